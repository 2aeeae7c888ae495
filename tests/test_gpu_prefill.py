"""First-time (cold-start) verification and chunked prefill on the GPU, against the oracle
(Sec. 4.4's two verification types: hundreds of uncached prompt tokens in front of the
drafts, next to follow-up requests with a cached history).

Each batch mixes cold starts (ctx_len = 0, prefill_len > 0), follow-ups (prefill_len = 0),
continuations of a chunked prompt (ctx_len > 0 and prefill_len > 0) and prompt chunks with
no drafts (gamma = 0).  The oracle forwards every new row (prompt, root, drafts) through its
plain model on the same pools; the GPU's logits must match the oracle's on the verification
rows (fp32: 1e-4 relative per row; bf16: 2e-2 max-abs), every new K/V slot must match and
every other slot stay bit-identical, and the acceptance decisions must agree except on
flagged near-ties.  Prompt, root and draft tokens are uniform random ids; q rows are
softmax of standard-normal noise.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2601_11652_amd as W
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import (check_decisions_on_gpu_logits, check_written, compare_decisions, gpu_model, log,
                         pools_from_dev, pools_to_dev, rel_row_err, to_dev)

pytestmark = pytest.mark.gpu

MINI_BF16 = wi.ModelShape("mini-bf16-gqa", 2, 256, 8, 2, 64, 512, 1024, "bf16", 10000.0)


def _case(shape, ctx, pre, gam, name, T=1.0):
    ctx = np.asarray(ctx, np.int32)
    pre = np.asarray(pre, np.int32)
    gam = np.asarray(gam, np.int32)
    B = ctx.shape[0]
    mix = wi.custom_mix(shape, ctx, gam, kv_source="prefill", name=name)
    # page tables sized for every new row (prompt, root, drafts)
    layout = wi.custom_mix(shape, ctx, pre + gam, name=name)
    pt, nb = wi.page_table(layout)
    model = fx.host_model(shape)
    pools0 = fx.empty_pools(shape, nb)
    fx.prefill_context(model, mix, pools0, pt)

    rng = np.random.default_rng(zlib.crc32(name.encode()))
    toks = [rng.integers(0, shape.vocab, size=int(pre[i] + gam[i] + 1)).astype(np.int32) for i in range(B)]
    tokens = np.concatenate(toks)
    vtokens = np.concatenate([t[pre[i]:] for i, t in enumerate(toks)])
    S = int(gam.sum())
    z = rng.standard_normal((S, shape.vocab))
    q = (np.exp(z - z.max(axis=1, keepdims=True)))
    q = (q / q.sum(axis=1, keepdims=True)).astype(np.float32)
    seed = 0x5EED0000 + B

    pools_ref = (pools0[0].copy(), pools0[1].copy())
    n_new = (pre + gam + 1).astype(np.int32)
    logits_all = oracle.forward(model, pools_ref[0], pools_ref[1], pt, ctx, n_new, tokens)
    pools_ref32 = None
    if shape.dtype == "bf16":      # the fp32-sum oracle: the floor of the K/V check
        pools_ref32 = (pools0[0].copy(), pools0[1].copy())
        oracle.forward(model, pools_ref32[0], pools_ref32[1], pt, ctx, n_new, tokens, acc32=True)
    ends = np.cumsum(n_new)
    logits_ref = np.concatenate([logits_all[ends[i] - gam[i] - 1:ends[i]] for i in range(B)])
    return dict(mix=mix, ctx=ctx, pre=pre, gam=gam, pt=pt, pools0=pools0, pools_ref=pools_ref,
                pools_ref32=pools_ref32, tokens=tokens,
                vtokens=vtokens, q=q, seed=seed, logits_ref=logits_ref, T=T)


def _run(shape, c):
    gm = gpu_model(shape)
    B = c["ctx"].shape[0]
    M = int((c["gam"] + 1).sum())
    kv = W.KVPool(*pools_to_dev(c["pools0"], shape.head_dim))
    desc = W.BatchDesc(c["ctx"], c["gam"], to_dev(c["pt"]), c["T"], np.arange(B, dtype=np.uint32),
                       prefill_len=c["pre"])
    assert desc.M == M and desc.rows == c["tokens"].shape[0]
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    q = to_dev(c["q"]) if c["q"].shape[0] else torch.zeros(1, dtype=torch.float32, device="cuda")
    acc = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((M,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((M, shape.vocab), float("nan"), dtype=torch.float32, device="cuda")
    W.wisp_verify(gm.c, kv, desc, to_dev(c["tokens"]), q, c["seed"], acc, out, logits, ws)
    W.wisp_check(ws)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), out.cpu().numpy(), logits.cpu().numpy(), pools_from_dev(kv.k, kv.v, shape.head_dim)


def _check_kv(shape, c, pools):
    worst = check_written(pools, c["pools_ref"], c["pools0"], c["pt"], c["ctx"], c["pre"] + c["gam"] + 1,
                          shape.head_dim, shape.dtype == "bf16", pools_ref32=c["pools_ref32"])
    log(f"  new K/V slots: worst error / bound {worst:.2f}")


def _verify_case(shape, ctx, pre, gam, name, logit_check):
    c = _case(shape, ctx, pre, gam, name)
    log(f"{shape.name}: ctx={list(c['ctx'])} prefill={list(c['pre'])} gamma={list(c['gam'])} "
        f"(rows {c['tokens'].shape[0]}, verification rows {int((c['gam'] + 1).sum())})")
    acc, out, logits, pools = _run(shape, c)
    logit_check(logits, c["logits_ref"])
    _check_kv(shape, c, pools)
    ref = oracle.accept(c["logits_ref"], c["vtokens"], c["q"], c["gam"], c["T"], c["seed"],
                        req_id=np.arange(c["ctx"].shape[0], dtype=np.uint32))
    gap = float(np.abs(logits - c["logits_ref"]).max())
    n_dec, mism, unflagged = compare_decisions(acc, out, ref, c["gam"], c["vtokens"], 1e-3, 1e-3,
                                               residual_exempt=shape.dtype == "bf16", logit_gap=gap)
    log(f"  decisions {n_dec}, mismatches {mism}, unflagged {unflagged}")
    assert not unflagged
    n_id, m_id = check_decisions_on_gpu_logits(acc, out, logits, c["vtokens"], c["q"], c["gam"], c["T"], c["seed"],
                                               req_id=np.arange(c["ctx"].shape[0], dtype=np.uint32))
    log(f"  on the GPU's own logits: {n_id} decisions, {m_id} flagged mismatches")


def _fp32_rows(logits, ref):
    err = rel_row_err(logits, ref)
    log(f"  max relative row error {err.max():.2e}")
    assert err.max() <= 1e-4


def _bf16_abs(logits, ref):
    d = np.abs(logits - ref).max()
    log(f"  max-abs logits error {d:.3e}")
    assert d <= 2e-2


def test_cold_start_and_chunked_prefill_fp32():
    # cold starts (0, 3), follow-ups (1, 4), a chunk continuing a cached prompt (2), gamma = 0 (2)
    _verify_case(wi.TINY, [0, 30, 17, 0, 50], [40, 0, 21, 15, 0], [3, 2, 0, 4, 1], "prefill-f32",
                 _fp32_rows)


def test_cold_start_and_chunked_prefill_bf16():
    # request 0: a 300-token prompt (306 rows x 4 query heads per kv head = 26 row groups)
    _verify_case(MINI_BF16, [0, 64, 33, 0], [300, 0, 47, 9], [5, 3, 2, 0], "prefill-bf16",
                 _bf16_abs)


def test_prompt_split_over_two_calls_matches_one_call():
    """Chunked prefill: the prompt's first part in one call (as a gamma = 0 request whose
    root is the part's last token), the rest plus the drafts in a second call over the
    first call's KV, gives the one-call logits (fp32, 1e-4 relative per row)."""
    shape = wi.TINY
    P, gamma, split = 70, 3, 33
    c = _case(shape, [0], [P], [gamma], "prefill-split")
    gm = gpu_model(shape)
    kv = W.KVPool(*pools_to_dev(c["pools0"], shape.head_dim))
    pt = to_dev(c["pt"])

    def call(ctx, pre, gam, toks, q):
        desc = W.BatchDesc([ctx], [gam], pt, 1.0, np.zeros(1, np.uint32), prefill_len=[pre])
        ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
        M = gam + 1
        acc = torch.empty(1, dtype=torch.int32, device="cuda")
        out = torch.empty(M, dtype=torch.int32, device="cuda")
        logits = torch.empty(M, shape.vocab, dtype=torch.float32, device="cuda")
        qd = to_dev(q) if q.shape[0] else torch.zeros(1, dtype=torch.float32, device="cuda")
        W.wisp_verify(gm.c, kv, desc, to_dev(toks), qd, 5, acc, out, logits, ws)
        W.wisp_check(ws)
        torch.cuda.synchronize()
        return logits.cpu().numpy()

    toks = c["tokens"]
    call(0, split - 1, 0, toks[:split], np.zeros((0, shape.vocab), np.float32))
    second = call(split, P - split, gamma, toks[split:], c["q"])
    err = rel_row_err(second, c["logits_ref"])
    log(f"two calls vs the oracle's one forward: max relative row error {err.max():.2e}")
    assert err.max() <= 1e-4
