"""First-time verification at full model width (Sec. 4.4's cold starts: hundreds of
uncached prompt tokens in front of the drafts), in one batch with follow-ups over long
cached contexts, against the oracle.

The model is the Llama-3-8B shape (d 4096, 32 / 8 heads, F 14336, vocabulary 128256, bf16)
cut to its first 2 layers, so that the oracle can recompute a cold start of a few hundred
rows on the host; every kernel runs at the 8B shape's widths.  The whole batch goes through
one wisp_verify call; the oracle reproduces each cold-start request alone, with fp64 sums
and again with fp32 sums (another correct accumulation order, whose distance from the fp64
result is the bf16 contract's own floor).  As in the full-size tests: logits within
max(2e-2, 2 * floor) max-abs and max(2e-3, 2 * mean floor) mean-abs; every K and V value
the request writes, prompt rows included, within max(two bf16 ulps at its head vector's
scale, 2 * the layer's floor); slots the request does not write stay bit-identical; decisions
bit-exact on the GPU's own logits (whole batch), and end to end agreeing except where the
observed logit gap could flip them.  Prompt, root and draft tokens are uniform random ids; q rows are
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
from gpu_harness import (check_decisions_on_gpu_logits, compare_decisions, gpu_model, kv_bound, log,
                         storage_to_f64, to_host_storage)

pytestmark = pytest.mark.gpu

SHAPE = wi.LLAMA3_8B.replace(n_layers=2, name="llama3-8b-shape-2L")
LOGIT_ATOL = 2e-2
LOGIT_MEAN = 2e-3
FLOOR_FACTOR = 2.0
# per request: cached context, prompt rows in front of the root, drafts
CTX = [0, 700, 0, 1500, 300, 0]
PRE = [128, 0, 256, 0, 0, 48]
GAM = [5, 4, 3, 7, 2, 0]
COLD = [0, 2, 5]


@pytest.mark.timeout(900)
def test_cold_starts_at_full_width():
    s = SHAPE
    ctx, pre, gam = (np.asarray(x, np.int32) for x in (CTX, PRE, GAM))
    B = len(CTX)
    rng = np.random.default_rng(zlib.crc32(b"prefill-full-width"))
    toks = [rng.integers(0, s.vocab, size=int(pre[i] + gam[i] + 1)).astype(np.int32) for i in range(B)]
    S = int(gam.sum())
    z = rng.standard_normal((S, s.vocab))
    q_np = np.exp(z - z.max(axis=1, keepdims=True))
    q_np = (q_np / q_np.sum(axis=1, keepdims=True)).astype(np.float32)
    qoff = np.concatenate([[0], np.cumsum(gam)])
    seed = 0x5EED1234
    log(f"full-width prefill: rows {int((pre + gam + 1).sum())} (verification rows {int((gam + 1).sum())}), "
        f"cold starts {COLD} with prompts {[int(pre[i]) for i in COLD]}")

    # --- oracle: each cold start alone, from nothing --------------------------------------
    model = fx.host_model(s)
    ref = {}
    for i in COLD:
        n_new = int(pre[i] + gam[i] + 1)
        n_pages = (n_new + wi.PAGE - 1) // wi.PAGE
        pt = np.arange(n_pages, dtype=np.int32)[None, :]
        after = fx.empty_pools(s, n_pages)
        lg = oracle.forward(model, after[0], after[1], pt, [0], [n_new], toks[i])
        after32 = fx.empty_pools(s, n_pages)
        lg32 = oracle.forward(model, after32[0], after32[1], pt, [0], [n_new], toks[i], acc32=True)
        ref[i] = dict(logits=lg[-(gam[i] + 1):], logits32=lg32[-(gam[i] + 1):], after=after, after32=after32)
        log(f"  oracle request {i}: {n_new} new rows")
    del model

    # --- the whole batch on the GPU ---------------------------------------------------------
    gm = gpu_model(s)
    layout = wi.custom_mix(s, ctx, pre + gam, name="prefill-full-width")
    pt_np, n_blocks = wi.page_table(layout)
    kv = W.KVPool.zeros(s.n_layers, n_blocks, s.n_kv_heads, s.head_dim, torch.bfloat16)
    wi.fill_kv_pool(kv.k, kv.v, wi.custom_mix(s, ctx, gam, name="prefill-full-width"), pt_np)
    before = (to_host_storage(kv.k), to_host_storage(kv.v))
    desc = W.BatchDesc(ctx, gam, torch.as_tensor(pt_np, device="cuda"), 1.0, np.arange(B, dtype=np.uint32),
                       prefill_len=pre)
    M = int((gam + 1).sum())
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    acc = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((M,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((M, s.vocab), float("nan"), dtype=torch.float32, device="cuda")
    W.wisp_verify(gm.c, kv, desc, torch.as_tensor(np.concatenate(toks), device="cuda"),
                  torch.from_numpy(q_np).cuda(), seed, acc, out, logits, ws)
    W.wisp_check(ws)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(logits).all())
    acc_np, out_np, lg_np = acc.cpu().numpy(), out.cpu().numpy(), logits.cpu().numpy()
    hd = s.head_dim
    slotted = lambda p, which: np.ascontiguousarray(   # library page order -> slot-major
        wi.slots_from_pages(p, which, hd).reshape(p.shape))
    got_pools = (slotted(to_host_storage(kv.k), "k"), slotted(to_host_storage(kv.v), "v"))
    before = (slotted(before[0], "k"), slotted(before[1], "v"))
    voff = np.concatenate([[0], np.cumsum(gam + 1)])
    vtok_all = np.concatenate([t[pre[i]:] for i, t in enumerate(toks)])
    n_id, m_id = check_decisions_on_gpu_logits(acc_np, out_np, lg_np, vtok_all, q_np, gam, 1.0, seed,
                                               req_id=np.arange(B, dtype=np.uint32))
    log(f"  whole batch on the GPU's own logits: {n_id} decisions, {m_id} flagged mismatches")

    # every request: an accepted prefix of its drafts, one valid extra token, -1 padding
    for i in range(B):
        L, o = int(acc_np[i]), out_np[voff[i]:voff[i + 1]]
        assert 0 <= L <= gam[i]
        np.testing.assert_array_equal(o[:L], toks[i][pre[i] + 1:pre[i] + 1 + L])
        assert 0 <= o[L] < s.vocab and np.all(o[L + 1:] == -1)

    for i, r in ref.items():
        lg = lg_np[voff[i]:voff[i + 1]]
        d = np.abs(lg - r["logits"])
        fl = np.abs(r["logits32"] - r["logits"])
        err = float(d.max())
        log(f"  request {i}: logits max-abs error {err:.3e} (floor {fl.max():.3e}), mean-abs {d.mean():.3e} "
            f"(floor {fl.mean():.3e})")
        assert err <= max(LOGIT_ATOL, FLOOR_FACTOR * fl.max()), (i, err, fl.max())
        assert d.mean() <= max(LOGIT_MEAN, FLOOR_FACTOR * fl.mean()), (i, d.mean(), fl.mean())
        n_new = int(pre[i] + gam[i] + 1)
        blocks = pt_np[i, :(n_new + wi.PAGE - 1) // wi.PAGE]
        for w in range(2):
            got = storage_to_f64(got_pools[w][:, blocks])
            pre_w = storage_to_f64(before[w][:, blocks])
            exp, exp32 = storage_to_f64(r["after"][w]), storage_to_f64(r["after32"][w])
            written = np.zeros(got.shape[1:], bool)
            wv = written.reshape(written.shape[:2] + (wi.PAGE, hd))
            for pos in range(n_new):
                wv[pos // wi.PAGE, :, pos % wi.PAGE, :] = True
            ulp = kv_bound(exp, hd)
            for l in range(s.n_layers):
                dk = np.abs(got[l][written] - exp[l][written])
                f_l = np.abs(exp32[l][written] - exp[l][written]).max()
                bad = dk > np.maximum(ulp[l][written], FLOOR_FACTOR * f_l)
                assert not bad.any(), (i, "KV"[w], l, float(dk.max()), f_l)
            np.testing.assert_array_equal(got[:, ~written], pre_w[:, ~written])
        vt = toks[i][pre[i]:]
        res = oracle.accept(r["logits"], vt, q_np[qoff[i]:qoff[i + 1]], gam[i:i + 1], 1.0, seed,
                            req_id=np.array([i], np.uint32))
        n_dec, mism, unflagged = compare_decisions(acc_np[i:i + 1], out_np[voff[i]:voff[i + 1]], res, gam[i:i + 1],
                                                   vt, 1e-3, 1e-3, residual_exempt=True, logit_gap=err)
        log(f"  request {i}: oracle L={int(res.accept_len[0])} gpu L={int(acc_np[i])}, mismatches {mism}")
        assert not unflagged, (i, unflagged)
