"""First-time verification at full model width (Sec. 4.4's cold starts: hundreds of
uncached prompt tokens in front of the drafts), in one batch with follow-ups over long
cached contexts, against the oracle.

The model is the Llama-3-8B shape (d 4096, 32 / 8 heads, F 14336, vocabulary 128256, bf16)
cut to its first 2 layers, so that the oracle can recompute a cold start of a few hundred
rows on the host; every kernel runs at the 8B shape's widths.  The whole batch goes through
one wisp_verify call; the oracle reproduces each cold-start request alone.  As in the
full-size tests, each quantity (the verification rows' logits, every K and V row the
request writes, prompt rows included) is checked against max(bound, 2 * floor), floor being
the oracle's own change under a one-ulp move of the first prompt token's embedding (for
K/V also one bf16 ulp of the value itself: one rounding flip); slots
the request does not write stay bit-identical; decisions agree except where the observed
logit gap could flip them.  Prompt, root and draft tokens are uniform random ids; q rows are
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
from gpu_harness import compare_decisions, gpu_model, log, storage_to_f64, to_host_storage

pytestmark = pytest.mark.gpu

SHAPE = wi.LLAMA3_8B.replace(n_layers=2, name="llama3-8b-shape-2L")
LOGIT_ATOL = 2e-2
KV_ATOL = 6e-2
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
        pert = fx.empty_pools(s, n_pages)
        with fx.perturbed_embedding(model, toks[i][0]):
            lg_p = oracle.forward(model, pert[0], pert[1], pt, [0], [n_new], toks[i])
        ref[i] = dict(logits=lg[-(gam[i] + 1):], logits_p=lg_p[-(gam[i] + 1):], after=after, after_p=pert)
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
    got_pools = (to_host_storage(kv.k), to_host_storage(kv.v))
    voff = np.concatenate([[0], np.cumsum(gam + 1)])

    # every request: an accepted prefix of its drafts, one valid extra token, -1 padding
    for i in range(B):
        L, o = int(acc_np[i]), out_np[voff[i]:voff[i + 1]]
        assert 0 <= L <= gam[i]
        np.testing.assert_array_equal(o[:L], toks[i][pre[i] + 1:pre[i] + 1 + L])
        assert 0 <= o[L] < s.vocab and np.all(o[L + 1:] == -1)

    kidx, vidx = wi.k_page_index(s.head_dim), wi.v_page_index(s.head_dim)
    for i, r in ref.items():
        lg = lg_np[voff[i]:voff[i + 1]]
        err = float(np.abs(lg - r["logits"]).max())
        floor = float(np.abs(r["logits_p"] - r["logits"]).max())
        log(f"  request {i}: logits max-abs error {err:.3e}, oracle 1-ulp floor {floor:.3e}")
        assert err <= max(LOGIT_ATOL, 2.0 * floor), (i, err, floor)
        n_new = int(pre[i] + gam[i] + 1)
        blocks = pt_np[i, :(n_new + wi.PAGE - 1) // wi.PAGE]
        for w, idx in enumerate((kidx, vidx)):
            got = storage_to_f64(got_pools[w][:, blocks])
            pre_w = storage_to_f64(before[w][:, blocks])
            exp, expp = storage_to_f64(r["after"][w]), storage_to_f64(r["after_p"][w])
            written = np.zeros(got.shape[1:], bool)
            for pos in range(n_new):
                written[pos // wi.PAGE, :, idx[pos % wi.PAGE]] = True
            for l in range(s.n_layers):
                d = np.abs(got[l][written] - exp[l][written])
                f_l = np.abs(expp[l][written] - exp[l][written]).max()
                # one rounding flip of a stored bf16 value costs one ulp of that value
                ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(exp[l][written]), 1e-30))) - 7)
                bad = d > np.maximum(max(KV_ATOL, 2.0 * f_l), ulp)
                assert not bad.any(), (i, "KV"[w], l, float(d.max()), f_l)
            np.testing.assert_array_equal(got[:, ~written], pre_w[:, ~written])
        vt = toks[i][pre[i]:]
        res = oracle.accept(r["logits"], vt, q_np[qoff[i]:qoff[i + 1]], gam[i:i + 1], 1.0, seed,
                            req_id=np.array([i], np.uint32))
        n_dec, mism, unflagged = compare_decisions(acc_np[i:i + 1], out_np[voff[i]:voff[i + 1]], res, gam[i:i + 1],
                                                   vt, 1e-3, 1e-3, residual_exempt=True, logit_gap=err)
        log(f"  request {i}: oracle L={int(res.accept_len[0])} gpu L={int(acc_np[i])}, mismatches {mism}")
        assert not unflagged, (i, unflagged)
