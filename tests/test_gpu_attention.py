"""GPU parity of the ragged paged causal attention (wisp_attention) against the oracle.

Cases cover scattered pages, contexts that are not a multiple of the 16-token page,
new rows straddling a page boundary, long contexts split into several KV chunks (up to 8
per group, combined in one round, and 12, combined in pipelined rounds), GQA groups G
in {1, 4, 8} and gamma up to 16 (more than 64 query rows per kv head).
bf16 tolerance: K, V, q are bf16 on both sides; the kernel rounds the softmax weights to
bf16 for the PV product and rounds the output to bf16, so |error| <= ~2^-8 * max|V|.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2601_11652_amd as W
import wisp_inputs as wi
from gpu_harness import log, to_dev

pytestmark = pytest.mark.gpu


def _case(ctx, gamma, n_q, n_kv, hd, bf16, seed):
    rng = np.random.default_rng(seed)
    B = len(ctx)
    ctx = np.asarray(ctx, np.int32)
    gamma = np.asarray(gamma, np.int32)
    need = (ctx + gamma + 1 + 15) // 16
    n_blocks = int(need.sum()) + 5
    perm = rng.permutation(n_blocks).astype(np.int32)
    pt = np.full((B, int(need.max()) + 1), -1, np.int32)
    o = 0
    for i in range(B):
        pt[i, :need[i]] = perm[o:o + need[i]]
        o += need[i]
    kd = rng.standard_normal((n_blocks, n_kv, 16, hd)).astype(np.float32)
    vd = rng.standard_normal((n_blocks, n_kv, 16, hd)).astype(np.float32)
    M = int((gamma + 1).sum())
    q = (rng.standard_normal((M, n_q, hd))).astype(np.float32)
    if bf16:
        r = lambda a: (a.view(np.uint32) + 0x7FFF + ((a.view(np.uint32) >> 16) & 1)) >> 16
        kp, vp, qs = [r(a).astype(np.uint16) for a in (kd, vd, q)]
    else:
        kp, vp, qs = kd, vd, q
    # the oracle reads slot-major pages, the library its own page order
    kn, vn = kp.reshape(n_blocks, n_kv, 16 * hd), vp.reshape(n_blocks, n_kv, 16 * hd)
    kp, vp = wi.pages_from_slots(kp, "k"), wi.pages_from_slots(vp, "v")
    return ctx, gamma, pt, kp, vp, qs, kn, vn


def _f64(a):
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


@pytest.mark.parametrize("ctx,gamma,n_q,n_kv,hd", [
    ([15, 40, 0, 129], [1, 4, 0, 3], 32, 8, 128),
    ([700, 33, 2500], [8, 16, 2], 32, 8, 128),
    ([1000, 17], [16, 5], 64, 8, 128),
    ([300, 64, 5], [3, 7, 1], 8, 8, 64),
    ([64, 900], [2, 9], 16, 2, 64),
    # a 12000-token context: even at the longest items (32 page pairs) each of its groups
    # has 12 chunks, so the combine takes its multi-round path; the short request's groups
    # (one chunk) take the one-round branch of the same launch
    ([12000, 900], [6, 3], 32, 8, 128),
])
@pytest.mark.parametrize("bf16", [True, False])
def test_attention_matches_oracle(ctx, gamma, n_q, n_kv, hd, bf16):
    log(f"attention ctx={ctx} gamma={gamma} nq={n_q} nkv={n_kv} hd={hd} bf16={bf16}")
    ctx, gamma, pt, kp, vp, q, kn, vn = _case(ctx, gamma, n_q, n_kv, hd, bf16, seed=sum(ctx) + n_q)
    shape = wi.ModelShape("attn", 1, 256, n_q, n_kv, hd, 256, 256, "bf16" if bf16 else "f32", 1e4)
    model = W.GpuModel.shape_only(shape)
    kv = W.KVPool(to_dev(kp[None]), to_dev(vp[None]))
    dpt = to_dev(pt)
    desc = W.BatchDesc(ctx, gamma, dpt, 1.0)
    ws = W.workspace(W.wisp_workspace_size(model, desc))
    dq = to_dev(q)
    out = torch.zeros_like(dq)
    W.wisp_attention(model, kv, desc, dq, out, ws)
    W.wisp_check(ws)
    got = _f64(out.cpu().view(torch.int16).numpy().view(np.uint16)) if bf16 else out.cpu().numpy().astype(np.float64)
    want = oracle.paged_attention(_f64(q), kn, vn, pt, ctx, gamma + 1, n_kv, bf16)
    err = np.abs(got - want)
    if bf16:
        assert err.max() < 2.5e-2, err.max()
        assert err.mean() < 3e-3, err.mean()
    else:
        assert err.max() < 1e-5, err.max()


def test_fp32_attention_at_its_longest_context():
    """The fp32 path keeps a request's scores in dynamic LDS (4 bytes per token): at the
    documented maximum of 32768 tokens per request that is 128 KB in one workgroup."""
    ctx, gamma = [32768 - 5], [4]
    log(f"fp32 attention at {ctx[0] + gamma[0] + 1} tokens")
    ctx, gamma, pt, kp, vp, q, kn, vn = _case(ctx, gamma, 4, 2, 32, False, seed=32768)
    shape = wi.ModelShape("attn", 1, 128, 4, 2, 32, 128, 256, "f32", 1e4)
    model = W.GpuModel.shape_only(shape)
    kv = W.KVPool(to_dev(kp[None]), to_dev(vp[None]))
    desc = W.BatchDesc(ctx, gamma, to_dev(pt), 1.0)
    ws = W.workspace(W.wisp_workspace_size(model, desc))
    dq = to_dev(q)
    out = torch.zeros_like(dq)
    W.wisp_attention(model, kv, desc, dq, out, ws)
    W.wisp_check(ws)
    want = oracle.paged_attention(q.astype(np.float64), kn, vn, pt, ctx, gamma + 1, 2, False)
    got = out.cpu().numpy().astype(np.float64)
    # each output sums 32768 fp32 products in order: relative bar of the fp32 path
    rel = np.abs(got - want).max() / np.abs(want).max()
    log(f"  max relative error {rel:.2e}")
    assert rel < 1e-4, rel
