"""Pin of the oracle's paged causal attention against a dense fp64 brute force.

The brute force gathers each request's keys/values into dense arrays and computes
softmax(Q K^T / sqrt(hd) + causal mask) V with numpy; the oracle walks the page
table.  Cases: scattered (permuted) pages, context lengths not a multiple of the
16-token page, new rows straddling a page boundary, GQA groups G in {1, 4, 8}.
"""
import numpy as np
import pytest

import oracle
import wisp_inputs as wi

PAGE = 16


def _case(B, n_q, n_kv, hd, seed, bf16):
    rng = np.random.default_rng(seed)
    ctx = rng.integers(0, 70, size=B).astype(np.int32)
    ctx[0] = 15                        # rows straddle the first page boundary
    n_new = rng.integers(1, 6, size=B).astype(np.int32)
    need = (ctx + n_new + PAGE - 1) // PAGE
    n_blocks = int(need.sum()) + 2
    perm = rng.permutation(n_blocks).astype(np.int32)
    pt = np.full((B, int(need.max())), -1, np.int32)
    o = 0
    for i in range(B):
        pt[i, :need[i]] = perm[o:o + need[i]]
        o += need[i]
    kd = rng.standard_normal((n_blocks, n_kv, PAGE, hd))     # [block][kv][slot][dim]
    vd = rng.standard_normal((n_blocks, n_kv, PAGE, hd))
    if bf16:
        kd, vd = oracle.round_bf16(kd).reshape(kd.shape), oracle.round_bf16(vd).reshape(vd.shape)
        kp = (kd.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        vp = (vd.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    else:
        kd, vd = kd.astype(np.float32).astype(np.float64), vd.astype(np.float32).astype(np.float64)
        kp, vp = kd.astype(np.float32), vd.astype(np.float32)
    kp, vp = kp.reshape(n_blocks, n_kv, PAGE * hd), vp.reshape(n_blocks, n_kv, PAGE * hd)   # slot-major pages
    M = int(n_new.sum())
    q = rng.standard_normal((M, n_q, hd))
    return ctx, n_new, pt, kd, vd, kp, vp, q


def _brute(ctx, n_new, pt, kd, vd, q, n_kv):
    M, n_q, hd = q.shape
    G = n_q // n_kv
    out = np.zeros_like(q)
    r = 0
    for i in range(len(ctx)):
        T = ctx[i] + n_new[i]
        blk = pt[i, np.arange(T) // PAGE]
        slot = np.arange(T) % PAGE
        for j in range(n_new[i]):
            for h in range(n_q):
                K = kd[blk, h // G, slot, :]              # [T][hd]
                Vv = vd[blk, h // G, slot, :]             # [T][hd]
                s = K @ q[r, h] / np.sqrt(hd)
                s[ctx[i] + j + 1:] = -np.inf              # causal: keys <= own position
                w = np.exp(s - s.max())
                out[r, h] = (w / w.sum()) @ Vv
            r += 1
    return out


@pytest.mark.parametrize("n_q,n_kv,hd", [(4, 4, 64), (8, 2, 32), (16, 2, 64), (32, 8, 128)])
@pytest.mark.parametrize("bf16", [False, True])
def test_paged_attention_matches_brute_force(n_q, n_kv, hd, bf16):
    ctx, n_new, pt, kd, vd, kp, vp, q = _case(5, n_q, n_kv, hd, 17 + n_q + hd, bf16)
    got = oracle.paged_attention(q, kp, vp, pt, ctx, n_new, n_kv, bf16)
    want = _brute(ctx, n_new, pt, kd, vd, q, n_kv)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-12)


def test_empty_context_row_sees_only_itself():
    ctx, n_new, pt, kd, vd, kp, vp, q = _case(3, 4, 4, 64, 3, False)
    ctx[:] = 0
    n_new[:] = 1
    q = q[:3]
    got = oracle.paged_attention(q, kp, vp, pt, ctx, n_new, 4, False)
    for i in range(3):
        blk = pt[i, 0]
        for h in range(4):
            np.testing.assert_allclose(got[i, h], vd[blk, h, 0, :], rtol=1e-12)
