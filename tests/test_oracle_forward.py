"""Pins of the oracle's forward pass (Sec. 4.5 batched one-step verification).

* incremental consistency: one call over rows [t_0..t_g] equals g+1 successive
  single-row calls (pins causal masking and the in-place KV append);
* batch invariance and page-permutation invariance;
* RoPE at position 0 is the identity and q_m . k_n depends only on m - n;
  RMSNorm is invariant to scaling its input;
* a dense reformulation built from torch library routines in fp64
  (F.rms_norm, F.linear, complex-rotation RoPE, F.scaled_dot_product_attention,
  F.silu) reproduces the oracle's logits, fp32 and bf16 modes.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import wisp_inputs as wi
from oracle import fixtures as fx

MINI_BF16 = wi.ModelShape("mini-bf16-gqa", 2, 128, 4, 2, 32, 256, 512, "bf16", 10000.0)
MINI_F32 = wi.ModelShape("mini-f32-gqa", 2, 128, 4, 2, 32, 192, 300, "f32", 10000.0)


@pytest.fixture(scope="module", params=["tiny", "mini_bf16", "mini_f32"])
def setup(request):
    shape = {"tiny": wi.TINY, "mini_bf16": MINI_BF16, "mini_f32": MINI_F32}[request.param]
    mix = wi.custom_mix(shape, [37, 16, 0, 50], [4, 2, 3, 0], kv_source="prefill", name=request.param)
    model = fx.host_model(shape)
    pt, nb = wi.page_table(mix)
    pools = fx.empty_pools(shape, nb)
    fx.prefill_context(model, mix, pools, pt)
    rng = np.random.default_rng(1)
    toks = rng.integers(0, shape.vocab, size=mix.M).astype(np.int32)
    return shape, mix, model, pt, pools, toks


def _fwd(model, pools, pt, ctx, n_new, toks):
    k, v = pools[0].copy(), pools[1].copy()
    return oracle.forward(model, k, v, pt, ctx, n_new, toks), (k, v)


def test_incremental_consistency(setup):
    shape, mix, model, pt, pools, toks = setup
    full, _ = _fwd(model, pools, pt, mix.ctx_len, mix.rows, toks)
    k, v = pools[0].copy(), pools[1].copy()
    off = np.concatenate([[0], np.cumsum(mix.rows)])
    for i in range(mix.B):
        for j in range(mix.rows[i]):
            lg = oracle.forward(model, k, v, pt[i:i + 1], [mix.ctx_len[i] + j], [1], toks[off[i] + j:off[i] + j + 1])
            np.testing.assert_allclose(lg[0], full[off[i] + j], rtol=1e-6, atol=1e-6)


def test_batch_and_page_permutation_invariance(setup):
    shape, mix, model, pt, pools, toks = setup
    full, _ = _fwd(model, pools, pt, mix.ctx_len, mix.rows, toks)
    off = np.concatenate([[0], np.cumsum(mix.rows)])
    i = 1
    alone, _ = _fwd(model, pools, pt[i:i + 1], mix.ctx_len[i:i + 1], mix.rows[i:i + 1], toks[off[i]:off[i + 1]])
    np.testing.assert_array_equal(alone, full[off[i]:off[i + 1]])
    # move every block to a new id
    nb = pools[0].shape[1]
    perm = np.random.default_rng(3).permutation(nb)
    k2 = np.empty_like(pools[0])
    v2 = np.empty_like(pools[1])
    k2[:, perm] = pools[0]
    v2[:, perm] = pools[1]
    pt2 = np.where(pt >= 0, perm[np.maximum(pt, 0)], -1).astype(np.int32)
    moved = oracle.forward(model, k2, v2, pt2, mix.ctx_len, mix.rows, toks)
    np.testing.assert_array_equal(moved, full)


def test_rope_identities():
    rng = np.random.default_rng(0)
    hd, base = 64, 10000.0
    q, k = rng.standard_normal(hd), rng.standard_normal(hd)
    np.testing.assert_array_equal(oracle.rope_apply(q, 0, base), q)
    for m, n, s in [(5, 2, 7), (100, 3, 1000), (31, 31, 12345)]:
        a = oracle.rope_apply(q, m, base) @ oracle.rope_apply(k, n, base)
        b = oracle.rope_apply(q, m + s, base) @ oracle.rope_apply(k, n + s, base)
        assert abs(a - b) < 1e-9 * (1 + abs(a))
        assert abs(np.linalg.norm(oracle.rope_apply(q, m, base)) - np.linalg.norm(q)) < 1e-12
    # rotate-half pairing: dimension i pairs with i + hd/2, angle pos * base^(-2i/hd)
    e = np.zeros(hd)
    e[3] = 1.0
    r = oracle.rope_apply(e, 2, base)
    ang = 2 * base ** (-6.0 / hd)
    np.testing.assert_allclose([r[3], r[3 + hd // 2]], [np.cos(ang), np.sin(ang)], atol=1e-15)


def test_rmsnorm_scale_invariance():
    rng = np.random.default_rng(2)
    h = rng.standard_normal((4, 256))
    a = oracle.rmsnorm_apply(h, 1e-12)
    b = oracle.rmsnorm_apply(h * 37.5, 1e-12)
    np.testing.assert_allclose(a, b, rtol=1e-12)
    np.testing.assert_allclose((a ** 2).mean(1), 1.0, rtol=1e-10)


# ------------------------------------------------------------------------------------
# dense reformulation through torch library routines (fp64)
# ------------------------------------------------------------------------------------
def _t(x):
    return torch.as_tensor(x).to(torch.float64)


def _round(x, bf16):
    return x.to(torch.bfloat16).to(torch.float64) if bf16 else x


def _store(x, bf16):
    return x.to(torch.bfloat16).to(torch.float64) if bf16 else x.to(torch.float32).to(torch.float64)


def _rope_complex(x, pos, base):
    # x [..., hd]: (x_i, x_{i+hd/2}) as one complex number rotated by pos * base^(-2i/hd)
    hd = x.shape[-1]
    inv = base ** (-torch.arange(0, hd // 2, dtype=torch.float64) * 2.0 / hd)
    ang = pos[:, None].to(torch.float64) * inv[None, :]
    z = torch.complex(x[..., : hd // 2], x[..., hd // 2:]) * torch.polar(torch.ones_like(ang), ang)[:, None, :]
    return torch.cat([z.real, z.imag], dim=-1)


def _dense_forward(shape, layers, glob, pools, pt, ctx, n_new, toks):
    bf16 = shape.dtype == "bf16"
    G = shape.group
    hd = shape.head_dim
    kp = torch.from_numpy(pools[0].astype(np.int32) << 16).view(torch.float32) if bf16 else torch.from_numpy(pools[0])
    vp = torch.from_numpy(pools[1].astype(np.int32) << 16).view(torch.float32) if bf16 else torch.from_numpy(pools[1])
    # slot-major pages -> [layer][block][kv][slot][dim]
    kp = kp.to(torch.float64).reshape(kp.shape[:3] + (16, hd))
    vp = vp.to(torch.float64).reshape(vp.shape[:3] + (16, hd))
    out = []
    off = 0
    for i in range(len(ctx)):
        n = int(n_new[i])
        c = int(ctx[i])
        tk = torch.as_tensor(toks[off:off + n], dtype=torch.long)
        off += n
        pos = torch.arange(c, c + n)
        h = _t(glob["embed"])[tk]
        tpos = torch.arange(c)
        blk = torch.as_tensor(pt[i])[tpos // 16]
        for l in range(shape.n_layers):
            w = {k: _t(v) for k, v in layers[l].items()}
            x = _round(F.rms_norm(h, (shape.d_model,), w["attn_norm"], shape.rms_eps), bf16)
            q = F.linear(x, w["wq"]).view(n, shape.n_q_heads, hd)
            k = F.linear(x, w["wk"]).view(n, shape.n_kv_heads, hd)
            v = F.linear(x, w["wv"]).view(n, shape.n_kv_heads, hd)
            q = _round(_rope_complex(q, pos, shape.rope_base), bf16)
            k = _store(_rope_complex(k, pos, shape.rope_base), bf16)
            v = _store(v, bf16)
            kc = kp[l][blk, :, tpos % 16, :]                       # [c][n_kv][hd]
            vc = vp[l][blk, :, tpos % 16, :]                       # [c][n_kv][hd]
            K = torch.cat([kc, k], 0).repeat_interleave(G, dim=1).transpose(0, 1)   # [n_q][T][hd]
            Vv = torch.cat([vc, v], 0).repeat_interleave(G, dim=1).transpose(0, 1)
            T = c + n
            mask = torch.arange(T)[None, :] <= pos[:, None]
            o = F.scaled_dot_product_attention(q.transpose(0, 1), K, Vv, attn_mask=mask)
            o = _round(o.transpose(0, 1).reshape(n, -1), bf16)
            h = h + F.linear(o, w["wo"])
            x2 = _round(F.rms_norm(h, (shape.d_model,), w["mlp_norm"], shape.rms_eps), bf16)
            a = _round(F.silu(F.linear(x2, w["w_gate"])) * F.linear(x2, w["w_up"]), bf16)
            h = h + F.linear(a, w["w_down"])
        x = _round(F.rms_norm(h, (shape.d_model,), _t(glob["final_norm"]), shape.rms_eps), bf16)
        out.append(F.linear(x, _t(glob["lm_head"])))
    return torch.cat(out).numpy()


def test_dense_library_reformulation(setup):
    shape, mix, model, pt, pools, toks = setup
    got, _ = _fwd(model, pools, pt, mix.ctx_len, mix.rows, toks)
    layers = [wi.layer_weights(shape, l) for l in range(shape.n_layers)]
    glob = wi.global_weights(shape)
    want = _dense_forward(shape, layers, glob, pools, pt, mix.ctx_len, mix.rows, toks)
    if shape.dtype == "f32":
        np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)
    else:
        # torch rounds fp64 -> bf16 through fp32, the oracle rounds directly: rare 1-ulp
        # differences at rounding points are the only expected deviations
        err = np.abs(got - want).max()
        assert err < 2e-2, err
        assert np.mean(np.abs(got - want) < 1e-5) > 0.5


# ------------------------------------------------------------------------------------
# the fp32-accumulation mode (a second correct rounding order)
# ------------------------------------------------------------------------------------
def test_fp32_sums_stay_within_the_textbook_bound():
    """A projection with fp32 sums in natural order: |fl(sum) - sum| <= gamma_n * sum |x_k w_k|
    with gamma_n = n u / (1 - n u), u = 2^-24 (the standard bound for recursive summation
    of exact products: the products of bf16-valued operands are exact in fp32).  The fp64
    mode agrees with numpy's fp64 matmul."""
    rng = np.random.default_rng(3)
    n = 4096
    W_ = oracle.round_bf16(rng.standard_normal((64, n)) * 0.02).astype(np.float32)
    x = oracle.round_bf16(rng.standard_normal((5, n)))
    y64 = oracle.linear_apply(W_, x)
    y32 = oracle.linear_apply(W_, x, acc32=True)
    np.testing.assert_allclose(y64, x @ W_.astype(np.float64).T, rtol=1e-12, atol=1e-12)
    u = 2.0 ** -24
    gam = n * u / (1 - n * u)
    bound = gam * (np.abs(x) @ np.abs(W_.astype(np.float64)).T)
    assert np.all(np.abs(y32 - y64) <= bound)
    assert np.any(y32 != y64)                          # the sums really are fp32
    assert np.all(y32 == y32.astype(np.float32))       # and the results fp32 values


@pytest.mark.parametrize("shape", [wi.TINY, MINI_BF16], ids=["fp32", "bf16"])
def test_fp32_accumulation_mode_stays_near_the_fp64_forward(shape):
    """fp32 model: the fp32-summed forward is within 1e-5 relative per row of the fp64 one.
    bf16 model: within the bf16 logits bound, and not identical (the rounding points see
    different sums, which is what the mode is for)."""
    mix = wi.custom_mix(shape, [37, 16, 0, 50], [4, 2, 3, 0], kv_source="prefill", name="acc32")
    model = fx.host_model(shape)
    pt, nb = wi.page_table(mix)
    pools = fx.empty_pools(shape, nb)
    fx.prefill_context(model, mix, pools, pt)
    toks = np.random.default_rng(2).integers(0, shape.vocab, size=mix.M).astype(np.int32)
    a = oracle.forward(model, pools[0].copy(), pools[1].copy(), pt, mix.ctx_len, mix.rows, toks)
    b = oracle.forward(model, pools[0].copy(), pools[1].copy(), pt, mix.ctx_len, mix.rows, toks, acc32=True)
    if shape.dtype == "f32":
        rel = np.abs(a - b).max(axis=1) / np.abs(a).max(axis=1)
        assert rel.max() <= 1e-5, rel.max()
    else:
        d = np.abs(a - b)
        assert d.max() <= 2e-2 and d.max() > 0, d.max()
