"""End-to-end GPU parity of wisp_verify against the oracle on small models.

* tiny workload (2 layers, d 256, 4 x 64 heads, SwiGLU 1024, vocab 1024, fp32, B = 4,
  contexts U[32, 128] prefilled by the oracle, gamma U{1..4}): logits within 1e-4
  relative per row (max |diff| / max |ref|), KV pages written in place match, untouched
  pages unchanged, decisions equal except at flagged near-ties;
* a small bf16 GQA model: logits within 2e-2 max-abs, same KV and decision checks.
"""
import numpy as np
import pytest

import oracle
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import Workload, check_written, compare_decisions, gpu_model, log, rel_row_err, run_gpu

pytestmark = pytest.mark.gpu

MINI_BF16 = wi.ModelShape("mini-bf16-gqa", 2, 256, 8, 2, 64, 512, 1024, "bf16", 10000.0)


def _check_pools(wl, pools_gpu):
    """New positions match the oracle's writes; every other slot is untouched."""
    mix = wl.mix
    check_written(pools_gpu, wl.pools_ref, wl.pools0, wl.pt, mix.ctx_len, mix.rows, mix.shape.head_dim,
                  mix.shape.dtype == "bf16", pools_ref32=wl.pools_ref32)


@pytest.mark.parametrize("T", [1.0, 0.0])
def test_tiny_verify_matches_oracle(T):
    mix = wi.make_mix("tiny")
    log(f"tiny verify T={T} ctx={mix.ctx_len.tolist()} gamma={mix.gamma.tolist()}")
    model = fx.host_model(mix.shape)
    wl = Workload(mix, model, temperature=T)
    gm = gpu_model(mix.shape)
    acc, out, logits, pools = run_gpu(gm, wl)
    err = rel_row_err(logits, wl.logits_ref)
    assert err.max() <= 1e-4, err.max()
    _check_pools(wl, pools)
    ref = oracle.accept(wl.logits_ref, wl.tokens, wl.q, mix.gamma, T, wl.seed, req_id=mix.req_id)
    n_dec, mism, unflagged = compare_decisions(acc, out, ref, mix.gamma, wl.tokens, 1e-3, 1e-3)
    assert not unflagged and mism == 0, (mism, unflagged)


def test_tiny_verify_is_idempotent():
    """Repeating a call on the same inputs gives bitwise identical outputs."""
    mix = wi.make_mix("tiny")
    model = fx.host_model(mix.shape)
    wl = Workload(mix, model)
    gm = gpu_model(mix.shape)
    a1 = run_gpu(gm, wl)
    a2 = run_gpu(gm, wl)
    for x, y in zip(a1[:3], a2[:3]):
        np.testing.assert_array_equal(x, y)


def test_mini_bf16_verify_matches_oracle():
    mix = wi.custom_mix(MINI_BF16, [37, 200, 16, 500, 3, 90], [4, 2, 16, 0, 7, 1], kv_source="prefill",
                        name="mini-bf16", t_draft=1.0, sigma=0.5)
    log(f"mini bf16 verify ctx={mix.ctx_len.tolist()} gamma={mix.gamma.tolist()}")
    model = fx.host_model(mix.shape)
    wl = Workload(mix, model)
    gm = gpu_model(mix.shape)
    acc, out, logits, pools = run_gpu(gm, wl)
    d = np.abs(logits - wl.logits_ref)
    log(f"  max-abs logits error {d.max():.3e}, mean {d.mean():.3e}")
    assert d.max() <= 2e-2
    _check_pools(wl, pools)
    ref = oracle.accept(wl.logits_ref, wl.tokens, wl.q, mix.gamma, 1.0, wl.seed, req_id=mix.req_id)
    # logits differ by up to 2e-2, so p/q may move by up to ~4 %: decisions are compared
    # where the oracle's draw is clear of that margin
    n_dec, mism, unflagged = compare_decisions(acc, out, ref, mix.gamma, wl.tokens, 0.05, 0.05, True)
    assert not unflagged, unflagged
