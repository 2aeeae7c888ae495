"""Seeded random verification batches on the GPU, each against the oracle.

Each case draws a batch the fixed cases do not spell out:
* B in 1..12 requests;
* gamma in 0..16, a quarter of them plain decodes;
* contexts from empty to 700 tokens, a mix of short, medium and long;
* a target temperature of 1, 0.6 or 0 (greedy), in turn.

It runs one wisp_verify call on the fp32 model or the bf16 GQA model and checks:
* the logits of every row: 1e-4 row-relative (fp32) or 2e-2 max-abs (bf16);
* every K and V row the step writes, and that no other slot changes;
* the decisions: on the GPU's own logits bit-exact except flagged near-ties (< 0.1 %);
  end to end (each side on its own logits) agreeing except where a draw lies within the
  margin the logit difference allows; the fp32 model's end-to-end mismatches stay under
  0.1 % of the decisions over all its cases.
"""
import numpy as np
import pytest

import oracle
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import Workload, check_decisions_on_gpu_logits, compare_decisions, gpu_model, log, run_gpu
from test_gpu_edge_cases import MINI_BF16, _bf16_abs, _check_written, _fp32_rows

pytestmark = pytest.mark.gpu

N_FP32, N_BF16 = 8, 6
_FP32_TALLY = [0, 0]      # end-to-end decisions and mismatches over the fp32 cases run so far


def _draw(k: int):
    r = np.random.default_rng(0xBA7C4 + k)
    B = int(r.integers(1, 13))
    gamma = r.integers(0, 17, size=B)
    gamma[r.random(B) < 0.25] = 0
    kind = r.random(B)
    ctx = np.where(kind < 0.3, r.integers(0, 21, size=B),
                   np.where(kind < 0.8, r.integers(21, 301, size=B), r.integers(301, 701, size=B)))
    T = (1.0, 0.6, 0.0)[k % 3]
    return ctx.astype(np.int32), gamma.astype(np.int32), T


@pytest.mark.parametrize("k", range(N_FP32 + N_BF16))
def test_random_batch_matches_oracle(k):
    shape, check = (wi.TINY, _fp32_rows) if k < N_FP32 else (MINI_BF16, _bf16_abs)
    ctx, gamma, T = _draw(k)
    mix = wi.custom_mix(shape, ctx, gamma, seed=1000 + k, name=f"random-{k}", kv_source="prefill",
                        t_draft=1.0, sigma=0.5)
    log(f"case {k}: {shape.name} T={T} ctx={ctx.tolist()} gamma={gamma.tolist()} (M = {mix.M})")
    wl = Workload(mix, fx.host_model(shape), temperature=T)
    acc, out, logits, pools = run_gpu(gpu_model(shape), wl)
    check(logits, wl.logits_ref)
    _check_written(wl, pools)
    ref = oracle.accept(wl.logits_ref, wl.tokens, wl.q, mix.gamma, T, wl.seed, req_id=mix.req_id)
    gap = float(np.abs(logits - wl.logits_ref).max())
    n_dec, mism, unflagged = compare_decisions(acc, out, ref, mix.gamma, wl.tokens, 1e-3, 1e-3,
                                               residual_exempt=shape.dtype == "bf16", logit_gap=gap)
    log(f"  decisions {n_dec}, mismatches {mism}, unflagged {unflagged}")
    assert not unflagged
    if shape.dtype == "f32":
        _FP32_TALLY[0] += n_dec
        _FP32_TALLY[1] += mism
        assert _FP32_TALLY[1] <= max(1, int(1e-3 * _FP32_TALLY[0])), _FP32_TALLY
    n_id, m_id = check_decisions_on_gpu_logits(acc, out, logits, wl.tokens, wl.q, mix.gamma, T, wl.seed,
                                               req_id=mix.req_id)
    log(f"  on the GPU's own logits: {n_id} decisions, {m_id} flagged mismatches")
