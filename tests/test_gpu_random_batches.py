"""Seeded random verification batches on the GPU, each against the oracle.

Each case draws a batch the fixed cases do not spell out:
* B in 1..12 requests;
* gamma in 0..16, a quarter of them plain decodes;
* contexts from empty to 700 tokens, a mix of short, medium and long;
* a target temperature of 1, 0.6 or 0 (greedy), in turn.

It runs one wisp_verify call on the fp32 model or the bf16 GQA model and checks:
* the logits of every row: 1e-4 row-relative (fp32) or 2e-2 max-abs (bf16);
* every K and V row the step writes, and that no other slot changes;
* the decisions: they agree except where a draw lies within the margin the logit
  difference allows.
"""
import numpy as np
import pytest

import oracle
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import Workload, compare_decisions, gpu_model, log, run_gpu
from test_gpu_edge_cases import MINI_BF16, _bf16_abs, _check_written, _fp32_rows

pytestmark = pytest.mark.gpu

N_FP32, N_BF16 = 8, 6


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
    shape, check, kv_atol = (wi.TINY, _fp32_rows, 1e-4) if k < N_FP32 else (MINI_BF16, _bf16_abs, 6e-2)
    ctx, gamma, T = _draw(k)
    mix = wi.custom_mix(shape, ctx, gamma, seed=1000 + k, name=f"random-{k}", kv_source="prefill",
                        t_draft=1.0, sigma=0.5)
    log(f"case {k}: {shape.name} T={T} ctx={ctx.tolist()} gamma={gamma.tolist()} (M = {mix.M})")
    wl = Workload(mix, fx.host_model(shape), temperature=T)
    acc, out, logits, pools = run_gpu(gpu_model(shape), wl)
    check(logits, wl.logits_ref)
    _check_written(wl, pools, kv_atol)
    ref = oracle.accept(wl.logits_ref, wl.tokens, wl.q, mix.gamma, T, wl.seed, req_id=mix.req_id)
    gap = float(np.abs(logits - wl.logits_ref).max())
    n_dec, mism, unflagged = compare_decisions(acc, out, ref, mix.gamma, wl.tokens, 1e-3, 1e-3,
                                               residual_exempt=shape.dtype == "bf16", logit_gap=gap)
    log(f"  decisions {n_dec}, mismatches {mism}, unflagged {unflagged}")
    assert not unflagged
