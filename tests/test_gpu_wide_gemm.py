"""The wide-output projections at the stated bf16 bound.

The 8B / 70B shapes have gate/up and LM-head outputs of at least 16384 columns, which the
small test models never had.  This model makes both wide at a width the oracle recomputes
in seconds: d_model 512, 8 query heads on 2 kv heads of 64, d_ff 8192 (gate/up 16384
columns), vocabulary 65536 (wide enough for the LM head's own plan), bf16, 2 layers.

Cases: 14 rows (gate/up on 64 x 128 tiles in one K range with the SwiGLU epilogue, the LM
head on 32 x 256 tiles with the row-maxima epilogue, the narrower projections on the
weight ring), 44 rows (the LM head on the 64-column weight ring, the rest on 64 x 128
tiles), 153 rows (the LM head on the 64-column weight ring, the rest on 192-row tiles,
gate/up in one K range with SwiGLU in its epilogue), 476 and 680 rows (every projection on
256 x 256 tiles, gate/up with two K ranges at 476 rows and with SwiGLU in its epilogue at
680, the narrow ones with K split).  Checks: logits within 2e-2 max-abs of the oracle, every written K/V value within
max(two bf16 ulps at its head vector's scale, twice the oracle's floor of its layer),
untouched slots bit-identical, decisions on the GPU's own logits bit-exact except flagged
near-ties.
"""
import numpy as np
import pytest

import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import Workload, check_decisions_on_gpu_logits, check_written, gpu_model, log, run_gpu

pytestmark = pytest.mark.gpu

WIDE_BF16 = wi.ModelShape("wide-bf16", 2, 512, 8, 2, 64, 8192, 65536, "bf16", 10000.0)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("B", [3, 8, 9, 28, 40], ids=["14rows", "44rows", "153rows", "476rows", "680rows"])
def test_wide_projections_match_the_oracle(B):
    r = np.random.default_rng(8192 + B)
    ctx = r.integers(0, 64, size=B).astype(np.int32)
    # 3 requests of 11 drafts: 14 rows; 8 requests of 36 drafts in all: 44 rows; otherwise
    # B requests of 16 drafts: 17 B rows
    gamma = np.array({3: [6, 1, 4], 8: [7, 1, 5, 3, 6, 4, 2, 8]}.get(B, [16] * B), np.int32)
    mix = wi.custom_mix(WIDE_BF16, ctx, gamma, kv_source="prefill", name=f"wide-{B}", t_draft=1.0,
                        sigma=0.5)
    log(f"{WIDE_BF16.name}: B={B} M={mix.M} ctx={ctx.tolist()} gamma={gamma.tolist()}")
    wl = Workload(mix, fx.host_model(WIDE_BF16))
    acc, out, logits, pools = run_gpu(gpu_model(WIDE_BF16), wl)
    d = np.abs(logits - wl.logits_ref)
    log(f"  logits max-abs error {d.max():.3e}, mean {d.mean():.3e} (|ref| max {np.abs(wl.logits_ref).max():.2f})")
    assert d.max() <= 2e-2
    worst = check_written(pools, wl.pools_ref, wl.pools0, wl.pt, mix.ctx_len, mix.rows, WIDE_BF16.head_dim, True,
                          pools_ref32=wl.pools_ref32)
    log(f"  written K/V: worst error / bound {worst:.2f}")
    n_id, m_id = check_decisions_on_gpu_logits(acc, out, logits, wl.tokens, wl.q, mix.gamma, 1.0, wl.seed,
                                               req_id=mix.req_id)
    log(f"  on the GPU's own logits: {n_id} decisions, {m_id} flagged mismatches")
