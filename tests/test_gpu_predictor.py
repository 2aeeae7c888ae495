"""Draft-side rejection predictor on the GPU (Sec. 3.3, Sec. 4.1, App. B) against the
oracle: the four statistics of draft-logit rows (16-byte and scalar load paths, vocabularies
of 1 .. 128256 entries, padded row strides, repeated maxima, large logits, temperature)
and the MLP (4 and 5 inputs).

Tolerances: the kernel forms z and exp(z - m) in fp32 (about one ulp each) and sums in
fp64, so confidence and margin carry a relative error near 1e-7 and the entropy an absolute
one near 1e-6; the bound is 1e-5 (relative for confidence, margin and dispersion, absolute
for entropy).  The MLP sums at most 512 fp32 products of unit-size terms per output: the
bound on the probability is 1e-5 absolute."""
import numpy as np
import pytest
import torch

import paper_2601_11652_amd as W
from gpu_harness import log
from oracle.predictor import draft_stats, reject_mlp

pytestmark = pytest.mark.gpu


def _rows(rng, V, n, scale):
    return (rng.standard_normal((n, V)) * scale).astype(np.float32)


@pytest.mark.parametrize("V,ld,T", [(128256, 128256, 1.0), (1000, 1003, 0.7), (7, 8, 1.3), (1, 4, 1.0),
                                    (4099, 4100, 1.0)])
def test_draft_stats_match_the_oracle(V, ld, T):
    rng = np.random.default_rng(V)
    x = np.concatenate([_rows(rng, V, 5, s) for s in (0.3, 2.0, 9.0)])
    if V > 2:
        x[0, :] = 1.25                                   # flat row
        x[1, 3] = x[1, V - 1] = x[1].max() + 2.0         # repeated maximum
        x[2] *= 6.0                                      # logits up to ~60
    host = np.zeros((x.shape[0], ld), np.float32)
    host[:, :V] = x
    dev = torch.from_numpy(host).cuda()
    stats = torch.empty(x.shape[0], 4, dtype=torch.float32, device="cuda")
    W.wisp_draft_stats(dev, V, T, stats)
    torch.cuda.synchronize()
    got = stats.cpu().numpy().astype(np.float64)
    ref = draft_stats(x, T)
    rel = lambda a, b: np.abs(a - b) / np.maximum(np.abs(b), 1e-30)   # noqa: E731
    e_conf = rel(got[:, 0], ref[:, 0]).max()
    e_ent = np.abs(got[:, 1] - ref[:, 1]).max()
    e_mar = (np.abs(got[:, 2] - ref[:, 2]) / np.maximum(np.abs(ref[:, 2]), 1e-2)).max()
    e_std = (np.abs(got[:, 3] - ref[:, 3]) / np.maximum(ref[:, 3], 1e-6)).max()
    log(f"  V {V} ld {ld} T {T}: confidence {e_conf:.1e}, entropy {e_ent:.1e}, margin {e_mar:.1e}, std {e_std:.1e}")
    assert e_conf <= 1e-5 and e_ent <= 1e-5 and e_mar <= 1e-5 and e_std <= 1e-5
    if V > 2:
        assert got[1, 2] == 0.0                          # a repeated maximum has no margin


@pytest.mark.parametrize("n_in,rows", [(4, 1), (4, 33), (5, 257)])
def test_reject_mlp_matches_the_oracle(n_in, rows):
    rng = np.random.default_rng(100 + n_in)
    p = {"mean": rng.standard_normal(n_in), "inv_std": rng.uniform(0.5, 2, n_in),
         "w1": rng.standard_normal((512, n_in)) * 0.5, "b1": rng.standard_normal(512) * 0.1,
         "w2": rng.standard_normal((128, 512)) / 16, "b2": rng.standard_normal(128) * 0.1,
         "w3": rng.standard_normal((64, 128)) / 8, "b3": rng.standard_normal(64) * 0.1,
         "w4": rng.standard_normal(64) / 4, "b4": 0.3}
    p32 = {k: (np.float32(v) if k == "b4" else v.astype(np.float32)) for k, v in p.items()}
    f = rng.standard_normal((rows, n_in)).astype(np.float32)
    mlp = W.RejectMLP({k: (float(v) if k == "b4" else torch.from_numpy(v).cuda()) for k, v in p32.items()})
    out = torch.empty(rows, dtype=torch.float32, device="cuda")
    W.wisp_reject_predict(mlp, torch.from_numpy(f).cuda(), out)
    torch.cuda.synchronize()
    ref = reject_mlp({k: np.float64(v) if k == "b4" else v.astype(np.float64) for k, v in p32.items()}, f)
    err = np.abs(out.cpu().numpy() - ref).max()
    log(f"  MLP n_in {n_in}, {rows} rows: max |dp| {err:.1e} (p in [{ref.min():.3f}, {ref.max():.3f}])")
    assert err <= 1e-5
