"""Oracle of the draft-side rejection predictor -- test infrastructure.

Sec. 3.3 observes that a drafted token's acceptance tracks summary statistics of the draft
model's next-token distribution, and Sec. 4.1 / App. B feed four of them to a small MLP
(hidden widths 512, 128, 64, ReLU, sigmoid output trained with binary cross-entropy).
Written out from their definitions, in float64, for one row of logits with z = logits / T
and p = softmax(z):
  confidence  max_k p_k
  entropy     -sum_k p_k ln p_k                  (nats; terms with p_k = 0 contribute 0)
  margin      p_(1) - p_(2), the two largest probabilities (as a multiset)
  dispersion  population standard deviation of z
Readings: the paper's text names these four features while App. B's dataset table lists
five dimensions; the fifth is left to the caller (the draft position, say).  "Standard
deviation" is taken of the scaled logits z (with T = 1, of the logits).
Only tests may import this module.
"""
from __future__ import annotations

import numpy as np


def draft_stats(logits, temperature: float = 1.0) -> np.ndarray:
    """[rows][4] float64 statistics of fp32 logits rows (z is formed in float32, as the
    logits are stored, then widened)."""
    z = (np.asarray(logits, np.float32) / np.float32(temperature)).astype(np.float64)
    out = np.empty((z.shape[0], 4))
    for r in range(z.shape[0]):
        zr = z[r]
        w = np.exp(zr - zr.max())
        p = w / w.sum()
        nz = p > 0
        top = np.sort(p)[::-1]
        out[r, 0] = top[0]
        out[r, 1] = -np.sum(p[nz] * np.log(p[nz]))
        out[r, 2] = top[0] - (top[1] if zr.shape[0] > 1 else 0.0)
        out[r, 3] = np.sqrt(np.mean((zr - zr.mean()) ** 2))
    return out


def reject_mlp(params: dict, features) -> np.ndarray:
    """Probability of acceptance per feature row: standardise, three ReLU layers, sigmoid."""
    f = {k: np.asarray(v, np.float64) for k, v in params.items()}
    x = (np.asarray(features, np.float64) - f["mean"]) * f["inv_std"]
    h = np.maximum(x @ f["w1"].T + f["b1"], 0.0)
    h = np.maximum(h @ f["w2"].T + f["b2"], 0.0)
    h = np.maximum(h @ f["w3"].T + f["b3"], 0.0)
    return 1.0 / (1.0 + np.exp(-(h @ f["w4"] + f["b4"])))
