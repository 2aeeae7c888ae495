"""Speculative sampling is lossless through the whole GPU path (Sec. 2.4: accept with
min(1, p/q), stop at the first rejection, then draw from norm(max(0, p - q)); Leviathan et
al., cited in Sec. 4.5).  Whatever the drafter's distribution q, the first token a request
emits follows the target's p.

The batch is 4096 independent requests on the fp32 model.  They share one cached 16-token
context page (each writes its own page for the new rows), have the same root, and draw
gamma = 3 drafts from a fixed q unrelated to p.  Over 25 calls with distinct seeds, that
is 102 400 first tokens.  The oracle forwards the context and root from nothing to get p.

Checks:
* a chi-square test of the first tokens against p passes;
* the same counts against q_1 fail, so the test can tell the two apart;
* the fraction that accept y_1 matches sum_y min(p, q_1).
"""
import numpy as np
import pytest
import torch
from scipy import stats

import oracle
import paper_2601_11652_amd as W
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import gpu_model, log, pools_to_dev, to_dev

pytestmark = pytest.mark.gpu

B, GAMMA, CALLS, CTX = 4096, 3, 25, 16


def _chi2_pvalue(counts: np.ndarray, probs: np.ndarray) -> float:
    n = counts.sum()
    exp = n * probs
    big = exp >= 5.0                       # small bins pooled into one
    obs = np.append(counts[big], counts[~big].sum())
    e = np.append(exp[big], exp[~big].sum())
    keep = e > 0
    chi2 = float(((obs[keep] - e[keep]) ** 2 / e[keep]).sum())
    return float(stats.chi2.sf(chi2, int(keep.sum()) - 1))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("T", [1.0, 0.7])
def test_first_emitted_token_follows_the_target(T):
    s = wi.TINY
    V = s.vocab
    rng = np.random.default_rng(2601 + int(10 * T))
    ctx_toks = rng.integers(0, V, CTX).astype(np.int32)
    root = int(rng.integers(0, V))

    # the oracle forwards context + root from nothing: p of the root row, and page 0's KV
    model = fx.host_model(s)
    k0, v0 = fx.empty_pools(s, 2)
    lg = oracle.forward(model, k0, v0, np.array([[0, 1]], np.int32), [0], [CTX + 1], np.append(ctx_toks, root))
    p = oracle.row_probs(lg[CTX], T).astype(np.float64)
    p /= p.sum()
    z = rng.standard_normal((GAMMA, V))
    q = np.exp(z - z.max(axis=1, keepdims=True))
    q = (q / q.sum(axis=1, keepdims=True)).astype(np.float32)
    q64 = q.astype(np.float64) / q.astype(np.float64).sum(axis=1, keepdims=True)
    cdf = np.cumsum(q64, axis=1)

    gm = gpu_model(s)
    kp, vp = fx.empty_pools(s, 1 + B)
    kp[:, 0], vp[:, 0] = k0[:, 0], v0[:, 0]
    kv = W.KVPool(*pools_to_dev((kp, vp), s.head_dim))
    pt = np.stack([np.zeros(B, np.int32), 1 + np.arange(B, dtype=np.int32)], axis=1)
    desc = W.BatchDesc(np.full(B, CTX, np.int32), np.full(B, GAMMA, np.int32), to_dev(pt), T,
                       np.arange(B, dtype=np.uint32))
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    dq = to_dev(np.tile(q, (B, 1)))
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    out = torch.empty(B * (GAMMA + 1), dtype=torch.int32, device="cuda")
    logits = torch.empty((B * (GAMMA + 1), V), dtype=torch.float32, device="cuda")

    counts = np.zeros(V, np.int64)
    accepted_first = 0
    for c in range(CALLS):
        drafts = np.stack([np.minimum(np.searchsorted(cdf[j], rng.random(B), side="right"), V - 1)
                           for j in range(GAMMA)], axis=1)
        toks = np.concatenate([np.full((B, 1), root), drafts], axis=1).reshape(-1).astype(np.int32)
        W.wisp_verify(gm.c, kv, desc, to_dev(toks), dq, 0xC0FFEE + 7919 * c, acc, out, logits, ws)
        W.wisp_check(ws)
        first = out.cpu().numpy().reshape(B, GAMMA + 1)[:, 0]
        counts += np.bincount(first, minlength=V)
        accepted_first += int((acc.cpu().numpy() >= 1).sum())
    n = CALLS * B
    pv_p, pv_q = _chi2_pvalue(counts, p), _chi2_pvalue(counts, q64[0])
    a = float(np.minimum(p, q64[0]).sum())
    rate = accepted_first / n
    sd = np.sqrt(a * (1 - a) / n)
    log(f"T={T}: {n} first tokens; chi-square p-value vs p {pv_p:.3g}, vs q_1 {pv_q:.3g}; "
        f"y_1 accepted {rate:.4f} (expected {a:.4f} +- {sd:.4f})")
    assert pv_p > 1e-3
    assert pv_q < 1e-6
    assert abs(rate - a) < 5 * sd
