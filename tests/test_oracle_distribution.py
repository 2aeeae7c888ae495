"""Distributional pins of the oracle's acceptance stage on a tiny vocabulary (V = 8).

Speculative sampling with the residual distribution is lossless (Leviathan et al.,
which the paper cites for its verification engine, Sec. 4.5): the emitted tokens
follow the target's autoregressive law.  10^6 seeded trials are checked with
chi-square tests (alpha = 1e-3), the acceptance-length law P(L >= k) = alpha^k
with alpha = sum_k min(p_k, q_k) is checked with z-tests, and a negative control
(the literal reading "extra token ~ p" even after a rejection) must be rejected.
"""
import numpy as np
import pytest
from scipy import stats

import oracle

V = 8
GAMMA = 4
N = 1_000_000
ALPHA_TEST = 1e-3

P = np.array([0.30, 0.05, 0.20, 0.02, 0.15, 0.08, 0.12, 0.08])
Q = np.array([0.05, 0.30, 0.10, 0.15, 0.05, 0.20, 0.05, 0.10])


def _sample(rng, probs, n):
    c = np.cumsum(probs)
    c = c / c[-1]
    return np.minimum(np.searchsorted(c, rng.random(n), side="right"), len(probs) - 1)


def _context_free_round(seed, n, rng):
    """n independent rounds with fixed p (logits = log p) and q; req_id = trial index."""
    lp = np.log(P).astype(np.float32)
    drafts = np.stack([_sample(rng, Q, n) for _ in range(GAMMA)], axis=1)
    toks = np.concatenate([np.zeros((n, 1), np.int64), drafts], axis=1).reshape(-1)
    logits = np.broadcast_to(lp, (n * (GAMMA + 1), V))
    q = np.broadcast_to(Q.astype(np.float32), (n * GAMMA, V))
    r = oracle.accept(logits, toks, q, np.full(n, GAMMA, np.int32), 1.0, seed)
    out = r.out_tokens.reshape(n, GAMMA + 1)
    return r, out, drafts


def _chi2_p(counts, expected):
    m = expected > 0
    return stats.chi2.sf((((counts - expected) ** 2)[m] / expected[m]).sum(), m.sum() - 1)


@pytest.fixture(scope="module")
def cf():
    rng = np.random.default_rng(2024)
    return _context_free_round(0xC0FFEE, N, rng)


def test_first_token_follows_p(cf):
    _, out, _ = cf
    p32 = oracle.row_probs(np.log(P).astype(np.float32), 1.0).astype(np.float64)
    counts = np.bincount(out[:, 0], minlength=V)
    assert _chi2_p(counts, N * p32) > ALPHA_TEST


def test_acceptance_length_law(cf):
    r, _, _ = cf
    a = np.minimum(P, Q).sum()
    L = r.accept_len
    for k in range(1, GAMMA + 1):
        pk = a ** k
        obs = (L >= k).sum()
        z = (obs - N * pk) / np.sqrt(N * pk * (1 - pk))
        assert abs(z) < 5.0, (k, obs / N, pk)
    assert abs(L.mean() - sum(a ** k for k in range(1, GAMMA + 1))) < 0.01


def test_bigrams_follow_p_product(cf):
    _, out, _ = cf
    r0, _, _ = cf
    # second emitted token: within the round when L >= 1, else from a second round
    o1 = out[:, 0]
    o2 = out[:, 1].copy()
    need = r0.accept_len == 0
    n2 = int(need.sum())
    rng = np.random.default_rng(7)
    _, out2, _ = _context_free_round(0xBEEF, n2, rng)
    o2[need] = out2[:, 0]
    p32 = oracle.row_probs(np.log(P).astype(np.float32), 1.0).astype(np.float64)
    counts = np.bincount(o1 * V + o2, minlength=V * V)
    assert _chi2_p(counts, N * np.outer(p32, p32).reshape(-1)) > ALPHA_TEST


def test_negative_control_literal_reading_fails(cf):
    # Reading Eq. (3) literally (extra token ~ p even after a rejection) is biased:
    # P(first = x) = min(p, q)(x) + (1 - alpha) p(x).  The test must detect it.
    r, out, _ = cf
    rng = np.random.default_rng(99)
    first = out[:, 0].copy()
    rej0 = r.accept_len == 0
    first[rej0] = _sample(rng, P, int(rej0.sum()))
    counts = np.bincount(first, minlength=V)
    assert _chi2_p(counts, N * P) < 1e-6


def test_markov_bigrams():
    """p(.|prev) and q(.|prev) depend on the previous token; drafts run autoregressively."""
    rng = np.random.default_rng(5)
    Pm = rng.dirichlet(np.ones(V) * 0.7, size=V)
    Qm = rng.dirichlet(np.ones(V) * 0.7, size=V)
    lPm = np.log(Pm).astype(np.float32)
    n = N

    def run(roots, seed):
        m = roots.shape[0]
        toks = np.zeros((m, GAMMA + 1), np.int64)
        toks[:, 0] = roots
        for j in range(1, GAMMA + 1):
            c = np.cumsum(Qm[toks[:, j - 1]], axis=1)
            toks[:, j] = np.minimum((c < rng.random((m, 1)) * c[:, -1:]).sum(1), V - 1)
        logits = lPm[toks].reshape(-1, V)
        q = Qm[toks[:, :GAMMA]].astype(np.float32).reshape(-1, V)
        r = oracle.accept(logits, toks.reshape(-1), q, np.full(m, GAMMA, np.int32), 1.0, seed)
        return r, r.out_tokens.reshape(m, GAMMA + 1)

    r1, out = run(np.zeros(n, np.int64), 31)
    o1 = out[:, 0]
    o2 = out[:, 1].copy()
    need = r1.accept_len == 0
    _, out2 = run(o1[need], 32)
    o2[need] = out2[:, 0]
    p_row = np.stack([oracle.row_probs(lPm[k], 1.0) for k in range(V)]).astype(np.float64)
    expected = n * (p_row[0][:, None] * p_row).reshape(-1)
    counts = np.bincount(o1 * V + o2, minlength=V * V)
    assert _chi2_p(counts, expected) > ALPHA_TEST
