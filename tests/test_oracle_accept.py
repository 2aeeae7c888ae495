"""Pins of the oracle's acceptance stage (Sec. 2.4, Eq. (1)-(3), residual at rejection).

Worked example (constructed from Eq. (1)): V = 4, p = [1/2, 1/4, 1/8, 1/8],
q = [1/4, 1/2, 1/8, 1/8].  Draft y = 1 has a = p/q = 1/2: u = 0.4 accepts, u = 0.6
rejects, and the residual max(0, p - q) = [1/4, 0, 0, 0] makes the extra token 0 for
every noise.  Draft y = 0 has a = min(1, 2) = 1 and is always accepted.
"""
import numpy as np
import pytest

import oracle

P4 = np.array([0.5, 0.25, 0.125, 0.125])
Q4 = np.array([0.25, 0.5, 0.125, 0.125])
L4 = np.log(P4).astype(np.float32)


def _one(gamma, rows, toks, qrows, u=None, T=1.0, seed=1, req=0):
    r = oracle.accept(np.stack(rows), np.array(toks), np.stack(qrows) if gamma else np.zeros((0, rows[0].shape[0])),
                      [gamma], T, seed, req_id=[req], u_inject=None if u is None else np.array(u))
    return r


def test_worked_example_single_draft():
    p = oracle.row_probs(L4, 1.0)
    np.testing.assert_allclose(p, P4, rtol=1e-6)
    q = Q4.astype(np.float32)
    r = _one(1, [L4, L4], [3, 1], [q], u=[0.4])
    assert r.accept_len[0] == 1 and r.out_tokens[0] == 1
    assert abs(r.acc_a[0] - 0.5) < 1e-6
    for seed in range(200):
        r = _one(1, [L4, L4], [3, 1], [q], u=[0.6], seed=seed)
        assert r.accept_len[0] == 0 and r.R[0] == 1
        assert r.out_tokens[0] == 0 and r.out_tokens[1] == -1
        assert r.degenerate[0] == 0


def test_worked_example_two_drafts():
    q = Q4.astype(np.float32)
    # y = (0, 1): first draft a = 1 always accepted; second accepted iff u2 <= 1/2
    r = _one(2, [L4, L4, L4], [2, 0, 1], [q, q], u=[0.999, 0.5])
    assert r.accept_len[0] == 2 and list(r.out_tokens[:2]) == [0, 1] and r.out_tokens[2] >= 0
    for seed in range(100):
        r = _one(2, [L4, L4, L4], [2, 0, 1], [q, q], u=[0.999, 0.51], seed=seed)
        assert r.accept_len[0] == 1 and list(r.out_tokens) == [0, 0, -1]


def _random_batch(B, V, gmax, seed, gamma_min=0):
    rng = np.random.default_rng(seed)
    gamma = rng.integers(gamma_min, gmax + 1, size=B).astype(np.int32)
    M = int((gamma + 1).sum())
    logits = (rng.standard_normal((M, V)) * 2).astype(np.float32)
    z = rng.standard_normal((int(gamma.sum()), V)) * 2
    q = np.exp(z - z.max(1, keepdims=True))
    q = (q / q.sum(1, keepdims=True)).astype(np.float32)
    toks = rng.integers(0, V, size=M).astype(np.int32)
    return gamma, logits, q, toks


def test_q_equals_p_accepts_everything():
    B, V = 300, 64
    gamma, logits, _, toks = _random_batch(B, V, 8, 5, gamma_min=1)
    off = np.concatenate([[0], np.cumsum(gamma + 1)])
    q = []
    for i in range(B):
        for j in range(1, gamma[i] + 1):
            q.append(oracle.row_probs(logits[off[i] + j - 1], 1.0))   # bitwise the oracle's p
    r = oracle.accept(logits, toks, np.stack(q), gamma, 1.0, 77)
    np.testing.assert_array_equal(r.accept_len, gamma)
    for i in range(B):
        o = r.out_tokens[off[i]:off[i + 1]]
        np.testing.assert_array_equal(o[:gamma[i]], toks[off[i] + 1:off[i + 1]])
        # bonus token = Gumbel race on the last row = a plain sample from p_gamma
        assert o[gamma[i]] == oracle.plain_decode(logits[off[i] + gamma[i]], 1.0, 77, i, int(gamma[i]))


@pytest.mark.parametrize("T", [1.0, 0.7, 0.0])
def test_gamma_zero_is_plain_decoding(T):
    B, V = 200, 128
    rng = np.random.default_rng(3)
    logits = (rng.standard_normal((B, V)) * 3).astype(np.float32)
    toks = rng.integers(0, V, size=B).astype(np.int32)
    r = oracle.accept(logits, toks, np.zeros((0, V), np.float32), np.zeros(B, np.int32), T, 1234)
    assert np.all(r.accept_len == 0)
    for i in range(B):
        want = oracle.plain_decode(logits[i], T, 1234, i, 0)
        assert r.out_tokens[i] == want
        if T == 0.0:
            assert want == int(np.argmax(logits[i]))


def test_greedy_accepts_iff_argmax():
    B, V = 200, 50
    gamma, logits, q, toks = _random_batch(B, V, 6, 11, gamma_min=1)
    off = np.concatenate([[0], np.cumsum(gamma + 1)])
    # make about half of the drafts equal to the argmax of the previous row
    rng = np.random.default_rng(12)
    for i in range(B):
        for j in range(1, gamma[i] + 1):
            if rng.random() < 0.7:
                toks[off[i] + j] = int(np.argmax(logits[off[i] + j - 1]))
    r = oracle.accept(logits, toks, q, gamma, 0.0, 5)
    for i in range(B):
        L = 0
        while L < gamma[i] and toks[off[i] + L + 1] == np.argmax(logits[off[i] + L]):
            L += 1
        assert r.accept_len[i] == L
        assert r.out_tokens[off[i] + L] == int(np.argmax(logits[off[i] + L]))


def test_invariants_random():
    B, V = 500, 200
    gamma, logits, q, toks = _random_batch(B, V, 16, 21)
    # mix in drafts that q likes, so both accept and reject paths occur
    r = oracle.accept(logits, toks, q, gamma, 1.0, 99)
    off = np.concatenate([[0], np.cumsum(gamma + 1)])
    assert np.all((r.accept_len >= 0) & (r.accept_len <= gamma))
    for i in range(B):
        L = r.accept_len[i]
        o = r.out_tokens[off[i]:off[i + 1]]
        np.testing.assert_array_equal(o[:L], toks[off[i] + 1:off[i] + 1 + L])
        assert 0 <= o[L] < V
        assert np.all(o[L + 1:] == -1)
        assert r.R[i] == L + 1


def test_zero_draft_probability_accepts():
    V = 16
    rng = np.random.default_rng(0)
    l = rng.standard_normal((2, V)).astype(np.float32)
    q = np.full((1, V), 1.0 / (V - 1), np.float32)
    q[0, 5] = 0.0
    for s in range(50):
        r = oracle.accept(l, np.array([0, 5]), q, [1], 1.0, s)
        assert r.accept_len[0] == 1 and r.acc_a[0] == 1.0


def test_degenerate_residual_samples_p():
    # q = 2p (unnormalised): every ratio is 1/2 and the residual max(0, p - q) is empty,
    # so a rejection falls back to a sample from p and is flagged.
    V = 32
    rng = np.random.default_rng(4)
    l = rng.standard_normal((2, V)).astype(np.float32)
    p = oracle.row_probs(l[0], 1.0)
    q = (2 * p)[None, :]
    for s in range(40):
        r = oracle.accept(l, np.array([1, 7]), q, [1], 1.0, s, u_inject=[0.9])
        assert r.accept_len[0] == 0 and r.degenerate[0] == 1
        assert r.out_tokens[0] == oracle.plain_decode(l[0], 1.0, s, 0, 0)


def test_request_keys_rng_stream():
    # identical inputs, different req_id -> independent draws; same req_id -> identical
    V = 64
    gamma, logits, q, toks = _random_batch(1, V, 4, 8, gamma_min=4)
    a = oracle.accept(logits, toks, q, gamma, 1.0, 1, req_id=[5])
    b = oracle.accept(logits, toks, q, gamma, 1.0, 1, req_id=[5])
    np.testing.assert_array_equal(a.out_tokens, b.out_tokens)
    outs = {tuple(oracle.accept(logits, toks, q, gamma, 1.0, 1, req_id=[k]).out_tokens) for k in range(40)}
    assert len(outs) > 3
