"""Oracle-side construction of verification workloads (test infrastructure only).

Builds host copies of a seeded model, the context KV of each request (a real
prefill through the oracle for the tiny model, or the synthetic pages of the
input generator), and the autoregressive draft fixture: for position j the draft
distribution is q_j = softmax(l_{j-1} / T_i + sigma_i * eps) built from the
oracle's own logits of row j-1, and y_j is drawn from q_j.
"""
from __future__ import annotations

import numpy as np
import torch

import wisp_inputs as wi

from . import OracleModel, forward


def host_model(shape: wi.ModelShape, seed: int = wi.MASTER_SEED) -> OracleModel:
    layers = [wi.layer_weights(shape, l, seed, "cpu") for l in range(shape.n_layers)]
    glob = wi.global_weights(shape, seed, "cpu")
    return OracleModel(shape, layers, glob)


def empty_pools(shape: wi.ModelShape, n_blocks: int):
    dt = np.float32 if shape.dtype == "f32" else np.uint16
    k = np.zeros((shape.n_layers, n_blocks, shape.n_kv_heads, wi.PAGE * shape.head_dim), dtype=dt)
    v = np.zeros((shape.n_layers, n_blocks, shape.n_kv_heads, wi.PAGE * shape.head_dim), dtype=dt)
    return k, v


def _to_storage(t: torch.Tensor, shape: wi.ModelShape) -> np.ndarray:
    if shape.dtype == "f32":
        return t.to(torch.float32).numpy()
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def place_synthetic_kv(mix: wi.Mix, pools, page_table, requests=None, layers=None, req_keys=None):
    """Write the input generator's synthetic context KV of the given requests into host pools
    (slot-major pages: token t of request i at block page_table[i][t // 16], slot t % 16).
    req_keys[i] (default i) is the request index that keys request i's generated values, so a
    request of a large batch can be reproduced on its own."""
    s = mix.shape
    hd = s.head_dim
    kp = pools[0].reshape(pools[0].shape[:3] + (wi.PAGE, hd))
    vp = pools[1].reshape(pools[1].shape[:3] + (wi.PAGE, hd))
    assert np.shares_memory(kp, pools[0]) and np.shares_memory(vp, pools[1]), "pools must be contiguous"
    dt = torch.float32 if s.dtype == "f32" else torch.bfloat16
    reqs = range(mix.B) if requests is None else requests
    lays = range(s.n_layers) if layers is None else layers
    for i in reqs:
        n = int(mix.ctx_len[i])
        if n == 0:
            continue
        key = i if req_keys is None else int(req_keys[i])
        t = np.arange(n)
        blk = page_table[i, t // wi.PAGE]
        slot = t % wi.PAGE
        for li, l in enumerate(lays):
            K, V = wi.kv_values(mix.seed, l, key, 0, n, s.n_kv_heads, hd, "cpu", dt)
            kp[li, blk, :, slot] = _to_storage(K, s)          # [n][n_kv][hd]
            vp[li, blk, :, slot] = _to_storage(V, s)


def prefill_context(model: OracleModel, mix: wi.Mix, pools, page_table, requests=None):
    """Real prefill of each request's random context tokens through the oracle."""
    reqs = list(range(mix.B)) if requests is None else list(requests)
    ctx = np.zeros(len(reqs), dtype=np.int32)
    n_new = np.array([mix.ctx_len[i] for i in reqs], dtype=np.int32)
    toks = np.concatenate([wi.context_tokens(mix, i) for i in reqs]).astype(np.int32)
    forward(model, pools[0], pools[1], page_table[reqs], ctx, n_new, toks)


def draft_fixture(model: OracleModel, mix: wi.Mix, pools, page_table, roots, requests=None):
    """Autoregressive drafts built from the oracle's own logits.

    Returns (tokens per request [root, y_1..y_gamma], q rows per request [gamma][V] fp32,
    logits per request [gamma][V] of rows 0..gamma-1).  Writes KV at the draft
    positions into the pools (the verification step overwrites them with the same rows)."""
    reqs = list(range(mix.B)) if requests is None else list(requests)
    V = mix.shape.vocab
    toks = {i: [int(roots[i])] for i in reqs}
    qs = {i: [] for i in reqs}
    lgs = {i: [] for i in reqs}
    gmax = max(int(mix.gamma[i]) for i in reqs) if reqs else 0
    for j in range(1, gmax + 1):
        act = [i for i in reqs if mix.gamma[i] >= j]
        ctx = np.array([mix.ctx_len[i] + j - 1 for i in act], dtype=np.int32)
        tk = np.array([toks[i][j - 1] for i in act], dtype=np.int32)
        lg = forward(model, pools[0], pools[1], page_table[act], ctx, np.ones(len(act), np.int32), tk)
        for a, i in enumerate(act):
            z = lg[a].astype(np.float64) / float(mix.t_draft[i]) + float(mix.sigma[i]) * wi.draft_noise(mix, i, j)
            e = np.exp(z - z.max())
            q = (e / e.sum()).astype(np.float32)
            c = np.cumsum(q.astype(np.float64))
            y = int(np.searchsorted(c, wi.draft_uniform(mix, i, j) * c[-1], side="right"))
            y = min(y, V - 1)
            toks[i].append(y)
            qs[i].append(q)
            lgs[i].append(lg[a])
    return ({i: np.array(toks[i], np.int32) for i in reqs},
            {i: (np.stack(qs[i]) if qs[i] else np.zeros((0, V), np.float32)) for i in reqs},
            {i: (np.stack(lgs[i]) if lgs[i] else np.zeros((0, V), np.float32)) for i in reqs})


def random_drafts(mix: wi.Mix, requests, roots, tag: int = 9):
    """Drafts that do not depend on the model (q = softmax of N(0, 1.3^2) noise, y ~ q),
    for requests whose outputs a test does not compare."""
    V = mix.shape.vocab
    toks, qs = {}, {}
    for i in requests:
        r = np.random.default_rng([mix.seed, tag, i])
        g = int(mix.gamma[i])
        z = r.standard_normal((g, V)) * 1.3
        e = np.exp(z - z.max(axis=1, keepdims=True))
        q = (e / e.sum(axis=1, keepdims=True)).astype(np.float32)
        ys = [int(r.choice(V, p=q[j].astype(np.float64) / q[j].astype(np.float64).sum())) for j in range(g)]
        toks[i] = np.array([int(roots[i])] + ys, np.int32)
        qs[i] = q
    return toks, qs
