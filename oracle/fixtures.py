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
    """Write the input generator's synthetic context KV of the given requests into host pools.
    req_keys[i] (default i) is the request index that keys request i's generated values, so a
    request of a large batch can be reproduced on its own."""
    s = mix.shape
    kp, vp = pools
    dt = torch.float32 if s.dtype == "f32" else torch.bfloat16
    reqs = range(mix.B) if requests is None else requests
    lays = range(s.n_layers) if layers is None else layers
    hd = s.head_dim
    kidx = wi.k_page_index(hd)
    vidx = wi.v_page_index(hd)
    for i in reqs:
        n = int(mix.ctx_len[i])
        if n == 0:
            continue
        key = i if req_keys is None else int(req_keys[i])
        nf = n // wi.PAGE                     # full pages
        full = page_table[i, :nf]
        for li, l in enumerate(lays):
            K, V = wi.kv_values(mix.seed, l, key, 0, n, s.n_kv_heads, hd, "cpu", dt)
            Kn = _to_storage(K, s)
            Vn = _to_storage(V, s)
            if nf:
                # whole pages by axis permutation (the layout's index tables, split into axes):
                # K (slot s = 8a + 4b + c, dim e = 32f + 8g + h) sits at [f][b][g][a][c][h],
                # V (slot s = 8a + c, dim e = 16f + h) sits at [f][a][h][c]
                k = Kn[:nf * wi.PAGE].reshape(nf, 2, 2, 4, s.n_kv_heads, hd // 32, 4, 8)
                kp[li, full] = k.transpose(0, 4, 5, 2, 6, 1, 3, 7).reshape(nf, s.n_kv_heads, -1)
                v = Vn[:nf * wi.PAGE].reshape(nf, 2, 8, s.n_kv_heads, hd // 16, 16)
                vp[li, full] = v.transpose(0, 3, 4, 1, 5, 2).reshape(nf, s.n_kv_heads, -1)
            if n > nf * wi.PAGE:
                blk = page_table[i, nf]
                sl = np.arange(n - nf * wi.PAGE)
                kp[li, blk][:, kidx[sl]] = Kn[nf * wi.PAGE:].transpose(1, 0, 2)
                vp[li, blk][:, vidx[sl]] = Vn[nf * wi.PAGE:].transpose(1, 0, 2)


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


class perturbed_embedding:
    """Context manager: moves embedding entries (token, col) of a host model by one unit in
    the last place of their storage format, and restores them on exit.  Used to measure how
    far the model's own rounding noise carries a minimal input change."""

    def __init__(self, model: OracleModel, token: int, cols=(17, 2011)):
        self.e = model.embed
        self.token = int(token)
        self.cols = [c % self.e.shape[1] for c in cols]
        self.saved = None

    def __enter__(self):
        self.saved = self.e[self.token, self.cols].copy()
        if self.e.dtype == np.uint16:
            self.e[self.token, self.cols] = self.saved + 1          # next bf16 bit pattern
        else:
            self.e[self.token, self.cols] = np.nextafter(self.saved, np.float32(np.inf))
        return self

    def __exit__(self, *exc):
        self.e[self.token, self.cols] = self.saved
        return False


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
