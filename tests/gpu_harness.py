"""Shared set-up of the GPU parity tests: seeded inputs on both sides, the oracle run on
the host, the HIP path through the C ABI.  Inputs come from wisp_inputs or the oracle,
never from the HIP path."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2601_11652_amd as W
import wisp_inputs as wi
from oracle import fixtures as fx


def log(msg: str):
    print(msg, flush=True)


def to_dev(a: np.ndarray, dtype=None) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    t = torch.from_numpy(np.ascontiguousarray(a))
    return (t.to(dtype) if dtype is not None else t).cuda()


def to_host_storage(t: torch.Tensor) -> np.ndarray:
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def pools_to_dev(pools, hd: int):
    """Oracle pools (slot-major pages, [..., 16 * hd]) -> device pools in the library's page
    layout (the K and V page orders of the C ABI)."""
    k = wi.pages_from_slots(pools[0].reshape(pools[0].shape[:-1] + (wi.PAGE, hd)), "k")
    v = wi.pages_from_slots(pools[1].reshape(pools[1].shape[:-1] + (wi.PAGE, hd)), "v")
    return to_dev(k), to_dev(v)


def pools_from_dev(k: torch.Tensor, v: torch.Tensor, hd: int):
    """Device pools in the library's page layout -> host storage, slot-major pages."""
    out = []
    for t, which in ((k, "k"), (v, "v")):
        p = wi.slots_from_pages(to_host_storage(t), which, hd)
        out.append(np.ascontiguousarray(p.reshape(p.shape[:-2] + (wi.PAGE * hd,))))
    return out[0], out[1]


def written_mask(pool_shape, page_table, ctx_len, n_new, hd: int) -> np.ndarray:
    """Boolean mask over a slot-major pool [layers][blocks][n_kv][16 * hd]: the slots at
    positions ctx_len[i] .. ctx_len[i] + n_new[i] - 1 of every request."""
    m = np.zeros(pool_shape, bool)
    v = m.reshape(pool_shape[:3] + (wi.PAGE, hd))
    for i in range(len(ctx_len)):
        for pos in range(int(ctx_len[i]), int(ctx_len[i]) + int(n_new[i])):
            v[:, page_table[i, pos // wi.PAGE], :, pos % wi.PAGE, :] = True
    return m


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """One unit in the last place of bf16 at |x| (8 significant bits; the smallest normal's
    quantum below it)."""
    a = np.maximum(np.abs(np.asarray(x, np.float64)), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def kv_bound(ref: np.ndarray, hd: int) -> np.ndarray:
    """Two bf16 ulps at the scale of each K/V value, the scale being its head vector's
    largest magnitude (one token's K or V row of one kv head): one ulp for the rounding of
    the stored value itself (the two sides may round to either neighbour), one for the
    rounding flips of earlier values that reach its sum.  A sum's rounding error scales with
    its terms, not with its result, so a value near a cancelling zero carries the error of
    its vector's scale.  ref: slot-major pools [..., 16 * hd]."""
    v = np.abs(ref).reshape(ref.shape[:-1] + (wi.PAGE, hd))
    scale = v.max(axis=-1, keepdims=True) + 0.0 * v
    return 2.0 * bf16_ulp(scale).reshape(ref.shape)


def check_written(pools_gpu, pools_ref, pools_before, page_table, ctx_len, n_new, hd: int, bf16: bool,
                  f32_atol: float = 1e-4, pools_ref32=None):
    """K/V written at the new positions match the oracle's, every other slot is untouched
    bit for bit.  bf16: each value within max(two bf16 ulps at its scale (kv_bound), twice
    the layer's floor), the floor being max |oracle with fp32 sums - oracle with fp64 sums|
    over the layer's written K (or V) values (pools_ref32: the fp32-sum oracle's pools).
    Two correct accumulation orders round some values on different sides of a bf16 boundary,
    and each layer's flips move the next layer's sums.  fp32: within f32_atol."""
    worst = 0.0
    for w in range(2):
        g = storage_to_f64(pools_gpu[w])
        r = storage_to_f64(pools_ref[w])
        r32 = storage_to_f64(pools_ref32[w]) if pools_ref32 is not None else None
        before = storage_to_f64(pools_before[w])
        written = written_mask(g.shape, page_table, ctx_len, n_new, hd)
        ulp = kv_bound(r, hd) if bf16 else None
        for l in range(g.shape[0]):
            gl, rl = g[l][written[l]], r[l][written[l]]
            if gl.size == 0:
                continue
            if bf16:
                bound = ulp[l][written[l]]
                if r32 is not None:
                    bound = np.maximum(bound, 2.0 * np.abs(r32[l][written[l]] - rl).max())
            else:
                bound = np.full(rl.shape, f32_atol)
            ratio = float((np.abs(gl - rl) / bound).max())
            assert ratio <= 1.0, ("KV"[w], l, ratio, float(np.abs(gl - rl).max()))
            worst = max(worst, ratio)
        np.testing.assert_array_equal(g[~written], before[~written])
    return worst


def gpu_model(shape: wi.ModelShape, seed: int = wi.MASTER_SEED) -> W.GpuModel:
    glob = wi.global_weights(shape, seed, "cuda")
    return W.GpuModel(shape, lambda l: wi.layer_weights(shape, l, seed, "cuda"), glob)


def storage_to_f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


class Workload:
    """A verification batch prepared by the oracle: context KV, drafts, q, reference outputs."""

    def __init__(self, mix: wi.Mix, model: oracle.OracleModel, temperature: float = 1.0, requests=None):
        self.mix = mix
        self.T = temperature
        s = mix.shape
        self.pt, self.n_blocks = wi.page_table(mix)
        self.pools0 = fx.empty_pools(s, self.n_blocks)
        reqs = list(range(mix.B)) if requests is None else list(requests)
        if mix.kv_source == "prefill":
            fx.prefill_context(model, mix, self.pools0, self.pt, reqs)
        else:
            fx.place_synthetic_kv(mix, self.pools0, self.pt, reqs)
        self.roots = wi.root_tokens(mix)
        work = (self.pools0[0].copy(), self.pools0[1].copy())
        toks, qs, _ = fx.draft_fixture(model, mix, work, self.pt, self.roots, reqs)
        self.tokens = np.concatenate([toks[i] for i in range(mix.B)]).astype(np.int32)
        S = int(mix.gamma.sum())
        self.q = (np.concatenate([qs[i] for i in range(mix.B)]).astype(np.float32)
                  if S else np.zeros((0, s.vocab), np.float32))
        self.seed = wi.verify_seed(mix)
        # reference forward on the pre-step pools (bf16: also with fp32 sums, the floor)
        self.pools_ref = (self.pools0[0].copy(), self.pools0[1].copy())
        self.logits_ref = oracle.forward(model, self.pools_ref[0], self.pools_ref[1], self.pt, mix.ctx_len,
                                         mix.rows, self.tokens)
        self.pools_ref32 = None
        if s.dtype == "bf16":
            self.pools_ref32 = (self.pools0[0].copy(), self.pools0[1].copy())
            self.logits_ref32 = oracle.forward(model, self.pools_ref32[0], self.pools_ref32[1], self.pt,
                                               mix.ctx_len, mix.rows, self.tokens, acc32=True)


def run_gpu(gm: W.GpuModel, wl: Workload):
    """One wisp_verify call on the workload; returns numpy outputs and the pools after it
    (slot-major, as the oracle holds them)."""
    mix = wl.mix
    kv = W.KVPool(*pools_to_dev(wl.pools0, mix.shape.head_dim))
    pt = to_dev(wl.pt)
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, pt, wl.T, mix.req_id)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    tokens = to_dev(wl.tokens)
    q = to_dev(wl.q) if wl.q.shape[0] else torch.zeros(1, dtype=torch.float32, device="cuda")
    acc = torch.full((mix.B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((mix.M,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((mix.M, mix.shape.vocab), float("nan"), dtype=torch.float32, device="cuda")
    W.wisp_verify(gm.c, kv, desc, tokens, q, wl.seed, acc, out, logits, ws)
    W.wisp_check(ws)
    torch.cuda.synchronize()
    return (acc.cpu().numpy(), out.cpu().numpy(), logits.cpu().numpy(),
            pools_from_dev(kv.k, kv.v, mix.shape.head_dim))


def rel_row_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per row: max_k |got - ref| / max_k |ref|."""
    return np.abs(got - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)


def compare_decisions(acc_gpu, out_gpu, ref: oracle.AcceptResult, gamma, tokens, u_margin: float,
                      key_margin: float, residual_exempt: bool = False, logit_gap=0.0):
    """GPU decisions vs the oracle's on its own logits.  Returns (n_decisions, mismatches,
    unflagged) where a mismatch is unflagged if no draw of the oracle's path was within the
    margins (|u - a| < u_margin on an acceptance, or top-two race keys within key_margin).
    With residual_exempt, the extra token after a rejection is not compared (used when the
    two sides' logits differ by more than rounding).  logit_gap (scalar or per request) is
    the max-abs difference of the two sides' logits: p/q moves by at most a factor
    exp(2 * gap), which widens the acceptance margin by that relative amount, and the race
    margin by 4 * gap."""
    gaps = np.broadcast_to(np.asarray(logit_gap, dtype=np.float64), (len(gamma),))
    off = np.concatenate([[0], np.cumsum(gamma + 1)])
    doff = np.concatenate([[0], np.cumsum(gamma)])
    n_dec = 0
    mism = 0
    unflagged = []
    for i in range(len(gamma)):
        L = int(ref.accept_len[i])
        nd = min(L + 1, int(gamma[i]))
        n_dec += nd + 1
        o_ref = ref.out_tokens[off[i]:off[i + 1]]
        o_gpu = out_gpu[off[i]:off[i + 1]]
        if acc_gpu[i] == L and np.array_equal(o_ref, o_gpu):
            continue
        mism += 1
        u = ref.acc_u[doff[i]:doff[i] + nd]
        a = ref.acc_a[doff[i]:doff[i] + nd]
        widen = np.expm1(2.0 * gaps[i])
        flag = bool(np.any(np.abs(u - a) < u_margin + a * widen))
        k1, k2 = ref.race_key1[i], ref.race_key2[i]
        # race keys are score - ln(-ln u) with score a log-probability or scaled logit: a
        # logit gap moves each key by at most 2 * gap, the difference of two by 4 * gap
        if acc_gpu[i] == L and abs(k1 - k2) < key_margin * max(1.0, abs(k1)) + 4.0 * gaps[i]:
            flag = True
        if residual_exempt and acc_gpu[i] == L and L < gamma[i]:
            flag = True       # residual keys ln(p - q) are not Lipschitz in the logits
        if not flag:
            unflagged.append(i)
    # validity of every GPU output
    for i in range(len(gamma)):
        L = int(acc_gpu[i])
        assert 0 <= L <= gamma[i]
        o = out_gpu[off[i]:off[i + 1]]
        np.testing.assert_array_equal(o[:L], tokens[off[i] + 1:off[i] + 1 + L])
        assert o[L] >= 0 and np.all(o[L + 1:] == -1)
    return n_dec, mism, unflagged


def check_decisions_on_gpu_logits(acc_gpu, out_gpu, logits_gpu, tokens, q, gamma, temperature, seed,
                                  req_id=None):
    """The acceptance contract on identical logits: the oracle's acceptance run on the GPU's
    own logits must take the GPU's decisions.  A mismatch is allowed only on a flagged
    near-tie (|u - p/q| < 1e-3, or top-two race keys within 1e-5 relative) and such
    mismatches stay under 0.1 % of the decisions (at most one below 1000 decisions).
    Returns (decisions, mismatches)."""
    ref = oracle.accept(logits_gpu, tokens, q, gamma, temperature, seed, req_id=req_id)
    n_dec, mism, unflagged = compare_decisions(acc_gpu, out_gpu, ref, np.asarray(gamma), tokens, 1e-3, 1e-5)
    assert not unflagged, ("unflagged decision mismatches on identical logits", unflagged)
    assert mism <= max(1, int(1e-3 * n_dec)), (mism, n_dec)
    return n_dec, mism

