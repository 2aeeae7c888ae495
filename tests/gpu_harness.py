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
        # reference forward on the pre-step pools
        self.pools_ref = (self.pools0[0].copy(), self.pools0[1].copy())
        self.logits_ref = oracle.forward(model, self.pools_ref[0], self.pools_ref[1], self.pt, mix.ctx_len,
                                         mix.rows, self.tokens)


def run_gpu(gm: W.GpuModel, wl: Workload):
    """One wisp_verify call on the workload; returns numpy outputs and the pools after it."""
    mix = wl.mix
    kv = W.KVPool(to_dev(wl.pools0[0]), to_dev(wl.pools0[1]))
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
            (to_host_storage(kv.k), to_host_storage(kv.v)))


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
