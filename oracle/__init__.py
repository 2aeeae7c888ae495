"""CPU oracle of the batched speculative-verification step (WISP, arXiv 2601.11652).

TEST INFRASTRUCTURE ONLY.  The test suite, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` are the only code allowed to import it; the product
library (``paper_2601_11652_amd``) never does, and the two share no code.

The arithmetic lives in plain C (``wisp_oracle.c``, fp64 forward / fp32 acceptance)
and is reached through ctypes.  The forward also has an fp32-accumulation mode
(``acc32``: every sum in fp32, natural index order, and in bf16 models the attention
weights rounded to bf16 before they weight the values, as a bf16 matrix-core product
takes them), a second correct rounding order whose distance from the fp64 result
measures the bf16 contract's own noise floor.
KV pools are natural ``[n_layers][n_blocks][n_kv][16][head_dim]`` arrays (slot-major
pages); the GPU library's page order is a separate interface layout, converted at the
test boundary.  What each function follows in the paper:

* ``forward``          -- Sec. 4.5, batched one-step verification over a paged,
                          prefix-cached KV (new rows written in place).
* ``paged_attention``  -- the attention inside that forward (causal, per request).
* ``accept``           -- Sec. 2.4, Eq. (1) acceptance, Eq. (2) stopping position,
                          Eq. (3) extra token, with the residual norm(max(0, p - q))
                          at a rejection (Leviathan et al., cited for losslessness).
* ``plain_decode``     -- ordinary sampling of one token from p (the gamma = 0 case).
* ``philox4x32_10`` / ``uniform`` -- the counter-based generator (Salmon et al., SC'11)
                          that keys every random draw of the method.

Pins (tests/test_oracle_*.py): a hand-worked acceptance example, closed forms
(q = p accepts everything, gamma = 0 is plain decoding, T = 0 is greedy), chi-square
tests of the output law on V = 8, the acceptance-length law P(L >= k) = alpha^k,
a negative control (the literal "extra token ~ p" reading must fail), an fp64 dense
brute-force attention, Philox known-answer vectors, forward invariants, and a dense
fp64 reformulation of the forward from torch library routines (rms_norm, linear,
complex-rotation RoPE, scaled_dot_product_attention, silu), compared logit by logit.
The weights are random-init, so no external reference logits exist to match.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wisp_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libwisp_oracle.so")
_lib = None

TAG_ACCEPT = 1
TAG_RACE = 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (ISO C11: no fast-math, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        _lib = C.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


_P = C.c_void_p


def _declare(L):
    L.orc_philox4x32_10.argtypes = [_P, _P, _P]
    L.orc_uniform.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32]
    L.orc_uniform.restype = C.c_float
    L.orc_uniform_array.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32, _P]
    L.orc_accept_batch.argtypes = [C.c_int, C.c_int, _P, _P, _P, _P, _P, C.c_float, C.c_uint64,
                                   _P, _P, _P, _P, _P, _P, _P, _P, _P]
    L.orc_plain_decode.argtypes = [C.c_int, _P, C.c_float, C.c_uint64, C.c_uint32, C.c_uint32]
    L.orc_plain_decode.restype = C.c_int32
    L.orc_paged_attention.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, _P, _P, _P,
                                      C.c_int, C.c_int, _P, _P, _P, _P]
    L.orc_forward.argtypes = [_P, _P, _P, C.c_int, C.c_int, _P, _P, _P, C.c_int, _P, _P]
    L.orc_round_bf16_array.argtypes = [_P, _P, C.c_int64]
    L.orc_row_probs.argtypes = [_P, C.c_int, C.c_float, _P]
    L.orc_rope_apply.argtypes = [_P, C.c_int, C.c_int, C.c_double]
    L.orc_linear_apply.argtypes = [_P, _P, _P, C.c_int, C.c_int, C.c_int, C.c_int]
    L.orc_rmsnorm_apply.argtypes = [_P, _P, C.c_int, C.c_int, C.c_double, C.c_int]


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


# ------------------------------------------------------------------------------------
# RNG
# ------------------------------------------------------------------------------------
def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    o = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(o))
    return o


def uniform(seed: int, req_id: int, tag: int, row: int, idx: int) -> float:
    return float(lib().orc_uniform(seed, req_id, tag, row, idx))


def uniform_array(seed: int, req_id: int, tag: int, row: int, n: int) -> np.ndarray:
    o = np.empty(n, dtype=np.float32)
    lib().orc_uniform_array(seed, req_id, tag, row, n, _ptr(o))
    return o


def round_bf16(x) -> np.ndarray:
    x = _c(x, np.float64)
    y = np.empty_like(x)
    lib().orc_round_bf16_array(_ptr(x), _ptr(y), x.size)
    return y


# ------------------------------------------------------------------------------------
# acceptance (Sec. 2.4)
# ------------------------------------------------------------------------------------
class AcceptResult:
    def __init__(self, B, M, S):
        self.accept_len = np.zeros(B, dtype=np.int32)
        self.out_tokens = np.zeros(M, dtype=np.int32)
        self.acc_u = np.zeros(max(S, 1), dtype=np.float32)
        self.acc_a = np.zeros(max(S, 1), dtype=np.float32)
        self.R = np.zeros(B, dtype=np.int32)
        self.degenerate = np.zeros(B, dtype=np.int32)
        self.race_key1 = np.zeros(B, dtype=np.float32)
        self.race_key2 = np.zeros(B, dtype=np.float32)


def accept(logits, tokens, q, gamma, temperature: float, seed: int, req_id=None,
           u_inject=None) -> AcceptResult:
    """Acceptance stage for a batch.

    logits [M][V] fp32 (M = sum(gamma+1), request-major), tokens [M] = per request
    [root, y_1..y_gamma], q [sum(gamma)][V] fp32 (row j-1 of a request holds q_j).
    Returns accept lengths, output tokens (y_1..y_L, extra, then -1), the acceptance
    draws/ratios of each decision taken, R, degenerate-residual flags and the top-two
    race keys (for near-tie accounting).
    """
    gamma = _c(gamma, np.int32)
    B = gamma.shape[0]
    logits = _c(logits, np.float32)
    V = logits.shape[-1]
    logits = logits.reshape(-1, V)
    M = int((gamma + 1).sum())
    S = int(gamma.sum())
    assert logits.shape[0] == M
    tokens = _c(tokens, np.int32).reshape(-1)
    assert tokens.shape[0] == M
    q = _c(q, np.float32).reshape(-1, V) if S > 0 else np.zeros((1, V), np.float32)
    assert S == 0 or q.shape[0] == S
    rid = _c(req_id, np.uint32) if req_id is not None else None
    ui = _c(u_inject, np.float32) if u_inject is not None else None
    res = AcceptResult(B, M, S)
    lib().orc_accept_batch(B, V, _ptr(gamma), _ptr(rid), _ptr(logits), _ptr(tokens), _ptr(q),
                           float(temperature), seed & ((1 << 64) - 1), _ptr(ui),
                           _ptr(res.accept_len), _ptr(res.out_tokens), _ptr(res.acc_u),
                           _ptr(res.acc_a), _ptr(res.R), _ptr(res.degenerate),
                           _ptr(res.race_key1), _ptr(res.race_key2))
    return res


def row_probs(logits_row, temperature: float) -> np.ndarray:
    """fp32 target distribution p of one logits row, exactly as the acceptance computes it."""
    l = _c(logits_row, np.float32).reshape(-1)
    p = np.empty_like(l)
    lib().orc_row_probs(_ptr(l), l.shape[0], float(temperature), _ptr(p))
    return p


def rope_apply(v, pos: int, base: float) -> np.ndarray:
    v = _c(v, np.float64).copy()
    lib().orc_rope_apply(_ptr(v), v.shape[0], int(pos), float(base))
    return v


def rmsnorm_apply(h, eps: float, bf16: bool = False) -> np.ndarray:
    h = _c(h, np.float64)
    rows, d = h.shape
    x = np.empty_like(h)
    lib().orc_rmsnorm_apply(_ptr(h), _ptr(x), rows, d, float(eps), int(bf16))
    return x


def plain_decode(logits_row, temperature: float, seed: int, req_id: int, row: int) -> int:
    l = _c(logits_row, np.float32).reshape(-1)
    return int(lib().orc_plain_decode(l.shape[0], _ptr(l), float(temperature),
                                      seed & ((1 << 64) - 1), req_id, row))


# ------------------------------------------------------------------------------------
# forward (Sec. 4.5)
# ------------------------------------------------------------------------------------
def paged_attention(q, k_pool, v_pool, page_table, ctx_len, n_new, n_kv: int, bf16: bool,
                    acc32: bool = False):
    """q [M][n_q][hd] float64; pools of ONE layer ([blocks][n_kv][16][hd], slot-major) as
    float32 or bf16 bits (uint16).  Returns [M][n_q][hd] fp64."""
    q = _c(q, np.float64)
    M, n_q, hd = q.shape
    out = np.empty_like(q)
    pt = _c(page_table, np.int32)
    ctx = _c(ctx_len, np.int32)
    nn = _c(n_new, np.int32)
    kp = np.ascontiguousarray(k_pool)
    vp = np.ascontiguousarray(v_pool)
    lib().orc_paged_attention(n_q, n_kv, hd, int(bf16), int(acc32), _ptr(kp), _ptr(vp), _ptr(pt),
                              pt.shape[1], ctx.shape[0], _ptr(ctx), _ptr(nn), _ptr(q), _ptr(out))
    return out


class _OrcModel(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d", C.c_int32), ("n_q", C.c_int32),
                ("n_kv", C.c_int32), ("hd", C.c_int32), ("F", C.c_int32), ("V", C.c_int32),
                ("bf16", C.c_int32), ("acc32", C.c_int32), ("eps", C.c_double),
                ("rope_base", C.c_double),
                ("embed", C.c_void_p), ("lm_head", C.c_void_p), ("final_norm", C.c_void_p),
                ("attn_norm", C.POINTER(C.c_void_p)), ("wq", C.POINTER(C.c_void_p)),
                ("wk", C.POINTER(C.c_void_p)), ("wv", C.POINTER(C.c_void_p)),
                ("wo", C.POINTER(C.c_void_p)), ("mlp_norm", C.POINTER(C.c_void_p)),
                ("w_gate", C.POINTER(C.c_void_p)), ("w_up", C.POINTER(C.c_void_p)),
                ("w_down", C.POINTER(C.c_void_p))]


def _np_storage(t):
    """torch tensor (float32 / bfloat16, CPU) or numpy array -> contiguous numpy storage."""
    try:
        import torch
        if isinstance(t, torch.Tensor):
            t = t.detach().contiguous().cpu()
            if t.dtype == torch.bfloat16:
                return t.view(torch.int16).numpy().view(np.uint16)
            return t.numpy()
    except ImportError:
        pass
    return np.ascontiguousarray(t)


class OracleModel:
    """Holds host copies of a model's weights in natural layout for the C oracle.

    ``layers`` is a list of dicts with keys wq, wk, wv, wo, w_gate, w_up, w_down,
    attn_norm, mlp_norm; ``glob`` has embed, lm_head, final_norm.  Weights are fp32
    arrays (fp32 model) or bf16 bit patterns (bf16 model)."""

    def __init__(self, shape, layers, glob):
        self.shape = shape
        self.bf16 = shape.dtype == "bf16"
        self._keep = []
        L = len(layers)

        def arr(t):
            a = _np_storage(t)
            self._keep.append(a)
            return a.ctypes.data_as(C.c_void_p)

        def vec(key):
            v = (C.c_void_p * L)(*[arr(layers[l][key]).value for l in range(L)])
            self._keep.append(v)
            return C.cast(v, C.POINTER(C.c_void_p))

        s = shape
        # the embedding table stays reachable so tests can perturb single entries
        self.embed = _np_storage(glob["embed"])
        self._keep.append(self.embed)
        self.s = _OrcModel(L, s.d_model, s.n_q_heads, s.n_kv_heads, s.head_dim, s.d_ff, s.vocab,
                           int(self.bf16), 0, s.rms_eps, s.rope_base, self.embed.ctypes.data_as(C.c_void_p),
                           arr(glob["lm_head"]), arr(glob["final_norm"]), vec("attn_norm"),
                           vec("wq"), vec("wk"), vec("wv"), vec("wo"), vec("mlp_norm"),
                           vec("w_gate"), vec("w_up"), vec("w_down"))


def forward(model: OracleModel, k_pool, v_pool, page_table, ctx_len, n_new, tokens,
            acc32: bool = False) -> np.ndarray:
    """Forward the new rows; updates the host pools in place (numpy arrays
    [n_layers][n_blocks][n_kv][16 * hd], each page slot-major, float32 or uint16 bf16
    bits).  Returns fp32 logits [M][V].  acc32: every sum accumulates in fp32 in natural
    index order (the fp64 result is the reference; this mode measures the rounding floor)."""
    assert k_pool.flags["C_CONTIGUOUS"] and v_pool.flags["C_CONTIGUOUS"]
    n_blocks = k_pool.shape[1]
    pt = _c(page_table, np.int32)
    ctx = _c(ctx_len, np.int32)
    nn = _c(n_new, np.int32)
    tok = _c(tokens, np.int32)
    M = int(nn.sum())
    assert tok.shape[0] == M
    logits = np.empty((M, model.shape.vocab), dtype=np.float32)
    model.s.acc32 = int(acc32)
    try:
        lib().orc_forward(C.byref(model.s), _ptr(k_pool), _ptr(v_pool), n_blocks, ctx.shape[0],
                          _ptr(ctx), _ptr(nn), _ptr(pt), pt.shape[1], _ptr(tok), _ptr(logits))
    finally:
        model.s.acc32 = 0
    return logits


def linear_apply(W, x, acc32: bool = False) -> np.ndarray:
    """y = x W^T exactly as the forward's projections compute it: W [out][in] fp32 values,
    x [rows][in]; fp64 sums, or fp32 sums in natural k order with acc32."""
    W = _c(W, np.float32)
    x = _c(x, np.float64)
    y = np.empty((x.shape[0], W.shape[0]), np.float64)
    lib().orc_linear_apply(_ptr(W), _ptr(x), _ptr(y), x.shape[0], x.shape[1], W.shape[0], int(acc32))
    return y
