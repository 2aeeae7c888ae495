"""MI355X (gfx950) batched speculative-verification step of WISP (arXiv 2601.11652).

Thin ctypes binding of ``libwisp.so`` (C ABI in include/wisp.h).  Every step of the
verification path runs in the library's HIP kernels; this module only marshals
arguments (torch tensors supply device memory and the stream).  Any call raises if
the library has not been built -- there is no fallback implementation.

Entry points keep the C names: wisp_verify, wisp_accept, wisp_attention,
wisp_pack_linear, wisp_workspace_size, wisp_accept_workspace_size, wisp_uniform,
wisp_check, wisp_last_error, wisp_schedule, wisp_draft_stats, wisp_reject_predict;
``KVManager`` wraps the wisp_kvm_* calls and ``RejectMLP`` the predictor's weights.
``GpuModel`` and ``BatchDesc`` assemble the C structs.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwisp.so")

WISP_OK = 0
WISP_E_INVALID = -1
WISP_E_CAPACITY = -2
WISP_E_WORKSPACE = -3
WISP_E_UNSUPPORTED = -4
WISP_E_HIP = -5
WISP_E_DEVICE_INPUT = -6
WISP_E_HOST_MEMORY = -7
WISP_F32 = 0
WISP_BF16 = 1
PAGE = 16
GAMMA_MAX = 16
PREFILL_MAX = 32768
ROWS_MAX = 262144
TAG_ACCEPT = 1
TAG_RACE = 2

EXPORTS = ("wisp_workspace_size", "wisp_logits_workspace_size", "wisp_accept_workspace_size", "wisp_pack_linear",
           "wisp_pack_gate_up", "wisp_verify",
           "wisp_accept", "wisp_attention", "wisp_uniform", "wisp_check", "wisp_profile_enable",
           "wisp_profile_read", "wisp_profile_reset", "wisp_last_error", "wisp_schedule", "wisp_kvm_create",
           "wisp_kvm_destroy", "wisp_kvm_lookup", "wisp_kvm_reserve", "wisp_kvm_commit", "wisp_kvm_release",
           "wisp_kvm_get_stats", "wisp_draft_stats_workspace_size", "wisp_draft_stats", "wisp_reject_predict",
           "wisp_gemm_plan", "wisp_verify_noalloc")


class WispError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"wisp status {status}: {msg}")
        self.status = status


_VP = C.c_void_p
_PVP = C.POINTER(C.c_void_p)


class wisp_model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ff", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_float), ("rope_base", C.c_float),
                ("dtype", C.c_int32), ("embed", _VP), ("final_norm", _VP), ("lm_head", _VP),
                ("attn_norm", _PVP), ("w_qkv", _PVP), ("w_o", _PVP), ("mlp_norm", _PVP),
                ("w_gate_up", _PVP), ("w_down", _PVP)]


class wisp_kv(C.Structure):
    _fields_ = [("k_pool", _VP), ("v_pool", _VP), ("n_blocks", C.c_int32), ("page_size", C.c_int32)]


class wisp_batch_desc(C.Structure):
    _fields_ = [("B", C.c_int32), ("ctx_len", C.POINTER(C.c_int32)), ("gamma", C.POINTER(C.c_int32)),
                ("req_id", C.POINTER(C.c_uint32)), ("kv_page_table", _VP), ("pt_stride", C.c_int32),
                ("temperature", C.c_float), ("prefill_len", C.POINTER(C.c_int32))]


class wisp_latency_model(C.Structure):
    _fields_ = [("a", C.c_double), ("b_compute", C.c_double), ("b_read", C.c_double), ("c", C.c_double)]


class wisp_sched_request(C.Structure):
    _fields_ = [("arrival", C.c_double), ("deadline", C.c_double), ("g_hat", C.c_double),
                ("m_hat", C.c_double), ("ctx_len", C.c_int32), ("l_new", C.c_int32)]


class wisp_kvm_stats(C.Structure):
    _fields_ = [("n_pages", C.c_int32), ("free_pages", C.c_int32), ("sessions", C.c_int32),
                ("evictions", C.c_int64), ("pages_evicted", C.c_int64), ("pages_allocated", C.c_int64),
                ("pages_freed", C.c_int64), ("lookup_hits", C.c_int64), ("lookup_misses", C.c_int64)]


class wisp_reject_mlp(C.Structure):
    _fields_ = [("n_in", C.c_int32), ("mean", C.c_void_p), ("inv_std", C.c_void_p), ("w1", C.c_void_p),
                ("b1", C.c_void_p), ("w2", C.c_void_p), ("b2", C.c_void_p), ("w3", C.c_void_p),
                ("b3", C.c_void_p), ("w4", C.c_void_p), ("b4", C.c_float)]


WISP_SCHED_SLO = 0
WISP_SCHED_FCFS = 1
WISP_SCHED_SLO_LIVE = 2

_lib = None


def load_library():
    """The loaded libwisp.so (raises ImportError when it has not been built)."""
    global _lib
    if _lib is None:
        _lib = _load()
    return _lib


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2601_11652_amd.build.build() "
                          "(or __graft_entry__.build()); there is no fallback path")
    L = C.CDLL(LIB_PATH)
    L.wisp_workspace_size.argtypes = [C.POINTER(wisp_model), C.POINTER(wisp_batch_desc)]
    L.wisp_workspace_size.restype = C.c_size_t
    L.wisp_logits_workspace_size.argtypes = [C.POINTER(wisp_model), C.POINTER(wisp_batch_desc)]
    L.wisp_logits_workspace_size.restype = C.c_size_t
    L.wisp_accept_workspace_size.argtypes = [C.POINTER(wisp_batch_desc), C.c_int32]
    L.wisp_accept_workspace_size.restype = C.c_size_t
    L.wisp_pack_linear.argtypes = [_VP, _VP, C.c_int32, C.c_int32, C.c_int32, _VP]
    L.wisp_pack_gate_up.argtypes = [_VP, _VP, _VP, C.c_int32, C.c_int32, C.c_int32, _VP]
    L.wisp_verify.argtypes = [C.POINTER(wisp_model), C.POINTER(wisp_kv), C.POINTER(wisp_batch_desc),
                              _VP, _VP, C.c_uint64, _VP, _VP, _VP, _VP, C.c_size_t, _VP]
    L.wisp_verify_noalloc.argtypes = [C.POINTER(wisp_model), C.POINTER(wisp_kv), C.POINTER(wisp_batch_desc),
                                      _VP, _VP, C.c_uint64, _VP, _VP, _VP, _VP, _VP]
    L.wisp_accept.argtypes = [C.POINTER(wisp_batch_desc), C.c_int32, _VP, _VP, _VP, C.c_uint64, _VP,
                              _VP, _VP, C.c_size_t, _VP]
    L.wisp_attention.argtypes = [C.POINTER(wisp_model), C.POINTER(wisp_kv), C.POINTER(wisp_batch_desc),
                                 _VP, _VP, _VP, C.c_size_t, _VP]
    L.wisp_uniform.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32, _VP, _VP]
    L.wisp_check.argtypes = [_VP, _VP]
    L.wisp_gemm_plan.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_int32)]
    L.wisp_profile_enable.argtypes = [C.c_int]
    L.wisp_profile_read.argtypes = [C.c_int, C.POINTER(C.c_double), C.POINTER(C.c_int64),
                                    C.POINTER(C.c_double), C.POINTER(C.c_double)]
    L.wisp_profile_reset.argtypes = []
    L.wisp_last_error.argtypes = []
    L.wisp_last_error.restype = C.c_char_p
    L.wisp_schedule.argtypes = [C.c_int32, C.POINTER(wisp_sched_request), C.c_int32, C.c_double, C.c_double,
                                C.c_double, C.POINTER(wisp_latency_model), C.POINTER(C.c_int32),
                                C.POINTER(C.c_int32)]
    _I32P, _I64P = C.POINTER(C.c_int32), C.POINTER(C.c_int64)
    L.wisp_kvm_create.argtypes = [C.c_int32, C.c_int32, C.POINTER(_VP)]
    L.wisp_kvm_destroy.argtypes = [_VP]
    L.wisp_kvm_destroy.restype = None
    L.wisp_kvm_lookup.argtypes = [_VP, _I64P, C.c_int32, _I32P]
    L.wisp_kvm_reserve.argtypes = [_VP, _I64P, _I32P, C.c_int32, _I32P, C.c_int32, _I32P]
    L.wisp_kvm_commit.argtypes = [_VP, _I64P, _I32P, C.c_int32]
    L.wisp_kvm_release.argtypes = [_VP, _I64P, C.c_int32]
    L.wisp_kvm_get_stats.argtypes = [_VP, C.POINTER(wisp_kvm_stats)]
    L.wisp_draft_stats_workspace_size.argtypes = [C.c_int32, C.c_int32]
    L.wisp_draft_stats_workspace_size.restype = C.c_size_t
    L.wisp_draft_stats.argtypes = [_VP, C.c_int32, C.c_int32, C.c_int64, C.c_float, _VP, _VP, C.c_size_t, _VP]
    L.wisp_reject_predict.argtypes = [C.POINTER(wisp_reject_mlp), _VP, C.c_int32, _VP, _VP]
    for name in ("wisp_pack_linear", "wisp_pack_gate_up", "wisp_verify", "wisp_verify_noalloc", "wisp_accept", "wisp_attention", "wisp_uniform",
                 "wisp_check", "wisp_gemm_plan", "wisp_profile_enable", "wisp_profile_read", "wisp_profile_reset",
                 "wisp_schedule", "wisp_kvm_create", "wisp_kvm_lookup", "wisp_kvm_reserve", "wisp_kvm_commit",
                 "wisp_kvm_release", "wisp_kvm_get_stats", "wisp_draft_stats", "wisp_reject_predict"):
        getattr(L, name).restype = C.c_int
    return L


class _Lazy:
    def __getattr__(self, name):
        return getattr(load_library(), name)


lib = _Lazy()


def wisp_last_error() -> str:
    return lib.wisp_last_error().decode()


def _ok(status: int):
    if status != WISP_OK:
        raise WispError(status, wisp_last_error())


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr()


def _dev(t, what: str, numel: int = 0, dtype=None, elem: int | None = None, contiguous: bool = True) -> int:
    """Device pointer of a torch tensor after the checks a C caller would owe the library:
    on the GPU, of the element type the entry point reads, contiguous, and holding at least
    `numel` elements.  A host tensor's pointer must never reach a kernel."""
    import torch
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{what}: expected a device tensor, got {type(t).__name__}"
                         + (f" on {t.device}" if isinstance(t, torch.Tensor) else ""))
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what}: dtype {t.dtype}, expected {dtype}")
    if elem is not None and t.element_size() != elem:
        raise ValueError(f"{what}: {t.element_size()}-byte elements, expected {elem}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{what}: must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{what}: {t.numel()} elements, needs at least {numel}")
    return t.data_ptr()


def _i32():
    import torch
    return torch.int32


def _f32():
    import torch
    return torch.float32


def _check_kv(model: "wisp_model", kv: "KVPool", layers: int):
    es = 2 if model.dtype == WISP_BF16 else 4
    per_layer = kv.c.n_blocks * model.n_kv_heads * PAGE * model.head_dim
    for name, t in (("kv.k", kv.k), ("kv.v", kv.v)):
        _dev(t, name, layers * per_layer, elem=es)


def _check_desc(desc: "BatchDesc"):
    if desc.B > 0:
        pt = desc.page_table
        _dev(pt, "desc.page_table", dtype=_i32())
        if pt.dim() != 2 or pt.shape[0] < desc.B:
            raise ValueError(f"desc.page_table: expected [>= {desc.B}][pt_stride], got {tuple(pt.shape)}")


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# ------------------------------------------------------------------------------------------
# struct builders
# ------------------------------------------------------------------------------------------
class BatchDesc:
    """Owns the host arrays behind a wisp_batch_desc."""

    def __init__(self, ctx_len, gamma, page_table=None, temperature: float = 1.0, req_id=None,
                 prefill_len=None):
        self.ctx_len = np.ascontiguousarray(ctx_len, dtype=np.int32)
        self.gamma = np.ascontiguousarray(gamma, dtype=np.int32)
        self.req_id = None if req_id is None else np.ascontiguousarray(req_id, dtype=np.uint32)
        self.prefill_len = None if prefill_len is None else np.ascontiguousarray(prefill_len, dtype=np.int32)
        self.page_table = page_table          # torch int32 [B][stride] on the device
        B = self.ctx_len.shape[0]
        self.c = wisp_batch_desc()
        self.c.B = B
        self.c.ctx_len = self.ctx_len.ctypes.data_as(C.POINTER(C.c_int32))
        self.c.gamma = self.gamma.ctypes.data_as(C.POINTER(C.c_int32))
        self.c.req_id = (self.req_id.ctypes.data_as(C.POINTER(C.c_uint32))
                         if self.req_id is not None else None)
        if page_table is not None:
            assert page_table.dtype.__str__() == "torch.int32" and page_table.is_contiguous()
            self.c.kv_page_table = page_table.data_ptr()
            self.c.pt_stride = page_table.shape[1]
        self.c.temperature = float(temperature)
        self.c.prefill_len = (self.prefill_len.ctypes.data_as(C.POINTER(C.c_int32))
                              if self.prefill_len is not None else None)

    @property
    def B(self):
        return int(self.c.B)

    @property
    def M(self):
        """Verification rows (logits rows): sum(gamma + 1)."""
        return int((self.gamma.astype(np.int64) + 1).sum())

    @property
    def rows(self):
        """Forwarded rows (token count): sum(prefill_len + gamma + 1)."""
        pre = 0 if self.prefill_len is None else int(self.prefill_len.astype(np.int64).sum())
        return self.M + pre

    @property
    def S(self):
        return int(self.gamma.sum())


class KVPool:
    """Two device pools [n_layers][n_blocks][n_kv][16 * head_dim] in the page layout."""

    def __init__(self, k, v):
        assert k.shape == v.shape and k.is_contiguous() and v.is_contiguous()
        self.k, self.v = k, v
        self.c = wisp_kv(k.data_ptr(), v.data_ptr(), k.shape[1], PAGE)

    @staticmethod
    def zeros(n_layers, n_blocks, n_kv, head_dim, dtype, device="cuda"):
        import torch
        shp = (n_layers, n_blocks, n_kv, PAGE * head_dim)
        return KVPool(torch.zeros(shp, dtype=dtype, device=device), torch.zeros(shp, dtype=dtype, device=device))

    def layer(self, l: int) -> "KVPool":
        return KVPool(self.k[l:l + 1], self.v[l:l + 1])


class GpuModel:
    """Packed device weights plus the wisp_model struct pointing at them.

    ``layer_source(l)`` returns the natural-layout device tensors of layer l (keys wq, wk,
    wv, wo, w_gate, w_up, w_down, attn_norm, mlp_norm); ``glob`` holds embed, lm_head,
    final_norm.  Natural tensors are released after packing."""

    def __init__(self, shape, layer_source, glob, stream=None):
        import torch
        self.shape = shape
        s = shape
        dt = torch.float32 if s.dtype == "f32" else torch.bfloat16
        code = WISP_F32 if s.dtype == "f32" else WISP_BF16
        self.dtype_code = code
        st = _stream(stream)
        dev = glob["embed"].device

        def pack(dst, src, rows, cols, row0=0):
            assert src.is_contiguous() and src.dtype == dt and tuple(src.shape) == (rows, cols)
            _ok(lib.wisp_pack_linear(dst.data_ptr() + row0 * cols * dst.element_size(), src.data_ptr(),
                                     rows, cols, code, st))

        self.layers = []
        for l in range(s.n_layers):
            w = layer_source(l)
            qd, kd = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim
            qkv = torch.empty((qd + 2 * kd) * s.d_model, dtype=dt, device=dev)
            pack(qkv, w["wq"], qd, s.d_model, 0)
            pack(qkv, w["wk"], kd, s.d_model, qd)
            pack(qkv, w["wv"], kd, s.d_model, qd + kd)
            wo = torch.empty(s.d_model * qd, dtype=dt, device=dev)
            pack(wo, w["wo"], s.d_model, qd)
            gu = torch.empty(2 * s.d_ff * s.d_model, dtype=dt, device=dev)
            for x in ("w_gate", "w_up"):
                assert w[x].is_contiguous() and w[x].dtype == dt and tuple(w[x].shape) == (s.d_ff, s.d_model)
            wisp_pack_gate_up(gu, w["w_gate"], w["w_up"], s.d_ff, s.d_model, code, stream)
            wd = torch.empty(s.d_model * s.d_ff, dtype=dt, device=dev)
            pack(wd, w["w_down"], s.d_model, s.d_ff)
            self.layers.append({"attn_norm": w["attn_norm"].contiguous(), "mlp_norm": w["mlp_norm"].contiguous(),
                                "w_qkv": qkv, "w_o": wo, "w_gate_up": gu, "w_down": wd})
            torch.cuda.current_stream().synchronize()
            del w
        self.embed = glob["embed"].contiguous()
        self.final_norm = glob["final_norm"].contiguous()
        self.lm_head = torch.empty(s.vocab * s.d_model, dtype=dt, device=dev)
        pack(self.lm_head, glob["lm_head"], s.vocab, s.d_model)
        torch.cuda.current_stream().synchronize()

        L = s.n_layers

        def arr(key):
            a = (C.c_void_p * L)(*[self.layers[l][key].data_ptr() for l in range(L)])
            return a

        self._arrs = {k: arr(k) for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")}
        self.c = wisp_model(L, s.d_model, s.n_q_heads, s.n_kv_heads, s.head_dim, s.d_ff, s.vocab,
                            s.rms_eps, s.rope_base, code, self.embed.data_ptr(), self.final_norm.data_ptr(),
                            self.lm_head.data_ptr(),
                            *[C.cast(self._arrs[k], _PVP) for k in ("attn_norm", "w_qkv", "w_o",
                                                                    "mlp_norm", "w_gate_up", "w_down")])

    @staticmethod
    def shape_only(shape) -> wisp_model:
        code = WISP_F32 if shape.dtype == "f32" else WISP_BF16
        return wisp_model(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                          shape.d_ff, shape.vocab, shape.rms_eps, shape.rope_base, code)


# ------------------------------------------------------------------------------------------
# entry points (C names)
# ------------------------------------------------------------------------------------------
def wisp_workspace_size(model: wisp_model, desc: BatchDesc) -> int:
    return int(lib.wisp_workspace_size(C.byref(model), C.byref(desc.c)))


def wisp_logits_workspace_size(model: wisp_model, desc: BatchDesc) -> int:
    """Extra workspace bytes wisp_verify needs when target_logits is None."""
    return int(lib.wisp_logits_workspace_size(C.byref(model), C.byref(desc.c)))


def wisp_accept_workspace_size(desc: BatchDesc, vocab: int) -> int:
    return int(lib.wisp_accept_workspace_size(C.byref(desc.c), vocab))


def wisp_pack_linear(dst, src, rows: int, cols: int, dtype: int, stream=None):
    es = 2 if dtype == WISP_BF16 else 4
    n = max(rows, 0) * max(cols, 0)
    _ok(lib.wisp_pack_linear(_dev(dst, "dst", n, elem=es), _dev(src, "src", n, elem=es), rows, cols, dtype,
                             _stream(stream)))


def wisp_pack_gate_up(dst, w_gate, w_up, d_ff: int, d_model: int, dtype: int, stream=None):
    es = 2 if dtype == WISP_BF16 else 4
    n = max(d_ff, 0) * max(d_model, 0)
    _ok(lib.wisp_pack_gate_up(_dev(dst, "dst", 2 * n, elem=es), _dev(w_gate, "w_gate", n, elem=es),
                              _dev(w_up, "w_up", n, elem=es), d_ff, d_model, dtype, _stream(stream)))


def _ws(workspace) -> tuple[int, int]:
    return _dev(workspace, "workspace"), workspace.numel() * workspace.element_size()


def wisp_verify(model: wisp_model, kv: KVPool, desc: BatchDesc, tokens, draft_probs, rng_seed: int,
                accept_len, out_tokens, target_logits, workspace, stream=None):
    _check_desc(desc)
    _check_kv(model, kv, model.n_layers)
    V = model.vocab
    probs = _dev(draft_probs, "draft_probs", desc.S * V, dtype=_f32()) if desc.S > 0 else _ptr(draft_probs)
    logits = None if target_logits is None else _dev(target_logits, "target_logits", desc.M * V, dtype=_f32())
    _ok(lib.wisp_verify(C.byref(model), C.byref(kv.c), C.byref(desc.c),
                        _dev(tokens, "tokens", desc.rows, dtype=_i32()), probs, rng_seed & ((1 << 64) - 1),
                        _dev(accept_len, "accept_len", desc.B, dtype=_i32()),
                        _dev(out_tokens, "out_tokens", desc.M, dtype=_i32()), logits, *_ws(workspace),
                        _stream(stream)))


def wisp_verify_noalloc(model: wisp_model, kv: KVPool, desc: BatchDesc, tokens, draft_probs, rng_seed: int,
                        accept_len, out_tokens, target_logits, fault=None, stream=None):
    """wisp_verify without a workspace (the library's static per-device scratch); `fault`
    (device int32 [1] or None) accumulates device-side input faults."""
    _check_desc(desc)
    _check_kv(model, kv, model.n_layers)
    V = model.vocab
    probs = _dev(draft_probs, "draft_probs", desc.S * V, dtype=_f32()) if desc.S > 0 else _ptr(draft_probs)
    logits = None if target_logits is None else _dev(target_logits, "target_logits", desc.M * V, dtype=_f32())
    flt = None if fault is None else _dev(fault, "fault", 1, dtype=_i32())
    _ok(lib.wisp_verify_noalloc(C.byref(model), C.byref(kv.c), C.byref(desc.c),
                                _dev(tokens, "tokens", desc.rows, dtype=_i32()), probs, rng_seed & ((1 << 64) - 1),
                                _dev(accept_len, "accept_len", desc.B, dtype=_i32()),
                                _dev(out_tokens, "out_tokens", desc.M, dtype=_i32()), logits, flt,
                                _stream(stream)))


def wisp_accept(desc: BatchDesc, vocab: int, logits, tokens, draft_probs, rng_seed: int, accept_len,
                out_tokens, workspace, stream=None):
    probs = _dev(draft_probs, "draft_probs", desc.S * vocab, dtype=_f32()) if desc.S > 0 else _ptr(draft_probs)
    _ok(lib.wisp_accept(C.byref(desc.c), vocab, _dev(logits, "logits", desc.M * max(vocab, 0), dtype=_f32()),
                        _dev(tokens, "tokens", desc.M, dtype=_i32()), probs, rng_seed & ((1 << 64) - 1),
                        _dev(accept_len, "accept_len", desc.B, dtype=_i32()),
                        _dev(out_tokens, "out_tokens", desc.M, dtype=_i32()), *_ws(workspace), _stream(stream)))


def wisp_attention(model: wisp_model, kv: KVPool, desc: BatchDesc, q, out, workspace, stream=None):
    _check_desc(desc)
    _check_kv(model, kv, 1)
    es = 2 if model.dtype == WISP_BF16 else 4
    n = desc.rows * model.n_q_heads * model.head_dim
    _ok(lib.wisp_attention(C.byref(model), C.byref(kv.c), C.byref(desc.c), _dev(q, "q", n, elem=es),
                           _dev(out, "out", n, elem=es), *_ws(workspace), _stream(stream)))


def wisp_uniform(rng_seed: int, req_id: int, tag: int, row: int, n: int, out, stream=None):
    _ok(lib.wisp_uniform(rng_seed & ((1 << 64) - 1), req_id, tag, row, n, _dev(out, "out", n, dtype=_f32()),
                         _stream(stream)))


def wisp_schedule(policy: int, requests, t_now: float, mem_budget: float, guard: float, model) -> list:
    """Batch for the dispatch epoch t_now (Sec. 4.3, Alg. 1; host code).  requests: sequence of
    objects with arrival, deadline, g_hat, m_hat, ctx_len, l_new; model: (a, b_compute,
    b_read, c) in seconds.  Returns the admitted request indices in admission order."""
    n = len(requests)
    arr = (wisp_sched_request * max(n, 1))()
    for i, r in enumerate(requests):
        arr[i] = wisp_sched_request(r.arrival, r.deadline, r.g_hat, r.m_hat, r.ctx_len, r.l_new)
    out = (C.c_int32 * max(n, 1))()
    k = C.c_int32(0)
    m = wisp_latency_model(*[float(x) for x in model])
    _ok(lib.wisp_schedule(policy, arr, n, t_now, mem_budget, guard, C.byref(m), out, C.byref(k)))
    return list(out[:k.value])


def wisp_draft_stats(logits, vocab: int, temperature: float, stats, ws=None, stream=None):
    """stats [rows][4] fp32 (confidence, entropy, top-2 margin, std of z) of logits rows
    [rows][ld] fp32 (the first `vocab` entries of each row), z = logits / temperature.
    `ws` (a device byte tensor of wisp_draft_stats_workspace_size bytes) is allocated when
    not given."""
    rows = logits.shape[0]
    if logits.dim() != 2 or logits.stride(1) != 1 or logits.shape[1] < vocab:
        raise ValueError(f"logits: expected [rows][>= {vocab}] with unit column stride")
    if ws is None:
        ws = workspace(lib.wisp_draft_stats_workspace_size(rows, vocab))
    _ok(lib.wisp_draft_stats(_dev(logits, "logits", dtype=_f32(), contiguous=False), rows, vocab, logits.stride(0),
                             temperature, _dev(stats, "stats", rows * 4, dtype=_f32()), *_ws(ws), _stream(stream)))


class RejectMLP:
    """Device weights of the rejection predictor MLP (hidden 512, 128, 64; fp32 tensors
    w1 [512][n_in], b1, w2 [128][512], b2, w3 [64][128], b3, w4 [64], scalar b4, and the input
    standardisation mean / inv_std [n_in])."""

    def __init__(self, params: dict):
        self.t = {k: v.contiguous() for k, v in params.items() if k != "b4"}
        for k, v in self.t.items():
            _dev(v, f"params[{k!r}]", dtype=_f32())
        self.c = wisp_reject_mlp(int(self.t["w1"].shape[1]), *[self.t[k].data_ptr() for k in
                                 ("mean", "inv_std", "w1", "b1", "w2", "b2", "w3", "b3", "w4")], float(params["b4"]))


def wisp_reject_predict(mlp: RejectMLP, features, p_accept, stream=None):
    rows = features.shape[0]
    _ok(lib.wisp_reject_predict(C.byref(mlp.c), _dev(features, "features", rows * mlp.c.n_in, dtype=_f32()), rows,
                                _dev(p_accept, "p_accept", rows, dtype=_f32()), _stream(stream)))


class KVManager:
    """A wisp_kv_manager (host code): page ids for multi-round sessions over a pool of
    n_pages pages (Sec. 4.5's in-place, prefix-cached KV).  Arrays are numpy."""

    def __init__(self, n_pages: int, page_size: int = PAGE):
        h = _VP()
        _ok(lib.wisp_kvm_create(n_pages, page_size, C.byref(h)))
        self._h = h
        self.page_size = page_size

    @staticmethod
    def _ids(sids):
        a = np.ascontiguousarray(sids, dtype=np.int64)
        return a, a.ctypes.data_as(C.POINTER(C.c_int64))

    @staticmethod
    def _i32(x, n):
        a = np.ascontiguousarray(np.broadcast_to(np.asarray(x, dtype=np.int32), (n,)))
        return a, a.ctypes.data_as(C.POINTER(C.c_int32))

    def lookup(self, sids) -> np.ndarray:
        ids, pid = self._ids(sids)
        out = np.zeros(ids.shape[0], np.int32)
        _ok(lib.wisp_kvm_lookup(self._h, pid, ids.shape[0], out.ctypes.data_as(C.POINTER(C.c_int32))))
        return out

    def reserve(self, sids, n_tokens, pt_stride: int):
        """(page table [n][pt_stride] int32, sessions evicted by the call)."""
        ids, pid = self._ids(sids)
        n = ids.shape[0]
        nt, pnt = self._i32(n_tokens, n)
        table = np.full((n, pt_stride), -1, np.int32)
        ev = C.c_int32(0)
        _ok(lib.wisp_kvm_reserve(self._h, pid, pnt, n, table.ctypes.data_as(C.POINTER(C.c_int32)), pt_stride,
                                 C.byref(ev)))
        return table, ev.value

    def commit(self, sids, cached):
        ids, pid = self._ids(sids)
        c, pc = self._i32(cached, ids.shape[0])
        _ok(lib.wisp_kvm_commit(self._h, pid, pc, ids.shape[0]))

    def release(self, sids):
        ids, pid = self._ids(sids)
        _ok(lib.wisp_kvm_release(self._h, pid, ids.shape[0]))

    def stats(self) -> dict:
        st = wisp_kvm_stats()
        _ok(lib.wisp_kvm_get_stats(self._h, C.byref(st)))
        return {k: getattr(st, k) for k, _ in wisp_kvm_stats._fields_}

    def close(self):
        if getattr(self, "_h", None):
            lib.wisp_kvm_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def gemm_plan(M: int, N: int, K: int) -> dict:
    """The launch plan of one bf16 projection (wisp_gemm_plan): kernel variant, row blocks,
    32-row fragments per block, K ranges."""
    out = (C.c_int32 * 4)()
    _ok(lib.wisp_gemm_plan(int(M), int(N), int(K), out))
    return dict(kind=out[0], rb=out[1], mt=out[2], splits=out[3])


def wisp_check(workspace, stream=None):
    _ok(lib.wisp_check(_dev(workspace, "workspace"), _stream(stream)))


def workspace(nbytes: int, device="cuda"):
    """A device byte buffer for the workspace argument (torch allocation), its fault record
    (the first 256 bytes) cleared as the library requires before first use."""
    import torch
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    ws[:256].zero_()
    return ws
