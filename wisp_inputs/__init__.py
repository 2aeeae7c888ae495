"""Seeded synthetic inputs for the batched speculative-verification step.

This module only draws numbers: model weights, request mixes, token ids,
context KV values, page tables and draft noise.  It holds none of the
verification method's arithmetic, so the CPU oracle and the GPU path may both
consume what it produces.

Large tensors (weights, context KV) come from an integer-exact counter-based
generator evaluated with torch integer ops, so a tensor produced on the GPU is
bitwise identical to the same tensor produced on the host, and any slice of it
(one layer, one request) can be regenerated on its own.

Workloads follow the paper's verification setting (Sec. 4.4 and Sec. 4.5): each
request carries a cached context of ctx_len tokens and gamma drafted tokens; the
step forwards gamma+1 rows per request.  The five named workloads and their
distributions are described in the repository's design notes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import zlib
from dataclasses import dataclass, field

import numpy as np
import torch

MASTER_SEED = 11652
PAGE = 16  # tokens per KV page


# --------------------------------------------------------------------------------------
# model shapes
# --------------------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    dtype: str          # "f32" or "bf16": storage of weights, activations at GEMM inputs, KV
    rope_base: float
    rms_eps: float = 1e-5

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def replace(self, **kw) -> "ModelShape":
        d = dict(self.__dict__)
        d.update(kw)
        return ModelShape(**d)


TINY = ModelShape("tiny-2L-d256", 2, 256, 4, 4, 64, 1024, 1024, "f32", 10000.0)
LLAMA3_8B = ModelShape("llama3-8b-shape", 32, 4096, 32, 8, 128, 14336, 128256, "bf16", 500000.0)
LLAMA3_70B = ModelShape("llama3-70b-shape", 80, 8192, 64, 8, 128, 28672, 128256, "bf16", 500000.0)


# --------------------------------------------------------------------------------------
# integer-exact counter-based generator (identical on every torch device)
# --------------------------------------------------------------------------------------
_M32 = 0xFFFFFFFF
_MIX = 0x45D9F3B   # 27-bit multiplier: products of 32-bit values stay below 2**63


def _key32(*parts) -> tuple[int, int]:
    s = ":".join(str(p) for p in parts).encode()
    return zlib.crc32(b"a|" + s) & _M32, zlib.crc32(b"b|" + s) & _M32


def _mix32_(h: torch.Tensor) -> torch.Tensor:
    """In-place 32-bit integer mixer on an int64 tensor holding values in [0, 2**32)."""
    h ^= h >> 16
    h.mul_(_MIX).bitwise_and_(_M32)
    h ^= h >> 16
    h.mul_(_MIX).bitwise_and_(_M32)
    h ^= h >> 16
    return h


def hashed_u32(key: tuple[int, int], start: int, n: int, device) -> torch.Tensor:
    """32-bit hash values for element indices start .. start+n-1 of the stream `key`."""
    assert 0 <= start and start + n <= (1 << 32), "stream index must fit in 32 bits"
    h = torch.arange(start, start + n, dtype=torch.int64, device=device)
    h ^= key[0]
    _mix32_(h)
    h ^= key[1]
    _mix32_(h)
    return h


# host implementation of the same generator (C, OpenMP): bitwise the same values
_HERE = os.path.dirname(os.path.abspath(__file__))
_GEN_SRC = os.path.join(_HERE, "gen.c")
_GEN_LIB = os.path.join(_HERE, "libwisp_inputs.so")
_gen = None


def build_host_generator(force: bool = True) -> str:
    if force or not os.path.exists(_GEN_LIB) or os.path.getmtime(_GEN_LIB) < os.path.getmtime(_GEN_SRC):
        tmp = _GEN_LIB + ".tmp"
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _GEN_SRC])
        os.replace(tmp, _GEN_LIB)
    return _GEN_LIB


def _host_gen():
    global _gen
    if _gen is None:
        build_host_generator(force=False)
        L = ctypes.CDLL(_GEN_LIB)
        vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
        for f in ("gen_table16", "gen_table32"):
            getattr(L, f).argtypes = [vp, u32, u32, u64, u64, vp]
        for f in ("gen_kv16", "gen_kv32"):
            getattr(L, f).argtypes = [u32, u32, u64, u64, vp]
        _gen = L
    return _gen


_QTABLE: dict = {}


def _normal_table(std: float, dtype: torch.dtype) -> torch.Tensor:
    """65536 midpoint quantiles of N(0, std^2), rounded once on the host to `dtype`."""
    k = (std, dtype)
    if k not in _QTABLE:
        from scipy.special import ndtri
        p = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
        t = torch.from_numpy(ndtri(p) * std)            # float64 on the host
        _QTABLE[k] = t.to(torch.float32).to(dtype)      # float32 then (for bf16) RNE
    return _QTABLE[k]


_CHUNK = 1 << 24
_FORCE_TORCH_GEN = False   # tests flip this to compare the two implementations


def normal_tensor(seed: int, name: str, shape, std: float, dtype: torch.dtype,
                  device="cpu", out: torch.Tensor | None = None) -> torch.Tensor:
    """N(0, std) values (through a 16-bit quantile table) for the named tensor.

    The value of flat element e depends only on (seed, name, e), on every device.
    """
    n = int(np.prod(shape))
    table = _normal_table(std, dtype).to(device)
    if out is None:
        out = torch.empty(n, dtype=dtype, device=device)
    flat = out.view(-1)
    assert flat.numel() == n
    key = _key32(seed, name)
    if flat.device.type == "cpu" and not _FORCE_TORCH_GEN:
        f = _host_gen().gen_table16 if dtype == torch.bfloat16 else _host_gen().gen_table32
        assert dtype in (torch.bfloat16, torch.float32)
        f(table.data_ptr(), key[0], key[1], 0, n, flat.data_ptr())
        return out.view(*shape)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        h = hashed_u32(key, s, m, device)
        flat[s:s + m] = table[h >> 16]
        del h
    return out.view(*shape)


def kv_values(seed: int, layer: int, req: int, start_pos: int, n_pos: int, n_kv: int, hd: int,
              device="cpu", dtype=torch.bfloat16):
    """Synthetic cached K and V for positions start_pos .. start_pos+n_pos-1 of one request.

    Each element is (2k - 255) / 128 with k an 8-bit field of the hash: odd multiples of
    2^-7 in [-1.99, 1.99], exactly representable in bf16 and fp32.  Returns (K, V), each
    of logical shape [n_pos][n_kv][hd].
    """
    per_pos = 2 * n_kv * hd
    key = _key32(seed, "kv", layer, req)
    if torch.device(device).type == "cpu" and not _FORCE_TORCH_GEN:
        n = n_pos * per_pos
        out = torch.empty(n, dtype=dtype)
        f = _host_gen().gen_kv16 if dtype == torch.bfloat16 else _host_gen().gen_kv32
        assert dtype in (torch.bfloat16, torch.float32)
        f(key[0], key[1], start_pos * per_pos, n, out.data_ptr())
        v = out.view(n_pos, 2, n_kv, hd)
        return v[:, 0], v[:, 1]
    h = hashed_u32(key, start_pos * per_pos, n_pos * per_pos, device)
    k8 = (h >> 24).to(torch.float32)
    v = ((k8 * 2.0 - 255.0) * (1.0 / 128.0)).to(dtype).view(n_pos, 2, n_kv, hd)
    return v[:, 0], v[:, 1]


# --------------------------------------------------------------------------------------
# KV page placement (the documented page layout; used to place inputs and read pages)
# --------------------------------------------------------------------------------------
def k_page_index(hd: int) -> np.ndarray:
    """[16][hd] -> flat position inside a K page:
    (((e/32)*2 + (s/4)%2)*4 + (e%32)/8)*64 + ((s/8)*4 + s%4)*8 + e%8."""
    s = np.arange(PAGE)[:, None]
    e = np.arange(hd)[None, :]
    return (((e // 32) * 2 + (s // 4) % 2) * 4 + (e % 32) // 8) * 64 + ((s // 8) * 4 + s % 4) * 8 + e % 8


def v_page_index(hd: int) -> np.ndarray:
    """[16][hd] -> flat position inside a V page: ((e/16)*2 + s/8)*128 + (e%16)*8 + s%8."""
    s = np.arange(PAGE)[:, None]
    e = np.arange(hd)[None, :]
    return ((e // 16) * 2 + s // 8) * 128 + (e % 16) * 8 + s % 8


def pages_from_slots(x, which: str):
    """x [..., 16, hd] (slot-major) -> [..., 16*hd] pages in the K or V page layout."""
    hd = x.shape[-1]
    idx = (k_page_index if which == "k" else v_page_index)(hd).reshape(-1)
    if isinstance(x, torch.Tensor):
        out = torch.empty(*x.shape[:-2], PAGE * hd, dtype=x.dtype, device=x.device)
        out[..., torch.as_tensor(idx, device=x.device)] = x.reshape(*x.shape[:-2], -1)
        return out
    out = np.empty(x.shape[:-2] + (PAGE * hd,), dtype=x.dtype)
    out[..., idx] = x.reshape(x.shape[:-2] + (-1,))
    return out


def slots_from_pages(p, which: str, hd: int):
    """Inverse of pages_from_slots: [..., 16*hd] -> [..., 16, hd]."""
    idx = (k_page_index if which == "k" else v_page_index)(hd)
    if isinstance(p, torch.Tensor):
        return p[..., torch.as_tensor(idx, device=p.device)]
    return p[..., idx]


def fill_kv_pool(k_pool: torch.Tensor, v_pool: torch.Tensor, mix: "Mix", page_table: np.ndarray,
                 requests=None, req_keys=None):
    """Place the synthetic cached context of the given requests (default: all) into pools
    [n_layers][n_blocks][n_kv][16 * head_dim] on any device, through the page table.
    req_keys[r] (default the request index) keys request r's generated values."""
    s = mix.shape
    dev = k_pool.device
    dt = k_pool.dtype
    kidx = torch.as_tensor(k_page_index(s.head_dim), device=dev)
    vidx = torch.as_tensor(v_page_index(s.head_dim), device=dev)
    heads = torch.arange(s.n_kv_heads, device=dev)[None, :, None]
    reqs = range(mix.B) if requests is None else requests
    for n_i, i in enumerate(reqs):
        n = int(mix.ctx_len[i])
        if n == 0:
            continue
        key = i if req_keys is None else int(req_keys[n_i])
        t = torch.arange(n, device=dev)
        blk = torch.as_tensor(page_table[n_i if requests is not None else i], device=dev)[t // PAGE][:, None, None]
        slot = t % PAGE
        for l in range(s.n_layers):
            K, V = kv_values(mix.seed, l, key, 0, n, s.n_kv_heads, s.head_dim, dev, dt)
            k_pool[l][blk, heads, kidx[slot][:, None, :]] = K
            v_pool[l][blk, heads, vidx[slot][:, None, :]] = V


# --------------------------------------------------------------------------------------
# model weights (natural layout: every linear map is [out_features][in_features])
# --------------------------------------------------------------------------------------
WEIGHT_STD = 0.02


def torch_dtype(shape: ModelShape) -> torch.dtype:
    return torch.float32 if shape.dtype == "f32" else torch.bfloat16


def layer_weight_shapes(s: ModelShape) -> dict:
    return {
        "wq": (s.n_q_heads * s.head_dim, s.d_model),
        "wk": (s.n_kv_heads * s.head_dim, s.d_model),
        "wv": (s.n_kv_heads * s.head_dim, s.d_model),
        "wo": (s.d_model, s.n_q_heads * s.head_dim),
        "w_gate": (s.d_ff, s.d_model),
        "w_up": (s.d_ff, s.d_model),
        "w_down": (s.d_model, s.d_ff),
    }


def layer_weights(s: ModelShape, layer: int, seed: int = MASTER_SEED, device="cpu") -> dict:
    """One decoder layer's weights.  Norm gains are 1."""
    dt = torch_dtype(s)
    w = {k: normal_tensor(seed, f"L{layer}.{k}", shp, WEIGHT_STD, dt, device)
         for k, shp in layer_weight_shapes(s).items()}
    w["attn_norm"] = torch.ones(s.d_model, dtype=dt, device=device)
    w["mlp_norm"] = torch.ones(s.d_model, dtype=dt, device=device)
    return w


def global_weights(s: ModelShape, seed: int = MASTER_SEED, device="cpu") -> dict:
    dt = torch_dtype(s)
    return {
        "embed": normal_tensor(seed, "embed", (s.vocab, s.d_model), WEIGHT_STD, dt, device),
        "lm_head": normal_tensor(seed, "lm_head", (s.vocab, s.d_model), WEIGHT_STD, dt, device),
        "final_norm": torch.ones(s.d_model, dtype=dt, device=device),
    }


# --------------------------------------------------------------------------------------
# request mixes
# --------------------------------------------------------------------------------------
@dataclass
class Mix:
    config: str
    shape: ModelShape
    ctx_len: np.ndarray        # int32 [B]
    gamma: np.ndarray          # int32 [B]
    req_id: np.ndarray         # uint32 [B]
    t_draft: np.ndarray        # float64 [B] draft temperature for the q fixture
    sigma: np.ndarray          # float64 [B] draft noise scale for the q fixture
    kv_source: str             # "prefill" (real context tokens) or "synthetic"
    seed: int = MASTER_SEED
    extra: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return int(self.ctx_len.shape[0])

    @property
    def rows(self) -> np.ndarray:
        return self.gamma.astype(np.int64) + 1

    @property
    def M(self) -> int:
        return int(self.rows.sum())


CONFIG_IDS = {"tiny": 1, "8b_b32": 2, "8b_b256": 3, "8b_dyn128": 4, "70b_b64": 5}


def _rng(seed: int, cfg: int | str, tag: int, *more) -> np.random.Generator:
    cid = CONFIG_IDS.get(cfg, cfg) if isinstance(cfg, str) else cfg
    if isinstance(cid, str):
        cid = zlib.crc32(cid.encode())
    return np.random.default_rng([seed, cid, tag, *more])


def _log_uniform_int(rng, lo, hi, n):
    x = np.exp(rng.uniform(np.log(lo), np.log(hi), size=n))
    return np.clip(np.rint(x), lo, hi).astype(np.int32)


def make_mix(config: str, seed: int = MASTER_SEED, B: int | None = None) -> Mix:
    """Request mix of one named workload (B may be overridden for sweeps)."""
    r = _rng(seed, config, 3)
    if config == "tiny":
        n = B or 4
        ctx = r.integers(32, 128, size=n, endpoint=True).astype(np.int32)
        gam = r.integers(1, 4, size=n, endpoint=True).astype(np.int32)
        t = np.ones(n)
        sg = np.ones(n)
        return Mix(config, TINY, ctx, gam, np.arange(n, dtype=np.uint32), t, sg, "prefill", seed)
    if config == "8b_b32":
        n = B or 32
        ctx = r.integers(512, 2048, size=n, endpoint=True).astype(np.int32)
        gam = r.integers(1, 8, size=n, endpoint=True).astype(np.int32)
        shape = LLAMA3_8B
    elif config == "8b_b256":
        n = B or 256
        ctx = _log_uniform_int(r, 1024, 8192, n)
        gam = r.integers(2, 6, size=n, endpoint=True).astype(np.int32)
        shape = LLAMA3_8B
    elif config == "8b_dyn128":
        n = B or 128
        ctx = _log_uniform_int(r, 256, 32768, n)
        plain = r.random(n) < 0.25
        geo = np.minimum(r.geometric(1.0 / 3.0, size=n), 16)
        gam = np.where(plain, 0, geo).astype(np.int32)
        shape = LLAMA3_8B
    elif config == "70b_b64":
        n = B or 64
        ctx = r.integers(1024, 4096, size=n, endpoint=True).astype(np.int32)
        gam = r.integers(1, 8, size=n, endpoint=True).astype(np.int32)
        shape = LLAMA3_70B
    else:
        raise KeyError(config)
    t = r.uniform(0.8, 1.2, size=n)
    sg = r.uniform(0.2, 2.0, size=n) if config == "8b_dyn128" else np.full(n, 0.5)
    return Mix(config, shape, ctx, gam, np.arange(n, dtype=np.uint32), t, sg, "synthetic", seed)


def custom_mix(shape: ModelShape, ctx_len, gamma, seed: int = MASTER_SEED, name="custom",
               kv_source="synthetic", t_draft=1.0, sigma=0.5) -> Mix:
    ctx = np.asarray(ctx_len, dtype=np.int32)
    gam = np.asarray(gamma, dtype=np.int32)
    n = ctx.shape[0]
    return Mix(name, shape, ctx, gam, np.arange(n, dtype=np.uint32), np.full(n, float(t_draft)),
               np.full(n, float(sigma)), kv_source, seed)


# --------------------------------------------------------------------------------------
# page tables, tokens, noise
# --------------------------------------------------------------------------------------
def page_table(mix: Mix, spare_blocks: int = 3, extra_pages: int = 0):
    """Scattered block ids: request i owns ceil((ctx+gamma+1)/16)+extra_pages pages drawn
    from a seeded random permutation of the pool.  Returns (table int32 [B][stride], n_blocks).
    Unused table entries are -1."""
    need = (mix.ctx_len.astype(np.int64) + mix.gamma + 1 + PAGE - 1) // PAGE + extra_pages
    n_blocks = int(need.sum()) + spare_blocks
    perm = _rng(mix.seed, mix.config, 7).permutation(n_blocks).astype(np.int32)
    stride = int(need.max())
    tab = np.full((mix.B, stride), -1, dtype=np.int32)
    o = 0
    for i in range(mix.B):
        tab[i, :need[i]] = perm[o:o + need[i]]
        o += need[i]
    return tab, n_blocks


def context_tokens(mix: Mix, req: int) -> np.ndarray:
    """Random context token ids of one request (used when the context is prefilled)."""
    r = _rng(mix.seed, mix.config, 4, req)
    return r.integers(0, mix.shape.vocab, size=int(mix.ctx_len[req])).astype(np.int32)


def root_tokens(mix: Mix) -> np.ndarray:
    r = _rng(mix.seed, mix.config, 4, 1 << 20)
    return r.integers(0, mix.shape.vocab, size=mix.B).astype(np.int32)


def draft_noise(mix: Mix, req: int, j: int) -> np.ndarray:
    """Standard-normal noise vector [V] (float64) for the draft of request req, position j."""
    return _rng(mix.seed, mix.config, 5, req, j).standard_normal(mix.shape.vocab)


def draft_uniform(mix: Mix, req: int, j: int) -> float:
    """Uniform draw in [0, 1) used to sample the draft token of request req, position j."""
    return float(_rng(mix.seed, mix.config, 8, req, j).random())


def verify_seed(mix: Mix) -> int:
    """The rng_seed handed to the verification step."""
    cid = CONFIG_IDS.get(mix.config, 0)
    return ((mix.seed << 32) | (cid << 8) | 6) & ((1 << 64) - 1)


def random_logits(seed: int, rows: int, vocab: int, scale: float = 1.3, tag: str = "logits") -> np.ndarray:
    """Seeded fp32 logits [rows][vocab] ~ N(0, scale^2), for sampler-only workloads."""
    r = np.random.default_rng([seed, zlib.crc32(tag.encode()), rows, vocab])
    return (r.standard_normal((rows, vocab)) * scale).astype(np.float32)


def random_uniforms(seed: int, n: int, tag: str = "u") -> np.ndarray:
    r = np.random.default_rng([seed, zlib.crc32(tag.encode()), n])
    return r.random(n)
