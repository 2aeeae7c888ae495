"""The C ABI on the CPU: every function declared in include/wisp.h is exported by
libwisp.so, and host-side validation returns the documented status before any launch."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wisp.h")


@pytest.fixture(scope="module")
def W():
    import paper_2601_11652_amd as W
    if not os.path.exists(W.LIB_PATH):
        from paper_2601_11652_amd import build
        build.build()
    W.load_library()
    return W


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(wisp_[a-z_0-9]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported(W):
    names = _declared()
    assert "wisp_verify" in names and "wisp_accept" in names and len(names) >= 10
    for n in names:
        assert hasattr(W.load_library(), n), n
    assert set(W.EXPORTS) == set(names)


FAKE = 0x1000  # never dereferenced: validation fails first


def _model(W, **kw):
    m = W.wisp_model(2, 256, 4, 4, 64, 1024, 1024, 1e-5, 1e4, W.WISP_F32, FAKE, FAKE, FAKE)
    arr = (C.c_void_p * 2)(FAKE, FAKE)
    for f in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down"):
        setattr(m, f, C.cast(arr, C.POINTER(C.c_void_p)))
    m._keep = arr
    for k, v in kw.items():
        setattr(m, k, v)
    return m


def _desc(W, ctx, gamma, stride=16, T=1.0, prefill=None):
    d = W.BatchDesc(ctx, gamma, None, T, prefill_len=prefill)
    d.c.kv_page_table = FAKE
    d.c.pt_stride = stride
    return d


def _verify(W, model, desc, ws_bytes=1 << 40, kv_pages=16, tokens=FAKE):
    L = W.load_library()
    kv = W.wisp_kv(FAKE, FAKE, 100, kv_pages)
    return L.wisp_verify(C.byref(model), C.byref(kv), C.byref(desc.c), tokens, FAKE, 1, FAKE, FAKE, FAKE,
                         FAKE, ws_bytes, None)


def test_validation_statuses(W):
    m = _model(W)
    assert _verify(W, m, _desc(W, [10], [17])) == W.WISP_E_INVALID
    assert "gamma" in W.wisp_last_error()
    assert _verify(W, m, _desc(W, [-1], [2])) == W.WISP_E_INVALID
    assert _verify(W, m, _desc(W, [10], [2], T=-1.0)) == W.WISP_E_INVALID
    assert _verify(W, m, _desc(W, [250], [8], stride=16)) == W.WISP_E_CAPACITY     # 259 > 256
    assert _verify(W, m, _desc(W, [10], [2]), ws_bytes=64) == W.WISP_E_WORKSPACE
    assert _verify(W, m, _desc(W, [10], [2]), kv_pages=8) == W.WISP_E_UNSUPPORTED
    assert _verify(W, m, _desc(W, [10], [2]), tokens=None) == W.WISP_E_INVALID
    assert _verify(W, _model(W, head_dim=48), _desc(W, [10], [2])) == W.WISP_E_UNSUPPORTED
    assert _verify(W, _model(W, n_kv_heads=3), _desc(W, [10], [2])) == W.WISP_E_UNSUPPORTED
    assert _verify(W, _model(W, dtype=W.WISP_BF16, head_dim=96, n_q_heads=4), _desc(W, [10], [2])) == W.WISP_E_UNSUPPORTED
    assert _verify(W, _model(W, embed=None), _desc(W, [10], [2])) == W.WISP_E_INVALID
    assert _verify(W, _model(W, d_model=8192 + 32), _desc(W, [10], [2])) == W.WISP_E_UNSUPPORTED
    assert "d_model" in W.wisp_last_error()
    assert _verify(W, _model(W, head_dim=288, n_q_heads=1, n_kv_heads=1), _desc(W, [10], [2])) == W.WISP_E_UNSUPPORTED
    assert W.wisp_workspace_size(_model(W, d_model=8192), _desc(W, [10], [2])) > 0
    L = W.load_library()
    assert L.wisp_verify(None, None, None, None, None, 0, None, None, None, None, 0, None) == W.WISP_E_INVALID
    assert _verify(W, m, _desc(W, [], [])) == W.WISP_OK          # empty batch: nothing to do


def test_prefill_validation_and_sizes(W):
    """Prompt rows in front of the root: bounds, page capacity over all new rows, and the
    workspace growing with the forwarded rows while the acceptance sizes stay per draft."""
    m = _model(W)
    assert _verify(W, m, _desc(W, [10], [2], prefill=[-1])) == W.WISP_E_INVALID
    assert "prefill_len" in W.wisp_last_error()
    assert _verify(W, m, _desc(W, [10], [2], prefill=[32769], stride=4096)) == W.WISP_E_INVALID   # > WISP_PREFILL_MAX
    # 200 cached + 50 prompt + 2 drafts + root = 253 tokens fit 16 pages; 60 prompt tokens do not
    assert _verify(W, m, _desc(W, [200], [2], prefill=[60])) == W.WISP_E_CAPACITY
    base = W.wisp_workspace_size(m, _desc(W, [200], [2]))
    with_prompt = W.wisp_workspace_size(m, _desc(W, [200], [2], prefill=[50]))
    assert with_prompt > base > 0
    assert W.wisp_workspace_size(m, _desc(W, [0], [3], prefill=[0])) == W.wisp_workspace_size(m, _desc(W, [0], [3]))
    d = _desc(W, [0, 5], [3, 1], prefill=[40, 2])
    assert d.M == 6 and d.rows == 48


def test_batch_size_limits(W):
    """Totals that the plan keeps in int: at most ROWS_MAX rows per call (prompt rows count
    only where the model runs) and at most 2^22 split-KV work items; beyond either the call
    returns WISP_E_UNSUPPORTED and the workspace sizes are 0."""
    m = _model(W)
    n = W.ROWS_MAX // (W.PREFILL_MAX + 1)                 # requests of a full prompt that fit
    fits = _desc(W, [0] * n, [0] * n, stride=4096, prefill=[W.PREFILL_MAX] * n)
    over = _desc(W, [0] * (n + 1), [0] * (n + 1), stride=4096, prefill=[W.PREFILL_MAX] * (n + 1))
    assert n * (W.PREFILL_MAX + 1) <= W.ROWS_MAX < (n + 1) * (W.PREFILL_MAX + 1)
    assert W.wisp_workspace_size(m, fits) > 0
    assert W.wisp_workspace_size(m, over) == 0
    assert W.wisp_logits_workspace_size(m, over) == 0
    assert _verify(W, m, over) == W.WISP_E_UNSUPPORTED
    assert "rows" in W.wisp_last_error()
    # the acceptance stage ignores prompt rows, and takes more rows than the model
    assert W.wisp_accept_workspace_size(over, 1024) > 0
    # exactly ROWS_MAX forwarded rows pass, one more does not (drafts only)
    B = W.ROWS_MAX // (W.GAMMA_MAX + 1)
    tail = W.ROWS_MAX - B * (W.GAMMA_MAX + 1)
    gam = [W.GAMMA_MAX] * B + ([tail - 1] if tail else [])
    assert sum(g + 1 for g in gam) == W.ROWS_MAX
    assert W.wisp_workspace_size(m, _desc(W, [0] * len(gam), gam)) > 0
    assert W.wisp_workspace_size(m, _desc(W, [0] * (len(gam) + 1), gam + [0])) == 0
    assert W.wisp_accept_workspace_size(_desc(W, [0] * (len(gam) + 1), gam + [0]), 8) > 0
    # contexts whose split-KV work list would pass 2^22 items (bf16 path: 1024 tokens
    # per item at most, one item list per kv head and 48-row group)
    mb = _model(W, dtype=W.WISP_BF16)
    ctx = 1 << 29                                         # 2^19 items per kv head
    few = _desc(W, [ctx] * 1, [0], stride=(ctx >> 4) + 1)
    many = _desc(W, [ctx] * 2, [0, 0], stride=(ctx >> 4) + 1)   # 2 x 4 heads x 2^19 = 2^22
    assert W.wisp_workspace_size(mb, few) > 0
    assert W.wisp_workspace_size(mb, many) == 0
    assert _verify(W, mb, many) == W.WISP_E_UNSUPPORTED
    assert "work items" in W.wisp_last_error()


def test_workspace_size_and_pack_validation(W):
    m = _model(W)
    assert W.wisp_workspace_size(m, _desc(W, [10], [2])) > 0
    assert W.wisp_workspace_size(m, _desc(W, [10], [17])) == 0
    small = W.wisp_workspace_size(m, _desc(W, [10], [2]))
    big = W.wisp_workspace_size(m, _desc(W, [10, 100, 7], [2, 16, 0]))
    assert big > small
    assert W.wisp_accept_workspace_size(_desc(W, [0], [3]), 0) == 0
    L = W.load_library()
    assert L.wisp_pack_linear(FAKE, FAKE, 30, 64, W.WISP_BF16, None) == W.WISP_E_UNSUPPORTED
    assert L.wisp_pack_linear(FAKE, FAKE, 32, 8, W.WISP_BF16, None) == W.WISP_E_UNSUPPORTED
    assert L.wisp_pack_linear(None, FAKE, 32, 16, W.WISP_BF16, None) == W.WISP_E_INVALID
    assert L.wisp_pack_linear(FAKE, FAKE, 32, 16, 7, None) == W.WISP_E_UNSUPPORTED
    assert L.wisp_pack_gate_up(FAKE, FAKE, FAKE, 48, 64, W.WISP_BF16, None) == W.WISP_E_UNSUPPORTED
    assert L.wisp_pack_gate_up(FAKE, FAKE, FAKE, 64, 8, W.WISP_BF16, None) == W.WISP_E_UNSUPPORTED
    assert L.wisp_pack_gate_up(FAKE, None, FAKE, 64, 64, W.WISP_BF16, None) == W.WISP_E_INVALID
    assert L.wisp_pack_gate_up(FAKE, FAKE, FAKE, 0, 64, W.WISP_BF16, None) == W.WISP_E_INVALID
    assert L.wisp_pack_gate_up(FAKE, FAKE, FAKE, 64, 64, 7, None) == W.WISP_E_UNSUPPORTED


def test_logits_in_workspace_sizes(W):
    """Without a target_logits buffer, wisp_verify keeps the logits (verification rows x
    vocab fp32, 256-byte aligned) after its own workspace and asks for both."""
    m = _model(W)
    d = _desc(W, [10, 0], [2, 4], prefill=[0, 30])
    rows = (2 + 1) + (4 + 1)                            # prompt rows produce no logits
    assert W.wisp_logits_workspace_size(m, d) == -(-rows * 1024 * 4 // 256) * 256
    base = W.wisp_workspace_size(m, d)
    L = W.load_library()
    kv = W.wisp_kv(FAKE, FAKE, 100, 16)
    args = (C.byref(m), C.byref(kv), C.byref(d.c), FAKE, FAKE, 1, FAKE, FAKE, None, FAKE)
    assert L.wisp_verify(*args, base, None) == W.WISP_E_WORKSPACE
    assert L.wisp_verify(*args, base + W.wisp_logits_workspace_size(m, d) - 1, None) == W.WISP_E_WORKSPACE


def test_binding_rejects_host_and_mistyped_tensors(W):
    """The binding hands the library device pointers only: a host tensor, a wrong element
    type or too few elements raise before any call (no GPU needed to see it)."""
    import torch
    with pytest.raises(ValueError, match="device tensor"):
        W.wisp_uniform(1, 0, 1, 0, 4, torch.zeros(4))
    with pytest.raises(ValueError, match="device tensor"):
        W.wisp_check(torch.zeros(256, dtype=torch.uint8))
    desc = W.BatchDesc([10], [2], torch.zeros((1, 4), dtype=torch.int32))
    m = _model(W)
    kv = W.KVPool(torch.zeros((2, 4, 4, 16 * 64)), torch.zeros((2, 4, 4, 16 * 64)))
    with pytest.raises(ValueError, match="page_table"):
        W.wisp_verify(m, kv, desc, None, None, 1, None, None, None, torch.zeros(256, dtype=torch.uint8))
    with pytest.raises(ValueError, match="device tensor"):
        W.wisp_accept(desc, 8, torch.zeros((3, 8)), torch.zeros(3, dtype=torch.int32), torch.zeros((2, 8)), 1,
                      torch.zeros(1, dtype=torch.int32), torch.zeros(3, dtype=torch.int32),
                      torch.zeros(256, dtype=torch.uint8))
    with pytest.raises(ValueError, match="unit column stride"):
        W.wisp_draft_stats(torch.zeros((8, 4)).t(), 8, 1.0, torch.zeros((4, 4)))


def test_gemm_plan_of_the_wide_projections(W):
    """The launch plan by row fragments (32 rows each).  The weight ring where it streams
    faster: the output projection at <= 32 rows, the LM head (>= 65536 columns) at 33-160
    rows (64-column wave tiles), small projections at <= 32 rows.  Elsewhere the LDS-staged
    tiles (variant 4) with K split into as many ranges as the work items fit one round of
    256 workgroups, at most 8 (16 at <= 32 rows), each keeping >= 8 chunks (5 ranges for 48
    tiles, 3 for 80); at <= 32 rows outputs of 16384-32768 columns on 64-row tiles in one K
    range; 129-160 rows gate/up on the 192-row tile in one K range; 225-256 rows one 256-row
    tile, 256 columns wide for the LM head; beyond 384 rows 256 x 256 tiles for every
    projection."""
    ring = {  # (M, N, K): kind
        (7, 4096, 4096): 1, (7, 1024, 256): 1, (44, 128256, 4096): 2, (150, 128256, 4096): 2,
        (44, 65536, 512): 2, (153, 65536, 512): 2,
    }
    for (M, N, K), kind in ring.items():
        assert W.gemm_plan(M, N, K)["kind"] == kind, (M, N, K, W.gemm_plan(M, N, K))
    tiles = {  # (M, N, K): (row tiles, fragments per row tile, K ranges)
        (7, 6144, 4096): (1, 1, 8), (32, 28672, 4096): (1, 2, 1), (7, 57344, 8192): (1, 1, 1), (7, 4096, 14336): (1, 1, 16),
        (7, 128256, 4096): (1, 1, 1),
        (44, 16384, 512): (1, 2, 1), (41, 6144, 4096): (1, 2, 5), (64, 4096, 4096): (1, 2, 8),
        (87, 28672, 4096): (1, 4, 1), (128, 4096, 14336): (1, 4, 8),
        (150, 6144, 4096): (1, 6, 5), (150, 4096, 14336): (1, 6, 8),
        (150, 28672, 4096): (1, 6, 1), (153, 16384, 512): (1, 6, 1),
        (171, 6144, 4096): (1, 6, 5), (171, 4096, 4096): (1, 6, 8), (171, 28672, 4096): (1, 6, 1),
        (171, 4096, 14336): (1, 6, 8), (171, 128256, 4096): (1, 6, 1),
        (343, 6144, 4096): (1, 12, 5), (343, 4096, 14336): (1, 12, 8), (343, 28672, 4096): (1, 12, 1),
        (370, 10240, 8192): (1, 12, 3), (370, 8192, 28672): (1, 12, 4),
        (476, 16384, 512): (2, 8, 2), (680, 16384, 512): (3, 8, 1), (680, 6144, 4096): (3, 8, 3),
        (680, 4096, 14336): (3, 8, 5), (512, 4096, 4096): (2, 8, 8),
        (1237, 4096, 14336): (5, 8, 3), (1237, 128256, 4096): (5, 8, 1), (1237, 6144, 4096): (5, 8, 2),
        (240, 128256, 4096): (1, 8, 1), (240, 28672, 4096): (1, 8, 1), (2108, 1024, 256): (9, 8, 2),
    }
    for (M, N, K), (rb, mt, splits) in tiles.items():
        t = W.gemm_plan(M, N, K)
        assert t["kind"] == 4 and (t["rb"], t["mt"], t["splits"]) == (rb, mt, splits), (M, N, K, t)
    with pytest.raises(W.WispError):
        W.gemm_plan(0, 1024, 256)


def test_noalloc_rejects_batches_beyond_its_static_scratch(W):
    """wisp_verify_noalloc refuses a batch whose scratch exceeds WISP_NOALLOC_SCRATCH_BYTES
    with WISP_E_WORKSPACE, before any GPU work (fake device pointers are never touched)."""
    L = W.load_library()
    m = _model(W, n_layers=2, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128, d_ff=14336,
               vocab=128256, dtype=W.WISP_BF16)
    big = _desc(W, [2048] * 256, [8] * 256, stride=160)
    kv = W.wisp_kv(FAKE, FAKE, 100000, 16)
    st = L.wisp_verify_noalloc(C.byref(m), C.byref(kv), C.byref(big.c), FAKE, FAKE, 1, FAKE, FAKE, FAKE, None, None)
    assert st == W.WISP_E_WORKSPACE, st
    assert "static" in W.wisp_last_error()
    assert W.wisp_workspace_size(m, big) > 128 << 20
