"""Edge cases of the verification step on the GPU, each against the oracle.

* an empty batch is a no-op (outputs untouched);
* requests with no cached context (ctx_len = 0: the rows attend only to each other),
  single-token contexts and the longest draft (gamma = 16) next to plain-decode requests
  (gamma = 0), on the fp32 model (1e-4 relative per row) and the bf16 model (2e-2
  max-abs);
* a batch of plain-decode requests only (no draft rows; the draft distributions may be
  NULL);
* more than 256 rows (24 requests x 17 rows = 408) and 2108 rows (124 x 17), which the
  LDS-staged tile GEMM serves in two and nine rows of 256 x 256 tiles;
* 129-256 rows, where the 32-column weight-ring GEMM runs 8 waves on two row halves: an
  odd number of 32-row fragments (150 rows: one half carries a zero fragment) and an even
  one (192 rows);
* an out-of-range block id in the page table: the kernels clamp it, write nothing through
  it, and wisp_check reports a device input error;
* a bf16 model of odd widths: d_model 96, d_ff 160, 3 query heads on 1 kv head, vocabulary
  1056.  Every projection then has a partly filled last column tile and a K shorter than
  one weight ring, and the GQA group is not a power of two; at 34 rows (weight ring) and
  612 rows (256 x 256 tiles, most columns of the narrow projections past the edge).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2601_11652_amd as W
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import (Workload, check_written, compare_decisions, gpu_model, log, pools_to_dev, rel_row_err,
                         run_gpu, to_dev)

pytestmark = pytest.mark.gpu

MINI_BF16 = wi.ModelShape("mini-bf16-gqa", 2, 256, 8, 2, 64, 512, 1024, "bf16", 10000.0)


def _check_written(wl, pools_gpu):
    mix = wl.mix
    check_written(pools_gpu, wl.pools_ref, wl.pools0, wl.pt, mix.ctx_len, mix.rows, mix.shape.head_dim,
                  mix.shape.dtype == "bf16", pools_ref32=wl.pools_ref32)


def _run_case(shape, ctx, gamma, logit_check, u_margin=1e-3):
    mix = wi.custom_mix(shape, ctx, gamma, kv_source="prefill", name="edge", t_draft=1.0, sigma=0.5)
    log(f"{shape.name}: ctx={list(ctx)} gamma={list(gamma)} (M = {mix.M})")
    model = fx.host_model(shape)
    wl = Workload(mix, model)
    gm = gpu_model(shape)
    acc, out, logits, pools = run_gpu(gm, wl)
    logit_check(logits, wl.logits_ref)
    _check_written(wl, pools)
    ref = oracle.accept(wl.logits_ref, wl.tokens, wl.q, mix.gamma, 1.0, wl.seed, req_id=mix.req_id)
    gap = float(np.abs(logits - wl.logits_ref).max())
    n_dec, mism, unflagged = compare_decisions(acc, out, ref, mix.gamma, wl.tokens, u_margin, 1e-3,
                                               residual_exempt=shape.dtype == "bf16", logit_gap=gap)
    log(f"  decisions {n_dec}, mismatches {mism}, unflagged {unflagged}")
    assert not unflagged


def _fp32_rows(logits, ref):
    err = rel_row_err(logits, ref)
    log(f"  max relative row error {err.max():.2e}")
    assert err.max() <= 1e-4


def _bf16_abs(logits, ref):
    d = np.abs(logits - ref).max()
    log(f"  max-abs logits error {d:.3e}")
    assert d <= 2e-2


def test_empty_batch_is_a_no_op():
    shape = wi.TINY
    gm = gpu_model(shape)
    kv = W.KVPool.zeros(shape.n_layers, 4, shape.n_kv_heads, shape.head_dim, torch.float32)
    pt = torch.zeros((0, 1), dtype=torch.int32, device="cuda")
    desc = W.BatchDesc(np.zeros(0, np.int32), np.zeros(0, np.int32), pt, 1.0)
    ws = W.workspace(max(256, W.wisp_workspace_size(gm.c, desc)))
    sentinel = torch.full((4,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((4,), 3.0, device="cuda")
    W.wisp_verify(gm.c, kv, desc, sentinel, None, 1, sentinel, sentinel, logits, ws)
    torch.cuda.synchronize()
    assert torch.all(sentinel == -7) and torch.all(logits == 3.0)
    assert torch.all(kv.k == 0) and torch.all(kv.v == 0)


@pytest.mark.parametrize("shape,check", [(wi.TINY, _fp32_rows), (MINI_BF16, _bf16_abs)], ids=["fp32", "bf16"])
def test_zero_and_short_contexts_with_longest_drafts(shape, check):
    _run_case(shape, [0, 0, 1, 15, 16, 33], [3, 0, 16, 16, 0, 7], check)


@pytest.mark.parametrize("shape,check", [(wi.TINY, _fp32_rows), (MINI_BF16, _bf16_abs)], ids=["fp32", "bf16"])
def test_plain_decode_batch_without_draft_rows(shape, check):
    mix = wi.custom_mix(shape, [5, 40, 0, 17], [0, 0, 0, 0], kv_source="prefill", name="decode")
    log(f"{shape.name}: plain decode, ctx={list(mix.ctx_len)}")
    model = fx.host_model(shape)
    wl = Workload(mix, model)
    gm = gpu_model(shape)
    kv = W.KVPool(*pools_to_dev(wl.pools0, shape.head_dim))
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(wl.pt), 1.0, mix.req_id)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    acc = torch.full((mix.B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((mix.M,), -7, dtype=torch.int32, device="cuda")
    logits = torch.empty(mix.M, shape.vocab, dtype=torch.float32, device="cuda")
    W.wisp_verify(gm.c, kv, desc, to_dev(wl.tokens), None, wl.seed, acc, out, logits, ws)   # NULL q
    W.wisp_check(ws)
    torch.cuda.synchronize()
    check(logits.cpu().numpy(), wl.logits_ref)
    ref = oracle.accept(wl.logits_ref, wl.tokens, wl.q, mix.gamma, 1.0, wl.seed, req_id=mix.req_id)
    assert np.all(acc.cpu().numpy() == 0)
    # gamma = 0: the one output token is a draw from p; identical unless the race is a near tie
    o = out.cpu().numpy()
    gap = float(np.abs(logits.cpu().numpy() - wl.logits_ref).max())
    for i in range(mix.B):
        if o[i] != ref.out_tokens[i]:
            assert abs(ref.race_key1[i] - ref.race_key2[i]) < 1e-3 + 4 * gap, (i, o[i], ref.out_tokens[i])


def test_more_than_256_rows_in_two_row_tiles():
    """408 rows: two rows of 256 x 256 tiles of the LDS-staged GEMM, the second mostly
    padding, with K split."""
    B = 24
    ctx = [int(c) for c in np.random.default_rng(5).integers(0, 96, size=B)]
    _run_case(MINI_BF16, ctx, [16] * B, _bf16_abs)


def test_2108_rows_in_lds_staged_tiles():
    B = 124
    ctx = [int(c) for c in np.random.default_rng(6).integers(0, 40, size=B)]
    _run_case(MINI_BF16, ctx, [16] * B, _bf16_abs)


@pytest.mark.parametrize("B,gamma", [(10, 14), (12, 15)], ids=["150rows", "192rows"])
def test_rows_around_the_ring_to_tile_switch(B, gamma):
    """150 rows (5 fragments) and 192 rows (6): the 192-row LDS-staged tile with its K split,
    partly and wholly filled (the paired-wave weight ring at these row counts is covered by
    the odd-width model at 192 rows)."""
    ctx = [int(c) for c in np.random.default_rng(B).integers(0, 80, size=B)]
    _run_case(MINI_BF16, ctx, [gamma] * B, _bf16_abs)


def test_odd_widths_bf16_at_192_rows():
    """The odd-width model at 192 rows: the projections whose K is an odd multiple of 32
    (QKV, gate/up and the LM head over d_model 96, down over d_ff 160) keep the paired-wave
    weight ring at 6 fragments; the output projection (K = 192) runs the 192-row tile on a
    partly filled column tile."""
    B = 12
    ctx = [int(c) for c in np.random.default_rng(8).integers(0, 60, size=B)]
    _run_case(ODD_BF16, ctx, [15] * B, _bf16_abs)


def test_out_of_range_block_id_is_reported():
    shape = wi.TINY
    mix = wi.custom_mix(shape, [20, 40], [2, 3], name="badblock")
    pt_np, nb = wi.page_table(mix)
    bad = pt_np.copy()
    bad[1, 1] = nb + 1000                 # a context page of request 1
    bad[0, 1] = nb                        # the page request 0's new rows are written to
    gm = gpu_model(shape)
    kv = W.KVPool.zeros(shape.n_layers, nb, shape.n_kv_heads, shape.head_dim, torch.float32)
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(bad), 1.0)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    tokens = torch.zeros(mix.M, dtype=torch.int32, device="cuda")
    q = torch.full((int(mix.gamma.sum()), shape.vocab), 1.0 / shape.vocab, device="cuda")
    acc = torch.empty(mix.B, dtype=torch.int32, device="cuda")
    out = torch.empty(mix.M, dtype=torch.int32, device="cuda")
    logits = torch.empty(mix.M, shape.vocab, device="cuda")
    W.wisp_verify(gm.c, kv, desc, tokens, q, 3, acc, out, logits, ws)
    with pytest.raises(W.WispError) as e:
        W.wisp_check(ws)
    assert "block id" in str(e.value)
    # nothing was written through the invalid ids: the pool stays finite, and the first
    # call after the report starts clean
    torch.cuda.synchronize()
    assert bool(torch.isfinite(kv.k).all()) and bool(torch.isfinite(kv.v).all())
    good = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(pt_np), 1.0)
    W.wisp_verify(gm.c, kv, good, tokens, q, 3, acc, out, logits, ws)
    W.wisp_check(ws)


def test_logits_kept_in_the_workspace():
    """target_logits = NULL: the logits live in the caller's workspace and every output is
    the same as with a logits buffer."""
    mix = wi.make_mix("tiny")
    wl = Workload(mix, fx.host_model(mix.shape))
    gm = gpu_model(mix.shape)
    acc_a, out_a, _, _ = run_gpu(gm, wl)
    kv = W.KVPool(*pools_to_dev(wl.pools0, mix.shape.head_dim))
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(wl.pt), wl.T, mix.req_id)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc) + W.wisp_logits_workspace_size(gm.c, desc))
    acc = torch.full((mix.B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((mix.M,), -7, dtype=torch.int32, device="cuda")
    W.wisp_verify(gm.c, kv, desc, to_dev(wl.tokens), to_dev(wl.q), wl.seed, acc, out, None, ws)
    W.wisp_check(ws)
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy(), acc_a) and np.array_equal(out.cpu().numpy(), out_a)


ODD_BF16 = wi.ModelShape("odd-bf16", 2, 96, 3, 1, 64, 160, 1056, "bf16", 10000.0)


def test_odd_widths_bf16():
    _run_case(ODD_BF16, [0, 37, 200, 5, 1], [16, 3, 0, 9, 1], _bf16_abs)


# fp32 head widths whose rotate-half partner is not a power-of-two lane offset away (96:
# 12 threads per head, heads straddle waves; 160: 20 threads per head)
HD96_F32 = wi.ModelShape("f32-hd96", 2, 192, 2, 1, 96, 384, 512, "f32", 10000.0)
HD160_F32 = wi.ModelShape("f32-hd160", 2, 320, 4, 2, 160, 512, 512, "f32", 10000.0)


@pytest.mark.parametrize("shape", [HD96_F32, HD160_F32], ids=["hd96", "hd160"])
def test_fp32_head_dims_off_the_power_of_two_grid(shape):
    _run_case(shape, [0, 21, 70], [4, 1, 9], _fp32_rows)


def test_fault_record_is_sticky_across_calls():
    """A token id out of range in one call is still reported after a later clean call on
    the same workspace; wisp_check clears the record."""
    shape = wi.TINY
    mix = wi.custom_mix(shape, [20, 40], [2, 3], name="sticky")
    pt_np, nb = wi.page_table(mix)
    gm = gpu_model(shape)
    kv = W.KVPool.zeros(shape.n_layers, nb, shape.n_kv_heads, shape.head_dim, torch.float32)
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(pt_np), 1.0)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    bad = torch.zeros(mix.M, dtype=torch.int32, device="cuda")
    bad[1] = shape.vocab + 5
    good = torch.zeros(mix.M, dtype=torch.int32, device="cuda")
    q = torch.full((int(mix.gamma.sum()), shape.vocab), 1.0 / shape.vocab, device="cuda")
    acc = torch.empty(mix.B, dtype=torch.int32, device="cuda")
    out = torch.empty(mix.M, dtype=torch.int32, device="cuda")
    logits = torch.empty(mix.M, shape.vocab, device="cuda")
    W.wisp_verify(gm.c, kv, desc, bad, q, 3, acc, out, logits, ws)
    W.wisp_verify(gm.c, kv, desc, good, q, 4, acc, out, logits, ws)
    with pytest.raises(W.WispError) as e:
        W.wisp_check(ws)
    assert "token id" in str(e.value)
    W.wisp_verify(gm.c, kv, desc, good, q, 5, acc, out, logits, ws)
    W.wisp_check(ws)


def test_odd_widths_bf16_at_tile_row_counts():
    """The odd-width model with 612 rows: every projection runs the LDS-staged tile kernel
    with partly filled last row and column tiles (1056 = 4 x 256 + 32 columns, 96 = 3 x 32
    inputs) and a K of 3 to 5 stages."""
    B = 36
    ctx = [int(c) for c in np.random.default_rng(7).integers(0, 60, size=B)]
    _run_case(ODD_BF16, ctx, [16] * B, _bf16_abs)

