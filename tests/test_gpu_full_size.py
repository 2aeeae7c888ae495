"""Parity at the full sizes of the benchmarked workloads, in the launch configuration the
benchmark times: the whole batch goes through ONE wisp_verify call (same batch
descriptor, page table and workspace sizing), and the oracle recomputes sampled
requests one at a time on the host.

Tolerance at depth.  The bf16 rounding contract has a noise floor of its own: two correct
implementations that sum in different orders round some values on different sides of a
bf16 boundary, and every later rounding point carries those one-ulp flips on.  The floor
is measured, not assumed: the oracle runs each sampled request twice, with fp64 sums (the
reference) and with fp32 sums in natural index order (another correct order), and
floor_Q = max |Q_fp32 - Q_fp64| for each checked quantity Q (logits; the K and V rows
written at each layer).  The GPU must then stay within

  logits: max-abs  <= max(2e-2, 2 * floor), mean-abs <= max(2e-3, 2 * mean floor);
  K / V:  per value <= max(two bf16 ulps at the scale of its head vector -- one token's
          K or V row of one kv head --, 2 * the layer's floor).

A wrong index, position, page, row or a dropped term shows up far above the floor.

Decisions.  Bit-exact on identical logits: the oracle's acceptance run on the GPU's logits
of the WHOLE batch must take the GPU's decisions, except on flagged near-ties (< 0.1 %).
End to end (each side on its own logits), the sampled requests' decisions must agree where
the observed logit gap cannot flip them (acceptance margin widened by exp(2 gap) - 1, race
margin by 4 gap, residual resample exempt).  Every request: finite logits, an accepted
prefix equal to the drafts, one valid extra token, -1 padding, no error flag.

The 8b_b32 request mix is also run at B = 3 (at most 27 rows: the QKV, gate/up and down
projections then take the 32-row GEMM tile with deep K splits, the others the weight ring).

Sampled requests (drafts from the oracle's own autoregressive fixture): the first, a
plain-decode request where the mix has one, the longest context and the largest gamma;
the other requests take model-independent seeded drafts.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2601_11652_amd as W
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import (check_decisions_on_gpu_logits, compare_decisions, gpu_model, kv_bound, log,
                         storage_to_f64, to_host_storage)

pytestmark = pytest.mark.gpu

LOGIT_ATOL = 2e-2      # bf16 logits bound, max-abs
LOGIT_MEAN = 2e-3      # bf16 logits bound, mean-abs
FLOOR_FACTOR = 2.0     # allowance over the measured fp32-vs-fp64 floor


def _samples(mix, n):
    cand = [0, int(np.argmax(mix.ctx_len)), int(np.argmax(mix.gamma))]
    zero = np.flatnonzero(mix.gamma == 0)
    if zero.size:
        cand.insert(1, int(zero[0]))
    out = []
    for c in cand:
        if c not in out:
            out.append(c)
    return out[:n]


def _oracle_request(model, mix, i, roots):
    """Request i reproduced alone on the host: its context pages, oracle drafts, the
    oracle's logits of its gamma + 1 rows and its pools after the step, with fp64 sums and
    again with fp32 sums (the floor)."""
    s = mix.shape
    sub = wi.custom_mix(s, [mix.ctx_len[i]], [mix.gamma[i]], seed=mix.seed, name=mix.config)
    sub.t_draft[:] = mix.t_draft[i]
    sub.sigma[:] = mix.sigma[i]
    n_pages = (int(mix.ctx_len[i]) + int(mix.gamma[i]) + 1 + wi.PAGE - 1) // wi.PAGE
    pt = np.arange(n_pages, dtype=np.int32)[None, :]
    before = fx.empty_pools(s, n_pages)
    fx.place_synthetic_kv(sub, before, pt, req_keys=[i])
    work = (before[0].copy(), before[1].copy())
    toks, qs, _ = fx.draft_fixture(model, sub, work, pt, roots[i:i + 1])
    del work
    after = (before[0].copy(), before[1].copy())
    logits = oracle.forward(model, after[0], after[1], pt, sub.ctx_len, sub.rows, toks[0])
    after32 = (before[0].copy(), before[1].copy())
    logits32 = oracle.forward(model, after32[0], after32[1], pt, sub.ctx_len, sub.rows, toks[0], acc32=True)
    return dict(tokens=toks[0], q=qs[0], logits=logits, before=before, after=after,
                logits32=logits32, after32=after32)


def _gather_pages(pool: torch.Tensor, blocks: np.ndarray) -> np.ndarray:
    idx = torch.as_tensor(blocks.astype(np.int64), device=pool.device)
    return to_host_storage(pool.index_select(1, idx))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("config,n_samples,B", [("8b_b32", 4, None), ("8b_b32", 3, 3), ("8b_b256", 3, None),
                                                ("8b_dyn128", 4, None), ("70b_b64", 2, None)],
                         ids=["8b_b32", "8b_b32-B3", "8b_b256", "8b_dyn128", "70b_b64"])
def test_full_size_verify(config, n_samples, B):
    mix = wi.make_mix(config, B=B)
    s = mix.shape
    samples = _samples(mix, n_samples)
    log(f"{config}: B={mix.B} M={mix.M} ctx [{mix.ctx_len.min()}, {mix.ctx_len.max()}] "
        f"gamma [{mix.gamma.min()}, {mix.gamma.max()}], sampled requests {samples}")
    roots = wi.root_tokens(mix)

    # --- oracle side: sampled requests reproduced alone --------------------------------
    model = fx.host_model(s, mix.seed)
    ref = {}
    for i in samples:
        ref[i] = _oracle_request(model, mix, i, roots)
        log(f"  oracle request {i}: ctx {mix.ctx_len[i]} gamma {mix.gamma[i]}")
    del model

    # --- the batch's drafts: oracle fixture for sampled requests, seeded noise elsewhere --
    others = [i for i in range(mix.B) if i not in ref]
    rtoks, rqs = fx.random_drafts(mix, others, roots)
    toks = [ref[i]["tokens"] if i in ref else rtoks[i] for i in range(mix.B)]
    qs = [ref[i]["q"] if i in ref else rqs[i] for i in range(mix.B)]
    tokens_np = np.concatenate(toks).astype(np.int32)
    S = int(mix.gamma.sum())
    q_np = np.concatenate(qs).astype(np.float32) if S else np.zeros((0, s.vocab), np.float32)
    off = np.concatenate([[0], np.cumsum(mix.rows)])

    # --- HIP side: the whole batch as the benchmark launches it ------------------------
    gm = gpu_model(s, mix.seed)
    pt_np, n_blocks = wi.page_table(mix)
    dt = torch.bfloat16 if s.dtype == "bf16" else torch.float32
    kv = W.KVPool.zeros(s.n_layers, n_blocks, s.n_kv_heads, s.head_dim, dt)
    wi.fill_kv_pool(kv.k, kv.v, mix, pt_np)
    pt = torch.as_tensor(pt_np, device="cuda")
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, pt, 1.0, mix.req_id)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    tokens = torch.as_tensor(tokens_np, device="cuda")
    q = torch.from_numpy(q_np).cuda() if S else torch.zeros(1, dtype=torch.float32, device="cuda")
    acc = torch.full((mix.B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((mix.M,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((mix.M, s.vocab), float("nan"), dtype=torch.float32, device="cuda")
    log(f"  HIP step on the full batch ({kv.k.numel() * 2 * kv.k.element_size() / 2**30:.1f} GiB of KV)")
    W.wisp_verify(gm.c, kv, desc, tokens, q, wi.verify_seed(mix), acc, out, logits, ws)
    W.wisp_check(ws)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(logits).all())
    acc_np = acc.cpu().numpy()
    out_np = out.cpu().numpy()

    # --- every request: valid outputs ---------------------------------------------------
    for i in range(mix.B):
        L = int(acc_np[i])
        g = int(mix.gamma[i])
        assert 0 <= L <= g, (i, L, g)
        o = out_np[off[i]:off[i + 1]]
        np.testing.assert_array_equal(o[:L], tokens_np[off[i] + 1:off[i] + 1 + L])
        assert 0 <= o[L] < s.vocab and np.all(o[L + 1:] == -1), (i, o)

    # --- decisions on identical logits: the whole batch ---------------------------------
    seed = wi.verify_seed(mix)
    logits_np = logits.cpu().numpy()
    n_id, m_id = check_decisions_on_gpu_logits(acc_np, out_np, logits_np, tokens_np, q_np, mix.gamma, 1.0, seed,
                                               req_id=mix.req_id)
    log(f"  whole batch on the GPU's own logits: {n_id} decisions, {m_id} flagged mismatches")

    # --- sampled requests against the oracle --------------------------------------------
    for i, r in ref.items():
        g = int(mix.gamma[i])
        lref = r["logits"]
        lg = logits_np[off[i]:off[i + 1]]
        d = np.abs(lg - lref)
        fl = np.abs(r["logits32"] - lref)
        log(f"  request {i}: logits max-abs error {d.max():.3e} (floor {fl.max():.3e}), mean-abs "
            f"{d.mean():.3e} (floor {fl.mean():.3e}), |ref| max {np.abs(lref).max():.2f}")
        assert d.max() <= max(LOGIT_ATOL, FLOOR_FACTOR * fl.max()), (i, d.max(), fl.max())
        assert d.mean() <= max(LOGIT_MEAN, FLOOR_FACTOR * fl.mean()), (i, d.mean(), fl.mean())

        blocks = pt_np[i, :r["before"][0].shape[1]]
        hd = s.head_dim
        for w, (pool, which) in enumerate(((kv.k, "k"), (kv.v, "v"))):
            pages = wi.slots_from_pages(_gather_pages(pool, blocks), which, hd)     # [L][pages][kv][16][hd]
            got = storage_to_f64(pages.reshape(pages.shape[:3] + (-1,)))
            exp = storage_to_f64(r["after"][w])
            exp32 = storage_to_f64(r["after32"][w])
            pre = storage_to_f64(r["before"][w])
            written = np.zeros(got.shape[1:], bool)
            wv = written.reshape(written.shape[:2] + (wi.PAGE, hd))
            for pos in range(int(mix.ctx_len[i]), int(mix.ctx_len[i]) + g + 1):
                wv[pos // wi.PAGE, :, pos % wi.PAGE, :] = True
            worst = 0.0
            ulp = kv_bound(exp, hd)
            for l in range(s.n_layers):
                e_l = np.abs(got[l][written] - exp[l][written])
                f_l = np.abs(exp32[l][written] - exp[l][written]).max()
                bound = np.maximum(ulp[l][written], FLOOR_FACTOR * f_l)
                ratio = float((e_l / bound).max())
                assert ratio <= 1.0, (i, "KV"[w], l, float(e_l.max()), f_l)
                worst = max(worst, ratio)
            np.testing.assert_array_equal(got[:, ~written], pre[:, ~written])
            log(f"  request {i}: {'KV'[w]} rows written in place, worst error / bound {worst:.2f}")

        res = oracle.accept(lref, r["tokens"], r["q"], mix.gamma[i:i + 1], 1.0, seed,
                            req_id=mix.req_id[i:i + 1])
        n_dec, mism, unflagged = compare_decisions(acc_np[i:i + 1], out_np[off[i]:off[i + 1]], res,
                                                   mix.gamma[i:i + 1], r["tokens"], 1e-3, 1e-3,
                                                   residual_exempt=True, logit_gap=float(d.max()))
        log(f"  request {i}: oracle L={int(res.accept_len[0])} gpu L={int(acc_np[i])}, end-to-end "
            f"mismatches {mism}")
        assert not unflagged, (i, unflagged)
    del gm, kv, logits, ws
    torch.cuda.empty_cache()
