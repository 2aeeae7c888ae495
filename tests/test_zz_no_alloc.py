"""wisp_verify_noalloc (the entry point for callers that cannot allocate) against
wisp_verify through the C ABI: two calls in a row on one GPU, the second with a smaller
batch, on the fp32 and the bf16 model.  Same kernels and plan, so the outputs (logits,
accept lengths, emitted tokens) and the KV written into the pools must be identical to
the workspace path's, bit for bit; a token id out of range is reported through the
caller's fault word and not through later clean calls."""
import numpy as np
import pytest
import torch

import paper_2601_11652_amd as W
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import Workload, gpu_model, log, pools_to_dev, to_dev

pytestmark = pytest.mark.gpu

MINI_BF16 = wi.ModelShape("mini-bf16-gqa", 2, 256, 8, 2, 64, 512, 1024, "bf16", 10000.0)


def _run_both(gm, wl):
    mix = wl.mix
    hd = mix.shape.head_dim
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(wl.pt), wl.T, mix.req_id)
    tokens = to_dev(wl.tokens)
    q = to_dev(wl.q) if wl.q.shape[0] else torch.zeros(1, dtype=torch.float32, device="cuda")
    outs = []
    for path in ("workspace", "noalloc"):
        kv = W.KVPool(*pools_to_dev(wl.pools0, hd))
        acc = torch.full((mix.B,), -7, dtype=torch.int32, device="cuda")
        out = torch.full((mix.M,), -7, dtype=torch.int32, device="cuda")
        logits = torch.full((mix.M, mix.shape.vocab), float("nan"), dtype=torch.float32, device="cuda")
        if path == "workspace":
            ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
            W.wisp_verify(gm.c, kv, desc, tokens, q, wl.seed, acc, out, logits, ws)
            W.wisp_check(ws)
        else:
            fault = torch.zeros(1, dtype=torch.int32, device="cuda")
            W.wisp_verify_noalloc(gm.c, kv, desc, tokens, q, wl.seed, acc, out, logits, fault)
            torch.cuda.synchronize()
            assert int(fault.item()) == 0
        torch.cuda.synchronize()
        outs.append((acc.cpu().numpy(), out.cpu().numpy(), logits.cpu().numpy(), kv.k.cpu(), kv.v.cpu()))
    return outs


@pytest.mark.parametrize("shape", [wi.TINY, MINI_BF16], ids=["fp32", "bf16"])
def test_noalloc_matches_the_workspace_path_twice(shape):
    gm = gpu_model(shape)
    model = fx.host_model(shape)
    # a batch, then a smaller one: the shared scratch keeps the first call's contents
    for name, ctx, gamma in (("first", [37, 0, 90, 15, 120, 3], [4, 16, 2, 0, 7, 1]), ("second", [50, 8], [3, 1])):
        mix = wi.custom_mix(shape, ctx, gamma, kv_source="prefill", name=f"noalloc-{name}", t_draft=1.0, sigma=0.5)
        log(f"{shape.name} {name}: ctx={ctx} gamma={gamma} (M = {mix.M})")
        (a1, o1, l1, k1, v1), (a2, o2, l2, k2, v2) = _run_both(gm, Workload(mix, model))
        np.testing.assert_array_equal(a1, a2)
        np.testing.assert_array_equal(o1, o2)
        np.testing.assert_array_equal(l1, l2)
        assert torch.equal(k1, k2) and torch.equal(v1, v2)


def test_noalloc_reports_faults_in_the_callers_word():
    shape = wi.TINY
    mix = wi.custom_mix(shape, [20, 40], [2, 3], name="noalloc-fault")
    pt_np, nb = wi.page_table(mix)
    gm = gpu_model(shape)
    kv = W.KVPool.zeros(shape.n_layers, nb, shape.n_kv_heads, shape.head_dim, torch.float32)
    desc = W.BatchDesc(mix.ctx_len, mix.gamma, to_dev(pt_np), 1.0)
    q = torch.full((int(mix.gamma.sum()), shape.vocab), 1.0 / shape.vocab, device="cuda")
    acc = torch.empty(mix.B, dtype=torch.int32, device="cuda")
    out = torch.empty(mix.M, dtype=torch.int32, device="cuda")
    logits = torch.empty(mix.M, shape.vocab, device="cuda")
    bad = torch.zeros(mix.M, dtype=torch.int32, device="cuda")
    bad[2] = shape.vocab
    good = torch.zeros(mix.M, dtype=torch.int32, device="cuda")
    fault = torch.zeros(1, dtype=torch.int32, device="cuda")
    W.wisp_verify_noalloc(gm.c, kv, desc, bad, q, 1, acc, out, logits, fault)
    W.wisp_verify_noalloc(gm.c, kv, desc, good, q, 2, acc, out, logits, fault)
    torch.cuda.synchronize()
    assert int(fault.item()) == 1            # the token-id bit, kept across the clean call
    fault.zero_()
    W.wisp_verify_noalloc(gm.c, kv, desc, good, q, 3, acc, out, logits, fault)
    torch.cuda.synchronize()
    assert int(fault.item()) == 0
