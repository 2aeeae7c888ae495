"""Verification-interference micro-benchmark (Sec. 3.3, Fig. 4) on this GPU.

Three cases, each one wisp_verify call:
  * solo A: a first-time (cold-start) verification: L_new new tokens (the uncached prompt,
    then the root, then 5 drafts) on an empty cache;
  * solo B: a follow-up verification: a cached 500-token prefix plus 5 drafts;
  * batched A+B: both requests in one call.
L_new is swept; the paper's point is that the batched call takes as long as solo A, so the
short request B inherits the long request's latency (head-of-line blocking).

Timing: 5 warm-up calls, then `runs` calls each bracketed by HIP events on the calling
stream (the call is idempotent); the median is reported.  Weights are the seeded
random-init weights of the model shape, context KV synthetic, tokens uniform random ids,
q rows uniform over the vocabulary.

Run on a GPU:  python -m paper_2601_11652_amd.interference --out profiles/interference_8b.json
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
from .records import command_line

PAGE = 16


def measure(shape, l_new_values, prefix: int = 500, drafts: int = 5, runs: int = 20, seed: int = 1, log=print):
    import torch
    from . import BatchDesc, GpuModel, KVPool, wisp_verify, wisp_workspace_size, workspace
    import wisp_inputs as wi

    torch.cuda.set_device(0)
    gm = GpuModel(shape, lambda l: wi.layer_weights(shape, l, seed, "cuda"), wi.global_weights(shape, seed, "cuda"))
    max_a = max(l_new_values)
    pages_a = (max_a + PAGE - 1) // PAGE
    pages_b = (prefix + drafts + 1 + PAGE - 1) // PAGE
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    kv = KVPool.zeros(shape.n_layers, pages_a + pages_b, shape.n_kv_heads, shape.head_dim, dt)
    # request B's cached prefix: synthetic bf16-exact values in its pages
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    kv.k.copy_((torch.randint(-255, 256, kv.k.shape, device="cuda", generator=g) | 1).to(dt) * 2.0 ** -7)
    kv.v.copy_((torch.randint(-255, 256, kv.v.shape, device="cuda", generator=g) | 1).to(dt) * 2.0 ** -7)
    stride = max(pages_a, pages_b)
    pt_a = torch.full((1, stride), -1, dtype=torch.int32)
    pt_a[0, :pages_a] = torch.arange(pages_a, dtype=torch.int32)
    pt_b = torch.full((1, stride), -1, dtype=torch.int32)
    pt_b[0, :pages_b] = torch.arange(pages_a, pages_a + pages_b, dtype=torch.int32)
    stream = torch.cuda.current_stream()
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed + 1)

    def timed(ctx, pre, gam, pt):
        ctx = np.asarray(ctx, np.int32)
        gam = np.asarray(gam, np.int32)
        pre = np.asarray(pre, np.int32)
        B = ctx.shape[0]
        desc = BatchDesc(ctx, gam, pt.cuda(), 1.0, np.arange(B, dtype=np.uint32), prefill_len=pre)
        ws = workspace(wisp_workspace_size(gm.c, desc))
        tokens = torch.randint(0, shape.vocab, (desc.rows,), dtype=torch.int32, device="cuda", generator=gen)
        q = torch.full((max(desc.S, 1), shape.vocab), 1.0 / shape.vocab, device="cuda")
        acc = torch.empty(B, dtype=torch.int32, device="cuda")
        out = torch.empty(desc.M, dtype=torch.int32, device="cuda")
        logits = torch.empty(desc.M, shape.vocab, dtype=torch.float32, device="cuda")
        for _ in range(5):
            wisp_verify(gm.c, kv, desc, tokens, q, 7, acc, out, logits, ws)
        ts = []
        for _ in range(runs):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            wisp_verify(gm.c, kv, desc, tokens, q, 7, acc, out, logits, ws)
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    solo_b = timed([prefix], [0], [drafts], pt_b)
    log(f"solo B (cached {prefix} + {drafts} drafts): {solo_b:.3f} ms")
    rows = []
    for L in l_new_values:
        pre = L - drafts - 1
        assert pre >= 0
        a = timed([0], [pre], [drafts], pt_a)
        ab = timed([0, prefix], [pre, 0], [drafts, drafts], torch.cat([pt_a, pt_b]))
        rows.append({"L_new": L, "solo_a_ms": a, "solo_b_ms": solo_b, "batched_ms": ab,
                     "b_slowdown": ab / solo_b})
        log(f"L_new {L:5d}: solo A {a:8.3f} ms | solo B {solo_b:6.3f} ms | batched A+B {ab:8.3f} ms "
            f"(B waits {ab / solo_b:5.1f}x its solo time)")
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default="profiles/interference_8b.json")
    ap.add_argument("--model", default="8b", choices=("8b", "70b"))
    ap.add_argument("--l-new", default="16,64,128,256,512,1024,2048,4096")
    args = ap.parse_args(argv)
    import wisp_inputs as wi
    shape = wi.LLAMA3_8B if args.model == "8b" else wi.LLAMA3_70B
    t0 = time.time()
    rows = measure(shape, [int(x) for x in args.l_new.split(",")], log=lambda m: print(m, flush=True))
    rec = {"model": shape.name, "prefix_b": 500, "drafts": 5,
           "protocol": "5 warm-up calls, median of 20 HIP-event-timed calls per case", "rows": rows,
           "seconds": time.time() - t0}
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        rec["command"] = command_line("paper_2601_11652_amd.interference", argv)
        json.dump(rec, f, indent=1)


if __name__ == "__main__":
    sys.exit(main())
