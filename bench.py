#!/usr/bin/env python3
"""Benchmark of the batched speculative-verification step (WISP, Sec. 4.5) on one MI355X.

Workload (default): Llama-3-8B-shaped random-init model in bf16 (32 layers, d 4096,
32 q / 8 kv heads x 128, SwiGLU 14336, vocab 128256), B = 32 requests with cached
contexts U[512, 2048] in 16-token pages and gamma U{1..8} drafts, draft distributions
q = softmax(logits / T + N(0, 0.5)) with T ~ U[0.8, 1.2] per request.

One step = one wisp_verify call: forward of all sum(gamma+1) rows over the paged KV plus
acceptance.  Inputs are resident in HBM before timing; the call is idempotent, so the
same batch is verified W + K times, each time with its own acceptance seed.  Metric:
committed (accepted + extra) tokens per second, sum(L_i + 1) averaged over the K timed
steps' draws / step time, with the step latency alongside.

Prints ONE JSON line.  Also reports the median and p90 step time, the whole step against
its roofline lower bound (each kernel class's algorithmic bytes or flops at the HBM or
MFMA peak), the dominant kernel class against its roofline (algorithmic bytes per launch
over the HIP-event-timed average launch) and the CPU oracle timed on a bounded sample of
the same batch, on its exact inputs.  The same line carries the other workloads of the
curve (`configs`: 8b_b256, 8b_dyn128, 70b_b64 by default) with their step times, rates,
lower bounds and per-class rooflines.  The parent process touches no GPU: each workload
is measured by a child process of its own (`--worker`), which is also the form to run
under a profiler.  `--sweep 1,2,4,...` prints the batch-size curve instead.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# timing classes of the library's profiling hook (include/wisp.h) and the kernels they cover
KERNEL_CLASSES = ((0, "gemm_ring1"), (1, "gemm_ring2"), (2, "gemm_tiled"), (3, "attention"),
                  (4, "attention_combine"), (5, "rows"), (6, "sampler"), (7, "gemm_tile"))
KERNEL_NAMES = {"gemm_ring1": "gemm_ring_kernel<2, 4, MT/2, 1, 8, 2> (M > 128) / <1, 4, MT, 1, 8, 1>", "gemm_ring2": "gemm_ring_kernel<1, 4, MT, 2, 4, 2>",
                "gemm_tiled": "gemm_f32_kernel", "attention": "attn_bf16_kernel",
                "attention_combine": "attn_combine_kernel", "rows": "row kernels", "sampler": "sampler kernels",
                "gemm_tile": "gemm_tile_kernel (LDS-staged output tiles)"}
# algorithmic bytes behind every GB/s figure (the library's profiling hook counts these)
BYTES_DEFINITION = ("GEMM classes: bf16 weights read once (2 N K per projection); attention: the K and V "
                    "bytes of every cached and new token per kv head; sampler: two fp32 passes over the "
                    "logits plus one row per request")
EXTRA_CONFIGS = "8b_b256,8b_dyn128,70b_b64"
BF16_PEAK_TFLOPS = 2516.6
FP32_PEAK_TFLOPS = 157.3


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def gpu_draft_fixture(W, gm, kv, mix, pt, roots):
    """Draft tokens and q rows for the timed batch: q_j = softmax(l_{j-1} / T_i + sigma_i eps)
    from the target's own row j-1 (gamma = 0 verification calls), y_j ~ q_j."""
    import numpy as np
    import torch
    s = mix.shape
    V = s.vocab
    gen = torch.Generator(device="cuda")
    gen.manual_seed(mix.seed * 7 + 5)
    toks = {i: [int(roots[i])] for i in range(mix.B)}
    qs = {i: [] for i in range(mix.B)}
    for j in range(1, int(mix.gamma.max()) + 1):
        act = [i for i in range(mix.B) if mix.gamma[i] >= j]
        a = torch.as_tensor(act, device="cuda")
        ptj = pt.index_select(0, a).contiguous()
        desc = W.BatchDesc(mix.ctx_len[act] + j - 1, np.zeros(len(act), np.int32), ptj, 1.0, mix.req_id[act])
        ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
        tk = torch.as_tensor([toks[i][j - 1] for i in act], dtype=torch.int32, device="cuda")
        logits = torch.empty(len(act), V, dtype=torch.float32, device="cuda")
        acc = torch.empty(len(act), dtype=torch.int32, device="cuda")
        out = torch.empty(len(act), dtype=torch.int32, device="cuda")
        W.wisp_verify(gm.c, kv, desc, tk, None, 12345 + j, acc, out, logits, ws)
        T = torch.as_tensor(mix.t_draft[act], dtype=torch.float32, device="cuda")[:, None]
        sg = torch.as_tensor(mix.sigma[act], dtype=torch.float32, device="cuda")[:, None]
        z = logits / T + sg * torch.randn(logits.shape, generator=gen, device="cuda")
        q = torch.softmax(z, dim=-1)
        y = torch.multinomial(q, 1, generator=gen)[:, 0].cpu().numpy()
        for r, i in enumerate(act):
            toks[i].append(int(y[r]))
            qs[i].append(q[r])
    tokens = torch.as_tensor(np.concatenate([toks[i] for i in range(mix.B)]), dtype=torch.int32, device="cuda")
    qrows = [r for i in range(mix.B) for r in qs[i]]
    q = torch.stack(qrows).contiguous() if qrows else torch.zeros(1, V, device="cuda")
    return tokens, q


def traffic_from_counters(kernel_key: str):
    """HBM bytes per launch from committed counter runs, if they were taken on the current
    kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", f"{kernel_key}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
        return None
    return rec.get("bytes_per_launch")


def host_info() -> dict:
    """CPU model, sockets, physical cores and logical CPUs of this host (from /proc/cpuinfo),
    and the OpenMP thread setting the oracle runs with."""
    model, phys = None, set()
    pid = cid = None
    try:
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k, v = k.strip(), v.strip()
            if k == "model name" and model is None:
                model = v
            elif k == "physical id":
                pid = v
            elif k == "core id":
                cid = v
            elif not k and pid is not None:
                phys.add((pid, cid))
                pid = cid = None
        if pid is not None:
            phys.add((pid, cid))
    except OSError:
        pass
    return {"cpu": model, "sockets": len({p for p, _ in phys}) or None, "physical_cores": len(phys) or None,
            "logical_cpus": os.cpu_count(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(mix, order, inputs, min_seconds: float = 10.0):
    """The CPU oracle on a bounded sample of the timed batch, on its exact inputs: for the
    requests in the given order, the same weights, the same context KV (regenerated on the
    host by the same integer-exact generator, bit for bit), the timed batch's own tokens and
    draft rows q (copied from the device) and the first timed step's seed, until at least
    min_seconds of oracle time are spent.  Times the oracle's verification of each sampled
    request: the forward of its gamma+1 rows plus acceptance; the rate is the sample's
    committed tokens over that time."""
    import numpy as np
    import oracle
    import wisp_inputs as wi
    from oracle import fixtures as fx
    s = mix.shape
    t0 = time.time()
    model = fx.host_model(s, mix.seed)
    log(f"cpu baseline: host weights generated in {time.time() - t0:.1f} s")
    off = np.concatenate([[0], np.cumsum(mix.rows)])
    doff = np.concatenate([[0], np.cumsum(mix.gamma)])
    dt = 0.0
    committed = 0
    done = []
    for i in order:
        i = int(i)
        sub = wi.custom_mix(s, [mix.ctx_len[i]], [mix.gamma[i]], seed=mix.seed, name=mix.config)
        n_pages = (int(mix.ctx_len[i]) + int(mix.gamma[i]) + 1 + 15) // 16
        pt = np.arange(n_pages, dtype=np.int32)[None, :]
        pools = fx.empty_pools(s, n_pages)
        fx.place_synthetic_kv(sub, pools, pt, req_keys=[i])
        toks = inputs["tokens"][off[i]:off[i + 1]]
        q = inputs["q"][doff[i]:doff[i + 1]]
        t1 = time.time()
        logits = oracle.forward(model, pools[0], pools[1], pt, sub.ctx_len, sub.rows, toks)
        res = oracle.accept(logits, toks, q, sub.gamma, 1.0, inputs["seed"], req_id=mix.req_id[i:i + 1])
        dt += time.time() - t1
        committed += int(res.accept_len[0]) + 1
        done.append(i)
        log(f"cpu baseline: request {i} (ctx {int(mix.ctx_len[i])}, gamma {int(mix.gamma[i])}), "
            f"{dt:.1f} s of oracle time so far")
        if dt >= min_seconds:
            break
    host = host_info()
    threads = int(host["omp_num_threads"] or os.cpu_count() or 1)
    ctx = [int(mix.ctx_len[i]) for i in done]
    gam = [int(mix.gamma[i]) for i in done]
    return {"value": committed / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"{len(done)} requests of the timed {mix.config} batch around its median context "
                       f"(ctx {min(ctx)}-{max(ctx)}, gamma {min(gam)}-{max(gam)}) on the timed step's exact "
                       f"inputs (tokens, draft rows q, context KV, seed): forward of their gamma+1 rows through "
                       f"all {s.n_layers} layers plus acceptance, {committed} committed tokens in {dt:.2f} s of "
                       f"oracle time on {threads} OpenMP threads"),
            "host": host}


def measure_workload(W, wi, gm, mix, steps: int, warmup: int, profile: bool = True, keep_inputs: bool = False):
    """Fill the KV pool and draft fixture of `mix`, then time `steps` verification steps
    (after `warmup` untimed ones) back to back on the current stream.  Returns the step
    figures and, with `profile`, the per-kernel-class durations."""
    import ctypes as C
    import numpy as np
    import torch
    s = mix.shape
    pt_np, n_blocks = wi.page_table(mix)
    dt = torch.bfloat16 if s.dtype == "bf16" else torch.float32
    kv = W.KVPool.zeros(s.n_layers, n_blocks, s.n_kv_heads, s.head_dim, dt)
    t0 = time.time()
    wi.fill_kv_pool(kv.k, kv.v, mix, pt_np)
    torch.cuda.synchronize()
    log(f"B = {mix.B}: KV pool {kv.k.numel() * 2 * kv.k.element_size() / 2**30:.2f} GiB filled in {time.time() - t0:.1f} s")
    pt = torch.as_tensor(pt_np, device="cuda")
    roots = wi.root_tokens(mix)
    tokens, q = gpu_draft_fixture(W, gm, kv, mix, pt, roots)

    desc = W.BatchDesc(mix.ctx_len, mix.gamma, pt, 1.0, mix.req_id)
    ws = W.workspace(W.wisp_workspace_size(gm.c, desc))
    M = mix.M
    # every timed step draws its own acceptance randomness (seed + step) into its own row of
    # accepted lengths, so the committed-token count is a mean over the K steps' draws
    accs = torch.empty((warmup + steps, mix.B), dtype=torch.int32, device="cuda")
    out = torch.empty(M, dtype=torch.int32, device="cuda")
    logits = torch.empty(M, s.vocab, dtype=torch.float32, device="cuda")
    seed = wi.verify_seed(mix)

    def step(i=0):
        W.wisp_verify(gm.c, kv, desc, tokens, q, seed + i, accs[i], out, logits, ws)

    for i in range(warmup):
        step(i)
    W.wisp_check(ws)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for k, i in enumerate(range(warmup, warmup + steps)):
        step(i)
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    W.wisp_check(ws)        # device-side input faults of the timed steps
    ms_step = ev[0].elapsed_time(ev[-1]) / steps
    per_step = np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(steps)])
    log(f"B = {mix.B}: {steps} steps: {ms_step:.3f} ms/step (events), {wall / steps * 1e3:.3f} ms/step (wall)")
    L = accs[warmup:].cpu().numpy().astype(np.int64)
    committed = float((L + 1).sum()) / steps
    res = {"ms_per_step": ms_step, "ms_p50": float(np.median(per_step)), "ms_p90": float(np.percentile(per_step, 90)),
           "committed": committed, "accepted": float(L.sum()) / steps, "M": M}
    if keep_inputs:
        res["inputs"] = {"tokens": tokens.cpu().numpy(), "q": q.cpu().numpy(), "seed": seed + warmup}

    classes = {}
    if profile:
        # per-kernel-class durations: HIP events stamped by each dispatch on the library's stream
        prof_steps = max(3, min(10, steps))
        W.lib.wisp_profile_enable(1)
        W.lib.wisp_profile_reset()
        for _ in range(prof_steps):
            step()
        torch.cuda.synchronize()
        for kind, name in KERNEL_CLASSES:
            ms, n, by, fl = C.c_double(), C.c_int64(), C.c_double(), C.c_double()
            W.lib.wisp_profile_read(kind, C.byref(ms), C.byref(n), C.byref(by), C.byref(fl))
            if n.value:
                classes[name] = {"ms_per_step": ms.value / prof_steps, "launches_per_step": n.value / prof_steps,
                                 "avg_launch_us": ms.value / n.value * 1e3, "bytes_per_launch": by.value / n.value,
                                 "flops_per_launch": fl.value / n.value,
                                 "achieved_GBs": by.value / ms.value / 1e6 if ms.value else 0.0,
                                 "achieved_TFLOPs": fl.value / ms.value / 1e9 if ms.value else 0.0}
        W.lib.wisp_profile_enable(0)
        W.wisp_check(ws)
    res["classes"] = classes
    del kv, ws, logits, q
    return res


def step_lower_bound(classes: dict) -> dict:
    """Roofline lower bound of a whole step: each kernel class's algorithmic bytes at the HBM
    peak or its flops at the bf16 MFMA peak, whichever is longer, summed over the classes."""
    lb = 0.0
    by = 0.0
    for c in classes.values():
        b = c["bytes_per_launch"] * c["launches_per_step"]
        f = c["flops_per_launch"] * c["launches_per_step"]
        by += b
        lb += max(b / (HBM_PEAK_GBS * 1e9), f / (BF16_PEAK_TFLOPS * 1e12))
    return {"lower_bound_ms": lb * 1e3, "bytes_per_step": by}


def class_roofline(name: str, c: dict, M: int) -> dict | None:
    """One kernel class against its roofline: GEMMs at large row counts (>= 630, twice the
    MFMA ridge) against the bf16 MFMA peak, everything with algorithmic bytes against the
    HBM peak; overhead classes (no algorithmic bytes) have none."""
    if name.startswith("gemm") and M >= 630 and c["flops_per_launch"] > 0:
        r = {"bound": "mfma", "achieved": c["achieved_TFLOPs"], "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    elif c["bytes_per_launch"] > 0:
        r = {"bound": "hbm", "achieved": c["achieved_GBs"], "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        return None
    r["frac"] = r["achieved"] / r["peak"]
    return r


def config_summary(mix, r) -> dict:
    """Step time, committed tokens/s, step lower bound and per-class rooflines of one
    measured workload."""
    lb = step_lower_bound(r["classes"])
    classes = {}
    for name, c in r["classes"].items():
        classes[name] = {"ms_per_step": c["ms_per_step"], "launches_per_step": c["launches_per_step"],
                         "avg_launch_us": c["avg_launch_us"], "roofline": class_roofline(name, c, r["M"])}
    return {"workload": f"{mix.config}: {mix.shape.name} verification step", "B": mix.B, "rows": r["M"],
            "sum_ctx": int(mix.ctx_len.sum()), "sum_gamma": int(mix.gamma.sum()),
            "ms_per_step": r["ms_per_step"], "ms_p50": r["ms_p50"], "ms_p90": r["ms_p90"],
            "committed_tokens_per_step": r["committed"], "tokens_per_s": r["committed"] / (r["ms_per_step"] / 1e3),
            "step_lower_bound_ms": lb["lower_bound_ms"], "step_frac": lb["lower_bound_ms"] / r["ms_per_step"],
            "classes": classes}


def sweep(args, W, wi, gm):
    """The batch-size curve: the same request distributions at B = 1 .. 256, one JSON line
    per batch size (tokens/s and step latency), written to --sweep-out as well."""
    rows = []
    for B in [int(b) for b in args.sweep.split(",")]:
        mix = wi.make_mix(args.config, B=B)
        r = measure_workload(W, wi, gm, mix, args.steps, args.warmup, profile=True,
                         keep_inputs=not args.no_cpu_baseline)
        lb = step_lower_bound(r["classes"])
        row = {"B": B, "rows": r["M"], "sum_ctx": int(mix.ctx_len.sum()), "ms_per_step": r["ms_per_step"],
               "ms_p50": r["ms_p50"], "ms_p90": r["ms_p90"], "committed_tokens_per_step": r["committed"],
               "tokens_per_s": r["committed"] / (r["ms_per_step"] / 1e3),
               "accepted_drafts_per_s": r["accepted"] / (r["ms_per_step"] / 1e3),
               "step_lower_bound_ms": lb["lower_bound_ms"], "step_frac": lb["lower_bound_ms"] / r["ms_per_step"]}
        rows.append(row)
        print(json.dumps(row), flush=True)
    if args.sweep_out:
        with open(args.sweep_out, "w") as f:
            from paper_2601_11652_amd.records import command_line
            json.dump({"config": args.config, "steps": args.steps, "warmup": args.warmup, "rows": rows,
                       "command": command_line(None)}, f, indent=1)


def worker(args) -> None:
    """GPU side: one workload measured in this process; prints its record as one JSON line
    (and, with --dump-inputs, writes the timed batch's inputs for the CPU baseline)."""
    import numpy as np
    import torch
    import paper_2601_11652_amd as W
    import wisp_inputs as wi

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    mix = wi.make_mix(args.config, B=args.B)
    s = mix.shape
    t0 = time.time()
    gm = W.GpuModel(s, lambda l: wi.layer_weights(s, l, mix.seed, "cuda"), wi.global_weights(s, mix.seed, "cuda"))
    log(f"{args.config}: weights generated and packed in {time.time() - t0:.1f} s")
    if args.sweep:
        sweep(args, W, wi, gm)
        return

    r = measure_workload(W, wi, gm, mix, args.steps, args.warmup, profile=True, keep_inputs=bool(args.dump_inputs))
    if args.dump_inputs:
        inp = r.pop("inputs")
        np.savez(args.dump_inputs, tokens=inp["tokens"], q=inp["q"], seed=np.uint64(inp["seed"]))
    ms_step = r["ms_per_step"]
    committed = r["committed"]
    classes = r["classes"]
    M = mix.M
    dom = max((k for k in classes if classes[k]["bytes_per_launch"] > 0), key=lambda k: classes[k]["ms_per_step"])
    c = classes[dom]
    if dom.startswith("gemm") and M >= 630:
        roof = {"bound": "mfma", "achieved": c["achieved_TFLOPs"], "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": c["achieved_GBs"], "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["kernel"] = KERNEL_NAMES[dom]
    roof["traffic"] = traffic_from_counters(f"{dom}_{args.config}")
    roof["bytes_definition"] = BYTES_DEFINITION
    for name, cl in classes.items():
        cl["roofline"] = class_roofline(name, cl, M)
    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        log("copy calibration: 1 GiB device-to-device copy done")
    rec = config_summary(mix, r)
    rec.update({"dtype": "bf16" if s.dtype == "bf16" else "f32", "layers": s.n_layers, "vocab": s.vocab,
                "accepted_drafts_per_s": r["accepted"] / (ms_step / 1e3),
                "acceptance_rate": r["accepted"] / max(1, int(mix.gamma.sum())),
                "roofline": roof, "kernels": classes})
    print(json.dumps(rec), flush=True)


def run_worker(args, config: str, steps: int, warmup: int, dump: str | None = None) -> dict:
    """One workload in a child process of its own: device memory a process frees is not
    handed back for its own reuse on this stack, so each workload starts from a whole GPU."""
    import subprocess
    cmd = [sys.executable, os.path.abspath(__file__), "--worker", "--config", config, "--steps", str(steps),
           "--warmup", str(warmup)]
    if args.B is not None and config == args.config:
        cmd += ["--B", str(args.B)]
    if dump:
        cmd += ["--dump-inputs", dump]
    if args.copy_calibration and config == args.config:
        cmd += ["--copy-calibration"]
    p = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
    if p.returncode != 0:
        raise SystemExit(f"bench worker for {config} failed with status {p.returncode}")
    return json.loads(p.stdout.strip().splitlines()[-1])


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="8b_b32")
    ap.add_argument("--B", type=int, default=None, help="override the batch size")
    ap.add_argument("--sweep", default=None, help="comma-separated batch sizes: print the batch-size curve instead")
    ap.add_argument("--sweep-out", default=None, help="also write the curve to this JSON file")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--configs", default=EXTRA_CONFIGS,
                    help="further workloads measured after the headline one ('' for none)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM counter scaling)")
    ap.add_argument("--worker", action="store_true",
                    help="measure --config in this process and print its record (what the parent runs)")
    ap.add_argument("--dump-inputs", default=None, help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one MI355X only; --gpus {args.gpus} is not supported (requests are "
              "independent, so N GPUs run N replicas; see the design notes)", file=sys.stderr)
        sys.exit(2)
    if args.worker or args.sweep:
        worker(args)
        return

    # parent: touches no GPU itself; each workload runs in a child process
    import tempfile
    import numpy as np
    import wisp_inputs as wi
    tmp = tempfile.mkdtemp(prefix="wisp_bench_")
    dump = None if args.no_cpu_baseline else os.path.join(tmp, "inputs.npz")
    h = run_worker(args, args.config, args.steps, args.warmup, dump)
    mix = wi.make_mix(args.config, B=args.B)
    result = {
        "metric": "accepted tokens/s + verify-step latency (ms) vs batch B, 8B-shape bf16",
        "value": h["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": h["dtype"],
        "data": "synthetic (seeded random-init weights, synthetic paged context KV, drafts from the target's own logits plus noise)",
        "config": {"workload": h["workload"], "B": h["B"], "rows": h["rows"], "sum_ctx": h["sum_ctx"],
                   "sum_gamma": h["sum_gamma"], "page": 16, "layers": h["layers"], "vocab": h["vocab"]},
        "ms_p50": h["ms_p50"],
        "ms_p90": h["ms_p90"],
        "accepted_drafts_per_s": h["accepted_drafts_per_s"],
        "acceptance_rate": h["acceptance_rate"],
        "committed_tokens_per_step": h["committed_tokens_per_step"],
        "step_roofline": {"lower_bound_ms": h["step_lower_bound_ms"], "frac": h["step_frac"]},
        "roofline": h["roofline"],
        "kernels": h["kernels"],
    }
    # the other workloads of the "vs batch B" curve: step time, tokens/s, lower bound and the
    # per-class rooflines of each (fewer steps each)
    extra = [c for c in args.configs.split(",") if c and c != args.config]
    if extra:
        result["configs"] = {}
        for name in extra:
            result["configs"][name] = run_worker(args, name, min(args.steps, 8), min(args.warmup, 2))
            log(f"{name}: {result['configs'][name]['ms_per_step']:.2f} ms/step, "
                f"{result['configs'][name]['tokens_per_s']:.0f} tokens/s")
    if dump:
        # requests outward from the median context: median, next above, next below, ...
        by_ctx = np.argsort(mix.ctx_len, kind="stable")
        mid = mix.B // 2
        order = [by_ctx[mid + (k + 1) // 2 * (1 if k % 2 else -1)] for k in range(2 * mix.B)
                 if 0 <= mid + (k + 1) // 2 * (1 if k % 2 else -1) < mix.B]
        z = np.load(dump)
        inputs = {"tokens": z["tokens"], "q": z["q"], "seed": int(z["seed"])}
        try:
            result["cpu_baseline"] = cpu_baseline(mix, order, inputs)
        except MemoryError as e:   # report rather than fail the GPU measurement
            result["cpu_baseline"] = {"value": None, "error": str(e)}
        os.remove(dump)
    os.rmdir(tmp)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
