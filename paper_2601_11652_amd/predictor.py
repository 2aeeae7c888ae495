"""Draft-side rejection predictor (Sec. 3.3, Sec. 4.1, App. B): timing of its two kernels.

wisp_draft_stats reads each logits row once (4 bytes per vocabulary entry) and writes 16
bytes per row, so its roofline is HBM bandwidth; wisp_reject_predict is a 512-128-64 MLP
whose 0.3 MB of weights stay in cache, bound by its per-row latency.

The MLP's weights are the caller's (seeded in the tests and here); training it needs the
paper's draft traces, which are not part of this library.

    python -m paper_2601_11652_amd.predictor --out profiles/predictor_8b.json
"""
from __future__ import annotations

import argparse
import json
import os
import sys


from . import RejectMLP, wisp_draft_stats, wisp_reject_predict
from .records import command_line

HBM_PEAK_GBS = 8000.0


def _time(fn, reps: int = 50, warmup: int = 5) -> float:
    """Average milliseconds of fn() over reps calls, HIP events on the current stream."""
    import torch
    for _ in range(warmup):
        fn()
    s = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        fn()
    e1.record(s)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def bench_stats(rows: int, vocab: int) -> dict:
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(rows * 7 + vocab)
    x = torch.randn(rows, vocab, generator=g, device="cuda") * 2.0
    st = torch.empty(rows, 4, device="cuda")
    ms = _time(lambda: wisp_draft_stats(x, vocab, 1.0, st))
    nbytes = rows * (vocab * 4 + 16)
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"rows": rows, "vocab": vocab, "us": ms * 1e3, "bytes": nbytes, "GBs": gbs, "frac": gbs / HBM_PEAK_GBS}


def bench_mlp(rows: int, n_in: int = 5) -> dict:
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(rows)
    p = {"mean": torch.zeros(n_in, device="cuda"), "inv_std": torch.ones(n_in, device="cuda"),
         "w1": torch.randn(512, n_in, generator=g, device="cuda"), "b1": torch.zeros(512, device="cuda"),
         "w2": torch.randn(128, 512, generator=g, device="cuda") / 16, "b2": torch.zeros(128, device="cuda"),
         "w3": torch.randn(64, 128, generator=g, device="cuda") / 8, "b3": torch.zeros(64, device="cuda"),
         "w4": torch.randn(64, generator=g, device="cuda") / 8, "b4": 0.0}
    mlp = RejectMLP(p)
    f = torch.randn(rows, n_in, generator=g, device="cuda")
    out = torch.empty(rows, device="cuda")
    ms = _time(lambda: wisp_reject_predict(mlp, f, out))
    flops = rows * 2 * (512 * n_in + 512 * 128 + 128 * 64 + 64)
    return {"rows": rows, "n_in": n_in, "us": ms * 1e3, "TFLOPs": flops / (ms / 1e3) / 1e12}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default="profiles/predictor_8b.json")
    args = ap.parse_args(argv)
    import torch
    torch.cuda.set_device(0)
    rec = {"stats": [], "mlp": []}
    for rows in (1, 32, 256, 1024):
        r = bench_stats(rows, 128256)
        rec["stats"].append(r)
        print(f"draft_stats {rows:5d} x 128256: {r['us']:8.2f} us, {r['GBs']:7.0f} GB/s ({100 * r['frac']:.0f} % of HBM)",
              flush=True)
    for rows in (1, 32, 256, 1024):
        r = bench_mlp(rows)
        rec["mlp"].append(r)
        print(f"reject_mlp {rows:5d} rows: {r['us']:8.2f} us ({r['TFLOPs']:.2f} TFLOP/s)", flush=True)
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        rec["command"] = command_line("paper_2601_11652_amd.predictor", argv)
        json.dump(rec, f, indent=1)


if __name__ == "__main__":
    sys.exit(main())
