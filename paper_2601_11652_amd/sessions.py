"""Multi-round speculative-verification sessions over the KV page-pool manager (Sec. 4.5).

Each session is one response in progress: its committed tokens (prompt, then everything
verification commits) and, on the server, the KV of its committed prefix in pages that a
KVManager hands out.  A round of a batch of sessions is
  1. drafting, on the device side: a draft model with its own KV pool and manager proposes
     gamma tokens per session, y_{j+1} ~ q_j = softmax(l_j / T_d + sigma * eps) where l_j
     are the draft model's logits (here the target's own weights, so the acceptance rate
     is set by T_d and sigma; sigma may be drawn per token, for drafts of varying
     difficulty); its first call also catches up on committed tokens it has
     not seen (as prompt rows);
  2. verification, on the server: one wisp_verify call over the batch; a session whose
     prefix the server holds sends only its root and drafts (a follow-up), one the server
     does not hold (new, or evicted) sends its whole committed prefix as prompt rows in
     front of them (a first-time verification, Sec. 4.4);
  3. commit: the server keeps the KV of the committed prefix (ctx_len + prefill_len + 1 +
     L tokens; rollback by length), the draft model the KV of what it drafted correctly.
With `recompute`, the server keeps nothing between rounds and every round is a first-time
verification of the whole prefix (no prefix cache), the baseline of the paper's
state-efficiency argument.

    python -m paper_2601_11652_amd.sessions --out profiles/sessions_8b.json
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

from . import (PAGE, BatchDesc, KVManager, KVPool, wisp_verify,
               wisp_workspace_size, workspace)
from .records import command_line


class Sessions:
    def __init__(self, gm, shape, server_pages: int, draft_pages: int, *, recompute: bool = False,
                 pt_stride: int = 512, seed: int = 1, t_draft: float = 1.0, sigma: float = 0.5,
                 max_rows: int = 4096):
        import torch
        self.torch = torch
        self.gm, self.shape = gm, shape
        dt = torch.float32 if shape.dtype == "f32" else torch.bfloat16
        self.kv = KVPool.zeros(shape.n_layers, server_pages, shape.n_kv_heads, shape.head_dim, dt)
        self.kv_d = KVPool.zeros(shape.n_layers, draft_pages, shape.n_kv_heads, shape.head_dim, dt)
        self.sm = KVManager(server_pages)
        self.dm = KVManager(draft_pages)
        self.recompute = recompute
        self.stride = pt_stride
        self.seed = seed
        self.t_draft, self.sigma = t_draft, sigma
        self.max_rows = max_rows
        self.seq = {}
        self.gen = torch.Generator(device="cuda")
        self.gen.manual_seed(seed)

    def open(self, sid: int, prompt):
        self.seq[int(sid)] = [int(t) for t in prompt]

    def close(self, sids):
        self.sm.release(sids)
        self.dm.release(sids)
        for s in sids:
            self.seq.pop(int(s), None)

    # one wisp_verify call; returns (accept_len, out_tokens, logits) as device tensors and the
    # call's time in ms when time_it
    def _call(self, kv, ctx, gamma, prefill, table, tokens, q, rng_seed, req_id, time_it=False):
        torch = self.torch
        pt = torch.as_tensor(table, device="cuda")
        desc = BatchDesc(ctx, gamma, pt, 1.0, req_id, prefill_len=prefill)
        ws = workspace(wisp_workspace_size(self.gm.c, desc))
        tk = torch.as_tensor(np.asarray(tokens, np.int32), device="cuda")
        acc = torch.empty(desc.c.B, dtype=torch.int32, device="cuda")
        out = torch.empty(desc.M, dtype=torch.int32, device="cuda")
        logits = torch.empty(desc.M, self.shape.vocab, dtype=torch.float32, device="cuda")
        ms = None
        if time_it:
            s = torch.cuda.current_stream()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
        wisp_verify(self.gm.c, kv, desc, tk, q, rng_seed, acc, out, logits, ws)
        if time_it:
            e1.record(s)
            e1.synchronize()
            ms = e0.elapsed_time(e1)
        return acc, out, logits, ms

    def _chunks(self, rows):
        """Consecutive groups of sessions whose new rows stay within max_rows per call."""
        groups, cur, acc = [], [], 0
        for i, r in enumerate(rows):
            if cur and acc + r > self.max_rows:
                groups.append(cur)
                cur, acc = [], 0
            cur.append(i)
            acc += int(r)
        if cur:
            groups.append(cur)
        return groups

    def draft(self, sids, gammas, rnd: int):
        """Draft up to gamma_i tokens per session with the device-side model.  Returns the
        drafts (list of lists) and the q rows (fp32 [sum gamma][V], request-major)."""
        torch = self.torch
        B = len(sids)
        n = np.array([len(self.seq[s]) for s in sids], np.int64)
        g = np.asarray(gammas, np.int32)
        cached = self.dm.lookup(sids).astype(np.int64)
        drafts = [[] for _ in range(B)]
        qrows = [[] for _ in range(B)]
        req = np.asarray(sids, np.int64).astype(np.uint32)
        for grp in self._chunks(n - cached):
            gs = [sids[i] for i in grp]
            table, ev = self.dm.reserve(gs, (n[grp] + g[grp] - 1).astype(np.int32), self.stride)
            assert ev == 0, "the draft-side pool holds every session"
            for j in range(int(g[grp].max())):
                act = [k for k, i in enumerate(grp) if g[i] > j]
                if not act:
                    break
                idx = [grp[k] for k in act]
                if j == 0:
                    ctx = cached[idx]
                    pre = n[idx] - 1 - ctx
                    toks = [t for i in idx for t in self.seq[sids[i]][int(cached[i]):]]
                else:
                    ctx = n[idx] + j - 1
                    pre = np.zeros(len(idx), np.int64)
                    toks = [drafts[i][j - 1] for i in idx]
                _, _, logits, _ = self._call(self.kv_d, ctx.astype(np.int32), np.zeros(len(idx), np.int32),
                                             pre.astype(np.int32), table[act], toks, None,
                                             (self.seed << 20) + 2 * rnd + 1, req[idx])
                eps = torch.randn(logits.shape, generator=self.gen, device="cuda")
                z = logits / self.t_draft + self.sigma * eps
                q = torch.softmax(z, dim=-1)
                y = torch.multinomial(q, 1, generator=self.gen)[:, 0].tolist()
                for r, i in enumerate(idx):
                    drafts[i].append(int(y[r]))
                    qrows[i].append(q[r])
        return drafts, qrows

    def verify(self, sids, drafts, qrows, rnd: int):
        """The server's verification of one round: one wisp_verify call per chunk of
        consecutive sessions with at most max_rows new rows.  Each chunk looks its sessions
        up, reserves, runs and commits before the next chunk is formed, so a session that
        an earlier chunk's reservation evicts is sent again in full.  Returns per-session
        accepted lengths and committed tokens, the logits of the last chunk, the summed call
        time (ms) and the row counts."""
        torch = self.torch
        B = len(sids)
        n = np.array([len(self.seq[s]) for s in sids], np.int64)
        g = np.array([len(d) for d in drafts], np.int32)
        cached = np.zeros(B, np.int64)
        acc = np.zeros(B, np.int32)
        new = [None] * B
        ms_total, evicted, logits = 0.0, 0, None
        req = np.asarray(sids, np.int64).astype(np.uint32)
        i0 = 0
        while i0 < B:
            rest = sids[i0:]
            c = np.zeros(len(rest), np.int64) if self.recompute else self.sm.lookup(rest).astype(np.int64)
            rows = n[i0:] - c + g[i0:]
            if rows[0] > self.max_rows:
                raise ValueError(f"session {sids[i0]} needs {rows[0]} new rows, more than {self.max_rows}")
            k = int(np.searchsorted(np.cumsum(rows), self.max_rows, side="right"))
            grp = list(range(i0, i0 + k))
            cached[grp] = c[:k]
            pre = n[grp] - 1 - cached[grp]
            gs = [sids[i] for i in grp]
            table, ev = self.sm.reserve(gs, (n[grp] + g[grp]).astype(np.int32), self.stride)
            evicted += ev
            toks = []
            for i in grp:
                toks += self.seq[sids[i]][int(cached[i]):] + drafts[i]
            qr = [r for i in grp for r in qrows[i]]
            q = torch.stack(qr).contiguous() if qr else None
            a, out, logits, ms = self._call(self.kv, cached[grp].astype(np.int32), g[grp], pre.astype(np.int32),
                                            table, toks, q, (self.seed << 20) + 2 * rnd, req[grp], time_it=True)
            ms_total += ms
            a = a.cpu().numpy()
            out = out.cpu().numpy()
            off = np.concatenate([[0], np.cumsum(g[grp] + 1)])
            for j, i in enumerate(grp):
                acc[i] = a[j]
                new[i] = out[off[j]:off[j] + a[j] + 1].tolist()
            if self.recompute:
                self.sm.release(gs)
            else:
                self.sm.commit(gs, (n[grp] + a).astype(np.int32))
            i0 += k
        self.dm.commit(sids, (n + np.minimum(acc, g - 1)).astype(np.int32))
        for i, s in enumerate(sids):
            self.seq[s] += new[i]
        pre_all = n - 1 - cached
        return {"accept_len": acc, "committed": new, "logits": logits, "ms": ms_total, "evicted": evicted,
                "new_rows": int((pre_all + g + 1).sum()), "prompt_rows": int(pre_all.sum()), "cached": cached}

    def round(self, sids, gammas, rnd: int) -> dict:
        sids = [int(s) for s in sids]
        t0 = time.perf_counter()
        drafts, qrows = self.draft(sids, gammas, rnd)
        self.torch.cuda.synchronize()
        r = self.verify(sids, drafts, qrows, rnd)
        r["draft_s"] = time.perf_counter() - t0 - r["ms"] / 1e3
        r["drafts"] = drafts
        return r


def _prompts(vocab: int, n: int, length, seed: int):
    rng = np.random.default_rng([seed, 604])
    lens = np.broadcast_to(np.asarray(length), (n,))
    return [rng.integers(0, vocab, size=int(lens[i])).astype(np.int32) for i in range(n)]


def run(shape, gm, n_sessions: int, batch: int, rounds: int, prompt_len, gamma, *, recompute=False,
        server_pages=None, pick="all", seed: int = 1, log=print) -> dict:
    """`rounds` rounds; each serves `batch` of the `n_sessions` sessions (all of them, or a
    seeded random subset with pick="random").  Returns per-round records."""
    pl = int(np.max(prompt_len))
    per = (pl + rounds * (gamma + 1) + gamma + 1 + PAGE - 1) // PAGE + 1
    draft_pages = n_sessions * per
    sp = server_pages or n_sessions * per
    S = Sessions(gm, shape, sp, draft_pages, recompute=recompute, pt_stride=per + 1, seed=seed)
    for i, p in enumerate(_prompts(shape.vocab, n_sessions, prompt_len, seed)):
        S.open(i, p)
    rng = np.random.default_rng([seed, 17])
    recs = []
    for rnd in range(rounds):
        sids = list(range(n_sessions)) if pick == "all" else sorted(rng.choice(n_sessions, batch, replace=False))
        r = S.round(sids, [gamma] * len(sids), rnd)
        ctx_mean = float(np.mean([len(S.seq[s]) for s in sids]))
        recs.append({"round": rnd, "ms": r["ms"], "committed": int(sum(len(c) for c in r["committed"])),
                     "accepted": int(r["accept_len"].sum()), "new_rows": r["new_rows"],
                     "prompt_rows": r["prompt_rows"], "evicted": r["evicted"], "ctx_mean": ctx_mean,
                     "hits": int((r["cached"] > 0).sum())})
        if rnd % 50 == 0 or rnd == rounds - 1:
            log(f"round {rnd}: {r['ms']:.2f} ms, {recs[-1]['committed']} committed, {r['new_rows']} new rows, "
                f"{r['evicted']} evicted, mean length {ctx_mean:.0f}")
    return {"rounds": recs, "stats": S.sm.stats(), "server_pages": sp, "n_sessions": n_sessions, "batch": batch,
            "gamma": gamma, "recompute": recompute, "pick": pick}


def summarize(rec: dict, window: int = 50) -> list:
    out = []
    rs = rec["rounds"]
    for w0 in range(0, len(rs), window):
        part = rs[w0:w0 + window]
        ms = float(np.mean([r["ms"] for r in part]))
        tok = float(np.sum([r["committed"] for r in part]))
        out.append({"rounds": f"{w0}-{w0 + len(part) - 1}", "ms_mean": ms,
                    "goodput_tok_s": tok / (np.sum([r["ms"] for r in part]) / 1e3),
                    "ctx_mean": float(np.mean([r["ctx_mean"] for r in part])),
                    "new_rows_mean": float(np.mean([r["new_rows"] for r in part])),
                    "hit_share": float(np.sum([r["hits"] for r in part]) / (len(part) * rec["batch"]))})
    return out


def report(res: dict) -> str:
    """Markdown summary of a sessions record."""
    L = ["# Multi-round verification sessions over the KV page-pool manager (Llama-3-8B shape, one MI355X)\n",
         "Command (repository root, on a GPU):\n",
         "    python -m paper_2601_11652_amd.sessions --out profiles/sessions_8b.json\n",
         "Each round drafts gamma = 4 tokens per served session with the device-side draft model (the target's "
         "weights, q = softmax(logits + 0.5 N(0, 1)), its own KV pool and manager) and verifies them in one "
         "wisp_verify call per chunk of at most 4096 new rows (HIP events around the verification only). "
         "Goodput = committed tokens / verification time.\n"]
    titles = {"cache_b2": "2 sessions, 256-token prompts, prefix cached between rounds",
              "recompute_b2": "the same 2 sessions, prefix recomputed every round (no prefix cache)",
              "cache_b32": "32 sessions, 512-token prompts, prefix cached",
              "evict_fit": "8 of 24 sessions per round at random, 128-token prompts, pool holding all",
              "evict_tight": "the same, pool holding 8 sessions at their longest (LRU eviction)"}
    for name, e in res["experiments"].items():
        st = e["stats"]
        L.append(f"## {name}: {titles.get(name, name)}\n")
        L.append(f"Server pool {e['server_pages']} pages; evictions {st['evictions']} ({st['pages_evicted']} pages); "
                 f"lookups hit {st['lookup_hits']} / missed {st['lookup_misses']}.\n")
        L.append("| rounds | verify ms (mean) | goodput tok/s | mean sequence length | new rows / round | "
                 "sessions found cached |")
        L.append("|---|---|---|---|---|---|")
        for w in e["summary"]:
            L.append(f"| {w['rounds']} | {w['ms_mean']:.2f} | {w['goodput_tok_s']:.0f} | {w['ctx_mean']:.0f} | "
                     f"{w['new_rows_mean']:.0f} | {100 * w['hit_share']:.0f} % |")
        L.append("")
    return "\n".join(L)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default="profiles/sessions_8b.json")
    ap.add_argument("--rounds", type=int, default=300)
    ap.add_argument("--report", default="", help="only write the markdown summary of this record")
    ap.add_argument("--md", default="profiles/sessions_8b.md")
    args = ap.parse_args(argv)
    if args.report:
        with open(args.md, "w") as f:
            f.write(report(json.load(open(args.report))))
        return
    import torch
    import wisp_inputs as wi
    from . import GpuModel
    torch.cuda.set_device(0)
    shape = wi.LLAMA3_8B
    gm = GpuModel(shape, lambda l: wi.layer_weights(shape, l, 1, "cuda"), wi.global_weights(shape, 1, "cuda"))
    log = lambda m: print(m, flush=True)   # noqa: E731
    res = {"model": shape.name, "experiments": {}}
    t0 = time.time()
    # 1. prefix cache vs recomputing the prefix every round (2 sessions, 256-token prompts)
    for name, rc in (("cache_b2", False), ("recompute_b2", True)):
        log(f"[{name}]")
        r = run(shape, gm, 2, 2, args.rounds, 256, 4, recompute=rc, log=log)
        res["experiments"][name] = {"summary": summarize(r), **r}
    # 2. a batch of 32 sessions over the rounds (512-token prompts)
    log("[cache_b32]")
    r = run(shape, gm, 32, 32, args.rounds, 512, 4, log=log)
    res["experiments"]["cache_b32"] = {"summary": summarize(r), **r}
    # 3. eviction: 8 of 24 sessions per round at random, the server pool holding 8 sessions
    #    at their longest (a round's batch always fits), against a pool that holds them all
    per = (128 + args.rounds // 3 * 5 + 5 + PAGE - 1) // PAGE + 1
    for name, pages in (("evict_fit", None), ("evict_tight", 8 * per)):
        log(f"[{name}]")
        r = run(shape, gm, 24, 8, args.rounds, 128, 4, pick="random", server_pages=pages, log=log)
        res["experiments"][name] = {"summary": summarize(r), **r}
    res["seconds"] = time.time() - t0
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        res["command"] = command_line("paper_2601_11652_amd.sessions", argv)
        json.dump(res, f)
    for name, e in res["experiments"].items():
        s = e["summary"]
        log(f"{name}: first {s[0]['ms_mean']:.2f} ms / {s[0]['goodput_tok_s']:.0f} tok/s, last "
            f"{s[-1]['ms_mean']:.2f} ms / {s[-1]['goodput_tok_s']:.0f} tok/s, evictions {e['stats']['evictions']}")


if __name__ == "__main__":
    sys.exit(main())
