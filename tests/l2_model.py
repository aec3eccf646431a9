"""A model of one XCD's L2 under the aggregation's X gathers (test support:
not a measurement, and not part of the library).

One 128-byte column slice pass of the block-level aggregation is replayed on
the CPU. Each nonzero gathers one line (its column's piece of X), so the line
id is the column. The model follows one XCD: every eighth launch position of
the plan's launch order (workgroups are dealt to the eight XCDs in turn), with
C workgroups in flight (32 CUs x 16). Each in-flight workgroup advances by
rounds in which every vwarp issues its next G gathers (k_spmm keeps 8 loads in
flight per lane); workgroups advance in a seeded random interleaving, and a
finished workgroup's slot takes the next launch position.

The L2 is a fully associative cache of K lines (4 MB / 128 B = 32768):
  lru        least recently used replacement (what the measured hit rates
             follow closely);
  opt        Belady's MIN on the same stream: the best any replacement
             policy could do with this schedule;
  compulsory one miss per distinct line: the floor for any schedule that
             gathers each column's line on this XCD at least once.
Schedules:
  launch     the library's: hub chunks first, then the other entries
             heaviest first (reverse metadata order);
  light      lightest entries first; random: a seeded random launch order;
  sweep      a schedule this design does not have: every workgroup of the
             XCD walks its nonzeros in column windows, in lockstep, with the
             row partial sums held on chip for the whole pass.

Usage: python tests/l2_model.py [--workload sweep_powerlaw] [--xcd 0]
Prints one JSON line per (schedule, policy).
"""
from __future__ import annotations

import argparse
import collections
import heapq
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

N_XCD = 8


def lru_hits(seq, K):
    """Hits of a K-line LRU cache on the line sequence `seq`."""
    cache = collections.OrderedDict()
    hits = 0
    for c in seq:
        if c in cache:
            hits += 1
            cache.move_to_end(c)
        else:
            cache[c] = None
            if len(cache) > K:
                cache.popitem(last=False)
    return hits


def opt_hits(seq, K):
    """Hits of Belady's MIN (evict the line whose next use is farthest)."""
    seq = np.asarray(seq)
    n = seq.size
    nxt = np.full(n, n + 1, dtype=np.int64)
    last = {}
    for i in range(n - 1, -1, -1):
        c = int(seq[i])
        nxt[i] = last.get(c, n + 1 + i)   # distinct "never" keys keep the heap ordered
        last[c] = i
    cached = {}                            # line -> its next use
    heap = []                              # (-next use, line), stale entries skipped
    hits = 0
    for i in range(n):
        c = int(seq[i])
        if c in cached:
            hits += 1
        elif len(cached) >= K:
            while True:
                nu, v = heapq.heappop(heap)
                if cached.get(v) == -nu:
                    del cached[v]
                    break
        cached[c] = int(nxt[i])
        heapq.heappush(heap, (-int(nxt[i]), c))
    return hits


def entry_vwarps(m, cs, W, deg_bound):
    """The column sequences of an entry's vwarps (the paper's warp workloads)."""
    d, loc, row, info = (int(x) for x in m)
    if d > deg_bound:
        n = info
        sl = -(-n // W)
        return [cs[loc + v * sl: loc + min(n, (v + 1) * sl)] for v in range(W)]
    rows, wn = info & 0xFFFF, info >> 16
    if d == 0:
        return []
    wpr = -(-d // wn)
    out = []
    for r in range(rows):
        base = loc + r * d
        for q in range(wpr):
            out.append(cs[base + q * wn: base + min(d, (q + 1) * wn)])
    return out


def launch_stream(meta, cs, order, W, deg_bound, xcd=0, C=512, G=8, seed=1):
    """Line sequence one XCD sees under the workgroup schedule of `order`."""
    rng = np.random.default_rng(seed)
    positions = order[xcd::N_XCD]
    nxt = 0
    slots = []

    def load():
        nonlocal nxt
        while nxt < len(positions):
            seqs = [s for s in entry_vwarps(meta[positions[nxt]], cs, W, deg_bound) if len(s)]
            nxt += 1
            if seqs:
                return [seqs, 0, max(len(s) for s in seqs)]
        return None

    for _ in range(C):
        s = load()
        if s is None:
            break
        slots.append(s)
    out = []
    while slots:
        live = []
        for s in slots:
            if rng.random() < 0.5:       # workgroups advance at varying rates
                live.append(s)
                continue
            seqs, r, mx = s
            for q in seqs:
                out.extend(q[r * G: r * G + G].tolist())
            s[1] = r + 1
            if s[1] * G >= mx:
                s = load()
                if s is None:
                    continue
            live.append(s)
        slots = live
    return np.asarray(out, dtype=np.int64)


def sweep_stream(meta, cs, W, deg_bound, n_cols, xcd=0, tiles=32, windows=32):
    """Line sequence of the column-window sweep: entries dealt round-robin to
    the GPU's workgroups (one per CU), the XCD's workgroups walking their
    nonzeros window by window in lockstep."""
    n_wg = tiles * N_XCD
    ents = np.arange(len(meta))[::-1]
    mine = [ents[t::n_wg] for t in range(xcd, n_wg, N_XCD)]
    streams = []
    for es in mine:
        parts = [np.concatenate(v) for v in (entry_vwarps(meta[e], cs, W, deg_bound) for e in es) if v]
        c = np.concatenate(parts) if parts else np.zeros(0, np.int64)
        w = (c.astype(np.int64) * windows) // max(n_cols, 1)
        o = np.argsort(w, kind="stable")
        c, w = c[o], w[o]
        pos = np.empty(len(c))
        for ww in range(windows):
            idx = np.nonzero(w == ww)[0]
            pos[idx] = ww + (np.arange(len(idx)) + 0.5) / max(len(idx), 1)
        streams.append((c, pos))
    allc = np.concatenate([s[0] for s in streams])
    allk = np.concatenate([s[1] for s in streams])
    return allc[np.argsort(allk, kind="stable")].astype(np.int64)


def main():
    import graphgen
    import oracle
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="sweep_powerlaw")
    ap.add_argument("--xcd", type=int, default=0)
    ap.add_argument("--K", type=int, default=32768)
    ap.add_argument("--W", type=int, default=16)
    ap.add_argument("--Z", type=int, default=32)
    ap.add_argument("--no-opt", action="store_true")
    args = ap.parse_args()
    g = graphgen.make(args.workload)
    p = oracle.plan(g.rowptr, g.colidx, g.vals, args.W, args.Z, 0)
    meta, cs = p["meta"], p["colidx_s"].astype(np.int64)
    W, deg_bound = args.W, args.W * args.Z
    rev = np.arange(len(meta))[::-1]
    # the library's launch order: hub chunks in column order (16-bit key of
    # their first column) when hub rows are long or chunks many, otherwise in
    # reverse metadata order; then the other entries heaviest first
    hub = np.nonzero(meta[:, 0] > deg_bound)[0]
    n_hub_rows = len(np.unique(meta[hub, 2])) if len(hub) else 0
    launch = rev
    if len(hub) and (len(hub) >= 8 * n_hub_rows or len(hub) >= 32768):
        key = (cs[meta[hub, 1]].astype(np.int64) << 16) // g.n_cols
        launch = np.concatenate([hub[np.argsort(key, kind="stable")], rev[len(hub):]])
    rng = np.random.default_rng(7)
    schedules = {"launch": launch, "light": np.arange(len(meta)), "random": rng.permutation(len(meta))}
    rows = []
    for name, order in schedules.items():
        seq = launch_stream(meta, cs, order, W, deg_bound, xcd=args.xcd)
        rows.append((name, seq))
    rows.append(("sweep", sweep_stream(meta, cs, W, deg_bound, g.n_cols, xcd=args.xcd)))
    for name, seq in rows:
        n = len(seq)
        res = {"workload": args.workload, "schedule": name, "accesses": n, "K": args.K,
               "lru": round(lru_hits(seq.tolist(), args.K) / n, 4),
               "compulsory": round(1 - len(np.unique(seq)) / n, 4)}
        if name == "launch" and not args.no_opt:
            res["opt"] = round(opt_hits(seq, args.K) / n, 4)
        print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
