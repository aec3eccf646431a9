"""Benchmark of the Accel-GCN aggregation path on one MI355X.

One step = the whole path over one synthetic graph: the device plan (degree
sort, relayout, Alg. 1/2 partition, one host sync) followed by the SpMM at
every feature width of the workload (default: the 230,000-node Chung-Lu
power-law graph, mean degree 50, F = 16, 32, 64, 128, 256), then the plan is
released. Inputs (CSR and X for every F) are resident in HBM before timing.

Prints ONE JSON line. value = whole-step throughput in GFLOP/s, FLOPs being
2 * nnz * F summed over the F sweep (the plan adds time, not FLOPs). Every step
builds its own plan; --overlap-steps builds the next step's plan on a second
stream while the current step's executes run.
Extra keys: per-F execute timings, plan time, the roofline of the dominant
kernel (measured with HIP events the library attaches to that kernel's
launch; each timed step marks the executes of one F, rotating through the
sweep, since every mark costs launch time) and the single-threaded CPU oracle
on a row sample.

--variant warp_level / column_loop times one of the two ablation baselines of
Table II instead (same workload, same step), for the ablation ratios.
--gcn-layer times one GCNConv forward of Sec. II-A instead (plan built once,
outside the timed steps): H = X W on the matrix cores, then the aggregation
with the ReLU epilogue, X of width --fin, W fin x --fout (default 128 x 128).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--F 16,32,...] [--variant block|warp_level|column_loop]
                       [--no-cpu-baseline] [--copy-probe]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import graphgen  # noqa: E402

METRIC = "SpMM GFLOP/s (2·nnz·F) and % of HBM roofline, F=16..256"
HBM_PEAK_GBPS = 8000.0
# Rates of random 128-byte gathers on this GPU (profiles/gather_ceiling_probe.md):
# served by L2 (working set within one XCD's 4 MB) 26-28 TB/s, served past L2
# (Infinity Cache or HBM) 6.8-7.3 TB/s; 64-byte gathers run at the same
# request rates. In requests per second for the whole GPU:
L2_GATHER_REQ_PER_S = 220e9
PAST_L2_GATHER_REQ_PER_S = 55e9
KERNEL_SRC = os.path.join(ROOT, "paper_2308_11825_amd", "csrc", "agcn_spmm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "spmm_traffic.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_bytes(st, F, n_ref, variant="block"):
    """Algorithmic HBM bytes of one launch of each execute kernel.

    k_spmm (and k_spmm_colloop, same plan):
                  8 nnz (sorted column index + value) + 16 per entry (metadata)
                  + 4 per non-hub row (perm) + 4 F per referenced X row (each once)
                  + 4 F per non-hub Y row + 4 F per hub chunk (partial row written)
    k_hub_reduce: 4 F per hub chunk (partial row read) + 4 F per hub row (Y)
                  + 8 per hub row (perm, chunk offset)
    k_spmm_wl:    8 nnz + 16 per group (metadata) + 4 F per referenced X row
                  + 4 F per Y row (rows cut by workgroups counted once)
    k_wl_fixup:   8 per row (group offsets)
    """
    if variant == "warp_level":
        return 8 * st.nnz + 16 * st.n_entries + 4 * F * n_ref + 4 * F * st.n_rows, 8 * st.n_rows
    nonhub = st.n_rows - st.n_hub_rows
    k7 = (8 * st.nnz + 16 * st.n_entries + 4 * nonhub + 4 * F * n_ref + 4 * F * nonhub
          + 4 * F * st.n_hub_chunks)
    k8 = 4 * F * st.n_hub_chunks + 4 * F * st.n_hub_rows + 8 * st.n_hub_rows
    return k7, k8


# Hub-row windows (plans whose agcn_plan_stats.hub_windows > 0, at F >= 64 on
# the float4 path): the library's launch shape, as agcn_spmm.hip computes it.
WIN_COLS, WIN_ROWS, WIN_SLICE, WIN_TARGET_GROUPS = 512, 1024, 64, 512
# LDS read bandwidth of the chip (the window kernel's gathers are LDS reads):
# 256 bytes per clock per CU, 256 CUs, 2.4 GHz. A read-only probe of ds_read_b128
# measured 135.7 TB/s (221 B/clk/CU) conflict-free and 111.5 TB/s with the
# window kernel's pattern (16-lane groups reading random 256-byte rows).
LDS_PEAK_GBPS = 256 * 256 * 2.4


def windows_used(st, F, variant="block"):
    return variant == "block" and st.hub_windows > 0 and F >= 64 and F % 4 == 0


def win_shape(st, F):
    n_slices = -(-F // WIN_SLICE)
    n_b = -(-st.n_hub_rows // WIN_ROWS)
    want = max(1, -(-WIN_TARGET_GROUPS // max(1, n_slices * n_b)))
    G = max(1, -(-st.hub_windows // want))
    return n_slices, n_b, G, -(-st.hub_windows // G)


def window_bytes(st, F, hub):
    """Algorithmic HBM bytes of the hub phase on windows (k_hub_win +
    k_hub_win_reduce), and of the aggregation of the other rows (k_spmm).

    k_hub_win + reduce: 8 per hub nonzero; X once per row batch (4 F per X
                  row); 8 per (hub row, window, slice) of window ranges;
                  (4 F + 4) per (hub row, window group) written and read
                  back (partial row, stray flag); 4 F + 4 per hub row (Y, perm)
    k_spmm:       as kernel_bytes, over the rows of degree <= deg_bound only
    hub: dict(hub_nnz, n_cols, low_nnz, low_ref, low_entries)."""
    n_slices, n_b, G, n_grp = win_shape(st, F)
    nh = st.n_hub_rows
    b_hub = (8 * hub["hub_nnz"] + 4 * F * hub["n_cols"] * n_b + 8 * nh * st.hub_windows * n_slices
             + 2 * (4 * F + 4) * nh * n_grp + (4 * F + 4) * nh)
    nonhub = st.n_rows - nh
    b_low = (8 * hub["low_nnz"] + 16 * hub["low_entries"] + 4 * nonhub + 4 * F * hub["low_ref"]
             + 4 * F * nonhub)
    return b_low, b_hub


def gather_requests(st, F):
    """Gather requests one aggregation launch issues for X: every nonzero
    loads its X row's piece of every column slice of 32 floats (one 128-byte
    line; a single 64-byte piece when F = 16)."""
    return st.nnz * ((F + 31) // 32)


def small_path(st):
    """Plans the library aggregates with k_spmm_rows (one vwarp per row, no
    staging): no hub rows, every degree <= min(Z, 32), nnz <= 2^18, rows <= 2^16."""
    return (st.n_hub_rows == 0 and st.max_deg <= min(st.max_wave_nzs, 32) and st.nnz <= 1 << 18
            and st.n_rows <= 1 << 16)


def spmm_kernel_name(F, variant="block", st=None):
    """Instantiation the library picks for an aligned float32 X: 32-column
    slices (AGCN_SLICE_COLS overrides), lanes = slice columns / 4."""
    if variant == "column_loop":
        return "k_spmm_colloop"
    if variant == "block" and st is not None and small_path(st):
        sc = min(F, 32) if F % 4 == 0 else min(F, 64)
        L = sc // 4 if F % 4 == 0 else sc
        return f"k_spmm_rows<{4 if F % 4 == 0 else 1}, {L if L in (4, 8) else 0}>"
    sc = int(os.environ.get("AGCN_SLICE_COLS", "32"))
    sc = sc if (4 <= sc <= 256 and sc % 4 == 0) else 32
    sc = min(F, sc)
    if variant == "warp_level":
        L = sc // 4 if F % 4 == 0 else min(F, sc)
        return f"k_spmm_wl<{4 if F % 4 == 0 else 1}, {L if L in (4, 8) else 0}>"
    return f"k_spmm<4, {sc // 4}>" if F % 4 == 0 else f"k_spmm<1, {min(F, sc, 64)}>"


def source_hash(path=KERNEL_SRC):
    """Hash of the aggregation kernels' code with comments and whitespace
    removed: a comment edit keeps stored counter figures valid, a code edit
    voids them."""
    import re
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    text = "".join(text.split())
    return hashlib.sha256(text.encode()).hexdigest()[:16]


def cpu_baseline(g, name, Fs, params, frac, seed=0):
    """Single-threaded oracle: full plan + SpMM of a random row sample for
    every F, extrapolated to all rows by nnz."""
    import oracle
    W, Z, H = params
    t0 = time.perf_counter()
    p = oracle.plan(g.rowptr, g.colidx, g.vals, W, Z, H)
    t_plan = time.perf_counter() - t0
    del p
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(g.n_rows, size=max(1, int(frac * g.n_rows)), replace=False)).astype(np.int32)
    nnz_s = int(g.degrees[rows].sum())
    t_spmm = 0.0
    for F in Fs:
        X = graphgen.workload_features(name, g, F)
        t0 = time.perf_counter()
        oracle.spmm_rows(g.rowptr, g.colidx, g.vals, X, rows)
        t_spmm += time.perf_counter() - t0
    scale = g.nnz / max(nnz_s, 1)
    t_step = t_plan + t_spmm * scale
    flops = sum(2.0 * g.nnz * F for F in Fs)
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": round(flops / t_step / 1e9, 4), "unit": "GFLOP/s", "cores": 1, "kind": "oracle",
        "cpu_model": model, "host_cpus": os.cpu_count(),
        "sample": (f"full oracle plan ({t_plan:.2f}s) + oracle SpMM over {rows.size} random rows "
                   f"({nnz_s} nnz, {100 * nnz_s / g.nnz:.1f}% of nnz) for F={Fs} "
                   f"({t_spmm:.2f}s), extrapolated by nnz to the full step"),
        "measured_s": round(t_plan + t_spmm, 3),
    }


def cache_protocol(agcn, plan, Fs, Xs, Ys, ws, stream, reps, dev):
    """Execute timings per F in the two cache states: cold (a 1 GiB buffer is
    written before every rep, outside the events, so X, the CSR and Y start
    outside L2 and the Infinity Cache) and warm (reps back to back).
    Median, p10 and p90 of the per-rep times, in ms: the whole execute, and
    the aggregation kernel alone (the events the library attaches to it)."""
    import torch
    flush = torch.empty(256 * 2**20, dtype=torch.float32, device=dev)
    sh = stream.cuda_stream

    def ev():
        e = torch.cuda.Event(enable_timing=True)
        e.record(stream)  # creates the underlying hipEvent_t
        return e

    def stats(t):
        return {"median_ms": round(float(np.median(t)), 5),
                "p10_ms": round(float(np.percentile(t, 10)), 5),
                "p90_ms": round(float(np.percentile(t, 90)), 5)}

    out = {}
    for F in Fs:
        res = {}
        for mode in ("cold", "warm"):
            marks = [(ev(), ev(), ev(), ev()) for _ in range(reps)]
            torch.cuda.synchronize()
            for a, b, m, c in marks:
                if mode == "cold":
                    flush.fill_(float(len(res)))
                a.record(stream)
                agcn.agcn_spmm_timed(plan, F, Xs[F].data_ptr(), F, Ys[F].data_ptr(), F,
                                     ws.data_ptr(), sh, b.cuda_event, m.cuda_event, None)
                c.record(stream)
            torch.cuda.synchronize()
            res[mode] = stats(np.array([a.elapsed_time(c) for a, _, _, c in marks]))
            res[mode]["spmm"] = stats(np.array([b.elapsed_time(m) for _, b, m, _ in marks]))
        out[F] = res
    del flush
    return out


ROCSPARSE_ALGS = {"default": 0, "csr": 1, "csr_row_split": 4, "csr_nnz_split": 5, "csr_merge_path": 9}


def rocsparse_compare(g, Fs, Xs, Ys, d_rowptr, d_colidx, d_vals, stream, reps):
    """rocSPARSE's generic CSR SpMM (torch's bundled librocsparse) on the same
    device arrays: row-major X and Y, fp32, original row order. Times the
    compute stage only (buffer sizing and preprocessing excluded, as the plan
    is excluded from `exec_ms`) for every CSR algorithm, and reports the
    largest difference between its Y and the library's Y. Context for the
    comparison, not a target."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "librocsparse.so"))
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    h = vp()
    assert lib.rocsparse_create_handle(ctypes.byref(h)) == 0
    assert lib.rocsparse_set_stream(h, vp(stream.cuda_stream)) == 0
    A = vp()
    st = lib.rocsparse_create_csr_descr(ctypes.byref(A), i64(g.n_rows), i64(g.n_cols), i64(g.nnz),
                                        vp(d_rowptr.data_ptr()), vp(d_colidx.data_ptr()),
                                        vp(d_vals.data_ptr()), 2, 2, 0, 151)
    assert st == 0, st
    alpha, beta = ctypes.c_float(1.0), ctypes.c_float(0.0)
    out = {}
    for F in Fs:
        Yr = torch.empty_like(Ys[F])
        B, C = vp(), vp()
        assert lib.rocsparse_create_dnmat_descr(ctypes.byref(B), i64(g.n_cols), i64(F), i64(F),
                                                vp(Xs[F].data_ptr()), 151, 0) == 0
        assert lib.rocsparse_create_dnmat_descr(ctypes.byref(C), i64(g.n_rows), i64(F), i64(F),
                                                vp(Yr.data_ptr()), 151, 0) == 0
        res = {}
        for name, alg in ROCSPARSE_ALGS.items():
            def call(stage, nbytes, buf):
                return lib.rocsparse_spmm(h, 111, 111, ctypes.byref(alpha), A, B, ctypes.byref(beta),
                                          C, 151, alg, stage, nbytes, buf)
            nbytes = ctypes.c_size_t(0)
            if call(1, ctypes.byref(nbytes), None) != 0:
                res[name] = "unsupported"
                continue
            buf = torch.empty(max(1, nbytes.value), dtype=torch.uint8, device=Ys[F].device)
            t0 = time.perf_counter()
            if call(2, ctypes.byref(nbytes), vp(buf.data_ptr())) != 0:
                res[name] = "preprocess failed"
                continue
            torch.cuda.synchronize()
            t_pre = time.perf_counter() - t0
            Yr.fill_(float("nan"))
            if call(3, ctypes.byref(nbytes), vp(buf.data_ptr())) != 0:
                res[name] = "compute failed"
                continue
            torch.cuda.synchronize()
            diff = float((Yr - Ys[F]).abs().max()) if Yr.numel() else 0.0
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                call(3, ctypes.byref(nbytes), vp(buf.data_ptr()))
            e1.record(stream)
            torch.cuda.synchronize()
            res[name] = {"ms": round(e0.elapsed_time(e1) / reps, 5), "preprocess_s": round(t_pre, 4),
                         "max_abs_diff_vs_agcn": diff}
            del buf
        out[F] = res
        lib.rocsparse_destroy_dnmat_descr(B)
        lib.rocsparse_destroy_dnmat_descr(C)
    lib.rocsparse_destroy_spmat_descr(A)
    lib.rocsparse_destroy_handle(h)
    return out


MFMA_FP32_PEAK_TFLOPS = 157.3


def linear_kernel_name(fin, fout):
    """Instantiation agcn_linear picks for compact, 16-byte aligned float32 X and
    W (AGCN_LINEAR_RW=0 forces the tiled kernel)."""
    vec = fin % 4 == 0 and fout % 4 == 0
    if vec and 1 <= fin <= 128 and fout <= 128 and os.environ.get("AGCN_LINEAR_RW", "1") != "0":
        nb = 2 if fout <= 32 else 4 if fout <= 64 else 8
        ks = 2 if fin <= 32 else 4 if fin <= 64 else 8
        return f"k_linear_rw<{nb}, {ks}>"
    return f"k_linear<{32 if fout <= 32 else 64 if fout <= 64 else 128}, {'true' if vec else 'false'}>"


def bench_layer(args):
    """One GCNConv forward per step over a plan built once."""
    import torch
    import paper_2308_11825_amd as agcn
    name, fin, fout = args.workload, args.fin, args.fout
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = graphgen.make(name, verbose=False)
    log(f"workload {name}: {graphgen.stats(g)}; layer {fin} -> {fout}")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_rowptr, d_colidx, d_vals = t(g.rowptr), t(g.colidx), t(g.vals)
    X = t(graphgen.workload_features(name, g, fin))
    W = t(graphgen.weights(fin, fout, seed=7))
    Y = torch.empty((g.n_rows, fout), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    prm = agcn.agcn_default_params()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    p0, p1 = ev(), ev()
    p0.record(stream)
    plan = agcn.agcn_plan_create(g.n_rows, g.n_cols, g.nnz, d_rowptr.data_ptr(), d_colidx.data_ptr(),
                                 d_vals.data_ptr(), prm, sh)
    p1.record(stream)
    torch.cuda.synchronize()
    plan_ms = p0.elapsed_time(p1)
    st = agcn.agcn_plan_info(plan)
    nb = agcn.agcn_gcn_workspace_size(plan, fout)
    ws = torch.empty((nb + 3) // 4, dtype=torch.float32, device=dev)
    H = ws[: g.n_cols * fout].view(g.n_cols, fout)
    relu = agcn.AGCN_EPILOGUE_RELU

    def layer():
        agcn.agcn_gcn_layer(plan, fin, fout, X.data_ptr(), fin, W.data_ptr(), fout, Y.data_ptr(),
                            fout, ws.data_ptr(), sh, relu)

    for _ in range(args.warmup):
        layer()
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record(stream)
    for _ in range(args.steps):
        layer()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    log(f"timed {args.steps} layer steps: {ms_step:.4f} ms/step")
    # The two halves of the same call, timed on their own for the roofline:
    # agcn_linear into the same workspace, then the aggregation with ReLU.
    marks = [(ev(), ev(), ev()) for _ in range(args.steps)]
    for a, b, c in marks:
        a.record(stream)
        agcn.agcn_linear(g.n_cols, fin, fout, X.data_ptr(), fin, W.data_ptr(), fout, H.data_ptr(),
                         fout, sh)
        b.record(stream)
        agcn.agcn_spmm_ex(plan, fout, H.data_ptr(), fout, Y.data_ptr(), fout,
                          ws[(nb - agcn.agcn_spmm_workspace_size(plan, fout)) // 4:].data_ptr()
                          if agcn.agcn_spmm_workspace_size(plan, fout) else None, sh, relu)
        c.record(stream)
    torch.cuda.synchronize()
    lin_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in marks]))
    agg_ms = float(np.mean([b.elapsed_time(c) for _, b, c in marks]))
    agcn.agcn_plan_destroy(plan)
    fl_lin = 2.0 * g.n_cols * fin * fout
    fl_agg = 2.0 * g.nnz * fout
    ach = fl_lin / (lin_ms * 1e-3) / 1e12
    kname = linear_kernel_name(fin, fout)
    out = {
        "metric": "GCNConv layer forward GFLOP/s (2·N·fin·fout + 2·nnz·fout)",
        "value": round((fl_lin + fl_agg) / (ms_step * 1e-3) / 1e9, 3), "unit": "GFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "n_rows": g.n_rows, "nnz": g.nnz, "fin": fin, "fout": fout,
                   "activation": "relu", "parallelism": "single GPU"},
        "plan_ms_once": round(plan_ms, 4), "linear_ms": round(lin_ms, 5),
        "aggregation_ms": round(agg_ms, 5),
        "roofline": {"bound": "mfma", "achieved": round(ach, 2), "peak": MFMA_FP32_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(ach / MFMA_FP32_PEAK_TFLOPS, 4),
                     "traffic": None, "kernel": kname,
                     "hbm_bytes_alg": int(4 * g.n_cols * (fin + fout) + 4 * fin * fout)},
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="sweep_powerlaw", choices=sorted(graphgen.CONFIGS))
    ap.add_argument("--F", default=None, help="comma-separated feature widths")
    ap.add_argument("--W", type=int, default=None)
    ap.add_argument("--Z", type=int, default=None)
    ap.add_argument("--H", type=int, default=None)
    ap.add_argument("--variant", default="block", choices=["block", "warp_level", "column_loop"],
                    help="ablation baselines of Table II (default: the block-level path)")
    ap.add_argument("--rocsparse", action="store_true",
                    help="also time rocSPARSE's CSR SpMM on the same inputs (context)")
    ap.add_argument("--gcn-layer", action="store_true",
                    help="time one GCNConv layer forward (linear + aggregation + ReLU)")
    ap.add_argument("--fin", type=int, default=128)
    ap.add_argument("--fout", type=int, default=128)
    ap.add_argument("--cache-reps", type=int, default=20,
                    help="reps per F for the cold/warm execute protocol (0 skips it)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-frac", type=float, default=0.4)
    ap.add_argument("--overlap-steps", action="store_true",
                    help="build the next step's plan on a second stream during the current "
                         "step's executes (default: plan, executes, release in order on one stream)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="accepted for older profile commands: the 1 GiB device copy (counter "
                         "calibration, measured copy bandwidth) now always runs after timing")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(row or column sharding of the aggregation is described, not implemented).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2308_11825_amd as agcn

    if args.gcn_layer:
        return bench_layer(args)
    name = args.workload
    Fs = [int(f) for f in args.F.split(",")] if args.F else list(graphgen.CONFIGS[name]["F"])
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = graphgen.make(name, verbose=False)
    log(f"workload {name}: {graphgen.stats(g)}")
    n_ref = int(np.count_nonzero(np.bincount(g.colidx, minlength=g.n_cols)))

    prm = agcn.agcn_default_params()
    if args.W is not None:
        prm.max_block_waves = args.W
    if args.Z is not None:
        prm.max_wave_nzs = args.Z
    if args.H is not None:
        prm.hub_chunk_nnz = args.H
    prm.flags = {"block": 0, "warp_level": agcn.AGCN_PLAN_WARP_LEVEL,
                 "column_loop": agcn.AGCN_PLAN_COLUMN_LOOP}[args.variant]

    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_rowptr, d_colidx, d_vals = t(g.rowptr), t(g.colidx), t(g.vals)
    Xs = {F: t(graphgen.workload_features(name, g, F)) for F in Fs}
    Ys = {F: torch.empty((g.n_rows, F), dtype=torch.float32, device=dev) for F in Fs}
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream

    # Workspace sized from a probe plan (same parameters, same graph).
    probe = agcn.agcn_plan_create(g.n_rows, g.n_cols, g.nnz, d_rowptr.data_ptr(),
                                  d_colidx.data_ptr(), d_vals.data_ptr(), prm, sh)
    st = agcn.agcn_plan_info(probe)
    ws_bytes = max(agcn.agcn_spmm_workspace_size(probe, F) for F in Fs)
    agcn.agcn_plan_destroy(probe)
    ws = torch.empty(max(1, (ws_bytes + 3) // 4), dtype=torch.float32, device=dev)
    log(f"plan: entries={st.n_entries} hub_rows={st.n_hub_rows} hub_chunks={st.n_hub_chunks} "
        f"W={st.max_block_waves} Z={st.max_wave_nzs} H={st.hub_chunk_nnz} ws={ws_bytes}B")

    def new_event():
        e = torch.cuda.Event(enable_timing=True)
        e.record(stream)  # creates the underlying hipEvent_t
        return e

    # Timing marks cost several microseconds per marked launch, so each timed
    # step marks the executes of one F only, rotating through the F sweep
    # (every F when there are fewer steps than widths).
    def timed_fs(k):
        return [Fs[k % len(Fs)]] if args.steps >= len(Fs) else list(Fs)

    # Every step builds its own plan and runs the five executes with it, plan,
    # executes and release one after the other on one stream. With
    # --overlap-steps the plan of step k+1 is built on a second stream
    # (default priority) while the executes of step k run, as a pipeline that
    # plans the next graph during the current aggregation would; the executes
    # wait for their plan on the device (the library orders an execute on
    # another stream after the plan's kernels).
    serial = not args.overlap_steps
    plan_stream = stream if serial else torch.cuda.Stream(dev)
    psh = plan_stream.cuda_stream

    def make_plan():
        return agcn.agcn_plan_create(g.n_rows, g.n_cols, g.nnz, d_rowptr.data_ptr(),
                                     d_colidx.data_ptr(), d_vals.data_ptr(), prm, psh)

    def executes(plan, evs):
        # evs: per marked F (k_spmm start, k_spmm end, after the execute); the
        # library records the first two on the launch stream.
        for F in Fs:
            b, m, a = evs[F] if evs is not None and F in evs else (None, None, None)
            agcn.agcn_spmm_timed(plan, F, Xs[F].data_ptr(), F, Ys[F].data_ptr(), F, ws.data_ptr(),
                                 sh, b.cuda_event if b else None, m.cuda_event if m else None, None)
            if a is not None:
                a.record(stream)

    def run_steps(n, evs_of):
        if serial:
            for k in range(n):
                plan = make_plan()
                executes(plan, evs_of(k))
                agcn.agcn_plan_destroy(plan)
            return
        cur = make_plan()
        for k in range(n):
            executes(cur, evs_of(k))
            nxt = make_plan() if k + 1 < n else None
            agcn.agcn_plan_destroy(cur)
            cur = nxt

    run_steps(args.warmup, lambda k: None)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    events = [{F: (new_event(), new_event(), new_event()) for F in timed_fs(k)}
              for k in range(args.steps)]
    torch.cuda.synchronize()
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(plan_stream)     # the first step's plan is the first work timed
    run_steps(args.steps, lambda k: events[k])
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    log(f"timed {args.steps} steps: {ms_step:.4f} ms/step")
    # the plan alone (serial, for reference): create + destroy on one stream
    pe0, pe1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    pe0.record(stream)
    for _ in range(5):
        agcn.agcn_plan_destroy(agcn.agcn_plan_create(g.n_rows, g.n_cols, g.nnz, d_rowptr.data_ptr(),
                                                     d_colidx.data_ptr(), d_vals.data_ptr(), prm, sh))
    pe1.record(stream)
    torch.cuda.synchronize()
    plan_alone_ms = pe0.elapsed_time(pe1) / 5

    hub = None
    if st.hub_windows > 0:
        deg = np.diff(g.rowptr.astype(np.int64))
        low_rows = deg <= st.deg_bound
        low_cols = g.colidx[np.repeat(low_rows, deg)]
        hub = {"hub_nnz": int(deg[~low_rows].sum()), "n_cols": g.n_cols,
               "low_nnz": int(deg[low_rows].sum()), "low_entries": st.hub_first_entry,
               "low_ref": int(np.count_nonzero(np.bincount(low_cols, minlength=g.n_cols)))}
    per_f = {}
    flops_step = 0.0
    exec_ms_sum = 0.0
    for F in Fs:
        marks = [ev[F] for ev in events if F in ev]
        k7 = np.array([b.elapsed_time(m) for b, m, _ in marks])
        # hub phase (hub-chunk reduction, or the windows and their reduction)
        # and the launch gap before it
        k8 = np.array([m.elapsed_time(a) for _, m, a in marks])
        win = windows_used(st, F, args.variant)
        b7, b8 = window_bytes(st, F, hub) if win else kernel_bytes(st, F, n_ref, args.variant)
        ex_ms = float(np.mean(k7 + k8))
        exec_ms_sum += ex_ms
        fl = 2.0 * g.nnz * F
        flops_step += fl
        per_f[F] = {
            "exec_ms": round(ex_ms, 5), "spmm_ms": round(float(k7.mean()), 5),
            "hub_reduce_ms": round(float(k8.mean()), 5), "timed_launches": len(marks),
            "gflops": round(fl / (ex_ms * 1e-3) / 1e9, 2),
            "alg_GBps": round((b7 + b8) / (ex_ms * 1e-3) / 1e9, 1),
            "frac_hbm": round((b7 + b8) / (ex_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "spmm_bytes": int(b7), "spmm_GBps": round(b7 / (k7.mean() * 1e-3) / 1e9, 1),
        }
        if win:
            # k_spmm covers the rows of degree <= deg_bound; the hub phase is
            # k_hub_win + k_hub_win_reduce, whose X reads are LDS reads (4 F
            # bytes per hub nonzero)
            lds = 4 * F * hub["hub_nnz"]
            per_f[F].update({"hub_path": "windows", "hub_bytes": int(b8),
                             "hub_GBps": round(b8 / (k8.mean() * 1e-3) / 1e9, 1),
                             "hub_lds_bytes": int(lds),
                             "hub_lds_GBps": round(lds / (k8.mean() * 1e-3) / 1e9, 1)})
    # serial steps: the plan plus the launch gaps between executes; overlapped
    # steps: whatever of the plan and the gaps the executes did not hide
    plan_ms = ms_step - exec_ms_sum
    # Group the aggregation launches by kernel instantiation (lanes per vwarp),
    # as rocprofv3 reports them; the dominant one is the group with the most
    # time per step. achieved = mean algorithmic bytes per launch / mean
    # launch duration over that group's launches.
    groups = {}
    for F in Fs:
        groups.setdefault(spmm_kernel_name(F, args.variant, st), []).append(F)
    dom = max(groups, key=lambda k: sum(per_f[F]["spmm_ms"] for F in groups[k]))
    dom_F = groups[dom]
    mean_bytes = float(np.mean([per_f[F]["spmm_bytes"] for F in dom_F]))
    mean_ms = float(np.mean([per_f[F]["spmm_ms"] for F in dom_F]))
    ach = mean_bytes / (mean_ms * 1e-3) / 1e9
    # traffic: calibrated FETCH_SIZE + WRITE_SIZE per launch, i.e. the bytes
    # moved between L2 and the memory side; gfx950 has no counter that tells
    # Infinity Cache hits from HBM accesses, so part of it may never reach HBM.
    traffic = past_l2_req = None
    try:
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if (tr.get("source_hash") == source_hash() and tr.get("workload") == name
                and tr.get("F") == dom_F and tr.get("kernel") == dom):
            traffic = tr.get("past_l2_bytes_per_launch")
            past_l2_req = tr.get("past_l2_read_requests_per_launch")
    except (OSError, ValueError):
        pass
    # Model ceiling of any kernel that gathers X rows per nonzero: its gather
    # requests all served by L2 at the measured L2 gather rate.
    req = float(np.mean([gather_requests(st, F) * (hub["low_nnz"] / st.nnz
                                                   if windows_used(st, F, args.variant) else 1.0)
                         for F in dom_F]))
    cap_ms = req / L2_GATHER_REQ_PER_S * 1e3
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBPS, 4), "traffic": traffic,
                "kernel": dom, "launches_per_step": len(dom_F), "F": dom_F,
                "alg_bytes_per_launch": int(mean_bytes), "avg_launch_ms": round(mean_ms, 5),
                "l2_gather_cap": {"requests_per_launch": int(req), "cap_ms": round(cap_ms, 5),
                                  "frac_at_cap": round(mean_bytes / (cap_ms * 1e-3) / 1e9
                                                       / HBM_PEAK_GBPS, 4),
                                  "achieved_over_cap": round(cap_ms / mean_ms, 4)}}
    win_F = [F for F in Fs if windows_used(st, F, args.variant)]
    win_roof = bool(win_F) and (sum(per_f[F]["hub_reduce_ms"] for F in win_F)
                                > sum(per_f[F]["spmm_ms"] for F in dom_F))
    if win_roof:
        # The hub windows dominate: their bound is the LDS reads of the staged
        # X windows. The marks frame the whole hub phase (k_hub_win,
        # k_hub_win_reduce and the gap before them), so achieved is a lower
        # bound for k_hub_win alone.
        lds_b = float(np.mean([per_f[F]["hub_lds_bytes"] for F in win_F]))
        hub_ms = float(np.mean([per_f[F]["hub_reduce_ms"] for F in win_F]))
        lds_ach = lds_b / (hub_ms * 1e-3) / 1e9
        hbm_b = float(np.mean([per_f[F]["hub_bytes"] for F in win_F]))
        roofline = {"bound": "lds", "achieved": round(lds_ach, 1), "peak": LDS_PEAK_GBPS,
                    "unit": "GB/s", "frac": round(lds_ach / LDS_PEAK_GBPS, 4), "traffic": None,
                    "kernel": "k_hub_win", "launches_per_step": len(win_F), "F": win_F,
                    "alg_bytes_per_launch": int(lds_b), "avg_launch_ms": round(hub_ms, 5),
                    "timed": "k_hub_win + k_hub_win_reduce",
                    "alg_hbm_bytes_per_launch": int(hbm_b),
                    "alg_hbm_GBps": round(hbm_b / (hub_ms * 1e-3) / 1e9, 1)}
    if traffic is not None and not win_roof:
        # counter-measured bytes past L2 (Infinity Cache hits included) over the same time
        tg = traffic / (mean_ms * 1e-3) / 1e9
        roofline["past_l2_GBps"] = round(tg, 1)
        roofline["past_l2_frac_of_hbm_peak"] = round(tg / HBM_PEAK_GBPS, 4)
    if past_l2_req and not win_roof:
        # the binding ceiling: random line requests past L2 (the L2 misses)
        rate = past_l2_req / (mean_ms * 1e-3)
        roofline["past_l2_request_cap"] = {
            "requests_per_launch": int(past_l2_req), "achieved_G_per_s": round(rate / 1e9, 2),
            "cap_G_per_s": PAST_L2_GATHER_REQ_PER_S / 1e9,
            "achieved_over_cap": round(rate / PAST_L2_GATHER_REQ_PER_S, 4)}

    # A measured streaming ceiling beside the 8 TB/s peak: a 1 GiB device copy
    # (read + write), timed after the timed region; with --copy-probe it is
    # also the counter calibration kernel.
    src = torch.empty(256 * 2**20, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(3):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_GBps = 3 * 2 * src.numel() * 4 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst
    roofline["copy_GBps"] = round(copy_GBps, 1)
    if not win_roof:
        roofline["frac_of_copy"] = round(ach / copy_GBps, 4)
    log(f"copy probe: 1 GiB device copy at {copy_GBps:.0f} GB/s (read + write)")

    out = {
        "metric": METRIC, "value": round(flops_step / (ms_step * 1e-3) / 1e9, 3), "unit": "GFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "n_rows": g.n_rows, "nnz": g.nnz, "F": Fs,
                   "max_block_waves": st.max_block_waves, "max_wave_nzs": st.max_wave_nzs,
                   "hub_chunk_nnz": st.hub_chunk_nnz, "n_entries": st.n_entries,
                   "n_hub_rows": st.n_hub_rows, "variant": args.variant,
                   "parallelism": "single GPU"},
        "steps_overlap": (None if serial else
                          "the plan of step k+1 is built on a second stream during the executes of "
                          "step k; every step still builds its own plan"),
        "plan_ms": round(plan_ms, 4), "plan_alone_ms": round(plan_alone_ms, 4),
        "spmm_only_gflops": round(flops_step / (exec_ms_sum * 1e-3) / 1e9, 2),
        "per_F": per_f,
        "roofline": roofline,
    }
    if args.cache_reps > 0:
        log("cold / warm execute protocol ...")
        plan = agcn.agcn_plan_create(g.n_rows, g.n_cols, g.nnz, d_rowptr.data_ptr(),
                                     d_colidx.data_ptr(), d_vals.data_ptr(), prm, sh)
        cw = cache_protocol(agcn, plan, Fs, Xs, Ys, ws, stream, args.cache_reps, dev)
        out["execute_cold_warm"] = cw
        agcn.agcn_plan_destroy(plan)
        # the dominant kernel's roofline fraction from its cold launches (X, the
        # CSR and Y outside L2 and the Infinity Cache when each launch starts)
        if win_roof:  # the hub phase of the cold executes: the execute minus k_spmm
            cold_ms = float(np.mean([cw[F]["cold"]["median_ms"] - cw[F]["cold"]["spmm"]["median_ms"]
                                     for F in win_F]))
            roofline["frac_cold"] = round(lds_b / (cold_ms * 1e-3) / 1e9 / LDS_PEAK_GBPS, 4)
        else:
            cold_ms = float(np.mean([cw[F]["cold"]["spmm"]["median_ms"] for F in dom_F]))
            roofline["frac_cold"] = round(mean_bytes / (cold_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)
        roofline["avg_launch_ms_cold"] = round(cold_ms, 5)
    if args.rocsparse:
        log("rocSPARSE comparison ...")
        rs = rocsparse_compare(g, Fs, Xs, Ys, d_rowptr, d_colidx, d_vals, stream, reps=10)
        # this path timed the way rocSPARSE is: 10 executes back to back between two events
        plan = agcn.agcn_plan_create(g.n_rows, g.n_cols, g.nnz, d_rowptr.data_ptr(),
                                     d_colidx.data_ptr(), d_vals.data_ptr(), prm, sh)
        b2b = {}
        for F in Fs:
            agcn.agcn_spmm(plan, F, Xs[F].data_ptr(), F, Ys[F].data_ptr(), F, ws.data_ptr(), sh)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(10):
                agcn.agcn_spmm(plan, F, Xs[F].data_ptr(), F, Ys[F].data_ptr(), F, ws.data_ptr(), sh)
            e1.record(stream)
            torch.cuda.synchronize()
            b2b[F] = e0.elapsed_time(e1) / 10
        agcn.agcn_plan_destroy(plan)
        summary = {}
        for F in Fs:
            timed = {k: v["ms"] for k, v in rs[F].items() if isinstance(v, dict)}
            best = min(timed, key=timed.get) if timed else None
            summary[F] = {"algs": rs[F], "best": best, "exec_ms_back_to_back": round(b2b[F], 5),
                          "exec_ms_ratio": (round(timed[best] / b2b[F], 3) if best else None)}
        out["rocsparse"] = summary
    if not args.no_cpu_baseline and args.variant == "block":
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(g, name, Fs, (st.max_block_waves, st.max_wave_nzs,
                                                         st.hub_chunk_nnz), args.cpu_frac)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
