"""Benchmark: exact Kernel K-means on one MI355X through the engine's C ABI.

A step is one whole clustering job on synthetic input already resident in
HBM: build K = kappa(X X^T), then run the workload's number of assignment
updates (E = K V^T, z, D, argmin, sizes) from the seeded initial ids.
``value`` is clustering updates per second over the whole job (K build
included), timed with no kernel instrumented.  Per-kernel times come from
HIP events the library records on its stream in as many further jobs; the
K-build and per-update roofline figures are derived from them.

Default workload: the largest, n=200,000 points, d=54, k=7, Gaussian kernel
gamma=1/54, 50 updates, K stored packed (its upper block triangle, 80 GB;
by default each workload takes the storage the library's planner picks for
its kernel and k).  Beside it, under their
own keys, the same workload with the full K resident (160 GB) and with K
tiles recomputed on the fly each update (nothing stored), each over fewer
jobs.  ``--config N`` picks another workload and ``--mode`` another storage.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, 8 TB/s
FP32_MFMA_PEAK_TF = 157.3    # MI355X dense fp32 matrix peak
METRIC = "clustering iters/sec + K-build TFLOP/s, % of HBM / MFMA peak, 1 GPU"

# HBM bytes per launch from two rocprofv3 counter runs (FETCH_SIZE, then
# WRITE_SIZE; KiB per dispatch) on a workload, scaled by what the same
# counters read for a plain 1 GiB device copy (fetch x1.9999, write x1.0).
# Reported only while the kernel's sources still hash to what was counted
# (the counter summaries are profiles/pmc_traffic_*).
FETCH_SCALE, WRITE_SCALE = 1.9999, 1.0
TRAFFIC = {
    # workload 2 (n=20000, d=784)
    ("spmm_sym", 2, "packed"): (("csrc/spmm_sym.hip",), ("891ad7dd7a334b15",), 397407.718, 21343.150),
    ("spmm_sym", 2, "packed-f16"): (("csrc/spmm_sym.hip",), ("891ad7dd7a334b15",), 198961.010, 21342.954),
    ("spmm_onehot", 2, "resident"): (("csrc/cluster_ops.hip",), ("ffc98cf809a2ba97",), 782834.6, 1578.0),
    # workload 3 (n=60000, d=780)
    ("spmm_sym", 3, "packed"): (("csrc/spmm_sym.hip",), ("891ad7dd7a334b15",), 3529196.106, 93745.717),
    ("spmm_onehot", 3, "resident"): (("csrc/cluster_ops.hip",), ("ffc98cf809a2ba97",), 7035962.829, 14074.69),
    ("gemm_kappa", 3, "packed"): (("csrc/gemm_kappa.hip", "csrc/tile_mma.h"),
                                  ("cd3f5d45226675f0", "366f902efcd9e5e8"), 22316348.562, 7053978.375),
    ("gemm_kappa", 3, "resident"): (("csrc/gemm_kappa.hip", "csrc/tile_mma.h"),
                                    ("cd3f5d45226675f0", "366f902efcd9e5e8"), 22302415.188, 14070234.375),
    # workload 4 (n=100000, d=128, k=64)
    ("spmm_sym", 4, "packed"): (("csrc/spmm_sym.hip",), ("891ad7dd7a334b15",), 9801771.536, 361881.540),
    ("gemm_kappa", 4, "packed"): (("csrc/gemm_kappa.hip", "csrc/tile_mma.h"),
                                  ("cd3f5d45226675f0", "366f902efcd9e5e8"), 9804441.500, 19721405.719),
    # workload 5 (n=200000, d=54)
    ("spmm_sym", 5, "packed"): (("csrc/spmm_sym.hip",), ("891ad7dd7a334b15",), 39117459.279, 886687.096),
    ("spmm_onehot", 5, "resident"): (("csrc/cluster_ops.hip",), ("ffc98cf809a2ba97",), 78128224.638, 153234.375),
    ("gemm_kappa", 5, "packed"): (("csrc/gemm_kappa.hip", "csrc/tile_mma.h"),
                                  ("cd3f5d45226675f0", "366f902efcd9e5e8"), 2543482.312, 78225773.438),
    ("gemm_kappa", 5, "resident"): (("csrc/gemm_kappa.hip", "csrc/tile_mma.h"),
                                    ("cd3f5d45226675f0", "366f902efcd9e5e8"), 2530310.188, 156250781.250),
}


def counted_traffic(kernel, cfg, mode):
    """Scaled HBM bytes per launch (GB) if the counters match the current sources, else None."""
    import hashlib
    entry = TRAFFIC.get((kernel, cfg, mode))
    if entry is None:
        return None
    srcs, hashes, fetch_kib, write_kib = entry
    for src, h in zip(srcs, hashes):
        path = os.path.join(ROOT, "paper_2601_17136_amd", src)
        if hashlib.sha256(open(path, "rb").read()).hexdigest()[:16] != h:
            return None
    return round((fetch_kib * FETCH_SCALE + write_kib * WRITE_SCALE) * 1024 / 1e9, 4)


def time_seeding(kkm, ctx, n, k, d_pad, reps=5):
    """K-means++ seeding on the built context (not part of the timed steps):
    events on the context's stream around whole calls, so no launch inside is
    bracketed.  Each of its k distance passes reads the staged points once
    (n * d_pad * 4 bytes), the algorithmic bytes of the roofline figure."""
    import numpy as np
    import torch
    u = np.random.default_rng(4242).random(k)
    V = torch.empty(n, dtype=torch.int32, device="cuda")
    kkm.kkm_init_kmeanspp(ctx, k, u, V)  # first call allocates the scratch
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms = []
    for _ in range(reps):
        a.record()
        kkm.kkm_init_kmeanspp(ctx, k, u, V)
        b.record()
        b.synchronize()
        ms.append(a.elapsed_time(b))
    t = min(ms)
    gbs = k * n * d_pad * 4 / (t * 1e-3) / 1e9
    return {"ms": round(t, 4), "k": k, "launches": 2 * k - 1, "bound": "hbm", "achieved": round(gbs, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
            "work": "k passes over the staged points, n * d_pad * 4 bytes each"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=5,
                    help="workload 1-5 (default 5: n=200000, d=54, k=7, the largest)")
    ap.add_argument("--mode", choices=["packed", "resident", "onthefly"], default=None,
                    help="K storage (default: the planner's choice for the workload's kernel, k and storage)")
    ap.add_argument("--storage", choices=["f32", "f16"], default="f32",
                    help="number format of the stored K (f16: binary16 with fp32 sums, a mixed-precision "
                         "option with its own error bound; the default keeps fp32)")
    ap.add_argument("--extra", default=None,
                    help="comma-separated further storage modes measured beside the headline, or none "
                         "(default: resident,onthefly for workload 5, none otherwise)")
    ap.add_argument("--extra-steps", type=int, default=3, help="timed jobs per further mode (after 1 warm-up)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="oracle sample sized for about this much host time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-timing", action="store_true", help="do not record per-kernel events")
    ap.add_argument("--panel", type=int, default=0, metavar="G",
                    help="measure one GPU's share of a G-GPU 1D split instead: GPU 0's column panel "
                         "of K (n x n/G), its build and its updates, without the exchanges")
    ap.add_argument("--block", type=int, default=0, metavar="Q",
                    help="measure one GPU's share of a Q x Q-GPU 1.5D split instead: GPU (0, 0)'s block "
                         "of K (n/Q x n/Q), its build and its updates, without the exchanges")
    ap.add_argument("--peaks", action="store_true",
                    help="measure the achievable peaks instead (16 GiB non-temporal streaming read and "
                         "write, fp32 MFMA register loop, the packed SpMM's load pattern alone over 80 GB) "
                         "and print them as one JSON line")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="first run one plain device-to-device copy of MIB MiB (a known-size "
                         "reference for memory-traffic counters)")
    return ap.parse_args()


def cpu_baseline_sized(w, X, cl0, seconds):
    """Pilot on 256 rows, then a sample sized for about ``seconds`` of host work
    (at most 4 GB of fp64 kernel rows)."""
    pilot = cpu_baseline(w, X, cl0, 256)
    per_row = (w.iters / pilot["value"]) / X.shape[0]      # seconds of oracle work per row
    cap = max(256, int(4e9 / (8.0 * X.shape[0])))
    rows = int(min(X.shape[0], cap, max(256, seconds / max(per_row, 1e-9))))
    return cpu_baseline(w, X, cl0, rows)


def cpu_baseline(w, X, cl0, rows):
    """The oracle (fp64 kernel entries from their definitions + NumPy steps) on a
    row sample: K rows and w.iters updates restricted to those rows, scaled by
    n / rows to the whole job (labelled extrapolated when rows < n).  The
    self-terms z are taken from the sample rows' own-cluster sums (what the
    update needs besides E)."""
    import numpy as np

    from oracle import kkm_oracle as oracle
    n = X.shape[0]
    rows = min(rows, n)
    rng = np.random.default_rng(7)
    sample = np.sort(rng.choice(n, size=rows, replace=False)).astype(np.int64)
    kern = oracle.Kernel(w.kind, w.gamma, w.coef0, w.degree)
    t0 = time.perf_counter()
    K_rows = kern.block(X, sample, None)
    diag = kern.pairs(X, sample, sample)
    t1 = time.perf_counter()
    cl = cl0.copy()
    fixed = 0.0   # per-update work over all n points (sizes, one-hot ids): not scaled by n / rows
    for _ in range(w.iters):
        ta = time.perf_counter()
        oracle.cluster_sizes(cl, w.k)
        oracle.one_hot(cl, w.k)
        fixed += time.perf_counter() - ta
        counts = oracle.cluster_sizes(cl, w.k)
        E = oracle.one_hot_product(K_rows, cl, w.k)
        own = oracle.mask(E, cl[sample])
        z = oracle.self_terms(own, cl[sample], np.maximum(oracle.cluster_sizes(cl[sample], w.k), 1))
        D = oracle.distances(diag, E, z, counts)
        new = oracle.assign(D)
        cl = cl.copy()
        cl[sample] = new
    t2 = time.perf_counter()
    scale = n / rows
    upd = (t2 - t1 - 2.0 * fixed)         # the oracle's own update calls, less their all-n part
    total = (t1 - t0) * scale + fixed + max(upd, 0.0) * scale
    threads = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
    how = "extrapolated" if rows < n else "measured"
    return {"value": w.iters / total, "unit": "iters/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "estimate": how,
            "sample": f"{how}: K rows and {w.iters} updates on {rows} of {n} rows (fp64), "
                      f"times scaled by n/rows={scale:.1f}: K {1e3 * (t1 - t0) * scale:.0f} ms, "
                      f"updates {1e3 * (fixed + max(upd, 0.0) * scale):.0f} ms "
                      f"(of which {1e3 * fixed:.0f} ms over all n points, not scaled)"}


def cpu_model() -> str:
    """The host CPU's model name (lscpu's "Model name"), for the oracle baseline."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def measure(args, w, X, cl0, mode, steps, warmup, kkm, torch):
    """One storage mode: `warmup` + `steps` whole jobs (build + w.iters updates),
    the timed ones with no launch bracketed; then, unless --no-timing, as many
    jobs again with HIP events around the dominant kernels only, and one job
    with every launch bracketed for the per-phase breakdown.  The context (and
    its K) is freed before returning, so the next mode has the memory."""
    n, d, k = w.n, w.d, w.k
    Xd = torch.from_numpy(X).cuda()
    V0 = torch.from_numpy(cl0).cuda()
    Vs = [V0.clone() for _ in range(steps + warmup)]
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    params = kkm.make_params(w.gamma, w.coef0, w.degree, kkm.MODES[mode], kkm.STORAGES[args.storage])
    kind = kkm.KINDS[w.kind]

    def job(V):
        kkm.kkm_build_kernel(ctx, Xd, n, d, kind, params)
        return kkm.kkm_iterate(ctx, V, k, w.iters, -1.0)

    res = {}
    try:
        for s in range(warmup):
            job(Vs[s])
            print(f"bench: {mode}: warmup step {s} done", file=sys.stderr, flush=True)
        # Timed steps, uninstrumented: a HIP event bracket costs several us of
        # stream time, so no kernel is bracketed here.
        kkm.kkm_set_timing(ctx, 0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            it, hist = job(Vs[warmup + s])
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        assert it == w.iters
        info = kkm.kkm_get_info(ctx)
        print(f"bench: {mode}: timed {steps} steps in {t1 - t0:.3f} s", file=sys.stderr, flush=True)
        ms_per_step = 1e3 * (t1 - t0) / steps
        res.update(value=w.iters / (ms_per_step / 1e3), ms_per_step=ms_per_step, steps=steps, warmup=warmup,
                   info=info, J_final=float(hist[-1]))
        # The update loop alone, uninstrumented, on the K the last job built;
        # short jobs run 200 updates, so the call's own fixed cost (the label
        # pass, the copy of the ids and the final synchronisation) is spread thin.
        n_loop = max(w.iters, 200) if ms_per_step < 100 else w.iters
        V = V0.clone()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        kkm.kkm_iterate(ctx, V, k, n_loop, -1.0)
        torch.cuda.synchronize()
        res["loop_ms_per_update"] = 1e3 * (time.perf_counter() - t0) / n_loop
        res["loop_updates"] = n_loop
        if not args.no_timing:
            # Kernel durations for the roofline: the same jobs again with events
            # around the dominant kernels only.
            kkm.kkm_set_timing(ctx, kkm.phase_mask("gemm", "spmm", "onthefly"))
            for s in range(steps):
                job(V0.clone())
            res["phases"] = kkm.kkm_get_timing(ctx)
            # One more job with every launch bracketed, for the per-phase breakdown.
            kkm.kkm_set_timing(ctx, kkm.KKM_TIME_ALL)
            job(V0.clone())
            res["breakdown"] = kkm.kkm_get_timing(ctx)
            kkm.kkm_set_timing(ctx, 0)
            res["kmeanspp"] = time_seeding(kkm, ctx, n, k, info["d_pad"])
    finally:
        kkm.kkm_destroy(ctx)
        del Xd, V0, Vs
        torch.cuda.empty_cache()
    return res


def roofline_fields(args, w, mode, res):
    """The roofline objects of one measured mode (needs its event timings)."""
    n, d = w.n, w.d
    phases, breakdown = res["phases"], res["breakdown"]

    def avg(ph):
        ms, cnt = phases[ph]
        return (ms / cnt if cnt else float("nan")), cnt

    f16 = args.storage == "f16"
    traffic_tag = "-f16" if f16 else ""   # counted traffic is kept per storage format
    out = {}
    spmm_ms, spmm_cnt = avg("spmm")
    gemm_ms, gemm_cnt = avg("gemm")
    kbuild_ms = sum(breakdown[p][0] for p in ("stage", "gemm", "fixup"))
    iter_ms = sum(breakdown[p][0] for p in ("labels", "scatter", "spmm", "reduce", "assign", "onthefly", "other"))
    flops = float(n) * (n + 1) * d                     # symmetric half of X X^T, 2 flops per MAC
    out["kbuild_ms"] = round(kbuild_ms, 4)
    out["kbuild_tflops"] = round(flops / (gemm_ms * 1e-3) / 1e12, 3) if gemm_cnt else None
    out["kbuild_frac_mfma"] = round(out["kbuild_tflops"] / FP32_MFMA_PEAK_TF, 4) if out["kbuild_tflops"] else None
    # per update: the uninstrumented loop (a launch bracketed by events costs
    # a few us of stream time, which counts on the small workloads), and the
    # sum of the bracketed launches of one job
    out["update_ms"] = round(res["loop_ms_per_update"], 4)
    out["updates_per_s_loop"] = round(1e3 / res["loop_ms_per_update"], 2)
    out["loop_updates"] = res["loop_updates"]
    out["update_ms_bracketed"] = round(iter_ms / w.iters, 4)
    from paper_2601_17136_amd.kkm import PHASES
    out["phases_ms_one_step"] = {p: round(breakdown[p][0], 4) for p in PHASES if breakdown[p][1]}
    if mode in ("resident", "packed"):
        # K streamed once per update: all of it, or its upper triangle
        # n(n+1)/2 (what symmetry leaves to read; the stored diagonal
        # tiles and column padding count against the kernel)
        kname = "spmm_onehot" if mode == "resident" else "spmm_sym"
        esize = 2.0 if f16 else 4.0   # bytes per stored entry
        bytes_per = esize * n * n if mode == "resident" else esize * n * (n + 1) / 2
        gbs = bytes_per / (spmm_ms * 1e-3) / 1e9
        out["roofline"] = {"kernel": kname, "bound": "hbm", "achieved": round(gbs, 1),
                           "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                           "traffic": counted_traffic(kname, w.cfg, mode + traffic_tag),
                           "traffic_unit": "GB per launch (algorithmic %.4f)" % (bytes_per / 1e9),
                           "avg_launch_ms": round(spmm_ms, 5), "launches": spmm_cnt,
                           "stored_K_bytes": res["info"]["bytes_K"]}
    else:
        otf_ms, otf_cnt = avg("onthefly")
        otf_tf = flops / (otf_ms * 1e-3) / 1e12   # the symmetric half, per update
        out["roofline"] = {"kernel": "onthefly", "bound": "mfma", "achieved": round(otf_tf, 2),
                           "peak": FP32_MFMA_PEAK_TF, "unit": "TFLOP/s",
                           "frac": round(otf_tf / FP32_MFMA_PEAK_TF, 4),
                           "traffic": counted_traffic("onthefly", w.cfg, mode),
                           "traffic_unit": "GB per launch", "avg_launch_ms": round(otf_ms, 5),
                           "launches": otf_cnt,
                           "work": "n(n+1)d flop per update (symmetric half of X X^T)"}
    tf = out["kbuild_tflops"]
    if gemm_cnt:
        out["roofline_kbuild"] = {"kernel": "gemm_kappa", "bound": "mfma", "achieved": tf,
                                  "peak": FP32_MFMA_PEAK_TF, "unit": "TFLOP/s",
                                  "frac": round(tf / FP32_MFMA_PEAK_TF, 4) if tf else None,
                                  "traffic": counted_traffic("gemm_kappa", w.cfg, mode + traffic_tag),
                                  "traffic_unit": "GB per launch", "avg_launch_ms": round(gemm_ms, 5),
                                  "work": "n(n+1)d flop (symmetric half of X X^T)",
                                  "gauss_fixups": res["info"]["fixups"]}
        if mode == "resident" or (mode == "packed" and not f16):
            # the write roof: the stored bytes of K at the HBM peak
            wbytes = float(res["info"]["bytes_K"])
            out["roofline_kbuild"]["write_gbs"] = round(wbytes / (gemm_ms * 1e-3) / 1e9, 1)
            out["roofline_kbuild"]["write_frac"] = round(wbytes / (gemm_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the engine is single-GPU; multi-GPU sharding is a design note, not built)", file=sys.stderr)
        sys.exit(2)
    import numpy as np  # noqa: F401
    import torch

    from paper_2601_17136_amd import datagen, kkm

    w = datagen.WORKLOADS[args.config]
    if args.mode is None:
        # the mode the library's planner (AUTO) picks for this workload on one
        # MI355X's memory (288 GB less 5%)
        m, _ = kkm.kkm_plan(w.n, w.d, w.k, kkm.KINDS[w.kind], int(0.95 * (288 << 30)), kkm.KKM_MODE_AUTO,
                            kkm.STORAGES[args.storage])
        args.mode = {v: name for name, v in kkm.MODES.items()}[m]
    extra = [m for m in (args.extra.split(",") if args.extra is not None else
                         (["resident", "onthefly"] if args.config == 5 else []))
             if m and m != "none" and m != args.mode]
    X, _ = datagen.make_points(args.config)
    cl0 = datagen.make_init(args.config, w.n, w.k)
    n, d, k = w.n, w.d, w.k
    print(f"bench: {w.describe()} mode={args.mode} steps={args.steps} warmup={args.warmup} "
          f"extra={','.join(extra) or '-'}", file=sys.stderr, flush=True)

    torch.cuda.set_device(0)
    torch.cuda.empty_cache()
    if args.copy_calibration > 0:
        src = torch.ones(args.copy_calibration << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"bench: calibration copy of {args.copy_calibration} MiB done", file=sys.stderr, flush=True)
        del src, dst
        torch.cuda.empty_cache()
    if args.peaks:
        peaks_main(kkm, torch)
        return
    if args.panel:
        panel_main(args, w, X, cl0, kkm, torch)
        return
    if args.block:
        block_main(args, w, X, cl0, kkm, torch)
        return

    res = measure(args, w, X, cl0, args.mode, args.steps, args.warmup, kkm, torch)
    f16 = args.storage == "f16"
    value, ms_per_step = res["value"], res["ms_per_step"]
    out = {"metric": METRIC, "value": round(value, 3), "unit": "iters/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic",
           "config": {"workload": w.describe() + f", K {args.mode}" + (", binary16 K" if f16 else ""),
                      "n": n, "d": d, "k": k, "iters": w.iters, "kernel": w.kind, "mode": args.mode,
                      "storage": args.storage, "parallelism": "1 GPU"}}
    if not args.no_timing:
        out.update(roofline_fields(args, w, args.mode, res))
        out["kmeanspp"] = res["kmeanspp"]
    # The other storage modes of the same workload (the resident K and the
    # on-the-fly sweep of workload 5): fewer jobs each, reported beside the
    # headline under their own keys.
    for m in extra:
        steps_x, warm_x = max(1, min(args.steps, args.extra_steps)), 1
        rx = measure(args, w, X, cl0, m, steps_x, warm_x, kkm, torch)
        key = {"resident": "run_resident", "onthefly": "run_onthefly", "packed": "run_packed"}[m]
        ent = {"mode": m, "value": round(rx["value"], 3), "unit": "iters/s", "steps": steps_x,
               "warmup": warm_x, "ms_per_step": round(rx["ms_per_step"], 4),
               "stored_K_bytes": rx["info"]["bytes_K"]}
        if not args.no_timing:
            ent.update(roofline_fields(args, w, m, rx))
        out[key] = ent
    if not args.no_cpu_baseline:
        print("bench: timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline_sized(w, X, cl0, args.cpu_seconds)
    print(json.dumps(out), flush=True)


ROWS_CHUNKS, ROWS_SEGS, ROWS_SEG = 1562, 49, 2048   # 199936 x 100352 fp32 = 80.3 GB


def peak_row_orders(nrows, seed=5):
    """Row tables for the row-pattern read: cluster-sorted (k = 7 random labels,
    members in index order, cut into 128-row chunks that may straddle two
    clusters), random, and consecutive."""
    import numpy as np
    rng = np.random.default_rng(seed)
    lab = rng.integers(0, 7, nrows)
    return {"cluster_sorted_k7": np.lexsort((np.arange(nrows), lab)).astype(np.int32),
            "random": rng.permutation(nrows).astype(np.int32),
            "consecutive": np.arange(nrows, dtype=np.int32)}


def peaks_main(kkm, torch):
    """What this GPU sustains, for the roofline fractions against measured peaks:
    a 16 GiB streaming read and write with non-temporal 16-byte accesses, and a
    register loop of v_mfma_f32_32x32x2_f32 (about 18 ms per launch, long enough
    for the clocks to settle); then the packed SpMM's load pattern alone over an
    80 GB matrix (workload 5's footprint) in three row orders.  One warm-up
    launch each, then the average of 5."""
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    rows_res = {}
    try:
        buf = torch.empty(4 << 30, dtype=torch.float32, device="cuda")   # 16 GiB
        sums = torch.zeros(kkm.PEAK_READ_GROUPS, dtype=torch.float32, device="cuda")
        kkm.kkm_peak_write(ctx, buf, 1.0, 1)
        w_ms = kkm.kkm_peak_write(ctx, buf, 1.0, 5)
        kkm.kkm_peak_read(ctx, buf, sums, 1)
        r_ms = kkm.kkm_peak_read(ctx, buf, sums, 5)
        read_ok = float(sums.double().sum().item()) == float(buf.numel())
        nbytes = buf.numel() * 4
        del buf
        out = torch.zeros(4096, dtype=torch.float32, device="cuda")
        kkm.kkm_peak_mfma(ctx, 40000, out, 1)
        m_ms, flops = kkm.kkm_peak_mfma(ctx, 40000, out, 5)
        A = torch.empty((ROWS_CHUNKS * 128, ROWS_SEGS * ROWS_SEG), dtype=torch.float32, device="cuda")
        kkm.kkm_peak_write(ctx, A, 1.0, 1)
        rsums = torch.zeros(ROWS_CHUNKS * ROWS_SEGS, dtype=torch.float32, device="cuda")
        for name, order in peak_row_orders(A.shape[0]).items():
            R = torch.from_numpy(order).cuda()
            kkm.kkm_peak_read_rows(ctx, A, R, ROWS_SEG, rsums, 1)
            ms = kkm.kkm_peak_read_rows(ctx, A, R, ROWS_SEG, rsums, 5)
            gbs = A.numel() * 4 / (ms * 1e-3) / 1e9
            rows_res[name] = {"GBps": round(gbs, 1), "frac_of_8TBps": round(gbs / 8e3, 4), "ms": round(ms, 4),
                              "sums_exact": bool((rsums == 128.0 * ROWS_SEG).all())}
            print(f"bench: row-pattern read, {name}: {gbs:.1f} GB/s", file=sys.stderr, flush=True)
        rows_bytes = A.numel() * 4
        del A
    finally:
        kkm.kkm_destroy(ctx)
    res = {"metric": "achievable peaks (measurement aids, not the clustering path)",
           "read_GBps": round(nbytes / (r_ms * 1e-3) / 1e9, 1), "write_GBps": round(nbytes / (w_ms * 1e-3) / 1e9, 1),
           "mfma_f32_TFLOPs": round(flops / (m_ms * 1e-3) / 1e12, 2),
           "read_frac_of_8TBps": round(nbytes / (r_ms * 1e-3) / 8e12, 4),
           "write_frac_of_8TBps": round(nbytes / (w_ms * 1e-3) / 8e12, 4),
           "mfma_frac_of_157.3TF": round(flops / (m_ms * 1e-3) / 157.3e12, 4),
           "bytes": nbytes, "read_ms": round(r_ms, 4), "write_ms": round(w_ms, 4), "mfma_ms": round(m_ms, 4),
           "mfma_flop_per_launch": flops, "read_sums_exact": read_ok,
           "row_pattern_read": {"bytes": rows_bytes, "rows": ROWS_CHUNKS * 128, "ld": ROWS_SEGS * ROWS_SEG,
                                "segment_floats": ROWS_SEG, "orders": rows_res}}
    print(json.dumps(res), flush=True)


def panel_main(args, w, X, cl0, kkm, torch):
    """One GPU's share of a G-GPU 1D split at its real shape: GPU 0's points
    [0, c1) (the first of G ranges cut at multiples of 128), the column panel
    K[:, 0:c1] built and updated on this GPU.  The exchanges a multi-GPU run
    adds (an all-reduce of k doubles, an all-gather of 4n bytes) are replaced
    by their local stand-ins: this GPU's z parts alone, and its new ids copied
    into the id vector."""
    import numpy as np
    n, d, k, G = w.n, w.d, w.k, args.panel
    c1 = n if G == 1 else max(128, (n // G) // 128 * 128)
    Xd = torch.from_numpy(X).cuda()
    V = torch.from_numpy(cl0).cuda()
    cl_out = torch.empty(c1, dtype=torch.int32, device="cuda")
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    params = kkm.make_params(w.gamma, w.coef0, w.degree, kkm.KKM_MODE_RESIDENT)
    kind = kkm.KINDS[w.kind]

    def build():
        kkm.kkm_build_panel(ctx, Xd, n, d, kind, params, 0, c1)

    def update():
        zpart, counts = kkm.kkm_panel_spmm(ctx, V, k)
        c = counts.astype(np.float64)
        z = np.where(counts > 0, zpart / np.where(counts > 0, c * c, 1.0), 0.0)
        kkm.kkm_panel_assign(ctx, k, z, cl_out)
        V[:c1].copy_(cl_out)

    for _ in range(args.warmup):
        build()
        update()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        build()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(args.steps * w.iters):
        update()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    kkm.kkm_set_timing(ctx, kkm.phase_mask("gemm", "spmm"))
    build()
    for _ in range(w.iters):
        update()
    ph = kkm.kkm_get_timing(ctx)
    kkm.kkm_set_timing(ctx, 0)
    kkm.kkm_destroy(ctx)
    upd_ms = 1e3 * (t2 - t1) / (args.steps * w.iters)
    build_ms = 1e3 * (t1 - t0) / args.steps
    spmm_ms = ph["spmm"][0] / max(ph["spmm"][1], 1)
    gemm_ms = ph["gemm"][0] / max(ph["gemm"][1], 1)
    nbytes = 4.0 * n * c1                      # the panel, read once per update
    flops = 2.0 * n * c1 * d                   # every tile of the panel (no symmetry inside it)
    gbs = nbytes / (spmm_ms * 1e-3) / 1e9
    tf = flops / (gemm_ms * 1e-3) / 1e12
    out = {"metric": "one GPU's share of a %d-GPU 1D split: updates/s of its panel" % G,
           "value": round(1e3 / upd_ms, 3), "unit": "updates/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(upd_ms, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": w.describe() + f", GPU 0 of {G}: column panel K[:, 0:{c1}]",
                      "n": n, "d": d, "k": k, "panel_points": c1, "panel_bytes": int(nbytes),
                      "parallelism": f"1 GPU's share of {G} (exchanges not included)"},
           "panel_build_ms": round(build_ms, 4),
           "roofline": {"kernel": "spmm_onehot (panel)", "bound": "hbm", "achieved": round(gbs, 1),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                        "traffic": None, "traffic_unit": "GB per launch (algorithmic %.3f)" % (nbytes / 1e9),
                        "avg_launch_ms": round(spmm_ms, 5), "launches": ph["spmm"][1]},
           "roofline_kbuild": {"kernel": "gemm_kappa (panel)", "bound": "mfma", "achieved": round(tf, 2),
                               "peak": FP32_MFMA_PEAK_TF, "unit": "TFLOP/s",
                               "frac": round(tf / FP32_MFMA_PEAK_TF, 4), "avg_launch_ms": round(gemm_ms, 5),
                               "work": "2 n c1 d flop (the panel's tiles)"}}
    print(json.dumps(out), flush=True)


def block_main(args, w, X, cl0, kkm, torch):
    """One GPU's share of a Q x Q-GPU 1.5D split at its real shape: grid
    position (0, 0), whose block is K[0:b, 0:b] for the first of Q point
    ranges cut at multiples of 128, and whose piece of the 1D partition is
    the first Q-th of that range.  The exchanges a multi-GPU run adds (the
    all-gather of row-block ids, the reduce-scatter of the partial E, the
    all-reduce of 2k words) are replaced by local stand-ins: this GPU's own
    partial E for its piece, its own z parts and sizes, and its new ids
    copied into the id vector."""
    import numpy as np
    n, d, k, Q = w.n, w.d, w.k, args.block
    b = n if Q == 1 else max(128, (n // Q) // 128 * 128)
    a1 = max(1, b // Q)                        # the piece [0, a1)
    Xd = torch.from_numpy(X).cuda()
    V = torch.from_numpy(cl0).cuda()
    part = torch.empty((b, k), device="cuda")
    cl_out = torch.empty(a1, dtype=torch.int32, device="cuda")
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    params = kkm.make_params(w.gamma, w.coef0, w.degree, kkm.KKM_MODE_RESIDENT)
    kind = kkm.KINDS[w.kind]

    def build():
        kkm.kkm_build_block(ctx, Xd, n, d, kind, params, 0, b, 0, b)

    def update():
        kkm.kkm_block_spmm(ctx, V[:b], k, part)
        Ep = part[:a1]
        zpart, counts = kkm.kkm_block_zpart(ctx, Ep, V[:a1], 0, a1, k)
        c = counts.astype(np.float64)
        z = np.where(counts > 0, zpart / np.where(counts > 0, c * c, 1.0), 0.0)
        kkm.kkm_block_assign(ctx, Ep, 0, a1, k, z, counts, cl_out)
        V[:a1].copy_(cl_out)

    for _ in range(args.warmup):
        build()
        update()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        build()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(args.steps * w.iters):
        update()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    kkm.kkm_set_timing(ctx, kkm.phase_mask("gemm", "spmm"))
    build()
    for _ in range(w.iters):
        update()
    ph = kkm.kkm_get_timing(ctx)
    kkm.kkm_set_timing(ctx, 0)
    kkm.kkm_destroy(ctx)
    upd_ms = 1e3 * (t2 - t1) / (args.steps * w.iters)
    build_ms = 1e3 * (t1 - t0) / args.steps
    spmm_ms = ph["spmm"][0] / max(ph["spmm"][1], 1)
    gemm_ms = ph["gemm"][0] / max(ph["gemm"][1], 1)
    nbytes = 4.0 * b * b                       # the block, read once per update
    flops = 2.0 * b * b * d                    # every tile of the block
    gbs = nbytes / (spmm_ms * 1e-3) / 1e9
    tf = flops / (gemm_ms * 1e-3) / 1e12
    out = {"metric": "one GPU's share of a %dx%d-GPU 1.5D split: updates/s of its block" % (Q, Q),
           "value": round(1e3 / upd_ms, 3), "unit": "updates/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(upd_ms, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": w.describe() + f", GPU (0, 0) of {Q}x{Q}: block K[0:{b}, 0:{b}], "
                                                 f"piece [0, {a1})",
                      "n": n, "d": d, "k": k, "block_points": b, "piece_points": a1, "block_bytes": int(nbytes),
                      "parallelism": f"1 GPU's share of {Q * Q} (exchanges not included)"},
           "block_build_ms": round(build_ms, 4),
           "roofline": {"kernel": "spmm_onehot (block)", "bound": "hbm", "achieved": round(gbs, 1),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                        "traffic": None, "traffic_unit": "GB per launch (algorithmic %.3f)" % (nbytes / 1e9),
                        "avg_launch_ms": round(spmm_ms, 5), "launches": ph["spmm"][1]},
           "roofline_kbuild": {"kernel": "gemm_kappa (block)", "bound": "mfma", "achieved": round(tf, 2),
                               "peak": FP32_MFMA_PEAK_TF, "unit": "TFLOP/s",
                               "frac": round(tf / FP32_MFMA_PEAK_TF, 4), "avg_launch_ms": round(gemm_ms, 5),
                               "work": "2 b^2 d flop (the block's tiles)"}}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
