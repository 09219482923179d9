#!/usr/bin/env python3
"""ROCKET transform throughput on one MI355X.

One step = one full transform pass over the workload's series (every row,
every kernel: X[n, L] -> F[n, 2K]) with X already resident in HBM.  Prints
one JSON line: series x kernels per second, the roofline position of the
fused kernel (fp32 MFMA bound, 157.3 TFLOP/s peak) and, on the side, the
fp64 oracle timed on this host's cores over a bounded row sample.

    python bench.py [--steps K] [--warmup W] [--workload manufacturing]
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_TFLOPS = 157.3      # MI355X dense fp32 (matrix and vector, published)
PEAK_FP32_FMA_NOPACK = 78.6   # fp32 vector FMA without packed instructions
F_RESIDENT_LIMIT = 16 << 30   # above this the feature matrix is streamed in row batches
DEFAULT_BATCH_ROWS = 100000


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


class ClockSampler:
    """The GPU's shader (GFX) clock, read from the AMD SMI library in a
    background thread while the timed passes run (the device is found by its
    PCI address).  The SMI refreshes its readings about once a second, and
    the first refresh after the start may still cover idle time before it,
    so only the readings from the second refresh inside the timed region on
    count: a region shorter than about two refreshes reports no clock.  The
    reading is the mean over the XCDs of their current GFX clocks (the
    per-XCD list of the GPU metrics table; the single clock reading where
    the table lacks it)."""

    def __init__(self, device_index=0, interval_s=0.02):
        import threading
        self.interval_s = interval_s
        self.samples = []  # (time, value in MHz, refresh signature)
        self._stop = threading.Event()
        self._thread = None
        self._smi = None
        self._handle = None
        self.error = None
        try:
            import amdsmi
            import torch
            pr = torch.cuda.get_device_properties(device_index)
            bdf = "%04x:%02x:%02x.0" % (pr.pci_domain_id, pr.pci_bus_id, pr.pci_device_id)
            amdsmi.amdsmi_init()
            self._smi = amdsmi
            self._handle = amdsmi.amdsmi_get_processor_handle_from_bdf(bdf)
            if self._read() is None:  # one read up front: fail here, not in the thread
                raise RuntimeError("no GFX clock reading")
        except Exception as e:  # no SMI access: the line says so
            self.error = "%s: %s" % (type(e).__name__, e)
            self._handle = None

    def _read(self):
        try:
            m = self._smi.amdsmi_get_gpu_metrics_info(self._handle)
            xcd = [float(c) for c in (m.get("current_gfxclks") or []) if isinstance(c, (int, float)) and c > 0]
            if xcd:
                return float(np.mean(xcd)), tuple(xcd)
        except Exception:
            pass
        info = self._smi.amdsmi_get_clock_info(self._handle, self._smi.AmdSmiClkType.GFX)
        clk = info.get("clk")
        return (float(clk), (float(clk),)) if isinstance(clk, (int, float)) and clk > 0 else None

    def _run(self):
        while not self._stop.is_set():
            try:
                r = self._read()
                if r is not None:
                    self.samples.append((time.perf_counter(), r[0], r[1]))
            except Exception as e:
                self.error = "%s: %s" % (type(e).__name__, e)
                return
            self._stop.wait(self.interval_s)

    def start(self):
        if self._handle is not None:
            import threading
            self._thread = threading.Thread(target=self._run, daemon=True)
            self._thread.start()
        return self

    def stop(self, t_end=None):
        """Readings taken after t_end (a perf_counter time: when the device
        went idle) are dropped."""
        if self._thread is not None:
            self._stop.set()
            self._thread.join()
        if self._smi is not None:
            try:
                self._smi.amdsmi_shut_down()
            except Exception:
                pass
        if self._handle is None:
            return {"mhz": None, "source": "amdsmi (unavailable: %s)" % self.error}
        pts = [(v, sig) for t, v, sig in self.samples if t_end is None or t <= t_end]
        refresh = [i for i in range(1, len(pts)) if pts[i][1] != pts[i - 1][1]]
        if len(refresh) < 2:
            return {"mhz": None, "refreshes": len(refresh),
                    "source": "amdsmi GFX clock: the timed region saw fewer than two refreshes of the "
                              "SMI readings (about one a second)"}
        a = np.array([v for v, _ in pts[refresh[1]:]])
        return {"mhz": float(np.median(a)), "min": float(a.min()), "max": float(a.max()),
                "refreshes": len(refresh) - 1,
                "source": "amdsmi GFX clock (mean over XCDs), read every %d ms during the timed passes, "
                          "from the second SMI refresh inside them on" % int(self.interval_s * 1e3)}


def timed_passes(torch, stream, one_pass, steps):
    """Time `steps` calls of one_pass on `stream`: a HIP event between
    consecutive passes (all on the launch stream), synchronised before and
    after.  Returns (total ms, per-pass ms list, clock record)."""
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    clock = ClockSampler()
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(steps):
        one_pass()
        evs[i + 1].record(stream)
        if i == 0:
            clock.start()  # the device is busy from here on
    torch.cuda.synchronize()
    clk = clock.stop(t_end=time.perf_counter())
    per = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    return evs[0].elapsed_time(evs[-1]), per, clk


def pass_stats(per):
    a = np.array(per, dtype=np.float64)
    return {"median": float(np.median(a)), "min": float(a.min()), "max": float(a.max()), "n": int(a.size)}


def valid_taps(kernels, L):
    """Products whose series index lands inside [0, L) (padding zeros excluded),
    summed over kernels (and, for multivariate sets, over the channels each
    kernel reads): the algorithmic FMA count of one series."""
    ln = kernels["length"].astype(np.int64)
    d = kernels["dilation"].astype(np.int64)
    p = kernels["padding"].astype(np.int64)
    ch = (kernels["channel_count"].astype(np.int64) if int(kernels.get("n_channels", 1)) > 1
          else np.ones_like(ln))
    O = L + 2 * p - (ln - 1) * d
    total = 0
    for j in range(11):
        on = j < ln
        lo = np.maximum(0, p - j * d)
        hi = np.minimum(O, p - j * d + L)
        total += int((np.where(on, np.maximum(0, hi - lo), 0) * ch).sum())
    nominal = int((ln * O * ch).sum())
    return total, nominal


def source_digest():
    h = hashlib.sha256()
    for name in ("transform.hip", "plan.cpp", "rocket_internal.h", "minirocket.cpp"):
        with open(os.path.join(ROOT, "paper_2601_17091_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload, digest, kernel="rocket_fused_kernel"):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it
    was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "%s_%s_pmc.json" % (kernel, workload))
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_digest") != digest:
        return None
    return rec.get("hbm_bytes_per_launch")


def add_clock_frac(out):
    """The roofline fraction against the peak at the shader clock the timed
    passes ran at (the published peak assumes 2.4 GHz), when it was read."""
    mhz = out.get("sclk_mhz")
    out["roofline"]["frac_at_sclk"] = (out["roofline"]["frac"] * 2400.0 / mhz) if mhz else None


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="manufacturing")
    ap.add_argument("--batch-rows", type=int, default=0,
                    help="rows per F batch (0: whole F if it fits %d GiB)" % (F_RESIDENT_LIMIT >> 30))
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle sample budget")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--direct", action="store_true", help="time the plain kernel instead")
    ap.add_argument("--mpv", action="store_true",
                    help="also compute the third feature, MPV (F has 3 columns per kernel)")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="also run one elementwise copy of this many MiB (reference for "
                         "hardware byte counters)")
    ap.add_argument("--sweep", action="store_true",
                    help="time the paper's one-factor sweep instead (n, L, K around "
                         "1,000 x 10,000 x 10,000), device-resident and host-to-host")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the transform runs on a single MI355X "
              "(rows would shard across GPUs with no exchange). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2601_17091_amd as rk
    from paper_2601_17091_amd.workloads import WORKLOADS, sample_rows, workload_series

    if args.sweep:
        return sweep(args)
    if args.workload == "minirocket":
        return bench_minirocket(args)

    if not os.path.exists(rk.rocket.LIB_PATH):
        from paper_2601_17091_amd import build_lib
        build_lib.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    props = torch.cuda.get_device_properties(dev)

    log("workload %s: n=%d L=%d K=%d" % (w.name, w.n, w.L, w.n_kernels))
    if w.channels > 1:
        ks = rk.generate_kernels_multi(w.kernel_seed, w.n_kernels, w.L, w.channels)
    else:
        ks = rk.generate_kernels(w.kernel_seed, w.n_kernels, w.L)
    t0 = time.perf_counter()
    X_np = workload_series(w.name)
    log("series generated in %.1f s" % (time.perf_counter() - t0))
    X = torch.from_numpy(X_np).to(dev)

    t0 = time.perf_counter()
    plan = rk.Plan(ks, w.L, direct=args.direct, mpv=args.mpv)
    torch.cuda.synchronize()
    plan_ms = (time.perf_counter() - t0) * 1e3
    info = plan.info()
    log("plan: %s (%.1f ms)" % (info, plan_ms))

    K2 = plan.n_features
    batch = args.batch_rows or (w.n if w.n * K2 * 4 <= F_RESIDENT_LIMIT else DEFAULT_BATCH_ROWS)
    batch = min(batch, w.n)
    F = torch.empty((batch, K2), dtype=torch.float32, device=dev)
    n_batches = (w.n + batch - 1) // batch
    stream = torch.cuda.current_stream()

    def one_pass():
        for r0 in range(0, w.n, batch):
            nb = min(batch, w.n - r0)
            plan.transform_into(X[r0:r0 + nb], F[:nb], stream)

    if args.copy_mb > 0:
        src = torch.ones(args.copy_mb << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        log("copy reference: %d MiB read, %d MiB written" % (args.copy_mb, args.copy_mb))
        del src, dst

    for i in range(args.warmup):
        one_pass()
        torch.cuda.synchronize()
        log("warmup %d/%d done" % (i + 1, args.warmup))
    torch.cuda.synchronize()
    total_ms, per_pass, clock = timed_passes(torch, stream, one_pass, args.steps)
    ms_per_step = total_ms / args.steps
    log("timed %d passes: %.3f ms per pass (median %.3f), shader clock %s" % (
        args.steps, ms_per_step, float(np.median(per_pass)), clock))

    valid_per_row, nominal_per_row = valid_taps(ks, w.L)
    flops_per_pass = 2.0 * w.n * valid_per_row
    launches = n_batches
    per_launch_ms = ms_per_step / launches
    achieved = (flops_per_pass / launches) / (per_launch_ms * 1e-3) / 1e12
    mfma_fma_per_pass = 256.0 * info["mfma_per_row"] * w.n
    pairs_per_s = w.n * w.n_kernels / (ms_per_step * 1e-3)
    digest = source_digest()
    # the layout the timed calls ran: series-lane for short univariate series
    # in calls of at least 4,096 series (then a permutation kernel writes F)
    series_path = bool(info.get("series_lane")) and batch >= 4096
    traffic = None if (args.direct or args.mpv) else traffic_from_profile(
        w.name, digest, "rocket_series_kernel" if series_path else "rocket_fused_kernel")

    # parity of sampled rows and the CPU baseline on the same rows
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        from oracle import rocket_oracle
        rocket_oracle.build()
        threads = rocket_oracle.max_threads()
        rng_rows = sample_rows(w.n, batch, 4096)
        t0 = time.perf_counter()
        rocket_oracle.transform(X_np, ks, rows=rng_rows[:2], threads=threads)
        per_row = max((time.perf_counter() - t0) / 2.0, 1e-6)
        m = int(max(2, min(rng_rows.shape[0], args.cpu_seconds / per_row * threads)))
        rows = np.unique(np.concatenate([rng_rows[:2], rng_rows[-2:],
                                         np.random.default_rng(3).choice(rng_rows, m, replace=False)]))
        log("oracle on %d rows (%d threads)" % (rows.shape[0], threads))
        t0 = time.perf_counter()
        ref = rocket_oracle.transform(X_np, ks, rows=rows, threads=threads)
        cpu_s = time.perf_counter() - t0
        cpu = {"value": rows.shape[0] * w.n_kernels / cpu_s, "unit": "series*kernels/s",
               "cores": threads, "kind": "oracle",
               "sample": "%d of %d %s rows (first/last row, first/last of each batch, seeded "
                         "random), all %d kernels, fp64, %.1f s" % (rows.shape[0], w.n, w.name,
                                                                     w.n_kernels, cpu_s)}
        cpu["single_thread"] = single_thread_rate(rocket_oracle.transform, X_np, ks, rows, per_row, threads,
                                                  w.n_kernels, args.cpu_seconds / 5)
        # GPU features of the same rows
        got = np.zeros((rows.shape[0], K2), np.float32)
        for r0 in range(0, w.n, batch):
            nb = min(batch, w.n - r0)
            sel = rows[(rows >= r0) & (rows < r0 + nb)]
            if sel.size == 0:
                continue
            plan.transform_into(X[r0:r0 + nb], F[:nb], stream)
            torch.cuda.synchronize()
            got[np.searchsorted(rows, sel)] = F[torch.from_numpy(sel - r0).to(dev)].cpu().numpy()
        O = ref["O"][None, :]
        nf = plan.features_per_kernel
        ppv, mxv = got[:, 0::nf], got[:, 1::nf]
        cnt = np.rint(ppv.astype(np.float64) * O)
        parity = {
            "rows": int(rows.shape[0]),
            "max_abs_err_max": float(np.abs(mxv - ref["F"][:, 1::2]).max()),
            "max_count_err": int(np.abs(cnt - ref["cnt"]).max()),
            "outside_certified": int(((cnt < ref["cnt_lo"]) | (cnt > ref["cnt_hi"])).sum()
                                     + (np.abs(mxv - ref["F"][:, 1::2]) > ref["beta"]).sum()),
        }
        if nf == 3:
            mpv = got[:, 2::3].astype(np.float64)
            parity["mpv_outside_certified"] = int(((mpv < ref["mpv_lo"]) | (mpv > ref["mpv_hi"])).sum())
            same = cnt == ref["cnt"]
            # error beyond the test rule 1e-4 * MPV + beta (0 when inside)
            excess = np.abs(mpv - ref["mpv"]) - (1e-4 * np.abs(ref["mpv"]) + ref["beta"])
            parity["mpv_max_excess_over_rule"] = float(max(0.0, excess[same].max()))
        log("parity %s" % parity)

    path = "direct" if info["direct"] else ("series-lane-mfma" if series_path else "fused-mfma")
    kernel_name = ("rocket_direct_kernel" if info["direct"] else
                   ("rocket_series_kernel + rocket_slot_permute_kernel" if series_path else
                    ("rocket_fused_kernel + rocket_toeplitz_kernel" if info.get("toeplitz_items") else
                     "rocket_fused_kernel")))
    out = {
        "metric": "series*kernels/s (ROCKET transform, fp32, 1 MI355X)",
        "value": pairs_per_s,
        "unit": "series*kernels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic (seeded %s series, z-normalised; seeded ROCKET kernels)" % w.kind,
        "config": {"workload": w.name, "n_series": w.n, "series_length": w.L, "channels": w.channels,
                   "n_kernels": w.n_kernels, "features": K2, "f_batch_rows": batch,
                   "kernel_seed": w.kernel_seed, "data_seed": w.data_seed,
                   "path": path},
        "pct_fp32_peak": 100.0 * achieved / PEAK_FP32_TFLOPS,
        "pct_fp32_fma_nopack_peak": 100.0 * achieved / PEAK_FP32_FMA_NOPACK,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_FP32_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_TFLOPS, "traffic": traffic,
                     "kernel": kernel_name,
                     "launches_per_step": launches, "launch_ms": per_launch_ms,
                     "algorithmic_flops_per_launch": flops_per_pass / launches,
                     "valid_fma_per_series": valid_per_row,
                     "nominal_fma_per_series": nominal_per_row,
                     "mfma_fma_issued_per_series": 256 * info["mfma_per_row"],
                     "valu_fma_issued_per_series": 64 * info.get("valu_fma_per_row", 0),
                     "mfma_pipe_frac": mfma_fma_issued_frac(mfma_fma_per_pass, ms_per_step),
                     "hbm_gbps": (traffic / (per_launch_ms * 1e-3) / 1e9) if traffic else None},
        "pass_ms": pass_stats(per_pass),
        "sclk_mhz": clock["mhz"],
        "sclk": clock,
        "plan": dict(info, create_ms=plan_ms),
        "device": {"name": props.name, "cu": props.multi_processor_count},
        "source_digest": digest,
        "cpu_baseline": cpu,
        "parity": parity,
    }
    add_clock_frac(out)
    print(json.dumps(out), flush=True)


def single_thread_rate(fn, X_np, params, rows, per_row_all_threads, threads, per_row_units, seconds):
    """The oracle on one thread over the first rows of the sample, sized to
    about `seconds`: units (series x kernels or features) per second."""
    # per_row_all_threads was timed on two rows, which keep at most two
    # threads busy: about one thread's time per row
    m = int(max(1, min(rows.shape[0], seconds / max(per_row_all_threads, 1e-6))))
    t0 = time.perf_counter()
    fn(X_np, params, rows=rows[:m], threads=1)
    dt = time.perf_counter() - t0
    return {"value": m * per_row_units / dt, "rows": m, "seconds": dt}


def minirocket_valid_taps(params, L):
    """Algorithmic FMAs of one series under MINIROCKET: the valid taps of
    every (dilation, kernel) pair, counted once per pair (its biases share
    the pair's dot products)."""
    total = 0
    for i, d in enumerate(params["dilations"]):
        if int(params["features_per_dilation"][i]) == 0:
            continue
        d = int(d)
        for k in range(84):
            p = 4 * d if (i + k) % 2 == 0 else 0
            O = L + 2 * p - 8 * d
            for j in range(9):
                lo, hi = max(0, p - j * d), min(O, p - j * d + L)
                total += max(0, hi - lo)
    return total


PEAK_COMPARE_TOPS = 256 * 4 * 64 * 2.4e9 / 4 / 1e12  # fp32 compares: one 64-lane VALU op per SIMD per 4 cycles


def minirocket_compares(params, L):
    """Algorithmic compares of one series under MINIROCKET: one per (feature,
    output), C_t > b (each feature's count needs every one of them)."""
    total = 0
    for i, d in enumerate(params["dilations"]):
        nf = int(params["features_per_dilation"][i])
        for k in range(84):
            O = L if (i + k) % 2 == 0 else L - 8 * int(d)
            total += nf * O
    return total


def bench_minirocket(args):
    """MINIROCKET (Sec. 5 names it): the manufacturing workload's 100,000
    series of 1,000 samples, 10,000 features fitted on the first 1,000
    series; one step = one transform pass over every series (F [n,
    n_features] of PPVs)."""
    import torch

    import paper_2601_17091_amd as rk
    from paper_2601_17091_amd.workloads import WORKLOADS, sample_rows, workload_series

    if not os.path.exists(rk.rocket.LIB_PATH):
        from paper_2601_17091_amd import build_lib
        build_lib.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = WORKLOADS["minirocket"]
    dev = torch.device("cuda:0")
    props = torch.cuda.get_device_properties(dev)
    log("workload minirocket: n=%d L=%d features requested=%d" % (w.n, w.L, w.n_kernels))
    t0 = time.perf_counter()
    X_np = workload_series(w.name)
    log("series generated in %.1f s" % (time.perf_counter() - t0))
    t0 = time.perf_counter()
    params = rk.minirocket_fit(X_np[:1000], w.n_kernels, w.kernel_seed)
    fit_ms = (time.perf_counter() - t0) * 1e3
    nf = int(params["biases"].shape[0])
    log("fit on 1000 series: %d dilations, %d features (%.1f ms)" % (len(params["dilations"]), nf, fit_ms))
    X = torch.from_numpy(X_np).to(dev)
    t0 = time.perf_counter()
    plan = rk.MiniRocketPlan(params)
    torch.cuda.synchronize()
    plan_ms = (time.perf_counter() - t0) * 1e3
    info = plan.info()
    log("plan: %s (%.1f ms)" % (info, plan_ms))
    F = torch.empty((w.n, nf), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    if args.copy_mb > 0:
        src = torch.ones(args.copy_mb << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        log("copy reference: %d MiB read, %d MiB written" % (args.copy_mb, args.copy_mb))
        del src, dst
    for i in range(args.warmup):
        plan.transform_into(X, F, stream)
        torch.cuda.synchronize()
        log("warmup %d/%d done" % (i + 1, args.warmup))
    total_ms, per_pass, clock = timed_passes(torch, stream, lambda: plan.transform_into(X, F, stream),
                                             max(args.steps, 1))
    ms = total_ms / max(args.steps, 1)
    log("timed %d passes: %.3f ms per pass, shader clock %s" % (args.steps, ms, clock))
    valid = minirocket_valid_taps(params, w.L)
    flops = 2.0 * w.n * valid
    achieved = flops / (ms * 1e-3) / 1e12
    compares = float(w.n) * minirocket_compares(params, w.L)
    cmp_rate = compares / (ms * 1e-3) / 1e12
    digest = source_digest()
    mr_traffic = traffic_from_profile("minirocket", digest, "rocket_minirocket_kernel")
    cpu = parity = None
    if not args.no_cpu_baseline:
        from oracle import minirocket_oracle, rocket_oracle
        rocket_oracle.build()
        threads = rocket_oracle.max_threads()
        rng_rows = sample_rows(w.n, w.n, 4096)
        t0 = time.perf_counter()
        minirocket_oracle.transform(X_np, params, rows=rng_rows[:2], threads=threads)
        per_row = max((time.perf_counter() - t0) / 2.0, 1e-6)
        m = int(max(2, min(rng_rows.shape[0], args.cpu_seconds / per_row * threads)))
        rows = np.unique(np.concatenate([rng_rows[:2], rng_rows[-2:],
                                         np.random.default_rng(3).choice(rng_rows, m, replace=False)]))
        log("oracle on %d rows (%d threads)" % (rows.shape[0], threads))
        t0 = time.perf_counter()
        ref = minirocket_oracle.transform(X_np, params, rows=rows, threads=threads)
        cpu_s = time.perf_counter() - t0
        cpu = {"value": rows.shape[0] * nf / cpu_s, "unit": "series*features/s", "cores": threads,
               "kind": "oracle",
               "sample": "%d of %d minirocket rows (first/last row, seeded random), all %d features, fp64, "
                         "%.1f s" % (rows.shape[0], w.n, nf, cpu_s)}
        cpu["single_thread"] = single_thread_rate(minirocket_oracle.transform, X_np, params, rows, per_row,
                                                  threads, nf, args.cpu_seconds / 5)
        plan.transform_into(X, F, stream)
        torch.cuda.synchronize()
        got = F[torch.from_numpy(rows).to(dev)].cpu().numpy().astype(np.float64)
        cnt = np.rint(got * ref["O"][None, :])
        parity = {"rows": int(rows.shape[0]), "max_count_err": int(np.abs(cnt - ref["cnt"]).max()),
                  "outside_certified": int(((cnt < ref["cnt_lo"]) | (cnt > ref["cnt_hi"])).sum())}
        log("parity %s" % parity)
    out = {
        "metric": "series*features/s (MINIROCKET transform, fp32, 1 MI355X)",
        "value": w.n * nf / (ms * 1e-3),
        "unit": "series*features/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp32",
        "data": "synthetic (seeded ar1 series, z-normalised; MINIROCKET fitted on the first 1000)",
        "config": {"workload": "minirocket", "n_series": w.n, "series_length": w.L, "features": nf,
                   "dilations": [int(d) for d in params["dilations"]], "fit_seed": w.kernel_seed,
                   "data_seed": w.data_seed, "fit_ms": fit_ms},
        "pct_fp32_peak": 100.0 * achieved / PEAK_FP32_TFLOPS,
        "algorithmic_tflops": achieved,
        # the kernel is bound by its compares (vector unit) and their
        # popcounts (scalar unit); its roofline is the compare rate of the
        # vector unit, one fp32 compare per lane per issue slot
        "roofline": {"bound": "alu", "achieved": cmp_rate, "peak": PEAK_COMPARE_TOPS, "unit": "Tcompare/s",
                     "frac": cmp_rate / PEAK_COMPARE_TOPS,
                     "algorithmic_compares_per_launch": compares,
                     "traffic": mr_traffic,
                     "hbm_gbps": (mr_traffic / (ms * 1e-3) / 1e9) if mr_traffic else None,
                     "kernel": "rocket_minirocket_kernel", "launches_per_step": 1, "launch_ms": ms,
                     "algorithmic_flops_per_launch": flops, "valid_fma_per_series": valid},
        "pass_ms": pass_stats(per_pass),
        "sclk_mhz": clock["mhz"],
        "sclk": clock,
        "plan": dict(info, create_ms=plan_ms),
        "device": {"name": props.name, "cu": props.multi_processor_count},
        "source_digest": digest,
        "cpu_baseline": cpu,
        "parity": parity,
    }
    add_clock_frac(out)
    print(json.dumps(out), flush=True)


SWEEP_DEFAULT = (1000, 10000, 10000)
SWEEP_POINTS = ([SWEEP_DEFAULT]
                + [(n, 10000, 10000) for n in (100, 500, 2000)]
                + [(1000, L, 10000) for L in (1000, 5000, 20000)]
                + [(1000, 10000, K) for K in (1000, 5000, 20000)])


def sweep(args):
    """The paper's timing sweep (Sec. 4): defaults n = 1,000 series, length
    L = 10,000, K = 10,000 kernels, one factor varied at a time.  Each point
    is timed with the series resident on the device, and host-to-host with
    pinned buffers through rocket_transform_host (copies overlapped with
    the transform).  The paper finds time linear in n, L and K; the line
    reports time per series x kernel x sample relative to the default."""
    import torch

    import paper_2601_17091_amd as rk
    from paper_2601_17091_amd.workloads import make_series

    dev = torch.device("cuda:0")
    points = []
    for (n, L, K) in SWEEP_POINTS:
        ks = rk.generate_kernels(206, K, L)
        X_np = make_series("random_walk", n, L, 106)
        X = torch.from_numpy(X_np).to(dev)
        plan = rk.Plan(ks, L)
        info = plan.info()
        F = torch.empty((n, 2 * K), dtype=torch.float32, device=dev)
        stream = torch.cuda.current_stream()
        for _ in range(max(1, args.warmup)):
            plan.transform_into(X, F, stream)
        torch.cuda.synchronize()
        reps = max(1, args.steps)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            plan.transform_into(X, F, stream)
        t1.record(stream)
        torch.cuda.synchronize()
        dev_ms = t0.elapsed_time(t1) / reps
        Xh = torch.empty((n, L), dtype=torch.float32, pin_memory=True)
        Xh.copy_(torch.from_numpy(X_np))
        Fh = torch.empty((n, 2 * K), dtype=torch.float32, pin_memory=True)
        plan.transform_host(Xh, Fh)
        h_reps = 2
        w0 = time.perf_counter()
        for _ in range(h_reps):
            plan.transform_host(Xh, Fh)
        host_ms = (time.perf_counter() - w0) * 1e3 / h_reps
        same = bool(torch.equal(Fh, F.cpu()))
        valid, _ = valid_taps(ks, L)
        flops = 2.0 * n * valid
        pt = {"n": n, "L": L, "K": K, "device_ms": dev_ms, "host_to_host_ms": host_ms,
              "host_matches_device": same, "tflops": flops / (dev_ms * 1e-3) / 1e12,
              "series_kernels_per_s": n * K / (dev_ms * 1e-3),
              "ns_per_series_kernel_sample": dev_ms * 1e6 / (n * K * L),
              "clamped": info["clamped"], "direct": info["direct"], "toeplitz_items": info["toeplitz_items"]}
        log("sweep %s" % json.dumps(pt))
        points.append(pt)
        plan.close()
        del X, F, Xh, Fh
    base = points[0]["ns_per_series_kernel_sample"]
    rel = [p["ns_per_series_kernel_sample"] / base for p in points]
    for p, r in zip(points, rel):
        p["time_per_unit_vs_default"] = r
    # per factor: the exponent of a least-squares fit log(time) = a + e log(x)
    # over the points that vary it (with the default point); 1 is linear
    exponents = {}
    d0 = SWEEP_POINTS[0]
    for i, name in enumerate(("n", "L", "K")):
        sel = [p for p, q in zip(points, SWEEP_POINTS)
               if all(q[j] == d0[j] for j in range(3) if j != i)]
        x = np.log([float(p[name]) for p in sel])
        y = np.log([p["device_ms"] for p in sel])
        exponents[name] = float(np.polyfit(x, y, 1)[0]) if len(sel) > 1 else None
    out = {"metric": "ROCKET transform time over the paper's n/L/K sweep (fp32, 1 MI355X)",
           "unit": "ms", "dtype": "fp32", "data": "synthetic (seeded random walks; seeded ROCKET kernels)",
           "config": {"workload": "paper_sweep", "default": {"n": 1000, "L": 10000, "K": 10000}},
           "points": points,
           "linearity": {"time_per_unit_vs_default_min": min(rel), "time_per_unit_vs_default_max": max(rel),
                         "time_exponent": exponents},
           "source_digest": source_digest()}
    print(json.dumps(out), flush=True)


def mfma_fma_issued_frac(fma_per_pass, ms_per_step):
    """Share of the fp32 MFMA peak the issued MFMA work (incl. padding and
    empty slots) represents."""
    return 2.0 * fma_per_pass / (ms_per_step * 1e-3) / 1e12 / PEAK_FP32_TFLOPS


if __name__ == "__main__":
    main()
