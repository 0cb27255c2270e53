#!/usr/bin/env python3
"""Throughput of the multiple-double product C = A.B on one MI355X.

One step = one ``mdgemm_ex`` call over the whole path (row/column exponents,
exact splits of A and B, the level GEMMs on the FP64 matrix cores, exact
accumulation and rounding), with A, B, C and the workspace resident in HBM.

Prints one JSON line:
* ``value``: effective multiple-double GFLOP/s = 2 m n k / (time per step);
* ``roofline``: the level-GEMM kernel (the dominant one) against the FP64 MFMA
  peak: algorithmic flops 2 m n k |pairs| per launch over its average duration
  from HIP events recorded on the launch stream around it in every timed step;
  ``traffic`` is the HBM bytes per launch from the committed rocprofv3 counter
  summary of this kernel and workload, or null when the kernel source changed
  after the counters were taken;
* ``stages``: every stage's average time and algorithmic rate;
* ``adaptive_width``: the same workload with the adaptive digit width (fewer,
  wider digits whose level sums stay exact at this k; at least the digit bits of
  four 13-bit digits per limb), timed over a few steps; the headline ``value``
  keeps the workload's 13-bit digits unless ``--slice-bits`` says otherwise;
* ``calibration``: the FP64 MFMA rate and the HBM copy rate measured on the
  same device in the same run (the library's probe kernels), beside the
  published 78.6 TFLOP/s and 8 TB/s; ``roofline.frac_of_measured`` is taken
  against the former; every memory-bound stage gets ``frac_of_peak`` (against
  8 TB/s) and ``frac_of_probe``, against the library's plain stream probe run
  at the stage's own size and read/write mix (``probe_GB/s``, ``probe_mix``);
* ``parity``: outside the timed region, the last timed step's C at sampled
  entries (corners, the rows and columns of extreme exponents, random ones)
  against the CPU oracle's chain (bit-exact limbs) and against the exact
  rational product (largest error over the stated tolerance);
* ``exponent_classes`` (workloads with a range, c7): the same product grouped
  by exponent class over that range (section 3's balancing), timed over a few
  steps, with a sampled parity check against the oracle's grouped chain;
* ``karatsuba`` (the Karatsuba schedule of the level products: fewer
  products, bit-identical limbs) and ``int8`` (the level products of 7-bit
  digits on the int8 matrix cores, within the same error bound), a few timed
  steps each beside the headline, which keeps the paper's separate pair
  products on the FP64 matrix cores;
* ``--extras`` adds ``karatsuba_adaptive``, ``sign_groups`` (section 3's
  sign grouping, four products, the same limbs), ``taylor_dd`` (the QR's
  application to power-series systems, timed) and ``qr_dd`` (the
  double-double Householder QR built on the product) lines;
* ``cpu_baseline``: the CPU oracle's classic multiple-double GEMM (one
  sequential inner product per element, all host cores) timed on a bounded
  sample of the same product's rows.
"""

from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_F64_PEAK_TFLOPS = 78.6  # MI355X dense FP64 matrix peak (published)
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E (published)
INT8_PEAK_TOPS = 5000.0  # MI355X dense int8 matrix peak (published)
METRIC = "effective dd/qd GEMM GFLOP/s; % FP64 MFMA peak; bit-exact+tol vs CPU oracle"
# the level-GEMM kernel is built from its source and the tile constants of internal.h
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_06881_amd", "csrc", "slice_gemm.hip")
GEMM_CONSTANTS = os.path.join(ROOT, "paper_2607_06881_amd", "csrc", "internal.h")
DEFAULT_CONFIG = "c2"


def kernel_source_hash() -> str:
    """First 16 hex digits of the sha256 of the level-GEMM source followed by the
    lines of internal.h that define its tile constants (``constexpr int kTile``)."""
    h = hashlib.sha256()
    with open(GEMM_SOURCE, "rb") as fh:
        h.update(fh.read())
    with open(GEMM_CONSTANTS, "rb") as fh:
        for ln in fh:
            if ln.lstrip().startswith(b"constexpr int kTile"):
                h.update(ln)
    return h.hexdigest()[:16]


def stored_traffic(config: str):
    """HBM bytes per level-GEMM launch from profiles/slice_gemm_<config>_pmc.txt
    (lines ``key = value``), if its recorded source hash matches the kernel."""
    path = os.path.join(ROOT, "profiles", f"slice_gemm_{config}_pmc.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for ln in fh:
            if "=" in ln and not ln.lstrip().startswith("#"):
                key, v = ln.split("=", 1)
                vals[key.strip()] = v.strip()
    if vals.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def calibrate(md, torch, dev, stream):
    """Measured FP64 MFMA rate (TFLOP/s) and copy rate (GB/s, read + write) of this device."""
    sink = torch.empty(2048 * 256, dtype=torch.float64, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    md.mdgemm_probe_mfma_f64(sink, 200, stream=stream)  # warm-up
    e0.record(stream)
    flops = md.mdgemm_probe_mfma_f64(sink, 20000, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    mfma = flops / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del sink
    n = 1 << 28  # 2 GiB per buffer
    src = torch.ones(n, dtype=torch.float64, device=dev)
    dst = torch.empty_like(src)
    md.mdgemm_probe_copy(src, dst, stream=stream)
    e0.record(stream)
    reps = 5
    for _ in range(reps):
        md.mdgemm_probe_copy(src, dst, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    copy = 2.0 * 8.0 * n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    return {"mfma_f64_TFLOP/s": round(mfma, 2), "mfma_f64_published_TFLOP/s": MFMA_F64_PEAK_TFLOPS,
            "copy_GB/s": round(copy, 1), "hbm_published_GB/s": HBM_PEAK_GBS,
            "probes": "mdgemm_probe_mfma_f64 (2048 x 256 threads, 8 independent v_mfma_f64_16x16x4f64 chains per "
                      "wave, 20000 rounds); mdgemm_probe_copy (2 GiB, read + write bytes, 5 copies)"}


def stage_probes(md, torch, dev, stream, mixes, reps=3):
    """The library's plain stream probe at each memory-bound stage's own size and
    read/write mix (count elements, reads and writes planes of doubles each)."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {}
    for key, (count, reads, writes) in mixes.items():
        src = torch.ones(reads * count, dtype=torch.float64, device=dev)
        dst = torch.empty(writes * count, dtype=torch.float64, device=dev) if writes else None
        md.mdgemm_probe_stream(src, reads, dst, writes, count, stream=stream)  # warm-up
        e0.record(stream)
        for _ in range(reps):
            md.mdgemm_probe_stream(src, reads, dst, writes, count, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        gbs = 8.0 * count * (reads + writes) * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
        out[key] = {"GB/s": round(gbs, 1), "count": count, "reads": reads, "writes": writes}
        del src, dst
    return out


def taylor_dd_line(md, torch, dev, stream, no_cpu, n=1024, r=64, d=8, reps=3):
    """The QR's application: the Taylor coefficients of the solution of
    A(t) X(t) = B(t) modulo t^(d+1) (mdgemm_taylor_dd) for a seeded series of
    n x n double-double coefficients (A_i normal / sqrt(n), A_0 + 2 I, so A_0 is
    well conditioned) and n x r right-hand sides, timed with HIP events around
    the call; its parity is the Taylor tests'.  Beside it, the oracle's
    degree-by-degree QR solve of a 128 x 128, r = 8, d = 4 series (CPU)."""
    import numpy as np

    def series(nn, rr, dd, seed):
        rng = np.random.default_rng(seed)
        A = rng.standard_normal((dd + 1, 2, nn, nn)) / np.sqrt(nn)
        A[:, 1] *= 2.0 ** -60 * rng.uniform(-1, 1, size=(dd + 1, nn, nn))
        A[0, 0] += 2.0 * np.eye(nn)
        B = rng.standard_normal((dd + 1, 2, nn, rr))
        B[:, 1] *= 2.0 ** -60 * rng.uniform(-1, 1, size=(dd + 1, nn, rr))
        return A, B

    A_h, B_h = series(n, r, d, 7)
    Ag, Bg = torch.from_numpy(A_h).to(dev), torch.from_numpy(B_h).to(dev)
    need = int(md.lib().mdgemm_taylor_dd_workspace_bytes(n, r, d))
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    X = md.mdgemm_taylor_dd(Ag, Bg, workspace=ws, stream=stream)  # warm-up
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        e0.record(stream)
        md.mdgemm_taylor_dd(Ag, Bg, X=X, workspace=ws, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    res = {"n": n, "r": r, "d": d, "ms": round(float(np.median(times)), 3), "workspace_bytes": need}
    del ws, X, Ag, Bg
    if not no_cpu:
        from oracle import coracle

        a, b = series(128, 8, 4, 8)
        t0 = time.perf_counter()
        coracle.taylor_dd(a, b)
        res["cpu_oracle_128_r8_d4_ms"] = round((time.perf_counter() - t0) * 1e3, 1)
    return res


def qr_dd_line(md, torch, dev, stream, A, no_cpu, nb=64, reps=3):
    """The downstream use: blocked Householder QR (mdgemm_qr_dd) of the
    workload's double-double A, and of its leading 1024 x 1024 block.  Rate in
    effective double-double flops, 2 m n^2 - 2 n^3 / 3 per factorization (each
    double-double operation counted once).  Its parity (residual and
    orthogonality in double-double against the CPU oracle) is the QR tests';
    beside it, the oracle's unblocked QR on a 256 x 256 block (CPU)."""
    import numpy as np

    res = {"nb": nb}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for key, (mm, nn) in (("full", (A.shape[1], A.shape[2])), ("block_1024", (1024, 1024))):
        if nn > mm or mm > A.shape[1] or nn > A.shape[2]:
            continue
        src = A[:, :mm, :nn].contiguous()
        need = int(md.lib().mdgemm_qr_dd_workspace_bytes(mm, nn, nb))
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        work = src.clone()
        md.mdgemm_qr_dd(work, nb=nb, workspace=ws, stream=stream)  # warm-up
        times = []
        for _ in range(reps):
            work.copy_(src)
            torch.cuda.synchronize()
            e0.record(stream)
            md.mdgemm_qr_dd(work, nb=nb, workspace=ws, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        ms = float(np.median(times))
        flops = 2.0 * mm * nn * nn - 2.0 * nn ** 3 / 3.0
        res[key] = {"m": mm, "n": nn, "ms": round(ms, 3), "dd_GFLOP/s": round(flops / (ms * 1e-3) / 1e9, 2),
                    "workspace_bytes": need}
        del ws, work, src
    if not no_cpu:
        from oracle import coracle

        blk = A[:, :256, :256].cpu().numpy()
        t0 = time.perf_counter()
        coracle.qr_dd(blk)
        sec = time.perf_counter() - t0
        flops = 2.0 * 256 ** 3 - 2.0 * 256 ** 3 / 3.0
        res["cpu_oracle_256"] = {"seconds": round(sec, 3), "dd_GFLOP/s": round(flops / sec / 1e9, 4),
                                 "kind": "oracle", "sample": "unblocked double-double Householder QR, 256 x 256"}
    return res


def parity(w, A_h, B_h, C_h, S, T, bits, count=32):
    """The timed product's C at sampled entries against the CPU oracle (test
    infrastructure, outside the timed region): bit-exact greedy limbs of the
    oracle's chain, and the error against the exact rational product over the
    stated tolerance 4 k 2^-(53L-4) (|A||B|)_ij."""
    import numpy as np

    from oracle import coracle, exact, pipeline

    L, m, k = A_h.shape
    n = B_h.shape[2]
    EA, EB = coracle.exponents(A_h[0], 0), coracle.exponents(B_h[0], 1)
    rng = np.random.default_rng(w.seed + 1000)
    rows = {0, m - 1, int(np.argmin(EA)), int(np.argmax(EA))}
    cols = {0, n - 1, int(np.argmin(EB)), int(np.argmax(EB))}
    entries = {(i, j) for i in rows for j in cols}
    while len(entries) < count:
        entries.add((int(rng.integers(m)), int(rng.integers(n))))
    entries = sorted(entries)
    t0 = time.perf_counter()
    ref = pipeline.reference_entries(A_h, B_h, S, T, entries, bits)
    mismatch = [e for e in entries if C_h[:, e[0], e[1]].tolist() != ref[e]["limbs"]]
    worst = 0.0
    for (i, j) in entries:
        want, mag = exact.exact_product(A_h, B_h, i, j)
        err = abs(exact.value(C_h[:, i, j]) - want)
        bound = exact.tolerance(k, L, mag)
        if bound > 0:
            worst = max(worst, float(err / bound))
        elif err != 0:
            worst = float("inf")
    return {"entries": len(entries), "bit_exact_vs_oracle": not mismatch, "mismatches": len(mismatch),
            "max_err_over_tolerance": worst, "within_tolerance": worst <= 1.0,
            "tolerance": "4 k 2^-(53L-4) (|A||B|)_ij vs the exact rational product",
            "seconds": round(time.perf_counter() - t0, 2)}


def cpu_baseline(w, A, B, target_s: float):
    """Classic multiple-double GEMM of the CPU oracle on a sample of rows of C."""
    import numpy as np  # noqa: F401

    from oracle import coracle

    coracle.lib()
    # calibrate on one row per thread, four times more until the run lasts half a
    # second (or covers C), then size the sample to about target_s seconds
    threads = coracle.num_threads()
    rows = min(w.m, threads)
    while True:
        t = time.perf_counter()
        coracle.classic_gemm(A[:, :rows, :], B)
        dt = max(time.perf_counter() - t, 1e-3)
        if dt >= 0.5 or rows >= w.m:
            break
        rows = min(w.m, 4 * rows)
    rows = int(min(w.m, max(threads, rows * target_s / dt)))
    t = time.perf_counter()
    _, used = coracle.classic_gemm(A[:, :rows, :], B)
    dt = time.perf_counter() - t
    flops = 2.0 * rows * w.n * w.k
    return {
        "value": flops / dt / 1e9,
        "unit": "GFLOP/s",
        "cores": int(used),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": f"classic {'double-double (Dekker/Hida-Li-Bailey add+mul)' if w.limbs == 2 else f'{w.limbs}-limb exact-expansion'}"
                  f" GEMM, rows 0..{rows - 1} of C ({rows} x {w.n} x {w.k}), {dt:.1f} s on {used} threads",
        "seconds": dt,
    }


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=DEFAULT_CONFIG, help="workload c0..c7 (default c2)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--slice-bits", default="13",
                    help="digit width of the timed product: 13 (the workload's digits and cutoff, default), "
                         "'auto' (the adaptive width) or 14..26")
    ap.add_argument("--adaptive-steps", type=int, default=5,
                    help="steps of each extra measurement (adaptive width, Karatsuba schedule) reported beside "
                         "the headline (0: none)")
    ap.add_argument("--products", choices=("fp64", "int8"), default="fp64",
                    help="level products on the FP64 matrix cores (the paper's, default) or on the int8 "
                         "matrix cores (MDGEMM_INT8, 7-bit digits)")
    ap.add_argument("--schedule", choices=("pairs", "karatsuba"), default="pairs",
                    help="schedule of the level products of the timed product: the paper's digit pairs (default) "
                         "or the Karatsuba schedule")
    ap.add_argument("--extras", action="store_true",
                    help="also time the Karatsuba schedule and the int8 level products beside the headline")
    ap.add_argument("--no-calibration", action="store_true", help="skip the MFMA and copy probes")
    ap.add_argument("--no-parity", action="store_true", help="skip the sampled parity check of the timed C")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed steps, run 3 device copies of this many MiB (calibrates the HBM byte "
                         "counters of a profiler run against a known size)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on one GPU only (the product has no multi-GPU path); use --gpus 1",
              file=sys.stderr)
        return 2
    if args.products == "int8" and (args.schedule != "pairs" or args.slice_bits != "13"):
        print("bench.py: --products int8 takes its own digit width and the pair schedule", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2607_06881_amd import mdgemm as md
    from paper_2607_06881_amd import workloads

    w = workloads.WORKLOADS[args.config]
    dev = torch.device("cuda:0")
    md.lib()  # fail loudly if the HIP library is missing

    A_h, B_h = workloads.make_workload(w)
    A = torch.from_numpy(A_h).to(dev)
    B = torch.from_numpy(B_h).to(dev)
    C = torch.empty((w.limbs, w.m, w.n), dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()

    def mode_opts(slice_bits):
        """Options of one digit mode: the workload's 13-bit digits and cutoff, the
        adaptive width or an explicit width (with the workload's range balancing)."""
        if slice_bits == 13:
            return w.options()
        if slice_bits == md.MDGEMM_SLICE_BITS_AUTO:
            return w.options(adaptive=True)
        opts = {"slice_bits": slice_bits}
        if w.range_bits:
            opts["range_bits"] = w.range_bits
        return opts

    def measure(opts, steps, warmup, base_flags=0):
        """ms per step and per-stage ms of mdgemm_ex with these options: K steps
        back to back (torch events around them; the options are marshalled once
        and the C entry point called directly, so that a small product is not
        bound by the host), then K steps with the library's stage events
        (MDGEMM_TIME_STAGES, each step read back before the next)."""
        ws = torch.empty(max(1, md.mdgemm_workspace_bytes(w.m, w.n, w.k, w.limbs, flags=base_flags, **opts)),
                         dtype=torch.uint8, device=dev)
        o_plain = md.make_opts(flags=base_flags, stream=stream, workspace=ws, **opts)
        o_timed = md.make_opts(flags=base_flags | md.MDGEMM_TIME_STAGES, stream=stream, workspace=ws, **opts)
        lib = md.lib()
        L_, m_, k_ = A.shape
        n_ = B.shape[2]
        pa, pb, pc = A.data_ptr(), B.data_ptr(), C.data_ptr()
        ref_plain, ref_timed = ctypes.byref(o_plain), ctypes.byref(o_timed)

        def step(o):
            st = lib.mdgemm_ex(m_, n_, k_, L_, pa, pb, pc, o)
            if st != md.MDGEMM_OK:
                raise md.MdgemmError(st, "mdgemm_ex")

        for _ in range(warmup):
            step(ref_plain)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            step(ref_plain)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        stage_sum = np.zeros(4)
        for _ in range(steps):
            step(ref_timed)
            stage_sum += np.array(md.mdgemm_stage_times())  # waits for this step's last event
        torch.cuda.synchronize()
        del ws
        return ms, stage_sum / steps

    bits_arg = md.MDGEMM_SLICE_BITS_AUTO if args.slice_bits == "auto" else int(args.slice_bits)
    sched_flags = md.MDGEMM_KARATSUBA if args.schedule == "karatsuba" else 0
    int8 = args.products == "int8"
    if int8:
        sched_flags = md.MDGEMM_INT8
    opts = {"range_bits": w.range_bits} if int8 and w.range_bits else ({} if int8 else mode_opts(bits_arg))
    bits, S, T = md.mdgemm_plan(w.m, w.n, w.k, w.limbs, flags=sched_flags, **opts)
    ms_per_step, stage_ms = measure(opts, args.steps, args.warmup, sched_flags)
    C_h = None if args.no_parity else C.cpu().numpy()  # the last timed step's product, for the parity check

    if args.copy_probe_mib > 0:
        src = torch.ones(args.copy_probe_mib * (1 << 20) // 8, dtype=torch.float64, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    m, n, k, L = w.m, w.n, w.k, w.limbs
    pairs = workloads.pair_count(S, T)
    info = md.mdgemm_schedule_info(m, n, k, S, T, bits=bits, flags=0 if int8 else sched_flags)
    panels_f32 = bool(info["panels_f32"])  # digit panels kept in FP32 (every digit sum below 2^24)
    # small outputs run the fused small-product kernel (all five steps in one
    # launch), whose stages leave nothing in the workspace: the library refuses
    # to describe a workspace layout for them
    fused = False
    if not int8 and not sched_flags:
        try:
            md.mdgemm_workspace_layout(w.m, w.n, w.k, w.limbs, **opts)
        except md.MdgemmError:
            fused = True
    md_flops = w.md_flops()
    # the GEMMs actually run: one per digit pair, or the Karatsuba schedule's products
    slice_flops = 2.0 * m * n * k * info["terms"]
    value = md_flops / (ms_per_step * 1e-3) / 1e9

    bytes_exp = 8.0 * (m * k + k * n) + 4.0 * (m + n)
    pe = 4.0 if panels_f32 else 8.0  # bytes per panel value
    bytes_split = 8.0 * L * (m * k + k * n) + pe * S * (m * k + k * n) + 4.0 * (m + n)
    # the Karatsuba schedule's combinations (digit sums), written by the split beside the digits
    bytes_split += pe * k * ((info["combos_a"] - S) * m + (info["combos_b"] - S) * n)
    bytes_acc = 8.0 * info["planes"] * m * n + 8.0 * L * m * n + 4.0 * (m + n)
    gemm_ms = stage_ms[2]
    achieved = slice_flops / (gemm_ms * 1e-3) / 1e12
    if int8:
        # int8 digits (1 byte), B's also transposed once; int32 level planes
        bytes_split = 8.0 * L * (m * k + k * n) + S * (m * k + 3.0 * k * n) + 4.0 * (m + n)
        bytes_acc = 4.0 * info["planes"] * m * n + 8.0 * L * m * n + 4.0 * (m + n)
    roofline = {
        "bound": "mfma",
        "achieved": round(achieved, 3),
        "peak": MFMA_F64_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(achieved / MFMA_F64_PEAK_TFLOPS, 4),
        # the stored counters were taken with the workload's 13-bit digits and pair schedule
        "traffic": stored_traffic(args.config) if bits_arg == 13 and not sched_flags else None,
        "kernel": ("slice_gemm32_kernel (level GEMMs on FP32 digit panels, v_mfma_f64_16x16x4f64)"
                   if panels_f32 else "slice_gemm_kernel (level GEMMs on FP64 digit panels, v_mfma_f64_16x16x4f64)"),
        "flops_per_launch": slice_flops,
        "avg_launch_ms": round(gemm_ms, 4),
    }
    if int8:
        roofline.update({"peak": INT8_PEAK_TOPS, "unit": "TOP/s", "frac": round(achieved / INT8_PEAK_TOPS, 4),
                         "traffic": None,
                         "kernel": f"level_gemm_i8_kernel: int8 level products ({T + 1} levels, int32 sums) "
                                   "in one launch",
                         "ops_per_step": roofline.pop("flops_per_launch"),
                         "avg_step_ms": roofline.pop("avg_launch_ms")})
    if fused:
        roofline.update({"kernel": "small_product_kernel (the five steps fused per 16 x 16 tile of C, "
                                   "v_mfma_f64_16x16x4f64)", "traffic": None})
    stages = {
        "exponents": {"ms": round(stage_ms[0], 4), "GB/s": round(bytes_exp / (stage_ms[0] * 1e-3) / 1e9, 1),
                      "bytes": bytes_exp},
        "split": {"ms": round(stage_ms[1], 4), "GB/s": round(bytes_split / (stage_ms[1] * 1e-3) / 1e9, 1),
                  "bytes": bytes_split},
        "slice_gemm": {"ms": round(stage_ms[2], 4), ("TOP/s" if int8 else "TFLOP/s"): round(achieved, 3)},
        "accum_renorm": {"ms": round(stage_ms[3], 4), "GB/s": round(bytes_acc / (stage_ms[3] * 1e-3) / 1e9, 1),
                         "bytes": bytes_acc},
        "hbm_peak_GB/s": HBM_PEAK_GBS,
    }
    if fused:  # one kernel: its time is the level-product stage's, the others are event gaps
        stages = {"fused_small_product": {"ms": round(stage_ms[2], 4), "TFLOP/s": round(achieved, 3)},
                  "event_gaps_ms": [round(float(x), 4) for x in (stage_ms[0], stage_ms[1], stage_ms[3])]}
    config = {"workload": f"{w.name}: {w.description}", "m": m, "n": n, "k": k, "limbs": L, "slices": S,
              "cutoff": T, "pairs": pairs, "seed": w.seed, "panels": "f32" if panels_f32 else "f64"}
    if sched_flags and not int8:
        config["schedule"] = "karatsuba"
        config["products"] = info["terms"]
        config["workload"] += f"; Karatsuba schedule: {info['terms']} digit-sum products for the {pairs} pairs"
    if w.range_bits:
        config["range_bits"] = w.range_bits
    if int8:
        config["products"] = "int8"
        config["slice_bits"] = bits
        config["panels"] = "int8"
        config["workload"] += f"; int8 level products: {S} digits of {bits} bits, pairs p+q <= {T}"
    elif bits != 13:
        config["slice_bits"] = bits
        config["workload"] += f"; adaptive width: {S} digits of {bits} bits, pairs p+q <= {T}"
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8" if int8 else "f64",
        "data": "synthetic",
        "config": config,
        "roofline": roofline,
        "stages": stages,
        "slice_gemm_share": round(stage_ms[2] / stage_ms.sum(), 4),
    }
    def extra(a_opts, flags):
        """A few timed steps of the same workload with other digit options or schedule."""
        a_bits, a_S, a_T = md.mdgemm_plan(m, n, k, L, flags=flags, **a_opts)
        a_info = md.mdgemm_schedule_info(m, n, k, a_S, a_T, bits=a_bits, flags=flags)
        a_ms, a_stage = measure(a_opts, args.adaptive_steps, 2, flags)
        a_pairs = workloads.pair_count(a_S, a_T)
        a_tflops = 2.0 * m * n * k * a_info["terms"] / (a_stage[2] * 1e-3) / 1e12
        return {
            "slice_bits": a_bits, "slices": a_S, "cutoff": a_T, "pairs": a_pairs, "products": a_info["terms"],
            "planes": a_info["planes"], "steps": args.adaptive_steps, "ms_per_step": round(a_ms, 4),
            "value": round(md_flops / (a_ms * 1e-3) / 1e9, 3),
            "stage_ms": [round(float(x), 4) for x in a_stage],
            "slice_gemm_TFLOP/s": round(a_tflops, 3), "frac": round(a_tflops / MFMA_F64_PEAK_TFLOPS, 4),
        }

    def int8_mode():
        """A few timed steps of the same workload with the int8 level products."""
        i_opts = {"range_bits": w.range_bits} if w.range_bits else {}
        I8 = md.MDGEMM_INT8
        try:
            i_bits, i_S, i_T = md.mdgemm_plan(m, n, k, L, flags=I8, **i_opts)
        except md.MdgemmError as e:  # e.g. more than 8 limbs: S > 64 at 7 bits
            return {"skipped": str(e)}
        i_ms, i_stage = measure(i_opts, args.adaptive_steps, 2, I8)
        i_pairs = workloads.pair_count(i_S, i_T)
        tops = 2.0 * m * n * k * i_pairs / (i_stage[2] * 1e-3) / 1e12
        return {
            "slice_bits": i_bits, "slices": i_S, "cutoff": i_T, "pairs": i_pairs, "gemms": i_T + 1,
            "steps": args.adaptive_steps, "ms_per_step": round(i_ms, 4),
            "value": round(md_flops / (i_ms * 1e-3) / 1e9, 3),
            "stage_ms": [round(float(x), 4) for x in i_stage],
            "level_gemm_TOPS": round(tops, 1), "frac": round(tops / INT8_PEAK_TOPS, 4),
        }

    if not args.no_parity:
        out["parity"] = parity(w, A_h, B_h, C_h, S, T, bits)
    if not args.no_calibration:
        cal = calibrate(md, torch, dev, stream)
        out["calibration"] = cal
        roofline["peak_measured"] = cal["mfma_f64_TFLOP/s"]
        roofline["frac_of_measured"] = round(achieved / cal["mfma_f64_TFLOP/s"], 4)
        # every memory-bound stage against the published 8 TB/s and against a
        # plain stream of its own size and read/write mix (planes of doubles,
        # the stage's read and write bytes per element rounded to whole planes)
        if "split" in stages:
            cnt_s = m * k + k * n
            w_split = bytes_split - 8.0 * L * cnt_s - 4.0 * (m + n)
            mixes = {"exponents": (cnt_s, 1, 0),
                     "split": (cnt_s, L, max(1, round(w_split / (8.0 * cnt_s)))),
                     "accum_renorm": (m * n, max(1, round((bytes_acc - 8.0 * L * m * n - 4.0 * (m + n)) /
                                                          (8.0 * m * n))), L)}
            probes = stage_probes(md, torch, dev, stream, mixes)
            for key, pr in probes.items():
                stages[key]["frac_of_peak"] = round(stages[key]["GB/s"] / HBM_PEAK_GBS, 4)
                stages[key]["probe_GB/s"] = pr["GB/s"]
                stages[key]["frac_of_probe"] = round(stages[key]["GB/s"] / pr["GB/s"], 4)
                stages[key]["probe_mix"] = f"{pr['reads']} read + {pr['writes']} write planes of {pr['count']}"
    if bits_arg == 13 and not sched_flags and args.adaptive_steps > 0:
        # the same workload with the adaptive width reported beside the paper's
        # 13-bit digit pairs (and, on request, the Karatsuba schedule and the
        # int8 level products)
        out["adaptive_width"] = extra(mode_opts(md.MDGEMM_SLICE_BITS_AUTO), 0)
        out["karatsuba"] = extra(mode_opts(13), md.MDGEMM_KARATSUBA)
        out["int8"] = int8_mode()
        if args.extras:
            out["karatsuba_adaptive"] = extra(mode_opts(md.MDGEMM_SLICE_BITS_AUTO), md.MDGEMM_KARATSUBA)
    def grouped(g_flags):
        """A few timed steps of the same workload as a grouped product (section 3's
        exponent classes over the workload's range, or sign groups), with a
        sampled parity check against the oracle's grouped chain."""
        from oracle import exact as ex
        from oracle import pipeline as pl

        g_opts = {"range_bits": w.range_bits} if w.range_bits else {}
        g_bits, g_S, g_T = md.mdgemm_plan(m, n, k, L, flags=g_flags, **g_opts)
        classes = 1 + -(-w.range_bits // g_bits) if (g_flags & md.MDGEMM_GROUP_EXPONENT) and w.range_bits else 1
        groups = classes * (2 if g_flags & md.MDGEMM_GROUP_SIGN else 1)
        g_ms, g_stage = measure(g_opts, args.adaptive_steps, 1, g_flags)
        terms = groups * groups * workloads.pair_count(g_S, g_T)
        tflops = 2.0 * m * n * k * terms / (g_stage[2] * 1e-3) / 1e12
        res = {"classes": classes, "groups": groups, "slices": g_S, "cutoff": g_T, "levels": g_T + 1 + 2 * (classes - 1),
               "pairs": terms, "steps": args.adaptive_steps, "ms_per_step": round(g_ms, 4),
               "value": round(md_flops / (g_ms * 1e-3) / 1e9, 3), "stage_ms": [round(float(x), 4) for x in g_stage],
               "slice_gemm_TFLOP/s": round(tflops, 3), "frac": round(tflops / MFMA_F64_PEAK_TFLOPS, 4)}
        if not args.no_parity:
            Cg = C.cpu().numpy()
            rng = np.random.default_rng(w.seed + 2000)
            entries = sorted({(int(rng.integers(m)), int(rng.integers(n))) for _ in range(8)})
            ref = pl.reference_entries_groups(A_h, B_h, g_S, g_T, classes, bool(g_flags & md.MDGEMM_GROUP_SIGN),
                                              entries, g_bits)
            worst = 0.0
            for (i, j) in entries:
                want, mag = ex.exact_product(A_h, B_h, i, j)
                worst = max(worst, float(abs(ex.value(Cg[:, i, j]) - want) / ex.tolerance(k, L, mag)))
            res["parity"] = {"entries": len(entries),
                             "bit_exact_vs_oracle": all(Cg[:, i, j].tolist() == ref[(i, j)]["limbs"]
                                                        for (i, j) in entries),
                             "max_err_over_tolerance": worst}
        return res

    if w.range_bits and bits_arg == 13 and not sched_flags and args.adaptive_steps > 0:
        # the paper's own balancing (exponent classes) beside the range balancing of the headline
        out["exponent_classes"] = grouped(md.MDGEMM_GROUP_EXPONENT)
    if args.extras and bits_arg == 13 and not sched_flags and args.adaptive_steps > 0:
        out["sign_groups"] = grouped(md.MDGEMM_GROUP_SIGN)
    if args.extras and L == 2:
        out["qr_dd"] = qr_dd_line(md, torch, dev, stream, A, args.no_cpu_baseline)
        out["taylor_dd"] = taylor_dd_line(md, torch, dev, stream, args.no_cpu_baseline)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, A_h, B_h, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
