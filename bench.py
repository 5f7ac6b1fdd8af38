"""Benchmark of the MI355X SC GEMM: one step = one full sc_gemm call per GEMM of the
workload (comparator sequences, row-length scheduler, operand layout and per-cycle-group
stream tables, the counting GEMM on the matrix cores and the decode) over one batch of
synthetic input already resident in HBM.

Prints ONE JSON line.  ``value`` is whole-call throughput in stream-bit-ops/s
(N * K * sum_i L_i per step / seconds per step).  ``roofline`` is for the dominant kernel
(the counting GEMM of the largest GEMM and, when its tiles are split, the pass that sums
the splits), timed with HIP events that the library records around exactly those launches
on the call's stream: one stream-bit-op is one fp4 product on the matrix cores (2 flops),
against the dense fp4 MFMA peak.  ``valu_bitop_peak`` is the measured rate of the same
work done as packed words on the vector ALUs (AND + accumulating popcount, 2 instructions
per 32 bit pairs: libscpeak), with the clock under that load; ``value`` is also given as a
multiple of it.  ``cpu_baseline`` times the CPU oracle on a bounded row sample.

Before the warm-up steps the call runs untimed until its time per call settles
(``clock_settle`` in the line): the GPU raises its clock over tens of milliseconds of load,
and the timed steps are meant to show the sustained rate.  ``--no-settle`` skips that.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SC stream-bit-ops/sec (M·N·K·L) and % of gfx950 bitop+popcount peak"
PEAK_FP4_FLOPS = 10.1e15                         # dense fp4 (e2m1) MFMA, MI355X (published)
# the paper's one speed figure for this path (Sec. 4.2): its fused GPU SC matmul against a
# direct CPU simulation, hardware of both sides not stated
PAPER_GPU_VS_CPU = 95000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="vitb16_fc1_L128")
    p.add_argument("--rng", choices=("lfsr", "cbsg"), default="lfsr",
                   help="comparator source: 32-bit LFSR, or scrambled Sobol-8 with "
                        "conditional generation of B's stream (C-BSG, L_max <= 256)")
    p.add_argument("--cpu-rows", type=int, default=0,
                   help="rows of A for the oracle sample (0 = size it to ~15 s)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-valu-peak", action="store_true",
                   help="skip the VALU AND + popcount peak measurement")
    p.add_argument("--no-settle", action="store_true",
                   help="start the warm-up steps without first running the call until its time "
                        "settles (the GPU's clock then still ramps up during the timed steps)")
    p.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                   help="only run a plain device copy of BYTES bytes (3 times), to calibrate "
                        "the HBM byte counters against a kernel of known traffic")
    return p.parse_args()


def kernel_source_digest():
    import hashlib
    h = hashlib.sha256()
    for name in ("sc_internal.h", "sc_kernels.hip", "sc_mfma.hip"):
        with open(os.path.join(ROOT, "paper_2609_32922_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per GEMM launch from the committed rocprofv3 counter summary, or None
    when the summary is missing or the kernel source changed since it was taken."""
    import glob
    import re
    for path in glob.glob(os.path.join(ROOT, "profiles", "*counters*.md")):
        with open(path) as f:
            text = f.read()
        m = re.search(r"^traffic_bytes_per_launch:\s*(\d+)\s+workload:\s*(\S+)\s+"
                      r"kernel_source_sha256:\s*([0-9a-f]+)", text, re.M)
        if m and m.group(2) == workload and m.group(3) == kernel_source_digest():
            return int(m.group(1))
    return None


EV_EVERY = 4


def copy_probe(nbytes):
    import torch
    x = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "reads": nbytes, "writes": nbytes}))


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only (--gpus 1): the SC GEMM runs on a single MI355X; "
              "across GPUs the rows of A would shard with no collective",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2609_32922_amd as scg
    import workloads as W

    w = W.WORKLOADS[args.workload]()
    rng = scg.SC_RNG_SOBOL8_CBSG if args.rng == "cbsg" else scg.SC_RNG_LFSR32
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    staged = []
    for g in w.gemms:
        t = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in (g.A, g.sA, g.B, g.sB, g.L)]
        out = torch.empty((g.batch, g.M, g.N), dtype=torch.float32, device=dev)
        d = scg.make_desc(t[0], t[2], g.L_max, g.polarity, g.seed, int(round(float(g.L.mean()))), rng)
        ws = scg.Workspace(scg.sc_gemm_workspace_size(d), dev)
        staged.append((g, t, out, ws))
    bitops = w.bitops()
    nsteps = args.steps
    # kernel timing events on every EV_EVERY-th timed step (and the last): a timestamped
    # dispatch leaves the GPU idle for several microseconds before and after it, a cost that
    # calls without profiling events do not have
    timed = [s for s in range(nsteps) if s % EV_EVERY == EV_EVERY - 1 or s == nsteps - 1]
    ev_pairs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in w.gemms] if s in timed else None for s in range(nsteps)]
    for pairs in ev_pairs:             # create the underlying HIP events
        for e0, e1 in pairs or []:
            e0.record(stream)
            e1.record(stream)
    torch.cuda.synchronize()

    def step(pairs=None):
        for k, (g, t, out, ws) in enumerate(staged):
            pe = None if pairs is None else (pairs[k][0].cuda_event, pairs[k][1].cuda_event)
            scg.gemm(t[0], t[1], t[2], t[3], t[4], L_max=g.L_max, polarity=g.polarity,
                     seed=g.seed, out=out, workspace=ws, stream=stream, prof_events=pe,
                     L_hint=int(round(float(g.L.mean()))), rng=rng)

    settle = None if args.no_settle else settle_clock(step, stream)
    for _ in range(args.warmup):
        step()
    for k in range(len(staged)):
        rc = scg.sc_gemm_status(staged[k][3].ptr, int(stream.cuda_stream))
        if rc != 0:
            raise SystemExit("device status error: %s" % scg.strerror(rc))
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for s in range(nsteps):
        step(ev_pairs[s])
    t1.record(stream)
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_per_step = ms_total / nsteps
    value = bitops / (ms_per_step * 1e-3)

    # dominant kernel: the counting GEMM of the largest GEMM in the workload
    kidx = int(np.argmax([g.bitops() for g in w.gemms]))
    gemm_ms = float(np.mean([ev_pairs[s][kidx][0].elapsed_time(ev_pairs[s][kidx][1]) for s in timed]))
    g_dom = w.gemms[kidx]
    achieved = g_dom.bitops() / (gemm_ms * 1e-3)
    traffic = measured_traffic("%s:%s" % (args.workload, args.rng))
    # one bit-pair product = one fp4 multiply-add = 2 flops on the matrix cores
    roofline = {"bound": "mfma", "achieved": 2 * achieved / 1e12, "peak": PEAK_FP4_FLOPS / 1e12,
                "unit": "TFLOP/s", "frac": 2 * achieved / PEAK_FP4_FLOPS, "traffic": traffic,
                "kernel": "%s<%s>" % (gemm_kernel_name(g_dom, rng == scg.SC_RNG_LFSR32),
                                      "bipolar" if g_dom.polarity == 0 else "unipolar"),
                "kernel_ms": gemm_ms, "kernel_ms_steps": len(timed), "kernel_stream_bit_ops_per_s": achieved}

    valu = None
    if not args.no_valu_peak:
        valu = valu_peak()
        valu["value_over_peak"] = value / valu["bitops_per_s"]
        valu["kernel_over_peak"] = achieved / valu["bitops_per_s"]

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_rows, args.rng == "cbsg")
        cpu["gpu_over_oracle"] = value / cpu["value"]
        cpu["paper_gpu_over_cpu"] = PAPER_GPU_VS_CPU

    g0 = w.gemms[0]
    cfg = {"workload": w.name, "gemms": [{"name": g.name, "batch": g.batch, "M": g.M, "N": g.N,
                                          "K": g.K, "L_mean": float(g.L.mean()),
                                          "L_max": g.L_max} for g in w.gemms],
           "polarity": "bipolar_xnor" if g0.polarity == 0 else "unipolar_and_sign_magnitude",
           "rng": "sobol8_cbsg" if args.rng == "cbsg" else "lfsr32", "seed": g0.seed,
           "bitops_per_step": bitops}
    line = {"metric": METRIC, "value": value, "unit": "stream-bit-ops/s", "n_gpus": 1,
            "steps": nsteps, "warmup": args.warmup, "ms_per_step": ms_per_step,
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "fp4", "data": "synthetic", "config": cfg, "roofline": roofline,
            "valu_bitop_peak": valu, "cpu_baseline": cpu, "clock_settle": settle}
    print(json.dumps(line), flush=True)


def settle_clock(step, stream, batch=10, min_s=0.1, max_s=3.0, tol=0.01):
    """Run the call untimed until its time per call settles, before the warm-up steps.

    Under sustained load the GPU raises its shader clock over tens of milliseconds (ViT-B fc1 at
    L = 128 measured 0.58 ms per call after 5 warm-up calls, 0.50 ms after 100), so a short
    benchmark would time the ramp rather than the sustained rate a continuously running
    deployment sees.  Batches of `batch` calls run until two consecutive batches differ by less
    than `tol` and at least `min_s` seconds have passed (at most `max_s`).  Returns what it did.
    """
    import torch
    t_start = time.perf_counter()
    first = prev = last = None
    n = 0
    while True:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(batch):
            step()
        e1.record(stream)
        e1.synchronize()
        n += batch
        last = e0.elapsed_time(e1) / batch
        if first is None:
            first = last
        el = time.perf_counter() - t_start
        if el >= max_s or (el >= min_s and prev is not None and abs(last - prev) <= tol * prev):
            break
        prev = last
    return {"calls": n, "seconds": time.perf_counter() - t_start, "first_batch_ms_per_step": first,
            "last_batch_ms_per_step": last,
            "kind": "untimed calls before the warm-up steps, until the time per call settles"}


def gemm_kernel_name(g, comparator):
    """The counting kernel the library takes for this shape (see make_layout): 256-row blocks
    for M > 128 (fragments from int8 chunks with comparator streams, 256 or, for N <= 64, 64
    columns wide; fp4 planes with C-BSG when N > 128); fragments from the int8 rows for other
    N <= 128 with comparator streams; 128-row planes otherwise."""
    if comparator and g.M > 128 and (g.N > 128 or g.N <= 64):
        return "k_rgemm"
    if g.M > 128 and g.N > 128:
        return "k_qgemm"
    if comparator and g.N <= 128:
        return "k_fgemm"
    return "k_mgemm"


def valu_peak():
    """The measured VALU rate of packed AND + accumulating popcount (libscpeak), best over
    1, 2, 4 and 8 waves per SIMD, with the shader clock under that load."""
    from paper_2609_32922_amd import peak
    best = None
    for wps in (1, 2, 4, 8):
        r = peak.sc_peak_valu_bitop(wps, 50000)
        if best is None or r.bitops_per_s > best.bitops_per_s:
            best = r
    return {"bitops_per_s": best.bitops_per_s, "unit": "stream-bit-ops/s",
            "lane_ops_per_s": best.lane_ops_per_s, "clock_ghz": best.clock_hz / 1e9,
            "cus": best.cus, "waves_per_simd": best.waves_per_simd,
            "lane_ops_per_cu_per_clock": best.lane_ops_per_s / (best.cus * best.clock_hz),
            "kind": "measured: 16 AND -> v_bcnt_u32_b32 chains per lane, registers only"}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, rows, cbsg=False):
    """The CPU oracle, as it stands, on the first rows of the dominant GEMM: all the host
    threads this process may use (capped by OMP_NUM_THREADS when it is set, the CPU share
    of one GPU on a shared host), then one thread on a small slice for the per-core rate."""
    import oracle
    ref = oracle.sc_gemm_cbsg if cbsg else oracle.sc_gemm
    visible = len(os.sched_getaffinity(0))
    cap = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    threads = min(visible, cap) if cap > 0 else visible
    g = max(w.gemms, key=lambda x: x.bitops())
    b = 0
    bB = 0 if g.B.shape[0] == 1 else b

    def run(n, nthreads):
        t = time.perf_counter()
        ref(g.A[b][:n], g.B[bB], g.sA[b][:n], g.sB[bB], g.L[b][:n], g.L_max,
            g.polarity, g.seed, nthreads=nthreads, want_out=True)
        return time.perf_counter() - t

    def ops(n):
        return int(g.N) * int(g.K) * int(g.L[b][:n].astype(np.int64).sum())

    target = 15.0
    if rows <= 0:
        # size the sample so that the timed oracle run takes about 15 s: two probes give
        # the fixed cost (B streams) and the per-row cost
        r1, r2 = 16, 64
        t1, t2 = run(r1, threads), run(r2, threads)
        per_row = max((t2 - t1) / (r2 - r1), 1e-6)
        rows = int(max(r2, min(g.M, (target - max(t1 - r1 * per_row, 0.0)) / per_row)))
    dt = run(rows, threads)
    # one thread: the difference of two slices removes the fixed cost of B's streams
    s1, s2 = 2, 10
    d1, d2 = run(s1, 1), run(s2, 1)
    one = (ops(s2) - ops(s1)) / max(d2 - d1, 1e-9)
    return {"value": ops(rows) / dt, "unit": "stream-bit-ops/s", "cores": threads, "kind": "oracle",
            "seconds": dt, "cpu_model": cpu_model(), "host_threads_visible": visible,
            "one_thread_value": one,
            "sample": "%s/%s rows 0..%d of %d, all %d columns, K=%d, %d stream-bit-ops "
                      "(every stream materialised inside the timed run); one-thread rate from "
                      "rows %d..%d" % (w.name, g.name, rows - 1, g.M, g.N, g.K, ops(rows), s1, s2 - 1)}


if __name__ == "__main__":
    main()
