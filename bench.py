#!/usr/bin/env python3
"""Benchmark of the continual convolution step on one MI355X.

A step is one forward_step call: every one of the B streams consumes one
frame, the per-step contraction runs, the partial-sum ring is updated and the
completed output frame is emitted (for the depthwise workload a step is the
depthwise convolution step followed by the continual average-pool step).
Inputs (the whole synthetic clip, split into contiguous frames), weights and
the state are resident in HBM before timing starts; runs longer than the clip
cycle through its frames, continuing the same state (streams are infinite).

Prints one JSON line: stream-frames/s (B x steps / s, eager forward_step
calls), the roofline of the dominant kernel (the convolution step, launched
back to back and timed with HIP events around the region), the same steps
replayed from a HIP graph and through forward_steps, and the CPU oracle timed
on a bounded sample of the same workload on the host cores.
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

DEFAULT_WORKLOAD = "conv3d_b1_c24_k3_56x56_f32"
METRIC = "stream-frames/sec for CoConv3d forward_step; % of MFMA peak or HBM GB/s"

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
# Non-packed fp32 FMA on the vector ALUs: 256 CUs x 4 SIMDs x 16 lanes x 2
# FLOP x 2.4 GHz (packed fp32 instructions are not used).
PEAK_VALU_F32_TFLOPS = 78.6


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--algo", default="auto")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="bounded CPU-oracle sample (seconds of oracle work)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-modes", action="store_true", help="skip graph / forward_steps modes")
    ap.add_argument("--copy-mib", type=float, default=0.0,
                    help="instead of the benchmark, run --steps plain device copies of this many "
                         "MiB (calibrates the HBM traffic counters)")
    return ap.parse_args()


def copy_calibration(mib, steps):
    """Plain device copies of a known size -- the runtime's copy kernel
    (Tensor.copy_) and an elementwise kernel (torch.neg) -- for scaling
    FETCH_SIZE and WRITE_SIZE counter readings to bytes."""
    import torch
    n = int(mib * 1024 * 1024 / 4)
    a = torch.randn(n, device="cuda")
    b = torch.empty_like(a)
    for _ in range(steps):
        b.copy_(a)
    for _ in range(steps):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "steps": steps, "kernels": ["copy_", "neg"]}))


def sources_digest():
    """sha256 prefix over the library's kernel sources (sorted file names and
    contents): the key under which measured counters stay valid."""
    import hashlib
    d = os.path.join(ROOT, "paper_2204_03418_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        h.update(name.encode())
        with open(os.path.join(d, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per launch of the workload's dominant kernel, from the
    rocprofv3 FETCH_SIZE / WRITE_SIZE passes summarised in profiles/traffic.txt
    (already scaled by the plain-copy calibration); None when the kernel
    sources changed after those counters were taken, or none were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    try:
        with open(path) as f:
            lines = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    except OSError:
        return None
    kv = {ln[0]: ln[1] for ln in lines if len(ln) == 2}
    if kv.get("sources") != sources_digest():
        return None
    for ln in lines:
        if len(ln) == 5 and ln[0] == workload:
            return int(ln[4])
    return None


def kT_of(c):
    return (tuple(c.kernel) + (1, 1))[0]


def per_step_work(c, Ho, Wo):
    """Algorithmic FLOPs and bytes of one conv step (eager partial sums, stride 1):
    FLOPs = 2 B Ho Wo C_out kT (C_in/G) kH kW;
    bytes = |x_n| + |W| + 2 (kT - 1) |Y frame| * 4 (float32 ring RMW) + |y|."""
    kT, kH, kW = (tuple(c.kernel) + (1, 1))[:3]
    esz = 2 if c.dtype == "bf16" else 4
    cg = c.in_channels // c.groups
    S = 1
    for s in c.in_size:
        S *= s
    So = Ho * Wo
    flops = 2 * c.batch * So * c.out_channels * kT * cg * kH * kW
    x_bytes = c.batch * c.in_channels * S * esz
    w_bytes = c.out_channels * cg * kT * kH * kW * esz
    ring_bytes = 2 * (kT - 1) * c.batch * c.out_channels * So * 4
    y_bytes = c.batch * c.out_channels * So * esz
    return flops, x_bytes + w_bytes + ring_bytes + y_bytes


def main():
    args = parse()
    if args.copy_mib > 0:
        copy_calibration(args.copy_mib, args.steps)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; multi-GPU sharding is "
                                   "not built (streams would shard over the batch)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2204_03418_amd import coinf, synth

    wl = synth.WORKLOADS[args.workload]
    c = wl.conv
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    x, w, b = synth.workload_inputs(args.workload)
    T = x.shape[2]
    frames = [x[:, :, t].contiguous().to(dev) for t in range(T)]
    co = coinf.CoConv(w.to(dev), b.to(dev) if b is not None else None, batch=c.batch,
                      in_size=c.in_size, stride=c.stride, padding=c.padding,
                      dilation=c.dilation, groups=c.groups, algo=args.algo)
    y = co.new_output()
    po = None
    if wl.pool is not None:
        pl = wl.pool
        po = coinf.CoPool(pl.kind, batch=pl.batch, channels=pl.channels, kernel=pl.kernel,
                          in_size=pl.in_size, stride=pl.stride, padding=pl.padding,
                          count_include_pad=pl.count_include_pad,
                          dtype=synth.torch_dtype(pl.dtype), device=dev)
        z = torch.empty(po.out_frame_shape(), dtype=synth.torch_dtype(pl.dtype), device=dev)

    fptr = [ctypes.c_void_p(f.data_ptr()) for f in frames]
    yptr = ctypes.c_void_p(y.data_ptr())
    zptr = ctypes.c_void_p(z.data_ptr()) if po is not None else None
    conv_step = coinf.co_conv_forward_step
    pool_step = coinf.co_pool_forward_step
    hconv = co.handle
    hpool = po.handle if po is not None else None

    def run(n0, count, stream_ptr):
        for i in range(n0, n0 + count):
            st = conv_step(hconv, fptr[i % T], yptr, 1, stream_ptr)
            if hpool is not None and st == coinf.CO_OK:
                pool_step(hpool, yptr, zptr, 1, stream_ptr)

    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    # warm-up: past the delay so every timed step emits
    warm = max(args.warmup, co.delay + (po.delay if po is not None else 0) + 2)
    run(0, warm, sp)
    torch.cuda.synchronize()
    n = warm

    # (i) eager forward_step calls: the headline number
    K = args.steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    run(n, K, sp)
    e1.record(stream)
    torch.cuda.synchronize()
    n += K
    ms = e0.elapsed_time(e1)
    ms_per_step = ms / K
    value = c.batch * K / (ms / 1e3)

    # dominant kernel: the conv step alone, launched back to back (every step
    # emits, so each launch is one full contraction + ring update + emit);
    # HIP events bracket the region on the launch stream
    Ho, Wo = (tuple(co.out_size) + (1, 1))[:2]
    flops, nbytes = per_step_work(c, Ho, Wo)
    Kk = K
    k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    k0.record(stream)
    for i in range(Kk):
        conv_step(hconv, fptr[(n + i) % T], yptr, 1, sp)
    k1.record(stream)
    torch.cuda.synchronize()
    n += Kk
    kern_ms = k0.elapsed_time(k1) / Kk
    if c.dtype == "bf16" or co.algo.startswith("gemm"):
        bound_compute = "mfma"
        peak_c = PEAK_MFMA_TFLOPS[c.dtype]
    else:
        bound_compute = "alu"
        peak_c = PEAK_VALU_F32_TFLOPS
    ai = flops / nbytes
    ridge = peak_c * 1e12 / (PEAK_HBM_GBS * 1e9)
    if ai >= ridge:
        achieved = flops / (kern_ms / 1e3) / 1e12
        roof = {"bound": bound_compute, "achieved": round(achieved, 3), "peak": peak_c,
                "unit": "TFLOP/s", "frac": round(achieved / peak_c, 5), "traffic": None}
    else:
        achieved = nbytes / (kern_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 5), "traffic": None}
    roof["traffic"] = measured_traffic(args.workload)
    roof.update({"kernel": f"conv step ({co.algo})", "kernel_avg_us": round(kern_ms * 1e3, 3),
                 "flops_per_launch": flops, "bytes_per_launch": nbytes})

    modes = {"eager_forward_step": round(value, 1)}
    modes_roof = {}
    if not args.no_modes:
        # (ii) the same steps replayed from a HIP graph: one schedule period
        # (ring slots x stride) per capture, so replays keep the state coherent
        period = co.info.ring_slots * c.stride[0]
        if po is not None:
            period *= po.info.fifo_slots * wl.pool.stride[0]
        period *= max(1, -(-64 // period))  # at least 64 steps per replay
        reps = max(1, K // period)
        gstream = torch.cuda.Stream()
        gstream.wait_stream(stream)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(gstream):
            with torch.cuda.graph(graph, stream=gstream):
                gp = ctypes.c_void_p(gstream.cuda_stream)
                run(n, period, gp)
        n += period
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(reps):
            graph.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        modes["graph_replay"] = round(c.batch * reps * period / (g0.elapsed_time(g1) / 1e3), 1)
        # (iii) forward_steps over the resident clip (the depthwise workload
        # chains the convolution's output clip into the pool's forward_steps)
        xc = x.to(dev)
        calls = max(1, K // T)

        def clip_pass():
            yc = co.forward_steps(xc)
            if po is not None and yc is not None:
                po.forward_steps(yc)

        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        clip_pass()
        torch.cuda.synchronize()
        s0.record(stream)
        for _ in range(calls):
            clip_pass()
        s1.record(stream)
        torch.cuda.synchronize()
        modes["forward_steps"] = round(c.batch * calls * T / (s0.elapsed_time(s1) / 1e3), 1)
        # the same roofline terms for forward_steps: per frame the persistent
        # launch does the step's FLOPs but moves only the frame and its output
        # (the partial sums stay on chip), so it is priced on compute
        us_frame = s0.elapsed_time(s1) * 1e3 / (calls * T)
        io_bytes = nbytes - 2 * (kT_of(c) - 1) * c.batch * c.out_channels * Ho * Wo * 4
        tf = flops / (us_frame * 1e-6) / 1e12
        gbs = io_bytes / (us_frame * 1e-6) / 1e9
        fs = {"persistent": bool(co.steps_fused(T)), "us_per_frame": round(us_frame, 3),
              "flops_per_frame": flops, "io_bytes_per_frame": io_bytes}
        if flops / io_bytes >= ridge:
            fs.update({"bound": bound_compute, "achieved": round(tf, 3), "peak": peak_c,
                       "unit": "TFLOP/s", "frac": round(tf / peak_c, 5)})
        else:
            fs.update({"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS,
                       "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 5)})
        modes_roof["forward_steps"] = fs

        # (iv) a depthwise convolution feeding a global pool: the fused step
        # (one launch per step, the same results as the two-launch chain)
        if po is not None and coinf.ConvPool.fits(co, po):
            cp = coinf.ConvPool(co, po)
            cp_step = coinf.co_convpool_forward_step
            for i in range(2 * T):
                cp_step(cp.handle, fptr[(n + i) % T], zptr, 1, sp)
            n += 2 * T
            f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            f0.record(stream)
            for i in range(K):
                cp_step(cp.handle, fptr[(n + i) % T], zptr, 1, sp)
            f1.record(stream)
            torch.cuda.synchronize()
            n += K
            modes["fused_convpool_step"] = round(c.batch * K / (f0.elapsed_time(f1) / 1e3), 1)
            # and the fused clip: one launch per forward_steps call where it fits
            cp.forward_steps(xc)
            torch.cuda.synchronize()
            f0.record(stream)
            for _ in range(calls):
                cp.forward_steps(xc)
            f1.record(stream)
            torch.cuda.synchronize()
            modes["fused_convpool_forward_steps"] = round(
                c.batch * calls * T / (f0.elapsed_time(f1) / 1e3), 1)

    if not args.no_modes:
        # (v) cold: the same eager conv steps rotating over enough independent
        # layer states (rings and packed weights) that their footprint passes
        # 512 MB, twice the 256 MB Infinity Cache, so the ring's reads and
        # writes come from HBM rather than the cache; frames rotate too
        nh = int(min(1024, max(2, -(-512 * 2**20 // co.info.state_bytes))))
        cold = [coinf.CoConv(w.to(dev), b.to(dev) if b is not None else None, batch=c.batch,
                             in_size=c.in_size, stride=c.stride, padding=c.padding,
                             dilation=c.dilation, groups=c.groups, algo=args.algo)
                for _ in range(nh)]
        ch = [cc.handle for cc in cold]
        for r in range(co.delay + 1):  # past the delay: every timed step emits
            for k in range(nh):
                conv_step(ch[k], fptr[r % T], yptr, 1, sp)
        Kc = max(K, 2 * nh)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        c0.record(stream)
        for i in range(Kc):
            conv_step(ch[i % nh], fptr[(i // nh) % T], yptr, 1, sp)
        c1.record(stream)
        torch.cuda.synchronize()
        cms = c0.elapsed_time(c1) / Kc
        modes["cold_conv_step"] = round(c.batch / (cms / 1e3), 1)
        cr = {"states": nh, "footprint_mb": round(nh * co.info.state_bytes / 2**20, 1),
              "kernel_avg_us": round(cms * 1e3, 3)}
        if roof["bound"] == "hbm":
            cg = nbytes / (cms / 1e3) / 1e9
            cr.update({"bound": "hbm", "achieved": round(cg, 2), "peak": PEAK_HBM_GBS,
                       "unit": "GB/s", "frac": round(cg / PEAK_HBM_GBS, 5)})
        else:
            ct = flops / (cms / 1e3) / 1e12
            cr.update({"bound": roof["bound"], "achieved": round(ct, 3), "peak": peak_c,
                       "unit": "TFLOP/s", "frac": round(ct / peak_c, 5)})
        modes_roof["cold_conv_step"] = cr
        del cold, ch

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wl, x, w, b, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "stream-frames/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": warm,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": c.dtype,
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": c.batch, "in_channels": c.in_channels,
                   "out_channels": c.out_channels, "groups": c.groups,
                   "kernel": list(c.kernel), "in_size": list(c.in_size),
                   "padding": list(c.padding), "frames": T, "algo": co.algo,
                   "pool": None if wl.pool is None else
                   {"kind": wl.pool.kind, "kernel": list(wl.pool.kernel),
                    "stride": list(wl.pool.stride)}},
        "roofline": roof,
        "cpu_baseline": cpu,
        "modes": modes,
        "modes_roofline": modes_roof,
    }
    print(json.dumps(out))


def cpu_baseline(wl, x, w, b, seconds):
    """The oracle's sliding-window driver stepping the same frames on the host
    cores (float64, OpenMP over (b, o)); bounded to about `seconds` of work."""
    import numpy as np

    import oracle

    c = wl.conv
    xs = x.float().double().numpy()
    co = oracle.ContinualConv(w.float().double().numpy(),
                              None if b is None else b.float().double().numpy(),
                              stride=c.stride, padding=c.padding, dilation=c.dilation,
                              groups=c.groups)
    po = None
    if wl.pool is not None:
        po = oracle.ContinualPool(wl.pool.kind, wl.pool.kernel, wl.pool.stride, wl.pool.padding,
                                  count_include_pad=wl.pool.count_include_pad,
                                  spatial_dims=len(wl.pool.in_size))
    T = xs.shape[2]

    def step(i):
        y = co.forward_step(xs[:, :, i % T])
        if po is not None and y is not None:
            po.forward_step(y)

    for i in range(co.delay + (po.delay if po else 0) + 1):
        step(i)
    i0 = co.delay + (po.delay if po else 0) + 1
    t0 = time.perf_counter()
    k = 0
    while time.perf_counter() - t0 < seconds or k == 0:
        step(i0 + k)
        k += 1
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or os.cpu_count()
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(c.batch * k / dt, 3), "unit": "stream-frames/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{k} steps of the same workload after the delay ({dt:.1f} s, float64, "
                      f"OpenMP over (b, o)); cpu: {cpu_model}"}


if __name__ == "__main__":
    main()
