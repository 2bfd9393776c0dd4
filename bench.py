#!/usr/bin/env python3
"""Benchmark of the continual convolution step on one MI355X.

A step is one forward_step call: every one of the B streams consumes one
frame, the per-step contraction runs, the partial-sum ring is updated and the
completed output frame is emitted (for the depthwise workload a step is the
depthwise convolution step followed by the continual average-pool step).
Inputs (the whole synthetic clip, split into contiguous frames), weights and
the state are resident in HBM before timing starts; runs longer than the clip
cycle through its frames, continuing the same state (streams are infinite).

The headline line is the 64-stream 192->192 3x3x3 14x14 bf16 layer, the
largest of the named workloads.  Every timed region runs exactly --steps
steps and is repeated (at least 5 times, and until the repetitions cover
10 ms); the median repetition is reported.  The line carries:

* value: stream-frames/s of eager forward_step calls (B x steps / s);
* roofline: the convolution step kernel alone, launched back to back, timed
  with HIP events on its launch stream (median repetition), priced on the
  step's algorithmic FLOPs or bytes;
* modes: the same steps replayed from a HIP graph, through forward_steps
  over the resident clip, and (depthwise) through the fused conv+pool step;
* workloads: the eager step, its kernel and forward_steps, with rooflines,
  for every named workload;
* bottleneck: the fused X3D bottleneck front against its layers stepped
  separately;
* cpu_baseline: the oracle timed on a bounded sample of the same workload on
  the host cores, at the host's thread count and at one thread.
"""
import argparse
import ctypes
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

DEFAULT_WORKLOAD = "conv3d_b64_c192_k3_14x14_bf16"
METRIC = "stream-frames/sec for CoConv3d forward_step; % of MFMA peak or HBM GB/s"

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
# Non-packed fp32 FMA on the vector ALUs: 256 CUs x 4 SIMDs x 16 lanes x 2
# FLOP x 2.4 GHz (packed fp32 instructions are not used).
PEAK_VALU_F32_TFLOPS = 78.6

MIN_REPS = 5
MIN_REGION_MS = 10.0
WARM_MS = 250.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--algo", default="auto")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="bounded CPU-oracle sample (seconds of oracle work per thread count)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-modes", action="store_true", help="skip graph / forward_steps modes")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the per-workload table (headline workload only)")
    ap.add_argument("--cold", action="store_true",
                    help="also time the eager conv step rotating over >512 MB of layer states")
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


def timed(fn, stream, est_ms=None):
    """Median wall time (ms, HIP events on `stream`) of repetitions of fn():
    at least MIN_REPS, and enough that they cover MIN_REGION_MS together.
    Returns (median ms, repetitions)."""
    import torch
    if est_ms is None:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        est_ms = max(e0.elapsed_time(e1), 1e-3)
    reps = max(MIN_REPS, min(200, int(math.ceil(MIN_REGION_MS / est_ms))))
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in ev), reps


class Workload:
    """One named workload resident on the GPU: frames, layer handles and
    output buffers; a running step counter keeps every timed step emitting."""

    def __init__(self, name, dev, algo="auto"):
        import torch

        from paper_2204_03418_amd import coinf, synth

        self.name = name
        self.wl = wl = synth.WORKLOADS[name]
        self.c = c = wl.conv
        self.dev = dev
        self.coinf = coinf
        x, w, b = synth.workload_inputs(name)
        self.x_cpu, self.w_cpu, self.b_cpu = x, w, b
        self.T = x.shape[2]
        self.frames = [x[:, :, t].contiguous().to(dev) for t in range(self.T)]
        self.xc = x.to(dev)
        self.w, self.b = w.to(dev), (b.to(dev) if b is not None else None)
        self.algo = algo
        self.co = self.new_conv()
        self.y = self.co.new_output()
        self.po = None
        if wl.pool is not None:
            pl = wl.pool
            self.po = coinf.CoPool(pl.kind, batch=pl.batch, channels=pl.channels,
                                   kernel=pl.kernel, in_size=pl.in_size, stride=pl.stride,
                                   padding=pl.padding, count_include_pad=pl.count_include_pad,
                                   dtype=synth.torch_dtype(pl.dtype), device=dev)
            self.z = torch.empty(self.po.out_frame_shape(), dtype=synth.torch_dtype(pl.dtype),
                                 device=dev)
        self.fptr = [ctypes.c_void_p(f.data_ptr()) for f in self.frames]
        self.yptr = ctypes.c_void_p(self.y.data_ptr())
        self.zptr = ctypes.c_void_p(self.z.data_ptr()) if self.po is not None else None
        self.stream = torch.cuda.current_stream()
        self.sp = ctypes.c_void_p(self.stream.cuda_stream)
        self.n = 0
        Ho, Wo = (tuple(self.co.out_size) + (1, 1))[:2]
        self.flops, self.nbytes = per_step_work(c, Ho, Wo)
        self.io_bytes = self.nbytes - 2 * (kT_of(c) - 1) * c.batch * c.out_channels * Ho * Wo * 4
        self.in_bytes = c.batch * c.in_channels * math.prod(c.in_size) * (2 if c.dtype == "bf16" else 4)
        # the GEMM family runs on the matrix cores, the depthwise and direct
        # kernels on the vector ALUs
        if self.co.algo.startswith("gemm"):
            self.bound_compute, self.peak_c = "mfma", PEAK_MFMA_TFLOPS[c.dtype]
        else:
            self.bound_compute, self.peak_c = "alu", PEAK_VALU_F32_TFLOPS
        self.ridge = self.peak_c * 1e12 / (PEAK_HBM_GBS * 1e9)

    def new_conv(self):
        c = self.c
        return self.coinf.CoConv(self.w, self.b, batch=c.batch, in_size=c.in_size,
                                 stride=c.stride, padding=c.padding, dilation=c.dilation,
                                 groups=c.groups, algo=self.algo)

    @property
    def delay(self):
        return self.co.delay + (self.po.delay if self.po is not None else 0)

    def steps(self, count, stream_ptr=None):
        """`count` eager forward_step calls (conv, then pool when it emitted)."""
        sp = self.sp if stream_ptr is None else stream_ptr
        conv_step, pool_step = self.coinf.co_conv_forward_step, self.coinf.co_pool_forward_step
        hc = self.co.handle
        hp = self.po.handle if self.po is not None else None
        for i in range(self.n, self.n + count):
            st = conv_step(hc, self.fptr[i % self.T], self.yptr, 1, sp)
            if hp is not None and st == self.coinf.CO_OK:
                pool_step(hp, self.yptr, self.zptr, 1, sp)
        self.n += count

    def conv_steps(self, count):
        """`count` convolution step launches alone (every one emits)."""
        conv_step = self.coinf.co_conv_forward_step
        hc = self.co.handle
        for i in range(self.n, self.n + count):
            conv_step(hc, self.fptr[i % self.T], self.yptr, 1, self.sp)
        self.n += count

    def roofline(self, us, flops=None, nbytes=None):
        """Roofline entry of a kernel taking `us` per launch: compute-priced
        when the arithmetic intensity on `nbytes` is above the ridge, else
        HBM-priced."""
        flops = self.flops if flops is None else flops
        nbytes = self.nbytes if nbytes is None else nbytes
        if flops / nbytes >= self.ridge:
            a = flops / (us * 1e-6) / 1e12
            return {"bound": self.bound_compute, "achieved": round(a, 3), "peak": self.peak_c,
                    "unit": "TFLOP/s", "frac": round(a / self.peak_c, 5)}
        a = nbytes / (us * 1e-6) / 1e9
        return {"bound": "hbm", "achieved": round(a, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(a / PEAK_HBM_GBS, 5)}

    def eager(self, K):
        """Median ms of K eager steps; stream-frames/s."""
        ms, reps = timed(lambda: self.steps(K), self.stream)
        return ms, reps, self.c.batch * K / (ms / 1e3)

    def kernel_us(self, K):
        """The convolution step kernel alone, K launches back to back on its
        stream, bracketed by HIP events: median µs per launch."""
        ms, _ = timed(lambda: self.conv_steps(K), self.stream)
        return ms * 1e3 / K

    def forward_steps(self, K):
        """forward_steps over the resident clip (the depthwise workload chains
        the convolution's output clip into the pool's forward_steps): calls of
        T frames covering at least K frames; median µs per frame."""
        calls = max(1, -(-K // self.T))

        def clip_pass():
            for _ in range(calls):
                yc = self.co.forward_steps(self.xc)
                if self.po is not None and yc is not None:
                    self.po.forward_steps(yc)

        clip_pass()
        ms, _ = timed(clip_pass, self.stream)
        return ms * 1e3 / (calls * self.T)

    def graph(self, K):
        """The same eager steps replayed from a HIP graph of whole schedule
        periods (ring slots x stride, at least 64 steps), so replays keep the
        state coherent: stream-frames/s."""
        import torch
        period = self.co.info.ring_slots * self.c.stride[0]
        if self.po is not None:
            period *= self.po.info.fifo_slots * self.wl.pool.stride[0]
        period *= max(1, -(-64 // period))
        gstream = torch.cuda.Stream()
        gstream.wait_stream(self.stream)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(gstream):
            with torch.cuda.graph(graph, stream=gstream):
                self.steps(period, ctypes.c_void_p(gstream.cuda_stream))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        reps = max(1, K // period)

        def replay():
            for _ in range(reps):
                graph.replay()

        ms, _ = timed(replay, self.stream)
        return self.c.batch * reps * period / (ms / 1e3)

    def fused_convpool(self, K):
        """Depthwise conv + global pool fused into one launch per step, and
        over the clip: stream-frames/s of each (None when the pair does not
        fuse)."""
        coinf = self.coinf
        if self.po is None or not coinf.ConvPool.fits(self.co, self.po):
            return None
        co2 = self.new_conv()
        c = self.wl.pool
        po2 = coinf.CoPool(c.kind, batch=c.batch, channels=c.channels, kernel=c.kernel,
                           in_size=c.in_size, stride=c.stride, padding=c.padding,
                           count_include_pad=c.count_include_pad,
                           dtype=self.z.dtype, device=self.dev)
        cp = coinf.ConvPool(co2, po2)
        cp_step = coinf.co_convpool_forward_step
        state = {"n": 0}

        def run(count):
            for i in range(state["n"], state["n"] + count):
                cp_step(cp.handle, self.fptr[i % self.T], self.zptr, 1, self.sp)
            state["n"] += count

        run(2 * self.T)
        ms, _ = timed(lambda: run(K), self.stream)
        step = self.c.batch * K / (ms / 1e3)
        calls = max(1, -(-K // self.T))

        def clip():
            for _ in range(calls):
                cp.forward_steps(self.xc)

        clip()
        ms, _ = timed(clip, self.stream)
        return step, self.c.batch * calls * self.T / (ms / 1e3)

    def cold(self, K):
        """The eager conv step rotating over enough independent layer states
        (rings and packed weights) that their footprint passes 512 MB, twice
        the 256 MB Infinity Cache, so the ring's reads and writes come from
        HBM rather than the cache; frames rotate too."""
        nh = int(min(1024, max(2, -(-512 * 2**20 // self.co.info.state_bytes))))
        cold = [self.new_conv() for _ in range(nh)]
        ch = [cc.handle for cc in cold]
        conv_step = self.coinf.co_conv_forward_step
        for r in range(self.co.delay + 1):
            for k in range(nh):
                conv_step(ch[k], self.fptr[r % self.T], self.yptr, 1, self.sp)
        Kc = max(K, 2 * nh)
        state = {"i": 0}

        def run():
            for i in range(state["i"], state["i"] + Kc):
                conv_step(ch[i % nh], self.fptr[(i // nh) % self.T], self.yptr, 1, self.sp)
            state["i"] += Kc

        ms, _ = timed(run, self.stream)
        us = ms * 1e3 / Kc
        out = {"states": nh, "footprint_mb": round(nh * self.co.info.state_bytes / 2**20, 1),
               "kernel_avg_us": round(us, 3)}
        out.update(self.roofline(us))
        return self.c.batch / (us * 1e-6), out


def bottleneck_entry(dev, K):
    """The fused X3D bottleneck front (pointwise conv+BN+ReLU, depthwise
    conv+BN+ReLU, average pool; one co_bneck launch per step) against the
    same modules stepped separately (pointwise layer on the kernel AUTO
    picks, then the activation, depthwise and pool launches), and the fused
    forward_steps over the resident clip.  Priced on the block's algorithmic
    FLOPs (pointwise + depthwise) and bytes (input frame, the depthwise
    ring's kT-1 slots read and written, the pool's reduced frames, output,
    weights once)."""
    import torch

    from paper_2204_03418_amd import coinf, synth

    sp = synth.BOTTLENECK
    x, w1, b1, w2, st1, st2 = synth.bottleneck_inputs(sp)
    B, Ci, C, (H, W) = sp.batch, sp.in_channels, sp.channels, sp.in_size
    T = x.shape[2]
    tdt = synth.torch_dtype(sp.dtype)
    xd = x.to(dev)
    frames = [x[:, :, t].contiguous().to(dev) for t in range(T)]
    fptr = [ctypes.c_void_p(f.data_ptr()) for f in frames]
    bn1 = tuple(t.to(dev) for t in st1) + (1e-5,)
    bn2 = tuple(t.to(dev) for t in st2) + (1e-5,)
    kT = sp.kernel[0]
    Ho, Wo = H + 2 * sp.padding[1] - sp.kernel[1] + 1, W + 2 * sp.padding[2] - sp.kernel[2] + 1

    def modules(pw_algo):
        pw = coinf.CoConv(w1.to(dev), b1.to(dev), batch=B, in_size=sp.in_size, algo=pw_algo,
                          bn=bn1)
        dw = coinf.CoConv(w2.to(dev), None, batch=B, in_size=sp.in_size, padding=sp.padding,
                          groups=C, bn=bn2)
        pool = coinf.CoPool("avg", batch=B, channels=C, kernel=sp.pool_kernel,
                            in_size=(Ho, Wo), stride=(1, Ho, Wo), dtype=tdt, device=dev)
        return pw, dw, pool

    stream = torch.cuda.current_stream()
    spp = ctypes.c_void_p(stream.cuda_stream)
    z = torch.empty((B, C, 1, 1), dtype=tdt, device=dev)
    zp = ctypes.c_void_p(z.data_ptr())
    fused_mods = modules("auto")
    bn = coinf.Bottleneck(fused_mods[0], True, fused_mods[1], True, fused_mods[2])
    step = coinf.co_bneck_forward_step
    state = {"n": 0}

    def run_fused(count):
        for i in range(state["n"], state["n"] + count):
            step(bn.handle, fptr[i % T], zp, 1, spp)
        state["n"] += count

    run_fused(2 * T)
    ms, _ = timed(lambda: run_fused(K), stream)
    fused_us = ms * 1e3 / K

    pw, dw, pool = modules("auto")
    y1 = torch.empty((B, C) + tuple(sp.in_size), dtype=tdt, device=dev)
    y2 = torch.empty((B, C, Ho, Wo), dtype=tdt, device=dev)
    y1p, y2p = ctypes.c_void_p(y1.data_ptr()), ctypes.c_void_p(y2.data_ptr())
    act = coinf.co_act_forward
    dt_code = coinf.DTYPES[tdt]
    cstep, pstep = coinf.co_conv_forward_step, coinf.co_pool_forward_step
    sep = {"n": 0}

    def run_separate(count):
        for i in range(sep["n"], sep["n"] + count):
            cstep(pw.handle, fptr[i % T], y1p, 1, spp)
            act(y1p, y1p, y1.numel(), dt_code, coinf.CO_ACT_RELU, spp)
            if cstep(dw.handle, y1p, y2p, 1, spp) == coinf.CO_OK:
                act(y2p, y2p, y2.numel(), dt_code, coinf.CO_ACT_RELU, spp)
                pstep(pool.handle, y2p, zp, 1, spp)
        sep["n"] += count

    run_separate(2 * T)
    ms, _ = timed(lambda: run_separate(K), stream)
    sep_us = ms * 1e3 / K

    calls = max(1, -(-K // T))

    def clip():
        for _ in range(calls):
            bn.forward_steps(xd)

    clip()
    ms, _ = timed(clip, stream)
    fs_us = ms * 1e3 / (calls * T)

    esz = 2 if sp.dtype == "bf16" else 4
    flops = 2 * B * H * W * C * Ci + 2 * B * C * Ho * Wo * kT * sp.kernel[1] * sp.kernel[2]
    pk = sp.pool_kernel[0]
    nbytes = (B * Ci * H * W * esz + 2 * (kT - 1) * B * C * Ho * Wo * 4
              + (pk + 1) * B * C * 4 + B * C * esz + C * Ci * 4 + C * kT * 9 * 4)
    ridge = PEAK_VALU_F32_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)

    def roof(us):
        if flops / nbytes >= ridge:
            a = flops / (us * 1e-6) / 1e12
            return {"bound": "alu", "achieved": round(a, 3), "peak": PEAK_VALU_F32_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(a / PEAK_VALU_F32_TFLOPS, 5)}
        a = nbytes / (us * 1e-6) / 1e9
        return {"bound": "hbm", "achieved": round(a, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(a / PEAK_HBM_GBS, 5)}

    return {"workload": sp.name, "batch": B, "dtype": sp.dtype,
            "fused_step": round(B / (fused_us * 1e-6), 1), "fused_us_per_step": round(fused_us, 3),
            "separate_step": round(B / (sep_us * 1e-6), 1),
            "separate_us_per_step": round(sep_us, 3), "separate_pointwise_algo": pw.algo,
            "fused_forward_steps": round(B / (fs_us * 1e-6), 1),
            "fused_forward_steps_us_per_frame": round(fs_us, 3),
            "flops_per_step": flops, "bytes_per_step": nbytes, "roofline": roof(fused_us)}


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

    import torch

    from paper_2204_03418_amd import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    K = args.steps

    wk = Workload(args.workload, dev, args.algo)
    c = wk.c
    # warm-up: past the delay so every timed step emits, and long enough
    # (WARM_MS of steps) that the clocks have left their idle state
    warm = warm_up(wk, args.warmup)

    # (i) eager forward_step calls: the headline number
    ms, reps, value = wk.eager(K)
    ms_per_step = ms / K

    # dominant kernel: the conv step alone, launched back to back (every step
    # emits, so each launch is one full contraction + ring update + emit)
    kern_us = wk.kernel_us(K)
    roof = wk.roofline(kern_us)
    roof["traffic"] = measured_traffic(args.workload)
    roof.update({"kernel": f"conv step ({wk.co.algo})", "kernel_avg_us": round(kern_us, 3),
                 "flops_per_launch": wk.flops, "bytes_per_launch": wk.nbytes,
                 "launches_per_region": K, "regions": reps})

    modes = {"eager_forward_step": round(value, 1)}
    modes_roof = {}
    if not args.no_modes:
        modes["graph_replay"] = round(wk.graph(K), 1)
        us_frame = wk.forward_steps(K)
        modes["forward_steps"] = round(c.batch / (us_frame * 1e-6), 1)
        fs = {"persistent": bool(wk.co.steps_fused(wk.T)), "us_per_frame": round(us_frame, 3),
              "flops_per_frame": wk.flops, "io_bytes_per_frame": wk.io_bytes}
        # per frame the persistent launch does the step's FLOPs but moves only
        # the frame and its output (the partial sums stay on chip)
        fs.update(wk.roofline(us_frame, nbytes=wk.io_bytes))
        modes_roof["forward_steps"] = fs
        fused = wk.fused_convpool(K)
        if fused is not None:
            modes["fused_convpool_step"] = round(fused[0], 1)
            modes["fused_convpool_forward_steps"] = round(fused[1], 1)
        if args.cold:
            v, cr = wk.cold(K)
            modes["cold_conv_step"] = round(v, 1)
            modes_roof["cold_conv_step"] = cr

    table = {}
    bneck = None
    if not args.no_workloads:
        for name in synth.WORKLOADS:
            table[name] = workload_entry(wk if name == args.workload else None, name, dev, K,
                                         args.algo, args.warmup)
        bneck = bottleneck_entry(dev, K)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wk, args.cpu_seconds)

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
                   "padding": list(c.padding), "frames": wk.T, "algo": wk.co.algo,
                   "pool": None if wk.wl.pool is None else
                   {"kind": wk.wl.pool.kind, "kernel": list(wk.wl.pool.kernel),
                    "stride": list(wk.wl.pool.stride)},
                   "timing": f"median of >= {MIN_REPS} repetitions of {K} steps "
                             f"({reps} here), HIP events on the launch stream"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "modes": modes,
        "modes_roofline": modes_roof,
        "workloads": table,
        "bottleneck": bneck,
    }
    print(json.dumps(out))


def warm_up(wk, steps):
    """At least `steps` untimed steps, past the layer's delay, and more until
    WARM_MS of them have run; returns the number of warm-up steps."""
    import torch
    n = max(steps, wk.delay + 2)
    wk.steps(n)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < WARM_MS:
        wk.steps(16)
        n += 16
        torch.cuda.synchronize()
    return n


def workload_entry(wk, name, dev, K, algo, warmup):
    """Eager step, its convolution kernel and forward_steps of one named
    workload, each with its roofline entry."""
    import torch
    if wk is None:
        wk = Workload(name, dev, algo)
        warm_up(wk, warmup)
    ms, _, value = wk.eager(K)
    kern_us = wk.kernel_us(K)
    us_frame = wk.forward_steps(K)
    e = {"batch": wk.c.batch, "algo": wk.co.algo, "dtype": wk.c.dtype,
         "eager_forward_step": round(value, 1), "ms_per_step": round(ms / K, 6),
         "kernel_avg_us": round(kern_us, 3), "flops_per_step": wk.flops,
         "bytes_per_step": wk.nbytes, "roofline": wk.roofline(kern_us),
         "forward_steps": round(wk.c.batch / (us_frame * 1e-6), 1),
         "forward_steps_us_per_frame": round(us_frame, 3),
         "forward_steps_persistent": bool(wk.co.steps_fused(wk.T)),
         "forward_steps_roofline": wk.roofline(us_frame, nbytes=wk.io_bytes)}
    fused = wk.fused_convpool(K)
    if fused is not None:
        # depthwise conv + global pool in one launch per step / per clip (the
        # intermediate frame stays on chip); priced on the conv's FLOPs and
        # the clip bytes read
        us_fused = wk.c.batch / fused[1] * 1e6
        e["fused_convpool_step"] = round(fused[0], 1)
        e["fused_convpool_forward_steps"] = round(fused[1], 1)
        e["fused_convpool_forward_steps_us_per_frame"] = round(us_fused, 3)
        e["fused_convpool_forward_steps_roofline"] = wk.roofline(us_fused, nbytes=wk.in_bytes)
    traffic = measured_traffic(name)
    if traffic is not None:
        e["roofline"]["traffic"] = traffic
    return e


def cpu_baseline(wk, seconds):
    """The oracle's sliding-window driver stepping the same frames on the host
    cores (float64, OpenMP over (b, o)), bounded to about `seconds` of work:
    all streams at the host's thread count, and one stream at one thread
    (streams are independent, so one stream is 1/B of a step's work)."""
    import oracle

    wl, c = wk.wl, wk.c
    xs = wk.x_cpu.float().double().numpy()
    w = wk.w_cpu.float().double().numpy()
    b = None if wk.b_cpu is None else wk.b_cpu.float().double().numpy()
    T = xs.shape[2]

    def driver():
        co = oracle.ContinualConv(w, b, stride=c.stride, padding=c.padding,
                                  dilation=c.dilation, groups=c.groups)
        po = None
        if wl.pool is not None:
            po = oracle.ContinualPool(wl.pool.kind, wl.pool.kernel, wl.pool.stride,
                                      wl.pool.padding, count_include_pad=wl.pool.count_include_pad,
                                      spatial_dims=len(wl.pool.in_size))
        return co, po

    def run(frames, secs):
        co, po = driver()

        def step(i):
            y = co.forward_step(frames[:, :, i % T])
            if po is not None and y is not None:
                po.forward_step(y)

        i0 = co.delay + (po.delay if po else 0) + 1
        for i in range(i0):
            step(i)
        t0 = time.perf_counter()
        k = 0
        while time.perf_counter() - t0 < secs or k == 0:
            step(i0 + k)
            k += 1
        return k, time.perf_counter() - t0

    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    threads = oracle.max_threads()
    k, dt = run(xs, seconds)
    out = {"value": round(c.batch * k / dt, 3), "unit": "stream-frames/s", "cores": threads,
           "kind": "oracle",
           "sample": f"{k} steps of all {c.batch} streams after the delay ({dt:.1f} s, float64, "
                     f"OpenMP over (b, o), {threads} threads); cpu: {cpu_model}"}
    oracle.set_threads(1)
    try:
        k1, dt1 = run(xs[:1], seconds)
    finally:
        oracle.set_threads(threads)
    out["one_thread"] = {"value": round(k1 / dt1, 3), "unit": "stream-frames/s", "cores": 1,
                         "sample": f"{k1} steps of one of the {c.batch} streams after the delay "
                                   f"({dt1:.1f} s, float64, one thread)"}
    return out


if __name__ == "__main__":
    main()
