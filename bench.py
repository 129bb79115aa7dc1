#!/usr/bin/env python3
"""Benchmark: one DeepSeek-V3-shape pruned, mixed-precision MoE layer, decode.

Workload (synthetic, seeded): hidden 7168, expert intermediate 2048, 256 routed
experts pruned to 192 (r = 0.75), 1 shared expert, sigmoid router with 8
groups / 4 groups per token / 8 experts per token, routed scale 2.5; routed
gate/up 3-bit, routed down 4-bit, shared expert 4-bit, blocks of 32 with
binary16 scales; weights N(0, 0.02) generated on the GPU and quantized by the
library's quantizer; activations bf16 N(0, 1), router logits fp32 N(0, 1);
batch 1 (one token per forward).

A step is one full layer forward (route, bucket, gate/up + SwiGLU, down,
combine) on the next of 64 pre-generated input sets, rotating over 4
independently seeded layers so that neither the routed experts nor the shared
expert are served from the 256 MB Infinity Cache between uses.  Steps are
replayed from a HIP graph; every input is resident in HBM before timing.

Reported: tokens/s (the value), effective weight GB/s per step (codes + scales
of the distinct tensors each step touches), the dominant kernel's roofline
(gate/up dequant-GEMV, HBM bound, timed with HIP events recorded by the
library around each stage), and the CPU oracle on a bounded sample.
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

METRIC = "V3-shape MoE layer decode tokens/s + effective weight GB/s vs HBM peak"
HBM_PEAK_GBPS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0   # dense fp16 / bf16 matrix peak of one MI355X

# HBM bytes per gate/up launch at batch 1 from rocprofv3 FETCH_SIZE + WRITE_SIZE,
# each scaled by the same counter's reading for a plain 1 GiB copy (factors
# 2.0 and 1.0; see profiles/gateup1_route_kernel_decode_b1_traffic.md).  Valid
# only for the kernel sources the counters were taken on, identified by their
# sha256: any change to them reports traffic as null until the counters are
# retaken.
GATEUP_TRAFFIC = {
    "bytes": 127422233,
    "sources": {
        "paper_2509_25689_amd/csrc/decode.hip": "115a87a545c2200d351c0a348f881c93749bd8e2a0a9df9136ea075383b65585",
        "paper_2509_25689_amd/csrc/layout.h": "ec9f6185567429769228f45977ef62d3009e3530746c8104eb4a54119a1468b5",
        "paper_2509_25689_amd/csrc/route_wave.h": "eb3854b178047d6ade2936070a4e74a0b27d75ca6945b4e3099ddd0a53941b6d",
    },
}


def gateup_traffic():
    """The measured traffic if the gate/up kernel is still the one measured, else None."""
    import hashlib
    for rel, digest in GATEUP_TRAFFIC["sources"].items():
        try:
            with open(os.path.join(ROOT, rel), "rb") as f:
                if hashlib.sha256(f.read()).hexdigest() != digest:
                    return None
        except OSError:
            return None
    return GATEUP_TRAFFIC["bytes"]


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=2560, help="timed batch-1 forwards (exactly this many)")
    p.add_argument("--warmup", type=int, default=256, help="untimed forwards before the timed ones")
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--layers", type=int, default=4, help="independently seeded layers rotated per step")
    p.add_argument("--sets", type=int, default=64, help="input sets (x, logits) per layer")
    p.add_argument("--kernel-steps", type=int, default=256, help="eager forwards timed per stage")
    p.add_argument("--cpu-steps", type=int, default=3,
                   help="oracle forwards per timed group in the CPU baseline; the value is the median of 3 "
                        "groups (0 = skip)")
    p.add_argument("--prefill-steps", type=int, default=10, help="2048-token prefill forwards timed (0 = skip)")
    p.add_argument("--b16-steps", type=int, default=2560, help="16-token decode steps timed (0 = skip)")
    p.add_argument("--k6-steps", type=int, default=2560,
                   help="batch-1 decode steps timed with 6 experts per token (0 = skip)")
    p.add_argument("--gate-steps", type=int, default=2560,
                   help="batch-1 decode steps timed with logits from the router gate (0 = skip)")
    p.add_argument("--wide-steps", type=int, default=2560,
                   help="batch-1 decode steps timed with a 6-bit shared expert (0 = skip)")
    p.add_argument("--stack-steps", type=int, default=580,
                   help="timed layer forwards of the 58-layer stack leg (0 = skip)")
    p.add_argument("--peak-reps", type=int, default=5, help="timed launches of each peak probe (0 = skip)")
    p.add_argument("--mode", choices=("all", "decode", "prefill", "copy", "stack", "sweep", "peaks"),
                   default="all",
                   help="all: batch-1 decode line with 16-token, prefill and CPU legs; decode / prefill: "
                        "one leg only (for profiling); copy: a plain 1 GiB device copy whose HBM counters "
                        "calibrate the profiler's byte counts; stack: 58 independent layers; sweep: kept "
                        "experts x widths x tokens x routing on the decode path; peaks: measured streaming-read "
                        "and MFMA rates")
    return p.parse_args()


class Hip:
    """The few HIP runtime calls the benchmark needs for events (torch's runtime)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so.7")
        for name, args in (("hipEventCreate", [ctypes.POINTER(ctypes.c_void_p)]),
                           ("hipEventCreateWithFlags", [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]),
                           ("hipEventDestroy", [ctypes.c_void_p]),
                           ("hipEventSynchronize", [ctypes.c_void_p]),
                           ("hipEventRecord", [ctypes.c_void_p, ctypes.c_void_p]),
                           ("hipEventElapsedTime", [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                    ctypes.c_void_p])):
            getattr(self.lib, name).argtypes = args
            getattr(self.lib, name).restype = ctypes.c_int

    # timing-only events: no system-scope fence (cache writeback and
    # invalidation) when they are recorded, so they barely perturb the kernels
    # they bracket
    DISABLE_SYSTEM_FENCE = 0x20000000

    def event(self):
        e = ctypes.c_void_p()
        assert self.lib.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE) == 0
        return e.value

    def record(self, e, stream):
        assert self.lib.hipEventRecord(e, stream) == 0

    def elapsed_ms(self, a, b, strict=True):
        assert self.lib.hipEventSynchronize(b) == 0
        ms = ctypes.c_float()
        rc = self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b)
        if rc != 0:
            if strict:
                raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
            return None
        return ms.value

    def destroy(self, e):
        self.lib.hipEventDestroy(e)

    def graph_upload(self, graph_exec, stream):
        """Upload an instantiated graph before it is timed, so that its first
        replay does not carry the upload."""
        fn = self.lib.hipGraphUpload
        fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        fn.restype = ctypes.c_int
        assert fn(graph_exec, stream) == 0


def build_layer(torch, moeq, synth, shape, plan, key, max_tokens):
    """N(0, 0.02) weights drawn on the GPU (seeded per tensor), quantized by
    moeq_quantize into the canonical packing, handed over as device pointers."""
    mask = synth.expert_mask(shape, key)
    bits_r, bits_s = synth.bit_plan(shape, plan, key)
    gen = torch.Generator(device="cuda")

    def tensor(kind, e, p, bits):
        rows, K = shape.rows_cols(p)
        gen.manual_seed(synth.seed_int("bench-w", key, kind, e, p))
        w = torch.randn((rows, K), generator=gen, device="cuda", dtype=torch.float32) * 0.02
        codes, scales = moeq.quantize(w, bits)
        return dict(bits=bits, codes=codes, scales=scales)

    routed = {int(e): tuple(tensor("r", e, p, int(bits_r[e, p])) for p in range(3))
              for e in range(shape.n_experts) if mask[e]}
    shared = [tuple(tensor("s", s, p, int(bits_s[s, p])) for p in range(3)) for s in range(shape.n_shared)]
    torch.cuda.synchronize()
    layer = moeq.Layer(shape, mask, routed, shared, max_tokens=max_tokens, device_weights=True)
    return layer, mask, bits_r, bits_s


def tensor_bytes(shape, bits, p):
    rows, K = shape.rows_cols(p)
    return rows * K * bits // 8 + rows * (K // 32) * 2


def prefill_bench(torch, np, moeq, synth, hip, steps, n=2048):
    """The 2048-token prefill: Zipf(1.1)-routed, per-tensor widths from {2,3,4}
    (p = 0.6, 0.2, 0.2), grouped GEMM path.  Returns a dict of measurements."""
    shape = synth.V3
    layer, mask, _, _ = build_layer(torch, moeq, synth, shape, "p234_602020", "bench-prefill", max_tokens=n)
    sets = 4
    xs = [torch.from_numpy(synth.activations(n, shape.hidden, "bench-pf-x", i).view(np.int16)).cuda()
          .view(torch.bfloat16) for i in range(sets)]
    lgs = [torch.from_numpy(synth.zipf_logits(n, mask, "bench-pf-l", i)).cuda() for i in range(sets)]
    y = torch.empty((n, shape.hidden), device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    for i in range(2):
        moeq.moeq_forward(layer.handle, xs[i % sets].data_ptr(), lgs[i % sets].data_ptr(), n, y.data_ptr(), stream)
    torch.cuda.synchronize()
    events = [[hip.event() for _ in range(moeq.MOEQ_STAGE_EVENTS)] for _ in range(steps)]
    for j in range(steps):
        moeq.moeq_set_stage_events(layer.handle, events[j])
        moeq.moeq_forward(layer.handle, xs[j % sets].data_ptr(), lgs[j % sets].data_ptr(), n, y.data_ptr(), stream)
    moeq.moeq_set_stage_events(layer.handle, None)
    torch.cuda.synchronize()
    st = np.array([[hip.elapsed_ms(ev[s], ev[s + 1]) for s in range(4)] for ev in events]).mean(axis=0)
    total = np.array([hip.elapsed_ms(ev[0], ev[4]) for ev in events]).mean()
    for ev in events:
        for e in ev:
            hip.destroy(e)
    layer.close()
    rows = n * (shape.top_k + shape.n_shared)
    f_gu = 2.0 * 2 * shape.hidden * shape.inter * rows
    f_dn = 2.0 * shape.hidden * shape.inter * rows
    tf = lambda f, ms: f / (ms * 1e-3) / 1e12
    return {"workload": f"DeepSeek-V3-shape layer prefill, {n} tokens, Zipf(1.1) routing over 192 kept experts, "
                        "per-tensor widths from {2,3,4} (p=0.6,0.2,0.2)",
            "tokens_per_s": round(n / (total * 1e-3), 1), "ms_per_step": round(total, 4),
            "useful_tflop_per_step": round((f_gu + f_dn) / 1e12, 4),
            "tflops": round(tf(f_gu + f_dn, total), 1),
            "mfma_frac": round(tf(f_gu + f_dn, total) / MFMA_F16_PEAK_TFLOPS, 4),
            "stage_ms": {"route_bucket": round(st[0], 4), "gate_up": round(st[1], 4), "down": round(st[2], 4),
                         "combine": round(st[3], 4)},
            "gate_up_tflops": round(tf(f_gu, st[1]), 1), "down_tflops": round(tf(f_dn, st[2]), 1),
            "gate_up_mfma_frac": round(tf(f_gu, st[1]) / MFMA_F16_PEAK_TFLOPS, 4),
            "steps": steps, "dtype": "fp16 MFMA, fp32 accumulate"}


def copy_calibration(torch, hip, nbytes=1 << 30, reps=4):
    """A plain device-to-device copy of known size: under rocprofv3 --pmc its
    FETCH_SIZE / WRITE_SIZE per dispatch give the factor that turns those
    counters into bytes."""
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").normal_()
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    e0, e1 = hip.event(), hip.event()
    stream = torch.cuda.current_stream().cuda_stream
    hip.record(e0, stream)
    for _ in range(reps):
        dst.copy_(src)
    hip.record(e1, stream)
    torch.cuda.synchronize()
    ms = hip.elapsed_ms(e0, e1) / reps
    hip.destroy(e0)
    hip.destroy(e1)
    return {"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "reps": reps, "ms_per_copy": round(ms, 4),
            "GBps_read_plus_write": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}


def peaks_leg(torch, hip, reps, read_bytes=4 << 30, mfma_wgs=2048, mfma_iters=4000):
    """Measured roofline denominators on this GPU: a streaming read of
    read_bytes (larger than every cache) with 16-byte coalesced loads, and a
    register-only binary16 MFMA loop over 8 workgroups of 4 waves per compute
    unit.  Median and best of `reps` timed launches after two untimed ones."""
    import statistics
    from paper_2509_25689_amd import peaks
    lib = peaks.load()
    stream = torch.cuda.current_stream().cuda_stream
    src = torch.randint(0, 1 << 30, (read_bytes // 4,), dtype=torch.int32, device="cuda")
    sink = torch.empty(lib.moeq_peaks_read_workgroups(read_bytes), dtype=torch.int32, device="cuda")
    fsink = torch.empty(mfma_wgs * 256, dtype=torch.float32, device="cuda")
    read_ms, mfma_ms = [], []
    for i in range(reps + 2):
        e = [hip.event() for _ in range(4)]
        hip.record(e[0], stream)
        assert lib.moeq_peaks_stream_read(src.data_ptr(), read_bytes, sink.data_ptr(), stream) == 0
        hip.record(e[1], stream)
        hip.record(e[2], stream)
        assert lib.moeq_peaks_mfma(mfma_wgs, mfma_iters, fsink.data_ptr(), stream) == 0
        hip.record(e[3], stream)
        torch.cuda.synchronize()
        if i >= 2:
            read_ms.append(hip.elapsed_ms(e[0], e[1]))
            mfma_ms.append(hip.elapsed_ms(e[2], e[3]))
        for x in e:
            hip.destroy(x)
    del src
    flops = lib.moeq_peaks_mfma_flops(mfma_wgs, mfma_iters)
    gbps = [read_bytes / (m * 1e-3) / 1e9 for m in read_ms]
    tflops = [flops / (m * 1e-3) / 1e12 for m in mfma_ms]
    return {"stream_read_GBps_median": round(statistics.median(gbps), 1), "stream_read_GBps_best": round(max(gbps), 1),
            "stream_read_bytes": read_bytes,
            "mfma_f16_TFLOPs_median": round(statistics.median(tflops), 1), "mfma_f16_TFLOPs_best": round(max(tflops), 1),
            "mfma_workgroups": mfma_wgs, "mfma_iters": mfma_iters, "reps": reps}


def cpu_baseline(shape, steps, batch):
    """The oracle, as it stands, on `steps` forwards of the same workload shape.

    Inputs: a seeded layer whose touched experts hold random packed codes
    (the oracle's cost does not depend on code values), seeded x and logits.
    Timed: routing, bucketing, dequantization of every touched tensor and the
    float64 expert products and combine -- the whole forward."""
    import numpy as np
    from inputs import synth
    from oracle import bucket, moe, router
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    key = "bench-cpu"
    mask = synth.expert_mask(shape, key)
    bits_r, bits_s = synth.bit_plan(shape, "gu3_d4_sh4", key)

    def packed(kind, e, p):
        rows, K = shape.rows_cols(p)
        bits = int(bits_r[e, p] if kind == "r" else bits_s[e, p])
        codes, scales = synth.random_packed(rows, K, bits, key, kind, e, p)
        return dict(bits=bits, codes=codes, scales=scales)

    xs = [synth.activations(batch, shape.hidden, key, "x", i) for i in range(3 * steps)]
    lgs = [synth.normal_logits(batch, shape.n_experts, key, "l", i) for i in range(3 * steps)]
    # untimed: materialise the packed tensors the sample touches
    need = set()
    for lg in lgs:
        idx, _ = router.route(lg, mask, n_group=shape.n_group, topk_group=shape.topk_group,
                              top_k=shape.top_k, routed_scale=shape.routed_scale)
        need |= set(int(e) for e in np.unique(idx))
    store = {e: tuple(packed("r", e, p) for p in range(3)) for e in need}
    shared_t = [tuple(packed("s", s, p) for p in range(3)) for s in range(shape.n_shared)]
    Ks = [shape.rows_cols(p)[1] for p in range(3)]

    def forward(i):
        idx, w = router.route(lgs[i], mask, n_group=shape.n_group, topk_group=shape.topk_group,
                              top_k=shape.top_k, routed_scale=shape.routed_scale)
        bucket.bucket(idx, shape.n_experts)
        shared = [tuple(moe.dequant_tensor(t, K) for t, K in zip(tr, Ks)) for tr in shared_t]
        moe.moe_forward(xs[i], idx, w,
                        lambda e: tuple(moe.dequant_tensor(t, K) for t, K in zip(store[e], Ks)), shared)

    group_s = []
    for g in range(3):
        t0 = time.perf_counter()
        for i in range(g * steps, (g + 1) * steps):
            forward(i)
        group_s.append(time.perf_counter() - t0)
    med = sorted(group_s)[1]
    cores = len(os.sched_getaffinity(0))
    return {"value": steps * batch / med, "unit": "tokens/s",
            "cores": blas_threads if blas_threads else cores, "kind": "oracle",
            "sample": f"median of 3 groups of {steps} forwards of {batch} token(s) each (group times "
                      f"{', '.join(f'{t:.2f}' for t in group_s)} s), same V3 shape and bit plan, random packed "
                      f"codes; host cores visible {cores}"}


def random_layer(torch, moeq, synth, shape, plan, key, max_tokens):
    """A layer whose codes are uniform random bytes and whose scales are
    spread around the block quantizer's typical d for N(0, 0.02) weights
    (synth.device_random_packed, keyed per tensor), generated directly on the
    GPU: used where quantizing real draws would take too long (the 58-layer
    stack, the sweep)."""
    mask = synth.expert_mask(shape, key)
    bits_r, bits_s = synth.bit_plan(shape, plan, key)

    def tensor(kind, e, p, bits):
        rows, K = shape.rows_cols(p)
        codes, scales = synth.device_random_packed(torch, rows, K, bits, key, kind, e, p)
        return dict(bits=bits, codes=codes, scales=scales)

    routed = {int(e): tuple(tensor("r", e, p, int(bits_r[e, p])) for p in range(3))
              for e in range(shape.n_experts) if mask[e]}
    shared = [tuple(tensor("s", s, p, int(bits_s[s, p])) for p in range(3)) for s in range(shape.n_shared)]
    torch.cuda.synchronize()
    layer = moeq.Layer(shape, mask, routed, shared, max_tokens=max_tokens, device_weights=True)
    del routed, shared
    return layer, mask, bits_r, bits_s


def step_bytes_of(np, shape, layer, bits_r, bits_s, logits):
    """Algorithmic bytes of one forward: codes + scales of every distinct
    tensor it touches (routed experts chosen by any token, plus the shared
    experts), and of each kind (gate/up, down)."""
    idx, _ = layer.route(logits)
    experts = np.unique(idx.cpu().numpy())
    g = sum(tensor_bytes(shape, int(bits_r[e, 0]), 0) + tensor_bytes(shape, int(bits_r[e, 1]), 1) for e in experts)
    d = sum(tensor_bytes(shape, int(bits_r[e, 2]), 2) for e in experts)
    for s in range(shape.n_shared):
        g += tensor_bytes(shape, int(bits_s[s, 0]), 0) + tensor_bytes(shape, int(bits_s[s, 1]), 1)
        d += tensor_bytes(shape, int(bits_s[s, 2]), 2)
    return g, d, len(experts)


def decode_leg(torch, np, moeq, synth, hip, shape, layers, B, R, steps, warmup, kernel_steps, key,
               zipf=False, path=None, gate=False):
    """Batch-B decode over the given layers (step s uses layer s % NL and
    input set s), replayed from one HIP graph with inputs resident in HBM.
    With gate, each layer holds a float32 router weight and computes its own
    logits (moeq_forward with NULL logits).  Returns timing, bytes and
    per-stage kernel durations."""
    NL = len(layers)
    n_sets = R * NL
    if path is not None:
        for L, *_ in layers:
            L.set_path(path)
    xs, lgs = [], []
    for i in range(n_sets):
        xb = synth.activations(B, shape.hidden, key, "x", i)
        xs.append(torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16))
        mask = layers[i % NL][1]
        lg = synth.zipf_logits(B, mask, key, "l", i) if zipf else synth.normal_logits(B, shape.n_experts, key, "l", i)
        lgs.append(torch.from_numpy(lg).cuda())
    if gate:
        for li, (L, *_) in enumerate(layers):
            L.set_router_weight(synth.router_weight(shape.n_experts, shape.hidden, key, "wr", li))
        lgs = [layers[i % NL][0].router_logits(xs[i]) for i in range(n_sets)]
    ys = [torch.empty((B, shape.hidden), device="cuda") for _ in range(NL)]
    gu_bytes, down_bytes, n_exp = [], [], []
    for i in range(n_sets):
        layer, mask, bits_r, bits_s = layers[i % NL]
        g, d, ne = step_bytes_of(np, shape, layer, bits_r, bits_s, lgs[i])
        gu_bytes.append(g)
        down_bytes.append(d)
        n_exp.append(ne)
    io_bytes = B * (shape.hidden * 2 + shape.n_experts * 4 + shape.hidden * 4)
    if gate:
        io_bytes += shape.n_experts * shape.hidden * 4

    def run_step(i, stream):
        layer = layers[i % NL][0]
        moeq.moeq_forward(layer.handle, xs[i].data_ptr(), 0 if gate else lgs[i].data_ptr(), B,
                          ys[i % NL].data_ptr(), stream)

    # one eager forward per layer before any capture (first-use set-up of
    # the library's kernels happens outside a graph)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(NL):
            run_step(i, side.cuda_stream)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    def capture(order):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            st = torch.cuda.current_stream().cuda_stream
            for i in order:
                run_step(i % n_sets, st)
        return g

    # warm-up: `warmup` forwards, then exactly `steps` timed forwards that
    # continue the rotation (forward i of the timed run uses set warmup + i)
    if warmup > 0:
        capture(list(range(warmup))).replay()
    timed = capture([(warmup + i) % n_sets for i in range(steps)])
    hip.graph_upload(timed.raw_cuda_graph_exec(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    timed.replay()
    t1.record()
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    ms_per_step = total_ms / steps
    del timed

    # per-stage kernel durations: timing-only events recorded by the library
    # between its kernels, over kernel_steps eager forwards
    KT = min(kernel_steps, n_sets)
    events = [[hip.event() for _ in range(moeq.MOEQ_STAGE_EVENTS)] for _ in range(KT)]
    stream = torch.cuda.current_stream().cuda_stream
    for j in range(KT):
        moeq.moeq_set_stage_events(layers[j % NL][0].handle, events[j])
        run_step(j, stream)
    for L, *_ in layers:
        moeq.moeq_set_stage_events(L.handle, None)
    torch.cuda.synchronize()
    stage_ms = np.array([[hip.elapsed_ms(ev[q], ev[q + 1]) for q in range(4)] for ev in events])
    for ev in events:
        for e in ev:
            hip.destroy(e)
    if path is not None:
        for L, *_ in layers:
            L.set_path(moeq.MOEQ_PATH_AUTO)
    if gate:
        for L, *_ in layers:
            L.set_router_weight(None)
    stage_mean = stage_ms.mean(axis=0)
    mean_step_bytes = float(np.mean(gu_bytes) + np.mean(down_bytes) + io_bytes)
    gu_launch = float(np.mean(gu_bytes[:KT]))
    dn_launch = float(np.mean(down_bytes[:KT]))
    return {
        "tokens_per_s": steps * B / (total_ms * 1e-3), "ms_per_step": ms_per_step, "steps": steps,
        "bytes_per_step": mean_step_bytes, "GBps": mean_step_bytes / (ms_per_step * 1e-3) / 1e9,
        "distinct_experts_per_step": float(np.mean(n_exp)),
        "stage_ms": stage_mean,
        "gu_launch_bytes": gu_launch, "dn_launch_bytes": dn_launch,
        "gu_GBps": gu_launch / (stage_mean[1] * 1e-3) / 1e9, "dn_GBps": dn_launch / (stage_mean[2] * 1e-3) / 1e9,
    }


def stack_leg(torch, np, moeq, synth, hip, steps, n_layers=58):
    """58 independent layers of the V3 decode shape (per-tensor widths from
    {2,3,4} with p = 0.7, 0.1, 0.2), batch 1: one step is the 58 layer
    forwards in sequence, each on its own x and logits."""
    shape = synth.V3
    t0 = time.perf_counter()
    layers = [random_layer(torch, moeq, synth, shape, "p234_701020", f"bench-stack-{li}", max_tokens=1)
              for li in range(n_layers)]
    build_s = time.perf_counter() - t0
    resident = sum(L.bytes()[0] for L, *_ in layers)
    r = decode_leg(torch, np, moeq, synth, hip, shape, layers, 1, 2, max(steps, 2 * n_layers), n_layers,
                   n_layers, "bench-stack")
    per_stack_ms = r["ms_per_step"] * n_layers
    out = {"workload": f"{n_layers} independent V3-shape layers (192 of 256 experts kept each), batch 1, "
                       "per-tensor widths from {2,3,4} with p = (0.7, 0.1, 0.2), random codes",
           "resident_weight_GB": round(resident / 1e9, 2), "build_s": round(build_s, 1),
           "ms_per_stack_step": round(per_stack_ms, 4), "tokens_per_s": round(1e3 / per_stack_ms, 1),
           "bytes_per_stack_step_GB": round(r["bytes_per_step"] * n_layers / 1e9, 3),
           "GBps": round(r["GBps"], 1), "hbm_frac": round(r["GBps"] / HBM_PEAK_GBPS, 4),
           "layer_forwards_timed": r["steps"]}
    for L, *_ in layers:
        L.close()
    return out


def sweep_leg(torch, np, moeq, synth, hip, steps):
    """Decode-path sweep: kept experts {256, 192, 128} x widths {uniform 2,
    uniform 4, mixed (shared 4-bit, routed 2-bit)} x tokens {1, 16, 64} x
    routing {N(0,1) logits, Zipf(1.1)}."""
    import dataclasses
    rows = []
    for kept in (256, 192, 128):
        shape = dataclasses.replace(synth.V3, n_kept=kept)
        for plan in ("all2", "all4", "mixed"):
            layer = random_layer(torch, moeq, synth, shape, plan, f"bench-sweep-{kept}-{plan}", max_tokens=64)
            for n in (1, 16, 64):
                for zipf in (False, True):
                    r = decode_leg(torch, np, moeq, synth, hip, shape, [layer], n, 32, steps, 32, 32,
                                   f"bench-sweep-{kept}-{plan}-{n}-{int(zipf)}", zipf=zipf,
                                   path=moeq.MOEQ_PATH_DECODE)
                    rows.append({"kept": kept, "bits": plan, "tokens": n, "routing": "zipf" if zipf else "normal",
                                 "tokens_per_s": round(r["tokens_per_s"], 1), "us_per_step": round(r["ms_per_step"] * 1e3, 2),
                                 "distinct_experts": round(r["distinct_experts_per_step"], 1),
                                 "GBps": round(r["GBps"], 1), "hbm_frac": round(r["GBps"] / HBM_PEAK_GBPS, 4)})
                    print(f"sweep point {len(rows)}/54: {rows[-1]}", file=sys.stderr, flush=True)
            layer[0].close()
    return rows


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(every run uses exactly one MI355X); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from inputs import synth
    from paper_2509_25689_amd import moeq

    shape = synth.V3
    B, NL, R = args.batch, args.layers, args.sets
    hip = Hip()
    torch.cuda.set_device(0)
    if args.mode == "copy":
        print(json.dumps(copy_calibration(torch, hip)), flush=True)
        return
    if args.mode == "prefill":
        print(json.dumps({"prefill": prefill_bench(torch, np, moeq, synth, hip, max(1, args.prefill_steps))}),
              flush=True)
        return
    if args.mode == "stack":
        print(json.dumps({"stack": stack_leg(torch, np, moeq, synth, hip, args.stack_steps)}), flush=True)
        return
    if args.mode == "peaks":
        print(json.dumps({"peaks": peaks_leg(torch, hip, max(1, args.peak_reps))}), flush=True)
        return
    peaks = peaks_leg(torch, hip, args.peak_reps) if args.mode == "all" and args.peak_reps > 0 else None
    if args.mode == "sweep":
        print(json.dumps({"sweep": sweep_leg(torch, np, moeq, synth, hip, args.steps)}), flush=True)
        return

    layers = [build_layer(torch, moeq, synth, shape, "gu3_d4_sh4", f"bench-layer-{li}", max_tokens=64)
              for li in range(NL)]
    resident = sum(L.bytes()[0] for L, *_ in layers)
    r = decode_leg(torch, np, moeq, synth, hip, shape, layers, B, R, args.steps, args.warmup,
                   args.kernel_steps, "bench")
    st = r["stage_ms"]
    out = {
        "metric": METRIC,
        "value": round(r["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": r["steps"],
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "arithmetic": "binary16 operands (bf16 x exact after a power-of-two prescale per block of 32; exact "
                      "code values; SwiGLU h rounded once to binary16 after a power-of-two prescale per block), "
                      "float32 accumulation; router scores float64 rounded once to float32",
        "data": "synthetic",
        "config": {
            "workload": f"DeepSeek-V3-shape MoE layer decode, batch {B}: hidden 7168, inter 2048, "
                        "192 of 256 routed experts kept, 1 shared, 8 groups / top-4 groups / top-8, "
                        "routed gate/up 3-bit, down 4-bit, shared 4-bit, block 32, fp16 scales",
            "global_batch": B, "seq_len": 1, "parallelism": "none (1 GPU)",
            "layers_rotated": NL, "input_sets_per_layer": R, "graph_replay": True,
            "resident_weight_GB": round(resident / 1e9, 3),
        },
        "effective_weight_GBps": round(r["GBps"], 1),
        "hbm_frac": round(r["GBps"] / HBM_PEAK_GBPS, 4),
        "bytes_per_step": int(r["bytes_per_step"]),
        "stage_us": {"route_bucket": round(st[0] * 1e3, 2), "gate_up": round(st[1] * 1e3, 2),
                     "down": round(st[2] * 1e3, 2), "combine": round(st[3] * 1e3, 2)},
        "stage_note": ("eager forwards timed by events between the stages; at batch 1 the routing runs inside "
                       "the gate/up kernel and the combine inside the down kernel, so those two stages hold no "
                       "launch and show only the events' own cost"),
        "down_GBps": round(r["dn_GBps"], 1),
        "roofline": {"bound": "hbm",
                     "kernel": ("gateup1_route_kernel (routing + fused dequant-GEMV gate/up + SwiGLU)" if B == 1
                                else "gateupn_kernel (fused dequant-GEMV gate/up + SwiGLU, 2 tokens per pass)"),
                     "achieved": round(r["gu_GBps"], 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(r["gu_GBps"] / HBM_PEAK_GBPS, 4), "traffic": gateup_traffic() if B == 1 else None,
                     "bytes_per_launch": int(r["gu_launch_bytes"])},
    }
    if peaks:
        meas = peaks["stream_read_GBps_median"]
        out["peaks_measured"] = peaks
        out["roofline"]["peak_measured"] = meas
        out["roofline"]["frac_of_measured_peak"] = round(r["gu_GBps"] / meas, 4)
        out["hbm_frac_of_measured_read"] = round(r["GBps"] / meas, 4)
    if args.mode == "all" and args.gate_steps > 0:
        # the same layers, logits computed in the forward by the router gate x W_r^T
        rg = decode_leg(torch, np, moeq, synth, hip, shape, layers, 1, R, args.gate_steps, 64, 64, "bench-gate",
                        gate=True)
        out["decode_b1_with_gate"] = {"tokens_per_s": round(rg["tokens_per_s"], 1),
                                      "us_per_step": round(rg["ms_per_step"] * 1e3, 2),
                                      "route_stage_us": round(rg["stage_ms"][0] * 1e3, 2),
                                      "bytes_per_step": int(rg["bytes_per_step"]), "GBps": round(rg["GBps"], 1)}
    if args.mode == "all" and args.b16_steps > 0:
        r16 = decode_leg(torch, np, moeq, synth, hip, shape, layers, 16, 16, args.b16_steps, 64, 64, "bench-b16")
        out["decode_b16"] = {"tokens_per_s": round(r16["tokens_per_s"], 1),
                             "us_per_step": round(r16["ms_per_step"] * 1e3, 2),
                             "distinct_experts_per_step": round(r16["distinct_experts_per_step"], 1),
                             "bytes_per_step": int(r16["bytes_per_step"]), "GBps": round(r16["GBps"], 1),
                             "hbm_frac": round(r16["GBps"] / HBM_PEAK_GBPS, 4)}
    for L, *_ in layers:
        L.close()
    if args.mode == "all" and args.k6_steps > 0:
        # Section 3.2: after keeping r = 0.75 of the experts, ceil(r * 8) = 6 per token
        import dataclasses
        shape6 = dataclasses.replace(shape, top_k=6)
        layers6 = [random_layer(torch, moeq, synth, shape6, "gu3_d4_sh4", f"bench-k6-{li}", max_tokens=1)
                   for li in range(NL)]
        r6 = decode_leg(torch, np, moeq, synth, hip, shape6, layers6, 1, R, args.k6_steps, 64, 64, "bench-k6")
        out["decode_b1_k6"] = {"tokens_per_s": round(r6["tokens_per_s"], 1),
                               "us_per_step": round(r6["ms_per_step"] * 1e3, 2),
                               "bytes_per_step": int(r6["bytes_per_step"]), "GBps": round(r6["GBps"], 1),
                               "hbm_frac": round(r6["GBps"] / HBM_PEAK_GBPS, 4)}
        for L, *_ in layers6:
            L.close()
    if args.mode == "all" and args.wide_steps > 0:
        # Section 3.3's Q6 upgrade of a medium tensor: the shared expert at 6 bits
        layers_w = [random_layer(torch, moeq, synth, shape, "gu3_d4_sh6", f"bench-sh6-{li}", max_tokens=1)
                    for li in range(NL)]
        rw = decode_leg(torch, np, moeq, synth, hip, shape, layers_w, 1, R, args.wide_steps, 64, 64, "bench-sh6")
        st = rw["stage_ms"]
        out["decode_b1_shared_6bit"] = {"tokens_per_s": round(rw["tokens_per_s"], 1),
                                        "us_per_step": round(rw["ms_per_step"] * 1e3, 2),
                                        "stage_us": {"route_bucket": round(st[0] * 1e3, 2),
                                                     "gate_up": round(st[1] * 1e3, 2),
                                                     "down": round(st[2] * 1e3, 2), "combine": round(st[3] * 1e3, 2)},
                                        "bytes_per_step": int(rw["bytes_per_step"]), "GBps": round(rw["GBps"], 1),
                                        "hbm_frac": round(rw["GBps"] / HBM_PEAK_GBPS, 4)}
        for L, *_ in layers_w:
            L.close()
    if args.mode == "all" and args.prefill_steps > 0:
        out["prefill"] = prefill_bench(torch, np, moeq, synth, hip, args.prefill_steps)
        if peaks:
            m = peaks["mfma_f16_TFLOPs_median"]
            out["prefill"]["mfma_peak_measured_TFLOPs"] = m
            out["prefill"]["mfma_frac_of_measured_peak"] = round(out["prefill"]["tflops"] / m, 4)
    if args.mode == "all" and args.stack_steps > 0:
        out["stack"] = stack_leg(torch, np, moeq, synth, hip, args.stack_steps)
        if peaks:
            out["stack"]["frac_of_measured_read"] = round(out["stack"]["GBps"] / peaks["stream_read_GBps_median"], 4)
    if args.mode == "all" and args.cpu_steps > 0:
        out["cpu_baseline"] = cpu_baseline(shape, args.cpu_steps, B)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
