"""Benchmark of the FGQ inference hot path on one MI355X.

One step = quantize the layer's fp32 input to uint8 with a dynamic per-tensor
scale (fgq_quantize_act) + the FGQ convolution (fgq_conv2d), on the
ResNet-50 conv3_x layer: 3x3, 128 -> 128 channels, 28x28, batch 32, stride 1,
pad 1, weights ternarized in groups of 4 input channels.  Weight preparation
(ternarization, folded-scale constants) happens once before timing, as for a
deployed model.

Timing: every step is captured into a HIP graph and replayed; the inputs and
outputs rotate over enough buffer sets (> 1 GiB) that neither the L2 nor the
256 MB Infinity Cache can hold them.  `value` is effective TOPS =
2*M*O*K / (wall time per step) with M = B*Ho*Wo, K = C*R*S.  The dominant
kernel (the convolution) is also timed alone with HIP events around graphs of
convolution launches on the same stream; its algorithmic bytes per launch
give the roofline object.  The CPU baseline is the plain oracle, timed on a
bounded row sample of the same layer.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective TOPS (2*M*N*K/s) of fgq_conv2d at N=4 and N=64; % of int8/HBM roofline"
HBM_PEAK_GBS = 8000.0
INT8_PEAK_TOPS = 5000.0

LAYER = dict(B=32, H=28, W=28, C=128, O=128, R=3, S=3, stride=1, pad=1)
LAYER_1X1 = dict(B=32, H=56, W=56, C=256, O=64, R=1, S=1, stride=1, pad=0)
CALIB_COPY_BYTES = 64 << 20  # plain device copy used to calibrate FETCH_SIZE / WRITE_SIZE
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_conv_b32.json")
_CSRC = "paper_1705_01462_amd/csrc/"
# Sources of the convolution kernel that runs at each group size.
KERNEL_SOURCES = {
    4: [_CSRC + f for f in ("fold.hip", "fold_kernel.h", "igemm.h", "epilogue.h", "qcode.h", "prepare.hip",
                            "fgq_internal.h", "xexpand.h", "xlayout.h", "bufcheck.h")],
    64: [_CSRC + f for f in ("group.hip", "group_kernel.h", "igemm.h", "epilogue.h", "qcode.h", "prepare.hip",
                             "fgq_internal.h", "xexpand.h", "bufcheck.h")],
}


CONFIGS = {"conv3x_g4": (LAYER, 4), "conv3x_g64": (LAYER, 64), "1x1_g64": (LAYER_1X1, 64)}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def layer_dims(L):
    Ho = (L["H"] + 2 * L["pad"] - L["R"]) // L["stride"] + 1
    Wo = (L["W"] + 2 * L["pad"] - L["S"]) // L["stride"] + 1
    M = L["B"] * Ho * Wo
    K = L["C"] * L["R"] * L["S"]
    return M, K, Ho, Wo


def algorithmic_bytes(L, G, bits, out_bits=32, alpha_bytes=4):
    """Activations in + 2-bit codes + alpha (fp32, or one byte as a fixed-point
    code) + output (fp32, or the next layer's 8-/4-bit codes), per launch."""
    M, K, _, _ = layer_dims(L)
    act = L["B"] * L["H"] * L["W"] * L["C"] * bits // 8
    return act + L["O"] * K // 4 + alpha_bytes * L["O"] * K // G + M * L["O"] * out_bits // 8


class Setup:
    """Device buffers of one timed configuration (prepared weights + rotating sets)."""

    def __init__(self, torch, fgq, fi, L, G, bits, nsets, folded=True):
        self.torch, self.fgq, self.L, self.G, self.bits = torch, fgq, L, G, bits
        M, K, Ho, Wo = layer_dims(L)
        self.M, self.K = M, K
        w = fi.he_weights(L["O"], L["C"], L["R"], L["S"], "bench", G)
        self.codes, self.alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
        self.prep = fgq.fgq_prepare_weights(self.codes, self.alpha, L["O"], K, G) if folded else None
        # the same layer with 8-bit fixed-point group scales
        self.prep_dfp = fgq.fgq_prepare_weights_dfp(self.codes, self.alpha, L["O"], K, G, 8)
        n = L["B"] * L["H"] * L["W"] * L["C"]
        base = [torch.from_numpy(fi.relu_gauss((n,), "bench-x", i)).cuda() for i in range(4)]
        wsb = fgq.fgq_quantize_ws_bytes(n)
        self.sets = []
        for i in range(nsets):
            x = base[i % 4].clone()
            q = torch.empty(n * bits // 8, dtype=torch.uint8, device="cuda")
            sx = torch.empty(1, dtype=torch.float32, device="cuda")
            ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
            y = torch.empty((L["B"], Ho, Wo, L["O"]), dtype=torch.float32, device="cuda")
            self.sets.append((x, q, sx, ws, y))
        self.shape = (L["B"], L["H"], L["W"], L["C"])
        # fused next-layer quantization: one output code buffer per set and a
        # static scale, calibrated from one fp32 output by calibrate()
        self.q_out = [torch.empty(M * L["O"] * bits // 8, dtype=torch.uint8, device="cuda")
                      for _ in range(nsets)]
        self.out_scale = torch.ones(1, dtype=torch.float32, device="cuda")

    def calibrate(self):
        """Static output scale: the largest fp32 output of set 0 maps to the top code."""
        self.step(0)
        self.out_scale.fill_(float(self.sets[0][4].max()) / (2 ** self.bits - 1))

    def quantize(self, i):
        x, q, sx, ws, y = self.sets[i]
        self.fgq.fgq_quantize_act(x, self.bits, q=q, scale_out=sx, ws=ws)

    def conv_dfp(self, i):
        x, q, sx, ws, y = self.sets[i]
        L = self.L
        self.fgq.fgq_conv2d_dfp(q, self.bits, sx, self.shape, self.codes, self.prep_dfp, L["O"], L["R"],
                                L["S"], L["stride"], L["pad"], self.G, out=y)

    def conv(self, i):
        x, q, sx, ws, y = self.sets[i]
        L = self.L
        self.fgq.fgq_conv2d(q, self.bits, sx, self.shape, self.codes, self.alpha, L["O"], L["R"],
                            L["S"], L["stride"], L["pad"], self.G, prepared=self.prep, y=y)

    def conv_q(self, i):
        x, q, sx, ws, y = self.sets[i]
        L = self.L
        self.fgq.fgq_conv2d_q(q, self.bits, sx, self.shape, self.codes, self.alpha, L["O"], L["R"],
                              L["S"], L["stride"], L["pad"], self.G, self.bits, self.out_scale,
                              prepared=self.prep, q_out=self.q_out[i])

    def step(self, i):
        self.quantize(i)
        self.conv(i)

    def graph(self, fn, count):
        torch = self.torch
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(count):
                fn(i % len(self.sets))
        return g


def branch_graph(st, count, branches):
    """One graph of steps 0..count-1 of the rotation dealt round-robin over
    `branches` independent chains (step i on chain i % branches, so a set's
    buffers are never used by two chains), forked from and joined back into
    the capturing stream: a replay runs the chains concurrently, one batch's
    quantization and tail overlapping another's convolution."""
    torch = st.torch
    g = torch.cuda.CUDAGraph()
    side = [torch.cuda.Stream() for _ in range(branches)]
    with torch.cuda.graph(g):
        cap = torch.cuda.current_stream()
        for s in side:
            s.wait_stream(cap)
        for r, s in enumerate(side):
            with torch.cuda.stream(s):
                for i in range(r, count, branches):
                    st.step(i % len(st.sets))
        for s in side:
            cap.wait_stream(s)
    return g


def time_graphs(torch, graphs_and_reps):
    """Run each (graph, reps) pair in order between two events; wall and GPU ms."""
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for g, reps in graphs_and_reps:
        for _ in range(reps):
            g.replay()
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return (t1 - t0) * 1e3, ev0.elapsed_time(ev1)


def measure(torch, st, steps, warmup, conv_reps=20, trials=1, streams=4):
    """Times exactly `steps` steps (the reported figure): independent
    batches (buffer sets) dealt round-robin over `streams` concurrent chains
    of one graph, so one batch's quantization and tail overlap another's
    convolution; then, for trials > 1, repeats the same timed region
    trials - 1 more times for a median and spread.  The same steps on one
    stream, and the component kernels alone, are timed separately."""
    nsets = len(st.sets)
    if nsets % streams:
        raise ValueError("the buffer sets must divide evenly over the chains")
    # eager warm-up and graph-replay correctness checks against eager results
    for i in range(nsets):
        st.step(i)
    torch.cuda.synchronize()
    y_eager = [s[4].clone() for s in st.sets]
    full = st.graph(st.step, nsets)
    full.replay()
    full.replay()
    torch.cuda.synchronize()
    if not torch.equal(st.sets[0][4], y_eager[0]):
        raise RuntimeError("graph replay differs from eager execution")
    full_b = branch_graph(st, nsets, streams)
    for s in st.sets:
        s[4].zero_()
    full_b.replay()
    torch.cuda.synchronize()
    if not all(torch.equal(s[4], y) for s, y in zip(st.sets, y_eager)):
        raise RuntimeError("replay of the concurrent chains differs from eager execution")
    del y_eager
    rem = steps % nsets
    rem_graph = st.graph(st.step, rem) if rem else None
    rem_b = branch_graph(st, rem, streams) if rem else None
    # warm-up replays (whole sets), then exactly `steps` timed steps
    for _ in range(max(1, -(-warmup // nsets))):
        full.replay()
        full_b.replay()
    for _ in range(2):
        full_b.replay()
    plan_b = [(full_b, steps // nsets)] + ([(rem_b, 1)] if rem_b else [])
    wall_ms, gpu_ms = time_graphs(torch, plan_b)
    trial_ms = [wall_ms] + [time_graphs(torch, plan_b)[0] for _ in range(trials - 1)]
    # the same steps on one stream
    plan = [(full, steps // nsets)] + ([(rem_graph, 1)] if rem_graph else [])
    one_ms = sorted(time_graphs(torch, plan)[0] for _ in range(max(1, min(trials, 3))))
    # the convolution alone, same stream, same rotation
    conv_g = st.graph(st.conv, nsets)
    conv_g.replay()
    _, conv_ms = time_graphs(torch, [(conv_g, conv_reps)])
    conv_us = conv_ms * 1e3 / (conv_reps * nsets)
    quant_g = st.graph(st.quantize, nsets)
    quant_g.replay()
    _, quant_ms = time_graphs(torch, [(quant_g, conv_reps)])
    quant_us = quant_ms * 1e3 / (conv_reps * nsets)
    # the convolution with the next layer's quantization fused (static scale);
    # its graph replay is checked against an eager call first
    st.calibrate()
    st.conv_q(0)
    torch.cuda.synchronize()
    q_eager = st.q_out[0].clone()
    fused_g = st.graph(st.conv_q, nsets)
    fused_g.replay()
    torch.cuda.synchronize()
    if not torch.equal(st.q_out[0], q_eager):
        raise RuntimeError("fused graph replay differs from eager execution")
    _, fused_ms = time_graphs(torch, [(fused_g, conv_reps)])
    fused_us = fused_ms * 1e3 / (conv_reps * nsets)
    # the layer with 8-bit fixed-point scales
    dfp_g = st.graph(st.conv_dfp, nsets)
    dfp_g.replay()
    _, dfp_ms = time_graphs(torch, [(dfp_g, conv_reps)])
    dfp_us = dfp_ms * 1e3 / (conv_reps * nsets)
    return dict(wall_ms=wall_ms, gpu_ms=gpu_ms, conv_us=conv_us, quant_us=quant_us, conv_fused_us=fused_us,
                conv_dfp_us=dfp_us, trial_ms=trial_ms, streams=streams,
                one_stream_ms=one_ms[len(one_ms) // 2])


def host_cpu():
    """The host the oracle runs on: CPU model, the CPUs of this process's
    affinity mask, and the oracle's thread count (all of those CPUs, capped by
    OMP_NUM_THREADS when the environment sets it), passed to every oracle
    call so that the reported count is the count used."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    affinity = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    threads = min(affinity, int(env)) if env.isdigit() and int(env) > 0 else affinity
    return {"cpu_model": model, "affinity_cpus": affinity, "threads": threads}


def cpu_baseline(fi, L, G, bits, budget_s=15.0, tag="bench"):
    """The plain oracle on the host: quantize of the whole input plus the
    convolution of a bounded sample of output rows, scaled to the metric."""
    import oracle
    hc = host_cpu()
    nt = hc["threads"]
    M, K, Ho, Wo = layer_dims(L)
    w = fi.he_weights(L["O"], L["C"], L["R"], L["S"], tag, G)
    x = fi.relu_gauss((L["B"], L["H"], L["W"], L["C"]), tag + "-x", 0)
    t, a, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    t0 = time.perf_counter()
    q, s = oracle.quantize_act(x, bits)
    t_q = time.perf_counter() - t0
    args = (q, bits, s, x.shape, codes, a, L["O"], L["R"], L["S"], (L["stride"],) * 2, (L["pad"],) * 2, G)
    probe = 256
    t0 = time.perf_counter()
    oracle.conv2d(*args, rows=(0, probe), nthreads=nt)
    t_probe = time.perf_counter() - t0
    nrows = int(min(M, max(probe, probe * budget_s / max(t_probe, 1e-6))))
    reps = 3 if nrows == M and t_probe * M / probe * 3 < budget_s * 2 else 1
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        oracle.conv2d(*args, rows=(0, nrows), nthreads=nt)
        times.append(time.perf_counter() - t0)
    t_c = sorted(times)[len(times) // 2]
    t_total = t_c + t_q * nrows / M
    ops = 2.0 * nrows * L["O"] * K
    return {"value": ops / t_total / 1e12, "unit": "TOPS", "cores": nt, "kind": "oracle",
            "cpu_model": hc["cpu_model"], "affinity_cpus": hc["affinity_cpus"],
            "sample": f"quantize of the full {L['B']}x{L['H']}x{L['W']}x{L['C']} input "
                      f"({t_q:.3f} s, prorated) + convolution of output rows [0, {nrows}) of {M} "
                      f"({t_c:.2f} s, median of {reps}); scaled per row",
            "seconds": round(t_total, 3)}


def cpu_baseline_gemm(fi, M=64, K=256, O=128, G=4, bits=8, budget_s=2.0):
    """The oracle on the single FGQ GEMM (whole layer, repeated until
    `budget_s` of CPU time; quantize + GEMM per call)."""
    import oracle
    hc = host_cpu()
    nt = hc["threads"]
    w = fi.gauss_weights(O, K, 0.05, "bench-gemm")
    x = fi.relu_gauss((M, K), "bench-gemm", 0)
    t, a, _ = oracle.ternarize(w.reshape(O, K, 1, 1), G)
    codes = oracle.pack_codes(t)
    calls, t0 = 0, time.perf_counter()
    while True:
        q, s = oracle.quantize_act(x, bits)
        oracle.gemm(q, bits, s, M, K, codes, a, O, G, nthreads=nt)
        calls += 1
        dt = time.perf_counter() - t0
        if dt >= budget_s or calls >= 100000:
            break
    us = dt / calls * 1e6
    return {"value": 2.0 * M * K * O / (us * 1e-6) / 1e12, "unit": "TOPS", "us_per_call": round(us, 2),
            "cores": nt, "kind": "oracle", "cpu_model": hc["cpu_model"], "affinity_cpus": hc["affinity_cpus"],
            "sample": f"the whole M={M} K={K} O={O} layer (quantize + GEMM), {calls} calls"}


def stack_cpu_estimate(fi, depth, G, bits, batch=64, rows=256):
    """The oracle's time for a stack's convolutions (and FC), extrapolated
    from a row sample: for every distinct layer, the oracle convolution of
    the first `rows` output rows of one image (a row depends only on its own
    image, so the cost per row is that of the full batch), scaled to the
    layer's M = batch * Ho * Wo rows and its multiplicity."""
    import oracle
    hc = host_cpu()
    total_s, ops, sampled = 0.0, 0.0, 0
    for L, count in stack_layers(fi, depth, 1):
        B1, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        st, pd = L["stride"], L["pad"]
        g = G if C % G == 0 else 4
        w = fi.he_weights(O, C, R, S, "stack-cpu", depth, L["name"])
        x = fi.relu_gauss((B1, H, W, C), "stack-cpu", depth, L["name"])
        if L["name"] == "conv1":
            w[:, 3:] = 0.0
            x[..., 3:] = 0.0
        t, a, _ = oracle.ternarize(w, g)
        codes = oracle.pack_codes(t)
        q, sx = oracle.quantize_act(x, bits)
        Ho, Wo = (H + 2 * pd - R) // st + 1, (W + 2 * pd - S) // st + 1
        n = min(rows, Ho * Wo)
        t0 = time.perf_counter()
        oracle.conv2d(q, bits, sx, x.shape, codes, a, O, R, S, (st, st), (pd, pd), g, rows=(0, n),
                      nthreads=hc["threads"])
        dt = time.perf_counter() - t0
        M = batch * Ho * Wo
        total_s += count * dt * M / n
        ops += count * 2.0 * M * O * R * S * (3 if L["name"] == "conv1" else C)
        sampled += n
    return {"seconds_extrapolated": round(total_s, 2), "effective_tops": ops / total_s / 1e12,
            "cores": hc["threads"], "kind": "oracle", "cpu_model": hc["cpu_model"],
            "affinity_cpus": hc["affinity_cpus"],
            "sample": f"first {rows} output rows (fewer on small maps) of one image per distinct layer, "
                      f"{sampled} rows in all, scaled to batch {batch} and each layer's multiplicity"}


def measured_peaks(torch, fgq, reps=5):
    """Measured peaks beside the published ones: the int8 matrix-instruction
    rate (fgq_probe_mfma_i8: two workgroups per compute unit, four
    independent 32x32x32 chains per wave) and a plain 1 GiB device copy
    (read plus written bytes over its time); medians of `reps` launches timed
    with events on the current stream."""
    def timed(fn):
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts)[len(ts) // 2]

    blocks = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    iters = 8192
    sink = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    fgq.fgq_probe_mfma_i8(blocks, 64, sink)
    torch.cuda.synchronize()
    ms = timed(lambda: fgq.fgq_probe_mfma_i8(blocks, iters, sink))
    mfma_tops = blocks * iters * 16 * 65536 / (ms * 1e-3) / 1e12
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    ms_copy = timed(lambda: dst.copy_(src))
    del src, dst
    torch.cuda.empty_cache()
    return {"int8_mfma_tops": round(mfma_tops, 1), "spec_int8_mfma_tops": INT8_PEAK_TOPS,
            "copy_gbs": round(2 * nbytes / (ms_copy * 1e-3) / 1e9, 1), "spec_hbm_gbs": HBM_PEAK_GBS,
            "method": f"fgq_probe_mfma_i8 ({blocks} workgroups x {iters} rounds) and a 1 GiB device copy, "
                      f"median of {reps} event-timed launches"}


def valu_floor_us(L, G):
    """The vector-ALU floor of a per-group fp32 epilogue: one multiply-add per
    row, channel and group, 64 lanes x 256 compute units per cycle at
    2.4 GHz."""
    M, K, _, _ = layer_dims(L)
    return 2.0 * M * L["O"] * (K // G) / (64 * 256 * 2.4e9) * 1e6


def stack_layers(fi, depth, batch):
    """Distinct layer shapes of the ResNet stack with their multiplicities."""
    out, index = [], {}
    for L in fi.resnet_convs(depth, batch):
        key = tuple(L[k] for k in ("H", "W", "C", "O", "R", "S", "stride", "pad"))
        if key in index:
            out[index[key]][1] += 1
        else:
            index[key] = len(out)
            out.append([L, 1])
    return out


def stack_layer_roofline(L, g, bits):
    """(ops, algorithmic bytes, roofline us) of one stack layer: 2*M*O*K with
    the unpadded reduction for conv1 (3 image channels), activations in +
    2-bit codes + fp32 scales + fp32 output, and the larger of the int8 and
    HBM times at the published peaks."""
    M, K, _, _ = layer_dims(L)
    k_true = L["R"] * L["S"] * (3 if L["name"] == "conv1" else L["C"])
    ops = 2.0 * M * L["O"] * k_true
    nbytes = L["B"] * L["H"] * L["W"] * L["C"] * bits // 8 + L["O"] * K // 4 + 4 * L["O"] * K // g + 4 * M * L["O"]
    return ops, nbytes, max(ops / (INT8_PEAK_TOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e6


def stack_measure(torch, fgq, fi, depth, G, bits, batch=64, nsets=3, reps=50):
    """Per-layer kernel times of a batch-`batch` ResNet-`depth` stack, every
    distinct layer timed at its full shape (graph replays over `nsets`
    rotating buffer sets) and counted with its multiplicity.  Inputs are
    seeded ReLU-Gaussian activations of each layer's shape (the layers are
    not chained); conv1 has its 3 input channels padded to 4 and uses
    groups of 4.  Effective ops use the unpadded conv1 reduction (147).
    Each layer is also timed with the next layer's quantization fused
    (fgq_conv2d_q, `bits`-bit codes, static scale from one fp32 output): a
    chain of such layers needs one fgq_quantize_act, for the network input.
    Finally each layer runs as the paper's own pipeline (Sec. 4): 8-bit
    fixed-point group scales (fgq_conv2d_dfp) with the fused output codes,
    and conv1 at 8-bit weights (fgq_conv2d_w8)."""
    layers, direct_layers = [], []
    tot = dict(conv_us=0.0, quant_us=0.0, fused_us=0.0, dfp_us=0.0, ops=0.0, roof_us=0.0, bytes=0.0,
               first_quant_us=0.0)
    gen = torch.Generator(device="cuda")
    for li, (L, count) in enumerate(stack_layers(fi, depth, batch)):
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        st, pd = L["stride"], L["pad"]
        g = G if C % G == 0 else 4
        w = fi.he_weights(O, C, R, S, "stack-bench", depth, L["name"])
        if L["name"] == "conv1":
            w[:, 3:] = 0.0
        codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), g)
        K = R * S * C
        # a layer whose group scales fail the folded layout's accuracy guard
        # runs the direct kernel (prepared = None), as a network would
        prep = fgq.fgq_prepare_weights(codes, alpha, O, K, g, fallback=True)
        if prep is None:
            direct_layers.append(L["name"])
        prep_dfp = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, g, 8)
        # the paper keeps the first layer at 8-bit weights (8w-8a)
        prep_w8 = fgq.fgq_prepare_weights_w8(torch.from_numpy(w).cuda()) if L["name"] == "conv1" else None
        n = B * H * W * C
        Ho, Wo = (H + 2 * pd - R) // st + 1, (W + 2 * pd - S) // st + 1
        M = B * Ho * Wo
        gen.manual_seed(fi.SEED + 1000 * depth + li)
        sets = []
        for _ in range(nsets):
            x = torch.randn(n, generator=gen, device="cuda").clamp_(min=0.0)
            if L["name"] == "conv1":
                x.view(B, H, W, C)[..., 3:] = 0.0
            q = torch.empty(n * bits // 8, dtype=torch.uint8, device="cuda")
            sx = torch.empty(1, dtype=torch.float32, device="cuda")
            ws = torch.empty(fgq.fgq_quantize_ws_bytes(n), dtype=torch.uint8, device="cuda")
            y = torch.empty((B, Ho, Wo, O), dtype=torch.float32, device="cuda")
            sets.append((x, q, sx, ws, y))
        q_outs = [torch.empty(M * O * bits // 8, dtype=torch.uint8, device="cuda") for _ in range(nsets)]
        out_scale = torch.ones(1, dtype=torch.float32, device="cuda")
        # the fully-connected layer (a 1x1 layer on a 1x1 map) runs as the
        # GEMM at small batch: K split over workgroups, weights read as codes
        fc = H == 1 and W == 1 and R == 1 and S == 1
        ws_fc = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, K, O, g, False), 4), dtype=torch.uint8, device="cuda")
        ws_fc_dfp = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, K, O, g, True), 4), dtype=torch.uint8, device="cuda")

        def quant(i):
            x, q, sx, ws, y = sets[i]
            fgq.fgq_quantize_act(x, bits, q=q, scale_out=sx, ws=ws)

        def conv(i):
            x, q, sx, ws, y = sets[i]
            if fc:
                fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, g, prepared=prep, out=y.view(M, O), ws=ws_fc)
                return
            fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, g, prepared=prep, y=y)

        def conv_q(i):
            x, q, sx, ws, y = sets[i]
            if fc:
                fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, g, prepared=prep, out_bits=bits,
                                out_scale=out_scale, out=q_outs[i], ws=ws_fc)
                return
            fgq.fgq_conv2d_q(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, g, bits, out_scale,
                             prepared=prep, q_out=q_outs[i])

        def conv_dfp_q(i):
            x, q, sx, ws, y = sets[i]
            if fc:
                fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep_dfp, O, g, bits, out_scale, out=q_outs[i],
                                    ws=ws_fc_dfp)
                return
            if prep_w8 is not None:
                fgq.fgq_conv2d_w8(q, bits, sx, (B, H, W, C), prep_w8, O, R, S, st, pd, bits, out_scale,
                                  out=q_outs[i])
            else:
                fgq.fgq_conv2d_dfp(q, bits, sx, (B, H, W, C), codes, prep_dfp, O, R, S, st, pd, g, bits,
                                   out_scale, out=q_outs[i])

        def graph(fn):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                for i in range(nsets):
                    fn(i)
            return gr

        for i in range(nsets):
            quant(i)
            conv(i)
        out_scale.fill_(float(sets[0][4].max()) / (2 ** bits - 1))
        for i in range(nsets):
            conv_q(i)
            conv_dfp_q(i)
        torch.cuda.synchronize()
        gq, gc, gf, gd = graph(quant), graph(conv), graph(conv_q), graph(conv_dfp_q)
        gq.replay()
        gc.replay()
        gf.replay()
        gd.replay()
        _, q_ms = time_graphs(torch, [(gq, reps)])
        _, c_ms = time_graphs(torch, [(gc, reps)])
        _, f_ms = time_graphs(torch, [(gf, reps)])
        _, d_ms = time_graphs(torch, [(gd, reps)])
        conv_us = c_ms * 1e3 / (reps * nsets)
        quant_us = q_ms * 1e3 / (reps * nsets)
        fused_us = f_ms * 1e3 / (reps * nsets)
        dfp_us = d_ms * 1e3 / (reps * nsets)
        ops, nbytes, roof_us = stack_layer_roofline(L, g, bits)
        layers.append([L["name"], count, round(conv_us, 2), round(roof_us / conv_us, 3), round(fused_us, 2),
                       round(dfp_us, 2)])
        tot["conv_us"] += count * conv_us
        tot["quant_us"] += count * quant_us
        tot["fused_us"] += count * fused_us
        tot["dfp_us"] += count * dfp_us
        if li == 0:
            tot["first_quant_us"] = quant_us
        tot["ops"] += count * ops
        tot["roof_us"] += count * roof_us
        tot["bytes"] += count * nbytes
        del sets, q_outs, gq, gc, gf, gd, prep, prep_dfp, prep_w8, codes, alpha
        torch.cuda.empty_cache()
    return {"workload": f"ResNet-{depth} conv stack, batch {batch}, G={G}, u{bits} (conv1 at G=4)",
            "layers_total": sum(c for _, c in stack_layers(fi, depth, batch)), "distinct": len(layers),
            "sum_conv_us": round(tot["conv_us"], 1), "sum_quantize_us": round(tot["quant_us"], 1),
            "effective_tops_conv": round(tot["ops"] / (tot["conv_us"] * 1e-6) / 1e12, 1),
            "effective_tops_with_quantize": round(tot["ops"] / ((tot["conv_us"] + tot["quant_us"]) * 1e-6) / 1e12, 1),
            "sum_conv_fused_us": round(tot["fused_us"], 1),
            "effective_tops_fused_chain": round(tot["ops"] / ((tot["fused_us"] + tot["first_quant_us"]) * 1e-6) / 1e12, 1),
            "sum_conv_dfp_fused_us": round(tot["dfp_us"], 1),
            "effective_tops_dfp_fused_chain": round(tot["ops"] / ((tot["dfp_us"] + tot["first_quant_us"]) * 1e-6) / 1e12, 1),
            "sum_roofline_us": round(tot["roof_us"], 1),
            "roofline_frac": round(tot["roof_us"] / tot["conv_us"], 4),
            "algorithmic_bytes": int(tot["bytes"]),
            "per_layer_columns": ["layer", "count", "conv_us", "roofline_frac", "conv_fused_us",
                                  "conv_dfp8_fused_us"],
            "per_layer": layers,
            "direct_kernel_layers": direct_layers}


class ResNetChain:
    """A whole ResNet-`depth` forward pass on the library (torchvision v1.5
    bottlenecks, hw x hw input, batch `batch`).  Every convolution and the
    fully-connected layer is an FGQ layer on prepared weights (fgq_conv2d;
    the fully-connected layer through fgq_gemm_ws), and every layer's input
    is quantized by fgq_quantize_act with its own dynamic per-tensor scale.
    The glue between layers is plain torch on fp32 NHWC tensors: the
    stem's 3x3 max pooling and the global average pooling; each block's
    shortcut addition and its ReLU are fused into the block's last
    convolution (fgq_conv2d_residual writes max(conv + shortcut, 0) into the
    block output), or with residual_fused=False run as a torch addition and
    ReLU after it.  The ReLU after the stem and after the first two
    convolutions of a block is the quantizer's own clamp at zero (the codes
    and the scale of y and of ReLU(y) are the same), so those layers'
    outputs are quantized as they are.  With dfp=True the layers follow the
    paper's pipeline: group scales as an 8-bit fixed point (fgq_conv2d_dfp
    and its residual form, fgq_gemm_dfp_ws) and the first layer at 8-bit
    weights (fgq_conv2d_w8).  The network input is pixel-like uint8 codes (128 + 32 z,
    clamped, scale 1/255; a zero fourth channel), the weights He-initialised
    and ternarized per layer (conv1 in groups of 4).  Every buffer is
    allocated up front, so forward() can be captured in a HIP graph; after
    it, each layer's input codes (`q`, `sx`) and fp32 output (`y`) stay in
    `self.layers`, and the stem and block outputs in `self.stem` and
    `self.blocks`, for checks."""

    def __init__(self, torch, fgq, fi, depth, G, bits, batch, hw=224, tag="chain", residual_fused=True,
                 dfp=False):
        self.torch, self.fgq, self.bits = torch, fgq, bits
        self.residual_fused = residual_fused
        # dfp: the paper's pipeline -- group scales as an 8-bit fixed point
        # (fgq_conv2d_dfp, fgq_gemm_dfp_ws) and the first layer at 8-bit
        # weights (fgq_conv2d_w8)
        self.dfp = dfp
        self.convs = fi.resnet_convs(depth, batch, hw)
        self.layers = {}
        self.ops = 0.0
        for L in self.convs:
            B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
            g = G if C % G == 0 else 4
            w = fi.he_weights(O, C, R, S, tag, depth, L["name"])
            if L["name"] == "conv1":
                w[:, 3:] = 0.0
            codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), g)
            K = R * S * C
            Ho, Wo = fi.conv_out(H, W, R, S, L["stride"], L["pad"])
            n = B * H * W * C
            e = dict(L=L, g=g, K=K, codes=codes, alpha=alpha,
                     prep=None if dfp else fgq.fgq_prepare_weights(codes, alpha, O, K, g, fallback=True),
                     q=torch.empty(n * bits // 8, dtype=torch.uint8, device="cuda"),
                     sx=torch.empty(1, dtype=torch.float32, device="cuda"),
                     ws=torch.empty(max(fgq.fgq_quantize_ws_bytes(n), 4), dtype=torch.uint8, device="cuda"),
                     y=torch.empty((B, Ho, Wo, O), dtype=torch.float32, device="cuda"))
            if dfp:
                e["prep_dfp"] = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, g, 8)
                if L["name"] == "conv1":
                    e["prep_w8"] = fgq.fgq_prepare_weights_w8(torch.from_numpy(w).cuda())
            if L["name"] == "fc":
                e["wsfc"] = torch.empty(max(fgq.fgq_gemm_ws_bytes(B, K, O, g, dfp), 4), dtype=torch.uint8,
                                        device="cuda")
            self.layers[L["name"]] = e
            self.ops += 2.0 * B * Ho * Wo * O * R * S * (3 if L["name"] == "conv1" else C)
        # the network input: pixel-like codes with a zero fourth channel
        L0 = self.convs[0]
        z = fi.rng("chain-input", depth, batch, hw).standard_normal((L0["B"], L0["H"], L0["W"], 4))
        x0 = np.clip(np.rint(128.0 + 32.0 * z), 0, 255).astype(np.uint8)
        x0[..., 3] = 0
        if bits == 4:
            x0 = x0 >> 4
            x0 = (x0[..., 0::2] | (x0[..., 1::2] << 4)).astype(np.uint8)
        c1 = self.layers["conv1"]
        c1["q"].copy_(torch.from_numpy(x0.reshape(-1)))
        c1["sx"].fill_(1.0 / (255.0 if bits == 8 else 15.0))
        # block outputs (and the stem's pooled output)
        y1 = c1["y"]
        Hp = (y1.shape[1] + 2 - 3) // 2 + 1
        self.stem = torch.empty((y1.shape[0], Hp, Hp, y1.shape[3]), dtype=torch.float32, device="cuda")
        self.blocks = {}
        for L in self.convs:
            if L["name"].endswith(".c3"):
                p = L["name"][:-3]
                self.blocks[p] = torch.empty_like(self.layers[L["name"]]["y"])
        # a downsampling convolution reads the block input's codes (the
        # stride is the convolution's), quantized once for both
        for p in self.blocks:
            ds = self.layers.get(f"{p}.ds")
            if ds is not None:
                c1 = self.layers[f"{p}.c1"]
                ds["q"], ds["sx"], ds["ws"] = c1["q"], c1["sx"], c1["ws"]
        last = self.blocks[list(self.blocks)[-1]]
        self.pooled = torch.empty((last.shape[0], last.shape[3]), dtype=torch.float32, device="cuda")
        self.logits = self.layers["fc"]["y"]

    def calibrate(self):
        """Static input scales for the fused form: each layer's scale from one
        forward pass with dynamic scales (the paper's per-layer scales)."""
        self.forward()
        for e in self.layers.values():
            e["sx_static"] = e["sx"].clone()

    def _quant(self, src, e):
        self.fgq.fgq_quantize_act(src, self.bits, q=e["q"], scale_out=e["sx"], ws=e["ws"])

    def _conv_q(self, e, nxt, sx=None):
        """Layer e (input scale sx, default its own) with the next layer's
        quantization fused: its codes written straight into nxt's input, at
        nxt's static scale."""
        L = e["L"]
        sx = e["sx"] if sx is None else sx
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        if self.dfp:
            self.fgq.fgq_conv2d_dfp(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["prep_dfp"], O, R, S,
                                    L["stride"], L["pad"], e["g"], self.bits, nxt["sx_static"], out=nxt["q"])
            return
        self.fgq.fgq_conv2d_q(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["alpha"], O, R, S,
                              L["stride"], L["pad"], e["g"], self.bits, nxt["sx_static"], prepared=e["prep"],
                              q_out=nxt["q"])

    def _conv(self, e, sx=None):
        """Layer e on its input codes, at scale sx (default: its own, as
        quantized)."""
        L = e["L"]
        sx = e["sx"] if sx is None else sx
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        if self.dfp:
            if L["name"] == "fc":
                self.fgq.fgq_gemm_dfp_ws(e["q"], self.bits, sx, B, e["K"], e["codes"], e["prep_dfp"], O, e["g"],
                                         out=e["y"].view(B, O), ws=e["wsfc"])
            elif L["name"] == "conv1":
                self.fgq.fgq_conv2d_w8(e["q"], self.bits, sx, (B, H, W, C), e["prep_w8"], O, R, S, L["stride"],
                                       L["pad"], out=e["y"])
            else:
                self.fgq.fgq_conv2d_dfp(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["prep_dfp"], O, R, S,
                                        L["stride"], L["pad"], e["g"], out=e["y"])
            return
        if L["name"] == "fc":
            self.fgq.fgq_gemm_ws(e["q"], self.bits, sx, B, e["K"], e["codes"], e["alpha"], O, e["g"],
                                 prepared=e["prep"], out=e["y"].view(B, O), ws=e["wsfc"])
        else:
            self.fgq.fgq_conv2d(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["alpha"], O, R, S,
                                L["stride"], L["pad"], e["g"], prepared=e["prep"], y=e["y"])

    def _conv_res(self, e, res, out, sx=None):
        """Layer e with the block's shortcut addition and ReLU fused:
        out = max(layer + res, 0)."""
        L = e["L"]
        sx = e["sx"] if sx is None else sx
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        if self.dfp:
            self.fgq.fgq_conv2d_dfp_residual(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["prep_dfp"], O, R,
                                             S, L["stride"], L["pad"], e["g"], res, y=out)
            return
        self.fgq.fgq_conv2d_residual(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["alpha"], O, R, S,
                                     L["stride"], L["pad"], e["g"], res, prepared=e["prep"], y=out)

    def _conv_res_q(self, e, res, out, nxt, sx=None):
        """Layer e with the block's shortcut addition and ReLU fused, writing
        out and also its codes as nxt's input at nxt's static scale."""
        L = e["L"]
        sx = e["sx"] if sx is None else sx
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        if self.dfp:
            self.fgq.fgq_conv2d_dfp_residual(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["prep_dfp"], O, R,
                                             S, L["stride"], L["pad"], e["g"], res, self.bits, nxt["sx_static"],
                                             y=out, q_out=nxt["q"])
            return
        self.fgq.fgq_conv2d_residual_q(e["q"], self.bits, sx, (B, H, W, C), e["codes"], e["alpha"], O, R, S,
                                       L["stride"], L["pad"], e["g"], res, self.bits, nxt["sx_static"],
                                       prepared=e["prep"], y=out, q_out=nxt["q"])

    def forward(self, fused=False):
        """fused=False: every layer's input quantized with a dynamic scale.
        fused=True (after calibrate()): the first two convolutions of each
        block write the next layer's codes at its static scale
        (fgq_conv2d_q), and with residual_fused the last one also writes the
        next block's input codes at that block's static scale
        (fgq_conv2d_residual_q), so only the stem's output and the head are
        quantized separately."""
        torch, F = self.torch, self.torch.nn.functional
        c1 = self.layers["conv1"]
        self._conv(c1)
        pooled = F.max_pool2d(c1["y"].permute(0, 3, 1, 2), 3, 2, 1)
        self.stem.copy_(pooled.permute(0, 2, 3, 1))
        h = self.stem
        names = list(self.blocks)
        coded = False  # the block input's codes already written (static scale)
        for bi, (p, out) in enumerate(self.blocks.items()):
            a, b, c = (self.layers[f"{p}.c{j}"] for j in (1, 2, 3))
            ds = self.layers.get(f"{p}.ds")
            if not coded:
                self._quant(h, a)
            sx_a = a["sx_static"] if coded else None
            if ds is not None:
                self._conv(ds, sx=sx_a)
            if fused:
                self._conv_q(a, b, sx=sx_a)
                self._conv_q(b, c, sx=b["sx_static"])
                sx_c = c["sx_static"]
            else:
                self._conv(a)
                self._quant(a["y"], b)
                self._conv(b)
                self._quant(b["y"], c)
                sx_c = None
            shortcut = ds["y"] if ds is not None else h
            nxt = self.layers[f"{names[bi + 1]}.c1"] if bi + 1 < len(names) else None
            coded = False
            if self.residual_fused and fused and nxt is not None:
                self._conv_res_q(c, shortcut, out, nxt, sx=sx_c)
                coded = True
            elif self.residual_fused:
                self._conv_res(c, shortcut, out, sx=sx_c)
            else:
                self._conv(c, sx=sx_c)
                torch.add(c["y"], shortcut, out=out)
                out.relu_()
            h = out
        torch.mean(h, dim=(1, 2), out=self.pooled)
        fc = self.layers["fc"]
        self._quant(self.pooled, fc)
        self._conv(fc)
        return fc["y"]


def _time_nets(torch, nets, reps):
    """One network's forward pass (dynamic scales, then the fused form with
    static scales) captured in one graph, and the networks' passes as
    concurrent chains of one graph; each checked against eager logits."""
    net = nets[0]
    res, conc = {}, {}
    for fused in (False, True):
        refs = []
        for n in nets:
            n.forward(fused)
            torch.cuda.synchronize()
            refs.append(n.forward(fused).clone())
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            net.forward(fused)
        g.replay()
        torch.cuda.synchronize()
        if not torch.equal(net.logits, refs[0]):
            raise RuntimeError("graph replay of the network differs from eager execution")
        _, ms = time_graphs(torch, [(g, reps)])
        res[fused] = (ms * 1e3 / reps, bool(torch.isfinite(refs[0]).all().item()))
        del g
        if len(nets) > 1:
            gc = torch.cuda.CUDAGraph()
            side = [torch.cuda.Stream() for _ in nets]
            with torch.cuda.graph(gc):
                cap = torch.cuda.current_stream()
                for s in side:
                    s.wait_stream(cap)
                for s, n in zip(side, nets):
                    with torch.cuda.stream(s):
                        n.forward(fused)
                for s in side:
                    cap.wait_stream(s)
            for n in nets:
                n.logits.zero_()
            gc.replay()
            torch.cuda.synchronize()
            if not all(torch.equal(n.logits, r) for n, r in zip(nets, refs)):
                raise RuntimeError("concurrent replay of the networks differs from eager execution")
            gc.replay()
            _, ms = time_graphs(torch, [(gc, reps)])
            conc[fused] = ms * 1e3 / (reps * len(nets))
            del gc
    out = {"end_to_end_us": round(res[False][0], 1),
           "effective_tops_end_to_end": round(net.ops / (res[False][0] * 1e-6) / 1e12, 1),
           "end_to_end_fused_us": round(res[True][0], 1),
           "effective_tops_end_to_end_fused": round(net.ops / (res[True][0] * 1e-6) / 1e12, 1),
           "logits_finite": res[False][1] and res[True][1]}
    if len(nets) > 1:
        out["in_flight"] = {"batches": len(nets),
                            "us_per_batch": round(conc[False], 1),
                            "effective_tops": round(net.ops / (conc[False] * 1e-6) / 1e12, 1),
                            "fused_us_per_batch": round(conc[True], 1),
                            "effective_tops_fused": round(net.ops / (conc[True] * 1e-6) / 1e12, 1)}
    return out


def chain_measure(torch, fgq, fi, depth, G, bits, batch=64, reps=10, in_flight=3):
    """End-to-end time of ResNetChain's forward pass, captured in one HIP
    graph: every layer's quantization, every FGQ layer and the torch glue.
    Also `in_flight` independent batches (one ResNetChain each, own buffers)
    as concurrent chains of one graph, forked from and joined into the
    capturing stream: the time per batch when batches overlap.  The same
    for the paper's pipeline (8-bit fixed-point group scales, the first
    layer at 8-bit weights: `paper_pipeline`)."""
    nets = [ResNetChain(torch, fgq, fi, depth, G, bits, batch) for _ in range(in_flight)]
    for net in nets:
        net.calibrate()
    out = {"workload": f"ResNet-{depth} forward pass, batch {batch}, 224x224, G={G}, u{bits}: every layer's "
                       "quantization, FGQ layer (each block's last one with the block's shortcut addition and ReLU "
                       "fused, fgq_conv2d_residual) and the torch glue (max pooling, average pooling) in one "
                       "graph; fused: the first two convolutions of each block write the next layer's codes and "
                       "the last one the next block's input codes, at calibrated static scales"}
    out.update(_time_nets(torch, nets, reps))
    # the same pass with each block's shortcut addition and ReLU as torch ops
    net = nets[0]
    net.residual_fused = False
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        net.forward(False)
    g.replay()
    _, ms = time_graphs(torch, [(g, reps)])
    out["end_to_end_torch_residual_us"] = round(ms * 1e3 / reps, 1)
    del g, net, nets
    torch.cuda.empty_cache()
    nets = [ResNetChain(torch, fgq, fi, depth, G, bits, batch, dfp=True) for _ in range(in_flight)]
    for net in nets:
        net.calibrate()
    out["paper_pipeline"] = {"layers": "group scales as an 8-bit fixed point (fgq_conv2d_dfp, "
                                       "fgq_conv2d_dfp_residual, fgq_gemm_dfp_ws), the first layer at 8-bit "
                                       "weights (fgq_conv2d_w8)"}
    out["paper_pipeline"].update(_time_nets(torch, nets, reps))
    del nets
    torch.cuda.empty_cache()
    return out


class AlexNetChain:
    """A whole AlexNet forward pass on the library (single tower, 227x227
    pixel-like uint8 input with a zero fourth channel, batch `batch`):
    conv1 -> 3x3/2 max pooling -> conv2 -> pooling -> conv3 -> conv4 ->
    conv5 -> pooling -> fc6 -> fc7 -> fc8, every convolution and
    fully-connected layer an FGQ layer (fgq_conv2d, fgq_gemm_ws) with its
    input quantized by fgq_quantize_act; the ReLUs are the quantizer's clamp
    at zero (a max pooling of y and of ReLU(y) gives the same codes), and
    the pooling is torch on fp32 NHWC.  Fused form (after calibrate()):
    conv3 -> conv4 -> conv5 and fc6 -> fc7 -> fc8 write the next layer's
    codes at calibrated static scales.  dfp=True: the paper's pipeline, the
    first layer at 8-bit weights (fgq_conv2d_w8) and the others with 8-bit
    fixed-point group scales (fgq_conv2d_dfp, fgq_gemm_dfp_ws).  Every
    buffer is allocated up front, so forward() can be captured in a graph;
    each layer's input codes, scale and fp32 output stay in `self.layers`,
    the pooled tensors in `self.pooled`.  The weights are those the per-layer
    AlexNet measurement draws (the same tag); a layer whose scales fail the
    folded layout's accuracy guard runs on the exact direct kernel and is
    listed in `self.direct_layers`."""

    def __init__(self, torch, fgq, fi, G, bits, batch, tag="alexnet-bench", dfp=False):
        self.torch, self.fgq, self.bits, self.dfp = torch, fgq, bits, dfp
        self.convs = fi.alexnet_layers(batch)
        self.layers, self.ops = {}, 0.0
        for L in self.convs:
            B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
            g = G if C % G == 0 else 4
            w = fi.he_weights(O, C, R, S, tag, L["name"])
            if L["name"] == "conv1":
                w[:, 3:] = 0.0
            codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), g)
            K = R * S * C
            Ho, Wo = fi.conv_out(H, W, R, S, L["stride"], L["pad"])
            n = B * H * W * C
            e = dict(L=L, g=g, K=K, codes=codes, alpha=alpha, fc=H == 1 and W == 1,
                     q=torch.empty(n * bits // 8, dtype=torch.uint8, device="cuda"),
                     sx=torch.empty(1, dtype=torch.float32, device="cuda"),
                     ws=torch.empty(max(fgq.fgq_quantize_ws_bytes(n), 4), dtype=torch.uint8, device="cuda"),
                     y=torch.empty((B, Ho, Wo, O), dtype=torch.float32, device="cuda"))
            if dfp:
                e["prep"] = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, g, 8)
                if L["name"] == "conv1":
                    e["prep_w8"] = fgq.fgq_prepare_weights_w8(torch.from_numpy(w).cuda())
            else:
                e["prep"] = fgq.fgq_prepare_weights(codes, alpha, O, K, g, fallback=True)
            if e["fc"]:
                e["wsfc"] = torch.empty(max(fgq.fgq_gemm_ws_bytes(B, K, O, g, dfp), 4), dtype=torch.uint8,
                                        device="cuda")
            self.layers[L["name"]] = e
            self.ops += 2.0 * B * Ho * Wo * O * R * S * (3 if L["name"] == "conv1" else C)
        self.direct_layers = [n for n, e in self.layers.items() if e["prep"] is None]
        L0 = self.convs[0]
        z = fi.rng("alexnet-chain-input", batch).standard_normal((L0["B"], L0["H"], L0["W"], 4))
        x0 = np.clip(np.rint(128.0 + 32.0 * z), 0, 255).astype(np.uint8)
        x0[..., 3] = 0
        if bits == 4:
            x0 = x0 >> 4
            x0 = (x0[..., 0::2] | (x0[..., 1::2] << 4)).astype(np.uint8)
        c1 = self.layers["conv1"]
        c1["q"].copy_(torch.from_numpy(x0.reshape(-1)))
        c1["sx"].fill_(1.0 / (255.0 if bits == 8 else 15.0))
        self.pooled = {}
        for a, b in (("conv1", "conv2"), ("conv2", "conv3"), ("conv5", "fc6")):
            y = self.layers[a]["y"]
            Hp = (y.shape[1] - 3) // 2 + 1
            self.pooled[a] = torch.empty((y.shape[0], Hp, Hp, y.shape[3]), dtype=torch.float32, device="cuda")
        self.logits = self.layers["fc8"]["y"]

    def calibrate(self):
        """Static input scales for the fused form, from one dynamic pass."""
        self.forward()
        for e in self.layers.values():
            e["sx_static"] = e["sx"].clone()

    def _quant(self, src, e):
        self.fgq.fgq_quantize_act(src, self.bits, q=e["q"], scale_out=e["sx"], ws=e["ws"])

    def _layer(self, e, sx=None, nxt=None):
        """Layer e at input scale sx (default: its own); with nxt, writing
        nxt's input codes at nxt's static scale instead of fp32."""
        f, L, bits = self.fgq, e["L"], self.bits
        sx = e["sx"] if sx is None else sx
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        ob, osc = (bits, nxt["sx_static"]) if nxt is not None else (0, None)
        if e["fc"]:
            out = nxt["q"] if nxt is not None else e["y"].view(B, O)
            if self.dfp:
                f.fgq_gemm_dfp_ws(e["q"], bits, sx, B, e["K"], e["codes"], e["prep"], O, e["g"], ob, osc, out=out,
                                  ws=e["wsfc"])
            else:
                f.fgq_gemm_ws(e["q"], bits, sx, B, e["K"], e["codes"], e["alpha"], O, e["g"], prepared=e["prep"],
                              out_bits=ob, out_scale=osc, out=out, ws=e["wsfc"])
        elif self.dfp and L["name"] == "conv1":
            f.fgq_conv2d_w8(e["q"], bits, sx, (B, H, W, C), e["prep_w8"], O, R, S, L["stride"], L["pad"],
                            out=e["y"])
        elif self.dfp:
            f.fgq_conv2d_dfp(e["q"], bits, sx, (B, H, W, C), e["codes"], e["prep"], O, R, S, L["stride"], L["pad"],
                             e["g"], ob, osc, out=nxt["q"] if nxt is not None else e["y"])
        elif nxt is not None:
            f.fgq_conv2d_q(e["q"], bits, sx, (B, H, W, C), e["codes"], e["alpha"], O, R, S, L["stride"], L["pad"],
                           e["g"], bits, osc, prepared=e["prep"], q_out=nxt["q"])
        else:
            f.fgq_conv2d(e["q"], bits, sx, (B, H, W, C), e["codes"], e["alpha"], O, R, S, L["stride"], L["pad"],
                         e["g"], prepared=e["prep"], y=e["y"])

    def _pool(self, name):
        F = self.torch.nn.functional
        p = F.max_pool2d(self.layers[name]["y"].permute(0, 3, 1, 2), 3, 2)
        self.pooled[name].copy_(p.permute(0, 2, 3, 1))
        return self.pooled[name]

    def forward(self, fused=False):
        """fused=False: every layer's input quantized with a dynamic scale;
        fused=True (after calibrate()): conv3 -> conv5 and fc6 -> fc8 write
        the next layer's codes at its static scale, and the layers after a
        pooling quantize their input with a dynamic scale."""
        Ls = self.layers
        self._layer(Ls["conv1"])
        self._quant(self._pool("conv1"), Ls["conv2"])
        self._layer(Ls["conv2"])
        self._quant(self._pool("conv2"), Ls["conv3"])
        chain = (("conv3", "conv4"), ("conv4", "conv5"))
        for i, (a, b) in enumerate(chain):
            sx = Ls[a]["sx_static"] if (fused and i > 0) else None
            if fused:
                self._layer(Ls[a], sx=sx, nxt=Ls[b])
            else:
                self._layer(Ls[a])
                self._quant(Ls[a]["y"], Ls[b])
        self._layer(Ls["conv5"], sx=Ls["conv5"]["sx_static"] if fused else None)
        self._quant(self._pool("conv5").reshape(Ls["fc6"]["L"]["B"], -1), Ls["fc6"])
        for i, (a, b) in enumerate((("fc6", "fc7"), ("fc7", "fc8"))):
            sx = Ls[a]["sx_static"] if (fused and i > 0) else None
            if fused:
                self._layer(Ls[a], sx=sx, nxt=Ls[b])
            else:
                self._layer(Ls[a])
                self._quant(Ls[a]["y"], Ls[b])
        self._layer(Ls["fc8"], sx=Ls["fc8"]["sx_static"] if fused else None)
        return self.logits


def alexnet_chain_measure(torch, fgq, fi, batch=64, G=4, bits=8, reps=10, in_flight=3):
    """End-to-end AlexNet forward passes (AlexNetChain), with fp32 group
    scales and as the paper's pipeline, one batch and `in_flight` batches
    at a time (as chain_measure)."""
    out = {"workload": f"AlexNet forward pass, batch {batch}, 227x227, G={G}, u{bits}: every layer's "
                       "quantization and FGQ layer and the torch max pooling in one graph; fused: conv3-conv5 "
                       "and fc6-fc8 write the next layer's codes at calibrated static scales"}
    for key, dfp in (("fp32_scales", False), ("paper_pipeline", True)):
        nets = [AlexNetChain(torch, fgq, fi, G, bits, batch, dfp=dfp) for _ in range(in_flight)]
        for n in nets:
            n.calibrate()
        out[key] = _time_nets(torch, nets, reps)
        out[key]["direct_kernel_layers"] = nets[0].direct_layers
        del nets
        torch.cuda.empty_cache()
    return out


def alexnet_measure(torch, fgq, fi, batch=64, G=4, bits=8, nsets=3, reps=50):
    """The AlexNet-shaped layers at batch `batch`, G=4, uint8: each layer timed
    at its full shape (graph replays over rotating sets) two ways: ternary
    weights with fp32 group scales and fp32 output (fgq_conv2d; the
    fully-connected layers, M = batch, through fgq_gemm_ws with split K),
    and the paper's pipeline (conv1 at 8-bit weights, the others with 8-bit
    fixed-point scales, fused 8-bit outputs; fgq_conv2d_w8 / fgq_conv2d_dfp /
    fgq_gemm_dfp_ws)."""
    layers, tot = [], dict(fp=0.0, paper=0.0, ops=0.0, roof=0.0)
    gen = torch.Generator(device="cuda")
    for li, L in enumerate(fi.alexnet_layers(batch)):
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        st, pd = L["stride"], L["pad"]
        fc = H == 1 and W == 1 and R == 1 and S == 1
        w = fi.he_weights(O, C, R, S, "alexnet-bench", L["name"])
        if L["name"] == "conv1":
            w[:, 3:] = 0.0
        codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
        K = R * S * C
        prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G, fallback=True)
        prep_dfp = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
        prep_w8 = fgq.fgq_prepare_weights_w8(torch.from_numpy(w).cuda()) if L["name"] == "conv1" else None
        Ho, Wo = (H + 2 * pd - R) // st + 1, (W + 2 * pd - S) // st + 1
        M = B * Ho * Wo
        ws = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, K, O, G), 4), dtype=torch.uint8, device="cuda")
        wsd = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, K, O, G, True), 4), dtype=torch.uint8, device="cuda")
        gen.manual_seed(fi.SEED + 7000 + li)
        sets = []
        for _ in range(nsets):
            x = torch.randn(B * H * W * C, generator=gen, device="cuda").clamp_(min=0.0)
            if L["name"] == "conv1":
                x.view(B, H, W, C)[..., 3:] = 0.0
            q, sx = fgq.fgq_quantize_act(x, bits)
            y = torch.empty((M, O), dtype=torch.float32, device="cuda")
            qo = torch.empty(M * O, dtype=torch.uint8, device="cuda")
            sets.append((q, sx, y, qo))
        out_scale = torch.ones(1, dtype=torch.float32, device="cuda")

        def plain(i):
            q, sx, y, qo = sets[i]
            if fc:
                fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep, out=y, ws=ws)
            else:
                fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G, prepared=prep,
                               y=y.view(B, Ho, Wo, O))

        def paper(i):
            q, sx, y, qo = sets[i]
            if prep_w8 is not None:
                fgq.fgq_conv2d_w8(q, bits, sx, (B, H, W, C), prep_w8, O, R, S, st, pd, 8, out_scale, out=qo)
            elif fc:
                fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep_dfp, O, G, 8, out_scale, out=qo, ws=wsd)
            else:
                fgq.fgq_conv2d_dfp(q, bits, sx, (B, H, W, C), codes, prep_dfp, O, R, S, st, pd, G, 8, out_scale,
                                   out=qo)

        for i in range(nsets):
            plain(i)
        out_scale.fill_(float(sets[0][2].max()) / 255)
        times = []
        for fn in (plain, paper):
            for i in range(nsets):
                fn(i)
            torch.cuda.synchronize()
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                for i in range(nsets):
                    fn(i)
            gr.replay()
            _, ms = time_graphs(torch, [(gr, reps)])
            times.append(ms * 1e3 / (reps * nsets))
        k_true = R * S * (3 if L["name"] == "conv1" else C)
        ops = 2.0 * M * O * k_true
        nbytes = B * H * W * C + O * K // 4 + 4 * O * K // G + 4 * M * O
        roof_us = max(ops / (INT8_PEAK_TOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e6
        layers.append([L["name"], round(times[0], 2), round(roof_us / times[0], 3), round(times[1], 2)])
        tot["fp"] += times[0]
        tot["paper"] += times[1]
        tot["ops"] += ops
        tot["roof"] += roof_us
        del sets, prep, prep_dfp, prep_w8, ws, wsd, codes, alpha
        torch.cuda.empty_cache()
    return {"workload": f"AlexNet-shaped layers, batch {batch}, G={G}, u{bits} (conv1 channels padded to 4; "
                        "fully-connected layers as GEMMs with split K)",
            "sum_us": round(tot["fp"], 1), "effective_tops": round(tot["ops"] / (tot["fp"] * 1e-6) / 1e12, 1),
            "sum_roofline_us": round(tot["roof"], 1), "roofline_frac": round(tot["roof"] / tot["fp"], 4),
            "sum_paper_pipeline_us": round(tot["paper"], 1),
            "effective_tops_paper_pipeline": round(tot["ops"] / (tot["paper"] * 1e-6) / 1e12, 1),
            "per_layer_columns": ["layer", "us", "roofline_frac", "paper_pipeline_us"],
            "per_layer": layers}


def gemm_measure(torch, fgq, fi, M=64, K=256, O=128, G=4, bits=8, nsets=8, reps=50):
    """Latency of the single FGQ GEMM (M=64, K=256, O=128, W ~ N(0, 0.05^2),
    G=4, uint8): a launch-latency-bound size, reported in microseconds."""
    w = fi.gauss_weights(O, K, 0.05, "bench-gemm")
    codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    sets = []
    for i in range(nsets):
        x = torch.from_numpy(fi.relu_gauss((M, K), "bench-gemm", i)).cuda()
        q, sx = fgq.fgq_quantize_act(x, bits)
        y = torch.empty((M, O), dtype=torch.float32, device="cuda")
        sets.append((q, sx, y))

    def run(i):
        q, sx, y = sets[i]
        fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep, y=y)

    for i in range(nsets):
        run(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(nsets):
            run(i)
    g.replay()
    _, ms = time_graphs(torch, [(g, reps)])
    us = ms * 1e3 / (reps * nsets)
    return {"workload": f"FGQ GEMM M={M} K={K} O={O}, G={G}, u{bits}", "us_per_call": round(us, 3),
            "effective_tops": round(2.0 * M * K * O / (us * 1e-6) / 1e12, 3)}


def kernel_source_hash(G):
    """sha256 of the conv kernel's sources with // comments and blank lines
    removed, so that a comment edit does not invalidate the counters."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[4 if G % 64 else 64]:
        for line in open(os.path.join(ROOT, f), encoding="utf-8"):
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()


def layer_key(L, G):
    return f"{L['R']}x{L['S']}_{L['C']}to{L['O']}_{L['H']}x{L['W']}_b{L['B']}_G{G}"


def measured_traffic(L, G):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources (else None)."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    e = t.get("per_launch", {}).get(layer_key(L, G))
    if e is None or e.get("kernel_source_sha256") != kernel_source_hash(G):
        return None
    return int(e["fetch_bytes"] + e["write_bytes"])


def roofline(L, G, bits, conv_us, out_bits=32, kernel=None, alpha_bytes=4):
    M, K, _, _ = layer_dims(L)
    nbytes = algorithmic_bytes(L, G, bits, out_bits, alpha_bytes)
    kernel = kernel or ("fgq_conv2d" if out_bits == 32 else "fgq_conv2d_q")
    traffic = measured_traffic(L, G) if kernel == "fgq_conv2d" else None
    ops = 2.0 * M * L["O"] * K
    t_hbm = nbytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = ops / (INT8_PEAK_TOPS * 1e12)
    if t_hbm >= t_mfma:
        achieved = nbytes / (conv_us * 1e-6) / 1e9
        return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": kernel, "kernel_us": round(conv_us, 3),
                "algorithmic_bytes": int(nbytes)}
    achieved = ops / (conv_us * 1e-6) / 1e12
    return {"bound": "mfma", "achieved": round(achieved, 1), "peak": INT8_PEAK_TOPS, "unit": "TFLOP/s",
            "frac": round(achieved / INT8_PEAK_TOPS, 4), "traffic": traffic,
            "kernel": kernel, "kernel_us": round(conv_us, 3), "algorithmic_ops": ops}


def dfp_entry(L, G, bits, r, ops):
    """fgq_conv2d_dfp: the same layer with 8-bit fixed-point group scales
    (one exponent per layer; one int8 matrix pass, exact integer result)."""
    return {"kernel": "fgq_conv2d_dfp", "alpha_bits": 8, "conv_us": round(r["conv_dfp_us"], 3),
            "conv_only_tops": round(ops / (r["conv_dfp_us"] * 1e-6) / 1e12, 1),
            "roofline": roofline(L, G, bits, r["conv_dfp_us"], kernel="fgq_conv2d_dfp", alpha_bytes=1)}


def fused_entry(L, G, bits, r, ops):
    """fgq_conv2d_q (8-bit codes of the next layer's activations, static
    scale) against fgq_conv2d + that layer's separate fgq_quantize_act."""
    return {"kernel": "fgq_conv2d_q", "out_bits": bits, "conv_fused_us": round(r["conv_fused_us"], 3),
            "conv_fp32_us": round(r["conv_us"], 3),
            "chained_layer_tops": round(ops / (r["conv_fused_us"] * 1e-6) / 1e12, 1),
            "roofline": roofline(L, G, bits, r["conv_fused_us"], out_bits=bits)}


def profile_fc(torch, fgq, fi, M, K, O, G, steps):
    """For profilers: `steps` eager calls of fgq_gemm_dfp_ws (8-bit scales,
    uint8 activations, fp32 output) on one prepared M x K x O layer."""
    w = fi.gauss_weights(O, K, 0.01, "fc", K, O)
    codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
    q, sx = fgq.fgq_quantize_act(torch.from_numpy(fi.relu_gauss((M, K), "fc")).cuda(), 8)
    y = torch.empty((M, O), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, K, O, G, True), 4), dtype=torch.uint8, device="cuda")
    for _ in range(steps):
        fgq.fgq_gemm_dfp_ws(q, 8, sx, M, K, codes, prep, O, G, out=y, ws=ws)
    torch.cuda.synchronize()
    log(f"[bench] profile fc M={M} K={K} O={O} G={G}: {steps} eager calls done")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--sets", type=int, default=96,
                    help="rotating buffer sets (~32 MB each; the 96 sets of 3.2 MB layer inputs "
                         "exceed the 256 MB memory-side cache)")
    ap.add_argument("--streams", type=int, default=4,
                    help="concurrent chains (streams forked inside one graph) the timed batches are "
                         "dealt over (1: one after another); the buffer sets must divide evenly")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-stacks", action="store_true", help="skip the ResNet stack measurements")
    ap.add_argument("--direct", action="store_true", help="time the direct per-group kernels")
    ap.add_argument("--profile-steps", type=int, default=0,
                    help="for profilers: run this many eager steps per group size (no graphs, "
                         "no timing) and exit")
    ap.add_argument("--layers", default="conv3x_g4,conv3x_g64,1x1_g64",
                    help="layer configurations for --profile-steps")
    ap.add_argument("--profile-fused", action="store_true",
                    help="with --profile-steps: each step also runs fgq_conv2d_q (8-bit output codes)")
    ap.add_argument("--profile-fc", default="",
                    help="with --profile-steps: instead of the conv layers, call fgq_gemm_dfp_ws on a "
                         "fully-connected layer given as M,K,O,G")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the FGQ layer is "
              "single-device here and its multi-GPU sharding is a design note, not a run.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import fgq_inputs as fi
    import paper_1705_01462_amd as fgq

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    bits = 8
    M, K, Ho, Wo = layer_dims(LAYER)
    ops = 2.0 * M * LAYER["O"] * K

    if args.profile_steps:
        fc = [int(v) for v in args.profile_fc.split(",")] if args.profile_fc else None
        for name in ([] if fc else args.layers.split(",")):
            L, G = CONFIGS[name]
            st = Setup(torch, fgq, fi, L, G, bits, 4, folded=not args.direct)
            if args.profile_fused:
                st.calibrate()
            for i in range(args.profile_steps):
                st.step(i % 4)
                if args.profile_fused:
                    st.conv_q(i % 4)
            torch.cuda.synchronize()
            log(f"[bench] profile {name} ({layer_key(L, G)}): {args.profile_steps} eager steps done")
            del st
        if fc:
            profile_fc(torch, fgq, fi, *fc, args.profile_steps)
        # calibration: one plain device copy of known size (FETCH_SIZE and
        # WRITE_SIZE of this dispatch give the counter-to-bytes factor)
        src = torch.ones(CALIB_COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {CALIB_COPY_BYTES} bytes done")
        return

    log(f"[bench] setting up G=4 ({args.sets} buffer sets)")
    st4 = Setup(torch, fgq, fi, LAYER, 4, bits, args.sets, folded=not args.direct)
    r4 = measure(torch, st4, args.steps, args.warmup, trials=5, streams=args.streams)
    log(f"[bench] G=4: {r4}")
    ms_per_step = r4["wall_ms"] / args.steps
    n_act = LAYER["B"] * LAYER["H"] * LAYER["W"] * LAYER["C"]
    # a step's algorithmic bytes: fp32 input read and codes written by the
    # quantization, then the convolution's own
    step_bytes = 4 * n_act + n_act * bits // 8 + algorithmic_bytes(LAYER, 4, bits)
    del st4
    torch.cuda.empty_cache()

    log("[bench] setting up G=64")
    st64 = Setup(torch, fgq, fi, LAYER, 64, bits, args.sets, folded=not args.direct)
    steps64 = max(args.sets, args.steps // 4)
    r64 = measure(torch, st64, steps64, args.sets, streams=args.streams)
    log(f"[bench] G=64: {r64}")
    del st64
    torch.cuda.empty_cache()

    log("[bench] setting up the 1x1 layer, G=64")
    st11 = Setup(torch, fgq, fi, LAYER_1X1, 64, bits, args.sets, folded=not args.direct)
    r11 = measure(torch, st11, steps64, args.sets, streams=args.streams)
    log(f"[bench] 1x1 G=64: {r11}")
    del st11
    torch.cuda.empty_cache()
    M11, K11, _, _ = layer_dims(LAYER_1X1)
    ops11 = 2.0 * M11 * LAYER_1X1["O"] * K11

    out = {
        "metric": METRIC,
        "value": round(ops / (ms_per_step * 1e-3) / 1e12, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "ResNet-50 conv3_x 3x3 conv 128->128, 28x28, batch 32, stride 1, pad 1; "
                               "ternary weights in groups of G=4 input channels; uint8 activations "
                               "(dynamic per-tensor scale); fp32 NHWC output",
                   "B": LAYER["B"], "H": LAYER["H"], "W": LAYER["W"], "C": LAYER["C"], "O": LAYER["O"],
                   "R": 3, "S": 3, "G": 4, "bits": bits, "M": M, "K": K,
                   "kernel": "direct" if args.direct else "folded-scale int8 MFMA (G=4); per-group int8 MFMA + fp32 epilogue (G=64)",
                   "step": "fgq_quantize_act + fgq_conv2d",
                   "streams": args.streams},
        "roofline": roofline(LAYER, 4, bits, r4["conv_us"]),
        "step_detail": {"conv_us": round(r4["conv_us"], 3), "quantize_us": round(r4["quant_us"], 3),
                        "gpu_ms_per_step": round(r4["gpu_ms"] / args.steps, 5),
                        "trials_ms_per_step": [round(t / args.steps, 5) for t in r4["trial_ms"]],
                        "median_of_5_tops": round(ops / (sorted(r4["trial_ms"])[2] / args.steps * 1e-3) / 1e12, 2),
                        "one_stream_ms_per_step": round(r4["one_stream_ms"] / args.steps, 5),
                        "one_stream_tops": round(ops / (r4["one_stream_ms"] / args.steps * 1e-3) / 1e12, 2),
                        "step_algorithmic_bytes": int(step_bytes),
                        "step_hbm_gbs": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                        "step_hbm_frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "conv_only_tops": round(ops / (r4["conv_us"] * 1e-6) / 1e12, 1)},
        "fused": fused_entry(LAYER, 4, bits, r4, ops),
        "dfp": dfp_entry(LAYER, 4, bits, r4, ops),
        "g64": {"workload": "same layer, G=64", "steps": steps64,
                "value": round(ops / (r64["wall_ms"] / steps64 * 1e-3) / 1e12, 2),
                "ms_per_step": round(r64["wall_ms"] / steps64, 5),
                "one_stream_tops": round(ops / (r64["one_stream_ms"] / steps64 * 1e-3) / 1e12, 2),
                "conv_us": round(r64["conv_us"], 3),
                "conv_only_tops": round(ops / (r64["conv_us"] * 1e-6) / 1e12, 1),
                "roofline": roofline(LAYER, 64, bits, r64["conv_us"]),
                "fused": fused_entry(LAYER, 64, bits, r64, ops),
                "dfp": dfp_entry(LAYER, 64, bits, r64, ops)},
        "g64_1x1": {"workload": "ResNet-50 1x1 conv 256->64, 56x56, batch 32, G=64", "steps": steps64,
                    "value": round(ops11 / (r11["wall_ms"] / steps64 * 1e-3) / 1e12, 2),
                    "ms_per_step": round(r11["wall_ms"] / steps64, 5),
                    "one_stream_tops": round(ops11 / (r11["one_stream_ms"] / steps64 * 1e-3) / 1e12, 2),
                    "conv_us": round(r11["conv_us"], 3), "quantize_us": round(r11["quant_us"], 3),
                    "conv_only_tops": round(ops11 / (r11["conv_us"] * 1e-6) / 1e12, 1),
                    "roofline": roofline(LAYER_1X1, 64, bits, r11["conv_us"]),
                    "fused": fused_entry(LAYER_1X1, 64, bits, r11, ops11),
                    "dfp": dfp_entry(LAYER_1X1, 64, bits, r11, ops11)},
    }
    out["gemm_m64"] = gemm_measure(torch, fgq, fi)
    log("[bench] measured peaks")
    peaks = measured_peaks(torch, fgq)
    out["measured_peaks"] = peaks
    out["roofline"]["frac_of_measured_copy"] = round(out["roofline"]["achieved"] / peaks["copy_gbs"], 4)
    fl64 = valu_floor_us(LAYER, 64)
    out["g64"]["valu_floor_us"] = round(fl64, 3)
    out["g64"]["valu_floor_frac"] = round(fl64 / r64["conv_us"], 4)
    if not args.no_stacks:
        out["stacks"] = {}
        for depth, G, sbits in ((50, 4, 8), (101, 64, 4)):
            log(f"[bench] ResNet-{depth} stack, G={G}, u{sbits}")
            out["stacks"][f"resnet{depth}_b64_g{G}_u{sbits}"] = stack_measure(torch, fgq, fi, depth, G, sbits)
            if not args.no_cpu:
                out["stacks"][f"resnet{depth}_b64_g{G}_u{sbits}"]["cpu_oracle"] = stack_cpu_estimate(fi, depth, G, sbits)
            log(f"[bench] ResNet-{depth}: sum conv {out['stacks'][f'resnet{depth}_b64_g{G}_u{sbits}']['sum_conv_us']} us")
            out["stacks"][f"resnet{depth}_b64_g{G}_u{sbits}"]["end_to_end"] = chain_measure(torch, fgq, fi, depth,
                                                                                            G, sbits)
            log(f"[bench] ResNet-{depth} forward pass: "
                f"{out['stacks'][f'resnet{depth}_b64_g{G}_u{sbits}']['end_to_end']['end_to_end_us']} us")
    if not args.no_stacks:
        log("[bench] AlexNet-shaped layers, batch 64, G=4, u8")
        out["alexnet_b64_g4_u8"] = alexnet_measure(torch, fgq, fi)
        out["alexnet_b64_g4_u8"]["end_to_end"] = alexnet_chain_measure(torch, fgq, fi)
        log(f"[bench] AlexNet: sum {out['alexnet_b64_g4_u8']['sum_us']} us, "
            f"paper pipeline {out['alexnet_b64_g4_u8']['sum_paper_pipeline_us']} us")
    if not args.no_cpu:
        log("[bench] CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(fi, LAYER, 4, bits)
        out["g64"]["cpu_baseline"] = cpu_baseline(fi, LAYER, 64, bits, budget_s=6.0)
        out["g64_1x1"]["cpu_baseline"] = cpu_baseline(fi, LAYER_1X1, 64, bits, budget_s=4.0)
        out["gemm_m64"]["cpu_baseline"] = cpu_baseline_gemm(fi)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
