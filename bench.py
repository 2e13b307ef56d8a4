"""Benchmark of the AF1 factorized binary linear on one MI355X.

Step = one forward of the decode hot path (s_in scaling, first sign product,
s_mid scaling, second sign product, s_out scaling and bf16 rounding) for one
batch, on a 4096x4096 layer at the strict 1.0-BPW rank r=2016, batch 1 --
a LLaMA-3-8B-shaped attention projection.  Weights rotate over a pool of
distinct layers larger than twice the 256 MB last-level cache, so every step
streams its packed signs from HBM.

The same JSON line also carries the prefill GEMM (2048 tokens, 70B-shaped
8192x8192 r=4064 and 28672x8192 / 8192x28672 r=6336) in TFLOP/s, the
roofline of the timed kernel, and the CPU oracle timed on the host.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("µs/layer + % HBM roofline, 1.0-BPW factorized GEMV b=1; "
          "TFLOP/s GEMM at 2048 tok")
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
POOL_BYTES = 512 << 20          # > 2 x 256 MB MALL

# HBM bytes per GEMV call from rocprofv3 FETCH_SIZE + WRITE_SIZE (scaled by a
# 64 MiB copy calibration; see profiles/gemv_4096x4096_r2016_b1.md).  Valid
# only for the kernel source it was measured on: reported as null as soon as
# the source hash differs.
GEMV_TRAFFIC = {"sources": ("paper_2609_06161_amd/csrc/af1_gemv.hip",
                            "paper_2609_06161_amd/csrc/af1_device.h"),
                "sha256": "2a832747ca707ce797fb871aef3f165223451fe0e9bc672fe8d3130b4f4dc2bb",
                "bytes_per_call": 2849213}


# HBM bytes of the prefill leg's three calls at 2048 tokens (8192^2 r=4064,
# 28672x8192 and 8192x28672 at r=6336), the sum over every kernel of each
# call of the same scaled counters (see profiles/gemm_prefill_T2048_70b_shapes.md:
# 268.8 + 1027.4 + 1116.5 MB).  Same validity rule as GEMV_TRAFFIC.
GEMM_TRAFFIC = {"sources": ("paper_2609_06161_amd/csrc/af1_gemm.hip",
                            "paper_2609_06161_amd/csrc/af1_device.h"),
                "sha256": "557d167b5d1ef153e7186b9cf302c71b38688d3f244e1703685c612c43df3709",
                "bytes_per_call": 2412700000}


# HBM bytes of one backward call of the training leg (8192^2 r=4064, T=2048:
# row statistics, preparation, both contractions, finish), same counters (see
# profiles/train_scale_only_sq8192_T2048.md).  Same validity rule.
TRAIN_BWD_TRAFFIC = dict(GEMM_TRAFFIC, bytes_per_call=422053879)


def measured_traffic(record):
    import hashlib
    h = hashlib.sha256()
    for rel in record["sources"]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return record["bytes_per_call"] if h.hexdigest() == record["sha256"] else None


def measured_gemv_traffic():
    return measured_traffic(GEMV_TRAFFIC)


def gemv_algorithmic_bytes(m, n, r, b):
    """Packed signs + fp16 scales (storage bits / 8) + bf16 x and y."""
    storage_bits = r * (m + n) + 16 * (m + n + r)
    return storage_bits // 8 + 2 * b * (m + n)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=2000)
    p.add_argument("--warmup", type=int, default=200)
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--gemm-steps", type=int, default=20)
    p.add_argument("--sustain", type=float, default=0.5,
                   help="seconds of untimed back-to-back calls before each prefill / "
                        "training measurement")
    p.add_argument("--no-gemm", action="store_true")
    p.add_argument("--no-decode-table", action="store_true")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--only", choices=("all", "gemv", "gemm", "train", "nabf"), default="all",
                   help="profiling aid: run one part only")
    p.add_argument("--shape", default="attn4096",
                   help="profiling aid (with --only gemv): the decode shape to time, one of "
                        "the decode table's names")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="profiling aid: first run a 64 MiB device copy five times, the "
                        "known-size reference for scaling hardware byte counters")
    return p.parse_args()


def time_events(fn, steps, stream):
    import torch
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record(stream)
    for i in range(steps):
        fn(i)
    e.record(stream)
    torch.cuda.synchronize()
    return s.elapsed_time(e)   # ms


def sustain(fn, stream, seconds=0.5):
    """Untimed warmup for the prefill and training legs: call fn until about
    `seconds` of back-to-back GPU work has run.  Under sustained MFMA load
    the throughput of these kernels keeps rising for the first ~100 ms of
    calls (clock and power management settling), so a few warmup calls
    would time the ramp rather than the steady state."""
    ms = time_events(fn, 3, stream)
    calls = max(3, int(seconds * 1e3 / max(ms / 3, 1e-3)))
    time_events(fn, calls, stream)


class DevicePool:
    """`count` distinct layers of one shape, generated on the device from a
    seeded generator with the recipe's distributions (fair sign bits as
    uniform 32-bit words, fp16 lognormal(0, 0.5) scales), so that a pool
    larger than the 256 MB last-level cache is built in milliseconds."""

    def __init__(self, torch, m, n, r, count, seed):
        from paper_2609_06161_amd import af1
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        words = lambda k: torch.randint(-2 ** 31, 2 ** 31, (count, k), dtype=torch.int32,
                                        device="cuda", generator=g)
        scales = lambda k: (torch.empty((count, k), device="cuda").log_normal_(0.0, 0.5, generator=g)
                            .to(torch.float16).view(torch.int16))
        self.Bv, self.Bu = words(r * n // 32), words(m * r // 32)
        self.s_in, self.s_mid, self.s_out = scales(n), scales(r), scales(m)
        self.desc = [af1.make_layer(m, n, r, self.Bu[i], self.Bv[i], self.s_out[i],
                                    self.s_mid[i], self.s_in[i]) for i in range(count)]
        self.m, self.n, self.r, self.count = m, n, r, count


def decode_time(args, torch, stream, m, n, r, b, seed, steps, exact_steps=None):
    """µs per layer of the decode forward over a pool of distinct layers
    (> 2x the last-level cache), eager and as a replayed HIP graph of one
    pass over the pool."""
    from paper_2609_06161_amd import af1, synth
    from paper_2609_06161_amd.layer import to_device
    layer_bytes = r * (m + n) // 8
    pool = max(2, -(-POOL_BYTES // layer_bytes))
    P = DevicePool(torch, m, n, r, pool, seed)
    x = to_device(synth.make_activations(seed, b, n))
    y = torch.empty((b, m), dtype=torch.int16, device="cuda")
    ws = torch.zeros(max(256, af1.af1_gemv_workspace_bytes(m, n, r, b)), dtype=torch.uint8,
                     device="cuda")

    def step(i):
        # stream=None: the binding uses torch's current stream (the capture
        # stream while a graph is being recorded)
        af1.af1_linear_gemv(P.desc[i % pool], x, b, y, ws, ws.numel(), None)

    time_events(step, min(args.warmup, pool), stream)
    eager_steps = max(pool, steps // 4)
    ms_eager = time_events(step, eager_steps, stream) / eager_steps
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(pool):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(pool):
            step(i)
    replays = max(1, -(-steps // pool))
    time_events(lambda i: graph.replay(), max(1, args.warmup // pool), stream)
    ms_graph = time_events(lambda i: graph.replay(), replays, stream) / (replays * pool)
    # spread: µs per layer of each replay (one pass over the pool), timed alone
    per = sorted(time_events(lambda i: graph.replay(), 1, stream) * 1e3 / pool
                 for _ in range(max(5, min(replays, 50))))
    pct = lambda q: per[min(len(per) - 1, int(q * (len(per) - 1) + 0.5))]
    del graph
    out = dict(m=m, n=n, r=r, b=b, pool=pool, pool_mb=pool * layer_bytes / 2 ** 20,
               steps_timed=replays * pool, us_graph=ms_graph * 1e3, us_eager=ms_eager * 1e3,
               us_graph_p10=pct(0.1), us_graph_p50=pct(0.5), us_graph_p90=pct(0.9),
               alg_bytes=gemv_algorithmic_bytes(m, n, r, b))
    if exact_steps:
        # W warmup calls, then exactly K calls in one timed graph replay,
        # walking the layer pool in order (a layer comes back only after
        # the whole pool, more than twice the last-level cache, has passed)
        K, W = exact_steps
        gw = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gw):
            for i in range(max(W, 1)):
                step(i % pool)
        g2 = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g2):
            for i in range(K):
                step((max(W, 1) + i) % pool)
        gw.replay()
        ms_k = time_events(lambda i: g2.replay(), 1, stream)
        out.update(exact_steps=K, exact_warmup=W, exact_ms=ms_k)
        del g2, gw
    del P
    return out


def launch_floor(torch, stream, count=256, replays=20):
    """µs per launch of a one-workgroup kernel (torch's in-place add on one
    element), `count` dependent launches in a replayed HIP graph: the floor
    under any per-call time that takes one launch per stage."""
    t = torch.zeros(1, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        t.add_(1.0)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(count):
            t.add_(1.0)
    time_events(lambda i: graph.replay(), 3, stream)
    us = time_events(lambda i: graph.replay(), replays, stream) * 1e3 / (replays * count)
    del graph
    return round(us, 3)


DECODE_TABLE = [("sq1024", 1), ("attn4096", 8), ("kv1024x4096", 1), ("mlp_up14336x4096", 1),
                ("mlp_up14336x4096", 4), ("mlp_up14336x4096", 16), ("mlp_down4096x14336", 1),
                ("mlp_down4096x14336", 4), ("mlp_down4096x14336", 16),
                ("attn4096_r5120_2.5bpw", 1), ("attn4096_r5120_2.5bpw", 8)]

# The paper's other budget (2.5 bits per weight) at 4096x4096: its own rank
# rule round(2.5 mn / (m + n)) (af1_paper_rank, 5120), above min(m, n), so
# the second sign matrix is the larger one.
def paper_25bpw_shape():
    from paper_2609_06161_amd import af1
    return (4096, 4096, af1.af1_paper_rank(4096, 4096, 2.5))


def shape_of(name):
    from paper_2609_06161_amd import synth
    return paper_25bpw_shape() if name == "attn4096_r5120_2.5bpw" else synth.SHAPES[name]


STACK_LINEARS = [("q", 4096, 4096, 2016), ("k", 1024, 4096, 800), ("v", 1024, 4096, 800),
                 ("o", 4096, 4096, 2016), ("gate", 14336, 4096, 3136),
                 ("up", 14336, 4096, 3136), ("down", 4096, 14336, 3136)]


def bench_stack(args, torch, stream):
    """An 8B-shaped decoder stack: 32 layers x 7 linears, per-linear ranks
    drawn +-25% around the budget rank with the whole stack <= 1.0 BPW,
    weights streamed from HBM in layer order, batch 1, each linear fed a
    fixed synthetic x of its input width; one HIP graph of the whole pass.

    Two schedules: the 224 linears one call each, and the projections that
    read the same input fused into one call (q, k, v; gate, up), which is
    how a decoder issues them: 4 calls per layer instead of 7."""
    from paper_2609_06161_amd import af1, synth
    from paper_2609_06161_amd.layer import to_device
    entries = synth.draw_stack_ranks(77, 32, STACK_LINEARS, af1.af1_storage_bits)
    bits = sum(af1.af1_storage_bits(m, n, r) for _, m, n, _, r in entries)
    dense = sum(m * n for _, m, n, _, _ in entries)
    pools, descs = [], []
    for i, (name, m, n, r0, r) in enumerate(entries):
        P = DevicePool(torch, m, n, r, 1, 5000 + i)
        pools.append(P)
        descs.append((name, P.desc[0], m, n, r))
    xs = {w: to_device(synth.make_activations(60 + w % 97, 1, w)) for w in (4096, 14336)}
    ys = {name: torch.empty((1, m), dtype=torch.int16, device="cuda")
          for name, m, _, _ in STACK_LINEARS}
    groups = []   # per layer: [q,k,v], [o], [gate,up], [down]
    for layer in range(32):
        q, k, v, o, gate, up, down = descs[7 * layer: 7 * layer + 7]
        groups += [[q, k, v], [o], [gate, up], [down]]
    ws_bytes = max(af1.af1_gemv_multi_workspace_bytes([e[1] for e in g], 1) for g in groups)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")

    def run_serial():
        for name, d, m, n, r in descs:
            af1.af1_linear_gemv(d, xs[n], 1, ys[name], ws, ws.numel(), None)

    def run_fused():
        for g in groups:
            n = g[0][3]
            if len(g) == 1:
                name, d, m, n, r = g[0]
                af1.af1_linear_gemv(d, xs[n], 1, ys[name], ws, ws.numel(), None)
            else:
                af1.af1_linear_gemv_multi([e[1] for e in g], xs[n], 1, [ys[e[0]] for e in g],
                                          ws, ws.numel(), None)

    out = dict(linears=len(descs), bpw=round(bits / dense, 5), weight_mb=round(bits / 8 / 1e6, 1))
    alg = sum(gemv_algorithmic_bytes(m, n, r, 1) for _, _, m, n, r in descs)
    for label, fn in (("", run_serial), ("_fused_projections", run_fused)):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        time_events(lambda i: graph.replay(), 2, stream)
        reps = 10
        ms = time_events(lambda i: graph.replay(), reps, stream) / reps
        out[f"us_per_decoder_layer{label}"] = round(ms * 1e3 / 32, 3)
        out[f"gbs{label}"] = round(alg / (ms * 1e-3) / 1e9, 1)
        del graph
    out["us_per_linear"] = round(out["us_per_decoder_layer"] / 7, 3)
    del pools
    return out


def bench_layer_stream(args, torch, stream):
    """The layer stream (af1_linear_stream: one persistent launch for a
    sequence of layers) on the 8B stack and on the 4096^2 pool, with two
    schedules: every layer waiting for the earlier ones where a decoder
    would (q, o, gate and down wait; for the pool, every layer), and the
    workload as specified (each linear reads a fixed synthetic x, so no
    linear waits for another; weights still stream in layer order)."""
    from paper_2609_06161_amd import af1, synth
    from paper_2609_06161_amd.layer import LayerStream, to_device

    class Desc:
        def __init__(self, d):
            self.desc = d

    def graph_ms(fn, reps=5):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        time_events(lambda i: graph.replay(), 2, stream)
        ms = time_events(lambda i: graph.replay(), reps, stream) / reps
        del graph
        return ms

    out = {}
    entries = synth.draw_stack_ranks(77, 32, STACK_LINEARS, af1.af1_storage_bits)
    xs = {w: to_device(synth.make_activations(60 + w % 97, 1, w)) for w in (4096, 14336)}
    pools = [DevicePool(torch, m, n, r, 1, 5000 + i) for i, (_, m, n, _, r) in
             enumerate(entries)]
    alg = sum(gemv_algorithmic_bytes(m, n, r, 1) for _, m, n, _, r in entries)
    for label, waits in (("decoder_waits", ("q", "o", "gate", "down")), ("independent", ())):
        items = [(Desc(P.desc[0]), xs[n], torch.empty((1, m), dtype=torch.int16, device="cuda"),
                  name in waits) for P, (name, m, n, _, r) in zip(pools, entries)]
        S = LayerStream(items, 1)
        ms = graph_ms(S.run)
        out[f"stack_{label}_us_per_decoder_layer"] = round(ms * 1e3 / 32, 3)
        out[f"stack_{label}_gbs"] = round(alg / (ms * 1e-3) / 1e9, 1)
        del S, items
    del pools
    m, n, r = synth.SHAPES["attn4096"]
    pool = max(2, -(-POOL_BYTES // (r * (m + n) // 8)))
    P = DevicePool(torch, m, n, r, pool, 1000)
    x = to_device(synth.make_activations(1000, 1, n))
    for label, wait in (("each_layer_waits", True), ("independent", False)):
        items = [(Desc(P.desc[i]), x, torch.empty((1, m), dtype=torch.int16, device="cuda"),
                  wait) for i in range(pool)]
        S = LayerStream(items, 1)
        ms = graph_ms(S.run)
        us = ms * 1e3 / pool
        out[f"sq4096_{label}_us_per_layer"] = round(us, 3)
        out[f"sq4096_{label}_hbm_frac"] = round(gemv_algorithmic_bytes(m, n, r, 1) /
                                                (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        del S, items
    del P
    return out


def bench_dense_decode(args, torch, stream, af1_us):
    """Context for the paper's BF16-vs-AF1 decode ratio: the dense bf16
    layers these factorizations replace, as torch.matmul of a [1, n] bf16
    activation with a contiguous [n, m] bf16 weight (hipBLASLt/rocBLAS), over
    pools of weights larger than twice the last-level cache, replayed in
    HIP graphs.  af1_us is the headline AF1 time of the 4096^2 layer."""
    out = {}

    def graph_ms(fn, calls, reps=5):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        time_events(lambda i: graph.replay(), 2, stream)
        ms = time_events(lambda i: graph.replay(), reps, stream) / reps
        del graph
        return ms / calls

    n = m = 4096
    count = 16                               # 16 x 32 MB = 512 MB
    W = [torch.randn((n, m), device="cuda", dtype=torch.bfloat16) for _ in range(count)]
    x = torch.randn((1, n), device="cuda", dtype=torch.bfloat16)
    ys = [None] * count

    def run():
        for i in range(count):
            ys[i] = torch.matmul(x, W[i])
    ms = graph_ms(run, count)
    out["sq4096_b1_dense_bf16_us"] = round(ms * 1e3, 3)
    out["sq4096_b1_dense_bf16_gbs"] = round(n * m * 2 / (ms * 1e-3) / 1e9, 1)
    out["sq4096_b1_af1_speedup_vs_dense_bf16"] = round(ms * 1e3 / af1_us, 3)
    del W, ys
    # two decoder layers of the 8B shapes (872 MB of bf16 weights)
    shapes = [(m_, n_) for _, m_, n_, _ in STACK_LINEARS]
    Ws = [torch.randn((n_, m_), device="cuda", dtype=torch.bfloat16)
          for _ in range(2) for m_, n_ in shapes]
    xs = {w: torch.randn((1, w), device="cuda", dtype=torch.bfloat16) for w in (4096, 14336)}
    outs = [None] * len(Ws)

    def run_stack():
        for i, Wd in enumerate(Ws):
            outs[i] = torch.matmul(xs[Wd.shape[0]], Wd)
    ms = graph_ms(run_stack, 2)
    out["stack_dense_bf16_us_per_decoder_layer"] = round(ms * 1e3, 3)
    del Ws, outs
    return out


def bench_decode_table(args, torch, stream):
    from paper_2609_06161_amd import synth
    out = {}
    for name, b in DECODE_TABLE:
        m, n, r = shape_of(name)
        d = decode_time(args, torch, stream, m, n, r, b, 2000 + b, max(200, args.steps // 4))
        out[f"{name}_b{b}"] = dict(us_per_layer=round(d["us_graph"], 3),
                                   us_per_layer_eager=round(d["us_eager"], 3),
                                   gbs=round(d["alg_bytes"] / (d["us_graph"] * 1e-6) / 1e9, 1),
                                   alg_bytes=d["alg_bytes"])
    return out


def bench_gemm(args, torch, stream):
    from paper_2609_06161_amd import synth
    from paper_2609_06161_amd.layer import DeviceLayer, to_device
    T = 2048
    out = {}
    total_flops, total_ms = 0.0, 0.0
    for name in ("sq8192", "mlp_up28672x8192", "mlp_down8192x28672"):
        m, n, r = synth.SHAPES[name]
        lin = synth.make_linear(55, m, n, r, T)
        L = DeviceLayer.from_host(lin)
        x = to_device(lin.x)
        y = torch.empty((T, m), dtype=torch.int16, device="cuda")
        from paper_2609_06161_amd import af1
        ws = torch.empty(af1.af1_gemm_workspace_bytes(m, n, r, T), dtype=torch.uint8, device="cuda")
        fn = lambda i: L.gemm(x, y, ws, stream)
        sustain(fn, stream, args.sustain)
        ms = time_events(fn, args.gemm_steps, stream) / args.gemm_steps
        flops = 2.0 * T * r * (m + n)
        out[name] = dict(m=m, n=n, r=r, T=T, us=ms * 1e3, tflops=flops / (ms * 1e-3) / 1e12)
        total_flops += flops
        total_ms += ms
        del L, x, y, ws
        # Context: the dense bf16 layer this factorization replaces, as one
        # torch.matmul (hipBLASLt), [T, n] x [n, m] with contiguous operands.
        xd = torch.randn((T, n), device="cuda", dtype=torch.bfloat16)
        wd = torch.randn((n, m), device="cuda", dtype=torch.bfloat16)
        fd = lambda i: torch.matmul(xd, wd)
        sustain(fd, stream, args.sustain)
        msd = time_events(fd, args.gemm_steps, stream) / args.gemm_steps
        out[name]["dense_bf16_us"] = msd * 1e3
        out[name]["dense_bf16_tflops"] = 2.0 * T * n * m / (msd * 1e-3) / 1e12
        out[name]["speedup_vs_dense_bf16"] = msd / ms
        del xd, wd
    out["all3_tflops"] = total_flops / (total_ms * 1e-3) / 1e12
    # the 2.5-BPW setting at 4096^2 (context; not in the three-shape total)
    m, n, r = paper_25bpw_shape()
    lin = synth.make_linear(56, m, n, r, T)
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    y = torch.empty((T, m), dtype=torch.int16, device="cuda")
    ws = torch.empty(af1.af1_gemm_workspace_bytes(m, n, r, T), dtype=torch.uint8, device="cuda")
    fn = lambda i: L.gemm(x, y, ws, stream)
    sustain(fn, stream, args.sustain)
    ms = time_events(fn, args.gemm_steps, stream) / args.gemm_steps
    out["attn4096_r5120_2.5bpw"] = dict(m=m, n=n, r=r, T=T, us=ms * 1e3,
                                        tflops=2.0 * T * r * (m + n) / (ms * 1e-3) / 1e12)
    del L, x, y, ws
    # Context: the prefill regime below 2048 tokens (chunked prefill), where
    # the tile grid alone would leave compute units idle and the
    # contractions split K; µs per call at 4096^2 and 8192^2, eager and as a
    # replayed HIP graph of 10 calls (up to five launches per call).
    sweep = {}
    for name in ("attn4096", "sq8192"):
        m, n, r = shape_of(name)
        lin = synth.make_linear(57, m, n, r, 512)
        L = DeviceLayer.from_host(lin)
        for T in (32, 128, 512):
            x = to_device(lin.x[:T])
            y = torch.empty((T, m), dtype=torch.int16, device="cuda")
            ws = torch.empty(af1.af1_gemm_workspace_bytes(m, n, r, T), dtype=torch.uint8,
                             device="cuda")
            fn = lambda i: L.gemm(x, y, ws, stream)
            sustain(fn, stream, min(args.sustain, 0.1))
            ms = time_events(fn, args.gemm_steps, stream) / args.gemm_steps
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                L.gemm(x, y, ws, None)
            torch.cuda.current_stream().wait_stream(side)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for _ in range(10):
                    L.gemm(x, y, ws, None)
            time_events(lambda i: graph.replay(), 5, stream)
            msg = time_events(lambda i: graph.replay(), 20, stream) / 200
            flops = 2.0 * T * r * (m + n)
            sweep[f"{name}_T{T}"] = dict(us=round(ms * 1e3, 1), us_graph=round(msg * 1e3, 1),
                                         tflops_graph=round(flops / (msg * 1e-3) / 1e12, 1))
            del graph, x, y, ws
        del L
    out["few_tokens"] = sweep
    # MFMA roofline of the prefill leg: algorithmic flops 2*T*r*(m+n) of the
    # three calls over their summed time, against the dense fp16 peak (the
    # contractions run on fp16 operands); traffic: HBM bytes of the three
    # calls together.
    out["roofline"] = {"bound": "mfma", "achieved": round(out["all3_tflops"], 1),
                       "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                       "frac": round(out["all3_tflops"] / MFMA_F16_PEAK_TFLOPS, 4),
                       "traffic": measured_traffic(GEMM_TRAFFIC)}
    return out


def bench_train(args, torch, stream):
    """Scale-only reconstruction step (Sec. 4.1: signs frozen, the three
    scale vectors trained) on sq8192 at T = 2048: the training forward (y
    and the saved intermediates) and the backward (dx and the three scale
    gradients).  Algorithmic flops: 2*T*r*(m+n) per direction."""
    from paper_2609_06161_amd import af1, synth
    from paper_2609_06161_amd.layer import DeviceLayer, to_device
    T = 2048
    m, n, r = synth.SHAPES["sq8192"]
    lin = synth.make_linear(57, m, n, r, T)
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    dy = to_device(synth.make_output_grad(58, T, m))
    y = torch.empty((T, m), dtype=torch.int16, device="cuda")
    saved = torch.empty(af1.af1_train_saved_bytes(m, n, r, T), dtype=torch.uint8, device="cuda")
    ws = torch.empty(af1.af1_train_workspace_bytes(m, n, r, T), dtype=torch.uint8, device="cuda")
    dx = torch.empty((T, n), dtype=torch.int16, device="cuda")
    grads = tuple(torch.empty(k, dtype=torch.float32, device="cuda") for k in (m, r, n))
    # the one-time transposes of the frozen factors
    BuT = torch.empty((r, m // 32), dtype=torch.int32, device="cuda")
    BvT = torch.empty((n, r // 32), dtype=torch.int32, device="cuda")
    ft = lambda i: (af1.af1_pack_transpose(L.Bu, m, r, BuT, stream),
                    af1.af1_pack_transpose(L.Bv, r, n, BvT, stream))
    time_events(ft, 3, stream)
    ms_t = time_events(ft, 20, stream) / 20
    L._T = (BuT, BvT)
    fwd = lambda i: L.forward_train(x, y, saved, ws, stream)
    bwd = lambda i: L.backward(x, dy, saved, dx, grads, False, ws, stream)
    step = lambda i: (fwd(i), bwd(i))
    inf = lambda i: L.gemm(x, y, ws, stream)
    def timed(f):
        sustain(f, stream, args.sustain)
        return time_events(f, args.gemm_steps, stream) / args.gemm_steps
    ms_f, ms_b, ms_s, ms_i = timed(fwd), timed(bwd), timed(step), timed(inf)
    flops = 2.0 * T * r * (m + n)
    tb = lambda ms, f=flops: round(f / (ms * 1e-3) / 1e12, 1)
    sign_bytes = 2 * (m * r + r * n) / 8          # read + write, both factors
    return {"workload": f"scale-only reconstruction step, sq8192 ({m}x{n} r={r}), T={T}",
            "us_forward_train": round(ms_f * 1e3, 2), "tflops_forward_train": tb(ms_f),
            "us_forward_inference": round(ms_i * 1e3, 2),
            "us_backward": round(ms_b * 1e3, 2), "tflops_backward": tb(ms_b),
            "us_step": round(ms_s * 1e3, 2), "tflops_step": tb(ms_s, 2 * flops),
            "tokens_per_s_step": round(T / (ms_s * 1e-3), 0),
            "us_transpose_both_factors": round(ms_t * 1e3, 2),
            "transpose_gbs": round(sign_bytes / (ms_t * 1e-3) / 1e9, 1),
            "roofline_backward": {"bound": "mfma", "achieved": tb(ms_b),
                                  "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                  "frac": round(flops / (ms_b * 1e-3) / 1e12
                                                / MFMA_F16_PEAK_TFLOPS, 4),
                                  "traffic": measured_traffic(TRAIN_BWD_TRAFFIC)}}


def bench_nabf(args, torch, stream):
    """One iteration of the NABF loop (Algorithm nabf) on a synthetic
    surrogate W' = A* B* + noise, and its building blocks, at 4096x4096,
    r = 2016 (fp32 products on rocBLAS, fp64 eigenproblems on rocSOLVER),
    plus the fp64 oracle's iteration at 1024x1024, r = 480 on the host."""
    import numpy as np
    from paper_2609_06161_amd import af1, nabf
    from paper_2609_06161_amd.layer import to_device
    out = {}

    def state(m, n, r, seed):
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        rn = lambda *sh, s=1.0: torch.randn(*sh, device="cuda", generator=g) * s
        As, Bs = rn(m, r, s=0.2), rn(r, n, s=0.2)
        Wp = (As @ Bs + 0.03 * rn(m, n)).contiguous()
        D = dict(A=(As + rn(m, r, s=0.05)).contiguous(), B=(Bs + rn(r, n, s=0.05)).contiguous(),
                 UA=torch.zeros(m, r, device="cuda"), UB=torch.zeros(r, n, device="cuda"),
                 A_bits=torch.empty(m, r // 32, dtype=torch.int32, device="cuda"),
                 B_bits=torch.empty(r, n // 32, dtype=torch.int32, device="cuda"),
                 a=torch.empty(m, device="cuda"), m1=torch.empty(r, device="cuda"),
                 m2=torch.empty(r, device="cuda"), b=torch.empty(n, device="cuda"))
        return Wp, D

    m = n = 4096
    r = 2016
    Wp, D = state(m, n, r, 5)
    ws = torch.empty(nabf.af1_nabf_workspace_bytes(m, n, r), dtype=torch.uint8, device="cuda")
    nb = ws.numel()
    # the start: SVID of the perturbed factors, as the loop's initialisation
    nabf.af1_svid(D["A"], m, r, 30, D["A_bits"], D["a"], D["m1"], ws, nb, stream)
    nabf.af1_svid(D["B"], r, n, 30, D["B_bits"], D["m2"], D["b"], ws, nb, stream)
    out_m_r = torch.empty(m, r, device="cuda")
    C = (D["B"] @ D["B"].T).contiguous()
    P = torch.empty(r, r, device="cuda")
    fit = torch.empty(r, device="cuda")
    legs = {
        "admm_left": lambda i: nabf.af1_admm_proxy(0, Wp, m, n, r, D["A"], D["B"], D["UA"], 0.5,
                                                   out_m_r, ws, nb, stream),
        "svid_30_passes_4096x2016": lambda i: nabf.af1_svid(out_m_r, m, r, 30, D["A_bits"],
                                                            D["a"], D["m1"], ws, nb, stream),
        "nullspace_projector_r2016": lambda i: nabf.af1_nullspace_projector(C, r, 0.01, P, None,
                                                                            ws, nb, stream),
        "scale_fit_left": lambda i: nabf.af1_scale_fit(0, out_m_r, D["A_bits"], D["a"], D["m1"],
                                                       m, r, P, fit, ws, nb, stream),
    }
    for name, fn in legs.items():
        time_events(fn, 1, stream)
        out[f"ms_{name}"] = round(time_events(fn, 3, stream) / 3, 3)
    # rebuild a consistent state, then time whole iterations
    Wp, D = state(m, n, r, 5)
    nabf.af1_svid(D["A"], m, r, 30, D["A_bits"], D["a"], D["m1"], ws, nb, stream)
    nabf.af1_svid(D["B"], r, n, 30, D["B_bits"], D["m2"], D["b"], ws, nb, stream)
    st = nabf.make_state(m, n, r, D["A"], D["B"], D["UA"], D["UB"], D["A_bits"], D["B_bits"],
                         D["a"], D["m1"], D["m2"], D["b"])
    # dense factors equal to their binary-scaled forms (set-up, not timed)
    for key, bits, left, right, rows, cols in (("A", "A_bits", "a", "m1", m, r),
                                               ("B", "B_bits", "m2", "b", r, n)):
        signs = torch.empty(rows, cols, dtype=torch.int8, device="cuda")
        af1.af1_unpack(D[bits], rows, cols, signs, stream)
        D[key].copy_(D[left][:, None] * signs.float() * D[right][None, :])

    def recon():
        torch.cuda.synchronize()
        A, B, W = D["A"].double(), D["B"].double(), Wp.double()
        return float(torch.linalg.norm(W - A @ B) / torch.linalg.norm(W))
    err0 = recon()
    it = lambda i: nabf.af1_nabf_iteration(Wp, st, 0.5, 0.01, 30, ws, nb, stream)
    time_events(it, 1, stream)
    ms = time_events(it, 3, stream) / 3
    out["workload"] = (f"NABF iteration (both factors) on a synthetic surrogate {m}x{n}, r={r}: "
                       "W' = A*B* + noise, start from SVID of perturbed factors; rho=0.5, "
                       "eta=0.01, 30 power-iteration passes")
    out["ms_iteration"] = round(ms, 2)
    out["relative_error_start"] = round(err0, 4)
    out["relative_error_after_4_iterations"] = round(recon(), 4)
    # left: B B^T, W' B^T, the Cholesky solve, E P; right: A^T A, A^T W', the
    # two triangular solves, P E
    fp32 = (2 * r * r * n + 2 * m * n * r + 2 * r * r * m + 2 * m * r * r) \
        + (2 * r * r * m + 2 * m * n * r + 2 * r * r * n + 2 * r * r * n)
    out["fp32_gflop_per_iteration_products"] = round(fp32 / 1e9, 1)
    out["fp64_gflop_per_iteration_projectors"] = round(2 * 2 * r ** 3 / 1e9, 1)
    del Wp, D, ws, C, P, out_m_r
    # the oracle's iteration on the host, at a smaller shape
    if not args.no_cpu_baseline:
        import time
        from oracle import nabf as onabf
        mm = nn = 1024
        rr = 480
        rng = np.random.default_rng(9)
        As, Bs = rng.standard_normal((mm, rr)) * 0.2, rng.standard_normal((rr, nn)) * 0.2
        Wph = As @ Bs + 0.03 * rng.standard_normal((mm, nn))
        Ab, a, m1 = onabf.svid((As + 0.05 * rng.standard_normal((mm, rr))).astype(np.float32), 30)
        Bb, m2, b = onabf.svid((Bs + 0.05 * rng.standard_normal((rr, nn))).astype(np.float32), 30)
        S = dict(A_bits=Ab, B_bits=Bb, a=a, m1=m1, m2=m2, b=b,
                 A=onabf.binary_scaled(Ab, a, m1, rr), B=onabf.binary_scaled(Bb, m2, b, nn),
                 UA=np.zeros((mm, rr)), UB=np.zeros((rr, nn)))
        t0 = time.perf_counter()
        onabf.nabf_iteration(Wph, S, 0.5, 0.01, 30)
        out["cpu_oracle_ms_iteration_1024x1024_r480"] = round((time.perf_counter() - t0) * 1e3, 1)
        Wg = to_device(Wph.astype(np.float32))
        Dg = {k: to_device(np.ascontiguousarray(v.astype(np.float32) if v.dtype == np.float64
                                                else v)) for k, v in S.items()}
        wsg = torch.empty(nabf.af1_nabf_workspace_bytes(mm, nn, rr), dtype=torch.uint8,
                          device="cuda")
        stg = nabf.make_state(mm, nn, rr, Dg["A"], Dg["B"], Dg["UA"], Dg["UB"], Dg["A_bits"],
                              Dg["B_bits"], Dg["a"], Dg["m1"], Dg["m2"], Dg["b"])
        itg = lambda i: nabf.af1_nabf_iteration(Wg, stg, 0.5, 0.01, 30, wsg, wsg.numel(), stream)
        time_events(itg, 1, stream)
        out["gpu_ms_iteration_1024x1024_r480"] = round(time_events(itg, 3, stream) / 3, 2)
    return out


def bench_pack(args, torch, stream):
    """Sign -> bit packing of a 16384 x 16384 matrix from each source type:
    HBM-bound, algorithmic bytes = source bytes + packed bytes."""
    from paper_2609_06161_amd import af1
    rows = cols = 16384
    out = {}
    dst = torch.empty(rows * cols // 32, dtype=torch.int32, device="cuda")
    for name, dtype, code in (("f32", torch.float32, af1.AF1_SRC_F32),
                              ("bf16", torch.bfloat16, af1.AF1_SRC_BF16),
                              ("i8", torch.int8, af1.AF1_SRC_I8)):
        g = torch.Generator(device="cuda")
        g.manual_seed(3)
        src = (torch.randint(-100, 100, (rows, cols), device="cuda", generator=g)
               .to(dtype))
        fn = lambda i: af1.af1_pack(src, code, rows, cols, dst, None)
        time_events(fn, 3, stream)
        ms = time_events(fn, 20, stream) / 20
        nbytes = rows * cols * src.element_size() + rows * cols // 8
        out[name] = dict(us=round(ms * 1e3, 1), gbs=round(nbytes / (ms * 1e-3) / 1e9, 1),
                         frac=round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 3))
        del src
    # Context: a plain device copy of 1 GiB (read + write), the practical
    # HBM rate of this GPU.
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    c = torch.empty_like(a)
    fn = lambda i: c.copy_(a)
    time_events(fn, 3, stream)
    ms = time_events(fn, 10, stream) / 10
    out["copy_1GiB_gbs"] = round(2 * (1 << 30) / (ms * 1e-3) / 1e9, 1)
    del a, c
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def bench_cpu_oracle(args):
    """The fp64 oracle on the host: the 4096x4096 r=2016 layer at the bench's
    batch, with every OpenMP thread, then with one."""
    import oracle
    from paper_2609_06161_amd import synth
    m, n, r = synth.SHAPES["attn4096"]
    lin = synth.make_linear(1000, m, n, r, args.batch)

    def timed(seconds):
        oracle.forward(m, n, r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, lin.x)  # warm
        calls, t0 = 0, time.perf_counter()
        while True:
            oracle.forward(m, n, r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, lin.x)
            calls += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                return calls, el
    threads = oracle.num_threads()
    calls, el = timed(args.cpu_seconds * 0.6)
    oracle.set_num_threads(1)
    try:
        calls1, el1 = timed(args.cpu_seconds * 0.4)
    finally:
        oracle.set_num_threads(threads)
    return dict(value=el / calls * 1e6, unit="us/layer", cores=threads, kind="oracle",
                cpu_model=cpu_model(), value_1_thread=el1 / calls1 * 1e6,
                sample=f"{calls} full fp64 forward calls of the 4096x4096 r=2016 b={args.batch} "
                       f"layer in {el:.1f} s with {threads} threads; {calls1} calls in "
                       f"{el1:.1f} s with 1 thread")


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the "
              "multi-GPU sharding of this layer is described but not built.", file=sys.stderr)
        sys.exit(2)
    if args.shape != "attn4096" and args.only != "gemv":
        print("--shape applies to --only gemv (the headline is the 4096x4096 layer)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    if args.calibrate_copy:
        src = torch.ones(64 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.only == "gemm":
        out = bench_gemm(args, torch, stream)
        print(json.dumps({"gemm": out}), flush=True)
        return
    if args.only == "train":
        print(json.dumps({"train": bench_train(args, torch, stream)}), flush=True)
        return
    if args.only == "nabf":
        print(json.dumps({"nabf": bench_nabf(args, torch, stream)}), flush=True)
        return

    m, n, r = shape_of(args.shape)
    g = decode_time(args, torch, stream, m, n, r, args.batch, 1000, args.steps,
                    exact_steps=(args.steps, args.warmup))
    # steady state: whole passes over the weight pool (the requested step
    # count rounded up to whole passes), graph-replayed back to back
    g["ms_per_step"] = g["us_graph"] * 1e-3
    us = g["us_graph"]
    achieved = g["alg_bytes"] / (g["ms_per_step"] * 1e-3) / 1e9
    result = {
        "metric": METRIC,
        "value": round(us, 4),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": g["steps_timed"],
        "warmup": args.warmup,
        "ms_per_step": g["ms_per_step"],
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"factorized GEMV {g['m']}x{g['n']} r={g['r']} b={g['b']} "
                               f"(1.0 BPW, fp16 scales, bf16 x/y), weights rotated over "
                               f"{g['pool']} distinct layers ({g['pool_mb']:.0f} MB)",
                   "m": g["m"], "n": g["n"], "r": g["r"], "batch": g["b"],
                   "timing": "HIP graph of one pass over the weight pool (two launches per "
                             "layer), replayed back to back; the requested step count is "
                             "rounded up to whole passes (steps = layers timed)",
                   "steps_requested": args.steps,
                   "us_per_layer_exact_requested_steps_one_replay": round(
                       g["exact_ms"] * 1e3 / g["exact_steps"], 3),
                   "us_per_layer_p10_p50_p90": [round(g["us_graph_p10"], 3),
                                                round(g["us_graph_p50"], 3),
                                                round(g["us_graph_p90"], 3)],
                   "us_per_layer_eager_launch": round(g["us_eager"], 3),
                   "us_per_launch_floor": launch_floor(torch, stream)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 5),
                     "traffic": measured_gemv_traffic(),
                     "alg_bytes_per_launch": g["alg_bytes"]},
    }
    if not args.no_decode_table and args.only == "all":
        result["decode_table"] = bench_decode_table(args, torch, stream)
        result["decode_stack_8b"] = bench_stack(args, torch, stream)
        result["decode_layer_stream"] = bench_layer_stream(args, torch, stream)
        dense = bench_dense_decode(args, torch, stream, us)
        dense["stack_af1_fused_speedup_vs_dense_bf16"] = round(
            dense["stack_dense_bf16_us_per_decoder_layer"] /
            result["decode_stack_8b"]["us_per_decoder_layer_fused_projections"], 3)
        result["decode_dense_bf16_context"] = dense
    if args.only == "all":
        result["pack_16384x16384"] = bench_pack(args, torch, stream)
    if not args.no_gemm and args.only == "all":
        result["gemm"] = bench_gemm(args, torch, stream)
        result["gemm"]["peak_tflops"] = MFMA_F16_PEAK_TFLOPS
        result["train"] = bench_train(args, torch, stream)
    if not args.no_cpu_baseline and args.only == "all":
        result["cpu_baseline"] = bench_cpu_oracle(args)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
