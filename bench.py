#!/usr/bin/env python3
"""Throughput of the W4A8 MoE layer on one MI355X.

Headline workload (one "step" = one whole MoE layer at decode M = 1: Q8_0 of
the token, routing, gate/up W4A8 GEMV, SiLU * up, Q8_0(h), down W4A8 GEMV,
weighted combine with the shared expert): hidden 2048, expert intermediate
512, 256 routed experts + 1 shared, top-8 from softmax of N(0,1) router
logits, Q4_0 expert weights quantized from N(0, 0.02^2), fp32 hidden ~ N(0,1).

Timing: eight distinct layers (3.6 GB of Q4_0) are cycled with fresh routing
and a fresh token every step, so the experts a step touches are not resident
in the 256 MB last-level cache; all inputs are in HBM before the timed region;
the K steps are captured in one HIP graph and replayed once between HIP events
recorded on the stream the kernels run on.  `value` is algorithmic bytes
(Q4_0 bytes of the distinct experts each step touches, plus the fp32 token in
and out, ids and weights) / time, in GB/s.

The line also carries the 947-token prefill of the same layer (router bias
~ N(0,1)) in tokens/s per layer, the same layer at batched decode (32 tokens),
a 40-layer stack (947-token prefill, then single-token decode steps, layers
chained by a residual RMSNorm), the roofline of the dominant kernel, and the
CPU oracle timed on this host on a bounded sample of the decode workload.
"""
from __future__ import annotations

import os
import re


def _host_setup():
    """Runs before torch or the CPU oracle load (OpenMP reads its settings
    when it starts): one OpenMP thread per physical core -- at most the CPU
    share the host gives this process, an OMP_NUM_THREADS already set --
    bound close, and, when more than one NUMA node is allowed, page
    interleaving over them for this process (the paper interleaves its expert
    block over both sockets, Sec. 4.3; hyper-threads hurt, Sec. 5.5)."""
    info = {}
    try:
        out = os.popen("lscpu").read()
        soc = int(re.search(r"Socket\(s\):\s+(\d+)", out).group(1))
        cps = int(re.search(r"Core\(s\) per socket:\s+(\d+)", out).group(1))
        info["physical_cores"] = soc * cps
    except Exception:
        info["physical_cores"] = os.cpu_count() or 1
    n = info["physical_cores"]
    share = os.environ.get("OMP_NUM_THREADS", "")
    if share.isdigit() and int(share) > 0:
        n = min(n, int(share))
        info["cpu_share"] = int(share)
    os.environ["OMP_NUM_THREADS"] = str(n)
    os.environ["OMP_PROC_BIND"] = "close"
    os.environ["OMP_PLACES"] = "cores"
    info["omp_threads"] = n
    nodes = []
    try:
        with open("/proc/self/status") as f:
            for line in f:
                if line.startswith("Mems_allowed_list:"):
                    for part in line.split(":", 1)[1].strip().split(","):
                        a, _, b = part.partition("-")
                        nodes += list(range(int(a), int(b or a) + 1))
    except Exception:
        pass
    info["numa_nodes"] = len(nodes) or 1
    info["numa_policy"] = "default"
    if len(nodes) > 1:
        import ctypes
        mask = 0
        for nd in nodes:
            mask |= 1 << nd
        words = (ctypes.c_ulong * 16)(*[(mask >> (64 * i)) & ((1 << 64) - 1) for i in range(16)])
        libc = ctypes.CDLL(None, use_errno=True)
        MPOL_INTERLEAVE, SYS_set_mempolicy = 3, 238
        rc = libc.syscall(SYS_set_mempolicy, MPOL_INTERLEAVE, words, ctypes.c_ulong(16 * 64))
        info["numa_policy"] = "interleave" if rc == 0 else f"interleave failed (errno {ctypes.get_errno()})"
    return info


HOST = _host_setup()

import argparse   # noqa: E402
import hashlib    # noqa: E402
import json       # noqa: E402
import sys        # noqa: E402
import time       # noqa: E402

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

H, I, E, K_TOP = 2048, 512, 256, 8
EXPERT_BYTES = (2 * I * (H // 32) + H * (I // 32)) * 18   # 1,769,472
HBM_PEAK_GBPS = 8000.0
INT8_PEAK_TOPS = 5000.0    # dense int8 matrix-core peak, TOP/s
METRIC = "MoE-layer W4A8 GEMV GB/s (% HBM peak) at M=1; prefill tokens/s per layer"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--layers", type=int, default=8, help="distinct weight sets cycled")
    ap.add_argument("--prefill-steps", type=int, default=8)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="launch steps eagerly")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--m32-steps", type=int, default=64)
    ap.add_argument("--stack-layers", type=int, default=40)
    ap.add_argument("--stack-decode-steps", type=int, default=128)
    ap.add_argument("--no-m32", action="store_true")
    ap.add_argument("--no-stack", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the E/k invariants, router, LM-head and 1024x1024 GEMV lines")
    ap.add_argument("--section", choices=["gemm", "sym_layer", "gdn"],
                    help="run only this extra section and print its result as JSON "
                         "(for profiling one kernel family)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy 5 times (for scaling the "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def make_layer(torch, w4, gen, dev):
    """One layer's Q4_0 weights from N(0, 0.02^2) fp32, quantized on the GPU
    by the library's Q4_0 kernel, 16 experts at a time."""
    w_gu = torch.empty((E, 2 * I, H // 32 * 18), dtype=torch.uint8, device=dev)
    w_d = torch.empty((E, H, I // 32 * 18), dtype=torch.uint8, device=dev)
    chunk = 16
    for e0 in range(0, E, chunk):
        f = torch.randn((chunk * 2 * I, H), generator=gen, device=dev) * 0.02
        w4.q4_0_quantize(f, out=w_gu[e0:e0 + chunk].view(chunk * 2 * I, -1))
        f = torch.randn((chunk * H, I), generator=gen, device=dev) * 0.02
        w4.q4_0_quantize(f, out=w_d[e0:e0 + chunk].view(chunk * H, -1))
    s_gu = w4.q4_0_quantize(torch.randn((2 * I, H), generator=gen, device=dev) * 0.02)
    s_d = w4.q4_0_quantize(torch.randn((H, I), generator=gen, device=dev) * 0.02)
    return w_gu, w_d, s_gu, s_d


def step_bytes(ids_row) -> int:
    distinct = len({int(e) for e in ids_row if 0 <= e < E})
    return (distinct + 1) * EXPERT_BYTES + 2 * H * 4 * (len(ids_row) // K_TOP) + ids_row.size * 8


def source_sha(files) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


DECODE_SOURCES = ["paper_2606_24031_amd/csrc/decode.hip", "paper_2606_24031_amd/csrc/w4a8_dev.h",
                  "paper_2606_24031_amd/csrc/router_dev.h"]


def measured_traffic():
    """HBM bytes per launch of the decode kernel from the committed rocprofv3
    PMC summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "decode_m1_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_sha = re.search(r"source_sha:\s*([0-9a-f]+)", text)
    m_val = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_sha or not m_val or m_sha.group(1) != source_sha(DECODE_SOURCES):
        return None
    return float(m_val.group(1))


def bench_decode(torch, w4, synth, layers, args, dev):
    rng = synth.rng(args.seed + 1)
    nsteps = args.steps
    total = nsteps + args.warmup
    ids_all, wts_all = synth.routing(rng, total, E, K_TOP)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 2)
    x_all = torch.randn((total, 1, H), generator=gen, device=dev)
    ids_d = torch.from_numpy(ids_all).to(dev).view(total, 1, K_TOP)
    wts_d = torch.from_numpy(wts_all).to(dev).view(total, 1, K_TOP)
    ws = w4.moe_workspace(1, H, I, E, K_TOP, device=dev)
    out = torch.empty((1, H), dtype=torch.float32, device=dev)

    def step(i):
        L = layers[i % len(layers)]
        w4.moe_forward(x_all[i], ids_d[i], wts_d[i], L[0], L[1], L[2], L[3], H, I, E, K_TOP,
                       ws, out=out)

    log(f"decode: warmup {args.warmup} steps")
    for i in range(args.warmup):
        step(nsteps + i)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    if args.no_graph:
        torch.cuda.synchronize()
        ev0.record()
        for i in range(nsteps):
            step(i)
        ev1.record()
        torch.cuda.synchronize()
    else:
        log(f"decode: capturing {nsteps} steps in a HIP graph")
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(nsteps):
                step(i)
        graph.replay()   # untimed first replay
        torch.cuda.synchronize()
        log("decode: timed replay")
        ev0.record()
        graph.replay()
        ev1.record()
        torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    nbytes = sum(step_bytes(ids_all[i]) for i in range(nsteps))
    return ms, nbytes


def bench_decode_invariants(torch, w4, synth, layers, args, dev, n=500):
    """Single-token layer at E = 128 (the first 128 experts of the same
    weight sets: the bytes per step are those of E = 256, so the time should
    be too) and at k = 4 (5 experts per step instead of 9)."""
    res = {}
    for name, e_, k_ in (("E128_k8", 128, 8), ("E256_k4", 256, 4)):
        rng = synth.rng(args.seed + 11)
        ids_all, wts_all = synth.routing(rng, n, e_, k_)
        gen = torch.Generator(device=dev)
        gen.manual_seed(args.seed + 12)
        x_all = torch.randn((n, 1, H), generator=gen, device=dev)
        ids_d = torch.from_numpy(ids_all).to(dev).view(n, 1, k_)
        wts_d = torch.from_numpy(wts_all).to(dev).view(n, 1, k_)
        ws = w4.moe_workspace(1, H, I, e_, k_, device=dev)
        out = torch.empty((1, H), dtype=torch.float32, device=dev)

        def step(i):
            L = layers[i % len(layers)]
            w4.moe_forward(x_all[i], ids_d[i], wts_d[i], L[0], L[1], L[2], L[3], H, I, e_, k_,
                           ws, out=out)

        for i in range(20):
            step(i)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(n):
                step(i)
        graph.replay()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        graph.replay()
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1)
        nbytes = sum((len({int(e) for e in ids_all[i]}) + 1) * EXPERT_BYTES + 2 * H * 4 + k_ * 8
                     for i in range(n))
        gbps = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"us_per_step": round(ms * 1e3 / n, 2), "GBps": round(gbps, 1),
                     "hbm_peak_frac": round(gbps / HBM_PEAK_GBPS, 4), "launch": "hipGraph"}
    return res


def bench_prefill(torch, w4, synth, layers, args, dev, T=947, n=None):
    """T tokens through one layer call (top-8 of 256 with a per-expert router
    bias, so group sizes are uneven as in a real prompt), cycling the weight
    sets; int8 operations counted over every valid pair's three products."""
    rng = synth.rng(args.seed + 3 + T)
    n = args.prefill_steps if n is None else n
    ids_l, wts_l, byts = [], [], []
    for _ in range(n + 2):
        ids, wts = synth.routing(rng, T, E, K_TOP, bias_std=1.0)
        ids_l.append(torch.from_numpy(ids).to(dev))
        wts_l.append(torch.from_numpy(wts).to(dev))
        touched = len(set(ids.ravel().tolist()))
        byts.append((touched + 1) * EXPERT_BYTES + 2 * T * H * 4 + ids.size * 8)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 4)
    xs = [torch.randn((T, H), generator=gen, device=dev) for _ in range(n + 2)]
    ws = w4.moe_workspace(T, H, I, E, K_TOP, device=dev)
    out = torch.empty((T, H), dtype=torch.float32, device=dev)

    def step(i):
        L = layers[i % len(layers)]
        w4.moe_forward(xs[i], ids_l[i], wts_l[i], L[0], L[1], L[2], L[3], H, I, E, K_TOP, ws,
                       out=out)

    log(f"prefill {T} tokens: warmup 2, timed {n}")
    step(n)
    step(n + 1)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for i in range(n):
        step(i)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / n
    ops = 2.0 * T * (K_TOP + 1) * 3 * H * I
    return {"tokens": T, "ms_per_layer": round(ms, 4),
            "tokens_per_s_per_layer": round(T / (ms / 1e3), 1),
            "GBps": round(sum(byts[:n]) / n / (ms / 1e3) / 1e9, 1),
            "hbm_peak_frac": round(sum(byts[:n]) / n / (ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
            "int8_TOPs": round(ops / (ms / 1e3) / 1e12, 1),
            "int8_peak_frac": round(ops / (ms / 1e3) / 1e12 / INT8_PEAK_TOPS, 4)}


def bench_one_expert(torch, w4, synth, args, dev, T=947, n=20):
    """One expert alone over T token rows (E = 1, k = 1, no shared expert:
    one group of T rows through the grouped int8-MFMA kernels), the point of
    the matrix-core sweep where the group is as large as the prompt."""
    g = synth.rng(args.seed + 12)
    w_gu = torch.from_numpy(synth.q4_0_random_blocks(g, 2 * I, H)).to(dev)
    w_d = torch.from_numpy(synth.q4_0_random_blocks(g, H, I)).to(dev)
    x = torch.from_numpy(synth.normal_f32(g, (T, H))).to(dev)
    ids = torch.zeros((T, 1), dtype=torch.int32, device=dev)
    wts = torch.ones((T, 1), dtype=torch.float32, device=dev)
    ws = w4.moe_workspace(T, H, I, 1, 1, device=dev)
    out = torch.empty((T, H), dtype=torch.float32, device=dev)
    for _ in range(3):
        w4.moe_forward(x, ids, wts, w_gu, w_d, None, None, H, I, 1, 1, ws, out=out)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(n):
        w4.moe_forward(x, ids, wts, w_gu, w_d, None, None, H, I, 1, 1, ws, out=out)
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / n * 1e3
    ops = 2.0 * T * 3 * H * I
    return {"tokens": T, "us_per_layer": round(us, 2), "int8_TOPs": round(ops / us / 1e6, 1),
            "int8_peak_frac": round(ops / us / 1e6 / INT8_PEAK_TOPS, 4)}


def bench_m32(torch, w4, synth, layers, args, dev, T=32, n=None):
    """Batched decode, T tokens (32) per layer call, each routed independently
    (top-8 of 256, no router bias); the calls cycle the weight sets and are
    replayed from one HIP graph."""
    n = args.m32_steps if n is None else n
    rng = synth.rng(args.seed + 5 + T)
    ids_l, wts_l, byts = [], [], []
    for _ in range(n):
        ids, wts = synth.routing(rng, T, E, K_TOP)
        ids_l.append(torch.from_numpy(ids).to(dev))
        wts_l.append(torch.from_numpy(wts).to(dev))
        byts.append((len(set(ids.ravel().tolist())) + 1) * EXPERT_BYTES + 2 * T * H * 4 + ids.size * 8)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 6)
    xs = torch.randn((n, T, H), generator=gen, device=dev)
    ws = w4.moe_workspace(T, H, I, E, K_TOP, device=dev)
    out = torch.empty((T, H), dtype=torch.float32, device=dev)

    def step(i):
        L = layers[i % len(layers)]
        w4.moe_forward(xs[i], ids_l[i], wts_l[i], L[0], L[1], L[2], L[3], H, I, E, K_TOP, ws, out=out)

    for i in range(min(n, 4)):
        step(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n):
            step(i)
    graph.replay()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / n
    gbps = sum(byts) / n / (ms / 1e3) / 1e9
    return {"tokens": T, "us_per_layer": round(ms * 1e3, 2),
            "tokens_per_s_per_layer": round(T / (ms / 1e3), 1), "GBps": round(gbps, 1),
            "hbm_peak_frac": round(gbps / HBM_PEAK_GBPS, 4), "calls": n}


def bench_router(torch, w4, synth, args, dev):
    """Router top-k on fp32 logits ~ N(0,1) (plus the per-expert bias for the
    947-token case): 947 tokens and 1 token, E = 256, k = 8."""
    res = {}
    for T, bias in ((947, 1.0), (1, 0.0)):
        g = synth.rng(args.seed + 7)
        b = synth.normal_f32(g, (E,), bias) if bias > 0 else 0.0
        logits = torch.from_numpy(synth.normal_f32(g, (T, E)) + b).to(dev)
        ids = torch.empty((T, K_TOP), dtype=torch.int32, device=dev)
        wts = torch.empty((T, K_TOP), dtype=torch.float32, device=dev)
        n = 200
        for _ in range(5):
            w4.router_topk(logits, K_TOP, ids, wts)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(n):
                w4.router_topk(logits, K_TOP, ids, wts)
        graph.replay()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        graph.replay()
        ev1.record()
        torch.cuda.synchronize()
        us = ev0.elapsed_time(ev1) / n * 1e3
        res[f"T{T}"] = {"us_per_call": round(us, 2), "tokens_per_s": round(T / (us / 1e6), 1),
                        "launch": "hipGraph"}
    return res


def bench_gemv_1024(torch, w4, synth, args, dev, copies=2048, n=2048):
    """The single W4A8 GEMV of 1024 x 1024 (Q4_0 weights from N(0, 0.02^2),
    one Q8_0 vector from N(0, 1)).  Its 0.59 MB of weights fit in L2, so the
    streaming rate is taken over `copies` distinct weight copies (1.2 GB,
    several times the last-level cache) replayed from one HIP graph; the
    latency of repeated calls on one copy (cache-resident) is reported
    beside it."""
    N = K = 1024
    g = synth.rng(args.seed)
    W = torch.from_numpy(synth.normal_f32(g, (N, K), 0.02)).to(dev)
    wq0 = w4.q4_0_quantize(W)
    blk = synth.q4_0_random_blocks(g, N, K)
    wbytes = N * (K // 32) * 18
    pool = torch.empty((copies, wbytes), dtype=torch.uint8, device=dev)
    pool[0].copy_(wq0.reshape(-1))
    src = torch.from_numpy(blk.reshape(-1)).to(dev)
    for c in range(1, copies):
        pool[c].copy_(src)
    xq = w4.q8_0_quantize(torch.from_numpy(synth.normal_f32(g, (1, K))).to(dev))
    y = torch.empty(N, dtype=torch.float32, device=dev)
    nbytes = wbytes + (K // 32) * 34 + N * 4

    def timed(sel):
        for i in range(8):
            w4.q4q8_gemv(pool[sel(i)], xq, N, K, y=y)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(n):
                w4.q4q8_gemv(pool[sel(i)], xq, N, K, y=y)
        graph.replay()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        graph.replay()
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / n * 1e3

    us_stream = timed(lambda i: i % copies)
    us_hot = timed(lambda i: 0)
    del pool
    return {"N": N, "K": K, "bytes_per_call": nbytes, "weight_copies": copies,
            "us_per_call": round(us_stream, 3),
            "GBps": round(nbytes / (us_stream / 1e6) / 1e9, 1),
            "hbm_peak_frac": round(nbytes / (us_stream / 1e6) / 1e9 / HBM_PEAK_GBPS, 4),
            "us_per_call_cache_resident": round(us_hot, 3),
            "launch": "hipGraph"}


def bench_gemv_sym(torch, w4, synth, args, dev):
    """The GEMV in the paper's own block format (symmetric 4-bit weights with an
    fp32 scale per 32, 20-byte blocks; 8-bit activations with an fp32 scale)
    at the output projection's shape (N = 151936, K = 2048, 195 MB), two
    weight copies alternated so successive calls stream from HBM."""
    N, K = 151936, H
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 10)
    ws = []
    for _ in range(2):
        wq = torch.empty((N, K // 32 * 20), dtype=torch.uint8, device=dev)
        for r0 in range(0, N, 16384):   # quantize in slabs: bounded fp32 staging
            r1 = min(N, r0 + 16384)
            W = torch.randn((r1 - r0, K), generator=gen, device=dev) * 0.02
            w4.q4_sym_quantize(W, out=wq[r0:r1])
        ws.append(wq)
    xq = w4.q8_f32_quantize(torch.randn((1, K), generator=gen, device=dev))
    y = torch.empty(N, dtype=torch.float32, device=dev)
    n = 40
    for i in range(4):
        w4.q4sym_q8f32_gemv(ws[i % 2], xq, N, K, y=y)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n):
            w4.q4sym_q8f32_gemv(ws[i % 2], xq, N, K, y=y)
    graph.replay()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / n * 1e3
    nbytes = N * (K // 32) * 20 + (K // 32) * 36 + N * 4
    del ws
    return {"N": N, "K": K, "format": "q4_sym x q8_f32 (fp32 scales)",
            "us_per_call": round(us, 2),
            "GBps": round(nbytes / (us / 1e6) / 1e9, 1),
            "hbm_peak_frac": round(nbytes / (us / 1e6) / 1e9 / HBM_PEAK_GBPS, 4),
            "launch": "hipGraph"}


def bench_lm_head(torch, w4, synth, args, dev):
    """The dense W4A8 GEMV at the output projection's shape (N = 151936
    vocabulary rows, K = H = 2048; random Q4_0 blocks, 175 MB), two weight
    copies alternated so successive calls stream from HBM."""
    N, K = 151936, H
    g = synth.rng(args.seed + 9)
    ws = [torch.from_numpy(synth.q4_0_random_blocks(g, N, K)).to(dev) for _ in range(2)]
    xq = w4.q8_0_quantize(torch.from_numpy(synth.normal_f32(g, (1, K))).to(dev))
    y = torch.empty(N, dtype=torch.float32, device=dev)
    n = 40
    for i in range(4):
        w4.q4q8_gemv(ws[i % 2], xq, N, K, y=y)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n):
            w4.q4q8_gemv(ws[i % 2], xq, N, K, y=y)
    graph.replay()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / n * 1e3
    nbytes = N * (K // 32) * 18 + (K // 32) * 34 + N * 4
    del ws
    return {"N": N, "K": K, "us_per_call": round(us, 2),
            "GBps": round(nbytes / (us / 1e6) / 1e9, 1),
            "hbm_peak_frac": round(nbytes / (us / 1e6) / 1e9 / HBM_PEAK_GBPS, 4),
            "launch": "hipGraph"}


def bench_gemm(torch, w4, synth, args, dev):
    """Dense W4A8 products of M activation rows (q4q8_gemm, one Q8_0
    alignment launch and one int8-MFMA launch): the output projection at
    M = 32 (HBM-bound: 175 MB of Q4_0 weights) and an M-sweep at the
    dense-layer shape N = K = 2048 (int8 operations against the matrix
    cores' peak), each timed over a hipGraph of back-to-back calls."""
    out = {}

    def timed(w_list, M, N, K, n):
        g = synth.rng(args.seed + 11 + M)
        xq = w4.q8_0_quantize(torch.from_numpy(synth.normal_f32(g, (M, K))).to(dev))
        y = torch.empty((M, N), dtype=torch.float32, device=dev)
        ws = w4.gemm_workspace(M, K, device=dev)
        for i in range(3):
            w4.q4q8_gemm(w_list[i % len(w_list)], xq, M, N, K, y=y, workspace=ws)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(n):
                w4.q4q8_gemm(w_list[i % len(w_list)], xq, M, N, K, y=y, workspace=ws)
        graph.replay()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        graph.replay()
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / n * 1e3

    N, K, M = 151936, H, 32
    g = synth.rng(args.seed + 10)
    ws = [torch.from_numpy(synth.q4_0_random_blocks(g, N, K)).to(dev) for _ in range(2)]
    us = timed(ws, M, N, K, 20)
    nbytes = N * (K // 32) * 18 + M * (K // 32) * 34 + M * N * 4
    out["lm_head_m32"] = {"M": M, "N": N, "K": K, "us_per_call": round(us, 2),
                          "GBps": round(nbytes / us / 1e3, 1),
                          "hbm_peak_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBPS, 4)}
    del ws
    N = K = H
    ws = [torch.from_numpy(synth.q4_0_random_blocks(g, N, K)).to(dev)]
    sweep = []
    for M in (32, 128, 947, 4096, 16384):
        us = timed(ws, M, N, K, 20)
        tops = 2.0 * M * N * K / us / 1e6
        sweep.append({"M": M, "us_per_call": round(us, 2), "int8_TOPs": round(tops, 1),
                      "int8_peak_frac": round(tops / INT8_PEAK_TOPS, 4)})
    out["dense_2048x2048_sweep"] = sweep
    return out


def bench_sym_layer(torch, w4, synth, args, dev, n=200):
    """The MoE layer in the paper's own format (Q4_SYM weights, Q8_F32
    activations; four launches) at one token, top-8 of 256 plus the shared
    expert, two weight sets alternated, replayed from a hipGraph."""
    g = synth.rng(args.seed + 13)
    sets = []
    for _ in range(2):
        sets.append([torch.from_numpy(synth.q4_sym_random_blocks(g, E * 2 * I, H)).to(dev),
                     torch.from_numpy(synth.q4_sym_random_blocks(g, E * H, I)).to(dev),
                     torch.from_numpy(synth.q4_sym_random_blocks(g, 2 * I, H)).to(dev),
                     torch.from_numpy(synth.q4_sym_random_blocks(g, H, I)).to(dev)])
    ids_all, wts_all = synth.routing(g, n, E, K_TOP)
    ids_d = torch.from_numpy(ids_all).to(dev).view(n, 1, K_TOP)
    wts_d = torch.from_numpy(wts_all).to(dev).view(n, 1, K_TOP)
    x = torch.from_numpy(synth.normal_f32(g, (n, 1, H))).to(dev)
    ws = w4.moe_sym_workspace(1, H, I, E, K_TOP, device=dev)
    out = torch.empty((1, H), dtype=torch.float32, device=dev)

    def step(i):
        L = sets[i % 2]
        w4.moe_sym_forward(x[i], ids_d[i], wts_d[i], L[0], L[1], L[2], L[3], H, I, E, K_TOP, ws,
                           out=out)

    for i in range(4):
        step(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n):
            step(i)
    graph.replay()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / n * 1e3
    expert = (2 * I * (H // 32) + H * (I // 32)) * 20
    nbytes = sum((len(set(r.tolist())) + 1) * expert for r in ids_all) / n
    del sets
    return {"T": 1, "us_per_layer": round(us, 2), "GBps": round(nbytes / us / 1e3, 1),
            "hbm_peak_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBPS, 4), "launch": "hipGraph"}


def bench_gdn(torch, w4, synth, args, dev):
    """The gated-delta-net recurrence of one linear-attention layer at the
    paper's head shape (32 value heads, dk = dv = 128) as a chunked scan:
    the 947-token prompt and a single decode token, each continuing a given
    state, replayed from a hipGraph."""
    out = {}
    for T, n in ((947, 20), (1, 200)):
        g = synth.rng(args.seed + 14 + T)
        q, k, v, gate, beta, s0 = synth.gdn_inputs(g, T, 32, 128, 128)
        d = [torch.from_numpy(a).to(dev) for a in (q, k, v, gate, beta, s0)]
        o = torch.empty((T, 32, 128), dtype=torch.float32, device=dev)
        s_out = torch.empty_like(d[5])
        ws = torch.empty(int(w4.lib().gdn_workspace_size(T, 32, 128, 128)), dtype=torch.uint8,
                         device=dev)
        for _ in range(3):
            w4.gdn_scan(*d, out=o, s_out=s_out, workspace=ws)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(n):
                w4.gdn_scan(*d, out=o, s_out=s_out, workspace=ws)
        graph.replay()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        graph.replay()
        ev1.record()
        torch.cuda.synchronize()
        us = ev0.elapsed_time(ev1) / n * 1e3
        out[f"T{T}"] = {"us_per_layer": round(us, 2), "tokens_per_s": round(T / us * 1e6, 1),
                        "heads": 32, "dk": 128, "dv": 128, "chunk": 32, "launch": "hipGraph"}
    return out


def bench_stack(torch, w4, synth, args, dev):
    """40 chained pre-norm residual layers (x <- x + MoE_l(RMSNorm_l(x)), one
    moe_w4a8_layer call each, the residual add and norm fused into the layer
    and, at one token, into its single decode launch): a 947-token prefill,
    then single-token decode steps through all layers; every layer has its own
    seed-generated weights (18.2 GB of Q4_0 resident in HBM), RMSNorm gains
    1 + N(0, 0.1^2) and its own routing per call."""
    nl, nd, Tp = args.stack_layers, args.stack_decode_steps, 947
    log(f"stack: generating {nl} layers of Q4_0 weights")
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 100)
    layers = [make_layer(torch, w4, gen, dev) for _ in range(nl)]
    gammas = [1.0 + 0.1 * torch.randn((H,), generator=gen, device=dev) for _ in range(nl)]
    rng = synth.rng(args.seed + 101)
    pre = [synth.routing(rng, Tp, E, K_TOP, bias_std=1.0) for _ in range(nl)]
    pre_ids = [torch.from_numpy(a).to(dev) for a, _ in pre]
    pre_wts = [torch.from_numpy(b).to(dev) for _, b in pre]
    dec_ids, dec_wts = synth.routing(rng, nd * nl, E, K_TOP)
    dec_ids = torch.from_numpy(dec_ids).to(dev).view(nd, nl, 1, K_TOP)
    dec_wts = torch.from_numpy(dec_wts).to(dev).view(nd, nl, 1, K_TOP)
    ws_p = w4.moe_workspace(Tp, H, I, E, K_TOP, device=dev)
    ws_d = w4.moe_workspace(1, H, I, E, K_TOP, device=dev)
    x_p0 = torch.randn((Tp, H), generator=gen, device=dev)
    x_d0 = torch.randn((nd, 1, H), generator=gen, device=dev)
    # residual stream and layer outputs ping-pong between two buffers each, so
    # no layer writes a buffer it reads
    xs_p = [torch.empty_like(x_p0) for _ in range(2)]
    ys_p = [torch.empty_like(x_p0) for _ in range(2)]
    xs_d = [torch.empty((1, H), device=dev) for _ in range(2)]
    ys_d = [torch.empty((1, H), device=dev) for _ in range(2)]

    def forward(xs, ys, ids, wts, ws):
        for l in range(nl):
            L = layers[l]
            w4.moe_layer(xs[l % 2], ys[(l + 1) % 2] if l else None, gammas[l], ids(l), wts(l),
                         L[0], L[1], L[2], L[3], H, I, E, K_TOP, ws,
                         x_out=xs[(l + 1) % 2], out=ys[l % 2])
        x = xs[nl % 2]
        w4.rmsnorm_residual(x, ys[(nl - 1) % 2], None, x_out=x, want_norm=False)
        return x

    def prefill():
        xs_p[0].copy_(x_p0)
        return forward(xs_p, ys_p, lambda l: pre_ids[l], lambda l: pre_wts[l], ws_p)

    def decode(s):
        xs_d[0].copy_(x_d0[s])
        return forward(xs_d, ys_d, lambda l: dec_ids[s, l], lambda l: dec_wts[s, l], ws_d)

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    prefill()
    torch.cuda.synchronize()
    ev0.record()
    x_p = prefill()
    ev1.record()
    torch.cuda.synchronize()
    ms_p = ev0.elapsed_time(ev1)
    decode(0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for s in range(nd):
            x_d = decode(s)
    graph.replay()
    torch.cuda.synchronize()
    ev0.record()
    graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms_d = ev0.elapsed_time(ev1) / nd

    # the same decode steps with the router in front of every layer: fresh
    # N(0,1) logits and a sigmoid gate on the shared expert per layer and step
    # (moe_w4a8_layer_routed: a router launch, then the layer's launch)
    dec_logits = torch.randn((nd, nl, 1, E), generator=gen, device=dev)
    dec_gate = torch.randn((nd, nl, 1), generator=gen, device=dev)
    r_ids = torch.empty((1, K_TOP), dtype=torch.int32, device=dev)
    r_wts = torch.empty((1, K_TOP), dtype=torch.float32, device=dev)

    def decode_routed(s):
        xs, ys = xs_d, ys_d
        xs[0].copy_(x_d0[s])
        for l in range(nl):
            L = layers[l]
            w4.moe_layer_routed(xs[l % 2], ys[(l + 1) % 2] if l else None, gammas[l],
                                dec_logits[s, l], L[0], L[1], L[2], L[3], H, I, E, K_TOP, ws_d,
                                shared_gate=dec_gate[s, l], x_out=xs[(l + 1) % 2],
                                out=ys[l % 2], topk_ids=r_ids, topk_w=r_wts)
        x = xs[nl % 2]
        w4.rmsnorm_residual(x, ys[(nl - 1) % 2], None, x_out=x, want_norm=False)
        return x

    decode_routed(0)
    torch.cuda.synchronize()
    graph_r = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph_r):
        for s in range(nd):
            x_r = decode_routed(s)
    graph_r.replay()
    torch.cuda.synchronize()
    ev0.record()
    graph_r.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms_r = ev0.elapsed_time(ev1) / nd
    assert torch.isfinite(x_r).all()
    ids_h = dec_ids.cpu().numpy().reshape(nd * nl, K_TOP)
    dbytes = sum(step_bytes(ids_h[i]) for i in range(nd * nl)) / nd
    assert torch.isfinite(x_p).all() and torch.isfinite(x_d).all()
    del layers
    return {"layers": nl, "weights_GB": round(nl * (E + 1) * EXPERT_BYTES / 1e9, 2),
            "prefill_tokens": Tp, "prefill_ms": round(ms_p, 3),
            "prefill_tokens_per_s": round(Tp / (ms_p / 1e3), 1),
            "decode_steps": nd, "decode_ms_per_token": round(ms_d, 4),
            "decode_tokens_per_s": round(1e3 / ms_d, 1),
            "decode_GBps": round(dbytes / (ms_d / 1e3) / 1e9, 1),
            "decode_routed_ms_per_token": round(ms_r, 4),
            "decode_routed_tokens_per_s": round(1e3 / ms_r, 1),
            "launch": "prefill eager; decode steps replayed from one HIP graph"}


def cpu_baseline(synth, seconds):
    """The oracle as it stands (plain C, scalar, fp64 accumulation) on this
    host's cores, for every workload: one thread, then one per physical core
    (OpenMP across tokens; the oracle takes a token's experts one after the
    other, so a single token runs on one core).  Expert weights are eight
    random experts' Q4_0 bytes tiled over the 256 (the time does not depend
    on the values).  `value` is the all-core decode rate of the headline
    workload, in the same algorithmic GB/s as the GPU figure.  The 40-layer
    stack is timed on two layers and extrapolated x20 (labelled)."""
    import numpy as np
    import oracle
    g = synth.rng(7)
    gu8 = synth.q4_0_random_blocks(g, 8 * 2 * I, H).reshape(8, 2 * I, -1)
    d8 = synth.q4_0_random_blocks(g, 8 * H, I).reshape(8, H, -1)
    w_gu = np.ascontiguousarray(np.tile(gu8, (E // 8, 1, 1)))
    w_d = np.ascontiguousarray(np.tile(d8, (E // 8, 1, 1)))
    s_gu, s_d = gu8[0].copy(), d8[0].copy()
    gamma = np.ones(H, np.float32)
    n_all = oracle.threads()

    def timed(fn, budget, min_reps=1):
        reps, t = 0, 0.0
        while reps < min_reps or t < budget:
            t0 = time.perf_counter()
            fn()
            t += time.perf_counter() - t0
            reps += 1
        return t / reps, reps

    def moe(x, ids, wts):
        oracle.moe(x, ids, wts, w_gu, w_d, s_gu, s_d, H, I, E, K_TOP, want_intermediates=False)

    res = {}
    for label, nt in (("1_thread", 1), ("all_cores", n_all)):
        oracle.set_threads(nt)
        r = {}
        # C1: the 1024 x 1024 GEMV
        W = synth.q4_0_random_blocks(g, 1024, 1024)
        xq = oracle.q8_0_quantize(synth.normal_f32(g, (1, 1024)))
        t, n = timed(lambda: oracle.gemv(W, xq, 1024, 1024), 0.5, 3)
        nb = 1024 * 32 * 18 + 32 * 34 + 1024 * 4
        r["gemv_1024"] = {"us_per_call": round(t * 1e6, 1), "GBps": round(nb / t / 1e9, 3),
                          "calls": n}
        # C2: single-token decode layer, latency; all cores: throughput over
        # independent tokens (the headline value)
        x = synth.normal_f32(g, (1, H))
        ids, wts = synth.routing(g, 1, E, K_TOP)
        t, n = timed(lambda: moe(x, ids, wts), 1.0, 2)
        r["decode_m1"] = {"ms_per_step": round(t * 1e3, 2),
                          "GBps": round(step_bytes(ids[0]) / t / 1e9, 3), "steps": n}
        if nt > 1:
            batch = 2 * nt
            done_t, done_b, used = 0, 0, 0.0
            while used < seconds:
                xb = synth.normal_f32(g, (batch, H))
                ib, wb = synth.routing(g, batch, E, K_TOP)
                t0 = time.perf_counter()
                moe(xb, ib, wb)
                used += time.perf_counter() - t0
                done_t += batch
                done_b += sum(step_bytes(ib[t_]) for t_ in range(batch))
            r["decode_m1_throughput"] = {"GBps": round(done_b / used / 1e9, 3),
                                         "tokens_per_s": round(done_t / used, 1),
                                         "steps": done_t, "seconds": round(used, 1)}
        # C3: the 32-token batched decode layer
        x = synth.normal_f32(g, (32, H))
        ids, wts = synth.routing(g, 32, E, K_TOP)
        t, n = timed(lambda: moe(x, ids, wts), 1.0)
        r["decode_m32"] = {"ms_per_layer": round(t * 1e3, 2),
                           "tokens_per_s": round(32 / t, 1), "calls": n}
        # C4: the 947-token prefill layer (biased routing); on one thread a
        # sample of 24 of its tokens (the oracle's time is per token)
        Tp = 947 if nt > 1 else 24
        x = synth.normal_f32(g, (947, H))
        ids, wts = synth.routing(g, 947, E, K_TOP, bias_std=1.0)
        t, n = timed(lambda: moe(x[:Tp], ids[:Tp], wts[:Tp]), 0.5)
        r["prefill_947"] = {"tokens_timed": Tp, "tokens_per_s": round(Tp / t, 1),
                            "ms_per_layer": round(947 / (Tp / t) * 1e3, 1),
                            "extrapolated_from_sample": Tp != 947}
        # C5: two chained layers (residual add + RMSNorm + layer), x20
        Tp5 = 947 if nt > 1 else 24
        t0 = time.perf_counter()
        xs, y = x[:Tp5], None
        for _ in range(2):
            xs, xn = oracle.rmsnorm_residual(xs, y, gamma)
            y = oracle.moe(xn.astype(np.float32), ids[:Tp5], wts[:Tp5], w_gu, w_d, s_gu, s_d, H,
                           I, E, K_TOP, want_intermediates=False).out.astype(np.float32)
        t_pre = (time.perf_counter() - t0) * 20 * 947 / Tp5
        ids1, wts1 = synth.routing(g, 4, E, K_TOP)
        t0 = time.perf_counter()
        for s_ in range(2):                      # two decode steps through two layers
            xs, y = synth.normal_f32(g, (1, H)), None
            for l in range(2):
                xs, xn = oracle.rmsnorm_residual(xs, y, gamma)
                y = oracle.moe(xn.astype(np.float32), ids1[2 * s_ + l:2 * s_ + l + 1],
                               wts1[2 * s_ + l:2 * s_ + l + 1], w_gu, w_d, s_gu, s_d, H, I, E,
                               K_TOP, want_intermediates=False).out.astype(np.float32)
        t_dec = (time.perf_counter() - t0) / 2 * 20
        r["stack_40_extrapolated"] = {"prefill_947_s": round(t_pre, 2),
                                      "decode_ms_per_token": round(t_dec * 1e3, 1),
                                      "decode_tokens_per_s": round(1.0 / t_dec, 2),
                                      "note": "two layers timed, x20; prefill on one thread "
                                              "from a 24-token sample" if nt == 1 else
                                              "two layers timed, x20"}
        res[label] = r
    oracle.set_threads(n_all)
    # the GDN recurrence's oracle (numpy fp64, one token at a time, all 32
    # heads at once): a 64-token sample of the 947-token prompt, scaled
    from oracle.gdn import gdn_recurrent
    q, k, v, gate, beta, s0 = synth.gdn_inputs(g, 64, 32, 128, 128)
    t, n = timed(lambda: gdn_recurrent(q, k, v, gate, beta, s0), 0.5)
    res["gdn_recurrence_numpy"] = {"tokens_timed": 64, "tokens_per_s": round(64 / t, 1),
                                   "ms_per_layer_947": round(947 / (64 / t) * 1e3, 1),
                                   "extrapolated_from_sample": True}
    main = res["all_cores"]["decode_m1_throughput"]
    return {"value": main["GBps"], "unit": "GB/s", "cores": n_all, "kind": "oracle",
            "sample": f"{main['steps']} independent M=1 decode steps of the same layer shape "
                      f"(256+1 experts, top-8), {main['seconds']} s, OpenMP across tokens on "
                      f"{n_all} threads ({HOST['physical_cores']} physical cores on this host, "
                      f"OMP_PROC_BIND=close, NUMA {HOST['numa_policy']} over "
                      f"{HOST['numa_nodes']} node(s)); per-workload single-thread and all-core "
                      f"times under 'configs'",
            "configs": res, "host": HOST}


def hbm_copy_rate(torch, dev, nbytes=2 << 30, reps=10):
    """Practical HBM rate on this machine: a plain device-to-device copy of 2 GiB
    (bytes read plus bytes written over time), beside the 8 TB/s
    specification.  A measured reference, not a ceiling: the read-only GEMV
    at the output projection's shape streams faster (a reduction such as
    torch.sum reads at only about 4 TB/s here)."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(reps):
        dst.copy_(src)
    ev1.record()
    torch.cuda.synchronize()
    s = ev0.elapsed_time(ev1) / reps / 1e3
    del src, dst
    return {"GBps": round(2 * nbytes / s / 1e9, 1), "kernel": "device copy of 2 GiB (read + write)",
            "frac_of_spec": round(2 * nbytes / s / 1e9 / HBM_PEAK_GBPS, 4)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the library runs "
              "a layer on a single MI355X and has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2606_24031_amd as w4
    from paper_2606_24031_amd import synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.section:
        fn = {"gemm": bench_gemm, "sym_layer": bench_sym_layer, "gdn": bench_gdn}[args.section]
        print(json.dumps({args.section: fn(torch, w4, synth, args, dev)}), flush=True)
        return

    log(f"generating {args.layers} layers of Q4_0 weights on the GPU")
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    layers = [make_layer(torch, w4, gen, dev) for _ in range(args.layers)]
    torch.cuda.synchronize()

    ms, nbytes = bench_decode(torch, w4, synth, layers, args, dev)
    ms_step = ms / args.steps
    gbps = nbytes / (ms / 1e3) / 1e9
    bytes_per_launch = nbytes / args.steps
    log(f"decode: {ms_step * 1e3:.2f} us/step, {gbps:.0f} GB/s")

    if args.calibrate_copy:
        src = torch.randint(0, 255, (256 << 20,), dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: 5 copies of {256 << 20} bytes")

    prefill = None
    if not args.no_prefill:
        prefill = bench_prefill(torch, w4, synth, layers, args, dev)
        log(f"prefill: {prefill}")

    prefill_5k = one_expert = None
    if not args.no_prefill and not args.no_extras:
        prefill_5k = bench_prefill(torch, w4, synth, layers, args, dev, T=5120, n=4)
        log(f"prefill 5120: {prefill_5k}")
        one_expert = bench_one_expert(torch, w4, synth, args, dev)
        log(f"one expert, 947 rows: {one_expert}")

    m32 = batch_sweep = None
    if not args.no_m32:
        m32 = bench_m32(torch, w4, synth, layers, args, dev)
        log(f"decode M=32: {m32}")
        if not args.no_extras:
            # batches on either side of the switch from the small-group VALU
            # kernels (up to 128 tokens) to the MFMA tiles
            batch_sweep = [bench_m32(torch, w4, synth, layers, args, dev, T=t, n=16)
                           for t in (64, 128, 129, 256)]
            log(f"batch sweep: {batch_sweep}")

    invariants = router = lm_head = gemv_1024 = gemv_sym = gemm = sym_layer = gdn = None
    if not args.no_extras:
        invariants = bench_decode_invariants(torch, w4, synth, layers, args, dev)
        log(f"decode invariants: {invariants}")
        router = bench_router(torch, w4, synth, args, dev)
        log(f"router top-k: {router}")
        lm_head = bench_lm_head(torch, w4, synth, args, dev)
        log(f"lm-head gemv: {lm_head}")
        gemv_1024 = bench_gemv_1024(torch, w4, synth, args, dev)
        log(f"gemv 1024x1024: {gemv_1024}")
        gemv_sym = bench_gemv_sym(torch, w4, synth, args, dev)
        log(f"gemv, paper's fp32-scale format: {gemv_sym}")
        gemm = bench_gemm(torch, w4, synth, args, dev)
        log(f"dense gemm: {gemm}")
        sym_layer = bench_sym_layer(torch, w4, synth, args, dev)
        log(f"layer in the paper's format: {sym_layer}")
        gdn = bench_gdn(torch, w4, synth, args, dev)
        log(f"GDN recurrence, chunked scan: {gdn}")

    stack = None
    if not args.no_stack:
        del layers
        torch.cuda.empty_cache()
        stack = bench_stack(torch, w4, synth, args, dev)
        log(f"stack: {stack}")

    cpu = None
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle for ~{args.cpu_seconds:.0f} s")
        cpu = cpu_baseline(synth, args.cpu_seconds)
        log(f"cpu baseline: {cpu}")

    traffic = measured_traffic()
    copy_rate = hbm_copy_rate(torch, dev)
    log(f"hbm copy rate: {copy_rate}")
    rec = {
        "metric": METRIC,
        "value": round(gbps, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "moe_layer_decode_m1", "T": 1, "hidden": H, "expert_intermediate": I,
                   "routed_experts": E, "top_k": K_TOP, "shared_experts": 1,
                   "weight_sets_cycled": args.layers,
                   "launch": "eager" if args.no_graph else "hipGraph",
                   "bytes_per_step": round(bytes_per_launch)},
        "roofline": {"bound": "hbm", "kernel": "decode_kernel (whole layer, one launch per step)",
                     "achieved": round(bytes_per_launch / (ms_step / 1e3) / 1e9, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(bytes_per_launch / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
        "cpu_baseline": cpu,
        "hbm_copy_rate": dict(copy_rate, decode_frac_of_copy_rate=round(gbps / copy_rate["GBps"], 4)),
        "prefill_947": prefill,
        "prefill_5120": prefill_5k,
        "one_expert_947_rows": one_expert,
        "decode_m32": m32,
        "batch_sweep": batch_sweep,
        "stack_40": stack,
        "decode_invariants": invariants,
        "router_topk": router,
        "gemv_lm_head": lm_head,
        "gemv_1024": gemv_1024,
        "gemv_lm_head_paper_format": gemv_sym,
        "gemm": gemm,
        "moe_layer_paper_format_m1": sym_layer,
        "gdn_recurrence": gdn,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
