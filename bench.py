"""Benchmark: batched paged GQA decode attention on one MI355X.

One step = one call of the whole path (plan, decode, combine kernels) over one
batch: every request of the batch decodes one token through one attention
layer. The default workload is the largest one-GPU configuration, the
Llama-3.1-70B layer shape (64 q heads, 8 kv heads, head_dim 128, block 16),
batch 512, lengths uniform in [256, 4096] (the paper's 70B setting, Sec. 5.1,
with code-generation-like lengths), shuffled physical blocks, bf16 q/K/V
~ N(0,1) (synthetic, seeded): 4.6 GB of KV per call. `--config 1..6` picks
the other workloads.

Inputs are resident in HBM before timing. The KV cache is replicated (at least
two copies, rotated, and at least 4x the 256 MB Infinity Cache in total) so that
consecutive steps never find their data in that cache; a third pass also
times each call alone after 1 GiB of other data is read. Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--config N] [--variant auto|valu|mfma]
    python bench.py --copy-calibration     # plain copy of known size, for rocprofv3 --pmc
    python bench.py --op kv_swap_out|kv_swap_in|kv_copy_d2d|kv_append   # cache operations
    python bench.py --op cpu_decode [--cpu-threads N] [--cpu-isa ...]   # host-CPU attention
    python bench.py --op profile_costs [--out F]   # T_ga / T_ca grids for the cost model
    python bench.py --op schedule_sim [--costs F]  # load-aware scheduler vs GPU-only, simulated
    python bench.py --op overlap_demo              # asymmetric pipelining, measured on the box
    python bench.py --op read_ceiling              # the device's streaming-read rate (4 GiB)
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, published
PEAK_PCIE_GBS = 64.0           # PCIe 5.0 x16 host link, one direction (32 GT/s x 16 lanes)
MALL_BYTES = 256 * 2 ** 20     # Infinity Cache
METRIC = "decode-attention achieved HBM GB/s (% of peak) + tokens/sec per layer, 1 GPU"
KERNEL_SOURCES = ("decode_mfma.hip", "decode_valu.hip", "decode_common.h", "neo_internal.h")
SEQ_DESC = {1: "U[64,512]", 2: "U[512,2048]", 3: "lognormal(median 1500, sigma 0.6) clip [128,8192]",
            4: "U[256,4096]", 5: "8 x 32768 + 1016 x U[16,256]",
            6: "U[256,4096] (one GPU's share of the 70B layer at 8-way tensor parallelism)"}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def pct(values, qs):
    """Percentiles (nearest rank) of a list of numbers."""
    xs = sorted(values)
    return [xs[min(len(xs) - 1, max(0, math.ceil(q / 100 * len(xs)) - 1))] for q in qs]


def kernel_source_sha(variant: str) -> str:
    from paper_2411_01142_amd import _build
    h = hashlib.sha256()
    # The source's own compiler flags (none for most) are part of the kernel.
    h.update(" ".join(_build.HIPCC_SOURCE_FLAGS.get(f"decode_{variant.split('_')[0]}.hip",
                                                    [])).encode())
    for name in KERNEL_SOURCES:
        if name.startswith("decode_") and name != "decode_common.h" and \
                name != f"decode_{variant.split('_')[0]}.hip":
            continue
        with open(os.path.join(ROOT, "paper_2411_01142_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(workload_key: str, variant: str, launches_per_step: int = 1,
                 reads_only: bool = False):
    """HBM bytes per decode launch (read + written, or read only) from committed
    rocprofv3 --pmc summaries, or None when they are missing or were taken on
    different kernel sources."""
    path = os.path.join(ROOT, "profiles", f"counters__decode_{variant}__{workload_key}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"TRAFFIC_JSON:\s*(\{.*\})", open(path).read())
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("kernel_sha") != kernel_source_sha(variant):
        return None
    if reads_only:
        return float(rec["fetch_kib_per_launch"]) * 1024 * float(rec["copy_factor_fetch"])
    return float(rec["traffic_bytes_per_launch"])


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch loaded (same soname)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so.7")
        self.lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                                     ctypes.c_uint]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    # Timing events without the system-scope release at record time: cheaper,
    # so the interval they bracket is closer to the kernel's own duration.
    FLAGS = 0x20000000  # hipEventDisableSystemFence

    def create(self):
        ev = ctypes.c_void_p()
        rc = self.lib.hipEventCreateWithFlags(ctypes.byref(ev), self.FLAGS)
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed: {rc}")
        return ev

    def elapsed_ms(self, a, b) -> float:
        ms = ctypes.c_float()
        rc = self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return float(ms.value)

    def record(self, ev, stream):
        rc = self.lib.hipEventRecord(ev, stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed: {rc}")

    def destroy(self, ev):
        self.lib.hipEventDestroy(ev)


def cpu_baseline(case, min_seconds: float = 10.0):
    """The fp64 oracle on the host cores over the whole batch, repeated until
    ``min_seconds`` have passed; same units as the GPU figure."""
    import numpy as np

    import oracle
    threads = oracle.max_threads()
    passes, t0 = 0, time.perf_counter()
    while True:
        oracle.decode_attention(case, threads=0)
        passes += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    gbs = case.algorithmic_bytes() * passes / el / 1e9
    # One thread over the first requests (a bounded sample: ~3 s).
    nreq = min(case.batch, 8)
    L = np.maximum(case.seq_lens[:nreq].astype(np.int64), 0)
    sample_bytes = (int(L.sum()) * case.num_kv_heads * case.head_dim * 4 +
                    nreq * case.num_q_heads * case.head_dim * 6 +
                    4 * int(((L + case.block_size - 1) // case.block_size).sum()) + 4 * nreq)
    passes1, t1 = 0, time.perf_counter()
    while True:
        oracle.decode_attention(case, rows=(0, nreq * case.num_q_heads), threads=1)
        passes1 += 1
        el1 = time.perf_counter() - t1
        if el1 >= min(3.0, min_seconds):
            break
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"full batch ({case.batch} requests x {case.num_q_heads} heads), "
                      f"{passes} pass(es) in {el:.1f} s, fp64 naive softmax, OpenMP",
            "tokens_per_s_per_layer": round(case.batch * passes / el, 2),
            "single_thread": {"value": round(sample_bytes * passes1 / el1 / 1e9, 4),
                              "unit": "GB/s", "cores": 1,
                              "sample": f"first {nreq} requests, {passes1} pass(es) in "
                                        f"{el1:.1f} s"}}


def copy_calibration(nbytes: int = 2 ** 30, reps: int = 5):
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "reps": reps}), flush=True)


def bench_kv_op(args, torch, neo, W):
    """Cache operations on the workload's KV: swap every in-use block out to a
    pinned host cache (kv_swap_out), back in (kv_swap_in), between two device
    caches (kv_copy_d2d), or append one token per request (kv_append). Each is
    one kernel on the current stream; a plain DMA copy of the same byte count
    (hipMemcpyAsync through torch) is timed beside the swaps for reference."""
    seed = args.config if args.seed is None else args.seed
    case = W.make_config(args.config, seed, poison=False)
    q, k, v, bt, sl = case.to_torch("cuda")
    used = sorted({int(x) for b, L in enumerate(case.seq_lens.tolist())
                   for x in case.block_table[b, :(L + 15) // 16]})
    n = len(used)
    ids = torch.tensor(used, dtype=torch.int32, device="cuda")
    seq = torch.arange(n, dtype=torch.int32, device="cuda")
    blk_bytes = 2 * case.num_kv_heads * 2048 * 2  # K and V of one block, all kv heads
    hip = HipEvents()
    sh = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    dma = None
    if args.op in ("kv_swap_out", "kv_swap_in", "kv_copy_d2d"):
        pinned = args.op != "kv_copy_d2d"
        shape_k, shape_v = (n,) + tuple(k.shape[1:]), (n,) + tuple(v.shape[1:])
        if pinned:
            ok_ = torch.empty(shape_k, dtype=torch.bfloat16, pin_memory=True)
            ov = torch.empty(shape_v, dtype=torch.bfloat16, pin_memory=True)
        else:
            ok_ = torch.empty(shape_k, dtype=torch.bfloat16, device="cuda")
            ov = torch.empty(shape_v, dtype=torch.bfloat16, device="cuda")
        if args.op == "kv_swap_in":
            neo.copy_blocks(k, v, ok_, ov, ids, seq)
            torch.cuda.synchronize()

            def one():
                neo.copy_blocks(ok_, ov, k, v, seq, ids)
        else:
            def one():
                neo.copy_blocks(k, v, ok_, ov, ids, seq)
        nbytes = n * blk_bytes
        bytes_per_call = 2 * nbytes  # read + write
        link_bytes = nbytes
        if pinned:
            dk = k[:n].contiguous() if args.op == "kv_swap_in" else k[:n]
            dv = v[:n].contiguous() if args.op == "kv_swap_in" else v[:n]

            def dma_one():
                if args.op == "kv_swap_out":
                    ok_.copy_(dk, non_blocking=True)
                    ov.copy_(dv, non_blocking=True)
                else:
                    dk.copy_(ok_, non_blocking=True)
                    dv.copy_(ov, non_blocking=True)
            dma = dma_one
    elif args.op == "kv_append":
        rng = __import__("numpy").random.default_rng(seed)
        shape = (case.batch, case.num_kv_heads, case.head_dim)
        kn = torch.from_numpy(rng.integers(0, 1 << 16, size=shape, dtype="uint16").view(
            "int16")).to("cuda").view(torch.bfloat16)
        vn = kn.clone()

        def one():
            neo.kv_append(k, v, kn, vn, bt, sl)
        nbytes = 2 * kn.numel() * 2
        bytes_per_call = 2 * nbytes + 4 * case.batch * 2
        link_bytes = None
    else:
        raise SystemExit(f"unknown --op {args.op}")

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        a, b = hip.create(), hip.create()
        hip.record(a, sh)
        for _ in range(args.steps):
            fn()
        hip.record(b, sh)
        torch.cuda.synchronize()
        ms = hip.elapsed_ms(a, b) / args.steps
        hip.destroy(a)
        hip.destroy(b)
        return ms

    def per_call(fn):
        """Mean GPU time of one call from an event pair around each call."""
        evs = [(hip.create(), hip.create()) for _ in range(args.steps)]
        for a, b in evs:
            hip.record(a, sh)
            fn()
            hip.record(b, sh)
        torch.cuda.synchronize()
        ms = sum(hip.elapsed_ms(a, b) for a, b in evs) / len(evs)
        for a, b in evs:
            hip.destroy(a)
            hip.destroy(b)
        return ms

    log(f"[bench] {args.op} on {case.name}: {n} blocks in use, {nbytes / 1e6:.1f} MB per call")
    ms = timed(one)
    kernel_ms = per_call(one)
    result = {
        "metric": f"{args.op} GB/s",
        "op": args.op,
        "value": round((link_bytes or bytes_per_call) / (ms * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "us_per_call": round(ms * 1e3, 3),
        "kernel_us": round(kernel_ms * 1e3, 3),
        "bytes_per_call": bytes_per_call,
        "config": {"workload": f"{case.name}: KV of {case.batch} requests, "
                               f"{case.num_kv_heads} kv heads, {n} blocks"},
        "steps": args.steps, "warmup": args.warmup,
    }
    if link_bytes is not None:
        result["roofline"] = {"bound": "pcie", "achieved": result["value"],
                              "peak": PEAK_PCIE_GBS, "unit": "GB/s",
                              "frac": round(result["value"] / PEAK_PCIE_GBS, 4)}
        if args.op == "kv_copy_d2d":
            hbm = bytes_per_call / (ms * 1e-3) / 1e9
            result["roofline"] = {"bound": "hbm", "achieved": round(hbm, 2),
                                  "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                  "frac": round(hbm / PEAK_HBM_GBS, 4)}
            result["value"] = round(hbm, 2)
    if dma is not None:
        dms = timed(dma)
        result["dma_reference"] = {"what": "hipMemcpyAsync of the same bytes, contiguous",
                                   "GBs": round(nbytes / (dms * 1e-3) / 1e9, 2),
                                   "us_per_call": round(dms * 1e3, 3)}
    print(json.dumps(result), flush=True)
    return 0


def bench_read_ceiling(args, torch, neo):
    """The device's read rate over 4 GiB with two probes: the strided probe
    (every thread 16 bytes, 8 loads in flight, the whole grid sweeping the
    buffer), nontemporal and plain loads; and the tile probe, the decode
    kernel's own pattern without its arithmetic (contiguous 8 KiB steps per
    wave through 4 KiB buffer resources, nontemporal), over a sweep of waves per
    compute unit and steps in flight, with equal per-wave ranges and with
    ranges weighted by XCD. Each configuration is timed two ways: its
    calls back to back between two events (as the decode benchmark's timed
    region runs), and one call at a time with the device idle in between (the
    median of those). The best back-to-back rate is the measured read ceiling:
    the one-at-a-time intervals also hold the dispatch latency of a kernel
    launched onto an idle stream (25-30 us), which back-to-back calls hide."""
    nbytes = 4 << 30
    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    sink = torch.empty(neo.READ_PROBE_SINK_WORDS, dtype=torch.int32, device="cuda")
    hip = HipEvents()
    sh = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    reps = max(args.steps // 10, 5)

    def back_to_back(fn):
        for _ in range(2):
            fn()
        a, b = hip.create(), hip.create()
        hip.record(a, sh)
        for _ in range(2 * reps):
            fn()
        hip.record(b, sh)
        torch.cuda.synchronize()
        ms = hip.elapsed_ms(a, b) / (2 * reps)
        hip.destroy(a)
        hip.destroy(b)
        return round(nbytes / (ms * 1e-3) / 1e9, 1)

    def rate(fn):
        for _ in range(2):
            fn()
        ms = []
        for _ in range(reps):
            a, b = hip.create(), hip.create()
            hip.record(a, sh)
            fn()
            hip.record(b, sh)
            torch.cuda.synchronize()
            ms.append(hip.elapsed_ms(a, b))
            hip.destroy(a)
            hip.destroy(b)
        return [round(nbytes / (m * 1e-3) / 1e9, 1) for m in ms]
    rates, b2b = {}, {}
    for nt in (True, False):
        key = "strided_" + ("nontemporal" if nt else "plain")
        rates[key] = rate(lambda: neo.read_probe(src, sink, nontemporal=nt))
        b2b[key] = back_to_back(lambda: neo.read_probe(src, sink, nontemporal=nt))
    # Waves per CU that the kernel's registers allow at each depth (51, 107,
    # 144 and 175 VGPRs: 8, 4, 3 and 2 waves per SIMD).
    fits = {1: (4, 8, 12, 16), 2: (4, 8, 12, 16), 3: (4, 8, 12), 4: (4, 8)}
    # Each with equal per-wave ranges and with ranges weighted by XCD as the
    # decode kernel weighs its slices (suffix _xcd): waves on odd-numbered XCDs
    # read more slowly, so equal ranges end when those do.
    configs = [(w, d, c) for w in (False, True) for d, cs in fits.items() for c in cs]
    for weighted, depth, wpc in configs:
        key = f"tiles_w{wpc}_d{depth}" + ("_xcd" if weighted else "")

        def fn(wpc=wpc, depth=depth, weighted=weighted):
            neo.read_probe_tiles(src, sink, waves_per_cu=wpc, depth=depth, xcd_weighted=weighted)
        b2b[key] = back_to_back(fn)
        rates[key] = rate(fn)
        log(f"[bench] tile probe {key}: back to back {b2b[key]} GB/s, "
            f"one call at a time {pct(rates[key], (50,))[0]} GB/s (median)")
    med = {k: pct(v, (50,))[0] for k, v in rates.items()}
    best_key = max(b2b, key=b2b.get)
    print(json.dumps({
        "metric": "device read rate (measured read ceiling for HBM-bound kernels)",
        "value": b2b[best_key], "unit": "GB/s", "n_gpus": 1, "higher_is_better": True,
        "bytes": nbytes, "best_pattern": best_key,
        "decode_pattern_gbs": b2b["tiles_w4_d1_xcd"], "back_to_back_gbs": b2b,
        "single_call_median_gbs": med, "single_call_runs_gbs": rates,
        "roofline": {"bound": "hbm", "achieved": b2b[best_key], "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(b2b[best_key] / PEAK_HBM_GBS, 4)},
    }), flush=True)
    return 0


def bench_cpu_decode(args, neo, W):
    """Decode attention on the host CPU over the workload's KV in host memory,
    against the host's measured read ceiling (the library's read probe over a
    buffer twice the cache size, same thread count)."""
    import numpy as np
    seed = args.config if args.seed is None else args.seed
    case = W.make_config(args.config, seed, poison=False)
    threads = args.cpu_threads or neo.cpu_default_threads()
    isa = neo.cpu_best_isa() if args.cpu_isa == "auto" else args.cpu_isa
    out = np.empty((case.batch, case.num_q_heads, case.head_dim), np.float32)

    def one():
        neo.cpu_decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                 case.seq_lens, case.scale, out, num_threads=threads, isa=isa)
    log(f"[bench] cpu_decode {case.name}: {threads} threads, isa {isa}")
    for _ in range(max(1, args.warmup)):
        one()
    times = []
    for _ in range(args.steps):
        t0 = time.perf_counter()
        one()
        times.append(time.perf_counter() - t0)
    times.sort()
    med = times[len(times) // 2]
    alg = case.algorithmic_bytes()
    gbs = alg / med / 1e9
    probe = np.ones(max(2 * (case.k_cache.nbytes + case.v_cache.nbytes), 1 << 30) // 4,
                    np.float32)
    neo.cpu_read_probe(probe, threads)
    pt = []
    for _ in range(5):
        t0 = time.perf_counter()
        neo.cpu_read_probe(probe, threads)
        pt.append(time.perf_counter() - t0)
    ceiling = probe.nbytes / sorted(pt)[2] / 1e9
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    result = {
        "metric": "cpu decode-attention achieved host-memory GB/s",
        "op": "cpu_decode",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "ms_per_call": round(med * 1e3, 3),
        "p10_ms": round(times[len(times) // 10] * 1e3, 3),
        "p90_ms": round(times[(len(times) * 9) // 10] * 1e3, 3),
        "tokens_per_s_per_layer": round(case.batch / med, 1),
        "steps": args.steps, "warmup": args.warmup,
        "dtype": "bf16", "accumulate": "fp32",
        "config": {"workload": f"{case.name}: decode attention on the host CPU, "
                               f"{case.num_q_heads}/{case.num_kv_heads} heads, batch "
                               f"{case.batch}, seq_lens {SEQ_DESC[args.config]}",
                   "threads": threads, "isa": isa, "cpu": cpu_model},
        "roofline": {"bound": "host-dram", "achieved": round(gbs, 2),
                     "peak": round(ceiling, 2), "unit": "GB/s",
                     "frac": round(gbs / ceiling, 4),
                     "peak_kind": "measured read ceiling (library read probe, same threads)"},
    }
    print(json.dumps(result), flush=True)
    return 0


COST_AXES = {"b": [1, 4, 16, 64, 256, 1024], "s": [2048, 16384, 131072, 524288]}
COST_SHAPE = {"num_q_heads": 32, "num_kv_heads": 8, "head_dim": 128, "block_size": 16}
DEFAULT_COSTS = os.path.join(ROOT, "paper_2411_01142_amd", "cost_profiles",
                             "mi355x_epyc16__llama3-8b_attention.json")


def bench_profile_costs(args, torch, neo):
    """Per-layer decode-attention time of the GPU path (T_ga) and of the CPU path
    (T_ca) on a grid of (requests, total context tokens): the offline profile of
    the cost model (Sec. 3.2). Each point is a batch of equal-length requests
    over shuffled blocks of one pool of N(0,1) bf16 K/V."""
    import numpy as np
    hq, hkv, D, bs = (COST_SHAPE[k] for k in ("num_q_heads", "num_kv_heads", "head_dim",
                                               "block_size"))
    B_axis, S_axis = COST_AXES["b"], COST_AXES["s"]
    nb_pool = max(S_axis) // bs + max(B_axis)
    log(f"[bench] cost profile: pool {nb_pool} blocks, grid {len(B_axis)} x {len(S_axis)}")
    gen = torch.Generator(device="cuda").manual_seed(7)
    k = torch.randn((nb_pool, hkv, D // 8, bs, 8), generator=gen, device="cuda").to(torch.bfloat16)
    v = torch.randn((nb_pool, hkv, D, bs), generator=gen, device="cuda").to(torch.bfloat16)
    k_host = k.view(torch.int16).cpu().numpy().view(np.uint16)
    v_host = v.view(torch.int16).cpu().numpy().view(np.uint16)
    perm = np.random.default_rng(7).permutation(nb_pool).astype(np.int32)
    threads = args.cpu_threads or neo.cpu_default_threads()
    hip = HipEvents()
    sh = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    gpu_t, cpu_t = [], []
    for B in B_axis:
        grow, crow = [], []
        for S in S_axis:
            lens = np.full(B, S // B, np.int32)
            lens[: S % B] += 1
            nbs = (lens + bs - 1) // bs
            mbps = int(nbs.max())
            table = np.full((B, mbps), -1, np.int32)
            o = 0
            for b in range(B):
                table[b, : nbs[b]] = perm[o: o + nbs[b]]
                o += nbs[b]
            q = torch.randn((B, hq, D), generator=gen, device="cuda").to(torch.bfloat16)
            bt = torch.from_numpy(table).to("cuda")
            sl = torch.from_numpy(lens).to("cuda")
            ws = neo.new_workspace(B, hq, hkv)
            out = torch.empty((B, hq, D), dtype=torch.float32, device="cuda")
            for _ in range(3):
                neo.decode_attention(q, k, v, bt, sl, out=out, workspace=ws)
            torch.cuda.synchronize()
            a, e = hip.create(), hip.create()
            reps = 20
            hip.record(a, sh)
            for _ in range(reps):
                neo.decode_attention(q, k, v, bt, sl, out=out, workspace=ws)
            hip.record(e, sh)
            torch.cuda.synchronize()
            grow.append(hip.elapsed_ms(a, e) / reps * 1e-3)
            hip.destroy(a)
            hip.destroy(e)
            qh = q.view(torch.int16).cpu().numpy().view(np.uint16)
            oh = np.empty((B, hq, D), np.float32)
            neo.cpu_decode_attention(qh, k_host, v_host, table, lens, out=oh, num_threads=threads)
            ts = []
            for _ in range(5):
                t0 = time.perf_counter()
                neo.cpu_decode_attention(qh, k_host, v_host, table, lens, out=oh,
                                         num_threads=threads)
                ts.append(time.perf_counter() - t0)
            crow.append(sorted(ts)[2])
            log(f"[bench]   B={B} S={S}: T_ga {grow[-1] * 1e6:.1f} us, T_ca {crow[-1] * 1e6:.1f} us")
        gpu_t.append(grow)
        cpu_t.append(crow)
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    prof = {"what": "per-layer decode-attention seconds, GPU path (t_ga) and CPU path (t_ca), "
                    "on a grid of (requests b, total context tokens s); equal-length requests",
            "shape": COST_SHAPE, "b": B_axis, "s": S_axis, "t_ga": gpu_t, "t_ca": cpu_t,
            "gpu": torch.cuda.get_device_name(0), "cpu": cpu_model, "cpu_threads": threads,
            "cpu_isa": neo.cpu_best_isa(), "command": "python3 bench.py --op profile_costs"}
    if args.out:
        with open(args.out, "w") as f:
            json.dump(prof, f, indent=1)
    print(json.dumps({"metric": "cost profile", "op": "profile_costs", **prof}), flush=True)
    return 0


def bench_schedule_sim(args):
    """The load-aware scheduler against GPU-only scheduling, simulated over a
    synthetic request mix with the measured attention costs (T_ga, T_ca) and a
    synthetic linear stage for a Llama-3-8B-shaped layer on MI355X
    (max(436 MB of weights / 6 TB/s, 2 x 218 M params x tokens / 1.75 PFLOP/s))."""
    import random
    from paper_2411_01142_amd import sched as S
    with open(args.costs or DEFAULT_COSTS) as f:
        prof = json.load(f)
    ga = S.CostGrid(prof["b"], prof["s"], prof["t_ga"])
    ca = S.CostGrid(prof["b"], prof["s"], prof["t_ca"])
    xs = [1.0, 64.0, 256.0, 1024.0, 8192.0]
    tl = S.CostCurve(xs, [max(436e6 / 6e12, 2 * 218e6 * x / 1.75e15) for x in xs])
    rng = random.Random(args.seed or 0)
    reqs = [(i, rng.randint(64, 2048), rng.randint(16, 512)) for i in range(2000)]
    results = {}
    # GPU KV cache for 16 K tokens per layer-set (a memory-bound regime) and a
    # CPU cache 16x larger; the GPU-only baseline preempts instead of swapping.
    for policy, cpu_blocks in (("neo", 16384), ("gpu_only", 0)):
        sc = S.Scheduler(S.SchedConfig(num_layers=32, block_size=16, gpu_blocks=1024,
                                       cpu_blocks=cpu_blocks, max_batch_tokens=8192, t_ga=ga,
                                       t_ca=ca, t_l=tl, policy=policy))
        for r in reqs:
            sc.add(*r)
        t0 = time.perf_counter()
        its = sc.run()
        wall = time.perf_counter() - t0
        st = sc.stats()
        results[policy] = {"tokens_per_s": round(st["tokens"] / st["now"], 1),
                           "iterations": st["iterations"],
                           "two_batch_iterations": st["two_batch_iterations"],
                           "swapped_out": st["swapped_out"], "swapped_in": st["swapped_in"],
                           "preempted": st["preempted"],
                           "scheduler_us_per_iteration": round(wall / max(1, len(its)) * 1e6, 2)}
    out = {"metric": "simulated decode throughput, load-aware scheduler vs GPU-only",
           "op": "schedule_sim", "unit": "tokens/s (simulated)",
           "value": results["neo"]["tokens_per_s"],
           "gain": round(results["neo"]["tokens_per_s"] / results["gpu_only"]["tokens_per_s"], 4),
           "results": results,
           "config": {"workload": "2000 requests, prompt U[64,2048], output U[16,512], all at t=0; "
                                  "32 layers; GPU KV 1024 blocks x 16 tokens, CPU KV 16384 blocks",
                      "costs": os.path.relpath(args.costs or DEFAULT_COSTS, ROOT),
                      "gpu": prof.get("gpu"), "cpu": prof.get("cpu")}}
    print(json.dumps(out), flush=True)
    return 0


def bench_overlap_demo(args, torch):
    """Asymmetric pipelining of Llama-3-8B-shaped layers (random weights): batch-0
    = 64 GPU-requests (KV in HBM), batch-1 = CPU-requests (KV in pinned host
    memory), per-iteration time with the host attention overlapped, run
    sequentially, and with both batches' KV in HBM (GPU-only)."""
    import numpy as np
    from paper_2411_01142_amd import pipeline as PL
    L = 8
    rng = np.random.default_rng(args.seed or 0)
    gpu_lens = rng.integers(512, 2048, size=64, endpoint=True)
    layers = [PL.LayerWeights(seed=100 + l) for l in range(L)]
    res = []
    for b1 in (2, 4, 8, 16):
        cpu_lens = rng.integers(512, 2048, size=b1, endpoint=True)
        gpu, cpu = PL.make_batches(L, gpu_lens, cpu_lens, seed=b1)
        pipe = PL.AsymmetricPipeline(layers, gpu, cpu)
        merged = PL.merge_caches(gpu, cpu, layers)

        def timed(fn, reps):
            for _ in range(2):
                fn()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(reps):
                fn()
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) / reps
        t_async = timed(lambda: pipe.iteration(overlap=True), args.steps)
        t_seq = timed(lambda: pipe.iteration(overlap=False), args.steps)
        t_gpu = timed(lambda: PL.gpu_only_iteration(layers, gpu, cpu, merged), args.steps)
        gpipe = PL.GraphedPipeline(layers, gpu, cpu)
        gg, _ = PL.graphed_gpu_only(layers, gpu, cpu, merged)
        tg_async = timed(lambda: gpipe.replay(overlap=True), args.steps)
        tg_seq = timed(lambda: gpipe.replay(overlap=False), args.steps)
        tg_gpu = timed(gg.replay, args.steps)
        gpipe.close()
        # stage times alone: GPU work of batch-0 per layer; host attention of batch-1 per layer
        t_cpu_att = timed(lambda: pipe._cpu_job(0, torch.cuda.Event()), args.steps)
        B = 64 + b1
        res.append({"cpu_requests": b1, "cpu_tokens": int(cpu_lens.sum()),
                    "iteration_ms": {"asymmetric": round(t_async * 1e3, 3),
                                     "sequential": round(t_seq * 1e3, 3),
                                     "gpu_only": round(t_gpu * 1e3, 3)},
                    "graphed_iteration_ms": {"asymmetric": round(tg_async * 1e3, 3),
                                             "sequential": round(tg_seq * 1e3, 3),
                                             "gpu_only": round(tg_gpu * 1e3, 3)},
                    "host_attention_ms_per_layer": round(t_cpu_att * 1e3, 3),
                    "graphed_tokens_per_s": {"asymmetric": round(B / tg_async, 1),
                                             "sequential": round(B / tg_seq, 1),
                                             "gpu_only": round(B / tg_gpu, 1)},
                    "overlap_saving": round(1 - t_async / t_seq, 4),
                    "graphed_overlap_saving": round(1 - tg_async / tg_seq, 4)})
        log(f"[bench] overlap demo b1={b1}: eager {res[-1]['iteration_ms']} "
            f"graphed {res[-1]['graphed_iteration_ms']}")
        pipe.close()
        del gpu, cpu, merged, pipe, gpipe, gg
        torch.cuda.empty_cache()
    out = {"metric": "asymmetric pipelining: decode iteration time, host attention overlapped",
           "op": "overlap_demo", "unit": "ms per iteration (8 layers)", "results": res,
           "config": {"workload": "8 Llama-3-8B-shaped layers (random bf16 weights, torch "
                                  "GEMMs); batch-0 64 GPU-requests U[512,2048]; batch-1 2-16 "
                                  "CPU-requests U[512,2048] in pinned host memory",
                      "cpu_threads": max(1, __import__("paper_2411_01142_amd").cpu_default_threads() - 1)}}
    print(json.dumps(out), flush=True)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=4, choices=[1, 2, 3, 4, 5, 6])
    ap.add_argument("--kv-layout", default="interleaved", choices=["interleaved", "separate"],
                    help="interleaved: K and V caches in one allocation, each block's K and V "
                         "adjacent (block stride 2 x num_kv_heads x 4 KiB); separate: two dense "
                         "caches")
    ap.add_argument("--no-flush-pass", action="store_true",
                    help="skip the per-call pass with a 1 GiB read before each call")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--variant", default="auto", choices=["auto", "valu", "mfma"])
    ap.add_argument("--schedule", default="auto",
                    choices=["auto", "fused", "staged", "two_kernel"])
    ap.add_argument("--max-slices", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--op", default="decode",
                    choices=["decode", "kv_swap_out", "kv_swap_in", "kv_copy_d2d", "kv_append",
                             "cpu_decode", "profile_costs", "schedule_sim", "overlap_demo",
                             "read_ceiling"])
    ap.add_argument("--out", default="")
    ap.add_argument("--costs", default="")
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--cpu-isa", default="auto",
                    choices=["auto", "generic", "avx512", "avx512_bf16"])
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the decode-attention path needs no "
              "collective, and the benchmark runs on a single MI355X (--gpus 1).", file=sys.stderr)
        return 2

    if args.op == "schedule_sim":
        return bench_schedule_sim(args)
    if args.op == "cpu_decode":
        import paper_2411_01142_amd as neo
        from paper_2411_01142_amd import workloads as W
        return bench_cpu_decode(args, neo, W)

    import torch
    if args.copy_calibration:
        copy_calibration()
        return 0

    import paper_2411_01142_amd as neo
    from paper_2411_01142_amd import workloads as W

    if args.op == "profile_costs":
        return bench_profile_costs(args, torch, neo)
    if args.op == "overlap_demo":
        return bench_overlap_demo(args, torch)
    if args.op == "read_ceiling":
        return bench_read_ceiling(args, torch, neo)
    if args.op != "decode":
        return bench_kv_op(args, torch, neo, W)

    seed = args.config if args.seed is None else args.seed
    log(f"[bench] generating config {args.config} seed {seed}")
    case = W.make_config(args.config, seed, poison=False)
    workload_key = W.CONFIGS[args.config]["name"]
    q, k, v, bt, sl = case.to_torch("cuda")
    kv_bytes = k.numel() * 2 + v.numel() * 2
    # At least two copies of the cache, rotated, and at least 4x the Infinity
    # Cache in total: no step finds the tiles of the step before it there.
    nrep = max(2, math.ceil(4 * MALL_BYTES / kv_bytes))
    if args.kv_layout == "interleaved":
        # Each copy one allocation, each block's K and V in one run (new_kv_cache).
        reps = []
        for _ in range(nrep):
            kk, vv = neo.new_kv_cache(case.num_blocks, case.num_kv_heads)
            kk.copy_(k)
            vv.copy_(v)
            reps.append((kk, vv))
        del k, v
        torch.cuda.empty_cache()
    else:
        reps = [(k, v)] + [(k.clone(), v.clone()) for _ in range(nrep - 1)]
    kv_stride = reps[0][0].stride(0)
    out = torch.empty((case.batch, case.num_q_heads, case.head_dim), dtype=torch.float32,
                      device="cuda")
    ws = neo.new_workspace(case.batch, case.num_q_heads, case.num_kv_heads)
    lib = neo.load_library()
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(stream.cuda_stream)
    variant_id = neo.VARIANTS[args.variant]
    schedule_id = neo.SCHEDULES[args.schedule]
    schedule = "fused" if args.schedule == "auto" else args.schedule
    resolved = "mfma" if args.variant == "auto" else args.variant
    hip = HipEvents()
    ev = [(hip.create(), hip.create()) for _ in range(args.steps)]

    def step(i, evs=(None, None)):
        kk, vv = reps[i % nrep]
        rc = lib.neo_decode_attention_events(
            q.data_ptr(), kk.data_ptr(), vv.data_ptr(), bt.data_ptr(), sl.data_ptr(),
            case.num_q_heads, case.num_kv_heads, case.head_dim, case.block_size,
            float(case.scale), out.data_ptr(), case.batch, case.max_blocks_per_seq,
            case.num_blocks, ws.data_ptr(), ws.numel(), variant_id, schedule_id,
            args.max_slices, kv_stride, evs[0], evs[1], sh)
        if rc != 0:
            raise neo.NeoError(rc, lib.neo_last_error().decode())

    log(f"[bench] {case.name}: B={case.batch} sumL={case.total_tokens()} "
        f"KV={kv_bytes / 1e6:.1f} MB x{nrep} replicas, {args.kv_layout} layout; "
        f"warmup {args.warmup}")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Timed region: K steps back to back; events only at its two ends.
    log(f"[bench] timing {args.steps} steps")
    region = (hip.create(), hip.create())
    hip.record(region[0], sh)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i)
    hip.record(region[1], sh)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    region_ms = hip.elapsed_ms(*region) / args.steps

    # Separate pass: events right before and after the decode kernel of each
    # step (they add a little GPU time per step, so they stay out of the
    # timed region above).
    for i in range(args.steps):
        step(args.warmup + args.steps + i, ev[i])
    torch.cuda.synchronize()
    decode_ms = [hip.elapsed_ms(a, b) for a, b in ev]

    # Third pass, one call at a time: 1 GiB of other data read between calls
    # (outside the events) evicts the Infinity Cache, so each call starts with
    # none of its cache lines there; events right around the decode kernel. A
    # read, not a write: a written flush leaves up to 256 MB of dirty lines
    # whose write-back would land inside the next call (measured +35 us).
    flushed_ms = []
    if not args.no_flush_pass:
        scratch = torch.ones(2 ** 30 // 4, dtype=torch.float32, device="cuda")
        sink = torch.empty(1, dtype=torch.float32, device="cuda")
        for i in range(args.steps):
            torch.sum(scratch, dim=0, out=sink[0])
            step(2 * args.steps + args.warmup + i, ev[i])
        torch.cuda.synchronize()
        flushed_ms = [hip.elapsed_ms(a, b) for a, b in ev]
        del scratch, sink
    for a, b in ev + [region]:
        hip.destroy(a)
        hip.destroy(b)

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    alg_bytes = case.algorithmic_bytes()
    value = alg_bytes / (ms_per_step * 1e-3) / 1e9
    dec_ms = sum(decode_ms) / len(decode_ms)
    # Average duration of the decode kernel: with the fused schedule a step is
    # that one kernel, launched back to back, so the timed region's event time
    # per step is it (it matches the rocprofv3 kernel mean); with several
    # kernels per step, the events recorded right around the decode kernel
    # (which add ~1 us of their own).
    kernel_ms = region_ms if schedule == "fused" else dec_ms
    achieved = alg_bytes / (kernel_ms * 1e-3) / 1e9
    traffic = load_traffic(workload_key, f"{resolved}_{schedule}")
    fetched = load_traffic(workload_key, f"{resolved}_{schedule}", reads_only=True)
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "accumulate": "fp32",
        "data": "synthetic",
        "pct_of_peak": round(100.0 * value / PEAK_HBM_GBS, 2),
        "tokens_per_s_per_layer": round(case.batch / (ms_per_step * 1e-3), 1),
        "config": {
            "workload": f"{case.name}: decode attention, {case.num_q_heads} q heads / "
                        f"{case.num_kv_heads} kv heads, head_dim {case.head_dim}, block "
                        f"{case.block_size}, batch {case.batch}, seq_lens {SEQ_DESC[args.config]}",
            "batch": case.batch, "num_q_heads": case.num_q_heads,
            "num_kv_heads": case.num_kv_heads, "head_dim": case.head_dim,
            "block_size": case.block_size, "sum_seq_len": case.total_tokens(),
            "algorithmic_bytes_per_step": alg_bytes, "kv_replicas": nrep,
            "kv_layout": (f"{args.kv_layout}: block stride {kv_stride} elements "
                          f"({'K and V of a block in one run' if args.kv_layout == 'interleaved' else 'two dense caches'})"),
            "variant": resolved, "schedule": schedule, "max_slices": args.max_slices,
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": f"decode_{resolved}_kernel<{case.group}, {schedule}>",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "kernel_ms": round(kernel_ms, 5),
            "kernel_ms_event_pair": round(dec_ms, 5),
            # Per-call spread of the event pairs around the decode kernel.
            "kernel_ms_event_pair_p10_p50_p90": [round(x, 5) for x in pct(decode_ms, (10, 50, 90))],
            # The same with the Infinity Cache evicted (1 GiB read) before each call.
            "kernel_ms_flushed_p10_p50_p90": ([round(x, 5) for x in pct(flushed_ms, (10, 50, 90))]
                                              if flushed_ms else None),
            "achieved_flushed_median": (round(alg_bytes / (pct(flushed_ms, (50,))[0] * 1e-3)
                                              / 1e9, 2) if flushed_ms else None),
            "gpu_ms_per_step": round(region_ms, 5),
            "algorithmic_bytes_per_launch": alg_bytes,
            # Where `traffic` and the two counter rates below come from: not this run
            # but a separate rocprofv3 --pmc run of the same command on the same kernel
            # sources (FETCH_SIZE, then WRITE_SIZE, one counter per run), scaled by what
            # each counter reads for a plain 1 GiB copy.
            "traffic_source": (f"rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, separate profiled run: "
                               f"profiles/counters__decode_{resolved}_{schedule}__{workload_key}.md"
                               if traffic else None),
            # HBM bytes the counters saw (FETCH + WRITE, copy-calibrated) over the same
            # kernel time, beside the algorithmic rate above.
            "achieved_traffic_gbs": (round(traffic / (kernel_ms * 1e-3) / 1e9, 2)
                                     if traffic else None),
            # Bytes read only (FETCH_SIZE), the read rate over the same time.
            "achieved_fetch_gbs": (round(fetched / (kernel_ms * 1e-3) / 1e9, 2)
                                   if fetched else None),
        },
    }
    if not args.no_cpu_baseline:
        log("[bench] CPU baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(case, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
