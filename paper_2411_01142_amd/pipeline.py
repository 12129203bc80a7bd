"""Asymmetric pipelining over one or more transformer layers (Sec. 3.1), driven
from Python with the library's kernels: a demonstration of the offloaded
decoding path on one MI355X and its host.

Two sub-batches per iteration (asymmetric batch division, Sec. 3.1):

* batch-0: GPU-requests, their KV in the GPU cache (HBM); attention on the GPU;
* batch-1: CPU-requests, their KV in the CPU cache (pinned host memory);
  attention on the host CPU.

Per layer l, with the linear stages of a Llama-3-8B-shaped layer (random bf16
weights: QKV projection, output projection, gated MLP; torch GEMMs):

* the GPU runs batch-0's post-projection of layer l-1 and pre-projection of
  layer l, appends batch-0's new K/V to the GPU cache, and runs batch-0's
  attention (T_l0 + T_ga0),
* while a host thread appends batch-1's new K/V to the CPU cache and runs
  batch-1's attention for layer l (T_ca1), on Q/K/V the GPU produced one stage
  earlier and copied to pinned host memory (TrQKV);
* then the output comes back to the GPU (TrO) and the GPU runs batch-1's
  post-projection of layer l and pre-projection of layer l+1 (T_l1), whose
  Q/K/V go to the host for the next layer.

``AsymmetricPipeline.iteration(overlap=False)`` does exactly the same work with
the host attention run while the GPU is idle (no overlap);
``gpu_only_iteration`` keeps both batches' KV in HBM with one attention call
per layer (the non-offloading schedule); ``GraphedPipeline`` replays each
stage's GPU work from a HIP graph.
"""
from __future__ import annotations

import concurrent.futures as cf
from dataclasses import dataclass
from typing import List

import numpy as np

from . import copy_blocks, cpu_decode_attention, cpu_default_threads, cpu_kv_append
from . import decode_attention, kv_append, new_workspace


def _torch():
    import torch
    return torch


class LayerWeights:
    """Random bf16 weights of one Llama-3-8B-shaped layer (no norms)."""

    def __init__(self, hidden=4096, hq=32, hkv=8, d=128, ffn=14336, *, seed=0, device="cuda"):
        torch = _torch()
        g = torch.Generator(device=device).manual_seed(seed)
        bf = torch.bfloat16

        def w(rows, cols):
            return (torch.randn(rows, cols, generator=g, device=device) * rows ** -0.5).to(bf)
        self.hidden, self.hq, self.hkv, self.d = hidden, hq, hkv, d
        self.wqkv = w(hidden, (hq + 2 * hkv) * d)
        self.wo = w(hq * d, hidden)
        self.w1 = w(hidden, ffn)
        self.w3 = w(hidden, ffn)
        self.w2 = w(ffn, hidden)

    def pre(self, x):
        """Pre-projection: x [B, hidden] -> q [B, hq, d], k, v [B, hkv, d] (bf16)."""
        B = x.shape[0]
        qkv = x @ self.wqkv
        nq, nk = self.hq * self.d, self.hkv * self.d
        q = qkv[:, :nq].reshape(B, self.hq, self.d).contiguous()
        k = qkv[:, nq:nq + nk].reshape(B, self.hkv, self.d).contiguous()
        v = qkv[:, nq + nk:].reshape(B, self.hkv, self.d).contiguous()
        return q, k, v

    def post(self, x, o):
        """Post-projection: attention output o [B, hq, d] (fp32) -> next x."""
        torch = _torch()
        B = x.shape[0]
        h = x + o.to(torch.bfloat16).reshape(B, -1) @ self.wo
        m = torch.nn.functional.silu(h @ self.w1) * (h @ self.w3)
        return h + m @ self.w2


@dataclass
class GpuBatch:
    """batch-0: per-layer KV caches in HBM."""
    k: List  # per layer [NB, Hkv, 16, 16, 8] bf16
    v: List  # per layer [NB, Hkv, 128, 16] bf16
    table: object  # [B, MBPS] int32 (device)
    lens: object   # [B] int32 (device)
    x: object      # [B, hidden] bf16 (device)


@dataclass
class CpuBatch:
    """batch-1: per-layer KV caches in pinned host memory."""
    k: List  # per layer, pinned CPU bf16
    v: List
    table: np.ndarray
    lens: np.ndarray
    x: object  # [B, hidden] bf16 (device)


def _lens_table(lens, rng):
    nbs = (lens + 15) // 16
    mbps = int(nbs.max())
    total = int(nbs.sum())
    nb = total + max(1, total // 20)
    perm = rng.permutation(nb).astype(np.int32)
    table = np.full((len(lens), mbps), -1, np.int32)
    o = 0
    for b, n in enumerate(nbs):
        table[b, :n] = perm[o:o + n]
        o += n
    return table, nb


def make_batches(num_layers, gpu_lens, cpu_lens, *, hidden=4096, hkv=8, seed=0, device="cuda"):
    """Caches of N(0,1) bf16 K/V for every layer (the slot of each request's
    newest token is overwritten by the append) and N(0,1) hidden states."""
    torch = _torch()
    rng = np.random.default_rng(seed)
    g = torch.Generator(device=device).manual_seed(seed + 1)
    gl = np.asarray(gpu_lens, np.int32)
    cl = np.asarray(cpu_lens, np.int32)
    gt, gnb = _lens_table(gl, rng)
    ct, cnb = _lens_table(cl, rng)
    bf = torch.bfloat16

    def kv(nb):
        k = torch.randn((nb, hkv, 16, 16, 8), generator=g, device=device).to(bf)
        v = torch.randn((nb, hkv, 128, 16), generator=g, device=device).to(bf)
        return k, v
    gk, gv, ck, cv = [], [], [], []
    for _ in range(num_layers):
        k, v = kv(gnb)
        gk.append(k)
        gv.append(v)
        k, v = kv(cnb)
        ck.append(k.cpu().pin_memory())
        cv.append(v.cpu().pin_memory())
    x0 = torch.randn((len(gl), hidden), generator=g, device=device).to(bf)
    x1 = torch.randn((len(cl), hidden), generator=g, device=device).to(bf)
    gpu = GpuBatch(gk, gv, torch.from_numpy(gt).to(device), torch.from_numpy(gl).to(device), x0)
    cpu = CpuBatch(ck, cv, ct, cl, x1)
    return gpu, cpu


class AsymmetricPipeline:
    """Runs iterations of the two-sub-batch schedule over `layers`."""

    def __init__(self, layers: List[LayerWeights], gpu: GpuBatch, cpu: CpuBatch, *,
                 cpu_threads: int = 0, cpu_isa: str = "auto"):
        torch = _torch()
        self.torch = torch
        self.layers, self.gpu, self.cpu = layers, gpu, cpu
        self.threads = cpu_threads or max(1, cpu_default_threads() - 1)  # one core launches
        self.isa = cpu_isa
        L0 = layers[0]
        B1 = cpu.x.shape[0]
        self.ws = new_workspace(gpu.x.shape[0], L0.hq, L0.hkv)
        self.q1_h = torch.empty((B1, L0.hq, L0.d), dtype=torch.bfloat16, pin_memory=True)
        self.k1_h = torch.empty((B1, L0.hkv, L0.d), dtype=torch.bfloat16, pin_memory=True)
        self.v1_h = torch.empty((B1, L0.hkv, L0.d), dtype=torch.bfloat16, pin_memory=True)
        self.o1_h = torch.empty((B1, L0.hq, L0.d), dtype=torch.float32, pin_memory=True)
        self.pool = cf.ThreadPoolExecutor(max_workers=1)
        # Per layer, when recording: both sub-batches' attention inputs and
        # outputs (q0, o0 on the GPU; q1, o1 in host memory).
        self.records = []

    def _to_host(self, q, k, v):
        self.q1_h.copy_(q, non_blocking=True)
        self.k1_h.copy_(k, non_blocking=True)
        self.v1_h.copy_(v, non_blocking=True)
        ev = self.torch.cuda.Event()
        ev.record()
        return ev

    def _cpu_job(self, layer, ready):
        ready.synchronize()  # TrQKV landed in pinned memory
        c = self.cpu
        cpu_kv_append(c.k[layer], c.v[layer], self.k1_h, self.v1_h, c.table, c.lens)
        cpu_decode_attention(self.q1_h, c.k[layer], c.v[layer], c.table, c.lens,
                             out=self.o1_h, num_threads=self.threads, isa=self.isa)

    def iteration(self, *, overlap=True, record=False):
        """One decoding iteration through every layer; returns (x0, x1)."""
        torch = self.torch
        g, c, Ls = self.gpu, self.cpu, self.layers
        x0, x1 = g.x, c.x
        q1, k1, v1 = Ls[0].pre(x1)
        ready = self._to_host(q1, k1, v1)
        o0 = None
        for l, W in enumerate(Ls):
            fut = self.pool.submit(self._cpu_job, l, ready) if overlap else None
            # GPU, batch-0: post-projection of l-1, pre-projection of l, append, attention
            if o0 is not None:
                x0 = Ls[l - 1].post(x0, o0)
            q0, k0, v0 = W.pre(x0)
            kv_append(g.k[l], g.v[l], k0, v0, g.table, g.lens)
            o0 = decode_attention(q0, g.k[l], g.v[l], g.table, g.lens, workspace=self.ws)
            if overlap:
                fut.result()
            else:
                torch.cuda.synchronize()
                self._cpu_job(l, ready)
            if record:
                self.records.append({"q0": q0.clone(), "o0": o0.clone(),
                                     "q1": self.q1_h.clone(), "o1": self.o1_h.clone()})
            # GPU, batch-1: output back (TrO), post-projection of l, pre-projection of l+1
            o1 = self.o1_h.to(x1.device, non_blocking=True)
            x1 = W.post(x1, o1)
            if l + 1 < len(Ls):
                q1, k1, v1 = Ls[l + 1].pre(x1)
                ready = self._to_host(q1, k1, v1)
        x0 = Ls[-1].post(x0, o0)
        return x0, x1

    def close(self):
        self.pool.shutdown()


def gpu_only_iteration(layers, gpu: GpuBatch, cpu: CpuBatch, caches=None):
    """Both sub-batches with their KV in HBM: one attention call per layer
    (the non-offloading schedule). `caches` from ``merge_caches``."""
    torch = _torch()
    x = torch.cat([gpu.x, cpu.x])
    k_all, v_all, table, lens, ws = caches
    o = None
    for l, W in enumerate(layers):
        if o is not None:
            x = layers[l - 1].post(x, o)
        q, k, v = W.pre(x)
        kv_append(k_all[l], v_all[l], k, v, table, lens)
        o = decode_attention(q, k_all[l], v_all[l], table, lens, workspace=ws)
    x = layers[-1].post(x, o)
    B0 = gpu.x.shape[0]
    return x[:B0], x[B0:]


def merge_caches(gpu: GpuBatch, cpu: CpuBatch, layers):
    """HBM caches holding both batches (batch-1's blocks swapped in after
    batch-0's with the library's block copy), for ``gpu_only_iteration``."""
    torch = _torch()
    dev = gpu.x.device
    NB0 = gpu.k[0].shape[0]
    NB1 = cpu.k[0].shape[0]
    ks, vs = [], []
    ids_src = torch.arange(NB1, dtype=torch.int32, device=dev)
    ids_dst = ids_src + NB0
    for l in range(len(layers)):
        k = torch.empty((NB0 + NB1,) + tuple(gpu.k[l].shape[1:]), dtype=torch.bfloat16, device=dev)
        v = torch.empty((NB0 + NB1,) + tuple(gpu.v[l].shape[1:]), dtype=torch.bfloat16, device=dev)
        k[:NB0].copy_(gpu.k[l])
        v[:NB0].copy_(gpu.v[l])
        copy_blocks(cpu.k[l], cpu.v[l], k, v, ids_src, ids_dst)
        ks.append(k)
        vs.append(v)
    t0 = gpu.table.cpu().numpy()
    t1 = np.where(cpu.table >= 0, cpu.table + NB0, -1).astype(np.int32)
    w = max(t0.shape[1], t1.shape[1])
    table = np.full((t0.shape[0] + t1.shape[0], w), -1, np.int32)
    table[:t0.shape[0], :t0.shape[1]] = t0
    table[t0.shape[0]:, :t1.shape[1]] = t1
    lens = np.concatenate([gpu.lens.cpu().numpy(), cpu.lens])
    L0 = layers[0]
    ws = new_workspace(len(lens), L0.hq, L0.hkv)
    return ks, vs, torch.from_numpy(table).to(dev), torch.from_numpy(lens).to(dev), ws


class GraphedPipeline(AsymmetricPipeline):
    """The same schedule with each stage's GPU work captured once as a HIP
    graph and replayed (launch overhead off the critical path, Sec. 4, "Reducing
    Kernel Launching Overhead"): per layer, graph A (batch-0: post-projection
    of l-1, pre-projection of l, append, attention) and graph B (batch-1: TrO,
    post-projection of l, pre-projection of l+1, TrQKV), plus a prologue and an
    epilogue graph. The host attention stays on the worker thread between the
    two replays. Every graph reads and writes fixed buffers, so each replay
    recomputes the iteration from the batches' stored hidden states."""

    def __init__(self, layers, gpu, cpu, *, cpu_threads: int = 0, cpu_isa: str = "auto"):
        super().__init__(layers, gpu, cpu, cpu_threads=cpu_threads, cpu_isa=cpu_isa)
        torch = self.torch
        g, c, Ls = gpu, cpu, layers
        self._keep = []
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        # warm up every op once on the capture stream (library workspaces, GEMM plans)
        with torch.cuda.stream(s):
            self.iteration(overlap=False)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()

        def capture(fn):
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                out = fn()
            self._keep.append(out)
            return graph, out

        state = {}

        def prologue():
            q1, k1, v1 = Ls[0].pre(c.x)
            self.q1_h.copy_(q1, non_blocking=True)
            self.k1_h.copy_(k1, non_blocking=True)
            self.v1_h.copy_(v1, non_blocking=True)
            return q1, k1, v1
        self.g_pro, _ = capture(prologue)
        self.g_a, self.g_b = [], []
        x0, x1, o0 = g.x, c.x, None
        for l, W in enumerate(Ls):
            def stage_a(l=l, W=W, x0=x0, o0=o0):
                x = Ls[l - 1].post(x0, o0) if o0 is not None else x0
                q0, k0, v0 = W.pre(x)
                kv_append(g.k[l], g.v[l], k0, v0, g.table, g.lens)
                o = decode_attention(q0, g.k[l], g.v[l], g.table, g.lens, workspace=self.ws)
                return x, o
            ga, (x0, o0) = capture(stage_a)

            def stage_b(l=l, W=W, x1=x1):
                o1 = self.o1_h.to(x1.device, non_blocking=True)
                x = W.post(x1, o1)
                if l + 1 < len(Ls):
                    q1, k1, v1 = Ls[l + 1].pre(x)
                    self.q1_h.copy_(q1, non_blocking=True)
                    self.k1_h.copy_(k1, non_blocking=True)
                    self.v1_h.copy_(v1, non_blocking=True)
                return x
            gb, x1 = capture(stage_b)
            self.g_a.append(ga)
            self.g_b.append(gb)

        def epilogue(x0=x0, o0=o0):
            return Ls[-1].post(x0, o0)
        self.g_epi, self.out0 = capture(epilogue)
        self.out1 = x1
        torch.cuda.synchronize()

    def replay(self, *, overlap=True):
        """One iteration from the graphs; returns (x0, x1) (graph-owned buffers)."""
        torch = self.torch
        self.g_pro.replay()
        ready = torch.cuda.Event()
        ready.record()
        for l in range(len(self.layers)):
            fut = self.pool.submit(self._cpu_job, l, ready) if overlap else None
            self.g_a[l].replay()
            if overlap:
                fut.result()
            else:
                torch.cuda.synchronize()
                self._cpu_job(l, ready)
            self.g_b[l].replay()
            ready = torch.cuda.Event()
            ready.record()
        self.g_epi.replay()
        return self.out0, self.out1


def graphed_gpu_only(layers, gpu, cpu, caches):
    """``gpu_only_iteration`` captured as one HIP graph; returns (graph, (x0, x1))."""
    torch = _torch()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        gpu_only_iteration(layers, gpu, cpu, caches)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        out = gpu_only_iteration(layers, gpu, cpu, caches)
    torch.cuda.synchronize()
    return graph, out
