"""Tests of the offloaded path on the machine that holds the GPU.

The asymmetric pipelining demo (Sec. 3.1): both sub-batches' attention inside
the pipeline (batch-0 on the GPU, batch-1 on the host CPU) matches the fp64
oracle element by element on the same q/K/V, for every host instruction-set
path; overlapping the host attention with GPU work changes no result
(bit-identical to running it sequentially); keeping every request's KV in HBM
(one attention call per layer) gives the same outputs up to bf16 GEMM
rounding. The host-CPU path (Sec. 4) also runs a full workload on this
machine's CPU against the oracle.
"""
import math
import sys

import numpy as np
import pytest

import oracle
import paper_2411_01142_amd as neo
from paper_2411_01142_amd import workloads as W
from parity_report import record

torch = pytest.importorskip("torch")

ABS_TOL = 1e-2
REL_TOL = 2e-2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


def test_asymmetric_matches_sequential_and_gpu_only():
    from paper_2411_01142_amd import pipeline as PL
    print("[pipeline] 2 layers, 8 GPU + 4 CPU requests", flush=True)
    L = 2
    layers = [PL.LayerWeights(seed=10 + l) for l in range(L)]
    gpu, cpu = PL.make_batches(L, [37, 200, 16, 129, 300, 64, 1, 90], [250, 17, 48, 400], seed=3)
    merged = PL.merge_caches(gpu, cpu, layers)
    pipe = PL.AsymmetricPipeline(layers, gpu, cpu, cpu_threads=4)
    a0, a1 = pipe.iteration(overlap=True)
    s0, s1 = pipe.iteration(overlap=False)
    torch.cuda.synchronize()
    assert torch.equal(a0, s0) and torch.equal(a1, s1)
    g0, g1 = PL.gpu_only_iteration(layers, gpu, cpu, merged)
    torch.cuda.synchronize()
    for a, g in ((a0, g0), (a1, g1)):
        a, g = a.float(), g.float()
        assert torch.isfinite(a).all()
        rel = ((a - g).norm() / g.norm()).item()
        print(f"[pipeline] rel diff vs gpu-only {rel:.2e}", flush=True)
        assert rel < 2e-2
    pipe.close()


def test_graph_replays_match_eager():
    """Each stage captured once as a HIP graph: every replay (with eager work and
    synchronisations in between) gives the eager iteration's results."""
    from paper_2411_01142_amd import pipeline as PL
    print("[pipeline] graphs: 2 layers, 8 GPU + 4 CPU requests", flush=True)
    L = 2
    layers = [PL.LayerWeights(seed=20 + l) for l in range(L)]
    gpu, cpu = PL.make_batches(L, [37, 200, 16, 129, 300, 64, 1, 90], [250, 17, 48, 400], seed=5)
    merged = PL.merge_caches(gpu, cpu, layers)
    eager = PL.AsymmetricPipeline(layers, gpu, cpu, cpu_threads=4)
    e0, e1 = [t.clone() for t in eager.iteration(overlap=False)]
    eager.close()
    pipe = PL.GraphedPipeline(layers, gpu, cpu, cpu_threads=4)
    for r in range(3):
        a0, a1 = pipe.replay(overlap=(r != 1))
        torch.cuda.synchronize()
        assert torch.equal(a0, e0) and torch.equal(a1, e1), r
        _ = (torch.randn(256, 256, device="cuda") @ torch.randn(256, 256, device="cuda")).sum().item()
    gg, (g0, g1) = PL.graphed_gpu_only(layers, gpu, cpu, merged)
    ref0, ref1 = [t.clone() for t in PL.gpu_only_iteration(layers, gpu, cpu, merged)]
    for r in range(3):
        gg.replay()
        torch.cuda.synchronize()
        assert torch.equal(g0, ref0) and torch.equal(g1, ref1), r
    pipe.close()


def _u16(t):
    """bf16 tensor (any device) -> numpy uint16 bit patterns."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _case(q, k, v, table, lens, name):
    q, k, v = _u16(q), _u16(k), _u16(v)
    return W.Case(q=q, k_cache=k, v_cache=v, block_table=np.ascontiguousarray(table, np.int32),
                  seq_lens=np.ascontiguousarray(lens, np.int32), num_q_heads=q.shape[1],
                  num_kv_heads=k.shape[1], head_dim=128, block_size=16,
                  scale=1.0 / math.sqrt(128), name=name)


def _errors(y, r):
    y = y.reshape(-1, y.shape[-1]).astype(np.float64)
    r = r.reshape(-1, r.shape[-1]).astype(np.float64)
    ae = np.abs(y - r)
    return float(ae.max()), float((ae.max(axis=1) / np.maximum(np.abs(r).max(axis=1), 1e-30)).max())


def _isa_available(isa):
    try:
        q = np.zeros((1, 8, 128), np.uint16)
        k = np.zeros((1, 8, 16, 16, 8), np.uint16)
        v = np.zeros((1, 8, 128, 16), np.uint16)
        neo.cpu_decode_attention(q, k, v, np.zeros((1, 1), np.int32), np.ones(1, np.int32),
                                 num_threads=1, isa=isa)
        return True
    except neo.NeoError as e:
        if e.status == 2:
            return False
        raise


@pytest.mark.parametrize("isa", ["avx512", "avx512_bf16", "generic"])
def test_pipeline_attention_matches_oracle(isa):
    """Each layer's attention of both sub-batches, taken inside an overlapped
    iteration (GPU batch-0 through the HIP kernels, host batch-1 through the
    CPU path with the given instruction set), against the oracle on the same
    q and the caches as the attention read them (each layer's cache is only
    appended to by that layer's step, so after the iteration it holds what the
    attention saw)."""
    from paper_2411_01142_amd import pipeline as PL
    if not _isa_available(isa):
        pytest.skip(f"this host CPU has no {isa} path")
    print(f"[pipeline-oracle] isa={isa}: 3 layers, 12 GPU + 6 CPU requests", flush=True)
    L = 3
    layers = [PL.LayerWeights(seed=40 + l) for l in range(L)]
    gpu_lens = [37, 200, 16, 129, 300, 64, 1, 90, 1000, 2047, 513, 17]
    cpu_lens = [250, 17, 48, 400, 1, 1500]
    gpu, cpu = PL.make_batches(L, gpu_lens, cpu_lens, seed=7)
    pipe = PL.AsymmetricPipeline(layers, gpu, cpu, cpu_threads=4, cpu_isa=isa)
    pipe.iteration(overlap=True, record=True)
    torch.cuda.synchronize()
    assert len(pipe.records) == L
    g_table, g_lens = gpu.table.cpu().numpy(), gpu.lens.cpu().numpy()
    worst = (0.0, 0.0)
    for l, rec in enumerate(pipe.records):
        c0 = _case(rec["q0"], gpu.k[l], gpu.v[l], g_table, g_lens, f"layer {l} batch-0")
        c1 = _case(rec["q1"], cpu.k[l], cpu.v[l], cpu.table, cpu.lens, f"layer {l} batch-1")
        for c, y in ((c0, rec["o0"]), (c1, rec["o1"])):
            y = y.cpu().numpy()
            ref = oracle.decode_attention(c)
            assert np.all(np.isfinite(y)), c.name
            ae, re = _errors(y, ref)
            print(f"[pipeline-oracle] {isa} {c.name}: max_abs={ae:.3e} max_rel_rownorm={re:.3e}",
                  flush=True)
            worst = (max(worst[0], ae), max(worst[1], re))
            assert ae <= ABS_TOL and re <= REL_TOL, (c.name, ae, re)
    record(f"pipeline ({isa} host path): {L} layers x 2 sub-batches, max_abs={worst[0]:.2e} "
           f"max_rel_rownorm={worst[1]:.2e}")
    pipe.close()


@pytest.mark.parametrize("isa", ["avx512", "avx512_bf16", "generic"])
def test_host_path_on_this_host_full_batch(isa):
    """The host-CPU path on the CPU of the machine that holds the GPU (the one
    an offloaded sub-batch would run on), over the full batch-64 Llama-3-8B
    workload with poisoned unused slots, element by element against the
    oracle, for each instruction-set path this CPU has."""
    if not _isa_available(isa):
        pytest.skip(f"this host CPU has no {isa} path")
    case = W.make_config(2, 2)
    print(f"[host-path] isa={isa} threads={neo.cpu_default_threads()} {case.name}", flush=True)
    y = neo.cpu_decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                 case.seq_lens, scale=case.scale, isa=isa)
    ref = oracle.decode_attention(case)
    assert np.all(np.isfinite(y))
    ae, re = _errors(y, ref)
    print(f"[host-path] {isa}: max_abs={ae:.3e} max_rel_rownorm={re:.3e}", flush=True)
    record(f"host CPU path ({isa}, {neo.cpu_default_threads()} threads) {case.name}: "
           f"max_abs={ae:.2e} max_rel_rownorm={re:.2e}")
    assert ae <= ABS_TOL and re <= REL_TOL
