"""Cost model and load-aware scheduler (Sec. 3.2): the oracle pinned by closed
forms and hand-traced scenarios, then the library's C++ scheduler compared with
the oracle decision by decision (bit-exact lists and modes; times within
1e-12 relative, both computed in double with the same formulas). CPU only."""
import math
import random

import numpy as np
import pytest

from oracle.scheduler import OracleScheduler, interp_curve, interp_grid
from paper_2411_01142_amd import NeoError
from paper_2411_01142_amd import sched as S


# ------------------------------------------------------------------ cost model

def planar_grid(bs, ss, a=3.0, kb=0.25, ks=0.002):
    return [[a + kb * b + ks * s for s in ss] for b in bs]


def test_bilinear_reproduces_planes_and_grid_points():
    bs, ss = [1, 4, 16, 64], [100, 1000, 5000]
    t = planar_grid(bs, ss)
    lib = S.CostGrid(bs, ss, t)
    rng = np.random.default_rng(0)
    for b, s in list(zip(rng.uniform(0, 100, 50), rng.uniform(0, 8000, 50))) + [(1, 100), (64, 5000)]:
        exact = 3.0 + 0.25 * b + 0.002 * s  # inside and outside the grid
        assert lib(b, s) == pytest.approx(exact, rel=1e-12, abs=1e-12)
        assert interp_grid(bs, ss, t, b, s) == pytest.approx(exact, rel=1e-12, abs=1e-12)
    for i, b in enumerate(bs):
        for j, s in enumerate(ss):
            assert lib(b, s) == t[i][j] == interp_grid(bs, ss, t, b, s)


def test_bilinear_cell_values():
    # one cell: f = t00 (1-u)(1-v) + t01 (1-u) v + t10 u (1-v) + t11 u v
    bs, ss, t = [0.0, 2.0], [0.0, 10.0], [[1.0, 5.0], [3.0, 11.0]]
    for b, s in [(1.0, 5.0), (0.5, 2.5), (2.0, 0.0), (1.5, 7.5)]:
        u, v = b / 2, s / 10
        want = 1 * (1 - u) * (1 - v) + 5 * (1 - u) * v + 3 * u * (1 - v) + 11 * u * v
        assert S.CostGrid(bs, ss, t)(b, s) == pytest.approx(want, rel=1e-14)
        assert interp_grid(bs, ss, t, b, s) == pytest.approx(want, rel=1e-14)


def test_single_point_axes_and_curves():
    g = S.CostGrid([8], [100, 200], [[1.0, 2.0]])
    assert g(1, 150) == g(1000, 150) == pytest.approx(1.5)
    c = S.CostCurve([1, 10, 100], [1.0, 10.0, 40.0])
    for x, want in [(5, 5.0), (55, 25.0), (0, 0.0), (200, 40.0 + 100 * 30 / 90)]:
        assert c(x) == pytest.approx(want) == pytest.approx(interp_curve([1, 10, 100], [1.0, 10.0, 40.0], x))
    assert S.CostCurve([7], [3.0])(1000) == 3.0


def test_cost_tables_are_validated():
    with pytest.raises(NeoError):
        S.CostGrid([1, 1], [1], [[0.0], [0.0]])(1, 1)
    with pytest.raises(NeoError):
        S.CostCurve([2, 1], [0.0, 0.0])(1)
    with pytest.raises(NeoError):
        S.CostCurve([1], [float("nan")])(1)


# ------------------------------------------------------------------ scheduler

def linear_costs(ga_per_tok, ca_per_tok):
    """T_ga = ga * s, T_ca = ca * s (independent of b), T_l(x) = x."""
    ga = ([1.0, 2.0], [1.0, 100.0], [[ga_per_tok, 100 * ga_per_tok]] * 2)
    ca = ([1.0, 2.0], [1.0, 100.0], [[ca_per_tok, 100 * ca_per_tok]] * 2)
    tl = ([1.0, 100.0], [1.0, 100.0])
    return ga, ca, tl


def make_pair(ga, ca, tl, **kw):
    o = OracleScheduler(t_ga=ga, t_ca=ca, t_l=tl, **kw)
    c = S.Scheduler(S.SchedConfig(t_ga=S.CostGrid(*ga), t_ca=S.CostGrid(*ca),
                                  t_l=S.CostCurve(*tl), **kw))
    return o, c


def small_kw(**over):
    kw = dict(num_layers=1, block_size=4, gpu_blocks=3, cpu_blocks=100, max_batch_tokens=100,
              swap_in_reserve_blocks=0, policy="neo")
    kw.update(over)
    return kw


def run_both(o, c, reqs):
    for rid, p, out, arr in reqs:
        o.add(rid, p, out, arr)
        c.add(rid, p, out, arr)
    trace_o, trace_c = [], []
    for _ in range(100000):
        a = o.step()
        b = c.step()
        assert (a is None) == (b is None)
        if a is None:
            break
        trace_o.append(a)
        trace_c.append(b)
    return trace_o, trace_c


def check_same(trace_o, trace_c):
    assert len(trace_o) == len(trace_c)
    for k, (a, b) in enumerate(zip(trace_o, trace_c)):
        for key in ("mode", "prefill", "gpu_decode", "cpu_decode0", "cpu_decode1", "swap_out",
                    "swap_in", "n_prefill_to_cpu", "n_tokens"):
            assert a[key] == getattr(b, key), (k, key, a[key], getattr(b, key))
        for key in ("t_iter", "t_two_batch", "t_gpu_only", "t_l0", "t_l1", "t_ga0", "t_ca0",
                    "t_ca1", "now"):
            assert getattr(b, key) == pytest.approx(a[key], rel=1e-12, abs=1e-15), (k, key)


def test_hand_traced_cpu_too_slow():
    # CPU attention 5x slower per token than T_l per token: the CPU is never used.
    o, c = make_pair(*linear_costs(0.1, 0.5), **small_kw())
    to, tc = run_both(o, c, [(0, 4, 3, 0.0), (1, 4, 3, 0.0), (2, 4, 2, 0.0)])
    check_same(to, tc)
    got = [(t["mode"], t["prefill"], t["gpu_decode"], t["swap_out"], t["swap_in"],
            round(t["t_iter"], 9)) for t in to]
    assert got == [
        ("gpu_only", [0, 1, 2], [], [], [], 12.0),     # three prefills, KV kept on the GPU
        ("gpu_only", [], [0], [2, 1], [], 1.5),        # next tokens need 6 blocks: swap out 2, 1
        ("gpu_only", [], [0], [], [], 1.6),            # CPU decodes fit neither inequality
        ("gpu_only", [], [2], [], [2], 1.5),           # 0 finished: swap 2 back in
        ("gpu_only", [], [1], [], [1], 1.5),
        ("gpu_only", [], [1], [], [], 1.6),
    ]
    assert o.total_tokens == 8 and c.stats()["tokens"] == 8


def test_hand_traced_two_batches():
    # CPU attention cheap: the swapped-out requests decode in batch-1.
    o, c = make_pair(*linear_costs(0.1, 0.05), **small_kw())
    to, tc = run_both(o, c, [(0, 4, 3, 0.0), (1, 4, 3, 0.0), (2, 4, 2, 0.0)])
    check_same(to, tc)
    got = [(t["mode"], t["gpu_decode"], t["cpu_decode0"], t["cpu_decode1"], t["swap_out"],
            round(t["t_iter"], 9), round(t["t_ca1"], 9), round(t["t_l1"], 9)) for t in to]
    assert got == [
        ("gpu_only", [], [], [], [], 12.0, 0.0, 0.0),
        # T_two = max(1, 0.5) + max(2 + 0.5, 0) = 3.5; 3 x 1.5 > 1 x 3.5
        ("two_batch", [0], [], [2, 1], [2, 1], 3.5, 0.5, 2.0),
        # T_two = max(1, 0.3) + max(1 + 0.6, 0) = 2.6; 2 x 1.6 > 1 x 2.6
        ("two_batch", [0], [], [1], [], 2.6, 0.3, 1.0),
    ]
    assert to[-1]["now"] == pytest.approx(12 + 3.5 + 2.6)


def test_iteration_time_closed_form():
    # constant stage times: T_two = L (max(l, c) + max(l + a, c))
    a, cc, l, L = 0.7, 2.0, 1.5, 3
    ga = ([1.0], [1.0], [[a]])
    ca = ([1.0], [1.0], [[cc]])
    tl = ([1.0], [l])
    o, c = make_pair(ga, ca, tl, **small_kw(num_layers=L, gpu_blocks=2, block_size=4))
    to, tc = run_both(o, c, [(i, 4, 4, 0.0) for i in range(4)])
    check_same(to, tc)
    for t in to:
        if t["mode"] == "two_batch":
            l0 = l if t["prefill"] or t["gpu_decode"] or t["cpu_decode0"] else 0.0
            c1 = cc if t["cpu_decode1"] else 0.0
            l1 = l if t["cpu_decode1"] else 0.0
            c0 = cc if t["cpu_decode0"] else 0.0
            a0 = a if t["gpu_decode"] else 0.0
            assert t["t_iter"] == pytest.approx(L * (max(l0, c1) + max(l1 + a0, c0)))
        else:
            l0 = l if t["prefill"] or t["gpu_decode"] else 0.0
            assert t["t_iter"] == pytest.approx(L * (l0 + (a if t["gpu_decode"] else 0.0)))


def bandwidth_costs(gpu_bw=5.5e12, cpu_bw=150e9, flops=1.75e15):
    """Per-layer times of a Llama-3-8B-shaped layer (8 kv heads, 436 MB of bf16
    weights, 218 M parameters) from simple bandwidth / compute models: attention
    streams 512 B per (token, kv head) at the device's bandwidth, the linear
    stage takes max(weights / GPU bandwidth, 2 x params x tokens / flops).
    Defaults: MI355X-like GPU attention and linear stage, a ~150 GB/s host."""
    bs = [1.0, 16.0, 64.0, 256.0, 1024.0]
    ss = [16.0, 4096.0, 65536.0, 1048576.0]
    ga = [[5e-6 + 0.1e-6 * b + s * 8 * 512 / gpu_bw for s in ss] for b in bs]
    ca = [[20e-6 + 0.5e-6 * b + s * 8 * 512 / cpu_bw for s in ss] for b in bs]
    xs = [1.0, 64.0, 256.0, 1024.0, 8192.0]
    tl = [max(436e6 / gpu_bw, 2 * 218e6 * x / flops) for x in xs]
    return (bs, ss, ga), (bs, ss, ca), (xs, tl)


def random_workload(seed, n, max_prompt=2048, max_out=256, spread=0.0):
    rng = random.Random(seed)
    return [(i, rng.randint(16, max_prompt), rng.randint(1, max_out),
             rng.uniform(0, spread) if spread else 0.0) for i in range(n)]


@pytest.mark.parametrize("seed,gpu_blocks,cpu_blocks,act,reserve,policy,spread", [
    (1, 2000, 20000, 4096, 0, "neo", 0.0),
    (2, 800, 20000, 2048, 16, "neo", 0.0),
    (3, 3000, 1500, 8192, 0, "neo", 0.5),
    (4, 1200, 0, 4096, 0, "neo", 0.0),        # no CPU cache: preemption instead of swaps
    (5, 2000, 20000, 4096, 0, "gpu_only", 0.0),
    (6, 500, 3000, 1024, 8, "neo", 2.0),
])
def test_library_matches_oracle(seed, gpu_blocks, cpu_blocks, act, reserve, policy, spread):
    ga, ca, tl = bandwidth_costs()
    kw = dict(num_layers=32, block_size=16, gpu_blocks=gpu_blocks, cpu_blocks=cpu_blocks,
              max_batch_tokens=act, swap_in_reserve_blocks=reserve, policy=policy)
    o, c = make_pair(ga, ca, tl, **kw)
    reqs = random_workload(seed, 120, spread=spread)
    to, tc = run_both(o, c, reqs)
    check_same(to, tc)
    st = c.stats()
    assert st["finished"] == len(reqs)
    assert st["tokens"] == sum(r[2] for r in reqs) == o.total_tokens
    assert st["now"] == pytest.approx(o.clock, rel=1e-12)
    if cpu_blocks == 0 or policy == "gpu_only":
        assert all(t["mode"] == "gpu_only" for t in to)


def test_invariants_during_a_run():
    ga, ca, tl = bandwidth_costs()
    cap_gpu, cap_cpu = 900, 6000
    c = S.Scheduler(S.SchedConfig(num_layers=32, block_size=16, gpu_blocks=cap_gpu,
                                  cpu_blocks=cap_cpu, max_batch_tokens=2048,
                                  t_ga=S.CostGrid(*ga), t_ca=S.CostGrid(*ca),
                                  t_l=S.CostCurve(*tl)))
    reqs = random_workload(9, 200)
    for r in reqs:
        c.add(*r)
    two = 0
    while True:
        it = c.step()
        if it is None:
            break
        st = c.stats()
        assert st["gpu_blocks_held"] <= cap_gpu and st["cpu_blocks_held"] <= cap_cpu
        if it.mode == "two_batch" and (it.prefill or it.gpu_decode):
            two += 1
            # Balancing and hiding the CPU (step 4's inequalities)
            assert it.t_ca1 <= it.t_l0 + 1e-15 and it.t_ca0 <= it.t_l1 + it.t_ga0 + 1e-15
        if it.mode == "two_batch":
            assert it.n_tokens * it.t_gpu_only >= (len(it.prefill) + len(it.gpu_decode)) * it.t_two_batch
    st = c.stats()
    assert st["finished"] == len(reqs) and st["tokens"] == sum(r[2] for r in reqs)
    assert two > 0


def test_offloading_beats_gpu_only_when_gpu_memory_binds():
    """The paper's premise (Sec. 2.2): when GPU memory limits the batch and the
    host's bandwidth is within a small factor of the GPU's (an A10G-like GPU,
    600 GB/s, against a 200 GB/s host), the two-batch schedule serves more tokens
    per second than GPU-only."""
    ga, ca, tl = bandwidth_costs(gpu_bw=600e9, cpu_bw=200e9, flops=75e12)
    reqs = random_workload(11, 400, max_prompt=1500, max_out=400)
    res = {}
    for policy, cpu in (("neo", 200000), ("gpu_only", 0)):
        c = S.Scheduler(S.SchedConfig(num_layers=32, block_size=16, gpu_blocks=3800,
                                      cpu_blocks=cpu, max_batch_tokens=4096,
                                      t_ga=S.CostGrid(*ga), t_ca=S.CostGrid(*ca),
                                      t_l=S.CostCurve(*tl), policy=policy))
        for r in reqs:
            c.add(*r)
        c.run()
        st = c.stats()
        assert st["tokens"] == sum(r[2] for r in reqs)
        res[policy] = st["tokens"] / st["now"]
    assert res["neo"] > 1.05 * res["gpu_only"], res


def test_bad_configs_and_requests():
    ga, ca, tl = bandwidth_costs()
    base = dict(num_layers=1, block_size=16, gpu_blocks=10, cpu_blocks=10, max_batch_tokens=64,
                t_ga=S.CostGrid(*ga), t_ca=S.CostGrid(*ca), t_l=S.CostCurve(*tl))
    with pytest.raises(NeoError):
        S.Scheduler(S.SchedConfig(**{**base, "num_layers": 0}))
    with pytest.raises(KeyError):
        S.Scheduler(S.SchedConfig(**base, policy="other"))
    c = S.Scheduler(S.SchedConfig(**base))
    with pytest.raises(NeoError):
        c.add(0, 0, 5)
    with pytest.raises(NeoError):
        c.add(0, 5, 5, float("nan"))
    c.add(1, 16 * 25, 2)  # 25 blocks: fits neither cache
    with pytest.raises(NeoError, match="fits neither"):
        c.step()
