"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Bar (decode attention with bf16 q/K/V and fp32 accumulation): max abs error
<= 1e-2 and row-normwise relative error <= 2e-2 (max over (request, head) of
max_d |y - r| / max_d |r|); block-table indexing bit-exact (the gather kernel,
and bit-identical outputs under physical-block relabeling).
"""
import ctypes
import math
import sys
import time

import numpy as np
import pytest

import oracle
import paper_2411_01142_amd as neo
from parity_report import record
from paper_2411_01142_amd import workloads as W

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

ABS_TOL = 1e-2
REL_TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    neo.load_library()
    yield


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run(case, kv_layout="separate", kv_pad=0, **kw):
    q, k, v, bt, sl = case.to_torch("cuda", kv_layout=kv_layout, kv_pad=kv_pad)
    out = neo.decode_attention(q, k, v, bt, sl, scale=case.scale, **kw)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def errors(y, r, rows=None):
    """(max abs error, max row-normwise rel error) over the given flat rows."""
    y = y.reshape(-1, y.shape[-1])
    r = r.reshape(-1, r.shape[-1])
    if rows is not None:
        y, r = y[rows], r[rows]
    ae = np.abs(y.astype(np.float64) - r.astype(np.float64))
    denom = np.maximum(np.abs(r).max(axis=1), 1e-30)
    return float(ae.max()), float((ae.max(axis=1) / denom).max())


def assert_parity(y, r, label, rows=None):
    assert np.all(np.isfinite(y.reshape(-1, y.shape[-1])[rows] if rows is not None else y)), label
    ae, re = errors(y, r, rows)
    say(f"[parity] {label}: max_abs={ae:.3e} max_rel_rownorm={re:.3e}")
    assert ae <= ABS_TOL and re <= REL_TOL, (label, ae, re)
    return ae, re


# --------------------------------------------------------------------- indexing

@pytest.mark.parametrize("which", ["k", "v"])
@pytest.mark.parametrize("shuffle", [True, False])
def test_gather_is_bit_exact(which, shuffle):
    case = W.build_case([1, 15, 16, 17, 100, 333, 0, 64], 8, 4, 128, 16, seed=3,
                        shuffle=shuffle, extra_table_cols=2)
    q, k, v, bt, sl = case.to_torch("cuda")
    dense = neo.paged_gather(k if which == "k" else v, which, bt, sl)
    got = dense.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = oracle.paged_gather(case, which)
    assert got.shape == ref.shape and np.array_equal(got, ref)


def test_gather_config1_bit_exact():
    case = W.make_config(1, 1)
    q, k, v, bt, sl = case.to_torch("cuda")
    for which, cache in (("k", k), ("v", v)):
        got = neo.paged_gather(cache, which, bt, sl).view(torch.int16).cpu().numpy()
        assert np.array_equal(got.view(np.uint16), oracle.paged_gather(case, which))


def test_debug_validate_counts_bad_indices():
    case = W.build_case([20, 40, 5], 4, 2, 128, 16, seed=4, extra_table_cols=1)
    q, k, v, bt, sl = case.to_torch("cuda")
    assert neo.debug_validate(bt, sl, case.num_blocks) == 0
    bt2 = bt.clone()
    bt2[1, 2] = case.num_blocks       # in use (40 tokens -> blocks 0..2): counted
    bt2[2, 3] = 10 ** 6               # past request 2's one block: never read
    bt2[0, 0] = -5                    # request 0 gets a negative length below: unused
    sl2 = sl.clone()
    sl2[0] = -3                       # counted
    assert neo.debug_validate(bt2, sl2, case.num_blocks) == 2
    # A length past the table is counted, and clamping it brings the -1 padding
    # of that row into use (3 more entries).
    sl3 = sl.clone()
    sl3[2] = 16 * case.max_blocks_per_seq + 1
    assert neo.debug_validate(bt, sl3, case.num_blocks) == 1 + 3


# --------------------------------------------------------------------- parity, small

SMALL_LENS = [1, 15, 16, 17, 31, 33, 100, 257, 1000, 2]


@pytest.mark.parametrize("group", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("variant", ["valu", "mfma"])
@pytest.mark.parametrize("schedule", ["fused", "staged", "two_kernel"])
def test_small_cases_all_groups(group, variant, schedule):
    hkv = 2
    case = W.build_case(SMALL_LENS, hkv * group, hkv, 128, 16, seed=10 + group)
    ref = oracle.decode_attention(case)
    for slices in (0, 1, 7, 333, neo.MAX_SLICES):
        y = run(case, variant=variant, schedule=schedule, max_slices=slices)
        assert_parity(y, ref, f"G={group} {variant} {schedule} slices={slices}")


@pytest.mark.parametrize("variant", ["valu", "mfma"])
def test_softmax_range_stress(variant):
    # Outlier keys x8 and a large scale push scores far apart.
    case = W.build_case([50, 300, 700, 16], 32, 8, 128, 16, seed=5, k_outlier_frac=0.05,
                        scale=0.5)
    ref = oracle.decode_attention(case)
    assert_parity(run(case, variant=variant), ref, f"stress {variant}")


# --------------------------------------------------------------------- parity, configs

@pytest.mark.parametrize("cfg,seed", [
    (1, 1), (1, 101), (2, 2), (2, 102), (3, 3), (3, 103), (4, 4), (4, 104), (5, 5), (5, 105),
    (6, 6), (6, 106),
])
def test_config_parity(cfg, seed):
    # Every row of every workload at full size, in the launch the benchmark
    # times (default schedule and slice count): the large batches are the only
    # runs of the default plan's XCD-weighted slices and of cut pairs merged
    # across workgroups with many contributors. The oracle runs on all host
    # cores (a few hundred ms per batch on a 16-core host).
    say(f"[config] cfg={cfg} seed={seed}: generating")
    t0 = time.perf_counter()
    case = W.make_config(cfg, seed)
    say(f"[config] {case.name} B={case.batch} NB={case.num_blocks} sumL={case.total_tokens()} "
        f"(generated in {time.perf_counter() - t0:.1f} s)")
    y = run(case)
    t0 = time.perf_counter()
    ref = oracle.decode_attention(case)
    say(f"[config] oracle over {case.batch * case.num_q_heads} rows in "
        f"{time.perf_counter() - t0:.1f} s")
    ae, re = assert_parity(y, ref, f"{case.name} (all {case.batch * case.num_q_heads} rows)")
    record(f"{case.name}: all {case.batch * case.num_q_heads} rows, max_abs={ae:.2e} "
           f"max_rel_rownorm={re:.2e}")


# --------------------------------------------------------------------- block stride

@pytest.mark.parametrize("cfg", [2, 3, 4, 5, 6])
def test_interleaved_caches_full_size(cfg):
    # Both caches in one allocation, each block's K then V (the layout the
    # benchmark uses): every row against the oracle, and the same bits as two
    # dense caches (only the addresses differ).
    case = W.make_config(cfg, cfg)
    say(f"[layout] {case.name}: interleaved caches")
    a = run(case, kv_layout="interleaved")
    ae, re = assert_parity(a, oracle.decode_attention(case), f"{case.name} interleaved")
    record(f"{case.name}, K and V of each block in one run: max_abs={ae:.2e} "
           f"max_rel_rownorm={re:.2e}")
    assert np.array_equal(a, run(case))


@pytest.mark.parametrize("pad", [8, 2048, 12288 + 8])
@pytest.mark.parametrize("variant", ["mfma", "valu"])
@pytest.mark.parametrize("schedule", ["fused", "staged", "two_kernel"])
def test_block_stride_with_padding(pad, variant, schedule):
    # Strides that are not twice a block (padding after each block's K and V,
    # NaN-filled, never read), on every kernel family and launch.
    case = W.build_case([1, 15, 16, 17, 300, 1000, 0, 2500], 32, 8, 128, 16, seed=61)
    ref = oracle.decode_attention(case)
    a = run(case, kv_layout="interleaved", kv_pad=pad, variant=variant, schedule=schedule,
            max_slices=0 if schedule == "fused" else 97)
    assert_parity(a, ref, f"stride pad {pad} {variant} {schedule}")
    assert np.array_equal(a, run(case, variant=variant, schedule=schedule,
                                 max_slices=0 if schedule == "fused" else 97))


def test_binding_checks_cache_strides():
    case = W.build_case([10, 40], 8, 2, 128, 16, seed=62)
    q, k, v, bt, sl = case.to_torch("cuda", kv_layout="interleaved")
    with pytest.raises(ValueError, match="block stride"):
        neo.decode_attention(q, k, v.contiguous(), bt, sl)      # strides differ
    kt = k.transpose(3, 4)                                       # not dense within a block
    with pytest.raises(ValueError, match="dense"):
        neo.decode_attention(q, kt, v, bt, sl)
    kk, vv = neo.new_kv_cache(case.num_blocks, case.num_kv_heads)
    assert kk.stride(0) == vv.stride(0) == 2 * case.num_kv_heads * 2048
    assert vv.data_ptr() - kk.data_ptr() == case.num_kv_heads * 2048 * 2


# --------------------------------------------------------------------- edge cases

@pytest.mark.parametrize("variant", ["valu", "mfma"])
def test_empty_and_single_token_requests(variant):
    case = W.build_case([0, 1, 0, 17, 1, 0], 8, 2, 128, 16, seed=6)
    y = run(case, variant=variant)
    ref = oracle.decode_attention(case)
    assert np.all(y[[0, 2, 5]] == 0.0)
    # One token: its weight is exactly 1, so the output is that V row bit for bit.
    assert np.array_equal(y[1], ref[1]) and np.array_equal(y[4], ref[4])
    assert_parity(y, ref, f"empty/single {variant}")


def test_all_requests_empty():
    case = W.build_case([0, 0, 0], 8, 2, 128, 16, seed=7)
    q, k, v, bt, sl = case.to_torch("cuda")
    out = torch.full((3, 8, 128), float("nan"), device="cuda")
    neo.decode_attention(q, k, v, bt, sl, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 0).item()


def test_batch_of_one_long_request():
    case = W.build_case([9000], 32, 8, 128, 16, seed=8)
    ref = oracle.decode_attention(case)
    for variant in ("valu", "mfma"):
        assert_parity(run(case, variant=variant), ref, f"B=1 L=9000 {variant}")


def test_maximum_sizes_many_requests_and_one_very_long_request():
    # Sizes beyond every workload: 16384 requests of 0-64 tokens (the in-kernel
    # plan reads the lengths in 16 rounds of 1024 requests; most pairs are one
    # block), then one request of 131072 tokens at group 8 (8192 blocks per
    # pair, every slice of the default plan inside one of its 8 pairs, cut
    # pairs merged with ~128 contributors each). Every row against the oracle.
    rng = np.random.default_rng(51)
    lens = rng.integers(0, 65, 16384)
    lens[rng.random(16384) < 0.05] = 0
    case = W.build_case(lens.tolist(), 8, 2, 128, 16, seed=51)
    say(f"[max] B={case.batch} sumL={case.total_tokens()}")
    ref = oracle.decode_attention(case)
    for variant in ("mfma", "valu"):
        a = run(case, variant=variant)
        ae, re = assert_parity(a, ref, f"16384 short requests {variant}")
        record(f"16384 requests of 0-64 tokens ({variant}): max_abs={ae:.2e} max_rel_rownorm={re:.2e}")
    case = W.build_case([131072], 64, 8, 128, 16, seed=52)
    say(f"[max] B=1 L=131072 G=8")
    ref = oracle.decode_attention(case)
    for variant in ("mfma", "valu"):
        a = run(case, variant=variant)
        ae, re = assert_parity(a, ref, f"one request of 131072 tokens {variant}")
        record(f"one request of 131072 tokens, G=8 ({variant}): max_abs={ae:.2e} "
               f"max_rel_rownorm={re:.2e}")


def test_lengths_beyond_the_table_are_clamped():
    case = W.build_case([40, 64], 4, 2, 128, 16, seed=9)
    clamped = W.Case(**{**case.__dict__, "seq_lens": np.array([40, 64], np.int32)})
    over = W.Case(**{**case.__dict__, "seq_lens": np.array([40, 10 ** 6], np.int32)})
    assert np.array_equal(run(over), run(clamped))


# --------------------------------------------------------------------- invariants

def relabel(case, seed):
    rng = np.random.default_rng(seed)
    new_of_old = rng.permutation(case.num_blocks)
    k = np.empty_like(case.k_cache)
    v = np.empty_like(case.v_cache)
    k[new_of_old] = case.k_cache
    v[new_of_old] = case.v_cache
    bt = case.block_table.copy()
    m = bt >= 0
    bt[m] = new_of_old[bt[m]]
    return W.Case(**{**case.__dict__, "k_cache": k, "v_cache": v, "block_table": bt})


@pytest.mark.parametrize("variant", ["valu", "mfma"])
@pytest.mark.parametrize("schedule", ["fused", "staged", "two_kernel"])
def test_block_relabeling_is_bit_identical(variant, schedule):
    case = W.make_config(2, 2, batch_limit=24)
    a = run(case, variant=variant, schedule=schedule)
    b = run(relabel(case, 1), variant=variant, schedule=schedule)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("variant", ["valu", "mfma"])
@pytest.mark.parametrize("schedule", ["fused", "staged", "two_kernel"])
def test_repeated_runs_are_bit_identical(variant, schedule):
    # The fused schedule's arrival counters must be back at zero after each
    # call, or a later call would merge too early or never.
    case = W.make_config(5, 5, batch_limit=200)
    q, k, v, bt, sl = case.to_torch("cuda")
    ws = neo.new_workspace(case.batch, case.num_q_heads, case.num_kv_heads)
    first = neo.decode_attention(q, k, v, bt, sl, variant=variant, schedule=schedule,
                                 workspace=ws).clone()
    for i in range(30):
        again = neo.decode_attention(q, k, v, bt, sl, variant=variant, schedule=schedule,
                                     workspace=ws, max_slices=[0, 97, 0, 2000][i % 4])
        if i % 2 == 0:
            assert torch.equal(first, again)
        else:
            assert torch.max(torch.abs(first - again)).item() <= 1e-5


def test_request_permutation():
    case = W.build_case([5, 300, 17, 1000, 64, 1], 16, 4, 128, 16, seed=11)
    perm = np.random.default_rng(0).permutation(case.batch)
    pc = W.Case(**{**case.__dict__, "q": case.q[perm], "block_table": case.block_table[perm],
                   "seq_lens": case.seq_lens[perm]})
    for variant in ("valu", "mfma"):
        a = run(case, variant=variant, max_slices=1)
        b = run(pc, variant=variant, max_slices=1)
        assert np.array_equal(a[perm], b)        # no split: same arithmetic per request
        a = run(case, variant=variant)
        b = run(pc, variant=variant)
        assert np.max(np.abs(a[perm] - b)) <= 1e-5


def test_split_matches_unsplit_and_variants_agree():
    case = W.make_config(5, 105, batch_limit=300)
    base = run(case, variant="mfma", max_slices=1)
    for variant in ("valu", "mfma"):
        for schedule in ("fused", "staged", "two_kernel"):
            for slices in (0, 64, 1024, neo.MAX_SLICES):
                y = run(case, variant=variant, schedule=schedule, max_slices=slices)
                d = float(np.max(np.abs(y - base)))
                say(f"[split] {variant} {schedule} slices={slices}: max diff vs unsplit {d:.2e}")
                assert d <= 1e-5


def test_schedules_agree_bit_for_bit():
    # Same slices, same per-slice arithmetic and the same merge: only the
    # launch differs.
    case = W.make_config(3, 3, batch_limit=64)
    for variant in ("valu", "mfma"):
        a = run(case, variant=variant, schedule="fused")
        b = run(case, variant=variant, schedule="staged")
        c = run(case, variant=variant, schedule="two_kernel")
        assert np.array_equal(a, b) and np.array_equal(a, c)


@pytest.mark.parametrize("variant", ["valu", "mfma"])
def test_group_merge_mixes_contributor_counts(variant):
    # Pairs of 3-190 weighted positions cut by 8-40 slices of >= 8 positions:
    # cut pairs with 2..7 contributors, some inside one 4-wave workgroup
    # (merged through LDS), some across workgroups (merged through the
    # workspace). Fused must match the oracle and, slice for slice, the
    # two-kernel schedule bit for bit (same merge arithmetic).
    lens = [800, 40, 1600, 16, 500, 3000, 1, 257]
    case = W.build_case(lens, 8, 2, 128, 16, seed=31)
    ref = oracle.decode_attention(case)
    for slices in (8, 12, 16, 24, 40):
        a = run(case, variant=variant, schedule="fused", max_slices=slices)
        b = run(case, variant=variant, schedule="two_kernel", max_slices=slices)
        assert_parity(a, ref, f"group merge {variant} slices={slices}")
        assert np.array_equal(a, b), f"fused != two_kernel at {slices} slices"


@pytest.mark.parametrize("variant", ["valu", "mfma"])
def test_xcd_weighted_slices(variant):
    # On a part with eight XCDs, slice counts that are multiples of 8 with at
    # least 16 positions per slice weigh the slices by XCD (34 : 30 units):
    # 8, 16 and 24 slices here (~300, ~150 and ~100 positions), 256 slices
    # stay equal (~9). Every schedule must match the oracle and each other bit
    # for bit.
    lens = [3000, 40, 5000, 16, 2500, 7000, 1, 1257]
    case = W.build_case(lens, 8, 2, 128, 16, seed=37)
    ref = oracle.decode_attention(case)
    for slices in (8, 16, 24, 256):
        a = run(case, variant=variant, schedule="fused", max_slices=slices)
        b = run(case, variant=variant, schedule="two_kernel", max_slices=slices)
        c = run(case, variant=variant, schedule="staged", max_slices=slices)
        assert_parity(a, ref, f"xcd weights {variant} slices={slices}")
        assert np.array_equal(a, b) and np.array_equal(a, c), f"schedules differ at {slices}"


def test_batch_beyond_one_plan_round():
    # More than 1024 requests: the in-kernel plan reads seq_lens in rounds of
    # 1024 requests; slices must start in the right request in every round
    # (the staged schedule computes the same slices in a separate kernel).
    rng = np.random.default_rng(41)
    lens = rng.integers(0, 80, 2100)
    lens[rng.random(2100) < 0.1] = 0
    case = W.build_case(lens.tolist(), 8, 2, 128, 16, seed=41)
    ref = oracle.decode_attention(case)
    for variant in ("valu", "mfma"):
        a = run(case, variant=variant, schedule="fused")
        assert_parity(a, ref, f"batch 2100 {variant}")
        for schedule in ("staged", "two_kernel"):
            assert np.array_equal(a, run(case, variant=variant, schedule=schedule)), schedule


def random_case(i):
    rng = np.random.default_rng(1000 + i)
    hkv = int(rng.choice([1, 2, 4, 8]))
    group = int(rng.choice([1, 2, 4, 8, 16]))
    batch = int(rng.integers(1, 301))
    kind = i % 4  # short, long, mixed, exact block multiples
    if kind == 0:
        lens = rng.integers(0, 130, batch)
    elif kind == 1:
        lens = rng.integers(500, 3001, batch)
    elif kind == 2:
        lens = np.where(rng.random(batch) < 0.1, rng.integers(1000, 3001, batch),
                        rng.integers(0, 200, batch))
    else:
        lens = 16 * rng.integers(0, 120, batch)
    lens[rng.random(batch) < 0.05] = 0
    # Keep each case small enough for the oracle (a few M token-heads).
    while lens.sum() * hkv * group > 4_000_000 and batch > 1:
        batch //= 2
        lens = lens[:batch]
    slices = int(rng.choice([0, 0, 1, 3, 64, 256, 1024, neo.MAX_SLICES]))
    return W.build_case(lens.tolist(), hkv * group, hkv, 128, 16, seed=2000 + i,
                        poison=bool(i % 2)), slices


@pytest.mark.parametrize("i", range(120))
def test_random_shapes(i):
    # Seeded random batches: lengths from empty to 3000 tokens (short, long,
    # mixed and exact block multiples), groups 1-16, 1-8 kv heads, default or
    # forced slice counts (so long and short slices, workgroup-local and
    # workspace merges all occur). Fused must match the oracle and, slice for
    # slice, the two-kernel schedule bit for bit.
    case, slices = random_case(i)
    say(f"[random] case {i}: B={case.batch} Hq={case.num_q_heads} Hkv={case.num_kv_heads} "
        f"sumL={case.total_tokens()} slices={slices}")
    ref = oracle.decode_attention(case)
    a = run(case, variant="mfma", schedule="fused", max_slices=slices)
    assert_parity(a, ref, f"random {i}")
    b = run(case, variant="mfma", schedule="two_kernel", max_slices=slices)
    assert np.array_equal(a, b), f"random {i}: fused != two_kernel"


def mixed_random_case(i):
    """Shapes beyond the power-of-two kv head counts (3, 5, 16 kv heads), lengths
    around block multiples, runs of 0-1 token requests, equal lengths, a few long
    requests among short ones; random kernel family, launch schedule, slice cap
    and cache layout (two caches, or both in one buffer with or without padding)."""
    rng = np.random.default_rng(90000 + i)
    hkv = int(rng.choice([1, 2, 3, 4, 5, 8, 16]))
    group = int(rng.choice([1, 2, 4, 8, 16]))
    batch = int(rng.integers(1, 600))
    kind = i % 6
    if kind == 0:
        lens = rng.integers(0, 40, batch)
    elif kind == 1:
        lens = 16 * rng.integers(0, 200, batch) + rng.integers(-1, 2, batch)
    elif kind == 2:
        lens = np.where(rng.random(batch) < 0.05, rng.integers(2000, 12000, batch),
                        rng.integers(0, 100, batch))
    elif kind == 3:
        lens = rng.integers(1, 5000, batch)
    elif kind == 4:
        lens = np.full(batch, int(rng.integers(1, 3000)))
    else:
        lens = rng.integers(0, 2, batch)
    lens = np.clip(lens, 0, None)
    while int(lens.sum()) * hkv * group > 6_000_000 and batch > 1:
        batch = max(1, batch // 2)
        lens = lens[:batch]
    case = W.build_case(lens.tolist(), hkv * group, hkv, 128, 16, seed=91000 + i,
                        poison=bool(i % 2), extra_table_cols=int(rng.integers(0, 3)))
    variant = str(rng.choice(["mfma", "mfma", "valu"]))
    schedule = str(rng.choice(["fused", "fused", "staged", "two_kernel"]))
    slices = int(rng.choice([0, 0, 0, 1, 2, 5, 63, 200, 777, 1024, 2048, 4096]))
    layout = str(rng.choice(["separate", "interleaved"]))
    pad = int(rng.choice([0, 0, 8, 1024])) if layout == "interleaved" else 0
    return case, variant, schedule, slices, layout, pad


@pytest.mark.parametrize("i", range(60))
def test_mixed_random_shapes_and_launches(i):
    case, variant, schedule, slices, layout, pad = mixed_random_case(i)
    say(f"[mixed] case {i}: B={case.batch} Hq={case.num_q_heads} Hkv={case.num_kv_heads} "
        f"sumL={case.total_tokens()} {variant} {schedule} slices={slices} {layout} pad={pad}")
    ref = oracle.decode_attention(case)
    assert_parity(run(case, variant=variant, schedule=schedule, max_slices=slices,
                      kv_layout=layout, kv_pad=pad), ref,
                  f"mixed random {i}")


def large_random_case(i):
    rng = np.random.default_rng(5000 + i)
    hkv = int(rng.choice([1, 2, 4, 8]))
    group = [1, 2, 4, 8, 16][i % 5]
    batch = int(rng.integers(64, 2049))
    mix = i % 3  # uniform long, lognormal, few very long among short
    if mix == 0:
        lens = rng.integers(200, 6000, batch)
    elif mix == 1:
        lens = np.clip(np.round(1200 * np.exp(0.8 * rng.standard_normal(batch))), 1, 20000)
    else:
        lens = np.where(rng.random(batch) < 0.02, rng.integers(8000, 30000, batch),
                        rng.integers(0, 300, batch))
    lens = lens.astype(np.int64)
    # At most ~2M (token, kv head) pairs: ~1 GB of KV, a fraction of a second of oracle.
    while int(lens.sum()) * hkv > 2_000_000 and batch > 8:
        batch //= 2
        lens = lens[:batch]
    return W.build_case(lens.tolist(), hkv * group, hkv, 128, 16, seed=6000 + i, poison=True)


@pytest.mark.parametrize("i", range(15))
def test_large_random_batches(i):
    # Seeded batches at the workloads' scale with the groups they lack (1, 2, 16 beside 4 and
    # 8), 1-8 kv heads, up to 2048 requests, in the default launch: every row against the
    # oracle, and the fused schedule equal to the two-kernel one bit for bit.
    case = large_random_case(i)
    say(f"[large] case {i}: B={case.batch} Hq={case.num_q_heads} Hkv={case.num_kv_heads} "
        f"sumL={case.total_tokens()}")
    ref = oracle.decode_attention(case)
    a = run(case)
    ae, re = assert_parity(a, ref, f"large random {i}")
    record(f"large random {i} (B={case.batch}, G={case.group}, Hkv={case.num_kv_heads}): "
           f"max_abs={ae:.2e} max_rel_rownorm={re:.2e}")
    b = run(case, schedule="two_kernel")
    assert np.array_equal(a, b), f"large random {i}: fused != two_kernel"


def test_poisoned_slots_do_not_leak():
    lens = [1, 15, 17, 64, 99, 250]
    a = W.build_case(lens, 16, 4, 128, 16, seed=12, poison=True)
    b = W.build_case(lens, 16, 4, 128, 16, seed=12, poison=False)
    for variant in ("valu", "mfma"):
        ya, yb = run(a, variant=variant), run(b, variant=variant)
        assert np.all(np.isfinite(ya)) and np.array_equal(ya, yb)


def test_integer_coded_v_counts_every_position_once():
    L = [1, 2, 15, 16, 17, 255, 256, 257, 600, 4097]

    def vf(b, t, g):
        v = np.zeros(128, dtype=np.float32)
        v[0], v[1] = t % 256, t // 256
        return v
    case = W.build_case(L, 4, 2, 128, 16, seed=13, q_values=np.zeros((len(L), 4, 128)),
                        v_values=vf)
    for variant in ("valu", "mfma"):
        y = run(case, variant=variant).astype(np.float64)
        for b, n in enumerate(L):
            got = y[b, :, 0] + 256.0 * y[b, :, 1]
            assert np.max(np.abs(got - (n - 1) / 2.0)) <= 1e-6 * max(1.0, n), (variant, n)
            assert np.all(y[b, :, 2:] == 0.0)


def test_runs_on_a_side_stream():
    case = W.build_case([100, 200, 3], 8, 2, 128, 16, seed=14)
    ref = run(case)
    q, k, v, bt, sl = case.to_torch("cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = neo.decode_attention(q, k, v, bt, sl, scale=case.scale)
    s.synchronize()
    assert np.array_equal(out.cpu().numpy(), ref)


def test_workspace_init_through_the_c_abi():
    # A workspace full of stale bytes (arrival counters included) is cleared by
    # neo_decode_workspace_init on the call's stream; every later call then
    # leaves the counters at zero for the next one.
    case = W.build_case([100, 2000, 37, 900, 3000, 16], 16, 4, 128, 16, seed=16)
    ref = oracle.decode_attention(case)
    q, k, v, bt, sl = case.to_torch("cuda")
    lib = neo.load_library()
    n = neo.workspace_bytes(case.batch, case.num_q_heads, case.num_kv_heads)
    ws = torch.full((n,), 0x5A, dtype=torch.uint8, device="cuda")
    out = torch.empty((case.batch, case.num_q_heads, 128), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    sh = ctypes.c_void_p(s.cuda_stream)
    assert lib.neo_decode_workspace_init(ws.data_ptr(), n, sh) == 0
    for i in range(3):
        rc = lib.neo_decode_attention(q.data_ptr(), k.data_ptr(), v.data_ptr(), bt.data_ptr(),
                                      sl.data_ptr(), case.num_q_heads, case.num_kv_heads, 128,
                                      16, float(case.scale), out.data_ptr(), case.batch,
                                      case.max_blocks_per_seq, case.num_blocks, ws.data_ptr(),
                                      n, sh)
        assert rc == 0, lib.neo_last_error()
        s.synchronize()
        assert_parity(out.cpu().numpy(), ref, f"workspace init, call {i}")


def test_cached_workspace_is_cleared_on_the_call_stream():
    # The binding's cached workspace for a new stream is allocated in that
    # stream's pool and cleared on it, so the first call there sees zeroed
    # counters even when the stream starts with no dependency on another.
    case = W.build_case([700, 1500, 9, 2500], 32, 8, 128, 16, seed=17)
    ref = oracle.decode_attention(case)
    q, k, v, bt, sl = case.to_torch("cuda")
    torch.cuda.synchronize()
    for _ in range(2):
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            out = neo.decode_attention(q, k, v, bt, sl, scale=case.scale)
        s.synchronize()
        assert_parity(out.cpu().numpy(), ref, "cached workspace on a new stream")


def test_binding_errors_are_raised():
    case = W.build_case([10], 8, 2, 128, 16, seed=15)
    q, k, v, bt, sl = case.to_torch("cuda")
    ws = torch.empty(1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(neo.NeoError) as ei:
        neo.decode_attention(q, k, v, bt, sl, workspace=ws)
    assert ei.value.status == 3
    with pytest.raises(neo.NeoError):
        neo.decode_attention(q, k, v, bt, sl, scale=math.inf)


def test_matches_golden_fixture():
    import json
    import os
    here = os.path.dirname(os.path.abspath(__file__))
    rec = json.load(open(os.path.join(here, "golden", "oracle_small.json")))
    s = rec["spec"]
    case = W.build_case(s["seq_lens"], s["num_q_heads"], s["num_kv_heads"], s["head_dim"],
                        s["block_size"], seed=s["seed"])
    expect = np.array([[[float.fromhex(x) for x in row] for row in head]
                       for head in rec["out_f32_hex"]], dtype=np.float32)
    for variant in ("valu", "mfma"):
        for schedule in ("staged", "fused", "two_kernel"):
            assert_parity(run(case, variant=variant, schedule=schedule), expect,
                          f"golden {variant} {schedule}")
