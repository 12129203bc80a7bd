"""Parity of the host-CPU decode attention (the library's CPU path) against the
fp64 oracle. Runs without a GPU: the CPU path is host code in the same library.

Bar: as for the GPU path, max abs error <= 1e-2 and row-normwise relative error
<= 2e-2; single-token requests bit-exact (their weight is exactly 1);
physical-block relabeling bit-identical. Every instruction-set path this CPU
has is tested; the others are skipped with the reason.
"""
import ctypes
import json
import os

import numpy as np
import pytest

import oracle
import paper_2411_01142_amd as neo
from kv_cases import drop_last_tokens
from paper_2411_01142_amd import workloads as W

ABS_TOL = 1e-2
REL_TOL = 2e-2
HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(neo.library_path()):
        import __graft_entry__
        __graft_entry__.build()
    return neo.load_library()


def has(isa):
    if isa == "generic":
        return True
    best = neo.cpu_best_isa()
    flags = open("/proc/cpuinfo").read()
    need = {"avx512": ["avx512f", "avx512bw", "avx512vl", "avx512dq"],
            "avx512_bf16": ["avx512f", "avx512bw", "avx512vl", "avx512dq", "avx512_bf16"]}[isa]
    return best == isa or all(f" {f}" in flags for f in need)


ISAS = [pytest.param(i, marks=pytest.mark.skipif(not has(i), reason=f"CPU lacks {i}"))
        for i in ("generic", "avx512", "avx512_bf16")]


def run(case, isa, threads=0, **kw):
    return neo.cpu_decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                    case.seq_lens, case.scale, num_threads=threads, isa=isa, **kw)


def assert_parity(y, r, label):
    y = y.reshape(-1, y.shape[-1]).astype(np.float64)
    r = r.reshape(-1, r.shape[-1]).astype(np.float64)
    assert np.all(np.isfinite(y)), label
    ae = np.abs(y - r)
    rel = (ae.max(axis=1) / np.maximum(np.abs(r).max(axis=1), 1e-30)).max()
    assert ae.max() <= ABS_TOL and rel <= REL_TOL, (label, ae.max(), rel)
    return ae.max()


@pytest.mark.parametrize("isa", ISAS)
@pytest.mark.parametrize("group", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("threads", [1, 3, 8])
def test_small_cases_all_groups(isa, group, threads):
    hkv = 2 if group < 16 else 1
    case = W.build_case([1, 17, 300, 1000, 0, 33, 16, 130], hkv * group, hkv, 128, 16,
                        seed=group * 10 + threads)
    err = assert_parity(run(case, isa, threads), oracle.decode_attention(case),
                        f"{isa} G={group} T={threads}")
    assert err < 1e-4  # fp32 accumulation of exact bf16 inputs


@pytest.mark.parametrize("isa", ISAS)
def test_softmax_range_stress(isa):
    case = W.build_case([700, 64, 2048], 32, 8, 128, 16, seed=9, k_outlier_frac=0.05,
                        k_outlier_mult=16)
    assert_parity(run(case, isa, 5), oracle.decode_attention(case), f"{isa} outliers")


@pytest.mark.parametrize("isa", ISAS)
def test_config2_full_batch(isa):
    case = W.make_config(2, 102)
    assert_parity(run(case, isa), oracle.decode_attention(case), f"{isa} cfg2")


@pytest.mark.parametrize("isa", ISAS)
def test_skewed_batch_splits_long_requests(isa):
    # a few long requests among many short ones: the long pairs are cut between threads
    case = W.build_case([4096, 16, 20, 3000] + [40] * 60, 32, 8, 128, 16, seed=4)
    ref = oracle.decode_attention(case)
    for threads in (2, 7, 16, 64):
        assert_parity(run(case, isa, threads), ref, f"{isa} T={threads}")


@pytest.mark.parametrize("isa", ISAS)
def test_single_token_requests_are_exact(isa):
    case = W.build_case([1, 1, 1, 1], 8, 2, 128, 16, seed=3)
    y = run(case, isa, 2)
    assert np.array_equal(y, oracle.decode_attention(case))


@pytest.mark.parametrize("isa", ISAS)
def test_empty_requests_and_batches(isa):
    case = W.build_case([0, 5, 0], 8, 2, 128, 16, seed=2)
    y = run(case, isa, 2, out=np.full((3, 8, 128), 7.0, np.float32))
    assert np.all(y[0] == 0) and np.all(y[2] == 0)
    assert_parity(y, oracle.decode_attention(case), "empty rows")
    case = W.build_case([0, 0], 8, 2, 128, 16, seed=2)
    assert np.all(run(case, isa) == 0)


@pytest.mark.parametrize("isa", ISAS)
def test_lengths_beyond_the_table_are_clamped(isa):
    case = W.build_case([40, 20], 8, 2, 128, 16, seed=8, poison=False)
    spare = sorted(set(range(case.num_blocks)) - set(case.block_table.ravel().tolist()))
    case.block_table[1, 2] = spare[0]
    case.seq_lens[:] = [40, 48]  # the table's three columns
    clamped = run(case, isa, 2)
    assert_parity(clamped, oracle.decode_attention(case), "clamped")
    case.seq_lens[:] = [40, 5000]  # clamped to the same 48 tokens
    assert np.array_equal(run(case, isa, 2), clamped)


@pytest.mark.parametrize("isa", ISAS)
def test_poisoned_slots_do_not_leak(isa):
    case = W.build_case([3, 19, 45], 8, 2, 128, 16, seed=12, poison=True)
    y = run(case, isa, 3)
    assert np.all(np.isfinite(y))
    assert_parity(y, oracle.decode_attention(case), "poison")


@pytest.mark.parametrize("isa", ISAS)
def test_block_relabeling_is_bit_identical(isa):
    case = W.build_case([100, 37, 260], 16, 4, 128, 16, seed=21)
    y0 = run(case, isa, 4)
    perm = np.random.default_rng(5).permutation(case.num_blocks)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(len(perm))
    relabeled = W.Case(**{**case.__dict__, "k_cache": case.k_cache[inv].copy(),
                          "v_cache": case.v_cache[inv].copy(),
                          "block_table": np.where(case.block_table >= 0,
                                                  perm[np.maximum(case.block_table, 0)],
                                                  -1).astype(np.int32)})
    assert np.array_equal(run(relabeled, isa, 4), y0)


@pytest.mark.parametrize("isa", ISAS)
def test_thread_counts_agree(isa):
    case = W.build_case([900, 5, 1500, 64], 32, 8, 128, 16, seed=30)
    ys = [run(case, isa, t) for t in (1, 2, 6, 13)]
    for y in ys[1:]:
        assert np.abs(y - ys[0]).max() <= 1e-5


def test_paths_agree():
    case = W.build_case([333, 1024, 17], 32, 8, 128, 16, seed=31)
    ref = run(case, "generic", 3)
    for isa in ("avx512", "avx512_bf16"):
        if has(isa):
            assert np.abs(run(case, isa, 3) - ref).max() <= 2e-5


def test_matches_golden_fixture():
    rec = json.load(open(os.path.join(HERE, "golden", "oracle_small.json")))
    s = rec["spec"]
    case = W.build_case(s["seq_lens"], s["num_q_heads"], s["num_kv_heads"], s["head_dim"],
                        s["block_size"], seed=s["seed"])
    expect = np.array([[[float.fromhex(x) for x in row] for row in head]
                       for head in rec["out_f32_hex"]], dtype=np.float32)
    assert_parity(run(case, "auto", 2), expect, "golden")


def test_bad_block_id_is_an_error_not_a_crash():
    case = W.build_case([40, 20], 8, 2, 128, 16, seed=8)
    case.block_table[1, 0] = case.num_blocks
    with pytest.raises(neo.NeoError, match="outside"):
        run(case, "auto")
    case.block_table[1, 0] = -1
    with pytest.raises(neo.NeoError, match="outside"):
        run(case, "auto")


def test_argument_errors(lib):
    case = W.build_case([4], 8, 2, 128, 16, seed=1)
    with pytest.raises(ValueError):
        neo.cpu_decode_attention(case.q.astype(np.float32), case.k_cache, case.v_cache,
                                 case.block_table, case.seq_lens)
    P = ctypes.c_void_p
    x = case.q.ctypes.data
    base = [x, x, x, x, x, 8, 2, 128, 16, 0.1, x, 1, 1, 4, 0, 0]

    def call(**kw):
        a = list(base)
        names = ["q", "k", "v", "t", "l", "hq", "hkv", "d", "bs", "scale", "out", "batch",
                 "mbps", "nb", "threads", "isa"]
        for k, v in kw.items():
            a[names.index(k)] = v
        return lib.neo_cpu_decode_attention_ex(*a)
    assert call(hq=7) == 1
    assert call(hq=6) == 2  # group 3
    assert call(hq=24, hkv=8) == 2
    assert call(d=64) == 2
    assert call(bs=32) == 2
    assert call(scale=float("nan")) == 1
    assert call(isa=9) == 2
    assert call(threads=-1) == 1
    assert call(q=None) == 1
    assert call(mbps=0) == 1
    assert call(batch=-1) == 1
    assert call(batch=0, q=None, k=None) == 0


def test_read_probe_sums_the_buffer():
    buf = np.arange(1 << 16, dtype=np.float32) % 7
    assert neo.cpu_read_probe(buf, 3) == pytest.approx(float(buf.sum()), rel=1e-6)
    with pytest.raises(neo.NeoError):
        neo.cpu_read_probe(np.ones(10, np.float32))


@pytest.mark.parametrize("hkv", [1, 2, 8])
def test_cpu_append_restores_the_dropped_token(hkv):
    case = W.build_case([1, 5, 16, 17, 40, 0, 33], 2 * hkv, hkv, 128, 16, seed=hkv)
    dropped, k_new, v_new = drop_last_tokens(case)
    neo.cpu_kv_append(dropped.k_cache, dropped.v_cache, k_new, v_new, case.block_table,
                      case.seq_lens)
    assert np.array_equal(dropped.k_cache, case.k_cache)
    assert np.array_equal(dropped.v_cache, case.v_cache)


def test_cpu_append_matches_oracle_with_clamps_and_bad_ids():
    case = W.build_case([20, 9, 16, 0], 2, 1, 128, 16, seed=6)
    case.seq_lens[:] = [20, 9, 1000, 0]
    case.block_table[2, 1] = 1
    case.block_table[1, 0] = case.num_blocks + 3
    rng = np.random.default_rng(4)
    k_new = rng.integers(0, 1 << 16, size=(4, 1, 128), dtype=np.uint16)
    v_new = rng.integers(0, 1 << 16, size=(4, 1, 128), dtype=np.uint16)
    k, v = case.k_cache.copy(), case.v_cache.copy()
    neo.cpu_kv_append(k, v, k_new, v_new, case.block_table, case.seq_lens)
    oracle.kv_append(case, k_new, v_new)
    assert np.array_equal(k, case.k_cache) and np.array_equal(v, case.v_cache)
