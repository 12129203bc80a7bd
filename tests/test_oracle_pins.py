"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Decode attention is defined in the paper (Sec. 2.1-2.2): the new token of a
request attends over every token in its paged KV cache; query heads share KV
heads in groups (GQA, Sec. 4); the block-granular split is aggregated per
request (Sec. 4). The paper prints no attention values, so the pins are a
library routine (torch's fp64 scaled-dot-product attention on dense tensors
built by the input generator's own layout code), brute force over a grid of
tiny shapes, closed forms, invariants and the exact split/merge identity.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2411_01142_amd import workloads as W


def dense_kv(case):
    """Per-request dense K/V float64 [Hkv][L][D] via the generator's unpack (not the oracle)."""
    k_log, v_log = case.logical_kv()
    k_log = W.bf16_to_f32(k_log).astype(np.float64)
    v_log = W.bf16_to_f32(v_log).astype(np.float64)
    out = []
    for b in range(case.batch):
        L = int(case.seq_lens[b])
        t = np.arange(L)
        p = case.block_table[b, t // case.block_size]
        o = t % case.block_size
        out.append((k_log[p, :, o, :].transpose(1, 0, 2), v_log[p, :, o, :].transpose(1, 0, 2)))
    return out


def torch_sdpa(case):
    """Library routine: torch CPU float64 scaled_dot_product_attention per request."""
    q = W.bf16_to_f32(case.q).astype(np.float64)
    G = case.group
    res = np.zeros((case.batch, case.num_q_heads, case.head_dim))
    for b, (K, V) in enumerate(dense_kv(case)):
        if K.shape[1] == 0:
            continue
        qt = torch.from_numpy(q[b]).reshape(1, case.num_q_heads, 1, case.head_dim)
        Kt = torch.from_numpy(np.ascontiguousarray(K)).repeat_interleave(G, dim=0)[None]
        Vt = torch.from_numpy(np.ascontiguousarray(V)).repeat_interleave(G, dim=0)[None]
        o = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, scale=case.scale)
        res[b] = o[0, :, 0, :].numpy()
    return res


# ----------------------------------------------------------------- library routine

@pytest.mark.parametrize("lens,hq,hkv,seed", [
    ([5, 17, 33], 4, 2, 0),
    ([64, 1, 100, 16], 8, 2, 1),
    ([200, 37], 8, 1, 2),
    ([48, 49, 47], 16, 16, 3),
])
def test_matches_torch_fp64_sdpa(lens, hq, hkv, seed):
    case = W.build_case(lens, hq, hkv, 128, 16, seed=seed)
    _, o64 = oracle.decode_attention(case, want_f64=True)
    ref = torch_sdpa(case)
    assert np.max(np.abs(o64 - ref)) <= 1e-12


def test_brute_force_tiny_grid():
    """Every combination of tiny shapes, random tables, against the library route."""
    rng = np.random.default_rng(7)
    n = 0
    for B, hkv, G, D, bs in itertools.product([1, 2, 3], [1, 2], [1, 2, 4], [8, 16], [1, 2, 4]):
        lens = rng.integers(0, 10, size=B)
        case = W.build_case(lens, hkv * G, hkv, D, bs, seed=int(rng.integers(1 << 30)),
                            scale=float(rng.uniform(0.05, 1.0)))
        _, o64 = oracle.decode_attention(case, want_f64=True)
        ref = torch_sdpa(case)
        for b in range(B):
            if lens[b] == 0:
                assert np.all(o64[b] == 0.0)
            else:
                assert np.max(np.abs(o64[b] - ref[b])) <= 1e-12, (B, hkv, G, D, bs, lens)
        n += 1
    assert n == 3 * 2 * 3 * 2 * 3


# ----------------------------------------------------------------- closed forms

def test_single_token_returns_its_v_row_exactly():
    rng = np.random.default_rng(11)
    case = W.build_case([1, 1, 1], 8, 2, 128, 16, seed=11)
    out = oracle.decode_attention(case)
    _, v_log = case.logical_kv()
    for b in range(3):
        p = case.block_table[b, 0]
        for h in range(8):
            assert np.array_equal(out[b, h], W.bf16_to_f32(v_log[p, h // 4, 0]))
    del rng


def test_zero_query_gives_exact_mean_of_small_integer_v():
    rng = np.random.default_rng(12)
    L = [3, 16, 17, 45]
    vals = {(b, t, g): rng.integers(-8, 9, size=128).astype(np.float32)
            for b in range(4) for t in range(L[b]) for g in range(2)}
    case = W.build_case(L, 4, 2, 128, 16, seed=12, q_values=np.zeros((4, 4, 128)),
                        v_values=lambda b, t, g: vals[(b, t, g)])
    _, o64 = oracle.decode_attention(case, want_f64=True)
    for b in range(4):
        for h in range(4):
            g = h // 2
            for d in (0, 5, 127):
                exact = Fraction(int(sum(vals[(b, t, g)][d] for t in range(L[b]))), L[b])
                assert o64[b, h, d] == float(exact)


def test_constant_v_returns_the_constant():
    case = W.build_case([7, 31, 90], 8, 4, 128, 16, seed=13,
                        v_values=lambda b, t, g: np.full(128, 0.625, dtype=np.float32))
    _, o64 = oracle.decode_attention(case, want_f64=True)
    assert np.max(np.abs(o64 - 0.625)) <= 1e-15


def test_two_tokens_sigmoid_form():
    # q = a e0, k_t = x_t e0: s_t = scale * a * x_t exactly (all values exact in bf16).
    a, x1, x2, scale = 1.5, 2.0, -0.75, 0.5
    v1 = np.linspace(-1, 1, 128).astype(np.float32)
    v2 = np.cos(np.arange(128)).astype(np.float32)
    v1b, v2b = W.bf16_to_f32(W.to_bf16(v1)), W.bf16_to_f32(W.to_bf16(v2))
    q = np.zeros((1, 1, 128), dtype=np.float32)
    q[0, 0, 0] = a

    def kf(b, t, g):
        k = np.zeros(128, dtype=np.float32)
        k[0] = x1 if t == 0 else x2
        return k
    case = W.build_case([2], 1, 1, 128, 16, seed=14, q_values=q, k_values=kf,
                        v_values=lambda b, t, g: v1 if t == 0 else v2, scale=scale)
    _, o64 = oracle.decode_attention(case, want_f64=True)
    s1, s2 = scale * a * x1, scale * a * x2
    sig = lambda z: 1.0 / (1.0 + math.exp(-z))
    expect = sig(s1 - s2) * v1b.astype(np.float64) + sig(s2 - s1) * v2b.astype(np.float64)
    assert np.max(np.abs(o64[0, 0] - expect)) <= 1e-15


def test_dominant_score_selects_that_row():
    L = 50
    q = np.zeros((1, 2, 128), dtype=np.float32)
    q[0, :, 0] = 8.0

    def kf(b, t, g):
        k = np.zeros(128, dtype=np.float32)
        k[0] = 64.0 if t == 23 else 0.25
        return k
    case = W.build_case([L], 2, 1, 128, 16, seed=15, q_values=q, k_values=kf, scale=0.125)
    _, o64 = oracle.decode_attention(case, want_f64=True)
    _, v_log = case.logical_kv()
    p = case.block_table[0, 23 // 16]
    row = W.bf16_to_f32(v_log[p, 0, 23 % 16]).astype(np.float64)
    # s(23) = 64, others = 0.25: the gap is 63.75 >= 40.
    rows = [W.bf16_to_f32(v_log[case.block_table[0, t // 16], 0, t % 16]) for t in range(L)]
    vmax = float(np.max(np.abs(np.stack(rows))))
    bound = (L - 1) * math.exp(-63.75) * vmax * 2
    assert np.max(np.abs(o64[0, 0] - row)) <= max(bound, 1e-300)


# ----------------------------------------------------------------- invariants

@pytest.mark.parametrize("seed", [0, 1])
def test_softmax_weights_sum_to_one(seed):
    case = W.build_case([1, 16, 17, 300], 8, 2, 128, 16, seed=seed, k_outlier_frac=0.05)
    for b in range(case.batch):
        for h in (0, 3, 7):
            w = oracle.softmax_weights(case, b, h)
            assert w.shape[0] == case.seq_lens[b]
            assert np.all(w >= 0)
            assert abs(w.sum() - 1.0) <= 1e-12


@pytest.mark.parametrize("lens,hq,hkv,seed", [
    ([1, 16, 17, 300], 8, 2, 0),
    ([5, 64, 129], 16, 4, 1),
    ([40, 2], 4, 4, 2),
])
def test_softmax_weights_match_torch_softmax(lens, hq, hkv, seed):
    # The weights themselves, position by position, against torch's fp64
    # softmax of scale * q K^T over the dense K the generator's own layout code
    # unpacks (so a permuted, shifted or mis-indexed weight vector fails).
    case = W.build_case(lens, hq, hkv, 128, 16, seed=seed, k_outlier_frac=0.05)
    q = W.bf16_to_f32(case.q).astype(np.float64)
    G = case.group
    for b, (K, _) in enumerate(dense_kv(case)):
        for h in range(hq):
            s = torch.from_numpy(K[h // G] @ q[b, h]) * case.scale
            ref = torch.softmax(s, dim=0).numpy()
            w = oracle.softmax_weights(case, b, h)
            assert w.shape == ref.shape
            assert np.max(np.abs(w - ref)) <= 1e-13, (b, h)
            # The largest weight sits at the largest score.
            assert int(np.argmax(w)) == int(torch.argmax(s))


def _relabel(case, rng):
    """Move every physical block to a new id; rewrite the table to match."""
    nb = case.num_blocks
    new_of_old = rng.permutation(nb)
    k = np.empty_like(case.k_cache)
    v = np.empty_like(case.v_cache)
    k[new_of_old] = case.k_cache
    v[new_of_old] = case.v_cache
    bt = case.block_table.copy()
    m = bt >= 0
    bt[m] = new_of_old[bt[m]]
    return W.Case(q=case.q, k_cache=k, v_cache=v, block_table=bt, seq_lens=case.seq_lens,
                  num_q_heads=case.num_q_heads, num_kv_heads=case.num_kv_heads,
                  head_dim=case.head_dim, block_size=case.block_size, scale=case.scale)


def test_block_relabeling_is_bit_identical():
    rng = np.random.default_rng(21)
    case = W.build_case([5, 16, 160, 77], 8, 2, 128, 16, seed=21)
    a = oracle.decode_attention(case, want_f64=True)[1]
    b = oracle.decode_attention(_relabel(case, rng), want_f64=True)[1]
    assert np.array_equal(a, b)


def test_request_permutation_permutes_outputs():
    rng = np.random.default_rng(22)
    case = W.build_case([5, 16, 160, 77, 1], 8, 4, 128, 16, seed=22)
    perm = rng.permutation(case.batch)
    pc = W.Case(q=case.q[perm], k_cache=case.k_cache, v_cache=case.v_cache,
                block_table=case.block_table[perm], seq_lens=case.seq_lens[perm],
                num_q_heads=8, num_kv_heads=4, head_dim=128, block_size=16, scale=case.scale)
    a = oracle.decode_attention(case, want_f64=True)[1]
    b = oracle.decode_attention(pc, want_f64=True)[1]
    assert np.array_equal(a[perm], b)


def test_integer_coded_v_uses_every_position_once():
    """q = 0 makes every weight exactly 1/L; V dim0 = t mod 256, dim1 = t // 256."""
    L = [1, 2, 15, 16, 17, 255, 256, 257, 600]

    def vf(b, t, g):
        v = np.zeros(128, dtype=np.float32)
        v[0], v[1] = t % 256, t // 256
        return v
    case = W.build_case(L, 2, 1, 128, 16, seed=23, q_values=np.zeros((len(L), 2, 128)),
                        v_values=vf)
    _, o64 = oracle.decode_attention(case, want_f64=True)
    for b, n in enumerate(L):
        e0 = Fraction(sum(t % 256 for t in range(n)), n)
        e1 = Fraction(sum(t // 256 for t in range(n)), n)
        assert o64[b, 0, 0] == float(e0) and o64[b, 0, 1] == float(e1)
        assert e0 + 256 * e1 == Fraction(n - 1, 2)
        assert np.all(o64[b, :, 2:] == 0.0)


def test_gqa_head_map_is_contiguous_groups():
    c = [0.5, -2.0, 4.0, 0.25]
    case = W.build_case([9, 40], 16, 4, 128, 16, seed=24,
                        v_values=lambda b, t, g: np.full(128, c[g], dtype=np.float32))
    _, o64 = oracle.decode_attention(case, want_f64=True)
    for h in range(16):
        assert np.max(np.abs(o64[:, h, :] - c[h // 4])) <= 1e-15


def test_split_and_lse_merge_equals_unsplit():
    rng = np.random.default_rng(25)
    case = W.build_case([16, 33, 300, 1000], 8, 2, 128, 16, seed=25, k_outlier_frac=0.02)
    _, o64 = oracle.decode_attention(case, want_f64=True)
    for b in range(case.batch):
        L = int(case.seq_lens[b])
        nblk = (L + 15) // 16
        for h in (0, 5):
            for _ in range(3):
                k = int(rng.integers(1, nblk + 1))
                cuts = sorted(set(int(x) for x in rng.integers(1, nblk, size=k - 1))) if nblk > 1 else []
                edges = [0] + [c * 16 for c in cuts] + [L]
                parts = [oracle.partial_attention(case, b, h, edges[i], edges[i + 1])
                         for i in range(len(edges) - 1)]
                merged, lse = oracle.lse_merge(np.stack([p[0] for p in parts]),
                                               np.array([p[1] for p in parts]))
                full, full_lse = oracle.partial_attention(case, b, h, 0, L)
                assert np.max(np.abs(merged - o64[b, h])) <= 1e-12
                assert np.max(np.abs(full - o64[b, h])) <= 1e-12
                assert abs(lse - full_lse) <= 1e-12 * max(1.0, abs(full_lse))


def test_lse_merge_closed_form():
    # Two partials with lse ln 1 and ln 3: weights 1/4 and 3/4.
    o = np.array([[1.0, 0.0], [0.0, 2.0]])
    out, lse = oracle.lse_merge(o, np.array([0.0, math.log(3.0)]))
    assert np.allclose(out, [0.25, 1.5], atol=1e-15, rtol=0)
    assert abs(lse - math.log(4.0)) <= 1e-15
    out, lse = oracle.lse_merge(o, np.array([-math.inf, 2.0]))
    assert np.array_equal(out, [0.0, 2.0]) and lse == 2.0


def test_power_of_two_rescaling_of_q_and_scale_is_bit_identical():
    case = W.build_case([30, 100], 8, 2, 128, 16, seed=26)
    a = oracle.decode_attention(case, want_f64=True)[1]
    q8 = W.to_bf16(W.bf16_to_f32(case.q) * np.float32(8.0))
    b = oracle.decode_attention(case, q=q8, scale=case.scale / 8.0, want_f64=True)[1]
    assert np.array_equal(a, b)


def test_poisoned_tails_and_spares_are_never_read():
    lens = [1, 15, 17, 64, 99]
    a = W.build_case(lens, 8, 2, 128, 16, seed=27, poison=True)
    b = W.build_case(lens, 8, 2, 128, 16, seed=27, poison=False)
    oa = oracle.decode_attention(a, want_f64=True)[1]
    ob = oracle.decode_attention(b, want_f64=True)[1]
    assert np.all(np.isfinite(oa))
    assert np.array_equal(oa, ob)


def test_zero_length_request_gives_zero_row():
    case = W.build_case([0, 5, 0], 4, 2, 128, 16, seed=28)
    out = oracle.decode_attention(case)
    assert np.all(out[0] == 0) and np.all(out[2] == 0) and np.any(out[1] != 0)


def test_oracle_gather_matches_generator_layout():
    case = W.build_case([1, 16, 17, 70], 4, 2, 128, 16, seed=29)
    k_log, v_log = case.logical_kv()
    for which, log in (("k", k_log), ("v", v_log)):
        dense = oracle.paged_gather(case, which)
        rows = []
        for b in range(case.batch):
            for t in range(int(case.seq_lens[b])):
                rows.append(log[case.block_table[b, t // 16], :, t % 16, :])
        assert np.array_equal(dense, np.stack(rows))


def test_bad_block_id_is_reported():
    case = W.build_case([20], 2, 1, 128, 16, seed=30)
    case.block_table[0, 1] = case.num_blocks + 3
    with pytest.raises(oracle.OracleError):
        oracle.decode_attention(case)


# ----------------------------------------------------------------- input generator

def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(31)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 7,
                        np.array([1.00390625, 1.01171875, -3.0e38, 1e-40, 0.0, -0.0], np.float32)])
    ours = W.to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_config_lengths_follow_recipes():
    L1 = W.config_seq_lens(1, 1)
    assert L1.shape == (4,) and L1.min() >= 64 and L1.max() <= 512
    L3 = W.config_seq_lens(3, 3)
    assert L3.shape == (256,) and L3.min() >= 128 and L3.max() <= 8192
    assert 1200 <= np.median(L3) <= 1800
    L5 = W.config_seq_lens(5, 5)
    assert L5.shape == (1024,) and int((L5 == 32768).sum()) == 8
    assert L5[L5 != 32768].max() <= 256 and L5.min() >= 16


# ----------------------------------------------------------------- regression fixture

def test_oracle_reproduces_golden_fixture():
    import json
    import os
    here = os.path.dirname(os.path.abspath(__file__))
    rec = json.load(open(os.path.join(here, "golden", "oracle_small.json")))
    s = rec["spec"]
    case = W.build_case(s["seq_lens"], s["num_q_heads"], s["num_kv_heads"], s["head_dim"],
                        s["block_size"], seed=s["seed"])
    expect = np.array([[[float.fromhex(x) for x in row] for row in head]
                       for head in rec["out_f32_hex"]], dtype=np.float32)
    assert np.array_equal(oracle.decode_attention(case), expect)
