"""Pins of the oracle's cache operations (append and block copy), CPU only.

Append is pinned to the generator's own packing: dropping each request's last
token from a generated case and appending it again must restore the caches
byte for byte. Block copy is pinned by brute force over small caches and by a
swap-out / swap-in round trip that must leave attention bit-identical.
"""
import numpy as np
import pytest

import oracle
from paper_2411_01142_amd import workloads as W
from kv_cases import POISON, drop_last_tokens, last_token_slots, used_blocks

@pytest.mark.parametrize("seed", [0, 1])
@pytest.mark.parametrize("hkv", [1, 2, 8])
def test_append_restores_the_dropped_token(seed, hkv):
    case = W.build_case([1, 5, 16, 17, 40, 0, 33], 2 * hkv, hkv, 128, 16, seed=seed)
    dropped, k_new, v_new = drop_last_tokens(case)
    assert not np.array_equal(dropped.k_cache, case.k_cache)
    n = oracle.kv_append(dropped, k_new, v_new)
    assert n == 6  # the empty request writes nothing
    assert np.array_equal(dropped.k_cache, case.k_cache)
    assert np.array_equal(dropped.v_cache, case.v_cache)


def test_append_touches_only_the_new_slots():
    case = W.build_case([3, 16, 31], 4, 2, 128, 16, seed=5)
    k0, v0 = case.k_cache.copy(), case.v_cache.copy()
    k_new = np.arange(3 * 2 * 128, dtype=np.uint16).reshape(3, 2, 128)
    v_new = k_new[::-1].copy()
    oracle.kv_append(case, k_new, v_new)
    k_log, v_log = case.logical_kv()
    k0_log, v0_log = W.unpack_k(k0), W.unpack_v(v0)
    changed = set()
    for b, blk, slot in last_token_slots(case):
        assert np.array_equal(k_log[blk, :, slot], k_new[b])
        assert np.array_equal(v_log[blk, :, slot], v_new[b])
        changed.add((blk, slot))
    for blk in range(case.num_blocks):
        for slot in range(16):
            if (blk, slot) not in changed:
                assert np.array_equal(k_log[blk, :, slot], k0_log[blk, :, slot])
                assert np.array_equal(v_log[blk, :, slot], v0_log[blk, :, slot])


def test_append_clamps_and_skips_bad_blocks():
    case = W.build_case([20, 9, 16], 2, 1, 128, 16, seed=6)
    case.seq_lens[:] = [20, 9, 1000]  # request 2 runs past its table row: token 31
    case.block_table[2, 1] = 1  # the spare block, so the clamped write lands somewhere valid
    case.block_table[1, 0] = case.num_blocks + 3  # request 1's block is out of range
    k_new = np.full((3, 1, 128), 7, np.uint16)
    before = case.k_cache.copy()
    n = oracle.kv_append(case, k_new, k_new)
    assert n == 2
    k_log = case.logical_kv()[0]
    cap = case.max_blocks_per_seq * 16
    t = min(1000, cap) - 1
    assert np.all(k_log[case.block_table[2, t // 16], 0, t % 16] == 7)
    diff = np.argwhere(W.unpack_k(before) != k_log)
    assert {tuple(x[:3]) for x in diff} == {
        (case.block_table[0, 19 // 16], 0, 19 % 16), (case.block_table[2, t // 16], 0, t % 16)}


def test_copy_blocks_brute_force():
    rng = np.random.default_rng(11)
    hkv, nsrc, ndst = 2, 9, 12
    src_k = rng.integers(0, 1 << 16, size=(nsrc, hkv, 16, 16, 8), dtype=np.uint16)
    src_v = rng.integers(0, 1 << 16, size=(nsrc, hkv, 128, 16), dtype=np.uint16)
    dst_k = rng.integers(0, 1 << 16, size=(ndst, hkv, 16, 16, 8), dtype=np.uint16)
    dst_v = rng.integers(0, 1 << 16, size=(ndst, hkv, 128, 16), dtype=np.uint16)
    src_ids = np.array([0, 8, 3, -1, 4, 9, 2], np.int32)
    dst_ids = np.array([11, 0, 5, 6, 12, 7, 3], np.int32)
    ek, ev = dst_k.copy(), dst_v.copy()
    valid = 0
    for s, d in zip(src_ids, dst_ids):
        if 0 <= s < nsrc and 0 <= d < ndst:
            ek[d] = src_k[s]
            ev[d] = src_v[s]
            valid += 1
    n = oracle.copy_blocks(src_k, src_v, dst_k, dst_v, src_ids, dst_ids, hkv)
    assert n == valid == 4
    assert np.array_equal(dst_k, ek) and np.array_equal(dst_v, ev)


def test_swap_out_and_in_leaves_attention_bit_identical():
    case = W.build_case([40, 7, 130, 0, 64], 8, 2, 128, 16, seed=12)
    ref = oracle.decode_attention(case)
    used = used_blocks(case)
    # swap out to a host cache at packed ids, poison the device blocks ...
    host_k = np.zeros((len(used), 2, 16, 16, 8), np.uint16)
    host_v = np.zeros((len(used), 2, 128, 16), np.uint16)
    ids = np.array(used, np.int32)
    assert oracle.copy_blocks(case.k_cache, case.v_cache, host_k, host_v, ids,
                              np.arange(len(used), dtype=np.int32), 2) == len(used)
    case.k_cache[ids] = POISON
    case.v_cache[ids] = POISON
    # ... then swap in at a permutation of free ids and remap the table
    new_ids = np.random.default_rng(1).permutation(case.num_blocks)[:len(used)].astype(np.int32)
    assert oracle.copy_blocks(host_k, host_v, case.k_cache, case.v_cache,
                              np.arange(len(used), dtype=np.int32), new_ids, 2) == len(used)
    remap = dict(zip(used, new_ids.tolist()))
    for b, L in enumerate(case.seq_lens):
        for j in range((L + 15) // 16):
            case.block_table[b, j] = remap[int(case.block_table[b, j])]
    assert np.array_equal(oracle.decode_attention(case), ref)
