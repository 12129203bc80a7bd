"""GPU tests of the cache operations (append, block copy, gather) through the C
ABI: bit-exact against the oracle's append and copy, on dense caches and on
caches with a block stride (K and V of a block in one run, with or without
padding), swap round trips through pinned host memory, and copies overlapping
attention on another stream."""
import ctypes
import sys

import numpy as np
import pytest

import oracle
import paper_2411_01142_amd as neo
from paper_2411_01142_amd import workloads as W
from kv_cases import POISON, drop_last_tokens, used_blocks

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    neo.load_library()
    yield


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_bf16(a, pinned=False):
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
    t = t.pin_memory() if pinned else t.to("cuda")
    return t.view(torch.bfloat16)


def host_u16(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda")


def decode(case, k, v, bt=None, **kw):
    q, _, _, bt0, sl = case.to_torch("cuda")
    out = neo.decode_attention(q, k, v, bt0 if bt is None else bt, sl, scale=case.scale, **kw)
    torch.cuda.synchronize()
    return out.cpu().numpy()


# ------------------------------------------------------------------- append

@pytest.mark.parametrize("hkv,seed", [(1, 0), (2, 1), (8, 2), (16, 3)])
def test_append_restores_the_dropped_token(hkv, seed):
    say(f"[kv] append hkv={hkv} seed={seed}")
    case = W.build_case([1, 5, 16, 17, 40, 0, 33, 300], 2 * hkv, hkv, 128, 16, seed=seed)
    dropped, k_new, v_new = drop_last_tokens(case)
    k, v = dev_bf16(dropped.k_cache), dev_bf16(dropped.v_cache)
    bt, sl = dev_i32(case.block_table), dev_i32(case.seq_lens)
    neo.kv_append(k, v, dev_bf16(k_new), dev_bf16(v_new), bt, sl)
    torch.cuda.synchronize()
    assert np.array_equal(host_u16(k), case.k_cache)
    assert np.array_equal(host_u16(v), case.v_cache)
    # the restored caches give the original attention, bit for bit
    q, k0, v0, _, _ = case.to_torch("cuda")
    assert np.array_equal(decode(case, k, v), decode(case, k0, v0))


def test_append_clamps_and_skips_like_the_oracle():
    case = W.build_case([20, 9, 16, 0], 2, 1, 128, 16, seed=6)
    case.seq_lens[:] = [20, 9, 1000, 0]
    case.block_table[2, 1] = 1
    case.block_table[1, 0] = case.num_blocks + 3
    rng = np.random.default_rng(4)
    k_new = rng.integers(0, 1 << 16, size=(4, 1, 128), dtype=np.uint16)
    v_new = rng.integers(0, 1 << 16, size=(4, 1, 128), dtype=np.uint16)
    k, v = dev_bf16(case.k_cache), dev_bf16(case.v_cache)
    neo.kv_append(k, v, dev_bf16(k_new), dev_bf16(v_new), dev_i32(case.block_table),
                  dev_i32(case.seq_lens))
    torch.cuda.synchronize()
    assert oracle.kv_append(case, k_new, v_new) == 2
    assert np.array_equal(host_u16(k), case.k_cache)
    assert np.array_equal(host_u16(v), case.v_cache)


def test_append_full_size_batch_matches_oracle():
    case = W.make_config(4, 7, poison=False)  # 512 requests, 8 kv heads
    say(f"[kv] append full batch={case.batch} blocks={case.num_blocks}")
    rng = np.random.default_rng(8)
    shape = (case.batch, case.num_kv_heads, 128)
    k_new = rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)
    v_new = rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)
    k, v = dev_bf16(case.k_cache), dev_bf16(case.v_cache)
    neo.kv_append(k, v, dev_bf16(k_new), dev_bf16(v_new), dev_i32(case.block_table),
                  dev_i32(case.seq_lens))
    torch.cuda.synchronize()
    assert oracle.kv_append(case, k_new, v_new) == case.batch
    assert np.array_equal(host_u16(k), case.k_cache)
    assert np.array_equal(host_u16(v), case.v_cache)


def test_append_empty_batch_is_a_noop():
    k = torch.zeros(4, 2, 16, 16, 8, dtype=torch.bfloat16, device="cuda")
    v = torch.zeros(4, 2, 128, 16, dtype=torch.bfloat16, device="cuda")
    e = torch.zeros(0, 2, 128, dtype=torch.bfloat16, device="cuda")
    neo.kv_append(k, v, e, e, torch.zeros(0, 1, dtype=torch.int32, device="cuda"),
                  torch.zeros(0, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert int(k.view(torch.int16).abs().sum()) == 0


# --------------------------------------------------------------------- copy

def random_caches(rng, nb, hkv, pinned=False):
    kk = rng.integers(0, 1 << 16, size=(nb, hkv, 16, 16, 8), dtype=np.uint16)
    vv = rng.integers(0, 1 << 16, size=(nb, hkv, 128, 16), dtype=np.uint16)
    return kk, vv, dev_bf16(kk, pinned), dev_bf16(vv, pinned)


@pytest.mark.parametrize("hkv", [1, 2, 8])
@pytest.mark.parametrize("src_pinned,dst_pinned", [(False, False), (False, True), (True, False)])
def test_copy_blocks_matches_oracle(hkv, src_pinned, dst_pinned):
    say(f"[kv] copy hkv={hkv} src_pinned={src_pinned} dst_pinned={dst_pinned}")
    rng = np.random.default_rng(100 + hkv)
    nsrc, ndst, n = 37, 53, 29
    sk, sv, tsk, tsv = random_caches(rng, nsrc, hkv, src_pinned)
    dk, dv, tdk, tdv = random_caches(rng, ndst, hkv, dst_pinned)
    src_ids = rng.integers(-2, nsrc + 2, size=n).astype(np.int32)
    dst_ids = rng.permutation(ndst + 4)[:n].astype(np.int32)  # distinct, some out of range
    neo.copy_blocks(tsk, tsv, tdk, tdv, dev_i32(src_ids), dev_i32(dst_ids))
    torch.cuda.synchronize()
    oracle.copy_blocks(sk, sv, dk, dv, src_ids, dst_ids, hkv)
    assert np.array_equal(host_u16(tdk), dk) and np.array_equal(host_u16(tdv), dv)
    assert np.array_equal(host_u16(tsk), sk)  # the source is untouched


def test_swap_round_trip_through_pinned_host_memory():
    case = W.make_config(2, 3, poison=True)
    say(f"[kv] swap round trip batch={case.batch} blocks={case.num_blocks}")
    q, k, v, bt, sl = case.to_torch("cuda")
    ref = decode(case, k, v)
    used = np.array(used_blocks(case), np.int32)
    n = len(used)
    host_k = torch.empty((n,) + tuple(k.shape[1:]), dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty((n,) + tuple(v.shape[1:]), dtype=torch.bfloat16, pin_memory=True)
    seq = dev_i32(np.arange(n))
    neo.copy_blocks(k, v, host_k, host_v, dev_i32(used), seq)  # swap out
    torch.cuda.synchronize()
    assert np.array_equal(host_u16(host_k), case.k_cache[used])
    assert np.array_equal(host_u16(host_v), case.v_cache[used])
    k.view(torch.int16).fill_(POISON)
    v.view(torch.int16).fill_(POISON)
    new_ids = np.random.default_rng(5).permutation(case.num_blocks)[:n].astype(np.int32)
    neo.copy_blocks(host_k, host_v, k, v, seq, dev_i32(new_ids))  # swap in elsewhere
    remap = np.full(case.num_blocks, -1, np.int32)
    remap[used] = new_ids
    table = case.block_table.copy()
    for b, L in enumerate(case.seq_lens.tolist()):
        nbk = (L + 15) // 16
        table[b, :nbk] = remap[table[b, :nbk]]
    torch.cuda.synchronize()
    assert np.array_equal(decode(case, k, v, bt=dev_i32(table)), ref)


def test_copy_refuses_pageable_host_memory():
    k = torch.zeros(4, 2, 16, 16, 8, dtype=torch.bfloat16)  # pageable
    v = torch.zeros(4, 2, 128, 16, dtype=torch.bfloat16)
    dk = torch.zeros(4, 2, 16, 16, 8, dtype=torch.bfloat16, device="cuda")
    dv = torch.zeros(4, 2, 128, 16, dtype=torch.bfloat16, device="cuda")
    ids = torch.arange(2, dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError, match="pinned"):
        neo.copy_blocks(k, v, dk, dv, ids, ids)
    # the C ABI refuses the pointer itself, before any launch
    lib = neo.load_library()
    rc = lib.neo_kv_copy_blocks(k.data_ptr(), v.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                ids.data_ptr(), ids.data_ptr(), 2, 2, 128, 16, 4, 4, 0, 0, None)
    assert rc == 1 and "pinned" in lib.neo_last_error().decode()
    torch.cuda.synchronize()


def test_copy_on_a_side_stream_overlaps_attention():
    case = W.make_config(2, 9, poison=True)
    say(f"[kv] overlap batch={case.batch}")
    q, k, v, bt, sl = case.to_torch("cuda")
    ref = decode(case, k, v)
    used = np.array(used_blocks(case), np.int32)
    n = len(used)
    host_k = torch.empty((n,) + tuple(k.shape[1:]), dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty((n,) + tuple(v.shape[1:]), dtype=torch.bfloat16, pin_memory=True)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    outs = []
    with torch.cuda.stream(side):
        neo.copy_blocks(k, v, host_k, host_v, dev_i32(used), dev_i32(np.arange(n)), stream=side)
    for _ in range(3):
        outs.append(neo.decode_attention(q, k, v, bt, sl, scale=case.scale))
    torch.cuda.synchronize()
    for o in outs:
        assert np.array_equal(o.cpu().numpy(), ref)
    assert np.array_equal(host_u16(host_k), case.k_cache[used])
    assert np.array_equal(host_u16(host_v), case.v_cache[used])


# ------------------------------------------------------------ strided caches

def one_buffer(kk, vv, pad=0, pinned=False):
    """(buf, k, v): k and v views of one bf16 buffer ``[nb][K | V | pad]``
    holding the uint16 arrays kk and vv, every padding element POISON."""
    nb, per = kk.shape[0], kk[0].size
    host = np.full((nb, 2 * per + pad), POISON, np.uint16)
    host[:, :per] = kk.reshape(nb, per)
    host[:, per:2 * per] = vv.reshape(nb, per)
    buf = dev_bf16(host, pinned)
    return buf, buf[:, :per].view(kk.shape), buf[:, per:2 * per].view(vv.shape)


def split_buffer(buf, kshape, vshape):
    """uint16 (k, v, padding) read back from a buffer made by one_buffer."""
    h = host_u16(buf)
    per = int(np.prod(kshape[1:]))
    return h[:, :per].reshape(kshape), h[:, per:2 * per].reshape(vshape), h[:, 2 * per:]


@pytest.mark.parametrize("hkv,pad", [(1, 0), (8, 0), (2, 8), (8, 4096 + 8)])
def test_append_into_strided_caches(hkv, pad):
    say(f"[kv] append strided hkv={hkv} pad={pad}")
    case = W.build_case([1, 5, 16, 17, 40, 0, 33, 300], 2 * hkv, hkv, 128, 16, seed=70 + hkv)
    dropped, k_new, v_new = drop_last_tokens(case)
    buf, k, v = one_buffer(dropped.k_cache, dropped.v_cache, pad)
    assert k.stride(0) == v.stride(0) == 2 * hkv * 2048 + pad
    neo.kv_append(k, v, dev_bf16(k_new), dev_bf16(v_new), dev_i32(case.block_table),
                  dev_i32(case.seq_lens))
    torch.cuda.synchronize()
    kk, vv, padding = split_buffer(buf, case.k_cache.shape, case.v_cache.shape)
    assert np.array_equal(kk, case.k_cache) and np.array_equal(vv, case.v_cache)
    assert np.all(padding == POISON)


def test_append_full_size_into_interleaved_caches():
    case = W.make_config(4, 7, poison=False)  # 512 requests, 8 kv heads
    say(f"[kv] append interleaved full batch={case.batch} blocks={case.num_blocks}")
    rng = np.random.default_rng(9)
    shape = (case.batch, case.num_kv_heads, 128)
    k_new = rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)
    v_new = rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)
    buf, k, v = one_buffer(case.k_cache, case.v_cache)
    neo.kv_append(k, v, dev_bf16(k_new), dev_bf16(v_new), dev_i32(case.block_table),
                  dev_i32(case.seq_lens))
    torch.cuda.synchronize()
    assert oracle.kv_append(case, k_new, v_new) == case.batch
    kk, vv, _ = split_buffer(buf, case.k_cache.shape, case.v_cache.shape)
    assert np.array_equal(kk, case.k_cache) and np.array_equal(vv, case.v_cache)


# (source layout, source pinned, destination layout, destination pinned); a
# layout is the padding after each block's K and V in one buffer, or None for
# two dense caches.
STRIDED_COPIES = [
    (0, False, None, True),      # swap out: interleaved device cache -> dense host cache
    (None, True, 0, False),      # swap in: dense host cache -> interleaved device cache
    (0, False, 24, False),       # between two strided device caches
    (64, True, 0, False),        # strided host cache -> interleaved device cache
]


@pytest.mark.parametrize("hkv", [1, 8])
@pytest.mark.parametrize("src_pad,src_pinned,dst_pad,dst_pinned", STRIDED_COPIES)
def test_copy_blocks_between_layouts(hkv, src_pad, src_pinned, dst_pad, dst_pinned):
    say(f"[kv] copy layouts hkv={hkv} src={src_pad},{src_pinned} dst={dst_pad},{dst_pinned}")
    rng = np.random.default_rng(200 + hkv)
    nsrc, ndst, n = 31, 45, 23
    kshape, vshape = (hkv, 16, 16, 8), (hkv, 128, 16)

    def caches(nb, pad, pinned):
        kk = rng.integers(0, 1 << 16, size=(nb,) + kshape, dtype=np.uint16)
        vv = rng.integers(0, 1 << 16, size=(nb,) + vshape, dtype=np.uint16)
        if pad is None:
            return kk, vv, None, dev_bf16(kk, pinned), dev_bf16(vv, pinned)
        buf, k, v = one_buffer(kk, vv, pad, pinned)
        return kk, vv, buf, k, v

    sk, sv, sbuf, tsk, tsv = caches(nsrc, src_pad, src_pinned)
    dk, dv, dbuf, tdk, tdv = caches(ndst, dst_pad, dst_pinned)
    src_ids = rng.integers(-2, nsrc + 2, size=n).astype(np.int32)
    dst_ids = rng.permutation(ndst + 4)[:n].astype(np.int32)
    neo.copy_blocks(tsk, tsv, tdk, tdv, dev_i32(src_ids), dev_i32(dst_ids))
    torch.cuda.synchronize()
    sk0, sv0 = sk.copy(), sv.copy()
    oracle.copy_blocks(sk, sv, dk, dv, src_ids, dst_ids, hkv)
    if dbuf is None:
        gk, gv = host_u16(tdk), host_u16(tdv)
    else:
        gk, gv, padding = split_buffer(dbuf, dk.shape, dv.shape)
        assert np.all(padding == POISON)
    assert np.array_equal(gk, dk) and np.array_equal(gv, dv)
    if sbuf is not None:
        gk, gv, padding = split_buffer(sbuf, sk.shape, sv.shape)
        assert np.array_equal(gk, sk0) and np.array_equal(gv, sv0) and np.all(padding == POISON)


@pytest.mark.parametrize("pad", [0, 8, 2048])
def test_gather_from_strided_caches(pad):
    case = W.build_case([1, 15, 16, 17, 100, 333, 0, 64], 8, 4, 128, 16, seed=71,
                        extra_table_cols=2)
    _, k, v = one_buffer(case.k_cache, case.v_cache, pad)
    bt, sl = dev_i32(case.block_table), dev_i32(case.seq_lens)
    for which, cache in (("k", k), ("v", v)):
        got = host_u16(neo.paged_gather(cache, which, bt, sl))
        assert np.array_equal(got, oracle.paged_gather(case, which)), which


def test_binding_refuses_mismatched_strides():
    rng = np.random.default_rng(72)
    kk = rng.integers(0, 1 << 16, size=(6, 2, 16, 16, 8), dtype=np.uint16)
    vv = rng.integers(0, 1 << 16, size=(6, 2, 128, 16), dtype=np.uint16)
    _, k, v = one_buffer(kk, vv)
    dense_v = dev_bf16(vv)
    ids = dev_i32(np.arange(2))
    e = torch.zeros(0, 2, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="block stride"):
        neo.kv_append(k, dense_v, e, e, dev_i32(np.zeros((0, 1))), dev_i32(np.zeros(0)))
    with pytest.raises(ValueError, match="block stride"):
        neo.copy_blocks(k, dense_v, k, v, ids, ids)
    with pytest.raises(ValueError, match="dense"):
        neo.paged_gather(k.transpose(2, 3), "k", dev_i32(np.zeros((1, 1))), dev_i32([1]))
    torch.cuda.synchronize()
