"""fp64 CPU oracle for batched paged GQA decode attention (ctypes wrapper of neo_ref.c).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the package's smoke check and
the benchmark's CPU-baseline leg; the library path never loads it.

Every function computes from the definition of decode attention (the paper,
Sec. 2.1-2.2) over the paged storage contract, in double precision. See
``neo_ref.c`` for the formulas and the storage layout.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "neo_ref.c")
_LIB = os.path.join(_HERE, "libneo_ref.so")

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_D = ctypes.c_double

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-Wall", _SRC,
                               "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    lib.neo_ref_decode_attention.argtypes = [_P, _P, _P, _P, _P, _I32, _I32, _I32, _I32, _D, _P, _P,
                                             _I32, _I32, _I32, _I64, _I64, _I32]
    lib.neo_ref_decode_attention.restype = ctypes.c_int
    lib.neo_ref_softmax_weights.argtypes = [_P, _P, _P, _P, _I32, _I32, _I32, _I32, _D, _I32, _I32,
                                            _I32, _I32, _I32, _P]
    lib.neo_ref_softmax_weights.restype = ctypes.c_int
    lib.neo_ref_partial_attention.argtypes = [_P, _P, _P, _P, _I32, _I32, _I32, _I32, _D, _I32,
                                              _I32, _I32, _I32, _I32, _I64, _I64, _P, _P]
    lib.neo_ref_partial_attention.restype = ctypes.c_int
    lib.neo_ref_lse_merge.argtypes = [_I32, _I32, _P, _P, _P, _P]
    lib.neo_ref_lse_merge.restype = ctypes.c_int
    lib.neo_ref_paged_gather.argtypes = [_P, _I32, _P, _P, _I32, _I32, _I32, _I32, _I32, _I32, _P]
    lib.neo_ref_paged_gather.restype = ctypes.c_int64
    lib.neo_ref_kv_append.argtypes = [_P, _P, _P, _P, _P, _P, _I32, _I32, _I32, _I32, _I32, _I32]
    lib.neo_ref_kv_append.restype = _I32
    lib.neo_ref_copy_blocks.argtypes = [_P, _P, _P, _P, _P, _P, _I32, _I32, _I32, _I32, _I32,
                                        _I32]
    lib.neo_ref_copy_blocks.restype = _I32
    lib.neo_ref_max_threads.argtypes = []
    lib.neo_ref_max_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class OracleError(RuntimeError):
    pass


def max_threads() -> int:
    return int(_load().neo_ref_max_threads())


def decode_attention(case, *, rows=None, threads: int = 0, want_f64: bool = False,
                     scale=None, q=None):
    """Oracle output for a ``workloads.Case``.

    Returns float32 ``[B][Hq][D]`` (or (float32, float64) with ``want_f64``).
    ``rows=(r0, r1)`` restricts work to flattened (request, q head) rows
    [r0, r1); other rows are left zero. ``q``/``scale`` override the case's.
    """
    lib = _load()
    B, Hq, D = case.batch, case.num_q_heads, case.head_dim
    qa = _c(case.q if q is None else q, np.uint16)
    kc, vc = _c(case.k_cache, np.uint16), _c(case.v_cache, np.uint16)
    bt, sl = _c(case.block_table, np.int32), _c(case.seq_lens, np.int32)
    out = np.zeros((B, Hq, D), dtype=np.float32)
    out64 = np.zeros((B, Hq, D), dtype=np.float64) if want_f64 else None
    r0, r1 = (0, B * Hq) if rows is None else rows
    rc = lib.neo_ref_decode_attention(
        _ptr(qa), _ptr(kc), _ptr(vc), _ptr(bt), _ptr(sl), Hq, case.num_kv_heads, D,
        case.block_size, float(case.scale if scale is None else scale), _ptr(out),
        _ptr(out64) if want_f64 else None, B, case.max_blocks_per_seq, case.num_blocks,
        int(r0), int(r1), int(threads))
    if rc != 0:
        raise OracleError(f"neo_ref_decode_attention failed: {rc}")
    return (out, out64) if want_f64 else out


def softmax_weights(case, b: int, h: int) -> np.ndarray:
    """Softmax weights (float64 [L]) of request ``b``, q head ``h``."""
    lib = _load()
    L = max(int(case.seq_lens[b]), 0)
    w = np.zeros(max(L, 1), dtype=np.float64)
    qa, kc = _c(case.q, np.uint16), _c(case.k_cache, np.uint16)
    bt, sl = _c(case.block_table, np.int32), _c(case.seq_lens, np.int32)
    rc = lib.neo_ref_softmax_weights(_ptr(qa), _ptr(kc), _ptr(bt), _ptr(sl), case.num_q_heads,
                                     case.num_kv_heads, case.head_dim, case.block_size,
                                     float(case.scale), case.batch, case.max_blocks_per_seq,
                                     case.num_blocks, int(b), int(h), _ptr(w))
    if rc != 0:
        raise OracleError(f"neo_ref_softmax_weights failed: {rc}")
    return w[:L]


def partial_attention(case, b: int, h: int, t0: int, t1: int):
    """(o float64 [D], lse float) of request ``b``, q head ``h`` over tokens [t0, t1)."""
    lib = _load()
    o = np.zeros(case.head_dim, dtype=np.float64)
    lse = np.zeros(1, dtype=np.float64)
    qa, kc, vc = _c(case.q, np.uint16), _c(case.k_cache, np.uint16), _c(case.v_cache, np.uint16)
    bt = _c(case.block_table, np.int32)
    rc = lib.neo_ref_partial_attention(_ptr(qa), _ptr(kc), _ptr(vc), _ptr(bt), case.num_q_heads,
                                       case.num_kv_heads, case.head_dim, case.block_size,
                                       float(case.scale), case.batch, case.max_blocks_per_seq,
                                       case.num_blocks, int(b), int(h), int(t0), int(t1),
                                       _ptr(o), _ptr(lse))
    if rc != 0:
        raise OracleError(f"neo_ref_partial_attention failed: {rc}")
    return o, float(lse[0])


def lse_merge(o: np.ndarray, lse: np.ndarray):
    """Merge partials ``o`` [n][D] with log-sum-exps ``lse`` [n]; returns (out [D], lse)."""
    lib = _load()
    o = _c(o, np.float64)
    lse = _c(lse, np.float64)
    n, d = o.shape
    out = np.zeros(d, dtype=np.float64)
    lo = np.zeros(1, dtype=np.float64)
    rc = lib.neo_ref_lse_merge(int(n), int(d), _ptr(o), _ptr(lse), _ptr(out), _ptr(lo))
    if rc != 0:
        raise OracleError(f"neo_ref_lse_merge failed: {rc}")
    return out, float(lo[0])


def paged_gather(case, which: str) -> np.ndarray:
    """Dense copy (uint16 [sum L][Hkv][D]) of the K (``which='k'``) or V cache."""
    lib = _load()
    cache = _c(case.k_cache if which == "k" else case.v_cache, np.uint16)
    bt, sl = _c(case.block_table, np.int32), _c(case.seq_lens, np.int32)
    total = int(np.maximum(case.seq_lens, 0).sum())
    dst = np.zeros((max(total, 1), case.num_kv_heads, case.head_dim), dtype=np.uint16)
    n = lib.neo_ref_paged_gather(_ptr(cache), 1 if which == "v" else 0, _ptr(bt), _ptr(sl),
                                 case.batch, case.max_blocks_per_seq, case.num_kv_heads,
                                 case.head_dim, case.block_size, case.num_blocks, _ptr(dst))
    if n < 0:
        raise OracleError(f"neo_ref_paged_gather failed: {n}")
    return dst[:total]


def kv_append(case, k_new: np.ndarray, v_new: np.ndarray) -> int:
    """Write each request's newest token (k_new, v_new: uint16 [B][Hkv][D]) into the
    case's caches in place, at token seq_lens[b] - 1. Returns requests written."""
    lib = _load()
    assert case.k_cache.flags.c_contiguous and case.v_cache.flags.c_contiguous
    kn, vn = _c(k_new, np.uint16), _c(v_new, np.uint16)
    bt, sl = _c(case.block_table, np.int32), _c(case.seq_lens, np.int32)
    return int(lib.neo_ref_kv_append(_ptr(case.k_cache), _ptr(case.v_cache), _ptr(kn), _ptr(vn),
                                      _ptr(bt), _ptr(sl), case.batch, case.max_blocks_per_seq,
                                      case.num_kv_heads, case.head_dim, case.block_size,
                                      case.num_blocks))


def copy_blocks(src_k, src_v, dst_k, dst_v, src_ids, dst_ids, num_kv_heads: int,
                head_dim: int = 128, block_size: int = 16) -> int:
    """dst block dst_ids[i] <- src block src_ids[i] (uint16 caches, in place)."""
    lib = _load()
    assert dst_k.flags.c_contiguous and dst_v.flags.c_contiguous
    sk, sv = _c(src_k, np.uint16), _c(src_v, np.uint16)
    si, di = _c(src_ids, np.int32), _c(dst_ids, np.int32)
    return int(lib.neo_ref_copy_blocks(_ptr(sk), _ptr(sv), _ptr(dst_k), _ptr(dst_v), _ptr(si),
                                       _ptr(di), int(si.shape[0]), num_kv_heads, head_dim,
                                       block_size, int(sk.shape[0]), int(dst_k.shape[0])))
