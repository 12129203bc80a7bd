"""The allocation-free decode entry point (a static device scratch array
instead of a caller workspace), called through the C ABI: its output matches
the workspace entry point's on two calls in a row, the second with a smaller
input (the scratch keeps the first call's contents), and the oracle."""
import ctypes
import sys

import numpy as np
import pytest

import oracle
import paper_2411_01142_amd as neo
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


def _errors(y, r):
    y = y.reshape(-1, y.shape[-1]).astype(np.float64)
    r = r.reshape(-1, r.shape[-1]).astype(np.float64)
    ae = np.abs(y - r)
    return float(ae.max()), float((ae.max(axis=1) / np.maximum(np.abs(r).max(axis=1), 1e-30)).max())


def _call(lib, case, fn, ws=None, kv_layout="separate"):
    q, k, v, bt, sl = case.to_torch("cuda", kv_layout=kv_layout)
    stride = k.stride(0) if kv_layout == "interleaved" else 0
    out = torch.full((case.batch, case.num_q_heads, 128), float("nan"), device="cuda")
    sh = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    common = (q.data_ptr(), k.data_ptr(), v.data_ptr(), bt.data_ptr(), sl.data_ptr(),
              case.num_q_heads, case.num_kv_heads, 128, 16, float(case.scale), out.data_ptr(),
              case.batch, case.max_blocks_per_seq, case.num_blocks)
    if fn == "noalloc":
        rc = lib.neo_decode_attention_noalloc(*common, stride, sh)
    else:
        rc = lib.neo_decode_attention_ex(*common, ws.data_ptr(), ws.numel(), 0, 0, 0, stride, sh)
    assert rc == 0, lib.neo_last_error().decode()
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_noalloc_matches_workspace_entry_point():
    lib = neo.load_library()
    # First a large batch with many requests split across workgroups (the
    # scratch's counters and partial slots in use), then a smaller one with a
    # different group, which must not see the first call's contents.
    cases = [W.make_config(5, 5, batch_limit=600),
             W.build_case([3000, 17, 900, 1, 0, 2500, 64], 32, 2, 128, 16, seed=77)]
    for i, case in enumerate(cases):
        print(f"[noalloc] call {i}: {case.name} B={case.batch} Hq={case.num_q_heads} "
              f"Hkv={case.num_kv_heads}", flush=True)
        sys.stdout.flush()
        ws = neo.new_workspace(case.batch, case.num_q_heads, case.num_kv_heads)
        want = _call(lib, case, "workspace", ws)
        got = _call(lib, case, "noalloc")
        ref = oracle.decode_attention(case)
        assert np.all(np.isfinite(got))
        ae, re = _errors(got, want)
        print(f"[noalloc] call {i}: vs workspace entry max_abs={ae:.2e} rel={re:.2e}; "
              f"bit-identical={np.array_equal(got, want)}", flush=True)
        assert ae <= ABS_TOL and re <= REL_TOL
        ae, re = _errors(got, ref)
        print(f"[noalloc] call {i}: vs oracle max_abs={ae:.2e} rel={re:.2e}", flush=True)
        assert ae <= ABS_TOL and re <= REL_TOL


def test_noalloc_with_interleaved_caches():
    # K and V of each block in one run (block stride twice a block): the same
    # bits as the workspace entry point given the same stride.
    lib = neo.load_library()
    case = W.make_config(6, 6)
    print(f"[noalloc] interleaved caches: {case.name} B={case.batch}", flush=True)
    ws = neo.new_workspace(case.batch, case.num_q_heads, case.num_kv_heads)
    want = _call(lib, case, "workspace", ws, kv_layout="interleaved")
    got = _call(lib, case, "noalloc", kv_layout="interleaved")
    assert np.all(np.isfinite(got))
    ae, re = _errors(got, oracle.decode_attention(case))
    print(f"[noalloc] interleaved: vs oracle max_abs={ae:.2e} rel={re:.2e}; "
          f"bit-identical to the workspace entry={np.array_equal(got, want)}", flush=True)
    assert ae <= ABS_TOL and re <= REL_TOL
    assert np.array_equal(got, want)


def test_noalloc_repeated_calls_are_bit_identical():
    lib = neo.load_library()
    case = W.make_config(2, 102)
    first = _call(lib, case, "noalloc")
    for _ in range(3):
        assert np.array_equal(_call(lib, case, "noalloc"), first)


def test_noalloc_rejects_bad_arguments_and_empty_batch():
    lib = neo.load_library()
    case = W.build_case([10, 20], 8, 2, 128, 16, seed=5)
    q, k, v, bt, sl = case.to_torch("cuda")
    out = torch.empty((2, 8, 128), device="cuda")
    args = [q.data_ptr(), k.data_ptr(), v.data_ptr(), bt.data_ptr(), sl.data_ptr(), 8, 2, 128, 16,
            0.1, out.data_ptr(), 2, case.max_blocks_per_seq, case.num_blocks, 0, None]
    bad = list(args)
    bad[7] = 64    # head_dim
    assert lib.neo_decode_attention_noalloc(*bad) == 2
    bad = list(args)
    bad[0] = None  # q
    assert lib.neo_decode_attention_noalloc(*bad) == 1
    empty = [None] * 5 + [8, 2, 128, 16, 0.1, None, 0, 1, 1, 0, None]
    assert lib.neo_decode_attention_noalloc(*empty) == 0
