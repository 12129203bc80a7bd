"""Decode attention captured in a HIP graph (torch.cuda.CUDAGraph) and replayed:
the allocation-free entry point and the workspace entry point, on interleaved
caches. Between replays the query rows are rewritten in place and the program
runs eager work of its own; every replay must give the bits the eager call
gives on the same inputs, and match the oracle."""
import ctypes

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


@pytest.mark.parametrize("entry", ["noalloc", "workspace"])
def test_graph_replays_match_eager_calls(entry):
    lib = neo.load_library()
    case = W.build_case([900, 17, 3000, 1, 0, 2048, 64, 511, 1500, 33], 32, 8, 128, 16, seed=91)
    print(f"[graph] {entry}: B={case.batch} Hq={case.num_q_heads} Hkv={case.num_kv_heads}",
          flush=True)
    q, k, v, bt, sl = case.to_torch("cuda", kv_layout="interleaved")
    stride = k.stride(0)
    ws = neo.new_workspace(case.batch, case.num_q_heads, case.num_kv_heads)
    out = torch.full((case.batch, case.num_q_heads, 128), float("nan"), device="cuda")

    def call(dst):
        sh = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        common = (q.data_ptr(), k.data_ptr(), v.data_ptr(), bt.data_ptr(), sl.data_ptr(),
                  case.num_q_heads, case.num_kv_heads, 128, 16, float(case.scale),
                  dst.data_ptr(), case.batch, case.max_blocks_per_seq, case.num_blocks)
        if entry == "noalloc":
            rc = lib.neo_decode_attention_noalloc(*common, stride, sh)
        else:
            rc = lib.neo_decode_attention_ex(*common, ws.data_ptr(), ws.numel(), 0, 0, 0, stride,
                                             sh)
        assert rc == 0, lib.neo_last_error().decode()

    # Eager first: the allocation-free entry point looks up its scratch on its
    # first call on a device, which stays outside the capture.
    call(out)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(out)
    rng = np.random.default_rng(92)
    for replay in range(4):
        # New query rows in place, eager work on the same stream, then the replay.
        new_q = rng.integers(0, 1 << 16, size=case.q.shape, dtype=np.uint16)
        new_q = np.where((new_q & 0x7F80) == 0x7F80, new_q & 0x3FFF, new_q)  # finite bf16 only
        new_q = (new_q & 0x3FFF) | (new_q & 0x8000)                           # |x| < 2
        q.copy_(torch.from_numpy(new_q.astype(np.uint16).view(np.int16)).cuda().view(torch.bfloat16))
        case.q = new_q.astype(np.uint16)
        scratch = torch.randn(1 << 20, device="cuda").sum()
        g.replay()
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        eager = torch.full_like(out, float("nan"))
        call(eager)
        torch.cuda.synchronize()
        want = eager.cpu().numpy()
        ae, re = _errors(got, oracle.decode_attention(case))
        print(f"[graph] {entry} replay {replay}: bit-identical to eager={np.array_equal(got, want)} "
              f"vs oracle max_abs={ae:.2e} rel={re:.2e} (scratch {float(scratch):.1f})", flush=True)
        assert np.array_equal(got, want)
        assert ae <= ABS_TOL and re <= REL_TOL
