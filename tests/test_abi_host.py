"""Host-side checks of the C ABI: the library loads, exports every entry point the
header declares, sizes workspaces, and rejects bad arguments before any HIP call
(so these run without a GPU)."""
import ctypes
import math
import os
import re

import pytest

import paper_2411_01142_amd as neo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libneoattn.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(neo.library_path()):
        import __graft_entry__
        __graft_entry__.build()
    return neo.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(neo_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("neo_decode_attention", "neo_decode_attention_ex", "neo_decode_workspace_bytes",
              "neo_decode_workspace_init", "neo_decode_attention_events",
              "neo_paged_gather", "neo_kv_append", "neo_kv_copy_blocks", "neo_debug_validate",
              "neo_last_error", "neo_version"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version(lib):
    assert re.fullmatch(r"\d+\.\d+\.\d+", neo.version())


def test_workspace_bytes_grow_with_batch_and_group():
    a = neo.workspace_bytes(64, 32, 8)
    b = neo.workspace_bytes(1024, 32, 8)
    c = neo.workspace_bytes(64, 64, 8)
    assert 0 < a < b and a < c
    assert a % 256 == 0
    # two partial slots per slice, group rows of (128 + 1) floats each, at least
    assert a >= 2 * neo.MAX_SLICES * 4 * 129 * 4


def _align256(x):
    return (x + 255) // 256 * 256


@pytest.mark.parametrize("batch,hq,hkv", [(0, 8, 8), (1, 32, 32), (64, 32, 8), (512, 64, 8),
                                          (1024, 32, 8), (3000, 128, 8)])
def test_workspace_bytes_match_the_documented_formula(batch, hq, hkv):
    # The header states the size: a fixed part sized for NEO_MAX_SLICES, one
    # int32 per request, and two partial slots per slice of group rows of
    # head_dim floats plus group log-sum-exps; no dependence on lengths or pool.
    S, D, G = neo.MAX_SLICES, 128, hq // hkv
    want = (_align256(16) + _align256(32 * (S + 1)) + _align256(4 * S) +
            _align256(4 * (batch + 1)) + _align256(8 * S * G) + _align256(8 * S * G * D))
    assert neo.workspace_bytes(batch, hq, hkv) == want


def test_header_documents_the_workspace_contract():
    text = open(HEADER).read()
    # The fused default is one kernel; the workspace is zeroed once and keeps
    # counters between calls.
    assert "Enqueues one kernel" in text
    assert "Enqueues two kernels" not in text
    assert "zero-filled once before its first use" in text
    assert "align256(8 * NEO_MAX_SLICES * group * head_dim)" in text


@pytest.mark.parametrize("args,code", [
    ((64, 32, 7, 128), INVALID),
    ((64, 0, 8, 128), INVALID),
    ((64, 32, 8, 64), UNSUPPORTED),
    ((64, 96, 8, 128), UNSUPPORTED),
    ((-1, 32, 8, 128), INVALID),
])
def test_workspace_bytes_rejects(lib, args, code):
    out = ctypes.c_size_t(0)
    assert lib.neo_decode_workspace_bytes(*args, ctypes.byref(out)) == code
    assert lib.neo_last_error().decode()


FAKE = 1 << 20  # non-null, 256-aligned host address; never dereferenced on these paths


def call(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, table=FAKE, lens=FAKE, hq=32, hkv=8, d=128, bs=16,
             scale=1 / math.sqrt(128), out=FAKE, batch=4, mbps=8, nb=100, ws=FAKE,
             ws_bytes=1 << 40, variant=0, schedule=0, slices=0, kv_stride=0, stream=None)
    a.update(kw)
    return lib.neo_decode_attention_ex(a["q"], a["k"], a["v"], a["table"], a["lens"], a["hq"],
                                       a["hkv"], a["d"], a["bs"], a["scale"], a["out"],
                                       a["batch"], a["mbps"], a["nb"], a["ws"], a["ws_bytes"],
                                       a["variant"], a["schedule"], a["slices"], a["kv_stride"],
                                       a["stream"])


@pytest.mark.parametrize("kw,code,needle", [
    (dict(q=None), INVALID, "NULL"),
    (dict(k=None), INVALID, "NULL"),
    (dict(v=None), INVALID, "NULL"),
    (dict(table=None), INVALID, "NULL"),
    (dict(lens=None), INVALID, "NULL"),
    (dict(out=None), INVALID, "NULL"),
    (dict(hkv=7), INVALID, "multiple"),
    (dict(hq=0), INVALID, "positive"),
    (dict(d=64), UNSUPPORTED, "head_dim"),
    (dict(bs=32), UNSUPPORTED, "block_size"),
    (dict(hq=96, hkv=8), UNSUPPORTED, "group"),
    (dict(scale=float("nan")), INVALID, "scale"),
    (dict(scale=float("inf")), INVALID, "scale"),
    (dict(batch=-3), INVALID, "batch"),
    (dict(mbps=0), INVALID, "positive"),
    (dict(nb=0), INVALID, "positive"),
    (dict(ws=None), WORKSPACE, "workspace"),
    (dict(ws_bytes=1000), WORKSPACE, "workspace"),
    (dict(q=FAKE + 8), INVALID, "aligned"),
    (dict(out=FAKE + 4), INVALID, "aligned"),
    (dict(ws=FAKE + 64), INVALID, "aligned"),
    (dict(variant=7), UNSUPPORTED, "variant"),
    (dict(schedule=4), UNSUPPORTED, "schedule"),
    (dict(slices=-1), INVALID, "max_slices"),
    (dict(slices=100000), INVALID, "max_slices"),
    (dict(batch=1 << 20, mbps=1 << 12), INVALID, "2^31"),
    (dict(batch=1 << 18, mbps=(1 << 10) - 3), INVALID, "+ 3)"),
    (dict(kv_stride=8 * 2048 - 8), INVALID, "kv_block_stride"),
    (dict(kv_stride=2 * 8 * 2048 + 4), INVALID, "kv_block_stride"),
    (dict(kv_stride=-2048), INVALID, "kv_block_stride"),
    (dict(kv_stride=1 << 41), INVALID, "kv_block_stride"),
    (dict(kv_stride=1 << 40, nb=1 << 22), INVALID, "kv_block_stride"),  # span of 2^62+ bytes
])
def test_decode_rejects_bad_arguments_before_any_hip_call(lib, kw, code, needle):
    assert call(lib, **kw) == code
    assert needle in lib.neo_last_error().decode()


def test_empty_batch_is_a_noop(lib):
    assert call(lib, batch=0, q=None, k=None, v=None, table=None, lens=None, out=None,
                ws=None) == OK
    assert lib.neo_last_error().decode() == ""


def test_plain_entry_point_validates_too(lib):
    rc = lib.neo_decode_attention(FAKE, FAKE, FAKE, FAKE, FAKE, 32, 8, 128, 16, 0.1, None, 4, 8,
                                  100, FAKE, 1 << 40, None)
    assert rc == INVALID


def test_gather_and_validate_reject(lib):
    assert lib.neo_paged_gather(FAKE, 2, FAKE, FAKE, FAKE, 4, 8, 8, 128, 16, 100, 0, FAKE,
                                None) == INVALID
    assert lib.neo_paged_gather(FAKE, 0, FAKE, FAKE, FAKE, 4, 8, 8, 100, 16, 100, 0, FAKE,
                                None) == INVALID
    assert lib.neo_paged_gather(None, 0, FAKE, FAKE, FAKE, 4, 8, 8, 128, 16, 100, 0, FAKE,
                                None) == INVALID
    assert lib.neo_paged_gather(None, 0, None, None, None, 0, 8, 8, 128, 16, 100, 0, None,
                                None) == OK
    # block strides below one block, not a multiple of 8, or beyond 2^40
    for bad in (8 * 128 * 16 - 8, 8 * 128 * 16 + 4, (1 << 40) + 8, -8):
        assert lib.neo_paged_gather(FAKE, 1, FAKE, FAKE, FAKE, 4, 8, 8, 128, 16, 100, bad, FAKE,
                                    None) == INVALID
        assert "block_stride" in lib.neo_last_error().decode()
    assert lib.neo_debug_validate(FAKE, FAKE, 4, 0, 16, 100, FAKE, None) == INVALID
    assert lib.neo_debug_validate(None, FAKE, 4, 8, 16, 100, FAKE, None) == INVALID
    assert lib.neo_decode_workspace_init(None, 1024, None) == INVALID
    assert lib.neo_decode_workspace_init(FAKE + 4, 1024, None) == INVALID


def append_call(lib, **kw):
    a = dict(k=FAKE, v=FAKE, kn=FAKE, vn=FAKE, table=FAKE, lens=FAKE, batch=4, mbps=8, hkv=8,
             d=128, bs=16, nb=100, stride=0)
    a.update(kw)
    return lib.neo_kv_append(a["k"], a["v"], a["kn"], a["vn"], a["table"], a["lens"], a["batch"],
                             a["mbps"], a["hkv"], a["d"], a["bs"], a["nb"], a["stride"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=-1), INVALID), (dict(hkv=0), INVALID), (dict(d=64), UNSUPPORTED),
    (dict(bs=8), UNSUPPORTED), (dict(k=None), INVALID), (dict(vn=None), INVALID),
    (dict(table=None), INVALID), (dict(mbps=0), INVALID), (dict(nb=0), INVALID),
    (dict(k=FAKE + 2), INVALID), (dict(kn=FAKE + 8), INVALID), (dict(v=FAKE + 1), INVALID),
    (dict(mbps=1 << 28), INVALID), (dict(batch=1 << 28, hkv=16), INVALID),
    (dict(stride=8 * 2048 - 8), INVALID), (dict(stride=8 * 2048 + 2), INVALID),
    (dict(stride=-1), INVALID), (dict(stride=1 << 40, nb=1 << 22), INVALID),
])
def test_kv_append_rejects(lib, kw, code):
    assert append_call(lib, **kw) == code
    assert lib.neo_last_error().decode()


def test_kv_append_empty_batch_is_a_noop(lib):
    assert append_call(lib, batch=0, k=None, v=None, kn=None, vn=None, table=None,
                       lens=None) == OK


def copy_call(lib, **kw):
    a = dict(sk=FAKE, sv=FAKE, dk=FAKE, dv=FAKE, si=FAKE, di=FAKE, n=4, hkv=8, d=128, bs=16,
             snb=100, dnb=100, sst=0, dst=0)
    a.update(kw)
    return lib.neo_kv_copy_blocks(a["sk"], a["sv"], a["dk"], a["dv"], a["si"], a["di"], a["n"],
                                  a["hkv"], a["d"], a["bs"], a["snb"], a["dnb"], a["sst"],
                                  a["dst"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(n=-1), INVALID), (dict(hkv=-2), INVALID), (dict(d=256), UNSUPPORTED),
    (dict(bs=32), UNSUPPORTED), (dict(sk=None), INVALID), (dict(dv=None), INVALID),
    (dict(di=None), INVALID), (dict(snb=0), INVALID), (dict(dnb=-5), INVALID),
    (dict(sv=FAKE + 8), INVALID), (dict(dk=FAKE + 4), INVALID),
    (dict(sst=8 * 2048 - 8), INVALID), (dict(dst=2 * 8 * 2048 + 6), INVALID),
    (dict(dst=(1 << 40) + 8), INVALID), (dict(sst=1 << 40, snb=1 << 22), INVALID),
    (dict(dst=1 << 39, dnb=1 << 23), INVALID),
])
def test_kv_copy_blocks_rejects(lib, kw, code):
    assert copy_call(lib, **kw) == code
    assert lib.neo_last_error().decode()


@pytest.mark.parametrize("src,nbytes,sink,words", [
    (None, 16, FAKE, 16384), (FAKE, 16, None, 16384), (FAKE, 0, FAKE, 16384),
    (FAKE, 24, FAKE, 16384), (FAKE + 8, 16, FAKE, 16384), (FAKE, 16, FAKE, 16383),
])
def test_read_probe_rejects(lib, src, nbytes, sink, words):
    assert lib.neo_read_probe(src, nbytes, 1, sink, words, None) == INVALID
    assert lib.neo_last_error().decode()


@pytest.mark.parametrize("src,nbytes,wpc,depth,weighted,sink", [
    (None, 8192, 4, 1, 0, FAKE), (FAKE, 8192, 4, 1, 0, None), (FAKE, 4096, 4, 1, 0, FAKE),
    (FAKE, 8192 << 31, 4, 1, 0, FAKE), (FAKE + 16, 8192, 4, 1, 0, FAKE),
    (FAKE, 8192, 6, 1, 0, FAKE), (FAKE, 8192, 4, 5, 0, FAKE), (FAKE, 8192, 4, 1, 2, FAKE),
])
def test_read_probe_tiles_rejects(lib, src, nbytes, wpc, depth, weighted, sink):
    assert lib.neo_read_probe_tiles(src, nbytes, wpc, depth, weighted, sink, 4096, None) == INVALID
    assert lib.neo_last_error().decode()


def test_read_probe_sink_size_matches_header():
    text = open(HEADER).read()
    assert int(re.search(r"#define NEO_READ_PROBE_SINK_WORDS (\d+)", text).group(1)) == \
        neo.READ_PROBE_SINK_WORDS


def test_kv_copy_blocks_zero_blocks_is_a_noop(lib):
    assert copy_call(lib, n=0, sk=None, sv=None, dk=None, dv=None, si=None, di=None) == OK


def test_python_binding_refuses_cpu_tensors():
    import torch
    q = torch.zeros(2, 8, 128, dtype=torch.bfloat16)
    k = torch.zeros(4, 2, 16, 16, 8, dtype=torch.bfloat16)
    v = torch.zeros(4, 2, 128, 16, dtype=torch.bfloat16)
    bt = torch.zeros(2, 2, dtype=torch.int32)
    sl = torch.ones(2, dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU"):
        neo.decode_attention(q, k, v, bt, sl)


def test_noalloc_entry_point_checks_arguments_before_any_hip_call(lib):
    def na(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, table=FAKE, lens=FAKE, hq=32, hkv=8, d=128, bs=16,
                 scale=0.1, out=FAKE, batch=4, mbps=8, nb=100)
        a.update(kw)
        return lib.neo_decode_attention_noalloc(a["q"], a["k"], a["v"], a["table"], a["lens"],
                                                a["hq"], a["hkv"], a["d"], a["bs"], a["scale"],
                                                a["out"], a["batch"], a["mbps"], a["nb"],
                                                a.get("stride", 0), None)
    assert na(hkv=7) == INVALID
    assert na(d=64) == UNSUPPORTED
    assert na(bs=8) == UNSUPPORTED
    assert na(scale=float("nan")) == INVALID
    assert na(out=None) == INVALID
    assert na(q=FAKE + 4) == INVALID
    assert na(stride=8 * 2048 - 8) == INVALID
    assert na(stride=2 * 8 * 2048 + 4) == INVALID
    assert na(batch=0, q=None, k=None, v=None, table=None, lens=None, out=None) == OK


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    # No fallback: with the shared library absent every entry point raises.
    monkeypatch.setattr(neo, "_LIB_PATH", str(tmp_path / "missing_libneoattn.so"))
    monkeypatch.setattr(neo, "_lib", None)
    with pytest.raises(ImportError):
        neo.load_library()
    with pytest.raises(ImportError):
        neo.workspace_bytes(4, 32, 8)
