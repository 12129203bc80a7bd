"""Batched paged GQA decode attention for AMD Instinct MI355X (gfx950).

Thin ctypes binding over ``libneoattn.so`` (C ABI in ``include/libneoattn.h``).
Every step of the operation runs in the library's HIP kernels; this module only
checks tensor shapes, derives the scalar arguments and passes device pointers
and torch's current stream. There is no CPU fallback: without the built library
or a GPU every call raises.

The operation (Neo, arXiv 2411.01142, Sec. 2.1-2.2 and Sec. 4): each request's
new query token attends over its own paged KV cache, query heads sharing KV
heads in groups. Layouts (torch tensors, all on one GPU):

* ``q``           bf16  ``[batch, num_q_heads, 128]``
* ``k_cache``     bf16  ``[num_blocks, num_kv_heads, 16, 16, 8]``  (piece-major keys)
* ``v_cache``     bf16  ``[num_blocks, num_kv_heads, 128, 16]``    (dim-major values)

  dense within each block; the blocks themselves may be strided (the same stride
  in both caches): ``new_kv_cache`` returns both as views of one allocation with
  each block's K and V adjacent, the fastest layout measured on MI355X.
* ``block_table`` int32 ``[batch, max_blocks_per_seq]``
* ``seq_lens``    int32 ``[batch]``
* result          fp32  ``[batch, num_q_heads, 128]``
"""
from __future__ import annotations

import ctypes
import math
import os
import threading

__all__ = [
    "NeoError", "decode_attention", "workspace_bytes", "paged_gather", "debug_validate",
    "library_path", "load_library", "VARIANTS", "SCHEDULES", "MAX_SLICES", "version",
    "new_workspace", "kv_append", "copy_blocks", "cpu_decode_attention", "CPU_ISAS",
    "cpu_best_isa", "cpu_default_threads", "cpu_read_probe", "cpu_kv_append",
    "read_probe", "read_probe_tiles", "READ_PROBE_SINK_WORDS", "new_kv_cache",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libneoattn.so")

CPU_ISAS = {"auto": 0, "generic": 1, "avx512_bf16": 2, "avx512": 3}
VARIANTS = {"auto": 0, "valu": 1, "mfma": 2}
SCHEDULES = {"auto": 0, "fused": 1, "staged": 2, "two_kernel": 3}
MAX_SLICES = 4096
READ_PROBE_SINK_WORDS = 16384
STATUS = {0: "NEO_OK", 1: "NEO_ERR_INVALID_ARG", 2: "NEO_ERR_UNSUPPORTED",
          3: "NEO_ERR_WORKSPACE", 4: "NEO_ERR_HIP"}

_lib = None
_lock = threading.Lock()
_workspaces = {}


class NeoError(RuntimeError):
    """A non-OK status from libneoattn; ``status`` holds the code."""

    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libneoattn.so (built by ``__graft_entry__.build()``); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is not built; run `python -c 'import __graft_entry__ "
                              "as g; g.build()'` first")
        try:
            # Import torch first so the library binds to the HIP runtime torch
            # already loaded (both carry the same soname): one runtime per process.
            import torch  # noqa: F401
        except ImportError:
            pass
        lib = ctypes.CDLL(_LIB_PATH)
        P, I, F, S = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
        lib.neo_decode_workspace_bytes.argtypes = [I, I, I, I, ctypes.POINTER(S)]
        lib.neo_decode_workspace_bytes.restype = ctypes.c_int
        lib.neo_decode_attention.argtypes = [P, P, P, P, P, I, I, I, I, F, P, I, I, I, P, S, P]
        lib.neo_decode_attention.restype = ctypes.c_int
        L = ctypes.c_int64
        lib.neo_decode_attention_ex.argtypes = [P, P, P, P, P, I, I, I, I, F, P, I, I, I, P, S,
                                                I, I, I, L, P]
        lib.neo_decode_attention_ex.restype = ctypes.c_int
        lib.neo_decode_attention_events.argtypes = [P, P, P, P, P, I, I, I, I, F, P, I, I, I, P,
                                                    S, I, I, I, L, P, P, P]
        lib.neo_decode_attention_events.restype = ctypes.c_int
        lib.neo_decode_attention_noalloc.argtypes = [P, P, P, P, P, I, I, I, I, F, P, I, I, I, L, P]
        lib.neo_decode_attention_noalloc.restype = ctypes.c_int
        lib.neo_decode_workspace_init.argtypes = [P, S, P]
        lib.neo_decode_workspace_init.restype = ctypes.c_int
        lib.neo_paged_gather.argtypes = [P, I, P, P, P, I, I, I, I, I, I, L, P, P]
        lib.neo_paged_gather.restype = ctypes.c_int
        lib.neo_kv_append.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, L, P]
        lib.neo_kv_append.restype = ctypes.c_int
        lib.neo_kv_copy_blocks.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, L, L, P]
        lib.neo_read_probe.argtypes = [P, S, I, P, S, P]
        lib.neo_read_probe.restype = ctypes.c_int
        lib.neo_read_probe_tiles.argtypes = [P, S, I, I, I, P, S, P]
        lib.neo_read_probe_tiles.restype = ctypes.c_int
        lib.neo_kv_copy_blocks.restype = ctypes.c_int
        lib.neo_cpu_decode_attention_ex.argtypes = [P, P, P, P, P, I, I, I, I, F, P, I, I, I, I, I]
        lib.neo_cpu_decode_attention_ex.restype = ctypes.c_int
        lib.neo_cpu_decode_attention.argtypes = [P, P, P, P, P, I, I, I, I, F, P, I, I, I, I]
        lib.neo_cpu_decode_attention.restype = ctypes.c_int
        lib.neo_cpu_kv_append.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I]
        lib.neo_cpu_kv_append.restype = ctypes.c_int
        lib.neo_cpu_read_probe.argtypes = [P, ctypes.c_size_t, I, ctypes.POINTER(ctypes.c_double)]
        lib.neo_cpu_read_probe.restype = ctypes.c_int
        lib.neo_cpu_best_isa.argtypes = []
        lib.neo_cpu_best_isa.restype = ctypes.c_int32
        lib.neo_cpu_default_threads.argtypes = []
        lib.neo_cpu_default_threads.restype = ctypes.c_int32
        lib.neo_debug_validate.argtypes = [P, P, I, I, I, I, P, P]
        lib.neo_debug_validate.restype = ctypes.c_int
        lib.neo_last_error.argtypes = []
        lib.neo_last_error.restype = ctypes.c_char_p
        lib.neo_version.argtypes = []
        lib.neo_version.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def version() -> str:
    return load_library().neo_version().decode()


def _check(status: int):
    if status != 0:
        msg = load_library().neo_last_error().decode(errors="replace")
        raise NeoError(status, msg)


def workspace_bytes(batch: int, num_q_heads: int, num_kv_heads: int, head_dim: int = 128) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().neo_decode_workspace_bytes(int(batch), int(num_q_heads),
                                                     int(num_kv_heads), int(head_dim),
                                                     ctypes.byref(out)))
    return int(out.value)


def _torch():
    import torch
    return torch


def _require(t, name, dtype, ndim):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU (got {t.device}); there is no CPU path")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims (got shape {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _require_cache(t, name, ndim, *, pinned_ok=False):
    """A bf16 GPU cache tensor (or, with ``pinned_ok``, one in pinned host
    memory) whose blocks (dim 0) may be strided: every dim but the first dense,
    the block stride a multiple of 8 elements of at least one block. Returns the
    block stride in elements."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda" and not (pinned_ok and t.is_pinned()):
        where = "on a GPU or in pinned host memory" if pinned_ok else "on a GPU"
        raise ValueError(f"{name} must be {where} (got {t.device}); there is no CPU path")
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be torch.bfloat16 (got {t.dtype})")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims (got shape {tuple(t.shape)})")
    inner = math.prod(t.shape[1:])
    want = [math.prod(t.shape[d + 1:]) for d in range(1, ndim)]
    if list(t.stride()[1:]) != want or t.stride(0) < inner or t.stride(0) % 8 != 0:
        raise ValueError(f"{name} must be dense within each block, with a block stride that is "
                         f"a multiple of 8 elements of at least {inner} (strides {t.stride()})")
    return int(t.stride(0))


def new_kv_cache(num_blocks: int, num_kv_heads: int, device="cuda", head_dim: int = 128,
                 block_size: int = 16):
    """(k_cache, v_cache) views of one allocation ``[num_blocks][K, V][num_kv_heads][tile]``:
    each block's K and V in one run, the caches' block stride twice a block. Shapes as the
    dense caches (``[NB, Hkv, 16, 16, 8]`` and ``[NB, Hkv, 128, 16]``); ``decode_attention``
    reads the stride from them. Uninitialised."""
    torch = _torch()
    tile = head_dim * block_size
    buf = torch.empty((num_blocks, 2, num_kv_heads, tile), dtype=torch.bfloat16, device=device)
    k = buf[:, 0].view(num_blocks, num_kv_heads, head_dim // 8, block_size, 8)
    v = buf[:, 1].view(num_blocks, num_kv_heads, head_dim, block_size)
    return k, v


def _stream_of(stream, device):
    torch = _torch()
    return torch.cuda.current_stream(device) if stream is None else stream


def _stream_handle(stream, device):
    return ctypes.c_void_p(_stream_of(stream, device).cuda_stream)


def new_workspace(batch: int, num_q_heads: int, num_kv_heads: int, device="cuda",
                  head_dim: int = 128, *, stream=None):
    """A workspace (uint8 GPU tensor) sized for these shapes, allocated for and
    zero-filled on ``stream`` (default: the current stream), so the first
    decode call on that stream sees it cleared."""
    torch = _torch()
    device = torch.device(device)
    if device.index is None:
        device = torch.device("cuda", torch.cuda.current_device())
    s = _stream_of(stream, device)
    nbytes = workspace_bytes(batch, num_q_heads, num_kv_heads, head_dim)
    with torch.cuda.device(device), torch.cuda.stream(s):
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _check(load_library().neo_decode_workspace_init(ws.data_ptr(), nbytes,
                                                        ctypes.c_void_p(s.cuda_stream)))
    return ws


def _workspace(nbytes: int, device, stream):
    """The cached workspace of (device, stream): allocated in that stream's
    pool and cleared on that stream, so the kernels that use it are ordered
    after the fill and a replaced buffer is reused only after them."""
    torch = _torch()
    key = (device.index, stream.cuda_stream)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        with torch.cuda.device(device), torch.cuda.stream(stream):
            ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
            _check(load_library().neo_decode_workspace_init(
                ws.data_ptr(), nbytes, ctypes.c_void_p(stream.cuda_stream)))
        _workspaces[key] = ws
    return ws


def decode_attention(q, k_cache, v_cache, block_table, seq_lens, scale=None, out=None, *,
                     workspace=None, variant: str = "auto", schedule: str = "auto",
                     max_slices: int = 0, stream=None):
    """Decode attention of the whole ragged batch; returns ``out`` (fp32 [B, Hq, 128]).

    ``scale`` defaults to 1/sqrt(head_dim). ``variant`` picks the kernel family
    ("auto", "valu", "mfma"); ``schedule`` the launch ("auto"/"fused": one
    kernel; "two_kernel": decode then combine; "staged": plan, decode and
    combine); ``max_slices`` caps
    the sequence slices of the plan (0 = library default, 1 = never split a
    request). ``workspace`` (a zero-filled uint8 GPU tensor of at least
    ``workspace_bytes(...)``, see ``new_workspace``; the fill must be ordered
    before this call's stream reaches the kernel) is allocated, cleared on
    ``stream`` and cached per device and stream when omitted. Runs on
    ``stream`` (default: torch's current stream) without synchronising.
    """
    torch = _torch()
    lib = load_library()
    _require(q, "q", torch.bfloat16, 3)
    k_stride = _shared_stride(k_cache, "k_cache", v_cache, "v_cache")
    _require(block_table, "block_table", torch.int32, 2)
    _require(seq_lens, "seq_lens", torch.int32, 1)
    B, Hq, D = q.shape
    NB, Hkv, npieces, bs, x = k_cache.shape
    if npieces * x != D or x != 8:
        raise ValueError(f"k_cache shape {tuple(k_cache.shape)} does not match head_dim {D}")
    if tuple(v_cache.shape) != (NB, Hkv, D, bs):
        raise ValueError(f"v_cache shape {tuple(v_cache.shape)} != {(NB, Hkv, D, bs)}")
    if block_table.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_table and seq_lens must have batch rows")
    devs = {t.device for t in (q, k_cache, v_cache, block_table, seq_lens)}
    if len(devs) != 1:
        raise ValueError("all tensors must be on one device")
    device = q.device
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.float32, device=device)
    else:
        _require(out, "out", torch.float32, 3)
        if tuple(out.shape) != (B, Hq, D) or out.device != device:
            raise ValueError("out must be fp32 [batch, num_q_heads, head_dim] on q's device")
    if variant not in VARIANTS:
        raise ValueError(f"variant must be one of {sorted(VARIANTS)}")
    if schedule not in SCHEDULES:
        raise ValueError(f"schedule must be one of {sorted(SCHEDULES)}")
    st = _stream_of(stream, device)
    sh = ctypes.c_void_p(st.cuda_stream)
    if B == 0:
        return out
    need = workspace_bytes(B, Hq, Hkv, D)
    if workspace is None:
        workspace = _workspace(need, device, st)
    else:
        _require(workspace, "workspace", torch.uint8, 1)
    with torch.cuda.device(device):
        _check(lib.neo_decode_attention_ex(
            q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
            seq_lens.data_ptr(), Hq, Hkv, D, bs, float(scale), out.data_ptr(), B,
            block_table.shape[1], NB, workspace.data_ptr(), workspace.numel(),
            VARIANTS[variant], SCHEDULES[schedule], int(max_slices), k_stride, sh))
    return out


def paged_gather(cache, kind: str, block_table, seq_lens, *, token_offsets=None, stream=None):
    """Dense bf16 copy ``[sum L, num_kv_heads, head_dim]`` of the K (``kind='k'``) or V cache."""
    torch = _torch()
    lib = load_library()
    if kind == "k":
        stride = _require_cache(cache, "cache", 5)
        NB, Hkv, npieces, bs, x = cache.shape
        D = npieces * x
    elif kind == "v":
        stride = _require_cache(cache, "cache", 4)
        NB, Hkv, D, bs = cache.shape
    else:
        raise ValueError("kind must be 'k' or 'v'")
    _require(block_table, "block_table", torch.int32, 2)
    _require(seq_lens, "seq_lens", torch.int32, 1)
    B = seq_lens.shape[0]
    device = cache.device
    if token_offsets is None:
        token_offsets = torch.zeros(B + 1, dtype=torch.int32, device=device)
        token_offsets[1:] = torch.cumsum(seq_lens.clamp(min=0), 0)
    total = int(token_offsets[-1].item()) if B else 0
    dst = torch.empty((max(total, 0), Hkv, D), dtype=torch.bfloat16, device=device)
    if B == 0 or total == 0:
        return dst
    sh = _stream_handle(stream, device)
    with torch.cuda.device(device):
        _check(lib.neo_paged_gather(cache.data_ptr(), 1 if kind == "v" else 0,
                                    block_table.data_ptr(), seq_lens.data_ptr(),
                                    token_offsets.data_ptr(), B, block_table.shape[1], Hkv, D,
                                    bs, NB, stride, dst.data_ptr(), sh))
    return dst


def debug_validate(block_table, seq_lens, num_blocks: int, block_size: int = 16, *,
                   stream=None) -> int:
    """Number of out-of-range lengths and in-use block ids (synchronises to read it)."""
    torch = _torch()
    lib = load_library()
    _require(block_table, "block_table", torch.int32, 2)
    _require(seq_lens, "seq_lens", torch.int32, 1)
    device = block_table.device
    cnt = torch.zeros(1, dtype=torch.int32, device=device)
    sh = _stream_handle(stream, device)
    with torch.cuda.device(device):
        _check(lib.neo_debug_validate(block_table.data_ptr(), seq_lens.data_ptr(),
                                      seq_lens.shape[0], block_table.shape[1], int(block_size),
                                      int(num_blocks), cnt.data_ptr(), sh))
    return int(cnt.item())


def kv_append(k_cache, v_cache, k_new, v_new, block_table, seq_lens, *, stream=None):
    """Write each request's newest token (k_new, v_new: bf16 [B, Hkv, 128]) into the
    paged caches at token seq_lens[b] - 1 (in place, on ``stream``). The caches may
    be dense or share one block stride (``new_kv_cache``)."""
    torch = _torch()
    lib = load_library()
    stride = _shared_stride(k_cache, "k_cache", v_cache, "v_cache")
    _require(k_new, "k_new", torch.bfloat16, 3)
    _require(v_new, "v_new", torch.bfloat16, 3)
    _require(block_table, "block_table", torch.int32, 2)
    _require(seq_lens, "seq_lens", torch.int32, 1)
    NB, Hkv, npieces, bs, x = k_cache.shape
    B = seq_lens.shape[0]
    if tuple(k_new.shape) != (B, Hkv, npieces * x) or k_new.shape != v_new.shape:
        raise ValueError("k_new and v_new must be [batch, num_kv_heads, head_dim]")
    sh = _stream_handle(stream, k_cache.device)
    with torch.cuda.device(k_cache.device):
        _check(lib.neo_kv_append(k_cache.data_ptr(), v_cache.data_ptr(), k_new.data_ptr(),
                                 v_new.data_ptr(), block_table.data_ptr(), seq_lens.data_ptr(),
                                 B, block_table.shape[1], Hkv, npieces * x, bs, NB, stride,
                                 sh))


def _shared_stride(k, k_name, v, v_name, *, pinned_ok=False):
    """Block stride of a K and V cache pair (both must have the same one)."""
    ks = _require_cache(k, k_name, 5, pinned_ok=pinned_ok)
    vs = _require_cache(v, v_name, 4, pinned_ok=pinned_ok)
    if ks != vs:
        raise ValueError(f"{k_name} and {v_name} must share one block stride ({ks} != {vs})")
    return ks


def copy_blocks(src_k, src_v, dst_k, dst_v, src_ids, dst_ids, *, stream=None, device=None):
    """dst block dst_ids[i] <- src block src_ids[i] for K and V. Caches may be GPU
    tensors or pinned host tensors (``pin_memory=True``), dense or with a block
    stride shared by the pair (source and destination strides may differ); ids
    are int32 GPU tensors. Runs as one kernel on ``stream`` (of ``device``,
    default: the ids')."""
    torch = _torch()
    lib = load_library()
    src_stride = _shared_stride(src_k, "src_k", src_v, "src_v", pinned_ok=True)
    dst_stride = _shared_stride(dst_k, "dst_k", dst_v, "dst_v", pinned_ok=True)
    _require(src_ids, "src_ids", torch.int32, 1)
    _require(dst_ids, "dst_ids", torch.int32, 1)
    if src_ids.shape != dst_ids.shape:
        raise ValueError("src_ids and dst_ids must have the same length")
    if src_k.shape[1:] != dst_k.shape[1:] or src_v.shape[1:] != dst_v.shape[1:]:
        raise ValueError("source and destination caches must share the block layout")
    NB_s, Hkv, npieces, bs, x = src_k.shape
    device = src_ids.device if device is None else device
    sh = _stream_handle(stream, device)
    with torch.cuda.device(device):
        _check(lib.neo_kv_copy_blocks(src_k.data_ptr(), src_v.data_ptr(), dst_k.data_ptr(),
                                      dst_v.data_ptr(), src_ids.data_ptr(), dst_ids.data_ptr(),
                                      src_ids.shape[0], Hkv, npieces * x, bs, NB_s,
                                      dst_k.shape[0], src_stride, dst_stride, sh))


def read_probe(src, sink, *, nontemporal: bool = True, stream=None):
    """Stream-read the GPU tensor ``src`` once (its bytes, a multiple of 16) and
    write ``READ_PROBE_SINK_WORDS`` per-wave xor words into ``sink`` (an int32 or
    uint32-sized GPU tensor): a measurement of the device's read rate. Runs on
    ``stream`` without synchronising."""
    torch = _torch()
    lib = load_library()
    if not (src.is_cuda and sink.is_cuda) or not src.is_contiguous() or not sink.is_contiguous():
        raise ValueError("src and sink must be contiguous GPU tensors")
    if sink.numel() * sink.element_size() < 4 * READ_PROBE_SINK_WORDS:
        raise ValueError(f"sink must hold {READ_PROBE_SINK_WORDS} 32-bit words")
    sh = _stream_handle(stream, src.device)
    with torch.cuda.device(src.device):
        _check(lib.neo_read_probe(src.data_ptr(), src.numel() * src.element_size(),
                                  int(bool(nontemporal)), sink.data_ptr(),
                                  sink.numel() * sink.element_size() // 4, sh))


def read_probe_tiles(src, sink, *, waves_per_cu: int = 4, depth: int = 1,
                     xcd_weighted: bool = False, stream=None):
    """Read the GPU tensor ``src`` (its bytes, a multiple of 8192) once in the
    decode kernel's pattern (contiguous 8 KiB steps per wave, ``waves_per_cu``
    waves per compute unit, ``depth`` steps in flight; ``xcd_weighted``: the
    ranges weighted by XCD like the decode kernel's slices) and write one xor
    word per wave into ``sink`` (``READ_PROBE_SINK_WORDS`` 32-bit words
    suffice). Runs on ``stream`` without synchronising."""
    torch = _torch()
    lib = load_library()
    if not (src.is_cuda and sink.is_cuda) or not src.is_contiguous() or not sink.is_contiguous():
        raise ValueError("src and sink must be contiguous GPU tensors")
    sh = _stream_handle(stream, src.device)
    with torch.cuda.device(src.device):
        _check(lib.neo_read_probe_tiles(src.data_ptr(), src.numel() * src.element_size(),
                                        int(waves_per_cu), int(depth), int(bool(xcd_weighted)),
                                        sink.data_ptr(),
                                        sink.numel() * sink.element_size() // 4, sh))


def cpu_best_isa() -> str:
    """The CPU attention path ``isa="auto"`` takes on this host."""
    code = load_library().neo_cpu_best_isa()
    return {v: k for k, v in CPU_ISAS.items()}[code]


def cpu_default_threads() -> int:
    return int(load_library().neo_cpu_default_threads())


def _host_array(a, name, dtype_np, ndim):
    """(pointer, keep-alive) of a C-contiguous host array: numpy of ``dtype_np``
    or a CPU torch tensor of the matching dtype (bf16 for uint16 storage)."""
    import numpy as np
    try:
        torch = _torch()
    except ImportError:  # pragma: no cover
        torch = None
    if torch is not None and isinstance(a, torch.Tensor):
        if a.device.type != "cpu":
            raise ValueError(f"{name} must be in host memory (got {a.device})")
        want = {np.uint16: torch.bfloat16, np.int32: torch.int32, np.float32: torch.float32}
        if a.dtype != want[dtype_np] or a.dim() != ndim or not a.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {want[dtype_np]} tensor with {ndim} dims")
        return a.data_ptr(), a
    if not isinstance(a, np.ndarray) or a.dtype != dtype_np or a.ndim != ndim or \
            not a.flags.c_contiguous:
        raise ValueError(f"{name} must be a C-contiguous {np.dtype(dtype_np)} array with {ndim} dims")
    return a.ctypes.data, a


def cpu_decode_attention(q, k_cache, v_cache, block_table, seq_lens, scale=None, out=None, *,
                         num_threads: int = 0, isa: str = "auto"):
    """Decode attention on the host CPU over host-memory caches (same layouts as
    ``decode_attention``). bf16 data is passed as numpy uint16 arrays (bit
    patterns) or CPU bf16 tensors. Returns ``out``: float32 [B, Hq, 128]."""
    import numpy as np
    lib = load_library()
    qp, _ = _host_array(q, "q", np.uint16, 3)
    kp, _ = _host_array(k_cache, "k_cache", np.uint16, 5)
    vp, _ = _host_array(v_cache, "v_cache", np.uint16, 4)
    bp, _ = _host_array(block_table, "block_table", np.int32, 2)
    lp, _ = _host_array(seq_lens, "seq_lens", np.int32, 1)
    B, Hq, D = q.shape
    NB, Hkv, npieces, bs, x = k_cache.shape
    if out is None:
        out = np.empty((B, Hq, D), dtype=np.float32)
    op, _ = _host_array(out, "out", np.float32, 3)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    _check(lib.neo_cpu_decode_attention_ex(qp, kp, vp, bp, lp, Hq, Hkv, D, bs, float(scale), op,
                                           B, block_table.shape[1], NB, int(num_threads),
                                           CPU_ISAS[isa]))
    return out


def cpu_read_probe(buf, num_threads: int = 0) -> float:
    """Read the whole host array ``buf`` (size a multiple of 64 bytes) once with the
    CPU attention's thread pool; returns the checksum (time the call for GB/s)."""
    import numpy as np
    if not isinstance(buf, np.ndarray) or not buf.flags.c_contiguous:
        raise ValueError("buf must be a C-contiguous numpy array")
    out = ctypes.c_double(0.0)
    _check(load_library().neo_cpu_read_probe(buf.ctypes.data, buf.nbytes, int(num_threads),
                                             ctypes.byref(out)))
    return out.value


def cpu_kv_append(k_cache, v_cache, k_new, v_new, block_table, seq_lens):
    """``kv_append`` for host-memory caches (numpy uint16 bit patterns or CPU bf16
    tensors), on the calling thread."""
    import numpy as np
    lib = load_library()
    kp, _ = _host_array(k_cache, "k_cache", np.uint16, 5)
    vp, _ = _host_array(v_cache, "v_cache", np.uint16, 4)
    knp, _ = _host_array(k_new, "k_new", np.uint16, 3)
    vnp, _ = _host_array(v_new, "v_new", np.uint16, 3)
    bp, _ = _host_array(block_table, "block_table", np.int32, 2)
    lp, _ = _host_array(seq_lens, "seq_lens", np.int32, 1)
    NB, Hkv, npieces, bs, x = k_cache.shape
    B = seq_lens.shape[0]
    if tuple(k_new.shape) != (B, Hkv, npieces * x) or tuple(v_new.shape) != tuple(k_new.shape):
        raise ValueError("k_new and v_new must be [batch, num_kv_heads, head_dim]")
    _check(lib.neo_cpu_kv_append(kp, vp, knp, vnp, bp, lp, B, block_table.shape[1], Hkv,
                                 npieces * x, bs, NB))
