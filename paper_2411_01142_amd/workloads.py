"""Seeded synthetic inputs for batched paged GQA decode attention.

This module only builds inputs: it draws random values, rounds them to bf16,
assigns physical KV-cache blocks to requests and writes values into the paged
storage layout. It computes nothing of the attention itself, and it is the one
module that both the HIP path's tests and the fp64 oracle's tests take inputs
from.

Storage contract (the paged KV cache of Sec. 2.1 and Sec. 4 of the paper,
whose layout the paper likens to vLLM's):

* ``q``           bf16 ``[batch][num_q_heads][head_dim]``
* ``k_cache``     bf16 ``[num_blocks][num_kv_heads][head_dim/8][block_size][8]``
  (each token's key is cut into 16-byte pieces of 8 dims; piece-major inside
  a block, so one (block, kv head) tile is one contiguous run)
* ``v_cache``     bf16 ``[num_blocks][num_kv_heads][head_dim][block_size]``
  (dim-major inside a block)
* ``block_table`` int32 ``[batch][max_blocks_per_seq]``; logical block ``j`` of
  request ``b`` lives in physical block ``block_table[b][j]``; unused entries
  hold -1
* ``seq_lens``    int32 ``[batch]``: tokens in the cache, including the token
  being decoded (its K/V already appended, Sec. 2.1).

Token ``t`` of request ``b`` is slot ``t % block_size`` of physical block
``block_table[b][t // block_size]``.

Workload recipes follow the five layer shapes the method is evaluated on
(Sec. 5.1: LLaMa-2-7B, LLaMa-3.1-8B, LLaMa-3.1-70B) with length mixes that
stand in for the coding and summarisation traces; see ``CONFIGS``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Optional, Sequence

import numpy as np

BF16_NAN = np.uint16(0x7FC0)
K_PACK = 8  # dims per 16-byte piece of a key row

__all__ = [
    "Case", "CONFIGS", "make_config", "build_case", "to_bf16", "bf16_to_f32",
    "pack_k", "pack_v", "unpack_k", "unpack_v", "BF16_NAN", "K_PACK",
]


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = ((u + rounding) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    """Widen bf16 bits (uint16) to float32 exactly."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def pack_k(k_logical: np.ndarray) -> np.ndarray:
    """[NB][Hkv][bs][D] -> storage [NB][Hkv][D/8][bs][8]."""
    nb, hkv, bs, d = k_logical.shape
    assert d % K_PACK == 0
    return np.ascontiguousarray(
        k_logical.reshape(nb, hkv, bs, d // K_PACK, K_PACK).transpose(0, 1, 3, 2, 4))


def unpack_k(k_cache: np.ndarray) -> np.ndarray:
    """Storage [NB][Hkv][D/8][bs][8] -> [NB][Hkv][bs][D]."""
    nb, hkv, dp, bs, x = k_cache.shape
    return np.ascontiguousarray(k_cache.transpose(0, 1, 3, 2, 4).reshape(nb, hkv, bs, dp * x))


def pack_v(v_logical: np.ndarray) -> np.ndarray:
    """[NB][Hkv][bs][D] -> storage [NB][Hkv][D][bs]."""
    return np.ascontiguousarray(v_logical.transpose(0, 1, 3, 2))


def unpack_v(v_cache: np.ndarray) -> np.ndarray:
    """Storage [NB][Hkv][D][bs] -> [NB][Hkv][bs][D]."""
    return np.ascontiguousarray(v_cache.transpose(0, 1, 3, 2))


@dataclasses.dataclass
class Case:
    """One batch of decode-attention inputs in the storage contract above."""
    q: np.ndarray            # uint16 [B][Hq][D]
    k_cache: np.ndarray      # uint16 [NB][Hkv][D/8][bs][8]
    v_cache: np.ndarray      # uint16 [NB][Hkv][D][bs]
    block_table: np.ndarray  # int32 [B][MBPS]
    seq_lens: np.ndarray     # int32 [B]
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    scale: float
    name: str = "case"

    @property
    def batch(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_blocks(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def total_tokens(self) -> int:
        return int(np.maximum(self.seq_lens, 0).sum())

    def algorithmic_bytes(self) -> int:
        """Bytes the operation must move at minimum: every valid K and V row once,
        q in, fp32 out, the block-table entries in use and the lengths."""
        L = np.maximum(self.seq_lens.astype(np.int64), 0)
        kv = int(L.sum()) * self.num_kv_heads * self.head_dim * 2 * 2
        qo = self.batch * self.num_q_heads * self.head_dim * (2 + 4)
        tbl = 4 * int(((L + self.block_size - 1) // self.block_size).sum()) + 4 * self.batch
        return kv + qo + tbl

    def algorithmic_flops(self) -> int:
        """2 flops per multiply-add: q.k and p.V, each head_dim per (token, q head)."""
        L = np.maximum(self.seq_lens.astype(np.int64), 0)
        return int(L.sum()) * self.num_q_heads * self.head_dim * 4

    def to_torch(self, device="cuda", kv_layout: str = "separate", kv_pad: int = 0):
        """(q, k_cache, v_cache, block_table, seq_lens) as torch tensors on ``device``
        (bf16 caches and q, int32 table and lengths).

        ``kv_layout="separate"``: two dense caches. ``"interleaved"``: both caches
        views of one buffer whose block b holds K's block then V's block, plus
        ``kv_pad`` elements (a multiple of 8) after each; the caches' block stride
        is then ``2 * Hkv * head_dim * block_size + kv_pad`` elements."""
        import torch

        def bf16(a):
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(
                torch.bfloat16)
        k, v = bf16(self.k_cache), bf16(self.v_cache)
        if kv_layout == "interleaved":
            nb, per = self.num_blocks, self.num_kv_heads * self.head_dim * self.block_size
            buf = torch.full((nb, 2 * per + kv_pad), float("nan"), dtype=torch.bfloat16,
                             device=device)
            kk = buf[:, :per].view(k.shape)
            vv = buf[:, per:2 * per].view(v.shape)
            kk.copy_(k)
            vv.copy_(v)
            k, v = kk, vv
        elif kv_layout != "separate":
            raise ValueError(f"unknown kv_layout {kv_layout!r}")
        return (bf16(self.q), k, v,
                torch.from_numpy(np.ascontiguousarray(self.block_table)).to(device),
                torch.from_numpy(np.ascontiguousarray(self.seq_lens)).to(device))

    def logical_kv(self):
        """Logical [NB][Hkv][bs][D] views (copies) of the caches, as uint16."""
        return unpack_k(self.k_cache), unpack_v(self.v_cache)


_NORMAL_TABLE = None


def normal_table() -> np.ndarray:
    """bf16 bits of the N(0,1) quantiles at (i + 1/2) / 65536, i = 0..65535.

    Indexing it with uniform 16-bit integers samples N(0,1) at 16-bit
    resolution (tails cut at |x| = 4.17), already rounded to bf16.
    """
    global _NORMAL_TABLE
    if _NORMAL_TABLE is None:
        from scipy.special import ndtri
        u = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
        _NORMAL_TABLE = to_bf16(ndtri(u).astype(np.float32))
    return _NORMAL_TABLE


def _draw_normal_bf16(rng: np.random.Generator, shape, chunk: int = 1 << 26) -> np.ndarray:
    """I.i.d. N(0,1) bf16 bits in C order of ``shape`` (inverse-CDF table sampler)."""
    table = normal_table()
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        idx = rng.integers(0, 65536, size=e - s, dtype=np.uint16)
        np.take(table, idx, out=out[s:e])
    return out.reshape(shape)


def build_case(seq_lens: Sequence[int], num_q_heads: int, num_kv_heads: int,
               head_dim: int = 128, block_size: int = 16, *,
               rng: Optional[np.random.Generator] = None, seed: int = 0,
               poison: bool = True, spare_frac: float = 0.05, shuffle: bool = True,
               k_outlier_frac: float = 0.0, k_outlier_mult: float = 8.0,
               q_values: Optional[np.ndarray] = None,
               k_values: Optional[Callable] = None,
               v_values: Optional[Callable] = None,
               scale: Optional[float] = None, extra_table_cols: int = 0,
               name: str = "case") -> Case:
    """Build a paged batch.

    Draw order from ``rng``: physical-block permutation, q, K, V (K and V
    i.i.d. in storage order), K-outlier mask (``seq_lens`` and any
    config-specific draws come before, from the caller). Random values are
    N(0,1) through ``normal_table``.

    ``q_values`` (float32 [B][Hq][D]) replaces the q draw. ``k_values`` /
    ``v_values`` are callables ``f(b, t, g) -> float32[D]`` giving the logical
    value of token ``t`` of request ``b`` at kv head ``g``; they replace the
    random draw for valid tokens (tests use them for closed-form inputs).
    ``poison`` fills slots past each request's length and unused blocks with
    bf16 NaN; otherwise they keep their N(0,1) draws.
    """
    if rng is None:
        rng = np.random.default_rng(seed)
    L = np.asarray(seq_lens, dtype=np.int64)
    B = int(L.shape[0])
    Hq, Hkv, D, bs = int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size)
    assert Hq % Hkv == 0 and D % K_PACK == 0 and bs >= 1
    nblk = (np.maximum(L, 0) + bs - 1) // bs
    needed = int(nblk.sum())
    nb = needed + int(math.ceil(spare_frac * needed))
    nb = max(nb, 1)
    perm = rng.permutation(nb) if shuffle else np.arange(nb)
    mbps = max(1, int(nblk.max()) if B else 1) + int(extra_table_cols)
    table = np.full((B, mbps), -1, dtype=np.int32)
    cur = 0
    for b in range(B):
        n = int(nblk[b])
        table[b, :n] = perm[cur:cur + n]
        cur += n

    if q_values is not None:
        q = to_bf16(np.asarray(q_values, dtype=np.float32).reshape(B, Hq, D))
    else:
        q = _draw_normal_bf16(rng, (B, Hq, D))
    # Random K and V are drawn i.i.d. directly in storage order.
    k_st = _draw_normal_bf16(rng, (nb, Hkv, D // K_PACK, bs, K_PACK))
    v_st = _draw_normal_bf16(rng, (nb, Hkv, D, bs))

    if k_values is not None or v_values is not None:
        k_log, v_log = unpack_k(k_st), unpack_v(v_st)
        for b in range(B):
            for t in range(int(max(L[b], 0))):
                p, o = int(table[b, t // bs]), t % bs
                for g in range(Hkv):
                    if k_values is not None:
                        k_log[p, g, o] = to_bf16(np.asarray(k_values(b, t, g), dtype=np.float32))
                    if v_values is not None:
                        v_log[p, g, o] = to_bf16(np.asarray(v_values(b, t, g), dtype=np.float32))
        k_st, v_st = pack_k(k_log), pack_v(v_log)

    if k_outlier_frac > 0.0:
        # Independent Bernoulli per (request, token, kv head) over valid tokens;
        # the key row is multiplied by a power of two, exact in bf16.
        for b in range(B):
            n_tok = int(max(L[b], 0))
            if n_tok == 0:
                continue
            mask = rng.random((n_tok, Hkv)) < k_outlier_frac
            ts, gs = np.nonzero(mask)
            for t, g in zip(ts.tolist(), gs.tolist()):
                p, o = int(table[b, t // bs]), t % bs
                row = bf16_to_f32(k_st[p, g, :, o, :]) * np.float32(k_outlier_mult)
                k_st[p, g, :, o, :] = to_bf16(row)

    if poison:
        used = np.zeros(nb, dtype=bool)
        for b in range(B):
            n = int(nblk[b])
            used[table[b, :n]] = True
            rem = int(L[b]) - (n - 1) * bs if n > 0 else bs
            if n > 0 and rem < bs:
                p = int(table[b, n - 1])
                k_st[p, :, :, rem:, :] = BF16_NAN
                v_st[p, :, :, rem:] = BF16_NAN
        k_st[~used] = BF16_NAN
        v_st[~used] = BF16_NAN

    return Case(q=q, k_cache=k_st, v_cache=v_st, block_table=table,
                seq_lens=L.astype(np.int32), num_q_heads=Hq, num_kv_heads=Hkv,
                head_dim=D, block_size=bs,
                scale=float(1.0 / math.sqrt(D)) if scale is None else float(scale),
                name=name)


# --------------------------------------------------------------------------------------
# The five layer-shaped workloads, and one GPU's share of the 70B layer under
# 8-way tensor parallelism. Shapes: LLaMa-2-7B (32 q / 32 kv heads), LLaMa-3-8B
# (32 / 8), LLaMa-3.1-70B (64 / 8; its TP-8 share 8 / 1); head_dim 128,
# block_size 16, bf16 q/K/V ~ N(0,1), scale 1/sqrt(128), shuffled physical blocks.
# --------------------------------------------------------------------------------------

def _lens_cfg1(rng):
    return rng.integers(64, 512, size=4, endpoint=True)


def _lens_cfg2(rng):
    return rng.integers(512, 2048, size=64, endpoint=True)


def _lens_cfg3(rng):
    # Summarisation-like: lognormal with median 1500 and sigma 0.6, clipped to [128, 8192].
    x = rng.lognormal(mean=math.log(1500.0), sigma=0.6, size=256)
    return np.clip(np.rint(x), 128, 8192).astype(np.int64)


def _lens_cfg4(rng):
    # Code-generation-like: uniform in [256, 4096].
    return rng.integers(256, 4096, size=512, endpoint=True)


def _lens_cfg5(rng):
    # Skewed: 8 requests of 32768 tokens at random positions, 1016 of U{16..256}.
    L = rng.integers(16, 256, size=1024, endpoint=True)
    longs = rng.choice(1024, size=8, replace=False)
    L[longs] = 32768
    return L


CONFIGS = {
    1: dict(name="llama2-7b_b4_u64-512", num_q_heads=32, num_kv_heads=32, lens=_lens_cfg1,
            k_outlier_frac=0.0),
    2: dict(name="llama3-8b_b64_u512-2048", num_q_heads=32, num_kv_heads=8, lens=_lens_cfg2,
            k_outlier_frac=0.0),
    3: dict(name="llama3-8b_b256_lognormal1500", num_q_heads=32, num_kv_heads=8, lens=_lens_cfg3,
            k_outlier_frac=0.01),
    4: dict(name="llama3.1-70b_b512_u256-4096", num_q_heads=64, num_kv_heads=8, lens=_lens_cfg4,
            k_outlier_frac=0.0),
    5: dict(name="llama3-8b_b1024_skew8x32k", num_q_heads=32, num_kv_heads=8, lens=_lens_cfg5,
            k_outlier_frac=0.0),
    # One GPU's share of the 70B layer under 8-way tensor parallelism (each GPU holds one kv
    # head and its 8 query heads): configuration 4's lengths and draw order, 1/8 of its KV.
    6: dict(name="llama3.1-70b-tp8share_b512_u256-4096", num_q_heads=8, num_kv_heads=1,
            lens=_lens_cfg4, k_outlier_frac=0.0),
}


def config_seq_lens(cfg: int, seed: int) -> np.ndarray:
    """Only the lengths of a config (first draw of its recipe)."""
    return CONFIGS[cfg]["lens"](np.random.default_rng(seed)).astype(np.int32)


def make_config(cfg: int, seed: Optional[int] = None, *, poison: bool = True,
                batch_limit: Optional[int] = None) -> Case:
    """Config ``cfg`` (1..6) with seed ``seed`` (default: ``cfg``).

    ``batch_limit`` keeps only the first requests (the draw order is unchanged
    for the lengths; later draws then cover the smaller batch).
    """
    spec = CONFIGS[cfg]
    seed = cfg if seed is None else seed
    rng = np.random.default_rng(seed)
    L = spec["lens"](rng)
    if batch_limit is not None:
        L = L[:batch_limit]
    return build_case(L, spec["num_q_heads"], spec["num_kv_heads"], 128, 16, rng=rng,
                      poison=poison, k_outlier_frac=spec["k_outlier_frac"],
                      name=f"cfg{cfg}:{spec['name']}:seed{seed}")
