// The decode driver shared by both kernel families: how a wavefront finds its
// slice of the batch, walks (request, kv head, block) tiles with loads
// issued ahead of use, and where a finished segment's result goes (straight
// to `out`, or to a partial slot that the last contributor merges).
//
// Tiles are numbered request-major, kv-head-next, block-minor; with T tiles
// and n slices, slice s owns [floor(sT/n), floor((s+1)T/n)). A (request, kv
// head) pair whose tiles cross a slice boundary is "cut": every slice that
// touches it writes a partial output normalised over its share plus the
// log-sum-exp of its scores, and the pair is aggregated afterwards (the
// block-granular split and per-request aggregation of Sec. 4 of the paper).
#pragma once

#include <math.h>

#include "neo_internal.h"

namespace neo {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.6931471805599453f;

// ----------------------------------------------------------------- coherent access

// Partials written by one slice and merged by another (possibly on another
// XCD, with its own L2) go through device-coherent accesses: stores that write
// through to the coherence point and loads that read from it. Ordering against
// the arrival counter comes from waiting for every store to complete before
// the counter is incremented, instead of a device-scope fence (which writes
// back and invalidates the whole L2).
__device__ inline void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void wait_all_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// ----------------------------------------------------------------- slice geometry

__device__ inline int32_t slice_first_tile(int64_t s, int32_t T, int32_t n) {
  return (int32_t)((s * T) / n);
}
// The slice holding tile t: the largest s with floor(sT/n) <= t.
__device__ inline int32_t slice_of_tile(int32_t t, int32_t T, int32_t n) {
  return (int32_t)((((int64_t)t + 1) * n - 1) / T);
}
// Partial slot of slice w for a pair starting at tile pair_first: a slice's
// first segment uses 2w, a later (end-cut) segment 2w+1. At most one of each.
__device__ inline int partial_slot(int32_t w, int32_t slice_first, int32_t pair_first) {
  return slice_first >= pair_first ? 2 * w : 2 * w + 1;
}

// Number of slices for T tiles. With min_tiles > 0: T / min_tiles, capped.
// With min_tiles == 0 (the default policy): whole multiples of `quantum` (one
// 4-wave workgroup per CU) so every CU gets the same share, stepping up to
// two workgroups per CU once slices still hold kAutoTilesPerSlice tiles;
// small batches get T / 8 slices.
constexpr int32_t kAutoTilesPerSlice = 40;
constexpr int32_t kSmallTilesPerSlice = 8;

__device__ inline int32_t slice_count(int32_t T, int32_t min_tiles, int32_t max_slices,
                                      int32_t quantum) {
  if (T <= 0) return 0;
  if (min_tiles > 0) return min(max(T / min_tiles, 1), max_slices);
  int32_t n;
  if (T >= 2 * quantum * kAutoTilesPerSlice) n = 2 * quantum;
  else if (T >= quantum * kSmallTilesPerSlice) n = quantum;
  else n = max(T / kSmallTilesPerSlice, 1);
  return min(n, max_slices);
}

struct SliceInfo {
  int32_t T, n;      // total tiles, slices
  int32_t s0, s1;    // this slice's tile range
  int32_t b, g, j;   // coordinates of tile s0
};

// ----------------------------------------------------------------- wave helpers

__device__ inline int32_t wave_sum_i32(int32_t v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ inline float wave_max_f32(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline float wave_sum_f32(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ inline int32_t wave_incl_scan_i32(int32_t v, int lane) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int32_t u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

// ----------------------------------------------------------------- planning

// Slice from the plan kernel's output (staged launch).
__device__ inline SliceInfo read_plan(const DecodeParams& p, int wave) {
  SliceInfo si;
  si.T = p.hdr->total_tiles;
  si.n = p.hdr->n_slices;
  if (wave >= si.n) return si;
  const SliceStart a = p.starts[wave];
  si.s0 = a.tile;
  si.s1 = p.starts[wave + 1].tile;
  si.b = a.b;
  si.g = a.g;
  si.j = a.j;
  return si;
}

// Slice computed by the wavefront itself from seq_lens (fused launch): a
// wave-wide reduction of the block counts gives T; a wave-wide scan locates
// the request holding the slice's first tile. Requests are read 64 per lane
// group, up to kPlanRegs groups per load round.
constexpr int kPlanRegs = 16;

// Block counts of requests base + 64r + lane, r < kPlanRegs (0 past the batch).
// Loads use a clamped index so that all of them issue before any is waited on.
__device__ inline void load_block_counts(const DecodeParams& p, int base, int lane,
                                         int32_t (&nb)[kPlanRegs]) {
  int32_t raw[kPlanRegs];
#pragma unroll
  for (int r = 0; r < kPlanRegs; ++r) raw[r] = p.lens[min(base + r * kWave + lane, p.batch - 1)];
#pragma unroll
  for (int r = 0; r < kPlanRegs; ++r)
    nb[r] = (base + r * kWave + lane < p.batch) ? blocks_of(raw[r], p.mbps) : 0;
}

__device__ inline SliceInfo plan_in_wave(const DecodeParams& p, int wave, int lane) {
  SliceInfo si;
  constexpr int kChunk = kWave * kPlanRegs;
  int32_t nb[kPlanRegs];
  int32_t total = 0;
  for (int base = 0; base < p.batch; base += kChunk) {
    load_block_counts(p, base, lane, nb);
    int32_t s = 0;
#pragma unroll
    for (int r = 0; r < kPlanRegs; ++r) s += nb[r];
    total += wave_sum_i32(s);
  }
  si.T = total * p.hkv;
  si.n = slice_count(si.T, p.min_tiles, p.max_slices, p.slice_quantum);
  if (wave >= si.n) return si;
  si.s0 = slice_first_tile(wave, si.T, si.n);
  si.s1 = slice_first_tile((int64_t)wave + 1, si.T, si.n);

  // Request b holds tiles [hkv*P_b, hkv*P_{b+1}) with P the block prefix sum.
  const int32_t u = si.s0 / p.hkv;
  int32_t carry = 0;
  int32_t found_b = -1, found_p = 0;
  for (int base = 0; base < p.batch && found_b < 0; base += kChunk) {
    if (p.batch > kChunk) load_block_counts(p, base, lane, nb);
#pragma unroll
    for (int r = 0; r < kPlanRegs; ++r) {
      if (found_b >= 0) break;
      const int32_t cs = wave_sum_i32(nb[r]);
      if (carry + cs > u) {
        const int32_t incl = wave_incl_scan_i32(nb[r], lane);
        const uint64_t hit = __ballot(carry + incl > u);
        const int first = __ffsll((unsigned long long)hit) - 1;
        found_b = base + r * kWave + first;
        found_p = carry + __shfl(incl - nb[r], first);
      } else {
        carry += cs;
      }
    }
  }
  const int32_t nbb = blocks_of(p.lens[found_b], p.mbps);
  const int32_t rem = si.s0 - p.hkv * found_p;
  si.b = found_b;
  si.g = rem / nbb;
  si.j = rem % nbb;
  return si;
}

// ----------------------------------------------------------------- outputs

// Requests with no tokens get a zero row; every wavefront takes a strided share.
__device__ inline void zero_empty_rows(const DecodeParams& p, int wave, int nwaves, int lane) {
  for (int b = wave; b < p.batch; b += nwaves) {
    if (clamp_len(p.lens[b], p.mbps) != 0) continue;
    f32x4_t* row = reinterpret_cast<f32x4_t*>(p.out + (size_t)b * p.hq * kHeadDim);
    const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
    for (int i = lane; i < p.hq * (kHeadDim / 4); i += kWave) row[i] = z;
  }
}

// Merge the partials of one cut pair into out[b][g*G .. g*G+G): M = max lse,
// out = sum_c e^(lse_c - M) o_c / sum_c e^(lse_c - M). Contributors are the
// slices c0..c1. Each lane owns dims 2*lane, 2*lane+1 of the sums.
template <int G>
__device__ inline int contributor_slot(int32_t c, int32_t T, int32_t n, int32_t pair_first) {
  return partial_slot(c, slice_first_tile(c, T, n), pair_first);
}

template <int G>
__device__ inline void store_merged(const DecodeParams& p, int32_t b, int32_t g, int h, int d,
                                    float a0, float a1, float z) {
  const float inv = 1.f / z;
  float2 r;
  r.x = a0 * inv;
  r.y = a1 * inv;
  *reinterpret_cast<float2*>(p.out + ((size_t)b * p.hq + g * G + h) * kHeadDim + d) = r;
}

template <int G>
__device__ inline void merge_pair(const DecodeParams& p, int32_t b, int32_t g, int32_t pair_first,
                                  int32_t c0, int32_t c1, int32_t T, int32_t n, int lane) {
  const int k = c1 - c0 + 1;
  const int d = 2 * lane;
  if (k <= kWave) {
    // Lane i reads the log-sum-exps of contributor c0 + i; partial rows are
    // then read kBatch contributors at a time with all loads issued together.
    constexpr int kBatch = 32 / G > 16 ? 16 : (32 / G > 0 ? 32 / G : 1);  // 64 registers
    const int mine = lane < k ? lane : 0;
    const int my_slot = contributor_slot<G>(c0 + mine, T, n, pair_first);
    float w[G], a0[G], a1[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float lse = lane < k ? load_coherent(p.part_lse + my_slot * G + h) : -INFINITY;
      w[h] = __expf(lse - wave_max_f32(lse));
      a0[h] = a1[h] = 0.f;
    }
    for (int i0 = 0; i0 < k; i0 += kBatch) {
      float ov[kBatch][G][2];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (i0 + u >= k) break;  // uniform
        const int slot = contributor_slot<G>(c0 + i0 + u, T, n, pair_first);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float* o = p.part_o + ((size_t)slot * G + h) * kHeadDim + d;
          ov[u][h][0] = load_coherent(o);
          ov[u][h][1] = load_coherent(o + 1);
        }
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (i0 + u >= k) break;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float wi = __shfl(w[h], i0 + u);
          a0[h] = fmaf(wi, ov[u][h][0], a0[h]);
          a1[h] = fmaf(wi, ov[u][h][1], a1[h]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) store_merged<G>(p, b, g, h, d, a0[h], a1[h], wave_sum_f32(w[h]));
    return;
  }
  // More than 64 contributors (a very long request cut into many slices):
  // global maximum first, then the weighted sums, one contributor at a time.
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int base = 0; base < k; base += kWave)
      if (base + lane < k)
        m = fmaxf(m, load_coherent(p.part_lse +
                                   contributor_slot<G>(c0 + base + lane, T, n, pair_first) * G +
                                   h));
    m = wave_max_f32(m);
    float z = 0.f, a0 = 0.f, a1 = 0.f;
    for (int i = 0; i < k; ++i) {
      const int slot = contributor_slot<G>(c0 + i, T, n, pair_first);
      const float wi = __expf(load_coherent(p.part_lse + slot * G + h) - m);
      const float* o = p.part_o + ((size_t)slot * G + h) * kHeadDim + d;
      z += wi;
      a0 = fmaf(wi, load_coherent(o), a0);
      a1 = fmaf(wi, load_coherent(o + 1), a1);
    }
    store_merged<G>(p, b, g, h, d, a0, a1, z);
  }
}

// Fused launch: after writing its partial for a cut pair, a slice counts itself
// in the pair's counter; the slice that completes the count merges the pair
// (returns true) and resets the counter to zero for the next call.
__device__ inline bool arrive_last(const DecodeParams& p, int32_t pair_first, int32_t pair_tiles,
                                   int32_t T, int32_t n, int lane) {
  const int32_t c0 = slice_of_tile(pair_first, T, n);
  const int32_t c1 = slice_of_tile(pair_first + pair_tiles - 1, T, n);
  wait_all_memory();  // this slice's partial has reached the coherence point
  int32_t old = 0;
  if (lane == 0)
    old = __hip_atomic_fetch_add(p.counters + c0, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  old = __shfl(old, 0);
  if (old != c1 - c0) return false;
  if (lane == 0)
    __hip_atomic_store(p.counters + c0, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

// ----------------------------------------------------------------- the driver

// Family provides: Tile, State, Q; load_q, init, load_tile, step, write.
// PF tiles are in flight ahead of the one being computed.
template <class F, int G, int PF, bool kFused>
__device__ inline void decode_driver(const DecodeParams& p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x >> 6;
  const int wave = blockIdx.x * kWavesPerGroup + wv;
  const int nwaves = gridDim.x * kWavesPerGroup;
  zero_empty_rows(p, wave, nwaves, lane);
  const SliceInfo si = kFused ? plan_in_wave(p, wave, lane) : read_plan(p, wave);
  if (wave >= si.n) return;

  __shared__ typename F::Shared shared[kWavesPerGroup];
  typename F::Shared& sh = shared[wv];
  const size_t blk_stride = (size_t)p.hkv * kTileElems;

  // A slice holds at most two cut pairs: the one it starts in and the one it
  // ends in.
  struct Pending {
    int32_t b, g, first, tiles;
  } pend[2];
  int npend = 0;

  int32_t t = si.s0;
  int b = si.b, g = si.g, j = si.j;
  while (t < si.s1 && b < p.batch) {
    const int32_t L = clamp_len(p.lens[b], p.mbps);
    const int32_t nb = (L + kBlock - 1) / kBlock;
    if (nb == 0) {
      ++b;
      g = 0;
      j = 0;
      continue;
    }
    const int32_t jend = min(nb, j + (si.s1 - t));
    const int32_t pair_first = t - j;

    // Block ids of this row, 64 at a time, one per lane.
    const int32_t* trow = p.table + (size_t)b * p.mbps;
    int32_t tbase = j;
    int32_t tvals = (tbase + lane < jend) ? trow[tbase + lane] : 0;
    auto tile_off = [&](int32_t jj) -> size_t {
      if (jj - tbase >= kWave) {
        tbase += kWave;
        tvals = (tbase + lane < jend) ? trow[tbase + lane] : 0;
      }
      const int32_t id = __builtin_amdgcn_readlane(tvals, jj - tbase);
      return (size_t)min((uint32_t)id, (uint32_t)(p.num_blocks - 1)) * blk_stride +
             (size_t)g * kTileElems;
    };

    typename F::Q qr;
    F::load_q(qr, p.q + ((size_t)b * p.hq + g * G) * kHeadDim, lane);
    typename F::State st;
    F::init(st);

    typename F::Tile buf[PF + 1];
#pragma unroll
    for (int i = 0; i < PF; ++i)
      if (j + i < jend) {
        const size_t off = tile_off(j + i);
        F::load_tile(buf[i], p.k + off, p.v + off, lane);
      }
    for (int32_t jj = j; jj < jend; jj += PF + 1) {
#pragma unroll
      for (int u = 0; u <= PF; ++u) {
        const int32_t cur = jj + u;
        if (cur >= jend) break;
        const int32_t ld = cur + PF;
        if (ld < jend) {
          const size_t off = tile_off(ld);
          F::load_tile(buf[(u + PF) % (PF + 1)], p.k + off, p.v + off, lane);
        }
        F::step(st, buf[u], qr, L - cur * kBlock, p.scale_log2, lane, sh);
      }
    }

    if (j == 0 && jend == nb) {
      F::template write<false>(st, p.out + ((size_t)b * p.hq + g * G) * kHeadDim, nullptr, lane);
    } else {
      const int slot = partial_slot(wave, si.s0, pair_first);
      F::template write<true>(st, p.part_o + (size_t)slot * G * kHeadDim, p.part_lse + slot * G,
                              lane);
      if (kFused && arrive_last(p, pair_first, nb, si.T, si.n, lane)) {
        // Merge after the tile loop, when the tile buffers are no longer live.
        pend[npend].b = b;
        pend[npend].g = g;
        pend[npend].first = pair_first;
        pend[npend].tiles = nb;
        ++npend;
      }
    }

    t += jend - j;
    j = jend;
    if (j == nb) {
      j = 0;
      if (++g == p.hkv) {
        g = 0;
        ++b;
      }
    }
  }
  if (kFused) {
    for (int i = 0; i < npend; ++i) {
      const int32_t c0 = slice_of_tile(pend[i].first, si.T, si.n);
      const int32_t c1 = slice_of_tile(pend[i].first + pend[i].tiles - 1, si.T, si.n);
      merge_pair<G>(p, pend[i].b, pend[i].g, pend[i].first, c0, c1, si.T, si.n, lane);
    }
  }
}

}  // namespace neo
