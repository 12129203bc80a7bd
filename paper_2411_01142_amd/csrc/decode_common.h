// The decode driver shared by both kernel families: how a wavefront finds its
// slice of the batch, walks (request, kv head, block) tiles with loads issued
// ahead of use, and where a finished segment's result goes (straight to `out`,
// or to a partial slot that is merged afterwards).
//
// Work is balanced on a weighted line: each (request, kv head) pair with nb > 0
// blocks occupies nb + pair_cost(nb) positions, its startup cost (q, block
// ids, pipeline fill, result write) followed by one position per block tile.
// The W positions are cut into n contiguous slices (equal ones, or, for long
// slices on an eight-XCD part, weighted by the XCD each runs on: SliceGeom),
// and each slice processes the tiles whose positions fall in it. A pair
// whose tiles cross a slice boundary is "cut": every slice holding some of
// its tiles writes a partial output normalised over its share plus the
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

// ----------------------------------------------------------------- tile loads

// KV tiles are read through buffer resources covering one 4 KiB tile. A tile
// past the end of a segment gets a resource of size 0: its loads still issue
// (and count) but return zeros without touching memory. Issuing the same
// number of loads on every path keeps the compiler's wait counts exact: with
// loads skipped by a branch, it must assume the fewest loads in flight and
// waits for the whole prefetch at every step.
constexpr int kTileBytes = kTileElems * 2;
constexpr int kBufferWord3 = 0x00020000;  // gfx9 buffer resource, dword 3
constexpr int kNontemporal = 2;           // cache policy bit: streaming access

__device__ inline int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ inline __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* base, bool valid) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void* u = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(u, (short)0, uniform(valid) ? kTileBytes : 0,
                                           kBufferWord3);
}
__device__ inline u32x4_t tile_load16(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_bit_cast(u32x4_t,
                            __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kNontemporal));
}
__device__ inline s16x4_t tile_load8(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_bit_cast(s16x4_t,
                            __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, kNontemporal));
}

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
// Two adjacent floats (8-byte aligned) in one coherent store.
__device__ inline void store_coherent2(float* p, float a, float b) {
  const uint64_t bits = (uint64_t)__builtin_bit_cast(uint32_t, a) |
                        ((uint64_t)__builtin_bit_cast(uint32_t, b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), bits, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Two adjacent floats (8-byte aligned) in one coherent load.
__device__ inline float2 load_coherent2(const float* p) {
  const uint64_t bits = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
  float2 r;
  r.x = __builtin_bit_cast(float, (uint32_t)bits);
  r.y = __builtin_bit_cast(float, (uint32_t)(bits >> 32));
  return r;
}
__device__ inline void wait_all_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// ----------------------------------------------------------------- slice geometry

// Geometry of a wave-uniform slice index or position, kept in scalar
// registers (the fp32 estimate runs on the vector ALU).
__device__ inline int32_t slice_start_u(int32_t s, const SliceGeom& g) {
  return uniform(slice_start(s, g));
}
__device__ inline int32_t slice_of_u(int32_t x, const SliceGeom& g) {
  return uniform(slice_of(x, g));
}
// Partial slot of slice s for a pair whose first tile sits at position
// first_tile: 2s when that tile is at or before the slice start (the pair runs
// into the slice: its first segment), else 2s+1 (a pair starting inside the
// slice and cut by its end). A slice has at most one of each.
__device__ inline int partial_slot(int32_t s, int32_t slice_first, int32_t first_tile) {
  return first_tile <= slice_first ? 2 * s : 2 * s + 1;
}

// Number of slices for W positions. With min_tiles > 0: W / min_tiles, capped.
// With min_tiles == 0 (the default policy): `quantum` slices, one 4-wave
// workgroup per CU, so every CU gets the same share; batches too small for
// that get W / 2 slices. Measured: two workgroups per CU are never faster
// (2-3 % slower on long requests: more streams in flight lower the HBM
// efficiency), counts that give some CUs two workgroups and others one are
// 10-25 % slower, and a small batch (4 requests of 64-512 tokens) is fastest
// with the most slices up to one workgroup per CU (W / 8 slices: 13 % slower).
constexpr int32_t kSmallTilesPerSlice = 2;

__host__ __device__ inline int32_t slice_count(int32_t W, int32_t min_tiles, int32_t max_slices,
                                               int32_t quantum) {
  if (W <= 0) return 0;
  if (min_tiles > 0) return min(max(W / min_tiles, 1), max_slices);
  const int32_t n = W >= quantum * kSmallTilesPerSlice ? quantum : max(W / kSmallTilesPerSlice, 1);
  return min(n, max_slices);
}

struct SliceInfo {
  SliceGeom geo;     // total positions, slices
  int32_t s0, s1;    // this slice's position range
  int32_t b, g, x;   // pair holding position s0 and the offset of s0 inside it
  int32_t L;         // clamped length of request b, or -1 when the plan does not hold it
};

// ----------------------------------------------------------------- wave helpers

// The plan is the same in every lane; saying so lets the compiler keep the
// slice walk in scalar registers (tile addresses must be scalar for buffer
// resources).
__device__ inline float uniform_f32(float v) {
  return __builtin_bit_cast(float, uniform(__builtin_bit_cast(int32_t, v)));
}
__device__ inline SliceGeom make_uniform(SliceGeom g) {
  g.W = uniform(g.W);
  g.n = uniform(g.n);
  g.weighted = uniform(g.weighted);
  g.cn = uniform(g.cn);
  g.a = uniform(g.a);
  g.r = uniform(g.r);
  g.r_over_cn = uniform_f32(g.r_over_cn);
  g.n_over_w = uniform_f32(g.n_over_w);
  return g;
}
__device__ inline SliceInfo make_uniform(SliceInfo si) {
  si.geo = make_uniform(si.geo);
  si.s0 = uniform(si.s0);
  si.s1 = uniform(si.s1);
  si.b = uniform(si.b);
  si.g = uniform(si.g);
  si.x = uniform(si.x);
  si.L = uniform(si.L);
  return si;
}

// Cross-lane arithmetic through DPP (operand modifiers of ordinary vector
// instructions) rather than shuffles, each of which is a round trip through
// the LDS crossbar: a 64-lane scan is four shifts inside each 16-lane row and
// two broadcasts from one row to the next. Measured: the plan's chain of
// shuffle reductions and scans took ~1.3 us per wave at any batch size.
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142;  // lane 15 of each row to the next row
constexpr int kDppRowBcast31 = 0x143;  // lane 31 to rows 2 and 3

// v moved by the DPP pattern; lanes with no source (outside the row, or rows
// left out by kRowMask) get `identity`.
template <int kCtrl, int kRowMask = 0xF>
__device__ inline int32_t dpp_move(int32_t identity, int32_t v) {
  return __builtin_amdgcn_update_dpp(identity, v, kCtrl, kRowMask, 0xF, false);
}
// Inclusive scan over the 64 lanes with an associative op and its identity.
template <class Op>
__device__ inline int32_t wave_scan_bits(int32_t v, int32_t identity, Op op) {
  v = op(v, dpp_move<kDppRowShr1>(identity, v));
  v = op(v, dpp_move<kDppRowShr2>(identity, v));
  v = op(v, dpp_move<kDppRowShr4>(identity, v));
  v = op(v, dpp_move<kDppRowShr8>(identity, v));
  v = op(v, dpp_move<kDppRowBcast15, 0xA>(identity, v));
  v = op(v, dpp_move<kDppRowBcast31, 0xC>(identity, v));
  return v;
}
__device__ inline int32_t wave_incl_scan_i32(int32_t v) {
  return wave_scan_bits(v, 0, [](int32_t a, int32_t b) { return a + b; });
}
// Reductions: the scan's last lane, read into a scalar register.
__device__ inline int32_t wave_sum_i32(int32_t v) {
  return __builtin_amdgcn_readlane(wave_incl_scan_i32(v), kWave - 1);
}
__device__ inline float wave_max_f32(float v) {
  const int32_t s = wave_scan_bits(
      __builtin_bit_cast(int32_t, v), __builtin_bit_cast(int32_t, -INFINITY),
      [](int32_t a, int32_t b) {
        return __builtin_bit_cast(int32_t,
                                  fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b)));
      });
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(s, kWave - 1));
}
__device__ inline float wave_sum_f32(float v) {
  const int32_t s = wave_scan_bits(
      __builtin_bit_cast(int32_t, v), 0, [](int32_t a, int32_t b) {
        return __builtin_bit_cast(int32_t,
                                  __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b));
      });
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(s, kWave - 1));
}

// Lane l combined with lane l ^ 16 (resp. l ^ 32) through the gfx950 row swap
// instructions, no LDS round trip: with the same value in both operands, the
// first result holds lane (l & ~16)'s value and the second lane (l | 16)'s, so
// both partners get op(lower lane's value, upper lane's value), the same bits.
// The results are copied to scalars before the bit cast: a cast applied to a
// vector-element subscript directly has been lowered as a read of element 0.
template <class Op>
__device__ inline float combine_xor16(float v, Op op) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const uint32_t lo = r[0], hi = r[1];
  return op(__builtin_bit_cast(float, lo), __builtin_bit_cast(float, hi));
}
template <class Op>
__device__ inline float combine_xor32(float v, Op op) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const uint32_t lo = r[0], hi = r[1];
  return op(__builtin_bit_cast(float, lo), __builtin_bit_cast(float, hi));
}
// Max / sum over the four lanes l, l^16, l^32, l^48 (one column of the
// 16 x 16 MFMA accumulator layout, or one head's four lane groups).
__device__ inline float max_over_rows(float v) {
  const auto mx = [](float a, float b) { return fmaxf(a, b); };
  return combine_xor32(combine_xor16(v, mx), mx);
}
__device__ inline float sum_over_rows(float v) {
  const auto add = [](float a, float b) { return a + b; };
  return combine_xor32(combine_xor16(v, add), add);
}

// ----------------------------------------------------------------- planning

// Slice from the plan kernel's output (staged launch).
__device__ inline SliceInfo read_plan(const DecodeParams& p, int wave) {
  SliceInfo si;
  si.geo = make_slice_geom(p.hdr->total, p.hdr->n_slices, p.xcd8 != 0);
  if (wave >= si.geo.n) return si;
  const SliceStart a = p.starts[wave];
  si.s0 = a.pos;
  si.s1 = p.starts[wave + 1].pos;
  si.b = a.b;
  si.g = a.g;
  si.x = a.x;
  si.L = -1;
  return make_uniform(si);
}

// Slice computed by the wavefront itself from seq_lens (fused launch): a
// wave-wide reduction of the request weights gives W; a wave-wide scan locates
// the request holding the slice's first position. Requests are read 64 per
// lane group, up to kPlanRegs groups per load round.
constexpr int kPlanRegs = 16;

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt == 0 and leaves the
// export and LDS/scalar counters alone.
constexpr int kWaitVmcnt0 = 0x0F70;
// ... that waits for lgkmcnt == 0 (LDS and scalar memory) only.
constexpr int kWaitLgkmcnt0 = 0xC07F;

// Slices of at least this many positions on average merge within a workgroup
// through LDS (fused launch).
constexpr int32_t kGroupMergeMinTiles = 8;

// Tiles before the end of a segment at which the fast-merge counter is read.
constexpr int32_t kMergeCheckAhead = 3;

// Weights of requests base + 64r + lane, r < kPlanRegs (0 past the batch), and
// their raw lengths. Loads use a clamped index so that all of them issue before
// any is waited on.
__device__ inline void load_weights(const DecodeParams& p, int base, int lane,
                                    int32_t (&w)[kPlanRegs], int32_t (&raw)[kPlanRegs]) {
#pragma unroll
  for (int r = 0; r < kPlanRegs; ++r)
    raw[r] = base + r * kWave < p.batch ? p.lens[min(base + r * kWave + lane, p.batch - 1)] : 0;
#pragma unroll
  for (int r = 0; r < kPlanRegs; ++r)
    w[r] = (base + r * kWave + lane < p.batch) ? pair_weight(raw[r], p.mbps) : 0;
}

__device__ inline SliceInfo plan_in_wave(const DecodeParams& p, int wave, int lane) {
  SliceInfo si;
  constexpr int kChunk = kWave * kPlanRegs;
  int32_t w[kPlanRegs], raw[kPlanRegs];
  int32_t total = 0;
  for (int base = 0; base < p.batch; base += kChunk) {
    load_weights(p, base, lane, w, raw);
    int32_t s = 0;
#pragma unroll
    for (int r = 0; r < kPlanRegs; ++r) s += w[r];
    total += wave_sum_i32(s);
  }
  const int32_t W = uniform(total * p.hkv);
  si.geo = make_uniform(
      make_slice_geom(W, slice_count(W, p.min_tiles, p.max_slices, p.slice_quantum), p.xcd8 != 0));
  if (wave >= si.geo.n) return si;
  si.s0 = slice_start_u(wave, si.geo);
  si.s1 = slice_start_u(wave + 1, si.geo);

  // Request b holds positions [hkv*P_b, hkv*P_{b+1}) with P the weight prefix
  // sum: the first b with hkv * P_{b+1} > s0 (no division by hkv).
  const int32_t s0 = si.s0;
  int32_t carry = 0;
  int32_t found_b = -1, found_p = 0, found_w = 1, found_len = 0;
  for (int base = 0; base < p.batch && found_b < 0; base += kChunk) {
    if (p.batch > kChunk) load_weights(p, base, lane, w, raw);
    // The register (64 requests) holding position s0, then the lane. In a
    // round of at most 64 requests the first register is it (every earlier
    // round was passed by its total); otherwise every register's sum is
    // reduced at once (the independent reductions pipeline).
    int32_t wr = w[0], rawr = raw[0], rr = 0;
    if (p.batch - base > kWave) {
      int32_t cs[kPlanRegs];
#pragma unroll
      for (int r = 0; r < kPlanRegs; ++r) cs[r] = w[r];
#pragma unroll
      for (int r = 0; r < kPlanRegs; ++r) cs[r] = wave_sum_i32(cs[r]);
      rr = -1;
#pragma unroll
      for (int r = 0; r < kPlanRegs; ++r) {
        const int32_t c = uniform(cs[r]);
        if (rr < 0) {
          if (p.hkv * (carry + c) > s0) rr = r; else carry += c;
        }
      }
      if (rr < 0) continue;  // past this round: carry holds its total
#pragma unroll
      for (int r = 0; r < kPlanRegs; ++r)
        if (r == rr) {
          wr = w[r];
          rawr = raw[r];
        }
    }
    const int32_t incl = wave_incl_scan_i32(wr);
    const uint64_t hit = __ballot(p.hkv * (carry + incl) > s0);
    const int first = __ffsll((unsigned long long)hit) - 1;
    found_b = base + rr * kWave + first;
    found_p = carry + __builtin_amdgcn_readlane(incl - wr, first);
    found_w = __builtin_amdgcn_readlane(wr, first);
    found_len = __builtin_amdgcn_readlane(rawr, first);
  }
  // The request's weight and length come from the registers already loaded:
  // no second round trip to seq_lens before the first table row.
  const int32_t rem = si.s0 - p.hkv * found_p;
  si.b = found_b;
  si.g = rem / found_w;
  si.x = rem % found_w;
  si.L = clamp_len(found_len, p.mbps);
  return make_uniform(si);
}

// ----------------------------------------------------------------- outputs

// Requests with no tokens get a zero row; every wavefront takes a strided share.
// len0: seq_lens[wave] (any value when wave >= batch), loaded by the caller
// before the plan so that its round trip overlaps the plan's.
__device__ inline void zero_empty_rows(const DecodeParams& p, int wave, int nwaves, int lane,
                                       int32_t len0) {
  for (int b = wave; b < p.batch; b += nwaves) {
    if (clamp_len(b == wave ? len0 : p.lens[b], p.mbps) != 0) continue;
    f32x4_t* row = reinterpret_cast<f32x4_t*>(p.out + (size_t)b * p.hq * kHeadDim);
    const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
    for (int i = lane; i < p.hq * (kHeadDim / 4); i += kWave) row[i] = z;
  }
}

// out rows of pair (b, g) from two contributors' log-sum-exps and rows (this
// lane's two dims): the two-contributor case of merge_pair, operation for
// operation.
template <int G, int GH = G>
__device__ inline void merge_two_values(const DecodeParams& p, int32_t b, int32_t g,
                                        const float* la, const float* lb, const float2* oa,
                                        const float2* ob, int lane, int h0 = 0) {
  const int d = 2 * lane;
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    const float m = fmaxf(la[h], lb[h]);
    const float wa = __expf(la[h] - m), wb = __expf(lb[h] - m);
    const float inv = 1.f / (wa + wb);
    float2 r;
    r.x = fmaf(wb, ob[h].x, wa * oa[h].x) * inv;
    r.y = fmaf(wb, ob[h].y, wa * oa[h].y) * inv;
    *reinterpret_cast<float2*>(p.out + ((size_t)b * p.hq + g * G + h0 + h) * kHeadDim + d) = r;
  }
}

// Merge the partials of one cut pair into out[b][g*G .. g*G+G): with M the
// largest log-sum-exp, out = sum_c e^(lse_c - M) o_c / sum_c e^(lse_c - M).
// Contributors are slices c0..c1, taken 64 at a time with a running maximum
// (earlier sums are rescaled when it grows). Lane i reads the log-sum-exps of
// contributor i of the chunk; each lane owns dims 2*lane, 2*lane+1 of the
// sums; partial rows are read kBatch contributors at a time, the first batch
// issued together with the log-sum-exps. Partial slot q lives at
// part_o[(q - slot0) * G * 128], part_lse[(q - slot0) * G] (the workspace, or a
// workgroup's shared copy). kCoherent: the partials were written by other
// wavefronts of the running kernel to the workspace. kMaxBatch caps the rows
// read per round (LDS reads need no batching; the sums are the same either way).
template <int G, int GH, bool kCoherent, int kMaxBatch>
__device__ inline void merge_pair_heads(const DecodeParams& p, const float* part_o,
                                        const float* part_lse, int32_t slot0, int32_t b,
                                        int32_t g, int h0, int32_t first_tile, int32_t c0,
                                        int32_t c1, const SliceGeom& geo, int lane) {
  constexpr int kFit = 32 / GH > 0 ? 32 / GH : 1;  // 64 registers of rows
  constexpr int kBatch = kFit < kMaxBatch ? kFit : kMaxBatch;
  auto ld = [](const float* a) -> float { return kCoherent ? load_coherent(a) : *a; };
  auto ld2 = [](const float* a) -> float2 {
    return kCoherent ? load_coherent2(a) : *reinterpret_cast<const float2*>(a);
  };
  const int k = c1 - c0 + 1;
  const int d = 2 * lane;
  float m[GH], z[GH], a0[GH], a1[GH];
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    m[h] = -INFINITY;
    z[h] = a0[h] = a1[h] = 0.f;
  }
  for (int base = 0; base < k; base += kWave) {
    const int cnt = min(kWave, k - base);
    float ov[kBatch][GH][2];
    auto load_rows = [&](int i0, bool clamp) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (!clamp && i0 + u >= cnt) break;  // uniform
        const int c = c0 + base + min(i0 + u, cnt - 1);
        const int slot = partial_slot(c, slice_start_u(c, geo), first_tile) - slot0;
#pragma unroll
        for (int h = 0; h < GH; ++h) {
          const float2 v = ld2(part_o + ((size_t)slot * G + h0 + h) * kHeadDim + d);
          ov[u][h][0] = v.x;
          ov[u][h][1] = v.y;
        }
      }
    };
    load_rows(0, true);
    const int mine = c0 + base + (lane < cnt ? lane : 0);
    const int my_slot = partial_slot(mine, slice_start(mine, geo), first_tile) - slot0;
    // Every head's log-sum-exp is loaded before any cross-lane step, so the
    // loads share one round trip.
    float lse_h[GH];
#pragma unroll
    for (int h = 0; h < GH; ++h) lse_h[h] = ld(part_lse + my_slot * G + h0 + h);
    float w[GH];
#pragma unroll
    for (int h = 0; h < GH; ++h) {
      const float lse = lane < cnt ? lse_h[h] : -INFINITY;
      const float mc = fmaxf(m[h], wave_max_f32(lse));
      const float rescale = __expf(m[h] - mc);  // 0 on the first chunk
      a0[h] *= rescale;
      a1[h] *= rescale;
      z[h] *= rescale;
      m[h] = mc;
      w[h] = __expf(lse - mc);
      z[h] += wave_sum_f32(w[h]);
    }
    for (int i0 = 0; i0 < cnt; i0 += kBatch) {
      if (i0 > 0) load_rows(i0, false);
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (i0 + u >= cnt) break;
#pragma unroll
        for (int h = 0; h < GH; ++h) {
          const float wi = __builtin_bit_cast(
              float, __builtin_amdgcn_readlane(__builtin_bit_cast(int32_t, w[h]), i0 + u));
          a0[h] = fmaf(wi, ov[u][h][0], a0[h]);
          a1[h] = fmaf(wi, ov[u][h][1], a1[h]);
        }
      }
    }
  }
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    const float inv = 1.f / z[h];
    float2 r;
    r.x = a0[h] * inv;
    r.y = a1[h] * inv;
    *reinterpret_cast<float2*>(p.out + ((size_t)b * p.hq + g * G + h0 + h) * kHeadDim + d) = r;
  }
}

// All heads of the pair, GH of them per pass (fewer live registers).
template <int G, bool kCoherent, int kMaxBatch = 16, int GH = G>
__device__ inline void merge_pair(const DecodeParams& p, const float* part_o,
                                  const float* part_lse, int32_t slot0, int32_t b, int32_t g,
                                  int32_t first_tile, int32_t c0, int32_t c1,
                                  const SliceGeom& geo, int lane) {
  static_assert(G % GH == 0, "head passes must tile the group");
  for (int h0 = 0; h0 < G; h0 += GH)
    merge_pair_heads<G, GH, kCoherent, kMaxBatch>(p, part_o, part_lse, slot0, b, g, h0,
                                                  first_tile, c0, c1, geo, lane);
}

// The merge of a pair with exactly two contributors, partial slots sa (the
// earlier slice) and sb of part_o / part_lse, with every load in one round
// trip. Same arithmetic, in the same order, as merge_pair for two
// contributors, so both give the same bits.
template <int G, bool kCoherent, int GH = G>
__device__ inline void merge_two(const DecodeParams& p, const float* part_o,
                                 const float* part_lse, int32_t b, int32_t g, int32_t sa,
                                 int32_t sb, int lane) {
  static_assert(G % GH == 0, "head passes must tile the group");
  const int d = 2 * lane;
  for (int h0 = 0; h0 < G; h0 += GH) {
    float la[GH], lb[GH];
    float2 oa[GH], ob[GH];
#pragma unroll
    for (int h = 0; h < GH; ++h) {
      const float* pa = part_o + ((size_t)sa * G + h0 + h) * kHeadDim + d;
      const float* pb = part_o + ((size_t)sb * G + h0 + h) * kHeadDim + d;
      if (kCoherent) {
        la[h] = load_coherent(part_lse + sa * G + h0 + h);
        lb[h] = load_coherent(part_lse + sb * G + h0 + h);
        oa[h] = load_coherent2(pa);
        ob[h] = load_coherent2(pb);
      } else {
        la[h] = part_lse[sa * G + h0 + h];
        lb[h] = part_lse[sb * G + h0 + h];
        oa[h] = *reinterpret_cast<const float2*>(pa);
        ob[h] = *reinterpret_cast<const float2*>(pb);
      }
    }
    merge_two_values<G, GH>(p, b, g, la, lb, oa, ob, lane, h0);
  }
}

// Fused launch: after writing its partial for a cut pair, a slice counts itself
// in the pair's counter; the slice that completes the count merges the pair
// (returns true) and resets the counter to zero for the next call.
__device__ inline bool arrive_last(const DecodeParams& p, int32_t c0, int32_t c1, int lane) {
  wait_all_memory();  // this slice's partial has reached the coherence point
  int32_t old = 0;
  if (lane == 0)
    old = __hip_atomic_fetch_add(p.counters + c0, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  old = __builtin_amdgcn_readlane(old, 0);
  if (old != c1 - c0) return false;
  if (lane == 0)
    __hip_atomic_store(p.counters + c0, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

// ----------------------------------------------------------------- the driver

// Cut pairs whose contributors are all slices of one workgroup (the four
// waves hold consecutive slices) are merged through LDS: partials, a counter
// per pair (indexed by its first slice), and the last arrival merges. No
// device-coherent store has to complete and no atomic crosses the chip, which
// under load takes several microseconds per cut segment. Pairs that cross a
// workgroup boundary use the workspace.
template <int G>
struct GroupMerge {
  static constexpr int kHeadsPerPass = G < 4 ? G : 4;  // merges from LDS: 4 heads at a time
  float o[2 * kWavesPerGroup][G * kHeadDim];  // partial slot 2s / 2s+1 of slice s, local
  float lse[2 * kWavesPerGroup][G];
  int32_t count[kWavesPerGroup];
};
// Launches that merge in a separate kernel keep no shared merge state.
template <int G, bool kOn>
struct GroupMergeOf {
  using type = GroupMerge<G>;
};
template <int G>
struct GroupMergeOf<G, false> {
  struct type {
    int32_t count[1];
  };
};

// Family provides: Tile, State, Q, Shared; load_q, init, load_tile, step, write.
// PF tiles are in flight ahead of the one being computed.
template <class F, int G, int PF, Schedule kSched>
__device__ inline void decode_driver(const DecodeParams& p) {
  constexpr bool kMergeHere = kSched == kFused;  // merge cut pairs in this kernel
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x >> 6;
  const int wave = blockIdx.x * kWavesPerGroup + wv;
  const int nwaves = gridDim.x * kWavesPerGroup;
  const int32_t len0 = wave < p.batch ? p.lens[wave] : 0;
  // Slices of this workgroup: first_slice .. first_slice + kWavesPerGroup - 1.
  const int32_t first_slice = blockIdx.x * kWavesPerGroup;
  __shared__ typename GroupMergeOf<G, kMergeHere>::type gm;
  const SliceInfo si = kSched == kStaged ? read_plan(p, wave) : plan_in_wave(p, wave, lane);
  zero_empty_rows(p, wave, nwaves, lane, len0);
  // Merges through LDS pay when slices are long enough to hold cut segments
  // of several tiles; for tiny slices the barrier that clears the counters
  // costs more than it saves. The plan is the same in every wave of the block,
  // so all of them take (or skip) the barrier, before any returns.
  const bool group_merge =
      kMergeHere && si.geo.n > 0 && si.geo.W >= kGroupMergeMinTiles * si.geo.n;
  if constexpr (kMergeHere) {
    if (group_merge) {
      if (threadIdx.x < kWavesPerGroup) gm.count[threadIdx.x] = 0;
      __syncthreads();
    }
  }
  if (kSched == kTwoKernel && lane == 0) {
    // Record the plan for the combine kernel.
    if (wave < si.geo.n) {
      SliceStart a;
      a.pos = si.s0;
      a.b = si.b;
      a.g = si.g;
      a.x = si.x;
      a.nb = blocks_of(p.lens[si.b], p.mbps);
      a.pad[0] = a.pad[1] = a.pad[2] = 0;
      p.starts[wave] = a;
    }
    if (wave == 0) {
      SliceStart e;
      e.pos = si.geo.W;
      e.b = p.batch;
      e.g = e.x = e.nb = 0;
      e.pad[0] = e.pad[1] = e.pad[2] = 0;
      p.starts[si.geo.n] = e;
      PlanHeader h;
      h.total = si.geo.W;
      h.n_slices = si.geo.n;
      h.batch = p.batch;
      h.pad = 0;
      *p.hdr = h;
    }
  }
  if (wave >= si.geo.n) return;

  __shared__ typename F::Shared shared[kWavesPerGroup];
  typename F::Shared& sh = shared[wv];
  const size_t blk_stride = (size_t)p.blk_stride;

  // A slice holds at most two cut pairs: the one it starts in and the one it
  // ends in. Their merges (fused launch) run after the tile loop. Two named
  // records, not an array: a dynamically indexed array would be placed in LDS
  // (measured: that allocation alone slows the whole kernel by ~15 %).
  struct Pending {
    int32_t b, g, first, c0, c1;
  } pend0{}, pend1{};
  int npend = 0;

  int32_t pos = si.s0;  // weighted position reached
  int b = si.b, g = si.g;
  int32_t x = si.x;     // offset of pos inside pair (b, g)
  // Known ahead of use: the length of request pf_b (from the plan for the
  // first pair, prefetched for later ones) and the first 64 block ids of
  // request pf_tb (prefetched while the previous pair streams), so that a new
  // pair's q and first tiles go out without dependent round trips.
  int32_t pf_b = si.L >= 0 ? si.b : -1, pf_L = si.L, pf_tb = -1, pf_vals = 0;
  while (b < p.batch) {
    const int32_t L = pf_b == b ? pf_L : clamp_len(p.lens[b], p.mbps);
    const int32_t nb = (L + kBlock - 1) / kBlock;
    if (nb == 0) {
      ++b;
      g = 0;
      x = 0;
      continue;
    }
    const int32_t pair_base = pos - x;
    const int32_t cost = pair_cost(nb);
    const int32_t first_tile = pair_base + cost;  // position of block 0
    const int32_t j = max(0, x - cost);
    const int32_t jend = min(nb, si.s1 - first_tile);
    if (jend <= j) break;  // the slice ends before this pair's next tile

    // Block ids of this row, 64 at a time, one per lane.
    const int32_t* trow = p.table + (size_t)b * p.mbps;
    int32_t tbase = j;
    int32_t tvals = (j == 0 && pf_tb == b) ? pf_vals : ((tbase + lane < jend) ? trow[tbase + lane] : 0);
    // The next pair is (b, g+1) or (b+1, 0); the next request's length is
    // requested now and used after this pair's first tile loads are out.
    const int32_t nq = g + 1 < p.hkv ? b : b + 1;
    const int32_t lq_raw = (nq != b && nq < p.batch) ? p.lens[nq] : 0;
    auto tile_off = [&](int32_t jj) -> size_t {
      if (jj - tbase >= kWave) {
        tbase += kWave;
        tvals = (tbase + lane < jend) ? trow[tbase + lane] : 0;
        // Wait for the new ids here, on the refresh path only. Without this
        // explicit wait the compiler puts a full vmcnt(0) after the branch
        // joins, on every tile, and that drains the tile prefetch each step.
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
      }
      const int32_t id = __builtin_amdgcn_readlane(tvals, jj - tbase);
      return (size_t)min((uint32_t)id, (uint32_t)(p.num_blocks - 1)) * blk_stride +
             (size_t)g * kTileElems;
    };

    typename F::Q qr;
    F::load_q(qr, p.q + ((size_t)b * p.hq + g * G) * kHeadDim, lane);
    typename F::State st;
    F::init(st);

    // Every step issues one tile's loads; tiles past jend are empty (their
    // index is clamped to a real tile, their resource has size 0).
    typename F::Tile buf[PF + 1];
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const size_t off = tile_off(min(j + i, jend - 1));
      F::load_tile(buf[i], p.k + off, p.v + off, j + i < jend, lane);
    }

    // Prefetch for the next pair (in bounds: lanes below its block count,
    // which is at most the table's row length).
    if (nq < p.batch) {
      const int32_t Lq = nq == b ? L : clamp_len(lq_raw, p.mbps);
      const int32_t nbq = (Lq + kBlock - 1) / kBlock;
      const int32_t* tq = p.table + (size_t)nq * p.mbps;
      pf_vals = lane < min(nbq, kWave) ? tq[lane] : 0;
      pf_b = pf_tb = nq;
      pf_L = Lq;
    }

    // The slices holding the pair's first and last tiles, if the pair is cut
    // (computed here, where their latency hides behind the first tile's
    // round trip; after the tiles it delayed every cut segment's result).
    const bool cut = j > 0 || jend < nb;
    const int32_t c0 = cut ? slice_of_u(first_tile, si.geo) : 0;
    const int32_t c1 = cut ? slice_of_u(first_tile + nb - 1, si.geo) : 0;

    // Fused launch, last pair of this slice cut with exactly one later slice
    // (the next one), which handles its share of the pair first: if it has
    // already arrived, this slice will be the last, so it merges straight
    // from registers after its tiles (no partial of its own, no atomic, one
    // round trip for the other partial). The counter is read a few tiles
    // before the segment ends (late enough that the next slice has usually
    // finished its share, early enough that the read's latency hides behind
    // the remaining tiles) and only looked at after the tiles.
    bool fast_cand = false;
    if constexpr (kMergeHere && F::kFastMerge)
      fast_cand = j == 0 && jend < nb &&
                  (!group_merge || wave + 1 == first_slice + kWavesPerGroup) && c1 == wave + 1;
    const int32_t check_at = fast_cand ? max(j, jend - kMergeCheckAhead) : -1;
    int32_t seen = 0;
    for (int32_t jj = j; jj < jend; jj += PF + 1) {
#pragma unroll
      for (int u = 0; u <= PF; ++u) {
        const int32_t cur = jj + u;
        if (cur >= jend) break;
        const int32_t ld = cur + PF;
        {
          const size_t off = tile_off(min(ld, jend - 1));
          F::load_tile(buf[(u + PF) % (PF + 1)], p.k + off, p.v + off, ld < jend, lane);
        }
        if (cur == check_at)
          seen = __hip_atomic_load(p.counters + wave, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        F::step(st, buf[u], qr, L - cur * kBlock, p.scale_log2, lane, sh);
      }
    }
    const bool merge_now = fast_cand && __builtin_amdgcn_readfirstlane(seen) == 1;

    if (j == 0 && jend == nb) {
      F::template write<false>(st, p.out + ((size_t)b * p.hq + g * G) * kHeadDim, nullptr, lane);
    } else if (merge_now) {
      if constexpr (kMergeHere && F::kFastMerge) {
        if (lane == 0)
          __hip_atomic_store(p.counters + wave, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int32_t nxt = wave + 1;
        const int slot = partial_slot(nxt, slice_start_u(nxt, si.geo), first_tile);
        F::merge_write(st, p.part_o + (size_t)slot * G * kHeadDim, p.part_lse + slot * G,
                       p.out + ((size_t)b * p.hq + g * G) * kHeadDim, lane);
      }
    } else if (group_merge && c0 >= first_slice && c1 < first_slice + kWavesPerGroup) {
      if constexpr (kMergeHere) {
        // Every contributor is a wave of this workgroup: merge through LDS.
        const int32_t slot0 = 2 * first_slice;
        constexpr int kLdsMergeHeads = GroupMerge<G>::kHeadsPerPass;
        const int ls = partial_slot(wave, si.s0, first_tile) - slot0;
        F::template write<false>(st, gm.o[ls], gm.lse[ls], lane);
        // LDS operations of a wave complete in order: once this wave's
        // partial writes are done (lgkmcnt 0), its count follows them, and a
        // wave that reads the count after it sees the partial. Waiting on LDS
        // only: an acquire-release atomic would also wait for every vector
        // memory operation in flight (vmcnt 0), including the empty tile load
        // queued behind other waves' loads, which costs up to a round trip.
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);
        int32_t old = 0;
        if (lane == 0)
          old = __hip_atomic_fetch_add(&gm.count[c0 - first_slice], 1, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_WORKGROUP);
        old = __builtin_amdgcn_readlane(old, 0);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (old == c1 - c0) {
          if (c1 == c0 + 1) {
            merge_two<G, false, kLdsMergeHeads>(p, &gm.o[0][0], &gm.lse[0][0], b, g,
                                partial_slot(c0, slice_start_u(c0, si.geo), first_tile) - slot0,
                                partial_slot(c1, slice_start_u(c1, si.geo), first_tile) - slot0,
                                lane);
          } else {
            merge_pair<G, false, 1, kLdsMergeHeads>(p, &gm.o[0][0], &gm.lse[0][0], slot0, b, g,
                                                    first_tile, c0, c1, si.geo, lane);
          }
        }
      }
    } else {
      const int slot = partial_slot(wave, si.s0, first_tile);
      F::template write<kMergeHere>(st, p.part_o + (size_t)slot * G * kHeadDim,
                                p.part_lse + slot * G, lane);
      if (kMergeHere) {
        if (arrive_last(p, c0, c1, lane)) {
          const Pending rec{b, g, first_tile, c0, c1};
          if (npend == 0) pend0 = rec; else pend1 = rec;
          ++npend;
        }
      }
    }

    pos = pair_base + nb + cost;
    x = 0;
    if (pos >= si.s1) break;
    if (++g == p.hkv) {
      g = 0;
      ++b;
    }
  }
  if (kMergeHere) {
    for (int i = 0; i < npend; ++i) {
      const Pending q = i == 0 ? pend0 : pend1;
      if (q.c1 == q.c0 + 1) {
        merge_two<G, true>(p, p.part_o, p.part_lse, q.b, q.g,
                           partial_slot(q.c0, slice_start_u(q.c0, si.geo), q.first),
                           partial_slot(q.c1, slice_start_u(q.c1, si.geo), q.first), lane);
      } else {
        merge_pair<G, true>(p, p.part_o, p.part_lse, 0, q.b, q.g, q.first, q.c0, q.c1, si.geo,
                            lane);
      }
    }
  }
}

}  // namespace neo
