// Internal definitions shared by the libneoattn translation units: the fixed
// tile geometry, the device workspace layout and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "libneoattn.h"

namespace neo {

constexpr int kHeadDim = 128;                   // dims per head
constexpr int kBlock = 16;                      // tokens per KV block
constexpr int kPiece = 8;                       // dims per 16-byte key piece
constexpr int kTileElems = kHeadDim * kBlock;   // bf16 elements per (block, kv head) tile
constexpr int kWave = 64;
constexpr int kWavesPerGroup = 4;               // wavefronts per workgroup (256 threads)
constexpr int kPlanThreads = 1024;

// Work plan. Each (request, kv head) pair with nb > 0 blocks occupies
// nb + pair_cost(nb) positions of a weighted line (its startup cost, then one
// position per block tile), pairs in request-major, kv-head-next order; slice
// s owns positions [starts[s].pos, starts[s+1].pos) and is run by one
// wavefront. The startup cost is what a wave loses between two pairs, in
// tiles: about two for a short pair (its rows are written, the next pair's
// first tile is a round trip away), three for a pair long enough to be cut
// between slices (a partial is written and counted; the merge follows).
// Measured: one cost for every pair gives 2 as the best compromise (1 is
// 2.7 points slower on a mix of short requests, 3 is 0.8 points faster on
// long requests but 0.6 slower on the short mix). On a mix of 1016 short
// requests, the waves holding them ended ~10 us before those streaming the
// long ones: a short pair's startup measured ~1.7 tiles. A cost of 1 for the
// shortest pairs (fewer than 4 blocks) brings the mix's average close to
// that: +0.2 points there (2 for pairs below 3 blocks: -0.2; below 6: +0.1).
constexpr int32_t kPairCost = 2;
constexpr int32_t kPairCostShort = 1;
constexpr int32_t kPairCostLong = 3;
constexpr int32_t kShortPairBlocks = 4;
constexpr int32_t kLongPairBlocks = 32;
__host__ __device__ inline int32_t pair_cost(int32_t nb) {
  return nb >= kLongPairBlocks ? kPairCostLong
                               : (nb >= kShortPairBlocks ? kPairCost : kPairCostShort);
}

// Slice geometry of the weighted line: W positions cut into n slices. Slice s
// owns [floor(C(s) W / C(n)), floor(C(s+1) W / C(n))), C(s) being the units of
// the slices before s: one per slice, or, on a part with eight XCDs and slices
// of at least kXcdWeightMinTiles positions, kXcdEvenUnits for a slice on an
// even-numbered XCD and kXcdOddUnits for one on an odd-numbered XCD.
// Workgroups are dispatched round-robin over the XCDs in index order (the
// hardware XCC id read back was workgroup index mod 8 in every run), and
// workgroup w holds slices 4w .. 4w+3, so slice s runs on XCD (s / 4) mod 8.
// Measured on MI355X: waves on the odd-numbered XCDs stream 8-15 % slower per
// tile, so with equal slices they end last. With K and V of a block in one
// run, 34 : 30 units gain 1.3 % on a 256-request lognormal mix, 1.8 % on a 70B
// layer, 1.0 % at batch 64 (~42 positions per slice) and 2.9 % on a 70B
// layer's tensor-parallel share (~70); 33 : 31 and 35 : 29 measured between
// equal slices and 34 : 30 or level with it. Slices below 16 positions are
// dominated by their fixed costs and stay equal.
//
// Evaluated without 64-bit division, which the GPU has no instruction for
// (the software sequence would run at every pair transition and merge): with
// W = a C(n) + r, floor(C(s) W / C(n)) = C(s) a + floor(C(s) r / C(n)); the
// fp32 estimate of the last term is within one of it (it is below 2^17) and
// one exact integer step corrects it.
constexpr int32_t kXcdEvenUnits = 34;
constexpr int32_t kXcdOddUnits = 30;
constexpr int32_t kXcdWeightMinTiles = 16;
constexpr int32_t kXcdPeriodUnits = 4 * (kXcdEvenUnits + kXcdOddUnits);  // 8 slices
struct SliceGeom {
  int32_t W, n;      // positions and slices, 0 < n <= min(W, NEO_MAX_SLICES) (n = 0: no slices)
  int32_t weighted;  // 1: slices weighed by XCD
  int32_t cn;        // C(n)
  int32_t a, r;      // W = a C(n) + r
  float r_over_cn;   // r / C(n)
  float n_over_w;    // n / W
};
static_assert((int64_t)(NEO_MAX_SLICES / 8) * kXcdPeriodUnits < ((int64_t)1 << 24),
              "C(s) must be exact in fp32");

// xcd8: the device has eight XCDs.
__host__ __device__ inline SliceGeom make_slice_geom(int32_t W, int32_t n, bool xcd8) {
  SliceGeom g;
  g.W = W;
  g.n = n;
  g.weighted = xcd8 && n > 0 && n % 8 == 0 && W / kXcdWeightMinTiles >= n;
  g.cn = g.weighted ? (n / 8) * kXcdPeriodUnits : n;
  g.a = g.cn > 0 ? W / g.cn : 0;
  g.r = W - g.a * g.cn;
  g.r_over_cn = g.cn > 0 ? (float)g.r / (float)g.cn : 0.f;
  g.n_over_w = W > 0 ? (float)n / (float)W : 0.f;
  return g;
}
// C(s), for 0 <= s <= n.
__host__ __device__ inline int32_t slice_units(int32_t s, const SliceGeom& g) {
  if (!g.weighted) return s;
  const int32_t k = s & 7;
  return (s >> 3) * kXcdPeriodUnits +
         (k < 4 ? k * kXcdEvenUnits : 4 * kXcdEvenUnits + (k - 4) * kXcdOddUnits);
}
// First position of slice s, for 0 <= s <= n.
__host__ __device__ inline int32_t slice_start(int32_t s, const SliceGeom& g) {
  const int32_t c = slice_units(s, g);
  int32_t q = (int32_t)((float)c * g.r_over_cn);
  const int64_t t = (int64_t)c * g.r - (int64_t)q * g.cn;
  q += t < 0 ? -1 : (t >= g.cn ? 1 : 0);
  return c * g.a + q;
}
// The slice holding position x, 0 <= x < W: the largest s with
// slice_start(s) <= x. For equal slices that is ceil((x+1) n / W) - 1, and the
// fp32 estimate of (x+1) n / W is within 2^-10 of it; XCD weights move a
// boundary by at most 4 (34 - 30) / 64 = 0.25 slices. Either way the estimate's
// floor is off by at most one.
// Branch-free (both neighbours' starts are computed): the kernels call it
// with wave-uniform x, but in vector registers, where a branch costs masking.
__host__ __device__ inline int32_t slice_of(int32_t x, const SliceGeom& g) {
  int32_t s = (int32_t)(((float)x + 1.f) * g.n_over_w);
  s = s < g.n - 1 ? s : g.n - 1;
  const bool down = slice_start(s, g) > x;
  const bool up = s + 1 < g.n && slice_start(s + 1, g) <= x;
  return down ? s - 1 : (up ? s + 1 : s);
}

struct alignas(16) PlanHeader {
  int32_t total;     // positions on the weighted line
  int32_t n_slices;
  int32_t batch;
  int32_t pad;
};

struct alignas(32) SliceStart {
  int32_t pos;  // first position of the slice
  int32_t b;    // request of the pair holding it
  int32_t g;    // kv head of that pair
  int32_t x;    // offset of pos inside the pair's nb + pair_cost(nb) positions
  int32_t nb;   // blocks of that pair
  int32_t pad[3];
};

// Launch schedules: plan kernel + decode + combine kernel; one fused kernel;
// decode (planning in-wave, recording slice starts) + combine kernel.
enum Schedule { kStaged = 0, kFused = 1, kTwoKernel = 2 };

struct WorkspaceLayout {
  size_t hdr, starts, counters, prefix, part_lse, part_o, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Partial outputs: two slots per slice (a slice cuts at most the pair it starts
// in and the pair it ends in), each slot `group` rows of head_dim floats plus
// `group` log-sum-exps (natural log).
inline WorkspaceLayout workspace_layout(int32_t batch, int32_t group) {
  WorkspaceLayout w;
  size_t off = 0;
  w.hdr = off;
  off = align256(off + sizeof(PlanHeader));
  w.starts = off;
  off = align256(off + sizeof(SliceStart) * (NEO_MAX_SLICES + 1));
  w.counters = off;  // arrival counts of cut pairs (fused launch); zero between calls
  off = align256(off + sizeof(int32_t) * NEO_MAX_SLICES);
  w.prefix = off;
  off = align256(off + sizeof(int32_t) * ((size_t)batch + 1));
  w.part_lse = off;
  off = align256(off + sizeof(float) * 2 * NEO_MAX_SLICES * (size_t)group);
  w.part_o = off;
  off = align256(off + sizeof(float) * 2 * NEO_MAX_SLICES * (size_t)group * kHeadDim);
  w.total = off;
  return w;
}

// Number of KV blocks of a request, with its length clamped to the table.
__host__ __device__ inline int32_t clamp_len(int32_t L, int32_t mbps) {
  int32_t cap = mbps * kBlock;
  return L < 0 ? 0 : (L > cap ? cap : L);
}
__host__ __device__ inline int32_t blocks_of(int32_t L, int32_t mbps) {
  return (clamp_len(L, mbps) + kBlock - 1) / kBlock;
}
// Positions of each (request, kv head) pair of a request with this length.
__host__ __device__ inline int32_t pair_weight(int32_t L, int32_t mbps) {
  const int32_t nb = blocks_of(L, mbps);
  return nb > 0 ? nb + pair_cost(nb) : 0;
}

struct DecodeParams {
  const uint16_t* q;          // [batch][hq][128] bf16
  const uint16_t* k;          // [nb][hkv][16][16][8] bf16
  const uint16_t* v;          // [nb][hkv][128][16] bf16
  const int32_t* table;       // [batch][mbps]
  const int32_t* lens;        // [batch]
  float* out;                 // [batch][hq][128]
  PlanHeader* hdr;
  SliceStart* starts;
  float* part_lse;            // [2*NEO_MAX_SLICES][group]
  float* part_o;              // [2*NEO_MAX_SLICES][group][128]
  int32_t* counters;          // [NEO_MAX_SLICES]
  int32_t batch, hq, hkv, mbps, num_blocks;
  int32_t max_slices, min_tiles;  // min_tiles == 0: the default slice policy
  int32_t slice_quantum;          // compute units x wavefronts per workgroup
  int32_t xcd8;                   // the device has eight XCDs (slice weights)
  float scale_log2;           // scale * log2(e)
  int64_t blk_stride;         // elements from one block of a cache to the next (K and V alike)
};

// Launchers (each returns the hipError_t of its launch).
hipError_t launch_plan(const int32_t* lens, int32_t batch, int32_t hkv, int32_t mbps,
                       int32_t max_slices, int32_t min_tiles, int32_t quantum, int32_t xcd8,
                       PlanHeader* hdr, SliceStart* starts, int32_t* prefix, hipStream_t stream);
hipError_t launch_decode_valu(const DecodeParams& p, int32_t group, Schedule sched,
                              int32_t grid, hipStream_t stream);
hipError_t launch_decode_mfma(const DecodeParams& p, int32_t group, Schedule sched,
                              int32_t grid, hipStream_t stream);
hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);
hipError_t launch_combine(const DecodeParams& p, int32_t group, int32_t grid, hipStream_t stream);
hipError_t launch_gather(const uint16_t* cache, int32_t is_v, const int32_t* table,
                         const int32_t* lens, const int32_t* offsets, int32_t batch,
                         int32_t mbps, int32_t hkv, int32_t head_dim, int32_t block_size,
                         int32_t num_blocks, int64_t blk_stride, uint16_t* dst,
                         hipStream_t stream);
hipError_t launch_validate(const int32_t* table, const int32_t* lens, int32_t batch,
                           int32_t mbps, int32_t block_size, int32_t num_blocks,
                           int32_t* error_count, hipStream_t stream);

}  // namespace neo
