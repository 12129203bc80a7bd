// Device helpers shared by the two decode-kernel families: the slice walk over
// (request, kv head, block) tiles, the block-table cursor and the zero rows of
// empty requests.
#pragma once

#include "neo_internal.h"

namespace neo {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.6931471805599453f;

// Requests with no tokens get a zero row; every wavefront of the grid takes a
// strided share of the batch.
__device__ inline void zero_empty_rows(const DecodeParams& p, int wave, int nwaves, int lane) {
  for (int b = wave; b < p.batch; b += nwaves) {
    if (clamp_len(p.lens[b], p.mbps) != 0) continue;
    f32x4_t* row = reinterpret_cast<f32x4_t*>(p.out + (size_t)b * p.hq * kHeadDim);
    const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
    for (int i = lane; i < p.hq * (kHeadDim / 4); i += kWave) row[i] = z;
  }
}

// Physical block ids of one request row, fetched 64 at a time (one per lane)
// and handed out with a uniform readlane; ids are clamped into the pool.
struct TableCursor {
  const int32_t* row;
  int32_t base, end, vals, last_block;
  int lane;
  __device__ TableCursor(const int32_t* row_, int32_t j0, int32_t jend, int32_t num_blocks,
                         int lane_)
      : row(row_), base(j0), end(jend), last_block(num_blocks - 1), lane(lane_) {
    vals = (base + lane < end) ? row[base + lane] : 0;
  }
  __device__ int32_t get(int32_t jj) {
    if (jj - base >= kWave) {
      base += kWave;
      vals = (base + lane < end) ? row[base + lane] : 0;
    }
    const int32_t id = __builtin_amdgcn_readlane(vals, jj - base);
    return (int32_t)min((uint32_t)id, (uint32_t)last_block);
  }
};

// Where a finished segment of pair (b, g) goes: straight to `out` when the
// segment is the whole pair, else to a partial slot of this slice. A slice's
// first segment uses slot 2w, a segment that starts later (and so is cut by the
// slice's end) uses 2w+1; the combine kernel recomputes the same rule.
__device__ inline int partial_slot(int wave, int32_t slice_first_tile, int32_t pair_first_tile) {
  return slice_first_tile >= pair_first_tile ? 2 * wave : 2 * wave + 1;
}

}  // namespace neo
