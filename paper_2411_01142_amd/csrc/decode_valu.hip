// Decode attention, vector-ALU family.
//
// One wavefront walks one slice of the batch's (request, kv head, block)
// tiles and reads each 4 KiB K tile and 4 KiB V tile once for the whole GQA
// query group. Lane l = 16r + c:
//
//   q.k : load i (0..3) gives the lane key piece c (dims 8c..8c+7) of token
//         4i + r (64 contiguous bytes per 4 lanes). The lane keeps the same
//         8 dims of every query head of the group in registers and forms
//         partial dots with v_dot2_f32_bf16; a 4-step DPP all-reduce inside the
//         16-lane row (xor 1, xor 2, half-mirror, mirror) completes them.
//   softmax: every lane of row r then holds the scores of tokens 4i + r for
//         all heads; the per-head max crosses the four rows with two shuffles.
//   p.V : the weights go through a small per-wave LDS buffer; load i gives
//         the lane 8 consecutive tokens of dim 32i + l/2 (1 KiB contiguous per
//         instruction), accumulated in fp32 per (dim, head); the two lanes
//         sharing a dim are summed once at the end of a segment.
#include <math.h>

#include "decode_common.h"

namespace neo {
namespace {

struct ValuTile {
  u32x4_t k[4];
  u32x4_t v[4];
};

__device__ inline void load_tile(ValuTile& x, const uint16_t* __restrict__ kbase,
                                 const uint16_t* __restrict__ vbase, int lane, int r, int c) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    x.k[i] = *reinterpret_cast<const u32x4_t*>(kbase + (c * kBlock + 4 * i + r) * kPiece);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    x.v[i] = *reinterpret_cast<const u32x4_t*>(vbase + 512 * i + 8 * lane);
}

__device__ inline float dpp_row_allreduce(float v) {
  v += __builtin_amdgcn_update_dpp(0.f, v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  v += __builtin_amdgcn_update_dpp(0.f, v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  v += __builtin_amdgcn_update_dpp(0.f, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += __builtin_amdgcn_update_dpp(0.f, v, 0x140, 0xF, 0xF, false);  // row_mirror
  return v;
}

__device__ inline float dot8(const u32x4_t& a, const u32x4_t& b) {
  float acc = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    // Bit-cast scalar copies: a cast applied to a vector-element subscript
    // directly has been lowered as a read of element 0.
    const uint32_t ae = a[e], be = b[e];
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ae),
                                          __builtin_bit_cast(bf16x2_t, be), acc, false);
  }
  return acc;
}

__device__ inline float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xFFFF0000u); }

template <int G>
struct ValuState {
  float acc[4][G];  // dim 32i + l/2, head h; this lane's half of each tile's tokens
  float m[G];       // running max per head (base-2 scaled), wave-uniform
  float l[G];       // this row's share of the denominator per head
};

template <int G>
__device__ inline void tile_step(ValuState<G>& st, ValuTile& x, const u32x4_t (&qv)[G],
                                 int32_t valid, float scale_log2, int lane, int r,
                                 float* __restrict__ plds) {
  float s[4][G];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int h = 0; h < G; ++h) s[i][h] = dpp_row_allreduce(dot8(qv[h], x.k[i]));

  float alpha[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i][h] = (4 * i + r < valid) ? s[i][h] * scale_log2 : -INFINITY;
      mt = fmaxf(mt, s[i][h]);
    }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float mn = fmaxf(st.m[h], mt);
    alpha[h] = __builtin_amdgcn_exp2f(st.m[h] - mn);
    st.m[h] = mn;
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i][h] = __builtin_amdgcn_exp2f(s[i][h] - mn);
      ps += s[i][h];
      plds[h * kBlock + 4 * i + r] = s[i][h];
    }
    st.l[h] = fmaf(st.l[h], alpha[h], ps);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  const int half = lane & 1;
  if (valid < kBlock) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // tokens 8*half + 2e (low half-word) and 8*half + 2e + 1 (high)
        const int t0 = 8 * half + 2 * e;
        uint32_t w = x.v[i][e];
        if (t0 >= valid) w &= 0xFFFF0000u;
        if (t0 + 1 >= valid) w &= 0x0000FFFFu;
        x.v[i][e] = w;
      }
  }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const f32x4_t p0 = *reinterpret_cast<const f32x4_t*>(plds + h * kBlock + 8 * half);
    const f32x4_t p1 = *reinterpret_cast<const f32x4_t*>(plds + h * kBlock + 8 * half + 4);
    const float pw[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float a = st.acc[i][h] * alpha[h];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a = fmaf(pw[2 * e], bf16_lo(x.v[i][e]), a);
        a = fmaf(pw[2 * e + 1], bf16_hi(x.v[i][e]), a);
      }
      st.acc[i][h] = a;
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int G>
__global__ __launch_bounds__(kWave * kWavesPerGroup) void decode_valu_kernel(DecodeParams p) {
  __shared__ float plds_all[kWavesPerGroup][G * kBlock];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x >> 6;
  const int wave = blockIdx.x * kWavesPerGroup + wv;
  const int nwaves = gridDim.x * kWavesPerGroup;
  zero_empty_rows(p, wave, nwaves, lane);
  const int n_slices = p.hdr->n_slices;
  if (wave >= n_slices) return;
  float* plds = plds_all[wv];

  const SliceStart s0 = p.starts[wave];
  const int32_t tend = p.starts[wave + 1].tile;
  const int r = lane >> 4, c = lane & 15;
  const size_t blk_stride = (size_t)p.hkv * kTileElems;

  int32_t t = s0.tile;
  int b = s0.b, g = s0.g, j = s0.j;
  while (t < tend && b < p.batch) {
    const int32_t L = clamp_len(p.lens[b], p.mbps);
    const int32_t nb = (L + kBlock - 1) / kBlock;
    if (nb == 0) {
      ++b;
      g = 0;
      j = 0;
      continue;
    }
    const int32_t jend = min(nb, j + (tend - t));
    const int32_t pair_first = t - j;

    u32x4_t qv[G];
    const uint16_t* qrow = p.q + ((size_t)b * p.hq + g * G) * kHeadDim + kPiece * c;
#pragma unroll
    for (int h = 0; h < G; ++h) qv[h] = *reinterpret_cast<const u32x4_t*>(qrow + h * kHeadDim);

    ValuState<G> st;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      st.m[h] = -INFINITY;
      st.l[h] = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) st.acc[i][h] = 0.f;
    }

    TableCursor tc(p.table + (size_t)b * p.mbps, j, jend, p.num_blocks, lane);
    const uint16_t* kg = p.k + (size_t)g * kTileElems;
    const uint16_t* vg = p.v + (size_t)g * kTileElems;
    ValuTile A, B;
    int32_t jj = j;
    {
      const size_t off = (size_t)tc.get(jj) * blk_stride;
      load_tile(A, kg + off, vg + off, lane, r, c);
    }
    while (true) {
      if (jj + 1 < jend) {
        const size_t off = (size_t)tc.get(jj + 1) * blk_stride;
        load_tile(B, kg + off, vg + off, lane, r, c);
      }
      tile_step<G>(st, A, qv, L - jj * kBlock, p.scale_log2, lane, r, plds);
      if (++jj >= jend) break;
      if (jj + 1 < jend) {
        const size_t off = (size_t)tc.get(jj + 1) * blk_stride;
        load_tile(A, kg + off, vg + off, lane, r, c);
      }
      tile_step<G>(st, B, qv, L - jj * kBlock, p.scale_log2, lane, r, plds);
      if (++jj >= jend) break;
    }

    const bool complete = (j == 0 && jend == nb);
    const int slot = partial_slot(wave, s0.tile, pair_first);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float lt = st.l[h] + __shfl_xor(st.l[h], 16);
      lt += __shfl_xor(lt, 32);
      const float inv = 1.f / lt;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a = st.acc[i][h] + __builtin_amdgcn_update_dpp(0.f, st.acc[i][h], 0xB1, 0xF,
                                                                    0xF, false);
        if ((lane & 1) == 0) {
          const int d = 32 * i + (lane >> 1);
          if (complete)
            p.out[((size_t)b * p.hq + g * G + h) * kHeadDim + d] = a * inv;
          else
            p.part_o[((size_t)slot * G + h) * kHeadDim + d] = a * inv;
        }
      }
      if (!complete && lane == 0) p.part_lse[slot * G + h] = (st.m[h] + __log2f(lt)) * kLn2;
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
}

}  // namespace

hipError_t launch_decode_valu(const DecodeParams& p, int32_t group, int32_t grid,
                              hipStream_t stream) {
  const dim3 block(kWave * kWavesPerGroup);
  switch (group) {
    case 1: decode_valu_kernel<1><<<grid, block, 0, stream>>>(p); break;
    case 2: decode_valu_kernel<2><<<grid, block, 0, stream>>>(p); break;
    case 4: decode_valu_kernel<4><<<grid, block, 0, stream>>>(p); break;
    case 8: decode_valu_kernel<8><<<grid, block, 0, stream>>>(p); break;
    case 16: decode_valu_kernel<16><<<grid, block, 0, stream>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace neo
