// Decode attention, vector-ALU family.
//
// For every KV block the wavefront reads the 4 KiB K tile and the 4 KiB V
// tile once for the whole GQA query group. Lane l = 16r + c:
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
#include "decode_common.h"

namespace neo {
namespace {

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

__device__ inline void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int G>
struct ValuFamily {
  struct Tile {
    u32x4_t k[4];
    u32x4_t v[4];
  };
  struct Q {
    u32x4_t v[G];  // dims 8c..8c+7 of each head of the group
  };
  struct State {
    float acc[4][G];  // dim 32i + l/2, head h; this lane's half of each tile's tokens
    float m[G];       // running max per head (base-2 scaled), wave-uniform
    float l[G];       // this row's share of the denominator per head
  };
  struct Shared {
    float p[G * kBlock];  // softmax weights of the current tile, [head][token]
  };
  static constexpr bool kFastMerge = false;  // no merge_write: the general path merges


  __device__ static void load_q(Q& q, const uint16_t* __restrict__ qpair, int lane) {
    const int c = lane & 15;
#pragma unroll
    for (int h = 0; h < G; ++h)
      q.v[h] = *reinterpret_cast<const u32x4_t*>(qpair + h * kHeadDim + kPiece * c);
  }

  __device__ static void init(State& st) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      st.m[h] = -INFINITY;
      st.l[h] = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) st.acc[i][h] = 0.f;
    }
  }

  // valid == false: the tile is past the segment; its registers read zeros
  // and no memory is touched.
  __device__ static void load_tile(Tile& x, const uint16_t* kbase, const uint16_t* vbase,
                                   bool valid, int lane) {
    const int r = lane >> 4, c = lane & 15;
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kbase, valid), rv = tile_rsrc(vbase, valid);
#pragma unroll
    for (int i = 0; i < 4; ++i) x.k[i] = tile_load16(rk, 2 * (c * kBlock + 4 * i + r) * kPiece);
#pragma unroll
    for (int i = 0; i < 4; ++i) x.v[i] = tile_load16(rv, 2 * (512 * i + 8 * lane));
  }

  __device__ static void step(State& st, Tile& x, const Q& q, int32_t valid, float scale_log2,
                              int lane, Shared& sh) {
    const int r = lane >> 4;
    float s[4][G];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int h = 0; h < G; ++h) s[i][h] = dpp_row_allreduce(dot8(q.v[h], x.k[i]));

    float alpha[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mt = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[i][h] = (4 * i + r < valid) ? s[i][h] * scale_log2 : -INFINITY;
        mt = fmaxf(mt, s[i][h]);
      }
      mt = max_over_rows(mt);
      const float mn = fmaxf(st.m[h], mt);
      alpha[h] = __builtin_amdgcn_exp2f(st.m[h] - mn);
      st.m[h] = mn;
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[i][h] = __builtin_amdgcn_exp2f(s[i][h] - mn);
        ps += s[i][h];
        sh.p[h * kBlock + 4 * i + r] = s[i][h];
      }
      st.l[h] = fmaf(st.l[h], alpha[h], ps);
    }
    wave_sync_lds();

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
      const f32x4_t p0 = *reinterpret_cast<const f32x4_t*>(sh.p + h * kBlock + 8 * half);
      const f32x4_t p1 = *reinterpret_cast<const f32x4_t*>(sh.p + h * kBlock + 8 * half + 4);
      const float pw[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = st.acc[i][h] * alpha[h];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t w = x.v[i][e];
          a = fmaf(pw[2 * e], bf16_lo(w), a);
          a = fmaf(pw[2 * e + 1], bf16_hi(w), a);
        }
        st.acc[i][h] = a;
      }
    }
    wave_sync_lds();
  }

  template <bool kCoherent>
  __device__ static void write(const State& st, float* __restrict__ rows,
                               float* __restrict__ lse, int lane) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float lt = sum_over_rows(st.l[h]);
      const float inv = 1.f / lt;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a =
            st.acc[i][h] + __builtin_amdgcn_update_dpp(0.f, st.acc[i][h], 0xB1, 0xF, 0xF, false);
        if ((lane & 1) == 0) {
          float* dst = rows + h * kHeadDim + 32 * i + (lane >> 1);
          if (kCoherent) store_coherent(dst, a * inv); else *dst = a * inv;
        }
      }
      if (lse && lane == 0) {
        const float x = (st.m[h] + __log2f(lt)) * kLn2;
        if (kCoherent) store_coherent(lse + h, x); else lse[h] = x;
      }
    }
  }
};

template <int G, Schedule kSched>
__global__ __launch_bounds__(kWave * kWavesPerGroup) void decode_valu_kernel(DecodeParams p) {
  decode_driver<ValuFamily<G>, G, 1, kSched>(p);
}

template <int G>
hipError_t launch_g(const DecodeParams& p, Schedule sched, int32_t grid, hipStream_t stream) {
  const dim3 block(kWave * kWavesPerGroup);
  switch (sched) {
    case kStaged: decode_valu_kernel<G, kStaged><<<grid, block, 0, stream>>>(p); break;
    case kFused: decode_valu_kernel<G, kFused><<<grid, block, 0, stream>>>(p); break;
    case kTwoKernel: decode_valu_kernel<G, kTwoKernel><<<grid, block, 0, stream>>>(p); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_valu(const DecodeParams& p, int32_t group, Schedule sched,
                              int32_t grid, hipStream_t stream) {
  switch (group) {
    case 1: return launch_g<1>(p, sched, grid, stream);
    case 2: return launch_g<2>(p, sched, grid, stream);
    case 4: return launch_g<4>(p, sched, grid, stream);
    case 8: return launch_g<8>(p, sched, grid, stream);
    case 16: return launch_g<16>(p, sched, grid, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace neo
