// Decode attention, matrix-core family (gfx950 bf16 MFMA).
//
// One wavefront walks one slice of the batch's (request, kv head, block)
// tiles. For every KV block it reads the 4 KiB K tile and the 4 KiB V tile
// once for the whole GQA query group (the group is padded to 16 columns):
//
//   S^T[16 tokens][16 heads] = K_tile[16][128] . Q^T[128][16]      4 x mfma 16x16x32 bf16
//   O^T[128 dims][16 heads] += V_tile^T[128][16] . P[16][16]        8 x mfma 16x16x16 bf16
//
// The storage layout makes every load land directly in MFMA operand order:
// K piece c of token t sits at 16*(16c + t) bytes, so lane l of load kb reads
// bytes 16*(64kb + l) (one contiguous 1 KiB per instruction) and holds token
// l%16, dims 8(4kb + l/16)..+8 -- the A-operand row l%16. V is dim-major, so
// lane l of load mb reads dim 16mb + l%16, tokens 4(l/16)..+4 (8 contiguous
// bytes; 512 contiguous bytes per instruction) -- the A operand of the second
// product. The score accumulator gives lane l tokens 4(l/16)+i of head l%16,
// which is exactly the B-operand order the second product needs, so softmax
// weights never leave registers.
//
// Online softmax in base 2 (scale * log2 e folded in): per head, the running
// max is reduced across the four lanes that share a head with two shuffles;
// each lane keeps a partial sum of its own tokens' weights. The weights enter
// the second product as bf16 hi + lo halves, which keeps ~16 mantissa bits.
#include <math.h>

#include "decode_common.h"

namespace neo {
namespace {

struct MfmaTile {
  bf16x8_t k[4];
  s16x4_t v[8];
};

__device__ inline void load_tile(MfmaTile& x, const uint16_t* __restrict__ kbase,
                                 const uint16_t* __restrict__ vbase, int lane, int col, int rq) {
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    x.k[kb] = *reinterpret_cast<const bf16x8_t*>(kbase + kPiece * (kWave * kb + lane));
#pragma unroll
  for (int mb = 0; mb < 8; ++mb)
    x.v[mb] = *reinterpret_cast<const s16x4_t*>(vbase + (16 * mb + col) * kBlock + 4 * rq);
}

struct MfmaState {
  f32x4_t acc[8];  // O^T: lane holds dims 16mb + 4(l/16) + i of head l%16
  float m;         // running max (base-2 scaled), identical across a head's lanes
  float l;         // this lane's share of the softmax denominator
};

template <int G>
__device__ inline void tile_step(MfmaState& st, MfmaTile& x, const bf16x8_t (&qf)[4],
                                 int32_t valid, float scale_log2, int rq) {
  f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x.k[kb], qf[kb], s, 0, 0, 0);

  float sc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) sc[i] = (4 * rq + i < valid) ? s[i] * scale_log2 : -INFINITY;
  if (valid < kBlock) {
    // Slots past the request's length may hold anything (even NaN): select
    // them out of V rather than multiplying by a zero weight.
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (4 * rq + i >= valid) x.v[mb][i] = 0;
  }
  float mt = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
  mt = fmaxf(mt, __shfl_xor(mt, 16));
  mt = fmaxf(mt, __shfl_xor(mt, 32));
  const float mn = fmaxf(st.m, mt);  // finite: every tile has a valid token
  const float alpha = __builtin_amdgcn_exp2f(st.m - mn);
  float pr[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) pr[i] = __builtin_amdgcn_exp2f(sc[i] - mn);
  st.l = fmaf(st.l, alpha, (pr[0] + pr[1]) + (pr[2] + pr[3]));
  st.m = mn;

  __bf16 hi[4], lo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi[i] = (__bf16)pr[i];
    lo[i] = (__bf16)(pr[i] - (float)hi[i]);
  }
  s16x4_t phi, plo;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    phi[i] = __builtin_bit_cast(short, hi[i]);
    plo[i] = __builtin_bit_cast(short, lo[i]);
  }
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) {
    st.acc[mb] *= alpha;
    st.acc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.v[mb], phi, st.acc[mb], 0, 0, 0);
    st.acc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.v[mb], plo, st.acc[mb], 0, 0, 0);
  }
}

template <int G>
__global__ __launch_bounds__(kWave * kWavesPerGroup) void decode_mfma_kernel(DecodeParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = blockIdx.x * kWavesPerGroup + (threadIdx.x >> 6);
  const int nwaves = gridDim.x * kWavesPerGroup;
  zero_empty_rows(p, wave, nwaves, lane);
  const int n_slices = p.hdr->n_slices;
  if (wave >= n_slices) return;

  const SliceStart s0 = p.starts[wave];
  const int32_t tend = p.starts[wave + 1].tile;
  const int col = lane & 15, rq = lane >> 4;
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

    bf16x8_t qf[4];
    const uint16_t* qrow = p.q + ((size_t)b * p.hq + g * G + (col < G ? col : 0)) * kHeadDim;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      bf16x8_t v = *reinterpret_cast<const bf16x8_t*>(qrow + kPiece * (4 * kb + rq));
      qf[kb] = (col < G) ? v : bf16x8_t{};
    }

    MfmaState st;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) st.acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m = -INFINITY;
    st.l = 0.f;

    TableCursor tc(p.table + (size_t)b * p.mbps, j, jend, p.num_blocks, lane);
    const uint16_t* kg = p.k + (size_t)g * kTileElems;
    const uint16_t* vg = p.v + (size_t)g * kTileElems;
    MfmaTile A, B;
    int32_t jj = j;
    {
      const size_t off = (size_t)tc.get(jj) * blk_stride;
      load_tile(A, kg + off, vg + off, lane, col, rq);
    }
    while (true) {
      if (jj + 1 < jend) {
        const size_t off = (size_t)tc.get(jj + 1) * blk_stride;
        load_tile(B, kg + off, vg + off, lane, col, rq);
      }
      tile_step<G>(st, A, qf, L - jj * kBlock, p.scale_log2, rq);
      if (++jj >= jend) break;
      if (jj + 1 < jend) {
        const size_t off = (size_t)tc.get(jj + 1) * blk_stride;
        load_tile(A, kg + off, vg + off, lane, col, rq);
      }
      tile_step<G>(st, B, qf, L - jj * kBlock, p.scale_log2, rq);
      if (++jj >= jend) break;
    }

    float lt = st.l + __shfl_xor(st.l, 16);
    lt += __shfl_xor(lt, 32);
    const float inv = 1.f / lt;
    if (j == 0 && jend == nb) {
      if (col < G) {
        float* orow = p.out + ((size_t)b * p.hq + g * G + col) * kHeadDim + 4 * rq;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
          *reinterpret_cast<f32x4_t*>(orow + 16 * mb) = st.acc[mb] * inv;
      }
    } else {
      const int slot = partial_slot(wave, s0.tile, pair_first);
      if (col < G) {
        float* orow = p.part_o + ((size_t)slot * G + col) * kHeadDim + 4 * rq;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
          *reinterpret_cast<f32x4_t*>(orow + 16 * mb) = st.acc[mb] * inv;
        if (rq == 0) p.part_lse[slot * G + col] = (st.m + __log2f(lt)) * kLn2;
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
}

}  // namespace

hipError_t launch_decode_mfma(const DecodeParams& p, int32_t group, int32_t grid,
                              hipStream_t stream) {
  const dim3 block(kWave * kWavesPerGroup);
  switch (group) {
    case 1: decode_mfma_kernel<1><<<grid, block, 0, stream>>>(p); break;
    case 2: decode_mfma_kernel<2><<<grid, block, 0, stream>>>(p); break;
    case 4: decode_mfma_kernel<4><<<grid, block, 0, stream>>>(p); break;
    case 8: decode_mfma_kernel<8><<<grid, block, 0, stream>>>(p); break;
    case 16: decode_mfma_kernel<16><<<grid, block, 0, stream>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace neo
