// Decode attention, matrix-core family (gfx950 bf16 MFMA).
//
// For every KV block the wavefront reads the 4 KiB K tile and the 4 KiB V tile
// once for the whole GQA query group (padded to 16 columns):
//
//   S^T[16 tokens][16 heads] = K_tile[16][128] . Q^T[128][16]      4 x mfma 16x16x32 bf16
//   O^T[128 dims][16 heads] += V_tile^T[128][16] . P[16][16]        16 x mfma 16x16x16 bf16
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
// the second product as bf16 hi + lo halves (two products), which keeps ~16
// mantissa bits of each weight.
#include "decode_common.h"

namespace neo {
namespace {

template <int G>
struct MfmaFamily {
  struct Tile {
    bf16x8_t k[4];
    s16x4_t v[8];
  };
  struct Q {
    bf16x8_t f[4];
  };
  struct State {
    f32x4_t acc[8];  // O^T: lane holds dims 16mb + 4(l/16) + i of head l%16
    float m;         // running max (base-2 scaled), identical across a head's lanes
    float l;         // this lane's share of the softmax denominator
  };
  struct Shared {
    int unused;
  };
  static constexpr bool kFastMerge = true;  // provides merge_write

  __device__ static void load_q(Q& q, const uint16_t* __restrict__ qpair, int lane) {
    const int col = lane & 15, rq = lane >> 4;
    const uint16_t* row = qpair + (col < G ? col : 0) * kHeadDim;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const bf16x8_t v = *reinterpret_cast<const bf16x8_t*>(row + kPiece * (4 * kb + rq));
      q.f[kb] = (col < G) ? v : bf16x8_t{};
    }
  }

  __device__ static void init(State& st) {
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) st.acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m = -INFINITY;
    st.l = 0.f;
  }

  // valid == false: the tile is past the segment; its registers read zeros
  // and no memory is touched.
  __device__ static void load_tile(Tile& x, const uint16_t* kbase, const uint16_t* vbase,
                                   bool valid, int lane) {
    const int col = lane & 15, rq = lane >> 4;
    // Each KV tile is read exactly once: nontemporal loads keep it from
    // displacing reusable lines in the caches.
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(kbase, valid), rv = tile_rsrc(vbase, valid);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      x.k[kb] = __builtin_bit_cast(bf16x8_t, tile_load16(rk, 2 * kPiece * (kWave * kb + lane)));
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
      x.v[mb] = tile_load8(rv, 2 * ((16 * mb + col) * kBlock + 4 * rq));
  }

  __device__ static void step(State& st, Tile& x, const Q& q, int32_t valid, float scale_log2,
                              int lane, Shared&) {
    const int rq = lane >> 4;
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x.k[kb], q.f[kb], s, 0, 0, 0);

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
    mt = max_over_rows(mt);
    const float mn = fmaxf(st.m, mt);  // finite: every tile has a valid token
    const float alpha = __builtin_amdgcn_exp2f(st.m - mn);
    float pr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pr[i] = __builtin_amdgcn_exp2f(sc[i] - mn);
    st.l = fmaf(st.l, alpha, (pr[0] + pr[1]) + (pr[2] + pr[3]));
    st.m = mn;

    s16x4_t phi, plo;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const __bf16 hi = (__bf16)pr[i];
      const __bf16 lo = (__bf16)(pr[i] - (float)hi);
      phi[i] = __builtin_bit_cast(short, hi);
      plo[i] = __builtin_bit_cast(short, lo);
    }
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      st.acc[mb] *= alpha;
      st.acc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.v[mb], phi, st.acc[mb], 0, 0, 0);
      st.acc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.v[mb], plo, st.acc[mb], 0, 0, 0);
    }
  }

  // rows: [G][128] destination (normalised); lse: [G] natural-log log-sum-exp or
  // null. kCoherent: partials another slice will merge (device-coherent stores).
  template <bool kCoherent>
  __device__ static void write(const State& st, float* __restrict__ rows,
                               float* __restrict__ lse, int lane) {
    const int col = lane & 15, rq = lane >> 4;
    const float lt = sum_over_rows(st.l);
    const float inv = 1.f / lt;
    if (col < G) {
      float* r = rows + col * kHeadDim + 4 * rq;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        const f32x4_t v = st.acc[mb] * inv;
        if (kCoherent) {
          store_coherent2(r + 16 * mb, v[0], v[1]);
          store_coherent2(r + 16 * mb + 2, v[2], v[3]);
        } else {
          *reinterpret_cast<f32x4_t*>(r + 16 * mb) = v;
        }
      }
      if (lse && rq == 0) {
        const float x = (st.m + __log2f(lt)) * kLn2;
        if (kCoherent) store_coherent(lse + col, x); else lse[col] = x;
      }
    }
  }

  // The pair's two-contributor merge done in registers: this slice's share
  // (st, not yet written) first, then the other slice's complete partial
  // (other_rows, other_lse, device-coherent loads); the same arithmetic as
  // merge_two_values on the stored partials, so the output bits are the same.
  __device__ static void merge_write(const State& st, const float* __restrict__ other_rows,
                                     const float* __restrict__ other_lse,
                                     float* __restrict__ out_rows, int lane) {
    const int col = lane & 15, rq = lane >> 4;
    const float lt = sum_over_rows(st.l);
    const float inv = 1.f / lt;
    if (col < G) {
      // Rounded exactly as the stored log-sum-exp of write(): the empty asm
      // makes la an opaque value, so the compiler cannot fuse its multiply
      // with the subtraction of the max below (the merge must see the same
      // value as the merge of stored partials).
      float la = (st.m + __log2f(lt)) * kLn2;
      asm volatile("" : "+v"(la));
      const float lb = load_coherent(other_lse + col);
      const float* ob = other_rows + col * kHeadDim + 4 * rq;
      float2 o2[8][2];
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        o2[mb][0] = load_coherent2(ob + 16 * mb);
        o2[mb][1] = load_coherent2(ob + 16 * mb + 2);
      }
      const float m = fmaxf(la, lb);
      const float wa = __expf(la - m), wb = __expf(lb - m);
      const float inv2 = 1.f / (wa + wb);
      float* r = out_rows + col * kHeadDim + 4 * rq;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        const f32x4_t oa = st.acc[mb] * inv;
        const float obv[4] = {o2[mb][0].x, o2[mb][0].y, o2[mb][1].x, o2[mb][1].y};
        f32x4_t res;
#pragma unroll
        for (int i = 0; i < 4; ++i) res[i] = fmaf(wb, obv[i], wa * oa[i]) * inv2;
        *reinterpret_cast<f32x4_t*>(r + 16 * mb) = res;
      }
    }
  }
};

template <int G, Schedule kSched>
__global__ __launch_bounds__(kWave * kWavesPerGroup, 2) void decode_mfma_kernel(
    const int32_t* __restrict__ lens, int32_t batch, int32_t hkv, int32_t mbps, DecodeParams p) {
  // The first step of every wave reads the request lengths: the arguments it
  // needs for that come first and separately, so that they can arrive in
  // registers with the wave (kernel-argument preload) instead of one scalar
  // load round trip later.
  p.lens = lens;
  p.batch = batch;
  p.hkv = hkv;
  p.mbps = mbps;
  // One tile in flight ahead of the one being computed: with 4 waves on every
  // CU that keeps HBM saturated; deeper prefetch measured equal or slower
  // (more requests in flight lower the HBM efficiency).
  decode_driver<MfmaFamily<G>, G, 1, kSched>(p);
}

template <int G>
hipError_t launch_g(const DecodeParams& p, Schedule sched, int32_t grid, hipStream_t stream) {
  const dim3 block(kWave * kWavesPerGroup);
  switch (sched) {
    case kStaged: decode_mfma_kernel<G, kStaged><<<grid, block, 0, stream>>>(p.lens, p.batch, p.hkv, p.mbps, p); break;
    case kFused: decode_mfma_kernel<G, kFused><<<grid, block, 0, stream>>>(p.lens, p.batch, p.hkv, p.mbps, p); break;
    case kTwoKernel: decode_mfma_kernel<G, kTwoKernel><<<grid, block, 0, stream>>>(p.lens, p.batch, p.hkv, p.mbps, p); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_mfma(const DecodeParams& p, int32_t group, Schedule sched,
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
