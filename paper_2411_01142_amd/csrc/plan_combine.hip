// Work plan (block-granular partition of the batch), log-sum-exp combine of
// split requests, and the test-facing gather / validation kernels.
//
// The partition follows the paper's Sec. 4 ("Efficient CPU Kernels"): every
// request's attention is cut along its sequence at KV-block granularity, each
// worker gets an equal number of blocks, and the partial outputs of a request
// are aggregated afterwards. Here a worker is one wavefront: the batch's tiles
// ((request, kv head, block) triples) are laid end to end and cut into equal
// contiguous slices, so the load is balanced whatever the length mix.
#include <algorithm>

#include "decode_common.h"

namespace neo {
namespace {

// One workgroup: pair weights, an exclusive scan over requests (weighted
// offsets), then each slice's first position located by binary search (over
// an LDS copy of the offsets when the batch fits).
constexpr int kPlanLdsBatch = 8192;

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(
    const int32_t* __restrict__ lens, int32_t batch, int32_t hkv, int32_t mbps,
    int32_t max_slices, int32_t min_tiles, int32_t quantum, int32_t xcd8,
    PlanHeader* __restrict__ hdr,
    SliceStart* __restrict__ starts, int32_t* __restrict__ prefix) {
  __shared__ int32_t sums[kPlanThreads];
  __shared__ int32_t sprefix[kPlanLdsBatch + 1];
  const bool in_lds = batch <= kPlanLdsBatch;
  const int tid = threadIdx.x;
  const int per = (batch + kPlanThreads - 1) / kPlanThreads;
  const int b0 = min(batch, tid * per);
  const int b1 = min(batch, b0 + per);
  int32_t local = 0;
  for (int b = b0; b < b1; ++b) local += pair_weight(lens[b], mbps);
  sums[tid] = local;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off <<= 1) {
    int32_t add = tid >= off ? sums[tid - off] : 0;
    __syncthreads();
    sums[tid] += add;
    __syncthreads();
  }
  int32_t run = tid == 0 ? 0 : sums[tid - 1];
  for (int b = b0; b < b1; ++b) {
    if (in_lds) sprefix[b] = run * hkv;
    else prefix[b] = run * hkv;
    run += pair_weight(lens[b], mbps);
  }
  const int32_t total = sums[kPlanThreads - 1] * hkv;
  __syncthreads();
  const int32_t* pre = in_lds ? sprefix : prefix;

  const int32_t n = slice_count(total, min_tiles, max_slices, quantum);
  const SliceGeom geo = make_slice_geom(total, n, xcd8 != 0);
  for (int s = tid; s <= n; s += kPlanThreads) {
    SliceStart st;
    st.pad[0] = st.pad[1] = st.pad[2] = 0;
    if (s == n) {
      st.pos = total;
      st.b = batch;
      st.g = 0;
      st.x = 0;
      st.nb = 0;
    } else {
      const int32_t pos = slice_start(s, geo);
      int lo = 0, hi = batch - 1;  // largest b with pre[b] <= pos
      while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= pos) lo = mid; else hi = mid - 1;
      }
      const int32_t w = pair_weight(lens[lo], mbps);
      const int32_t r = pos - pre[lo];
      st.pos = pos;
      st.b = lo;
      st.g = r / w;
      st.x = r % w;
      st.nb = blocks_of(lens[lo], mbps);
    }
    starts[s] = st;
  }
  if (tid == 0) {
    PlanHeader h;
    h.total = total;
    h.n_slices = n;
    h.batch = batch;
    h.pad = 0;
    *hdr = h;
  }
}

// Staged launch: aggregation of the partial outputs of pairs cut by slice
// boundaries (Sec. 4: the per-request partial results are combined). Wave
// w looks at boundary s = w + 1: when it falls strictly inside the tiles of a
// pair whose first tile lies in slice s - 1, that boundary is the first to cut
// the pair and the wave merges it. Every contributing slice stored its part
// normalised, with its log-sum-exp.
template <int G>
__global__ __launch_bounds__(kWave * kWavesPerGroup) void combine_kernel(DecodeParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int s = blockIdx.x * kWavesPerGroup + (threadIdx.x >> 6) + 1;
  if (s > NEO_MAX_SLICES) return;
  // The header and this boundary's record are loaded together (the record
  // array always holds NEO_MAX_SLICES + 1 entries; stale ones are not used).
  const SliceStart a = p.starts[s];
  const int32_t W = p.hdr->total;
  const int32_t n = p.hdr->n_slices;
  // A pair cut at this boundary nearly always has exactly two contributors:
  // slice s-1's end-cut segment (slot 2s-1) and slice s's first segment (slot
  // 2s). Their log-sum-exps and rows are loaded in the same round trip as the
  // record (all slots exist whatever the plan; unused values are ignored).
  // (s <= NEO_MAX_SLICES here; the slots read are clamped below 2 NEO_MAX_SLICES,
  // s = NEO_MAX_SLICES being a boundary no plan has.)
  const int d = 2 * lane;
  const int sa = 2 * min(s, NEO_MAX_SLICES - 1) - 1, sb = sa + 1;
  float la[G], lb[G];
  float2 oa[G], ob[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    la[h] = p.part_lse[sa * G + h];
    lb[h] = p.part_lse[sb * G + h];
    oa[h] = *reinterpret_cast<const float2*>(p.part_o + ((size_t)sa * G + h) * kHeadDim + d);
    ob[h] = *reinterpret_cast<const float2*>(p.part_o + ((size_t)sb * G + h) * kHeadDim + d);
  }
  // Every value above is an operand of this empty statement, so all the loads
  // are issued before the branches below (left alone, the compiler moves the
  // speculative ones after them, costing a second round trip).
  asm volatile("" ::"v"(a.pos), "v"(a.x), "v"(a.nb), "s"(W), "s"(n));
#pragma unroll
  for (int h = 0; h < G; ++h)
    asm volatile("" ::"v"(la[h]), "v"(lb[h]), "v"(oa[h].x), "v"(oa[h].y), "v"(ob[h].x),
                 "v"(ob[h].y));
  if (s >= n) return;
  const int32_t cost = pair_cost(a.nb);
  if (a.x <= cost) return;                      // no tile of the pair before the boundary
  const int32_t first_tile = a.pos - a.x + cost;
  const SliceGeom geo = make_slice_geom(W, n, p.xcd8 != 0);
  const int32_t prev_start = slice_start(s - 1, geo);
  if (first_tile < prev_start) return;          // an earlier boundary cuts it first
  const int32_t c1 = slice_of(first_tile + a.nb - 1, geo);
  if (c1 == s && first_tile > prev_start) {
    merge_two_values<G>(p, a.b, a.g, la, lb, oa, ob, lane);  // slots 2s-1, 2s
    return;
  }
  merge_pair<G, false>(p, p.part_o, p.part_lse, 0, a.b, a.g, first_tile, s - 1, c1, geo, lane);
}

__global__ __launch_bounds__(256) void fill_zero_kernel(uint32_t* __restrict__ dst, size_t words) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
       i += (size_t)gridDim.x * blockDim.x)
    dst[i] = 0u;
}

// Workgroup (j, b) copies block j of request b: thread -> (slot, 8-dim piece).
__global__ __launch_bounds__(256) void gather_kernel(
    const uint16_t* __restrict__ cache, int32_t is_v, const int32_t* __restrict__ table,
    const int32_t* __restrict__ lens, const int32_t* __restrict__ offsets, int32_t mbps,
    int32_t hkv, int32_t head_dim, int32_t block_size, int32_t num_blocks, int64_t blk_stride,
    uint16_t* __restrict__ dst) {
  const int j = blockIdx.x, b = blockIdx.y;
  const int32_t L = min(max(lens[b], 0), mbps * block_size);
  const int32_t t0 = j * block_size;
  if (t0 >= L) return;
  const int32_t valid = min(block_size, L - t0);
  int32_t phys = table[(size_t)b * mbps + j];
  phys = (int32_t)min((uint32_t)phys, (uint32_t)(num_blocks - 1));
  const int pieces = head_dim / kPiece;
  const int items = hkv * valid * pieces;
  const size_t row0 = (size_t)offsets[b] + t0;
  for (int it = threadIdx.x; it < items; it += blockDim.x) {
    const int c = it % pieces;
    const int o = (it / pieces) % valid;
    const int g = it / (pieces * valid);
    uint16_t vals[kPiece];
    for (int e = 0; e < kPiece; ++e) {
      const int d = c * kPiece + e;
      size_t src;
      if (is_v)
        src = ((size_t)g * head_dim + d) * block_size + o;
      else
        src = (((size_t)g * pieces + c) * block_size + o) * kPiece + e;
      src += (size_t)phys * (size_t)blk_stride;
      vals[e] = cache[src];
    }
    uint16_t* out = dst + ((row0 + o) * hkv + g) * head_dim + c * kPiece;
    for (int e = 0; e < kPiece; ++e) out[e] = vals[e];
  }
}

__global__ __launch_bounds__(256) void validate_kernel(const int32_t* __restrict__ table,
                                                       const int32_t* __restrict__ lens,
                                                       int32_t batch, int32_t mbps,
                                                       int32_t block_size, int32_t num_blocks,
                                                       int32_t* error_count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)batch * mbps) return;
  const int b = (int)(i / mbps), j = (int)(i % mbps);
  const int32_t L = lens[b];
  int bad = 0;
  if (j == 0 && (L < 0 || (int64_t)L > (int64_t)mbps * block_size)) bad++;
  const int32_t Lc = min(max(L, 0), mbps * block_size);
  if ((int64_t)j * block_size < Lc) {
    const int32_t phys = table[i];
    if (phys < 0 || phys >= num_blocks) bad++;
  }
  if (bad) atomicAdd(error_count, bad);
}

}  // namespace

hipError_t launch_plan(const int32_t* lens, int32_t batch, int32_t hkv, int32_t mbps,
                       int32_t max_slices, int32_t min_tiles, int32_t quantum, int32_t xcd8,
                       PlanHeader* hdr, SliceStart* starts, int32_t* prefix, hipStream_t stream) {
  plan_kernel<<<1, kPlanThreads, 0, stream>>>(lens, batch, hkv, mbps, max_slices, min_tiles,
                                              quantum, xcd8, hdr, starts, prefix);
  return hipGetLastError();
}

hipError_t launch_combine(const DecodeParams& p, int32_t group, int32_t grid, hipStream_t stream) {
  const dim3 block(kWave * kWavesPerGroup);
  switch (group) {
    case 1: combine_kernel<1><<<grid, block, 0, stream>>>(p); break;
    case 2: combine_kernel<2><<<grid, block, 0, stream>>>(p); break;
    case 4: combine_kernel<4><<<grid, block, 0, stream>>>(p); break;
    case 8: combine_kernel<8><<<grid, block, 0, stream>>>(p); break;
    case 16: combine_kernel<16><<<grid, block, 0, stream>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream) {
  const size_t words = bytes / 4;
  if (words == 0) return hipSuccess;
  const size_t blocks = std::min<size_t>((words + 255) / 256, 4096);
  fill_zero_kernel<<<(unsigned)blocks, 256, 0, stream>>>(static_cast<uint32_t*>(ptr), words);
  return hipGetLastError();
}

hipError_t launch_gather(const uint16_t* cache, int32_t is_v, const int32_t* table,
                         const int32_t* lens, const int32_t* offsets, int32_t batch,
                         int32_t mbps, int32_t hkv, int32_t head_dim, int32_t block_size,
                         int32_t num_blocks, int64_t blk_stride, uint16_t* dst,
                         hipStream_t stream) {
  gather_kernel<<<dim3(mbps, batch), 256, 0, stream>>>(cache, is_v, table, lens, offsets, mbps,
                                                       hkv, head_dim, block_size, num_blocks,
                                                       blk_stride, dst);
  return hipGetLastError();
}

hipError_t launch_validate(const int32_t* table, const int32_t* lens, int32_t batch,
                           int32_t mbps, int32_t block_size, int32_t num_blocks,
                           int32_t* error_count, hipStream_t stream) {
  const int64_t n = (int64_t)batch * mbps;
  const int blocks = (int)((n + 255) / 256);
  validate_kernel<<<blocks, 256, 0, stream>>>(table, lens, batch, mbps, block_size, num_blocks,
                                             error_count);
  return hipGetLastError();
}

}  // namespace neo
