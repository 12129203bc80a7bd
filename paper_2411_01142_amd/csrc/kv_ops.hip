// The two cache operations on either side of decode attention:
//
//  * append: the decoding phase reads and appends the KV cache (Sec. 2.1);
//    the new token's key and value rows are written into their paged slot;
//  * block copy: whole (block, all kv heads) runs of K and V moved between two
//    caches, e.g. the GPU cache in HBM and a CPU cache in pinned host memory
//    (partial offloading and layer-wise swapping, Sec. 3.1). The copy is a
//    kernel on the caller's stream, so it overlaps with attention running on
//    another stream, and pinned host memory is read or written directly over
//    the host link in 16-byte accesses.
#include "decode_common.h"
#include "kv_ops.h"
#include "neo_internal.h"

namespace neo {
namespace {

// One workgroup of 128 threads per (request, kv head): thread d writes dim d
// of the value row (a 2-byte store: V is dim-major, so the token's dims are
// 32 bytes apart), threads 0-15 also write one 16-byte key piece each.
// blk_stride: elements from one block of a cache to the next.
__global__ __launch_bounds__(128) void append_kernel(
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const int32_t* __restrict__ table, const int32_t* __restrict__ lens, int32_t mbps,
    int32_t hkv, int32_t num_blocks, int64_t blk_stride) {
  const int b = blockIdx.x / hkv, g = blockIdx.x % hkv;
  const int32_t L = clamp_len(lens[b], mbps);
  if (L <= 0) return;
  const int32_t t = L - 1;
  const int32_t blk = table[(size_t)b * mbps + t / kBlock];
  if (blk < 0 || blk >= num_blocks) return;
  const int slot = t % kBlock;
  const size_t tile = (size_t)blk * (size_t)blk_stride + (size_t)g * kTileElems;
  const size_t src = ((size_t)b * hkv + g) * kHeadDim;
  const int d = threadIdx.x;
  if (d < kHeadDim / kPiece) {
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(k_new + src + d * kPiece);
    *reinterpret_cast<u32x4_t*>(k_cache + tile + ((size_t)d * kBlock + slot) * kPiece) = v;
  }
  v_cache[tile + (size_t)d * kBlock + slot] = v_new[src + d];
}

// One workgroup per copied block: K and V, 16 bytes per access, four words of
// each cache loaded before any is stored so that reads over the host link
// keep eight requests in flight per thread. Every byte is touched once, so
// loads (and stores into device memory) are nontemporal: a block copy between
// two HBM caches measured 5.9 TB/s (read + write) against 5.3 with cached
// accesses.
template <bool kStreamStores>
__global__ __launch_bounds__(256) void copy_blocks_kernel(
    const uint16_t* __restrict__ src_k, const uint16_t* __restrict__ src_v,
    uint16_t* __restrict__ dst_k, uint16_t* __restrict__ dst_v,
    const int32_t* __restrict__ src_ids, const int32_t* __restrict__ dst_ids, int32_t hkv,
    int32_t src_blocks, int32_t dst_blocks, int64_t src_stride, int64_t dst_stride) {
  constexpr int kUnroll = 4;
  const int i = blockIdx.x;
  const int32_t s = src_ids[i], d = dst_ids[i];
  if (s < 0 || s >= src_blocks || d < 0 || d >= dst_blocks) return;
  // 16-byte words per block per cache: hkv * 256, a multiple of blockDim. The
  // block strides (elements) are multiples of 8, i.e. whole 16-byte words.
  const int words = hkv * (kTileElems / 8);
  const size_t so = (size_t)s * (size_t)(src_stride / 8), doff = (size_t)d * (size_t)(dst_stride / 8);
  const u32x4_t* sk = reinterpret_cast<const u32x4_t*>(src_k) + so;
  const u32x4_t* sv = reinterpret_cast<const u32x4_t*>(src_v) + so;
  u32x4_t* dk = reinterpret_cast<u32x4_t*>(dst_k) + doff;
  u32x4_t* dv = reinterpret_cast<u32x4_t*>(dst_v) + doff;
  for (int w0 = 0; w0 < words; w0 += kUnroll * 256) {
    // Rows of 256 words left in this step (fewer than kUnroll only at the end).
    const int rows = min(kUnroll, (words - w0) / 256);
    u32x4_t a[kUnroll], c[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (u < rows) {
        const int w = w0 + u * 256 + threadIdx.x;
        a[u] = __builtin_nontemporal_load(sk + w);
        c[u] = __builtin_nontemporal_load(sv + w);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (u < rows) {
        const int w = w0 + u * 256 + threadIdx.x;
        if (kStreamStores) {
          __builtin_nontemporal_store(a[u], dk + w);
          __builtin_nontemporal_store(c[u], dv + w);
        } else {
          dk[w] = a[u];
          dv[w] = c[u];
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_kv_append(uint16_t* k_cache, uint16_t* v_cache, const uint16_t* k_new,
                            const uint16_t* v_new, const int32_t* table, const int32_t* lens,
                            int32_t batch, int32_t mbps, int32_t hkv, int32_t num_blocks,
                            int64_t blk_stride, hipStream_t stream) {
  append_kernel<<<(unsigned)batch * hkv, kHeadDim, 0, stream>>>(
      k_cache, v_cache, k_new, v_new, table, lens, mbps, hkv, num_blocks, blk_stride);
  return hipGetLastError();
}

hipError_t launch_copy_blocks(const uint16_t* src_k, const uint16_t* src_v, uint16_t* dst_k,
                              uint16_t* dst_v, const int32_t* src_ids, const int32_t* dst_ids,
                              int32_t n, int32_t hkv, int32_t src_blocks, int32_t dst_blocks,
                              int64_t src_stride, int64_t dst_stride, bool dst_in_hbm,
                              hipStream_t stream) {
  if (dst_in_hbm)
    copy_blocks_kernel<true><<<n, 256, 0, stream>>>(src_k, src_v, dst_k, dst_v, src_ids, dst_ids,
                                                    hkv, src_blocks, dst_blocks, src_stride,
                                                    dst_stride);
  else
    copy_blocks_kernel<false><<<n, 256, 0, stream>>>(src_k, src_v, dst_k, dst_v, src_ids,
                                                     dst_ids, hkv, src_blocks, dst_blocks,
                                                     src_stride, dst_stride);
  return hipGetLastError();
}

// ----------------------------------------------------------------- read probe

namespace {

typedef uint32_t probe_u32x4 __attribute__((ext_vector_type(4)));

// Each thread reads words tid, tid + stride, ... with 8 loads in flight, xors
// them, and the wave's xor goes to sink: the loads cannot be dropped, and the
// result is checkable (the xor of all sink words is the xor of the buffer).
template <bool kNontemporal>
__global__ __launch_bounds__(256) void read_probe_kernel(const probe_u32x4* __restrict__ src,
                                                         size_t n16, uint32_t* __restrict__ sink) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  auto ld = [&](size_t i) -> probe_u32x4 {
    return kNontemporal ? __builtin_nontemporal_load(src + i) : src[i];
  };
  probe_u32x4 acc = {0u, 0u, 0u, 0u};
  size_t i = tid;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    probe_u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = ld(i + u * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u];
  }
  for (; i < n16; i += stride) acc ^= ld(i);
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x ^= __shfl_xor(x, o);
  if ((threadIdx.x & 63) == 0) sink[tid >> 6] = x;
}

// The decode kernel's access pattern without its arithmetic: one wave per
// contiguous range of 8 KiB steps (two 4 KiB tiles, each read through a buffer
// resource covering exactly that tile, 16-byte nontemporal loads, 1 KiB per
// instruction), kDepth steps in flight ahead of the one consumed; a step past
// the wave's range gets resources of size 0 (its loads return zeros without
// touching memory), so every step issues the same loads. Workgroups of four
// waves. The wave's xor goes to sink[wave]. xcd8: the ranges are cut by the
// decode kernel's slice geometry with its XCD weights (waves on even XCDs get
// 34 units, those on odd XCDs 30, where the geometry allows it), else equal.
template <int kDepth>
__global__ __launch_bounds__(256) void read_probe_tiles_kernel(const uint16_t* __restrict__ src,
                                                               int32_t nsteps, int32_t xcd8,
                                                               uint32_t* __restrict__ sink) {
  constexpr int kStepElems = 2 * kTileElems;  // 8 KiB of bf16
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t wave = (int32_t)blockIdx.x * kWavesPerGroup + uniform(threadIdx.x >> 6);
  const int32_t nw = (int32_t)gridDim.x * kWavesPerGroup;
  const SliceGeom geo = make_slice_geom(nsteps, nw, xcd8 != 0);
  const int64_t s0 = uniform(slice_start(wave, geo)), s1 = uniform(slice_start(wave + 1, geo));
  u32x4_t buf[kDepth + 1][8];
  auto issue = [&](u32x4_t(&b)[8], int64_t s) {
    const bool valid = s < s1;
    const uint16_t* base = src + (valid ? s : s0) * kStepElems;
    const __amdgpu_buffer_rsrc_t ra = tile_rsrc(base, valid);
    const __amdgpu_buffer_rsrc_t rb = tile_rsrc(base + kTileElems, valid);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      b[u] = tile_load16(ra, 16 * (kWave * u + lane));
      b[4 + u] = tile_load16(rb, 16 * (kWave * u + lane));
    }
  };
  u32x4_t acc = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < kDepth; ++i) issue(buf[i], s0 + i);
  for (int64_t s = s0; s < s1; s += kDepth + 1) {
#pragma unroll
    for (int u = 0; u <= kDepth; ++u) {
      const int64_t cur = s + u;
      if (cur >= s1) break;
      issue(buf[(u + kDepth) % (kDepth + 1)], cur + kDepth);
#pragma unroll
      for (int k = 0; k < 8; ++k) acc ^= buf[u][k];
    }
  }
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x ^= __shfl_xor(x, o);
  if (lane == 0) sink[wave] = x;
}

}  // namespace

hipError_t launch_read_probe_tiles(const void* src, int32_t nsteps, int32_t workgroups,
                                   int32_t depth, bool xcd8, uint32_t* sink, hipStream_t stream) {
  const uint16_t* s = static_cast<const uint16_t*>(src);
  const int32_t w = xcd8 ? 1 : 0;
  switch (depth) {
    case 1: read_probe_tiles_kernel<1><<<workgroups, 256, 0, stream>>>(s, nsteps, w, sink); break;
    case 2: read_probe_tiles_kernel<2><<<workgroups, 256, 0, stream>>>(s, nsteps, w, sink); break;
    case 3: read_probe_tiles_kernel<3><<<workgroups, 256, 0, stream>>>(s, nsteps, w, sink); break;
    default: read_probe_tiles_kernel<4><<<workgroups, 256, 0, stream>>>(s, nsteps, w, sink); break;
  }
  return hipGetLastError();
}

hipError_t launch_read_probe(const void* src, size_t n16, bool nontemporal, uint32_t* sink,
                             hipStream_t stream) {
  const probe_u32x4* s = static_cast<const probe_u32x4*>(src);
  if (nontemporal)
    read_probe_kernel<true><<<kReadProbeBlocks, 256, 0, stream>>>(s, n16, sink);
  else
    read_probe_kernel<false><<<kReadProbeBlocks, 256, 0, stream>>>(s, n16, sink);
  return hipGetLastError();
}

}  // namespace neo
