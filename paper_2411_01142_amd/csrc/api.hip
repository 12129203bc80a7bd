// C ABI of libneoattn: argument checks (all on the host, before any HIP
// call), workspace sizing, and the launches: by default one fused decode
// kernel (plan, tiles and merges), or plan -> decode -> combine (staged) and
// decode -> combine (two-kernel); the allocation-free entry point and its
// static scratch; the cache operations and the read probes.
#include <math.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "neo_error.h"
#include "kv_ops.h"
#include "neo_internal.h"


namespace {

using neo::set_error;

neo_status ok() { return neo::clear_error(); }

bool aligned(const void* p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// Address the device uses for `p`: `p` itself for device or managed memory,
// the mapped device address for pinned host memory, NULL for anything else
// (pageable host memory, unknown pointers). Clears the error HIP records for
// an unknown pointer.
void* device_address(const void* p, bool* in_device_memory = nullptr) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  if (in_device_memory) *in_device_memory = a.type == hipMemoryTypeDevice;
  switch (a.type) {
    case hipMemoryTypeDevice:
    case hipMemoryTypeManaged:
      return const_cast<void*>(p);
    case hipMemoryTypeHost:
      // The mapped address of `p` itself, whether the runtime reports the
      // allocation's base or `p` (the offset from hostPointer is kept).
      if (!a.devicePointer) return nullptr;
      return static_cast<char*>(a.devicePointer) +
             (a.hostPointer ? static_cast<const char*>(p) - static_cast<const char*>(a.hostPointer)
                            : 0);
    default:
      return nullptr;
  }
}

bool supported_group(int32_t g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

// Compute units of the current device, cached per device ordinal. The default
// plan uses at most CUs x wavefronts per workgroup slices (one workgroup per
// CU).
constexpr int kMaxDevices = 64;
// Per device ordinal: compute units in the low 16 bits, XCDs above (0: not
// read yet).
std::atomic<int32_t> g_device_shape[kMaxDevices];

// Compute units and XCDs of the current device.
neo_status device_shape(int32_t* cus, int32_t* xcds) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev >= 0 && dev < kMaxDevices) {
    const int32_t cached = g_device_shape[dev].load(std::memory_order_relaxed);
    if (cached > 0) {
      *cus = cached & 0xFFFF;
      *xcds = cached >> 16;
      return NEO_OK;
    }
  }
  int v = 0, x = 0;
  e = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess || v <= 0 || v > 0xFFFF)
    return set_error(NEO_ERR_HIP, "hipDeviceGetAttribute(cu count): %s", hipGetErrorString(e));
  // An XCD count the runtime cannot give only turns the slice weights off.
  if (hipDeviceGetAttribute(&x, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || x < 1 ||
      x > 0x7FFF) {
    (void)hipGetLastError();
    x = 1;
  }
  if (dev >= 0 && dev < kMaxDevices)
    g_device_shape[dev].store(v | (x << 16), std::memory_order_relaxed);
  *cus = v;
  *xcds = x;
  return NEO_OK;
}

neo_status check_heads(int32_t hq, int32_t hkv, int32_t head_dim) {
  if (hq <= 0 || hkv <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "num_q_heads (%d) and num_kv_heads (%d) must be positive",
                     hq, hkv);
  if (hq % hkv != 0)
    return set_error(NEO_ERR_INVALID_ARG, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)",
                     hq, hkv);
  if (head_dim != neo::kHeadDim)
    return set_error(NEO_ERR_UNSUPPORTED, "head_dim %d unsupported (only %d)", head_dim,
                     neo::kHeadDim);
  if (!supported_group(hq / hkv))
    return set_error(NEO_ERR_UNSUPPORTED, "query group %d unsupported (1, 2, 4, 8 or 16)",
                     hq / hkv);
  return NEO_OK;
}

// A cache's block stride in elements: 0 stands for `dense` (num_kv_heads tiles,
// blocks back to back); otherwise a multiple of 8 (whole 16-byte words) of at
// least `dense` -- the stride may leave room after a block (the other cache's
// block, padding) but not less -- and at most 2^40, so that block id * stride
// stays far inside 64 bits. *resolved gets the stride to use.
neo_status check_block_stride(int64_t stride, int64_t dense, const char* name,
                              int64_t* resolved) {
  if (stride != 0 &&
      (stride < dense || stride % neo::kPiece != 0 || stride > ((int64_t)1 << 40)))
    return set_error(NEO_ERR_INVALID_ARG,
                     "%s %lld must be 0 or a multiple of %d of at least %lld elements "
                     "(and at most 2^40)",
                     name, (long long)stride, neo::kPiece, (long long)dense);
  *resolved = stride != 0 ? stride : dense;
  return NEO_OK;
}

// The caches' byte span (num_blocks blocks at `stride` elements) must stay far
// inside 64 bits, so that no block offset the kernels form can wrap.
neo_status check_span(int64_t stride, int32_t num_blocks, const char* name) {
  if (num_blocks > 0 && stride > (((int64_t)1 << 61) / num_blocks))
    return set_error(NEO_ERR_INVALID_ARG,
                     "%s: %d blocks at a stride of %lld elements span 2^62 bytes or more",
                     name, num_blocks, (long long)stride);
  return NEO_OK;
}

// Host-side checks of a decode call, shared by every decode entry point (no
// HIP call). *noop is set for an empty batch, which needs no pointer.
neo_status check_decode(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* block_table, const int32_t* seq_lens,
                        int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                        int32_t block_size, float scale, const float* out, int32_t batch,
                        int32_t max_blocks_per_seq, int32_t num_blocks, int32_t variant,
                        int32_t schedule, int32_t max_slices, int64_t kv_block_stride,
                        bool* noop) {
  *noop = false;
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  const neo_status st = check_heads(num_q_heads, num_kv_heads, head_dim);
  if (st != NEO_OK) return st;
  if (block_size != neo::kBlock)
    return set_error(NEO_ERR_UNSUPPORTED, "block_size %d unsupported (only %d)", block_size,
                     neo::kBlock);
  if (!isfinite(scale)) return set_error(NEO_ERR_INVALID_ARG, "scale is not finite");
  if (variant != NEO_VARIANT_AUTO && variant != NEO_VARIANT_VALU && variant != NEO_VARIANT_MFMA)
    return set_error(NEO_ERR_UNSUPPORTED, "unknown variant %d", variant);
  if (schedule != NEO_SCHEDULE_AUTO && schedule != NEO_SCHEDULE_FUSED &&
      schedule != NEO_SCHEDULE_STAGED && schedule != NEO_SCHEDULE_TWO_KERNEL)
    return set_error(NEO_ERR_UNSUPPORTED, "unknown schedule %d", schedule);
  if (max_slices < 0 || max_slices > NEO_MAX_SLICES)
    return set_error(NEO_ERR_INVALID_ARG, "max_slices %d outside [0, %d]", max_slices,
                     NEO_MAX_SLICES);
  int64_t resolved = 0;
  const neo_status sst = check_block_stride(kv_block_stride, (int64_t)num_kv_heads * neo::kTileElems,
                                            "kv_block_stride", &resolved);
  if (sst != NEO_OK) return sst;
  if (batch == 0) {
    *noop = true;
    return ok();
  }
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !out)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (max_blocks_per_seq <= 0 || num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG,
                     "max_blocks_per_seq (%d) and num_blocks (%d) must be positive",
                     max_blocks_per_seq, num_blocks);
  {
    const neo_status span = check_span(resolved, num_blocks, "kv_block_stride");
    if (span != NEO_OK) return span;
  }
  if ((int64_t)batch * (max_blocks_per_seq + neo::kPairCostLong) * num_kv_heads >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG,
                     "batch * (max_blocks_per_seq + %d) * num_kv_heads must stay below 2^31",
                     neo::kPairCostLong);
  if ((int64_t)max_blocks_per_seq * neo::kBlock >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq too large");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16))
    return set_error(NEO_ERR_INVALID_ARG, "q, k_cache, v_cache and out must be 16-byte aligned");
  if (!aligned(block_table, 4) || !aligned(seq_lens, 4))
    return set_error(NEO_ERR_INVALID_ARG, "block_table and seq_lens must be 4-byte aligned");
  return NEO_OK;
}

// ----------------------------------------------------------------- static scratch
//
// The allocation-free entry point keeps the fused kernel's cross-workgroup
// merge state in a file-scope device array instead of a caller workspace:
// the arrival counters of cut pairs (one int32 per slice) and two partial
// slots per slice (group rows of head_dim floats plus group log-sum-exps).
// It is sized for kScratchSlices slices at the largest supported group; the
// plan of that entry point uses at most kScratchSlices slices (one per wave
// of one 4-wave workgroup per CU on a 256-CU part). Every GPU the library
// runs on holds one copy until the process ends (16.1 MiB).
constexpr int32_t kScratchSlices = 1024;
constexpr int32_t kScratchMaxGroup = 16;
constexpr size_t kScratchCountersOff = 0;
constexpr size_t kScratchLseOff =
    kScratchCountersOff + ((sizeof(int32_t) * kScratchSlices + 255) & ~size_t(255));
constexpr size_t kScratchOOff =
    kScratchLseOff + ((sizeof(float) * 2 * kScratchSlices * kScratchMaxGroup + 255) & ~size_t(255));
constexpr size_t kScratchBytes =
    kScratchOOff + sizeof(float) * 2 * kScratchSlices * kScratchMaxGroup * neo::kHeadDim;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each device ordinal (the host-side name is
// only a stand-in, never a device address), looked up once per device with
// that device current; set-up also clears the arrival counters, which every
// call then leaves at zero.
std::mutex g_scratch_mutex;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

neo_status scratch_address(hipStream_t stream, char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(NEO_ERR_HIP, "device ordinal %d outside [0, %d)", dev, kMaxDevices);
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      void* ptr = nullptr;
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !ptr)
        return set_error(NEO_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      e = neo::launch_fill_zero(static_cast<char*>(ptr) + kScratchCountersOff,
                                sizeof(int32_t) * kScratchSlices, stream);
      if (e != hipSuccess)
        return set_error(NEO_ERR_HIP, "scratch counter fill: %s", hipGetErrorString(e));
      g_scratch_ptr[dev].store(ptr, std::memory_order_release);
      p = ptr;
    }
  }
  *out = static_cast<char*>(p);
  return NEO_OK;
}

}  // namespace

extern "C" {

const char* neo_version(void) { return "0.1.0"; }

neo_status neo_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                      int32_t head_dim, size_t* bytes_out) {
  if (!bytes_out) return set_error(NEO_ERR_INVALID_ARG, "bytes_out is NULL");
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  neo_status st = check_heads(num_q_heads, num_kv_heads, head_dim);
  if (st != NEO_OK) return st;
  *bytes_out = neo::workspace_layout(batch, num_q_heads / num_kv_heads).total;
  return ok();
}

neo_status neo_decode_attention_events(const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* block_table, const int32_t* seq_lens,
                                       int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t head_dim, int32_t block_size, float scale,
                                       float* out, int32_t batch, int32_t max_blocks_per_seq,
                                       int32_t num_blocks, void* workspace,
                                       size_t workspace_bytes, int32_t variant,
                                       int32_t schedule, int32_t max_slices,
                                       int64_t kv_block_stride, void* decode_start_event,
                                       void* decode_end_event, void* stream) {
  bool noop = false;
  neo_status st = check_decode(q, k_cache, v_cache, block_table, seq_lens, num_q_heads,
                               num_kv_heads, head_dim, block_size, scale, out, batch,
                               max_blocks_per_seq, num_blocks, variant, schedule, max_slices,
                               kv_block_stride, &noop);
  if (st != NEO_OK || noop) return st;
  const int32_t group = num_q_heads / num_kv_heads;
  const neo::WorkspaceLayout wl = neo::workspace_layout(batch, group);
  if (!workspace || workspace_bytes < wl.total)
    return set_error(NEO_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", wl.total,
                     workspace ? workspace_bytes : (size_t)0);
  if (!aligned(workspace, 256))
    return set_error(NEO_ERR_INVALID_ARG, "workspace must be 256-byte aligned");

  int32_t cus = 0, xcds = 0;
  st = device_shape(&cus, &xcds);
  if (st != NEO_OK) return st;
  const int32_t quantum = cus * neo::kWavesPerGroup;
  // Default: at most one slice per wave of one workgroup per CU (the policy
  // in slice_count), so the grid has no workgroups without a slice.
  const int32_t slices =
      max_slices == 0 ? std::min<int32_t>(quantum, NEO_MAX_SLICES) : max_slices;
  const int32_t min_tiles = max_slices == 0 ? 0 : 1;
  if (variant == NEO_VARIANT_AUTO) variant = NEO_VARIANT_MFMA;
  // Default: the fused kernel. Any launch costs ~4.6 us on MI355X, so the
  // combine launch of the two-kernel schedule (~6 us) outweighs the in-kernel
  // merges at the end of the fused one; measured equal or faster on every
  // length mix tried.
  const neo::Schedule sched = schedule == NEO_SCHEDULE_TWO_KERNEL ? neo::kTwoKernel
                              : schedule == NEO_SCHEDULE_STAGED   ? neo::kStaged
                                                                  : neo::kFused;

  char* ws = static_cast<char*>(workspace);
  neo::DecodeParams p;
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k_cache);
  p.v = static_cast<const uint16_t*>(v_cache);
  p.table = block_table;
  p.lens = seq_lens;
  p.out = out;
  p.hdr = reinterpret_cast<neo::PlanHeader*>(ws + wl.hdr);
  p.starts = reinterpret_cast<neo::SliceStart*>(ws + wl.starts);
  p.part_lse = reinterpret_cast<float*>(ws + wl.part_lse);
  p.part_o = reinterpret_cast<float*>(ws + wl.part_o);
  p.counters = reinterpret_cast<int32_t*>(ws + wl.counters);
  p.batch = batch;
  p.hq = num_q_heads;
  p.hkv = num_kv_heads;
  p.mbps = max_blocks_per_seq;
  p.num_blocks = num_blocks;
  p.max_slices = slices;
  p.min_tiles = min_tiles;
  p.slice_quantum = quantum;
  p.xcd8 = xcds == 8;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.blk_stride = kv_block_stride != 0 ? kv_block_stride : (int64_t)num_kv_heads * neo::kTileElems;

  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (sched == neo::kStaged) {
    e = neo::launch_plan(seq_lens, batch, num_kv_heads, max_blocks_per_seq, slices, min_tiles,
                         quantum, p.xcd8, reinterpret_cast<neo::PlanHeader*>(ws + wl.hdr),
                         reinterpret_cast<neo::SliceStart*>(ws + wl.starts),
                         reinterpret_cast<int32_t*>(ws + wl.prefix), s);
    if (e != hipSuccess) return set_error(NEO_ERR_HIP, "plan launch: %s", hipGetErrorString(e));
  }
  const int32_t grid = (slices + neo::kWavesPerGroup - 1) / neo::kWavesPerGroup;
  if (decode_start_event) {
    e = hipEventRecord(static_cast<hipEvent_t>(decode_start_event), s);
    if (e != hipSuccess) return set_error(NEO_ERR_HIP, "event record: %s", hipGetErrorString(e));
  }
  e = variant == NEO_VARIANT_VALU ? neo::launch_decode_valu(p, group, sched, grid, s)
                                  : neo::launch_decode_mfma(p, group, sched, grid, s);
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
  if (decode_end_event) {
    e = hipEventRecord(static_cast<hipEvent_t>(decode_end_event), s);
    if (e != hipSuccess) return set_error(NEO_ERR_HIP, "event record: %s", hipGetErrorString(e));
  }
  if (sched != neo::kFused) {
    e = neo::launch_combine(p, group, grid, s);
    if (e != hipSuccess) return set_error(NEO_ERR_HIP, "combine launch: %s", hipGetErrorString(e));
  }
  return ok();
}

neo_status neo_decode_attention_ex(const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   int32_t block_size, float scale, float* out, int32_t batch,
                                   int32_t max_blocks_per_seq, int32_t num_blocks,
                                   void* workspace, size_t workspace_bytes, int32_t variant,
                                   int32_t schedule, int32_t max_slices, int64_t kv_block_stride,
                                   void* stream) {
  return neo_decode_attention_events(q, k_cache, v_cache, block_table, seq_lens, num_q_heads,
                                     num_kv_heads, head_dim, block_size, scale, out, batch,
                                     max_blocks_per_seq, num_blocks, workspace, workspace_bytes,
                                     variant, schedule, max_slices, kv_block_stride, nullptr,
                                     nullptr, stream);
}

neo_status neo_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const int32_t* seq_lens,
                                int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                int32_t block_size, float scale, float* out, int32_t batch,
                                int32_t max_blocks_per_seq, int32_t num_blocks, void* workspace,
                                size_t workspace_bytes, void* stream) {
  return neo_decode_attention_events(q, k_cache, v_cache, block_table, seq_lens, num_q_heads,
                                     num_kv_heads, head_dim, block_size, scale, out, batch,
                                     max_blocks_per_seq, num_blocks, workspace, workspace_bytes,
                                     NEO_VARIANT_AUTO, NEO_SCHEDULE_AUTO, 0, 0, nullptr, nullptr,
                                     stream);
}

neo_status neo_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                        const int32_t* block_table, const int32_t* seq_lens,
                                        int32_t num_q_heads, int32_t num_kv_heads,
                                        int32_t head_dim, int32_t block_size, float scale,
                                        float* out, int32_t batch, int32_t max_blocks_per_seq,
                                        int32_t num_blocks, int64_t kv_block_stride,
                                        void* stream) {
  bool noop = false;
  neo_status st = check_decode(q, k_cache, v_cache, block_table, seq_lens, num_q_heads,
                               num_kv_heads, head_dim, block_size, scale, out, batch,
                               max_blocks_per_seq, num_blocks, NEO_VARIANT_AUTO,
                               NEO_SCHEDULE_AUTO, 0, kv_block_stride, &noop);
  if (st != NEO_OK || noop) return st;
  const int32_t group = num_q_heads / num_kv_heads;
  if (group > kScratchMaxGroup)
    return set_error(NEO_ERR_WORKSPACE, "query group %d exceeds the static scratch (at most %d)",
                     group, kScratchMaxGroup);
  int32_t cus = 0, xcds = 0;
  st = device_shape(&cus, &xcds);
  if (st != NEO_OK) return st;
  const int32_t quantum = cus * neo::kWavesPerGroup;
  // The default slice policy, capped at what the scratch holds.
  const int32_t slices = std::min<int32_t>(quantum, kScratchSlices);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = nullptr;
  st = scratch_address(s, &base);
  if (st != NEO_OK) return st;

  neo::DecodeParams p;
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k_cache);
  p.v = static_cast<const uint16_t*>(v_cache);
  p.table = block_table;
  p.lens = seq_lens;
  p.out = out;
  p.hdr = nullptr;     // plan records: staged and two-kernel launches only
  p.starts = nullptr;
  p.part_lse = reinterpret_cast<float*>(base + kScratchLseOff);
  p.part_o = reinterpret_cast<float*>(base + kScratchOOff);
  p.counters = reinterpret_cast<int32_t*>(base + kScratchCountersOff);
  p.batch = batch;
  p.hq = num_q_heads;
  p.hkv = num_kv_heads;
  p.mbps = max_blocks_per_seq;
  p.num_blocks = num_blocks;
  p.max_slices = slices;
  p.min_tiles = 0;
  p.slice_quantum = quantum;
  p.xcd8 = xcds == 8;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.blk_stride = kv_block_stride != 0 ? kv_block_stride : (int64_t)num_kv_heads * neo::kTileElems;
  const int32_t grid = (slices + neo::kWavesPerGroup - 1) / neo::kWavesPerGroup;
  const hipError_t e = neo::launch_decode_mfma(p, group, neo::kFused, grid, s);
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
  return ok();
}

neo_status neo_decode_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace) return set_error(NEO_ERR_INVALID_ARG, "workspace is NULL");
  if (!aligned(workspace, 256))
    return set_error(NEO_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  hipError_t e = neo::launch_fill_zero(workspace, workspace_bytes & ~(size_t)3,
                                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "fill launch: %s", hipGetErrorString(e));
  return ok();
}

neo_status neo_paged_gather(const void* cache, int32_t is_v, const int32_t* block_table,
                            const int32_t* seq_lens, const int32_t* token_offsets, int32_t batch,
                            int32_t max_blocks_per_seq, int32_t num_kv_heads, int32_t head_dim,
                            int32_t block_size, int32_t num_blocks, int64_t block_stride,
                            void* dst, void* stream) {
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  if (is_v != 0 && is_v != 1) return set_error(NEO_ERR_INVALID_ARG, "is_v must be 0 or 1");
  if (num_kv_heads <= 0 || head_dim <= 0 || head_dim % neo::kPiece != 0 || block_size <= 0 ||
      (int64_t)num_kv_heads * head_dim * block_size >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "bad shape (num_kv_heads %d, head_dim %d, block_size %d)",
                     num_kv_heads, head_dim, block_size);
  int64_t stride = 0;
  const neo_status sst = check_block_stride(
      block_stride, (int64_t)num_kv_heads * head_dim * block_size, "block_stride", &stride);
  if (sst != NEO_OK) return sst;
  if (batch == 0) return ok();
  if (!cache || !block_table || !seq_lens || !token_offsets || !dst)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (max_blocks_per_seq <= 0 || num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq and num_blocks must be positive");
  {
    const neo_status span = check_span(stride, num_blocks, "block_stride");
    if (span != NEO_OK) return span;
  }
  if (batch > 65535) return set_error(NEO_ERR_INVALID_ARG, "batch above 65535");
  if ((int64_t)max_blocks_per_seq * block_size >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq too large");
  hipError_t e = neo::launch_gather(static_cast<const uint16_t*>(cache), is_v, block_table,
                                    seq_lens, token_offsets, batch, max_blocks_per_seq,
                                    num_kv_heads, head_dim, block_size, num_blocks, stride,
                                    static_cast<uint16_t*>(dst), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "gather launch: %s", hipGetErrorString(e));
  return ok();
}

neo_status neo_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                         const int32_t* block_table, const int32_t* seq_lens, int32_t batch,
                         int32_t max_blocks_per_seq, int32_t num_kv_heads, int32_t head_dim,
                         int32_t block_size, int32_t num_blocks, int64_t kv_block_stride,
                         void* stream) {
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  if (num_kv_heads <= 0) return set_error(NEO_ERR_INVALID_ARG, "num_kv_heads must be positive");
  if (head_dim != neo::kHeadDim || block_size != neo::kBlock)
    return set_error(NEO_ERR_UNSUPPORTED, "head_dim %d / block_size %d unsupported (128 / 16)",
                     head_dim, block_size);
  int64_t stride = 0;
  const neo_status sst = check_block_stride(
      kv_block_stride, (int64_t)num_kv_heads * neo::kTileElems, "kv_block_stride", &stride);
  if (sst != NEO_OK) return sst;
  if (batch == 0) return ok();
  if (!k_cache || !v_cache || !k_new || !v_new || !block_table || !seq_lens)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (max_blocks_per_seq <= 0 || num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq and num_blocks must be positive");
  {
    const neo_status span = check_span(stride, num_blocks, "kv_block_stride");
    if (span != NEO_OK) return span;
  }
  if ((int64_t)max_blocks_per_seq * neo::kBlock >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq too large");
  if ((int64_t)batch * num_kv_heads >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "batch * num_kv_heads must be below 2^31");
  if (!aligned(k_cache, 16) || !aligned(k_new, 16) || !aligned(v_cache, 2) || !aligned(v_new, 2))
    return set_error(NEO_ERR_INVALID_ARG, "k_cache and k_new must be 16-byte aligned");
  hipError_t e = neo::launch_kv_append(
      static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache),
      static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), block_table,
      seq_lens, batch, max_blocks_per_seq, num_kv_heads, num_blocks, stride,
      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "append launch: %s", hipGetErrorString(e));
  return ok();
}

neo_status neo_kv_copy_blocks(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                              const int32_t* src_ids, const int32_t* dst_ids, int32_t n,
                              int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                              int32_t src_num_blocks, int32_t dst_num_blocks,
                              int64_t src_block_stride, int64_t dst_block_stride, void* stream) {
  if (n < 0) return set_error(NEO_ERR_INVALID_ARG, "n (%d) is negative", n);
  if (num_kv_heads <= 0) return set_error(NEO_ERR_INVALID_ARG, "num_kv_heads must be positive");
  if (head_dim != neo::kHeadDim || block_size != neo::kBlock)
    return set_error(NEO_ERR_UNSUPPORTED, "head_dim %d / block_size %d unsupported (128 / 16)",
                     head_dim, block_size);
  const int64_t dense = (int64_t)num_kv_heads * neo::kTileElems;
  int64_t src_stride = 0, dst_stride = 0;
  neo_status sst = check_block_stride(src_block_stride, dense, "src_block_stride", &src_stride);
  if (sst != NEO_OK) return sst;
  sst = check_block_stride(dst_block_stride, dense, "dst_block_stride", &dst_stride);
  if (sst != NEO_OK) return sst;
  if (n == 0) return ok();
  if (!src_k || !src_v || !dst_k || !dst_v || !src_ids || !dst_ids)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (src_num_blocks <= 0 || dst_num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "block counts must be positive");
  sst = check_span(src_stride, src_num_blocks, "src_block_stride");
  if (sst != NEO_OK) return sst;
  sst = check_span(dst_stride, dst_num_blocks, "dst_block_stride");
  if (sst != NEO_OK) return sst;
  if (!aligned(src_k, 16) || !aligned(src_v, 16) || !aligned(dst_k, 16) || !aligned(dst_v, 16))
    return set_error(NEO_ERR_INVALID_ARG, "caches must be 16-byte aligned");
  // Every pointer the kernel dereferences must be device memory or pinned host
  // memory; pageable host memory would fault the kernel, so it is refused here.
  const void* ptrs[6] = {src_k, src_v, dst_k, dst_v, src_ids, dst_ids};
  void* dev[6];
  bool in_hbm[6];
  static const char* names[6] = {"src_k", "src_v", "dst_k", "dst_v", "src_ids", "dst_ids"};
  for (int i = 0; i < 6; ++i) {
    dev[i] = device_address(ptrs[i], &in_hbm[i]);
    if (!dev[i])
      return set_error(NEO_ERR_INVALID_ARG,
                       "%s is not device memory or pinned host memory the device can address",
                       names[i]);
  }
  hipError_t e = neo::launch_copy_blocks(
      static_cast<const uint16_t*>(dev[0]), static_cast<const uint16_t*>(dev[1]),
      static_cast<uint16_t*>(dev[2]), static_cast<uint16_t*>(dev[3]),
      static_cast<const int32_t*>(dev[4]), static_cast<const int32_t*>(dev[5]), n, num_kv_heads,
      src_num_blocks, dst_num_blocks, src_stride, dst_stride, in_hbm[2] && in_hbm[3],
      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "copy launch: %s", hipGetErrorString(e));
  return ok();
}

static_assert(neo::kReadProbeWaves == NEO_READ_PROBE_SINK_WORDS, "probe sink size");

neo_status neo_read_probe(const void* src, size_t bytes, int32_t nontemporal, uint32_t* sink,
                          size_t sink_words, void* stream) {
  if (!src || !sink) return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (bytes == 0 || bytes % 16 != 0)
    return set_error(NEO_ERR_INVALID_ARG, "bytes (%zu) must be a positive multiple of 16", bytes);
  if (!aligned(src, 16)) return set_error(NEO_ERR_INVALID_ARG, "src must be 16-byte aligned");
  if (sink_words < (size_t)NEO_READ_PROBE_SINK_WORDS)
    return set_error(NEO_ERR_INVALID_ARG, "sink holds %zu words, needs %d", sink_words,
                     NEO_READ_PROBE_SINK_WORDS);
  const hipError_t e = neo::launch_read_probe(src, bytes / 16, nontemporal != 0, sink,
                                              static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "probe launch: %s", hipGetErrorString(e));
  return ok();
}

neo_status neo_read_probe_tiles(const void* src, size_t bytes, int32_t waves_per_cu,
                                int32_t depth, int32_t xcd_weighted, uint32_t* sink,
                                size_t sink_words, void* stream) {
  if (!src || !sink) return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (bytes == 0 || bytes % 8192 != 0 || bytes / 8192 >= ((size_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG,
                     "bytes (%zu) must be a positive multiple of 8192 below 2^44", bytes);
  if (xcd_weighted != 0 && xcd_weighted != 1)
    return set_error(NEO_ERR_INVALID_ARG, "xcd_weighted must be 0 or 1");
  if (!aligned(src, 256)) return set_error(NEO_ERR_INVALID_ARG, "src must be 256-byte aligned");
  if (waves_per_cu < 4 || waves_per_cu > 16 || waves_per_cu % 4 != 0)
    return set_error(NEO_ERR_INVALID_ARG, "waves_per_cu %d must be 4, 8, 12 or 16",
                     waves_per_cu);
  if (depth < 1 || depth > 4)
    return set_error(NEO_ERR_INVALID_ARG, "depth %d outside [1, 4]", depth);
  int32_t cus = 0, xcds = 0;
  neo_status st = device_shape(&cus, &xcds);
  if (st != NEO_OK) return st;
  const size_t waves = (size_t)cus * waves_per_cu;
  if (sink_words < waves)
    return set_error(NEO_ERR_INVALID_ARG, "sink holds %zu words, needs %zu", sink_words, waves);
  const hipError_t e =
      neo::launch_read_probe_tiles(src, (int32_t)(bytes / 8192),
                                   (int32_t)(waves / neo::kWavesPerGroup), depth,
                                   xcd_weighted != 0 && xcds == 8, sink,
                                   static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "probe launch: %s", hipGetErrorString(e));
  return ok();
}

neo_status neo_debug_validate(const int32_t* block_table, const int32_t* seq_lens, int32_t batch,
                              int32_t max_blocks_per_seq, int32_t block_size, int32_t num_blocks,
                              int32_t* error_count, void* stream) {
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  if (batch == 0) return ok();
  if (!block_table || !seq_lens || !error_count)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (max_blocks_per_seq <= 0 || block_size <= 0 || num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "sizes must be positive");
  if ((int64_t)max_blocks_per_seq * block_size >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq too large");
  hipError_t e = neo::launch_validate(block_table, seq_lens, batch, max_blocks_per_seq,
                                      block_size, num_blocks, error_count,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return set_error(NEO_ERR_HIP, "validate launch: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
