// Launchers of the cache operations (append, block copy) on either side of
// decode attention.
#pragma once

#include "neo_internal.h"

namespace neo {

hipError_t launch_kv_append(uint16_t* k_cache, uint16_t* v_cache, const uint16_t* k_new,
                            const uint16_t* v_new, const int32_t* table, const int32_t* lens,
                            int32_t batch, int32_t mbps, int32_t hkv, int32_t num_blocks,
                            int64_t blk_stride, hipStream_t stream);
// Block strides in elements, multiples of 8. dst_in_hbm: the destination
// caches are device memory (streaming stores pay there; into pinned host
// memory over the link they measured slightly slower).
hipError_t launch_copy_blocks(const uint16_t* src_k, const uint16_t* src_v, uint16_t* dst_k,
                              uint16_t* dst_v, const int32_t* src_ids, const int32_t* dst_ids,
                              int32_t n, int32_t hkv, int32_t src_blocks, int32_t dst_blocks,
                              int64_t src_stride, int64_t dst_stride, bool dst_in_hbm,
                              hipStream_t stream);

// Streaming-read probe: reads n16 16-byte words once; sink gets one word per
// wave (kReadProbeWaves of them), the xor of every 32-bit word that wave read.
constexpr int kReadProbeBlocks = 4096;
constexpr int kReadProbeWaves = kReadProbeBlocks * 4;
hipError_t launch_read_probe(const void* src, size_t n16, bool nontemporal, uint32_t* sink,
                             hipStream_t stream);
// Tile-pattern probe: nsteps 8 KiB steps split into contiguous per-wave
// ranges over `workgroups` 4-wave workgroups (equal, or weighted by XCD like
// the decode kernel's slices when xcd8), `depth` (1-4) steps in flight; sink
// gets one word per wave (workgroups * 4).
hipError_t launch_read_probe_tiles(const void* src, int32_t nsteps, int32_t workgroups,
                                   int32_t depth, bool xcd8, uint32_t* sink, hipStream_t stream);

}  // namespace neo
