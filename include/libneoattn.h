/*
 * libneoattn -- batched paged GQA decode attention on AMD Instinct MI355X (gfx950).
 *
 * The operation (Neo, arXiv 2411.01142, Sec. 2.1-2.2): in the decoding phase each
 * request contributes one new query token per query head, and that token attends
 * over every token in the request's KV cache. It is the only step that touches the
 * KV cache, needs no weights and is bound by memory bandwidth (Sec. 2.2, Sec. 4).
 * The cache is paged (fixed-size blocks reached through a per-request block table,
 * Sec. 2.1 and Sec. 4); query heads share KV heads in groups (GQA, Sec. 4). Work is
 * partitioned along each request's sequence at block granularity and the partial
 * outputs of a request are aggregated (Sec. 4, after Flash-Decoding); the GPU
 * attention runs once per iteration over the whole GPU batch (Sec. 3.1), so the
 * library takes the whole ragged batch in one call.
 *
 * For request b with L = seq_lens[b] cached tokens (the token being decoded
 * included), query head h and kv head g = h / (num_q_heads / num_kv_heads):
 *
 *   s_t          = scale * sum_d q[b][h][d] * K[b][g][t][d],        t in [0, L)
 *   out[b][h][d] = sum_t exp(s_t - max s) * V[b][g][t][d] / sum_t exp(s_t - max s)
 *
 * A request with L = 0 gets a zero row. The exp is natural (the kernels use exp2
 * with log2(e) folded into the scale).
 *
 * Storage contract (all device buffers, row-major, no padding):
 *   q           bf16  [batch][num_q_heads][head_dim]
 *   k_cache     bf16  [num_blocks][num_kv_heads][head_dim/8][block_size][8]
 *                     (key of token t, dims 8c..8c+7, at [blk][g][c][t % block_size][:])
 *   v_cache     bf16  [num_blocks][num_kv_heads][head_dim][block_size]
 *                     (value of token t, dim d, at [blk][g][d][t % block_size])
 *   block_table int32 [batch][max_blocks_per_seq]; token t of request b lives in
 *                     block block_table[b][t / block_size], slot t % block_size.
 *                     Entries at and past ceil(L/block_size) are never read.
 *   seq_lens    int32 [batch]
 *   out         fp32  [batch][num_q_heads][head_dim]; every element is written.
 * One (block, kv head) tile of K or of V is one contiguous 4 KiB run.
 * Block stride: the entry points with a block stride argument accept blocks
 * that are that many elements apart (the same in a K and V cache pair)
 * instead of num_kv_heads * head_dim * block_size; within a block the layout
 * is as above. With kv_block_stride = 2 * num_kv_heads * head_dim * block_size
 * and v_cache = k_cache + num_kv_heads * head_dim * block_size, both caches
 * live in one allocation [num_blocks][K, V][num_kv_heads][tile], each block's
 * K and V in one run of 2 * num_kv_heads * 4 KiB (interleaved caches). On
 * MI355X decode attention streams such caches 1-6 % faster than two separate
 * allocations: the HBM read rate depends on where a block's K and V tiles lie
 * relative to each other, and of the placements measured this one (without
 * padding) was the fastest.
 *
 * Supported: head_dim 128, block_size 16, num_q_heads / num_kv_heads in {1,2,4,8,16}.
 * q, k_cache, v_cache and out must be 16-byte aligned; the workspace 256-byte aligned.
 *
 * Ownership: the caller owns every buffer. The library keeps no pointer after a
 * call returns and allocates nothing on any path.
 * Asynchrony: calls enqueue kernels on `stream` (a hipStream_t; NULL = the null
 * stream) and return without synchronising. Device faults surface at the caller's
 * next synchronisation.
 * Errors: arguments are checked on the host before any HIP call; a non-OK status
 * sets a message readable with neo_last_error(). Launch failures return NEO_ERR_HIP.
 * Block ids outside [0, num_blocks) are clamped to a valid block (no fault, wrong
 * result); seq_lens above max_blocks_per_seq * block_size are clamped to it and
 * negative ones read as 0. neo_debug_validate() reports both.
 * State: the library keeps no state between calls apart from the thread-local
 * error text and a per-device cache of the compute-unit and XCD counts. The
 * caller's decode workspace does carry state from one call to the next: the
 * arrival counters of split requests, which every call leaves at zero. A new
 * workspace must therefore be zero-filled once before its first use
 * (neo_decode_workspace_init, or any fill that has completed on the stream of
 * the first call); a workspace that was never zeroed gives wrong merges, not
 * an error. Calls that may overlap on the device need distinct workspaces.
 */
#ifndef LIBNEOATTN_H
#define LIBNEOATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NEO_OK = 0,
  NEO_ERR_INVALID_ARG = 1, /* null pointer, negative size, num_q_heads % num_kv_heads != 0,
                              non-finite scale, misaligned buffer, size overflow */
  NEO_ERR_UNSUPPORTED = 2, /* head_dim != 128, block_size != 16, group not in {1,2,4,8,16},
                              unknown variant */
  NEO_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than neo_decode_workspace_bytes() */
  NEO_ERR_HIP = 4          /* a HIP call or kernel launch failed; detail in neo_last_error() */
} neo_status;

/* Kernel family for the decode step (neo_decode_attention_ex). */
typedef enum {
  NEO_VARIANT_AUTO = 0, /* the fastest measured on MI355X for the group size */
  NEO_VARIANT_VALU = 1, /* vector-ALU dot products with DPP row reductions */
  NEO_VARIANT_MFMA = 2  /* q.K and p.V on bf16 matrix cores, query group padded to 16 */
} neo_variant;

/* How the call is launched (neo_decode_attention_ex). */
typedef enum {
  NEO_SCHEDULE_AUTO = 0,       /* fused (equal or fastest on MI355X for every length mix tried) */
  NEO_SCHEDULE_FUSED = 1,      /* one kernel: each wavefront plans its own slice from seq_lens
                                  and the last slice to finish a split request merges it */
  NEO_SCHEDULE_STAGED = 2,     /* three kernels: plan, decode, log-sum-exp combine */
  NEO_SCHEDULE_TWO_KERNEL = 3  /* decode (planning in-wave, recording the plan), then combine */
} neo_schedule;

/* Largest number of sequence slices (one wavefront each) a call may use. */
#define NEO_MAX_SLICES 4096

/*
 * Bytes of device workspace neo_decode_attention needs: the work plan (slice
 * starts, per-request tile offsets) and room for two partial outputs per slice
 * (group * head_dim fp32 values plus group log-sum-exps each), and the arrival
 * counters of split requests. Depends only on host scalars, so it can be
 * allocated ahead of time. Sized for NEO_MAX_SLICES, so it depends on the
 * batch (one int32 per request plus a fixed part) and on the query group
 * (num_q_heads / num_kv_heads), never on the lengths or the pool size: the
 * arguments are (batch, num_q_heads, num_kv_heads, head_dim), and the value is
 * align256(16) + align256(32 * (NEO_MAX_SLICES + 1)) + align256(4 * NEO_MAX_SLICES)
 * + align256(4 * (batch + 1)) + align256(8 * NEO_MAX_SLICES * group)
 * + align256(8 * NEO_MAX_SLICES * group * head_dim) bytes.
 *
 * The workspace must be zero-filled once before its first use
 * (neo_decode_workspace_init or any fill); every call leaves its counters at
 * zero again. Calls that may overlap on the device need distinct workspaces.
 */
neo_status neo_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                      int32_t head_dim, size_t* bytes_out);

/* Zero-fill a workspace on `stream` with a fill kernel (no memset node, so it
 * may be captured in a HIP graph). Enqueued like any kernel: a decode call on
 * another stream must wait for it. workspace_bytes: the bytes to clear (the
 * whole workspace); the workspace must be 256-byte aligned. */
neo_status neo_decode_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/*
 * Decode attention of the whole ragged batch (the operation and layouts above).
 * The first eleven arguments follow the problem statement in that order; the rest
 * are what a device pointer cannot carry: batch size, block-table row stride
 * (max_blocks_per_seq), pool size (num_blocks), the workspace and the stream.
 * Enqueues one kernel: each wavefront plans its own slice of the batch from
 * seq_lens, streams its tiles, and the last slice to finish a request that
 * was split merges the partial outputs in the same kernel (the staged and
 * two-kernel launches of neo_decode_attention_ex add a plan and a combine
 * kernel). Reads q, k_cache, v_cache, block_table and seq_lens; writes out and
 * the workspace.
 * Workspace: at least neo_decode_workspace_bytes(batch, num_q_heads,
 * num_kv_heads, head_dim) bytes, 256-byte aligned, zero-filled before its
 * first use and then reused as is (each call leaves its arrival counters at
 * zero); NEO_ERR_WORKSPACE when it is NULL or too small.
 * Limits: batch * (max_blocks_per_seq + 3) * num_kv_heads below 2^31 and
 * max_blocks_per_seq * block_size below 2^31 (NEO_ERR_INVALID_ARG otherwise).
 * batch == 0 is a no-op (pointers may then be NULL).
 */
neo_status neo_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const int32_t* seq_lens,
                                int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                int32_t block_size, float scale, float* out, int32_t batch,
                                int32_t max_blocks_per_seq, int32_t num_blocks, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * As neo_decode_attention, with the kernel family (neo_variant), the launch
 * schedule (neo_schedule), the number of sequence slices and the caches' block
 * stride chosen by the caller. max_slices = 0 picks the library default; any
 * value in [1, NEO_MAX_SLICES] caps the number of slices the plan may cut
 * (1 = no request is ever split). kv_block_stride: elements from one block to
 * the next in k_cache and in v_cache (see "Block stride" above); 0 means
 * num_kv_heads * head_dim * block_size (dense caches); otherwise a multiple
 * of 8 of at least that and at most 2^40, with num_blocks blocks at that
 * stride spanning less than 2^62 bytes (NEO_ERR_INVALID_ARG). The caller's
 * caches must hold num_blocks blocks at that stride. The result is the same
 * operation for every choice, up to fp32 summation order, and bit for bit the
 * same for every block stride.
 */
neo_status neo_decode_attention_ex(const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   int32_t block_size, float scale, float* out, int32_t batch,
                                   int32_t max_blocks_per_seq, int32_t num_blocks,
                                   void* workspace, size_t workspace_bytes, int32_t variant,
                                   int32_t schedule, int32_t max_slices,
                                   int64_t kv_block_stride, void* stream);

/*
 * As neo_decode_attention_ex, also recording two caller-created HIP events
 * (hipEvent_t, may be NULL) on `stream` immediately before and after the decode
 * kernel, so the main kernel can be timed apart from the plan and combine
 * launches of the staged schedule. Meant for measurement.
 */
neo_status neo_decode_attention_events(const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* block_table, const int32_t* seq_lens,
                                       int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t head_dim, int32_t block_size, float scale,
                                       float* out, int32_t batch, int32_t max_blocks_per_seq,
                                       int32_t num_blocks, void* workspace,
                                       size_t workspace_bytes, int32_t variant,
                                       int32_t schedule, int32_t max_slices,
                                       int64_t kv_block_stride, void* decode_start_event,
                                       void* decode_end_event, void* stream);

/*
 * For callers that cannot allocate device memory or a workspace (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * neo_decode_attention without the workspace arguments, with the caches'
 * block stride as for neo_decode_attention_ex (0: dense). The same operation,
 * layouts, checks and clamping rules, and the same single fused kernel
 * (MFMA family, default slice policy capped at 1024 slices); for a given
 * input the result equals neo_decode_attention's up to fp32 summation order
 * (bit for bit on a part with at most 256 compute units).
 * Instead of a workspace it uses a file-scope device array of the library
 * (16.1 MiB per GPU, held until the process ends): the arrival counters and
 * partial outputs of requests split across workgroups, for up to 1024 slices
 * at any supported query group (a larger group would be refused with
 * NEO_ERR_WORKSPACE). Its address on each device is looked up on the first
 * call made with that device current, which also clears its counters on
 * `stream`; every call leaves them at zero again. It calls no hipMalloc or
 * hipFree and no allocating library routine. Every call on one GPU shares
 * that GPU's array: calls that may overlap on one GPU (different streams with
 * no ordering between them, or different host threads) race and give wrong
 * results; order them, or use neo_decode_attention with distinct workspaces.
 */
neo_status neo_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                        const int32_t* block_table, const int32_t* seq_lens,
                                        int32_t num_q_heads, int32_t num_kv_heads,
                                        int32_t head_dim, int32_t block_size, float scale,
                                        float* out, int32_t batch, int32_t max_blocks_per_seq,
                                        int32_t num_blocks, int64_t kv_block_stride,
                                        void* stream);

/*
 * Bit-exact dense copy of one paged cache through the block table (the paged
 * layout of Sec. 2.1 / Sec. 4). is_v = 0 reads the K layout, 1 the V layout.
 * token_offsets: device int32 [batch+1], exclusive prefix sum of seq_lens
 * (token_offsets[batch] = total). dst: device bf16 [total][num_kv_heads][head_dim],
 * row token_offsets[b] + t holding token t of request b. Same clamping rules as
 * neo_decode_attention; head_dim must be a multiple of 8. block_stride:
 * elements from one block of `cache` to the next, 0 for dense
 * (num_kv_heads * head_dim * block_size), else a multiple of 8 of at least
 * that and at most 2^40 (NEO_ERR_INVALID_ARG).
 */
neo_status neo_paged_gather(const void* cache, int32_t is_v, const int32_t* block_table,
                            const int32_t* seq_lens, const int32_t* token_offsets, int32_t batch,
                            int32_t max_blocks_per_seq, int32_t num_kv_heads, int32_t head_dim,
                            int32_t block_size, int32_t num_blocks, int64_t block_stride,
                            void* dst, void* stream);

/*
 * Append one token per request (the decoding phase reads and appends the KV
 * cache, Sec. 2.1). k_new, v_new: device bf16 [batch][num_kv_heads][head_dim],
 * the key and value rows of each request's newest token; they are written as
 * token seq_lens[b] - 1 of request b (seq_lens counts the new token): block
 * block_table[b][(L-1)/block_size], slot (L-1) % block_size, into the K and V
 * layouts above. Requests with L <= 0 are skipped; lengths past the table are
 * clamped to it; a block id outside [0, num_blocks) skips the write.
 * kv_block_stride: the caches' block stride as for neo_decode_attention_ex
 * (0: dense). head_dim 128, block_size 16. k_cache and k_new must be 16-byte
 * aligned.
 */
neo_status neo_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                         const int32_t* block_table, const int32_t* seq_lens, int32_t batch,
                         int32_t max_blocks_per_seq, int32_t num_kv_heads, int32_t head_dim,
                         int32_t block_size, int32_t num_blocks, int64_t kv_block_stride,
                         void* stream);

/*
 * Copy whole blocks (all kv heads, K and V) between two caches of the layout
 * above: for i < n, dst block dst_ids[i] <- src block src_ids[i]. This is the
 * swap of partial offloading (a request's KV lives wholly in the GPU cache or
 * wholly in the CPU cache) and of layer-wise swapping (each layer's KV of newly
 * prefilled requests moves as soon as it is computed), Sec. 3.1. Each cache
 * pointer may be device memory or pinned host memory the device can address
 * (hipHostMalloc); any other pointer (pageable host memory) is refused with
 * NEO_ERR_INVALID_ARG before launch. The copy is one kernel on `stream`, so it
 * overlaps with attention on another stream. src_ids, dst_ids: int32 [n], same
 * memory rules; pairs with an id out of range are skipped. Destination blocks
 * must be distinct and must not be read by the same call (no in-place chains).
 * src_block_stride, dst_block_stride: block strides of the source caches and
 * of the destination caches as for neo_decode_attention_ex (0: dense), so a
 * copy can go between an interleaved device cache and a dense host one.
 * head_dim 128, block_size 16; all four caches 16-byte aligned.
 */
neo_status neo_kv_copy_blocks(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                              const int32_t* src_ids, const int32_t* dst_ids, int32_t n,
                              int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                              int32_t src_num_blocks, int32_t dst_num_blocks,
                              int64_t src_block_stride, int64_t dst_block_stride, void* stream);

/*
 * Measurement aid, not part of attention: the device's streaming-read rate,
 * the practical ceiling for an HBM-bound kernel (the decode kernel reads its
 * KV once). Reads `bytes` of device memory at `src` once (16-byte loads,
 * 8 per thread in flight, nontemporal when `nontemporal` != 0) and writes
 * NEO_READ_PROBE_SINK_WORDS words to `sink` (device memory, caller-owned):
 * word w is the xor of every 32-bit word wave w read, so the xor of all of
 * them is the xor of the buffer. One kernel on `stream`; time it with events.
 * bytes: a positive multiple of 16; src 16-byte aligned.
 */
#define NEO_READ_PROBE_SINK_WORDS 16384
neo_status neo_read_probe(const void* src, size_t bytes, int32_t nontemporal, uint32_t* sink,
                          size_t sink_words, void* stream);

/*
 * Measurement aid, not part of attention: the read rate of the decode kernel's
 * own access pattern without its arithmetic. `bytes` (a positive multiple of
 * 8192, below 2^44) at `src` (device memory, 256-byte aligned) are cut into
 * 8 KiB steps (two 4 KiB tiles, like the K and V tiles of one block), the
 * steps into one contiguous range per wavefront; waves_per_cu (4, 8, 12 or 16)
 * wavefronts per compute unit in workgroups of four, each with `depth` (1-4)
 * steps in flight ahead of the one it consumes; 16-byte nontemporal buffer
 * loads. xcd_weighted = 1: on a part with eight XCDs the ranges are weighted
 * by XCD as the decode kernel weighs its slices (34 units for a wave on an
 * even-numbered XCD, 30 on an odd one, when the geometry allows it); 0: equal
 * ranges. Writes one word per wavefront (compute units * waves_per_cu words,
 * at most 4096 on MI355X) to `sink`: the xor of every 32-bit word that wave
 * read, so the xor of all of them is the xor of the buffer. One kernel on
 * `stream`.
 */
neo_status neo_read_probe_tiles(const void* src, size_t bytes, int32_t waves_per_cu,
                                int32_t depth, int32_t xcd_weighted, uint32_t* sink,
                                size_t sink_words, void* stream);

/*
 * Decode attention on the host CPU over a KV cache in host memory (the CPU
 * half of offloaded decoding, Sec. 4: PACPU). Same arguments, layouts, result
 * and clamping rules as neo_decode_attention, but every pointer is host
 * memory (pageable or pinned) and the call is synchronous: it returns when
 * `out` is written. Work is split at block granularity into equal shares for
 * `num_threads` threads (0: NEO_CPU_THREADS, else OMP_NUM_THREADS, else the
 * CPUs this process may run on); the partial outputs of a request split
 * between threads are aggregated by their log-sum-exps. Block ids in use are
 * checked against [0, num_blocks) before any is read (NEO_ERR_INVALID_ARG).
 * The library keeps one pool of worker threads and a host scratch buffer for
 * the process; concurrent calls are serialised.
 */
neo_status neo_cpu_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                                    const int32_t* block_table, const int32_t* seq_lens,
                                    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                    int32_t block_size, float scale, float* out, int32_t batch,
                                    int32_t max_blocks_per_seq, int32_t num_blocks,
                                    int32_t num_threads);

/* neo_kv_append for a cache in host memory, on the calling thread (the CPU
 * side of a CPU-request's decode step). Same arguments, layouts and rules,
 * with dense caches (no block stride argument); every pointer is host memory;
 * synchronous. */
neo_status neo_cpu_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                             const int32_t* block_table, const int32_t* seq_lens, int32_t batch,
                             int32_t max_blocks_per_seq, int32_t num_kv_heads, int32_t head_dim,
                             int32_t block_size, int32_t num_blocks);

/* Instruction-set paths of the CPU attention. */
typedef enum {
  NEO_CPU_ISA_AUTO = 0,        /* the best this CPU supports */
  NEO_CPU_ISA_GENERIC = 1,     /* portable scalar code */
  NEO_CPU_ISA_AVX512_BF16 = 2, /* AVX-512 with BF16 dot products (vdpbf16ps) */
  NEO_CPU_ISA_AVX512 = 3       /* AVX-512F, bf16 widened to fp32, fp32 FMAs */
} neo_cpu_isa;

/* neo_cpu_decode_attention with an explicit path; a path this CPU lacks is
 * NEO_ERR_UNSUPPORTED. */
neo_status neo_cpu_decode_attention_ex(const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* block_table, const int32_t* seq_lens,
                                       int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t head_dim, int32_t block_size, float scale,
                                       float* out, int32_t batch, int32_t max_blocks_per_seq,
                                       int32_t num_blocks, int32_t num_threads, int32_t isa);

/* The path NEO_CPU_ISA_AUTO takes on this CPU: the environment variable
 * NEO_CPU_ISA (generic, avx512, avx512_bf16) when this CPU has it, else
 * AVX512 on any AVX-512 CPU, else GENERIC. */
int32_t neo_cpu_best_isa(void);

/* Threads a call with num_threads = 0 uses. */
int32_t neo_cpu_default_threads(void);

/*
 * Host memory read probe: `num_threads` threads (0: as above) of the CPU
 * attention's pool each sum one contiguous share of `bytes` (a multiple of
 * 64) at `buf`, with the widest loads this CPU has; *checksum receives the
 * sum. Timing a call gives the read bandwidth the CPU attention competes
 * for (its roofline, and the CPU-side input of a cost model).
 */
neo_status neo_cpu_read_probe(const void* buf, size_t bytes, int32_t num_threads,
                              double* checksum);

/* ------------------------------------------------------------------------
 * Cost model and load-aware scheduler (Sec. 3.2), host only.
 *
 * Per-layer stage times are profiled offline and linearly interpolated:
 * GPU decode attention T_ga and CPU decode attention T_ca on a grid of
 * (requests in the sub-batch, their total context tokens), the linear stage
 * T_l (pre- plus post-projection) on a curve over the sub-batch's tokens.
 * Interpolation is bilinear inside the grid; outside it the edge cell's
 * plane (line, for a curve) is extended; an axis of one point is constant.
 * An empty sub-batch costs 0.
 * ---------------------------------------------------------------------- */
typedef struct {
  int32_t n_b, n_s;   /* axis lengths, >= 1 */
  const double* b;    /* [n_b] requests, strictly ascending */
  const double* s;    /* [n_s] total context tokens, strictly ascending */
  const double* t;    /* [n_b][n_s] seconds per layer */
} neo_cost_grid;

typedef struct {
  int32_t n;          /* >= 1 */
  const double* x;    /* [n] tokens, strictly ascending */
  const double* t;    /* [n] seconds per layer */
} neo_cost_curve;

/* Interpolated value of a grid at (b, s) / of a curve at x. */
neo_status neo_cost_eval_grid(const neo_cost_grid* grid, double b, double s, double* out);
neo_status neo_cost_eval_curve(const neo_cost_curve* curve, double x, double* out);

typedef enum { NEO_SCHED_POLICY_NEO = 0, NEO_SCHED_POLICY_GPU_ONLY = 1 } neo_sched_policy;
typedef enum { NEO_SCHED_GPU_ONLY = 0, NEO_SCHED_TWO_BATCH = 1 } neo_sched_mode;

typedef struct {
  int32_t num_layers;              /* L of the iteration-time model */
  int32_t block_size;              /* tokens per KV block */
  int64_t gpu_blocks;              /* GPU KV cache capacity, blocks */
  int64_t cpu_blocks;              /* CPU KV cache capacity, blocks (0: no offloading) */
  int64_t max_batch_tokens;        /* activation capacity: tokens of both sub-batches' linear stages */
  int64_t swap_in_reserve_blocks;  /* GPU blocks left free after a swap-in */
  neo_cost_grid t_ga, t_ca;        /* copied at creation */
  neo_cost_curve t_l;              /* copied at creation */
  int32_t policy;                  /* neo_sched_policy: NEO = the six steps; GPU_ONLY = steps 1-3 */
} neo_sched_config;

/* One iteration's decision. ids (if given) receives, in order, the request
 * ids of: prefills, GPU decodes, CPU decodes in batch-0, CPU decodes in
 * batch-1 (both only for TWO_BATCH), swap-outs, swap-ins. */
typedef struct {
  int32_t done;                    /* 1: no request left; nothing else is set */
  int32_t mode;                    /* neo_sched_mode chosen */
  int32_t n_prefill, n_prefill_to_cpu, n_gpu_decode, n_cpu_decode0, n_cpu_decode1;
  int32_t n_swap_out, n_swap_in;
  int64_t n_tokens;                /* tokens produced (one per scheduled request) */
  double t_iter;                   /* estimated time of the chosen schedule, s */
  double t_two_batch, t_gpu_only;  /* both estimates */
  double t_l0, t_l1, t_ga0, t_ca0, t_ca1;  /* per-layer stage estimates of the two-batch schedule */
  double now;                      /* simulated time after the iteration */
} neo_sched_iter;

typedef struct {
  double now;
  int64_t tokens, iterations, two_batch_iterations, finished;
  int64_t swapped_out, swapped_in, preempted;
  int64_t gpu_blocks_held, cpu_blocks_held, waiting, gpu_running, cpu_running;
} neo_sched_stats;

typedef struct neo_sched neo_sched;

/* A simulator of the load-aware scheduler: each neo_sched_step makes one
 * iteration's schedule in the six steps of Sec. 3.2 and advances every
 * scheduled request by one token, simulated time by the estimate. */
neo_status neo_sched_create(const neo_sched_config* cfg, neo_sched** out);
/* Requests enter the prefill wait queue at `arrival` (simulated seconds). */
neo_status neo_sched_add_request(neo_sched* s, int64_t id, int32_t prompt_len, int32_t output_len,
                                 double arrival);
neo_status neo_sched_step(neo_sched* s, neo_sched_iter* info, int64_t* ids, int64_t ids_capacity);
neo_status neo_sched_get_stats(const neo_sched* s, neo_sched_stats* out);
void neo_sched_destroy(neo_sched* s);

/*
 * Opt-in check of the indexing inputs: counts seq_lens outside
 * [0, max_blocks_per_seq * block_size] and block-table entries in use
 * (j < ceil(L / block_size)) outside [0, num_blocks). Adds the count to
 * *error_count (device int32, caller zeroes it first).
 */
neo_status neo_debug_validate(const int32_t* block_table, const int32_t* seq_lens, int32_t batch,
                              int32_t max_blocks_per_seq, int32_t block_size, int32_t num_blocks,
                              int32_t* error_count, void* stream);

/* Message of this thread's last non-OK status; valid until its next neo_* call. */
const char* neo_last_error(void);

/* Library version, "major.minor.patch". */
const char* neo_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBNEOATTN_H */
