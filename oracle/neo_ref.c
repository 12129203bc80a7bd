/*
 * neo_ref.c -- fp64 CPU oracle for batched paged GQA decode attention.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, obviously-correct reference
 * that the HIP path is checked against. It shares no source, header, table or
 * helper with the HIP library; only tests, the package's smoke check and the
 * benchmark's CPU-baseline leg may load it.
 *
 * What it computes (the paper, Sec. 2.1-2.2 and Sec. 4): in the decoding
 * phase each request's single new query token attends over all tokens in that
 * request's KV cache, which is stored in fixed-size blocks addressed through a
 * per-request block table (paged attention); query heads share KV heads in
 * groups (GQA). The method's block-granular split with per-request
 * aggregation (Sec. 4, "Efficient CPU Kernels") reaches exactly standard
 * scaled-dot-product attention, so the oracle is that definition written out:
 *
 *   s_t = scale * sum_d q[b][h][d] * K[b][g][t][d]     g = h / (Hq/Hkv)
 *   w_t = exp(s_t - max_t s_t),  Z = sum_t w_t
 *   out[b][h][d] = (sum_t w_t * V[b][g][t][d]) / Z
 *
 * Everything is accumulated in double; bf16 inputs widen exactly; the result
 * is rounded once to float (round to nearest even). A request with zero
 * tokens yields a zero row. Sums run over ascending t and ascending d.
 *
 * Storage contract (same meaning as the library's, written independently):
 *   k_cache  [num_blocks][num_kv_heads][head_dim/8][block_size][8]
 *   v_cache  [num_blocks][num_kv_heads][head_dim][block_size]
 *   token t of request b: block block_table[b*mbps + t/block_size], slot t%block_size
 *
 * The split/merge functions restate the Flash-Decoding style partition and
 * aggregation of Sec. 4: attention over one block-aligned slice of a request
 * gives a normalised partial output and its log-sum-exp; partials merge by
 * weighting each with exp(lse_i - max lse).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { REF_OK = 0, REF_BAD_ARG = -1, REF_BAD_BLOCK = -2, REF_NOMEM = -3 };

static double bf16_bits_to_double(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

typedef struct {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* table;
  int32_t hkv, d, bs, mbps, nblocks;
} ref_cache;

/* Physical block holding token t of request b, or -1 if the table entry is out of range. */
static int64_t ref_block(const ref_cache* c, int64_t b, int64_t t) {
  int64_t j = t / c->bs;
  if (j >= c->mbps) return -1;
  int64_t p = c->table[b * c->mbps + j];
  if (p < 0 || p >= c->nblocks) return -1;
  return p;
}

static double ref_k(const ref_cache* c, int64_t p, int64_t g, int64_t slot, int64_t d) {
  int64_t idx = (((p * c->hkv + g) * (c->d / 8) + d / 8) * c->bs + slot) * 8 + d % 8;
  return bf16_bits_to_double(c->k[idx]);
}

static double ref_v(const ref_cache* c, int64_t p, int64_t g, int64_t slot, int64_t d) {
  int64_t idx = ((p * c->hkv + g) * c->d + d) * c->bs + slot;
  return bf16_bits_to_double(c->v[idx]);
}

/* Scores s_t (t in [t0,t1)) of query row qrow against kv head g of request b. */
static int ref_scores(const ref_cache* c, const uint16_t* qrow, int64_t b, int64_t g, double scale,
                      int64_t t0, int64_t t1, double* s) {
  for (int64_t t = t0; t < t1; ++t) {
    int64_t p = ref_block(c, b, t);
    if (p < 0) return REF_BAD_BLOCK;
    double dot = 0.0;
    for (int64_t d = 0; d < c->d; ++d)
      dot += bf16_bits_to_double(qrow[d]) * ref_k(c, p, g, t % c->bs, d);
    s[t - t0] = scale * dot;
  }
  return REF_OK;
}

/* Attention of one query row over tokens [t0,t1): normalised output o[D] and lse = M + ln Z. */
static int ref_attend(const ref_cache* c, const uint16_t* qrow, int64_t b, int64_t g, double scale,
                      int64_t t0, int64_t t1, double* s, double* o, double* lse) {
  int64_t n = t1 - t0;
  for (int64_t d = 0; d < c->d; ++d) o[d] = 0.0;
  if (n <= 0) {
    if (lse) *lse = -INFINITY;
    return REF_OK;
  }
  int rc = ref_scores(c, qrow, b, g, scale, t0, t1, s);
  if (rc) return rc;
  double m = -INFINITY;
  for (int64_t i = 0; i < n; ++i) m = s[i] > m ? s[i] : m;
  double z = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    s[i] = exp(s[i] - m);
    z += s[i];
  }
  for (int64_t i = 0; i < n; ++i) {
    int64_t t = t0 + i;
    int64_t p = ref_block(c, b, t);
    for (int64_t d = 0; d < c->d; ++d) o[d] += s[i] * ref_v(c, p, g, t % c->bs, d);
  }
  for (int64_t d = 0; d < c->d; ++d) o[d] /= z;
  if (lse) *lse = m + log(z);
  return REF_OK;
}

static int ref_check_shape(int32_t hq, int32_t hkv, int32_t d, int32_t bs, int32_t batch,
                           int32_t mbps, int32_t nblocks) {
  if (hq <= 0 || hkv <= 0 || hq % hkv != 0 || d <= 0 || d % 8 != 0 || bs <= 0 || batch < 0 ||
      mbps <= 0 || nblocks <= 0)
    return REF_BAD_ARG;
  return REF_OK;
}

/*
 * Full decode attention. out: float [batch][hq][d] (may be NULL); out64: double,
 * same shape (may be NULL). Rows [row_begin, row_end) of the flattened
 * (request, q head) index are computed (pass 0, batch*hq for all).
 * num_threads <= 0 means the OpenMP default. Returns 0, or a negative code.
 */
int neo_ref_decode_attention(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                             const int32_t* block_table, const int32_t* seq_lens,
                             int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                             int32_t block_size, double scale, float* out, double* out64,
                             int32_t batch, int32_t max_blocks_per_seq, int32_t num_blocks,
                             int64_t row_begin, int64_t row_end, int32_t num_threads) {
  int rc = ref_check_shape(num_q_heads, num_kv_heads, head_dim, block_size, batch,
                           max_blocks_per_seq, num_blocks);
  if (rc) return rc;
  ref_cache c = {k_cache, v_cache, block_table, num_kv_heads, head_dim, block_size,
                 max_blocks_per_seq, num_blocks};
  int64_t group = num_q_heads / num_kv_heads;
  int64_t maxlen = 0;
  for (int32_t b = 0; b < batch; ++b) maxlen = seq_lens[b] > maxlen ? seq_lens[b] : maxlen;
  if (maxlen > (int64_t)max_blocks_per_seq * block_size) return REF_BAD_ARG;
  if (row_end > (int64_t)batch * num_q_heads) row_end = (int64_t)batch * num_q_heads;
  int err = REF_OK;
#ifdef _OPENMP
  if (num_threads > 0) omp_set_num_threads(num_threads);
#endif
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * (size_t)(maxlen > 0 ? maxlen : 1));
    double* o = (double*)malloc(sizeof(double) * (size_t)head_dim);
    int ok = (s != NULL && o != NULL);
    if (!ok) {
#pragma omp atomic write
      err = REF_NOMEM;
    }
#pragma omp for schedule(static)
    for (int64_t row = row_begin; row < row_end; ++row) {
      if (!ok) continue;
      int64_t b = row / num_q_heads, h = row % num_q_heads;
      int64_t g = h / group;
      int64_t L = seq_lens[b] > 0 ? seq_lens[b] : 0;
      int r = ref_attend(&c, q + row * head_dim, b, g, scale, 0, L, s, o, NULL);
      if (r) {
#pragma omp atomic write
        err = r;
      }
      for (int64_t d = 0; d < head_dim; ++d) {
        if (out) out[row * head_dim + d] = (float)o[d];
        if (out64) out64[row * head_dim + d] = o[d];
      }
    }
    free(s);
    free(o);
  }
  return err;
}

/* Softmax weights w_t / Z (t in [0, L)) of one (request, q head); w must hold L doubles. */
int neo_ref_softmax_weights(const uint16_t* q, const uint16_t* k_cache, const int32_t* block_table,
                            const int32_t* seq_lens, int32_t num_q_heads, int32_t num_kv_heads,
                            int32_t head_dim, int32_t block_size, double scale, int32_t batch,
                            int32_t max_blocks_per_seq, int32_t num_blocks, int32_t b, int32_t h,
                            double* w) {
  int rc = ref_check_shape(num_q_heads, num_kv_heads, head_dim, block_size, batch,
                           max_blocks_per_seq, num_blocks);
  if (rc) return rc;
  if (b < 0 || b >= batch || h < 0 || h >= num_q_heads) return REF_BAD_ARG;
  ref_cache c = {k_cache, NULL, block_table, num_kv_heads, head_dim, block_size,
                 max_blocks_per_seq, num_blocks};
  int64_t L = seq_lens[b] > 0 ? seq_lens[b] : 0;
  if (L == 0) return REF_OK;
  int64_t g = h / (num_q_heads / num_kv_heads);
  rc = ref_scores(&c, q + ((int64_t)b * num_q_heads + h) * head_dim, b, g, scale, 0, L, w);
  if (rc) return rc;
  double m = -INFINITY, z = 0.0;
  for (int64_t t = 0; t < L; ++t) m = w[t] > m ? w[t] : m;
  for (int64_t t = 0; t < L; ++t) {
    w[t] = exp(w[t] - m);
    z += w[t];
  }
  for (int64_t t = 0; t < L; ++t) w[t] /= z;
  return REF_OK;
}

/*
 * Partial attention of one (request, q head) over tokens [t0, t1): o[D] is the
 * output normalised over the slice, *lse = max_t s_t + ln(sum_t exp(s_t - max)).
 * An empty slice gives o = 0 and lse = -inf.
 */
int neo_ref_partial_attention(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                              const int32_t* block_table, int32_t num_q_heads,
                              int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                              double scale, int32_t batch, int32_t max_blocks_per_seq,
                              int32_t num_blocks, int32_t b, int32_t h, int64_t t0, int64_t t1,
                              double* o, double* lse) {
  int rc = ref_check_shape(num_q_heads, num_kv_heads, head_dim, block_size, batch,
                           max_blocks_per_seq, num_blocks);
  if (rc) return rc;
  if (b < 0 || b >= batch || h < 0 || h >= num_q_heads || t0 < 0 || t1 < t0) return REF_BAD_ARG;
  ref_cache c = {k_cache, v_cache, block_table, num_kv_heads, head_dim, block_size,
                 max_blocks_per_seq, num_blocks};
  double* s = (double*)malloc(sizeof(double) * (size_t)(t1 > t0 ? t1 - t0 : 1));
  if (!s) return REF_NOMEM;
  int64_t g = h / (num_q_heads / num_kv_heads);
  rc = ref_attend(&c, q + ((int64_t)b * num_q_heads + h) * head_dim, b, g, scale, t0, t1, s, o,
                  lse);
  free(s);
  return rc;
}

/*
 * Aggregation of n partial outputs of one request row: M = max_i lse_i,
 * w_i = exp(lse_i - M), out = sum_i w_i o_i / sum_i w_i. o is [n][d].
 * Partials with lse = -inf carry no weight; if all are -inf the result is 0.
 */
int neo_ref_lse_merge(int32_t n, int32_t d, const double* o, const double* lse, double* out,
                      double* lse_out) {
  if (n < 0 || d <= 0) return REF_BAD_ARG;
  double m = -INFINITY;
  for (int32_t i = 0; i < n; ++i) m = lse[i] > m ? lse[i] : m;
  for (int32_t k = 0; k < d; ++k) out[k] = 0.0;
  if (m == -INFINITY) {
    if (lse_out) *lse_out = -INFINITY;
    return REF_OK;
  }
  double z = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    double w = exp(lse[i] - m);
    z += w;
    for (int32_t k = 0; k < d; ++k) out[k] += w * o[(int64_t)i * d + k];
  }
  for (int32_t k = 0; k < d; ++k) out[k] /= z;
  if (lse_out) *lse_out = m + log(z);
  return REF_OK;
}

/*
 * Dense copy of one cache through the block table: dst [sum_b L_b][num_kv_heads][head_dim]
 * (bf16 bits), requests in order, tokens ascending. is_v selects the V storage
 * layout, else the K layout. Returns the number of rows written, or a negative code.
 */
int64_t neo_ref_paged_gather(const uint16_t* cache, int32_t is_v, const int32_t* block_table,
                             const int32_t* seq_lens, int32_t batch, int32_t max_blocks_per_seq,
                             int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                             int32_t num_blocks, uint16_t* dst) {
  if (ref_check_shape(num_kv_heads, num_kv_heads, head_dim, block_size, batch, max_blocks_per_seq,
                      num_blocks))
    return REF_BAD_ARG;
  ref_cache c = {is_v ? NULL : cache, is_v ? cache : NULL, block_table, num_kv_heads, head_dim,
                 block_size, max_blocks_per_seq, num_blocks};
  int64_t row = 0;
  for (int64_t b = 0; b < batch; ++b) {
    int64_t L = seq_lens[b] > 0 ? seq_lens[b] : 0;
    for (int64_t t = 0; t < L; ++t, ++row) {
      int64_t p = ref_block(&c, b, t);
      if (p < 0) return REF_BAD_BLOCK;
      for (int64_t g = 0; g < num_kv_heads; ++g) {
        for (int64_t d = 0; d < head_dim; ++d) {
          int64_t idx = is_v ? ((p * num_kv_heads + g) * head_dim + d) * block_size + t % block_size
                             : (((p * num_kv_heads + g) * (head_dim / 8) + d / 8) * block_size +
                                t % block_size) * 8 + d % 8;
          dst[(row * num_kv_heads + g) * head_dim + d] = cache[idx];
        }
      }
    }
  }
  return row;
}

int neo_ref_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/*
 * Append (the decoding phase reads and appends the KV cache, Sec. 2.1): the
 * newest token of request b is token L-1 with L = seq_lens[b] (clamped to the
 * table); its key and value rows k_new[b][g][:], v_new[b][g][:] go to block
 * block_table[b][(L-1)/bs], slot (L-1) % bs. L <= 0 or an out-of-range block
 * id: nothing written. Returns the number of requests written.
 */
int32_t neo_ref_kv_append(uint16_t* k_cache, uint16_t* v_cache, const uint16_t* k_new,
                          const uint16_t* v_new, const int32_t* block_table,
                          const int32_t* seq_lens, int32_t batch, int32_t max_blocks_per_seq,
                          int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                          int32_t num_blocks) {
  int32_t written = 0;
  for (int64_t b = 0; b < batch; ++b) {
    int64_t L = seq_lens[b];
    int64_t cap = (int64_t)max_blocks_per_seq * block_size;
    if (L > cap) L = cap;
    if (L <= 0) continue;
    int64_t t = L - 1;
    int64_t p = block_table[b * max_blocks_per_seq + t / block_size];
    if (p < 0 || p >= num_blocks) continue;
    int64_t slot = t % block_size;
    for (int64_t g = 0; g < num_kv_heads; ++g) {
      for (int64_t d = 0; d < head_dim; ++d) {
        int64_t src = (b * num_kv_heads + g) * head_dim + d;
        k_cache[(((p * num_kv_heads + g) * (head_dim / 8) + d / 8) * block_size + slot) * 8 +
                d % 8] = k_new[src];
        v_cache[((p * num_kv_heads + g) * head_dim + d) * block_size + slot] = v_new[src];
      }
    }
    ++written;
  }
  return written;
}

/*
 * Block copy between two caches of the same layout: dst block dst_ids[i] <-
 * src block src_ids[i] for every i with both ids in range (all kv heads, K and V).
 */
int32_t neo_ref_copy_blocks(const uint16_t* src_k, const uint16_t* src_v, uint16_t* dst_k,
                            uint16_t* dst_v, const int32_t* src_ids, const int32_t* dst_ids,
                            int32_t n, int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                            int32_t src_num_blocks, int32_t dst_num_blocks) {
  int64_t per = (int64_t)num_kv_heads * head_dim * block_size;
  int32_t copied = 0;
  for (int32_t i = 0; i < n; ++i) {
    int64_t s = src_ids[i], d = dst_ids[i];
    if (s < 0 || s >= src_num_blocks || d < 0 || d >= dst_num_blocks) continue;
    for (int64_t e = 0; e < per; ++e) {
      dst_k[d * per + e] = src_k[s * per + e];
      dst_v[d * per + e] = src_v[s * per + e];
    }
    ++copied;
  }
  return copied;
}
