// Paged decode attention on the host CPU: the CPU half of the offloaded
// decoding path (Sec. 4, efficient CPU kernels), over the same paged layout as
// the GPU cache, so blocks move between the two caches unchanged.
//
// Parallel structure (the Flash-Decoding-like strategy of Sec. 4): every
// (request, kv head) pair is cut at block granularity into tasks; the threads
// get equal shares of blocks (plus a small per-pair cost), each task reads its
// own contiguous 4 KiB K and V tiles, and the partial outputs of a pair cut
// between threads are aggregated with the log-sum-exp identity at the end.
//
// Within a core (Sec. 4: SIMD loads, contiguous access): the AVX-512 BF16
// path scores a K tile for up to four heads of the query group with
// vdpbf16ps over 64-byte rows, and accumulates P*V with vdpbf16ps as well,
// P split into a bf16 high part and a bf16 remainder so the weights keep
// about 16 significant bits. A portable scalar path computes the same thing.
//
// Built with the host compiler; the ISA-specific functions carry target
// attributes and are chosen at run time.
#include <immintrin.h>
#include <pthread.h>
#include <sched.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "libneoattn.h"
#include "neo_error.h"

namespace neo {
namespace cpu {
namespace {

constexpr int kD = 128;          // head_dim
constexpr int kBs = 16;          // tokens per block
constexpr int kTile = kD * kBs;  // bf16 elements of one (block, kv head) tile
constexpr int kChunk = 8;        // tiles per online-softmax step
constexpr int kMaxGroup = 16;
constexpr int64_t kPairCost = 1;  // per-(request, kv head) overhead, in tiles
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ------------------------------------------------------------------ threads

// Fixed set of worker threads, created on first use and kept for the process.
// run(n, fn) calls fn(tid) for tid in [0, n): tid 0 on the calling thread,
// the rest on workers 1..n-1, each woken on its own (a call wakes only the
// workers it uses). A worker spins briefly after a job before sleeping, so
// back-to-back calls skip the wakeup. Calls are serialised.
class Pool {
 public:
  static Pool& get() {
    static Pool* pool = new Pool();  // never destroyed: workers live until exit
    return *pool;
  }

  void run(int n, const std::function<void(int)>& fn) {
    std::lock_guard<std::mutex> call_lock(call_m_);
    grow(n - 1);
    job_ = &fn;
    remaining_.store(n - 1, std::memory_order_relaxed);
    ++gen_;
    for (int i = 1; i < n; ++i) {
      Worker& w = *workers_[i - 1];
      {
        std::lock_guard<std::mutex> lk(w.m);
        w.gen.store(gen_, std::memory_order_release);
      }
      w.cv.notify_one();
    }
    fn(0);
    for (int i = 0; remaining_.load(std::memory_order_acquire) != 0; ++i) {
      if (i < 100000)
        _mm_pause();
      else
        sched_yield();
    }
  }

 private:
  struct Worker {
    std::mutex m;
    std::condition_variable cv;
    std::atomic<uint64_t> gen{0};
  };

  Pool() = default;

  void grow(int n) {
    while ((int)workers_.size() < n) {
      workers_.emplace_back(new Worker());
      Worker* w = workers_.back();
      const int tid = (int)workers_.size();
      std::thread([this, w, tid] { loop(*w, tid); }).detach();
    }
  }

  void loop(Worker& w, int tid) {
    uint64_t seen = 0;
    for (;;) {
      // Spin for a while (about 50 us), then sleep until signalled.
      for (int i = 0; i < 20000 && w.gen.load(std::memory_order_acquire) == seen; ++i)
        _mm_pause();
      if (w.gen.load(std::memory_order_acquire) == seen) {
        std::unique_lock<std::mutex> lk(w.m);
        w.cv.wait(lk, [&] { return w.gen.load(std::memory_order_acquire) != seen; });
      }
      seen = w.gen.load(std::memory_order_acquire);
      (*job_)(tid);
      remaining_.fetch_sub(1, std::memory_order_acq_rel);
    }
  }

  std::mutex call_m_;
  uint64_t gen_ = 0;
  const std::function<void(int)>* job_ = nullptr;
  std::atomic<int> remaining_{0};
  std::vector<Worker*> workers_;
};

// Barrier for the n threads of one run() call.
class Barrier {
 public:
  explicit Barrier(int n) : n_(n) {}
  void wait() {
    const int g = gen_.load(std::memory_order_acquire);
    if (count_.fetch_add(1, std::memory_order_acq_rel) == n_ - 1) {
      count_.store(0, std::memory_order_relaxed);
      gen_.store(g + 1, std::memory_order_release);
      return;
    }
    for (int i = 0; gen_.load(std::memory_order_acquire) == g; ++i) {
      if (i < 4000)
        _mm_pause();
      else
        sched_yield();
    }
  }

 private:
  const int n_;
  std::atomic<int> count_{0};
  std::atomic<int> gen_{0};
};

// ------------------------------------------------------------------ problem

struct Problem {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* table;
  const int32_t* lens;
  float* out;
  int32_t batch, hq, hkv, group, mbps;
  float scale_log2;  // scale * log2(e): scores are kept in base 2
};

inline int32_t clamp_len(int32_t L, int32_t mbps) {
  const int64_t cap = (int64_t)mbps * kBs;
  return L <= 0 ? 0 : (int32_t)std::min<int64_t>(L, cap);
}

inline float bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

// One task: pair (b, g), tiles [j0, j1) of the request's nb tiles. Writes the
// G normalised output rows to `o` (stride kD) and, when `lse` is non-null,
// the natural-log log-sum-exp of each head's scores over those tiles.
struct Task {
  int32_t b, g, j0, j1, L;
  float* o;
  float* lse;
};

// ------------------------------------------------------------------ generic

void task_generic(const Problem& P, const Task& t) {
  const int G = P.group;
  float qf[kMaxGroup][kD];
  float m[kMaxGroup], l[kMaxGroup];
  float acc[kMaxGroup][kD];
  for (int h = 0; h < G; ++h) {
    const uint16_t* qr = P.q + ((size_t)t.b * P.hq + (size_t)t.g * G + h) * kD;
    for (int d = 0; d < kD; ++d) qf[h][d] = bf16_to_f32(qr[d]);
    m[h] = -INFINITY;
    l[h] = 0.f;
    for (int d = 0; d < kD; ++d) acc[h][d] = 0.f;
  }
  const int32_t* row = P.table + (size_t)t.b * P.mbps;
  for (int j = t.j0; j < t.j1; ++j) {
    const size_t tile = ((size_t)row[j] * P.hkv + t.g) * kTile;
    const uint16_t* kt = P.k + tile;  // [16 pieces][16 tokens][8]
    const uint16_t* vt = P.v + tile;  // [128 dims][16 tokens]
    const int valid = std::min(kBs, t.L - j * kBs);
    for (int h = 0; h < G; ++h) {
      float s[kBs];
      float smax = -INFINITY;
      for (int tok = 0; tok < valid; ++tok) {
        float dot = 0.f;
        for (int d = 0; d < kD; ++d)
          dot += qf[h][d] * bf16_to_f32(kt[((d >> 3) * kBs + tok) * 8 + (d & 7)]);
        s[tok] = dot * P.scale_log2;
        smax = std::max(smax, s[tok]);
      }
      const float mn = std::max(m[h], smax);
      const float alpha = std::exp2(m[h] - mn);
      float p[kBs];
      float psum = 0.f;
      for (int tok = 0; tok < valid; ++tok) {
        p[tok] = std::exp2(s[tok] - mn);
        psum += p[tok];
      }
      l[h] = l[h] * alpha + psum;
      m[h] = mn;
      for (int d = 0; d < kD; ++d) {
        float a = acc[h][d] * alpha;
        for (int tok = 0; tok < valid; ++tok) a += p[tok] * bf16_to_f32(vt[d * kBs + tok]);
        acc[h][d] = a;
      }
    }
  }
  for (int h = 0; h < G; ++h) {
    const float inv = 1.f / l[h];
    for (int d = 0; d < kD; ++d) t.o[h * kD + d] = acc[h][d] * inv;
    if (t.lse) t.lse[h] = (m[h] + std::log2(l[h])) * kLn2;
  }
}

// ----------------------------------------------------------------- AVX-512
//
// Two AVX-512 formulations of the same chunked task, sharing the chunk loop,
// the softmax step and the final reduction:
//  * kDot (AVX-512 BF16): vdpbf16ps multiplies bf16 pairs straight from the
//    tiles; P is split into bf16 hi + lo parts.
//  * kFma (AVX-512F): bf16 pairs are widened to fp32 with one shift (even
//    elements) and one mask (odd elements) per 64 bytes, and multiplied with
//    fp32 FMAs; the query is pre-split into even and odd dims to match, and P
//    stays fp32.
// Which is faster depends on the core's vdpbf16ps and FMA throughputs.

#define NEO_AVX512 __attribute__((target("avx512f,avx512bw,avx512vl,avx512dq")))
#define NEO_AVX512BF16 __attribute__((target("avx512f,avx512bw,avx512vl,avx512dq,avx512bf16")))

enum class Math { kDot, kFma };

// 2^x for x <= 0: x = n + f with n = round(x), |f| <= 1/2, 2^f = e^(f ln 2)
// by its Taylor series to degree 7 (remainder below 6e-9 relative), then
// scaled by 2^n. Below x = -125 the result is 0 (x = -inf included): a weight
// that far under the running maximum changes nothing in fp32, and it keeps
// every intermediate a normal number (denormals take slow microcode assists
// on some cores).
NEO_AVX512 inline __m512 exp2_ps(__m512 x) {
  const __m512 lo = _mm512_set1_ps(-125.f);
  const __mmask16 keep = _mm512_cmp_ps_mask(x, lo, _CMP_GE_OQ);
  x = _mm512_max_ps(x, lo);
  const __m512 n = _mm512_roundscale_ps(x, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC);
  const __m512 f = _mm512_sub_ps(x, n);
  constexpr double c1 = 0.6931471805599453;  // ln 2
  constexpr double c2 = c1 * c1 / 2, c3 = c2 * c1 / 3, c4 = c3 * c1 / 4, c5 = c4 * c1 / 5;
  constexpr double c6 = c5 * c1 / 6, c7 = c6 * c1 / 7;
  __m512 p = _mm512_set1_ps((float)c7);
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps((float)c6));
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps((float)c5));
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps((float)c4));
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps((float)c3));
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps((float)c2));
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps((float)c1));
  p = _mm512_fmadd_ps(p, f, _mm512_set1_ps(1.f));
  return _mm512_maskz_mov_ps(keep, _mm512_scalef_ps(p, n));
}

// 32 bf16 (as 16 dwords) -> fp32 of the even elements / of the odd elements.
NEO_AVX512 inline __m512 even_ps(__m512i x) { return _mm512_castsi512_ps(_mm512_slli_epi32(x, 16)); }
NEO_AVX512 inline __m512 odd_ps(__m512i x) {
  return _mm512_castsi512_ps(_mm512_and_si512(x, _mm512_set1_epi32((int)0xFFFF0000u)));
}

NEO_AVX512 inline __m512 bf16x16_to_ps(__m256i h) {
  return _mm512_castsi512_ps(_mm512_slli_epi32(_mm512_cvtepu16_epi32(h), 16));
}

// Pairwise sums of adjacent lanes over the 32 lanes a ++ b:
// result lane i = x[2i] + x[2i+1].
NEO_AVX512 inline __m512 pair_sum(__m512 a, __m512 b) {
  const __m512i even = _mm512_set_epi32(30, 28, 26, 24, 22, 20, 18, 16, 14, 12, 10, 8, 6, 4, 2, 0);
  const __m512i odd = _mm512_set_epi32(31, 29, 27, 25, 23, 21, 19, 17, 15, 13, 11, 9, 7, 5, 3, 1);
  return _mm512_add_ps(_mm512_permutex2var_ps(a, even, b), _mm512_permutex2var_ps(a, odd, b));
}

// Scores from the accumulators acc[i] (i = token group 4i..4i+3), whose lane
// 4u + r holds a partial dot product of token 4i + u: a 4x4 transpose inside
// each 128-bit lane and a sum leave token 4i + u at lane 4u + i; one permute
// restores token order. Scaled to base 2; tokens >= valid get -inf.
NEO_AVX512 inline void finish_scores(const __m512* acc, int valid, float scale_log2, float* out) {
  const __m512i order = _mm512_set_epi32(15, 11, 7, 3, 14, 10, 6, 2, 13, 9, 5, 1, 12, 8, 4, 0);
  const __mmask16 live = valid >= 16 ? (__mmask16)0xFFFF : (__mmask16)((1u << valid) - 1);
  const __m512 t0 = _mm512_unpacklo_ps(acc[0], acc[1]);
  const __m512 t1 = _mm512_unpackhi_ps(acc[0], acc[1]);
  const __m512 t2 = _mm512_unpacklo_ps(acc[2], acc[3]);
  const __m512 t3 = _mm512_unpackhi_ps(acc[2], acc[3]);
  const __m512 r0 = _mm512_shuffle_ps(t0, t2, 0x44);
  const __m512 r1 = _mm512_shuffle_ps(t0, t2, 0xEE);
  const __m512 r2 = _mm512_shuffle_ps(t1, t3, 0x44);
  const __m512 r3 = _mm512_shuffle_ps(t1, t3, 0xEE);
  __m512 s = _mm512_add_ps(_mm512_add_ps(r0, r1), _mm512_add_ps(r2, r3));
  s = _mm512_mul_ps(_mm512_permutexvar_ps(order, s), _mm512_set1_ps(scale_log2));
  _mm512_storeu_ps(out, _mm512_mask_mov_ps(_mm512_set1_ps(-INFINITY), live, s));
}

// K tile rows: piece c (dims 8c..8c+7) of tokens 4i..4i+3 are 64 contiguous
// bytes at element c * 128 + i * 32.

// kDot scores for heads [0, HB) of qrow (bf16 rows).
template <int HB>
NEO_AVX512BF16 inline void score_tile_dot(const uint16_t* kt, const uint16_t* const* qrow,
                                          int valid, float scale_log2, float* const* s_out) {
  __m512 acc[HB][4];
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h)
    for (int i = 0; i < 4; ++i) acc[h][i] = _mm512_setzero_ps();
#pragma GCC unroll 2
  for (int c = 0; c < 16; ++c) {
    const __m512i k0 = _mm512_loadu_si512(kt + c * 128);
    const __m512i k1 = _mm512_loadu_si512(kt + c * 128 + 32);
    const __m512i k2 = _mm512_loadu_si512(kt + c * 128 + 64);
    const __m512i k3 = _mm512_loadu_si512(kt + c * 128 + 96);
#pragma GCC unroll 4
    for (int h = 0; h < HB; ++h) {
      const __m512i qv =
          _mm512_broadcast_i32x4(_mm_loadu_si128((const __m128i*)(qrow[h] + 8 * c)));
      acc[h][0] = _mm512_dpbf16_ps(acc[h][0], (__m512bh)k0, (__m512bh)qv);
      acc[h][1] = _mm512_dpbf16_ps(acc[h][1], (__m512bh)k1, (__m512bh)qv);
      acc[h][2] = _mm512_dpbf16_ps(acc[h][2], (__m512bh)k2, (__m512bh)qv);
      acc[h][3] = _mm512_dpbf16_ps(acc[h][3], (__m512bh)k3, (__m512bh)qv);
    }
  }
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h) finish_scores(acc[h], valid, scale_log2, s_out[h]);
}

// kFma scores for heads [0, HB); qsplit[h] holds, per piece c, the fp32 query
// dims (8c, 8c+2, 8c+4, 8c+6) then (8c+1, 8c+3, 8c+5, 8c+7).
template <int HB>
NEO_AVX512 inline void score_tile_fma(const uint16_t* kt, const float* const* qsplit, int valid,
                                      float scale_log2, float* const* s_out) {
  __m512 acc[HB][4];
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h)
    for (int i = 0; i < 4; ++i) acc[h][i] = _mm512_setzero_ps();
  for (int c = 0; c < 16; ++c) {
    __m512 qe[HB], qo[HB];
#pragma GCC unroll 4
    for (int h = 0; h < HB; ++h) {
      qe[h] = _mm512_broadcast_f32x4(_mm_load_ps(qsplit[h] + c * 8));
      qo[h] = _mm512_broadcast_f32x4(_mm_load_ps(qsplit[h] + c * 8 + 4));
    }
#pragma GCC unroll 4
    for (int i = 0; i < 4; ++i) {
      const __m512i k = _mm512_loadu_si512(kt + c * 128 + i * 32);
      const __m512 ke = even_ps(k), ko = odd_ps(k);
#pragma GCC unroll 4
      for (int h = 0; h < HB; ++h)
        acc[h][i] = _mm512_fmadd_ps(ko, qo[h], _mm512_fmadd_ps(ke, qe[h], acc[h][i]));
    }
  }
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h) finish_scores(acc[h], valid, scale_log2, s_out[h]);
}

// V tile rows (2dp, 2dp + 1) are the 64 bytes at element dp * 32. acc[h][dp]
// lanes 0-7 gather row 2dp, lanes 8-15 row 2dp+1 (token pairs), reduced at
// the end of the task. One call: d pairs [4 db, 4 db + 4), heads [h0, h0+HB),
// all tiles of the chunk; the stored accumulators are first scaled by alpha
// (on the task's first chunk, `fresh`, they start from zero instead).
// P per (head, tile): kDot: 16 bf16 hi then 16 bf16 lo (64 bytes);
// kFma: 8 fp32 weights of even tokens then 8 of odd tokens (64 bytes).
template <int HB>
NEO_AVX512BF16 inline void accumulate_v_dot(const uint16_t* const* vtiles, int ntiles, int db,
                                            const uint8_t* pbuf, int h0, float* accv,
                                            const float* alpha, bool fresh) {
  __m512 acc[HB][4];
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h) {
    const __m512 a = _mm512_set1_ps(alpha[h0 + h]);
    for (int i = 0; i < 4; ++i)
      acc[h][i] = fresh ? _mm512_setzero_ps()
                        : _mm512_mul_ps(_mm512_load_ps(accv + ((h0 + h) * 64 + db * 4 + i) * 16), a);
  }
  for (int tt = 0; tt < ntiles; ++tt) {
    const uint16_t* vt = vtiles[tt] + db * 4 * 32;
    const __m512i v0 = _mm512_loadu_si512(vt);
    const __m512i v1 = _mm512_loadu_si512(vt + 32);
    const __m512i v2 = _mm512_loadu_si512(vt + 64);
    const __m512i v3 = _mm512_loadu_si512(vt + 96);
#pragma GCC unroll 4
    for (int h = 0; h < HB; ++h) {
      const uint8_t* pp = pbuf + ((size_t)(h0 + h) * kChunk + tt) * 64;
      const __m512i ph = _mm512_broadcast_i64x4(_mm256_load_si256((const __m256i*)pp));
      const __m512i pl = _mm512_broadcast_i64x4(_mm256_load_si256((const __m256i*)(pp + 32)));
      acc[h][0] = _mm512_dpbf16_ps(acc[h][0], (__m512bh)v0, (__m512bh)ph);
      acc[h][1] = _mm512_dpbf16_ps(acc[h][1], (__m512bh)v1, (__m512bh)ph);
      acc[h][2] = _mm512_dpbf16_ps(acc[h][2], (__m512bh)v2, (__m512bh)ph);
      acc[h][3] = _mm512_dpbf16_ps(acc[h][3], (__m512bh)v3, (__m512bh)ph);
      acc[h][0] = _mm512_dpbf16_ps(acc[h][0], (__m512bh)v0, (__m512bh)pl);
      acc[h][1] = _mm512_dpbf16_ps(acc[h][1], (__m512bh)v1, (__m512bh)pl);
      acc[h][2] = _mm512_dpbf16_ps(acc[h][2], (__m512bh)v2, (__m512bh)pl);
      acc[h][3] = _mm512_dpbf16_ps(acc[h][3], (__m512bh)v3, (__m512bh)pl);
    }
  }
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h)
    for (int i = 0; i < 4; ++i)
      _mm512_store_ps(accv + ((h0 + h) * 64 + db * 4 + i) * 16, acc[h][i]);
}

template <int HB>
NEO_AVX512 inline void accumulate_v_fma(const uint16_t* const* vtiles, int ntiles, int db,
                                        const uint8_t* pbuf, int h0, float* accv,
                                        const float* alpha, bool fresh) {
  __m512 acc[HB][4];
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h) {
    const __m512 a = _mm512_set1_ps(alpha[h0 + h]);
    for (int i = 0; i < 4; ++i)
      acc[h][i] = fresh ? _mm512_setzero_ps()
                        : _mm512_mul_ps(_mm512_load_ps(accv + ((h0 + h) * 64 + db * 4 + i) * 16), a);
  }
  for (int tt = 0; tt < ntiles; ++tt) {
    const uint16_t* vt = vtiles[tt] + db * 4 * 32;
    __m512 pe[HB], po[HB];
#pragma GCC unroll 4
    for (int h = 0; h < HB; ++h) {
      const float* pp = reinterpret_cast<const float*>(pbuf + ((size_t)(h0 + h) * kChunk + tt) * 64);
      pe[h] = _mm512_broadcast_f32x8(_mm256_load_ps(pp));
      po[h] = _mm512_broadcast_f32x8(_mm256_load_ps(pp + 8));
    }
#pragma GCC unroll 4
    for (int i = 0; i < 4; ++i) {
      const __m512i v = _mm512_loadu_si512(vt + i * 32);
      const __m512 ve = even_ps(v), vo = odd_ps(v);
#pragma GCC unroll 4
      for (int h = 0; h < HB; ++h)
        acc[h][i] = _mm512_fmadd_ps(vo, po[h], _mm512_fmadd_ps(ve, pe[h], acc[h][i]));
    }
  }
#pragma GCC unroll 4
  for (int h = 0; h < HB; ++h)
    for (int i = 0; i < 4; ++i)
      _mm512_store_ps(accv + ((h0 + h) * 64 + db * 4 + i) * 16, acc[h][i]);
}

// fp32 query in the kFma order: per piece c, dims (8c, 8c+2, 8c+4, 8c+6)
// then (8c+1, 8c+3, 8c+5, 8c+7). 64 bytes of bf16 (pieces 4k..4k+3) widen to
// even and odd dims, interleaved four at a time.
NEO_AVX512 inline void split_query(const uint16_t* q, float* out) {
  const __m512i lo = _mm512_set_epi32(23, 22, 21, 20, 7, 6, 5, 4, 19, 18, 17, 16, 3, 2, 1, 0);
  const __m512i hi = _mm512_set_epi32(31, 30, 29, 28, 15, 14, 13, 12, 27, 26, 25, 24, 11, 10, 9, 8);
  for (int k = 0; k < 4; ++k) {
    const __m512i x = _mm512_loadu_si512(q + 32 * k);
    const __m512 e = even_ps(x), o = odd_ps(x);
    _mm512_store_ps(out + 32 * k, _mm512_permutex2var_ps(e, lo, o));
    _mm512_store_ps(out + 32 * k + 16, _mm512_permutex2var_ps(e, hi, o));
  }
}

// P of one (head, tile) from its 16 base-2 scores and the running max.
NEO_AVX512BF16 inline __m512 store_p_dot(__m512 s, __m512 mv, uint8_t* pp) {
  const __m512 p = exp2_ps(_mm512_sub_ps(s, mv));
  const __m256i hi = (__m256i)_mm512_cvtneps_pbh(p);
  const __m512 lo = _mm512_sub_ps(p, bf16x16_to_ps(hi));
  _mm256_store_si256((__m256i*)pp, hi);
  _mm256_store_si256((__m256i*)(pp + 32), (__m256i)_mm512_cvtneps_pbh(lo));
  return p;
}

NEO_AVX512 inline __m512 store_p_fma(__m512 s, __m512 mv, uint8_t* pp) {
  const __m512 p = exp2_ps(_mm512_sub_ps(s, mv));
  const __m512i split = _mm512_set_epi32(15, 13, 11, 9, 7, 5, 3, 1, 14, 12, 10, 8, 6, 4, 2, 0);
  _mm512_store_ps(reinterpret_cast<float*>(pp), _mm512_permutexvar_ps(split, p));
  return p;
}

// The chunked task. Per chunk of up to kChunk tiles: scores of every tile,
// one online-softmax step (running max, rescale factor alpha, P), then P*V
// accumulated d-block by d-block over the chunk. (Software prefetch of the
// next tiles measured slower than the hardware prefetchers.) A macro body, instantiated in
// two functions, because the two formulations need different target
// attributes and GCC will not inline target-specific code across them.

#define NEO_TASK_BODY                                                                        \
  constexpr int HB = G < 4 ? G : 4;                                                          \
  alignas(64) float accv[G * 64 * 16];                                                       \
  alignas(64) float sbuf[G][kChunk * kBs];                                                   \
  alignas(64) uint8_t pbuf[G * kChunk * 64];                                                 \
  alignas(64) uint16_t vtail[kTile];                                                         \
  alignas(64) float qsplit[M == Math::kFma ? G : 1][kD];                                     \
  float m[G], l[G], alpha[G];                                                                \
  const uint16_t* qrow[G];                                                                   \
  const float* qs[G];                                                                        \
  for (int h = 0; h < G; ++h) {                                                              \
    qrow[h] = P.q + ((size_t)t.b * P.hq + (size_t)t.g * G + h) * kD;                         \
    if (M == Math::kFma) {                                                                   \
      split_query(qrow[h], qsplit[h]);                                                       \
      qs[h] = qsplit[h];                                                                     \
    }                                                                                        \
    m[h] = -INFINITY;                                                                        \
    l[h] = 0.f;                                                                              \
  }                                                                                          \
  const int32_t* row = P.table + (size_t)t.b * P.mbps;                                       \
  for (int jc = t.j0; jc < t.j1; jc += kChunk) {                                             \
    const int n = std::min(kChunk, t.j1 - jc);                                               \
    const uint16_t* vtiles[kChunk];                                                          \
    for (int tt = 0; tt < n; ++tt) {                                                         \
      const int j = jc + tt;                                                                 \
      const size_t tile = ((size_t)row[j] * P.hkv + t.g) * kTile;                            \
      const int valid = std::min(kBs, t.L - j * kBs);                                        \
      vtiles[tt] = P.v + tile;                                                               \
      for (int h0 = 0; h0 < G; h0 += HB) {                                                   \
        float* so[HB];                                                                       \
        for (int h = 0; h < HB; ++h) so[h] = &sbuf[h0 + h][tt * kBs];                        \
        if (M == Math::kDot)                                                                 \
          score_tile_dot<HB>(P.k + tile, qrow + h0, valid, P.scale_log2, so);                \
        else                                                                                 \
          score_tile_fma<HB>(P.k + tile, qs + h0, valid, P.scale_log2, so);                  \
      }                                                                                      \
      if (valid < kBs) {                                                                     \
        /* unused slots of the last tile: weight 0, but 0 * NaN must not reach P*V. */      \
        /* Two dims per 64-byte store, the size P*V loads, so the loads are forwarded. */    \
        const uint32_t live16 = (1u << valid) - 1;                                           \
        const __mmask32 live = (__mmask32)(live16 | (live16 << 16));                         \
        for (int d = 0; d < kD; d += 2)                                                      \
          _mm512_store_si512(vtail + d * kBs,                                                \
                             _mm512_maskz_mov_epi16(live, _mm512_loadu_si512(                \
                                 P.v + tile + d * kBs)));                                    \
        vtiles[tt] = vtail;                                                                  \
      }                                                                                      \
    }                                                                                        \
    for (int h = 0; h < G; ++h) {                                                            \
      __m512 mx = _mm512_set1_ps(-INFINITY);                                                 \
      for (int tt = 0; tt < n; ++tt) mx = _mm512_max_ps(mx, _mm512_load_ps(&sbuf[h][tt * kBs])); \
      const float mn = std::max(m[h], _mm512_reduce_max_ps(mx));                             \
      alpha[h] = std::exp2(m[h] - mn); /* 0 on the first chunk */                            \
      const __m512 mv = _mm512_set1_ps(mn);                                                  \
      __m512 ls = _mm512_setzero_ps();                                                       \
      for (int tt = 0; tt < n; ++tt) {                                                       \
        uint8_t* pp = pbuf + ((size_t)h * kChunk + tt) * 64;                                 \
        const __m512 s = _mm512_load_ps(&sbuf[h][tt * kBs]);                                 \
        ls = _mm512_add_ps(ls, M == Math::kDot ? store_p_dot(s, mv, pp) : store_p_fma(s, mv, pp)); \
      }                                                                                      \
      l[h] = l[h] * alpha[h] + _mm512_reduce_add_ps(ls);                                     \
      m[h] = mn;                                                                             \
    }                                                                                        \
    for (int db = 0; db < 16; ++db)                                                          \
      for (int h0 = 0; h0 < G; h0 += HB) {                                                   \
        if (M == Math::kDot)                                                                 \
          accumulate_v_dot<HB>(vtiles, n, db, pbuf, h0, accv, alpha, jc == t.j0);            \
        else                                                                                 \
          accumulate_v_fma<HB>(vtiles, n, db, pbuf, h0, accv, alpha, jc == t.j0);            \
      }                                                                                      \
  }                                                                                          \
  for (int h = 0; h < G; ++h) {                                                              \
    const __m512 inv = _mm512_set1_ps(1.f / l[h]);                                           \
    const float* a = accv + h * 64 * 16;                                                     \
    for (int k = 0; k < 8; ++k) {                                                            \
      const float* x = a + k * 8 * 16;                                                       \
      const __m512 y0 = pair_sum(_mm512_load_ps(x + 0 * 16), _mm512_load_ps(x + 1 * 16));    \
      const __m512 y1 = pair_sum(_mm512_load_ps(x + 2 * 16), _mm512_load_ps(x + 3 * 16));    \
      const __m512 y2 = pair_sum(_mm512_load_ps(x + 4 * 16), _mm512_load_ps(x + 5 * 16));    \
      const __m512 y3 = pair_sum(_mm512_load_ps(x + 6 * 16), _mm512_load_ps(x + 7 * 16));    \
      const __m512 z = pair_sum(pair_sum(y0, y1), pair_sum(y2, y3));                         \
      _mm512_storeu_ps(t.o + h * kD + k * 16, _mm512_mul_ps(z, inv));                        \
    }                                                                                        \
    if (t.lse) t.lse[h] = (m[h] + std::log2(l[h])) * kLn2;                                   \
  }

template <int G>
NEO_AVX512BF16 void task_dot_g(const Problem& P, const Task& t) {
  constexpr Math M = Math::kDot;
  NEO_TASK_BODY
}

template <int G>
NEO_AVX512 void task_fma_g(const Problem& P, const Task& t) {
  constexpr Math M = Math::kFma;
  NEO_TASK_BODY
}

#undef NEO_TASK_BODY

NEO_AVX512BF16 void task_avx512_bf16(const Problem& P, const Task& t) {
  switch (P.group) {
    case 1: return task_dot_g<1>(P, t);
    case 2: return task_dot_g<2>(P, t);
    case 4: return task_dot_g<4>(P, t);
    case 8: return task_dot_g<8>(P, t);
    default: return task_dot_g<16>(P, t);
  }
}

NEO_AVX512 void task_avx512(const Problem& P, const Task& t) {
  switch (P.group) {
    case 1: return task_fma_g<1>(P, t);
    case 2: return task_fma_g<2>(P, t);
    case 4: return task_fma_g<4>(P, t);
    case 8: return task_fma_g<8>(P, t);
    default: return task_fma_g<16>(P, t);
  }
}

bool cpu_has_avx512() {
  __builtin_cpu_init();
  return __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
         __builtin_cpu_supports("avx512vl") && __builtin_cpu_supports("avx512dq");
}

bool cpu_has_avx512_bf16() { return cpu_has_avx512() && __builtin_cpu_supports("avx512bf16"); }

// The default path: NEO_CPU_ISA if set to one this CPU has; else the FMA
// formulation on any AVX-512 CPU (measured: as fast as vdpbf16ps on a
// Zen 5 host, where both run near the memory ceiling, and faster on Intel
// cores, where vdpbf16ps issues at a quarter of the FMA rate; and fp32 P
// is the more accurate); the generic code without AVX-512.
int32_t best_isa() {
  static const int32_t isa = [] {
    const char* e = getenv("NEO_CPU_ISA");
    if (e) {
      if (!strcmp(e, "generic")) return (int32_t)NEO_CPU_ISA_GENERIC;
      if (!strcmp(e, "avx512") && cpu_has_avx512()) return (int32_t)NEO_CPU_ISA_AVX512;
      if (!strcmp(e, "avx512_bf16") && cpu_has_avx512_bf16())
        return (int32_t)NEO_CPU_ISA_AVX512_BF16;
    }
    return (int32_t)(cpu_has_avx512() ? NEO_CPU_ISA_AVX512 : NEO_CPU_ISA_GENERIC);
  }();
  return isa;
}

// ------------------------------------------------------------------ driver

using TaskFn = void (*)(const Problem&, const Task&);

// Start of thread i's share of the weighted positions [0, W).
inline int64_t share_start(int64_t i, int64_t W, int64_t T) { return i * W / T; }
// Thread whose share holds position x.
inline int64_t share_of(int64_t x, int64_t W, int64_t T) { return ((x + 1) * T - 1) / W; }

// Merges the partials of one pair cut between threads [c0, c1]: thread c0
// wrote slot 2 c0 + 1, later threads slot 2 c.
void merge_pair(const Problem& P, int64_t b, int64_t g, int64_t c0, int64_t c1,
                const float* part_o, const float* part_lse) {
  const int G = P.group;
  for (int h = 0; h < G; ++h) {
    float mx = -INFINITY;
    for (int64_t c = c0; c <= c1; ++c) {
      const int64_t slot = c == c0 ? 2 * c + 1 : 2 * c;
      mx = std::max(mx, part_lse[slot * G + h]);
    }
    float acc[kD] = {0.f};
    float wsum = 0.f;
    for (int64_t c = c0; c <= c1; ++c) {
      const int64_t slot = c == c0 ? 2 * c + 1 : 2 * c;
      const float w = std::exp(part_lse[slot * G + h] - mx);
      wsum += w;
      const float* o = part_o + (slot * G + h) * kD;
      for (int d = 0; d < kD; ++d) acc[d] += w * o[d];
    }
    float* dst = P.out + ((size_t)b * P.hq + (size_t)g * G + h) * kD;
    const float inv = 1.f / wsum;
    for (int d = 0; d < kD; ++d) dst[d] = acc[d] * inv;
  }
}

struct Scratch {
  std::vector<int64_t> prefix;
  std::vector<float> part_o, part_lse;
};

Scratch& scratch() {
  static Scratch s;  // guarded by the pool's call serialisation
  return s;
}

std::mutex g_call_m;

int default_threads() {
  for (const char* var : {"NEO_CPU_THREADS", "OMP_NUM_THREADS"}) {
    const char* e = getenv(var);
    if (e && atoi(e) > 0) return atoi(e);
  }
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof set, &set) == 0) return std::max(1, CPU_COUNT(&set));
  return std::max(1u, std::thread::hardware_concurrency());
}

neo_status run(const Problem& P, int threads, TaskFn fn) {
  std::lock_guard<std::mutex> lock(g_call_m);
  Scratch& S = scratch();
  const int64_t npairs = (int64_t)P.batch * P.hkv;
  S.prefix.resize(npairs + 1);
  int64_t W = 0;
  for (int64_t b = 0; b < P.batch; ++b) {
    const int32_t L = clamp_len(P.lens[b], P.mbps);
    const int64_t nb = (L + kBs - 1) / kBs;
    if (nb == 0) memset(P.out + (size_t)b * P.hq * kD, 0, sizeof(float) * P.hq * kD);
    for (int64_t g = 0; g < P.hkv; ++g) {
      S.prefix[b * P.hkv + g] = W;
      W += nb > 0 ? nb + kPairCost : 0;
    }
  }
  S.prefix[npairs] = W;
  if (W == 0) return NEO_OK;
  // At least a few tiles per thread, so tiny batches do not pay for idle wakeups.
  const int64_t T = std::max<int64_t>(1, std::min<int64_t>(threads, W / 4));
  S.part_o.resize((size_t)2 * T * P.group * kD);
  S.part_lse.resize((size_t)2 * T * P.group);
  float* part_o = S.part_o.data();
  float* part_lse = S.part_lse.data();
  const int64_t* prefix = S.prefix.data();
  Barrier barrier((int)T);

  auto job = [&](int tid) {
    const int64_t s0 = share_start(tid, W, T), s1 = share_start(tid + 1, W, T);
    // First pair whose positions reach past s0.
    int64_t p = std::upper_bound(prefix, prefix + npairs + 1, s0) - prefix - 1;
    int64_t merge_b = -1, merge_g = 0, merge_c1 = 0;
    for (; p < npairs && prefix[p] < s1; ++p) {
      const int64_t w = prefix[p + 1] - prefix[p];
      if (w == 0) continue;
      const int64_t nb = w - kPairCost, first = prefix[p] + kPairCost;
      const int64_t j0 = std::max<int64_t>(0, s0 - first), j1 = std::min<int64_t>(nb, s1 - first);
      if (j1 <= j0) continue;
      const int64_t b = p / P.hkv, g = p % P.hkv;
      Task t{(int32_t)b, (int32_t)g, (int32_t)j0, (int32_t)j1, clamp_len(P.lens[b], P.mbps),
             nullptr, nullptr};
      if (j0 == 0 && j1 == nb) {
        t.o = P.out + ((size_t)b * P.hq + (size_t)g * P.group) * kD;
      } else {
        const int64_t slot = j0 > 0 ? 2 * tid : 2 * tid + 1;
        t.o = part_o + (size_t)slot * P.group * kD;
        t.lse = part_lse + (size_t)slot * P.group;
        if (j0 == 0) {
          merge_b = b;
          merge_g = g;
          merge_c1 = share_of(first + nb - 1, W, T);
        }
      }
      fn(P, t);
    }
    barrier.wait();
    if (merge_b >= 0) merge_pair(P, merge_b, merge_g, tid, merge_c1, part_o, part_lse);
  };
  Pool::get().run((int)T, job);
  return NEO_OK;
}

// Sum of 64-byte rows [r0, r1) of buf (keeps the loads live).
NEO_AVX512 double sum_rows_avx512(const float* buf, size_t r0, size_t r1) {
  __m512 a0 = _mm512_setzero_ps(), a1 = a0, a2 = a0, a3 = a0;
  size_t r = r0;
  for (; r + 4 <= r1; r += 4) {
    a0 = _mm512_add_ps(a0, _mm512_loadu_ps(buf + r * 16));
    a1 = _mm512_add_ps(a1, _mm512_loadu_ps(buf + r * 16 + 16));
    a2 = _mm512_add_ps(a2, _mm512_loadu_ps(buf + r * 16 + 32));
    a3 = _mm512_add_ps(a3, _mm512_loadu_ps(buf + r * 16 + 48));
  }
  for (; r < r1; ++r) a0 = _mm512_add_ps(a0, _mm512_loadu_ps(buf + r * 16));
  return _mm512_reduce_add_ps(_mm512_add_ps(_mm512_add_ps(a0, a1), _mm512_add_ps(a2, a3)));
}

double sum_rows_generic(const float* buf, size_t r0, size_t r1) {
  float acc[16] = {0.f};
  for (size_t r = r0; r < r1; ++r)
    for (int i = 0; i < 16; ++i) acc[i] += buf[r * 16 + i];
  double s = 0;
  for (float a : acc) s += a;
  return s;
}

}  // namespace
}  // namespace cpu
}  // namespace neo

extern "C" {

neo_status neo_cpu_read_probe(const void* buf, size_t bytes, int32_t num_threads,
                              double* checksum) {
  using neo::set_error;
  if (!buf || !checksum) return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (bytes % 64 != 0) return set_error(NEO_ERR_INVALID_ARG, "bytes must be a multiple of 64");
  if (num_threads < 0)
    return set_error(NEO_ERR_INVALID_ARG, "num_threads (%d) is negative", num_threads);
  const int T = num_threads > 0 ? num_threads : neo::cpu::default_threads();
  const size_t rows = bytes / 64;
  std::vector<double> part(T, 0.0);
  const float* f = static_cast<const float*>(buf);
  const bool wide = neo::cpu::cpu_has_avx512();
  std::lock_guard<std::mutex> lock(neo::cpu::g_call_m);
  neo::cpu::Pool::get().run(T, [&](int tid) {
    const size_t r0 = rows * tid / T, r1 = rows * (tid + 1) / T;
    part[tid] = wide ? neo::cpu::sum_rows_avx512(f, r0, r1) : neo::cpu::sum_rows_generic(f, r0, r1);
  });
  double s = 0;
  for (double x : part) s += x;
  *checksum = s;
  return neo::clear_error();
}


int32_t neo_cpu_best_isa(void) { return neo::cpu::best_isa(); }

neo_status neo_cpu_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                             const int32_t* block_table, const int32_t* seq_lens, int32_t batch,
                             int32_t max_blocks_per_seq, int32_t num_kv_heads, int32_t head_dim,
                             int32_t block_size, int32_t num_blocks) {
  using neo::set_error;
  namespace C = neo::cpu;
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  if (num_kv_heads <= 0) return set_error(NEO_ERR_INVALID_ARG, "num_kv_heads must be positive");
  if (head_dim != C::kD || block_size != C::kBs)
    return set_error(NEO_ERR_UNSUPPORTED, "head_dim %d / block_size %d unsupported (128 / 16)",
                     head_dim, block_size);
  if (batch == 0) return neo::clear_error();
  if (!k_cache || !v_cache || !k_new || !v_new || !block_table || !seq_lens)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (max_blocks_per_seq <= 0 || num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq and num_blocks must be positive");
  uint16_t* kc = static_cast<uint16_t*>(k_cache);
  uint16_t* vc = static_cast<uint16_t*>(v_cache);
  const uint16_t* kn = static_cast<const uint16_t*>(k_new);
  const uint16_t* vn = static_cast<const uint16_t*>(v_new);
  for (int64_t b = 0; b < batch; ++b) {
    const int32_t L = C::clamp_len(seq_lens[b], max_blocks_per_seq);
    if (L <= 0) continue;
    const int32_t t = L - 1;
    const int32_t blk = block_table[b * max_blocks_per_seq + t / C::kBs];
    if (blk < 0 || blk >= num_blocks) continue;
    const int slot = t % C::kBs;
    for (int64_t g = 0; g < num_kv_heads; ++g) {
      const size_t tile = ((size_t)blk * num_kv_heads + g) * C::kTile;
      const uint16_t* ks = kn + ((size_t)b * num_kv_heads + g) * C::kD;
      const uint16_t* vs = vn + ((size_t)b * num_kv_heads + g) * C::kD;
      for (int c = 0; c < C::kD / 8; ++c)
        memcpy(kc + tile + ((size_t)c * C::kBs + slot) * 8, ks + c * 8, 16);
      for (int d = 0; d < C::kD; ++d) vc[tile + (size_t)d * C::kBs + slot] = vs[d];
    }
  }
  return neo::clear_error();
}

int32_t neo_cpu_default_threads(void) { return neo::cpu::default_threads(); }

neo_status neo_cpu_decode_attention_ex(const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* block_table, const int32_t* seq_lens,
                                       int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t head_dim, int32_t block_size, float scale,
                                       float* out, int32_t batch, int32_t max_blocks_per_seq,
                                       int32_t num_blocks, int32_t num_threads, int32_t isa) {
  using neo::set_error;
  if (batch < 0) return set_error(NEO_ERR_INVALID_ARG, "batch (%d) is negative", batch);
  if (num_q_heads <= 0 || num_kv_heads <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "num_q_heads (%d) and num_kv_heads (%d) must be positive",
                     num_q_heads, num_kv_heads);
  if (num_q_heads % num_kv_heads != 0)
    return set_error(NEO_ERR_INVALID_ARG, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)",
                     num_q_heads, num_kv_heads);
  const int32_t group = num_q_heads / num_kv_heads;
  if (head_dim != neo::cpu::kD)
    return set_error(NEO_ERR_UNSUPPORTED, "head_dim %d unsupported (128)", head_dim);
  if (block_size != neo::cpu::kBs)
    return set_error(NEO_ERR_UNSUPPORTED, "block_size %d unsupported (16)", block_size);
  if (group != 1 && group != 2 && group != 4 && group != 8 && group != 16)
    return set_error(NEO_ERR_UNSUPPORTED, "group size %d unsupported (1, 2, 4, 8, 16)", group);
  if (!std::isfinite(scale)) return set_error(NEO_ERR_INVALID_ARG, "scale must be finite");
  if (num_threads < 0)
    return set_error(NEO_ERR_INVALID_ARG, "num_threads (%d) is negative", num_threads);
  if (isa < NEO_CPU_ISA_AUTO || isa > NEO_CPU_ISA_AVX512)
    return set_error(NEO_ERR_UNSUPPORTED, "isa %d unknown", isa);
  if (isa == NEO_CPU_ISA_AVX512_BF16 && !neo::cpu::cpu_has_avx512_bf16())
    return set_error(NEO_ERR_UNSUPPORTED, "this CPU has no AVX-512 BF16");
  if (isa == NEO_CPU_ISA_AVX512 && !neo::cpu::cpu_has_avx512())
    return set_error(NEO_ERR_UNSUPPORTED, "this CPU has no AVX-512");
  if (batch == 0) return neo::clear_error();
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !out)
    return set_error(NEO_ERR_INVALID_ARG, "a required pointer is NULL");
  if (max_blocks_per_seq <= 0 || num_blocks <= 0)
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq and num_blocks must be positive");
  if ((int64_t)max_blocks_per_seq * neo::cpu::kBs >= ((int64_t)1 << 31))
    return set_error(NEO_ERR_INVALID_ARG, "max_blocks_per_seq too large");
  // Every block id in use is checked before any thread reads a tile.
  for (int64_t b = 0; b < batch; ++b) {
    const int32_t L = neo::cpu::clamp_len(seq_lens[b], max_blocks_per_seq);
    const int32_t* row = block_table + b * max_blocks_per_seq;
    for (int32_t j = 0; j < (L + neo::cpu::kBs - 1) / neo::cpu::kBs; ++j)
      if (row[j] < 0 || row[j] >= num_blocks)
        return set_error(NEO_ERR_INVALID_ARG,
                         "block_table[%lld][%d] = %d is outside [0, %d)", (long long)b, j,
                         row[j], num_blocks);
  }
  neo::cpu::Problem P{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_cache),
                      static_cast<const uint16_t*>(v_cache), block_table, seq_lens, out,
                      batch, num_q_heads, num_kv_heads, group, max_blocks_per_seq,
                      scale * neo::cpu::kLog2e};
  if (isa == NEO_CPU_ISA_AUTO) isa = neo::cpu::best_isa();
  const neo::cpu::TaskFn fn = isa == NEO_CPU_ISA_AVX512_BF16 ? neo::cpu::task_avx512_bf16
                              : isa == NEO_CPU_ISA_AVX512    ? neo::cpu::task_avx512
                                                             : neo::cpu::task_generic;
  const int threads = num_threads > 0 ? num_threads : neo::cpu::default_threads();
  neo::cpu::run(P, threads, fn);
  return neo::clear_error();
}

neo_status neo_cpu_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                                    const int32_t* block_table, const int32_t* seq_lens,
                                    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                    int32_t block_size, float scale, float* out, int32_t batch,
                                    int32_t max_blocks_per_seq, int32_t num_blocks,
                                    int32_t num_threads) {
  return neo_cpu_decode_attention_ex(q, k_cache, v_cache, block_table, seq_lens, num_q_heads,
                                     num_kv_heads, head_dim, block_size, scale, out, batch,
                                     max_blocks_per_seq, num_blocks, num_threads,
                                     NEO_CPU_ISA_AUTO);
}

}  // extern "C"
