// Host-only driver of the library's CPU-side code, built with sanitizers
// (AddressSanitizer + UndefinedBehaviorSanitizer, and separately
// ThreadSanitizer) by tests/test_host_sanitizers.py:
//
//  * the CPU decode attention (every instruction-set path this CPU has, 1-8
//    threads, requests split between threads, empty and single-token
//    requests, NaN in every slot no request may read) against the fp64
//    oracle, including two host threads calling it at once;
//  * the CPU cache append and read probe;
//  * the error paths of the CPU entry points;
//  * the load-aware scheduler simulator run to completion, with its
//    capacity and token-count invariants.
//
// Prints "ok ..." and exits 0 when every check passes.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <random>
#include <thread>
#include <vector>

#include "libneoattn.h"

extern "C" int neo_ref_decode_attention(const uint16_t* q, const uint16_t* k_cache,
                                        const uint16_t* v_cache, const int32_t* block_table,
                                        const int32_t* seq_lens, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim,
                                        int32_t block_size, double scale, float* out,
                                        double* out64, int32_t batch,
                                        int32_t max_blocks_per_seq, int32_t num_blocks,
                                        int64_t row_begin, int64_t row_end, int32_t num_threads);

namespace {

constexpr int kD = 128, kBs = 16;
constexpr uint16_t kNaN = 0x7FC0;
int g_failures = 0;

#define CHECK(cond, ...)                          \
  do {                                            \
    if (!(cond)) {                                \
      ++g_failures;                               \
      fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      fprintf(stderr, __VA_ARGS__);               \
      fprintf(stderr, "\n");                      \
    }                                             \
  } while (0)

uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFF + ((u >> 16) & 1);  // round to nearest even (inputs are finite)
  return (uint16_t)(u >> 16);
}

struct Case {
  int32_t batch, hq, hkv, mbps, nb;
  std::vector<int32_t> lens, table;
  std::vector<uint16_t> q, k, v;  // k: [nb][hkv][16][16][8], v: [nb][hkv][128][16]
};

// Shuffled physical blocks, 3 spare blocks, -1 table padding, N(0,1) values
// (x8 on ~2 % of key rows), NaN in unused tail slots and spare blocks.
Case make_case(const std::vector<int32_t>& lens, int32_t hq, int32_t hkv, uint64_t seed) {
  Case c;
  c.batch = (int32_t)lens.size();
  c.hq = hq;
  c.hkv = hkv;
  c.lens = lens;
  std::mt19937_64 rng(seed);
  std::normal_distribution<float> nd(0.f, 1.f);
  int32_t used = 0, mbps = 1;
  for (int32_t L : lens) {
    const int32_t n = (std::max(L, 0) + kBs - 1) / kBs;
    used += n;
    mbps = std::max(mbps, n);
  }
  c.mbps = mbps;
  c.nb = used + 3;
  std::vector<int32_t> perm(c.nb);
  for (int32_t i = 0; i < c.nb; ++i) perm[i] = i;
  std::shuffle(perm.begin(), perm.end(), rng);
  c.table.assign((size_t)c.batch * mbps, -1);
  const size_t tile = (size_t)kD * kBs;
  c.k.assign((size_t)c.nb * hkv * tile, kNaN);
  c.v.assign((size_t)c.nb * hkv * tile, kNaN);
  c.q.resize((size_t)c.batch * hq * kD);
  for (auto& x : c.q) x = to_bf16(nd(rng));
  int32_t next = 0;
  for (int32_t b = 0; b < c.batch; ++b) {
    const int32_t L = std::max(lens[b], 0);
    for (int32_t j = 0; j < (L + kBs - 1) / kBs; ++j) c.table[(size_t)b * mbps + j] = perm[next++];
    for (int32_t t = 0; t < L; ++t) {
      const int32_t blk = c.table[(size_t)b * mbps + t / kBs], slot = t % kBs;
      for (int32_t g = 0; g < hkv; ++g) {
        const float mul = (rng() % 50 == 0) ? 8.f : 1.f;
        const size_t base = ((size_t)blk * hkv + g) * tile;
        for (int d = 0; d < kD; ++d) {
          c.k[base + ((size_t)(d / 8) * kBs + slot) * 8 + d % 8] = to_bf16(mul * nd(rng));
          c.v[base + (size_t)d * kBs + slot] = to_bf16(nd(rng));
        }
      }
    }
  }
  return c;
}

// max abs error and max row-normwise relative error
void compare(const std::vector<float>& y, const std::vector<float>& r, double* ae, double* re) {
  *ae = 0;
  *re = 0;
  for (size_t row = 0; row < r.size() / kD; ++row) {
    double m = 0, rmax = 0;
    for (int d = 0; d < kD; ++d) {
      const double a = y[row * kD + d], b = r[row * kD + d];
      m = std::max(m, fabs(a - b));
      rmax = std::max(rmax, fabs(b));
      if (!std::isfinite(a)) m = INFINITY;
    }
    *ae = std::max(*ae, m);
    *re = std::max(*re, m / std::max(rmax, 1e-30));
  }
}

std::vector<float> oracle(const Case& c) {
  std::vector<float> out((size_t)c.batch * c.hq * kD, 0.f);
  const int rc = neo_ref_decode_attention(c.q.data(), c.k.data(), c.v.data(), c.table.data(),
                                          c.lens.data(), c.hq, c.hkv, kD, kBs,
                                          1.0 / sqrt((double)kD), out.data(), nullptr, c.batch,
                                          c.mbps, c.nb, 0, (int64_t)c.batch * c.hq, 1);
  CHECK(rc == 0, "oracle rc %d", rc);
  return out;
}

neo_status run_cpu(const Case& c, std::vector<float>& out, int32_t threads, int32_t isa) {
  out.assign((size_t)c.batch * c.hq * kD, NAN);
  return neo_cpu_decode_attention_ex(c.q.data(), c.k.data(), c.v.data(), c.table.data(),
                                     c.lens.data(), c.hq, c.hkv, kD, kBs,
                                     (float)(1.0 / sqrt((double)kD)), out.data(), c.batch,
                                     c.mbps, c.nb, threads, isa);
}

int check_attention() {
  const std::vector<std::vector<int32_t>> lens_sets = {
      {1, 15, 16, 17, 0, 100, 333, 2},
      {3000, 5, 1, 0, 700},
      {16, 16, 16, 16},
      {0, 0},
      {2047},
  };
  const int32_t shapes[][2] = {{8, 2}, {32, 8}, {4, 4}, {16, 1}};
  const int32_t isas[] = {NEO_CPU_ISA_GENERIC, NEO_CPU_ISA_AVX512, NEO_CPU_ISA_AVX512_BF16};
  int runs = 0;
  uint64_t seed = 1;
  for (const auto& lens : lens_sets) {
    for (const auto& sh : shapes) {
      const Case c = make_case(lens, sh[0], sh[1], seed++);
      const std::vector<float> ref = oracle(c);
      for (int32_t isa : isas) {
        for (int32_t threads : {1, 3, 8}) {
          std::vector<float> y;
          const neo_status st = run_cpu(c, y, threads, isa);
          if (st == NEO_ERR_UNSUPPORTED) continue;  // this CPU lacks the path
          CHECK(st == NEO_OK, "cpu attention status %d: %s", (int)st, neo_last_error());
          double ae, re;
          compare(y, ref, &ae, &re);
          CHECK(ae <= 1e-2 && re <= 2e-2, "isa %d threads %d: abs %g rel %g", isa, threads, ae, re);
          ++runs;
        }
      }
    }
  }
  return runs;
}

// Two host threads calling at once (the library serialises them).
void check_concurrent_calls() {
  const Case a = make_case({500, 90, 1, 1200}, 32, 8, 101);
  const Case b = make_case({64, 3000, 17}, 16, 4, 102);
  const std::vector<float> ra = oracle(a), rb = oracle(b);
  std::vector<float> ya, yb;
  neo_status sa = NEO_OK, sb = NEO_OK;
  std::thread ta([&] {
    for (int i = 0; i < 3 && sa == NEO_OK; ++i) sa = run_cpu(a, ya, 4, NEO_CPU_ISA_AUTO);
  });
  std::thread tb([&] {
    for (int i = 0; i < 3 && sb == NEO_OK; ++i) sb = run_cpu(b, yb, 5, NEO_CPU_ISA_AUTO);
  });
  ta.join();
  tb.join();
  CHECK(sa == NEO_OK && sb == NEO_OK, "concurrent calls: %d %d", (int)sa, (int)sb);
  double ae, re;
  compare(ya, ra, &ae, &re);
  CHECK(ae <= 1e-2 && re <= 2e-2, "concurrent a: abs %g rel %g", ae, re);
  compare(yb, rb, &ae, &re);
  CHECK(ae <= 1e-2 && re <= 2e-2, "concurrent b: abs %g rel %g", ae, re);
}

void check_append_probe_and_errors() {
  Case c = make_case({5, 16, 40, 0}, 8, 2, 201);
  std::vector<uint16_t> kn((size_t)c.batch * c.hkv * kD, 0x3F80), vn(kn.size(), 0x4000);
  CHECK(neo_cpu_kv_append(c.k.data(), c.v.data(), kn.data(), vn.data(), c.table.data(),
                          c.lens.data(), c.batch, c.mbps, c.hkv, kD, kBs, c.nb) == NEO_OK,
        "append: %s", neo_last_error());
  // Request 2's last token (t = 39) now holds 1.0 in K and 2.0 in V.
  const int32_t blk = c.table[(size_t)2 * c.mbps + 39 / kBs], slot = 39 % kBs;
  const size_t base = ((size_t)blk * c.hkv + 1) * kD * kBs;
  CHECK(c.k[base + ((size_t)5 * kBs + slot) * 8 + 3] == 0x3F80, "append K slot");
  CHECK(c.v[base + (size_t)77 * kBs + slot] == 0x4000, "append V slot");

  std::vector<uint8_t> buf(1 << 20, 1);
  double sum = 0;
  CHECK(neo_cpu_read_probe(buf.data(), buf.size(), 3, &sum) == NEO_OK, "probe: %s",
        neo_last_error());
  CHECK(neo_cpu_read_probe(buf.data(), 100, 3, &sum) == NEO_ERR_INVALID_ARG, "probe size");

  std::vector<float> out((size_t)c.batch * c.hq * kD);
  const float sc = 0.1f;
  CHECK(neo_cpu_decode_attention(nullptr, c.k.data(), c.v.data(), c.table.data(), c.lens.data(),
                                 c.hq, c.hkv, kD, kBs, sc, out.data(), c.batch, c.mbps, c.nb,
                                 2) == NEO_ERR_INVALID_ARG,
        "null q");
  CHECK(neo_cpu_decode_attention(c.q.data(), c.k.data(), c.v.data(), c.table.data(),
                                 c.lens.data(), c.hq, c.hkv, 64, kBs, sc, out.data(), c.batch,
                                 c.mbps, c.nb, 2) == NEO_ERR_UNSUPPORTED,
        "head_dim 64");
  std::vector<int32_t> bad = c.table;
  bad[(size_t)1 * c.mbps] = c.nb + 7;  // in use by request 1
  CHECK(neo_cpu_decode_attention(c.q.data(), c.k.data(), c.v.data(), bad.data(), c.lens.data(),
                                 c.hq, c.hkv, kD, kBs, sc, out.data(), c.batch, c.mbps, c.nb,
                                 2) == NEO_ERR_INVALID_ARG,
        "bad block id");
  CHECK(strlen(neo_last_error()) > 0, "error text");
  CHECK(neo_cpu_decode_attention(nullptr, nullptr, nullptr, nullptr, nullptr, c.hq, c.hkv, kD,
                                 kBs, sc, nullptr, 0, c.mbps, c.nb, 2) == NEO_OK,
        "empty batch");
}

// Per-layer stage times from bandwidth and flops (seconds): GPU attention at
// 5 TB/s, CPU attention at 150 GB/s, 512 B per (token, kv head) x 8 kv heads;
// the linear stage reads 436 MB of weights or computes 436 MFLOP per token.
void check_scheduler() {
  std::vector<double> b = {1, 16, 64, 256}, s = {256, 4096, 65536, 524288};
  std::vector<double> ga(16), ca(16);
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) {
      ga[i * 4 + j] = 18e-6 + s[j] * 4096 / 5e12 + b[i] * 1e-8;
      ca[i * 4 + j] = 25e-6 + s[j] * 4096 / 150e9 + b[i] * 1e-7;
    }
  std::vector<double> x = {1, 64, 512, 4096}, tl(4);
  for (int i = 0; i < 4; ++i) tl[i] = std::max(436e6 / 5e12, 2 * 218e6 * x[i] / 1.5e15);
  neo_sched_config cfg;
  memset(&cfg, 0, sizeof cfg);
  cfg.num_layers = 32;
  cfg.block_size = 16;
  cfg.gpu_blocks = 900;
  cfg.cpu_blocks = 6000;
  cfg.max_batch_tokens = 2048;
  cfg.swap_in_reserve_blocks = 8;
  cfg.t_ga = {4, 4, b.data(), s.data(), ga.data()};
  cfg.t_ca = {4, 4, b.data(), s.data(), ca.data()};
  cfg.t_l = {4, x.data(), tl.data()};
  cfg.policy = NEO_SCHED_POLICY_NEO;
  neo_sched* sch = nullptr;
  CHECK(neo_sched_create(&cfg, &sch) == NEO_OK && sch, "sched create: %s", neo_last_error());
  if (!sch) return;
  std::mt19937_64 rng(7);
  int64_t want_tokens = 0;
  for (int i = 0; i < 150; ++i) {
    const int32_t prompt = 64 + (int32_t)(rng() % 1500), output = 16 + (int32_t)(rng() % 300);
    want_tokens += output;
    CHECK(neo_sched_add_request(sch, i, prompt, output, 0.01 * (i % 10)) == NEO_OK, "add");
  }
  std::vector<int64_t> ids(4096);
  int64_t iters = 0;
  for (;;) {
    neo_sched_iter it;
    CHECK(neo_sched_step(sch, &it, ids.data(), (int64_t)ids.size()) == NEO_OK, "step: %s",
          neo_last_error());
    if (it.done) break;
    neo_sched_stats st;
    neo_sched_get_stats(sch, &st);
    CHECK(st.gpu_blocks_held <= cfg.gpu_blocks && st.cpu_blocks_held <= cfg.cpu_blocks,
          "capacity exceeded");
    if (++iters > 1000000) {
      CHECK(false, "scheduler did not finish");
      break;
    }
  }
  neo_sched_stats st;
  neo_sched_get_stats(sch, &st);
  CHECK(st.finished == 150 && st.tokens == want_tokens, "finished %lld tokens %lld want %lld",
        (long long)st.finished, (long long)st.tokens, (long long)want_tokens);
  neo_sched_destroy(sch);
  neo_sched_config bad = cfg;
  bad.num_layers = 0;
  neo_sched* none = nullptr;
  CHECK(neo_sched_create(&bad, &none) != NEO_OK && !none, "bad config accepted");
}

}  // namespace

int main() {
  const int runs = check_attention();
  check_concurrent_calls();
  check_append_probe_and_errors();
  check_scheduler();
  if (g_failures) {
    fprintf(stderr, "%d check(s) failed\n", g_failures);
    return 1;
  }
  printf("ok: %d attention runs against the oracle, concurrent calls, append, probe, errors, "
         "scheduler\n", runs);
  return 0;
}
