// Host-side checks of the library's C ABI, meant to run under AddressSanitizer and
// UndefinedBehaviorSanitizer on a host-only build of the library sources (no GPU needed and no
// kernel launched): the routing templates of Appendix B (every layout over many geometries,
// ragged and full attention, per-sequence and variable-length layouts) write exactly the words
// the caller sized, coverage and the fitted parameters stay in range, and the validation and
// workspace plans of every entry point reject bad arguments before any device call.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "tilemix.h"

namespace {

uint64_t g_state = 0x9e3779b97f4a7c15ull;
uint32_t rnd() {   // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return (uint32_t)((g_state * 0x2545f4914f6cdd1dull) >> 32);
}
int rnd_in(int lo, int hi) { return lo + (int)(rnd() % (uint32_t)(hi - lo + 1)); }
float rnd_unit() { return (float)(rnd() % 10001) / 10000.0f; }

int g_fail = 0;
void check(bool ok, const char* what, int line) {
  if (!ok) {
    ++g_fail;
    fprintf(stderr, "FAILED line %d: %s (%s)\n", line, what, tilemix_last_error());
  }
}
#define CHECK(x) check((x), #x, __LINE__)

tilemix_params random_params() {
  tilemix_params p{};
  p.batch = rnd_in(1, 3);
  p.heads_kv = rnd_in(1, 3);
  p.heads_q = p.heads_kv * (1 << rnd_in(0, 2));
  p.len_k = rnd_in(1, 3000);
  p.len_q = (rnd() & 1) ? p.len_k : rnd_in(1, 3000);
  p.head_dim = (rnd() & 1) ? 128 : 64;
  p.block_m = (rnd() & 1) ? 128 : 64;
  p.block_n = 64;
  p.group_size = rnd_in(1, 17);
  p.causal = (int32_t)(rnd() & 1);
  p.scale = 0.125f;
  p.route_per_batch = (int32_t)(rnd() & 1);
  p.route_hint = -1;
  return p;
}

tilemix_template random_template(int kind, const tilemix_params& p) {
  tilemix_template t{};
  t.kind = kind;
  t.band_w = kind == TILEMIX_TEMPLATE_BIGBIRD ? rnd_in(-1, 6) : rnd_in(0, 6);
  t.global_groups = rnd_in(0, 8);
  t.rand_fp16 = rnd_unit();
  t.align_alpha = (float)rnd_in(0, 4);
  t.align_beta = rnd_unit() * 2.0f;
  t.sp_stride = rnd_in(1, 2 * p.len_k + 64);
  t.sp_tail = rnd_in(0, 200);
  t.seed = ((uint64_t)rnd() << 32) | rnd();
  return t;
}

void templates_fixed(int iters) {
  for (int it = 0; it < iters; ++it) {
    tilemix_params p = random_params();
    const int W = tilemix_route_words_per_row(&p);
    CHECK(W >= 1);
    const long long T_m = (p.len_q + p.block_m - 1) / p.block_m;
    const long long B_r = p.route_per_batch ? p.batch : 1;
    const size_t n = (size_t)(B_r * p.heads_kv * T_m * W);
    for (int kind = 0; kind <= TILEMIX_TEMPLATE_SPTRANS; ++kind) {
      tilemix_template t = random_template(kind, p);
      std::vector<uint64_t> words(n, 0xdeadbeefull);   // exactly the caller's size
      CHECK(tilemix_route_template(&p, &t, words.data()) == TILEMIX_OK);
      double rg = -1.0, rp = -1.0;
      CHECK(tilemix_route_coverage(&p, words.data(), &rg, &rp) == TILEMIX_OK);
      CHECK(rg >= 0.0 && rg <= 1.0 && rp >= 0.0 && rp <= 1.0);
      if (kind == TILEMIX_TEMPLATE_ONE) CHECK(rg == 1.0 && rp == 1.0);
      if (kind == TILEMIX_TEMPLATE_ZERO) CHECK(rg == 0.0 && rp == 0.0);
      const double rho = (double)(rnd() % 5) / 4.0;
      tilemix_template f = t;
      CHECK(tilemix_fit_template(&p, &f, rho) == TILEMIX_OK);
      CHECK(tilemix_route_template(&p, &f, words.data()) == TILEMIX_OK);
    }
  }
}

void templates_varlen(int iters) {
  for (int it = 0; it < iters; ++it) {
    tilemix_params p = random_params();
    p.route_per_batch = 0;
    p.batch = rnd_in(1, 5);
    std::vector<int32_t> lq(p.batch), lk(p.batch);
    long long rows = 0;
    for (int b = 0; b < p.batch; ++b) {
      lq[b] = rnd_in(0, p.len_q);
      lk[b] = p.len_q == p.len_k ? lq[b] : rnd_in(0, p.len_k);
      rows += (lq[b] + p.block_m - 1) / p.block_m;
    }
    const int W = tilemix_route_words_per_row(&p);
    for (int kind = 0; kind <= TILEMIX_TEMPLATE_SPTRANS; ++kind) {
      tilemix_template t = random_template(kind, p);
      std::vector<uint64_t> words((size_t)(rows * p.heads_kv * W) + (rows == 0 ? 1 : 0), 0ull);
      CHECK(tilemix_route_template_varlen(&p, lq.data(), lk.data(), &t, words.data()) == TILEMIX_OK);
    }
  }
}

void validation() {
  tilemix_params p{};
  p.batch = 1; p.heads_q = 32; p.heads_kv = 8; p.len_q = 8192; p.len_k = 8192; p.head_dim = 128;
  p.block_m = 128; p.block_n = 64; p.group_size = 1; p.causal = 1; p.scale = 0.0884f;
  p.route_per_batch = 0; p.route_hint = -1;
  size_t bytes = 0;
  CHECK(tilemix_workspace_size(&p, &bytes) == TILEMIX_OK && bytes > 0);
  CHECK(tilemix_fused_workspace_size(&p, &bytes) == TILEMIX_OK && bytes > 0);
  CHECK(tilemix_varlen_workspace_size(&p, 1000, 1000, &bytes) == TILEMIX_OK && bytes > 0);
  CHECK(tilemix_varlen_fused_workspace_size(&p, 1000, 1000, &bytes) == TILEMIX_OK);
  CHECK(tilemix_workspace_size(&p, nullptr) == TILEMIX_ERR_NULL);
  CHECK(tilemix_workspace_size(nullptr, &bytes) == TILEMIX_ERR_NULL);
  // every field out of range
  int32_t tilemix_params::*ints[] = {&tilemix_params::batch, &tilemix_params::heads_q,
                                           &tilemix_params::heads_kv, &tilemix_params::len_q,
                                           &tilemix_params::len_k, &tilemix_params::head_dim,
                                           &tilemix_params::block_m, &tilemix_params::block_n,
                                           &tilemix_params::group_size, &tilemix_params::causal,
                                           &tilemix_params::route_per_batch,
                                           &tilemix_params::route_hint};
  const int32_t bad_values[] = {0, -1, 3, 96, 1 << 30, -2147483647 - 1};
  for (auto f : ints) {
    for (int32_t v : bad_values) {
      tilemix_params q = p;
      q.*f = v;
      (void)tilemix_workspace_size(&q, &bytes);   // must return, not crash
      (void)tilemix_route_words_per_row(&q);
    }
  }
  tilemix_params q = p;
  q.scale = -1.0f;
  CHECK(tilemix_workspace_size(&q, &bytes) == TILEMIX_ERR_SHAPE);
  q.scale = 1.0f / 0.0f;
  CHECK(tilemix_workspace_size(&q, &bytes) == TILEMIX_ERR_SHAPE);
  // entry points reject before any device call
  void* fake = (void*)(uintptr_t)0x100000;
  void* odd = (void*)(uintptr_t)0x100001;
  const uint64_t* fw = (const uint64_t*)fake;
  CHECK(tilemix_prefill(&p, nullptr, fake, fake, fw, fake, fake, 1ull << 40, nullptr) == TILEMIX_ERR_NULL);
  CHECK(tilemix_prefill(&p, odd, fake, fake, fw, fake, fake, 1ull << 40, nullptr) == TILEMIX_ERR_ALIGN);
  CHECK(tilemix_prefill(&p, fake, fake, fake, fw, fake, fake, 16, nullptr) == TILEMIX_ERR_WORKSPACE);
  CHECK(tilemix_prefill_fused(&p, fake, fake, fake, fw, fake, nullptr, 0, nullptr) == TILEMIX_ERR_WORKSPACE);
  CHECK(tilemix_prefill_varlen(&p, 0, 10, (const int32_t*)fake, (const int32_t*)fake, fake, fake, fake,
                               fw, 1, fake, fake, 1ull << 40, nullptr) == TILEMIX_ERR_SHAPE);
  CHECK(tilemix_prefill_varlen(&p, 10, 10, nullptr, (const int32_t*)fake, fake, fake, fake, fw, 1, fake,
                               fake, 1ull << 40, nullptr) == TILEMIX_ERR_NULL);
  CHECK(tilemix_prefill_varlen(&p, 10, 10, (const int32_t*)fake, (const int32_t*)fake, fake, fake, fake,
                               fw, -1, fake, fake, 1ull << 40, nullptr) == TILEMIX_ERR_SHAPE);
  CHECK(tilemix_prefill_varlen_fused(&p, 10, 10, (const int32_t*)odd, (const int32_t*)fake, fake, fake,
                                     fake, fw, 1, fake, fake, 1ull << 40, nullptr) == TILEMIX_ERR_ALIGN);
  tilemix_params big = p;
  big.batch = 4; big.heads_q = 64; big.len_q = 65536; big.len_k = 65536; big.group_size = 8;
  CHECK(tilemix_prefill_noalloc(&big, fake, fake, fake, fw, fake, nullptr) == TILEMIX_ERR_WORKSPACE);
  CHECK(tilemix_prefill_noalloc(&p, nullptr, fake, fake, fw, fake, nullptr) == TILEMIX_ERR_NULL);
  tilemix_debug_export ex{};
  CHECK(tilemix_debug_prefill(&p, 0, -1, -1, nullptr, nullptr, fake, fake, fake, fw, 0, fake, fake,
                              1ull << 40, &ex, nullptr) == TILEMIX_ERR_NULL);
  CHECK(tilemix_debug_qk_int32(&p, (const int8_t*)fake, (const int8_t*)fake, (const int32_t*)fake, -1,
                               (int32_t*)fake, nullptr) == TILEMIX_ERR_SHAPE);
  tilemix_params dp = p;
  dp.len_q = 1;
  CHECK(tilemix_decode_workspace_size(&dp, &bytes) == TILEMIX_OK && bytes > 0);
  CHECK(tilemix_decode_varlen(&dp, nullptr, fake, fake, (const int8_t*)fake, (const uint16_t*)fake,
                              (const int8_t*)fake, (const uint16_t*)fake, fw, fake, fake, 1ull << 40,
                              nullptr) == TILEMIX_ERR_NULL);
  CHECK(tilemix_decode(&p, fake, fake, (const int8_t*)fake, (const uint16_t*)fake, (const int8_t*)fake,
                       (const uint16_t*)fake, fw, fake, fake, 1ull << 40, nullptr) == TILEMIX_ERR_UNSUPPORTED);
  // template argument errors
  tilemix_template t{};
  t.kind = 99;
  std::vector<uint64_t> w(4096);
  CHECK(tilemix_route_template(&p, &t, w.data()) != TILEMIX_OK);
  t.kind = TILEMIX_TEMPLATE_BAND;
  t.band_w = -5;
  CHECK(tilemix_route_template(&p, &t, w.data()) != TILEMIX_OK);
  CHECK(tilemix_route_template(&p, nullptr, w.data()) == TILEMIX_ERR_NULL);
  for (int len = -3; len < 300000; len += 997) (void)tilemix_auto_group_size(len, 64);
  CHECK(tilemix_auto_group_size(0, 64) == 0);
  for (int s = 0; s <= 6; ++s) CHECK(tilemix_status_string((tilemix_status)s)[0] != '\0');
}

// A deliberately undersized routing-word buffer (one word short): under AddressSanitizer the
// template write past its end must be reported, which shows that the library code is
// instrumented.
int undersized() {
  tilemix_params p{};
  p.batch = 1; p.heads_q = 2; p.heads_kv = 1; p.len_q = 1000; p.len_k = 1000; p.head_dim = 128;
  p.block_m = 128; p.block_n = 64; p.group_size = 1; p.causal = 1; p.scale = 0.0884f;
  p.route_per_batch = 0; p.route_hint = -1;
  tilemix_template t{};
  t.kind = TILEMIX_TEMPLATE_ONE;
  const int W = tilemix_route_words_per_row(&p);
  std::vector<uint64_t> words((size_t)(8 * W) - 1);
  return tilemix_route_template(&p, &t, words.data()) == TILEMIX_OK ? 0 : 1;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc > 1) return undersized();
  validation();
  templates_fixed(600);
  templates_varlen(400);
  if (g_fail) {
    fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  printf("host ABI checks ok\n");
  return 0;
}
