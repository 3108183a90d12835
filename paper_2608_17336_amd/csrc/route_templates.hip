// route_templates.hip -- host-side routing templates, coverage accounting and the automatic
// group size of Appendix B (TileMix, arXiv 2608.17336).  Plain C++ on the host: a template is
// a data-free 2-D map R[m, g_j] (1 = INT8, 0 = FP16) over query-tile rows m and key-tile
// groups g_j, broadcast over KV heads and packed into the routing words the fused kernel
// reads (Section 4.2, "Bitmask packing").
//
// Row m's legal groups G_m: because every query's legal keys form a prefix [0, last(i)] of the
// keys, G_m is the prefix {0, ..., gmax(m)} with gmax(m) = floor(last(q_hi(m)) / span), span =
// g * BLOCK_N the keys per group and last(i) = min(L_k - 1, i + L_k - L_q) (bottom-right causal)
// or L_k - 1 (full attention).  A row whose last query sees no key has no legal group.
// Every template chooses its FP16 set F_m inside G_m; bits outside G_m stay 0.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "tilemix.h"
#include "tilemix_internal.h"

namespace {

using tilemix::api::fail;
using tilemix::api::ok;

struct Geometry {
  long long Lq, Lk, BM, BN, g, span, T_m, T_mask, W, off;
  bool causal;
  // Lengths default to the params' (one sequence); a sequence of a variable-length batch
  // passes its own.
  explicit Geometry(const tilemix_params& p, long long len_q = -1, long long len_k = -1) {
    Lq = len_q >= 0 ? len_q : p.len_q;
    Lk = len_k >= 0 ? len_k : p.len_k;
    BM = p.block_m; BN = p.block_n; g = p.group_size;
    span = g * BN;
    T_m = (Lq + BM - 1) / BM;
    T_mask = ((Lk + BN - 1) / BN + g - 1) / g;
    W = (T_mask + 63) / 64;
    causal = p.causal != 0;
    off = Lk - Lq;
  }
  long long q_lo(long long m) const { return m * BM; }
  long long q_hi(long long m) const { return std::min(Lq, (m + 1) * BM) - 1; }
  long long last_key(long long i) const { return causal ? std::min(Lk - 1, i + off) : Lk - 1; }
  // Largest legal group of row m, or -1 when the row has none.
  long long gmax(long long m) const {
    const long long last = last_key(q_hi(m));
    return last < 0 ? -1 : last / span;
  }
  long long k_lo(long long gj) const { return gj * span; }
  long long k_hi(long long gj) const { return std::min(Lk, (gj + 1) * span) - 1; }
};

// SplitMix64 output function (Steele, Lea and Flood, 2014): the 64-bit value the generator
// returns from state x.  Used counter-style: the sampling key of (row m, group g) is
// mix64(seed ^ (m << 32 | g)).
uint64_t mix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// FP16 set of row m as a 0/1 vector over groups 0 .. T_mask - 1 (only legal groups set).
void fp16_row(const Geometry& G, const tilemix_template& t, long long m, std::vector<uint8_t>& f) {
  std::fill(f.begin(), f.end(), 0);
  const long long gm = G.gmax(m);
  if (gm < 0) return;
  const long long n_legal = gm + 1;
  auto set_range = [&](long long lo, long long hi) {
    lo = std::max(lo, 0LL);
    hi = std::min(hi, gm);
    for (long long x = lo; x <= hi; ++x) f[x] = 1;
  };
  auto band = [&](long long w) {   // |g_j - gamma(m)| <= w, gamma(m) = floor(m BLOCK_M / span)
    const long long gamma = (m * G.BM) / G.span;
    set_range(gamma - w, gamma + w);
  };
  auto global = [&](long long k) { set_range(0, k - 1); };
  auto rowrand = [&](double frac) {   // round((1 - rho) |G_m|) groups, uniform w/o replacement
    const long long k = (long long)floor(frac * (double)n_legal + 0.5);
    if (k <= 0) return;
    std::vector<std::pair<uint64_t, long long>> keys((size_t)n_legal);
    for (long long x = 0; x < n_legal; ++x)
      keys[(size_t)x] = {mix64(t.seed ^ (((uint64_t)m << 32) | (uint64_t)x)), x};
    const long long take = std::min(k, n_legal);
    std::partial_sort(keys.begin(), keys.begin() + take, keys.end());
    for (long long x = 0; x < take; ++x) f[keys[(size_t)x].second] = 1;
  };
  switch (t.kind) {
    case TILEMIX_TEMPLATE_ONE:
      return;
    case TILEMIX_TEMPLATE_ZERO:
      set_range(0, gm);
      return;
    case TILEMIX_TEMPLATE_BAND:
      band(t.band_w);
      return;
    case TILEMIX_TEMPLATE_GLOBAL:
      global(t.global_groups);
      return;
    case TILEMIX_TEMPLATE_ROWRAND:
      rowrand(t.rand_fp16);
      return;
    case TILEMIX_TEMPLATE_ALIGNED: {   // the last a(m) = min(|G_m|, ceil(alpha + beta m)) groups
      const double a = ceil((double)t.align_alpha + (double)t.align_beta * (double)m);
      const long long am = std::min(n_legal, (long long)std::max(0.0, a));
      set_range(gm - am + 1, gm);
      return;
    }
    case TILEMIX_TEMPLATE_BIGBIRD:
      if (t.band_w >= 0) band(t.band_w);
      global(t.global_groups);
      rowrand(t.rand_fp16);
      return;
    case TILEMIX_TEMPLATE_SPTRANS: {
      // Keys in FP16 for some query i of the row (key coordinate i' = i + L_k - L_q): the union
      // over i of [u(i') s, i'] and of the tails [max(r s, (r+1) s - c), (r+1) s - 1] of the
      // strides r < u(i').  Over the row this is [u(i_lo') s, i_hi'] plus the tails of every
      // stride r < u(i_hi').
      const long long s = t.sp_stride, c = std::min<long long>(t.sp_tail, s);
      const long long lo_i = std::max(G.q_lo(m) + G.off, 0LL), hi_i = G.q_hi(m) + G.off;
      if (hi_i < 0) return;
      const long long local_lo = (lo_i / s) * s, u_hi = hi_i / s;
      for (long long x = 0; x <= gm; ++x) {
        const long long a = G.k_lo(x), b = G.k_hi(x);
        bool hit = a <= hi_i && b >= local_lo;
        const long long r0 = a / s;
        if (!hit && c > 0 && r0 < u_hi && r0 <= b / s) hit = (r0 + 1) * s - c <= b;
        f[x] = hit ? 1 : 0;
      }
      return;
    }
    default:
      return;
  }
}

tilemix_status check_template(const tilemix_template* t) {
  if (!t) return fail(TILEMIX_ERR_NULL, "template is NULL");
  switch (t->kind) {
    case TILEMIX_TEMPLATE_ONE:
    case TILEMIX_TEMPLATE_ZERO:
      return TILEMIX_OK;
    case TILEMIX_TEMPLATE_BAND:
      if (t->band_w < 0) return fail(TILEMIX_ERR_SHAPE, "band_w must be >= 0");
      return TILEMIX_OK;
    case TILEMIX_TEMPLATE_GLOBAL:
      if (t->global_groups < 0) return fail(TILEMIX_ERR_SHAPE, "global_groups must be >= 0");
      return TILEMIX_OK;
    case TILEMIX_TEMPLATE_BIGBIRD:
      if (t->band_w < -1 || t->global_groups < 0)
        return fail(TILEMIX_ERR_SHAPE, "BigBird needs band_w >= -1 and global_groups >= 0");
      [[fallthrough]];
    case TILEMIX_TEMPLATE_ROWRAND:
      if (!(t->rand_fp16 >= 0.0f && t->rand_fp16 <= 1.0f))
        return fail(TILEMIX_ERR_SHAPE, "rand_fp16 must lie in [0, 1]");
      return TILEMIX_OK;
    case TILEMIX_TEMPLATE_ALIGNED:
      if (!(isfinite(t->align_alpha) && isfinite(t->align_beta)))
        return fail(TILEMIX_ERR_SHAPE, "align_alpha and align_beta must be finite");
      return TILEMIX_OK;
    case TILEMIX_TEMPLATE_SPTRANS:
      if (t->sp_stride < 1 || t->sp_tail < 0)
        return fail(TILEMIX_ERR_SHAPE, "SpTrans needs sp_stride >= 1 and sp_tail >= 0");
      return TILEMIX_OK;
  }
  return fail(TILEMIX_ERR_UNSUPPORTED, "unknown template kind %d", t->kind);
}

// Realized INT8 coverage of a 2-D template (FP16 sets from fp16_row) over legal groups.
double template_coverage(const Geometry& G, const tilemix_template& t) {
  std::vector<uint8_t> f((size_t)G.T_mask);
  long long legal = 0, fp16 = 0;
  for (long long m = 0; m < G.T_m; ++m) {
    const long long gm = G.gmax(m);
    if (gm < 0) continue;
    fp16_row(G, t, m, f);
    legal += gm + 1;
    for (long long x = 0; x <= gm; ++x) fp16 += f[x];
  }
  return legal ? (double)(legal - fp16) / (double)legal : 0.0;
}

}  // namespace

extern "C" {

int32_t tilemix_auto_group_size(int32_t len_k, int32_t block_n) {
  if (len_k < 1 || block_n < 1) return 0;
  // b_64 = ceil(L_k / 64); BLOCK_N^mask = BLOCK_N ceil(max(b_64, BLOCK_N) / BLOCK_N);
  // g = BLOCK_N^mask / BLOCK_N.
  const long long b64 = ((long long)len_k + 63) / 64;
  const long long mx = std::max<long long>(b64, block_n);
  return (int32_t)((mx + block_n - 1) / block_n);
}

tilemix_status tilemix_route_template(const tilemix_params* params, const tilemix_template* tmpl,
                                      uint64_t* words) {
  tilemix_status st = tilemix::api::validate(params);
  if (st != TILEMIX_OK) return st;
  if ((st = check_template(tmpl)) != TILEMIX_OK) return st;
  if (!words) return fail(TILEMIX_ERR_NULL, "words is NULL");
  const Geometry G(*params);
  const size_t row_words = (size_t)G.W;
  std::vector<uint8_t> f((size_t)G.T_mask);
  std::vector<uint64_t> plane((size_t)G.T_m * row_words, 0ull);
  for (long long m = 0; m < G.T_m; ++m) {
    fp16_row(G, *tmpl, m, f);
    uint64_t* row = plane.data() + (size_t)m * row_words;
    for (long long x = 0; x <= G.gmax(m); ++x)
      if (!f[x]) row[x >> 6] |= 1ull << (x & 63);
  }
  const long long planes = (long long)(params->route_per_batch ? params->batch : 1) * params->heads_kv;
  for (long long h = 0; h < planes; ++h)
    memcpy(words + (size_t)h * plane.size(), plane.data(), plane.size() * sizeof(uint64_t));
  return ok();
}

tilemix_status tilemix_route_template_varlen(const tilemix_params* params, const int32_t* seqlens_q,
                                             const int32_t* seqlens_k, const tilemix_template* tmpl,
                                             uint64_t* words) {
  tilemix_status st = tilemix::api::validate(params);
  if (st != TILEMIX_OK) return st;
  if ((st = check_template(tmpl)) != TILEMIX_OK) return st;
  if (!words || !seqlens_q || !seqlens_k) return fail(TILEMIX_ERR_NULL, "NULL pointer");
  const long long W = Geometry(*params).W;   // words per row of the longest key sequence
  std::vector<uint8_t> f;
  uint64_t* out = words;
  for (int b = 0; b < params->batch; ++b) {
    if (seqlens_q[b] < 0 || seqlens_q[b] > params->len_q || seqlens_k[b] < 0 ||
        seqlens_k[b] > params->len_k)
      return fail(TILEMIX_ERR_SHAPE, "sequence %d has lengths (%d, %d) outside [0, (%d, %d)]", b,
                  seqlens_q[b], seqlens_k[b], params->len_q, params->len_k);
    const Geometry G(*params, seqlens_q[b], seqlens_k[b]);
    f.assign((size_t)std::max(1LL, G.T_mask), 0);
    for (long long m = 0; m < G.T_m; ++m) {
      fp16_row(G, *tmpl, m, f);
      std::vector<uint64_t> row((size_t)W, 0ull);
      for (long long x = 0; x <= G.gmax(m); ++x)
        if (!f[x]) row[x >> 6] |= 1ull << (x & 63);
      for (int h = 0; h < params->heads_kv; ++h, out += W) memcpy(out, row.data(), W * sizeof(uint64_t));
    }
  }
  return ok();
}

tilemix_status tilemix_route_coverage(const tilemix_params* params, const uint64_t* words,
                                      double* rho_groups, double* rho_pairs) {
  tilemix_status st = tilemix::api::validate(params);
  if (st != TILEMIX_OK) return st;
  if (!words || !rho_groups || !rho_pairs) return fail(TILEMIX_ERR_NULL, "NULL pointer");
  const Geometry G(*params);
  const long long planes = (long long)(params->route_per_batch ? params->batch : 1) * params->heads_kv;
  long long n_groups = 0, int8_groups = 0;
  double n_pairs = 0.0, int8_pairs = 0.0;
  for (long long m = 0; m < G.T_m; ++m) {
    const long long gm = G.gmax(m);
    for (long long x = 0; x <= gm; ++x) {
      // legal (query, key) pairs of the row/group rectangle
      long long pairs = 0;
      for (long long i = G.q_lo(m); i <= G.q_hi(m); ++i)
        pairs += std::max(0LL, std::min(G.k_hi(x), G.last_key(i)) - G.k_lo(x) + 1);
      if (pairs == 0) continue;
      for (long long h = 0; h < planes; ++h) {
        const uint64_t w = words[((size_t)h * G.T_m + m) * G.W + (x >> 6)];
        const int bit = (int)((w >> (x & 63)) & 1ull);
        ++n_groups;
        int8_groups += bit;
        n_pairs += (double)pairs;
        if (bit) int8_pairs += (double)pairs;
      }
    }
  }
  *rho_groups = n_groups ? (double)int8_groups / (double)n_groups : 0.0;
  *rho_pairs = n_pairs > 0.0 ? int8_pairs / n_pairs : 0.0;
  return ok();
}

tilemix_status tilemix_fit_template(const tilemix_params* params, tilemix_template* tmpl,
                                    double rho_int8) {
  tilemix_status st = tilemix::api::validate(params);
  if (st != TILEMIX_OK) return st;
  if (!tmpl) return fail(TILEMIX_ERR_NULL, "template is NULL");
  if (!(rho_int8 >= 0.0 && rho_int8 <= 1.0)) return fail(TILEMIX_ERR_SHAPE, "rho_int8 must lie in [0, 1]");
  const Geometry G(*params);
  tilemix_template t = *tmpl;
  auto cov = [&](const tilemix_template& x) { return template_coverage(G, x); };
  // Integer parameter p in [lo, hi] whose coverage is closest to rho_int8 (first such p).
  auto best_int = [&](int32_t tilemix_template::*field, long long lo, long long hi) {
    long long best = lo;
    double err = 2.0;
    for (long long p = lo; p <= hi; ++p) {
      t.*field = (int32_t)p;
      const double e = fabs(cov(t) - rho_int8);
      if (e < err) { err = e; best = p; }
    }
    t.*field = (int32_t)best;
  };
  // Real parameter in [lo, hi] on which coverage decreases: bisection to rho_int8.
  auto bisect = [&](float tilemix_template::*field, double lo, double hi) {
    for (int it = 0; it < 60; ++it) {
      const double mid = 0.5 * (lo + hi);
      t.*field = (float)mid;
      if (cov(t) > rho_int8) lo = mid; else hi = mid;
    }
    t.*field = (float)lo;
    const double e_lo = fabs(cov(t) - rho_int8);
    t.*field = (float)hi;
    if (fabs(cov(t) - rho_int8) > e_lo) t.*field = (float)lo;
  };
  switch (t.kind) {
    case TILEMIX_TEMPLATE_ONE:
    case TILEMIX_TEMPLATE_ZERO:
      break;
    case TILEMIX_TEMPLATE_BAND:
      best_int(&tilemix_template::band_w, 0, G.T_mask);
      break;
    case TILEMIX_TEMPLATE_GLOBAL:
      best_int(&tilemix_template::global_groups, 0, G.T_mask);
      break;
    case TILEMIX_TEMPLATE_ROWRAND:
      t.rand_fp16 = (float)(1.0 - rho_int8);
      break;
    case TILEMIX_TEMPLATE_ALIGNED:
      t.align_alpha = 1.0f;
      bisect(&tilemix_template::align_beta, 0.0, (double)G.T_mask);
      break;
    case TILEMIX_TEMPLATE_BIGBIRD:
      t.band_w = 0;
      t.global_groups = 1;
      bisect(&tilemix_template::rand_fp16, 0.0, 1.0);
      break;
    case TILEMIX_TEMPLATE_SPTRANS:
      if (t.sp_stride < 1) return fail(TILEMIX_ERR_SHAPE, "SpTrans fitting needs sp_stride >= 1");
      best_int(&tilemix_template::sp_tail, 0, t.sp_stride);
      break;
    default:
      return fail(TILEMIX_ERR_UNSUPPORTED, "unknown template kind %d", t.kind);
  }
  *tmpl = t;
  return ok();
}

}  // extern "C"
