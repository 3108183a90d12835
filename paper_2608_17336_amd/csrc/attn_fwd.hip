// attn_fwd.hip -- fused routed prefill attention for gfx950 (TileMix, arXiv 2608.17336).
//
// One workgroup owns one routed tile row: query tile m (BLOCK_M rows) of one query head.
// It has BLOCK_M/32 waves; each wave owns 32 query rows.  The inner loop streams key
// tiles n of 64 keys through double-buffered LDS and, per tile:
//   1. reads the tile's routing bit: group g_j = n / g, word g_j / 64, bit g_j % 64
//      (Section 4.2, constant-time lookup).  The bit is the same for the whole
//      workgroup, so one branch selects which K form (FP16 K or INT8 K8) is staged;
//   2. computes the transposed score tile S^T (keys x queries) on the matrix cores:
//        FP16 route: v_mfma_f32_32x32x16_f16, K from LDS x Q from registers;
//        INT8 route: v_mfma_i32_32x32x32_i8 on the quantize-once codes, exact INT32,
//                    then one FP32 factor scale*log2(e)*dQ*dK (Appendix C rescale);
//      with keys on the matrix rows, every lane holds all scores of one query row for
//      16 keys of each 32-key block, so row max / row sum are in-lane plus one exchange
//      between the two half-waves;
//   3. updates the shared online-softmax state of Section 3.1 in FP32 (running max in
//      the log2 domain, normalizer, output accumulator).  The accumulator is rescaled
//      only when a row's max grows by more than 2^8, which leaves the result unchanged
//      and keeps P <= 256 in FP16;
//   4. packs P to FP16 in registers, in exactly the operand layout the P.V step needs,
//      and accumulates O^T += V^T P^T (v_mfma_f32_32x32x16_f16, FP32 accumulate).
// Legality (causal, sequence end) is applied only on tiles that cross it; tiles past
// the last legal key of the workgroup are never visited and waves whose rows see no
// key of a tile skip its math.  Rows are scheduled longest-first, and consecutive
// workgroups on one XCD share a KV head when the KV stream count allows it.
#include "tilemix_device.h"
#include "tilemix_internal.h"

namespace tilemix {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleThreshold = 8.0f;   // log2 units: rescale when the max grows > x256
constexpr float kNegInf = -__builtin_huge_valf();

template <int D, int BM>
struct TileCfg {
  static constexpr int kWaves = BM / 32;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int kKBytes = kBlockN * D * 2;     // FP16 K tile (K8 uses half of it)
  static constexpr int kVBytes = D * kBlockN * 2;     // V^T tile
  static constexpr int kStage = kKBytes + kVBytes;
  static constexpr int kKChunks = kKBytes / 16 / kThreads;   // 16-byte loads per thread
  static constexpr int kK8Chunks = kKChunks / 2;
  static constexpr int kVChunks = kVBytes / 16 / kThreads;
  static_assert(kKChunks * kThreads * 16 == kKBytes, "K split");
  static_assert(kK8Chunks * 2 == kKChunks, "K8 split");
  static_assert(kVChunks * kThreads * 16 == kVBytes, "V split");
};

// Registers holding one prefetched K/V tile on its way from HBM to LDS.
template <int D, int BM>
struct Prefetch {
  uint4 k[TileCfg<D, BM>::kKChunks];
  uint4 v[TileCfg<D, BM>::kVChunks];
};

template <int D, int BM, bool WITH_V>
__device__ __forceinline__ void load_tile(Prefetch<D, BM>& pf, const _Float16* __restrict__ K,
                                          const int8_t* __restrict__ K8,
                                          const _Float16* __restrict__ Vt, int b, int hk, int n,
                                          int Lk, int Hk, int T_n, bool int8) {
  using C = TileCfg<D, BM>;
  const int tid = threadIdx.x;
  const int key0 = n * kBlockN;
  if (!int8) {
#pragma unroll
    for (int i = 0; i < C::kKChunks; ++i) {
      const int c = tid + C::kThreads * i;
      const int row = c / (D / 8), ch = c % (D / 8);
      const int key = key0 + row;
      pf.k[i] = (key < Lk) ? ld_global_16(K + (((size_t)b * Lk + key) * Hk + hk) * D + ch * 8)
                           : make_uint4(0, 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < C::kK8Chunks; ++i) {
      const int c = tid + C::kThreads * i;
      const int row = c / (D / 16), ch = c % (D / 16);
      const int key = key0 + row;
      pf.k[i] = (key < Lk) ? ld_global_16(K8 + (((size_t)b * Lk + key) * Hk + hk) * D + ch * 16)
                           : make_uint4(0, 0, 0, 0);
    }
  }
  if constexpr (WITH_V) {
    const _Float16* vt = Vt + (((size_t)b * Hk + hk) * T_n + n) * (size_t)(D * kBlockN);
#pragma unroll
    for (int i = 0; i < C::kVChunks; ++i) {
      const int c = tid + C::kThreads * i;
      pf.v[i] = ld_global_16(vt + c * 8);
    }
  }
}

template <int D, int BM, bool WITH_V>
__device__ __forceinline__ void store_tile(const Prefetch<D, BM>& pf, char* stage, bool int8) {
  using C = TileCfg<D, BM>;
  const int tid = threadIdx.x;
  if (!int8) {
#pragma unroll
    for (int i = 0; i < C::kKChunks; ++i) {
      const int c = tid + C::kThreads * i;
      st_lds_16(stage, swz<2 * D>(c / (D / 8), c % (D / 8)), pf.k[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < C::kK8Chunks; ++i) {
      const int c = tid + C::kThreads * i;
      st_lds_16(stage, swz<D>(c / (D / 16), c % (D / 16)), pf.k[i]);
    }
  }
  if constexpr (WITH_V) {
    char* vs = stage + C::kKBytes;
#pragma unroll
    for (int i = 0; i < C::kVChunks; ++i) {
      const int c = tid + C::kThreads * i;
      st_lds_16(vs, swz<128>(c / 8, c % 8), pf.v[i]);
    }
  }
}

// S^T tile (64 keys x 32 queries of this wave) by the INT8 route: exact INT32 products.
template <int D>
__device__ __forceinline__ void qk_int8(const char* kst, const i32x4 (&q8f)[D / 32], int lane,
                                        i32x16& acc0, i32x16& acc1) {
  const int lq = lane & 31, hi = lane >> 5;
  acc0 = i32x16{};
  acc1 = i32x16{};
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    const i32x4 a0 = as_i32x4(ld_lds_16(kst, swz<D>(lq, 2 * s + hi)));
    const i32x4 a1 = as_i32x4(ld_lds_16(kst, swz<D>(32 + lq, 2 * s + hi)));
    acc0 = mfma_i8(a0, q8f[s], acc0);
    acc1 = mfma_i8(a1, q8f[s], acc1);
  }
}

// S^T tile by the FP16 route: FP16 products, FP32 accumulation.
template <int D>
__device__ __forceinline__ void qk_fp16(const char* kst, const half8 (&qf)[D / 16], int lane,
                                        f32x16& acc0, f32x16& acc1) {
  const int lq = lane & 31, hi = lane >> 5;
  acc0 = f32x16{};
  acc1 = f32x16{};
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    const half8 a0 = as_half8(ld_lds_16(kst, swz<2 * D>(lq, 2 * s + hi)));
    const half8 a1 = as_half8(ld_lds_16(kst, swz<2 * D>(32 + lq, 2 * s + hi)));
    acc0 = mfma_f16(a0, qf[s], acc0);
    acc1 = mfma_f16(a1, qf[s], acc1);
  }
}

// Map a linear workgroup id to (b, h_q, m): rows longest first (largest m first for causal
// attention); when the number of KV streams (b, h_k) is a multiple of 8, workgroups that
// share an XCD (id % 8) walk the same KV streams, so their K/V tiles meet in one L2.
__device__ __forceinline__ void decode_unit(int id, int B, int Hq, int Hk, int T_m, int& b,
                                            int& hq, int& hk, int& m) {
  const int G = Hq / Hk;
  const int P = B * Hk;
  int m_rev, p, qg;
  if ((P & 7) == 0) {
    const int x = id & 7, j = id >> 3;
    const int per_m = (P >> 3) * G;
    m_rev = j / per_m;
    const int rem = j - m_rev * per_m;
    p = (rem / G) * 8 + x;
    qg = rem % G;
  } else {
    const int per_m = P * G;
    m_rev = id / per_m;
    const int rem = id - m_rev * per_m;
    p = rem / G;
    qg = rem % G;
  }
  m = T_m - 1 - m_rev;
  b = p / Hk;
  hk = p - b * Hk;
  hq = hk * G + qg;
}

template <int D, int BM>
__global__ __launch_bounds__(2 * BM, 2) void routed_attn_fwd_kernel(AttnArgs a) {
  using C = TileCfg<D, BM>;
  __shared__ __align__(16) char smem[2 * C::kStage];

  int b, hq, hk, m;
  decode_unit(blockIdx.x, a.B, a.Hq, a.Hk, a.T_m, b, hq, hk, m);

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid & (kWave - 1);
  const int lq = lane & 31, hi = lane >> 5;
  const int q0 = m * BM + 32 * wave;          // first query row of this wave
  const int my_q = q0 + lq;
  const int off = a.Lk - a.Lq;                // bottom-right causal alignment
  const bool wave_active = q0 < a.Lq;

  // Last key any row of the workgroup / of this wave may see.
  const int wg_last_q = min(a.Lq - 1, m * BM + BM - 1);
  int wg_last_key = a.causal ? min(a.Lk - 1, wg_last_q + off) : a.Lk - 1;
  const int wave_last_q = min(a.Lq - 1, q0 + 31);
  const int wave_last_key = a.causal ? min(a.Lk - 1, wave_last_q + off) : a.Lk - 1;

  _Float16* orow = a.O + (((size_t)b * a.Lq + my_q) * a.Hq + hq) * D;
  if (wg_last_key < 0) {   // no legal key for any row of this tile: output is zero
    if (my_q < a.Lq) {   // the two lanes of a row each clear half of it
#pragma unroll
      for (int c = 0; c < D / 2; c += 8) *reinterpret_cast<half8*>(orow + hi * (D / 2) + c) = half8{};
    }
    return;
  }
  const int n_end = wg_last_key / kBlockN;

  const uint64_t* route_row =
      a.route + (size_t)b * a.route_batch_stride + ((size_t)hk * a.T_m + m) * a.W;
  auto route_of = [&](int n) -> bool {
    if (a.force_fp16) return false;
    const int gj = n / a.g;
    return (route_row[gj >> 6] >> (gj & 63)) & 1ull;
  };

  // Which operand forms this row needs (looked up once per row).
  bool need_int8 = false, need_fp16 = false;
  {
    const int g_last = n_end / a.g;
    for (int w = 0; w <= (g_last >> 6); ++w) {
      const int nb = min(64, g_last - 64 * w + 1);
      const uint64_t valid = (nb >= 64) ? ~0ull : ((1ull << nb) - 1ull);
      const uint64_t word = a.force_fp16 ? 0ull : route_row[w];
      need_int8 |= (word & valid) != 0ull;
      need_fp16 |= (~word & valid) != 0ull;
    }
  }

  // Q operands of this wave, kept in registers for the whole row.
  half8 qf[D / 16];
  i32x4 q8f[D / 32];
  const bool row_ok = my_q < a.Lq;
  const size_t qoff = (((size_t)b * a.Lq + (row_ok ? my_q : 0)) * a.Hq + hq) * D;
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
    qf[s] = (need_fp16 && row_ok) ? as_half8(ld_global_16(a.Q + qoff + 16 * s + 8 * hi)) : half8{};
#pragma unroll
  for (int s = 0; s < D / 32; ++s)
    q8f[s] = (need_int8 && row_ok) ? as_i32x4(ld_global_16(a.Q8 + qoff + 32 * s + 16 * hi)) : i32x4{};
  const float dq = (need_int8 && wave_active)
                       ? half_bits_to_float(a.dQ[((size_t)b * a.nQB + q0 / kQuantBlockQ) * a.Hq + hq])
                       : 0.0f;

  // Online-softmax state (Section 3.1), FP32; max kept in log2 units.
  float m_run = kNegInf;
  float z_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) oacc[c] = f32x16{};

  Prefetch<D, BM> pf;
  bool r_cur = route_of(0);
  load_tile<D, BM, true>(pf, a.K, a.K8, a.Vt, b, hk, 0, a.Lk, a.Hk, a.T_n, r_cur);
  store_tile<D, BM, true>(pf, smem, r_cur);
  __syncthreads();

  for (int n = 0; n <= n_end; ++n) {
    char* kst = smem + (n & 1) * C::kStage;
    const char* vst = kst + C::kKBytes;
    const bool has_next = n < n_end;
    bool r_next = false;
    if (has_next) {
      r_next = route_of(n + 1);
      load_tile<D, BM, true>(pf, a.K, a.K8, a.Vt, b, hk, n + 1, a.Lk, a.Hk, a.T_n, r_next);
    }

    const int key0 = n * kBlockN;
    if (wave_active && key0 <= wave_last_key) {
      float sv[32];
      float c;   // factor from raw score to log2-domain scaled score
      if (r_cur) {
        i32x16 i0, i1;
        qk_int8<D>(kst, q8f, lane, i0, i1);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sv[r] = (float)i0[r];
          sv[16 + r] = (float)i1[r];
        }
        const float dk = half_bits_to_float(a.dK[((size_t)b * a.nKB + n) * a.Hk + hk]);
        c = a.scale_log2e * dq * dk;
      } else {
        f32x16 f0, f1;
        qk_fp16<D>(kst, qf, lane, f0, f1);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sv[r] = f0[r];
          sv[16 + r] = f1[r];
        }
        c = a.scale_log2e;
      }

      // Row max of this tile, in the log2 domain.
      const bool masked = (key0 + kBlockN - 1 > (a.causal ? q0 + off : a.Lk - 1)) ||
                          (key0 + kBlockN > a.Lk);
      float mt;
      if (masked) {
        // Scale first, then mask, so a zero scale can never meet an infinity.
        float mx = kNegInf;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const int key = key0 + 32 * (i >> 4) + acc_row(i & 15, lane);
          const bool legal = key < a.Lk && (!a.causal || key <= my_q + off);
          sv[i] = legal ? sv[i] * c : kNegInf;
          mx = fmaxf(mx, sv[i]);
        }
        mt = fmaxf(mx, other_half(mx));
      } else {
        float mx = sv[0];
#pragma unroll
        for (int i = 1; i < 32; ++i) mx = fmaxf(mx, sv[i]);
        mx = fmaxf(mx, other_half(mx));
        mt = mx * c;
      }

      const float m_new = fmaxf(m_run, mt);
      const bool grow = m_new > m_run + kRescaleThreshold;
      if (__any(grow)) {
        const float alpha = (m_new == kNegInf) ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
        z_run *= alpha;
#pragma unroll
        for (int cc = 0; cc < D / 32; ++cc) oacc[cc] *= alpha;
        m_run = m_new;
      }
      const float msub = (m_run == kNegInf) ? 0.0f : m_run;

      // P = exp2(s*c - m), packed to FP16 in the P.V operand order; z += sum(P) (of the
      // FP16 values actually multiplied into V).
      half8 pfr[4];
      float zs = 0.0f;
      const half2v ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const int i = 16 * (t >> 1) + 8 * (t & 1) + e;
          float p0, p1;
          if (masked) {
            p0 = __builtin_amdgcn_exp2f(sv[i] - msub);
            p1 = __builtin_amdgcn_exp2f(sv[i + 1] - msub);
          } else {
            p0 = __builtin_amdgcn_exp2f(fmaf(sv[i], c, -msub));
            p1 = __builtin_amdgcn_exp2f(fmaf(sv[i + 1], c, -msub));
          }
          const half2v pr = {(_Float16)p0, (_Float16)p1};
          zs = __builtin_amdgcn_fdot2(pr, ones, zs, false);
          pfr[t][e] = pr[0];
          pfr[t][e + 1] = pr[1];
        }
      }
      z_run += zs;

      // O^T += V^T P^T
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int cc = 0; cc < D / 32; ++cc) {
          const half8 va = as_half8(ld_lds_16(vst, swz<128>(32 * cc + lq, 2 * t + hi)));
          oacc[cc] = mfma_f16(va, pfr[t], oacc[cc]);
        }
      }
    }

    if (has_next) store_tile<D, BM, true>(pf, smem + ((n + 1) & 1) * C::kStage, r_next);
    __syncthreads();
    r_cur = r_next;
  }

  // Epilogue: O = O~ / z~, FP16 (round to nearest even).
  if (wave_active && row_ok) {
    const float zt = z_run + other_half(z_run);
    const float inv = zt > 0.0f ? 1.0f / zt : 0.0f;
#pragma unroll
    for (int cc = 0; cc < D / 32; ++cc) {
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        half4 h;
#pragma unroll
        for (int e = 0; e < 4; ++e) h[e] = (_Float16)(oacc[cc][4 * rg + e] * inv);
        *reinterpret_cast<half4*>(orow + 32 * cc + 8 * rg + 4 * hi) = h;
      }
    }
  }
}

// INT32 tile products C = Q8_m K8_n^T through the same staging and matrix-core code as the
// INT8 route of the fused kernel.  One workgroup per requested tile.
template <int D, int BM>
__global__ __launch_bounds__(2 * BM) void debug_tiles_kernel(DebugTileArgs a) {
  using C = TileCfg<D, BM>;
  __shared__ __align__(16) char smem[C::kStage];
  const int e = blockIdx.x;
  const int b = a.tiles[4 * e + 0], hq = a.tiles[4 * e + 1];
  const int m = a.tiles[4 * e + 2], n = a.tiles[4 * e + 3];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid & (kWave - 1);
  const int lq = lane & 31, hi = lane >> 5;
  int32_t* out = a.out + (size_t)e * BM * kBlockN;
  const bool ok = b >= 0 && b < a.B && hq >= 0 && hq < a.Hq && m >= 0 && n >= 0 &&
                  m * BM < a.Lq && n * kBlockN < a.Lk;
  if (!ok) {
    for (int i = tid; i < BM * kBlockN; i += C::kThreads) out[i] = 0;
    return;
  }
  const int hk = hq / (a.Hq / a.Hk);
  Prefetch<D, BM> pf;
  load_tile<D, BM, false>(pf, nullptr, a.K8, nullptr, b, hk, n, a.Lk, a.Hk, 0, true);
  store_tile<D, BM, false>(pf, smem, true);
  __syncthreads();
  const int my_q = m * BM + 32 * wave + lq;
  i32x4 q8f[D / 32];
  const size_t qoff = (((size_t)b * a.Lq + (my_q < a.Lq ? my_q : 0)) * a.Hq + hq) * D;
#pragma unroll
  for (int s = 0; s < D / 32; ++s)
    q8f[s] = (my_q < a.Lq) ? as_i32x4(ld_global_16(a.Q8 + qoff + 32 * s + 16 * hi)) : i32x4{};
  i32x16 i0, i1;
  qk_int8<D>(smem, q8f, lane, i0, i1);
  const int row = 32 * wave + lq;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    out[row * kBlockN + acc_row(r, lane)] = i0[r];
    out[row * kBlockN + 32 + acc_row(r, lane)] = i1[r];
  }
}

template <int D, int BM>
hipError_t launch_attn_t(const AttnArgs& a, hipStream_t stream) {
  using C = TileCfg<D, BM>;
  const long long grid = (long long)a.B * a.Hq * a.T_m;
  if (grid <= 0 || grid > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL((routed_attn_fwd_kernel<D, BM>), dim3((unsigned)grid), dim3(C::kThreads), 0,
                     stream, a);
  return hipGetLastError();
}

template <int D, int BM>
hipError_t launch_debug_t(const DebugTileArgs& a, hipStream_t stream) {
  using C = TileCfg<D, BM>;
  hipLaunchKernelGGL((debug_tiles_kernel<D, BM>), dim3(a.count), dim3(C::kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_routed_attention(const AttnArgs& a, int d, int block_m, hipStream_t stream) {
  if (d == 128 && block_m == 128) return launch_attn_t<128, 128>(a, stream);
  if (d == 128 && block_m == 64) return launch_attn_t<128, 64>(a, stream);
  if (d == 64 && block_m == 128) return launch_attn_t<64, 128>(a, stream);
  if (d == 64 && block_m == 64) return launch_attn_t<64, 64>(a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_debug_tiles(const DebugTileArgs& a, int d, int block_m, hipStream_t stream) {
  if (a.count <= 0) return hipSuccess;
  if (d == 128 && block_m == 128) return launch_debug_t<128, 128>(a, stream);
  if (d == 128 && block_m == 64) return launch_debug_t<128, 64>(a, stream);
  if (d == 64 && block_m == 128) return launch_debug_t<64, 128>(a, stream);
  if (d == 64 && block_m == 64) return launch_debug_t<64, 64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace tilemix
