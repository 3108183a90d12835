// decode.hip -- routed decode over an INT8 key/value cache (TileMix, arXiv 2608.17336,
// Appendix C "Additional Execution Interfaces").
//
// One new query token per (sequence, query head) attends to the L_k cached keys.  Cached K8
// (with its FP16 block scales) feeds the INT8 score path, the FP16 key cache the FP16 path;
// the routing bit of the key's tile group chooses (Sections 4.2, 4.3).  Cached V8 is widened
// to float on chip and its block scale is folded into the probability before the P.V
// product.  Decode reads every cached byte once and does O(1) work per byte, so it is bound
// by HBM bandwidth; a split-K layout spreads each (sequence, KV head) stream over many
// workgroups.
//
//   decode_partial_kernel<D>: workgroup (chunk of keys, KV head, sequence), 8 waves.  The grid
//     is sized for one 8-wave workgroup per CU (256 on an MI355X): each wave streams
//     tiles_per_wave 64-key tiles (tile t of the chunk goes to wave t % 8, so the eight waves
//     read neighbouring tiles at a time) and keeps its own online-softmax state (max,
//     normalizer, output) in registers across them; the group's query heads (G <= 16) sit on
//     the columns of 16x16 matrix-core tiles (padding columns carry no weight).  Per tile the
//     wave issues the key rows on the routed path and the value rows together, scores the tile
//     (v_mfma_i32_16x16x64_i8 on K8 rows, v_mfma_f32_16x16x32_f16 on FP16 key rows), and adds
//     V^T (P dV)^T on v_mfma_f32_16x16x32_f16 with P in registers.  The group's query rows are
//     quantized on chip once per workgroup (the lone decode row is a whole 128-row
//     quantization block).  At the end the eight waves' states are merged through LDS with the
//     log-sum-exp rule; the workgroup writes (max, normalizer, unnormalized output) per
//     (sequence, query head, chunk).
//   decode_combine_kernel: merges the chunks of one (sequence, query head) with the
//     log-sum-exp rule and writes O in FP16.
// A ragged batch (per-sequence cache lengths in a padded cache) runs the same kernels: tiles
// and chunks past a sequence's length are skipped and not merged; a sequence with no key gets
// O = 0.
#include "tilemix_device.h"
#include "tilemix_internal.h"

#include <algorithm>

namespace tilemix {

namespace {

constexpr int kDecWaves = 8;                        // waves per workgroup
constexpr int kDecThreads = kDecWaves * kWave;      // 512
constexpr int kDecHeads = 16;                       // query heads per KV head on the MFMA columns
constexpr int kDecSlots = 256;                      // workgroups resident at once: one per CU
constexpr int kCombineThreads = 256;

// Eight int8 codes (one per byte of v) widened to FP16, exactly: with the sign bit flipped a
// byte b reads as 1024 + 128 + b in the FP16 pattern 0x64xx, and 1152 is then subtracted.
__device__ __forceinline__ half8 i8x8_to_half8(uint32_t w0, uint32_t w1) {
  const half2v bias = {(_Float16)-1152.0f, (_Float16)-1152.0f};
  half8 out;
  const uint32_t w[2] = {w0 ^ 0x80808080u, w1 ^ 0x80808080u};
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    // bytes 0,1 -> halves 0x64b0, 0x64b1; bytes 2,3 -> 0x64b2, 0x64b3
    const uint32_t p01 = __builtin_amdgcn_perm(0x64646464u, w[i], 0x07010700u);
    const uint32_t p23 = __builtin_amdgcn_perm(0x64646464u, w[i], 0x07030702u);
    const half2v h01 = __builtin_bit_cast(half2v, p01) + bias;
    const half2v h23 = __builtin_bit_cast(half2v, p23) + bias;
    out[4 * i + 0] = h01[0]; out[4 * i + 1] = h01[1];
    out[4 * i + 2] = h23[0]; out[4 * i + 3] = h23[1];
  }
  return out;
}

// Workgroup = (chunk of 8 * tiles_per_wave key tiles, KV head, sequence).
//
// Scores are computed transposed, S^T = K Q^T, with keys on the 16 rows and the group's query
// heads on the 16 columns of each tile product.  Score block blk (= 2 * st + h) of a tile puts
// key 16 * (i / 4) + 4 * blk + i % 4 on row i, so that lane (head, lq) receives the keys
// 16 * lq + 8 * st + 4 * h + r (r < 4): for each st these are the eight keys 16 * lq + 8 * st + e
// that the B operand of P.V step st needs in lane (head, lq), slot e.  P therefore never
// leaves the registers, and the V^T operand of step st is bytes [16 * lq + 8 * st, + 8) of a
// channel row of the transposed value tile: one 16-byte load per lane covers both steps.
// Registers (about 180 per lane: key rows, value rows, output, scores) allow two waves per
// SIMD, so one 8-wave workgroup fills a CU.
template <int D>
__global__ __launch_bounds__(kDecThreads) __attribute__((amdgpu_waves_per_eu(2)))
void decode_partial_kernel(DecodeArgs a) {
  constexpr int kCB = D / 16;      // 16-channel blocks of the output
  constexpr int kS16 = D / 32;     // FP16 score products per 16-key block
  constexpr int kS8 = D / 64;      // INT8 score products per 16-key block
  constexpr int kQ16 = D + 8, kQ8 = D + 16, kOS = D + 4;   // padded LDS row lengths
  const int chunk = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int G = a.Hq / a.Hk;
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, lq = lane >> 4;
  // Keys of this sequence: all L_k cached ones, or its own length in a ragged batch.  A chunk
  // past the end has nothing to contribute and is not merged.
  const int Lkb = a.seqlens ? min(max(a.seqlens[b], 0), a.Lk) : a.Lk;
  const int tpw = a.tiles_per_wave;
  const int tile0 = chunk * kDecWaves * tpw;   // first key tile of the chunk
  if (tile0 * kBlockN >= Lkb) return;
  const int nKBb = (Lkb + kBlockN - 1) / kBlockN;
  __shared__ __align__(16) _Float16 q16[kDecHeads][kQ16];
  __shared__ __align__(16) int8_t q8[kDecHeads][kQ8];
  __shared__ float cq[kDecHeads];                         // scale * log2(e) * dQ per head
  __shared__ float red_m[kDecWaves][kDecHeads], red_z[kDecWaves][kDecHeads];
  __shared__ __align__(16) float osum[kDecWaves][kDecHeads][kOS];

  // 1. The group's query rows and this (sequence, KV head)'s routing row (Section 4.2): lane w
  //    holds word w, so a tile's bit is a lane read plus a shift.
  _Float16 qx[kDecHeads / kDecWaves][D / 64];
#pragma unroll
  for (int i = 0; i < kDecHeads / kDecWaves; ++i) {
    const int g = wave + kDecWaves * i;
#pragma unroll
    for (int e = 0; e < D / 64; ++e)
      qx[i][e] = g < G ? a.Q[((size_t)b * a.Hq + hk * G + g) * D + lane + 64 * e] : (_Float16)0.0f;
  }
  const uint64_t my_word =
      (!a.force_fp16 && lane < a.W) ? a.route[((size_t)(a.route_per_batch ? b : 0) * a.Hk + hk) * a.W + lane] : 0ull;
  const uint32_t word_lo = (uint32_t)my_word, word_hi = (uint32_t)(my_word >> 32);
  auto route_of = [&](int n) -> bool {
    const int gj = n / a.g, w = gj >> 6, bit = gj & 63;
    const uint32_t h = bit < 32 ? __builtin_amdgcn_readlane(word_lo, w) : __builtin_amdgcn_readlane(word_hi, w);
    return (h >> (bit & 31)) & 1u;
  };

  // 2. FP16 copy, INT8 codes and FP16-stored scale of the query rows (Appendix C
  //    quantization; the lone decode row forms its own 128-row block).  Rows past G are 0.
#pragma unroll
  for (int i = 0; i < kDecHeads / kDecWaves; ++i) {
    const int g = wave + kDecWaves * i;
    float x[D / 64];
    float amax = 0.0f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      q16[g][lane + 64 * e] = qx[i][e];
      x[e] = (float)qx[i][e];
      amax = fmaxf(amax, fabsf(x[e]));
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, kWave));
    const float d32 = amax / 127.0f;   // IEEE FP32 division
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      const float c = amax > 0.0f ? fminf(127.0f, fmaxf(-127.0f, rintf(x[e] / d32))) : 0.0f;
      q8[g][lane + 64 * e] = (int8_t)(int)c;
    }
    if (lane == 0) cq[g] = a.scale_log2e * (amax > 0.0f ? (float)(_Float16)d32 : 0.0f);
  }
  __syncthreads();

  // 3. The wave's tiles tile0 + wave, tile0 + wave + 8, ...: per tile, key rows (routed path)
  //    and value rows are issued together; scores in log2 units; the running max, normalizer
  //    and output of the wave are rescaled when the max grows (Section 3.1); P = 2^(s - m)
  //    with the V block scale folded in is the FP16 B operand of the P.V products.
  const bool head_ok = l16 < G;   // columns past G are padding
  const float ninf = -__builtin_huge_valf();
  float m_w = ninf, z_w = 0.0f;   // z_w: this lane's share of the normalizer
  f32x4 acc[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) acc[cb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  for (int i = 0; i < tpw; ++i) {
    const int n = tile0 + i * kDecWaves + wave;
    if (n >= nKBb) break;
    asm volatile("" ::: "memory");   // keep the LDS operand reads inside the loop
    const bool int8 = route_of(n);
    const size_t si = ((size_t)b * a.nKB + n) * a.Hk + hk;
    const uint16_t dk_bits = a.dK[si], dv_bits = a.dV[si];
    uint4 kr[4][kS16];
    {
      const char* kbytes = int8 ? reinterpret_cast<const char*>(a.K8) : reinterpret_cast<const char*>(a.K);
      const size_t row_bytes = int8 ? D : 2 * D;
      // K8 and FP16 key rows differ only in their row length (D or 2 D bytes): lane lq reads
      // bytes 16 * lq + 64 * s of the row for product s of a 16-key block.
      const int kbase = n * kBlockN + 16 * (l16 >> 2) + (l16 & 3);
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) {
        const int key = min(kbase + 4 * blk, Lkb - 1);   // keys past the length are masked below
        const char* kp = kbytes + (((size_t)b * a.Lk + key) * a.Hk + hk) * row_bytes + 16 * lq;
#pragma unroll
        for (int s = 0; s < kS8; ++s) kr[blk][s] = ld_global_16(kp + 64 * s);
        if (!int8) {
#pragma unroll
          for (int s = kS8; s < kS16; ++s) kr[blk][s] = ld_global_16(kp + 64 * s);
        }
      }
    }
    uint4 vr[kCB];
    {
      const int8_t* vt = a.V8 + ((((size_t)b * a.Hk + hk) * a.nKB + n) * D + l16) * kBlockN + 16 * lq;
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) vr[cb] = ld_global_16(vt + cb * 16 * kBlockN);
    }
    float sc[4][4];
    if (int8) {
      i32x4 c[4];
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) c[blk] = i32x4{0, 0, 0, 0};
#pragma unroll
      for (int s = 0; s < kS8; ++s) {   // one query operand slice live at a time
        const i32x4 qb = *reinterpret_cast<const i32x4*>(&q8[l16][64 * s + 16 * lq]);
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
          c[blk] = __builtin_amdgcn_mfma_i32_16x16x64_i8(as_i32x4(kr[blk][s]), qb, c[blk], 0, 0, 0);
      }
      const float f = cq[l16] * half_bits_to_float(dk_bits);
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[blk][r] = (float)c[blk][r] * f;
    } else {
      f32x4 c[4];
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) c[blk] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int s = 0; s < kS16; ++s) {
        const half8 qb = *reinterpret_cast<const half8*>(&q16[l16][32 * s + 8 * lq]);
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
          c[blk] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_half8(kr[blk][s]), qb, c[blk], 0, 0, 0);
      }
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[blk][r] = c[blk][r] * a.scale_log2e;
    }
    const float dv = half_bits_to_float(dv_bits);
    float mt = ninf;
#pragma unroll
    for (int blk = 0; blk < 4; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool ok = head_ok && n * kBlockN + 16 * lq + 4 * blk + r < Lkb;
        sc[blk][r] = ok ? sc[blk][r] : ninf;
        mt = fmaxf(mt, sc[blk][r]);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, kWave));
    mt = fmaxf(mt, __shfl_xor(mt, 32, kWave));
    const float m_new = fmaxf(m_w, mt);
    const float alpha = m_w == ninf ? 0.0f : __builtin_amdgcn_exp2f(m_w - m_new);
    z_w *= alpha;
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) acc[cb] *= alpha;
    m_w = m_new;
    half8 pb[2];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = sc[blk][r] == ninf ? 0.0f : __builtin_amdgcn_exp2f(sc[blk][r] - m_new);
        z_w += p;
        pb[blk >> 1][4 * (blk & 1) + r] = (_Float16)(p * dv);
      }
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(i8x8_to_half8(vr[cb].x, vr[cb].y), pb[0], acc[cb], 0, 0, 0);
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(i8x8_to_half8(vr[cb].z, vr[cb].w), pb[1], acc[cb], 0, 0, 0);
    }
  }
  // 4. Merge of the eight waves (log-sum-exp rule through LDS), then (max, normalizer,
  //    unnormalized output) of the chunk per head.
  z_w += __shfl_xor(z_w, 16, kWave);
  z_w += __shfl_xor(z_w, 32, kWave);
  if (lq == 0) red_m[wave][l16] = m_w;
  __syncthreads();
  float mc = red_m[0][l16];
#pragma unroll
  for (int w = 1; w < kDecWaves; ++w) mc = fmaxf(mc, red_m[w][l16]);
  const float fw = m_w == ninf ? 0.0f : __builtin_amdgcn_exp2f(m_w - mc);
  if (lq == 0) red_z[wave][l16] = z_w * fw;
  if (head_ok) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb)
      *reinterpret_cast<f32x4*>(&osum[wave][l16][16 * cb + 4 * lq]) = acc[cb] * fw;
  }
  __syncthreads();
  for (int o = tid; o < G * D; o += kDecThreads) {
    const int g = o / D, c = o % D;
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) sum += osum[w][g][c];
    a.part_o[(((size_t)b * a.Hq + hk * G + g) * a.chunks + chunk) * D + c] = sum;
  }
  if (tid < G) {
    float zz = 0.0f, mm = red_m[0][tid];
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      zz += red_z[w][tid];
      mm = fmaxf(mm, red_m[w][tid]);
    }
    const size_t o = ((size_t)b * a.Hq + hk * G + tid) * a.chunks + chunk;
    a.part_m[o] = mm;
    a.part_z[o] = zz;
  }
}

// One workgroup per (sequence, query head).  Thread (part, c4) owns channels 4*c4 .. 4*c4+3
// and the chunks part, part + kRows, ...; it keeps a running (max, normalizer, output) merged
// with the log-sum-exp rule, loading kUnroll chunks ahead.  The parts are merged in LDS.
template <int D>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(DecodeArgs a) {
  constexpr int kLanes = D / 4;                     // float4 lanes per chunk row
  constexpr int kRows = kCombineThreads / kLanes;   // chunk rows per pass
  constexpr int kUnroll = 8;
  const int bh = blockIdx.x;   // b * Hq + hq
  const int tid = threadIdx.x, c4 = tid % kLanes, part = tid / kLanes;
  int chunks = a.chunks;       // the chunks that hold keys of this sequence
  if (a.seqlens) {
    const int len = min(max(a.seqlens[bh / a.Hq], 0), a.Lk);
    const int per = kDecWaves * a.tiles_per_wave;   // key tiles per chunk
    chunks = min(chunks, ((len + kBlockN - 1) / kBlockN + per - 1) / per);
  }
  __shared__ float sm[kRows], sz[kRows];
  __shared__ f32x4 so[kRows][kLanes];
  const float* pm = a.part_m + (size_t)bh * a.chunks;
  const float* pz = a.part_z + (size_t)bh * a.chunks;
  const f32x4* po = reinterpret_cast<const f32x4*>(a.part_o + (size_t)bh * a.chunks * D) + c4;
  const float ninf = -__builtin_huge_valf();
  float m = ninf, z = 0.0f;
  f32x4 o = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int i0 = part; i0 < chunks; i0 += kRows * kUnroll) {
    float mi[kUnroll], zi[kUnroll];
    f32x4 oi[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = i0 + u * kRows;
      const bool ok = i < chunks;
      mi[u] = ok ? pm[i] : ninf;
      zi[u] = ok ? pz[i] : 0.0f;
      oi[u] = ok ? po[(size_t)i * kLanes] : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    float mn = m;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) mn = fmaxf(mn, mi[u]);
    if (mn == ninf) continue;
    const float f = m == ninf ? 0.0f : __builtin_amdgcn_exp2f(m - mn);
    z *= f;
    o *= f;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const float fu = mi[u] == ninf ? 0.0f : __builtin_amdgcn_exp2f(mi[u] - mn);
      z += zi[u] * fu;
      o += oi[u] * fu;
    }
    m = mn;
  }
  if (c4 == 0) {
    sm[part] = m;
    sz[part] = z;
  }
  so[part][c4] = o;
  __syncthreads();
  if (tid < kLanes) {
    float mm = sm[0];
#pragma unroll
    for (int p = 1; p < kRows; ++p) mm = fmaxf(mm, sm[p]);
    float zz = 0.0f;
    f32x4 oo = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int p = 0; p < kRows; ++p) {
      const float fp = sm[p] == ninf ? 0.0f : __builtin_amdgcn_exp2f(sm[p] - mm);
      zz += sz[p] * fp;
      oo += so[p][tid] * fp;
    }
    const float inv = zz > 0.0f ? 1.0f / zz : 0.0f;
    half4 h;
#pragma unroll
    for (int r = 0; r < 4; ++r) h[r] = (_Float16)(oo[r] * inv);
    *reinterpret_cast<half4*>(a.O + (size_t)bh * D + 4 * tid) = h;
  }
}

template <int D>
hipError_t launch_decode_t(const DecodeArgs& a, hipStream_t stream) {
  if (a.Hq / a.Hk > kDecHeads) return hipErrorInvalidValue;
  hipLaunchKernelGGL((decode_partial_kernel<D>), dim3(a.chunks, a.Hk, a.B), dim3(kDecThreads), 0,
                     stream, a);
  hipLaunchKernelGGL(decode_combine_kernel<D>, dim3(a.B * a.Hq), dim3(kCombineThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int d, hipStream_t stream) {
  if (d == 128) return launch_decode_t<128>(a, stream);
  if (d == 64) return launch_decode_t<64>(a, stream);
  return hipErrorInvalidValue;
}

// Tiles each wave streams: the grid then holds about kDecSlots workgroups, one round on the
// chip, however long the cache.
int decode_tiles_per_wave(int batch, int heads_kv, int len_k) {
  const long long tiles = (long long)batch * heads_kv * ((len_k + kBlockN - 1) / kBlockN);
  const long long per = (long long)kDecWaves * kDecSlots;
  return (int)std::max<long long>(1, (tiles + per - 1) / per);
}

int decode_chunks(int batch, int heads_kv, int len_k) {
  const int per = kDecWaves * decode_tiles_per_wave(batch, heads_kv, len_k);
  return ((len_k + kBlockN - 1) / kBlockN + per - 1) / per;
}

}  // namespace tilemix
