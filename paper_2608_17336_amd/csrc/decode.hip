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
//   decode_partial_kernel<D>: workgroup (chunk of 512 keys, KV head, sequence), the G <= 16
//     query heads of the GQA group on the rows of 16x16 matrix-core tiles (padding rows carry
//     no weight).  The group's query rows are quantized on chip (the lone decode row is a
//     whole 128-row quantization block).  Each wave scores its 128 keys in 16-key blocks on
//     the block's routed path (v_mfma_i32_16x16x64_i8 on K8 rows, v_mfma_f32_16x16x32_f16 on
//     FP16 key rows); one max and one sum reduction give the chunk's max and normalizer per
//     head; P * dV goes to LDS in FP16 and the wave accumulates O^T += V^T (P dV)^T with
//     v_mfma_f32_16x16x32_f16, V^T read from the transposed value-cache tiles and widened to
//     FP16 exactly.  The waves' partial outputs are added through LDS.  Writes (max,
//     normalizer, unnormalized output) per (sequence, query head, chunk).
//   decode_combine_kernel: merges the chunks of one (sequence, query head) with the
//     log-sum-exp rule and writes O in FP16.
#include "tilemix_device.h"
#include "tilemix_internal.h"

namespace tilemix {

namespace {

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kDecChunk = 512;                  // keys per workgroup
constexpr int kDecHeads = 16;                   // query heads per KV head the MFMA rows hold
constexpr int kDecMaxChunks = (kMaxKeyTiles * kBlockN) / kDecChunk;   // chunks of the longest cache

__device__ __forceinline__ float wave_max(float v) {
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Eight int8 codes (one per byte of v) widened to FP16, exactly: with the sign bit flipped a
// byte b reads as 1024 + 128 + b in the FP16 pattern 0x64xx, and 1152 is then subtracted.
__device__ __forceinline__ half8 i8x8_to_half8(uint2 v) {
  const uint32_t lo = v.x ^ 0x80808080u, hi = v.y ^ 0x80808080u;
  const half2v bias = {(_Float16)-1152.0f, (_Float16)-1152.0f};
  half8 out;
  const uint32_t w[2] = {lo, hi};
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

template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_partial_kernel(DecodeArgs a) {
  constexpr int kKeysPerWave = kDecChunk / kDecWaves;   // 128
  constexpr int kBlocks = kKeysPerWave / 16;             // 16-key score blocks per wave
  constexpr int kSteps = kKeysPerWave / 32;              // 32-key P.V steps per wave
  constexpr int kCB = D / 16;                            // 16-channel output blocks
  const int chunk = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int G = a.Hq / a.Hk;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int l16 = lane & 15, lq = lane >> 4;
  __shared__ __align__(16) _Float16 q16[kDecHeads][D];
  __shared__ __align__(16) int8_t q8[kDecHeads][D];
  __shared__ float cq[kDecHeads];                         // scale * log2(e) * dQ per head
  // P * dV [head][key] in FP16 for the P.V step, then the waves' partial outputs [wave][head][D]
  constexpr int kPhBytes = kDecHeads * kDecChunk * 2, kOsumBytes = kDecWaves * kDecHeads * D * 4;
  __shared__ __align__(16) char buf[kPhBytes > kOsumBytes ? kPhBytes : kOsumBytes];
  auto ph = reinterpret_cast<_Float16(*)[kDecChunk]>(buf);
  auto osum = reinterpret_cast<float(*)[kDecHeads][D]>(buf);
  __shared__ float red[2][kDecWaves][kDecHeads];

  // 1. Query rows of the group: FP16 copy, INT8 codes and FP16-stored scale (Appendix C
  //    quantization; the lone decode row forms its own 128-row block).  Rows past G are 0.
  for (int g = wave; g < kDecHeads; g += kDecWaves) {
    const int hq = hk * G + g;
    float x[D / 64];
    float amax = 0.0f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      const _Float16 h = g < G ? a.Q[((size_t)b * a.Hq + hq) * D + lane + 64 * e] : (_Float16)0.0f;
      q16[g][lane + 64 * e] = h;
      x[e] = (float)h;
      amax = fmaxf(amax, fabsf(x[e]));
    }
    amax = wave_max(amax);
    const float d32 = amax / 127.0f;   // IEEE FP32 division
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      const float c = amax > 0.0f ? fminf(127.0f, fmaxf(-127.0f, rintf(x[e] / d32))) : 0.0f;
      q8[g][lane + 64 * e] = (int8_t)(int)c;
    }
    if (lane == 0) cq[g] = a.scale_log2e * (amax > 0.0f ? (float)(_Float16)d32 : 0.0f);
  }
  __syncthreads();

  // 2. Scores S[head][key] of the wave's 128 keys, 16 keys per block, on the matrix cores:
  //    v_mfma_i32_16x16x64_i8 (INT8 route) or v_mfma_f32_16x16x32_f16 (FP16 route), heads on
  //    the rows (A from LDS) and keys on the columns (B straight from the key rows).  Lane l
  //    holds heads 4*(l/16) + r of key l % 16.
  i32x4 qa8[D / 64];
  half8 qa16[D / 32];
#pragma unroll
  for (int s = 0; s < D / 64; ++s) qa8[s] = *reinterpret_cast<const i32x4*>(&q8[l16][64 * s + 16 * lq]);
#pragma unroll
  for (int s = 0; s < D / 32; ++s) qa16[s] = *reinterpret_cast<const half8*>(&q16[l16][32 * s + 8 * lq]);
  float cqr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) cqr[r] = cq[4 * lq + r];
  const int key_base = chunk * kDecChunk + wave * kKeysPerWave;
  float sc[kBlocks][4];
#pragma unroll
  for (int jb = 0; jb < kBlocks; ++jb) {
    const int k0 = key_base + 16 * jb;
    const int n = min(k0 >> 6, a.nKB - 1);   // key tile of the block (clamped past L_k)
    const int gj = n / a.g;
    const uint64_t word = a.route[((size_t)(a.route_per_batch ? b : 0) * a.Hk + hk) * a.W + (gj >> 6)];
    const bool int8 = !a.force_fp16 && ((word >> (gj & 63)) & 1ull);
    const int key = k0 + l16;
    const bool valid = key < a.Lk;
    const size_t row = ((size_t)b * a.Lk + (valid ? key : 0)) * a.Hk + hk;
    float v[4];
    if (int8) {
      const float dk = half_bits_to_float(a.dK[((size_t)b * a.nKB + n) * a.Hk + hk]);
      i32x4 acc = {0, 0, 0, 0};
#pragma unroll
      for (int s = 0; s < D / 64; ++s) {
        const i32x4 kb = as_i32x4(ld_global_16(a.K8 + row * D + 64 * s + 16 * lq));
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(qa8[s], kb, acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = (float)acc[r] * (cqr[r] * dk);
    } else {
      f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int s = 0; s < D / 32; ++s) {
        const half8 kb = as_half8(ld_global_16(a.K + row * D + 32 * s + 8 * lq));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa16[s], kb, acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = acc[r] * a.scale_log2e;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) sc[jb][r] = (valid && 4 * lq + r < G) ? v[r] : -__builtin_huge_valf();
  }

  // 3. Per-head chunk max and normalizer (the 16 lanes of a quarter-wave share their heads);
  //    P * dV to LDS in FP16 for the P.V step (the V block scale folded into P).
  float mx[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float m = sc[0][r];
#pragma unroll
    for (int jb = 1; jb < kBlocks; ++jb) m = fmaxf(m, sc[jb][r]);
#pragma unroll
    for (int x = 1; x < 16; x <<= 1) m = fmaxf(m, __shfl_xor(m, x, kWave));
    mx[r] = m;
  }
  if (l16 == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) red[0][wave][4 * lq + r] = mx[r];
  }
  __syncthreads();
  float zs[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float m = red[0][0][4 * lq + r];
#pragma unroll
    for (int w = 1; w < kDecWaves; ++w) m = fmaxf(m, red[0][w][4 * lq + r]);
    mx[r] = m;
    zs[r] = 0.0f;
  }
#pragma unroll
  for (int jb = 0; jb < kBlocks; ++jb) {
    const int t = wave * kKeysPerWave + 16 * jb + l16;           // key within the chunk
    const int n = min((chunk * kDecChunk + t) >> 6, a.nKB - 1);
    const float dv = half_bits_to_float(a.dV[((size_t)b * a.nKB + n) * a.Hk + hk]);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = (mx[r] == -__builtin_huge_valf()) ? 0.0f : __builtin_amdgcn_exp2f(sc[jb][r] - mx[r]);
      zs[r] += p;
      ph[4 * lq + r][t] = (_Float16)(p * dv);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float z = zs[r];
#pragma unroll
    for (int x = 1; x < 16; x <<= 1) z += __shfl_xor(z, x, kWave);
    zs[r] = z;
  }
  if (l16 == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) red[1][wave][4 * lq + r] = zs[r];
  }
  __syncthreads();
  if (tid < G) {
    float z = 0.0f, m = red[0][0][tid];
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      z += red[1][w][tid];
      m = fmaxf(m, red[0][w][tid]);
    }
    const size_t o = ((size_t)b * a.Hq + hk * G + tid) * a.chunks + chunk;
    a.part_m[o] = m;
    a.part_z[o] = z;
  }

  // 4. O^T[channel][head] += V^T[channel][key] (P dV)^T[key][head], v_mfma_f32_16x16x32_f16:
  //    A = 8 consecutive keys of one channel from the transposed V8 tile (widened to FP16),
  //    B = 8 keys of P dV for one head from LDS.  Lane l ends with channels 4*(l/16) + r of
  //    its 16-channel block for head l % 16.
  f32x4 acc[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) acc[cb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int kk = wave * kKeysPerWave + 32 * st;                // first key of the step (chunk)
    const int key0 = chunk * kDecChunk + kk;
    if (key0 >= a.Lk) break;                                     // the rest of the chunk is past L_k
    const int n = key0 >> 6;
    const half8 pb = *reinterpret_cast<const half8*>(&ph[l16][kk + 8 * lq]);
    const int8_t* vt = a.V8 + ((((size_t)b * a.Hk + hk) * a.nKB + n) * D + l16) * kBlockN +
                       (key0 & 63) + 8 * lq;
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      const uint2 raw = *reinterpret_cast<const uint2*>(vt + (size_t)cb * 16 * kBlockN);
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(i8x8_to_half8(raw), pb, acc[cb], 0, 0, 0);
    }
  }
  __syncthreads();   // every wave is done reading P before the buffer holds outputs
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) osum[wave][l16][16 * cb + 4 * lq + r] = acc[cb][r];
  __syncthreads();
  for (int o = tid; o < G * D; o += kDecThreads) {
    const int g = o / D, c = o % D;
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) sum += osum[w][g][c];
    a.part_o[(((size_t)b * a.Hq + hk * G + g) * a.chunks + chunk) * D + c] = sum;
  }
}

// One workgroup per (sequence, query head): the chunks' maxima give m; each chunk's weight
// 2^(m_i - m) goes to LDS with the normalizer z = sum z_i 2^(m_i - m); then threads over
// (channel, chunk residue) add the weighted chunk outputs and the residues are summed in LDS.
template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_combine_kernel(DecodeArgs a) {
  constexpr int kParts = kDecThreads / D;
  const int bh = blockIdx.x;   // b * Hq + hq
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  __shared__ float wgt[kDecMaxChunks];
  __shared__ float red[kDecWaves];
  __shared__ float opart[kParts][D];
  const float* pm = a.part_m + (size_t)bh * a.chunks;
  const float* pz = a.part_z + (size_t)bh * a.chunks;
  float m = -__builtin_huge_valf();
  for (int i = tid; i < a.chunks; i += kDecThreads) m = fmaxf(m, pm[i]);
  m = wave_max(m);
  if (lane == 0) red[wave] = m;
  __syncthreads();
  m = red[0];
#pragma unroll
  for (int w = 1; w < kDecWaves; ++w) m = fmaxf(m, red[w]);
  float zl = 0.0f;
  for (int i = tid; i < a.chunks; i += kDecThreads) {
    const float f = (m == -__builtin_huge_valf() || pm[i] == -__builtin_huge_valf())
                        ? 0.0f : __builtin_amdgcn_exp2f(pm[i] - m);
    wgt[i] = f;
    zl += pz[i] * f;
  }
  zl = wave_sum(zl);
  __syncthreads();   // red is reused
  if (lane == 0) red[wave] = zl;
  __syncthreads();
  float z = 0.0f;
#pragma unroll
  for (int w = 0; w < kDecWaves; ++w) z += red[w];
  const int c = tid % D, part = tid / D;
  const float* po = a.part_o + (size_t)bh * a.chunks * D + c;
  float o = 0.0f;
#pragma unroll 4
  for (int i = part; i < a.chunks; i += kParts) o += po[(size_t)i * D] * wgt[i];
  opart[part][c] = o;
  __syncthreads();
  if (tid < D) {
    float t = 0.0f;
#pragma unroll
    for (int r = 0; r < kParts; ++r) t += opart[r][tid];
    a.O[(size_t)bh * D + tid] = (_Float16)(z > 0.0f ? t / z : 0.0f);
  }
}

template <int D>
hipError_t launch_decode_t(const DecodeArgs& a, hipStream_t stream) {
  if (a.Hq / a.Hk > kDecHeads) return hipErrorInvalidValue;
  hipLaunchKernelGGL((decode_partial_kernel<D>), dim3(a.chunks, a.Hk, a.B), dim3(kDecThreads), 0,
                     stream, a);
  hipLaunchKernelGGL(decode_combine_kernel<D>, dim3(a.B * a.Hq), dim3(kDecThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int d, hipStream_t stream) {
  if (d == 128) return launch_decode_t<128>(a, stream);
  if (d == 64) return launch_decode_t<64>(a, stream);
  return hipErrorInvalidValue;
}

int decode_chunks(int len_k) { return (len_k + kDecChunk - 1) / kDecChunk; }

}  // namespace tilemix
