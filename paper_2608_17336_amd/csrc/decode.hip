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
//   decode_partial_kernel<D, GP>: workgroup (chunk of 512 keys, KV head, sequence), GP >= G
//     query heads of the GQA group (the padding heads carry no weight).  The group's query
//     rows are quantized on chip (the lone decode row is a whole 128-row quantization block);
//     each thread scores two keys on their routed path for every head; one max and one sum
//     reduction per chunk give the chunk's max and normalizer; then each wave accumulates
//     P * dV against V8 over its quarter of the chunk, lanes over 4-channel slots, and the
//     waves' partial outputs are added through LDS.  Writes (max, normalizer, unnormalized
//     output) per (sequence, query head, chunk).
//   decode_combine_kernel: merges the chunks of one (sequence, query head) with the
//     log-sum-exp rule and writes O in FP16.
#include "tilemix_device.h"
#include "tilemix_internal.h"

namespace tilemix {

namespace {

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kDecChunk = 512;                  // keys per workgroup
constexpr int kKeysPerThread = kDecChunk / kDecThreads;
constexpr int kDecMaxChunks = (kMaxKeyTiles * kBlockN) / kDecChunk;   // chunks of the longest cache

__device__ __forceinline__ float wave_max(float v) {
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

template <int D, int GP>
__global__ __launch_bounds__(kDecThreads) void decode_partial_kernel(DecodeArgs a) {
  constexpr int kRowDwords = D / 4;               // dwords of one V8 row
  constexpr int kKeysPerIter = kWave / kRowDwords; // keys one wave reads per load
  const int chunk = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int G = a.Hq / a.Hk;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  __shared__ __align__(16) _Float16 q16[GP][D];
  __shared__ __align__(16) int8_t q8[GP][D];
  __shared__ float cq[GP];                                   // scale * log2(e) * dQ per head
  __shared__ __align__(16) float pv[GP * kDecChunk];         // scores, P * dV; then outputs
  __shared__ float red[2][GP][kDecWaves];

  // 1. Query rows of the group: FP16 copy, INT8 codes and FP16-stored scale (Appendix C
  //    quantization; the lone decode row forms its own 128-row block).  Padding heads are 0.
  for (int g = wave; g < GP; g += kDecWaves) {
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

  // 2. Scores of this thread's keys for every head, log2 domain; lane max per head.
  float lmax[GP];
#pragma unroll
  for (int g = 0; g < GP; ++g) lmax[g] = -__builtin_huge_valf();
#pragma unroll
  for (int u = 0; u < kKeysPerThread; ++u) {
    const int t = u * kDecThreads + tid;                     // key within the chunk
    const int j = chunk * kDecChunk + t;
    const bool valid = j < a.Lk;
    // key tile of the wave's keys (clamped for the keys past L_k of the last chunk)
    const int n = min(__builtin_amdgcn_readfirstlane(j >> 6), a.nKB - 1);
    const int gj = n / a.g;
    const uint64_t word = a.route[((size_t)(a.route_per_batch ? b : 0) * a.Hk + hk) * a.W + (gj >> 6)];
    const bool int8 = !a.force_fp16 && ((word >> (gj & 63)) & 1ull);
    const float dk = half_bits_to_float(a.dK[((size_t)b * a.nKB + n) * a.Hk + hk]);
    const size_t row = ((size_t)b * a.Lk + (valid ? j : 0)) * a.Hk + hk;
    float s[GP];
    if (int8) {
      int kw[D / 4];
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const uint4 v = ld_global_16(a.K8 + row * D + 16 * c);
        kw[4 * c] = (int)v.x; kw[4 * c + 1] = (int)v.y; kw[4 * c + 2] = (int)v.z; kw[4 * c + 3] = (int)v.w;
      }
#pragma unroll
      for (int g = 0; g < GP; ++g) {
        const int* qw = reinterpret_cast<const int*>(q8[g]);
        int acc = 0;
#pragma unroll
        for (int c = 0; c < D / 4; ++c) acc = __builtin_amdgcn_sdot4(kw[c], qw[c], acc, false);
        s[g] = (float)acc * (cq[g] * dk);
      }
    } else {
      half2v kh[D / 2];
#pragma unroll
      for (int c = 0; c < D / 8; ++c) {
        const half8 v = as_half8(ld_global_16(a.K + row * D + 8 * c));
#pragma unroll
        for (int e = 0; e < 4; ++e) kh[4 * c + e] = half2v{v[2 * e], v[2 * e + 1]};
      }
#pragma unroll
      for (int g = 0; g < GP; ++g) {
        const half2v* qh = reinterpret_cast<const half2v*>(q16[g]);
        float acc = 0.0f;
#pragma unroll
        for (int c = 0; c < D / 2; ++c) acc = __builtin_amdgcn_fdot2(kh[c], qh[c], acc, false);
        s[g] = acc * a.scale_log2e;
      }
    }
#pragma unroll
    for (int g = 0; g < GP; ++g) {
      const float v = (valid && g < G) ? s[g] : -__builtin_huge_valf();
      pv[g * kDecChunk + t] = v;
      lmax[g] = fmaxf(lmax[g], v);
    }
  }
#pragma unroll
  for (int g = 0; g < GP; ++g) {
    const float m = wave_max(lmax[g]);
    if (lane == 0) red[0][g][wave] = m;
  }
  __syncthreads();

  // 3. Chunk max and normalizer per head; P * dV for the P.V step.
  float m[GP], lz[GP];
#pragma unroll
  for (int g = 0; g < GP; ++g) {
    m[g] = red[0][g][0];
#pragma unroll
    for (int w = 1; w < kDecWaves; ++w) m[g] = fmaxf(m[g], red[0][g][w]);
    lz[g] = 0.0f;
  }
#pragma unroll
  for (int u = 0; u < kKeysPerThread; ++u) {
    const int t = u * kDecThreads + tid;
    const int n = min((chunk * kDecChunk + t) >> 6, a.nKB - 1);
    const float dv = half_bits_to_float(a.dV[((size_t)b * a.nKB + n) * a.Hk + hk]);
#pragma unroll
    for (int g = 0; g < GP; ++g) {
      const float sc = pv[g * kDecChunk + t];
      const float p = (m[g] == -__builtin_huge_valf()) ? 0.0f : __builtin_amdgcn_exp2f(sc - m[g]);
      lz[g] += p;
      pv[g * kDecChunk + t] = p * dv;
    }
  }
#pragma unroll
  for (int g = 0; g < GP; ++g) {
    const float z = wave_sum(lz[g]);
    if (lane == 0) red[1][g][wave] = z;
  }
  __syncthreads();
  if (tid < G) {
    float z = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) z += red[1][tid][w];
    const size_t o = ((size_t)b * a.Hq + hk * G + tid) * a.chunks + chunk;
    float mm = red[0][tid][0];
#pragma unroll
    for (int w = 1; w < kDecWaves; ++w) mm = fmaxf(mm, red[0][tid][w]);
    a.part_m[o] = mm;
    a.part_z[o] = z;
  }

  // 4. O_g[c] = sum over the chunk's keys of (P dV)_g,j * V8[j][c]: wave w takes keys
  //    [w, w + kDecWaves, ...) in steps of kKeysPerIter, each lane one 4-channel slot of one key.
  const int kmax = min(kDecChunk, a.Lk - chunk * kDecChunk);
  const int c4 = lane % kRowDwords, ksub = lane / kRowDwords;
  const int8_t* vchunk = a.V8 + (((size_t)b * a.Lk + (size_t)chunk * kDecChunk) * a.Hk + hk) * D + 4 * c4;
  const size_t vstride = (size_t)a.Hk * D;   // bytes between consecutive keys
  float acc[GP][4];
#pragma unroll
  for (int g = 0; g < GP; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[g][e] = 0.0f;
  // Loads are issued kBatch keys at a time ahead of their arithmetic, so that each wave keeps
  // kBatch rows in flight; keys past L_k read as 0 and carry P = 0.
  constexpr int kStep = kDecWaves * kKeysPerIter;
  constexpr int kBatch = 16;
  for (int t0 = wave * kKeysPerIter; t0 < kmax; t0 += kStep * kBatch) {
    uint32_t w[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int t = t0 + u * kStep + ksub;
      w[u] = t < kmax ? *reinterpret_cast<const uint32_t*>(vchunk + (size_t)t * vstride) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int t = min(t0 + u * kStep + ksub, kDecChunk - 1);
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (float)(int8_t)(uint8_t)(w[u] >> (8 * e));
#pragma unroll
      for (int g = 0; g < GP; ++g) {
        const float p = pv[g * kDecChunk + t];
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[g][e] += p * v[e];
      }
    }
  }
  // Lanes holding the same slot for different keys are added by lane exchange, the waves'
  // partial outputs through LDS (pv is free again: [kDecWaves][GP][D] fits in it).
#pragma unroll
  for (int x = kRowDwords; x < kWave; x <<= 1)
#pragma unroll
    for (int g = 0; g < GP; ++g)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[g][e] += __shfl_xor(acc[g][e], x, kWave);
  static_assert(kDecWaves * GP * D <= GP * kDecChunk, "partial outputs fit in pv");
  __syncthreads();   // every wave is done reading pv
  float* osum = pv;
  if (ksub == 0) {
#pragma unroll
    for (int g = 0; g < GP; ++g)
#pragma unroll
      for (int e = 0; e < 4; ++e) osum[(wave * GP + g) * D + 4 * c4 + e] = acc[g][e];
  }
  __syncthreads();
  for (int o = tid; o < G * D; o += kDecThreads) {
    const int g = o / D, c = o % D;
    float sum = 0.0f;
#pragma unroll
    for (int r = 0; r < kDecWaves; ++r) sum += osum[(r * GP + g) * D + c];
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

template <int D, int GP>
void launch_partial(const DecodeArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((decode_partial_kernel<D, GP>), dim3(a.chunks, a.Hk, a.B), dim3(kDecThreads),
                     0, stream, a);
}

template <int D>
hipError_t launch_decode_t(const DecodeArgs& a, hipStream_t stream) {
  const int G = a.Hq / a.Hk;
  if (G <= 1) launch_partial<D, 1>(a, stream);
  else if (G <= 2) launch_partial<D, 2>(a, stream);
  else if (G <= 4) launch_partial<D, 4>(a, stream);
  else if (G <= 8) launch_partial<D, 8>(a, stream);
  else if (G <= 16) launch_partial<D, 16>(a, stream);
  else return hipErrorInvalidValue;
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
