// prepare.hip -- operand preparation for the routed attention kernel (bandwidth-bound).
//
// quantize_blocks_kernel: the quantize-once pass of Appendix C ("Blockwise INT8
//   Quantization", "Quantization Granularity", "Quantize-Once Execution"): for every
//   (sequence, head, block of 128 query / 64 key tokens) the FP32 absmax, the FP32
//   scale absmax/127, the codes round-half-even(x / scale) clamped to [-127, 127]
//   and the FP16 scale.  One workgroup per block; the block is read once into
//   registers, reduced, then converted and written.
//
// v_tiles_kernel: lays V out per 64-key tile as [d][64] so that the P.V matrix-core
//   step reads its A operand (V^T) as contiguous 16-byte runs.  Within each run of
//   16 keys the order is (0-3, 8-11 | 4-7, 12-15): this is the key order in which
//   the score accumulator hands P to the P.V step (accumulator rows 8*(r/4) +
//   4*(lane/32) + r%4), so P never leaves registers.  Keys past L are zero.
#include "tilemix_device.h"
#include "tilemix_internal.h"

namespace tilemix {

namespace {

constexpr int kPrepThreads = 256;

__device__ __forceinline__ float block_max(float v, float* red) {
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  const int wave = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
  for (int w = 1; w < kPrepThreads / kWave; ++w) r = fmaxf(r, red[w]);
  return r;
}

// Rows of sequence b in the packed tensor, and its first scale block: computed for one common
// length L, or read from the sequence table of a variable-length batch (fields f_start, f_len,
// f_blk of its 8-int rows).
struct SeqRows {
  long long start, blk;
  int len;
};
__device__ __forceinline__ SeqRows seq_rows(const int* seqs, int b, int L, int nblk, int f_start,
                                            int f_len, int f_blk) {
  if (!seqs) return SeqRows{(long long)b * L, (long long)b * nblk, L};
  const int* e = seqs + kSeqFields * b;
  return SeqRows{e[f_start], e[f_blk], e[f_len]};
}

// TRANSPOSED (64-row blocks only): the codes of block r of head h go out as one [D][64] tile,
// [B, H, nblk, D, 64], rows past the sequence end as 0 (the INT8 value-cache layout of decode);
// the tile is transposed in LDS and written in 16-byte runs.
template <int D, int BLK, bool TRANSPOSED = false>
__global__ __launch_bounds__(kPrepThreads) void quantize_blocks_kernel(
    const _Float16* __restrict__ X, int8_t* __restrict__ X8, uint16_t* __restrict__ dX,
    int L, int H, int nblk, const int* __restrict__ seqs, int f_start, int f_len, int f_blk) {
  constexpr int kChunksPerRow = D / 8;                          // 16-byte chunks of 8 halfs
  constexpr int kPer = BLK * kChunksPerRow / kPrepThreads;      // chunks per thread
  static_assert(kPer * kPrepThreads == BLK * kChunksPerRow, "block split");
  __shared__ float red[kPrepThreads / kWave];
  // TRANSPOSED: the block's codes as [D][BLK] (rows padded to keep 16-byte alignment)
  __shared__ __align__(16) uint8_t tile[TRANSPOSED ? D : 1][TRANSPOSED ? BLK + 16 : 16];

  const int r = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const SeqRows sq = seq_rows(seqs, b, L, nblk, f_start, f_len, f_blk);
  const int row0 = r * BLK;
  if (row0 >= sq.len) return;   // past the end of a shorter sequence
  const int rows = min(BLK, sq.len - row0);

  uint4 v[kPer];
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int c = threadIdx.x + kPrepThreads * i;
    const int row = c / kChunksPerRow, ch = c % kChunksPerRow;
    if (row < rows) {
      const size_t off = ((size_t)(sq.start + row0 + row) * H + h) * D + ch * 8;
      v[i] = ld_global_16(X + off);
      const half8 hv = as_half8(v[i]);
#pragma unroll
      for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)hv[e]));
    } else {
      v[i] = make_uint4(0, 0, 0, 0);
    }
  }
  amax = block_max(amax, red);
  const float d32 = amax / 127.0f;   // IEEE FP32 division (compiled without fast-math)

#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int c = threadIdx.x + kPrepThreads * i;
    const int row = c / kChunksPerRow, ch = c % kChunksPerRow;
    if (row < rows) {
      const half8 hv = as_half8(v[i]);
      uint32_t packed[2] = {0u, 0u};
      if (amax > 0.0f) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float q = rintf((float)hv[e] / d32);          // round half to even
          q = fminf(127.0f, fmaxf(-127.0f, q));
          const uint32_t byte = (uint32_t)((int)q) & 0xffu;
          packed[e >> 2] |= byte << (8 * (e & 3));
        }
      }
      if constexpr (TRANSPOSED) {
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[ch * 8 + e][row] = (uint8_t)(packed[e >> 2] >> (8 * (e & 3)));
      } else {
        const size_t off = ((size_t)(sq.start + row0 + row) * H + h) * D + ch * 8;
        *reinterpret_cast<uint2*>(X8 + off) = make_uint2(packed[0], packed[1]);
      }
    } else if constexpr (TRANSPOSED) {   // padding keys of the last tile
#pragma unroll
      for (int e = 0; e < 8; ++e) tile[ch * 8 + e][row] = 0;
    }
  }
  if constexpr (TRANSPOSED) {   // the [D][64] tile out in 16-byte runs
    __syncthreads();
    int8_t* t = X8 + (((size_t)b * H + h) * nblk + r) * (size_t)(D * BLK);
    for (int k = threadIdx.x; k < D * BLK / 16; k += kPrepThreads) {
      const int c = k / (BLK / 16), j = k % (BLK / 16);
      *reinterpret_cast<uint4*>(t + (size_t)c * BLK + 16 * j) =
          *reinterpret_cast<const uint4*>(&tile[c][16 * j]);
    }
  }
  if (threadIdx.x == 0) {
    const _Float16 s = (amax > 0.0f) ? (_Float16)d32 : (_Float16)0.0f;   // RNE
    uint16_t bits;
    __builtin_memcpy(&bits, &s, 2);
    dX[(size_t)(sq.blk + r) * H + h] = bits;
  }
}

// Position p (0..63) of a V tile row holds key (16*(p/16) + 8*((p%8)/4) + 4*((p/8)%2) + p%4).
__device__ __forceinline__ int vt_key_of_pos(int p) {
  const int t = p >> 4, h = (p >> 3) & 1, e = p & 7;
  return 16 * t + 8 * (e >> 2) + 4 * h + (e & 3);
}

// Tile n of KV head h of sequence b lands at tile index (b H + h) T_n + n for one common length,
// or h * (all key tiles of the batch) + (first key tile of b) + n for a variable-length batch.
template <int D>
__global__ __launch_bounds__(kPrepThreads) void v_tiles_kernel(
    const _Float16* __restrict__ V, _Float16* __restrict__ Vt, int L, int H, int T_n,
    const int* __restrict__ seqs, int batch) {
  constexpr int kRowHalfs = D + 8;                  // padded LDS row: 8 rows hit 8 bank groups
  constexpr int kInChunks = kBlockN * D / 8;        // 16-byte chunks of the input tile
  constexpr int kOutChunks = D * kBlockN / 8;
  __shared__ __align__(16) _Float16 tile[kBlockN * kRowHalfs];

  const int n = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  long long start = (long long)b * L, dst_tile = ((long long)b * H + h) * T_n + n;
  int len = L;
  if (seqs) {
    const int* e = seqs + kSeqFields * b;
    start = e[kSeqKStart];
    len = e[kSeqKLen];
    dst_tile = (long long)h * seqs[kSeqFields * batch + kSeqKTile] + e[kSeqKTile] + n;
  }
  const int key0 = n * kBlockN;
  if (key0 >= len) return;   // past the end of a shorter sequence
  for (int c = threadIdx.x; c < kInChunks; c += kPrepThreads) {
    const int row = c / (D / 8), ch = c % (D / 8);
    uint4 val = make_uint4(0, 0, 0, 0);
    if (key0 + row < len) val = ld_global_16(V + ((size_t)(start + key0 + row) * H + h) * D + ch * 8);
    *reinterpret_cast<uint4*>(&tile[row * kRowHalfs + ch * 8]) = val;
  }
  __syncthreads();
  _Float16* out = Vt + (size_t)dst_tile * (size_t)(D * kBlockN);
  for (int c = threadIdx.x; c < kOutChunks; c += kPrepThreads) {
    const int d = c / 8, ch = c % 8;
    half8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = tile[vt_key_of_pos(ch * 8 + e) * kRowHalfs + d];
    *reinterpret_cast<half8*>(out + d * kBlockN + ch * 8) = o;
  }
}

}  // namespace

namespace {

// Sequence table of a variable-length batch, built on the device from cu_seqlens so that the
// host never reads them: for each sequence its rows in the packed Q and K (clamped to the
// tensors, the maximum lengths and after the previous sequence, so that a malformed table
// stays in bounds) and the running totals of scale blocks, query-tile rows and key tiles;
// row B holds the totals.  Once a sequence's query-tile rows would run past the route_rows
// routing rows the caller passed, it and every later sequence are treated as empty (no query
// rows).  One thread walks the batch.
__global__ void seq_table_kernel(const int* __restrict__ cu_q, const int* __restrict__ cu_k,
                                 int batch, int total_q, int total_k, int max_q, int max_k,
                                 int block_m, int route_rows, int* __restrict__ seqs) {
  if (threadIdx.x != 0) return;
  int q_end = 0, k_end = 0, qblk = 0, kblk = 0, qtile = 0, ktile = 0;
  bool fits = true;
  for (int b = 0; b < batch; ++b) {
    const int qs = min(max(cu_q[b], q_end), total_q);
    const int qe = min(max(cu_q[b + 1], qs), total_q);
    const int ks = min(max(cu_k[b], k_end), total_k);
    const int ke = min(max(cu_k[b + 1], ks), total_k);
    int ql = min(qe - qs, max_q);
    const int kl = min(ke - ks, max_k);
    fits = fits && qtile + (ql + block_m - 1) / block_m <= route_rows;
    if (!fits) ql = 0;
    int* e = seqs + kSeqFields * b;
    e[kSeqQStart] = qs; e[kSeqQLen] = ql; e[kSeqKStart] = ks; e[kSeqKLen] = kl;
    e[kSeqQBlk] = qblk; e[kSeqKBlk] = kblk; e[kSeqQTile] = qtile; e[kSeqKTile] = ktile;
    qblk += (ql + kQuantBlockQ - 1) / kQuantBlockQ;
    kblk += (kl + kQuantBlockK - 1) / kQuantBlockK;
    qtile += (ql + block_m - 1) / block_m;
    ktile += (kl + kBlockN - 1) / kBlockN;
    q_end = qs + ql;
    k_end = ks + kl;
  }
  int* e = seqs + kSeqFields * batch;
  e[kSeqQStart] = q_end; e[kSeqQLen] = 0; e[kSeqKStart] = k_end; e[kSeqKLen] = 0;
  e[kSeqQBlk] = qblk; e[kSeqKBlk] = kblk; e[kSeqQTile] = qtile; e[kSeqKTile] = ktile;
}

}  // namespace

hipError_t launch_seq_table(const int* cu_q, const int* cu_k, int batch, int total_q, int total_k,
                            int max_q, int max_k, int block_m, int route_rows, int* seqs,
                            hipStream_t stream) {
  hipLaunchKernelGGL(seq_table_kernel, dim3(1), dim3(64), 0, stream, cu_q, cu_k, batch, total_q,
                     total_k, max_q, max_k, block_m, route_rows, seqs);
  return hipGetLastError();
}

hipError_t launch_quantize(const _Float16* X, int8_t* X8, uint16_t* dX, int B, int L, int H,
                           int d, int block_rows, const int* seqs, bool keys, hipStream_t stream,
                           bool transposed) {
  const int nblk = (L + block_rows - 1) / block_rows;
  dim3 grid(nblk, H, B), block(kPrepThreads);
  const int fs = keys ? kSeqKStart : kSeqQStart, fl = keys ? kSeqKLen : kSeqQLen;
  const int fb = keys ? kSeqKBlk : kSeqQBlk;
  if (transposed) {   // value cache: 64-row blocks, fixed lengths
    if (seqs || block_rows != 64) return hipErrorInvalidValue;
    if (d == 128)
      hipLaunchKernelGGL((quantize_blocks_kernel<128, 64, true>), grid, block, 0, stream, X, X8, dX, L, H, nblk, seqs, fs, fl, fb);
    else if (d == 64)
      hipLaunchKernelGGL((quantize_blocks_kernel<64, 64, true>), grid, block, 0, stream, X, X8, dX, L, H, nblk, seqs, fs, fl, fb);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (d == 128 && block_rows == 128)
    hipLaunchKernelGGL((quantize_blocks_kernel<128, 128>), grid, block, 0, stream, X, X8, dX, L, H, nblk, seqs, fs, fl, fb);
  else if (d == 128 && block_rows == 64)
    hipLaunchKernelGGL((quantize_blocks_kernel<128, 64>), grid, block, 0, stream, X, X8, dX, L, H, nblk, seqs, fs, fl, fb);
  else if (d == 64 && block_rows == 128)
    hipLaunchKernelGGL((quantize_blocks_kernel<64, 128>), grid, block, 0, stream, X, X8, dX, L, H, nblk, seqs, fs, fl, fb);
  else if (d == 64 && block_rows == 64)
    hipLaunchKernelGGL((quantize_blocks_kernel<64, 64>), grid, block, 0, stream, X, X8, dX, L, H, nblk, seqs, fs, fl, fb);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_v_tiles(const _Float16* V, _Float16* Vt, int B, int L, int H, int d,
                          const int* seqs, hipStream_t stream) {
  const int T_n = (L + kBlockN - 1) / kBlockN;
  dim3 grid(T_n, H, B), block(kPrepThreads);
  if (d == 128)
    hipLaunchKernelGGL((v_tiles_kernel<128>), grid, block, 0, stream, V, Vt, L, H, T_n, seqs, B);
  else if (d == 64)
    hipLaunchKernelGGL((v_tiles_kernel<64>), grid, block, 0, stream, V, Vt, L, H, T_n, seqs, B);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tilemix
