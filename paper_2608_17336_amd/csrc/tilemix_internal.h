// tilemix_internal.h -- host-side declarations shared by the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "tilemix.h"

namespace tilemix {

namespace api {
// Record a printf-style message as the calling thread's last error and return `st`.
tilemix_status fail(tilemix_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clear the calling thread's last error and return TILEMIX_OK.
tilemix_status ok();
const char* last_error();
// Check a parameter block (sizes, supported shapes, flags); TILEMIX_OK or an error status.
tilemix_status validate(const tilemix_params* p);
}  // namespace api

// Sequence table of a variable-length batch: int32 [B + 1][kSeqFields], row b = sequence b,
// row B = totals (first free row of Q and K, and the total numbers of Q / K scale blocks,
// query-tile rows and key tiles).
constexpr int kSeqFields = 8;
constexpr int kSeqQStart = 0, kSeqQLen = 1, kSeqKStart = 2, kSeqKLen = 3;
constexpr int kSeqQBlk = 4, kSeqKBlk = 5, kSeqQTile = 6, kSeqKTile = 7;

// Arguments of the fused routed attention kernel (plain values; passed by value).
struct AttnArgs {
  const _Float16* Q;      // [B, Lq, Hq, d]
  const _Float16* K;      // [B, Lk, Hk, d]
  const _Float16* Vt;     // [B, Hk, T_n, d, 64]: V per 64-key tile, d-major, keys permuted
  const int8_t* K8;       // [B, Lk, Hk, d]
  const uint16_t* dK;     // FP16 bits [B, nKB, Hk]
  const uint64_t* route;  // [B_r, Hk, T_m, W]
  _Float16* O;            // [B, Lq, Hq, d]
  // Variable-length batch: sequence table (see kSeqFields), or nullptr when every sequence has
  // the lengths Lq / Lk.  With a table, Lq / Lk are the maximum lengths, Q/K/V/O/K8 are
  // packed [rows, H, d], scales [blocks, H], V tiles [Hk, key tiles, d, 64] and routing rows
  // [query-tile rows, Hk, W].
  const int* seqs;
  int B, Hq, Hk, Lq, Lk;
  int T_m, T_n, W, g;
  int nKB;
  int causal;
  int force_fp16;         // 1: ignore routing words, every tile takes the FP16 path
  int on_the_fly;         // 1: no K8/scales either; the kernel quantizes INT8 key tiles on chip
  long long route_batch_stride;  // words between the maps of consecutive sequences (0 = shared)
  float scale_log2e;      // softmax scale * log2(e)
  // Test-only export of the INT8 operands the kernel itself makes and multiplies (all nullptr
  // in normal calls; a separate kernel instantiation writes them).  A query-tile row index r is
  // b * T_m + m (or, in a variable-length batch, the sequence's first routing row + m).
  int8_t* dbg_q8;         // like Q: the query codes of every row whose tile row has an INT8 group
  uint16_t* dbg_dq;       // FP16 bits [rows r, Hq]: the query-block scale each workgroup used
  int32_t* dbg_tiles;     // [rows r, Hq, T_n, BM, 64]: INT32 products of the INT8-routed tiles
  int32_t* dbg_kind;      // [rows r, Hq, T_n, BM / 32]: per wave, how the tile's products were
                          // formed (kDbg* below); untouched for tiles not on the INT8 route
};

// dbg_kind values.
constexpr int kDbgFolded = 1;   // pipelined, accumulator started at the 1.5 * 2^23 bias
constexpr int kDbgExact = 2;    // pipelined, accumulator started at 0
constexpr int kDbgMasked = 3;   // the per-tile masked path

// Arguments of the INT8 key/value cache decode kernels (one query token per sequence).
constexpr int kDecMaxGroup = 16;   // query heads per KV head
struct DecodeArgs {
  const _Float16* Q;       // [B, Hq, d]
  const _Float16* K;       // FP16 key cache [B, Lk, Hk, d] (FP16-routed groups)
  const int8_t* K8;        // [B, Lk, Hk, d]
  const uint16_t* dK;      // FP16 bits [B, nKB, Hk]
  const int8_t* V8;        // [B, Hk, nKB, d, 64]: per 64-key block, channel-major
  const uint16_t* dV;      // FP16 bits [B, nKB, Hk]
  const uint64_t* route;   // [B_r, Hk, 1, W]
  _Float16* O;             // [B, Hq, d]
  float* part_m;           // [B, Hq, chunks]: chunk max (log2 units)
  float* part_z;           // [B, Hq, chunks]: chunk normalizer
  float* part_o;           // [B, Hq, chunks, d]: chunk output, unnormalized
  // Per-sequence cache lengths [B] (device), or nullptr when every sequence holds Lk keys.
  // Sequence b uses its first min(max(seqlens[b], 0), Lk) cached keys; Lk is the capacity.
  const int* seqlens;
  int B, Hq, Hk, Lk, W, g, nKB, chunks;
  int tiles_per_wave;      // key tiles each wave of the partial kernel streams
  int route_per_batch, force_fp16;
  float scale_log2e;
};

// Arguments of the INT32 tile-product check kernel.
struct DebugTileArgs {
  const int8_t* Q8;
  const int8_t* K8;
  const int32_t* tiles;   // [count, 4] (b, h_q, m, n)
  int32_t* out;           // [count, BM, 64]
  int count;
  int B, Hq, Hk, Lq, Lk;
};

// seqs: sequence table or nullptr (every sequence of length L); keys selects its K fields.
// transposed: write 64-row blocks as [B, H, blocks, d, 64] tiles (the INT8 value cache).
hipError_t launch_quantize(const _Float16* X, int8_t* X8, uint16_t* dX, int B, int L, int H,
                           int d, int block_rows, const int* seqs, bool keys, hipStream_t stream,
                           bool transposed = false);
hipError_t launch_v_tiles(const _Float16* V, _Float16* Vt, int B, int L, int H, int d,
                          const int* seqs, hipStream_t stream);
hipError_t launch_seq_table(const int* cu_q, const int* cu_k, int batch, int total_q, int total_k,
                            int max_q, int max_k, int block_m, int route_rows, int* seqs,
                            hipStream_t stream);
hipError_t launch_routed_attention(const AttnArgs& args, int d, int block_m, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& args, int d, hipStream_t stream);
int decode_tiles_per_wave(int batch, int heads_kv, int len_k);
int decode_chunks(int batch, int heads_kv, int len_k);
hipError_t launch_debug_tiles(const DebugTileArgs& args, int d, int block_m, hipStream_t stream);

}  // namespace tilemix
