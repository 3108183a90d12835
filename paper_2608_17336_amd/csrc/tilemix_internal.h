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

// Arguments of the fused routed attention kernel (plain values; passed by value).
struct AttnArgs {
  const _Float16* Q;      // [B, Lq, Hq, d]
  const _Float16* K;      // [B, Lk, Hk, d]
  const _Float16* Vt;     // [B, Hk, T_n, d, 64]: V per 64-key tile, d-major, keys permuted
  const int8_t* Q8;       // [B, Lq, Hq, d]
  const int8_t* K8;       // [B, Lk, Hk, d]
  const uint16_t* dQ;     // FP16 bits [B, nQB, Hq]
  const uint16_t* dK;     // FP16 bits [B, nKB, Hk]
  const uint64_t* route;  // [B_r, Hk, T_m, W]
  _Float16* O;            // [B, Lq, Hq, d]
  int B, Hq, Hk, Lq, Lk;
  int T_m, T_n, W, g;
  int nQB, nKB;
  int causal;
  int force_fp16;         // 1: ignore routing words, every tile takes the FP16 path
  long long route_batch_stride;  // words between the maps of consecutive sequences (0 = shared)
  float scale_log2e;      // softmax scale * log2(e)
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

hipError_t launch_quantize(const _Float16* X, int8_t* X8, uint16_t* dX, int B, int L, int H,
                           int d, int block_rows, hipStream_t stream);
hipError_t launch_v_tiles(const _Float16* V, _Float16* Vt, int B, int L, int H, int d,
                          hipStream_t stream);
hipError_t launch_routed_attention(const AttnArgs& args, int d, int block_m, hipStream_t stream);
hipError_t launch_debug_tiles(const DebugTileArgs& args, int d, int block_m, hipStream_t stream);

}  // namespace tilemix
