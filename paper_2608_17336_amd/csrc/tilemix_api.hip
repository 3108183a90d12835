// tilemix_api.hip -- the C ABI declared in include/tilemix.h: argument validation, the
// workspace plan and the launch sequence.  No allocation, no synchronization, no state
// beyond a per-thread error message.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "tilemix.h"
#include "tilemix_device.h"
#include "tilemix_internal.h"

namespace tilemix {
namespace api {

namespace {
thread_local char g_last_error[512] = "";
}  // namespace

const char* last_error() { return g_last_error; }

tilemix_status fail(tilemix_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

tilemix_status ok() {
  g_last_error[0] = '\0';
  return TILEMIX_OK;
}

namespace {
long long cdiv_ll(long long a, long long b) { return (a + b - 1) / b; }
}  // namespace

tilemix_status validate(const tilemix_params* p) {
  if (!p) return fail(TILEMIX_ERR_NULL, "params is NULL");
  if (p->batch < 1 || p->heads_q < 1 || p->heads_kv < 1 || p->len_q < 1 || p->len_k < 1)
    return fail(TILEMIX_ERR_SHAPE, "batch, heads and lengths must be >= 1");
  if (p->heads_q % p->heads_kv != 0)
    return fail(TILEMIX_ERR_SHAPE, "heads_q (%d) must be a multiple of heads_kv (%d)", p->heads_q,
                p->heads_kv);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(TILEMIX_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", p->head_dim);
  if (p->block_m != 64 && p->block_m != 128)
    return fail(TILEMIX_ERR_UNSUPPORTED, "block_m %d not supported (64 or 128)", p->block_m);
  if (p->block_n != 64)
    return fail(TILEMIX_ERR_UNSUPPORTED, "block_n %d not supported (64)", p->block_n);
  if (p->group_size < 1) return fail(TILEMIX_ERR_SHAPE, "group_size must be >= 1");
  if (p->causal != 0 && p->causal != 1) return fail(TILEMIX_ERR_SHAPE, "causal must be 0 or 1");
  if (!(isfinite(p->scale) && p->scale > 0.0f))
    return fail(TILEMIX_ERR_SHAPE, "scale must be finite and > 0");
  if (p->route_per_batch != 0 && p->route_per_batch != 1)
    return fail(TILEMIX_ERR_SHAPE, "route_per_batch must be 0 or 1");
  if (p->route_hint != -1 && p->route_hint != 0)
    return fail(TILEMIX_ERR_SHAPE, "route_hint must be -1 or 0");
  const long long rows_q = (long long)p->batch * p->len_q * p->heads_q;
  const long long rows_k = (long long)p->batch * p->len_k * p->heads_kv;
  if (rows_q * p->head_dim > (1LL << 40) || rows_k * p->head_dim > (1LL << 40))
    return fail(TILEMIX_ERR_SHAPE, "tensor too large");
  if (cdiv_ll(p->len_k, p->block_n) > tilemix::kMaxKeyTiles)
    return fail(TILEMIX_ERR_UNSUPPORTED, "len_k %d exceeds the supported %d keys", p->len_k,
                tilemix::kMaxKeyTiles * tilemix::kBlockN);
  const long long grid = (long long)p->batch * p->heads_q * cdiv_ll(p->len_q, p->block_m);
  if (grid > 0x7fffffffLL) return fail(TILEMIX_ERR_SHAPE, "too many query tiles");
  if ((long long)p->heads_kv * p->batch > 65535 || p->heads_q > 65535)
    return fail(TILEMIX_ERR_SHAPE, "too many heads");
  return TILEMIX_OK;
}

}  // namespace api
}  // namespace tilemix

namespace {

using tilemix::api::fail;
using tilemix::api::ok;
using tilemix::api::validate;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
long long cdiv(long long a, long long b) { return (a + b - 1) / b; }

// Derived sizes of one problem.  A variable-length batch (total_q >= 0) sizes its buffers by
// the packed row counts: B sequences of total_q / total_k rows hold at most total / block + B
// blocks or tiles, and its workspace starts with the device-built sequence table.
struct Plan {
  long long T_m, T_n, T_mask, W;
  long long nKB;
  size_t seq_bytes, k8_bytes, dk_bytes, vt_bytes;
  size_t seq_off, k8_off, dk_off, vt_off, total;
};

// fused: the on-the-fly operand mode, whose workspace holds the V tiles only.
Plan make_plan(const tilemix_params* p, long long total_q = -1, long long total_k = -1,
               bool fused = false) {
  Plan pl{};
  pl.T_m = cdiv(p->len_q, p->block_m);
  pl.T_n = cdiv(p->len_k, p->block_n);
  pl.T_mask = cdiv(pl.T_n, p->group_size);
  pl.W = cdiv(pl.T_mask, 64);
  pl.nKB = cdiv(p->len_k, tilemix::kQuantBlockK);
  const size_t d = (size_t)p->head_dim;
  const bool varlen = total_q >= 0;
  const long long rows_k = varlen ? total_k : (long long)p->batch * p->len_k;
  const long long kblocks = varlen ? cdiv(total_k, tilemix::kQuantBlockK) + p->batch : p->batch * pl.nKB;
  const long long ktiles = varlen ? cdiv(total_k, tilemix::kBlockN) + p->batch : p->batch * pl.T_n;
  pl.seq_bytes = varlen ? (size_t)(p->batch + 1) * tilemix::kSeqFields * sizeof(int) : 0;
  // The attention kernel quantizes each query block itself (one workgroup per block), so only
  // the key operands of the quantize-once pass live in the workspace.
  pl.k8_bytes = fused ? 0 : (size_t)rows_k * p->heads_kv * d;
  pl.dk_bytes = fused ? 0 : (size_t)kblocks * p->heads_kv * 2;
  pl.vt_bytes = (size_t)ktiles * p->heads_kv * d * tilemix::kBlockN * 2;
  pl.seq_off = 0;
  pl.k8_off = align256(pl.seq_off + pl.seq_bytes);
  pl.dk_off = align256(pl.k8_off + pl.k8_bytes);
  pl.vt_off = align256(pl.dk_off + pl.dk_bytes);
  pl.total = align256(pl.vt_off + pl.vt_bytes);
  return pl;
}

bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr % a) == 0; }

tilemix_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return TILEMIX_OK;
  return fail(TILEMIX_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

int32_t tilemix_route_words_per_row(const tilemix_params* params) {
  if (validate(params) != TILEMIX_OK) return 0;
  return (int32_t)make_plan(params).W;
}

tilemix_status tilemix_workspace_size(const tilemix_params* params, size_t* bytes) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  if (!bytes) return fail(TILEMIX_ERR_NULL, "bytes is NULL");
  *bytes = make_plan(params).total;
  return ok();
}

namespace {

tilemix_status check_workspace(const Plan& pl, const void* workspace, size_t workspace_bytes) {
  if (!workspace) return fail(TILEMIX_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned(workspace, 256)) return fail(TILEMIX_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (workspace_bytes < pl.total)
    return fail(TILEMIX_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, pl.total);
  return TILEMIX_OK;
}

// seqs: the sequence table of a variable-length batch (in the workspace), or nullptr.
// fused: the on-the-fly operand mode (no quantize-once pass).
// Q is not read here: the attention kernel quantizes the query blocks itself.
tilemix_status prepare_impl(const tilemix_params& p, const Plan& pl, const void* /*Q*/, const void* K,
                            const void* V, void* workspace, hipStream_t s,
                            const int* seqs = nullptr, bool fused = false) {
  char* ws = static_cast<char*>(workspace);
  int8_t* k8 = reinterpret_cast<int8_t*>(ws + pl.k8_off);
  uint16_t* dk = reinterpret_cast<uint16_t*>(ws + pl.dk_off);
  _Float16* vt = reinterpret_cast<_Float16*>(ws + pl.vt_off);
  tilemix_status st;
  if (p.route_hint != 0 && !fused) {   // an all-FP16 map skips the quantize-once pass
    st = hip_status(tilemix::launch_quantize(static_cast<const _Float16*>(K), k8, dk, p.batch,
                                             p.len_k, p.heads_kv, p.head_dim,
                                             tilemix::kQuantBlockK, seqs, true, s), "quantize K");
    if (st != TILEMIX_OK) return st;
  }
  return hip_status(tilemix::launch_v_tiles(static_cast<const _Float16*>(V), vt, p.batch, p.len_k,
                                            p.heads_kv, p.head_dim, seqs, s), "V tiles");
}

tilemix_status attend_impl(const tilemix_params& p, const Plan& pl, const void* Q, const void* K,
                           const uint64_t* route_bits, void* O, const void* workspace,
                           hipStream_t s, const int* seqs = nullptr, bool fused = false,
                           const tilemix_debug_export* dbg = nullptr) {
  const char* ws = static_cast<const char*>(workspace);
  tilemix::AttnArgs a{};
  a.seqs = seqs;
  a.Q = static_cast<const _Float16*>(Q);
  a.K = static_cast<const _Float16*>(K);
  a.Vt = reinterpret_cast<const _Float16*>(ws + pl.vt_off);
  a.K8 = reinterpret_cast<const int8_t*>(ws + pl.k8_off);
  a.dK = reinterpret_cast<const uint16_t*>(ws + pl.dk_off);
  a.route = route_bits;
  a.O = static_cast<_Float16*>(O);
  a.B = p.batch; a.Hq = p.heads_q; a.Hk = p.heads_kv; a.Lq = p.len_q; a.Lk = p.len_k;
  a.T_m = (int)pl.T_m; a.T_n = (int)pl.T_n; a.W = (int)pl.W; a.g = p.group_size;
  a.nKB = (int)pl.nKB;
  a.causal = p.causal;
  a.force_fp16 = p.route_hint == 0 ? 1 : 0;
  a.on_the_fly = fused ? 1 : 0;
  a.route_batch_stride = p.route_per_batch ? (long long)p.heads_kv * pl.T_m * pl.W : 0;
  a.scale_log2e = p.scale * 1.4426950408889634f;
  if (dbg) {
    a.dbg_q8 = dbg->q8;
    a.dbg_dq = dbg->dq;
    a.dbg_tiles = dbg->tiles;
    a.dbg_kind = dbg->kinds;
  }
  return hip_status(tilemix::launch_routed_attention(a, p.head_dim, p.block_m, s), "routed attention");
}

tilemix_status check_qkv(const void* Q, const void* K, const void* V) {
  if (!Q || !K || !V) return fail(TILEMIX_ERR_NULL, "Q, K and V must be non-NULL");
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16))
    return fail(TILEMIX_ERR_ALIGN, "Q, K and V must be 16-byte aligned");
  return TILEMIX_OK;
}

tilemix_status check_out(const uint64_t* route_bits, const void* O) {
  if (!O || !route_bits) return fail(TILEMIX_ERR_NULL, "O and route_bits must be non-NULL");
  if (!aligned(O, 16)) return fail(TILEMIX_ERR_ALIGN, "O must be 16-byte aligned");
  if (!aligned(route_bits, 8)) return fail(TILEMIX_ERR_ALIGN, "route_bits must be 8-byte aligned");
  return TILEMIX_OK;
}

}  // namespace

namespace {

tilemix_status check_varlen(const tilemix_params* params, int32_t total_q, int32_t total_k) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  if (total_q < 1 || total_k < 1) return fail(TILEMIX_ERR_SHAPE, "total_q and total_k must be >= 1");
  if (params->route_per_batch != 0)
    return fail(TILEMIX_ERR_SHAPE, "route_per_batch must be 0 for a variable-length batch");
  if ((long long)total_q * params->heads_q * params->head_dim > (1LL << 40) ||
      (long long)total_k * params->heads_kv * params->head_dim > (1LL << 40))
    return fail(TILEMIX_ERR_SHAPE, "tensor too large");
  return TILEMIX_OK;
}

// A variable-length batch (total_q >= 0) or a fixed-length one (total_q < 0).
struct Varlen {
  int32_t total_q = -1, total_k = -1;
  const int32_t* cu_q = nullptr;
  const int32_t* cu_k = nullptr;
  int32_t route_rows = 0;
};

// Every prefill entry point: validation, the workspace plan, the sequence table of a
// variable-length batch, the operand preparation and the attention kernel.
tilemix_status run_prefill(const tilemix_params* params, bool fused, const Varlen& vl,
                           const void* Q, const void* K, const void* V,
                           const uint64_t* route_bits, void* O, void* workspace,
                           size_t workspace_bytes, void* stream,
                           const tilemix_debug_export* dbg = nullptr) {
  const bool varlen = vl.total_q >= 0;
  tilemix_status st = varlen ? check_varlen(params, vl.total_q, vl.total_k) : validate(params);
  if (st != TILEMIX_OK) return st;
  if (varlen) {
    if (!vl.cu_q || !vl.cu_k) return fail(TILEMIX_ERR_NULL, "cu_seqlens must be non-NULL");
    if (!aligned(vl.cu_q, 4) || !aligned(vl.cu_k, 4))
      return fail(TILEMIX_ERR_ALIGN, "cu_seqlens must be 4-byte aligned");
    if (vl.route_rows < 0) return fail(TILEMIX_ERR_SHAPE, "route_rows must be >= 0");
  }
  if ((st = check_qkv(Q, K, V)) != TILEMIX_OK) return st;
  if ((st = check_out(route_bits, O)) != TILEMIX_OK) return st;
  const Plan pl = varlen ? make_plan(params, vl.total_q, vl.total_k, fused)
                         : make_plan(params, -1, -1, fused);
  if ((st = check_workspace(pl, workspace, workspace_bytes)) != TILEMIX_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int* seqs = nullptr;
  if (varlen) {
    seqs = reinterpret_cast<int*>(static_cast<char*>(workspace) + pl.seq_off);
    st = hip_status(tilemix::launch_seq_table(vl.cu_q, vl.cu_k, params->batch, vl.total_q,
                                              vl.total_k, params->len_q, params->len_k,
                                              params->block_m, vl.route_rows, seqs, s),
                    "sequence table");
    if (st != TILEMIX_OK) return st;
  }
  if ((st = prepare_impl(*params, pl, Q, K, V, workspace, s, seqs, fused)) != TILEMIX_OK) return st;
  if ((st = attend_impl(*params, pl, Q, K, route_bits, O, workspace, s, seqs, fused, dbg)) != TILEMIX_OK)
    return st;
  return ok();
}

}  // namespace

tilemix_status tilemix_prefill(const tilemix_params* params, const void* Q, const void* K,
                               const void* V, const uint64_t* route_bits, void* O,
                               void* workspace, size_t workspace_bytes, void* stream) {
  return run_prefill(params, false, Varlen{}, Q, K, V, route_bits, O, workspace, workspace_bytes,
                     stream);
}

tilemix_status tilemix_fused_workspace_size(const tilemix_params* params, size_t* bytes) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  if (!bytes) return fail(TILEMIX_ERR_NULL, "bytes is NULL");
  *bytes = make_plan(params, -1, -1, true).total;
  return ok();
}

tilemix_status tilemix_prefill_fused(const tilemix_params* params, const void* Q, const void* K,
                                     const void* V, const uint64_t* route_bits, void* O,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  return run_prefill(params, true, Varlen{}, Q, K, V, route_bits, O, workspace, workspace_bytes,
                     stream);
}

tilemix_status tilemix_prepare(const tilemix_params* params, const void* Q, const void* K,
                               const void* V, void* workspace, size_t workspace_bytes,
                               void* stream) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  if ((st = check_qkv(Q, K, V)) != TILEMIX_OK) return st;
  const Plan pl = make_plan(params);
  if ((st = check_workspace(pl, workspace, workspace_bytes)) != TILEMIX_OK) return st;
  if ((st = prepare_impl(*params, pl, Q, K, V, workspace, static_cast<hipStream_t>(stream))) != TILEMIX_OK)
    return st;
  return ok();
}

tilemix_status tilemix_attend(const tilemix_params* params, const void* Q, const void* K,
                              const uint64_t* route_bits, void* O, const void* workspace,
                              size_t workspace_bytes, void* stream) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  if (!Q || !K) return fail(TILEMIX_ERR_NULL, "Q and K must be non-NULL");
  if (!aligned(Q, 16) || !aligned(K, 16)) return fail(TILEMIX_ERR_ALIGN, "Q and K must be 16-byte aligned");
  if ((st = check_out(route_bits, O)) != TILEMIX_OK) return st;
  const Plan pl = make_plan(params);
  if ((st = check_workspace(pl, workspace, workspace_bytes)) != TILEMIX_OK) return st;
  if ((st = attend_impl(*params, pl, Q, K, route_bits, O, workspace, static_cast<hipStream_t>(stream))) != TILEMIX_OK)
    return st;
  return ok();
}

namespace {

// The workspace of tilemix_prefill_noalloc: one file-scope device array, which the library's
// code object holds on every GPU it is loaded on until the process ends.  Host code never
// passes the array's name itself to a kernel (on the host it is a stand-in, not a device
// address): it uses the address hipGetSymbolAddress returns for the current device, looked up
// once per device on that device's first call.
__device__ __align__(256) unsigned char scratch[TILEMIX_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

tilemix_status scratch_of_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(TILEMIX_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(TILEMIX_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return TILEMIX_OK;
}

}  // namespace

tilemix_status tilemix_prefill_noalloc(const tilemix_params* params, const void* Q, const void* K,
                                       const void* V, const uint64_t* route_bits, void* O,
                                       void* stream) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  const Plan pl = make_plan(params);
  if (pl.total > (size_t)TILEMIX_NOALLOC_SCRATCH_BYTES)
    return fail(TILEMIX_ERR_WORKSPACE,
                "the problem needs %zu bytes of workspace; tilemix_prefill_noalloc serves at most "
                "%zu (use tilemix_prefill with a caller-owned workspace)",
                pl.total, (size_t)TILEMIX_NOALLOC_SCRATCH_BYTES);
  if ((st = check_qkv(Q, K, V)) != TILEMIX_OK) return st;
  if ((st = check_out(route_bits, O)) != TILEMIX_OK) return st;
  void* ws = nullptr;
  if ((st = scratch_of_current_device(&ws)) != TILEMIX_OK) return st;
  return run_prefill(params, false, Varlen{}, Q, K, V, route_bits, O, ws,
                     (size_t)TILEMIX_NOALLOC_SCRATCH_BYTES, stream);
}

tilemix_status tilemix_varlen_workspace_size(const tilemix_params* params, int32_t total_q,
                                             int32_t total_k, size_t* bytes) {
  tilemix_status st = check_varlen(params, total_q, total_k);
  if (st != TILEMIX_OK) return st;
  if (!bytes) return fail(TILEMIX_ERR_NULL, "bytes is NULL");
  *bytes = make_plan(params, total_q, total_k).total;
  return ok();
}

tilemix_status tilemix_prefill_varlen(const tilemix_params* params, int32_t total_q,
                                      int32_t total_k, const int32_t* cu_seqlens_q,
                                      const int32_t* cu_seqlens_k, const void* Q, const void* K,
                                      const void* V, const uint64_t* route_bits,
                                      int32_t route_rows, void* O, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  Varlen vl;
  vl.total_q = total_q; vl.total_k = total_k;
  vl.cu_q = cu_seqlens_q; vl.cu_k = cu_seqlens_k;
  vl.route_rows = route_rows;
  if (total_q < 0) return check_varlen(params, total_q, total_k);
  return run_prefill(params, false, vl, Q, K, V, route_bits, O, workspace, workspace_bytes, stream);
}

tilemix_status tilemix_varlen_fused_workspace_size(const tilemix_params* params, int32_t total_q,
                                                   int32_t total_k, size_t* bytes) {
  tilemix_status st = check_varlen(params, total_q, total_k);
  if (st != TILEMIX_OK) return st;
  if (!bytes) return fail(TILEMIX_ERR_NULL, "bytes is NULL");
  *bytes = make_plan(params, total_q, total_k, true).total;
  return ok();
}

tilemix_status tilemix_prefill_varlen_fused(const tilemix_params* params, int32_t total_q,
                                            int32_t total_k, const int32_t* cu_seqlens_q,
                                            const int32_t* cu_seqlens_k, const void* Q,
                                            const void* K, const void* V,
                                            const uint64_t* route_bits, int32_t route_rows,
                                            void* O, void* workspace, size_t workspace_bytes,
                                            void* stream) {
  Varlen vl;
  vl.total_q = total_q; vl.total_k = total_k;
  vl.cu_q = cu_seqlens_q; vl.cu_k = cu_seqlens_k;
  vl.route_rows = route_rows;
  if (total_q < 0) return check_varlen(params, total_q, total_k);
  return run_prefill(params, true, vl, Q, K, V, route_bits, O, workspace, workspace_bytes, stream);
}

tilemix_status tilemix_debug_prefill(const tilemix_params* params, int32_t fused, int32_t total_q,
                                     int32_t total_k, const int32_t* cu_seqlens_q,
                                     const int32_t* cu_seqlens_k, const void* Q, const void* K,
                                     const void* V, const uint64_t* route_bits, int32_t route_rows,
                                     void* O, void* workspace, size_t workspace_bytes,
                                     const tilemix_debug_export* dbg, void* stream) {
  if (!dbg || !dbg->q8 || !dbg->dq || !dbg->tiles || !dbg->kinds)
    return fail(TILEMIX_ERR_NULL, "every export buffer must be non-NULL");
  if (!aligned(dbg->q8, 16) || !aligned(dbg->dq, 2) || !aligned(dbg->tiles, 4) ||
      !aligned(dbg->kinds, 4))
    return fail(TILEMIX_ERR_ALIGN, "q8 must be 16-byte, dq 2-byte, tiles and kinds 4-byte aligned");
  if (fused != 0 && fused != 1) return fail(TILEMIX_ERR_SHAPE, "fused must be 0 or 1");
  Varlen vl;
  if (total_q >= 0) {
    vl.total_q = total_q; vl.total_k = total_k;
    vl.cu_q = cu_seqlens_q; vl.cu_k = cu_seqlens_k;
    vl.route_rows = route_rows;
  }
  return run_prefill(params, fused == 1, vl, Q, K, V, route_bits, O, workspace, workspace_bytes,
                     stream, dbg);
}

namespace {

tilemix_status check_decode(const tilemix_params* p) {
  tilemix_status st = validate(p);
  if (st != TILEMIX_OK) return st;
  if (p->len_q != 1) return fail(TILEMIX_ERR_UNSUPPORTED, "decode takes one query token (len_q = 1)");
  if (p->heads_q / p->heads_kv > tilemix::kDecMaxGroup)
    return fail(TILEMIX_ERR_UNSUPPORTED, "decode supports at most %d query heads per KV head",
                tilemix::kDecMaxGroup);
  return TILEMIX_OK;
}

size_t decode_workspace(const tilemix_params* p) {
  const size_t rows = (size_t)p->batch * p->heads_q * tilemix::decode_chunks(p->batch, p->heads_kv, p->len_k);
  return align256(rows * sizeof(float)) * 2 + align256(rows * p->head_dim * sizeof(float));
}

}  // namespace

tilemix_status tilemix_quantize_kv(const tilemix_params* params, const void* K, const void* V,
                                   int8_t* K8, uint16_t* dK, int8_t* V8, uint16_t* dV,
                                   void* stream) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  const tilemix_params& p = *params;
  if (!K || !V || !K8 || !dK || !V8 || !dV) return fail(TILEMIX_ERR_NULL, "NULL tensor pointer");
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(K8, 16) || !aligned(V8, 16) ||
      !aligned(dK, 2) || !aligned(dV, 2))
    return fail(TILEMIX_ERR_ALIGN, "K, V, K8, V8 must be 16-byte and dK, dV 2-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = hip_status(tilemix::launch_quantize(static_cast<const _Float16*>(K), K8, dK, p.batch, p.len_k,
                                           p.heads_kv, p.head_dim, tilemix::kQuantBlockK, nullptr,
                                           true, s), "quantize K");
  if (st != TILEMIX_OK) return st;
  st = hip_status(tilemix::launch_quantize(static_cast<const _Float16*>(V), V8, dV, p.batch, p.len_k,
                                           p.heads_kv, p.head_dim, tilemix::kQuantBlockK, nullptr,
                                           true, s, /*transposed=*/true), "quantize V");
  if (st != TILEMIX_OK) return st;
  return ok();
}

tilemix_status tilemix_decode_workspace_size(const tilemix_params* params, size_t* bytes) {
  tilemix_status st = check_decode(params);
  if (st != TILEMIX_OK) return st;
  if (!bytes) return fail(TILEMIX_ERR_NULL, "bytes is NULL");
  *bytes = decode_workspace(params);
  return ok();
}

namespace {

tilemix_status decode_impl(const tilemix_params* params, const int32_t* seqlens_k,
                           const void* Q, const void* K, const int8_t* K8, const uint16_t* dK,
                           const int8_t* V8, const uint16_t* dV, const uint64_t* route_bits,
                           void* O, void* workspace, size_t workspace_bytes, void* stream) {
  tilemix_status st = check_decode(params);
  if (st != TILEMIX_OK) return st;
  const tilemix_params& p = *params;
  if (!Q || !K || !K8 || !dK || !V8 || !dV || !route_bits || !O)
    return fail(TILEMIX_ERR_NULL, "NULL tensor pointer");
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(K8, 16) || !aligned(V8, 16) ||
      !aligned(dK, 2) || !aligned(dV, 2) || !aligned(route_bits, 8) || !aligned(O, 16))
    return fail(TILEMIX_ERR_ALIGN, "Q, K, K8, V8, O must be 16-byte, dK, dV 2-byte and "
                "route_bits 8-byte aligned");
  const size_t need = decode_workspace(params);
  if (!workspace) return fail(TILEMIX_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned(workspace, 256)) return fail(TILEMIX_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (workspace_bytes < need)
    return fail(TILEMIX_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  const Plan pl = make_plan(params);
  tilemix::DecodeArgs a{};
  a.Q = static_cast<const _Float16*>(Q);
  a.K = static_cast<const _Float16*>(K);
  a.K8 = K8; a.dK = dK; a.V8 = V8; a.dV = dV;
  a.route = route_bits;
  a.O = static_cast<_Float16*>(O);
  a.B = p.batch; a.Hq = p.heads_q; a.Hk = p.heads_kv; a.Lk = p.len_k;
  a.W = (int)pl.W; a.g = p.group_size; a.nKB = (int)pl.nKB;
  a.chunks = tilemix::decode_chunks(p.batch, p.heads_kv, p.len_k);
  a.tiles_per_wave = tilemix::decode_tiles_per_wave(p.batch, p.heads_kv, p.len_k);
  a.route_per_batch = p.route_per_batch;
  a.force_fp16 = p.route_hint == 0 ? 1 : 0;
  a.scale_log2e = p.scale * 1.4426950408889634f;
  a.seqlens = seqlens_k;
  const size_t rows = (size_t)p.batch * p.heads_q * a.chunks;
  char* ws = static_cast<char*>(workspace);
  a.part_m = reinterpret_cast<float*>(ws);
  a.part_z = reinterpret_cast<float*>(ws + align256(rows * sizeof(float)));
  a.part_o = reinterpret_cast<float*>(ws + 2 * align256(rows * sizeof(float)));
  st = hip_status(tilemix::launch_decode(a, p.head_dim, static_cast<hipStream_t>(stream)), "decode");
  if (st != TILEMIX_OK) return st;
  return ok();
}

}  // namespace

tilemix_status tilemix_decode(const tilemix_params* params, const void* Q, const void* K,
                              const int8_t* K8, const uint16_t* dK, const int8_t* V8,
                              const uint16_t* dV, const uint64_t* route_bits, void* O,
                              void* workspace, size_t workspace_bytes, void* stream) {
  return decode_impl(params, nullptr, Q, K, K8, dK, V8, dV, route_bits, O, workspace,
                     workspace_bytes, stream);
}

tilemix_status tilemix_decode_varlen(const tilemix_params* params, const int32_t* seqlens_k,
                                     const void* Q, const void* K, const int8_t* K8,
                                     const uint16_t* dK, const int8_t* V8, const uint16_t* dV,
                                     const uint64_t* route_bits, void* O, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  if (!seqlens_k) return fail(TILEMIX_ERR_NULL, "seqlens_k is NULL");
  if (!aligned(seqlens_k, 4)) return fail(TILEMIX_ERR_ALIGN, "seqlens_k must be 4-byte aligned");
  return decode_impl(params, seqlens_k, Q, K, K8, dK, V8, dV, route_bits, O, workspace,
                     workspace_bytes, stream);
}

tilemix_status tilemix_quantize(const tilemix_params* params, const void* Q, const void* K,
                                int8_t* Q8, uint16_t* dQ, int8_t* K8, uint16_t* dK, void* stream) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  const tilemix_params& p = *params;
  if (!Q || !K || !Q8 || !dQ || !K8 || !dK) return fail(TILEMIX_ERR_NULL, "NULL tensor pointer");
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(Q8, 16) || !aligned(K8, 16) ||
      !aligned(dQ, 2) || !aligned(dK, 2))
    return fail(TILEMIX_ERR_ALIGN, "Q, K, Q8, K8 must be 16-byte and dQ, dK 2-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = hip_status(tilemix::launch_quantize(static_cast<const _Float16*>(Q), Q8, dQ, p.batch, p.len_q,
                                           p.heads_q, p.head_dim, tilemix::kQuantBlockQ, nullptr,
                                           false, s),
                  "quantize Q");
  if (st != TILEMIX_OK) return st;
  st = hip_status(tilemix::launch_quantize(static_cast<const _Float16*>(K), K8, dK, p.batch, p.len_k,
                                           p.heads_kv, p.head_dim, tilemix::kQuantBlockK, nullptr,
                                           true, s),
                  "quantize K");
  if (st != TILEMIX_OK) return st;
  return ok();
}

tilemix_status tilemix_debug_qk_int32(const tilemix_params* params, const int8_t* Q8,
                                      const int8_t* K8, const int32_t* tiles, int32_t count,
                                      int32_t* out, void* stream) {
  tilemix_status st = validate(params);
  if (st != TILEMIX_OK) return st;
  const tilemix_params& p = *params;
  if (count < 0) return fail(TILEMIX_ERR_SHAPE, "count must be >= 0");
  if (count == 0) return ok();
  if (!Q8 || !K8 || !tiles || !out) return fail(TILEMIX_ERR_NULL, "NULL pointer");
  if (!aligned(Q8, 16) || !aligned(K8, 16) || !aligned(tiles, 4) || !aligned(out, 4))
    return fail(TILEMIX_ERR_ALIGN, "Q8, K8 must be 16-byte and tiles, out 4-byte aligned");
  tilemix::DebugTileArgs a{};
  a.Q8 = Q8; a.K8 = K8; a.tiles = tiles; a.out = out; a.count = count;
  a.B = p.batch; a.Hq = p.heads_q; a.Hk = p.heads_kv; a.Lq = p.len_q; a.Lk = p.len_k;
  st = hip_status(tilemix::launch_debug_tiles(a, p.head_dim, p.block_m, static_cast<hipStream_t>(stream)),
                  "debug tiles");
  if (st != TILEMIX_OK) return st;
  return ok();
}

const char* tilemix_status_string(tilemix_status status) {
  switch (status) {
    case TILEMIX_OK: return "ok";
    case TILEMIX_ERR_NULL: return "null pointer";
    case TILEMIX_ERR_SHAPE: return "invalid shape or parameter";
    case TILEMIX_ERR_UNSUPPORTED: return "unsupported configuration";
    case TILEMIX_ERR_ALIGN: return "misaligned pointer";
    case TILEMIX_ERR_WORKSPACE: return "workspace missing or too small";
    case TILEMIX_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* tilemix_last_error(void) { return tilemix::api::last_error(); }

}  // extern "C"
