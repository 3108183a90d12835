/*
 * tilemix.h -- C ABI of the MI355X (gfx950) TileMix routed prefill attention library.
 *
 * What the library computes (TileMix, arXiv 2608.17336):
 *   Causal (or full) softmax attention O = softmax(S) V over dense FP16 tensors
 *   (Section 3.1), where every legal score tile of BLOCK_M query rows by
 *   BLOCK_N keys is produced by one of two paths chosen by a packed routing
 *   bit (Sections 4.2 and 4.3):
 *     bit 0 (FP16):  S = scale * Q K^T with FP16 operands and FP32 accumulation;
 *     bit 1 (INT8):  S = scale * dQ * dK * (Q8 K8^T), Q8/K8 the blockwise
 *                    symmetric INT8 codes of Q and K with one FP16 scale per
 *                    128-token query block / 64-token key block and head,
 *                    the product accumulated exactly in INT32 (Appendix C).
 *   Both paths feed one online-softmax state; V and the P.V product stay FP16
 *   (Appendix C, "INT8 Score Computation" and "Quantize-Once Execution").
 *
 * Conventions shared by every entry point:
 *   - Tensors are dense and contiguous, token-major with interleaved heads:
 *       Q, O : FP16 [B, L_q, H_q, d]      K, V : FP16 [B, L_k, H_k, d]
 *     Query head h_q reads KV head h_k = h_q / (H_q / H_k) (Section 4.1).
 *   - Routing words: uint64 [B_r, H_k, T_m, W] with T_m = ceil(L_q / BLOCK_M),
 *     T_n = ceil(L_k / BLOCK_N), T_mask = ceil(T_n / g) routing groups per row
 *     and W = ceil(T_mask / 64) words per row.  Key tile n belongs to group
 *     g_j = n / g, found in word g_j / 64 at bit g_j % 64; 1 = INT8, 0 = FP16
 *     (Section 4.2, "Bitmask packing" and "Constant-time lookup").  With
 *     W == 1 this is the paper's one-word-per-row layout; longer rows continue
 *     into further words.  B_r is 1 (one map for every sequence, as in the
 *     paper) unless params.route_per_batch is 1, then B_r = B.
 *     Bits of groups that hold no legal (query, key) pair, and bits at
 *     positions >= T_mask, are ignored.
 *   - Legality (causal and sequence-boundary masks) is decided in the kernel,
 *     independently of routing (Section 4.1).  With causal = 1 key j is legal
 *     for query i iff j <= i + (L_k - L_q) (bottom-right alignment); a query
 *     row with no legal key produces zeros.
 *   - Pointers named "device" must be device memory (hipMalloc / torch CUDA
 *     tensors) on the current device; the caller owns every buffer.  The
 *     library allocates nothing, never synchronizes, and keeps no state
 *     between calls, so calls on different streams with distinct outputs and
 *     workspaces may run concurrently.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     All device work is enqueued on it; the call returns without waiting.
 *   - Errors: argument problems are detected before anything is enqueued and
 *     returned as a status (tilemix_last_error() gives a message, per thread).
 *     A failed kernel launch returns TILEMIX_ERR_HIP.  Faults during execution
 *     surface at the caller's next synchronization, as usual for HIP.
 */
#ifndef TILEMIX_H
#define TILEMIX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum tilemix_status {
  TILEMIX_OK = 0,
  TILEMIX_ERR_NULL = 1,         /* a required pointer is NULL */
  TILEMIX_ERR_SHAPE = 2,        /* sizes inconsistent or out of range */
  TILEMIX_ERR_UNSUPPORTED = 3,  /* d, tile shape or flags the library does not implement */
  TILEMIX_ERR_ALIGN = 4,        /* a pointer is not aligned as required */
  TILEMIX_ERR_WORKSPACE = 5,    /* workspace NULL or smaller than tilemix_workspace_size() */
  TILEMIX_ERR_HIP = 6           /* the HIP runtime rejected a launch */
} tilemix_status;

/* Problem description shared by all entry points. */
typedef struct tilemix_params {
  int32_t batch;          /* B >= 1 */
  int32_t heads_q;        /* H_q >= 1 */
  int32_t heads_kv;       /* H_k >= 1 and H_q % H_k == 0 */
  int32_t len_q;          /* L_q >= 1 */
  int32_t len_k;          /* 1 <= L_k <= 262144 */
  int32_t head_dim;       /* d: 64 or 128 */
  int32_t block_m;        /* BLOCK_M (query rows per routed tile): 64 or 128 */
  int32_t block_n;        /* BLOCK_N (keys per routed tile): 64 */
  int32_t group_size;     /* g >= 1: one routing bit per g adjacent key tiles */
  int32_t causal;         /* 0 or 1 */
  float scale;            /* softmax scale (1/sqrt(d) for standard attention); finite, > 0 */
  int32_t route_per_batch;/* 0: routing words shared by the batch (B_r = 1); 1: B_r = B */
  int32_t route_hint;     /* -1: unknown; 0: the map has no INT8 bit (quantization is skipped
                             and every tile takes the FP16 path); other values: invalid */
} tilemix_params;

/* Words per routing row, W = ceil(ceil(ceil(L_k / BLOCK_N) / g) / 64); 0 if params invalid. */
int32_t tilemix_route_words_per_row(const tilemix_params* params);

/* Bytes of device workspace tilemix_prefill needs (K8, its FP16 block scales and V laid out
 * per 64-key tile); the workspace must be 256-byte aligned.  No Q8 tensor is kept: a 128-row
 * query block belongs to one workgroup of the attention kernel (two when BLOCK_M is 64), which
 * quantizes it in its prologue with the same codes and scale as tilemix_quantize. */
tilemix_status tilemix_workspace_size(const tilemix_params* params, size_t* bytes);

/*
 * tilemix_prefill -- routed attention forward: O = Attention(Q, K, V) with per-tile-group
 * FP16/INT8 score routing (Sections 3.1, 4.1-4.3, Appendix C).
 *   Q          device FP16 [B, L_q, H_q, d], 16-byte aligned, read only
 *   K, V       device FP16 [B, L_k, H_k, d], 16-byte aligned, read only
 *   route_bits device uint64 [B_r, H_k, T_m, W], 8-byte aligned, read only
 *   O          device FP16 [B, L_q, H_q, d], 16-byte aligned, written (every element)
 *   workspace  device scratch of at least tilemix_workspace_size() bytes, 256-byte aligned;
 *              overwritten; must not be shared with a concurrently running call
 * Enqueues the operand preparation (skipped parts: see route_hint) and the fused kernel.
 */
tilemix_status tilemix_prefill(const tilemix_params* params,
                               const void* Q, const void* K, const void* V,
                               const uint64_t* route_bits, void* O,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * tilemix_prefill_noalloc -- tilemix_prefill for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * allocates nothing and takes no workspace: the workspace tilemix_prefill would need lives in
 * a device array of TILEMIX_NOALLOC_SCRATCH_BYTES (128 MiB) that the library's code object
 * holds on each GPU it runs on until the process ends.  Problems whose
 * tilemix_workspace_size() exceeds that are rejected with TILEMIX_ERR_WORKSPACE before
 * anything is enqueued (the workspace takes about 3 bytes per element of K, so problems with
 * B * L_k * H_k * d up to about 44 million fit, e.g. L_k = 32768 with 8 KV heads of d = 128).  Every call on one GPU uses
 * that GPU's one array: calls that overlap in time on one GPU (other streams, other host
 * threads) race and must not be issued.  Nothing in the array needs clearing between calls.
 * Arguments, results and errors otherwise as for tilemix_prefill; the output is the same bit
 * for bit.
 */
#define TILEMIX_NOALLOC_SCRATCH_BYTES (128u << 20)

tilemix_status tilemix_prefill_noalloc(const tilemix_params* params,
                                       const void* Q, const void* K, const void* V,
                                       const uint64_t* route_bits, void* O, void* stream);

/*
 * tilemix_prefill_fused -- tilemix_prefill in the fused on-the-fly operand mode (Appendix D,
 * "Storage and Execution Layout", the fused on-the-fly mode; Appendix C quantization rules):
 * no K8 / scale tensors and no quantization pass.  The kernel computes the scales and codes
 * on chip, only for what INT8-routed groups use: each workgroup quantizes the 128-row query
 * block of its rows once (as tilemix_prefill does too), and every INT8-routed 64-key tile (one
 * key scale block) after its FP16 copy reaches LDS.  Codes and scales equal those of
 * tilemix_quantize, so the output equals tilemix_prefill's bit for bit.  Arguments as in
 * tilemix_prefill; the workspace
 * (tilemix_fused_workspace_size bytes) holds only V laid out per 64-key tile.  The INT8 route
 * costs more per tile here (every workgroup requantizes the key tiles it reads); the mode
 * trades that time for the K8 scratch.
 */
tilemix_status tilemix_fused_workspace_size(const tilemix_params* params, size_t* bytes);

tilemix_status tilemix_prefill_fused(const tilemix_params* params,
                                     const void* Q, const void* K, const void* V,
                                     const uint64_t* route_bits, void* O,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * tilemix_prepare -- the first half of tilemix_prefill: the quantize-once pass over the keys
 * (K8 and its FP16 block scales, Appendix C "Quantize-Once Execution"; skipped when route_hint
 * is 0) and the per-64-key-tile V layout, written into `workspace`.  The query blocks are
 * quantized by tilemix_attend itself, once per block.  Arguments as in tilemix_prefill (Q is
 * not read).  The workspace then serves any number of tilemix_attend calls on the same K and V.
 */
tilemix_status tilemix_prepare(const tilemix_params* params, const void* Q, const void* K,
                               const void* V, void* workspace, size_t workspace_bytes,
                               void* stream);

/*
 * tilemix_attend -- the second half of tilemix_prefill: the fused routed attention kernel
 * (Sections 3.1, 4.2, 4.3) reading Q, K and the prepared workspace.  `params`, Q and K must
 * be those of the tilemix_prepare call that filled the workspace (route_hint included);
 * route_bits may differ between calls.  Arguments as in tilemix_prefill.
 */
tilemix_status tilemix_attend(const tilemix_params* params, const void* Q, const void* K,
                              const uint64_t* route_bits, void* O, const void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * tilemix_quantize -- the quantize-once operand preparation on its own (Appendix C,
 * "Blockwise INT8 Quantization", "Quantization Granularity", "Quantize-Once Execution").
 *   Q, K  device FP16 as in tilemix_prefill
 *   Q8    device int8 [B, L_q, H_q, d] written;  dQ device FP16 bits [B, ceil(L_q/128), H_q]
 *   K8    device int8 [B, L_k, H_k, d] written;  dK device FP16 bits [B, ceil(L_k/64), H_k]
 * Scale = block absmax / 127 in FP32 (IEEE division), code = round-half-even(x / scale)
 * clamped to [-127, 127], a zero block gets codes 0 and scale 0, the scale is stored as FP16
 * (round to nearest even).  Q8/K8 16-byte aligned, dQ/dK 2-byte aligned.
 */
tilemix_status tilemix_quantize(const tilemix_params* params, const void* Q, const void* K,
                                int8_t* Q8, uint16_t* dQ, int8_t* K8, uint16_t* dK, void* stream);

/*
 * tilemix_debug_qk_int32 -- the INT32 tile products C = Q8_m K8_n^T of the INT8 score path
 * (Appendix C, "INT8 Score Computation"), computed with the same MFMA code as the fused
 * kernel, for checking bit-exactness.
 *   Q8, K8  device int8 as written by tilemix_quantize
 *   tiles   device int32 [count, 4] rows (b, h_q, m, n): query tile m, key tile n
 *   out     device int32 [count, BLOCK_M, BLOCK_N] row-major (query row, key column);
 *           entries past L_q or L_k are 0
 * A tile row whose (b, h_q, m, n) lies out of range yields an all-zero tile; count < 0 is an
 * error and count == 0 enqueues nothing.
 */
tilemix_status tilemix_debug_qk_int32(const tilemix_params* params, const int8_t* Q8,
                                      const int8_t* K8, const int32_t* tiles, int32_t count,
                                      int32_t* out, void* stream);

/*
 * tilemix_debug_prefill -- a test entry point: tilemix_prefill (fused = 0) or
 * tilemix_prefill_fused (fused = 1), fixed-length (total_q < 0; the varlen arguments are then
 * ignored) or over a variable-length batch (as tilemix_prefill_varlen[_fused]), run by a
 * kernel instantiation that also writes out the INT8 operands it makes and multiplies
 * (Appendix C, "Quantization Granularity" and "INT8 Score Computation"), so that they can be
 * compared bit for bit with an independent implementation.  O is written as by the ordinary
 * call.  A query-tile row r is b * T_m + m for a fixed-length batch and the routing row index
 * (the rows of sequence b after those of b - 1) for a variable-length one; R is their number.
 *   q8     device int8, the shape of Q: the INT8 codes of each query row whose tile row has an
 *          INT8-routed group, as the kernel's prologue made them from Q (other rows untouched)
 *   dq     device FP16 bits [R, H_q]: the query-block scale the workgroup of (r, h_q) used, for
 *          tile rows with an INT8-routed group (others untouched)
 *   tiles  device int32 [R, H_q, T_n, BLOCK_M, 64]: for every INT8-routed tile the kernel
 *          visits, C = Q8 K8^T as its accumulators held it (entries past L_q or L_k
 *          unspecified; tiles not on the INT8 route untouched)
 *   kinds  device int32 [R, H_q, T_n, BLOCK_M / 32]: per 32-row wave of such a tile, 1 = the
 *          pipelined products started from the 1.5 * 2^23 bias, 2 = started from 0, 3 = the
 *          per-tile path of tiles crossing the diagonal or the sequence end (untouched for
 *          tiles not on the INT8 route)
 * The caller pre-fills the export buffers so that untouched entries can be recognised.
 */
typedef struct tilemix_debug_export {
  int8_t* q8;
  uint16_t* dq;
  int32_t* tiles;
  int32_t* kinds;
} tilemix_debug_export;

tilemix_status tilemix_debug_prefill(const tilemix_params* params, int32_t fused, int32_t total_q,
                                     int32_t total_k, const int32_t* cu_seqlens_q,
                                     const int32_t* cu_seqlens_k, const void* Q, const void* K,
                                     const void* V, const uint64_t* route_bits, int32_t route_rows,
                                     void* O, void* workspace, size_t workspace_bytes,
                                     const tilemix_debug_export* dbg, void* stream);

/* ------------------------------------------------------------ variable-length batching
 * A batch of B sequences of different lengths, packed without padding (Section 4.1: flattened
 * inputs with cu_seqlens prefix sums; Appendix C: per-sequence scale blocks).
 *   params          batch = B; len_q / len_k = the maximum query / key length of any
 *                   sequence (they size the grid and the routing rows); route_per_batch = 0;
 *                   every other field as for tilemix_prefill
 *   total_q/total_k rows of the packed Q / K tensors (>= 1)
 *   cu_seqlens_q/k  device int32 [B + 1]: sequence b owns Q rows cu_seqlens_q[b] ..
 *                   cu_seqlens_q[b+1] - 1 and K/V rows cu_seqlens_k[b] .. cu_seqlens_k[b+1] - 1
 *                   (cu[0] = 0, nondecreasing, lengths within the maxima).  The library reads
 *                   them only on the device; out-of-range entries are clamped so that every
 *                   access stays inside the tensors, with unspecified output.
 *   Q, O            device FP16 [total_q, H_q, d];  K, V device FP16 [total_k, H_k, d]
 *   route_bits      device uint64 [route_rows, H_k, W]: the routing rows of sequence b
 *                   (ceil(L_q,b / BLOCK_M) of them) follow those of sequence b - 1;
 *                   W = tilemix_route_words_per_row(params), i.e. from the maximum key length;
 *                   group bits as for tilemix_prefill against that sequence's own legal groups
 *   route_rows      rows of route_bits (>= 0).  From the first sequence whose routing rows
 *                   would run past them on, sequences are treated as empty: their O rows are
 *                   not written
 *   workspace       >= tilemix_varlen_workspace_size() bytes, 256-byte aligned
 * Each sequence is attended on its own: bottom-right causal alignment with its own lengths,
 * quantization blocks restart at its first row (Appendix C varlen scale layout).
 */
tilemix_status tilemix_varlen_workspace_size(const tilemix_params* params, int32_t total_q,
                                             int32_t total_k, size_t* bytes);

tilemix_status tilemix_prefill_varlen(const tilemix_params* params, int32_t total_q,
                                      int32_t total_k, const int32_t* cu_seqlens_q,
                                      const int32_t* cu_seqlens_k, const void* Q, const void* K,
                                      const void* V, const uint64_t* route_bits,
                                      int32_t route_rows, void* O, void* workspace,
                                      size_t workspace_bytes, void* stream);

/*
 * tilemix_prefill_varlen_fused -- tilemix_prefill_varlen in the fused on-the-fly operand mode
 * (Appendix D, "Storage and Execution Layout"; Section 4.1 prefix-sum metadata): no K8 or scale
 * tensors; each workgroup quantizes its sequence's 128-row query block (restarting at the
 * sequence's first row) and every INT8-routed key tile on chip, with the codes and scales of
 * the quantize-once rule, so the output equals tilemix_prefill_varlen's bit for bit.
 * Arguments as for tilemix_prefill_varlen; the workspace (tilemix_varlen_fused_workspace_size
 * bytes) holds the sequence table and V laid out per 64-key tile.
 */
tilemix_status tilemix_varlen_fused_workspace_size(const tilemix_params* params, int32_t total_q,
                                                   int32_t total_k, size_t* bytes);

tilemix_status tilemix_prefill_varlen_fused(const tilemix_params* params, int32_t total_q,
                                            int32_t total_k, const int32_t* cu_seqlens_q,
                                            const int32_t* cu_seqlens_k, const void* Q,
                                            const void* K, const void* V,
                                            const uint64_t* route_bits, int32_t route_rows,
                                            void* O, void* workspace, size_t workspace_bytes,
                                            void* stream);

/* --------------------------------------------------------------- INT8 key/value cache decode
 * Appendix C, "Additional Execution Interfaces": an INT8 key/value cache holds K8 and V8 with
 * FP16 per-block scales (64-token key blocks per KV head, the key quantization of Appendix C
 * applied to K and to V).  During decode, cached K8 takes the INT8 score path; cached V8 is
 * widened on chip with its block scale folded into the probabilities before P.V.
 *
 * tilemix_quantize_kv -- build the cache from device FP16 K, V [B, L_k, H_k, d] (same rules as
 * tilemix_quantize):
 *   K8      int8 [B, L_k, H_k, d] (key rows, the layout of K)
 *   V8      int8 [B, H_k, ceil(L_k/64), d, 64]: each 64-key block stored channel-major (V^T),
 *           keys past L_k in the last block 0
 *   dK, dV  FP16 bits [B, ceil(L_k/64), H_k]
 * K8, V8 16-byte and dK, dV 2-byte aligned.
 */
tilemix_status tilemix_quantize_kv(const tilemix_params* params, const void* K, const void* V,
                                   int8_t* K8, uint16_t* dK, int8_t* V8, uint16_t* dV,
                                   void* stream);

/* Bytes of device workspace tilemix_decode needs, 256-aligned: per (sequence, query head, chunk)
 * the chunk's max, normalizer and d FP32 output values.  A chunk is 8 t key tiles of 64, with
 * t = max(1, ceil(B H_k ceil(L_k/64) / 2048)) tiles per wave, so that the partial kernel runs
 * about 256 workgroups (one per CU); the size depends only on params. */
tilemix_status tilemix_decode_workspace_size(const tilemix_params* params, size_t* bytes);

/*
 * tilemix_decode -- one decode step: each sequence's newest query token attends to all L_k
 * cached keys (the last query row of causal attention).
 *   params      len_q = 1 (one token), len_k = cached keys, H_q / H_k <= 16, block_n = 64, g,
 *               scale, route_per_batch, route_hint as for tilemix_prefill (block_m is unused:
 *               the routing rows hold one query-tile row, T_m = 1)
 *   Q, O        device FP16 [B, 1, H_q, d]
 *   K           device FP16 key cache [B, L_k, H_k, d], read for FP16-routed groups
 *   K8, dK      device INT8 key cache and scales (tilemix_quantize_kv), INT8-routed groups
 *   V8, dV      device INT8 value cache (the transposed-block layout above) and scales
 *   route_bits  device uint64 [B_r, H_k, 1, W]
 *   workspace   >= tilemix_decode_workspace_size() bytes, 256-byte aligned
 * Scores follow tilemix_prefill (the query's INT8 codes use its own row as the block); the
 * output is O = sum_j P_j (dV_j V8_j) / sum_j P_j.
 */
tilemix_status tilemix_decode(const tilemix_params* params, const void* Q, const void* K,
                              const int8_t* K8, const uint16_t* dK, const int8_t* V8,
                              const uint16_t* dV, const uint64_t* route_bits, void* O,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * tilemix_decode_varlen -- tilemix_decode over a ragged batch: sequence b's cache holds
 * seqlens_k[b] keys (Section 4.1, per-sequence lengths; Appendix C, "Additional Execution
 * Interfaces").  The caches keep the layouts of tilemix_decode with params.len_k as their
 * capacity (K, K8 [B, len_k, H_k, d], V8 [B, H_k, ceil(len_k/64), d, 64], scales
 * [B, ceil(len_k/64), H_k]); sequence b attends to its first seqlens_k[b] cached keys and the
 * entries past them are never used.  Routing rows as for tilemix_decode, W from len_k.
 *   seqlens_k  device int32 [B], 4-byte aligned; values are clamped to [0, len_k] on the
 *              device; a sequence of length 0 gets O = 0
 * Other arguments, the workspace and errors as for tilemix_decode.
 */
tilemix_status tilemix_decode_varlen(const tilemix_params* params, const int32_t* seqlens_k,
                                     const void* Q, const void* K, const int8_t* K8,
                                     const uint16_t* dK, const int8_t* V8, const uint16_t* dV,
                                     const uint64_t* route_bits, void* O, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ routing templates
 * Host-side routing policies of Appendix B ("Policy Construction and Sharing", "Coverage
 * Accounting" and the layouts One, Zero, Band, Global, Row-Random, Aligned Sparse, BigBird,
 * SpTrans).  A template is a data-free 2-D map R[m, g_j] over query-tile rows m and key-tile
 * groups g_j (1 = INT8, 0 = FP16), broadcast over KV heads (and sequences) and packed into the
 * routing words tilemix_prefill reads.  Row m's legal groups G_m are the groups holding at
 * least one legal (query, key) pair of the row (a prefix 0 .. gmax(m) of the groups); each
 * layout picks its FP16 set F_m inside G_m, every other legal group is INT8 and every illegal
 * group's bit is 0.  These functions run on the host only and touch no device memory.
 */
typedef enum tilemix_template_kind {
  TILEMIX_TEMPLATE_ONE = 0,      /* F_m empty: every legal group INT8 */
  TILEMIX_TEMPLATE_ZERO = 1,     /* F_m = G_m: every legal group FP16 */
  TILEMIX_TEMPLATE_BAND = 2,     /* F_m = {g_j : |g_j - gamma(m)| <= band_w},
                                    gamma(m) = floor(m BLOCK_M / (g BLOCK_N)) */
  TILEMIX_TEMPLATE_GLOBAL = 3,   /* F_m = {g_j < global_groups} (the first key groups) */
  TILEMIX_TEMPLATE_ROWRAND = 4,  /* F_m = k_m groups of G_m drawn uniformly without replacement,
                                    k_m = floor(rand_fp16 |G_m| + 1/2); draw order: ascending
                                    SplitMix64 output of seed ^ (m << 32 | g_j), ties by g_j */
  TILEMIX_TEMPLATE_ALIGNED = 5,  /* F_m = the last a(m) = min(|G_m|, ceil(align_alpha +
                                    align_beta m)) groups of G_m (right-aligned) */
  TILEMIX_TEMPLATE_BIGBIRD = 6,  /* union of Band(band_w; none if -1), Global(global_groups)
                                    and Row-Random(rand_fp16, seed) */
  TILEMIX_TEMPLATE_SPTRANS = 7   /* F_m = groups meeting, for some query i of row m, the keys
                                    [u s, i'] and [max(r s, (r+1) s - c), (r+1) s - 1] for r < u,
                                    u = floor(i' / s), i' = i + L_k - L_q, s = sp_stride,
                                    c = sp_tail (tokens) */
} tilemix_template_kind;

typedef struct tilemix_template {
  int32_t kind;            /* tilemix_template_kind */
  int32_t band_w;          /* Band (>= 0), BigBird (>= -1): half-width in groups */
  int32_t global_groups;   /* Global, BigBird: number of leading FP16 groups (>= 0) */
  float rand_fp16;         /* Row-Random, BigBird: FP16 share of each row, 1 - rho (in [0, 1]) */
  float align_alpha;       /* Aligned Sparse: initial width */
  float align_beta;        /* Aligned Sparse: growth per query-tile row */
  int32_t sp_stride;       /* SpTrans: stride s in tokens (>= 1) */
  int32_t sp_tail;         /* SpTrans: tail c in tokens (>= 0) */
  uint64_t seed;           /* Row-Random, BigBird */
} tilemix_template;

/* The paper's automatic group size: b_64 = ceil(L_k / 64), BLOCK_N^mask = BLOCK_N *
 * ceil(max(b_64, BLOCK_N) / BLOCK_N), g = BLOCK_N^mask / BLOCK_N (Appendix B).  0 if an
 * argument is < 1. */
int32_t tilemix_auto_group_size(int32_t len_k, int32_t block_n);

/* Instantiate a template for `params` (lengths, tile, g, causal, route_per_batch) into HOST
 * memory `words`, uint64 [B_r, H_k, T_m, W] (B_r as for tilemix_prefill), every plane the
 * same map; illegal groups and padding bits are 0.  Errors: NULL pointers, invalid params or
 * template fields. */
tilemix_status tilemix_route_template(const tilemix_params* params, const tilemix_template* tmpl,
                                      uint64_t* words);

/* A template for each sequence of a variable-length batch, in the layout
 * tilemix_prefill_varlen reads: HOST uint64 [sum_b ceil(seqlens_q[b] / BLOCK_M), H_k, W] with
 * W from params->len_k.  seqlens_q / seqlens_k: HOST int32 [B] lengths, each within
 * params->len_q / len_k. */
tilemix_status tilemix_route_template_varlen(const tilemix_params* params, const int32_t* seqlens_q,
                                             const int32_t* seqlens_k, const tilemix_template* tmpl,
                                             uint64_t* words);

/* Realized coverage of HOST routing words [B_r, H_k, T_m, W] (Appendix B, "Coverage
 * Accounting"): rho_groups = INT8 share of the legal (h_k, m, g_j) groups; rho_pairs = INT8
 * share of the legal (query, key) pairs (over KV heads; each serves H_q / H_k query heads
 * alike). */
tilemix_status tilemix_route_coverage(const tilemix_params* params, const uint64_t* words,
                                      double* rho_groups, double* rho_pairs);

/* Choose the template's size parameter so that its realized group coverage is closest to
 * rho_int8 (Appendix B: parameters are selected at tile-group granularity to match the
 * requested coverage).  Band: band_w; Global: global_groups; Row-Random: rand_fp16 = 1 -
 * rho_int8; Aligned Sparse: align_beta with align_alpha = 1; BigBird: rand_fp16 with band_w = 0
 * and global_groups = 1; SpTrans: sp_tail for the given sp_stride (>= 1).  One and Zero are
 * left as they are. */
tilemix_status tilemix_fit_template(const tilemix_params* params, tilemix_template* tmpl,
                                    double rho_int8);

/* Static description of a status code. */
const char* tilemix_status_string(tilemix_status status);

/* Message describing the last error returned on the calling thread ("" if none). */
const char* tilemix_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TILEMIX_H */
