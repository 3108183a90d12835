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
//        INT8 route: v_mfma_i32_32x32x32_i8 on the INT8 codes, exact INT32, then one
//                    FP32 factor scale*log2(e)*dQ*dK (Appendix C rescale), applied in the
//                    exp argument.  The key codes come from the quantize-once pass; the
//                    query codes are made in the workgroup's prologue, since a 128-row query
//                    block belongs to one workgroup (two for BLOCK_M = 64);
//      with keys on the matrix rows, every lane holds all scores of one query row for
//      16 keys of each 32-key block, so row max / row sum are in-lane plus one exchange
//      between the two half-waves;
//   3. updates the shared online-softmax state of Section 3.1 in FP32 (running max in
//      the log2 domain, normalizer, output accumulator).  Tiles that every row sees in full
//      form P against the running max as it stands and refresh it (rescaling the
//      accumulator) only when a lane's FP16 P sum passes a limit; tiles that cross the
//      diagonal use their exact max and rescale when it grows by more than 2^8.  Either
//      way the result is the same softmax;
//   4. packs P to FP16 in registers, in exactly the operand layout the P.V step needs,
//      and accumulates O^T += V^T P^T (v_mfma_f32_32x32x16_f16, FP32 accumulate).
// Legality (causal, sequence end) is applied only on tiles that cross it; tiles past
// the last legal key of the workgroup are never visited and waves whose rows see no
// key of a tile skip its math.  Rows are scheduled longest-first, and consecutive
// workgroups on one XCD share a KV head when the KV stream count allows it.
//
// Staging: tiles move HBM -> LDS by direct-to-LDS copies (global_load_lds_dwordx4), so no
// registers hold the next tile.  Every LDS tile is made of 128-byte rows (an FP16 key tile
// of d = 128 is stored as two 64-row halves, one per 64 channels) whose 16-byte granules are
// XOR-swizzled by (row / 2) mod 8; each copying lane fetches the source granule that belongs
// at its destination.  gfx950's LDS serves 16 lanes of a 16-byte read per cycle over 64
// banks: those 16 lanes read 16 consecutive rows at one logical granule, and the swizzle
// spreads them over all 64 banks.  INT8 key tiles of d = 64 use 64-byte rows swizzled by
// (row / 4) mod 4 to the same effect.
#include <type_traits>

#include "tilemix_device.h"
#include "tilemix_internal.h"


namespace tilemix {

namespace {

// Compile-time loop: f(std::integral_constant<int, I>) for I = B .. E - 1, so every index the
// body derives from I is a constant (registers are never indexed dynamically).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

constexpr float kRescaleThreshold = 8.0f;   // log2 units: rescale when the max grows > x256
constexpr float kNegInf = -__builtin_huge_valf();
// Pipelined tiles do not recompute the row max: P = 2^(score - m) is formed against the
// running max m as it stands, which only ever holds an actual earlier score maximum, so P
// cannot underflow relative to the row's mass.  A lane whose 32 FP16 P values sum past this
// limit (or reach infinity) makes the wave refresh m from the tile's exact max and redo the
// tile; below it every P is a finite FP16 value well inside range.
constexpr float kSumLimit = 4096.0f;
// An INT8 accumulator may start at the bit pattern of 1.5 * 2^23: every exact INT32 product C
// (|C| <= 128 * 127^2 < 2^21) then leaves it holding the FP32 number 1.5 * 2^23 + C, read as
// float with no conversion instruction, and the bias is folded into the exp subtrahend
// k = 1.5 * 2^23 * c + m.  That fold rounds k once, by at most half an ulp of k; a tile takes
// it only when |k| < kFoldLimit, which keeps the error of the exp argument within 2^-11 (a
// relative 3.4e-4 on P, below the FP16 rounding P gets anyway).  Other INT8 tiles start at 0
// and convert the products exactly.
constexpr int kMagicBits = 0x4B400000;
constexpr float kMagic = 12582912.0f;
constexpr float kFoldLimit = 16384.0f;

template <int D, int BM, int HEADS>
struct TileCfg {
  static constexpr int kWavesPerHead = BM / 32;
  static constexpr int kWaves = HEADS * kWavesPerHead;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int kKHalves = D / 64;             // FP16 key tile: 64-channel halves
  static constexpr int kKRow = 128;                   // LDS bytes per FP16 key row (one half)
  static constexpr int kK8Row = D;                    // LDS bytes per INT8 key row
  static constexpr int kVRow = 2 * kBlockN;           // LDS bytes per d row of V^T
  static constexpr int kKHalfBytes = kBlockN * kKRow;
  static constexpr int kKBytes = kKHalves * kKHalfBytes;
  static constexpr int kK8Bytes = kBlockN * kK8Row;
  static constexpr int kVBytes = D * kVRow;
  static constexpr int kStage = kKBytes + kVBytes;
  // 1 KB direct-to-LDS copies issued per wave for each tile kind
  static constexpr int kKInstr = kKBytes / 1024 / kWaves;
  static constexpr int kK8Instr = kK8Bytes / 1024 / kWaves;
  static constexpr int kVInstr = kVBytes / 1024 / kWaves;
  static_assert(kKInstr * kWaves * 1024 == kKBytes, "K split");
  static_assert(kK8Instr * kWaves * 1024 == kK8Bytes, "K8 split");
  static_assert(kVInstr * kWaves * 1024 == kVBytes, "V split");
};

// Row-swizzle key of an LDS tile row: granule c of row r is stored at granule c ^ key(r).
template <int ROW_BYTES>
__device__ __forceinline__ int swz_key(int r) {
  static_assert(ROW_BYTES == 128 || ROW_BYTES == 64, "row size");
  if constexpr (ROW_BYTES == 128) return (r >> 1) & 7;
  else return (r >> 2) & 3;
}

// Direct-to-LDS copy plan of a tile with ROW_BYTES-byte rows: copy J (1 KB) has lane l write
// LDS byte 1024*J + 16*l, i.e. row r = J*(1024/ROW_BYTES) + l/(ROW_BYTES/16) and swizzled
// granule p = l % (ROW_BYTES/16); that slot holds logical granule c = p ^ swz_key(r), so the
// lane reads source row r, granule c.  swz_key(r) depends on the parity of J for 128-byte
// rows, not for 64-byte rows: the per-lane part of the source offset takes two values at most.
template <int ROW_BYTES>
struct DmaPlan {
  static constexpr int kCpr = ROW_BYTES / 16;
  static constexpr int kRowsPerCopy = 1024 / ROW_BYTES;
  uint32_t off_even, off_odd;   // lane part of the source byte offset for even / odd J
  int row_in_copy;              // l / kCpr
  __device__ __forceinline__ DmaPlan(int lane, int stride) {
    row_in_copy = lane / kCpr;
    off_even = lane_offset(lane, stride, 0);
    off_odd = lane_offset(lane, stride, 1);
  }
  __device__ __forceinline__ uint32_t lane_offset(int lane, int stride, int par) const {
    const int r = par * kRowsPerCopy + row_in_copy;
    const int c = (lane % kCpr) ^ swz_key<ROW_BYTES>(r);
    return (uint32_t)row_in_copy * (uint32_t)stride + (uint32_t)c * 16u;
  }
};

// Copy one tile into LDS.  `src` is the tile's first row (uniform), `stride` the bytes between
// source rows, `rows_valid` how many of its rows exist: rows past it re-read the last valid
// row, whose contents are never used unmasked.  Copies come in blocks of BLOCK_COPIES; block k
// covers source columns [k*COL_STEP, (k+1)*COL_STEP) of the same rows (the channel halves of
// an FP16 key tile) and lands right after block k-1 in LDS.
template <int ROW_BYTES, int INSTR, int ROWS, int BLOCK_COPIES = (1 << 20), int COL_STEP = 0>
__device__ __forceinline__ void dma_tile(const char* src, int stride, int rows_valid, uint32_t lds,
                                         int wave, int lane, const DmaPlan<ROW_BYTES> plan) {
  constexpr int kRpc = DmaPlan<ROW_BYTES>::kRowsPerCopy;
  if (rows_valid >= ROWS) {
#pragma unroll
    for (int j = 0; j < INSTR; ++j) {
      const int J = wave * INSTR + j;
      const int Jb = J / BLOCK_COPIES, Ji = J % BLOCK_COPIES;
      const char* s = src + (size_t)Jb * COL_STEP + (size_t)(Ji * kRpc) * stride;
      const uint32_t lo = (INSTR % 2 == 0) ? ((j & 1) ? plan.off_odd : plan.off_even)
                                           : (((wave * INSTR + j) & 1) ? plan.off_odd : plan.off_even);
      dma_16(s, lo, lds + J * 1024);
    }
  } else {
#pragma unroll
    for (int j = 0; j < INSTR; ++j) {
      const int J = wave * INSTR + j;
      const int Jb = J / BLOCK_COPIES, Ji = J % BLOCK_COPIES;
      const int r = Ji * kRpc + plan.row_in_copy;
      const int c = (lane % DmaPlan<ROW_BYTES>::kCpr) ^ swz_key<ROW_BYTES>(r);
      const int rs = min(r, rows_valid - 1);
      dma_16(src, (uint32_t)(Jb * COL_STEP + rs * stride + c * 16), lds + J * 1024);
    }
  }
}

// Per-lane LDS fragment offsets for a swizzled tile with ROW_BYTES-byte rows: logical
// granule 2*s + hi of row lq (+32 rows per 32-key block) is at at(s).  With key(r) =
// 2*x1 + x0 the stored granule is 2*(s ^ x1) + (hi ^ x0), so four registers cover s = 0..3
// (s = 0..1 for 64-byte rows).
template <int ROW_BYTES>
struct FragOffsets {
  int o[4];
  __device__ __forceinline__ explicit FragOffsets(int lane) {
    const int lq = lane & 31, hi = lane >> 5;
    const int key = swz_key<ROW_BYTES>(lq);
    const int x0 = key & 1, x1 = key >> 1;
#pragma unroll
    for (int u = 0; u < 4; ++u) o[u] = lq * ROW_BYTES + 16 * (hi ^ x0) + 32 * (u ^ x1);
  }
  __device__ __forceinline__ int at(int s) const { return o[s]; }
};

// S^T tile (64 keys x 32 queries of this wave) by the INT8 route: exact INT32 products.
template <int D>
__device__ __forceinline__ void qk_int8(const char* kst, const FragOffsets<D>& fo,
                                        const i32x4 (&q8f)[D / 32], i32x16& acc0, i32x16& acc1) {
  acc0 = i32x16{};
  acc1 = i32x16{};
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    const i32x4 a0 = as_i32x4(ld_lds_16(kst, fo.at(s)));
    const i32x4 a1 = as_i32x4(ld_lds_16(kst, fo.at(s) + 32 * D));
    acc0 = mfma_i8(a0, q8f[s], acc0);
    acc1 = mfma_i8(a1, q8f[s], acc1);
  }
}

// S^T tile by the FP16 route: FP16 products, FP32 accumulation.  Channel half h of the key
// tile (channels 64h .. 64h + 63) sits kKHalfBytes * h into the slot.
template <int D>
__device__ __forceinline__ void qk_fp16(const char* kst, const FragOffsets<128>& fo,
                                        const half8 (&qf)[D / 16], f32x16& acc0, f32x16& acc1) {
  acc0 = f32x16{};
  acc1 = f32x16{};
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    const int off = fo.at(s & 3) + (s >> 2) * (kBlockN * 128);
    const half8 a0 = as_half8(ld_lds_16(kst, off));
    const half8 a1 = as_half8(ld_lds_16(kst, off + 32 * 128));
    acc0 = mfma_f16(a0, qf[s], acc0);
    acc1 = mfma_f16(a1, qf[s], acc1);
  }
}

// One online-softmax step (Section 3.1) for the 64 scores a lane holds.  `sv` are raw
// scores (INT32 products or FP16-route dot products); `c` turns them into log2-domain
// scaled scores.  Produces P in FP16, packed in P.V operand order, and updates the state.
template <int D, bool MASKED>
__device__ __forceinline__ void softmax_step(float (&sv)[32], float c, int key0, int last_key,
                                             int lane, float& m_run, float& z_run,
                                             f32x16 (&oacc)[D / 32], half8 (&pfr)[4]) {
  float mt;
  if constexpr (MASKED) {
    // Scale first, then mask, so a zero scale can never meet an infinity.  Element i is key
    // key0 + 32*(i/16) + acc_row(i%16, lane); only the 4*(lane/32) part depends on the lane.
    const int lim = last_key - key0 - 4 * (lane >> 5);
    float mx = kNegInf;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int kc = 32 * (i >> 4) + 8 * ((i & 15) >> 2) + (i & 3);
      sv[i] = kc <= lim ? sv[i] * c : kNegInf;
      mx = fmaxf(mx, sv[i]);
    }
    mt = pair_max(mx);
  } else {
    float mx = sv[0];
#pragma unroll
    for (int i = 1; i < 32; ++i) mx = fmaxf(mx, sv[i]);
    mt = pair_max(mx) * c;
  }
  const float m_new = fmaxf(m_run, mt);
  if (__any(m_new > m_run + kRescaleThreshold)) {
    const float alpha = (m_new == kNegInf) ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
    z_run *= alpha;
#pragma unroll
    for (int cc = 0; cc < D / 32; ++cc) oacc[cc] *= alpha;
    m_run = m_new;
  }
  const float msub = (m_run == kNegInf) ? 0.0f : m_run;
  float zs = 0.0f;
  const half2v ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const int i = 16 * (t >> 1) + 8 * (t & 1) + e;
      float p0, p1;
      if constexpr (MASKED) {
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
}

// Map a linear workgroup id to (b, first query head, m).  A workgroup serves HEADS query heads
// of one GQA group (they share the KV head and its routing words).  Rows go longest first
// (largest m first for causal attention); when the number of KV streams (b, h_k) is a multiple
// of 8, workgroups that share an XCD (id % 8) walk the same KV streams, so their K/V tiles
// meet in one L2.
template <int HEADS>
__device__ __forceinline__ void decode_unit(int id, int B, int Hq, int Hk, int T_m, int& b,
                                            int& hq0, int& hk, int& m) {
  const int G = Hq / Hk / HEADS;   // workgroups per (KV stream, m)
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
  hq0 = hk * (Hq / Hk) + qg * HEADS;
}

// max(a, b, c) in one instruction.  The scores are never NaN, so the operand quieting that a
// library max would add is not needed.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Exp half of the online-softmax step for score pair J of a lane (elements i, i + 1 of its 32
// scores, held in two accumulator blocks, taken in P.V operand order): P = 2^(c*s - msub) rounded to FP16 into its operand
// slot, and the FP16 pair added to the row-sum partial, so the normalizer sums exactly the P
// that P.V multiplies.
template <int J>
__device__ __forceinline__ void exp_pair(const f32x16& x0, const f32x16& x1, float c, float msub,
                                         half8 (&pfr)[4], float& zs) {
  constexpr int t = J >> 2, e = 2 * (J & 3);
  constexpr int i = 16 * (t >> 1) + 8 * (t & 1) + e;
  float s0, s1;
  if constexpr (i < 16) {
    s0 = x0[i];
    s1 = x0[i + 1];
  } else {
    s0 = x1[i - 16];
    s1 = x1[i - 15];
  }
  const float p0 = __builtin_amdgcn_exp2f(fmaf(s0, c, -msub));
  const float p1 = __builtin_amdgcn_exp2f(fmaf(s1, c, -msub));
  const half2v pr = {(_Float16)p0, (_Float16)p1};
  const half2v ones = {(_Float16)1.0f, (_Float16)1.0f};
  zs = __builtin_amdgcn_fdot2(pr, ones, zs, false);
  pfr[t][e] = pr[0];
  pfr[t][e + 1] = pr[1];
}

// OTF: the fused on-the-fly operand mode (Appendix D, "Storage and Execution Layout"): no Q8 /
// K8 / scale tensors exist.  The workgroup quantizes its query block on chip in the prologue
// (a 128-row Q block is one or two workgroups' rows) and every INT8-routed key tile after its
// FP16 copy lands: the tile's absmax, scale and codes (the 64-key tile is exactly one key
// scale block) into an INT8 slot in the K8 layout, for the same INT8 products.
//
// DBG: a test-only instantiation that also writes out the INT8 operands the kernel makes and
// multiplies: each row's query codes and its workgroup's query-block scale after the prologue,
// and the INT32 products of every INT8-routed tile as its accumulators hold them (AttnArgs
// dbg_*).  The arithmetic is that of the ordinary instantiation.
template <int D, int BM, int HEADS, bool OTF = false, bool DBG = false>
__global__ __launch_bounds__(HEADS * 2 * BM, 2) void routed_attn_fwd_kernel(AttnArgs a) {
  using C = TileCfg<D, BM, HEADS>;
  static_assert(HEADS == 1, "the query-block quantization reduces over the whole workgroup");
  // Two K slots and two V slots: step n reads K of tile n + 1 and V of tile n while K of tile
  // n + 2 and V of tile n + 1 are copied into the slots that step n - 1 released.  72 KB at
  // d = 128, so two workgroups share a CU and each SIMD runs one wave of each.
  // OTF: one INT8 key slot after the K and V slots (the key scales come from the chip).
  constexpr int kK8Off = 2 * C::kKBytes + 2 * C::kVBytes;
  __shared__ __align__(16) char smem[kK8Off + (OTF ? C::kK8Bytes : 0)];
  __shared__ uint16_t key_scale[OTF ? 1 : kMaxKeyTiles];   // dK of this row's key tiles (FP16 bits)
  __shared__ float otf_red[OTF ? C::kWaves : 1];          // OTF: per-wave absmax partials

  int b, hq0, hk, m;
  decode_unit<HEADS>(blockIdx.x, a.B, a.Hq, a.Hk, a.T_m, b, hq0, hk, m);
  // This sequence: its lengths, first rows in Q and K, first scale blocks, and the addresses
  // of this routing row and of this KV head's first V tile.
  int Lq = a.Lq, Lk = a.Lk;
  long long q_row0 = (long long)b * a.Lq, k_row0 = (long long)b * a.Lk;
  long long kblk0 = (long long)b * a.nKB;
  const uint64_t* route_row =
      a.route + (size_t)b * a.route_batch_stride + ((size_t)hk * a.T_m + m) * a.W;
  long long vt_tile0 = ((long long)b * a.Hk + hk) * a.T_n;
  long long dbg_row = (long long)b * a.T_m + m;   // DBG: this query-tile row's export index
  if (a.seqs) {
    const int* e = a.seqs + kSeqFields * b;
    Lq = e[kSeqQLen];
    Lk = e[kSeqKLen];
    if (m * BM >= Lq) return;   // past the end of a shorter sequence: no rows to write
    q_row0 = e[kSeqQStart];
    k_row0 = e[kSeqKStart];
    kblk0 = e[kSeqKBlk];
    route_row = a.route + ((size_t)(e[kSeqQTile] + m) * a.Hk + hk) * a.W;
    dbg_row = e[kSeqQTile] + m;
    vt_tile0 = (long long)hk * a.seqs[kSeqFields * a.B + kSeqKTile] + e[kSeqKTile];
  }

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hq = hq0 + wave / C::kWavesPerHead;   // this wave's query head
  const int wave_in_head = wave % C::kWavesPerHead;
  const int lane = tid & (kWave - 1);
  const int lq = lane & 31, hi = lane >> 5;
  const int q0 = m * BM + 32 * wave_in_head;  // first query row of this wave
  const int my_q = q0 + lq;
  // Row i may see keys j <= i + off (bottom-right causal alignment); without the causal
  // mask every key up to L_k - 1 is legal.
  const int off = a.causal ? Lk - Lq : Lk;
  const bool wave_active = q0 < Lq;

  // Last key any row of the workgroup / of this wave may see.
  const int wg_last_key = min(Lk - 1, min(Lq - 1, m * BM + BM - 1) + off);
  const int wave_last_key = min(Lk - 1, min(Lq - 1, q0 + 31) + off);
  const int my_last_key = min(Lk - 1, my_q + off);

  _Float16* orow = a.O + ((size_t)(q_row0 + my_q) * a.Hq + hq) * D;
  if (wg_last_key < 0) {   // no legal key for any row of this tile: output is zero
    if (my_q < Lq) {       // the two lanes of a row each clear half of it
#pragma unroll
      for (int c = 0; c < D / 2; c += 8) *reinterpret_cast<half8*>(orow + hi * (D / 2) + c) = half8{};
    }
    return;
  }
  const int n_end = wg_last_key / kBlockN;

  // Routing words of this row: lane w holds word w (at most 64 words per row), so the
  // per-tile lookup is a lane read plus a shift-and-mask, with no memory access in the loop.
  const uint64_t my_word = (!a.force_fp16 && lane < a.W) ? route_row[lane] : 0ull;
  const uint32_t word_lo = (uint32_t)my_word, word_hi = (uint32_t)(my_word >> 32);
  auto group_route = [&](int gj) -> bool {   // routing bit of tile group gj
    const int w = gj >> 6, bit = gj & 63;
    const uint32_t half = bit < 32 ? __builtin_amdgcn_readlane(word_lo, w)
                                   : __builtin_amdgcn_readlane(word_hi, w);
    return (half >> (bit & 31)) & 1u;
  };

  // Which operand forms this row needs (looked up once per row).
  bool need_int8 = false, need_fp16 = false;
  {
    const int g_last = n_end / a.g;
    const int nb = g_last - 64 * lane + 1;      // groups of the row in this lane's word
    const uint64_t valid = nb <= 0 ? 0ull : (nb >= 64 ? ~0ull : ((1ull << nb) - 1ull));
    need_int8 = __any((my_word & valid) != 0ull);
    need_fp16 = __any((~my_word & valid) != 0ull);
  }

  // Tile sources (uniform bases).
  const int kstride = a.Hk * D * 2;                              // bytes between keys (FP16)
  const char* kbase = reinterpret_cast<const char*>(a.K) + ((size_t)k_row0 * a.Hk + hk) * D * 2;
  const char* k8base = reinterpret_cast<const char*>(a.K8) + ((size_t)k_row0 * a.Hk + hk) * D;
  const char* vbase = reinterpret_cast<const char*>(a.Vt) + (size_t)vt_tile0 * (size_t)(D * kBlockN * 2);
  const DmaPlan<C::kKRow> plan_k(lane, kstride);
  const DmaPlan<C::kK8Row> plan_k8(lane, kstride / 2);
  const DmaPlan<C::kVRow> plan_v(lane, C::kVRow);
  auto k_slot = [](int n) { return (n & 1) * C::kKBytes; };                   // LDS offsets
  auto v_slot = [](int n) { return 2 * C::kKBytes + (n & 1) * C::kVBytes; };
  const uint32_t smem_lds = lds_addr_of(smem);

  // Copies are issued in tile order, K and V each on their own.  The issue state advances by
  // additions only: the next tile, its routing group (tile = group * g + r) and its source
  // addresses.  The route of every issued K tile is kept in a 64-bit ring (bit t mod 64),
  // which the math reads back; at most two K tiles are ever in flight.
  int iss_kt = 0, iss_vt = 0, iss_g = 0, iss_r = 0;
  uint64_t route_ring = 0;
  const char* iss_k = kbase;
  const char* iss_k8 = k8base;
  const char* iss_v = vbase;
  auto issue_k_next = [&]() {
    const bool int8 = group_route(iss_g);
    const uint64_t bit = 1ull << (iss_kt & 63);
    route_ring = int8 ? (route_ring | bit) : (route_ring & ~bit);
    const uint32_t dst = smem_lds + (uint32_t)k_slot(iss_kt);
    const int rows = min(kBlockN, Lk - iss_kt * kBlockN);
    if (int8 && !OTF)   // OTF stages every key tile in FP16
      dma_tile<C::kK8Row, C::kK8Instr, kBlockN>(iss_k8, kstride / 2, rows, dst, wave, lane, plan_k8);
    else   // 8 copies per 64-channel half of the FP16 key tile
      dma_tile<C::kKRow, C::kKInstr, kBlockN, 8, 128>(iss_k, kstride, rows, dst, wave, lane, plan_k);
    ++iss_kt;
    if (++iss_r == a.g) {
      iss_r = 0;
      ++iss_g;
    }
    iss_k += (size_t)kBlockN * kstride;
    iss_k8 += (size_t)kBlockN * (kstride / 2);
  };
  auto issue_v_next = [&]() {
    dma_tile<C::kVRow, C::kVInstr, D>(iss_v, C::kVRow, D, smem_lds + (uint32_t)v_slot(iss_vt), wave,
                                      lane, plan_v);
    ++iss_vt;
    iss_v += (size_t)D * kBlockN * 2;
  };
  // Every sync below frees exactly one K and one V slot, so at most one tile of each kind is
  // pending at a call.
  auto issue = [&](int k_last, int v_last) {
    if (iss_kt <= min(k_last, n_end)) issue_k_next();
    if (iss_vt <= min(v_last, n_end)) issue_v_next();
  };
  auto route_of = [&](int n) -> bool { return (route_ring >> (n & 63)) & 1ull; };   // issued K n
  // Every copy issued so far has landed for every wave, then K through k_last and V through
  // v_last are issued.  Each call site issues exactly the tiles whose slots the barrier freed.
  auto sync = [&](int k_last, int v_last) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    issue(k_last, v_last);
  };
  // The first K and V tiles start copying now, so that their latency overlaps the query
  // operand set-up below.
  issue(0, 0);   // K and V of tile 0, then K of tile 1
  issue(1, 0);

  // Q operands of this wave, kept in registers for the whole row.  The lane's 64 FP16 query
  // values in the FP16 operand layout (lane l: row l % 32, channels 16 s + 8 (l / 32) + 0..7)
  // are loaded once; with 128-row tiles they also give the query block's scale and codes.
  half8 qf[D / 16];
  i32x4 q8f[D / 32];
  const bool row_ok = my_q < Lq;
  const size_t qoff = ((size_t)(q_row0 + (row_ok ? my_q : 0)) * a.Hq + hq) * D;
  constexpr bool kQBlockInRegs = BM == kQuantBlockQ;   // the workgroup's rows are one Q block
  half8 qv[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
    qv[s] = ((need_fp16 || (kQBlockInRegs && need_int8)) && row_ok)
                ? as_half8(ld_global_16(a.Q + qoff + 16 * s + 8 * hi)) : half8{};
#pragma unroll
  for (int s = 0; s < D / 16; ++s) qf[s] = need_fp16 ? qv[s] : half8{};
#pragma unroll
  for (int s = 0; s < D / 32; ++s)
    q8f[s] = i32x4{};
  float dq = 0.0f;   // the FP16-stored scale of this row's query block (set below)

  // OTF: maximum of a per-thread value over the workgroup (every thread gets it).
  auto wg_max = [&](float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    if (lane == 0) otf_red[wave] = v;
    __syncthreads();
    float r = otf_red[0];
#pragma unroll
    for (int w = 1; w < C::kWaves; ++w) r = fmaxf(r, otf_red[w]);
    return r;
  };
  // OTF: the code of x in a block with scale d32 = absmax / 127 and rcp = 1 / d32 (both
  // correctly rounded), as the low byte of the returned word.  x * rcp refined by one residual
  // step is the correctly rounded x / d32 (checked exhaustively over every FP16 x and block
  // absmax), the same quotient the quantize-once pass divides out; adding 1.5 * 2^23 rounds it
  // half to even into the low mantissa bits.  |x| <= absmax keeps the quotient within
  // 127 * (1 + 2^-23), so the clamp to [-127, 127] of the quantization rule never acts.
  auto code_word = [](float x, float d32, float rcp) {
    const float q0 = fmaf(x, rcp, 0.0f);   // x * rcp (an FMA takes x in FP16 directly)
    const float q = fmaf(fmaf(-q0, d32, x), rcp, q0);
    return __builtin_bit_cast(uint32_t, q + 12582912.0f);
  };
  // Low bytes of four code words, packed little-endian.
  auto pack4 = [](uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
    const uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm(w3, w2, 0x0c0c0400u);
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
  };
  // Largest |h| of eight FP16 values, as FP16 bits: finite non-negative FP16 values order like
  // their bit patterns, so packed unsigned 16-bit maxima of the magnitudes serve.
  auto absmax_bits = [](uint4 v, uint32_t m) {
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    u16x2 acc = __builtin_bit_cast(u16x2, m);
    acc = __builtin_elementwise_max(acc, __builtin_bit_cast(u16x2, v.x & 0x7fff7fffu));
    acc = __builtin_elementwise_max(acc, __builtin_bit_cast(u16x2, v.y & 0x7fff7fffu));
    acc = __builtin_elementwise_max(acc, __builtin_bit_cast(u16x2, v.z & 0x7fff7fffu));
    acc = __builtin_elementwise_max(acc, __builtin_bit_cast(u16x2, v.w & 0x7fff7fffu));
    return __builtin_bit_cast(uint32_t, acc);
  };
  auto bits_max_float = [](uint32_t m) {
    return half_bits_to_float((uint16_t)max(m & 0xffffu, m >> 16));
  };
  // 16 codes of the FP16 values in two 16-byte granules.
  auto codes16 = [&](uint4 g0, uint4 g1, float d32, float rcp) {
    const half8 h0 = as_half8(g0), h1 = as_half8(g1);
    uint32_t w[16];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      w[e] = code_word((float)h0[e], d32, rcp);
      w[8 + e] = code_word((float)h1[e], d32, rcp);
    }
    return make_uint4(pack4(w[0], w[1], w[2], w[3]), pack4(w[4], w[5], w[6], w[7]),
                      pack4(w[8], w[9], w[10], w[11]), pack4(w[12], w[13], w[14], w[15]));
  };
  // The query operands of the INT8 route are made here, in both operand modes: the 128-row
  // query block of this row (Appendix C) is this workgroup's own rows (BLOCK_M = 128) or those of
  // two workgroups (64), so each block is quantized once, with the codes and scale of the
  // quantize-once rule, and no Q8 tensor passes through HBM.
  {
    if (need_int8) {   // the same for every wave of the workgroup
      uint32_t mb = 0u;
      if constexpr (kQBlockInRegs) {   // the block's absmax from the values in registers
#pragma unroll
        for (int s = 0; s < D / 16; ++s) mb = absmax_bits(__builtin_bit_cast(uint4, qv[s]), mb);
      } else {   // the block spans two workgroups: read it (rows qb0 .. qb0 + 127 that exist)
        const int qb0 = (m * BM / kQuantBlockQ) * kQuantBlockQ;
        const int qrows = min(kQuantBlockQ, Lq - qb0);
        for (int c = tid; c < kQuantBlockQ * (D / 8); c += C::kThreads) {
          const int r = c / (D / 8), ch = 8 * (c % (D / 8));
          if (r < qrows)
            mb = absmax_bits(ld_global_16(a.Q + ((size_t)(q_row0 + qb0 + r) * a.Hq + hq) * D + ch), mb);
        }
      }
      const float amax = wg_max(bits_max_float(mb));
      const float d32 = amax / 127.0f;   // IEEE FP32 division
      const float rcp = amax > 0.0f ? 1.0f / d32 : 0.0f;
      dq = amax > 0.0f ? (float)(_Float16)d32 : 0.0f;
#pragma unroll
      for (int s = 0; s < D / 32; ++s) {   // codes of channels 32 s + 16 hi + 0..15
        uint4 g0, g1;
        if constexpr (kQBlockInRegs) {
          // FP16 fragment 2 s + hi of this lane holds 8 of them; its partner lane (l ^ 32)
          // holds the other 8 in its own fragment 2 s + hi, and sends it in exchange for ours.
          const uint4 f0 = __builtin_bit_cast(uint4, qv[2 * s]);
          const uint4 f1 = __builtin_bit_cast(uint4, qv[2 * s + 1]);
          const uint4 mine = hi ? f1 : f0;
          const uint4 send = hi ? f0 : f1;
          uint32_t o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t v = e == 0 ? send.x : e == 1 ? send.y : e == 2 ? send.z : send.w;
            const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
            o[e] = hi ? (uint32_t)r[0] : (uint32_t)r[1];   // the partner lane's value
          }
          const uint4 other = make_uint4(o[0], o[1], o[2], o[3]);
          g0 = hi ? other : mine;
          g1 = hi ? mine : other;
        } else {
          g0 = row_ok ? ld_global_16(a.Q + qoff + 32 * s + 16 * hi) : uint4{};
          g1 = row_ok ? ld_global_16(a.Q + qoff + 32 * s + 16 * hi + 8) : uint4{};
        }
        if (row_ok) {   // a zero block has rcp = 0: codes 0
          const uint4 c = codes16(g0, g1, d32, rcp);
          q8f[s] = i32x4{(int)c.x, (int)c.y, (int)c.z, (int)c.w};
        }
      }
    }
  }
  if constexpr (DBG) {   // the query operands of the INT8 route, as made above
    if (need_int8) {
      if (row_ok) {
#pragma unroll
        for (int s = 0; s < D / 32; ++s)
          *reinterpret_cast<i32x4*>(a.dbg_q8 + qoff + 32 * s + 16 * hi) = q8f[s];
      }
      if (tid == 0) a.dbg_dq[dbg_row * a.Hq + hq] = __builtin_bit_cast(uint16_t, (_Float16)dq);
    }
  }
  // DBG: the INT32 products of INT8-routed key tile n from this wave's 32 raw scores per lane
  // (element i is key 32*(i/16) + acc_row(i%16, lane)): 1.5 * 2^23 + C read as FP32 when the
  // accumulators started at the bias, the exactly converted float(C) otherwise.
  auto dbg_tile = [&](int n, const float (&v)[32], int kind) {
    if constexpr (DBG) {
      const size_t t = ((size_t)dbg_row * a.Hq + hq) * a.T_n + n;
      if (lane == 0) a.dbg_kind[t * C::kWavesPerHead + wave_in_head] = kind;
      int32_t* out = a.dbg_tiles + t * BM * kBlockN + (size_t)(32 * wave_in_head + lq) * kBlockN;
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const int key = 32 * (i >> 4) + acc_row(i & 15, lane);
        out[key] = kind == kDbgFolded ? __builtin_bit_cast(int, v[i]) - kMagicBits : (int)v[i];
      }
    }
  };
  auto dbg_tile2 = [&](int n, const f32x16& y0, const f32x16& y1, int kind) {
    if constexpr (DBG) {
      float v[32];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        v[r] = y0[r];
        v[16 + r] = y1[r];
      }
      dbg_tile(n, v, kind);
    }
  };
  const float c_fp16 = a.scale_log2e;
  const float c_int8_q = a.scale_log2e * dq;
  if (!OTF && need_int8) {   // key-block scales of the tiles this row visits (key block = key tile)
    for (int t = tid; t <= n_end; t += C::kThreads)
      key_scale[t] = a.dK[(size_t)(kblk0 + t) * a.Hk + hk];
  }

  // Per-lane LDS fragment offsets.
  const FragOffsets<128> fo_128(lane);      // K (FP16 halves), V^T, and K8 when d = 128
  const FragOffsets<C::kK8Row> fo_k8(lane);

  // OTF: quantize the FP16 key tile in slot koff into the INT8 slot (K8 layout), with the
  // blockwise rule of Appendix C over the tile's 64 keys; every thread of the workgroup takes
  // part (two barriers).  Rows past L_k hold copies of the last key, so they leave the absmax
  // unchanged.  Returns the FP16 bits of the tile's scale.
  auto convert_k = [&](int koff) -> uint16_t {
    constexpr int kGr = D / 16;                          // 16-code granules per key row
    constexpr int kPer = kBlockN * kGr / C::kThreads;    // granules per thread
    static_assert(kPer * C::kThreads == kBlockN * kGr, "granule split");
    const char* src = smem + koff;
    // FP16 granules 2*c8 and 2*c8 + 1 of 64-channel half c8 / 4 hold the 16 channels of
    // INT8 granule c8.
    auto fp16_off = [](int r, int c8, int j) {
      const int c16 = (2 * c8 + j) & 7;
      return ((2 * c8) >> 3) * C::kKHalfBytes + r * C::kKRow + 16 * (c16 ^ swz_key<128>(r));
    };
    uint32_t mb = 0u;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int gi = tid + i * C::kThreads, r = gi / kGr, c8 = gi % kGr;
#pragma unroll
      for (int j = 0; j < 2; ++j) mb = absmax_bits(ld_lds_16(src, fp16_off(r, c8, j)), mb);
    }
    const float amax = wg_max(bits_max_float(mb));
    const float d32 = amax / 127.0f;   // IEEE FP32 division
    const float rcp = amax > 0.0f ? 1.0f / d32 : 0.0f;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {   // a zero block has rcp = 0: codes 0
      const int gi = tid + i * C::kThreads, r = gi / kGr, c8 = gi % kGr;
      *reinterpret_cast<uint4*>(smem + kK8Off + r * C::kK8Row + 16 * (c8 ^ swz_key<C::kK8Row>(r))) =
          codes16(ld_lds_16(src, fp16_off(r, c8, 0)), ld_lds_16(src, fp16_off(r, c8, 1)), d32, rcp);
    }
    __syncthreads();   // codes visible to every wave; otf_red free again
    const _Float16 sc = amax > 0.0f ? (_Float16)d32 : (_Float16)0.0f;   // RNE
    return __builtin_bit_cast(uint16_t, sc);
  };

  // Online-softmax state (Section 3.1), FP32; max kept in log2 units.
  float m_run = kNegInf;
  float msub = 0.0f;   // the max that P subtracts (0 while no score has been seen)
  float z_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) oacc[c] = f32x16{};

  // ---- Straight per-tile path, used for tiles that cross the causal diagonal or the sequence
  // end.  Raw scores of key tile n (INT32 products converted to float, or FP32 dot products)
  // and the factor c that turns them into log2-domain scaled scores.
  // ks_otf: OTF only, the on-chip scale of tile n (its codes are in the INT8 slot).
  auto qk = [&](int n, float (&sv)[32], float& c, uint16_t ks_otf) {
    const char* kst = smem + k_slot(n);
    if (route_of(n)) {
      i32x16 i0, i1;
      qk_int8<D>(OTF ? smem + kK8Off : kst, fo_k8, q8f, i0, i1);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sv[r] = (float)i0[r];
        sv[16 + r] = (float)i1[r];
      }
      c = c_int8_q * half_bits_to_float(OTF ? ks_otf : key_scale[n]);
    } else {
      f32x16 f0, f1;
      qk_fp16<D>(kst, fo_128, qf, f0, f1);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sv[r] = f0[r];
        sv[16 + r] = f1[r];
      }
      c = c_fp16;
    }
  };
  // O^T += V^T P^T for key tile n: granule 2t + hi of V^T row 32*cc + lq holds the keys of
  // P^T slot t.
  auto pv = [&](int n, const half8 (&pfr)[4]) {
    const char* vst = smem + v_slot(n);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
        const half8 va = as_half8(ld_lds_16(vst, fo_128.at(t) + cc * 32 * C::kVRow));
        oacc[cc] = mfma_f16(va, pfr[t], oacc[cc]);
      }
    }
  };

  // ---- Software-pipelined path for the tiles every row of the workgroup sees in full.  Each
  // step interleaves, in one wave, matrix-core work of one tile with vector work of another:
  //   phase A: Q K^T of tile n + 1           | exp of tile n's softmax (P(n), row sum)
  //   phase B: O += V^T P^T of tile n (P.V)
  // Every chunk below is one MFMA plus its share of the vector work, kept in program order by
  // a scheduling barrier; LDS fragments are read kLeadA / kLeadB chunks ahead of the MFMA that
  // consumes them.  A tile's 32 scores per lane live in two accumulator blocks (elements 0-15, 16-31);
  // two such buffers alternate between "scores of tile n" and "scores of tile n + 1" from
  // step to step.  Raw scores are FP32 dot products (FP16 route) or 1.5 * 2^23 + C (INT8
  // route); a tile's log2-domain score is (raw - bias) * c with bias 0 or 1.5 * 2^23, and P
  // is 2^(raw * c - k) with k = bias * c + msub.
  constexpr int kLeadA = 2, kLeadB = 3;
  float c_cur = 0.0f, bias_cur = 0.0f, k_cur = 0.0f;
  i32x16 magic;
#pragma unroll
  for (int r = 0; r < 16; ++r) magic[r] = kMagicBits;

  // Phase A.  QK: 0 = none (exp only), 1 = FP16 route, 2 = INT8 route with the folded bias,
  // 3 = INT8 route with exact conversion, for tile n + 1, whose raw scores go to y0 / y1.
  auto phase_a = [&](auto qk_tag, auto exp_tag, int k_off, const f32x16& x0, const f32x16& x1,
                     f32x16& y0, f32x16& y1, half8 (&pfr)[4], float& zs) {
    constexpr int kQK = decltype(qk_tag)::value;
    constexpr bool kExp = decltype(exp_tag)::value;
    constexpr int NQ = kQK == 0 ? 4 : (kQK >= 2 ? 2 * (D / 32) : 2 * (D / 16));   // chunks
    // Chunk j feeds accumulator h = j % 2 with K slice s = j / 2: consecutive MFMAs write
    // different accumulators, so none waits for its predecessor's result.
    const char* kst = smem + k_off;
    uint4 kf[NQ];
    auto kload = [&](auto jc) {
      constexpr int j = decltype(jc)::value, s = j / 2, h = j % 2;
      if constexpr (kQK >= 2) kf[j] = ld_lds_16(kst, fo_k8.at(s) + h * 32 * D);
      else kf[j] = ld_lds_16(kst, fo_128.at(s & 3) + (s >> 2) * (kBlockN * 128) + h * 32 * 128);
    };
    if constexpr (kQK != 0) static_for<0, (kLeadA < NQ ? kLeadA : NQ)>(kload);
    // Every call site computes the same exp of tile n; an opaque copy of its inputs keeps
    // each copy inside its own branch, interleaved with that branch's MFMAs, instead of being
    // merged ahead of the branch.
    float c_x = c_cur, k_x = k_cur;
    asm volatile("" : "+v"(c_x), "+v"(k_x));
    float zs0 = 0.0f, zs1 = 0.0f;
    // Wave priorities (the SIMD's other wave belongs to the other workgroup on this CU): the
    // phase that mixes matrix-core and vector work issues first, the pure P.V phase next, and
    // the barrier and copy code last.
    __builtin_amdgcn_s_setprio(2);
    static_for<0, NQ>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      if constexpr (kQK != 0) {
        if constexpr (j + kLeadA < NQ) kload(std::integral_constant<int, j + kLeadA>{});
        constexpr int s = j / 2;
        f32x16& acc = (j % 2 == 0) ? y0 : y1;
        if constexpr (kQK >= 2) {
          const i32x16 init = kQK == 2 ? magic : i32x16{};
          const i32x16 cin = (s == 0) ? init : __builtin_bit_cast(i32x16, acc);
          acc = __builtin_bit_cast(f32x16, mfma_i8(as_i32x4(kf[j]), q8f[s], cin));
          if constexpr (kQK == 3 && j >= NQ - 2) {   // exact INT32 -> FP32
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float raw = acc[r];   // (bit-casting the element lvalue reads element 0)
              acc[r] = (float)__builtin_bit_cast(int, raw);
            }
          }
        } else {
          acc = mfma_f16(as_half8(kf[j]), qf[s], s == 0 ? f32x16{} : acc);
        }
      }
      if constexpr (kExp) {   // the 16 exp pairs, spread evenly over the chunks
        static_for<(16 * j) / NQ, (16 * (j + 1)) / NQ>([&](auto pc) {
          constexpr int J = decltype(pc)::value;
          exp_pair<J>(x0, x1, c_x, k_x, pfr, (J & 1) ? zs1 : zs0);
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    __builtin_amdgcn_s_setprio(0);
    zs = zs0 + zs1;
  };

  // Phase B: P.V of tile n.
  auto phase_b = [&](int v_off, const half8 (&pfr)[4]) {
    constexpr int NP = 4 * (D / 32);   // chunks
    const char* vst = smem + v_off;
    uint4 vf[NP];
    auto vload = [&](auto jc) {
      constexpr int j = decltype(jc)::value, t = j / (D / 32), cc = j % (D / 32);
      vf[j] = ld_lds_16(vst, fo_128.at(t) + cc * 32 * C::kVRow);
    };
    static_for<0, (kLeadB < NP ? kLeadB : NP)>(vload);
    __builtin_amdgcn_s_setprio(1);
    static_for<0, NP>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      if constexpr (j + kLeadB < NP) vload(std::integral_constant<int, j + kLeadB>{});
      constexpr int t = j / (D / 32), cc = j % (D / 32);
      oacc[cc] = mfma_f16(as_half8(vf[j]), pfr[t], oacc[cc]);
      __builtin_amdgcn_sched_barrier(0);
    });
    __builtin_amdgcn_s_setprio(0);
  };

  // Lane max of a tile's 32 raw scores.
  auto lane_max = [](const f32x16& y0, const f32x16& y1) {
    float mx = max3f(y0[0], y0[1], y0[2]);
#pragma unroll
    for (int i = 3; i < 15; i += 2) mx = max3f(mx, y0[i], y0[i + 1]);
    mx = max3f(mx, y0[15], y1[0]);
#pragma unroll
    for (int i = 1; i < 15; i += 2) mx = max3f(mx, y1[i], y1[i + 1]);
    return fmaxf(mx, y1[15]);
  };

  // Raise the running max to the tile max mt (log2 units) where it is larger, rescaling the
  // accumulator and the normalizer by 2^(m_old - m_new), and re-derive the exp subtrahend.
  auto raise_max = [&](float mt) {
    const float m_new = fmaxf(m_run, mt);
    const float alpha = (m_run == kNegInf) ? 0.0f : __builtin_amdgcn_exp2f(m_run - m_new);
    z_run *= alpha;
#pragma unroll
    for (int cc = 0; cc < D / 32; ++cc) oacc[cc] *= alpha;
    m_run = m_new;
    msub = m_run;
    k_cur = fmaf(bias_cur, c_cur, msub);
  };
  // Factor and bias of key tile t's raw scores.
  auto set_tile = [&](bool int8, bool fold, uint16_t ks) {
    c_cur = int8 ? c_int8_q * half_bits_to_float(ks) : c_fp16;
    bias_cur = fold ? kMagic : 0.0f;
    k_cur = fmaf(bias_cur, c_cur, msub);
  };
  // Whether an INT8 tile with score factor c may carry the folded bias against the current
  // subtrahend (the same decision in every lane of the wave).
  auto fold_ok_c = [&](float c) { return !__any(!(fmaf(kMagic, c, fabsf(msub)) < kFoldLimit)); };
  auto fold_ok = [&](uint16_t ks) { return fold_ok_c(c_int8_q * half_bits_to_float(ks)); };
  // Drop the bias from a folded tile's raw scores when the running max moved past the fold's
  // bound: raw - 1.5 * 2^23 = C exactly (both lie in [2^23, 2^24)), so the tile continues as an
  // exactly converted one.
  auto unfold = [&](f32x16& y0, f32x16& y1) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      y0[r] -= kMagic;
      y1[r] -= kMagic;
    }
  };

  using True = std::integral_constant<bool, true>;
  using False = std::integral_constant<bool, false>;
  using QKNone = std::integral_constant<int, 0>;
  using QKFp16 = std::integral_constant<int, 1>;
  using QKInt8 = std::integral_constant<int, 2>;
  using QKInt8Exact = std::integral_constant<int, 3>;

  // Tiles whose every key every row of the workgroup may see: keys <= the first row's last key.
  const int wg_first_row_last_key = min(Lk - 1, m * BM + off);
  const int n_split = max(0, min(n_end + 1, (wg_first_row_last_key + 1) / kBlockN));

  wait_all_memory();   // tiles 0 and 1, issued before the query set-up
  __syncthreads();

  f32x16 xa0, xa1, xb0 = {}, xb1 = {};   // the two score buffers
  uint16_t ks0 = 0;
  if constexpr (OTF) {
    if (n_split > 0 && route_of(0)) ks0 = convert_k(k_slot(0));
  } else {
    ks0 = key_scale[0];
  }
  if (n_split > 0 && wave_active) {   // Q K^T of tile 0 and the running max it starts
    half8 unused_p[4];
    float unused_z;
    const bool int8 = route_of(0);
    const bool fold = int8 && fold_ok(ks0);
    const int k8_off = OTF ? kK8Off : k_slot(0);
    if (fold) phase_a(QKInt8{}, False{}, k8_off, xb0, xb1, xa0, xa1, unused_p, unused_z);
    else if (int8) phase_a(QKInt8Exact{}, False{}, k8_off, xb0, xb1, xa0, xa1, unused_p, unused_z);
    else phase_a(QKFp16{}, False{}, k_slot(0), xb0, xb1, xa0, xa1, unused_p, unused_z);
    if (int8) dbg_tile2(0, xa0, xa1, fold ? kDbgFolded : kDbgExact);
    set_tile(int8, fold, ks0);
    raise_max((pair_max(lane_max(xa0, xa1)) - bias_cur) * c_cur);
    if (fold && !fold_ok(ks0)) {   // the tile's own max moved the subtrahend past the bound
      unfold(xa0, xa1);
      set_tile(true, false, ks0);
    }
  }
  // Step n: scores of tile n in x, tile n + 1's go to y.
  auto step = [&](int n, f32x16& x0, f32x16& x1, f32x16& y0, f32x16& y1) {
    sync(n + 2, n + 1);   // K of tile n + 1 and V of tile n landed; K n + 2, V n + 1 in flight
    const bool has_next = n + 1 < n_split;
    const bool int8 = has_next && route_of(n + 1);
    uint16_t ks;
    if constexpr (OTF) ks = int8 ? convert_k(k_slot(n + 1)) : (uint16_t)0;   // whole workgroup
    else ks = key_scale[min(n + 1, n_end)];
    if (!wave_active) return;
    bool fold = int8 && fold_ok(ks);
    const int k8_off = OTF ? kK8Off : k_slot(n + 1);
    half8 pfr[4];
    float zs;
    if (!has_next) {
      y0 = f32x16{};
      y1 = f32x16{};
      phase_a(QKNone{}, True{}, 0, x0, x1, y0, y1, pfr, zs);
    } else if (fold) {
      phase_a(QKInt8{}, True{}, k8_off, x0, x1, y0, y1, pfr, zs);
    } else if (int8) {
      phase_a(QKInt8Exact{}, True{}, k8_off, x0, x1, y0, y1, pfr, zs);
    } else {
      phase_a(QKFp16{}, True{}, k_slot(n + 1), x0, x1, y0, y1, pfr, zs);
    }
    if (int8) dbg_tile2(n + 1, y0, y1, fold ? kDbgFolded : kDbgExact);
    if (__builtin_expect(__any(!(zs <= kSumLimit)), 0)) {
      // Some P of tile n left the comfortable FP16 range: refresh the running max from the
      // tile's exact max and redo its exp.  A folded tile n or n + 1 whose bias no longer
      // fits the fold's bound against the new subtrahend is converted exactly first.
      raise_max((pair_max(lane_max(x0, x1)) - bias_cur) * c_cur);
      if (bias_cur != 0.0f && !fold_ok_c(c_cur)) {
        unfold(x0, x1);
        bias_cur = 0.0f;
        k_cur = msub;
      }
      if (fold && !fold_ok(ks)) {
        unfold(y0, y1);
        fold = false;
      }
      f32x16 u0, u1;
      phase_a(QKNone{}, True{}, 0, x0, x1, u0, u1, pfr, zs);
    }
    z_run += zs;
    phase_b(v_slot(n), pfr);
    if (has_next) set_tile(int8, fold, ks);
  };
  int n = 0;
  for (; n + 1 < n_split; n += 2) {
    step(n, xa0, xa1, xb0, xb1);
    step(n + 1, xb0, xb1, xa0, xa1);
  }
  if (n < n_split) step(n, xa0, xa1, xb0, xb1);

  // Tiles crossing the diagonal or the sequence end, one at a time with the masked softmax;
  // waves whose rows see no key of a tile skip its math.
  for (n = n_split; n <= n_end; ++n) {
    sync(n + 1, n + 1);   // tile n landed; the slots of tile n - 1 take tile n + 1
    uint16_t ks_otf = 0;
    if constexpr (OTF) {
      if (route_of(n)) ks_otf = convert_k(k_slot(n));   // whole workgroup
    }
    if (wave_active && n * kBlockN <= wave_last_key) {
      float svm[32], c;
      qk(n, svm, c, ks_otf);
      if (route_of(n)) dbg_tile(n, svm, kDbgMasked);
      half8 pfr[4];
      softmax_step<D, true>(svm, c, n * kBlockN, my_last_key, lane, m_run, z_run, oacc, pfr);
      pv(n, pfr);
    }
  }

  // Epilogue: O = O~ / z~, FP16 (round to nearest even).
  if (wave_active) {
    const float zt = pair_sum(z_run);
    const float inv = zt > 0.0f ? 1.0f / zt : 0.0f;
    if (row_ok) {
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
}

// INT32 tile products C = Q8_m K8_n^T through the same staging and matrix-core code as the
// INT8 route of the fused kernel.  One workgroup per requested tile.
template <int D, int BM>
__global__ __launch_bounds__(2 * BM) void debug_tiles_kernel(DebugTileArgs a) {
  using C = TileCfg<D, BM, 1>;
  __shared__ __align__(16) char smem[C::kStage];
  const int e = blockIdx.x;
  const int b = a.tiles[4 * e + 0], hq = a.tiles[4 * e + 1];
  const int m = a.tiles[4 * e + 2], n = a.tiles[4 * e + 3];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & (kWave - 1);
  const int lq = lane & 31, hi = lane >> 5;
  int32_t* out = a.out + (size_t)e * BM * kBlockN;
  const bool ok = b >= 0 && b < a.B && hq >= 0 && hq < a.Hq && m >= 0 && n >= 0 &&
                  m * BM < a.Lq && n * kBlockN < a.Lk;
  if (!ok) {
    for (int i = tid; i < BM * kBlockN; i += C::kThreads) out[i] = 0;
    return;
  }
  const int hk = hq / (a.Hq / a.Hk);
  const int kstride = a.Hk * D * 2;
  const char* k8t = reinterpret_cast<const char*>(a.K8) +
                    ((size_t)b * a.Lk * a.Hk + hk) * D + (size_t)n * kBlockN * (kstride / 2);
  const int rows = min(kBlockN, a.Lk - n * kBlockN);
  const DmaPlan<C::kK8Row> plan_k8(lane, kstride / 2);
  dma_tile<C::kK8Row, C::kK8Instr, kBlockN>(k8t, kstride / 2, rows, lds_addr_of(smem), wave, lane,
                                            plan_k8);
  wait_all_memory();
  __syncthreads();
  const int my_q = m * BM + 32 * wave + lq;
  i32x4 q8f[D / 32];
  const size_t qoff = (((size_t)b * a.Lq + (my_q < a.Lq ? my_q : 0)) * a.Hq + hq) * D;
#pragma unroll
  for (int s = 0; s < D / 32; ++s)
    q8f[s] = (my_q < a.Lq) ? as_i32x4(ld_global_16(a.Q8 + qoff + 32 * s + 16 * hi)) : i32x4{};
  const FragOffsets<C::kK8Row> fo_k8(lane);
  i32x16 i0, i1;
  qk_int8<D>(smem, fo_k8, q8f, i0, i1);
  const int row = 32 * wave + lq;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int k0 = acc_row(r, lane), k1 = 32 + acc_row(r, lane);
    out[row * kBlockN + k0] = k0 < rows ? i0[r] : 0;      // keys past L_k: 0
    out[row * kBlockN + k1] = k1 < rows ? i1[r] : 0;
  }
}

template <int D, int BM, int HEADS, bool OTF = false>
hipError_t launch_attn_t(const AttnArgs& a, hipStream_t stream) {
  using C = TileCfg<D, BM, HEADS>;
  const long long grid = (long long)a.B * (a.Hq / HEADS) * a.T_m;
  if (grid <= 0 || grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (a.dbg_tiles)
    hipLaunchKernelGGL((routed_attn_fwd_kernel<D, BM, HEADS, OTF, true>), dim3((unsigned)grid),
                       dim3(C::kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((routed_attn_fwd_kernel<D, BM, HEADS, OTF>), dim3((unsigned)grid),
                       dim3(C::kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D, int BM>
hipError_t launch_debug_t(const DebugTileArgs& a, hipStream_t stream) {
  using C = TileCfg<D, BM, 1>;
  hipLaunchKernelGGL((debug_tiles_kernel<D, BM>), dim3(a.count), dim3(C::kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_routed_attention(const AttnArgs& a, int d, int block_m, hipStream_t stream) {
  // One query head per workgroup; two workgroups share a CU.
  // On-the-fly operands: an all-FP16 map has nothing to quantize, and the quantize-once kernel
  // then reads neither Q8 nor K8 nor their scales.
  if (a.on_the_fly && !a.force_fp16) {
    if (d == 128 && block_m == 128) return launch_attn_t<128, 128, 1, true>(a, stream);
    if (d == 128 && block_m == 64) return launch_attn_t<128, 64, 1, true>(a, stream);
    if (d == 64 && block_m == 128) return launch_attn_t<64, 128, 1, true>(a, stream);
    if (d == 64 && block_m == 64) return launch_attn_t<64, 64, 1, true>(a, stream);
    return hipErrorInvalidValue;
  }
  if (d == 128 && block_m == 128) return launch_attn_t<128, 128, 1>(a, stream);
  if (d == 128 && block_m == 64) return launch_attn_t<128, 64, 1>(a, stream);
  if (d == 64 && block_m == 128) return launch_attn_t<64, 128, 1>(a, stream);
  if (d == 64 && block_m == 64) return launch_attn_t<64, 64, 1>(a, stream);
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
