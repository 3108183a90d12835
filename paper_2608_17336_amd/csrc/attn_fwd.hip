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

constexpr float kRescaleThreshold = 8.0f;   // log2 units: rescale when the max grows > x256
constexpr float kNegInf = -__builtin_huge_valf();

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

// s_waitcnt takes an immediate: wait until at most `n` vector-memory operations of this wave
// are outstanding (loads complete in issue order).  `n` is wave-uniform.
__device__ __forceinline__ void wait_vmem_at_most(int n) {
  switch (n) {
#define TM_WAIT_CASE(k) case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
    TM_WAIT_CASE(0) TM_WAIT_CASE(1) TM_WAIT_CASE(2) TM_WAIT_CASE(3) TM_WAIT_CASE(4)
    TM_WAIT_CASE(5) TM_WAIT_CASE(6) TM_WAIT_CASE(7) TM_WAIT_CASE(8) TM_WAIT_CASE(9)
    TM_WAIT_CASE(10) TM_WAIT_CASE(11) TM_WAIT_CASE(12) TM_WAIT_CASE(13) TM_WAIT_CASE(14)
    TM_WAIT_CASE(15) TM_WAIT_CASE(16) TM_WAIT_CASE(17) TM_WAIT_CASE(18) TM_WAIT_CASE(19)
    TM_WAIT_CASE(20) TM_WAIT_CASE(21) TM_WAIT_CASE(22) TM_WAIT_CASE(23) TM_WAIT_CASE(24)
    TM_WAIT_CASE(25) TM_WAIT_CASE(26) TM_WAIT_CASE(27) TM_WAIT_CASE(28) TM_WAIT_CASE(29)
    TM_WAIT_CASE(30) TM_WAIT_CASE(31) TM_WAIT_CASE(32)
#undef TM_WAIT_CASE
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
}

__device__ __forceinline__ float load_scale_uniform(const uint16_t* base, size_t idx) {
  // The scale arrays live in 256-byte aligned workspace slots, so reading the aligned
  // 32-bit word that holds element idx stays inside the slot.
  const uint32_t w = reinterpret_cast<const uint32_t*>(base)[idx >> 1];
  return half_bits_to_float((uint16_t)((idx & 1) ? (w >> 16) : (w & 0xffffu)));
}

template <int D, int BM, int HEADS, int NSTAGE, bool PINGPONG>
__global__ __launch_bounds__(HEADS * 2 * BM, 2) void routed_attn_fwd_kernel(AttnArgs a) {
  using C = TileCfg<D, BM, HEADS>;
  __shared__ __align__(16) char smem[NSTAGE * C::kStage];
  __shared__ uint16_t key_scale[kMaxKeyTiles];   // dK of this row's key tiles (FP16 bits)

  int b, hq0, hk, m;
  decode_unit<HEADS>(blockIdx.x, a.B, a.Hq, a.Hk, a.T_m, b, hq0, hk, m);

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
  const int off = a.causal ? a.Lk - a.Lq : a.Lk;
  const bool wave_active = q0 < a.Lq;

  // Last key any row of the workgroup / of this wave may see.
  const int wg_last_key = min(a.Lk - 1, min(a.Lq - 1, m * BM + BM - 1) + off);
  const int wave_last_key = min(a.Lk - 1, min(a.Lq - 1, q0 + 31) + off);
  const int first_row_last_key = min(a.Lk - 1, q0 + off);    // smallest last key of the wave
  const int my_last_key = min(a.Lk - 1, my_q + off);

  _Float16* orow = a.O + (((size_t)b * a.Lq + my_q) * a.Hq + hq) * D;
  if (wg_last_key < 0) {   // no legal key for any row of this tile: output is zero
    if (my_q < a.Lq) {     // the two lanes of a row each clear half of it
#pragma unroll
      for (int c = 0; c < D / 2; c += 8) *reinterpret_cast<half8*>(orow + hi * (D / 2) + c) = half8{};
    }
    return;
  }
  const int n_end = wg_last_key / kBlockN;

  // Routing words of this row: lane w holds word w (at most 64 words per row), so the
  // per-tile lookup is a lane read plus a shift-and-mask, with no memory access in the loop.
  const uint64_t* route_row =
      a.route + (size_t)b * a.route_batch_stride + ((size_t)hk * a.T_m + m) * a.W;
  const uint64_t my_word = (!a.force_fp16 && lane < a.W) ? route_row[lane] : 0ull;
  const uint32_t word_lo = (uint32_t)my_word, word_hi = (uint32_t)(my_word >> 32);
  auto route_of = [&](int n) -> bool {
    const int gj = n / a.g;
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
                       ? load_scale_uniform(a.dQ, ((size_t)b * a.nQB + q0 / kQuantBlockQ) * a.Hq + hq)
                       : 0.0f;
  const float c_fp16 = a.scale_log2e;
  const float c_int8_q = a.scale_log2e * dq;
  if (need_int8) {   // key-block scales of the tiles this row visits (key block = key tile)
    for (int t = tid; t <= n_end; t += C::kThreads)
      key_scale[t] = a.dK[((size_t)b * a.nKB + t) * a.Hk + hk];
  }

  // Tile sources (uniform bases) and per-lane LDS fragment offsets.
  const int kstride = a.Hk * D * 2;                              // bytes between keys (FP16)
  const char* kbase = reinterpret_cast<const char*>(a.K) + ((size_t)b * a.Lk * a.Hk + hk) * D * 2;
  const char* k8base = reinterpret_cast<const char*>(a.K8) + ((size_t)b * a.Lk * a.Hk + hk) * D;
  const char* vbase = reinterpret_cast<const char*>(a.Vt) +
                      ((size_t)b * a.Hk + hk) * a.T_n * (size_t)(D * kBlockN * 2);
  const DmaPlan<C::kKRow> plan_k(lane, kstride);
  const DmaPlan<C::kK8Row> plan_k8(lane, kstride / 2);
  const DmaPlan<C::kVRow> plan_v(lane, C::kVRow);
  auto stage_of = [&](int n) -> char* { return smem + (n % NSTAGE) * C::kStage; };
  const uint32_t smem_lds = lds_addr_of(smem);
  auto copies = [&](bool int8) -> int { return (int8 ? C::kK8Instr : C::kKInstr) + C::kVInstr; };
  auto issue = [&](int n, bool int8) {   // start copying key tile n into its stage
    const uint32_t st = smem_lds + (uint32_t)((n % NSTAGE) * C::kStage);
    const int rows = min(kBlockN, a.Lk - n * kBlockN);
    if (int8)
      dma_tile<C::kK8Row, C::kK8Instr, kBlockN>(k8base + (size_t)n * kBlockN * (kstride / 2),
                                                kstride / 2, rows, st, wave, lane, plan_k8);
    else   // 8 copies per 64-channel half of the FP16 key tile
      dma_tile<C::kKRow, C::kKInstr, kBlockN, 8, 128>(kbase + (size_t)n * kBlockN * kstride, kstride,
                                                      rows, st, wave, lane, plan_k);
    dma_tile<C::kVRow, C::kVInstr, D>(vbase + (size_t)n * (D * kBlockN * 2), C::kVRow, D,
                                      st + C::kKBytes, wave, lane, plan_v);
  };
  const FragOffsets<128> fo_128(lane);      // K (FP16 halves), V^T, and K8 when d = 128
  const FragOffsets<C::kK8Row> fo_k8(lane);

  // Online-softmax state (Section 3.1), FP32; max kept in log2 units.
  float m_run = kNegInf;
  float z_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) oacc[c] = f32x16{};

  // Raw scores of key tile n for this wave (INT32 products converted to float, or FP32 dot
  // products) and the factor c that turns them into log2-domain scaled scores.
  auto qk = [&](int n, float (&sv)[32], float& c) {
    const char* kst = stage_of(n);
    if (route_of(n)) {
      i32x16 i0, i1;
      qk_int8<D>(kst, fo_k8, q8f, i0, i1);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sv[r] = (float)i0[r];
        sv[16 + r] = (float)i1[r];
      }
      c = c_int8_q * half_bits_to_float(key_scale[n]);
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
    const char* vst = stage_of(n) + C::kKBytes;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int cc = 0; cc < D / 32; ++cc) {
        const half8 va = as_half8(ld_lds_16(vst, fo_128.at(t) + cc * 32 * C::kVRow));
        oacc[cc] = mfma_f16(va, pfr[t], oacc[cc]);
      }
    }
  };
  // Does this wave have a legal key in tile n (only in doubt on masked tiles)?
  auto sees = [&](int n, bool masked) { return wave_active && (!masked || n * kBlockN <= wave_last_key); };

  // Schedule.  Copies run PD tiles ahead of the math.  With PINGPONG the second head of the
  // pair runs each tile half an iteration late: while the first head's wave multiplies Q K^T of
  // tile n on the matrix cores, its SIMD partner (same SIMD, other head) runs the softmax of
  // tile n - 1 on the vector ALU, then takes the matrix cores for P.V of tile n - 1 and Q K^T of
  // tile n while the first head runs its softmax.  It keeps tile n - 1's scores in registers
  // across the tile barrier and needs V of tile n - 1 still resident: one extra LDS stage.
  constexpr int PD = PINGPONG ? NSTAGE - 2 : NSTAGE - 1;
  static_assert(PD >= 1, "at least one tile of copy lead");
  static_assert(!PINGPONG || HEADS == 2, "ping-pong pairs the two heads of a workgroup");
  const bool late = PINGPONG && (wave >= C::kWavesPerHead);

  for (int t = 0; t < PD; ++t)
    if (t <= n_end) issue(t, route_of(t));
  wait_all_memory();
  __syncthreads();

  // Start the copy of tile n + PD; at the end of a tile, tile n + 1 must have landed for every
  // wave while copies of tiles n + 2 .. n + PD may stay in flight.
  auto prefetch = [&](int n) {
    if (n + PD <= n_end) issue(n + PD, route_of(n + PD));
  };
  auto finish_tile = [&](int n) {
    int pending = 0;
    for (int t = n + 2; t <= min(n + PD, n_end); ++t) pending += copies(route_of(t));
    wait_vmem_at_most(pending);
    __syncthreads();   // tile n + 1 visible to every wave; the oldest stage released
  };
  auto early_tile = [&](int n, auto masked_tag) {
    constexpr bool kMasked = decltype(masked_tag)::value;
    prefetch(n);
    if (sees(n, kMasked)) {
      float sv[32], c;
      qk(n, sv, c);
      half8 pfr[4];
      softmax_step<D, kMasked>(sv, c, n * kBlockN, my_last_key, lane, m_run, z_run, oacc, pfr);
      pv(n, pfr);
    }
    finish_tile(n);
  };

  // Tiles whose every key every row of the workgroup may see: keys <= the first row's last key.
  const int wg_first_row_last_key = min(a.Lk - 1, m * BM + off);
  const int n_split = max(0, min(n_end + 1, (wg_first_row_last_key + 1) / kBlockN));
  using Unmasked = std::integral_constant<bool, false>;
  using Masked = std::integral_constant<bool, true>;
  if (!late) {
    int n = 0;
    for (; n < n_split; ++n) early_tile(n, Unmasked{});
    for (; n <= n_end; ++n) early_tile(n, Masked{});
  } else {
    float sv_late[32];   // scores of the previous tile, carried across the tile barrier
    float c_late = 0.0f;
    // Each tile's softmax uses the same (masked or unmasked) variant as in the early head, so
    // the two heads compute bit-identical results on identical inputs.
    auto late_tile = [&](int n, auto prev_masked_tag, auto cur_masked_tag) {
      constexpr bool kPrevMasked = decltype(prev_masked_tag)::value;
      constexpr bool kCurMasked = decltype(cur_masked_tag)::value;
      prefetch(n);
      if (n >= 1 && sees(n - 1, kPrevMasked)) {
        half8 pfr[4];
        softmax_step<D, kPrevMasked>(sv_late, c_late, (n - 1) * kBlockN, my_last_key, lane, m_run,
                                     z_run, oacc, pfr);
        pv(n - 1, pfr);
      }
      if (sees(n, kCurMasked)) qk(n, sv_late, c_late);
      finish_tile(n);
    };
    int n = 0;
    for (; n < n_split; ++n) late_tile(n, Unmasked{}, Unmasked{});
    if (n <= n_end) late_tile(n++, Unmasked{}, Masked{});
    for (; n <= n_end; ++n) late_tile(n, Masked{}, Masked{});
    half8 pfr[4];   // the last tile's softmax and P.V
    if (n_end < n_split) {
      if (sees(n_end, false)) {
        softmax_step<D, false>(sv_late, c_late, n_end * kBlockN, my_last_key, lane, m_run, z_run,
                               oacc, pfr);
        pv(n_end, pfr);
      }
    } else if (sees(n_end, true)) {
      softmax_step<D, true>(sv_late, c_late, n_end * kBlockN, my_last_key, lane, m_run, z_run,
                            oacc, pfr);
      pv(n_end, pfr);
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

template <int D, int BM, int HEADS, int NSTAGE, bool PINGPONG = false>
hipError_t launch_attn_t(const AttnArgs& a, hipStream_t stream) {
  using C = TileCfg<D, BM, HEADS>;
  const long long grid = (long long)a.B * (a.Hq / HEADS) * a.T_m;
  if (grid <= 0 || grid > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL((routed_attn_fwd_kernel<D, BM, HEADS, NSTAGE, PINGPONG>), dim3((unsigned)grid),
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
  // d = 128: two query heads of a GQA group per workgroup (one K/V copy serves both) when the
  // group has an even number of heads, with three LDS stages.  d = 64: one head, four stages.
  const bool pair = ((a.Hq / a.Hk) % 2) == 0;
  if (d == 128 && block_m == 128)
    return pair ? launch_attn_t<128, 128, 2, 3, true>(a, stream) : launch_attn_t<128, 128, 1, 2>(a, stream);
  if (d == 128 && block_m == 64)
    return pair ? launch_attn_t<128, 64, 2, 2>(a, stream) : launch_attn_t<128, 64, 1, 2>(a, stream);
  if (d == 64 && block_m == 128) return launch_attn_t<64, 128, 1, 4>(a, stream);
  if (d == 64 && block_m == 64) return launch_attn_t<64, 64, 1, 4>(a, stream);
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
