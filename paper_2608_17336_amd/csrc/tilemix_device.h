// tilemix_device.h -- shared gfx950 device helpers for the TileMix kernels.
//
// Matrix-core shapes used (CDNA4 / gfx950, wave64):
//   v_mfma_f32_32x32x16_f16 : A 32x16, B 16x32 FP16 -> D 32x32 FP32
//   v_mfma_i32_32x32x32_i8  : A 32x32, B 32x32 INT8 -> D 32x32 INT32 (exact)
// Operand lane layout (both shapes): lane l holds row/column (l % 32) and the
// contraction slice [kw*(l/32), kw*(l/32)+kw) with kw = 8 (f16) or 16 (i8).
// Accumulator layout: register r of lane l is D[8*(r/4) + 4*(l/32) + r%4][l%32].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tilemix {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kQuantBlockQ = 128;  // query rows per INT8 scale block (Appendix C)
constexpr int kQuantBlockK = 64;   // key rows per INT8 scale block (Appendix C)
constexpr int kBlockN = 64;        // keys per compute tile (= key scale block)
constexpr int kMaxKeyTiles = 4096; // key tiles per row whose scales the kernel holds in LDS
                                   // (L_k <= 262144); also bounds the routing words per row
                                   // to 64, which one register pair per wave holds

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

// Lanes l and l^32 of a 32x32 accumulator column hold the same query row.  After
// v_permlane32_swap with both operands equal to x, the two results of every lane are
// {x[l], x[l ^ 32]} (in lane-dependent order), so their max / sum is the pair value.
__device__ __forceinline__ float pair_max(float x) {
  const int v = __builtin_bit_cast(int, x);
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__builtin_bit_cast(float, (int)r[0]), __builtin_bit_cast(float, (int)r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
  const int v = __builtin_bit_cast(int, x);
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __builtin_bit_cast(float, (int)r[0]) + __builtin_bit_cast(float, (int)r[1]);
}

// Direct global -> LDS copy of 16 bytes per lane: lane l reads base + voff and writes LDS byte
// lds_addr + 16*l (base and lds_addr wave-uniform).  Completion is tracked by vmcnt like any
// vector load; it is issued as inline assembly so that the only waits on it are the explicit
// vmcnt waits of the caller (the compiler would otherwise wait for every copy in flight
// before any LDS read, whichever LDS bytes the copies write).
// base and lds_addr pass through readfirstlane (a no-op on values the compiler already holds in
// scalar registers), so that the scalar operands stay scalar where its uniformity analysis
// loses track of them.
// m0 is a register the compiler reserves (it warns that the clobber names one); the code it
// generates for these kernels never reads m0, so setting it here disturbs nothing else.
__device__ __forceinline__ void dma_16(const void* base, uint32_t voff, uint32_t lds_addr) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const uint64_t bs = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  const uint32_t ls = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds_addr);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"((const void*)(uintptr_t)bs), "s"(ls)
               : "m0");
}

// 32-bit LDS address of a __shared__ object.
template <typename T>
__device__ __forceinline__ uint32_t lds_addr_of(T* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)(p);
}

// Wait for every outstanding memory operation of the wave (vector, scalar, LDS).  Emitted with
// the builtin, so the compiler knows its own earlier loads are complete as well.
__device__ __forceinline__ void wait_all_memory() { __builtin_amdgcn_s_waitcnt(0); }

__device__ __forceinline__ uint4 ld_global_16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ void st_lds_16(char* lds, int off, uint4 v) {
  *reinterpret_cast<uint4*>(lds + off) = v;
}

__device__ __forceinline__ uint4 ld_lds_16(const char* lds, int off) {
  return *reinterpret_cast<const uint4*>(lds + off);
}

__device__ __forceinline__ half8 as_half8(uint4 v) { return __builtin_bit_cast(half8, v); }
__device__ __forceinline__ i32x4 as_i32x4(uint4 v) { return __builtin_bit_cast(i32x4, v); }

__device__ __forceinline__ f32x16 mfma_f16(half8 a, half8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ i32x16 mfma_i8(i32x4 a, i32x4 b, i32x16 c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

// Key (row of the 32x32 accumulator block) held by register r of lane l.
__device__ __forceinline__ int acc_row(int r, int lane) {
  return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}

}  // namespace tilemix
