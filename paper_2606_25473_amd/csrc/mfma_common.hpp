// mfma_common.hpp -- device helpers shared by the bf16 matrix-core kernels (gfx950):
// operand types, the LDS row swizzle, MFMA and transposed-LDS-read wrappers, and the
// direct global -> LDS load.  Device code only; included by the .hip kernel files.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace attn {
namespace dev {

typedef __bf16 bf16_t;
typedef bf16_t bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16_t bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// XOR swizzle of the 16-byte chunks within an LDS row (D / 8 chunks per row):
// conflict-free both for the 16 consecutive rows of a b128 score-operand read (16 lanes
// per pass over the 64 banks) and for the 4-row x 4-chunk footprint of a transposed read.
// It depends on row bits 0..3 only, and not on bit 4, so the offsets of rows r and r + 16
// differ by a constant (the transposed reads of both k steps share one base).
template <int D>
__device__ __forceinline__ int swz(int row) {
  static_assert(D == 64 || D == 128, "head_dim 64 or 128");
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);  // 128-byte rows: two per 64 banks
}

template <int D>
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * (2 * D) + ((chunk ^ swz<D>(row)) << 4);  // rows of D bf16
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x4 ld_tr(const char* p) {
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(p));
  return __builtin_bit_cast(bf16x4, v);
}

// The same reads from a 32-bit LDS byte address (ds_read_b64_tr_b16 / ds_read_b128).
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
__device__ __forceinline__ bf16x4 ld_tr_at(unsigned addr) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)addr));
}
__device__ __forceinline__ bf16x8 ld128_at(unsigned addr) { return *(lds_bf16x8*)(uintptr_t)addr; }

// u + v in a vector register, opaque to the compiler.  Offsets derived from the result
// (one XOR per operand read) are then formed where they are used instead of being
// hoisted out of the key-block loop, where each would hold a register for the whole
// loop.  The optional `dep` (unused by the instruction) ties the result to a loop-variant
// value when u and v are loop-invariant.
__device__ __forceinline__ unsigned vreg_add(unsigned u, unsigned v) {
  unsigned r;
  asm("v_add_u32 %0, %1, %2" : "=v"(r) : "s"(u), "v"(v));
  return r;
}
__device__ __forceinline__ unsigned vreg_add(unsigned u, unsigned v, int dep) {
  unsigned r;
  asm("v_add_u32 %0, %1, %2 ; %3" : "=v"(r) : "s"(u), "v"(v), "s"(dep));
  return r;
}

// Maximum of 16 floats (never NaN) in 8 v_max3_f32, one asm block (separate asm
// statements get a wait state between them).  The compiler's own fmaxf chain first
// quiets its inputs (IEEE mode): two more instructions per call.
__device__ __forceinline__ float max16(const float v[16]) {
  float m;
  asm("v_max3_f32 %0, %1, %2, %3\n\t"
      "v_max3_f32 %0, %0, %4, %5\n\t"
      "v_max3_f32 %0, %0, %6, %7\n\t"
      "v_max3_f32 %0, %0, %8, %9\n\t"
      "v_max3_f32 %0, %0, %10, %11\n\t"
      "v_max3_f32 %0, %0, %12, %13\n\t"
      "v_max3_f32 %0, %0, %14, %15\n\t"
      "v_max_f32 %0, %0, %16"
      : "=&v"(m)
      : "v"(v[0]), "v"(v[1]), "v"(v[2]), "v"(v[3]), "v"(v[4]), "v"(v[5]), "v"(v[6]), "v"(v[7]),
        "v"(v[8]), "v"(v[9]), "v"(v[10]), "v"(v[11]), "v"(v[12]), "v"(v[13]), "v"(v[14]), "v"(v[15]));
  return m;
}

__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32, 64); }

// Direct global -> LDS load of 16 bytes per lane (global_load_lds_dwordx4): lane l's
// bytes land at LDS address lds + 16 l.  Issued from inline assembly on purpose: the
// compiler then does not track these loads, so it never inserts waits for them before
// LDS reads of other pipeline stages (it cannot tell stages apart when the stage index
// is a run-time value).  The kernel waits for them itself (vmcnt) before a barrier.
// M0 carries the LDS base address (one wait state separates its write from the load);
// M0 is saved and restored around the load because the compiler reserves it.
__device__ __forceinline__ void lds_load16(const void* gbase, unsigned byte_off, unsigned lds) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(byte_off), "s"(gbase), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}

// Direct global -> LDS load of 4 bytes per lane (lane l's bytes land at lds + 4 l);
// same contract as lds_load16.
__device__ __forceinline__ void lds_load4(const void* gbase, unsigned byte_off, unsigned lds) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(byte_off), "s"(gbase), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}

__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Per-lane offsets of the transposed operand reads (ds_read_b64_tr_b16) of a 32-row
// tile whose rows are listed in the accumulator order of a 32x32 MFMA output:
// tro[t][p][dt] for k step t (16 rows), row half p (+0 / +8), d tile dt.  In each
// 16-lane group, lane j receives element j%4 of the 8-byte word addressed by lane
// 4e + j/4 (e = result element); the addresses below make the row order of the
// operand equal to that of the B operand taken from the lane's own accumulator.
template <int D>
__device__ __forceinline__ void tr_offsets(int lane, int tro[2][2][D / 32]) {
  const int g16 = lane >> 4, s16 = lane & 15;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const int r = 16 * t + 8 * p + 4 * (g16 >> 1) + (s16 >> 2);
        const int chunk = 4 * dt + 2 * (g16 & 1) + ((s16 & 3) >> 1);
        tro[t][p][dt] = lds_off<D>(r, chunk) + 8 * (s16 & 1);
      }
}

// The same offsets as two bases: with the row swizzle, tro[t][p][dt] equals
// 16 t ROWB + (trx[p] ^ (64 dt)), so a kernel keeps trx[0..1] in registers and forms
// each read's offset with one XOR.
template <int D>
__device__ __forceinline__ void tr_bases(int lane, unsigned trx[2]) {
  const int g16 = lane >> 4, s16 = lane & 15;
  const int r = 4 * (g16 >> 1) + (s16 >> 2), chunk = 2 * (g16 & 1) + ((s16 & 3) >> 1);
  trx[0] = lds_off<D>(r, chunk) + 8 * (s16 & 1);
  trx[1] = lds_off<D>(8 + r, chunk) + 8 * (s16 & 1);
}

}  // namespace dev
}  // namespace attn
