// Device-side vector types and conversions for gfx950 (CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace s2l {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

__device__ inline uint32_t f2u(float x) { return __builtin_bit_cast(uint32_t, x); }
__device__ inline float u2f(uint32_t x) { return __builtin_bit_cast(float, x); }

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ inline uint32_t pack_bf16x2(float a, float b) {
  f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Four E4M3 codes (one dword) -> four bf16 (two dwords), two codes per instruction
// (v_cvt_scalef32_pk_bf16_fp8 with scale 1).  Exact: every E4M3 value is a bf16 value, so
// the scaled conversion by 1 rounds nothing; NaN codes give bf16 NaN.
__device__ inline u32x2 fp8x4_to_bf16x4(uint32_t w) {
  u32x2 r;
  r[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false));
  r[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true));
  return r;
}

// Saturate to the finite E4M3 range; NaN passes through (comparisons with NaN are false).
__device__ inline float sat448(float x) { return x > 448.f ? 448.f : (x < -448.f ? -448.f : x); }

// Four fp32 -> four E4M3 codes (RNE, v_cvt_pk_fp8_f32), after saturation.
__device__ inline uint32_t f32x4_to_fp8x4(float a, float b, float c, float d) {
  uint32_t w = 0;
  w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(sat448(a), sat448(b), (int)w, false);
  w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(sat448(c), sat448(d), (int)w, true);
  return w;
}

// acc + lo + hi of a packed bf16 pair, in fp32 (v_dot2_f32_bf16 with (1, 1)).
__device__ inline float sum_bf16x2(uint32_t w, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), __builtin_bit_cast(bf16x2, 0x3F803F80u), acc,
                                         false);
}

__device__ inline float bf16lo(uint32_t w) { return u2f(w << 16); }
__device__ inline float bf16hi(uint32_t w) { return u2f(w & 0xFFFF0000u); }

// Combination over the lane pair (l, l ^ 32) with v_permlane32_swap, written as one
// assembly block: the compiler treats the two results of permlane32_swap(x, x) as equal and
// folds max(r0, r1) to r0 and r0 + r1 to 2 r0.  The s_nops keep the swap's operand reads
// and the combining read apart from the VALU writes before them.  The input must come from
// an ordinary VALU instruction (not an MFMA or a transcendental), whose hazards are the
// only ones these wait states cover.
__device__ inline float max_with_partner(float x) {
  float y;
  __asm__("s_nop 1\n\tv_mov_b32 %1, %0\n\ts_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1\n\t"
          "v_max_f32 %0, %0, %1"
          : "+v"(x), "=&v"(y));
  return x;
}
__device__ inline float sum_with_partner(float x) {
  float y;
  __asm__("s_nop 1\n\tv_mov_b32 %1, %0\n\ts_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1\n\t"
          "v_add_f32 %0, %0, %1"
          : "+v"(x), "=&v"(y));
  return x;
}

// Outputs of a launch whose device plan did not fit the host's sizing (its status word is
// not 0: the device length arrays disagree with the host copies, and nothing was planned).
// Every workgroup writes NaN over its share of the `rows` output rows the host sized the
// call for (rows blockIdx.x, blockIdx.x + gridDim.x, ...: out [rows][hq][128] bf16, lse
// [rows][hq] fp32), so that the failure shows in the results instead of stale memory.
__device__ inline void poison_outputs(uint16_t* out, float* lse, int64_t rows, int32_t hq) {
  const int64_t chunks = (int64_t)hq * 16;            // 16-byte chunks of one output row
  for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
    uint16_t* orow = out + r * hq * 128;
    for (int64_t c = threadIdx.x; c < chunks; c += blockDim.x)
      *reinterpret_cast<u32x4*>(orow + 8 * c) = u32x4{0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u};
    if (lse != nullptr)
      for (int h = threadIdx.x; h < hq; h += blockDim.x) lse[r * hq + h] = __builtin_nanf("");
  }
}

}  // namespace s2l
