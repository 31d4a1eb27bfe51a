// Shared device helpers for the gfx950 (CDNA4) kernels of libmapl.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mapl {

typedef uint16_t bf16_t;  // bf16 stored as its bit pattern

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

constexpr int WAVE = 64;

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 bits (lo in bits 0..15), round to nearest even:
// one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}
__device__ __forceinline__ uint32_t f2bf(float f) { return pack_bf2(f, 0.f) & 0xFFFFu; }
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// 32x32x16 bf16 MFMA, fp32 accumulate.
// Lane l holds A[m = l%32][k = 8(l/32) .. +7] and B[k = 8(l/32) .. +7][n = l%32];
// accumulator j of lane l is D[m = 8(j/4) + 4(l/32) + j%4][n = l%32].
__device__ __forceinline__ f32x16_t mfma32x32x16(const uint4& a, const uint4& b, f32x16_t c) {
  bf16x8_t av = __builtin_bit_cast(bf16x8_t, a);
  bf16x8_t bv = __builtin_bit_cast(bf16x8_t, b);
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, c, 0, 0, 0);
}

// 32x32x2 fp32 MFMA: lane l holds A[m = l%32][k = l/32], B[k = l/32][n = l%32];
// accumulator layout as above.
__device__ __forceinline__ f32x16_t mfma32x32x2f32(float a, float b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Token ids outside [0, V) read row 0 instead of faulting.
__device__ __forceinline__ int clamp_id(int id, int V) { return (unsigned)id < (unsigned)V ? id : 0; }

__device__ __forceinline__ int acc_row(int j, int lane) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

// Screening margin of the RVQ kernel for residual width R:
//   |s~_j - s_j| <= k1 ||R|| ||C_j|| + k2 ||C_j||^2, with
//   k1 = 2 (2^-7 (bf16 rounding of both operands) + R 2^-24 (fp32
//   accumulation)) plus the rounding of the fused add and of the fp32 norms,
//   and k2 covering the fp32 norm ||C_j||^2; both inflated.
__host__ __device__ constexpr float rvq_margin_k1(int R) {
  return 0.015625f * 1.0078125f + 8.0f * R / 16777216.0f + 1.0f / 1048576.0f;
}
__host__ __device__ constexpr float rvq_margin_k2(int R) { return 4.0f * (R + 2) / 16777216.0f; }

// Wave-wide reductions (wave64) through LDS-free cross-lane shuffles.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, WAVE));
  return v;
}

}  // namespace mapl
