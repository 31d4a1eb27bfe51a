// Shared device helpers for the gfx950 (CDNA4) kernels of libmapl.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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

// 32x32x16 fp16 MFMA, fp32 accumulate; same lane layout as mfma32x32x16.
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8_t;
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ f32x16_t mfma32x32x16h(const uint4& a, const uint4& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c,
                                                0, 0, 0);
}

// 16x16x32 bf16 MFMA, fp32 accumulate.
// Lane l holds A[m = l%16][k = 8(l/16) .. +7] and B[k = 8(l/16) .. +7][n = l%16];
// accumulator j of lane l is D[m = 4(l/16) + j][n = l%16].
__device__ __forceinline__ f32x4_t mfma16x16x32(const uint4& a, const uint4& b, f32x4_t c) {
  bf16x8_t av = __builtin_bit_cast(bf16x8_t, a);
  bf16x8_t bv = __builtin_bit_cast(bf16x8_t, b);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

// 32x32x2 fp32 MFMA: lane l holds A[m = l%32][k = l/32], B[k = l/32][n = l%32];
// accumulator layout as for mfma32x32x16.
__device__ __forceinline__ f32x16_t mfma32x32x2f32(float a, float b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Token ids outside [0, V) read row 0 instead of faulting.
__device__ __forceinline__ int clamp_id(int id, int V) { return (unsigned)id < (unsigned)V ? id : 0; }

__device__ __forceinline__ int acc_row(int j, int lane) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

// Screening margin of the RVQ kernel for residual width R.  With
// R~ = bf16(R), C~_j = bf16(C_j), eR = ||R - R~|| and e_j = ||C_j - C~_j||
// (bf16 has 8 significant bits, so e_j <= 2^-8 ||C_j||), the screen's score
// s~_j = ||C_j||^2 - 2 R~.C~_j (the squared norm exact after the first
// k-step: three bf16 pieces that sum to it exactly, times ones) satisfies
//   |s~_j - s_j| <= 2 ||R|| e_j + 2 eR (1 + 2^-8) ||C_j||
//                   + ka ||R|| ||C_j|| + k2 ||C_j||^2  =: Delta_j, where
// 2 R.C_j - 2 R~.C~_j = 2 R.(C_j - C~_j) + 2 (R - R~).C~_j gives the first
// two terms (Cauchy-Schwarz, ||C~_j|| <= ||C_j|| + e_j), and
//   ka = (8 R 2^-24            (fp32 accumulation of 2R~.C~, any order,
//                               relative error up to 2 u per addition)
//        + 2^-20 + 2^-12) (1 + 2^-7)  (norm rounding; an index tag in up
//                               to 9 low mantissa bits, which moves a score
//                               by at most 2^-14 of |s~_j| <= ||C_j||^2 +
//                               2.02 ||R|| ||C_j||, doubled; ||R~|| ||C~||
//                               against ||R|| ||C||)
//   k2 = 4 (R + 4) 2^-24 + 2^-13 (accumulation and fp32 rounding of
//                               ||C_j||^2; the index tag, doubled)
// The actual rounding-error norms replace the componentwise worst case
// 2^-8 ||.||: for data they are about 0.4 of it, and the candidate sets
// shrink accordingly.
__host__ __device__ constexpr float rvq_margin_ka(int R) {
  return (8.0f * R / 16777216.0f + 1.0f / 1048576.0f + 1.0f / 4096.0f) * 1.0078125f;
}
__host__ __device__ constexpr float rvq_margin_k2(int R) { return 4.0f * (R + 4) / 16777216.0f + 1.0f / 8192.0f; }

// The screen of the RVQ kernel computes, per codeword, a certified lower bound
// of the exact score s_j = ||C_j||^2 - 2 R . C_j rather than the score itself:
// the norm columns of a codeword row hold (1 - RVQ_K2_SLACK k2) ||C_j||^2
// (three bf16 pieces, exact), ||C_j|| rounded up (two bf16 pieces) and e_j
// rounded up (one piece); the token's operand multiplies them by ones, by -b
// with b = (2 eR (1 + 2^-7) + ka ||R||) RVQ_K1_SLACK and by -c with
// c = 2 ||R|| RVQ_K1_SLACK, each rounded up to bf16, so that the accumulator
// ends at
//   L_j = s~_j - k2' ||C_j||^2 - b ||C_j||' - c e_j'  <=  s_j.
// The subtracted amount is at most RVQ_SUB_FACTOR Delta_j (bf16 rounding up
// of the coefficients and of e_j, 2^-7 each, and the slack), so
// s_j <= L_j + (RVQ_SUB_FACTOR + 1) Delta_j.
constexpr float RVQ_K1_SLACK = 1.0002f * 1.01f;
constexpr float RVQ_K2_SLACK = 1.01f;
constexpr float RVQ_SUB_FACTOR = 1.03f;

// bf16 bit pattern of a non-negative finite float, rounded toward +infinity.
__device__ __forceinline__ uint32_t bf16_up(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b >> 16) + ((b & 0xFFFFu) ? 1u : 0u);
}

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

// ---- LDS access through inline asm
// The pipelined kernels fill LDS with buffer_load ... lds (direct-to-LDS)
// while reading earlier stages.  The compiler cannot prove that an ordinary
// LDS read does not alias a DMA still in flight and drains every
// outstanding DMA (s_waitcnt vmcnt(0)) before it, which serialises the
// pipeline.  Reads issued as inline asm are invisible to that analysis; the
// kernels order them with explicit s_waitcnt vmcnt + barriers (stage ready)
// and lds_wait() (data returned), whose in/out operands keep every use of
// the loaded registers after the wait.
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

template <int OFF = 0>
__device__ __forceinline__ u32x4 lds_read_b128(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset is 16 bits");
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
  return r;
}

template <int OFF = 0>
__device__ __forceinline__ void lds_write_b128(uint32_t addr, u32x4 v) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset is 16 bits");
  asm volatile("ds_write_b128 %0, %1 offset:%2" ::"v"(addr), "v"(v), "i"(OFF) : "memory");
}

// Wait until every LDS access of this wave has completed; the listed
// registers become defined only after the wait.
template <int N>
__device__ __forceinline__ void lds_wait(u32x4 (&v)[N]) {
  static_assert(N >= 1 && N <= 8, "lds_wait takes 1..8 registers per call");
  if constexpr (N == 1) asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0])::"memory");
  if constexpr (N == 2) asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1])::"memory");
  if constexpr (N == 3) asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2])::"memory");
  if constexpr (N == 4)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3])::"memory");
  if constexpr (N == 5)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4])::"memory");
  if constexpr (N == 6)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5])::"memory");
  if constexpr (N == 7)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6])::"memory");
  if constexpr (N == 8)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
                   "+v"(v[7])::"memory");
}

// Wait until every LDS access of this wave has completed; pair with
// reg_pin() on the registers loaded before it.
__device__ __forceinline__ void lds_wait0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Wait until at most N LDS operations of this wave are outstanding; v is
// defined only after the wait.  Valid only while no scalar memory load is in
// flight (those count too and complete out of order); LDS operations
// complete in order, so with the N reads issued after v's among the
// outstanding ones, v has landed.
template <int N>
__device__ __forceinline__ void lds_wait_n(u32x4& v) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt is 4 bits");
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(v) : "n"(N) : "memory");
}

// Pins registers after an earlier lds_wait0() / lds_wait() (no instruction
// emitted): both are volatile asm, so their order is kept, and every later
// use of the registers depends on the pin.
template <int N>
__device__ __forceinline__ void reg_pin(u32x4 (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}

// Chunk swizzle of token-major tiles: chunk c of row t is stored at
// c ^ wg_sw(t, cpr); it stays inside the row for every cpr >= 8.
__device__ __forceinline__ int wg_sw(int row, int cpr) { return (4 * (row & 3)) & (cpr - 1); }

// Transposed fragment read from a token-major LDS tile (rows = tokens,
// `cpr` 16 B chunks per row, swizzled by wg_sw).  ds_read_b64_tr_b16 gives
// lane i of each 16-lane group element (i & 3) of the 8 B read by lane
// 4j + (i >> 2), j = 0..3; pointing lane 4j + q at token t0 + j, columns
// 4q..4q+3 hands lane i column i of tokens t0..t0+3.  Two reads build the
// MFMA fragment: 8 consecutive tokens of column col0 + lane % 32, tokens
// 8 (lane / 32) .. +7 of the 16-token k-step.
//
// The reads are issued as inline asm (a kernel that fills LDS by
// direct-to-LDS loads would otherwise drain all of those first); the caller
// completes them with lds_wait() on the fragments.
__device__ __forceinline__ u32x4 tr_frag(const bf16_t* tile, int cpr, int k0, int col0, int lane) {
  const int g = lane >> 4, sidx = lane & 15, j = sidx >> 2, q = sidx & 3;
  const int col = col0 + 16 * (g & 1) + 4 * q;
  typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
  u32x2 h0, h1;
  {
    const int row = k0 + 8 * (g >> 1) + j;
    const int pc = (col >> 3) ^ wg_sw(row, cpr);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(h0) : "v"(lds_addr(tile + row * cpr * 8 + pc * 8 + (col & 7))) : "memory");
  }
  {
    const int row = k0 + 8 * (g >> 1) + 4 + j;
    const int pc = (col >> 3) ^ wg_sw(row, cpr);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(h1) : "v"(lds_addr(tile + row * cpr * 8 + pc * 8 + (col & 7))) : "memory");
  }
  return u32x4{h0.x, h0.y, h1.x, h1.y};
}

// Compile-time loop: f(std::integral_constant<int, I>) for I = B .. E-1.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

__device__ __forceinline__ uint4 as_uint4(u32x4 v) { return make_uint4(v.x, v.y, v.z, v.w); }
__device__ __forceinline__ u32x4 as_u32x4(uint4 v) { return u32x4{v.x, v.y, v.z, v.w}; }

}  // namespace mapl
