// Batched strided GEMM on the fp32 matrix units (v_mfma_f32_32x32x2_f32):
//   C[b](m,n) = alpha_b * sum_k A[b](m,k) B[b](k,n) + beta_b * Cin[b](m,n)
// with alpha_b = alpha * (alpha_ptr ? alpha_ptr[b] : 1), likewise beta.
// Operands may be fp32 or bf16 (widened exactly to fp32 in LDS); any
// element strides, so transposed operands need no copies.  This kernel
// carries every product of the Stiefel step and the fp32 codec path.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int GF_BM = 128, GF_BN = 128, GF_BK = 16, GF_PAD = 1;
constexpr int GF_THREADS = 256;

template <typename T>
__device__ __forceinline__ float ld_elem(const T* p);
template <>
__device__ __forceinline__ float ld_elem<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld_elem<bf16_t>(const bf16_t* p) { return bf2f(*p); }

// Load a [BM x BK] tile of op(A) (element (m,k) at A + m*sm + k*sk) into
// LDS as s[k][m].  Consecutive threads walk the operand's unit-stride index.
template <typename T, int ROWS>
__device__ __forceinline__ void load_tile(float (*s)[ROWS + GF_PAD], const T* A, int64_t sm, int64_t sk,
                                          int m0, int k0, int M, int K, int tid) {
  constexpr int N = ROWS * GF_BK;
  if (sk == 1) {
#pragma unroll 4
    for (int e = tid; e < N; e += GF_THREADS) {
      int m = e / GF_BK, k = e % GF_BK;
      int gm = m0 + m, gk = k0 + k;
      s[k][m] = (gm < M && gk < K) ? ld_elem<T>(A + gm * sm + gk) : 0.f;
    }
  } else {
#pragma unroll 4
    for (int e = tid; e < N; e += GF_THREADS) {
      int k = e / ROWS, m = e % ROWS;
      int gm = m0 + m, gk = k0 + k;
      s[k][m] = (gm < M && gk < K) ? ld_elem<T>(A + gm * sm + (int64_t)gk * sk) : 0.f;
    }
  }
}

template <typename TA, typename TB, typename TO>
__global__ __launch_bounds__(GF_THREADS) void k_gemm_f32(GemmF32Args g) {
  __shared__ float As[GF_BK][GF_BM + GF_PAD];
  __shared__ float Bs[GF_BK][GF_BN + GF_PAD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves, 64 x 64 each
  const int b = blockIdx.z;
  const int m0 = blockIdx.x * GF_BM, n0 = blockIdx.y * GF_BN;
  const TA* A = (const TA*)g.A + b * g.sAb;
  const TB* B = (const TB*)g.B + b * g.sBb;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  for (int k0 = 0; k0 < g.K; k0 += GF_BK) {
    load_tile<TA, GF_BM>(As, A, g.sAm, g.sAk, m0, k0, g.M, g.K, tid);
    // B is addressed as element (k,n) at B + k*sBk + n*sBn; load it as the
    // tile of B^T (rows n, cols k).
    load_tile<TB, GF_BN>(Bs, B, g.sBn, g.sBk, n0, k0, g.N, g.K, tid);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GF_BK; kk += 2) {
      float a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[kk + (lane >> 5)][wm * 64 + i * 32 + (lane & 31)];
#pragma unroll
      for (int j = 0; j < 2; ++j) bb[j] = Bs[kk + (lane >> 5)][wn * 64 + j * 32 + (lane & 31)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x2f32(a[i], bb[j], acc[i][j]);
    }
    __syncthreads();
  }

  const float alpha = g.alpha * (g.alpha_ptr ? g.alpha_ptr[b] : 1.f);
  const float beta = g.beta * (g.beta_ptr ? g.beta_ptr[b] : 1.f);
  const float* Cin = g.Cin ? g.Cin + b * g.sCinb : nullptr;
  TO* C = (TO*)g.C + b * g.sCb;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        int m = m0 + wm * 64 + i * 32 + acc_row(e, lane);
        int n = n0 + wn * 64 + j * 32 + (lane & 31);
        if (m < g.M && n < g.N) {
          float v = alpha * acc[i][j][e];
          if (Cin && beta != 0.f) v += beta * Cin[m * g.sCinm + n * g.sCinn];
          if constexpr (sizeof(TO) == 4)
            C[m * g.sCm + n * g.sCn] = v;
          else
            C[m * g.sCm + n * g.sCn] = (TO)f2bf(v);
        }
      }
}

}  // namespace

hipError_t launch_gemm_f32(const GemmF32Args& g, int ta, int tb, int to, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return hipSuccess;
  dim3 grid((g.M + GF_BM - 1) / GF_BM, (g.N + GF_BN - 1) / GF_BN, g.batch);
  dim3 block(GF_THREADS);
#define MAPL_GF(TA_, TB_, TO_) hipLaunchKernelGGL((k_gemm_f32<TA_, TB_, TO_>), grid, block, 0, s, g)
  if (ta == 0 && tb == 0 && to == 0) MAPL_GF(float, float, float);
  else if (ta == 1 && tb == 0 && to == 0) MAPL_GF(bf16_t, float, float);
  else if (ta == 0 && tb == 1 && to == 0) MAPL_GF(float, bf16_t, float);
  else if (ta == 1 && tb == 1 && to == 0) MAPL_GF(bf16_t, bf16_t, float);
  else if (ta == 1 && tb == 1 && to == 1) MAPL_GF(bf16_t, bf16_t, bf16_t);
  else if (ta == 0 && tb == 0 && to == 1) MAPL_GF(float, float, bf16_t);
  else if (ta == 1 && tb == 0 && to == 1) MAPL_GF(bf16_t, float, bf16_t);
  else if (ta == 0 && tb == 1 && to == 1) MAPL_GF(float, bf16_t, bf16_t);
  else return hipErrorInvalidValue;
#undef MAPL_GF
  return hipGetLastError();
}

}  // namespace mapl
