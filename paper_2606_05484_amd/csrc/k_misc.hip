// Small kernels: the fp32 codec path (gathers, exact fp32 RVQ, codebook
// sums) and the elementwise / reduction steps of the SPEL update
// (Sec. 3.3: Eq. 4 symmetrisation, Eq. 5 momentum, the normalisations that
// precede the two PolarExpress iterations of Eqs. 6-7).
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

__global__ void k_gather_rows_f32(const float* __restrict__ A, int k, const int32_t* __restrict__ ids,
                                  int V, int T, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)T * k) return;
  const int t = (int)(i / k), c = (int)(i % k);
  out[i] = A[(int64_t)clamp_id(ids[t], V) * k + c];
}

// One wave per token: residual in registers/LDS, exact fp32 squared
// distances sum_c (R_c - C_jc)^2 for every codeword, lowest index on ties.
__global__ void k_rvq_f32(const float* __restrict__ Z0, const float* __restrict__ C, int T, int r, int L,
                          int K, void* codes, int code_bytes) {
  extern __shared__ float sh[];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  if (t >= T) return;
  float* R = sh + wave * r;
  for (int c = lane; c < r; c += 64) R[c] = Z0[(int64_t)t * r + c];
  __builtin_amdgcn_wave_barrier();
  for (int l = 0; l < L; ++l) {
    const float* Cl = C + (int64_t)l * K * r;
    float best = INFINITY;
    int bj = 0x7fffffff;
    for (int j = lane; j < K; j += 64) {
      float s = 0.f;
      for (int c = 0; c < r; ++c) {
        const float df = R[c] - Cl[(int64_t)j * r + c];
        s = fmaf(df, df, s);
      }
      if (s < best) { best = s; bj = j; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o, WAVE);
      const int oj = __shfl_xor(bj, o, WAVE);
      if (ob < best || (ob == best && oj < bj)) { best = ob; bj = oj; }
    }
    if (bj >= K) bj = 0;  // only reachable with non-finite inputs
    if (lane == 0) {
      if (code_bytes == 1)
        ((uint8_t*)codes)[(int64_t)t * L + l] = (uint8_t)bj;
      else
        ((uint16_t*)codes)[(int64_t)t * L + l] = (uint16_t)bj;
    }
    __builtin_amdgcn_wave_barrier();
    for (int c = lane; c < r; c += 64) R[c] -= Cl[(int64_t)bj * r + c];
    __builtin_amdgcn_wave_barrier();
  }
}

// gdim 2: grouped codes [T, L, r/2] (u8), column c takes group c / 2's code.
__global__ void k_codes_sum_f32(const void* __restrict__ codes, int code_bytes, const float* __restrict__ C,
                                int T, int r, int L, int K, int gdim, float* __restrict__ Zhat) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)T * r) return;
  const int t = (int)(i / r), c = (int)(i % r);
  float v = 0.f;
  for (int l = 0; l < L; ++l) {
    int code = gdim == 2 ? ((const uint8_t*)codes)[((int64_t)t * L + l) * (r / 2) + c / 2]
               : code_bytes == 1 ? ((const uint8_t*)codes)[(int64_t)t * L + l]
                                 : ((const uint16_t*)codes)[(int64_t)t * L + l];
    code = code < K ? code : K - 1;
    v += C[((int64_t)l * K + code) * r + c];
  }
  Zhat[i] = v;
}

__global__ void k_copy_f32(const float* __restrict__ src, float* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

// S <- (S + S^T) / 2 per projector: one block per pair of 32 x 32 tiles
// (ta, tb), ta <= tb (row by row), both read and written in rows through LDS;
// element (a, b) and its mirror get the same 0.5 (S[a][b] + S[b][a]).
__global__ __launch_bounds__(256) void k_symmetrize(float* S, int r) {
  __shared__ float A[32][33], B[32][33];
  float* Sp = S + (int64_t)blockIdx.y * r * r;
  const int nt = (r + 31) / 32;
  int t = blockIdx.x, ta = 0;
  while (t >= nt - ta) {
    t -= nt - ta;
    ++ta;
  }
  const int tb = ta + t;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 8 rows of 32 per pass
  const int a0 = 32 * ta, b0 = 32 * tb;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = ty + 8 * u;
    A[i][tx] = (a0 + i < r && b0 + tx < r) ? Sp[(int64_t)(a0 + i) * r + b0 + tx] : 0.f;
    B[i][tx] = (b0 + i < r && a0 + tx < r) ? Sp[(int64_t)(b0 + i) * r + a0 + tx] : 0.f;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = ty + 8 * u;
    if (a0 + i < r && b0 + tx < r) Sp[(int64_t)(a0 + i) * r + b0 + tx] = 0.5f * (A[i][tx] + B[tx][i]);
    if (ta != tb && b0 + i < r && a0 + tx < r) Sp[(int64_t)(b0 + i) * r + a0 + tx] = 0.5f * (A[tx][i] + B[i][tx]);
  }
}

// grid (nblk, P): block-stride loop, one partial sum of M^2 per block.
// M <- beta M + (1 - beta) gR; per-block partial sums of M^2 (partial[p][b])
// and of G^2 (partial[P + p][b]: the gradient's norm for the zero rule).
__global__ void k_momentum(float* __restrict__ M, const float* __restrict__ gR, const float* __restrict__ G,
                           int64_t n, float beta, float* __restrict__ partial) {
  __shared__ float red[2][4];
  const int p = blockIdx.y;
  float* Mp = M + (int64_t)p * n;
  const float* gp = gR + (int64_t)p * n;
  const float* Gp = G + (int64_t)p * n;
  float s = 0.f, sg = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float v = beta * Mp[i] + (1.f - beta) * gp[i];
    Mp[i] = v;
    s = fmaf(v, v, s);
    const float gv = Gp[i];
    sg = fmaf(gv, gv, sg);
  }
  s = wave_sum(s);
  sg = wave_sum(sg);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = s;
    red[1][threadIdx.x >> 6] = sg;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t nb = gridDim.x, P = gridDim.y;
    partial[(int64_t)p * nb + blockIdx.x] = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    partial[(P + p) * nb + blockIdx.x] = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  }
}

// LMO normalisation of Eq. 6: scale = 1 / (||M||_F + eps), or 0 (so the LMO
// returns D = 0) when ||M||_F <= zero_rel ||G||_F: a momentum below the fp32
// resolution of the gradient carries no direction.
__global__ void k_fro_scale(const float* __restrict__ partial, int nblk, int P, float eps, float zero_rel,
                            float* scale) {
  const int p = blockIdx.x, lane = threadIdx.x;
  float s = 0.f, sg = 0.f;
  for (int i = lane; i < nblk; i += 64) {
    s += partial[(int64_t)p * nblk + i];
    sg += partial[(int64_t)(P + p) * nblk + i];
  }
  s = wave_sum(s);
  sg = wave_sum(sg);
  if (lane == 0) {
    const float nm = sqrtf(s);
    const float sc = nm <= zero_rel * sqrtf(sg) ? 0.f : 1.f / (nm + eps);
    scale[p] = sc;
  }
}

// nu2 = max_i sum_j |S_ij| per projector, in two launches: blocks of four
// waves take 16 rows each (a wave 4 rows, every load of the four rows issued
// before the sums: one round of loads per wave) and write their row maximum;
// one thread per projector then takes the maximum over its blocks.  r <= 1024.
__global__ __launch_bounds__(256) void k_inf_norm_partial(const float* __restrict__ S, int r,
                                                          float* __restrict__ part) {
  __shared__ float red[4];
  constexpr int RB = 4, QMAX = 16;
  const int p = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* Sp = S + (int64_t)p * r * r;
  const int nq = (r + 63) / 64;
  float m = 0.f;
  for (int i0 = blockIdx.x * 16 + wave * RB; i0 < min(r, blockIdx.x * 16 + wave * RB + RB); i0 += RB) {
    float v[RB][QMAX];
#pragma unroll
    for (int u = 0; u < RB; ++u)
#pragma unroll
      for (int q = 0; q < QMAX; ++q) {
        const int i = i0 + u, c = lane + 64 * q;
        v[u][q] = (q < nq && i < r && c < r) ? Sp[(int64_t)i * r + c] : 0.f;
      }
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      float sum = 0.f;
#pragma unroll
      for (int q = 0; q < QMAX; ++q) sum += fabsf(v[u][q]);
      m = fmaxf(m, wave_sum(sum));
    }
  }
  if (lane == 0) red[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0)
    part[(int64_t)p * gridDim.x + blockIdx.x] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__global__ void k_inf_norm_final(const float* __restrict__ part, int nb, int P, float* inv_nu, float* inv_nu2) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= P) return;
  float nu2 = 0.f;
  for (int j = 0; j < nb; ++j) nu2 = fmaxf(nu2, part[(int64_t)p * nb + j]);
  const float in2 = 1.f / nu2;
  inv_nu2[p] = in2;
  inv_nu[p] = sqrtf(in2);
}

// Streaming codebook synchronisation (Sec. 3.5): one wave per transmitted
// codeword row, 16-byte accesses across the row.  pack: buf[l][i] =
// C[l][rows[l][i]]; unpack: C[l][rows[l][i]] = buf[l][i].  Rows outside
// [0, K) are skipped (pack writes zeros for them).
__global__ void k_codebook_pack(const float* __restrict__ C, const int32_t* __restrict__ rows, int K, int r, int n,
                                float* __restrict__ buf) {
  const int i = blockIdx.x, l = blockIdx.y, lane = threadIdx.x;
  const int row = rows[(int64_t)l * n + i];
  const bool ok = (unsigned)row < (unsigned)K;
  const float4* src = (const float4*)(C + ((int64_t)l * K + (ok ? row : 0)) * r);
  float4* dst = (float4*)(buf + ((int64_t)l * n + i) * r);
  for (int c = lane; c < r / 4; c += 64) dst[c] = ok ? src[c] : make_float4(0.f, 0.f, 0.f, 0.f);
}

__global__ void k_codebook_unpack(const float* __restrict__ buf, const int32_t* __restrict__ rows, int K, int r,
                                  int n, float* __restrict__ C) {
  const int i = blockIdx.x, l = blockIdx.y, lane = threadIdx.x;
  const int row = rows[(int64_t)l * n + i];
  if ((unsigned)row >= (unsigned)K) return;
  const float4* src = (const float4*)(buf + ((int64_t)l * n + i) * r);
  float4* dst = (float4*)(C + ((int64_t)l * K + row) * r);
  for (int c = lane; c < r / 4; c += 64) dst[c] = src[c];
}

}  // namespace

hipError_t launch_gather_rows_f32(const float* A, int k, const int32_t* ids, int V, int T, float* out,
                                  hipStream_t s) {
  const int64_t n = (int64_t)T * k;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, A, k, ids, V, T, out);
  return hipGetLastError();
}

hipError_t launch_rvq_f32(const float* Z0, const float* C, int T, int r, int L, int K, void* codes,
                          int code_bytes, hipStream_t s) {
  if (T <= 0 || L <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_rvq_f32, dim3((T + 3) / 4), dim3(256), 4 * r * sizeof(float), s, Z0, C, T, r, L, K,
                     codes, code_bytes);
  return hipGetLastError();
}

hipError_t launch_codes_sum_f32(const void* codes, int code_bytes, const float* C, int T, int r, int L, int K,
                                float* Zhat, hipStream_t s, int gdim) {
  const int64_t n = (int64_t)T * r;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_codes_sum_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, codes, code_bytes, C,
                     T, r, L, K, gdim, Zhat);
  return hipGetLastError();
}

hipError_t launch_copy_f32(const float* src, float* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_symmetrize(float* S, int P, int r, hipStream_t s) {
  const int nt = (r + 31) / 32;
  hipLaunchKernelGGL(k_symmetrize, dim3((unsigned)(nt * (nt + 1) / 2), P), dim3(256), 0, s, S, r);
  return hipGetLastError();
}

hipError_t launch_momentum(float* M, const float* gR, const float* G, int64_t n, int P, float beta, float* partial,
                           int nblk, hipStream_t s) {
  hipLaunchKernelGGL(k_momentum, dim3(nblk, P), dim3(256), 0, s, M, gR, G, n, beta, partial);
  return hipGetLastError();
}

hipError_t launch_fro_scale(const float* partial, int nblk, int P, float eps, float zero_rel, float* scale,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_fro_scale, dim3(P), dim3(64), 0, s, partial, nblk, P, eps, zero_rel, scale);
  return hipGetLastError();
}

hipError_t launch_inf_norm_scales(const float* S, int P, int r, float* part, float* inv_nu, float* inv_nu2,
                                  hipStream_t s) {
  if (r > 1024) return hipErrorInvalidValue;
  const int nb = (r + 15) / 16;  // 16 rows per block, 4 per wave
  hipLaunchKernelGGL(k_inf_norm_partial, dim3(nb, P), dim3(256), 0, s, S, r, part);
  hipLaunchKernelGGL(k_inf_norm_final, dim3((P + 255) / 256), dim3(256), 0, s, part, nb, P, inv_nu, inv_nu2);
  return hipGetLastError();
}

hipError_t launch_codebook_pack(const float* C, const int32_t* rows, int L, int K, int r, int n, float* buf,
                                hipStream_t s) {
  if (n <= 0 || L <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_codebook_pack, dim3(n, L), dim3(64), 0, s, C, rows, K, r, n, buf);
  return hipGetLastError();
}

hipError_t launch_codebook_unpack(const float* buf, const int32_t* rows, int L, int K, int r, int n, float* C,
                                  hipStream_t s) {
  if (n <= 0 || L <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_codebook_unpack, dim3(n, L), dim3(64), 0, s, buf, rows, K, r, n, C);
  return hipGetLastError();
}

}  // namespace mapl
