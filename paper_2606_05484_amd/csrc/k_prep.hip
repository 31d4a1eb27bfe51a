// Per-call operand preparation and the receiver-side operand assembly.
//   prep_u          U (fp32 master) -> bf16 copies in both K-contiguous
//                   layouts the matrix units need (U~ [d,r] and U~^T [r,d])
//   transpose_into  scaled transposed copies (anchor companions into the
//                   concatenated weight operands)
//   prep_codebook   bf16 screening copy of the codebooks plus fp32 norms
//   assemble        [Zhat | a_r] rows for the lift: Zhat is the payload or
//                   the RVQ gather-sum sum_l C_l[code_l] (Sec. 3.5), a_r the
//                   receiver's anchor row (Eq. 2)
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

// 32x32 tiles through LDS so both the read of U and the write of U^T are
// coalesced.
__global__ void k_prep_u(const float* __restrict__ U, int d, int r, bf16_t* __restrict__ Ub,
                         int64_t ldub, bf16_t* __restrict__ Ut, int64_t ldut) {
  __shared__ bf16_t tile[32][33];
  const int j0 = blockIdx.x * 32, c0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int y = ty; y < 32; y += 8) {
    const int j = j0 + y, c = c0 + tx;
    bf16_t v = 0;
    if (j < d && c < r) v = (bf16_t)f2bf(U[(int64_t)j * r + c]);
    tile[y][tx] = v;
    if (Ub && j < d && c < ldub) Ub[(int64_t)j * ldub + c] = (c < r) ? v : (bf16_t)0;
  }
  __syncthreads();
  if (Ut) {
    for (int y = ty; y < 32; y += 8) {
      const int c = c0 + y, j = j0 + tx;
      if (c < r && j < ldut) Ut[(int64_t)c * ldut + j] = (j < d) ? tile[tx][y] : (bf16_t)0;
    }
  }
}

__global__ void k_transpose_into(const void* __restrict__ src, int src_f32, int rows, int cols,
                                 int64_t lds, float scale, bf16_t* __restrict__ dst, int64_t ldd,
                                 int off) {
  __shared__ float tile[32][33];
  const int i0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) {
    const int i = i0 + y, j = j0 + tx;
    float v = 0.f;
    if (i < rows && j < cols)
      v = src_f32 ? ((const float*)src)[(int64_t)i * lds + j] : bf2f(((const bf16_t*)src)[(int64_t)i * lds + j]);
    tile[y][tx] = v;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int j = j0 + y, i = i0 + tx;
    if (j < cols && i < rows) dst[(int64_t)j * ldd + off + i] = (bf16_t)f2bf(scale * tile[tx][y]);
  }
}

// One wave per codeword: bf16 copy and fp32 norms.
__global__ void k_prep_codebook(const float* __restrict__ C, int LK, int r, bf16_t* __restrict__ Cb,
                                float* __restrict__ cn2, float* __restrict__ cnrm) {
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (w >= LK) return;
  const float* row = C + (int64_t)w * r;
  float s = 0.f;
  for (int c = lane; c < r; c += 64) {
    const float v = row[c];
    s += v * v;
    Cb[(int64_t)w * r + c] = (bf16_t)f2bf(v);
  }
  s = wave_sum(s);
  if (lane == 0) {
    cn2[w] = s;
    cnrm[w] = sqrtf(s);
  }
}

// One wave per token row.
__global__ void k_assemble(AssembleArgs a) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (t >= a.T) return;
  bf16_t* out = a.out + (int64_t)t * a.ldo;
  const int id = (a.A != nullptr) ? clamp_id(a.ids[t], a.V) : 0;
  for (int c = lane; c < a.r; c += 64) {
    float v;
    if (a.L == 0) {
      v = bf2f(a.Zp[(int64_t)t * a.r + c]);
    } else {
      v = 0.f;
      for (int l = 0; l < a.L; ++l) {
        int code = a.code_bytes == 1 ? ((const uint8_t*)a.codes)[(int64_t)t * a.L + l]
                                     : ((const uint16_t*)a.codes)[(int64_t)t * a.L + l];
        code = code < a.K ? code : a.K - 1;
        v += a.C[((int64_t)l * a.K + code) * a.r + c];
      }
    }
    if (a.Bc != nullptr) {
      const bf16_t* arow = a.A + (int64_t)id * a.k;
      for (int i = 0; i < a.k; ++i) v += bf2f(arow[i]) * bf2f(a.Bc[(int64_t)i * a.r + c]);
    }
    out[c] = (bf16_t)f2bf(v);
  }
  int col = a.r;
  if (a.A != nullptr && a.Bc == nullptr) {
    const bf16_t* arow = a.A + (int64_t)id * a.k;
    for (int i = lane; i < a.k; i += 64) out[a.r + i] = arow[i];
    col += a.k;
  }
  for (int c = col + lane; c < a.ldo; c += 64) out[c] = 0;
}

__global__ void k_check_ids(const int32_t* __restrict__ ids, int T, int64_t V, int* flag) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < T && (ids[t] < 0 || (int64_t)ids[t] >= V)) atomicOr(flag, 1);
}

__global__ void k_zero_bytes(uint32_t* p, int64_t words) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < words) p[i] = 0;
}

}  // namespace

hipError_t launch_prep_u(const float* U, int d, int r, bf16_t* Ub, int64_t ldub, bf16_t* Ut,
                         int64_t ldut, hipStream_t s) {
  const int cols = (int)((Ub && ldub > r) ? ldub : r);
  const int rows = (int)((Ut && ldut > d) ? ldut : d);
  dim3 grid((rows + 31) / 32, (cols + 31) / 32);
  hipLaunchKernelGGL(k_prep_u, grid, dim3(256), 0, s, U, d, r, Ub, ldub, Ut, ldut);
  return hipGetLastError();
}

hipError_t launch_transpose_into(const void* src, int src_f32, int rows, int cols, int64_t lds,
                                 float scale, bf16_t* dst, int64_t ldd, int off, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  dim3 grid((cols + 31) / 32, (rows + 31) / 32);
  hipLaunchKernelGGL(k_transpose_into, grid, dim3(256), 0, s, src, src_f32, rows, cols, lds, scale, dst,
                     ldd, off);
  return hipGetLastError();
}

hipError_t launch_prep_codebook(const float* C, int L, int K, int r, bf16_t* Cb, float* cn2, float* cnrm,
                                hipStream_t s) {
  const int LK = L * K;
  if (LK <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_prep_codebook, dim3((LK + 3) / 4), dim3(256), 0, s, C, LK, r, Cb, cn2, cnrm);
  return hipGetLastError();
}

hipError_t launch_assemble(const AssembleArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_assemble, dim3((a.T + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_check_ids(const int32_t* ids, int T, int64_t V, int* flag, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_check_ids, dim3((T + 255) / 256), dim3(256), 0, s, ids, T, V, flag);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(void* p, int64_t bytes, hipStream_t s) {
  const int64_t words = bytes / 4;
  if (words <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero_bytes, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, s, (uint32_t*)p,
                     words);
  return hipGetLastError();
}

}  // namespace mapl
