// Projector gradient: dU-type products that contract over tokens,
//   part[s](m,n) = sum_{t in split s} P[t,m] Q[t,n],
// with P = dXhat (receiver, Eq. 2 backward) or [X | a_s] (sender, Eq. 1
// backward; the anchor columns a_s = A_s[ids] are gathered in flight).  Both
// operands are token-major in HBM, i.e. K-strided for the matrix units, so
// each thread loads an 8 token x 8 column block with 16 B row loads,
// transposes it in registers and writes 8 K-contiguous 16 B rows to LDS
// under an XOR swizzle of the 16 B chunks (conflict-free writes and
// fragment reads).  Splits over tokens fill the chip; a second kernel sums
// the splits in a fixed order, so results are bitwise reproducible.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int WG_BM = 128, WG_BK = 64, WG_LDK = WG_BK + 8, WG_THREADS = 256;

__device__ __forceinline__ void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
  // in[t] = 8 bf16 of token t (columns 0..7); out[c] = 8 bf16 of column c
  // (tokens 0..7).
  const uint32_t* x = reinterpret_cast<const uint32_t*>(in);
  uint32_t* y = reinterpret_cast<uint32_t*>(out);
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t a = x[(2 * w) * 4 + (c >> 1)], b = x[(2 * w + 1) * 4 + (c >> 1)];
      y[c * 4 + w] = (c & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
    }
}

template <int BN>
__global__ __launch_bounds__(WG_THREADS) void k_wgrad(WgradArgs g) {
  constexpr int FN = BN / 64;  // 2 x 2 waves; wave tile 64 x (BN/2)
  constexpr int QBLK = (BN / 8) * (WG_BK / 8);
  __shared__ __attribute__((aligned(16))) bf16_t Ps[2][WG_BM][WG_LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Qs[2][BN][WG_LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.x * WG_BM, n0 = blockIdx.y * BN;
  const int Mtot = g.Ma + g.Mg;
  const int t_begin = blockIdx.z * g.tokens_per_split;
  const int t_end = min(g.T, t_begin + g.tokens_per_split);

  // loader role: P block (tid < 128) or Q block (tid >= 128)
  const bool isP = tid < 128;
  const int bidx = isP ? tid : tid - 128;
  const int tb = bidx / (isP ? 16 : BN / 8), cb = bidx % (isP ? 16 : BN / 8);
  const bool active = isP || bidx < QBLK;
  uint4 rows[8];

  auto load = [&](int t0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) rows[i] = make_uint4(0, 0, 0, 0);
    if (!active) return;
    const int col = (isP ? m0 : n0) + 8 * cb;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int t = t0 + 8 * tb + i;
      if (t < t_end) {
        if (!isP) {
          rows[i] = *(const uint4*)(g.Q + (int64_t)t * g.ldq + col);
        } else if (col < g.Ma) {
          rows[i] = *(const uint4*)(g.Pa + (int64_t)t * g.ldp + col);
        } else if (col < Mtot) {
          rows[i] = *(const uint4*)(g.Tg + (int64_t)clamp_id(g.ids[t], g.V) * g.ldt + (col - g.Ma));
        }
      }
    }
  };
  auto store = [&](int buf) {
    if (!active) return;
    uint4 cols[8];
    transpose8x8(rows, cols);
    const int pc = 8 * (tb ^ (cb & 7));
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      if (isP)
        *(uint4*)&Ps[buf][8 * cb + c][pc] = cols[c];
      else
        *(uint4*)&Qs[buf][8 * cb + c][pc] = cols[c];
    }
  };

  f32x16_t acc[2][FN];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  const int nsteps = t_end > t_begin ? (t_end - t_begin + WG_BK - 1) / WG_BK : 0;
  if (nsteps > 0) {
    load(t_begin);
    store(0);
  }
  __syncthreads();
  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1;
    if (s + 1 < nsteps) load(t_begin + (s + 1) * WG_BK);
#pragma unroll
    for (int kk = 0; kk < WG_BK / 16; ++kk) {
      const int chunk = 2 * kk + (lane >> 5);
      uint4 af[2], bfr[FN];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int m = wm * 64 + i * 32 + (lane & 31);
        af[i] = *(const uint4*)&Ps[buf][m][8 * (chunk ^ ((m >> 3) & 7))];
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int n = wn * (BN / 2) + j * 32 + (lane & 31);
        bfr[j] = *(const uint4*)&Qs[buf][n][8 * (chunk ^ ((n >> 3) & 7))];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32x32x16(af[i], bfr[j], acc[i][j]);
    }
    if (s + 1 < nsteps) store(buf ^ 1);
    __syncthreads();
  }

  float* out = g.part + (int64_t)blockIdx.z * Mtot * g.N;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * (BN / 2) + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm * 64 + i * 32 + acc_row(e, lane);
        if (m < Mtot) out[(int64_t)m * g.N + n] = acc[i][j][e];
      }
    }
}

__global__ void k_reduce_splits(const float* __restrict__ part, int splits, int64_t n4,
                                int64_t stride, float* __restrict__ dst, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 v = accumulate ? ((const float4*)dst)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < splits; ++s) {
    float4 p = ((const float4*)(part + s * stride))[i];
    v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
  }
  ((float4*)dst)[i] = v;
}

__global__ void k_reduce_splits_t_bf16(const float* __restrict__ part, int splits, int M, int N,
                                       int64_t stride, float scale, bf16_t* __restrict__ dst, int64_t ldd,
                                       int off) {
  __shared__ float tile[32][33];
  const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) {
    const int m = m0 + y, n = n0 + tx;
    float v = 0.f;
    if (m < M && n < N)
      for (int s = 0; s < splits; ++s) v += part[s * stride + (int64_t)m * N + n];
    tile[y][tx] = v;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int n = n0 + y, m = m0 + tx;
    if (n < N && m < M) dst[(int64_t)n * ldd + off + m] = (bf16_t)f2bf(scale * tile[tx][y]);
  }
}

}  // namespace

hipError_t launch_reduce_splits_t_bf16(const float* part, int splits, int M, int N, int64_t part_stride,
                                       float scale, bf16_t* dst, int64_t ldd, int off, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + 31) / 32, (M + 31) / 32);
  hipLaunchKernelGGL(k_reduce_splits_t_bf16, grid, dim3(256), 0, s, part, splits, M, N, part_stride, scale, dst,
                     ldd, off);
  return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& g, hipStream_t s) {
  const int Mtot = g.Ma + g.Mg;
  if (Mtot <= 0 || g.N <= 0) return hipSuccess;
  if (g.N % 128 == 0) {
    dim3 grid((Mtot + WG_BM - 1) / WG_BM, g.N / 128, g.splits);
    hipLaunchKernelGGL(k_wgrad<128>, grid, dim3(WG_THREADS), 0, s, g);
  } else if (g.N % 64 == 0) {
    dim3 grid((Mtot + WG_BM - 1) / WG_BM, g.N / 64, g.splits);
    hipLaunchKernelGGL(k_wgrad<64>, grid, dim3(WG_THREADS), 0, s, g);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_reduce_splits(const float* part, int splits, int M, int N, int64_t part_stride,
                                float* dst, int accumulate, hipStream_t s) {
  const int64_t n4 = (int64_t)M * N / 4;
  if (n4 == 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce_splits, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, part, splits,
                     n4, part_stride, dst, accumulate);
  return hipGetLastError();
}

}  // namespace mapl
