// Token-major bf16 GEMM on the bf16 matrix units (v_mfma_f32_32x32x16_bf16):
//
//   out[t, n] = sum_{c < Ka} A[t, c] W[n, c]  +  sum_{i < Kg} T[ids[t], i] W[n, Ka + i]
//
// A [M, lda] and W [N, ldw] are both K-contiguous bf16; the optional second
// sum gathers anchor rows T[ids[t]] (bf16, [V, ldt]) -- the token-id lookup of
// Eqs. 1-2 -- straight into the K loop, so the anchored operand [X | a] is
// never materialised.  fp32 accumulation; the epilogue stores bf16 (RNE) or
// fp32.  One kernel serves the four dense products of the codec:
//   encode      Z0   = [X | a_s] [U~ ; -(B_s U~)]        (N = r)
//   decode_bwd  dZ   = dXhat U~                          (N = r)
//   decode      Xhat = [Zhat | a_r] [U~^T ; B_r]         (N = d)
//   encode_bwd  dX   = dZ U~^T                           (N = d)
// Tiles: BM tokens x BN outputs per workgroup of 4 waves (WM x WN), K staged
// through LDS 32 at a time, double-buffered, with a register prefetch of
// the next stage while the matrix units work on the current one.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int TB_BK = 32;
constexpr int TB_LDK = TB_BK + 8;  // +16 B per row: conflict-free 16 B fragment reads
constexpr int TB_THREADS = 256;

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(TB_THREADS) void k_gemm_tn(TnArgs g) {
  static_assert(WM * WN == 4, "4 waves");
  constexpr int FM = BM / (32 * WM), FN = BN / (32 * WN);
  static_assert(FM >= 1 && FN >= 1, "tile");
  constexpr int ACH = BM * TB_BK / 8 / TB_THREADS;  // 16 B chunks per thread
  constexpr int BCH = BN * TB_BK / 8 / TB_THREADS;
  constexpr int ACH1 = ACH > 0 ? ACH : 1;
  constexpr int BCH1 = BCH > 0 ? BCH : 1;

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][TB_LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Ws[2][BN][TB_LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int ka_steps = g.Ka / TB_BK;
  const int kg_steps = (g.Kg + TB_BK - 1) / TB_BK;
  const int nsteps = ka_steps + kg_steps;

  uint4 ra[ACH1], rw[BCH1];

  auto load_stage = [&](int s) {
    const bool gathered = s >= ka_steps;
    const int kc = gathered ? (s - ka_steps) * TB_BK : s * TB_BK;
#pragma unroll
    for (int i = 0; i < ACH1; ++i) {
      int c = tid + i * TB_THREADS;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (ACH > 0 || c < BM * TB_BK / 8) {
        int row = c >> 2, col = (c & 3) * 8;
        int t = m0 + row;
        if (t < g.M) {
          if (!gathered) {
            v = *(const uint4*)(g.A + (int64_t)t * g.lda + kc + col);
          } else if (kc + col < g.Kg) {
            int id = clamp_id(g.ids[t], g.V);
            v = *(const uint4*)(g.T + (int64_t)id * g.ldt + kc + col);
          }
        }
      }
      ra[i] = v;
    }
    const int kw = s * TB_BK;
#pragma unroll
    for (int i = 0; i < BCH1; ++i) {
      int c = tid + i * TB_THREADS;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (BCH > 0 || c < BN * TB_BK / 8) {
        int row = c >> 2, col = (c & 3) * 8;
        v = *(const uint4*)(g.W + (int64_t)(n0 + row) * g.ldw + kw + col);
      }
      rw[i] = v;
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH1; ++i) {
      int c = tid + i * TB_THREADS;
      if (ACH > 0 || c < BM * TB_BK / 8) *(uint4*)&As[buf][c >> 2][(c & 3) * 8] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH1; ++i) {
      int c = tid + i * TB_THREADS;
      if (BCH > 0 || c < BN * TB_BK / 8) *(uint4*)&Ws[buf][c >> 2][(c & 3) * 8] = rw[i];
    }
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  if (nsteps > 0) {
    load_stage(0);
    store_stage(0);
  }
  __syncthreads();
  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1;
    if (s + 1 < nsteps) load_stage(s + 1);
#pragma unroll
    for (int kk = 0; kk < TB_BK; kk += 16) {
      uint4 af[FM], wf[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *(const uint4*)&As[buf][wm * (BM / WM) + i * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
#pragma unroll
      for (int j = 0; j < FN; ++j)
        wf[j] = *(const uint4*)&Ws[buf][wn * (BN / WN) + j * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32x32x16(af[i], wf[j], acc[i][j]);
    }
    if (s + 1 < nsteps) store_stage(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds column n = lane%32 of each 32x32 fragment.
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * (BN / WN) + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = m0 + wm * (BM / WM) + i * 32 + acc_row(e, lane);
        if (t < g.M) {
          float v = acc[i][j][e];
          if (g.out_f32)
            ((float*)g.out)[(int64_t)t * g.ldo + n] = v;
          else
            ((bf16_t*)g.out)[(int64_t)t * g.ldo + n] = (bf16_t)f2bf(v);
        }
      }
    }
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_tn(const TnArgs& g, hipStream_t s) {
  dim3 grid((g.M + BM - 1) / BM, g.N / BN);
  hipLaunchKernelGGL((k_gemm_tn<BM, BN, WM, WN>), grid, dim3(TB_THREADS), 0, s, g);
  return hipGetLastError();
}

}  // namespace

// Tile choice: cover N with as few column tiles as possible (each A row is
// then streamed from HBM once) and shrink BM when the token count alone
// would leave compute units idle.
hipError_t launch_gemm_tn(const TnArgs& g, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  const int BN = g.N % 256 == 0 ? 256 : g.N % 128 == 0 ? 128 : g.N % 64 == 0 ? 64 : g.N % 32 == 0 ? 32 : 0;
  if (BN == 0) return hipErrorInvalidValue;
  const bool small = (int64_t)((g.M + 127) / 128) * (g.N / BN) < 256;
  switch (BN) {
    case 256: return small ? launch_tn<64, 256, 2, 2>(g, s) : launch_tn<128, 256, 2, 2>(g, s);
    case 128: return small ? launch_tn<64, 128, 2, 2>(g, s) : launch_tn<128, 128, 2, 2>(g, s);
    case 64: return small ? launch_tn<64, 64, 2, 2>(g, s) : launch_tn<128, 64, 2, 2>(g, s);
    default: return launch_tn<128, 32, 4, 1>(g, s);
  }
}

}  // namespace mapl
