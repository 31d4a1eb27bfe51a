// Grouped residual vector quantisation (Sec. 3.5, the coordinates
// decomposed into groups; App. E: group dimension 2, K = 256, R = 2): each
// token's r coordinates form r / 2 independent two-dimensional residuals,
// and group g is quantised round after round over the 2-D codewords
// C[l][j][2g : 2g + 2], the nearest by exact fp32 squared distance, the
// lowest index among equals.
//
// Layout: one lane per (token, group) query.  A workgroup owns GW
// consecutive groups (their 2 GW columns of every codebook round staged in
// LDS, group-major, so a wave reads each codeword as one broadcast) and a
// block of 256 tokens; wave w takes GW / 4 of the groups for 64 tokens at a
// time.  The codes of a wave's groups for one (token, round) are
// consecutive bytes of the [T, L, r/2] code array and leave as one store.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int GQ_THREADS = 256, GQ_TOK = 128, GQ_KMAX = 256, GQ_LDS_FLOATS = 16384;  // 64 KiB at most

template <int GPW>  // groups per wave, searched side by side (independent chains)
__global__ __launch_bounds__(GQ_THREADS) void k_grvq(const float* __restrict__ Z0, const float* __restrict__ C,
                                                     int T, int r, int L, int K, uint8_t* __restrict__ codes) {
  extern __shared__ float cb[];  // [L][GW][K][2]
  constexpr int GW = 4 * GPW;
  const int G = r / 2;
  const int g0 = blockIdx.y * GW;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // stage the workgroup's codebook columns: row (l, j) holds 2 GW floats
  for (int e = tid; e < L * K * GW; e += GQ_THREADS) {
    const int gi = e % GW, lj = e / GW, l = lj / K, j = lj % K;
    const float2 v = *(const float2*)(C + ((int64_t)l * K + j) * r + 2 * (g0 + gi));
    *(float2*)(cb + (((int64_t)l * GW + gi) * K + j) * 2) = v;
  }
  __syncthreads();
  for (int t0 = blockIdx.x * GQ_TOK; t0 < min(T, (blockIdx.x + 1) * GQ_TOK); t0 += 64) {
    const int t = t0 + lane;
    const bool valid = t < T;
    uint32_t word[8];  // codes of this wave's groups, per round (GPW <= 4 bytes each)
#pragma unroll
    for (int l = 0; l < 8; ++l) word[l] = 0;
    float2 R[GPW];
#pragma unroll
    for (int q = 0; q < GPW; ++q)
      R[q] = valid ? *(const float2*)(Z0 + (int64_t)t * r + 2 * (g0 + wave * GPW + q)) : make_float2(0.f, 0.f);
    for (int l = 0; l < L; ++l) {
      const float* cl[GPW];
      float best[GPW];
      int bj[GPW];
#pragma unroll
      for (int q = 0; q < GPW; ++q) {
        cl[q] = cb + ((int64_t)l * GW + wave * GPW + q) * K * 2;
        best[q] = INFINITY;
        bj[q] = 0;
      }
      for (int j = 0; j < K; j += 2) {
#pragma unroll
        for (int q = 0; q < GPW; ++q) {
          const float4 c2 = *(const float4*)(cl[q] + 2 * j);  // codewords j, j + 1 (broadcast)
          float dx = R[q].x - c2.x, dy = R[q].y - c2.y;
          float dd = fmaf(dy, dy, dx * dx);
          if (dd < best[q]) { best[q] = dd; bj[q] = j; }
          dx = R[q].x - c2.z;
          dy = R[q].y - c2.w;
          dd = fmaf(dy, dy, dx * dx);
          if (dd < best[q]) { best[q] = dd; bj[q] = j + 1; }
        }
      }
#pragma unroll
      for (int q = 0; q < GPW; ++q) {
        const float2 w = *(const float2*)(cl[q] + 2 * bj[q]);
        R[q].x -= w.x;
        R[q].y -= w.y;
#pragma unroll
        for (int ll = 0; ll < 8; ++ll)
          if (ll == l) word[ll] |= (uint32_t)bj[q] << (8 * q);
      }
    }
    if (valid) {
      uint8_t* crow = codes + (int64_t)t * L * G + g0 + wave * GPW;
#pragma unroll
      for (int l = 0; l < 8; ++l) {
        if (l < L) {
          if constexpr (GPW == 4) *(uint32_t*)(crow + (int64_t)l * G) = word[l];
          else if constexpr (GPW == 2) *(uint16_t*)(crow + (int64_t)l * G) = (uint16_t)word[l];
          else crow[(int64_t)l * G] = (uint8_t)word[l];
        }
      }
    }
  }
}

}  // namespace

// Groups per workgroup so that L rounds of K two-float codewords fit the LDS.
static int grvq_groups_per_wg(int L, int K, int G) {
  for (int gw = 8; gw >= 4; gw /= 2)
    if ((int64_t)L * K * gw * 2 <= GQ_LDS_FLOATS && G % gw == 0) return gw;
  return 0;
}

hipError_t launch_grvq(const float* Z0, const float* C, int T, int r, int L, int K, uint8_t* codes, hipStream_t s) {
  if (T <= 0 || L <= 0) return hipSuccess;
  const int G = r / 2;
  if (r % 8 || K > GQ_KMAX || K % 2 || L > 8) return hipErrorInvalidValue;
  const int gw = grvq_groups_per_wg(L, K, G);
  if (gw == 0) return hipErrorInvalidValue;
  dim3 grid((T + GQ_TOK - 1) / GQ_TOK, G / gw);
  const size_t lds = (size_t)L * K * gw * 2 * sizeof(float);
  switch (gw / 4) {
    case 4: hipLaunchKernelGGL(k_grvq<4>, grid, dim3(GQ_THREADS), lds, s, Z0, C, T, r, L, K, codes); break;
    case 2: hipLaunchKernelGGL(k_grvq<2>, grid, dim3(GQ_THREADS), lds, s, Z0, C, T, r, L, K, codes); break;
    default: hipLaunchKernelGGL(k_grvq<1>, grid, dim3(GQ_THREADS), lds, s, Z0, C, T, r, L, K, codes); break;
  }
  return hipGetLastError();
}

bool grvq_supported(int r, int L, int K) { return r % 8 == 0 && K <= GQ_KMAX && K % 2 == 0 && L >= 1 && L <= 8 &&
                                                  grvq_groups_per_wg(L, K, r / 2) > 0; }

}  // namespace mapl
