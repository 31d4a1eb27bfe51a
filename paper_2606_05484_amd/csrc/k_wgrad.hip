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

constexpr int WG_BM = 128, WG_KT = 64, WG_THREADS = 256;
constexpr uint32_t WG_OOB = 0x80000000u;

typedef __attribute__((address_space(3))) void* wg_lds_ptr;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short v4s_t;
typedef __attribute__((address_space(3))) v4s_t* lds_v4s_ptr;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t wg_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0x7fffffffull ? 0x7fffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n, 0x00020000);
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
// The reads are issued as inline asm: the compiler cannot tell them apart
// from the direct-to-LDS loads still in flight for later stages and would
// drain all of those first.  The caller completes them with tr_wait(),
// whose in/out operands keep every use of the fragments after the wait;
// stage completion itself is guaranteed by the pipeline's vmcnt + barrier.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

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

template <int BN>
struct WgSmem {
  bf16_t p[WG_KT * WG_BM];
  bf16_t q[WG_KT * BN];
};

// part[s][m][n] = sum_{t in split s} P[t][m] Q[t][n]; P columns < Ma come
// from Pa, columns in [Mao, Mao + Mg) from Pg (Mao = Ma rounded up to a tile).
template <int BN>
__global__ __launch_bounds__(WG_THREADS) void k_wgrad(WgradArgs g, int mtiles, int xcd_map) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature (launch stub)
  constexpr int FM = 2, FN = BN / 64;
  constexpr int PCPR = WG_BM / 8, QCPR = BN / 8;       // 16 B chunks per token row
  constexpr int PBLK = WG_KT * PCPR / 64 / 4;          // 1 KiB DMA blocks per wave per stage
  constexpr int QBLK = WG_KT * QCPR / 64 / 4;
  constexpr int LOADS = PBLK + QBLK;
  __shared__ __attribute__((aligned(1024))) WgSmem<BN> S0;
  __shared__ __attribute__((aligned(1024))) WgSmem<BN> S1;
  __shared__ __attribute__((aligned(1024))) WgSmem<BN> S2;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int G = gridDim.x;
  const int lin = blockIdx.x;
  // workgroups of one token split land on one XCD (dispatch is round-robin
  // over the 8 XCDs), so they share the split's Q rows in that XCD's L2
  const int idx = xcd_map ? (lin % 8) * (G / 8) + lin / 8 : lin;
  const int split = idx / mtiles, mt = idx % mtiles;
  const int Mao = (g.Ma + WG_BM - 1) / WG_BM * WG_BM;
  const int m0 = mt * WG_BM;
  const int n0 = blockIdx.y * BN;
  const int t_begin = split * g.tokens_per_split;
  const int t_end = min(g.T, t_begin + g.tokens_per_split);
  const int KS = t_end > t_begin ? (t_end - t_begin + WG_KT - 1) / WG_KT : 0;
  const int total = (KS + 2) / 3 * 3;
  const bool from_pg = m0 >= Mao;

  // resources cover this split's token rows only (32-bit offsets from there)
  const int nt_rows = t_end > t_begin ? t_end - t_begin : 0;
  const int pld = from_pg ? g.Mg : (int)g.ldp;
  const __amdgpu_buffer_rsrc_t rp = from_pg
      ? wg_rsrc(g.Tg + (int64_t)t_begin * g.Mg, (uint64_t)nt_rows * g.Mg * 2)
      : wg_rsrc(g.Pa + (int64_t)t_begin * g.ldp, (uint64_t)nt_rows * g.ldp * 2);
  const __amdgpu_buffer_rsrc_t rq = wg_rsrc(g.Q + (int64_t)t_begin * g.ldq, (uint64_t)nt_rows * g.ldq * 2);
  const int pcol0 = from_pg ? m0 - Mao : m0;
  const int plim = from_pg ? g.Mg : g.Ma;

  // DMA geometry: lane i of a 1 KiB block writes row b * rows_per_blk + i / cpr,
  // physical chunk i % cpr, holding logical chunk (i % cpr) ^ 4 (row & 3).
  uint32_t p_off[PBLK], q_off[QBLK];
  int p_row[PBLK], q_row[QBLK];
#pragma unroll
  for (int jb = 0; jb < PBLK; ++jb) {
    const int b = wave * PBLK + jb;
    const int row = b * (64 / PCPR) + lane / PCPR;
    const int c = (lane % PCPR) ^ wg_sw(row, PCPR);
    const int col = pcol0 + 8 * c;
    p_row[jb] = row;
    p_off[jb] = (col < plim) ? (uint32_t)col * 2u : WG_OOB;
  }
#pragma unroll
  for (int jb = 0; jb < QBLK; ++jb) {
    const int b = wave * QBLK + jb;
    const int row = b * (64 / QCPR) + lane / QCPR;
    const int c = (lane % QCPR) ^ wg_sw(row, QCPR);
    q_row[jb] = row;
    q_off[jb] = (uint32_t)(n0 + 8 * c) * 2u;
  }

  auto issue = [&](int step, bf16_t* sp, bf16_t* sq) {
    const int t0 = step * WG_KT;  // relative to t_begin
    const bool pad = step >= KS;
#pragma unroll
    for (int jb = 0; jb < PBLK; ++jb) {
      const int t = t0 + p_row[jb];
      const bool ok = !pad && t < nt_rows && p_off[jb] != WG_OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (wg_lds_ptr)(sp + (wave * PBLK + jb) * 512), 16,
                                               ok ? (uint32_t)t * (uint32_t)pld * 2u + p_off[jb] : WG_OOB, 0, 0,
                                               0);
    }
#pragma unroll
    for (int jb = 0; jb < QBLK; ++jb) {
      const int t = t0 + q_row[jb];
      const bool ok = !pad && t < nt_rows;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (wg_lds_ptr)(sq + (wave * QBLK + jb) * 512), 16,
                                               ok ? (uint32_t)t * (uint32_t)g.ldq * 2u + q_off[jb] : WG_OOB, 0,
                                               0, 0);
    }
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  // Fragments double-buffered in registers: the transposed reads of k-step
  // kk + 1 are in flight while the matrix units work on k-step kk.
  u32x4 fa[2][FM], fb[2][FN];
  auto load_frags = [&](const bf16_t* sp, const bf16_t* sq, int kk, u32x4 (&a)[FM], u32x4 (&b)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i) a[i] = tr_frag(sp, PCPR, 16 * kk, wm * 64 + i * 32, lane);
#pragma unroll
    for (int j = 0; j < FN; ++j) b[j] = tr_frag(sq, QCPR, 16 * kk, wn * (BN / 2) + j * 32, lane);
  };
  // complete the asm LDS reads; the in/out operands pin every use after it
  auto wait_frags = [&](u32x4 (&a)[FM], u32x4 (&b)[FN]) {
    if constexpr (FN == 4)
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3])::"memory");
    else if constexpr (FN == 2)
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1])::"memory");
    else
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0])::"memory");
  };
  auto compute = [&](const bf16_t* sp, const bf16_t* sq) {
    load_frags(sp, sq, 0, fa[0], fb[0]);
    wait_frags(fa[0], fb[0]);
#pragma unroll
    for (int kk = 0; kk < WG_KT / 16; ++kk) {
      const int cb = kk & 1, nb = cb ^ 1;
      if (kk + 1 < WG_KT / 16) load_frags(sp, sq, kk + 1, fa[nb], fb[nb]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = mfma32x32x16(__builtin_bit_cast(uint4, fa[cb][i]), __builtin_bit_cast(uint4, fb[cb][j]),
                                   acc[i][j]);
      if (kk + 1 < WG_KT / 16) wait_frags(fa[nb], fb[nb]);
    }
  };

  auto step = [&](int s, const bf16_t* cp, const bf16_t* cq, bf16_t* np, bf16_t* nq) {
    if (s + 1 < total)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    if (s + 2 < total) issue(s + 2, np, nq);
    if (s < KS) compute(cp, cq);
  };

  if (total > 0) {
    issue(0, S0.p, S0.q);
    issue(1, S1.p, S1.q);
  }
  for (int s = 0; s < total; s += 3) {
    step(s, S0.p, S0.q, S2.p, S2.q);
    step(s + 1, S1.p, S1.q, S0.p, S0.q);
    step(s + 2, S2.p, S2.q, S1.p, S1.q);
  }

  const int Mpart = Mao + g.Mg;
  float* out = g.part + (int64_t)split * Mpart * g.N;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * (BN / 2) + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm * 64 + i * 32 + acc_row(e, lane);
        if (m < Mpart) out[(int64_t)m * g.N + n] = acc[i][j][e];
      }
    }
#endif
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
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)M * N) return;
  const int m = (int)(e / N), n = (int)(e % N);
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[s * stride + e];
  dst[(int64_t)n * ldd + off + m] = (bf16_t)f2bf(scale * v);
}

// dU[i][c] (+)= sum_s part[s][i][c] - sum_j B[j][i] Wa[j][c]   (Wa may be null)
// One 64 x 64 tile of dU per block; B (bf16 [k,d]) and Wa (fp32 [k,r]) are
// staged through LDS in 32-row slices.
__global__ __launch_bounds__(256) void k_reduce_dU(const float* __restrict__ part, int splits, int64_t stride,
                                                   int d, int r, float* __restrict__ dU, int accumulate,
                                                   const bf16_t* __restrict__ B, const float* __restrict__ Wa,
                                                   int k) {
  __shared__ float Bs[32][64 + 1];
  __shared__ float Ws[32][64 + 1];
  const int i0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;  // 16 x 16 threads, 4 x 4 outputs each
  float acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = 0.f;
  if (Wa != nullptr) {
    for (int j0 = 0; j0 < k; j0 += 32) {
      for (int e = threadIdx.x; e < 32 * 64; e += 256) {
        const int jj = e / 64, q = e % 64;
        const int j = j0 + jj;
        Bs[jj][q] = (j < k && i0 + q < d) ? bf2f(B[(int64_t)j * d + i0 + q]) : 0.f;
        Ws[jj][q] = (j < k && c0 + q < r) ? Wa[(int64_t)j * r + c0 + q] : 0.f;
      }
      __syncthreads();
#pragma unroll 4
      for (int jj = 0; jj < 32; ++jj) {
        float bv[4], wv[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) bv[a] = Bs[jj][ty * 4 + a];
#pragma unroll
        for (int b = 0; b < 4; ++b) wv[b] = Ws[jj][tx * 4 + b];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = fmaf(bv[a], wv[b], acc[a][b]);
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int i = i0 + ty * 4 + a;
    if (i >= d) continue;
    const int c = c0 + tx * 4;
    if (c >= r) continue;
    const int64_t o = (int64_t)i * r + c;
    float4 v = accumulate ? *(const float4*)(dU + o) : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < splits; ++s) {
      const float4 p = *(const float4*)(part + s * stride + o);
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    v.x -= acc[a][0]; v.y -= acc[a][1]; v.z -= acc[a][2]; v.w -= acc[a][3];
    *(float4*)(dU + o) = v;
  }
}

}  // namespace

hipError_t launch_reduce_splits_t_bf16(const float* part, int splits, int M, int N, int64_t part_stride,
                                       float scale, bf16_t* dst, int64_t ldd, int off, hipStream_t s) {
  const int64_t n = (int64_t)M * N;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce_splits_t_bf16, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, part, splits, M, N,
                     part_stride, scale, dst, ldd, off);
  return hipGetLastError();
}

hipError_t launch_reduce_dU(const float* part, int splits, int64_t part_stride, int d, int r, float* dU,
                            int accumulate, const bf16_t* B, const float* Wa, int k, hipStream_t s) {
  dim3 grid((r + 63) / 64, (d + 63) / 64);
  hipLaunchKernelGGL(k_reduce_dU, grid, dim3(256), 0, s, part, splits, part_stride, d, r, dU, accumulate, B, Wa, k);
  return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& g, hipStream_t s) {
  const int Mao = (g.Ma + WG_BM - 1) / WG_BM * WG_BM;
  const int mtiles = Mao / WG_BM + (g.Mg + WG_BM - 1) / WG_BM;
  if (mtiles <= 0 || g.N <= 0) return hipSuccess;
  if (g.Ma % 8 || g.Mg % 8 || g.ldp % 8 || g.ldq % 8) return hipErrorInvalidValue;
  const int G = mtiles * g.splits;
  const int xcd = G % 8 == 0 ? 1 : 0;
  if (g.N % 256 == 0) {
    hipLaunchKernelGGL(k_wgrad<256>, dim3(G, g.N / 256), dim3(WG_THREADS), 0, s, g, mtiles, xcd);
  } else if (g.N % 128 == 0) {
    hipLaunchKernelGGL(k_wgrad<128>, dim3(G, g.N / 128), dim3(WG_THREADS), 0, s, g, mtiles, xcd);
  } else if (g.N % 64 == 0) {
    hipLaunchKernelGGL(k_wgrad<64>, dim3(G, g.N / 64), dim3(WG_THREADS), 0, s, g, mtiles, xcd);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int wgrad_row_offset(int Ma) { return (Ma + WG_BM - 1) / WG_BM * WG_BM; }

hipError_t launch_reduce_splits(const float* part, int splits, int M, int N, int64_t part_stride,
                                float* dst, int accumulate, hipStream_t s) {
  const int64_t n4 = (int64_t)M * N / 4;
  if (n4 == 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce_splits, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, part, splits,
                     n4, part_stride, dst, accumulate);
  return hipGetLastError();
}

}  // namespace mapl
