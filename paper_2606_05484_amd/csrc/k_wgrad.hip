// Projector gradient: dU-type products that contract over tokens,
//   part[s](m,n) = sum_{t in split s} P[t,m] Q[t,n],
// with P = dXhat (receiver, Eq. 2 backward) or [X | a_s] (sender, Eq. 1
// backward; the anchor columns come from the gathered copy of A_s[ids]).
// Both operands are token-major in HBM, i.e. K-strided for the matrix units:
// 64-token stages of both are copied as they are (16 B chunks, XOR-swizzled
// per row) into LDS by direct-to-LDS loads, and the matrix units' fragments
// are read transposed with ds_read_b64_tr_b16 (see tr_frag).  Splits over
// tokens fill the chip; a second kernel sums the splits in a fixed order, so
// results are bitwise reproducible.
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

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar LDS addresses
  const int wm = wave >> 1, wn = wave & 1;
  // Workgroup ids are dispatched round-robin over the 8 XCDs (id % 8).  The
  // k-th workgroup of XCD x takes work item x q' + k (q' = its share), so
  // every XCD owns a contiguous run of (split, m-tile, n-tile) items and the
  // workgroups of a token split share its Q rows in one L2.
  const int NY = gridDim.y;
  const int Gt = gridDim.x * NY;
  const int lin = blockIdx.x + blockIdx.y * gridDim.x;
  int item = lin;
  if (xcd_map) {
    const int xcd = lin % 8, k = lin / 8, q = Gt / 8, rem = Gt % 8;
    item = xcd < rem ? xcd * (q + 1) + k : rem * (q + 1) + (xcd - rem) * q + k;
  }
  const int ny = item % NY, idx = item / NY;
  const int split = idx / mtiles, mt = idx % mtiles;
  const int Mao = (g.Ma + WG_BM - 1) / WG_BM * WG_BM;
  const int m0 = mt * WG_BM;
  const int n0 = ny * BN;
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

  // lane part of each load's offset (row within the step, column chunk);
  // a step adds its first token's row offset, uniform across the wave
  uint32_t p_lane[PBLK], q_lane[QBLK];
#pragma unroll
  for (int jb = 0; jb < PBLK; ++jb)
    p_lane[jb] = p_off[jb] != WG_OOB ? (uint32_t)p_row[jb] * (uint32_t)pld * 2u + p_off[jb] : WG_OOB;
#pragma unroll
  for (int jb = 0; jb < QBLK; ++jb) q_lane[jb] = (uint32_t)q_row[jb] * (uint32_t)g.ldq * 2u + q_off[jb];

  // A real step issues exactly LOADS loads per wave, a padding step none
  // (the wait before a step accounts for that).  The next step's loads are
  // issued a few at a time between the products (see compute): a burst of
  // them would hold up the wave's instruction stream.  A step whose 64
  // tokens all exist takes the lane's fixed offset as the VGPR operand and
  // the step's row offset as the scalar one (no vector arithmetic); the last
  // step of a ragged split checks each lane's token.
  struct Plan {
    bf16_t *sp, *sq;
    int t0;
    bool live, full;
  };
  auto plan = [&](int step, bf16_t* sp, bf16_t* sq) {
    Plan p;
    p.sp = sp;
    p.sq = sq;
    p.t0 = __builtin_amdgcn_readfirstlane(step * WG_KT);  // relative to t_begin
    p.live = p.t0 < KS * WG_KT;
    p.full = p.t0 + WG_KT <= nt_rows;
    return p;
  };
  auto issue_range = [&](const Plan& p, auto b0c, auto b1c) {
    constexpr int B0 = decltype(b0c)::value, B1 = decltype(b1c)::value;
    if (!p.live) return;
    const int sP = (int)((uint32_t)p.t0 * (uint32_t)pld * 2u), sQ = (int)((uint32_t)p.t0 * (uint32_t)g.ldq * 2u);
    if (p.full) {
      static_for<B0, B1>([&](auto lic) {
        constexpr int LI = decltype(lic)::value;
        if constexpr (LI < PBLK)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (wg_lds_ptr)(p.sp + (wave * PBLK + LI) * 512), 16, p_lane[LI],
                                                   sP, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (wg_lds_ptr)(p.sq + (wave * QBLK + LI - PBLK) * 512), 16,
                                                   q_lane[LI - PBLK], sQ, 0, 0);
      });
    } else {
      static_for<B0, B1>([&](auto lic) {
        constexpr int LI = decltype(lic)::value;
        if constexpr (LI < PBLK) {
          const int t = p.t0 + p_row[LI];
          const bool ok = t < nt_rows && p_off[LI] != WG_OOB;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (wg_lds_ptr)(p.sp + (wave * PBLK + LI) * 512), 16,
                                                   ok ? (uint32_t)t * (uint32_t)pld * 2u + p_off[LI] : WG_OOB, 0, 0, 0);
        } else {
          constexpr int J = LI - PBLK;
          const int t = p.t0 + q_row[J];
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (wg_lds_ptr)(p.sq + (wave * QBLK + J) * 512), 16,
                                                   t < nt_rows ? (uint32_t)t * (uint32_t)g.ldq * 2u + q_off[J] : WG_OOB,
                                                   0, 0, 0);
        }
      });
    }
  };
  auto issue = [&](int step, bf16_t* sp, bf16_t* sq) {
    issue_range(plan(step, sp, sq), std::integral_constant<int, 0>{}, std::integral_constant<int, LOADS>{});
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
  constexpr int KSTEP = WG_KT / 16, PER = (LOADS + KSTEP - 1) / KSTEP;
  auto compute = [&](const bf16_t* sp, const bf16_t* sq, const Plan& nx) {
    load_frags(sp, sq, 0, fa[0], fb[0]);
    wait_frags(fa[0], fb[0]);
    static_for<0, KSTEP>([&](auto kkc) {
      constexpr int KK = decltype(kkc)::value, CB = KK & 1, NB = CB ^ 1;
      if constexpr (KK + 1 < KSTEP) load_frags(sp, sq, KK + 1, fa[NB], fb[NB]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = mfma32x32x16(__builtin_bit_cast(uint4, fa[CB][i]), __builtin_bit_cast(uint4, fb[CB][j]),
                                   acc[i][j]);
      constexpr int B0 = KK * PER < LOADS ? KK * PER : LOADS;
      constexpr int B1 = (KK + 1) * PER < LOADS ? (KK + 1) * PER : LOADS;
      issue_range(nx, std::integral_constant<int, B0>{}, std::integral_constant<int, B1>{});
      if constexpr (KK + 1 < KSTEP) wait_frags(fa[NB], fb[NB]);
    });
  };

  auto step = [&](int s, const bf16_t* cp, const bf16_t* cq, bf16_t* np, bf16_t* nq) {
    // step s must be complete; only step s + 1 (if it loads) may be in flight
    if (s + 1 < KS)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    const Plan nx = plan(s + 2, np, nq);  // not live past KS
    if (s < KS)
      compute(cp, cq, nx);
    else
      issue_range(nx, std::integral_constant<int, 0>{}, std::integral_constant<int, LOADS>{});
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

// dst (+)= sum_s part[s], the splits added in order; the loads of up to
// eight splits are in flight together.
__global__ void k_reduce_splits(const float* __restrict__ part, int splits, int64_t n4,
                                int64_t stride, float* __restrict__ dst, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 v = accumulate ? ((const float4*)dst)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  constexpr int B = 8;
  for (int s0 = 0; s0 < splits; s0 += B) {
    float4 p[B];
#pragma unroll
    for (int u = 0; u < B; ++u)
      if (s0 + u < splits) p[u] = ((const float4*)(part + (s0 + u) * stride))[i];
#pragma unroll
    for (int u = 0; u < B; ++u)
      if (s0 + u < splits) {
        v.x += p[u].x; v.y += p[u].y; v.z += p[u].z; v.w += p[u].w;
      }
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

// dU (+)= sum_s part[s][i][c] - sum_j B[j][i] Wa[j][c]: the split-K reduction
// of the weight gradient fused with the ambient-anchor correction
// -B_s^T (a_s^T dZ) of the encoder backward.  B is bf16 [k, d], Wa fp32
// [k, r] (already reduced).  A workgroup owns 32 rows x 64 columns of dU;
// thread (ty, tx) owns row ty and columns 8tx .. 8tx+7.  All loads of a
// chunk are issued before any LDS store so their latencies overlap.
constexpr int RD_I = 32, RD_C = 64, RD_KC = 128;

__global__ __launch_bounds__(256) void k_reduce_dU(const float* __restrict__ part, int splits, int64_t stride,
                                                   int d, int r, float* __restrict__ dU, int accumulate,
                                                   const bf16_t* __restrict__ B, const float* __restrict__ Wa,
                                                   int k) {
  __shared__ float Bs[RD_KC][RD_I + 1];
  __shared__ __attribute__((aligned(16))) float Ws[RD_KC][RD_C];
  const int i0 = blockIdx.y * RD_I, c0 = blockIdx.x * RD_C;
  const int tid = threadIdx.x, ty = tid >> 3, tx = tid & 7;
  const int i = i0 + ty, c = c0 + 8 * tx;
  const bool own = i < d && c < r;  // r % 32 == 0: c < r implies c + 7 < r
  const int64_t o = (int64_t)i * r + c;
  float v[8];
  if (own && accumulate) {
    const float4 p0 = *(const float4*)(dU + o), p1 = *(const float4*)(dU + o + 4);
    v[0] = p0.x; v[1] = p0.y; v[2] = p0.z; v[3] = p0.w; v[4] = p1.x; v[5] = p1.y; v[6] = p1.z; v[7] = p1.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = 0.f;
  }
  if (own) {
    // the splits added in order, the loads of up to eight in flight together
    constexpr int B = 8;
    for (int s = 0; s < splits; s += B) {
      float4 q[2 * B];
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (s + u < splits) {
          q[2 * u] = *(const float4*)(part + (s + u) * stride + o);
          q[2 * u + 1] = *(const float4*)(part + (s + u) * stride + o + 4);
        }
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (s + u < splits) {
          v[0] += q[2 * u].x; v[1] += q[2 * u].y; v[2] += q[2 * u].z; v[3] += q[2 * u].w;
          v[4] += q[2 * u + 1].x; v[5] += q[2 * u + 1].y; v[6] += q[2 * u + 1].z; v[7] += q[2 * u + 1].w;
        }
    }
  }
  if (Wa != nullptr && k > 0) {
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int j0 = 0; j0 < k; j0 += RD_KC) {
      const int kc = min(RD_KC, k - j0);
      // B rows j0.., columns i0 .. i0+31: 4 x 16 B per row, 2 per thread;
      // Wa rows j0.., columns c0 .. c0+63: 16 float4 per row, 8 per thread
      uint4 bq[2];
      float4 wq[8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int e = tid + 256 * u, jj = e >> 2, q = (e & 3) * 8;
        bq[u] = jj < kc ? *(const uint4*)(B + (int64_t)(j0 + jj) * d + i0 + q) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = tid + 256 * u, jj = e >> 4, q = (e & 15) * 4;
        wq[u] = (jj < kc && c0 + q < r) ? *(const float4*)(Wa + (int64_t)(j0 + jj) * r + c0 + q)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      __syncthreads();  // the previous chunk's readers are done
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int e = tid + 256 * u, jj = e >> 2, q = (e & 3) * 8;
        const uint32_t w4[4] = {bq[u].x, bq[u].y, bq[u].z, bq[u].w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          Bs[jj][q + 2 * h] = bf2f(w4[h] & 0xFFFFu);
          Bs[jj][q + 2 * h + 1] = bf2f(w4[h] >> 16);
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = tid + 256 * u, jj = e >> 4, q = (e & 15) * 4;
        *(float4*)&Ws[jj][q] = wq[u];
      }
      __syncthreads();
      for (int jj = 0; jj < kc; ++jj) {
        const float b = Bs[jj][ty];
        const float4 w0 = *(const float4*)&Ws[jj][8 * tx], w1 = *(const float4*)&Ws[jj][8 * tx + 4];
        acc[0] = fmaf(b, w0.x, acc[0]); acc[1] = fmaf(b, w0.y, acc[1]);
        acc[2] = fmaf(b, w0.z, acc[2]); acc[3] = fmaf(b, w0.w, acc[3]);
        acc[4] = fmaf(b, w1.x, acc[4]); acc[5] = fmaf(b, w1.y, acc[5]);
        acc[6] = fmaf(b, w1.z, acc[6]); acc[7] = fmaf(b, w1.w, acc[7]);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] -= acc[e];
  }
  if (own) {
    *(float4*)(dU + o) = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(dU + o + 4) = make_float4(v[4], v[5], v[6], v[7]);
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
  if (d % RD_I || r % 32 || (uintptr_t)B % 16) return hipErrorInvalidValue;
  dim3 grid((r + RD_C - 1) / RD_C, d / RD_I);
  hipLaunchKernelGGL(k_reduce_dU, grid, dim3(256), 0, s, part, splits, part_stride, d, r, dU, accumulate, B, Wa, k);
  return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& g, hipStream_t s) {
  const int Mao = (g.Ma + WG_BM - 1) / WG_BM * WG_BM;
  const int mtiles = Mao / WG_BM + (g.Mg + WG_BM - 1) / WG_BM;
  if (mtiles <= 0 || g.N <= 0) return hipSuccess;
  if (g.Ma % 8 || g.Mg % 8 || g.ldp % 8 || g.ldq % 8) return hipErrorInvalidValue;
  const int G = mtiles * g.splits;
  const int xcd = 1;
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
