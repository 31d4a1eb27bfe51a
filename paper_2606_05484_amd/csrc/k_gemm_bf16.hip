// Token-major bf16 GEMM on the bf16 matrix units (v_mfma_f32_32x32x16_bf16):
//
//   out[t, n] = sum_{c < Ka} A[t, c] W[n, c]  +  sum_{i < Kg} T[ids[t], i] W[n, Ka + i]
//
// A [M, lda] and W [N, ldw] are both K-contiguous bf16; the optional second
// sum gathers anchor rows T[ids[t]] (bf16, [V, ldt]) -- the token-id lookup of
// Eqs. 1-2 -- straight into the K loop, so the anchored operand [X | a] is
// never materialised.  fp32 accumulation; the epilogue stores bf16 (RNE) or
// fp32 (optionally accumulating).  One kernel serves the dense products of
// the codec:
//   encode      Z0   = [X | a_s] [U~ ; -(B_s U~)]        (N = r)
//   decode_bwd  dZ   = dXhat U~                          (N = r)
//   decode      Xhat = [Zhat | a_r] [U~^T ; B_r]         (N = d)
//   encode_bwd  dX   = dZ U~^T                           (N = d)
// and, with split-K over grid z, the small per-call operand products.
//
// Pipeline: a workgroup of 4 waves owns BM = 128 tokens and walks a run of
// BN-wide output tiles; K is staged 64 at a time through three LDS stages
// filled by buffer_load ... lds (direct-to-LDS, no register staging), two
// stages in flight while the matrix units consume the third.  Each stage
// lives in its own __shared__ array so the compiler's wait counting stays
// per-stage.  LDS rows are 128 B with the 16 B chunks XOR-swizzled by
// ((row >> 1) & 7): 16 consecutive rows reading one logical chunk then hit
// 16 distinct 16 B bank groups of the 64-bank LDS (rows alternate between
// the two halves of the bank space), and the lane-linear DMA writes are
// conflict-free by construction.  The matrix units are fed W as the first
// operand and the tokens as the second, so each lane ends up holding four
// consecutive output columns of one token: fp32 results leave as 16 B
// stores, bf16 results are paired across lane halves (v_permlane32_swap) into
// 16 B row segments and staged through LDS into full 128 B row writes.  Buffer resources bound every
// operand: lanes past the last token row, past Kg or past ldw read zeros.
#include "tn_gemm.hpp"

namespace mapl {

namespace {

// NS pipeline stages (2 or 3), one __shared__ array each.
template <int BN, int NS, bool FULLK>
__global__ __launch_bounds__(GTHREADS) void k_gemm_tn(TnArgs g, int ntiles_per_wg) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature (launch stub)
  __shared__ __attribute__((aligned(1024))) TnSmem<BN> S0;
  __shared__ __attribute__((aligned(1024))) TnSmem<BN> S1;
  // third stage (NS == 3 only; a token array otherwise)
  __shared__ __attribute__((aligned(1024))) bf16_t S2buf[NS == 3 ? (GM + BN) * GK : 8];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m0 = blockIdx.x * GM, nt0 = blockIdx.y * ntiles_per_wg;
  char* obase = (char*)g.out + (g.kz > 0 ? (int64_t)blockIdx.z * g.out_z * 4 : 0);
  tn_mainloop<BN, NS, FULLK>(g, ntiles_per_wg, S0.a, S0.w, S1.a, S1.w, S2buf, S2buf + GM * GK,
                             [&](f32x16_t (&acc)[2][BN / 64], int tile) {
                               // epilogue, staging bf16 results through the buffer consumed by the
                               // tile's last step (no DMA targets it before the next tile's first step)
                               if (!g.out_f32) __builtin_amdgcn_s_barrier();  // every wave is done reading it
                               tn_epilogue<BN, (GM + BN) * GK * 2>(acc, g, obase, m0, nt0 + tile,
                                                                  lds_addr(NS == 3 ? S2buf : S1.a), wave, lane);
                             });
#endif
}

// Short-K, write-heavy products with bf16 output (decode: K = r + k,
// encode_bwd: K = r; N = d), walked over many output tiles per 128-token
// block: 128 x 128 tiles, each of the 4 waves owning 32 token rows and all
// 128 columns.  A wave loads the token fragments of its rows for the whole
// K (up to 6 stages) once, straight from memory into registers in the
// matrix unit's operand layout (16 B per lane and fragment: token row
// l % 32, k 8 (l / 32) .. +7 of a 16-wide k-step; anchor rows gathered by
// id), so the token operand uses no LDS; W streams through a three-deep
// ring of 16 KiB stages.  48 KiB of LDS and at most 216 registers per lane
// let two workgroups share a CU, so one's output stores overlap the
// other's products.  Epilogue: as tn_epilogue, for 32-row waves.
template <int KS>
__global__ __launch_bounds__(GTHREADS, 2) void k_gemm_tn_short(TnArgs g, int ntiles_per_wg) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int BN = 128, NSW = 3, FN = BN / 32, KSTEP = GK / 16, KST = KS * KSTEP;
  constexpr int WBLK = BN / 8 / 4;  // W: 1 KiB blocks per wave per stage
  __shared__ __attribute__((aligned(1024))) bf16_t SW[NSW][BN * GK];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m0 = blockIdx.x * GM;
  const int nt0 = blockIdx.y * ntiles_per_wg;
  const int ntiles = min(ntiles_per_wg, g.N / BN - nt0);
  const int total = ntiles * KS;

  const int mrows = min(GM, g.M - m0);
  const __amdgpu_buffer_rsrc_t ra = rsrc(g.A + (int64_t)m0 * g.lda, (uint64_t)(mrows > 0 ? mrows : 0) * g.lda * 2);
  const __amdgpu_buffer_rsrc_t rt = rsrc(g.T, g.T ? (uint64_t)g.V * g.ldt * 2 : 0);
  const __amdgpu_buffer_rsrc_t rw = rsrc(g.W, (uint64_t)g.N * g.ldw * 2);

  // token fragments of rows 32 wave .. +31; rows past the last token read zeros
  u32x4 afr[KST];
  {
    const int row = wave * 32 + (lane & 31);
    const bool in = m0 + row < g.M;
    const uint32_t ch = 16u * (uint32_t)(lane >> 5);
    const uint32_t aoff = in ? (uint32_t)row * (uint32_t)g.lda * 2u + ch : OOB;
    const uint32_t toff =
        in && g.Kg > 0 ? (uint32_t)clamp_id(g.ids[m0 + row], g.V) * (uint32_t)g.ldt * 2u + ch : OOB;
#pragma unroll
    for (int q = 0; q < KST; ++q) {
      const int kc = q * 16;
      if (kc < g.Ka)
        afr[q] = __builtin_amdgcn_raw_buffer_load_b128(ra, aoff, kc * 2, 0);
      else
        afr[q] = __builtin_amdgcn_raw_buffer_load_b128(rt, toff, (kc - g.Ka) * 2, 0);
    }
  }

  const int lrow = lane >> 3;
  const uint32_t lchp[2] = {(uint32_t)((lane & 7) ^ (lane >> 4)), (uint32_t)((lane & 7) ^ (4 + (lane >> 4)))};
  uint32_t w_off[WBLK];
#pragma unroll
  for (int j = 0; j < WBLK; ++j) {
    const int row = 8 * (wave * WBLK + j) + lrow;
    w_off[j] = (uint32_t)row * (uint32_t)g.ldw * 2u + 16u * lchp[j & 1];
  }
  int pl_ks = 0, pl_nt = nt0, pl_s = 0;
  struct WPlan {
    bf16_t* sw;
    int soff;
    bool live;
  };
  auto plan_next = [&](bf16_t* sw) {
    WPlan p;
    p.sw = sw;
    const int ks = __builtin_amdgcn_readfirstlane(pl_ks), nt = __builtin_amdgcn_readfirstlane(pl_nt);
    p.live = __builtin_amdgcn_readfirstlane(pl_s) < total;
    ++pl_s;
    if (++pl_ks == KS) {
      pl_ks = 0;
      ++pl_nt;
    }
    p.soff = (int)((uint32_t)nt * BN * (uint32_t)g.ldw * 2u + (uint32_t)(ks * GK) * 2u);
    return p;
  };
  auto issue_range = [&](const WPlan& p, auto b0c, auto b1c) {
    if (!p.live) return;
    static_for<decltype(b0c)::value, decltype(b1c)::value>([&](auto jc) {
      constexpr int J = decltype(jc)::value;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(p.sw + (wave * WBLK + J) * 512), 16, w_off[J], p.soff, 0,
                                               0);
    });
  };

  f32x16_t acc[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) acc[j] = f32x16_t{};
  uint32_t koff[KSTEP];
#pragma unroll
  for (int kk = 0; kk < KSTEP; ++kk) koff[kk] = tn_koff(kk, lane);
  constexpr int PER = (WBLK + KSTEP - 1) / KSTEP;
  constexpr uint32_t WSTG = BN * GK * 2;
  const uint32_t swb = lds_addr(&SW[0][0]);
  auto wbuf = [&](int u) { return (bf16_t*)&SW[0][0] + u * (BN * GK); };

  issue_range(plan_next(wbuf(0)), std::integral_constant<int, 0>{}, std::integral_constant<int, WBLK>{});
  issue_range(plan_next(wbuf(1)), std::integral_constant<int, 0>{}, std::integral_constant<int, WBLK>{});
  // wait for the token fragments here, not inside the tile loop
#pragma unroll
  for (int q = 0; q < KST; ++q) asm volatile("" : "+v"(afr[q]));

  int s = 0, u = 0;
  for (int tile = 0; tile < ntiles; ++tile) {
    static_for<0, KS>([&](auto ksc) {
      constexpr int KSI = decltype(ksc)::value;
      if (s + 1 < total)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(WBLK) : "memory");
      else
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __builtin_amdgcn_s_barrier();
      const int un = u == 0 ? NSW - 1 : u - 1;
      const WPlan nx = plan_next(wbuf(un));
      const uint32_t bw = swb + u * WSTG;
      u32x4 fr[2][FN];
      auto load = [&](int kk, u32x4 (&f)[FN]) {
        static_for<0, FN>([&](auto jc) {
          constexpr int J = decltype(jc)::value;
          f[J] = lds_read_b128<J * 32 * GK * 2>(bw + koff[kk]);
        });
      };
      load(0, fr[0]);
      lds_wait(fr[0]);
      static_for<0, KSTEP>([&](auto kkc) {
        constexpr int KK = decltype(kkc)::value, CB = KK & 1;
        if constexpr (KK + 1 < KSTEP) load(KK + 1, fr[CB ^ 1]);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[j] = mfma32x32x16(as_uint4(fr[CB][j]), as_uint4(afr[KSI * KSTEP + KK]), acc[j]);
        constexpr int B0 = KK * PER < WBLK ? KK * PER : WBLK;
        constexpr int B1 = (KK + 1) * PER < WBLK ? (KK + 1) * PER : WBLK;
        issue_range(nx, std::integral_constant<int, B0>{}, std::integral_constant<int, B1>{});
        if constexpr (KK + 1 < KSTEP) lds_wait(fr[CB ^ 1]);
      });
      ++s;
      if (KSI + 1 < KS) u = u + 1 == NSW ? 0 : u + 1;
    });

    // epilogue through the W buffer the tile's last step consumed: per half
    // of the columns, each wave stages its 32 x 64 block (4 KiB) and stores
    // full 128 B row segments
    __builtin_amdgcn_s_barrier();  // every wave is done reading it
    {
      constexpr int COLS = 64, CPR = COLS / 8;
      const int half = lane >> 5;
      const uint32_t stg = swb + u * WSTG + wave * (32 * COLS * 2);
      const int nt = nt0 + tile;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const f32x16_t& c = acc[h * 2 + jj];
          uint32_t p[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) p[e] = pack_bf2(c[2 * e], c[2 * e + 1]);
#pragma unroll
          for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int w = 0; w < 2; ++w) {
              const auto sw2 = __builtin_amdgcn_permlane32_swap(p[4 * q + w], p[4 * q + 2 + w], false, false);
              p[4 * q + w] = sw2[0];
              p[4 * q + 2 + w] = sw2[1];
            }
          const int row = lane & 31;
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int chn = jj * 4 + 2 * q + half;
            lds_write_b128(stg + row * COLS * 2 + 16 * (chn ^ ((row >> 1) & (CPR - 1))),
                           u32x4{p[4 * q], p[4 * q + 1], p[4 * q + 2], p[4 * q + 3]});
          }
        }
        u32x4 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = lane + 64 * q;
          const int row = c / CPR, chn = c % CPR;
          v[q] = lds_read_b128(stg + row * COLS * 2 + 16 * (chn ^ ((row >> 1) & (CPR - 1))));
        }
        lds_wait(v);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = lane + 64 * q;
          const int row = c / CPR, chn = c % CPR;
          const int t = m0 + wave * 32 + row;
          if (t < g.M)
            *(uint4*)((bf16_t*)g.out + (int64_t)t * g.ldo + nt * BN + h * COLS + chn * 8) = as_uint4(v[q]);
        }
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[j] = f32x16_t{};
    }
    u = u + 1 == NSW ? 0 : u + 1;
  }
#endif
}


template <int BN, int NS>
hipError_t launch_bn(const TnArgs& g, hipStream_t s) {
  const int kz = g.kz > 0 ? g.kz : g.Ka;
  const bool fullk = kz % GK == 0 && g.Kg % GK == 0 && g.Ka + g.Kg <= g.ldw;
  const int mt = (g.M + GM - 1) / GM;
  const int nt = g.N / BN;
  const int zs = g.kz > 0 ? g.Ka / g.kz : 1;
  // enough workgroups to cover the chip once; each walks a run of N tiles
  int per = 1;
  while (per < nt && (int64_t)mt * ((nt + per * 2 - 1) / (per * 2)) * zs >= 256) per *= 2;
  dim3 grid(mt, (nt + per - 1) / per, zs);
  // a short K (2 to 6 stages) walked over many tiles with bf16 output
  // (decode, encode_bwd): token operand in registers, read once, 128-wide
  // tiles, two workgroups per CU; each workgroup walks per2 tiles and the
  // grid fills two workgroups per CU
  const int KS = (g.Ka + g.Kg) / GK;
  if constexpr (BN == 256) {
    const int nt2 = g.N / 128;
    int per2 = 1;
    while (per2 < nt2 && (int64_t)mt * ((nt2 + per2 * 2 - 1) / (per2 * 2)) >= 512) per2 *= 2;
    if (!g.out_f32 && fullk && g.kz == 0 && per2 >= 2 && KS >= 2 && KS <= 6) {
      dim3 grid2(mt, (nt2 + per2 - 1) / per2, 1);
      switch (KS) {
        case 2: hipLaunchKernelGGL((k_gemm_tn_short<2>), grid2, dim3(GTHREADS), 0, s, g, per2); break;
        case 3: hipLaunchKernelGGL((k_gemm_tn_short<3>), grid2, dim3(GTHREADS), 0, s, g, per2); break;
        case 4: hipLaunchKernelGGL((k_gemm_tn_short<4>), grid2, dim3(GTHREADS), 0, s, g, per2); break;
        case 5: hipLaunchKernelGGL((k_gemm_tn_short<5>), grid2, dim3(GTHREADS), 0, s, g, per2); break;
        default: hipLaunchKernelGGL((k_gemm_tn_short<6>), grid2, dim3(GTHREADS), 0, s, g, per2); break;
      }
      return hipGetLastError();
    }
  }
  if (fullk)
    hipLaunchKernelGGL((k_gemm_tn<BN, NS, true>), grid, dim3(GTHREADS), 0, s, g, per);
  else
    hipLaunchKernelGGL((k_gemm_tn<BN, NS, false>), grid, dim3(GTHREADS), 0, s, g, per);
  return hipGetLastError();
}

template <int BN>
hipError_t launch_ns(const TnArgs& g, hipStream_t s) {
  // Three stages, unless a short K would pad its step count (a multiple of
  // the stage count) by a large fraction: then two.
  const int kz = g.kz > 0 ? g.kz : g.Ka;
  const int KS = (kz + GK - 1) / GK + (g.Kg + GK - 1) / GK;
  if (KS % 3 != 0 && KS < 24 && KS % 2 == 0) return launch_bn<BN, 2>(g, s);
  return launch_bn<BN, 3>(g, s);
}

}  // namespace

hipError_t launch_gemm_tn(const TnArgs& g, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  if (g.kz > 0 && (g.kz % GK != 0 || g.Ka % g.kz != 0 || g.Kg != 0)) return hipErrorInvalidValue;
  if (g.N % 256 == 0) return launch_ns<256>(g, s);
  if (g.N % 128 == 0) return launch_ns<128>(g, s);
  if (g.N % 64 == 0) return launch_ns<64>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace mapl
