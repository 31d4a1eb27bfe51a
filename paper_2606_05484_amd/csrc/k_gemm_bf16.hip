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
#include "short_plan.hpp"

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

// Short-K, write-heavy products with bf16 output (decode: K = r + k <= 384,
// encode_bwd: K = r; N = d).  A workgroup of 4 waves owns a 256-token block
// and walks a run of 128-column output tiles; each wave owns 64 token rows
// (two 32-row fragments) x all 128 columns, so every W fragment read from
// LDS feeds two matrix products (half the LDS bytes per product of a 32-row
// wave).  A wave loads its token fragments for the whole K once, straight
// from memory into registers in the matrix unit's operand layout (16 B per
// lane and fragment; anchor rows gathered by id).  W streams through a ring
// of NSW 16 KiB stages filled by buffer_load ... lds, D = NSW - 1 stages
// ahead; the stage-ready wait and barrier sit after the third k-step of the
// stage before, so the first fragments of every stage are read while the
// last products of the previous one run.  The 128 accumulator registers per
// lane take one wave per SIMD.
//
// Output: at the end of a tile each wave packs its 64 x 128 block to bf16
// (the cross-half swap of tn_epilogue) into a wave-private 16 KiB LDS area
// as 128 B row segments; the 16 row-segment stores (8 rows x 128 B each)
// are then spread over the first k-steps of the next tile, one LDS read and
// one range-checked buffer store at a time, so the output leaves while the
// matrix units work instead of in a burst that stalls them (rows past the
// last token are dropped by the hardware; the last tile's stores drain
// after the loop).  Every wave issues the same memory operations in the same
// order every tile -- the first tile's stores go to an out-of-range offset,
// DMA past the last stage reads zeros into a slot nobody reads -- so each
// stage wait is a fixed vmcnt count, computed below from that order.
constexpr int SH_BM = 256, SH_BN = 128;

template <int KS>
__global__ __launch_bounds__(GTHREADS, 1) void k_gemm_tn_short(TnArgs g, int ntiles_per_wg) {
#if defined(__HIP_DEVICE_COMPILE__)
  using P = ShortPlan<KS>;
  static_assert(P::KSTEP == GK / 16, "64-deep stages");
  constexpr int BN = SH_BN, FM = 2, FN = BN / 32, KSTEP = P::KSTEP, KST = P::KST, D = P::D, NSW = P::NSW;
  constexpr int WBLK = P::WBLK;
  static_assert(WBLK == BN / 8 / 4 && WBLK == KSTEP, "one 1 KiB DMA block per wave and k-step");
  static_assert(KST >= 8, "at most two stores per k-step");
  constexpr uint32_t WSTG = BN * GK * 2;
  constexpr int COLS = 64, CPR = COLS / 8, STGB = 64 * BN * 2;  // per-wave staging: 64 rows x 128 columns
  __shared__ __attribute__((aligned(1024))) bf16_t SW[NSW * BN * GK + 4 * STGB / 2];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m0 = blockIdx.x * SH_BM;
  const int nt0 = blockIdx.y * ntiles_per_wg;
  const int ntiles = min(ntiles_per_wg, g.N / BN - nt0);
  const int total = ntiles * KS;

  const int mrows = min(SH_BM, g.M - m0);
  const __amdgpu_buffer_rsrc_t ra = rsrc(g.A + (int64_t)m0 * g.lda, (uint64_t)mrows * g.lda * 2);
  const __amdgpu_buffer_rsrc_t rt = rsrc(g.T, g.T ? (uint64_t)g.V * g.ldt * 2 : 0);
  const __amdgpu_buffer_rsrc_t rw = rsrc(g.W, (uint64_t)g.N * g.ldw * 2);
  const __amdgpu_buffer_rsrc_t ro = rsrc((bf16_t*)g.out + (int64_t)m0 * g.ldo, (uint64_t)mrows * g.ldo * 2);

  // token fragments of rows 64 wave + 32 i .. +31; rows past the last token read zeros
  u32x4 afr[FM][KST];
  if (!g.codes) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wave * 64 + i * 32 + (lane & 31);
      const bool in = row < mrows;
      const uint32_t ch = 16u * (uint32_t)(lane >> 5);
      const uint32_t aoff = in ? (uint32_t)row * (uint32_t)g.lda * 2u + ch : OOB;
      const uint32_t toff =
          in && g.Kg > 0 ? (uint32_t)clamp_id(g.ids[m0 + row], g.V) * (uint32_t)g.ldt * 2u + ch : OOB;
#pragma unroll
      for (int q = 0; q < KST; ++q) {
        const int kc = q * 16;
        const bool in_a = kc < g.Ka;
        afr[i][q] = __builtin_amdgcn_raw_buffer_load_b128(in_a ? ra : rt, in_a ? aoff : toff,
                                                          in_a ? kc * 2 : (kc - g.Ka) * 2, 0);
      }
    }
  } else {
    // the first Ka columns gathered from the codebooks: lane (row, half)
    // sums the 8 fp32 values k0 .. k0+7 (k0 = 16 q + 8 half) of its row's
    // codewords, l = 0 then 1, and rounds the sums to bf16
    const __amdgpu_buffer_rsrc_t rc = rsrc(g.C, (uint64_t)g.L * g.K * g.Ka * 4);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wave * 64 + i * 32 + (lane & 31);
      const bool in = row < mrows;
      const uint32_t ch = 16u * (uint32_t)(lane >> 5);
      uint32_t cw[2];
#pragma unroll
      for (int l = 0; l < 2; ++l) {
        cw[l] = OOB;
        if (in && l < g.L) {
          const int64_t e = (int64_t)(m0 + row) * g.L + l;
          const int c = g.code_bytes == 1 ? ((const uint8_t*)g.codes)[e] : ((const uint16_t*)g.codes)[e];
          cw[l] = (uint32_t)(l * g.K + (c < g.K ? c : g.K - 1)) * (uint32_t)g.Ka * 4u + 2u * ch;
        }
      }
      const uint32_t toff =
          in && g.Kg > 0 ? (uint32_t)clamp_id(g.ids[m0 + row], g.V) * (uint32_t)g.ldt * 2u + ch : OOB;
#pragma unroll
      for (int q = 0; q < KST; ++q) {
        const int kc = q * 16;
        if (kc < g.Ka) {
          const u32x4 a0 = __builtin_amdgcn_raw_buffer_load_b128(rc, cw[0], kc * 4, 0);
          const u32x4 a1 = __builtin_amdgcn_raw_buffer_load_b128(rc, cw[0], kc * 4 + 16, 0);
          const u32x4 b0 = __builtin_amdgcn_raw_buffer_load_b128(rc, cw[1], kc * 4, 0);
          const u32x4 b1 = __builtin_amdgcn_raw_buffer_load_b128(rc, cw[1], kc * 4 + 16, 0);
          float v[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = 0.f + __uint_as_float(a0[e]);
            v[4 + e] = 0.f + __uint_as_float(a1[e]);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] += __uint_as_float(b0[e]);
            v[4 + e] += __uint_as_float(b1[e]);
          }
          afr[i][q] = u32x4{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7])};
        } else {
          afr[i][q] = __builtin_amdgcn_raw_buffer_load_b128(rt, toff, (kc - g.Ka) * 2, 0);
        }
      }
    }
  }

  // W stage s (tile s / KS, k 64 (s % KS) ..) goes to ring slot s % NSW as
  // 128 B rows, 16 B chunks swizzled by ((row >> 1) & 7); block j of a wave
  // covers rows 8 (4 wave + j) .. +7
  uint32_t w_off[WBLK];
  {
    const int lrow = lane >> 3;
    const uint32_t lchp[2] = {(uint32_t)((lane & 7) ^ (lane >> 4)), (uint32_t)((lane & 7) ^ (4 + (lane >> 4)))};
#pragma unroll
    for (int j = 0; j < WBLK; ++j) {
      const int row = 8 * (wave * WBLK + j) + lrow;
      w_off[j] = (uint32_t)row * (uint32_t)g.ldw * 2u + 16u * lchp[j & 1];
    }
  }
  const uint32_t ntile_bytes = (uint32_t)BN * (uint32_t)g.ldw * 2u;
  // the DMA cursor: the stage it fills next, its ring slot, its byte offset in W
  int d_stage = 0, d_slot = 0, d_ks = 0;
  uint32_t d_off = (uint32_t)nt0 * ntile_bytes;
  auto dma_block = [&](int j) {
    const bool live = d_stage < total;
    bf16_t* dst = SW + d_slot * (BN * GK) + (wave * WBLK + j) * 512;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)dst, 16, live ? w_off[j] : OOB, (int)d_off, 0, 0);
  };
  auto dma_next = [&]() {
    ++d_stage;
    d_slot = d_slot + 1 == NSW ? 0 : d_slot + 1;
    if (++d_ks == KS) {
      d_ks = 0;
      d_off += ntile_bytes - (uint32_t)((KS - 1) * GK * 2);
    } else {
      d_off += GK * 2;
    }
  };
#pragma unroll
  for (int s = 0; s < D; ++s) {
#pragma unroll
    for (int j = 0; j < WBLK; ++j) dma_block(j);
    dma_next();
  }
  // the token fragments land here, not inside the stage loop
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int q = 0; q < KST; ++q) asm volatile("" : "+v"(afr[i][q]));

  uint32_t koff[KSTEP];
#pragma unroll
  for (int kk = 0; kk < KSTEP; ++kk) koff[kk] = tn_koff(kk, lane);
  const uint32_t swb = lds_addr(SW);
  const uint32_t stg = swb + NSW * WSTG + wave * STGB;
  const int half = lane >> 5;
  // staging chunk c (block b = c / 4 = 2 i + h, 32 rows x 64 columns; part
  // q = c % 4): lane l reads row (l + 64 q) / 8, 16 B chunk (l + 64 q) % 8
  auto chunk_lds = [&](int c) {
    const int cc = lane + 64 * (c & 3), row = cc / CPR, chn = cc % CPR;
    return stg + (c >> 2) * (32 * COLS * 2) + row * COLS * 2 + 16 * (chn ^ ((row >> 1) & (CPR - 1)));
  };
  auto chunk_out = [&](int c, int nt) {
    const int cc = lane + 64 * (c & 3), row = cc / CPR, chn = cc % CPR;
    const int i = c >> 3, h = (c >> 2) & 1;
    return (uint32_t)(wave * 64 + i * 32 + row) * (uint32_t)g.ldo * 2u +
           (uint32_t)(nt * BN + h * COLS + chn * 8) * 2u;
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  u32x4 fr[2][FN];
  auto wload = [&](uint32_t slot_base, int kk, u32x4 (&f)[FN]) {
    const uint32_t b = slot_base + koff[kk];
    static_for<0, FN>([&](auto jc) {
      constexpr int J = decltype(jc)::value;
      f[J] = lds_read_b128<J * 32 * GK * 2>(b);
    });
  };
  // stage 0 ready: the DMA of stages 1 .. D-1 may still be in flight
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(WBLK * (D - 1)) : "memory");
  __builtin_amdgcn_s_barrier();
  wload(swb, 0, fr[0]);
  lds_wait(fr[0]);

  int c_slot = 0;  // ring slot of the stage being consumed
  for (int tile = 0; tile < ntiles; ++tile) {
    // the previous tile's output, stored during this tile's first k-steps
    // (the first tile's stores go nowhere)
    const int pnt = nt0 + tile - 1;
    const bool pout = tile > 0;
    static_for<0, KS>([&](auto ksc) {
      constexpr int KSI = decltype(ksc)::value;
      const uint32_t bw = swb + (uint32_t)c_slot * WSTG;
      const int n_slot = c_slot + 1 == NSW ? 0 : c_slot + 1;
      static_for<0, KSTEP>([&](auto kkc) {
        constexpr int KK = decltype(kkc)::value, CB = KK & 1;
        constexpr int Q = KSI * KSTEP + KK, NS = P::st(Q), C0 = P::st0(Q);
        // the next k-step's W fragments (the next stage's first, after the barrier below)
        if constexpr (KK + 1 < KSTEP) wload(bw, KK + 1, fr[CB ^ 1]);
        if constexpr (KK + 1 == KSTEP) wload(swb + (uint32_t)n_slot * WSTG, 0, fr[CB ^ 1]);
        u32x4 sv[NS > 0 ? NS : 1];
        static_for<0, NS>([&](auto uc) {
          constexpr int U = decltype(uc)::value;
          sv[U] = lds_read_b128(chunk_lds(C0 + U));
        });
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int i = 0; i < FM; ++i) acc[i][j] = mfma32x32x16(as_uint4(fr[CB][j]), as_uint4(afr[i][Q]), acc[i][j]);
        dma_block(KK);
        lds_wait(fr[CB ^ 1]);
        if constexpr (KK == KSTEP - 2) {
          // stage s + 1 ready (the count of later operations is fixed by the
          // issue order), and every wave is done with stage s - 1's slot,
          // which the DMA refills from the next k-step on
          if (tile == 0)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(P::wait_n(KSI, true)) : "memory");
          else
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(P::wait_n(KSI, false)) : "memory");
          __builtin_amdgcn_s_barrier();
        }
        static_for<0, NS>([&](auto uc) {
          constexpr int U = decltype(uc)::value;
          __builtin_amdgcn_raw_buffer_store_b128(sv[U], ro, pout ? chunk_out(C0 + U, pnt) : OOB, 0, 0);
        });
      });
      dma_next();
      c_slot = n_slot;
    });

    // this tile's output into the staging area (its previous contents were
    // all read by the stores above)
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const f32x16_t& c = acc[i][j];
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
        const int row = lane & 31, h = j >> 1, jj = j & 1;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int chn = jj * 4 + 2 * q + half;
          lds_write_b128(stg + (2 * i + h) * (32 * COLS * 2) + row * COLS * 2 + 16 * (chn ^ ((row >> 1) & (CPR - 1))),
                         u32x4{p[4 * q], p[4 * q + 1], p[4 * q + 2], p[4 * q + 3]});
        }
        acc[i][j] = f32x16_t{};
      }
  }
  // the last tile's output
  {
    u32x4 v[8];
#pragma unroll
    for (int h8 = 0; h8 < 2; ++h8) {
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = lds_read_b128(chunk_lds(8 * h8 + u));
      lds_wait(v);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        __builtin_amdgcn_raw_buffer_store_b128(v[u], ro, chunk_out(8 * h8 + u, nt0 + ntiles - 1), 0, 0);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // and the zero-filling DMA past the last stage
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

// Tiles per workgroup of the short-K kernel for g, or 0 where it does not
// apply: bf16 output, 2 to 6 full stages, N a multiple of 128, and at least
// two tiles per workgroup with one 256-token workgroup per CU.
static int short_per(const TnArgs& g) {
  const int ks = (g.Ka + g.Kg) / GK;
  if (g.M <= 0 || g.out_f32 || g.kz != 0 || g.Ka % GK || g.Kg % GK || g.Ka + g.Kg > g.ldw || g.N % SH_BN ||
      ks < 2 || ks > 6)
    return 0;
  if (g.codes && (g.L < 1 || g.L > 2 || !g.C || g.K < 1 || (g.code_bytes != 1 && g.code_bytes != 2))) return 0;
  const int mt = (g.M + SH_BM - 1) / SH_BM, nt = g.N / SH_BN;
  int per = 1;
  while (per < nt && (int64_t)mt * ((nt + per * 2 - 1) / (per * 2)) >= 256) per *= 2;
  return per >= 2 ? per : 0;
}

bool gemm_tn_gathers(const TnArgs& g) { return short_per(g) >= 2; }

hipError_t launch_gemm_tn(const TnArgs& g, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  if (g.kz > 0 && (g.kz % GK != 0 || g.Ka % g.kz != 0 || g.Kg != 0)) return hipErrorInvalidValue;
  const int per = short_per(g);
  if (g.codes && per < 2) return hipErrorInvalidValue;
  // a short K (2 to 6 stages) walked over several 128-column tiles with bf16
  // output (decode, encode_bwd): one 256-token workgroup per CU, each walking
  // per tiles, as long as every workgroup gets at least two
  {
    const int ks = (g.Ka + g.Kg) / GK;
    if (per >= 2) {
      const int mt = (g.M + SH_BM - 1) / SH_BM, nt = g.N / SH_BN;
      const dim3 grid(mt, (nt + per - 1) / per);
      switch (ks) {
        case 2: hipLaunchKernelGGL((k_gemm_tn_short<2>), grid, dim3(GTHREADS), 0, s, g, per); break;
        case 3: hipLaunchKernelGGL((k_gemm_tn_short<3>), grid, dim3(GTHREADS), 0, s, g, per); break;
        case 4: hipLaunchKernelGGL((k_gemm_tn_short<4>), grid, dim3(GTHREADS), 0, s, g, per); break;
        case 5: hipLaunchKernelGGL((k_gemm_tn_short<5>), grid, dim3(GTHREADS), 0, s, g, per); break;
        default: hipLaunchKernelGGL((k_gemm_tn_short<6>), grid, dim3(GTHREADS), 0, s, g, per); break;
      }
      return hipGetLastError();
    }
  }
  if (g.N % 256 == 0) return launch_ns<256>(g, s);
  if (g.N % 128 == 0) return launch_ns<128>(g, s);
  if (g.N % 64 == 0) return launch_ns<64>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace mapl
