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
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

typedef __attribute__((address_space(3))) void* lds_ptr;

constexpr int GM = 128, GK = 64, GTHREADS = 256;
constexpr uint32_t OOB = 0x80000000u;  // any offset >= num_records reads zero

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0x7fffffffull ? 0x7fffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n, 0x00020000);
}

template <int BN>
struct TnSmem {
  bf16_t a[GM * GK];
  bf16_t w[BN * GK];
};

// Fragment geometry shared by the kernels: per 16-wide k-step kk the lane
// reads row lane % 32 (+ multiples of 16, which keep the swizzle), logical
// chunk 2 kk + lane / 32 of a 128 B-row stage.
__device__ __forceinline__ uint32_t tn_koff(int kk, int lane) {
  return (uint32_t)((lane & 31) * (GK * 2) + 16 * ((2 * kk + (lane >> 5)) ^ (((lane & 31) >> 1) & 7)));
}

// The products of one GK-deep stage for a wave's 64 x BN/2 sub-tile: A
// fragments at LDS byte address ba (token rows), W fragments at bw.
// acc[i][j] is the transposed 32 x 32 block: rows = output columns (W
// fragment j), columns = tokens (A fragment i).  Fragment reads are inline
// asm (see lds_read_b128), double-buffered in registers: the reads of
// k-step kk + 1 are in flight while the matrix units work on kk.  After the
// products of k-step kk, after(kk) runs (the caller issues a share of the
// next stage's loads there).
template <int BN, typename After>
__device__ __forceinline__ void tn_products(f32x16_t (&acc)[2][BN / 64], uint32_t ba, uint32_t bw,
                                            const uint32_t (&koff)[GK / 16], After&& after) {
  constexpr int FM = 2, FN = BN / 64, KSTEP = GK / 16;
  u32x4 fr[2][FM + FN];
  auto load = [&](int kk, u32x4 (&f)[FM + FN]) {
    static_for<0, FM>([&](auto ic) {
      constexpr int I = decltype(ic)::value;
      f[I] = lds_read_b128<I * 32 * GK * 2>(ba + koff[kk]);
    });
    static_for<0, FN>([&](auto jc) {
      constexpr int J = decltype(jc)::value;
      f[FM + J] = lds_read_b128<J * 32 * GK * 2>(bw + koff[kk]);
    });
  };
  load(0, fr[0]);
  lds_wait(fr[0]);
  static_for<0, KSTEP>([&](auto kkc) {
    constexpr int KK = decltype(kkc)::value, CB = KK & 1;
    if constexpr (KK + 1 < KSTEP) load(KK + 1, fr[CB ^ 1]);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = mfma32x32x16(as_uint4(fr[CB][FM + j]), as_uint4(fr[CB][i]), acc[i][j]);
    after(kkc);
    if constexpr (KK + 1 < KSTEP) lds_wait(fr[CB ^ 1]);
  });
}

// Epilogue of one 128 x BN output tile (columns nt BN ..): lane l holds
// token (l % 32) of fragment i and, for q = 0..3, output columns
// 8q + 4(l / 32) + 0..3 of fragment j.  fp32 results leave as 16 B stores
// (optionally accumulating).  bf16: after the cross-half swap lane (t, h)
// holds the 16 B segment of token t covering columns 8(2q + h) .. +7 of
// fragment j (q = 0, 1); segments are staged through STG_BYTES of LDS at
// byte address stg (free for the duration: the caller syncs the workgroup
// before), 128 B rows with chunks swizzled by ((row >> 1) & 7), then
// stored as full rows.  The accumulators are cleared.
template <int BN, int STG_BYTES>
__device__ __forceinline__ void tn_epilogue(f32x16_t (&acc)[2][BN / 64], const TnArgs& g, char* obase, int m0, int nt,
                                            uint32_t stg_base, int wave, int lane) {
  constexpr int FM = 2, FN = BN / 64;
  const int wm = wave >> 1, wn = wave & 1, half = lane >> 5;
  if (g.out_f32) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int t = m0 + wm * 64 + i * 32 + (lane & 31);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if (t < g.M) {
          float* o = (float*)obase + (int64_t)t * g.ldo + nt * BN + wn * (BN / 2) + j * 32 + 4 * half;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float4 v = make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
            if (g.out_accum) {
              const float4 p = *(const float4*)(o + 8 * q);
              v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
            }
            *(float4*)(o + 8 * q) = v;
          }
        }
        acc[i][j] = f32x16_t{};
      }
    }
    return;
  }
  constexpr int HALVES = FN >= 2 ? FN / 2 : 1;
  constexpr int FJ = FN >= 2 ? 2 : 1;            // fragments per half
  constexpr int COLS = FJ * 32, CPR = COLS / 8;  // staged columns, 16 B chunks per row
  static_assert(4 * 64 * COLS * 2 <= STG_BYTES, "staging fits the free buffer");
  const uint32_t stg = stg_base + wave * (64 * COLS * 2);
#pragma unroll
  for (int h = 0; h < HALVES; ++h) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int jj = 0; jj < FJ; ++jj) {
        const f32x16_t& c = acc[i][h * FJ + jj];
        uint32_t p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) p[e] = pack_bf2(c[2 * e], c[2 * e + 1]);
        // p[2g], p[2g+1]: columns 8g + 4h + 0..3; swap groups (0,1) and (2,3)
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int w = 0; w < 2; ++w) {
            const auto sw2 = __builtin_amdgcn_permlane32_swap(p[4 * q + w], p[4 * q + 2 + w], false, false);
            p[4 * q + w] = sw2[0];
            p[4 * q + 2 + w] = sw2[1];
          }
        const int row = i * 32 + (lane & 31);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int ch = jj * 4 + 2 * q + half;
          lds_write_b128(stg + row * COLS * 2 + 16 * (ch ^ ((row >> 1) & (CPR - 1))),
                         u32x4{p[4 * q], p[4 * q + 1], p[4 * q + 2], p[4 * q + 3]});
        }
      }
    u32x4 v[CPR];
#pragma unroll
    for (int q = 0; q < CPR; ++q) {
      const int c = lane + 64 * q;
      const int row = c / CPR, ch = c % CPR;
      v[q] = lds_read_b128(stg + row * COLS * 2 + 16 * (ch ^ ((row >> 1) & (CPR - 1))));
    }
    lds_wait(v);
#pragma unroll
    for (int q = 0; q < CPR; ++q) {
      const int c = lane + 64 * q;
      const int row = c / CPR, ch = c % CPR;
      const int t = m0 + wm * 64 + row;
      if (t < g.M)
        *(uint4*)((bf16_t*)obase + (int64_t)t * g.ldo + nt * BN + wn * (BN / 2) + h * COLS + ch * 8) = as_uint4(v[q]);
    }
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};
}

// NS pipeline stages (2 or 3), one __shared__ array each.
template <int BN, int NS, bool FULLK>
__global__ __launch_bounds__(GTHREADS) void k_gemm_tn(TnArgs g, int ntiles_per_wg) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature (launch stub)
  static_assert(NS == 2 || NS == 3, "stages");
  constexpr int FM = 2, FN = BN / 64;           // 2 x 2 waves, wave tile 64 x BN/2
  constexpr int ABLK = GM / 8 / 4;              // A: 1 KiB blocks (8 rows) per wave per stage
  constexpr int WBLK = BN / 8 / 4;              // W: 1 KiB blocks per wave per stage
  constexpr int LOADS = ABLK + WBLK;            // buffer_load...lds per wave per stage
  __shared__ __attribute__((aligned(1024))) TnSmem<BN> S0;
  __shared__ __attribute__((aligned(1024))) TnSmem<BN> S1;
  // third stage (NS == 3 only; a token array otherwise)
  __shared__ __attribute__((aligned(1024))) bf16_t S2buf[NS == 3 ? (GM + BN) * GK : 8];
  bf16_t* const S2a = S2buf;
  bf16_t* const S2w = S2buf + GM * GK;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar LDS addresses
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.x * GM;
  const int nt0 = blockIdx.y * ntiles_per_wg;
  const int ntiles = min(ntiles_per_wg, g.N / BN - nt0);
  const int kz = g.kz > 0 ? g.kz : g.Ka;
  const int kbase = g.kz > 0 ? blockIdx.z * g.kz : 0;
  const int ka_steps = (kz + GK - 1) / GK;
  const int kg_steps = (g.Kg + GK - 1) / GK;
  const int KS = ka_steps + kg_steps;
  const int KSP = (KS + NS - 1) / NS * NS;      // padded: stage buffers repeat every tile
  const int total = ntiles * KSP;
  // Workgroups start their K walk at different k-steps (the same for the
  // eight consecutive ids spread over the XCDs): at any moment the token
  // rows in flight then sit at different column offsets, which spreads the
  // strided row reads over more HBM channels and banks.
  const int rot = KS > 0 ? (int)(blockIdx.x >> 3) % KS : 0;

  // Buffer resources: A rows of this workgroup, the anchor table, W.
  const int mrows = min(GM, g.M - m0);
  const __amdgpu_buffer_rsrc_t ra = rsrc(g.A + (int64_t)m0 * g.lda, (uint64_t)(mrows > 0 ? mrows : 0) * g.lda * 2);
  const __amdgpu_buffer_rsrc_t rt = rsrc(g.T, g.T ? (uint64_t)g.V * g.ldt * 2 : 0);
  const __amdgpu_buffer_rsrc_t rw = rsrc(g.W, (uint64_t)g.N * g.ldw * 2);

  // Per-lane DMA geometry: lane i of block b fills row 8b + i/8, physical
  // chunk i%8, so it loads logical chunk (i%8) ^ ((row >> 1) & 7), which
  // depends only on the parity of b.  All offsets are 32-bit byte offsets
  // from the resource bases (validated on the host).  The per-lane part
  // (row, chunk) is fixed for the whole kernel; a stage adds its column
  // offset, uniform across the wave.
  const int lrow = lane >> 3;
  const uint32_t lchp[2] = {(uint32_t)((lane & 7) ^ (lane >> 4)), (uint32_t)((lane & 7) ^ (4 + (lane >> 4)))};
  uint32_t a_off[ABLK], t_off[ABLK], w_off[WBLK];
#pragma unroll
  for (int j = 0; j < ABLK; ++j) {
    const int row = 8 * (wave * ABLK + j) + lrow;
    const uint32_t lc = lchp[j & 1];
    a_off[j] = (uint32_t)row * (uint32_t)g.lda * 2u + 16u * lc;
    const bool has = g.Kg > 0 && m0 + row < g.M;
    t_off[j] = has ? (uint32_t)clamp_id(g.ids[m0 + row], g.V) * (uint32_t)g.ldt * 2u + 16u * lc : OOB;
  }
#pragma unroll
  for (int j = 0; j < WBLK; ++j) {
    const int row = 8 * (wave * WBLK + j) + lrow;
    w_off[j] = (uint32_t)row * (uint32_t)g.ldw * 2u + 16u * lchp[j & 1];
  }

  // A real step issues exactly LOADS loads per wave; a padding step issues
  // none (the wait before a step accounts for that).  A step's loads are
  // planned once (steps in order), then issued a few at a time between the
  // products of the step before (see compute): a burst of them would hold up
  // the wave's instruction stream while the memory pipeline drains it.
  // FULLK: every K dimension is a multiple of GK, so each real step covers
  // whole stages: a load takes the lane's fixed offset as its VGPR operand
  // and the stage's column offset as its scalar operand (rows past the last
  // token still fall outside the A resource and read zeros), and planning
  // costs no vector arithmetic.  Otherwise per-lane checks select each
  // offset or OOB.
  struct Plan {
    bf16_t *sa, *sw;
    int sA, sW;
    bool live, gathered;
    uint32_t vA[FULLK ? 1 : ABLK], vW[FULLK ? 1 : WBLK];  // per-lane offsets (not FULLK)
  };
  int pl_ks = 0, pl_nt = nt0;  // next step to plan
  auto plan_next = [&](bf16_t* sa, bf16_t* sw) {
    Plan p;
    p.sa = sa;
    p.sw = sw;
    // uniform by construction; readfirstlane lets the compiler see it, so
    // the choices and offsets below stay in scalar registers
    const int ks0 = __builtin_amdgcn_readfirstlane(pl_ks), nt = __builtin_amdgcn_readfirstlane(pl_nt);
    if (++pl_ks == KSP) {
      pl_ks = 0;
      ++pl_nt;
    }
    p.live = ks0 < KS;
    int ks = ks0 + rot;
    if (ks >= KS) ks -= KS;
    p.gathered = p.live && ks >= ka_steps;
    const int kc = p.gathered ? (ks - ka_steps) * GK : ks * GK;
    const uint32_t aadd = (uint32_t)(p.gathered ? kc : kbase + kc) * 2u;
    const int wcol0 = p.gathered ? g.Ka + kc : kbase + kc;
    const uint32_t wadd = (uint32_t)nt * BN * (uint32_t)g.ldw * 2u + (uint32_t)wcol0 * 2u;
    if constexpr (FULLK) {
      p.sA = (int)aadd;
      p.sW = (int)wadd;
    } else {
      const int alim = p.gathered ? g.Kg : kz;
      const int wlim = p.gathered ? g.Ka + g.Kg : kbase + kz;
      // this lane's first column in the stage, per block parity
      const int col0 = kc + 8 * (int)lchp[0], col1 = kc + 8 * (int)lchp[1];
      const int wc0 = wcol0 + 8 * (int)lchp[0], wc1 = wcol0 + 8 * (int)lchp[1];
      const bool ok0 = col0 < alim, ok1 = col1 < alim;
      const bool wok0 = wc0 < wlim && wc0 < g.ldw, wok1 = wc1 < wlim && wc1 < g.ldw;
#pragma unroll
      for (int j = 0; j < ABLK; ++j) {
        const uint32_t o = p.gathered ? t_off[j] : a_off[j];
        p.vA[j] = ((j & 1) ? ok1 : ok0) && o != OOB ? o + aadd : OOB;
      }
#pragma unroll
      for (int j = 0; j < WBLK; ++j) p.vW[j] = ((j & 1) ? wok1 : wok0) ? w_off[j] + wadd : OOB;
      p.sA = 0;
      p.sW = 0;
    }
    return p;
  };
  // loads [B0, B1) of a step: A (or anchor) block li < ABLK, else W block li - ABLK
  auto issue_range = [&](const Plan& p, auto b0c, auto b1c) {
    constexpr int B0 = decltype(b0c)::value, B1 = decltype(b1c)::value;
    if (!p.live) return;
    auto go = [&](auto gc) {
      constexpr bool GATH = decltype(gc)::value;
      static_for<B0, B1>([&](auto lic) {
        constexpr int LI = decltype(lic)::value;
        if constexpr (LI < ABLK) {
          const lds_ptr dst = (lds_ptr)(p.sa + (wave * ABLK + LI) * 512);
          const uint32_t v = FULLK ? (GATH ? t_off[LI] : a_off[LI]) : p.vA[FULLK ? 0 : LI];
          __builtin_amdgcn_raw_ptr_buffer_load_lds(GATH ? rt : ra, dst, 16, v, p.sA, 0, 0);
        } else {
          constexpr int J = LI - ABLK;
          const lds_ptr dst = (lds_ptr)(p.sw + (wave * WBLK + J) * 512);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, dst, 16, FULLK ? w_off[J] : p.vW[FULLK ? 0 : J], p.sW, 0, 0);
        }
      });
    };
    if (p.gathered)
      go(std::true_type{});
    else
      go(std::false_type{});
  };
  auto issue_next = [&](bf16_t* sa, bf16_t* sw) {
    const Plan p = plan_next(sa, sw);
    issue_range(p, std::integral_constant<int, 0>{}, std::integral_constant<int, LOADS>{});
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  uint32_t koff[GK / 16];
#pragma unroll
  for (int kk = 0; kk < GK / 16; ++kk) koff[kk] = tn_koff(kk, lane);
  // Products of one stage; the next step's loads (if any) are issued in
  // KSTEP groups after the products of each 16-wide k-step.
  constexpr int KSTEP = GK / 16, PER = (LOADS + KSTEP - 1) / KSTEP;
  auto compute = [&](const bf16_t* sa, const bf16_t* sw, const Plan& nx, bool has_next) {
    const uint32_t ba = lds_addr(sa) + wm * 64 * (GK * 2), bw = lds_addr(sw) + wn * (BN / 2) * (GK * 2);
    tn_products<BN>(acc, ba, bw, koff, [&](auto kkc) {
      constexpr int KK = decltype(kkc)::value;
      constexpr int B0 = KK * PER < LOADS ? KK * PER : LOADS;
      constexpr int B1 = (KK + 1) * PER < LOADS ? (KK + 1) * PER : LOADS;
      if (has_next) issue_range(nx, std::integral_constant<int, B0>{}, std::integral_constant<int, B1>{});
    });
  };

  // One pipeline step: stage s (in buffer `cur`) is consumed; stage s + NS - 1
  // is issued into `nxt` (the buffer consumed at step s - 1).
  auto step = [&](int s, int ks, const bf16_t* ca, const bf16_t* cw, bf16_t* na, bf16_t* nw) {
    // stage s must be complete; only stage s + 1 (if it loads anything) may
    // still be in flight (NS = 3)
    const bool next_loads = s + 1 < total && !(ks + 1 < KSP && ks + 1 >= KS);
    if (NS == 3 && next_loads)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    const bool has_next = s + NS - 1 < total;
    if (ks < KS) {
      Plan p{};
      if (has_next) p = plan_next(na, nw);
      compute(ca, cw, p, has_next);
    } else if (has_next) {
      issue_next(na, nw);
    }
  };

  issue_next(S0.a, S0.w);
  if (NS == 3 && total > 1) issue_next(S1.a, S1.w);
  char* obase = (char*)g.out + (g.kz > 0 ? (int64_t)blockIdx.z * g.out_z * 4 : 0);
  for (int tile = 0; tile < ntiles; ++tile) {
    for (int ks = 0; ks < KSP; ks += NS) {
      const int s = tile * KSP + ks;
      if constexpr (NS == 3) {
        step(s, ks, S0.a, S0.w, S2a, S2w);
        step(s + 1, ks + 1, S1.a, S1.w, S0.a, S0.w);
        step(s + 2, ks + 2, S2a, S2w, S1.a, S1.w);
      } else {
        step(s, ks, S0.a, S0.w, S1.a, S1.w);
        step(s + 1, ks + 1, S1.a, S1.w, S0.a, S0.w);
      }
    }
    // epilogue, staging bf16 results through the buffer consumed by the
    // tile's last step (no DMA targets it before the next tile's first step)
    if (!g.out_f32) __builtin_amdgcn_s_barrier();  // every wave is done reading that buffer
    tn_epilogue<BN, (GM + BN) * GK * 2>(acc, g, obase, m0, nt0 + tile, lds_addr(NS == 3 ? S2a : S1.a), wave, lane);
  }
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
