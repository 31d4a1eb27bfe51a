// The token-major bf16 GEMM's building blocks (layout, fragment geometry,
// the pipelined K loop and the epilogue), shared by the GEMM kernels and the
// fused encoder (projection followed by RVQ in one launch).  Device code;
// included by the kernel sources only.
#pragma once
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

// The K loop of one workgroup over its run of BN-wide output tiles, NS
// pipeline stages (2 or 3; stage i at (sia, siw), each stage its own
// __shared__ object so the compiler's wait counting stays per stage).
// After the last step of a tile, epi(acc, tile) receives the tile's
// accumulators (layout as for tn_epilogue) and must leave them cleared; no
// load is in flight then, and every wave has finished its fragment reads of
// the stages once the workgroup passes a barrier.
template <int BN, int NS, bool FULLK, bool ROT = true, typename Epi>
__device__ __forceinline__ void tn_mainloop(const TnArgs& g, int ntiles_per_wg, bf16_t* s0a, bf16_t* s0w,
                                            bf16_t* s1a, bf16_t* s1w, bf16_t* s2a, bf16_t* s2w, Epi&& epi) {
  static_assert(NS == 2 || NS == 3, "stages");
  constexpr int FM = 2, FN = BN / 64;           // 2 x 2 waves, wave tile 64 x BN/2
  constexpr int ABLK = GM / 8 / 4;              // A: 1 KiB blocks (8 rows) per wave per stage
  constexpr int WBLK = BN / 8 / 4;              // W: 1 KiB blocks per wave per stage
  constexpr int LOADS = ABLK + WBLK;            // buffer_load...lds per wave per stage

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
  // (ROT = false: every workgroup starts at step 0; measured faster for the
  // fused encoder, whose RVQ phase follows, and slower for the other uses)
  const int rot = ROT && KS > 0 ? (int)(blockIdx.x >> 3) % KS : 0;

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

  issue_next(s0a, s0w);
  if (NS == 3 && total > 1) issue_next(s1a, s1w);
  for (int tile = 0; tile < ntiles; ++tile) {
    for (int ks = 0; ks < KSP; ks += NS) {
      const int s = tile * KSP + ks;
      if constexpr (NS == 3) {
        step(s, ks, s0a, s0w, s2a, s2w);
        step(s + 1, ks + 1, s1a, s1w, s0a, s0w);
        step(s + 2, ks + 2, s2a, s2w, s1a, s1w);
      } else {
        step(s, ks, s0a, s0w, s1a, s1w);
        step(s + 1, ks + 1, s1a, s1w, s0a, s0w);
      }
    }
    epi(acc, tile);
  }
}

}  // namespace

}  // namespace mapl
