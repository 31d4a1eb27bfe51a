// Residual vector quantisation of the projected coordinates (Sec. 3.5):
// L rounds; round l picks, per token, the codeword of C_l nearest to the
// current residual R_l and subtracts it.  Ties go to the lowest index.
//
// Decision procedure (exact with respect to the fp32 residual):
//   screen  on the bf16 matrix units with R~ = bf16(R), C~ = bf16(C), the
//           first k-step of every tile multiplying the codeword's norm
//           columns by the token's norm operand, so the accumulator ends at
//           a certified lower bound of the exact score s_j = ||C_j||^2 -
//           2 R.C_j:  L_j = s~_j - Delta'_j,  s~_j = ||C_j||^2 - 2 R~.C~_j,
//           where Delta'_j >= Delta_j bounds |s~_j - s_j| from the actual
//           bf16 rounding-error norms of the token's residual and of the
//           codeword, fp32 accumulation and norms, and the index tag below
//           (see rvq_margin_ka/k2 and the norm columns in common.hpp): the
//           margin is each codeword's own, not the codebook's largest.
//   tag     the low 4 mantissa bits of L_j hold its slot among the 16
//           scores a lane sees per tile, so a plain float min / med3 also
//           yields the position; the tile of the smallest is tracked per
//           tile.
//   pass 1  per lane: the two smallest keys.  The nearest codeword j*
//           satisfies L_j* <= s_j* <= s_j1 <= U = L_j1 + (1 + 1.03) Delta_j1
//           for the smallest key j1, so it is among {j : L_j <= U}: a
//           single codeword when the token's second key exceeds U (final).
//   pass 2  (only in a workgroup with a token not final) lists every
//           codeword with L_j <= U of those tokens: their B operands are
//           compacted into 32-token tiles in LDS, and each wave screens a
//           quarter of the codeword tiles against them, codebook fragments
//           read straight from the L2-resident screening copy.
//   rescore the listed candidates exactly in fp32 as sum_c (R_c - C_jc)^2:
//           per wave a batch of up to 8 open tokens, their residual rows
//           staged in LDS, 8 (token, codeword) pairs per step with coalesced
//           codeword rows and one cross-lane reduction for all 8.
// The fp32 residual stays in registers across rounds, updated as
// R_{l+1} = R_l - C_l[code_l]; the rescoring reads it from there (through
// LDS rows), so screening and rescoring see the same R.
//
// Layout: a workgroup of 4 waves owns 128 tokens, 32 per wave.  A wave keeps
// its tokens' bf16(-2R) as the B operand of v_mfma_f32_32x32x16_bf16 in
// registers (tokens along N); 64-codeword chunks of C~ (with the norm
// columns) stream through three LDS stages filled by buffer_load ... lds
// (direct-to-LDS, one __shared__ array per stage) as the A operand
// (codewords along M).
// Each lane thus sees the scores of ONE token for 16 codewords per tile;
// the fold of one tile into (m1, m2) overlaps the matrix products of the
// next.  The two lane halves that share a token merge at the end of a pass.
#include "tn_gemm.hpp"

namespace mapl {

namespace {

typedef __attribute__((address_space(3))) void* rq_lds_ptr;
constexpr int RQ_THREADS = 256, RQ_TOK = 128, RQ_CW = 64, RQ_CAP = 16, RQ_LMAX = 8;
constexpr uint32_t RQ_OOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rq_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0x7fffffffull ? 0x7fffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n, 0x00020000);
}

// Codeword rows (R + 16 bf16: the coordinates, then the norm columns) are
// stored 2(R + 16) + 16 bytes apart, an odd number of 16 B chunks, so the 16
// rows that read one 16 B column chunk of a fragment hit 16 distinct bank
// groups: conflict-free reads whose addresses differ per k-step by an
// immediate offset only.
template <int R>
constexpr int rq_row_bytes() { return 2 * (R + 16) + 16; }
template <int R>
constexpr int rq_blocks() {  // 1 KiB DMA blocks per wave covering the 64 padded rows
  return (RQ_CW * rq_row_bytes<R>() + 4 * 1024 - 1) / (4 * 1024);
}

template <int R>
struct RqStage {
  bf16_t c[4 * rq_blocks<R>() * 512];  // 64 padded codeword rows (+ tail)
};

__device__ __forceinline__ int load_code(const void* codes, int cb, int64_t idx) {
  return cb == 1 ? ((const uint8_t*)codes)[idx] : ((const uint16_t*)codes)[idx];
}

// Row of a 32-codeword tile held by accumulator slot e of a lane in `half`.
__device__ __forceinline__ int rq_row(int e, int half) { return 8 * (e >> 2) + 4 * half + (e & 3); }

// A score tagged in its low 4 mantissa bits with its slot among the lane's
// 16 scores of a tile (inline constants, one operation): a plain float min /
// med3 then also carries the slot.  The tag moves a score by less than
// 2^-19 of its magnitude, inside the margin's allowance for it.
__device__ __forceinline__ float rq_tag_slot(float s, int e) {
  return __uint_as_float((__float_as_uint(s) & ~15u) | (uint32_t)e);
}

// Per-workgroup LDS of the rounds besides the three codebook stages.
struct RqSmall {
  int cand_cnt[RQ_TOK];
  uint16_t cand[RQ_TOK][RQ_CAP];
  float cthr[RQ_TOK];  // the open tokens, compacted: threshold U and token index
  int cmap[RQ_TOK];
  int wcnt[4];         // open tokens per wave
  int dec[4][8];       // per wave: the decisions of a rescoring batch
};

// The L rounds for the workgroup's 128 tokens (blockIdx.x), given each
// lane's fp32 residual R_0 = Z0 (columns 16 s + 8 (lane / 32) + 0..7 of
// token 32 wave + lane % 32; zeros past T).  s0, s1, s2: three stage
// buffers of at least sizeof(RqStage<R>) bytes, each its own __shared__
// object (stage 2 also holds the residuals of the tokens being rescored).
// No load may be in flight on entry and the workgroup must have passed a
// barrier after its last use of the buffers.
template <int R>
__device__ __forceinline__ void rvq_rounds(const RvqArgs& a, bf16_t* s0, bf16_t* s1, bf16_t* s2, RqSmall& sm,
                                           float (&res)[R / 16][8]) {
  constexpr int NK16 = R / 16;                     // k-steps of the coordinates
  constexpr int CPR = (R + 16) / 8;                // 16 B chunks per codeword row
  constexpr int LOADS = rq_blocks<R>();            // DMA blocks per wave per stage
  auto& cand_cnt = sm.cand_cnt;
  auto& cand = sm.cand;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int tl = wave * 32 + (lane & 31);  // token within the workgroup
  const int t = blockIdx.x * RQ_TOK + tl;
  const bool valid = t < a.T;
  const int nchunks = (a.K + RQ_CW - 1) / RQ_CW;
  const int total = (nchunks + 2) / 3 * 3;       // padded: stage buffers repeat every pass

  // DMA geometry: LDS byte 1024 b + 16 i of a stage (lane i of block b)
  // holds 16 B column chunk `ch` of codeword row `row` of the chunk, or a
  // padding slot (zeros).  Per lane the global offset is fixed up to the
  // chunk's base, so it is computed once.
  constexpr int RB = rq_row_bytes<R>();
  constexpr int CBLK = rq_blocks<R>();
  uint32_t c_off[CBLK];
#pragma unroll
  for (int jb = 0; jb < CBLK; ++jb) {
    const int byte = (wave * CBLK + jb) * 1024 + lane * 16;
    const int row = byte / RB, ch = (byte % RB) / 16;
    c_off[jb] = (row < RQ_CW && ch < CPR) ? (uint32_t)row * (uint32_t)((R + 16) * 2) + (uint32_t)ch * 16u : RQ_OOB;
  }

  // chunk q of round l's codebook into stage buffer sc
  auto issue_l = [&](int l, int q, bf16_t* sc) {
    const __amdgpu_buffer_rsrc_t rc =
        rq_rsrc(a.Cb + (int64_t)l * a.K * (R + 16), (uint64_t)a.K * (R + 16) * 2);
    const bool pad = q >= nchunks;
    // rows past K read zeros through the resource bound (K % 32 == 0)
#pragma unroll
    for (int jb = 0; jb < CBLK; ++jb)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (rq_lds_ptr)(sc + (wave * CBLK + jb) * 512), 16,
                                               (!pad && c_off[jb] != RQ_OOB)
                                                   ? (uint32_t)(q * RQ_CW) * (uint32_t)((R + 16) * 2) + c_off[jb]
                                                   : RQ_OOB,
                                               0, 0, 0);
  };
  // A round's first two chunks are requested before the previous round's
  // residual update, so their latencies overlap.
  issue_l(0, 0, s0);
  issue_l(0, 1, s1);

  // res: fp32 residual of the lane's token, R_{l+1} = R_l - C_l[code_l]
  for (int l = 0; l < a.L; ++l) {
    auto issue = [&](int q, bf16_t* sc) { issue_l(l, q, sc); };

    // bf16(-2 R_l) in B-fragment layout, ||R_l||^2 and ||R_l - bf16(R_l)||^2
    // from the fp32 residual (-2 bf16(v) = bf16(-2 v), and v - bf16(v) is
    // exact in fp32)
    uint4 rb[NK16];
    float rn2 = 0.f, er2 = 0.f;
#pragma unroll
    for (int s = 0; s < NK16; ++s) {
      const float* v = res[s];
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[e] = pack_bf2(-2.f * v[2 * e], -2.f * v[2 * e + 1]);
        const float d0 = fmaf(0.5f, __uint_as_float(w[e] << 16), v[2 * e]);
        const float d1 = fmaf(0.5f, __uint_as_float(w[e] & 0xFFFF0000u), v[2 * e + 1]);
        rn2 = fmaf(v[2 * e], v[2 * e], rn2);
        rn2 = fmaf(v[2 * e + 1], v[2 * e + 1], rn2);
        er2 = fmaf(d0, d0, er2);
        er2 = fmaf(d1, d1, er2);
      }
      rb[s] = make_uint4(w[0], w[1], w[2], w[3]);
    }
    rn2 += __shfl_xor(rn2, 32, WAVE);
    er2 += __shfl_xor(er2, 32, WAVE);
    // norms rounded up (each sum carries at most R ulps of accumulation error)
    const float rnorm = sqrtf(rn2) * (1.0f + 1.0f / 32768.0f);
    const float enorm = sqrtf(er2) * (1.0f + 1.0f / 32768.0f);
    // the margin's coefficient of ||C_j|| (b) and of e_j (c)
    const float bco = 2.0f * enorm * 1.0078125f + rvq_margin_ka(R) * rnorm;
    const float cco = 2.0f * rnorm;

    // One screening pass over all chunks.  Per 32-codeword tile the fold
    // callbacks see begin(), score(acc, tile, e) for e = 0..15, end(tile).
    // Software pipeline per 64-codeword chunk (asm LDS reads, see
    // lds_read_b128; sched_barrier keeps the interleave):
    //   first fragment reads
    //   tile 0 products, each followed by a later fragment read and a share
    //     of the fold of the previous chunk's tile 1
    //   tile 1 products, each followed by a later fragment read and a share
    //     of the fold of tile 0
    // Reads of an invalid second tile (K % 64 == 32) hit zero-filled rows and
    // are discarded.
    // Products per tile: the norm step, then the NK16 coordinate k-steps;
    // one fragment read per product.
    constexpr int P = NK16 + 1;
    constexpr int FPS = (16 + P - 1) / P;  // scores folded per product step
    // second operand of the norm step: ones in k = 0..2 (the reduced norm's
    // pieces), -b in k = 3, 4 (times the norm's pieces) and -c in k = 5
    // (times the rounding-error norm) of the block: the screen yields the
    // lower bound L_j of each codeword's score
    const uint32_t bbits = bf16_up(bco * RVQ_K1_SLACK) | 0x8000u;
    const uint32_t cbits = bf16_up(cco * RVQ_K1_SLACK) | 0x8000u;
    const uint4 rbn = half == 0 ? make_uint4(0x3F803F80u, 0x3F80u | (bbits << 16), bbits | (cbits << 16), 0u)
                                : make_uint4(0u, 0u, 0u, 0u);
    auto pass = [&](auto&& fbegin, auto&& fscore, auto&& fend, bool first) {
      if (!first) {
        issue(0, s0);
        issue(1, s1);
      }
      f32x16_t pend;
#pragma unroll
      for (int e = 0; e < 16; ++e) pend[e] = 3.0e38f;
      int pend_tile = -1;
      auto fold_all = [&](const f32x16_t& acc, int tile) {
        fbegin();
        static_for<0, 16>([&](auto ec) { fscore(acc, tile, ec); });
        fend(tile);
      };
      auto stage = [&](int q, const bf16_t* sc, bf16_t* nc) {
        if (q + 1 < total)
          asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS) : "memory");
        else
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        if (q + 2 < total) issue(q + 2, nc);
        if (q >= nchunks) return;
        const bool t1ok = q * RQ_CW + 32 < a.K;
        // rows lane % 32 of a tile, 16 B chunk 2s + lane / 32 (s = NK16: the
        // norm columns)
        const uint32_t cbase = lds_addr(sc) + (lane & 31) * RB + half * 16;
        // The chunk's 2P products read one fragment each, in order, through
        // a window of W registers: fragment p + W is read right after
        // product p, and product p waits until at most the reads issued
        // after fragment p are outstanding (LDS reads complete in order).
        constexpr int W = 4, NP2 = 2 * P;
        u32x4 fw[W];
        auto read = [&](auto pc) {
          constexpr int PI = decltype(pc)::value, CT = PI / P, RI = PI % P;
          if constexpr (RI == 0)
            fw[PI % W] = lds_read_b128<CT * 32 * RB + 32 * NK16>(cbase);
          else
            fw[PI % W] = lds_read_b128<CT * 32 * RB + 32 * (RI - 1)>(cbase);
        };
        auto opnd = [&](auto sc2) -> const uint4& {
          constexpr int S = decltype(sc2)::value;
          if constexpr (S == 0)
            return rbn;
          else
            return rb[S - 1];
        };
        static_for<0, W>([&](auto pc) { read(pc); });
        // an invalid second tile (K % 64 == 32) reads zero rows; its
        // products are computed and discarded
        f32x16_t acc0 = f32x16_t{}, acc1 = f32x16_t{};
        static_for<0, NP2>([&](auto pc) {
          constexpr int PI = decltype(pc)::value, CT = PI / P, S = PI % P;
          constexpr int AHEAD = (NP2 - 1 - PI) < (W - 1) ? (NP2 - 1 - PI) : (W - 1);
          lds_wait_n<AHEAD>(fw[PI % W]);
          if constexpr (CT == 0)
            acc0 = mfma32x32x16(as_uint4(fw[PI % W]), opnd(std::integral_constant<int, S>{}), acc0);
          else
            acc1 = mfma32x32x16(as_uint4(fw[PI % W]), opnd(std::integral_constant<int, S>{}), acc1);
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (PI + W < NP2) read(std::integral_constant<int, PI + W>{});
          constexpr int E0 = S * FPS < 16 ? S * FPS : 16, E1 = (S + 1) * FPS < 16 ? (S + 1) * FPS : 16;
          if constexpr (CT == 0) {
            // the previous chunk's second tile, folded a share per product
            // of this chunk's first
            if constexpr (S == 0) fbegin();
            static_for<E0, E1>([&](auto ec) { fscore(pend, pend_tile, ec); });
            if constexpr (S == P - 1) fend(pend_tile);
          } else {
            // the first tile's scores, folded a share per product of the second
            if constexpr (S == 0) fbegin();
            static_for<E0, E1>([&](auto ec) { fscore(acc0, 2 * q, ec); });
          }
          __builtin_amdgcn_sched_barrier(0);
        });
        fend(2 * q);
        if (t1ok) {
          pend = acc1;
          pend_tile = 2 * q + 1;
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) pend[e] = 3.0e38f;
          pend_tile = -1;
        }
      };
      for (int q = 0; q < total; q += 3) {
        stage(q, s0, s2);
        stage(q + 1, s1, s0);
        stage(q + 2, s2, s1);
      }
      fold_all(pend, pend_tile);
    };

    // Decision.  Each key is a lower bound L_j of its codeword's exact score
    // (the screen subtracts that codeword's own error bound), and s_j1 <= U =
    // L_j1 + (RVQ_SUB_FACTOR + 1) Delta_j1 for the smallest key j1 (of equal
    // keys, half 0's), so only codewords with L_j <= U can be nearest.
    //  pass 1: per lane the two smallest keys and the position of the
    //    first; a token is final when its second key exceeds U;
    //  pass 2 (only in a workgroup with an open token): every key <= U of
    //    the open tokens listed (the open tokens compacted); the candidates
    //    are rescored exactly in fp32.
    const float* n2l = a.meta + (int64_t)l * nchunks * 64;
    const float* e2l = n2l + (int64_t)a.L * nchunks * 64;
    auto margin = [&](int j) {  // Delta_j, rounded up
      const int jj = min(max(j, 0), nchunks * 64 - 1);
      const float n2 = n2l[jj];
      return (cco * e2l[jj] + bco * (sqrtf(n2) * (1.0f + 1.0f / 32768.0f)) + rvq_margin_k2(R) * n2) * 1.0002f +
             1e-30f;
    };
    // ---- pass 1: the two smallest keys per lane (slot tags) and the tile
    // of the smallest
    int j1;
    float thr;
    bool open;  // not final: the token's candidates are listed by pass 2
    {
      float m1 = INFINITY, m2 = INFINITY, m1_in = INFINITY;
      int tile1 = 0;
      pass([&]() { m1_in = m1; },
           [&](const f32x16_t& acc, int, auto ec) {
             constexpr int E = decltype(ec)::value;
             const float key = rq_tag_slot(acc[E], E);
             m2 = __builtin_amdgcn_fmed3f(m1, m2, key);
             m1 = __builtin_amdgcn_fmed3f(m1, key, -3.40282347e38f);  // min for finite keys
           },
           [&](int tile) { tile1 = m1 < m1_in ? tile : tile1; }, true);
      const float o1 = __shfl_xor(m1, 32, WAVE), o2 = __shfl_xor(m2, 32, WAVE);
      const int own_j1 = tile1 * 32 + rq_row((int)(__float_as_uint(m1) & 15u), half);
      const int o_j1 = __shfl_xor(own_j1, 32, WAVE);
      j1 = (m1 < o1 || (m1 == o1 && half == 0)) ? own_j1 : o_j1;
      const float k2 = fminf(fmaxf(m1, o1), fminf(m2, o2));
      thr = fminf(m1, o1) + (RVQ_SUB_FACTOR + 1.0f) * margin(j1);
      open = valid && !(k2 > thr);
      if (half == 0) cand_cnt[tl] = 0;
    }
    const int any_open = __syncthreads_or(open ? 1 : 0);
    if (a.stats && tid == 0) {
      atomicAdd(&a.stats[4], 1);
      if (any_open) atomicAdd(&a.stats[3], 1);
    }

    int jstar = j1;
    if (any_open) {
      // ---- pass 2: list every key <= U of the open tokens.  The open
      // tokens are compacted: each writes its MFMA B operand (the 17 k-steps
      // of bf16(-2R) and the norm operand, 16 B per lane half and k-step) to
      // a row of stages 0 and 1 (free until the next round's loads), its
      // threshold and index to a table; then every wave takes 32 compacted
      // tokens at a time against its quarter of the codeword tiles, the
      // codebook fragments read straight from the (L2-resident) screening
      // copy, with no LDS staging and no barrier between waves.
      constexpr int TB = (R + 16) * 2;                        // bytes of a compacted row
      constexpr int CAP0 = (int)(sizeof(RqStage<R>) / TB);     // rows in stage 0
      static_assert(2 * CAP0 >= RQ_TOK, "stages 0 and 1 hold every token's row");
      auto crow = [&](int c) -> char* {
        return c < CAP0 ? (char*)s0 + (int64_t)c * TB : (char*)s1 + (int64_t)(c - CAP0) * TB;
      };
      {
        const uint64_t ob = __ballot(half == 0 && open);
        if (lane == 0) sm.wcnt[wave] = __popcll(ob);
        __syncthreads();
        int base = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) base += w < wave ? sm.wcnt[w] : 0;
        if (open) {
          const int c = base + __popcll(ob & ((1ull << (lane & 31)) - 1ull));
          char* rw = crow(c) + 16 * half;
#pragma unroll
          for (int s = 0; s < NK16; ++s) *(uint4*)(rw + 32 * s) = rb[s];
          *(uint4*)(rw + 32 * NK16) = rbn;
          if (half == 0) {
            sm.cthr[c] = thr;
            sm.cmap[c] = tl;
          }
        }
        __syncthreads();
      }
      const int n_open = (sm.wcnt[0] + sm.wcnt[1]) + (sm.wcnt[2] + sm.wcnt[3]);
      const __amdgpu_buffer_rsrc_t rcb =
          rq_rsrc(a.Cb + (int64_t)l * a.K * (R + 16), (uint64_t)a.K * (R + 16) * 2);
      const int ntiles = a.K / 32;  // K % 32 == 0
      for (int ct = 0; ct * 32 < n_open; ++ct) {  // workgroup-uniform
        const int c = ct * 32 + (lane & 31);
        const bool cv = c < n_open;
        const int cc = cv ? c : n_open - 1;
        uint4 bq[NK16 + 1];  // [0]: the norm step, [1 + s]: k-step s
        {
          const char* rr = crow(cc) + 16 * half;
          bq[0] = *(const uint4*)(rr + 32 * NK16);
#pragma unroll
          for (int s = 0; s < NK16; ++s) bq[1 + s] = *(const uint4*)(rr + 32 * s);
        }
        const float cthr = cv ? sm.cthr[cc] : -INFINITY;
        const int ctl = sm.cmap[cc];
        // codeword tiles q = wave, wave + 4, ...; the next tile's fragments
        // are requested before the products of the current one
        constexpr int PF = NK16 + 1;  // the whole next tile
        auto frag = [&](int q, int p) -> uint4 {
          // row q * 32 + lane % 32; 16-byte chunk 2 s + half for k-step s =
          // p - 1, the norm columns (chunk 2 NK16 + half) for p = 0
          const uint32_t off = (uint32_t)(q * 32 + (lane & 31)) * (uint32_t)TB + 16u * (uint32_t)half +
                               32u * (uint32_t)(p == 0 ? NK16 : p - 1);
          const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rcb, off, 0, 0);
          return make_uint4(v[0], v[1], v[2], v[3]);
        };
        uint4 pre[PF];
        if (wave < ntiles) {
#pragma unroll
          for (int p = 0; p < PF; ++p) pre[p] = frag(wave, p);
        }
        for (int q = wave; q < ntiles; q += 4) {  // wave-uniform
          uint4 af[NK16 + 1];
#pragma unroll
          for (int p = 0; p < PF; ++p) af[p] = pre[p];
#pragma unroll
          for (int p = PF; p <= NK16; ++p) af[p] = frag(q, p);
          if (q + 4 < ntiles) {
#pragma unroll
            for (int p = 0; p < PF; ++p) pre[p] = frag(q + 4, p);
          }
          f32x16_t acc = f32x16_t{};
#pragma unroll
          for (int p = 0; p <= NK16; ++p) acc = mfma32x32x16(af[p], bq[p], acc);
          uint32_t hit = 0;
#pragma unroll
          for (int e = 0; e < 16; ++e) hit |= acc[e] <= cthr ? (1u << e) : 0u;
          for (uint32_t h = hit; h; h &= h - 1u) {
            const int e = __builtin_ctz(h);
            const int idx = atomicAdd(&cand_cnt[ctl], 1);
            if (idx < RQ_CAP) cand[ctl][idx] = (uint16_t)(q * 32 + rq_row(e, half));
          }
        }
      }
      __syncthreads();  // every list is complete, stages 0 and 1 are read
      // ---- exact fp32 rescoring of the open tokens, wave by wave (each wave
      // its own 32), a batch of up to 8 tokens at a time: their residuals go
      // to the wave's share of stage 2, their (token, codeword) pairs are
      // listed one per lane, and the wave scores G = 8 pairs per step, each
      // lane holding R / 64 coordinates of a pair (coalesced codeword rows),
      // with one reduction for all G pairs.  A list that overflowed stands
      // for every codeword of the round.
      constexpr int PER = R / 64, NB = 8, G = 8;
      static_assert(NB * R * 4 <= CBLK * 1024, "a batch of residuals fits the wave's share of a stage");
      static_assert(NB * RQ_CAP <= 128, "two pairs per lane");
      float* stg = reinterpret_cast<float*>(s2) + wave * (CBLK * 256);
      const float* Cl = a.C + (int64_t)l * a.K * R;
      uint32_t pend = (uint32_t)__ballot(half == 0 && open);
      const int u_own = lane & 31;
      int* dec = sm.dec[wave];
      // lane of the full sum of pair g after the reduction below
      auto glane = [](int g) { return 32 * (g >> 2) + 16 * ((g >> 1) & 1) + 8 * (g & 1); };
      while (pend) {  // wave-uniform
        uint32_t rest = pend;
#pragma unroll
        for (int i = 0; i < NB; ++i) rest &= rest - 1u;
        const uint32_t bm = pend & ~rest;
        pend = rest;
        const int nb = __popc(bm);
        const bool mine = (bm >> u_own) & 1u;
        const int slot = __popc(bm & ((1u << u_own) - 1u));
        if (mine) {
          float* rw = stg + slot * R + 8 * half;
#pragma unroll
          for (int s = 0; s < NK16; ++s) {
            *(float4*)(rw + 16 * s) = make_float4(res[s][0], res[s][1], res[s][2], res[s][3]);
            *(float4*)(rw + 16 * s + 4) = make_float4(res[s][4], res[s][5], res[s][6], res[s][7]);
          }
        }
        // lane i < nb: the token of batch slot i and its list length
        int tok = 0, cnt = 0;
        if (lane < nb) {
          uint32_t m = bm;
          for (int i = 0; i < lane; ++i) m &= m - 1u;
          tok = wave * 32 + __builtin_ctz(m);
          cnt = cand_cnt[tok];
        }
        // the slots' first pairs (scalar): listed pairs only, overflowed
        // lists apart
        int bs[NB];
        int npairs = 0;
        uint32_t ovm = 0;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int ci = __builtin_amdgcn_readlane(cnt, i);
          bs[i] = npairs;
          if (i < nb && ci > RQ_CAP) ovm |= 1u << i;
          npairs += (i < nb && ci <= RQ_CAP) ? ci : 0;
        }
        // pair p = lane + 64 h: (slot << 16) | codeword
        uint32_t pj[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int p = lane + 64 * h;
          int sl = 0, b0 = 0;
#pragma unroll
          for (int i = 1; i < NB; ++i)
            if (i < nb && p >= bs[i]) {
              sl = i;
              b0 = bs[i];
            }
          const int tk = __shfl(tok, sl, WAVE);
          pj[h] = p < npairs ? ((uint32_t)sl << 16) | (uint32_t)cand[tk][p - b0] : 0xFFFFFFFFu;
        }
        float best = INFINITY;
        int bj = 0x7fffffff;
        float cv[G][PER];
        int sg[G], jg[G];
        // request the rows of G pairs given by pair(g) = (slot, codeword),
        // slot -1 for none
        auto load = [&](auto&& pair) {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            pair(g, sg[g], jg[g]);
            const int jl = sg[g] >= 0 ? jg[g] : 0;
            const float* src = Cl + (int64_t)jl * R + PER * lane;
            if constexpr (PER == 4) {
              const float4 v = *(const float4*)src;
              cv[g][0] = v.x; cv[g][1] = v.y; cv[g][2] = v.z; cv[g][3] = v.w;
            } else if constexpr (PER == 2) {
              const float2 v = *(const float2*)src;
              cv[g][0] = v.x; cv[g][1] = v.y;
            } else {
              cv[g][0] = *src;
            }
          }
        };
        // score the requested pairs and keep each slot's best (lane = slot),
        // ties to the lower index
        auto score = [&]() {
          float v8[G];
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float* rsrc = stg + (sg[g] >= 0 ? sg[g] : 0) * R + PER * lane;
            float d = 0.f;
#pragma unroll
            for (int e = 0; e < PER; ++e) {
              const float df = rsrc[e] - cv[g][e];
              d = fmaf(df, df, d);
            }
            v8[g] = d;
          }
          // all G sums at once: the steps over lane bits 5, 4, 3 halve the
          // values a lane holds, then bits 2, 1, 0 finish the single one
          float w4[4], w2[2];
          const int b5 = (lane >> 5) & 1, b4 = (lane >> 4) & 1, b3 = (lane >> 3) & 1;
#pragma unroll
          for (int t = 0; t < 4; ++t) w4[t] = (b5 ? v8[4 + t] : v8[t]) + __shfl_xor(b5 ? v8[t] : v8[4 + t], 32, WAVE);
#pragma unroll
          for (int t = 0; t < 2; ++t) w2[t] = (b4 ? w4[2 + t] : w4[t]) + __shfl_xor(b4 ? w4[t] : w4[2 + t], 16, WAVE);
          float y = (b3 ? w2[1] : w2[0]) + __shfl_xor(b3 ? w2[0] : w2[1], 8, WAVE);
          y += __shfl_xor(y, 4, WAVE);
          y += __shfl_xor(y, 2, WAVE);
          y += __shfl_xor(y, 1, WAVE);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float dg = __shfl(y, glane(g), WAVE);
            if (sg[g] >= 0 && lane == sg[g] && (dg < best || (dg == best && jg[g] < bj))) {
              best = dg;
              bj = jg[g];
            }
          }
        };
        auto listed = [&](int p0) {
          return [&, p0](int g, int& sl, int& j) {
            const int p = p0 + g;
            const uint32_t e = p < 64 ? (uint32_t)__builtin_amdgcn_readlane((int)pj[0], p & 63)
                                      : (uint32_t)__builtin_amdgcn_readlane((int)pj[1], p & 63);
            const bool ok = p < npairs && (int)(e & 0xFFFFu) < a.K;
            sl = ok ? (int)(e >> 16) : -1;
            j = (int)(e & 0xFFFFu);
          };
        };
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        for (int p0 = 0; p0 < npairs; p0 += G) {  // wave-uniform
          load(listed(p0));
          score();
        }
        for (uint32_t ov = ovm; ov; ov &= ov - 1u) {  // overflowed lists: every codeword
          const int si = __builtin_ctz(ov);
          for (int q0 = 0; q0 < a.K; q0 += G) {
            load([&](int g, int& sl, int& j) {
              j = q0 + g;
              sl = j < a.K ? si : -1;
            });
            score();
          }
        }
        if (lane < nb) dec[lane] = bj < a.K ? bj : 0;  // bj >= K only with non-finite inputs
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (mine) jstar = dec[slot];
        if (a.stats && lane == 0) {
          atomicAdd(&a.stats[0], nb);
          atomicAdd(&a.stats[1], npairs);
          if (ovm) atomicAdd(&a.stats[2], __popc(ovm));
        }
        __builtin_amdgcn_wave_barrier();  // dec and the staging rows are reused by the next batch
      }
    }
    if (jstar < 0 || jstar >= a.K) jstar = 0;  // only reachable with non-finite inputs
    if (l + 1 < a.L) {
      // every wave is past this round's last stage barrier (and the
      // rescoring's), so stages 0 and 1 are free
      issue_l(l + 1, 0, s0);
      issue_l(l + 1, 1, s1);
      const float* cw = a.C + ((int64_t)l * a.K + jstar) * R + 8 * half;
#pragma unroll
      for (int s = 0; s < NK16; ++s) {
        const float4 p0 = *(const float4*)(cw + 16 * s), p1 = *(const float4*)(cw + 16 * s + 4);
        if (valid) {
          res[s][0] -= p0.x; res[s][1] -= p0.y; res[s][2] -= p0.z; res[s][3] -= p0.w;
          res[s][4] -= p1.x; res[s][5] -= p1.y; res[s][6] -= p1.z; res[s][7] -= p1.w;
        }
      }
    }
    if (half == 0 && valid) {
      if (a.code_bytes == 1)
        ((uint8_t*)a.codes)[(int64_t)t * a.L + l] = (uint8_t)jstar;
      else
        ((uint16_t*)a.codes)[(int64_t)t * a.L + l] = (uint16_t)jstar;
    }
    // no barrier: the next round's shared state (cand_cnt, cand, the
    // compacted tokens' table;
    // dec and the staging rows, which only the token's own wave touches) is
    // written after barriers that every wave reaches only once done with
    // this round
  }
}

template <int R>
__global__ __launch_bounds__(RQ_THREADS) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_rvq(RvqArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature (launch stub)
  __shared__ __attribute__((aligned(1024))) RqStage<R> S0;
  __shared__ __attribute__((aligned(1024))) RqStage<R> S1;
  __shared__ __attribute__((aligned(1024))) RqStage<R> S2;
  __shared__ RqSmall sm;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int t = blockIdx.x * RQ_TOK + (threadIdx.x >> 6) * 32 + (lane & 31);
  float res[R / 16][8];
#pragma unroll
  for (int s = 0; s < R / 16; ++s) {
    float4 z0 = make_float4(0.f, 0.f, 0.f, 0.f), z1 = z0;
    if (t < a.T) {
      const float4* zp = (const float4*)(a.Z0 + (int64_t)t * R + 16 * s + 8 * half);
      z0 = zp[0];
      z1 = zp[1];
    }
    res[s][0] = z0.x; res[s][1] = z0.y; res[s][2] = z0.z; res[s][3] = z0.w;
    res[s][4] = z1.x; res[s][5] = z1.y; res[s][6] = z1.z; res[s][7] = z1.w;
  }
  rvq_rounds<R>(a, S0.c, S1.c, S2.c, sm, res);
#endif
}

// Encoder in one launch for r = 256: the projection Z0 = [X | a] W of the
// workgroup's 128 tokens (the GEMM's K loop, one 128 x 256 tile), handed
// to the RVQ rounds through LDS instead of HBM, so the unquantised
// coordinates never leave the CU.  The GEMM's three stage buffers hold the
// fp32 tile (row t of 1 KiB: stage t / 48, 16 B chunks XOR-swizzled by
// t % 8 so 8 consecutive rows hit distinct bank groups) and then serve as
// the RVQ's codebook stages.
constexpr int FU_R = 256;
static_assert(sizeof(RqStage<FU_R>) <= sizeof(TnSmem<FU_R>), "RVQ stages fit the GEMM stages");
static_assert(sizeof(RqStage<FU_R>) <= (GM + FU_R) * GK * sizeof(bf16_t), "RVQ stage 2 fits the third GEMM stage");
static_assert(GM == RQ_TOK, "one token block");

template <bool FULLK>
__global__ __launch_bounds__(RQ_THREADS) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_enc_rvq(TnArgs g,
                                                                                                    RvqArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int R = FU_R, NK16 = R / 16;
  __shared__ __attribute__((aligned(1024))) TnSmem<R> S0;
  __shared__ __attribute__((aligned(1024))) TnSmem<R> S1;
  __shared__ __attribute__((aligned(1024))) bf16_t S2buf[(GM + R) * GK];
  __shared__ RqSmall sm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  constexpr int ROWS = (int)(sizeof(TnSmem<R>) / 1024);  // 1 KiB fp32 rows per stage buffer
  static_assert(3 * ROWS >= GM, "the tile fits the stage buffers");
  auto hrow = [&](int t) -> uint32_t {
    return t < ROWS ? lds_addr(&S0) + (uint32_t)t * 1024u
                    : t < 2 * ROWS ? lds_addr(&S1) + (uint32_t)(t - ROWS) * 1024u
                                   : lds_addr(S2buf) + (uint32_t)(t - 2 * ROWS) * 1024u;
  };
  tn_mainloop<R, 3, FULLK, false>(g, 1, S0.a, S0.w, S1.a, S1.w, S2buf, S2buf + GM * GK,
                           [&](f32x16_t (&acc)[2][R / 64], int) {
                             __syncthreads();  // every wave is done reading the stages
                             const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
                             for (int i = 0; i < 2; ++i) {
                               const int row = wm * 64 + i * 32 + (lane & 31);
                               const uint32_t base = hrow(row);
                               const int sw = row & 7;
#pragma unroll
                               for (int j = 0; j < R / 64; ++j) {
#pragma unroll
                                 for (int q = 0; q < 4; ++q) {
                                   // columns 128 wn + 32 j + 8 q + 4 half + 0..3
                                   const int ch = wn * 32 + 8 * j + 2 * q + half;
                                   lds_write_b128(base + 16u * (uint32_t)(ch ^ sw),
                                                  u32x4{__float_as_uint(acc[i][j][4 * q]),
                                                        __float_as_uint(acc[i][j][4 * q + 1]),
                                                        __float_as_uint(acc[i][j][4 * q + 2]),
                                                        __float_as_uint(acc[i][j][4 * q + 3])});
                                 }
                                 acc[i][j] = f32x16_t{};
                               }
                             }
                           });
  lds_wait0();
  __syncthreads();  // the tile is in LDS
  float res[NK16][8];
  {
    const int row = wave * 32 + (lane & 31), sw = row & 7;
    const uint32_t base = hrow(row);
#pragma unroll
    for (int s0 = 0; s0 < NK16; s0 += 4) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        // columns 16 (s0 + u) + 8 half + 0..7: chunks 4 (s0 + u) + 2 half (+1)
        const int ch = 4 * (s0 + u) + 2 * half;
        v[2 * u] = lds_read_b128(base + 16u * (uint32_t)(ch ^ sw));
        v[2 * u + 1] = lds_read_b128(base + 16u * (uint32_t)((ch + 1) ^ sw));
      }
      lds_wait(v);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          res[s0 + u][e] = __uint_as_float(v[2 * u][e]);
          res[s0 + u][4 + e] = __uint_as_float(v[2 * u + 1][e]);
        }
    }
  }
  __syncthreads();  // the stages are free for the codebook
  rvq_rounds<R>(a, S0.a, S1.a, S2buf, sm, res);
#endif
}

}  // namespace

bool enc_rvq_fusable(int r, int L) { return r == FU_R && L >= 1 && L <= RQ_LMAX; }

hipError_t launch_enc_rvq(const TnArgs& g, const RvqArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (!enc_rvq_fusable(a.r, a.L) || g.N != FU_R || g.M != a.T || g.kz != 0) return hipErrorInvalidValue;
  if (g.Ka % 32 || g.Kg % 16 || g.Ka + g.Kg > g.ldw || g.lda % 8 || g.ldt % 8 || g.ldw % 8)
    return hipErrorInvalidValue;
  const bool fullk = g.Ka % GK == 0 && g.Kg % GK == 0;
  dim3 grid((a.T + RQ_TOK - 1) / RQ_TOK);
  if (fullk)
    hipLaunchKernelGGL(k_enc_rvq<true>, grid, dim3(RQ_THREADS), 0, s, g, a);
  else
    hipLaunchKernelGGL(k_enc_rvq<false>, grid, dim3(RQ_THREADS), 0, s, g, a);
  return hipGetLastError();
}

hipError_t launch_rvq(const RvqArgs& a, hipStream_t s) {
  if (a.T <= 0 || a.L <= 0) return hipSuccess;
  if (a.L > RQ_LMAX) return hipErrorInvalidValue;
  dim3 grid((a.T + RQ_TOK - 1) / RQ_TOK);
  switch (a.r) {
    case 64: hipLaunchKernelGGL(k_rvq<64>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 128: hipLaunchKernelGGL(k_rvq<128>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 256: hipLaunchKernelGGL(k_rvq<256>, grid, dim3(RQ_THREADS), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mapl
