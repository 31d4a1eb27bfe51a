// Residual vector quantisation of the projected coordinates (Sec. 3.5):
// L rounds; round l picks, per token, the codeword of C_l nearest to the
// current residual R_l and subtracts it.  Ties go to the lowest index.
//
// Decision procedure (exact with respect to the fp32 residual):
//   screen  s~_j = ||C_j||^2 - 2 R~ . C~_j on the bf16 matrix units, with
//           R~ = bf16(R), C~ = bf16(C), fp32 accumulation.  The true
//           s_j = ||C_j||^2 - 2 R.C_j obeys |s~_j - s_j| <= delta_j with
//           delta_j = kappa ||R|| ||C_j|| + kappa2 ||C_j||^2 (bf16 rounding of
//           both operands, fp32 accumulation and the final fused add; the
//           constants carry a safety factor, see rvq_margin()).
//   bound   U* = min_j (s~_j + delta_j) >= min_j s_j; the nearest codeword is
//           among {j : s~_j - delta_j <= U*}.
//   pass 1  tracks U*, the smallest and second-smallest lower bound; if the
//           second-smallest exceeds U* the candidate set is a single
//           codeword and the decision is final.
//   pass 2  (only when a token of the workgroup is ambiguous) re-screens
//           and lists every candidate; the candidates are rescored exactly
//           in fp32 as sum_c (R_c - C_jc)^2.
// The residual is rebuilt in fp32 for every round from Z0 and the codes
// already chosen, so screening and rescoring see the same R.
//
// Layout: a workgroup of 4 waves owns 128 tokens, 32 per wave.  A wave keeps
// its tokens' bf16 residual as the B operand of v_mfma_f32_32x32x16_bf16 in
// registers (tokens along N); 64-codeword chunks of C~ stream through three
// LDS stages filled by buffer_load ... lds (direct-to-LDS, one __shared__
// array per stage) as the A operand (codewords along M), together with the
// chunk's per-codeword screen constants (||C||^2, ||C||, kappa2 ||C||^2).
// Each lane thus sees the scores of ONE token for 16 codewords per tile and
// tracks its bounds in registers; only the two lane halves that share a
// token merge at the end of a pass.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

typedef __attribute__((address_space(3))) void* rq_lds_ptr;
constexpr int RQ_THREADS = 256, RQ_TOK = 128, RQ_CW = 64, RQ_CAP = 16, RQ_LMAX = 8;
constexpr uint32_t RQ_OOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rq_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0x7fffffffull ? 0x7fffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n, 0x00020000);
}

template <int R>
struct RqStage {
  bf16_t c[RQ_CW * R];   // codewords, 2R bytes per row, 16 B chunks XOR-swizzled by row
  float meta[4][256];    // per wave: [n2 | cnr | n2k] x 64 codewords (wave-private copy)
};

__device__ __forceinline__ int load_code(const void* codes, int cb, int64_t idx) {
  return cb == 1 ? ((const uint8_t*)codes)[idx] : ((const uint16_t*)codes)[idx];
}

template <int R>
__global__ __launch_bounds__(RQ_THREADS) void k_rvq(RvqArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature (launch stub)
  constexpr int NK16 = R / 16;
  constexpr int CPR = R / 8;                       // 16 B chunks per codeword row
  constexpr int CBLK = RQ_CW * CPR / 64 / 4;       // 1 KiB DMA blocks per wave per stage
  constexpr int LOADS = CBLK + 1;                  // + the wave's meta copy
  __shared__ __attribute__((aligned(1024))) RqStage<R> S0;
  __shared__ __attribute__((aligned(1024))) RqStage<R> S1;
  __shared__ __attribute__((aligned(1024))) RqStage<R> S2;
  __shared__ uint16_t codes_s[RQ_TOK][RQ_LMAX];
  __shared__ int cand_cnt[RQ_TOK];
  __shared__ uint16_t cand[RQ_TOK][RQ_CAP];
  __shared__ int amb_s[RQ_TOK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int tl = wave * 32 + (lane & 31);  // token within the workgroup
  const int t = blockIdx.x * RQ_TOK + tl;
  const bool valid = t < a.T;
  const int nchunks = (a.K + RQ_CW - 1) / RQ_CW;
  const int total = (nchunks + 2) / 3 * 3;       // padded: stage buffers repeat every pass

  // DMA geometry (codeword chunk): lane i of block b writes row b*rpb + i/CPR,
  // physical chunk i%CPR holding logical chunk (i%CPR) ^ (row & 15 & (CPR-1)):
  // 16 consecutive rows read one logical chunk from 16 different bank groups.
  constexpr int RPB = 64 / CPR;
  uint32_t c_off[CBLK];
#pragma unroll
  for (int jb = 0; jb < CBLK; ++jb) {
    const int b = wave * CBLK + jb;
    const int row = b * RPB + lane / CPR;
    const int lch = (lane % CPR) ^ (row & 15 & (CPR - 1));
    c_off[jb] = (uint32_t)row * (uint32_t)(R * 2) + (uint32_t)lch * 16u;
  }

  for (int l = 0; l < a.L; ++l) {
    const __amdgpu_buffer_rsrc_t rc = rq_rsrc(a.Cb + (int64_t)l * a.K * R, (uint64_t)a.K * R * 2);
    const __amdgpu_buffer_rsrc_t rm = rq_rsrc(a.meta + (int64_t)l * nchunks * 192, (uint64_t)nchunks * 192 * 4);

    auto issue = [&](int q, bf16_t* sc, float* smeta) {
      const bool pad = q >= nchunks;
#pragma unroll
      for (int jb = 0; jb < CBLK; ++jb) {
        const int row = (wave * CBLK + jb) * RPB + lane / CPR;
        const bool ok = !pad && q * RQ_CW + row < a.K;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (rq_lds_ptr)(sc + (wave * CBLK + jb) * 512), 16,
                                                 ok ? (uint32_t)(q * RQ_CW) * (uint32_t)(R * 2) + c_off[jb] : RQ_OOB,
                                                 0, 0, 0);
      }
      // 768 B of constants: lanes 0..47 carry 16 B each, the rest read zeros
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rm, (rq_lds_ptr)(smeta + wave * 256), 16,
                                               (!pad && lane < 48) ? (uint32_t)q * 768u + (uint32_t)lane * 16u
                                                                   : RQ_OOB,
                                               0, 0, 0);
    };

    // ---- residual R_l in fp32 (B-fragment layout), its bf16 image and norm;
    // the first two codebook chunks are already in flight meanwhile
    issue(0, S0.c, &S0.meta[0][0]);
    issue(1, S1.c, &S1.meta[0][0]);
    uint4 rb[NK16];
    float rn2 = 0.f;
#pragma unroll
    for (int s = 0; s < NK16; ++s) {
      float v[8];
      const int c0 = 16 * s + 8 * half;
      if (valid) {
        const float4* zp = (const float4*)(a.Z0 + (int64_t)t * R + c0);
        float4 z0 = zp[0], z1 = zp[1];
        v[0] = z0.x; v[1] = z0.y; v[2] = z0.z; v[3] = z0.w;
        v[4] = z1.x; v[5] = z1.y; v[6] = z1.z; v[7] = z1.w;
        for (int i = 0; i < l; ++i) {
          const float4* cw = (const float4*)(a.C + ((int64_t)i * a.K + codes_s[tl][i]) * R + c0);
          const float4 p0 = cw[0], p1 = cw[1];
          v[0] -= p0.x; v[1] -= p0.y; v[2] -= p0.z; v[3] -= p0.w;
          v[4] -= p1.x; v[5] -= p1.y; v[6] -= p1.z; v[7] -= p1.w;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) rn2 += v[e] * v[e];
      rb[s] = make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
    }
    rn2 += __shfl_xor(rn2, 32, WAVE);
    const float kappa = rvq_margin_k1(R) * sqrtf(rn2) * 1.0001f;

    // One screening pass over all chunks; fn(j, score, margin) per codeword.
    auto pass = [&](auto&& fn, bool first) {
      if (!first) {
        issue(0, S0.c, &S0.meta[0][0]);
        issue(1, S1.c, &S1.meta[0][0]);
      }
      auto stage = [&](int q, const bf16_t* sc, const float* smeta, bf16_t* nc, float* nmeta) {
        if (q + 1 < total)
          asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS) : "memory");
        else
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        if (q + 2 < total) issue(q + 2, nc, nmeta);
        if (q >= nchunks) return;
        const float* mw = smeta + wave * 256;
#pragma unroll
        for (int ct = 0; ct < RQ_CW / 32; ++ct) {
          if (q * RQ_CW + ct * 32 >= a.K) continue;  // K % 32 == 0: whole tile valid or not
          f32x16_t acc = f32x16_t{};
#pragma unroll
          for (int s = 0; s < NK16; ++s) {
            const int row = ct * 32 + (lane & 31);
            const int lch = (2 * s + half) ^ (row & 15 & (CPR - 1));
            const uint4 af = *(const uint4*)(sc + row * R + lch * 8);
            acc = mfma32x32x16(af, rb[s], acc);
          }
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4) {
            const int jl0 = ct * 32 + 8 * e4 + 4 * half;  // rows jl0..jl0+3 of this lane
            const float4 n2 = *(const float4*)(mw + jl0);
            const float4 cr = *(const float4*)(mw + 64 + jl0);
            const float4 nk = *(const float4*)(mw + 128 + jl0);
            const float n2v[4] = {n2.x, n2.y, n2.z, n2.w}, crv[4] = {cr.x, cr.y, cr.z, cr.w},
                        nkv[4] = {nk.x, nk.y, nk.z, nk.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float sc2 = fmaf(-2.f, acc[4 * e4 + e], n2v[e]);
              const float dl = fmaf(kappa, crv[e], nkv[e]);
              fn(q * RQ_CW + jl0 + e, sc2, dl);
            }
          }
        }
      };
      for (int q = 0; q < total; q += 3) {
        stage(q, S0.c, &S0.meta[0][0], S2.c, &S2.meta[0][0]);
        stage(q + 1, S1.c, &S1.meta[0][0], S0.c, &S0.meta[0][0]);
        stage(q + 2, S2.c, &S2.meta[0][0], S1.c, &S1.meta[0][0]);
      }
    };

    // ---- pass 1
    float ub_min = INFINITY, lb1 = INFINITY, lb2 = INFINITY;
    int j1 = 0;
    pass(
        [&](int j, float sc, float dl) {
          const float ub = sc + dl, lb = sc - dl;
          ub_min = fminf(ub_min, ub);
          lb2 = fminf(lb2, fmaxf(lb1, lb));
          const bool better = lb < lb1;
          j1 = better ? j : j1;
          lb1 = fminf(lb1, lb);
        },
        true);
    {
      const float o_ub = __shfl_xor(ub_min, 32, WAVE);
      const float o_lb1 = __shfl_xor(lb1, 32, WAVE);
      const float o_lb2 = __shfl_xor(lb2, 32, WAVE);
      const int o_j1 = __shfl_xor(j1, 32, WAVE);
      ub_min = fminf(ub_min, o_ub);
      const float nlb2 = fminf(fmaxf(lb1, o_lb1), fminf(lb2, o_lb2));
      if (o_lb1 < lb1 || (o_lb1 == lb1 && o_j1 < j1)) j1 = o_j1;
      lb1 = fminf(lb1, o_lb1);
      lb2 = nlb2;
    }
    const bool amb = valid && !(lb2 > ub_min);
    if (half == 0) {
      amb_s[tl] = amb ? 1 : 0;
      cand_cnt[tl] = 0;
    }
    const int any_amb = __syncthreads_or(amb ? 1 : 0);

    int jstar = j1;
    if (any_amb) {
      // ---- pass 2: list every candidate of the ambiguous tokens
      const float ustar = ub_min;
      pass(
          [&](int j, float sc, float dl) {
            if (amb && sc - dl <= ustar) {
              const int idx = atomicAdd(&cand_cnt[tl], 1);
              if (idx < RQ_CAP) cand[tl][idx] = (uint16_t)j;
            }
          },
          false);
      // ---- exact fp32 rescoring, one wave per token of its own 32
      for (int u = 0; u < 32; ++u) {
        const int tu = wave * 32 + u;
        if (!amb_s[tu]) continue;  // wave-uniform
        const int tg = blockIdx.x * RQ_TOK + tu;
        constexpr int PER = (R + 63) / 64;
        float rv[PER];
#pragma unroll
        for (int p = 0; p < PER; ++p) {
          const int c = lane + 64 * p;
          float v = 0.f;
          if (c < R) {
            v = a.Z0[(int64_t)tg * R + c];
            for (int i = 0; i < l; ++i) v -= a.C[((int64_t)i * a.K + codes_s[tu][i]) * R + c];
          }
          rv[p] = v;
        }
        const float* Cl = a.C + (int64_t)l * a.K * R;
        auto dist = [&](int j) {
          float s = 0.f;
#pragma unroll
          for (int p = 0; p < PER; ++p) {
            const int c = lane + 64 * p;
            if (c < R) {
              const float df = rv[p] - Cl[(int64_t)j * R + c];
              s = fmaf(df, df, s);
            }
          }
          return wave_sum(s);
        };
        const int cnt = cand_cnt[tu];
        float best = INFINITY;
        int bj = 0x7fffffff;
        if (cnt <= RQ_CAP) {
          for (int q = 0; q < cnt; ++q) {
            const int j = cand[tu][q];
            const float dd = dist(j);
            if (dd < best || (dd == best && j < bj)) { best = dd; bj = j; }
          }
        } else {
          for (int j = 0; j < a.K; ++j) {
            const float dd = dist(j);
            if (dd < best) { best = dd; bj = j; }
          }
        }
        if (bj >= a.K) bj = 0;  // only reachable with non-finite inputs
        if (lane == 0) {
          cand_cnt[tu] = bj;  // reuse as the decision slot
          if (a.stats) {
            atomicAdd(&a.stats[0], 1);
            atomicAdd(&a.stats[1], cnt);
            if (cnt > RQ_CAP) atomicAdd(&a.stats[2], 1);
          }
        }
      }
      __syncthreads();
      if (amb) jstar = cand_cnt[tl];
    }
    if (half == 0 && valid) {
      codes_s[tl][l] = (uint16_t)jstar;
      if (a.code_bytes == 1)
        ((uint8_t*)a.codes)[(int64_t)t * a.L + l] = (uint8_t)jstar;
      else
        ((uint16_t*)a.codes)[(int64_t)t * a.L + l] = (uint16_t)jstar;
    }
    __syncthreads();
  }
#endif
}

}  // namespace

hipError_t launch_rvq(const RvqArgs& a, hipStream_t s) {
  if (a.T <= 0 || a.L <= 0) return hipSuccess;
  if (a.L > RQ_LMAX) return hipErrorInvalidValue;
  dim3 grid((a.T + RQ_TOK - 1) / RQ_TOK);
  switch (a.r) {
    case 32: hipLaunchKernelGGL(k_rvq<32>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 64: hipLaunchKernelGGL(k_rvq<64>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 128: hipLaunchKernelGGL(k_rvq<128>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 256: hipLaunchKernelGGL(k_rvq<256>, grid, dim3(RQ_THREADS), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mapl
