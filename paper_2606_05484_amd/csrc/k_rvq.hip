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
//           constants below carry a safety factor).
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
// registers (tokens along N), and streams 64-codeword chunks of C~ through
// LDS as the A operand (codewords along M).  Each lane therefore sees the
// scores of ONE token for 16 codewords per tile, and tracks its bounds in
// registers without cross-lane traffic; only the two lane halves that share
// a token merge at the end of a pass.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int RQ_THREADS = 256, RQ_TOK = 128, RQ_CW = 64, RQ_CAP = 16, RQ_LMAX = 8;

template <int R>
struct RvqConsts {
  // 2 * (2^-7 (bf16 rounding of both operands) + R 2^-24 (fp32 accumulation))
  // plus the rounding of the fused add and of the fp32 norms, inflated.
  static constexpr float K1 = 0.015625f * 1.0078125f + 8.0f * R / 16777216.0f + 1.0f / 1048576.0f;
  static constexpr float K2 = 4.0f * (R + 2) / 16777216.0f;
};

__device__ __forceinline__ int load_code(const void* codes, int cb, int64_t idx) {
  return cb == 1 ? ((const uint8_t*)codes)[idx] : ((const uint16_t*)codes)[idx];
}

template <int R>
__global__ __launch_bounds__(RQ_THREADS) void k_rvq(RvqArgs a) {
  constexpr int NK16 = R / 16;
  constexpr int LDC = R + 8;
  constexpr int CCH = RQ_CW * R / 8 / RQ_THREADS;  // 16 B chunks per thread per codebook chunk
  static_assert(CCH >= 1, "chunk");
  __shared__ __attribute__((aligned(16))) bf16_t Cs[2][RQ_CW][LDC];
  __shared__ float cn2s[2][RQ_CW], cnrs[2][RQ_CW];
  __shared__ uint16_t codes_s[RQ_TOK][RQ_LMAX];
  __shared__ int cand_cnt[RQ_TOK];
  __shared__ uint16_t cand[RQ_TOK][RQ_CAP];
  __shared__ float ustar_s[RQ_TOK];
  __shared__ int amb_s[RQ_TOK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int tl = wave * 32 + (lane & 31);  // token within the workgroup
  const int t = blockIdx.x * RQ_TOK + tl;
  const bool valid = t < a.T;
  const int nchunks = (a.K + RQ_CW - 1) / RQ_CW;

  for (int l = 0; l < a.L; ++l) {
    const bf16_t* Cbl = a.Cb + (int64_t)l * a.K * R;
    const float* cn2l = a.cn2 + (int64_t)l * a.K;
    const float* cnrl = a.cnrm + (int64_t)l * a.K;

    // ---- residual R_l in fp32 (B-fragment layout), its bf16 image and norm
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
          const float* cw = a.C + ((int64_t)i * a.K + codes_s[tl][i]) * R + c0;
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] -= cw[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) rn2 += v[e] * v[e];
      rb[s] = make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]),
                         pack_bf2(v[6], v[7]));
    }
    rn2 += __shfl_xor(rn2, 32, WAVE);
    const float kappa = RvqConsts<R>::K1 * sqrtf(rn2) * 1.0001f;
    constexpr float kappa2 = RvqConsts<R>::K2;

    // ---- codebook chunk loader (cooperative, register-prefetched)
    uint4 pre[CCH];
    float pre_n2 = 0.f, pre_nr = 0.f;
    auto fetch = [&](int q) {
#pragma unroll
      for (int i = 0; i < CCH; ++i) {
        const int c = tid + i * RQ_THREADS;
        const int row = c / (R / 8), col = (c % (R / 8)) * 8;
        const int j = q * RQ_CW + row;
        pre[i] = j < a.K ? *(const uint4*)(Cbl + (int64_t)j * R + col) : make_uint4(0, 0, 0, 0);
      }
      if (tid < RQ_CW) {
        const int j = q * RQ_CW + tid;
        pre_n2 = j < a.K ? cn2l[j] : 0.f;
        pre_nr = j < a.K ? cnrl[j] : 0.f;
      }
    };
    auto commit = [&](int buf) {
#pragma unroll
      for (int i = 0; i < CCH; ++i) {
        const int c = tid + i * RQ_THREADS;
        const int row = c / (R / 8), col = (c % (R / 8)) * 8;
        *(uint4*)&Cs[buf][row][col] = pre[i];
      }
      if (tid < RQ_CW) {
        cn2s[buf][tid] = pre_n2;
        cnrs[buf][tid] = pre_nr;
      }
    };

    // Runs the screen over all codewords; fn(j, screen score) per score.
    auto screen = [&](auto&& fn) {
      fetch(0);
      commit(0);
      __syncthreads();
      for (int q = 0; q < nchunks; ++q) {
        const int buf = q & 1;
        if (q + 1 < nchunks) fetch(q + 1);
#pragma unroll
        for (int ct = 0; ct < RQ_CW / 32; ++ct) {
          f32x16_t acc = f32x16_t{};
#pragma unroll
          for (int s = 0; s < NK16; ++s) {
            const uint4 af = *(const uint4*)&Cs[buf][ct * 32 + (lane & 31)][16 * s + 8 * half];
            acc = mfma32x32x16(af, rb[s], acc);
          }
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int jl = ct * 32 + acc_row(e, lane);
            const int j = q * RQ_CW + jl;
            if (j < a.K) {
              const float n2 = cn2s[buf][jl];
              const float sc = fmaf(-2.f, acc[e], n2);
              const float dl = fmaf(kappa, cnrs[buf][jl], kappa2 * n2);
              fn(j, sc, dl);
            }
          }
        }
        if (q + 1 < nchunks) commit(buf ^ 1);
        __syncthreads();
      }
    };

    // ---- pass 1
    float ub_min = INFINITY, lb1 = INFINITY, lb2 = INFINITY;
    int j1 = 0;
    screen([&](int j, float sc, float dl) {
      const float ub = sc + dl, lb = sc - dl;
      ub_min = fminf(ub_min, ub);
      lb2 = fminf(lb2, fmaxf(lb1, lb));
      const bool better = lb < lb1;
      j1 = better ? j : j1;
      lb1 = fminf(lb1, lb);
    });
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
      ustar_s[tl] = ub_min;
      amb_s[tl] = amb ? 1 : 0;
      cand_cnt[tl] = 0;
    }
    const int any_amb = __syncthreads_or(amb ? 1 : 0);

    int jstar = j1;
    if (any_amb) {
      // ---- pass 2: list every candidate of the ambiguous tokens
      const float ustar = ub_min;
      screen([&](int j, float sc, float dl) {
        if (amb && sc - dl <= ustar) {
          const int idx = atomicAdd(&cand_cnt[tl], 1);
          if (idx < RQ_CAP) cand[tl][idx] = (uint16_t)j;
        }
      });
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
}

}  // namespace

hipError_t launch_rvq(const RvqArgs& a, hipStream_t s) {
  if (a.T <= 0 || a.L <= 0) return hipSuccess;
  if (a.L > RQ_LMAX) return hipErrorInvalidValue;
  dim3 grid((a.T + RQ_TOK - 1) / RQ_TOK);
  switch (a.r) {
    case 32: hipLaunchKernelGGL(k_rvq<32>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 64: hipLaunchKernelGGL(k_rvq<64>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 96: hipLaunchKernelGGL(k_rvq<96>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 128: hipLaunchKernelGGL(k_rvq<128>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 160: hipLaunchKernelGGL(k_rvq<160>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 192: hipLaunchKernelGGL(k_rvq<192>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 224: hipLaunchKernelGGL(k_rvq<224>, grid, dim3(RQ_THREADS), 0, s, a); break;
    case 256: hipLaunchKernelGGL(k_rvq<256>, grid, dim3(RQ_THREADS), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mapl
