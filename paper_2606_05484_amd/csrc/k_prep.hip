// Per-call operand preparation and the receiver-side operand assembly.
//   prep_u          U (fp32 master) -> bf16 copies in both K-contiguous
//                   layouts the matrix units need (U~ [d,r] and U~^T [r,d])
//   transpose_into  scaled transposed copies (anchor companions into the
//                   concatenated weight operands)
//   prep_codebook   bf16 screening copy of the codebooks plus fp32 norms
//   assemble        [Zhat | a_r] rows for the lift: Zhat is the payload or
//                   the RVQ gather-sum sum_l C_l[code_l] (Sec. 3.5), a_r the
//                   receiver's anchor row (Eq. 2)
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

// 32x32 tiles through LDS so both the read of U and the write of U^T are
// coalesced.
__device__ __forceinline__ void prep_u_tile(int bx, int by, const float* __restrict__ U, int d, int r,
                                            bf16_t* __restrict__ Ub, int64_t ldub, bf16_t* __restrict__ Ut,
                                            int64_t ldut) {
  __shared__ bf16_t tile[32][33];
  const int j0 = bx * 32, c0 = by * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int y = ty; y < 32; y += 8) {
    const int j = j0 + y, c = c0 + tx;
    bf16_t v = 0;
    if (j < d && c < r) v = (bf16_t)f2bf(U[(int64_t)j * r + c]);
    tile[y][tx] = v;
    if (Ub && j < d && c < ldub) Ub[(int64_t)j * ldub + c] = (c < r) ? v : (bf16_t)0;
  }
  __syncthreads();
  if (Ut) {
    for (int y = ty; y < 32; y += 8) {
      const int c = c0 + y, j = j0 + tx;
      if (c < r && j < ldut) Ut[(int64_t)c * ldut + j] = (j < d) ? tile[tx][y] : (bf16_t)0;
    }
  }
}

__device__ __forceinline__ void transpose_tile(int bx, int by, const void* __restrict__ src, int src_f32,
                                               int rows, int cols, int64_t lds, float scale,
                                               bf16_t* __restrict__ dst, int64_t ldd, int off) {
  __shared__ float tile[32][33];
  const int i0 = by * 32, j0 = bx * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) {
    const int i = i0 + y, j = j0 + tx;
    float v = 0.f;
    if (i < rows && j < cols)
      v = src_f32 ? ((const float*)src)[(int64_t)i * lds + j] : bf2f(((const bf16_t*)src)[(int64_t)i * lds + j]);
    tile[y][tx] = v;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int j = j0 + y, i = i0 + tx;
    if (j < cols && i < rows) dst[(int64_t)j * ldd + off + i] = (bf16_t)f2bf(scale * tile[tx][y]);
  }
}

// One wave per (stage, codeword slot of a 64-codeword chunk): the bf16 copy
// with the norm columns of the RVQ screen appended (rows of r + 16), and the
// fp32 squared norm, laid out per chunk as 64 consecutive floats.  A squared
// norm x is stored as hi = bf16(x), mid = bf16(x - hi), lo = bf16(x - hi -
// mid); each difference is exact in fp32 and an fp32 value has 24
// significant bits, so hi + mid + lo = x exactly, in any order of addition.
__device__ __forceinline__ void prep_codebook_block(int bx, const float* __restrict__ C, int L, int K, int r,
                                                    bf16_t* __restrict__ Cb, float* __restrict__ meta) {
  const int nch = (K + 63) / 64;
  const int w = bx * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (w >= L * nch * 64) return;
  const int l = w / (nch * 64), slot = w % (nch * 64);
  const int j = slot;  // codeword index within stage l
  const int cols = rvq_cb_cols(r);
  float s = 0.f, es = 0.f;
  if (j < K) {
    const float* row = C + ((int64_t)l * K + j) * r;
    for (int c = lane; c < r; c += 64) {
      const float v = row[c];
      s += v * v;
      const uint32_t vb = f2bf(v);
      const float d = v - bf2f(vb);  // the rounding error, exact in fp32
      es += d * d;
      Cb[((int64_t)l * K + j) * cols + c] = (bf16_t)vb;
    }
  }
  s = wave_sum(s);
  es = wave_sum(es);
  // ||C_j - bf16(C_j)|| rounded up: es carries at most r ulps of accumulation error
  const float eu = sqrtf(es) * (1.0f + 1.0f / 32768.0f);
  if (j < K && lane < 16) {
    // columns r .. r+2: the reduced norm n' = s - 1.01 k2 s in three pieces
    // (each difference exact in fp32, so they sum to n' exactly); columns
    // r+3, r+4: ||C_j|| rounded up, c_hi + c_lo >= sqrt(s) (1 + 2^-15), which
    // bounds the norm of the fp32 codeword above (s carries at most r ulps
    // of accumulation error); r+5: the rounding-error norm, rounded up to
    // bf16; the rest zero
    const float np = s - s * (RVQ_K2_SLACK * rvq_margin_k2(r));
    const uint32_t hi = f2bf(np);
    const float r1 = np - bf2f(hi);
    const uint32_t mid = f2bf(r1);
    const uint32_t lo = f2bf(r1 - bf2f(mid));
    const float cu = sqrtf(s) * (1.0f + 1.0f / 32768.0f);
    const uint32_t chi = f2bf(cu);
    const float cr = cu - bf2f(chi);
    // toward +infinity: up for a positive remainder, magnitude truncated for a negative one
    const uint32_t clo = cr > 0.f ? bf16_up(cr) : (__float_as_uint(cr) >> 16);
    uint32_t v = 0u;
    if (lane == 0) v = hi;
    if (lane == 1) v = mid;
    if (lane == 2) v = lo;
    if (lane == 3) v = chi;
    if (lane == 4) v = clo;
    if (lane == 5) v = bf16_up(eu);
    Cb[((int64_t)l * K + j) * cols + r + lane] = (bf16_t)v;
  }
  if (lane == 0) {
    const int64_t m = ((int64_t)l * nch + j / 64) * 64 + (j % 64);
    meta[m] = s;
    meta[(int64_t)L * nch * 64 + m] = eu;
  }
}

// One thread per (token, 8 columns): 16 B stores, independent gathers.
// Requires r % 8 == 0 and, for the anchor columns, k % 8 == 0.
__device__ __forceinline__ void assemble_block(int bx, const AssembleArgs& a) {
  const int per_row = a.ldo / 8;
  const int64_t e = (int64_t)bx * blockDim.x + threadIdx.x;
  if (e >= (int64_t)a.T * per_row) return;
  const int t = (int)(e / per_row), c0 = (int)(e % per_row) * 8;
  bf16_t* out = a.out + (int64_t)t * a.ldo + c0;
  const bool anchor_cols = a.A != nullptr && a.Bc == nullptr;
  float v[8];
  if (c0 < a.r) {
    if (a.L == 0) {
      const uint4 z = *(const uint4*)(a.Zp + (int64_t)t * a.r + c0);
      const uint32_t w[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) { v[2 * q] = bf2f(w[q] & 0xFFFFu); v[2 * q + 1] = bf2f(w[q] >> 16); }
    } else if (a.gdim == 2) {
      // grouped codes [T, L, r/2]: columns c0 .. c0 + 7 are groups
      // c0/2 .. c0/2 + 3, four code bytes per round in one load
      constexpr int LMAX = 8;
      const int G = a.r / 2;
      uint32_t cw4[LMAX];
#pragma unroll
      for (int l = 0; l < LMAX; ++l)
        if (l < a.L) cw4[l] = *(const uint32_t*)((const uint8_t*)a.codes + ((int64_t)t * a.L + l) * G + c0 / 2);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = 0.f;
#pragma unroll
      for (int l = 0; l < LMAX; ++l) {
        if (l < a.L) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            int c = (int)((cw4[l] >> (8 * q)) & 255u);
            c = c < a.K ? c : a.K - 1;
            const float2 p = *(const float2*)(a.C + ((int64_t)l * a.K + c) * a.r + c0 + 2 * q);
            v[2 * q] += p.x;
            v[2 * q + 1] += p.y;
          }
        }
      }
    } else {
      // all codes, then all codeword rows, then the sum in stage order: the
      // loads of every stage are in flight together (L <= 8)
      constexpr int LMAX = 8;
      int code[LMAX];
#pragma unroll
      for (int l = 0; l < LMAX; ++l) {
        if (l < a.L) {
          const int c = a.code_bytes == 1 ? ((const uint8_t*)a.codes)[(int64_t)t * a.L + l]
                                          : ((const uint16_t*)a.codes)[(int64_t)t * a.L + l];
          code[l] = c < a.K ? c : a.K - 1;
        }
      }
      float4 cw[LMAX][2];
#pragma unroll
      for (int l = 0; l < LMAX; ++l) {
        if (l < a.L) {
          const float4* p = (const float4*)(a.C + ((int64_t)l * a.K + code[l]) * a.r + c0);
          cw[l][0] = p[0];
          cw[l][1] = p[1];
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = 0.f;
#pragma unroll
      for (int l = 0; l < LMAX; ++l) {
        if (l < a.L) {
          const float4 p = cw[l][0], q4 = cw[l][1];
          v[0] += p.x; v[1] += p.y; v[2] += p.z; v[3] += p.w;
          v[4] += q4.x; v[5] += q4.y; v[6] += q4.z; v[7] += q4.w;
        }
      }
    }
    if (a.Bc != nullptr) {
      const bf16_t* arow = a.A + (int64_t)clamp_id(a.ids[t], a.V) * a.k;
      for (int i = 0; i < a.k; ++i) {
        const float ai = bf2f(arow[i]);
        const uint4 b = *(const uint4*)(a.Bc + (int64_t)i * a.r + c0);
        const uint32_t w[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[2 * q] = fmaf(ai, bf2f(w[q] & 0xFFFFu), v[2 * q]);
          v[2 * q + 1] = fmaf(ai, bf2f(w[q] >> 16), v[2 * q + 1]);
        }
      }
    }
    *(uint4*)out = make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
  } else if (anchor_cols && c0 < a.r + a.k) {
    const bf16_t* arow = a.A + (int64_t)clamp_id(a.ids[t], a.V) * a.k;
    *(uint4*)out = *(const uint4*)(arow + (c0 - a.r));
  } else {
    *(uint4*)out = make_uint4(0, 0, 0, 0);
  }
}

// The common decode case of assemble_block: Zhat = sum of L <= 2 codewords,
// no anchor columns (ldo == r).  One thread per 8 columns of four tokens
// (4 g .. 4 g + 3): all codes, then all codeword rows of the four tokens are
// loaded before any sum, so a thread has up to sixteen independent loads in
// flight and a quarter of the threads cover the rows.  Same sums in the same
// order as assemble_block.
__device__ __forceinline__ void assemble_sum_block(int bx, const AssembleArgs& a) {
  constexpr int TPT = 4, LM = 2;
  const int per_row = a.r / 8;
  const int64_t e = (int64_t)bx * blockDim.x + threadIdx.x;
  if (e >= ((int64_t)a.T + TPT - 1) / TPT * per_row) return;
  const int g = (int)(e / per_row), c0 = (int)(e % per_row) * 8;
  int code[TPT][LM];
#pragma unroll
  for (int u = 0; u < TPT; ++u) {
    const int t = min(g * TPT + u, a.T - 1);
#pragma unroll
    for (int l = 0; l < LM; ++l) {
      if (l < a.L) {
        const int c = a.code_bytes == 1 ? ((const uint8_t*)a.codes)[(int64_t)t * a.L + l]
                                        : ((const uint16_t*)a.codes)[(int64_t)t * a.L + l];
        code[u][l] = c < a.K ? c : a.K - 1;
      }
    }
  }
  float4 cw[TPT][LM][2];
#pragma unroll
  for (int u = 0; u < TPT; ++u)
#pragma unroll
    for (int l = 0; l < LM; ++l) {
      if (l < a.L) {
        const float4* p = (const float4*)(a.C + ((int64_t)l * a.K + code[u][l]) * a.r + c0);
        cw[u][l][0] = p[0];
        cw[u][l][1] = p[1];
      }
    }
#pragma unroll
  for (int u = 0; u < TPT; ++u) {
    const int t = g * TPT + u;
    if (t < a.T) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = 0.f;
#pragma unroll
      for (int l = 0; l < LM; ++l) {
        if (l < a.L) {
          const float4 p = cw[u][l][0], q4 = cw[u][l][1];
          v[0] += p.x; v[1] += p.y; v[2] += p.z; v[3] += p.w;
          v[4] += q4.x; v[5] += q4.y; v[6] += q4.z; v[7] += q4.w;
        }
      }
      *(uint4*)(a.out + (int64_t)t * a.ldo + c0) =
          make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
    }
  }
}

// One thread per 8 columns of a gathered row (16 B copies).
__device__ __forceinline__ void gather_rows_block(int bx, const bf16_t* __restrict__ A, int k,
                                                  const int32_t* __restrict__ ids, int V, int T,
                                                  bf16_t* __restrict__ out) {
  const int cpr = k / 8;
  const int64_t e = (int64_t)bx * blockDim.x + threadIdx.x;
  if (e >= (int64_t)T * cpr) return;
  const int t = (int)(e / cpr), c = (int)(e % cpr) * 8;
  *(uint4*)(out + (int64_t)t * k + c) = *(const uint4*)(A + (int64_t)clamp_id(ids[t], V) * k + c);
}

__global__ void k_prep_u(const float* __restrict__ U, int d, int r, bf16_t* __restrict__ Ub, int64_t ldub,
                         bf16_t* __restrict__ Ut, int64_t ldut) {
  prep_u_tile(blockIdx.x, blockIdx.y, U, d, r, Ub, ldub, Ut, ldut);
}
__global__ void k_transpose_into(const void* __restrict__ src, int src_f32, int rows, int cols, int64_t lds,
                                 float scale, bf16_t* __restrict__ dst, int64_t ldd, int off) {
  transpose_tile(blockIdx.x, blockIdx.y, src, src_f32, rows, cols, lds, scale, dst, ldd, off);
}
__global__ void k_prep_codebook(const float* __restrict__ C, int L, int K, int r, bf16_t* __restrict__ Cb,
                                float* __restrict__ meta) {
  prep_codebook_block(blockIdx.x, C, L, K, r, Cb, meta);
}
__global__ void k_assemble(AssembleArgs a) { assemble_block(blockIdx.x, a); }
__global__ void k_gather_rows_bf16(const bf16_t* __restrict__ A, int k, const int32_t* __restrict__ ids, int V,
                                   int T, bf16_t* __restrict__ out) {
  gather_rows_block(blockIdx.x, A, k, ids, V, T, out);
}

// dst[c * ldd + off + i] = bf16(scale * sum_j P[i][j] bf16(Q(j, c))) for a
// 16 x 16 output tile (i0 = 16 by, c0 = 16 bx): P bf16 [M, Kd] row-major,
// Q(j, c) = Q[j * ldq + c] (qt = 0) or Q[c * ldq + j] (qt = 1), fp32, rounded
// to bf16 where it enters the matrix units; fp32 accumulation
// (v_mfma_f32_16x16x32_bf16).  The four waves take every fourth 32-wide
// k-step and add their partial tiles through LDS in a fixed order; small
// tiles give many workgroups, so each wave's chain of dependent loads over
// K stays short.  Kd % 32 == 0, N % 16 == 0; rows >= M are not written.
__device__ __forceinline__ void small_gemm_tile(int bx, int by, const PrepJob& j) {
  __shared__ float part[3][16 * 16];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, quad = lane >> 4;
  const int i0 = by * 16, c0 = bx * 16;
  const int prow = min(i0 + (lane & 15), j.M - 1);
  const bf16_t* P = (const bf16_t*)j.P + (int64_t)prow * j.ldp;
  const int c = c0 + (lane & 15);
  f32x4_t acc = f32x4_t{};
  // batches of up to four k-steps: every load of a batch is issued before
  // the first conversion, so their latencies overlap
  constexpr int NB = 4;
  for (int kb = 32 * wave; kb < j.Kd; kb += 128 * NB) {
    uint4 a[NB];
    float qv[NB][8];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int k0 = min(kb + 128 * u, j.Kd - 32);  // past the end: a repeat, not used
      a[u] = *(const uint4*)(P + k0 + 8 * quad);
      if (j.qt) {
        const float4* q4 = (const float4*)(j.Q + (int64_t)c * j.ldq + k0 + 8 * quad);
        const float4 x0 = q4[0], x1 = q4[1];
        qv[u][0] = x0.x; qv[u][1] = x0.y; qv[u][2] = x0.z; qv[u][3] = x0.w;
        qv[u][4] = x1.x; qv[u][5] = x1.y; qv[u][6] = x1.z; qv[u][7] = x1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qv[u][e] = j.Q[(int64_t)(k0 + 8 * quad + e) * j.ldq + c];
      }
    }
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const uint4 b = make_uint4(pack_bf2(qv[u][0], qv[u][1]), pack_bf2(qv[u][2], qv[u][3]),
                                 pack_bf2(qv[u][4], qv[u][5]), pack_bf2(qv[u][6], qv[u][7]));
      if (kb + 128 * u < j.Kd) acc = mfma16x16x32(a[u], b, acc);
    }
  }
  // acc e: row 4 quad + e of the tile, column lane % 16
  if (wave > 0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) part[wave - 1][(4 * quad + e) * 16 + (lane & 15)] = acc[e];
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 4 * quad + e, col = lane & 15;
      const float v = ((acc[e] + part[0][row * 16 + col]) + part[1][row * 16 + col]) + part[2][row * 16 + col];
      if (i0 + row < j.M) {
        const int64_t o = j.dst_rows ? (int64_t)(i0 + row) * j.ldd + j.off + c0 + col
                                     : (int64_t)(c0 + col) * j.ldd + j.off + i0 + row;
        j.dst[o] = (bf16_t)f2bf(j.scale * v);
      }
    }
  }
}

// Several independent preparation jobs in one launch: block b runs job q
// where q is the first job whose cumulative block count exceeds b.
__global__ __launch_bounds__(256) void k_prep_batch(PrepBatch batch) {
  int b = blockIdx.x, q = 0;
  while (q + 1 < batch.n && b >= batch.job[q].blocks) {
    b -= batch.job[q].blocks;
    ++q;
  }
  const PrepJob& j = batch.job[q];
  switch (j.kind) {
    case PJ_PREP_U: prep_u_tile(b % j.gx, b / j.gx, j.U, j.d, j.r, j.Ub, j.ldub, j.Ut, j.ldut); break;
    case PJ_TRANSPOSE:
      transpose_tile(b % j.gx, b / j.gx, j.src, j.src_f32, j.rows, j.cols, j.lds, j.scale, j.dst, j.ldd, j.off);
      break;
    case PJ_CODEBOOK: prep_codebook_block(b, j.C, j.L, j.K, j.r, j.Cb, j.meta); break;
    case PJ_ASSEMBLE: assemble_block(b, j.asm_args); break;
    case PJ_ASSEMBLE_SUM: assemble_sum_block(b, j.asm_args); break;
    case PJ_GATHER: gather_rows_block(b, j.A, j.k, j.ids, j.V, j.T, j.out); break;
    case PJ_SMALL_GEMM: small_gemm_tile(b % j.gx, b / j.gx, j); break;
    default: break;
  }
}

__global__ void k_check_ids(const int32_t* __restrict__ ids, int T, int64_t V, int* flag) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < T && (ids[t] < 0 || (int64_t)ids[t] >= V)) atomicOr(flag, 1);
}

__global__ void k_zero_bytes(uint32_t* p, int64_t words) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < words) p[i] = 0;
}

}  // namespace

hipError_t launch_prep_u(const float* U, int d, int r, bf16_t* Ub, int64_t ldub, bf16_t* Ut,
                         int64_t ldut, hipStream_t s) {
  const int cols = (int)((Ub && ldub > r) ? ldub : r);
  const int rows = (int)((Ut && ldut > d) ? ldut : d);
  dim3 grid((rows + 31) / 32, (cols + 31) / 32);
  hipLaunchKernelGGL(k_prep_u, grid, dim3(256), 0, s, U, d, r, Ub, ldub, Ut, ldut);
  return hipGetLastError();
}

hipError_t launch_transpose_into(const void* src, int src_f32, int rows, int cols, int64_t lds,
                                 float scale, bf16_t* dst, int64_t ldd, int off, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  dim3 grid((cols + 31) / 32, (rows + 31) / 32);
  hipLaunchKernelGGL(k_transpose_into, grid, dim3(256), 0, s, src, src_f32, rows, cols, lds, scale, dst,
                     ldd, off);
  return hipGetLastError();
}

hipError_t launch_prep_codebook(const float* C, int L, int K, int r, bf16_t* Cb, float* meta, hipStream_t s) {
  const int64_t slots = (int64_t)L * ((K + 63) / 64) * 64;
  if (slots <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_prep_codebook, dim3((unsigned)((slots + 3) / 4)), dim3(256), 0, s, C, L, K, r, Cb, meta);
  return hipGetLastError();
}

hipError_t launch_assemble(const AssembleArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (a.r % 8 || a.ldo % 8 || (a.A != nullptr && a.k % 8)) return hipErrorInvalidValue;
  const int64_t n = (int64_t)a.T * (a.ldo / 8);
  hipLaunchKernelGGL(k_assemble, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_rows_bf16(const bf16_t* A, int k, const int32_t* ids, int V, int T, bf16_t* out,
                                   hipStream_t s) {
  if (k % 8) return hipErrorInvalidValue;
  const int64_t n = (int64_t)T * (k / 8);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows_bf16, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, A, k, ids, V, T, out);
  return hipGetLastError();
}

PrepJob prep_job_u(const float* U, int d, int r, bf16_t* Ub, int64_t ldub, bf16_t* Ut, int64_t ldut) {
  PrepJob j{};
  j.kind = PJ_PREP_U;
  j.U = U; j.d = d; j.r = r; j.Ub = Ub; j.ldub = ldub; j.Ut = Ut; j.ldut = ldut;
  // only the d x r values: padding columns of the operands are never read
  j.gx = (d + 31) / 32;
  j.blocks = j.gx * ((r + 31) / 32);
  return j;
}

PrepJob prep_job_transpose(const void* src, int src_f32, int rows, int cols, int64_t lds, float scale, bf16_t* dst,
                           int64_t ldd, int off) {
  PrepJob j{};
  j.kind = PJ_TRANSPOSE;
  j.src = src; j.src_f32 = src_f32; j.rows = rows; j.cols = cols; j.lds = lds; j.scale = scale;
  j.dst = dst; j.ldd = ldd; j.off = off;
  j.gx = (cols + 31) / 32;
  j.blocks = rows > 0 && cols > 0 ? j.gx * ((rows + 31) / 32) : 0;
  return j;
}

PrepJob prep_job_codebook(const float* C, int L, int K, int r, bf16_t* Cb, float* meta) {
  PrepJob j{};
  j.kind = PJ_CODEBOOK;
  j.C = C; j.L = L; j.K = K; j.r = r; j.Cb = Cb; j.meta = meta;
  j.blocks = (int)(((int64_t)L * ((K + 63) / 64) * 64 + 3) / 4);
  return j;
}

PrepJob prep_job_assemble(const AssembleArgs& a) {
  PrepJob j{};
  j.asm_args = a;
  if (a.L >= 1 && a.L <= 2 && a.A == nullptr && a.Bc == nullptr && a.ldo == a.r && a.gdim == 0) {
    j.kind = PJ_ASSEMBLE_SUM;
    j.blocks = a.T > 0 ? (int)(((int64_t)(a.T + 3) / 4 * (a.r / 8) + 255) / 256) : 0;
  } else {
    j.kind = PJ_ASSEMBLE;
    j.blocks = a.T > 0 ? (int)(((int64_t)a.T * (a.ldo / 8) + 255) / 256) : 0;
  }
  return j;
}

PrepJob prep_job_gather(const bf16_t* A, int k, const int32_t* ids, int V, int T, bf16_t* out) {
  PrepJob j{};
  j.kind = PJ_GATHER;
  j.A = A; j.k = k; j.ids = ids; j.V = V; j.T = T; j.out = out;
  j.blocks = T > 0 ? (int)(((int64_t)T * (k / 8) + 255) / 256) : 0;
  return j;
}

PrepJob prep_job_small_gemm(const bf16_t* P, int64_t ldp, const float* Q, int64_t ldq, int qt, int M, int N,
                            int Kd, float scale, bf16_t* dst, int64_t ldd, int off) {
  PrepJob j{};
  j.kind = PJ_SMALL_GEMM;
  j.P = P; j.ldp = ldp; j.Q = Q; j.ldq = ldq; j.qt = qt; j.M = M; j.N = N; j.Kd = Kd; j.scale = scale;
  j.dst = dst; j.ldd = ldd; j.off = off;
  j.gx = N / 16;
  j.blocks = M > 0 ? ((M + 15) / 16) * (N / 16) : 0;
  return j;
}

hipError_t launch_prep_batch(const PrepJob* jobs, int n, hipStream_t s) {
  PrepBatch b{};
  int total = 0;
  for (int i = 0; i < n; ++i) {
    if (jobs[i].blocks <= 0) continue;
    if (b.n == PREP_MAX_JOBS) return hipErrorInvalidValue;
    if (jobs[i].kind == PJ_SMALL_GEMM &&
        (jobs[i].Kd % 32 || jobs[i].N % 16 || jobs[i].ldp % 8 || (jobs[i].qt && jobs[i].ldq % 4)))
      return hipErrorInvalidValue;
    if ((jobs[i].kind == PJ_ASSEMBLE || jobs[i].kind == PJ_ASSEMBLE_SUM) &&
        (jobs[i].asm_args.r % 8 || jobs[i].asm_args.ldo % 8 ||
                                        (jobs[i].asm_args.A != nullptr && jobs[i].asm_args.k % 8)))
      return hipErrorInvalidValue;
    if (jobs[i].kind == PJ_GATHER && jobs[i].k % 8) return hipErrorInvalidValue;
    b.job[b.n++] = jobs[i];
    total += jobs[i].blocks;
  }
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(k_prep_batch, dim3((unsigned)total), dim3(256), 0, s, b);
  return hipGetLastError();
}

hipError_t launch_check_ids(const int32_t* ids, int T, int64_t V, int* flag, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_check_ids, dim3((T + 255) / 256), dim3(256), 0, s, ids, T, V, flag);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(void* p, int64_t bytes, hipStream_t s) {
  const int64_t words = bytes / 4;
  if (words <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero_bytes, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, s, (uint32_t*)p,
                     words);
  return hipGetLastError();
}

}  // namespace mapl
