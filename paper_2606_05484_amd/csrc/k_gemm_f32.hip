// Batched strided GEMM with fp32 results:
//   C[b](m,n) = alpha_b * sum_k A[b](m,k) B[b](k,n) + beta_b * Cin[b](m,n)
// with alpha_b = alpha * (alpha_ptr ? alpha_ptr[b] : 1), likewise beta, on
// the fp32 matrix units (v_mfma_f32_32x32x2_f32) or, for fp32 operands with
// GEMM_SPLIT_F16, as products of fp16 pieces on the 16-bit matrix units
// (k_gemm_x3).  Operands may be fp32 or bf16 (widened exactly to fp32 in
// LDS); any element strides, so transposed operands need no copies.  These
// kernels carry every product of the Stiefel step and the fp32 codec path.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int GF_BM = 128, GF_BN = 128, GF_BK = 16, GF_PAD = 1;
constexpr int GF_THREADS = 256;

template <typename T>
__device__ __forceinline__ float ld_elem(const T* p);
template <>
__device__ __forceinline__ float ld_elem<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld_elem<bf16_t>(const bf16_t* p) { return bf2f(*p); }

// Load a [BM x BK] tile of op(A) (element (m,k) at A + m*sm + k*sk) into
// LDS as s[k][m].  Consecutive threads walk the operand's unit-stride index.
template <typename T, int ROWS>
__device__ __forceinline__ void load_tile(float (*s)[ROWS + GF_PAD], const T* A, int64_t sm, int64_t sk,
                                          int m0, int k0, int M, int K, int tid) {
  constexpr int N = ROWS * GF_BK;
  if (sk == 1) {
#pragma unroll 4
    for (int e = tid; e < N; e += GF_THREADS) {
      int m = e / GF_BK, k = e % GF_BK;
      int gm = m0 + m, gk = k0 + k;
      s[k][m] = (gm < M && gk < K) ? ld_elem<T>(A + gm * sm + gk) : 0.f;
    }
  } else {
#pragma unroll 4
    for (int e = tid; e < N; e += GF_THREADS) {
      int k = e / ROWS, m = e % ROWS;
      int gm = m0 + m, gk = k0 + k;
      s[k][m] = (gm < M && gk < K) ? ld_elem<T>(A + gm * sm + (int64_t)gk * sk) : 0.f;
    }
  }
}

template <typename TA, typename TB, typename TO>
__global__ __launch_bounds__(GF_THREADS) void k_gemm_f32(GemmF32Args g) {
  __shared__ float As[GF_BK][GF_BM + GF_PAD];
  __shared__ float Bs[GF_BK][GF_BN + GF_PAD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves, 64 x 64 each
  const int b = blockIdx.z;
  const int m0 = blockIdx.x * GF_BM, n0 = blockIdx.y * GF_BN;
  const TA* A = (const TA*)g.A + b * g.sAb;
  const TB* B = (const TB*)g.B + b * g.sBb;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  for (int k0 = 0; k0 < g.K; k0 += GF_BK) {
    load_tile<TA, GF_BM>(As, A, g.sAm, g.sAk, m0, k0, g.M, g.K, tid);
    // B is addressed as element (k,n) at B + k*sBk + n*sBn; load it as the
    // tile of B^T (rows n, cols k).
    load_tile<TB, GF_BN>(Bs, B, g.sBn, g.sBk, n0, k0, g.N, g.K, tid);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GF_BK; kk += 2) {
      float a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[kk + (lane >> 5)][wm * 64 + i * 32 + (lane & 31)];
#pragma unroll
      for (int j = 0; j < 2; ++j) bb[j] = Bs[kk + (lane >> 5)][wn * 64 + j * 32 + (lane & 31)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x2f32(a[i], bb[j], acc[i][j]);
    }
    __syncthreads();
  }

  const float alpha = g.alpha * (g.alpha_ptr ? g.alpha_ptr[b] : 1.f);
  const float beta = g.beta * (g.beta_ptr ? g.beta_ptr[b] : 1.f);
  const float* Cin = g.Cin ? g.Cin + b * g.sCinb : nullptr;
  TO* C = (TO*)g.C + b * g.sCb;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        int m = m0 + wm * 64 + i * 32 + acc_row(e, lane);
        int n = n0 + wn * 64 + j * 32 + (lane & 31);
        if (m < g.M && n < g.N) {
          float v = alpha * acc[i][j][e];
          if (Cin && beta != 0.f) v += beta * Cin[m * g.sCinm + n * g.sCinn];
          if (m == n) v += g.diag;
          if constexpr (sizeof(TO) == 4)
            C[m * g.sCm + n * g.sCn] = v;
          else
            C[m * g.sCm + n * g.sCn] = (TO)f2bf(v);
        }
      }
}


// Pipelined variant for the aligned case (every operand has a unit-stride
// dimension, the other stride and that dimension's extent multiples of 4,
// 16-byte (fp32) or 8-byte (bf16) aligned bases): 128 x 128 tiles, K staged
// 32 at a time with 16-byte global loads into registers one stage ahead and
// two LDS buffers, so the matrix units work on one stage while the next is
// in flight (one barrier per stage).  A is either m-contiguous (AK = false:
// A(m,k) at A + m + k*sAk) or k-contiguous (AK = true: A + m*sAm + k); B is
// n-contiguous.  LDS holds both operands as k-pairs: s[k/2][m'][k%2], so the
// 64 lanes of one operand read (rows m0 .. m0+31, k and k+1) touch one
// 64-float span, every bank once; m' permutes the rows inside each group of
// 32 so that the 8-byte stores of 32 lanes also land in distinct banks:
// m' = m ^ ((m / 32) % 4) for tiles loaded row by row (B, m-contiguous A),
// m' = m ^ 4 ((k / 2) % 8) for the k-contiguous A.
constexpr int GV_BM = 128, GV_BN = 128, GV_BK = 32;

// Tile coordinates and batch entry of a workgroup.  Workgroups are handed to
// the 8 XCDs round-robin by linear id, each XCD with its own L2; when the
// batch count is a multiple of 8, linear id w is given to batch entry
// b = (w % 8) + 8 j and tile t (w / 8 = j T + t, T tiles per entry), so that
// all tiles of one entry run on one XCD and share its L2 (its operands are
// read once from HBM instead of once per XCD).  Otherwise the grid's
// (x, y, z).  With sym_upper the tiles are those on or above the diagonal of
// an nt x nt tile grid, row by row.
template <int BT = GV_BM>
__device__ __forceinline__ void gv_tile(const GemmF32Args& g, int& bm, int& bn, int& b) {
  const int ntm = (g.M + BT - 1) / BT, ntn = (g.N + BT - 1) / BT;
  const int T = g.sym_upper ? ntm * (ntm + 1) / 2 : ntm * ntn;
  int t;
  if (g.batch % 8 == 0) {
    const int w = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const int q = w >> 3;
    b = (w & 7) + 8 * (q / T);
    t = q % T;
  } else {
    b = blockIdx.z;
    t = blockIdx.x + gridDim.x * blockIdx.y;
  }
  if (g.sym_upper) {
    int row = 0;
    while (t >= ntm - row) {
      t -= ntm - row;
      ++row;
    }
    bm = row;
    bn = row + t;
  } else {
    bm = t % ntm;
    bn = t / ntm;
  }
}

// Stream-K split of a symmetric product (sym_upper with a partial
// workspace): the (tile, k-stage) units, tile after tile (batch entries
// outermost), are dealt out in equal runs of U to two workgroups per CU, the
// runs of each XCD contiguous so that its workgroups share operands in its
// L2.  A run covers the end of one tile and the start of the next; each
// (tile, workgroup) piece of accumulators goes to its own fp32 slot, and
// k_gemm_sk_fix sums a tile's pieces in K order (bitwise reproducible) and
// applies the epilogue.  Without the split, 160 tiles of the c5 Gram products
// would leave 96 of the 256 CUs idle.
__device__ __forceinline__ void sk_tile(int t, int M, int& b, int& bm, int& bn) {
  const int ntm = (M + 127) / 128, Tb = ntm * (ntm + 1) / 2;
  b = t / Tb;
  int tl = t % Tb, row = 0;
  while (tl >= ntm - row) {
    tl -= ntm - row;
    ++row;
  }
  bm = row;
  bn = row + tl;
}

template <typename F>
__device__ __forceinline__ void sk_run(const GemmF32Args& g, F&& products, int tid) {
  const SkPlan p = gemm_f32_sk_plan(g.M, g.K, g.batch);
  const int w = blockIdx.x;
  const int v = p.nwg % 8 == 0 ? (w & 7) * (p.nwg >> 3) + (w >> 3) : w;
  const int64_t total = (int64_t)p.T * p.nk;
  const int64_t u1 = min((int64_t)(v + 1) * p.U, total);
  for (int64_t u = (int64_t)v * p.U; u < u1;) {
    const int t = (int)(u / p.nk), ks0 = (int)(u % p.nk);
    const int ks1 = (int)min((int64_t)p.nk, ks0 + (u1 - u));
    const int piece = v - (int)(((int64_t)t * p.nk) / p.U);
    int b, bm, bn;
    sk_tile(t, g.M, b, bm, bn);
    f32x16_t acc[2][2];
    products(b, bm, bn, ks0, ks1, acc);
    float* slot = g.sk_part + ((int64_t)t * p.maxp + piece) * (128 * 128);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) slot[((i * 2 + j) * 16 + e) * 256 + tid] = acc[i][j][e];
    u += ks1 - ks0;
  }
}

// The epilogue of the aligned kernels for one wave's 32F x 32F block of
// tile (tbm, tbn) (tiles of 64F x 64F, 2 x 2 waves): C = alpha acc +
// beta Cin, plus diag where m == n, and the mirrored element of an
// off-diagonal tile of a symmetric product.  Cin is
// read in full before the first store: C may alias Cin as far as the
// compiler knows, which would otherwise hold every load behind the store
// before it.
template <typename TO, int F = 2>
__device__ __forceinline__ void gv_epilogue(const GemmF32Args& g, const f32x16_t (&acc)[F][F], int b, int tbm,
                                            int tbn, int lane, int wm, int wn) {
  const int m0 = (tbm * 2 + wm) * 32 * F, n0 = (tbn * 2 + wn) * 32 * F;
  const bool second = g.A2 && b >= g.bsplit;  // the second product of a paired launch
  void* const Cbase = second ? g.C2 : g.C;
  if (second) b -= g.bsplit;
  const float alpha = g.alpha * (g.alpha_ptr ? g.alpha_ptr[b] : 1.f);
  const float beta = g.beta * (g.beta_ptr ? g.beta_ptr[b] : 1.f);
  const bool has_cin = g.Cin && beta != 0.f;
  float cin[F][F][16];
  if (has_cin) {
    const float* Cin = g.Cin + b * g.sCinb;
#pragma unroll
    for (int i = 0; i < F; ++i)
#pragma unroll
      for (int j = 0; j < F; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = m0 + i * 32 + acc_row(e, lane), n = n0 + j * 32 + (lane & 31);
          cin[i][j][e] = (m < g.M && n < g.N) ? Cin[m * g.sCinm + n * g.sCinn] : 0.f;
        }
  }
  TO* C = (TO*)Cbase + b * g.sCb;
#pragma unroll
  for (int i = 0; i < F; ++i)
#pragma unroll
    for (int j = 0; j < F; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + i * 32 + acc_row(e, lane), n = n0 + j * 32 + (lane & 31);
        if (m < g.M && n < g.N) {
          float v = alpha * acc[i][j][e];
          if (has_cin) v += beta * cin[i][j][e];
          if (m == n) v += g.diag;
          if constexpr (sizeof(TO) == 4) {
            C[m * g.sCm + n * g.sCn] = v;
            if (g.sym_upper && tbm != tbn) C[n * g.sCm + m * g.sCn] = v;
          } else {
            C[m * g.sCm + n * g.sCn] = (TO)f2bf(v);
            if (g.sym_upper && tbm != tbn) C[n * g.sCm + m * g.sCn] = (TO)f2bf(v);
          }
        }
      }
}

// Operand loads are raw buffer loads (out-of-range offsets read zero) into
// registers that are converted to fp32 only when the stage is written to LDS,
// so nothing waits for the loads before the products of the current stage.
constexpr uint32_t GV_OOB = 0x80000000u;  // any offset >= num_records reads zero

template <typename T>
struct Raw4;  // four consecutive elements as loaded
template <>
struct Raw4<float> {
  typedef __attribute__((ext_vector_type(4))) uint32_t type;
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  }
  static __device__ __forceinline__ float4 cvt(type v) {
    return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
  }
};
template <>
struct Raw4<bf16_t> {
  typedef __attribute__((ext_vector_type(2))) uint32_t type;
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  }
  static __device__ __forceinline__ float4 cvt(type v) {
    return make_float4(bf2f(v[0] & 0xFFFFu), bf2f(v[0] >> 16), bf2f(v[1] & 0xFFFFu), bf2f(v[1] >> 16));
  }
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t gv_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)(bytes > 0 ? bytes : 0), 0x00020000);
}

template <typename TA, typename TB, typename TO, bool AK>
__global__ __launch_bounds__(GF_THREADS) void k_gemm_f32v(GemmF32Args g) {
  __shared__ __attribute__((aligned(16))) float As[2][GV_BK / 2][GV_BM][2];
  __shared__ __attribute__((aligned(16))) float Bs[2][GV_BK / 2][GV_BN][2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves, 64 x 64 each
  const int nk = (g.K + GV_BK - 1) / GV_BK;
  // the products of tile (tbm, tbn) of batch entry b over k-stages [ks0, ks1)
  auto products = [&](int b, int tbm, int tbn, int ks0, int ks1, f32x16_t (&acc)[2][2]) {
  const int m0 = tbm * GV_BM, n0 = tbn * GV_BN;
  // the host guarantees that each operand's extent fits 31-bit byte offsets
  const __amdgpu_buffer_rsrc_t rA =
      gv_rsrc((const TA*)g.A + b * g.sAb,
              (AK ? (int64_t)(g.M - 1) * g.sAm + g.K : (int64_t)(g.K - 1) * g.sAk + g.M) * (int64_t)sizeof(TA));
  const __amdgpu_buffer_rsrc_t rB =
      gv_rsrc((const TB*)g.B + b * g.sBb, ((int64_t)(g.K - 1) * g.sBk + g.N) * (int64_t)sizeof(TB));

  // per thread and stage: B (and an m-contiguous A) as two k-pairs of four
  // consecutive columns ([pair][row of the pair]); a k-contiguous A as four
  // runs of four k
  typename Raw4<TA>::type ra[4];
  typename Raw4<TB>::type rb[4];
  auto load = [&](int k0) {
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int idx = tid + GF_THREADS * v;  // k-pair idx / 32, columns 4 (idx % 32) .. +3
      const int k = k0 + 2 * (idx >> 5), n = n0 + 4 * (idx & 31);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bool ok = k + h < g.K && n < g.N;
        rb[2 * v + h] = Raw4<TB>::load(rB, ok ? (uint32_t)(((int64_t)(k + h) * g.sBk + n) * sizeof(TB)) : GV_OOB);
      }
      if constexpr (!AK) {
        const int m = m0 + 4 * (idx & 31);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const bool ok = k + h < g.K && m < g.M;
          ra[2 * v + h] = Raw4<TA>::load(rA, ok ? (uint32_t)(((int64_t)(k + h) * g.sAk + m) * sizeof(TA)) : GV_OOB);
        }
      }
    }
    if constexpr (AK) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int idx = tid + GF_THREADS * v;  // m = idx / 8, k = 4 (idx % 8) .. +3
        const int m = m0 + (idx >> 3), k = k0 + 4 * (idx & 7);
        const bool ok = m < g.M && k < g.K;
        ra[v] = Raw4<TA>::load(rA, ok ? (uint32_t)(((int64_t)m * g.sAm + k) * sizeof(TA)) : GV_OOB);
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int idx = tid + GF_THREADS * v;
      const int kp = idx >> 5, c4 = 4 * (idx & 31), sw = (idx & 31) >> 3;
      const float4 r0 = Raw4<TB>::cvt(rb[2 * v]), r1 = Raw4<TB>::cvt(rb[2 * v + 1]);
      *(float2*)&Bs[buf][kp][c4 + (0 ^ sw)][0] = make_float2(r0.x, r1.x);
      *(float2*)&Bs[buf][kp][c4 + (1 ^ sw)][0] = make_float2(r0.y, r1.y);
      *(float2*)&Bs[buf][kp][c4 + (2 ^ sw)][0] = make_float2(r0.z, r1.z);
      *(float2*)&Bs[buf][kp][c4 + (3 ^ sw)][0] = make_float2(r0.w, r1.w);
      if constexpr (!AK) {
        const float4 a0 = Raw4<TA>::cvt(ra[2 * v]), a1 = Raw4<TA>::cvt(ra[2 * v + 1]);
        *(float2*)&As[buf][kp][c4 + (0 ^ sw)][0] = make_float2(a0.x, a1.x);
        *(float2*)&As[buf][kp][c4 + (1 ^ sw)][0] = make_float2(a0.y, a1.y);
        *(float2*)&As[buf][kp][c4 + (2 ^ sw)][0] = make_float2(a0.z, a1.z);
        *(float2*)&As[buf][kp][c4 + (3 ^ sw)][0] = make_float2(a0.w, a1.w);
      }
    }
    if constexpr (AK) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int idx = tid + GF_THREADS * v;
        const int m = (idx >> 3) ^ ((idx & 7) << 2), kp = 2 * (idx & 7);
        const float4 a = Raw4<TA>::cvt(ra[v]);
        *(float2*)&As[buf][kp][m][0] = make_float2(a.x, a.y);
        *(float2*)&As[buf][kp + 1][m][0] = make_float2(a.z, a.w);
      }
    }
  };

#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  load(ks0 * GV_BK);
  store(0);
  __syncthreads();
  for (int it = ks0; it < ks1; ++it) {
    const int buf = (it - ks0) & 1;
    if (it + 1 < ks1) load((it + 1) * GV_BK);
#pragma unroll
    for (int kp = 0; kp < GV_BK / 2; ++kp) {
      float a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int sw = AK ? (kp >> 1) << 2 : (2 * wm + i) & 3;
        a[i] = As[buf][kp][wm * 64 + i * 32 + ((lane & 31) ^ sw)][lane >> 5];
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) bb[j] = Bs[buf][kp][wn * 64 + j * 32 + ((lane & 31) ^ ((2 * wn + j) & 3))][lane >> 5];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x2f32(a[i], bb[j], acc[i][j]);
    }
    // the other buffer was last read in the previous stage, before the barrier
    if (it + 1 < ks1) store(buf ^ 1);
    __syncthreads();
  }
  };

  if (g.sk_part) {
    sk_run(g, products, tid);
    return;
  }
  int tbm, tbn, b;
  gv_tile(g, tbm, tbn, b);
  f32x16_t acc[2][2];
  products(b, tbm, tbn, 0, nk, acc);
  gv_epilogue<TO>(g, acc, b, tbm, tbn, lane, wm, wn);
}

// Split variant of the aligned fp32 GEMM (fp32 operands and output): the
// split of Ootomo and Yokota (2022) on fp16 pieces, with a power-of-two
// prescale instead of their scaled low piece.  Every operand element x is
// held as y = 2^8 x, hi = fp16(y), lo = fp16(y - hi) (both round to nearest
// even, subnormals kept), each product taken as hi.hi + hi.lo + lo.hi on
// v_mfma_f32_32x32x16_f16 (fp32 accumulation, lo.lo dropped) and the sums
// scaled by 2^-16 (exact), at five times the fp32 MFMA rate.  An operand may
// carry a per-batch factor (pre_a, pre_b) taken into the prescale, so the
// product is of the scaled operands.  hi + lo holds y to 22 bits where lo is
// normal (|x| >= 2^-11) and to an absolute 2^-33 below that, so each product
// term carries about 2^-21 relative error: fp32's accuracy for the sums over
// K of a few thousand.  The (scaled) operands must satisfy |x| < 255 (hi
// stays finite); callers use it only where a norm bound holds.
// Same tiling as k_gemm_f32v (128 x 128, K staged 32 at a time, 16-byte
// loads into registers one stage ahead, two LDS buffers).  Hi and lo pieces
// live apart in LDS, each operand in the layout its loads give:
//  - a k-contiguous A as [row][k], rows 80 bytes apart (an odd number of
//    16 B chunks: consecutive rows' 16-byte accesses hit distinct bank
//    groups), fragments read as 8 consecutive k of one row per lane;
//  - B and an m-contiguous A as [k][row] (k-major, 128 rows = 16 chunks per
//    k, chunk-swizzled by wg_sw), written 8 bytes per lane along the row and
//    read with transposing LDS reads (tr_frag).
constexpr int GX_LD = GV_BK + 8;  // 16-bit pieces per row of a [row][k] tile
constexpr int X3_SMALL_BELOW = 512;  // 128-tile workgroups under which the split kernel takes 64 x 64 tiles

template <bool AK, int BT>
__global__ __launch_bounds__(GF_THREADS) __attribute__((amdgpu_waves_per_eu(256 / BT, 256 / BT))) void k_gemm_x3(
    GemmF32Args g) {
  static_assert(BT == 128 || BT == 64, "tiles of 128 x 128 or 64 x 64");
  constexpr int F = BT / 64;        // 32 x 32 blocks per wave and dimension (wave tile BT/2 square)
  constexpr int CPR = BT / 8;       // 16-byte chunks per k of a [k][row] tile
  constexpr int KPT = 4 * BT / 128; // k per thread of a [k][row] operand's stage (4 column quads each)
  constexpr int TPR = 256 / BT;     // threads per row of a k-contiguous A's stage
  constexpr int KQ = BT / 32;       // 4-float loads per thread and stage of a k-contiguous A
  // [row][k] tiles (k-contiguous A) or [k][row] tiles (the rest), per buffer and piece
  constexpr int A_ELEMS = AK ? BT * GX_LD : GV_BK * BT;
  __shared__ __attribute__((aligned(16))) bf16_t Ah[2][A_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t Al[2][A_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t Bh[2][GV_BK * BT];
  __shared__ __attribute__((aligned(16))) bf16_t Bl[2][GV_BK * BT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves, BT/2 x BT/2 each
  const int nk = (g.K + GV_BK - 1) / GV_BK;
  // the products of tile (tbm, tbn) of batch entry b over k-stages [ks0, ks1)
  auto products = [&](int b, int tbm, int tbn, int ks0, int ks1, f32x16_t (&acc)[F][F]) {
  const int m0 = tbm * BT, n0 = tbn * BT;
  // a paired launch's second product: A2 and entry b - bsplit of the rest
  const bool second = g.A2 && b >= g.bsplit;
  const int e = second ? b - g.bsplit : b;
  const __amdgpu_buffer_rsrc_t rA =
      gv_rsrc((const float*)(second ? g.A2 : g.A) + e * g.sAb,
              (AK ? (int64_t)(g.M - 1) * g.sAm + g.K : (int64_t)(g.K - 1) * g.sAk + g.M) * 4);
  const __amdgpu_buffer_rsrc_t rB = gv_rsrc((const float*)g.B + e * g.sBb, ((int64_t)(g.K - 1) * g.sBk + g.N) * 4);
  typedef Raw4<float>::type raw_t;
  // two register sets: the loads of stages it + 1 and it + 2 are in flight
  // while stage it is multiplied
  raw_t ra0[4], rb0[4], ra1[4], rb1[4];
  // B (and an m-contiguous A): thread t loads rows 4 (t % (BT/4)) + 0..3 at
  // k = KPT (t / (BT/4)) + 0..KPT-1, one 16-byte piece per k; a
  // k-contiguous A: row t / TPR, k = 4 KQ (t % TPR) + 0..4 KQ-1
  auto load = [&](int k0, raw_t (&ra)[4], raw_t (&rb)[4]) {
    const int kb = k0 + KPT * (tid / (BT / 4)), c = 4 * (tid % (BT / 4));
#pragma unroll
    for (int h = 0; h < KPT; ++h) {
      const int k = kb + h;
      rb[h] = Raw4<float>::load(rB, (k < g.K && n0 + c < g.N) ? (uint32_t)(((int64_t)k * g.sBk + n0 + c) * 4) : GV_OOB);
      if constexpr (!AK)
        ra[h] = Raw4<float>::load(rA, (k < g.K && m0 + c < g.M) ? (uint32_t)(((int64_t)k * g.sAk + m0 + c) * 4) : GV_OOB);
    }
    if constexpr (AK) {
      const int m = m0 + tid / TPR, k = k0 + 4 * KQ * (tid % TPR);
#pragma unroll
      for (int h = 0; h < KQ; ++h)
        ra[h] = Raw4<float>::load(rA, (m < g.M && k + 4 * h < g.K) ? (uint32_t)(((int64_t)m * g.sAm + k + 4 * h) * 4)
                                                                    : GV_OOB);
    }
  };
  // the fp16 split's prescale: 2^8 times the operand's factor for this batch entry
  const float sa = 256.f * (g.pre_a ? g.pre_a[e] : 1.f);
  const float sb = 256.f * (g.pre_b ? g.pre_b[e] : 1.f);
  // hi and lo pieces of two floats, packed
  auto split2 = [](float x, float y, uint32_t& hi, uint32_t& lo, float sc) {
    const f32x2_t v = (f32x2_t){x, y} * sc;
    const f16x2_t h = __builtin_convertvector(v, f16x2_t);
    hi = __builtin_bit_cast(uint32_t, h);
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(v - __builtin_convertvector(h, f32x2_t), f16x2_t));
  };
  auto mma = [](const u32x4& a, const u32x4& b, f32x16_t c) { return mfma32x32x16h(as_uint4(a), as_uint4(b), c); };
  // 4 consecutive rows at KPT consecutive k (v[h]: k = h) into a [k][row] tile
  auto put_kmajor = [&](bf16_t* H, bf16_t* Lo, const raw_t (&v)[4], int row0, int kk, float sc) {
#pragma unroll
    for (int h = 0; h < KPT; ++h) {
      const int k = kk + h;
      const int off = k * CPR * 8 + (((row0 >> 3) ^ wg_sw(k, CPR)) << 3) + (row0 & 7);
      uint32_t h0, l0, h1, l1;
      split2(__uint_as_float(v[h][0]), __uint_as_float(v[h][1]), h0, l0, sc);
      split2(__uint_as_float(v[h][2]), __uint_as_float(v[h][3]), h1, l1, sc);
      *(uint2*)(H + off) = make_uint2(h0, h1);
      *(uint2*)(Lo + off) = make_uint2(l0, l1);
    }
  };
  auto store = [&](int buf, const raw_t (&ra)[4], const raw_t (&rb)[4]) {
    const int kk = KPT * (tid / (BT / 4)), c = 4 * (tid % (BT / 4));
    put_kmajor(Bh[buf], Bl[buf], rb, c, kk, sb);
    if constexpr (!AK) {
      put_kmajor(Ah[buf], Al[buf], ra, c, kk, sa);
    } else {
      const int m = tid / TPR, k = 4 * KQ * (tid % TPR);
      uint32_t hv[2 * KQ], lv[2 * KQ];
#pragma unroll
      for (int h = 0; h < KQ; ++h) {
        split2(__uint_as_float(ra[h][0]), __uint_as_float(ra[h][1]), hv[2 * h], lv[2 * h], sa);
        split2(__uint_as_float(ra[h][2]), __uint_as_float(ra[h][3]), hv[2 * h + 1], lv[2 * h + 1], sa);
      }
      bf16_t* H = Ah[buf] + m * GX_LD + k;
      bf16_t* Lo = Al[buf] + m * GX_LD + k;
#pragma unroll
      for (int q = 0; q < KQ / 2; ++q) {
        *(uint4*)(H + 8 * q) = make_uint4(hv[4 * q], hv[4 * q + 1], hv[4 * q + 2], hv[4 * q + 3]);
        *(uint4*)(Lo + 8 * q) = make_uint4(lv[4 * q], lv[4 * q + 1], lv[4 * q + 2], lv[4 * q + 3]);
      }
    }
  };

#pragma unroll
  for (int i = 0; i < F; ++i)
#pragma unroll
    for (int j = 0; j < F; ++j) acc[i][j] = f32x16_t{};

  // stage it: request stage it + 2 into (la, lb), multiply the LDS buffer of
  // stage it, write stage it + 1 from (sa, sb) into the other buffer (last
  // read in stage it - 1, before the barrier that ended it)
  auto stage = [&](int it, raw_t (&la)[4], raw_t (&lb)[4], const raw_t (&sa_)[4], const raw_t (&sb_)[4]) {
    const int buf = (it - ks0) & 1;
    if (it + 2 < ks1) load((it + 2) * GV_BK, la, lb);
#pragma unroll
    for (int ks = 0; ks < GV_BK / 16; ++ks) {
      u32x4 f[4 * F];  // a hi [F], a lo [F], b hi [F], b lo [F]
#pragma unroll
      for (int i = 0; i < F; ++i) {
        if constexpr (AK) {
          const int row = wm * 32 * F + i * 32 + (lane & 31), kc = 16 * ks + 8 * (lane >> 5);
          f[i] = *(const u32x4*)(Ah[buf] + row * GX_LD + kc);
          f[F + i] = *(const u32x4*)(Al[buf] + row * GX_LD + kc);
        } else {
          f[i] = tr_frag(Ah[buf], CPR, 16 * ks, wm * 32 * F + i * 32, lane);
          f[F + i] = tr_frag(Al[buf], CPR, 16 * ks, wm * 32 * F + i * 32, lane);
        }
      }
#pragma unroll
      for (int j = 0; j < F; ++j) {
        f[2 * F + j] = tr_frag(Bh[buf], CPR, 16 * ks, wn * 32 * F + j * 32, lane);
        f[3 * F + j] = tr_frag(Bl[buf], CPR, 16 * ks, wn * 32 * F + j * 32, lane);
      }
      lds_wait(f);
#pragma unroll
      for (int i = 0; i < F; ++i)
#pragma unroll
        for (int j = 0; j < F; ++j) {
          acc[i][j] = mma(f[F + i], f[2 * F + j], acc[i][j]);
          acc[i][j] = mma(f[i], f[3 * F + j], acc[i][j]);
          acc[i][j] = mma(f[i], f[2 * F + j], acc[i][j]);
        }
    }
    if (it + 1 < ks1) store(buf ^ 1, sa_, sb_);
    __syncthreads();
  };
  load(ks0 * GV_BK, ra0, rb0);
  if (ks0 + 1 < ks1) load((ks0 + 1) * GV_BK, ra1, rb1);
  store(0, ra0, rb0);
  __syncthreads();
  for (int it = ks0; it < ks1; it += 2) {
    stage(it, ra0, rb0, ra1, rb1);
    if (it + 1 < ks1) stage(it + 1, ra1, rb1, ra0, rb0);
  }
#pragma unroll
  for (int i = 0; i < F; ++i)
#pragma unroll
    for (int j = 0; j < F; ++j) acc[i][j] *= 1.f / 65536.f;
  };

  if constexpr (BT == GV_BM) {
    if (g.sk_part) {
      sk_run(g, products, tid);
      return;
    }
  }
  int tbm, tbn, b;
  gv_tile<BT>(g, tbm, tbn, b);
  f32x16_t acc[F][F];
  products(b, tbm, tbn, 0, nk, acc);
  gv_epilogue<float, F>(g, acc, b, tbm, tbn, lane, wm, wn);
}

// The stream-K fix-up: one workgroup per (tile, wave quarter), one wave per
// 32 x 32 block of the quarter, sums the pieces in piece (= K) order and
// applies the epilogue of the one-launch kernels (scaling, diagonal); an
// off-diagonal tile's mirror is written through a 64 x 64 LDS transpose, in
// whole rows.
__global__ __launch_bounds__(256) void k_gemm_sk_fix(GemmF32Args g) {
  __shared__ float L[64][65];
  const SkPlan p = gemm_f32_sk_plan(g.M, g.K, g.batch);
  const int t = blockIdx.x >> 2, wave = blockIdx.x & 3;
  const int lane = threadIdx.x & 63, blk = threadIdx.x >> 6;  // blk = (i, j) block of the quarter
  const int wm = wave >> 1, wn = wave & 1, i = blk >> 1, j = blk & 1;
  const int pf = (int)(((int64_t)t * p.nk) / p.U), pl = (int)(((int64_t)(t + 1) * p.nk - 1) / p.U);
  // a piece holds element e of block (i, j) of quarter w, lane l, at ((2i + j) 16 + e) 256 + 64 w + l
  const float* slot = g.sk_part + (int64_t)t * p.maxp * (128 * 128) + blk * 16 * 256 + 64 * wave + lane;
  float v[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = slot[e * 256];
  for (int pc = 1; pc <= pl - pf; ++pc) {
    float w[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) w[e] = slot[(int64_t)pc * (128 * 128) + e * 256];
#pragma unroll
    for (int e = 0; e < 16; ++e) v[e] += w[e];
  }
  int b, bm, bn;
  sk_tile(t, g.M, b, bm, bn);
  const int mb = bm * GV_BM + wm * 64, nb = bn * GV_BN + wn * 64;
  const float alpha = g.alpha * (g.alpha_ptr ? g.alpha_ptr[b] : 1.f);
  float* C = (float*)g.C + b * g.sCb;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int mm = i * 32 + acc_row(e, lane), nn = j * 32 + (lane & 31);
    float x = alpha * v[e];
    if (mb + mm == nb + nn) x += g.diag;
    if (mb + mm < g.M && nb + nn < g.N) C[(mb + mm) * g.sCm + (nb + nn) * g.sCn] = x;
    L[mm][nn] = x;
  }
  if (bm == bn) return;  // a diagonal tile has no mirror (uniform over the workgroup)
  __syncthreads();
  // mirror: C[nb + nn][mb + lane] = L[lane][nn], one 64-float row per wave and step
  for (int nn = blk; nn < 64; nn += 4)
    if (nb + nn < g.N && mb + lane < g.M) C[(nb + nn) * g.sCm + (mb + lane) * g.sCn] = L[lane][nn];
}

// The aligned case of the pipelined kernel: returns 0 (A m-contiguous), 1
// (A k-contiguous) or -1 (use the general kernel).
int gemm_f32_vec_mode(const GemmF32Args& g, int ta, int tb) {
  const int ea = ta ? 2 : 4, eb = tb ? 2 : 4;
  auto al = [](const void* p, int e) { return ((uintptr_t)p % (uintptr_t)(4 * e)) == 0; };
  auto m4 = [](int64_t v) { return v % 4 == 0; };
  if (g.K <= 0 || !al(g.A, ea) || !al(g.B, eb)) return -1;
  if (!(g.sBn == 1 && m4(g.sBk) && m4(g.N) && m4(g.sBb))) return -1;
  // buffer offsets are 31-bit byte offsets
  const int64_t lim = 0x7fffffffll - 16;
  if (((int64_t)(g.K - 1) * g.sBk + g.N) * eb > lim) return -1;
  if (g.sAm == 1 && m4(g.sAk) && m4(g.M) && m4(g.sAb) && ((int64_t)(g.K - 1) * g.sAk + g.M) * ea <= lim) return 0;
  if (g.sAk == 1 && m4(g.sAm) && m4(g.K) && m4(g.sAb) && ((int64_t)(g.M - 1) * g.sAm + g.K) * ea <= lim) return 1;
  return -1;
}

}  // namespace

hipError_t launch_gemm_f32(const GemmF32Args& g, int ta, int tb, int to, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return hipSuccess;
  const int vm = gemm_f32_vec_mode(g, ta, tb);
  if (g.sym_upper && (vm < 0 || g.M != g.N)) return hipErrorInvalidValue;
  if (g.sk_part && g.Cin) return hipErrorInvalidValue;  // the fix-up applies no Cin
  if (g.split < 0 || g.split > GEMM_SPLIT_F16) return hipErrorInvalidValue;
  if ((g.pre_a || g.pre_b) && g.split != GEMM_SPLIT_F16) return hipErrorInvalidValue;
  if (g.A2 && (g.split != GEMM_SPLIT_F16 || !g.C2 || g.sk_part || g.bsplit <= 0 || g.bsplit >= g.batch))
    return hipErrorInvalidValue;
  if (g.sk_part && !(g.sym_upper && ta == 0 && tb == 0 && to == 0)) return hipErrorInvalidValue;
  const int ntm = (g.M + GV_BM - 1) / GV_BM;
  const dim3 vgrid = g.sk_part      ? dim3(gemm_f32_sk_plan(g.M, g.K, g.batch).nwg)
                     : g.sym_upper ? dim3(ntm * (ntm + 1) / 2, 1, g.batch)
                                   : dim3(ntm, (g.N + GV_BN - 1) / GV_BN, g.batch);
  auto sk_fix = [&]() {
    if (!g.sk_part) return hipGetLastError();
    hipLaunchKernelGGL(k_gemm_sk_fix, dim3(4 * gemm_f32_sk_plan(g.M, g.K, g.batch).T), dim3(256), 0, s, g);
    return hipGetLastError();
  };
  if (g.split && (vm < 0 || ta || tb || to)) return hipErrorInvalidValue;
  if (g.split == GEMM_SPLIT_F16) {
    // 64 x 64 tiles where 128 x 128 ones would give fewer than X3_SMALL_BELOW
    // workgroups: such launches are bound by one workgroup's latency, and
    // four times the workgroups hide it better than the larger tiles' fewer
    // LDS bytes per product help
    const int ntn = (g.N + GV_BN - 1) / GV_BN;
    const int64_t t128 = (int64_t)(g.sym_upper ? ntm * (ntm + 1) / 2 : ntm * ntn) * g.batch;
    if (!g.sk_part && t128 < X3_SMALL_BELOW) {
      const int m64 = (g.M + 63) / 64, n64 = (g.N + 63) / 64;
      const dim3 grid64 = g.sym_upper ? dim3(m64 * (m64 + 1) / 2, 1, g.batch) : dim3(m64, n64, g.batch);
      if (vm) hipLaunchKernelGGL((k_gemm_x3<true, 64>), grid64, dim3(GF_THREADS), 0, s, g);
      else hipLaunchKernelGGL((k_gemm_x3<false, 64>), grid64, dim3(GF_THREADS), 0, s, g);
      return hipGetLastError();
    }
    if (vm) hipLaunchKernelGGL((k_gemm_x3<true, GV_BM>), vgrid, dim3(GF_THREADS), 0, s, g);
    else hipLaunchKernelGGL((k_gemm_x3<false, GV_BM>), vgrid, dim3(GF_THREADS), 0, s, g);
    const hipError_t e = hipGetLastError();
    return e != hipSuccess ? e : sk_fix();
  }
  if (vm >= 0) {
    const dim3 grid = vgrid;
#define MAPL_GV(TA_, TB_, TO_)                                                                        \
  do {                                                                                                \
    if (vm)                                                                                           \
      hipLaunchKernelGGL((k_gemm_f32v<TA_, TB_, TO_, true>), grid, dim3(GF_THREADS), 0, s, g);        \
    else                                                                                              \
      hipLaunchKernelGGL((k_gemm_f32v<TA_, TB_, TO_, false>), grid, dim3(GF_THREADS), 0, s, g);       \
  } while (0)
    if (ta == 0 && tb == 0 && to == 0) MAPL_GV(float, float, float);
    else if (ta == 1 && tb == 0 && to == 0) MAPL_GV(bf16_t, float, float);
    else if (ta == 0 && tb == 1 && to == 0) MAPL_GV(float, bf16_t, float);
    else if (ta == 1 && tb == 1 && to == 0) MAPL_GV(bf16_t, bf16_t, float);
    else if (ta == 1 && tb == 1 && to == 1) MAPL_GV(bf16_t, bf16_t, bf16_t);
    else if (ta == 0 && tb == 0 && to == 1) MAPL_GV(float, float, bf16_t);
    else if (ta == 1 && tb == 0 && to == 1) MAPL_GV(bf16_t, float, bf16_t);
    else if (ta == 0 && tb == 1 && to == 1) MAPL_GV(float, bf16_t, bf16_t);
    else return hipErrorInvalidValue;
#undef MAPL_GV
    const hipError_t e = hipGetLastError();
    return e != hipSuccess ? e : sk_fix();
  }
  if (g.sk_part) return hipErrorInvalidValue;
  dim3 grid((g.M + GF_BM - 1) / GF_BM, (g.N + GF_BN - 1) / GF_BN, g.batch);
  dim3 block(GF_THREADS);
#define MAPL_GF(TA_, TB_, TO_) hipLaunchKernelGGL((k_gemm_f32<TA_, TB_, TO_>), grid, block, 0, s, g)
  if (ta == 0 && tb == 0 && to == 0) MAPL_GF(float, float, float);
  else if (ta == 1 && tb == 0 && to == 0) MAPL_GF(bf16_t, float, float);
  else if (ta == 0 && tb == 1 && to == 0) MAPL_GF(float, bf16_t, float);
  else if (ta == 1 && tb == 1 && to == 0) MAPL_GF(bf16_t, bf16_t, float);
  else if (ta == 1 && tb == 1 && to == 1) MAPL_GF(bf16_t, bf16_t, bf16_t);
  else if (ta == 0 && tb == 0 && to == 1) MAPL_GF(float, float, bf16_t);
  else if (ta == 1 && tb == 0 && to == 1) MAPL_GF(bf16_t, float, bf16_t);
  else if (ta == 0 && tb == 1 && to == 1) MAPL_GF(float, bf16_t, bf16_t);
  else return hipErrorInvalidValue;
#undef MAPL_GF
  return hipGetLastError();
}

}  // namespace mapl
