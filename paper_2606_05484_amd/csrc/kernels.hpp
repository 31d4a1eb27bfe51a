// Launchers of the gfx950 kernels behind libmapl.  Host-side only
// declarations; every launcher enqueues on the given stream and returns
// hipGetLastError().
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mapl {

typedef uint16_t bf16_t;

// ---------------------------------------------------------------- bf16 GEMM
// out[t,n] = sum_{c<Ka} A[t,c] W[n,c] + sum_{i<Kg} T[ids[t],i] W[n,Ka+i]
// Ka % 32 == 0, Kg % 16 == 0, ldw >= Ka + roundup(Kg,32) with zero padding,
// lda, ldt, ldw multiples of 8 (16 B rows), N % 32 == 0.
// Split-K: with kz > 0 (and Kg == 0) grid z-slice s covers columns
// [s*kz, (s+1)*kz) of A and W and writes its own fp32 partial at out + s*out_z.
// out_accum (fp32 output only) adds to the existing output instead of storing.
// With codes != null the first Ka columns of the token operand are not read
// from A but gathered: sum_{l<L} C[l][codes[t][l]][c] (C fp32 [L][K][Ka],
// codes [M][L] of code_bytes each, clamped to K-1, L <= 2), summed in fp32
// in l order from 0 and rounded once to bf16 -- the decoder's Zhat.  Only
// the short-K kernel takes it: gemm_tn_gathers() says whether g does.
struct TnArgs {
  const bf16_t* A; int64_t lda;
  const bf16_t* T; int64_t ldt; const int32_t* ids; int Kg; int V;  // ids clamped to [0,V)
  const bf16_t* W; int64_t ldw;
  int M, N, Ka;
  void* out; int64_t ldo; int out_f32;
  int kz; int64_t out_z; int out_accum;
  const void* codes; int code_bytes; const float* C; int L; int K;
};
hipError_t launch_gemm_tn(const TnArgs& g, hipStream_t s);
bool gemm_tn_gathers(const TnArgs& g);

// ---------------------------------------------------------------- fp32 GEMM
// C[b](m,n) = alpha_b sum_k A[b](m,k) B[b](k,n) + beta_b Cin[b](m,n)
// element types: 0 = fp32, 1 = bf16 (A, B, C); Cin is fp32 (may be null).
enum { GEMM_SPLIT_NONE = 0, GEMM_SPLIT_F16 = 1 };
struct GemmF32Args {
  const void* A; int64_t sAm, sAk, sAb;
  const void* B; int64_t sBk, sBn, sBb;
  const float* Cin; int64_t sCinm, sCinn, sCinb;
  void* C; int64_t sCm, sCn, sCb;
  int M, N, K, batch;
  float alpha, beta;
  const float* alpha_ptr; const float* beta_ptr;
  float diag;  // added to every element with m == n after the scaling
  int split;  // fp32 operands and output, aligned: GEMM_SPLIT_F16 takes the products as
             // hi.hi + hi.lo + lo.hi of fp16 pieces of 2^8 x (|operands| < 255)
  const float* pre_a; const float* pre_b;  // GEMM_SPLIT_F16 only: per-batch factors of A and B
                                           // (null: 1), applied before the split
  const void* A2; void* C2; int bsplit;   // GEMM_SPLIT_F16 only, optional: batch entries b >= bsplit
                                           // multiply A2 and write C2 (their entry b - bsplit), with
                                           // B, Cin and the per-batch factors of entry b - bsplit: two
                                           // products that share B in one launch
  int sym_upper;   // C = A B known symmetric (M == N; Cin, if any, symmetric too): only tiles on or
                   // above the diagonal are computed, each off-diagonal one also written mirrored
                   // (aligned case)
  float* sk_part;  // sym_upper, fp32 operands and output: with this workspace (gemm_f32_sk_bytes)
                   // the tiles' K ranges are split evenly over two workgroups per CU (stream-K) and
                   // a second launch sums each tile's pieces in K order
};
hipError_t launch_gemm_f32(const GemmF32Args& g, int ta, int tb, int to, hipStream_t s);

// Stream-K plan of a symmetric product (M x M output, upper 128 x 128 tiles
// of batch entries, K in 32-deep stages): T tiles, nk stages each, runs of U
// consecutive (tile, stage) units per workgroup over nwg workgroups, at most
// maxp pieces per tile.
struct SkPlan {
  int T, nk, U, maxp, nwg;
};
constexpr int SK_WORKGROUPS = 512;  // two per compute unit of an MI355X
__host__ __device__ inline SkPlan gemm_f32_sk_plan(int M, int K, int batch) {
  SkPlan p;
  const int ntm = (M + 127) / 128;
  p.T = ntm * (ntm + 1) / 2 * batch;
  p.nk = (K + 31) / 32;
  const long long total = (long long)p.T * p.nk;
  p.U = (int)((total + SK_WORKGROUPS - 1) / SK_WORKGROUPS);
  p.nwg = (int)((total + p.U - 1) / p.U);
  p.maxp = (p.nk - 1) / p.U + 2;
  return p;
}
inline size_t gemm_f32_sk_bytes(int M, int K, int batch) {
  const SkPlan p = gemm_f32_sk_plan(M, K, batch);
  return (size_t)p.T * p.maxp * 128 * 128 * 4;
}

// ---------------------------------------------------------------- weight gradient
// part[s][m][n] = sum over tokens t of split s of P[t,m] Q[t,n], where
// P[t,m] = Pa[t,m] for m < Ma and Tg[t, m-Mao] for Mao <= m < Mao+Mg, with
// Mao = wgrad_row_offset(Ma) (Ma rounded up to a 128-row tile; rows in
// [Ma, Mao) are written as zeros).  Tg is token-major [T, Mg].
// Ma, Mg, ldp, ldq multiples of 8, N % 64 == 0; bf16 inputs, fp32 partials.
struct WgradArgs {
  const bf16_t* Pa; int64_t ldp; int Ma;
  const bf16_t* Tg; int Mg;
  const bf16_t* Q; int64_t ldq;
  int T, N, splits, tokens_per_split;
  float* part;  // [splits][Mao+Mg][N]
};
hipError_t launch_wgrad(const WgradArgs& g, hipStream_t s);
int wgrad_row_offset(int Ma);
// out[t][i] = A[ids[t]][i] (bf16) for i < k.
hipError_t launch_gather_rows_bf16(const bf16_t* A, int k, const int32_t* ids, int V, int T, bf16_t* out,
                                   hipStream_t s);
// dst[n*ldd + off + m] = bf16(scale * sum_s part[s][m][n]) (transposed, fixed order).
hipError_t launch_reduce_splits_t_bf16(const float* part, int splits, int M, int N, int64_t part_stride,
                                       float scale, bf16_t* dst, int64_t ldd, int off, hipStream_t s);
// dU[i][c] (+)= sum_s part[s][i][c] - sum_j B[j][i] Wa[j][c] (fixed order; B bf16
// [k,d], Wa fp32 [k,r]; Wa == null skips the correction).  r % 4 == 0.
hipError_t launch_reduce_dU(const float* part, int splits, int64_t part_stride, int d, int r, float* dU,
                            int accumulate, const bf16_t* B, const float* Wa, int k, hipStream_t s);
// dst[m][n] (+)= sum_s part[s][m][n] for m < M (fixed summation order).
hipError_t launch_reduce_splits(const float* part, int splits, int M, int N, int64_t part_stride,
                                float* dst, int accumulate, hipStream_t s);

// ---------------------------------------------------------------- operand prep
// Ub[j][c] = bf16(U[j][c]) (row stride ldub, c < r), Ut[c][j] = bf16(U[j][c])
// (row stride ldut, j < d); either pointer may be null.  Padding columns
// [r, ldub) of Ub and [d, ldut) of Ut are zeroed.
hipError_t launch_prep_u(const float* U, int d, int r, bf16_t* Ub, int64_t ldub, bf16_t* Ut,
                         int64_t ldut, hipStream_t s);
// dst[j*ldd + off + i] = bf16(scale * src[i*lds + j]) for i < rows, j < cols
// (a transposed, scaled copy of a [rows, cols] matrix); src_f32 selects fp32
// or bf16 source.
hipError_t launch_transpose_into(const void* src, int src_f32, int rows, int cols, int64_t lds,
                                 float scale, bf16_t* dst, int64_t ldd, int off, hipStream_t s);
// Screening copy of the codebooks, rows of rvq_cb_cols(r) = r + 16 bf16:
// Cb[l][j][0:r] = bf16(C[l][j]), Cb[l][j][r:r+3] = hi, mid, lo with
// hi + mid + lo = ||C_j||^2 exactly (fp32 split into three bf16 pieces),
// Cb[l][j][r+3:r+5] = ||C_j|| rounded up (two pieces), Cb[l][j][r+5] =
// ||C_j - bf16(C_j)|| rounded up, Cb[l][j][r+6:r+16] = 0.  meta[0][l][chunk][64]:
// ||C_j||^2 in fp32 per 64-codeword chunk, meta[1][l][chunk][64]:
// ||C_j - bf16(C_j)|| rounded up (zero past K).
hipError_t launch_prep_codebook(const float* C, int L, int K, int r, bf16_t* Cb, float* meta, hipStream_t s);
inline int64_t rvq_meta_floats(int L, int K) { return 2 * (int64_t)L * ((K + 63) / 64) * 64; }
__host__ __device__ constexpr int rvq_cb_cols(int r) { return r + 16; }

// ---------------------------------------------------------------- receiver-side operand
// out[t][0:r]   = Zhat[t]: payload row (bf16) or sum_l C[l][codes[t,l]] (fp32 -> bf16)
// out[t][r:r+k] = A[ids[t]] when A != null; remaining columns up to ldo zeroed.
// When Bc != null (coordinate anchor), out[t][0:r] = Zhat[t] + A[ids[t]] Bc
// (Bc [k,r] bf16) and no anchor columns are appended.
struct AssembleArgs {
  const bf16_t* Zp;                  // [T,r] bf16 payload (L == 0) or null
  const void* codes; int code_bytes; // [T,L] (L > 0)
  const float* C; int L, K;          // [L,K,r]
  const bf16_t* A; int k;            // anchor table [V,k] or null
  const bf16_t* Bc;                  // [k,r] coordinate anchor companion or null
  const int32_t* ids; int V;
  int T, r; int64_t ldo;
  bf16_t* out;
  int gdim;                          // 2: grouped u8 codes [T, L, r/2] (group dimension 2)
};
hipError_t launch_assemble(const AssembleArgs& a, hipStream_t s);

// ---------------------------------------------------------------- batched preparation
// Independent preparation jobs of one call issued as a single launch
// (launch_prep_batch); each job behaves like the corresponding launcher.
enum { PJ_PREP_U = 1, PJ_TRANSPOSE, PJ_CODEBOOK, PJ_ASSEMBLE, PJ_GATHER, PJ_SMALL_GEMM, PJ_ASSEMBLE_SUM };
struct PrepJob {
  int kind, blocks, gx;
  // PJ_PREP_U
  const float* U; int d, r; bf16_t* Ub; int64_t ldub; bf16_t* Ut; int64_t ldut;
  // PJ_TRANSPOSE, PJ_SMALL_GEMM (dst, ldd, off, scale)
  const void* src; int src_f32, rows, cols; int64_t lds; float scale; bf16_t* dst; int64_t ldd; int off;
  // PJ_CODEBOOK
  const float* C; int L, K; bf16_t* Cb; float* meta;
  // PJ_ASSEMBLE, PJ_ASSEMBLE_SUM (codeword sums only: L <= 2, no anchor columns)
  AssembleArgs asm_args;
  // PJ_GATHER
  const bf16_t* A; int k; const int32_t* ids; int V, T; bf16_t* out;
  // PJ_SMALL_GEMM: dst[c*ldd + off + i] (dst_rows = 0) or dst[i*ldd + off + c]
  // (dst_rows = 1) = bf16(scale * sum_j P[i][j] bf16(Q(j, c))),
  // Q(j, c) = Q[j*ldq + c] (qt = 0) or Q[c*ldq + j] (qt = 1)
  const void* P; int64_t ldp; const float* Q; int64_t ldq; int qt, M, N, Kd, dst_rows;
};
constexpr int PREP_MAX_JOBS = 4;
struct PrepBatch {
  PrepJob job[PREP_MAX_JOBS];
  int n;
};
PrepJob prep_job_u(const float* U, int d, int r, bf16_t* Ub, int64_t ldub, bf16_t* Ut, int64_t ldut);
PrepJob prep_job_transpose(const void* src, int src_f32, int rows, int cols, int64_t lds, float scale, bf16_t* dst,
                           int64_t ldd, int off);
PrepJob prep_job_codebook(const float* C, int L, int K, int r, bf16_t* Cb, float* meta);
PrepJob prep_job_assemble(const AssembleArgs& a);
PrepJob prep_job_gather(const bf16_t* A, int k, const int32_t* ids, int V, int T, bf16_t* out);
PrepJob prep_job_small_gemm(const bf16_t* P, int64_t ldp, const float* Q, int64_t ldq, int qt, int M, int N,
                            int Kd, float scale, bf16_t* dst, int64_t ldd, int off);
hipError_t launch_prep_batch(const PrepJob* jobs, int n, hipStream_t s);

// ---------------------------------------------------------------- RVQ (bf16 screen + fp32 rescore)
// r in {32, 64, 128, 256}.
struct RvqArgs {
  const float* Z0;     // [T,r] fp32 unquantised coordinates
  const bf16_t* Cb;    // [L,K,r+16] bf16 screening copy with the split norms (rvq_cb_cols)
  const float* C;      // [L,K,r] fp32 codebooks
  const float* meta;   // [2][L][ceil(K/64)][64]: ||C_j||^2, ||C_j - bf16(C_j)|| (rvq_meta_floats)
  int T, r, L, K;
  void* codes; int code_bytes;  // [T,L]
  int* stats;          // [8] optional counters, may be null: tokens rescored, their candidates,
                       // candidate-list overflows, (workgroup, round) pairs with the second
                       // (listing) pass, (workgroup, round) pairs in total
};
hipError_t launch_rvq(const RvqArgs& a, hipStream_t s);
// The encoder in one launch: Z0 = [X | a] W as launch_gemm_tn computes it
// (g.N == r, fp32, never stored; g.out unused), then the RVQ rounds of
// launch_rvq on it (a.Z0 unused).  Only where enc_rvq_fusable(r, L).
bool enc_rvq_fusable(int r, int L);
hipError_t launch_enc_rvq(const TnArgs& g, const RvqArgs& a, hipStream_t s);

// ---------------------------------------------------------------- fp32 codec path helpers
// out[t][i] = A[ids[t]][i] (fp32) for i < k.
hipError_t launch_gather_rows_f32(const float* A, int k, const int32_t* ids, int V, int T, float* out,
                                  hipStream_t s);
// fp32 residual quantisation with exact fp32 distances over all K.
hipError_t launch_rvq_f32(const float* Z0, const float* C, int T, int r, int L, int K, void* codes,
                          int code_bytes, hipStream_t s);
// Zhat[t] = sum_l C[l][codes[t,l]] (fp32); gdim 2: grouped u8 codes [T,L,r/2],
// Zhat[t][2g:2g+2] = sum_l C[l][codes[t,l,g]][2g:2g+2].
hipError_t launch_codes_sum_f32(const void* codes, int code_bytes, const float* C, int T, int r, int L,
                                int K, float* Zhat, hipStream_t s, int gdim = 0);
// Grouped RVQ (group dimension 2): codes[t][l][g] (u8) = the nearest 2-D codeword
// C[l][j][2g:2g+2] to the group's residual, exact fp32 distances, lowest index
// on ties; Z0 [T,r] fp32.  Needs grvq_supported(r, L, K).
hipError_t launch_grvq(const float* Z0, const float* C, int T, int r, int L, int K, uint8_t* codes, hipStream_t s);
bool grvq_supported(int r, int L, int K);
hipError_t launch_copy_f32(const float* src, float* dst, int64_t n, hipStream_t s);

// ---------------------------------------------------------------- Stiefel step helpers
// S <- (S + S^T)/2 for each of P [r,r] matrices, in place.
hipError_t launch_symmetrize(float* S, int P, int r, hipStream_t s);
// M <- beta M + (1-beta) gR (n elements per projector, P projectors);
// partial sums of M^2 -> partial[p][nblk], of G^2 -> partial[P + p][nblk].
hipError_t launch_momentum(float* M, const float* gR, const float* G, int64_t n, int P, float beta, float* partial,
                           int nblk, hipStream_t s);
// scale[p] = 1/(||M_p|| + eps), or 0 when ||M_p|| <= zero_rel ||G_p||
// (norms from launch_momentum's partials).
hipError_t launch_fro_scale(const float* partial, int nblk, int P, float eps, float zero_rel, float* scale,
                            hipStream_t s);
// For S [P][r][r]: nu2 = max_i sum_j |S_ij|; inv_nu = 1/sqrt(nu2), inv_nu2 = 1/nu2;
// part: P * ceil(r / 16) floats of scratch.
hipError_t launch_inf_norm_scales(const float* S, int P, int r, float* part, float* inv_nu, float* inv_nu2,
                                  hipStream_t s);

// ---------------------------------------------------------------- codebook synchronisation
// buf[l][i][:] = C[l][rows[l*n + i]][:] (zeros for rows outside [0, K)); r % 4 == 0.
hipError_t launch_codebook_pack(const float* C, const int32_t* rows, int L, int K, int r, int n, float* buf,
                                hipStream_t s);
// C[l][rows[l*n + i]][:] = buf[l][i][:] (rows outside [0, K) skipped); r % 4 == 0.
hipError_t launch_codebook_unpack(const float* buf, const int32_t* rows, int L, int K, int r, int n, float* C,
                                  hipStream_t s);

// ---------------------------------------------------------------- anchor-table gradient
// W[i][c] = B[i][c] (i < k), 0 for k <= i < kp; c < K; both row-major with K columns.
hipError_t launch_pad_rows_bf16(const bf16_t* B, int k, int K, int kp, bf16_t* W, hipStream_t s);
// Stable radix sort of (ids[i], i) by id over `passes` 8-bit digits; buffers of
// n int32 each (k0/v0, k1/v1 ping-pong) and hist of 256 * radix_tiles(n) ints;
// *skey / *sval receive the sorted ids and token indices.
int radix_tiles(int n);
hipError_t launch_sort_ids(const int32_t* ids, int n, int passes, int* hist, int32_t* k0, int32_t* v0, int32_t* k1,
                           int32_t* v1, const int32_t** skey, const int32_t** sval, hipStream_t s);
// dA[v] (+)= scale * sum of g[t] over the tokens t of id v, in sorted order
// (sub-chunks of 64 positions, then their boundary pieces in order).
struct AnchorSegArgs {
  const float* g; int64_t ldg; int k;
  const int32_t* skey; const int32_t* sval; int n;
  float* dA; int V; int accumulate; float scale;  // rows of ids outside [0, V) are skipped
  float* headp; float* tailp; int32_t* head_id; int32_t* head_thru; int32_t* tail_id; int nsub;
};
int anchor_sub_chunks(int n);
hipError_t launch_anchor_segsum(const AnchorSegArgs& a, hipStream_t s);

// ---------------------------------------------------------------- debug
// flag[0] = 1 if any ids[t] is outside [0, V).
hipError_t launch_check_ids(const int32_t* ids, int T, int64_t V, int* flag, hipStream_t s);
hipError_t launch_zero_bytes(void* p, int64_t bytes, hipStream_t s);

}  // namespace mapl
