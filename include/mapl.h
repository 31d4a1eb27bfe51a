/*
 * mapl.h -- C ABI of the MAPL stage-boundary codec and SPEL projector step
 * on AMD Instinct MI355X (gfx950).
 *
 * Method: "Learned Subspace Compression for Communication-Efficient Pipeline
 * Parallelism" (MAPL).  At each pipeline boundary the sender removes a
 * per-stage factorised anchor embedding from the boundary activations and
 * projects them onto an orthonormal projector (Sec. 3.2, Eq. 1), optionally
 * residual-vector-quantises the coordinates (Sec. 3.5); the receiver
 * rebuilds the activations (Eq. 2).  The projector is updated by SPEL
 * (Sec. 3.3, Eqs. 4-7; the projector-update half of Algorithm 1).
 *
 * Notation used below (paper -> argument):
 *   X^{b_p} [B,T,d] flattened to X [T,d]   boundary activations
 *   A_p in St(d,r)                 -> U [d,r] fp32 (orthonormal columns)
 *   E_p^small [V,k] (anchor table) -> A_s (sender), A_r (receiver) [V,k]
 *   P_p (frozen companion)         -> B_s, B_r: [k,d] for the ambient anchor
 *                                     of Eqs. 1-2, [k,r] for the coordinate
 *                                     reading (anchor added in r-space)
 *   t_ids                          -> ids [T] int32, 0 <= id < V
 *   Z^{b_p} [T,r]                  -> payload when L == 0
 *   R rounds of residual VQ        -> L stages, K codewords each,
 *                                     codebooks C [L,K,r] fp32
 *
 * Conventions shared by every call
 *   - Every array pointer is a DEVICE pointer owned by the caller; the
 *     library never allocates, frees or retains user memory.  Arrays are
 *     dense and row-major (last index fastest), 16-byte aligned.
 *   - Scratch memory comes only from the caller's workspace `ws` of
 *     `ws_bytes` bytes (256-byte aligned), sized by mapl_workspace_bytes().
 *     The workspace is not preserved between calls.
 *   - `stream` is a hipStream_t (passed as void*; NULL = default stream).
 *     Calls only enqueue work on it and never synchronise.
 *   - All arguments are validated on the host before anything is enqueued;
 *     on any error nothing is written and a negative mapl_status is
 *     returned; mapl_last_error() then describes it (thread-local string).
 *   - Outputs must not overlap inputs (except U and M of
 *     mapl_stiefel_step, which are updated in place).
 *   - Token ids are not range-checked on the device (the caller guarantees
 *     0 <= id < V); set MAPL_DEBUG=1 in the environment to have each codec
 *     call check them (this synchronises the stream) and fail with
 *     MAPL_E_RANGE.
 *   - Codes are written token-major, codes[t*L + l]; among codewords at
 *     equal distance the lowest index is chosen.
 *   - Calls that run concurrently on different streams must use different
 *     workspaces.
 */
#ifndef MAPL_H
#define MAPL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MAPL_VERSION 2

enum mapl_status {
  MAPL_OK = 0,
  MAPL_E_NULL = -1,        /* a required pointer is NULL                    */
  MAPL_E_SHAPE = -2,       /* sizes out of range or inconsistent            */
  MAPL_E_DTYPE = -3,       /* unknown or mismatched element type            */
  MAPL_E_RANGE = -4,       /* K too large for the code type; bad token id   */
  MAPL_E_ALIGN = -5,       /* pointer not 16-byte (workspace: 256) aligned  */
  MAPL_E_ALIAS = -6,       /* an output overlaps an input                   */
  MAPL_E_WORKSPACE = -7,   /* workspace missing or too small                */
  MAPL_E_UNSUPPORTED = -8, /* valid request this build does not implement   */
  MAPL_E_HIP = -9          /* a HIP launch or runtime call failed           */
};

enum mapl_dtype { MAPL_F32 = 0, MAPL_BF16 = 1, MAPL_U8 = 2, MAPL_U16 = 3 };

enum mapl_anchor_space {
  MAPL_ANCHOR_AMBIENT = 0, /* B is [k,d]: Eq. 1-2 (anchor removed/added in d-space) */
  MAPL_ANCHOR_COORD = 1    /* B is [k,r]: anchor removed after projection,
                              added back before the lift by U^T            */
};

enum mapl_call {
  MAPL_CALL_ENCODE = 0,
  MAPL_CALL_DECODE = 1,
  MAPL_CALL_DECODE_BWD = 2,
  MAPL_CALL_ENCODE_BWD = 3,
  MAPL_CALL_STIEFEL = 4
};

/* One boundary, one micro-batch.
 *   T  tokens (B*T of the paper flattened), 0 <= T < 2^31
 *   d  model width, multiple of 64, 64 <= d <= 16384
 *   r  projector rank, multiple of 32, 32 <= r <= min(d, 1024); the bf16
 *      path needs r % 64 == 0, and r in {64, 128, 256} when L > 0
 *      (MAPL_E_UNSUPPORTED otherwise)
 *   V  vocabulary size (rows of A), >= 1 when k > 0
 *   k  anchor rank, multiple of 16, 0 <= k <= min(d, 512); 0 = no anchor
 *   anchor_space  enum mapl_anchor_space
 *   L  RVQ stages, 0 <= L <= 8; 0 = no quantisation, payload is Z [T,r]
 *   K  codewords per stage (L > 0): multiple of 32, 32 <= K <= 65536
 *   x_dtype   MAPL_BF16 or MAPL_F32: X, Z, Xhat, dXhat, dZ, dX
 *   ab_dtype  element type of A and B; must equal x_dtype
 *   code_dtype MAPL_U8 (K <= 256) or MAPL_U16 (K <= 65536); ignored if L == 0
 *   group_dim 0: whole r-dimensional codewords; 2: the coordinates split into
 *      r/2 groups of two, each quantised on its own over the same two columns
 *      of every codebook round (Sec. 3.5 "decomposed into G groups"; App. E:
 *      group dimension 2, K = 256, R = 2).  Grouped codes are u8 [T, L, r/2]
 *      (codes[(t*L + l)*(r/2) + g]); needs L >= 1, K <= 256, MAPL_U8, and
 *      both element types are supported at any r above.
 *   On the bf16 path U is rounded to bf16 (round-to-nearest-even) where it
 *   enters the matrix units; accumulation is fp32.  On the fp32 path every
 *   operand stays fp32.
 */
typedef struct mapl_codec_desc {
  int64_t T, d, r, V, k;
  int32_t anchor_space;
  int32_t L, K;
  int32_t x_dtype, ab_dtype, code_dtype;
  int32_t group_dim;
} mapl_codec_desc;

/* Sender side, Eq. 1 (Alg. 1, "Project") followed by RVQ (Sec. 3.5).
 *   Z0[t] = (X[t] - A_s[ids[t]] B_s) U          (ambient)
 *   Z0[t] = X[t] U - A_s[ids[t]] B_s            (coord)
 *   L == 0: payload = Z0 rounded to x_dtype, [T,r].
 *   L  > 0: for l = 0..L-1, codes[t,l] = argmin_j ||R_l[t] - C[l,j]||^2 with
 *           R_0 = Z0, R_{l+1} = R_l - C[l, codes[t,l]]; payload = codes [T,L]
 *           of code_dtype.  Distances are decided in fp32 from Z0 computed
 *           with fp32 accumulation (bf16 matrix-unit screening, then exact
 *           fp32 rescoring of every codeword that could be nearest).
 *           group_dim 2: the same per group of two coordinates, codes
 *           [T, L, r/2] u8, exact fp32 distances.
 *   C may be NULL when L == 0.  A_s/B_s may be NULL when k == 0. */
int mapl_encode(const mapl_codec_desc* desc, const void* X, const int32_t* ids,
                const float* U, const void* A_s, const void* B_s, const float* C,
                void* payload, void* ws, size_t ws_bytes, void* stream);

/* Receiver side, Eq. 2 (Alg. 1, "Reconstruct").
 *   Zhat = payload (L == 0) or sum_l C[l, codes[t,l]] (L > 0; group_dim 2:
 *          Zhat[t, 2g:2g+2] = sum_l C[l, codes[t,l,g], 2g:2g+2])
 *   Xhat[t] = Zhat[t] U^T + A_r[ids[t]] B_r       (ambient)
 *   Xhat[t] = (Zhat[t] + A_r[ids[t]] B_r) U^T     (coord)
 *   Xhat is [T,d] of x_dtype.  Codes >= K are a caller error. */
int mapl_decode(const mapl_codec_desc* desc, const void* payload, const int32_t* ids,
                const float* U, const void* A_r, const void* B_r, const float* C,
                void* Xhat, void* ws, size_t ws_bytes, void* stream);

/* Backward of Eq. 2 (Sec. 3.2: the gradient is routed back through the
 * same projector).
 *   dZ = dXhat U                                   [T,r] of x_dtype
 *   dU (+)= dXhat^T Zhat                            (ambient)
 *   dU (+)= dXhat^T (Zhat + A_r[ids] B_r)           (coord)      [d,r] fp32
 * accumulate_dU = 0 overwrites dU, 1 adds to it (the sender's and the
 * receiver's contributions to the shared projector sum). */
int mapl_decode_bwd(const mapl_codec_desc* desc, const void* dXhat, const void* payload,
                    const int32_t* ids, const float* U, const void* A_r, const void* B_r,
                    const float* C, void* dZ, float* dU, int accumulate_dU, void* ws,
                    size_t ws_bytes, void* stream);

/* mapl_decode_bwd with the returned gradient quantised (Sec. 3.5: the
 * multi-codebook quantiser compresses "both forward activations and
 * backward gradients").  Instead of writing dZ it residual-vector-quantises
 * the r-dim gradient with its own codebooks:
 *   dZ0 = dXhat U  (fp32 accumulation, not rounded; bf16 U~ on the bf16 path)
 *   gcodes[t,l] = argmin_j ||R_l[t] - Cg[l,j]||^2, R_0 = dZ0,
 *                 R_{l+1} = R_l - Cg[l, gcodes[t,l]]   (as mapl_encode)
 *   dU (+)= exactly as mapl_decode_bwd.
 * Cg [Lg,Kg,r] fp32; gcodes [T,Lg] of gcode_dtype (MAPL_U8 for Kg <= 256,
 * MAPL_U16 otherwise).  1 <= Lg <= 8, 32 <= Kg <= 65536, Kg % 32 == 0; the
 * bf16 path needs r in {64, 128, 256}.  Workspace:
 * mapl_decode_bwd_q_workspace_bytes(desc, Lg, Kg).  The sending side turns
 * gcodes back into the gradient with mapl_grad_dequantize and passes it to
 * mapl_encode_bwd. */
int mapl_decode_bwd_q(const mapl_codec_desc* desc, const void* dXhat, const void* payload,
                      const int32_t* ids, const float* U, const void* A_r, const void* B_r,
                      const float* C, int32_t Lg, int32_t Kg, int32_t gcode_dtype, const float* Cg,
                      void* gcodes, float* dU, int accumulate_dU, void* ws, size_t ws_bytes,
                      void* stream);
size_t mapl_decode_bwd_q_workspace_bytes(const mapl_codec_desc* desc, int32_t Lg, int32_t Kg);

/* The quantised gradient's reconstruction (progressive refinement of
 * Sec. 3.5): dZ[t] = sum_l Cg[l, gcodes[t,l]], summed in fp32 and written as
 * out_dtype (MAPL_BF16, round-to-nearest-even, or MAPL_F32) [T,r].
 * 32 <= r <= 1024, r % 32 == 0; codes >= Kg are a caller error. */
int mapl_grad_dequantize(int64_t T, int64_t r, int32_t Lg, int32_t Kg, int32_t gcode_dtype,
                         const void* gcodes, const float* Cg, int32_t out_dtype, void* dZ,
                         void* stream);

/* Backward of Eq. 1; the quantiser is passed straight through (the gradient
 * of the codes' reconstruction is taken as the gradient of Z0).
 *   dX = dZ U^T                                    [T,d] of x_dtype
 *   dU (+)= (X - A_s[ids] B_s)^T dZ                 (ambient)
 *   dU (+)= X^T dZ                                   (coord)     [d,r] fp32 */
int mapl_encode_bwd(const mapl_codec_desc* desc, const void* dZ, const void* X,
                    const int32_t* ids, const float* U, const void* A_s, const void* B_s,
                    void* dX, float* dU, int accumulate_dU, void* ws, size_t ws_bytes,
                    void* stream);

/* SPEL step (Sec. 3.3, Eqs. 4-7) on P independent projectors, fp32 arrays
 * [P,d,r]:
 *   g_R = G - U sym(U^T G)                     (Eq. 4, sym(S) = (S+S^T)/2)
 *   M   = beta M + (1 - beta) g_R              (Eq. 5, in place)
 *   D   = PolarExpress_{lmo_steps}(M / (||M||_F + 1e-7))          (Eq. 6)
 *         and D = 0 when ||M||_F <= 2^-20 ||G||_F (a momentum below the
 *         fp32 resolution of the gradient has no direction)
 *   Y   = U - lr D
 *   U   = PolarExpress_{retract_steps}(Y / nu), nu^2 = max row sum of
 *         |Y^T Y| (an upper bound of sigma_max(Y)^2)                (Eq. 7)
 * PolarExpress step: X <- a X + X (b S + c S^2), S = X^T X, with the greedy
 * minimax odd-quintic schedule designed for singular values in [1e-3, 1]
 * (LMO) and [0.5, 1] (retraction).  Eq. 4 and Y^T Y are fp32 products; the
 * PolarExpress iterates are computed as X_0 times a product of the steps'
 * r x r polynomials, whose products multiply fp16 pieces of fp32 values
 * (hi + lo of 2^8 x, three products, fp32 accumulation: fp32's accuracy;
 * every operand is bounded by construction, for any U, G and M).  The
 * workspace (mapl_workspace_bytes, MAPL_CALL_STIEFEL) holds the iterates.
 * Requirements: 1 <= P, 32 <= r <= d,
 * r multiple of 32, d multiple of 32, r <= 1024, 1 <= lmo_steps,
 * retract_steps <= 16.  The retraction is accurate while lr*||D||_2 <= 1/3. */
int mapl_stiefel_step(int64_t P, int64_t d, int64_t r, float* U, const float* G, float* M,
                      float lr, float beta, int lmo_steps, int retract_steps, void* ws,
                      size_t ws_bytes, void* stream);

/* Gradient of an anchor table (Sec. 3.2: E_small is trainable, Eq. 3; the
 * sender's table enters Eq. 1, the receiver's Eq. 2).  Each token t gives a
 * row g[t] of length k, and
 *   dA[v] (+)= sum over the tokens t with ids[t] == v of g[t]      dA [V,k] fp32
 * side = MAPL_SENDER (table A_s, dY = dZ [T,r], the gradient of Eq. 1's
 * output; with RVQ it is the straight-through gradient):
 *   g[t] = -dZ[t] (B_s U)^T   (ambient; on the bf16 path B_s U~ rounded to bf16
 *                              as the encoder uses it)
 *   g[t] = -dZ[t] B_s^T       (coord)
 * side = MAPL_RECEIVER (table A_r):
 *   g[t] = dXhat[t] B_r^T     (ambient, dY = dXhat [T,d])
 *   g[t] = dZhat[t] B_r^T     (coord, dY = dZhat = dXhat U [T,r], e.g. the dZ
 *                              output of mapl_decode_bwd)
 * dY and B are of x_dtype; U is needed (fp32 [d,r]) only for the ambient
 * sender.  The rows of one id are summed in a fixed order (tokens sorted
 * stably by id, then in order), so repeated calls give identical bits;
 * fp32 accumulation of fp32 rows.  accumulate = 0 overwrites all of dA
 * (rows of absent ids become 0), 1 adds to it.  Requires k >= 1 and
 * T <= 2^24; ids must lie in [0, V) (MAPL_DEBUG=1 checks them).
 * Workspace: mapl_anchor_bwd_workspace_bytes(desc, side). */
enum mapl_side { MAPL_SENDER = 0, MAPL_RECEIVER = 1 };
int mapl_anchor_bwd(const mapl_codec_desc* desc, int side, const void* dY, const int32_t* ids,
                    const float* U, const void* B, float* dA, int accumulate, void* ws,
                    size_t ws_bytes, void* stream);
size_t mapl_anchor_bwd_workspace_bytes(const mapl_codec_desc* desc, int side);

/* Streaming codebook synchronisation (Sec. 3.5 "Codebook Synchronization",
 * App. F): instead of the whole codebook, each micro-batch carries a random
 * subset of its codewords (a 1/5 fraction per micro-batch in the paper's
 * hyperparameter table), so sender and receiver copies stay identical up to
 * a bounded staleness.  The subsets are the caller's: rows [L,n] int32 holds,
 * per round l, the n codeword indices sent this micro-batch (a random
 * partition of [0,K) into parts, one part per micro-batch, gives every
 * codeword once per cycle).  Indices of one round must be distinct for
 * unpack; indices outside [0,K) are skipped (pack writes a zero row).
 *   pack   (sender):   buf[l][i][:] = C[l][rows[l][i]][:],  buf [L,n,r] fp32
 *   unpack (receiver): C[l][rows[l][i]][:] = buf[l][i][:], other rows kept
 * C is [L,K,r] fp32.  Requirements: 1 <= L <= 8, 1 <= K <= 65536,
 * 4 <= r <= 1024 with r % 4 == 0, 0 <= n <= K; buf must not overlap C or
 * rows.  Device pointers, 16-byte aligned; enqueued on `stream` only. */
int mapl_codebook_pack(int32_t L, int32_t K, int64_t r, const float* C, const int32_t* rows,
                       int32_t n, float* buf, void* stream);
int mapl_codebook_unpack(int32_t L, int32_t K, int64_t r, const float* buf, const int32_t* rows,
                         int32_t n, float* C, void* stream);

/* mapl_encode without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, results and errors as mapl_encode;
 * scratch comes from a static device array of MAPL_NOALLOC_SCRATCH_BYTES
 * that the library holds on each GPU it runs on (the current device at the
 * call) until the process ends.  Requests whose workspace
 * (mapl_workspace_bytes(desc, MAPL_CALL_ENCODE)) exceeds it fail with
 * MAPL_E_WORKSPACE before anything is enqueued; at r = 256 this is about
 * 2.3 MiB for d = 2048, K = 1024, L = 2 at any T, while other ranks with
 * L > 0 also hold Z0 (4 r bytes per token).  The call allocates nothing.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (other threads, other streams) race and must be serialised by the
 * caller.  The first call on a device looks up the array's address there. */
#define MAPL_NOALLOC_SCRATCH_BYTES (16u << 20)
int mapl_encode_noalloc(const mapl_codec_desc* desc, const void* X, const int32_t* ids,
                        const float* U, const void* A_s, const void* B_s, const float* C,
                        void* payload, void* stream);

/* Workspace bytes needed by `call` (enum mapl_call).  Codec calls read
 * `desc` and ignore P, d, r; MAPL_CALL_STIEFEL ignores `desc`.  Returns 0
 * for an invalid request (mapl_last_error() says why). */
size_t mapl_workspace_bytes(const mapl_codec_desc* desc, int call, int64_t P, int64_t d,
                            int64_t r);

/* Thread-local description of the last error on this thread ("" if none). */
const char* mapl_last_error(void);

/* MAPL_VERSION of the built library. */
int mapl_version(void);

/* Tracing.  mapl_profile(1) makes every later call bracket each of its
 * kernel launches with a pair of HIP events on the call's stream (a small
 * per-launch overhead); mapl_profile(0) stops it.  mapl_profile(2) also
 * counts the decisions of the bf16 RVQ encoder (every such mapl_encode call
 * then synchronises its stream to read them).  mapl_profile_report()
 * waits for the recorded events, writes one line "name launches total_ms"
 * per kernel, in the order of each name's first launch (names are
 * "<call>:<kernel>"), followed, after RVQ counting, by lines "name count 0"
 * for rvq:tokens_rescored, rvq:candidates (summed over rescored tokens),
 * rvq:list_overflows, rvq:second_pass_blocks and rvq:blocks ((workgroup,
 * round) pairs with the second, candidate-listing screen, and in total),
 * into buf
 * (NUL-terminated, at most `bytes` bytes), and forgets the records.  Not for
 * use under stream capture.  Returns MAPL_OK, MAPL_E_HIP if an event could
 * not be resolved, or MAPL_E_WORKSPACE if buf was too small (the text is
 * truncated). */
int mapl_profile(int enable);
int mapl_profile_report(char* buf, size_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* MAPL_H */
