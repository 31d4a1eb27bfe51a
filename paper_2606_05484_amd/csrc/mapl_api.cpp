// libmapl host side: argument validation, workspace layout and kernel
// sequencing for the five C-ABI calls declared in include/mapl.h.
//
// Data flow per call (bf16 path; "~" = rounded to bf16 for the matrix units):
//   encode      prep U~^T | B_s U~ (ambient) -> Z0 = [X | a_s] [U~ ; -(B_s U~)]^T
//               (one token-major GEMM, anchors gathered in flight) -> bf16 Z
//               (L = 0) or fp32 Z0 -> RVQ screen/rescore -> codes
//   decode      prep [U~ | B_r^T] (and Zhat's codebook gather-sum where the
//               product cannot gather the codewords itself)
//               -> Xhat = [Zhat | a_r] [U~ | B_r^T]^T
//   decode_bwd  dZ = dXhat U~;  dU (+)= dXhat^T Zhat  (split over tokens,
//               fixed-order reduction)
//   encode_bwd  dX = dZ U~^T;  dU (+)= X^T dZ - B_s^T (a_s^T dZ)
//   stiefel     Eq. 4 tangent projection, Eq. 5 momentum, Eq. 6 LMO and
//               Eq. 7 retraction by PolarExpress, batched over projectors.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/mapl.h"
#include "kernels.hpp"
#include "polar_coeffs.h"

using namespace mapl;

namespace {

thread_local std::string g_err;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(MAPL_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define MAPL_HIP(expr)                                  \
  do {                                                  \
    hipError_t e_ = (expr);                             \
    if (e_ != hipSuccess) return hip_fail(e_, #expr);   \
  } while (0)

bool debug_ids() {
  static const int on = [] {
    const char* v = getenv("MAPL_DEBUG");
    return (v && v[0] && v[0] != '0') ? 1 : 0;
  }();
  return on != 0;
}

// ------------------------------------------------------------------ tracing
// mapl_profile(1) brackets every kernel launch with a pair of HIP events on
// the caller's stream; mapl_profile_report() resolves them into per-kernel
// launch counts and total milliseconds.
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof = false;
bool g_prof_rvq = false;      // mapl_profile(2): also collect the RVQ decision counters
constexpr int kRvqStats = 5;
long long g_rvq_stats[kRvqStats] = {0, 0, 0, 0, 0};
const char* const kRvqStatNames[kRvqStats] = {"rvq:tokens_rescored", "rvq:candidates", "rvq:list_overflows",
                                              "rvq:second_pass_blocks", "rvq:blocks"};
std::vector<ProfRec> g_prof_recs;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void prof_push(const char* name, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_recs.push_back({name, a, b});
}

#define LAUNCH(NAME, EXPR)                                              \
  do {                                                                  \
    hipEvent_t e0_ = nullptr, e1_ = nullptr;                            \
    if (g_prof && (e0_ = prof_event()) != nullptr) (void)hipEventRecord(e0_, s); \
    MAPL_HIP(EXPR);                                                     \
    if (e0_ && (e1_ = prof_event()) != nullptr) {                       \
      (void)hipEventRecord(e1_, s);                                     \
      prof_push(NAME, e0_, e1_);                                        \
    }                                                                   \
  } while (0)

inline int64_t rup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline size_t esize(int dt) { return dt == MAPL_F32 ? 4 : 2; }
inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// ------------------------------------------------------------------ workspace
struct Carve {
  size_t off = 0;
  size_t take(size_t bytes) {
    size_t o = off;
    off = (size_t)rup((int64_t)(off + bytes), 256);
    return o;
  }
};

// The Stiefel step's Gram products X^T X ([r, r] upper tiles over K = d)
// take the stream-K split where they have fewer tiles than two per CU and K
// is long enough for the split to pay for its fix-up launch.
bool gram_stream_k(int P, int d, int r) {
  const SkPlan p = gemm_f32_sk_plan(r, d, P);
  return p.T < SK_WORKGROUPS && p.nk >= 16;
}

struct SplitPlan {
  int splits, tps;
};

// Token splits of the weight-gradient kernel: it holds 144 KiB of LDS, so
// one workgroup per compute unit; the grid (tiles x splits) is kept within
// one wave of 256 workgroups.
SplitPlan plan_splits(int64_t T, int Ma, int Mg, int N) {
  const int bn = (N % 256 == 0) ? 256 : (N % 128 == 0) ? 128 : 64;
  const int64_t mt = wgrad_row_offset(Ma) / 128 + (Mg + 127) / 128;
  const int64_t tiles = mt * (int64_t)(N / bn);
  // one workgroup per CU (the kernel's LDS footprint) and a single wave of
  // workgroups: at most 256 in total
  int64_t want = tiles >= 256 ? 1 : 256 / tiles;
  int64_t maxs = (T + 63) / 64;
  if (want > maxs) want = maxs;
  if (want < 1) want = 1;
  int64_t tps = rup((T + want - 1) / want, 64);
  if (tps < 64) tps = 64;
  int64_t splits = (T + tps - 1) / tps;
  if (splits < 1) splits = 1;
  return {(int)splits, (int)tps};
}

struct Layout {
  size_t total = 0;
  size_t w = 0, w2 = 0, z0 = 0, cb = 0, cn2 = 0, cnr = 0, stats = 0, flag = 0;
  size_t ahat = 0, part = 0, wsum = 0, ga = 0, bu = 0, zh = 0, z2 = 0, bt = 0, wt = 0;
  int64_t kp = 0, kw = 0;
  SplitPlan sp{1, 64};
};


bool grouped(const mapl_codec_desc& D);

// Quantisation of the returned gradient (mapl_decode_bwd_q): its own RVQ
// codebooks over the r-dim gradient.
struct GradQ {
  int L, K, code_bytes;
  const float* C;
  void* codes;
};

Layout layout(const mapl_codec_desc& D, int call, const GradQ* q = nullptr) {
  Layout Lo;
  Carve c;
  c.take(0);
  const bool bf = D.x_dtype == MAPL_BF16;
  const int64_t T = D.T, d = D.d, r = D.r, k = D.k;
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  Lo.flag = c.take(256);
  Lo.kp = k > 0 ? rup(k, 32) : 0;
  if (bf) {
    switch (call) {
      case MAPL_CALL_ENCODE:
        Lo.kw = d + Lo.kp;
        Lo.w = c.take((size_t)r * Lo.kw * 2);
        if (grouped(D)) {
          Lo.z0 = c.take((size_t)T * r * 4);  // fp32 Z0 for the grouped quantiser
        } else if (D.L > 0) {
          // fp32 Z0 between the projection and the RVQ, unless one launch does both
          if (!enc_rvq_fusable((int)r, D.L)) Lo.z0 = c.take((size_t)T * r * 4);
          Lo.cb = c.take((size_t)D.L * D.K * rvq_cb_cols((int)r) * 2);
          Lo.cn2 = c.take((size_t)rvq_meta_floats(D.L, D.K) * 4);
          Lo.stats = c.take(32);
        }
        break;
      case MAPL_CALL_DECODE:
        Lo.kw = r + Lo.kp;
        Lo.w2 = c.take((size_t)d * Lo.kw * 2);
        if (D.L > 0) Lo.ahat = c.take((size_t)T * r * 2);
        break;
      case MAPL_CALL_DECODE_BWD:
        Lo.w = c.take((size_t)r * d * 2);
        if (D.L > 0 || (!amb && k > 0)) Lo.ahat = c.take((size_t)T * r * 2);
        Lo.sp = plan_splits(T, (int)d, 0, (int)r);
        Lo.part = c.take((size_t)Lo.sp.splits * wgrad_row_offset((int)d) * r * 4);
        if (q) {
          if (!enc_rvq_fusable((int)r, q->L)) Lo.z0 = c.take((size_t)T * r * 4);
          Lo.cb = c.take((size_t)q->L * q->K * rvq_cb_cols((int)r) * 2);
          Lo.cn2 = c.take((size_t)rvq_meta_floats(q->L, q->K) * 4);
          Lo.stats = c.take(32);
        }
        break;
      case MAPL_CALL_ENCODE_BWD: {
        Lo.w2 = c.take((size_t)d * r * 2);
        const int mg = (amb && k > 0) ? (int)k : 0;
        Lo.sp = plan_splits(T, (int)d, mg, (int)r);
        Lo.part = c.take((size_t)Lo.sp.splits * (wgrad_row_offset((int)d) + mg) * r * 4);
        if (mg) {
          Lo.wsum = c.take((size_t)k * r * 4);   // a_s^T dZ
          Lo.ga = c.take((size_t)T * k * 2);     // a_s = A_s[ids], token-major bf16
        }
        break;
      }
    }
  } else {
    switch (call) {
      case MAPL_CALL_ENCODE:
        if (k > 0) Lo.ga = c.take((size_t)T * k * 4);
        if (k > 0 && amb) Lo.bu = c.take((size_t)k * r * 4);
        if (D.L > 0) Lo.z0 = c.take((size_t)T * r * 4);
        break;
      case MAPL_CALL_DECODE:
      case MAPL_CALL_DECODE_BWD:
        if (k > 0) Lo.ga = c.take((size_t)T * k * 4);
        Lo.zh = c.take((size_t)T * r * 4);
        if (!amb && k > 0) Lo.z2 = c.take((size_t)T * r * 4);
        if (q && call == MAPL_CALL_DECODE_BWD) Lo.z0 = c.take((size_t)T * r * 4);
        break;
      case MAPL_CALL_ENCODE_BWD:
        if (k > 0 && amb) {
          Lo.ga = c.take((size_t)T * k * 4);
          Lo.wsum = c.take((size_t)k * r * 4);
        }
        break;
    }
  }
  Lo.total = c.off;
  return Lo;
}

// ------------------------------------------------------------------ validation
int check_desc(const mapl_codec_desc* D) {
  if (!D) return fail(MAPL_E_NULL, "desc is NULL");
  if (D->x_dtype != MAPL_BF16 && D->x_dtype != MAPL_F32)
    return fail(MAPL_E_DTYPE, "x_dtype must be MAPL_BF16 or MAPL_F32 (got %d)", D->x_dtype);
  if (D->ab_dtype != D->x_dtype)
    return fail(MAPL_E_DTYPE, "ab_dtype (%d) must equal x_dtype (%d)", D->ab_dtype, D->x_dtype);
  if (D->T < 0 || D->T >= ((int64_t)1 << 31)) return fail(MAPL_E_SHAPE, "T=%lld out of range", (long long)D->T);
  if (D->d < 64 || D->d > 16384 || D->d % 64) return fail(MAPL_E_SHAPE, "d=%lld: need 64 <= d <= 16384, d %% 64 == 0", (long long)D->d);
  if (D->r < 32 || D->r > 1024 || D->r % 32 || D->r > D->d)
    return fail(MAPL_E_SHAPE, "r=%lld: need 32 <= r <= min(d,1024), r %% 32 == 0", (long long)D->r);
  if (D->k < 0 || D->k > 512 || D->k % 16 || D->k > D->d)
    return fail(MAPL_E_SHAPE, "k=%lld: need 0 <= k <= min(d,512), k %% 16 == 0", (long long)D->k);
  if (D->k > 0 && (D->V < 1 || D->V * D->k * (D->x_dtype == MAPL_F32 ? 4 : 2) >= ((int64_t)1 << 31)))
    return fail(MAPL_E_SHAPE, "V=%lld: need V >= 1 and an anchor table under 2 GiB", (long long)D->V);
  if (D->anchor_space != MAPL_ANCHOR_AMBIENT && D->anchor_space != MAPL_ANCHOR_COORD)
    return fail(MAPL_E_SHAPE, "anchor_space=%d unknown", D->anchor_space);
  if (D->x_dtype == MAPL_BF16 && D->r % 64)
    return fail(MAPL_E_UNSUPPORTED, "the bf16 path needs r %% 64 == 0 (got r=%lld; r = 32 runs in fp32)",
                (long long)D->r);
  if (D->L < 0 || D->L > 8) return fail(MAPL_E_SHAPE, "L=%d: need 0 <= L <= 8", D->L);
  if (D->L > 0) {
    if (D->K < 32 || D->K > 65536 || D->K % 32) return fail(MAPL_E_SHAPE, "K=%d: need 32 <= K <= 65536, K %% 32 == 0", D->K);
    if (D->code_dtype == MAPL_U8) {
      if (D->K > 256) return fail(MAPL_E_RANGE, "K=%d does not fit MAPL_U8 codes", D->K);
    } else if (D->code_dtype != MAPL_U16) {
      return fail(MAPL_E_DTYPE, "code_dtype must be MAPL_U8 or MAPL_U16 (got %d)", D->code_dtype);
    }
    if (D->group_dim == 2) {
      if (D->K > 256 || D->code_dtype != MAPL_U8)
        return fail(MAPL_E_RANGE, "grouped RVQ (group_dim 2) needs K <= 256 and MAPL_U8 codes");
      if (!grvq_supported((int)D->r, D->L, D->K))
        return fail(MAPL_E_UNSUPPORTED, "grouped RVQ: r=%lld, L=%d, K=%d not supported", (long long)D->r, D->L, D->K);
    } else if (D->x_dtype == MAPL_BF16 && D->r != 64 && D->r != 128 && D->r != 256) {
      return fail(MAPL_E_UNSUPPORTED, "RVQ on the bf16 path supports r in {64, 128, 256} (got %lld)", (long long)D->r);
    }
  }
  if (D->group_dim != 0 && D->group_dim != 2)
    return fail(MAPL_E_SHAPE, "group_dim must be 0 (whole vectors) or 2 (got %d)", D->group_dim);
  if (D->group_dim == 2 && D->L == 0) return fail(MAPL_E_SHAPE, "group_dim 2 needs RVQ stages (L >= 1)");
  return MAPL_OK;
}

struct Span {
  const void* p;
  size_t bytes;
  const char* name;
};

int check_ptrs(std::initializer_list<Span> req, std::initializer_list<Span> outs, std::initializer_list<Span> ins) {
  for (const Span& s : req)
    if (s.bytes > 0 && !s.p) return fail(MAPL_E_NULL, "%s is NULL", s.name);
  for (const Span& s : req)
    if (s.p && !aligned(s.p, 16)) return fail(MAPL_E_ALIGN, "%s is not 16-byte aligned", s.name);
  for (const Span& o : outs) {
    if (!o.p || !o.bytes) continue;
    const uintptr_t a0 = (uintptr_t)o.p, a1 = a0 + o.bytes;
    for (const Span& i : ins) {
      if (!i.p || !i.bytes) continue;
      const uintptr_t b0 = (uintptr_t)i.p, b1 = b0 + i.bytes;
      if (a0 < b1 && b0 < a1) return fail(MAPL_E_ALIAS, "output %s overlaps input %s", o.name, i.name);
    }
  }
  return MAPL_OK;
}

int check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return MAPL_OK;
  if (!ws) return fail(MAPL_E_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (!aligned(ws, 256)) return fail(MAPL_E_ALIGN, "workspace is not 256-byte aligned");
  if (ws_bytes < need) return fail(MAPL_E_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  return MAPL_OK;
}

int run_id_check(const int32_t* ids, int64_t T, int64_t V, void* ws, const Layout& Lo, hipStream_t s) {
  if (!debug_ids() || T == 0) return MAPL_OK;
  int* flag = (int*)((char*)ws + Lo.flag);
  MAPL_HIP(launch_zero_bytes(flag, 4, s));
  MAPL_HIP(launch_check_ids(ids, (int)T, V, flag, s));
  int h = 0;
  MAPL_HIP(hipMemcpyAsync(&h, flag, 4, hipMemcpyDeviceToHost, s));
  MAPL_HIP(hipStreamSynchronize(s));
  if (h) return fail(MAPL_E_RANGE, "a token id is outside [0, V=%lld)", (long long)V);
  return MAPL_OK;
}

// Convenience builders for the fp32-unit GEMM.
GemmF32Args gemm(int M, int N, int K) {
  GemmF32Args g;
  memset(&g, 0, sizeof g);
  g.M = M; g.N = N; g.K = K; g.batch = 1;
  g.alpha = 1.f; g.beta = 0.f;
  return g;
}

template <typename P>
inline P* at(void* ws, size_t off) { return (P*)((char*)ws + off); }

size_t code_bytes(const mapl_codec_desc& D) { return D.code_dtype == MAPL_U8 ? 1 : 2; }
bool grouped(const mapl_codec_desc& D) { return D.L > 0 && D.group_dim == 2; }
size_t payload_bytes(const mapl_codec_desc& D) {
  if (grouped(D)) return (size_t)D.T * D.L * (D.r / 2);
  return D.L == 0 ? (size_t)D.T * D.r * esize(D.x_dtype) : (size_t)D.T * D.L * code_bytes(D);
}
size_t b_cols(const mapl_codec_desc& D) { return D.anchor_space == MAPL_ANCHOR_AMBIENT ? D.d : D.r; }

}  // namespace

// ===================================================================== API

extern "C" const char* mapl_last_error(void) { return g_err.c_str(); }
extern "C" int mapl_version(void) { return MAPL_VERSION; }

extern "C" size_t mapl_workspace_bytes(const mapl_codec_desc* desc, int call, int64_t P, int64_t d, int64_t r) {
  g_err.clear();
  if (call == MAPL_CALL_STIEFEL) {
    if (P < 1 || d < 32 || r < 32 || r > d || r > 1024 || r % 32 || d % 32) {
      fail(MAPL_E_SHAPE, "stiefel: need 1 <= P, 32 <= r <= min(d,1024), r and d multiples of 32");
      return 0;
    }
    Carve c;
    c.take((size_t)P * r * r * 4);   // S
    c.take((size_t)P * r * r * 4);   // Q
    c.take((size_t)P * d * r * 4);   // X0
    c.take((size_t)P * d * r * 4);   // X1
    c.take((size_t)P * 2048 * 4);    // partial sums of M^2 and G^2
    c.take((size_t)P * 8 * 4);       // scalars
    if (gram_stream_k((int)P, (int)d, (int)r)) c.take(gemm_f32_sk_bytes((int)r, (int)d, (int)P));  // Gram pieces
    for (int i = 0; i < 4; ++i) c.take((size_t)P * r * r * 4);  // retraction: Q', S Q, two products of Q's
    return c.off;
  }
  if (call < MAPL_CALL_ENCODE || call > MAPL_CALL_ENCODE_BWD) {
    fail(MAPL_E_SHAPE, "unknown call %d", call);
    return 0;
  }
  if (check_desc(desc) != MAPL_OK) return 0;
  return layout(*desc, call).total;
}

// --------------------------------------------------------------------- encode
extern "C" int mapl_encode(const mapl_codec_desc* desc, const void* X, const int32_t* ids, const float* U,
                           const void* A_s, const void* B_s, const float* C, void* payload, void* ws,
                           size_t ws_bytes, void* stream) {
  g_err.clear();
  int st = check_desc(desc);
  if (st) return st;
  const mapl_codec_desc& D = *desc;
  const int64_t T = D.T, d = D.d, r = D.r, k = D.k;
  const size_t xe = esize(D.x_dtype);
  st = check_ptrs({{X, (size_t)T * d * xe, "X"}, {ids, k > 0 ? (size_t)T * 4 : 0, "ids"},
                   {U, (size_t)d * r * 4, "U"}, {A_s, k > 0 ? (size_t)D.V * k * xe : 0, "A_s"},
                   {B_s, k > 0 ? (size_t)k * b_cols(D) * xe : 0, "B_s"},
                   {C, D.L > 0 ? (size_t)D.L * D.K * r * 4 : 0, "C"}, {payload, payload_bytes(D), "payload"}},
                  {{payload, payload_bytes(D), "payload"}},
                  {{X, (size_t)T * d * xe, "X"}, {ids, (size_t)T * 4, "ids"}, {U, (size_t)d * r * 4, "U"},
                   {A_s, (size_t)D.V * k * xe, "A_s"}, {B_s, (size_t)k * b_cols(D) * xe, "B_s"},
                   {C, (size_t)D.L * D.K * r * 4, "C"}, {ws, ws_bytes, "workspace"}});
  if (st) return st;
  const Layout Lo = layout(D, MAPL_CALL_ENCODE);
  if ((st = check_ws(ws, ws_bytes, Lo.total))) return st;
  hipStream_t s = (hipStream_t)stream;
  if (k > 0 && (st = run_id_check(ids, T, D.V, ws, Lo, s))) return st;
  if (T == 0) return MAPL_OK;
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  const int cbytes = (int)code_bytes(D);

  if (D.x_dtype == MAPL_BF16) {
    // one launch: Wt = [U~^T | -(B_s U~)^T] (or the coordinate anchor's
    // -B_s^T), and the bf16 codebook copy with its norms
    bf16_t* Wt = at<bf16_t>(ws, Lo.w);
    bf16_t* Cb = D.L > 0 ? at<bf16_t>(ws, Lo.cb) : nullptr;
    float* meta = D.L > 0 ? at<float>(ws, Lo.cn2) : nullptr;
    PrepJob jobs[3];
    int nj = 0;
    jobs[nj++] = prep_job_u(U, (int)d, (int)r, nullptr, 0, Wt, Lo.kw);
    if (k > 0) {
      if (amb)  // Wt[c][d+i] = -bf16( (B_s U~)[i][c] )
        jobs[nj++] = prep_job_small_gemm((const bf16_t*)B_s, d, U, r, 0, (int)k, (int)r, (int)d, -1.f, Wt, Lo.kw,
                                         (int)d);
      else
        jobs[nj++] = prep_job_transpose(B_s, 0, (int)k, (int)r, r, -1.f, Wt, Lo.kw, (int)d);
    }
    if (D.L > 0 && !grouped(D)) jobs[nj++] = prep_job_codebook(C, D.L, D.K, (int)r, Cb, meta);
    LAUNCH("enc:prep", launch_prep_batch(jobs, nj, s));
    TnArgs g{};
    g.A = (const bf16_t*)X; g.lda = d; g.Ka = (int)d;
    g.T = (const bf16_t*)A_s; g.ldt = k; g.ids = ids; g.Kg = (int)k; g.V = (int)D.V;
    g.W = Wt; g.ldw = Lo.kw;
    g.M = (int)T; g.N = (int)r;
    if (D.L == 0) {
      g.out = payload; g.ldo = r; g.out_f32 = 0;
      LAUNCH("enc:gemm_tn", launch_gemm_tn(g, s));
      return MAPL_OK;
    }
    if (grouped(D)) {
      float* Z0 = at<float>(ws, Lo.z0);
      g.out = Z0; g.ldo = r; g.out_f32 = 1;
      LAUNCH("enc:gemm_tn", launch_gemm_tn(g, s));
      LAUNCH("enc:grvq", launch_grvq(Z0, C, (int)T, (int)r, D.L, D.K, (uint8_t*)payload, s));
      return MAPL_OK;
    }
    RvqArgs a{};
    a.Z0 = nullptr; a.Cb = Cb; a.C = C; a.meta = meta;
    a.T = (int)T; a.r = (int)r; a.L = D.L; a.K = D.K;
    a.codes = payload; a.code_bytes = cbytes;
    a.stats = nullptr;
    if (g_prof_rvq) {
      a.stats = at<int>(ws, Lo.stats);
      MAPL_HIP(launch_zero_bytes(a.stats, 32, s));
    }
    if (enc_rvq_fusable((int)r, D.L)) {
      // projection and RVQ in one launch: Z0 stays on chip
      LAUNCH("enc:gemm_rvq", launch_enc_rvq(g, a, s));
    } else {
      float* Z0 = at<float>(ws, Lo.z0);
      g.out = Z0; g.ldo = r; g.out_f32 = 1;
      LAUNCH("enc:gemm_tn", launch_gemm_tn(g, s));
      a.Z0 = Z0;
      LAUNCH("enc:rvq", launch_rvq(a, s));
    }
    if (a.stats) {
      // diagnostics mode only: read the counters back (synchronises the stream)
      int h[8];
      MAPL_HIP(hipMemcpyAsync(h, a.stats, sizeof h, hipMemcpyDeviceToHost, s));
      MAPL_HIP(hipStreamSynchronize(s));
      std::lock_guard<std::mutex> lk(g_prof_mu);
      for (int i = 0; i < kRvqStats; ++i) g_rvq_stats[i] += h[i];
    }
    return MAPL_OK;
  }

  // ---------------- fp32 path
  float* out = D.L == 0 ? (float*)payload : at<float>(ws, Lo.z0);
  {
    GemmF32Args g = gemm((int)T, (int)r, (int)d);
    g.A = X; g.sAm = d; g.sAk = 1;
    g.B = U; g.sBk = r; g.sBn = 1;
    g.C = out; g.sCm = r; g.sCn = 1;
    LAUNCH("enc:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  if (k > 0) {
    float* a = at<float>(ws, Lo.ga);
    LAUNCH("enc:gather_rows_f32", launch_gather_rows_f32((const float*)A_s, (int)k, ids, (int)D.V, (int)T, a, s));
    const float* Bk = (const float*)B_s;  // coord: [k,r]
    if (amb) {
      float* BU = at<float>(ws, Lo.bu);
      GemmF32Args g = gemm((int)k, (int)r, (int)d);
      g.A = B_s; g.sAm = d; g.sAk = 1;
      g.B = U; g.sBk = r; g.sBn = 1;
      g.C = BU; g.sCm = r; g.sCn = 1;
      LAUNCH("enc:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
      Bk = BU;
    }
    GemmF32Args g = gemm((int)T, (int)r, (int)k);
    g.A = a; g.sAm = k; g.sAk = 1;
    g.B = Bk; g.sBk = r; g.sBn = 1;
    g.Cin = out; g.sCinm = r; g.sCinn = 1;
    g.C = out; g.sCm = r; g.sCn = 1;
    g.alpha = -1.f; g.beta = 1.f;
    LAUNCH("enc:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  if (grouped(D))
    LAUNCH("enc:grvq", launch_grvq(out, C, (int)T, (int)r, D.L, D.K, (uint8_t*)payload, s));
  else if (D.L > 0)
    LAUNCH("enc:rvq_f32", launch_rvq_f32(out, C, (int)T, (int)r, D.L, D.K, payload, cbytes, s));
  return MAPL_OK;
}

// --------------------------------------------------------------------- decode
extern "C" int mapl_decode(const mapl_codec_desc* desc, const void* payload, const int32_t* ids, const float* U,
                           const void* A_r, const void* B_r, const float* C, void* Xhat, void* ws,
                           size_t ws_bytes, void* stream) {
  g_err.clear();
  int st = check_desc(desc);
  if (st) return st;
  const mapl_codec_desc& D = *desc;
  const int64_t T = D.T, d = D.d, r = D.r, k = D.k;
  const size_t xe = esize(D.x_dtype);
  st = check_ptrs({{payload, payload_bytes(D), "payload"}, {ids, k > 0 ? (size_t)T * 4 : 0, "ids"},
                   {U, (size_t)d * r * 4, "U"}, {A_r, k > 0 ? (size_t)D.V * k * xe : 0, "A_r"},
                   {B_r, k > 0 ? (size_t)k * b_cols(D) * xe : 0, "B_r"},
                   {C, D.L > 0 ? (size_t)D.L * D.K * r * 4 : 0, "C"}, {Xhat, (size_t)T * d * xe, "Xhat"}},
                  {{Xhat, (size_t)T * d * xe, "Xhat"}},
                  {{payload, payload_bytes(D), "payload"}, {ids, (size_t)T * 4, "ids"}, {U, (size_t)d * r * 4, "U"},
                   {A_r, (size_t)D.V * k * xe, "A_r"}, {B_r, (size_t)k * b_cols(D) * xe, "B_r"},
                   {C, (size_t)D.L * D.K * r * 4, "C"}, {ws, ws_bytes, "workspace"}});
  if (st) return st;
  const Layout Lo = layout(D, MAPL_CALL_DECODE);
  if ((st = check_ws(ws, ws_bytes, Lo.total))) return st;
  hipStream_t s = (hipStream_t)stream;
  if (k > 0 && (st = run_id_check(ids, T, D.V, ws, Lo, s))) return st;
  if (T == 0) return MAPL_OK;
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  const int cbytes = (int)code_bytes(D);

  if (D.x_dtype == MAPL_BF16) {
    // one launch: W2 = [U~ | B_r^T] (or the coordinate anchor's (B_r U~^T)^T)
    // and, for codes, Zhat = sum_l C_l[code_l]
    bf16_t* W2 = at<bf16_t>(ws, Lo.w2);
    PrepJob jobs[3];
    int nj = 0;
    jobs[nj++] = prep_job_u(U, (int)d, (int)r, W2, Lo.kw, nullptr, 0);
    if (k > 0) {
      if (amb)
        jobs[nj++] = prep_job_transpose(B_r, 0, (int)k, (int)d, d, 1.f, W2, Lo.kw, (int)r);
      else  // W2[j][r+i] = bf16( sum_c B_r[i][c] U~[j][c] )
        jobs[nj++] = prep_job_small_gemm((const bf16_t*)B_r, r, U, r, 1, (int)k, (int)d, (int)r, 1.f, W2, Lo.kw,
                                         (int)r);
    }
    TnArgs g{};
    g.A = (const bf16_t*)payload; g.lda = r; g.Ka = (int)r;
    g.T = (const bf16_t*)A_r; g.ldt = k; g.ids = ids; g.Kg = (int)k; g.V = (int)D.V;
    g.W = W2; g.ldw = Lo.kw;
    g.M = (int)T; g.N = (int)d;
    g.out = Xhat; g.ldo = d; g.out_f32 = 0;
    if (D.L > 0) {
      // Zhat: gathered by code inside the product's token-operand load where
      // the short-K kernel runs it (whole-vector codewords, L <= 2), else
      // assembled in the preparation launch
      g.codes = payload; g.code_bytes = cbytes; g.C = C; g.L = D.L; g.K = D.K;
      if (grouped(D) || !gemm_tn_gathers(g)) {
        g.codes = nullptr;
        bf16_t* Ah = at<bf16_t>(ws, Lo.ahat);
        AssembleArgs a{};
        a.codes = payload; a.code_bytes = cbytes; a.C = C; a.L = D.L; a.K = D.K;
        a.T = (int)T; a.r = (int)r; a.ldo = r; a.out = Ah; a.gdim = grouped(D) ? 2 : 0;
        jobs[nj++] = prep_job_assemble(a);
        g.A = Ah;
      }
    }
    LAUNCH("dec:prep", launch_prep_batch(jobs, nj, s));
    LAUNCH("dec:gemm_tn", launch_gemm_tn(g, s));
    return MAPL_OK;
  }

  // ---------------- fp32 path
  const float* Zh = (const float*)payload;
  if (D.L > 0) {
    float* z = at<float>(ws, Lo.zh);
    LAUNCH("dec:codes_sum_f32", launch_codes_sum_f32(payload, cbytes, C, (int)T, (int)r, D.L, D.K, z, s, grouped(D) ? 2 : 0));
    Zh = z;
  }
  float* a = k > 0 ? at<float>(ws, Lo.ga) : nullptr;
  if (k > 0) LAUNCH("dec:gather_rows_f32", launch_gather_rows_f32((const float*)A_r, (int)k, ids, (int)D.V, (int)T, a, s));
  if (!amb && k > 0) {
    float* z2 = at<float>(ws, Lo.z2);
    GemmF32Args g = gemm((int)T, (int)r, (int)k);
    g.A = a; g.sAm = k; g.sAk = 1;
    g.B = B_r; g.sBk = r; g.sBn = 1;
    g.Cin = Zh; g.sCinm = r; g.sCinn = 1; g.beta = 1.f;
    g.C = z2; g.sCm = r; g.sCn = 1;
    LAUNCH("dec:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
    Zh = z2;
  }
  {
    GemmF32Args g = gemm((int)T, (int)d, (int)r);
    g.A = Zh; g.sAm = r; g.sAk = 1;
    g.B = U; g.sBk = 1; g.sBn = r;
    g.C = Xhat; g.sCm = d; g.sCn = 1;
    LAUNCH("dec:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  if (amb && k > 0) {
    GemmF32Args g = gemm((int)T, (int)d, (int)k);
    g.A = a; g.sAm = k; g.sAk = 1;
    g.B = B_r; g.sBk = d; g.sBn = 1;
    g.Cin = (const float*)Xhat; g.sCinm = d; g.sCinn = 1; g.beta = 1.f;
    g.C = Xhat; g.sCm = d; g.sCn = 1;
    LAUNCH("dec:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  return MAPL_OK;
}

// ----------------------------------------------------------------- decode_bwd
namespace {
// decode_bwd, and with q != null its gradient-quantising variant: the r-dim
// gradient dXhat U is RVQ-encoded over q's codebooks into q->codes instead
// of being written as dZ (dZ is then null).
int decode_bwd_impl(const mapl_codec_desc* desc, const void* dXhat, const void* payload, const int32_t* ids,
                    const float* U, const void* A_r, const void* B_r, const float* C, void* dZ, float* dU,
                    int accumulate_dU, void* ws, size_t ws_bytes, void* stream, const GradQ* q) {
  int st = check_desc(desc);
  if (st) return st;
  const mapl_codec_desc& D = *desc;
  const int64_t T = D.T, d = D.d, r = D.r, k = D.k;
  const size_t xe = esize(D.x_dtype);
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  const bool need_anchor = !amb && k > 0;
  st = check_ptrs({{dXhat, (size_t)T * d * xe, "dXhat"}, {payload, payload_bytes(D), "payload"},
                   {ids, need_anchor ? (size_t)T * 4 : 0, "ids"}, {U, (size_t)d * r * 4, "U"},
                   {A_r, need_anchor ? (size_t)D.V * k * xe : 0, "A_r"},
                   {B_r, need_anchor ? (size_t)k * r * xe : 0, "B_r"},
                   {C, D.L > 0 ? (size_t)D.L * D.K * r * 4 : 0, "C"}, {dZ, q ? 0 : (size_t)T * r * xe, "dZ"},
                   {dU, (size_t)d * r * 4, "dU"}},
                  {{dZ, q ? 0 : (size_t)T * r * xe, "dZ"}, {dU, (size_t)d * r * 4, "dU"}},
                  {{dXhat, (size_t)T * d * xe, "dXhat"}, {payload, payload_bytes(D), "payload"},
                   {ids, (size_t)T * 4, "ids"}, {U, (size_t)d * r * 4, "U"}, {A_r, (size_t)D.V * k * xe, "A_r"},
                   {B_r, (size_t)k * b_cols(D) * xe, "B_r"}, {C, (size_t)D.L * D.K * r * 4, "C"},
                   {ws, ws_bytes, "workspace"}});
  if (st) return st;
  if (q) {
    const size_t gb = (size_t)q->L * q->K * r * 4, cbn = (size_t)T * q->L * q->code_bytes;
    st = check_ptrs({{q->C, gb, "Cg"}, {q->codes, cbn, "gcodes"}},
                    {{q->codes, cbn, "gcodes"}},
                    {{dXhat, (size_t)T * d * xe, "dXhat"}, {payload, payload_bytes(D), "payload"},
                     {ids, (size_t)T * 4, "ids"}, {U, (size_t)d * r * 4, "U"}, {C, (size_t)D.L * D.K * r * 4, "C"},
                     {q->C, gb, "Cg"}, {dU, (size_t)d * r * 4, "dU"}, {ws, ws_bytes, "workspace"}});
    if (st) return st;
  }
  if (dZ && dU) {
    const uintptr_t a0 = (uintptr_t)dZ, a1 = a0 + T * r * xe, b0 = (uintptr_t)dU, b1 = b0 + d * r * 4;
    if (a0 < b1 && b0 < a1) return fail(MAPL_E_ALIAS, "output dZ overlaps output dU");
  }
  const Layout Lo = layout(D, MAPL_CALL_DECODE_BWD, q);
  if ((st = check_ws(ws, ws_bytes, Lo.total))) return st;
  hipStream_t s = (hipStream_t)stream;
  if (need_anchor && (st = run_id_check(ids, T, D.V, ws, Lo, s))) return st;
  const int cbytes = (int)code_bytes(D);
  if (T == 0) {
    if (!accumulate_dU) LAUNCH("dec_bwd:zero_bytes", launch_zero_bytes(dU, d * r * 4, s));
    return MAPL_OK;
  }

  if (D.x_dtype == MAPL_BF16) {
    // one launch: Ut = U~^T and the second operand of dU (Zhat, plus the
    // coordinate anchor)
    bf16_t* Ut = at<bf16_t>(ws, Lo.w);
    PrepJob jobs[3];
    int nj = 0;
    jobs[nj++] = prep_job_u(U, (int)d, (int)r, nullptr, 0, Ut, d);
    bf16_t* Cbq = q ? at<bf16_t>(ws, Lo.cb) : nullptr;
    float* metaq = q ? at<float>(ws, Lo.cn2) : nullptr;
    if (q) jobs[nj++] = prep_job_codebook(q->C, q->L, q->K, (int)r, Cbq, metaq);
    const bf16_t* Q = (const bf16_t*)payload;
    if (D.L > 0 || need_anchor) {
      bf16_t* Ah = at<bf16_t>(ws, Lo.ahat);
      AssembleArgs a{};
      a.Zp = D.L == 0 ? (const bf16_t*)payload : nullptr;
      a.codes = payload; a.code_bytes = cbytes; a.C = C; a.L = D.L; a.K = D.K;
      if (need_anchor) { a.A = (const bf16_t*)A_r; a.k = (int)k; a.Bc = (const bf16_t*)B_r; a.ids = ids; a.V = (int)D.V; }
      a.T = (int)T; a.r = (int)r; a.ldo = r; a.out = Ah; a.gdim = grouped(D) ? 2 : 0;
      jobs[nj++] = prep_job_assemble(a);
      Q = Ah;
    }
    LAUNCH("dec_bwd:prep", launch_prep_batch(jobs, nj, s));
    TnArgs g{};
    g.A = (const bf16_t*)dXhat; g.lda = d; g.Ka = (int)d;
    g.W = Ut; g.ldw = d;
    g.M = (int)T; g.N = (int)r;
    if (!q) {
      g.out = dZ; g.ldo = r; g.out_f32 = 0;
      LAUNCH("dec_bwd:gemm_tn", launch_gemm_tn(g, s));
    } else {
      // the gradient's RVQ, as the encoder's: fused with the GEMM at r = 256
      RvqArgs a{};
      a.Cb = Cbq; a.C = q->C; a.meta = metaq;
      a.T = (int)T; a.r = (int)r; a.L = q->L; a.K = q->K;
      a.codes = q->codes; a.code_bytes = q->code_bytes;
      if (enc_rvq_fusable((int)r, q->L)) {
        LAUNCH("dec_bwd_q:gemm_rvq", launch_enc_rvq(g, a, s));
      } else {
        float* Z0 = at<float>(ws, Lo.z0);
        g.out = Z0; g.ldo = r; g.out_f32 = 1;
        LAUNCH("dec_bwd_q:gemm_tn", launch_gemm_tn(g, s));
        a.Z0 = Z0;
        LAUNCH("dec_bwd_q:rvq", launch_rvq(a, s));
      }
    }
    WgradArgs w{};
    w.Pa = (const bf16_t*)dXhat; w.ldp = d; w.Ma = (int)d;
    w.Q = Q; w.ldq = r;
    w.T = (int)T; w.N = (int)r; w.splits = Lo.sp.splits; w.tokens_per_split = Lo.sp.tps;
    w.part = at<float>(ws, Lo.part);
    LAUNCH("dec_bwd:wgrad", launch_wgrad(w, s));
    LAUNCH("dec_bwd:reduce", launch_reduce_splits(w.part, w.splits, (int)d, (int)r,
                                                  (int64_t)wgrad_row_offset((int)d) * r, dU, accumulate_dU, s));
    return MAPL_OK;
  }

  // ---------------- fp32 path
  {
    GemmF32Args g = gemm((int)T, (int)r, (int)d);
    g.A = dXhat; g.sAm = d; g.sAk = 1;
    g.B = U; g.sBk = r; g.sBn = 1;
    g.C = q ? (void*)at<float>(ws, Lo.z0) : dZ; g.sCm = r; g.sCn = 1;
    LAUNCH("dec_bwd:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
    if (q)
      LAUNCH("dec_bwd_q:rvq_f32", launch_rvq_f32(at<float>(ws, Lo.z0), q->C, (int)T, (int)r, q->L, q->K, q->codes,
                                                 q->code_bytes, s));
  }
  const float* Zh = (const float*)payload;
  if (D.L > 0) {
    float* z = at<float>(ws, Lo.zh);
    LAUNCH("dec_bwd:codes_sum_f32", launch_codes_sum_f32(payload, cbytes, C, (int)T, (int)r, D.L, D.K, z, s, grouped(D) ? 2 : 0));
    Zh = z;
  }
  if (need_anchor) {
    float* a = at<float>(ws, Lo.ga);
    LAUNCH("dec_bwd:gather_rows_f32", launch_gather_rows_f32((const float*)A_r, (int)k, ids, (int)D.V, (int)T, a, s));
    float* z2 = at<float>(ws, Lo.z2);
    GemmF32Args g = gemm((int)T, (int)r, (int)k);
    g.A = a; g.sAm = k; g.sAk = 1;
    g.B = B_r; g.sBk = r; g.sBn = 1;
    g.Cin = Zh; g.sCinm = r; g.sCinn = 1; g.beta = 1.f;
    g.C = z2; g.sCm = r; g.sCn = 1;
    LAUNCH("dec_bwd:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
    Zh = z2;
  }
  {
    GemmF32Args g = gemm((int)d, (int)r, (int)T);
    g.A = dXhat; g.sAm = 1; g.sAk = d;
    g.B = Zh; g.sBk = r; g.sBn = 1;
    if (accumulate_dU) { g.Cin = dU; g.sCinm = r; g.sCinn = 1; g.beta = 1.f; }
    g.C = dU; g.sCm = r; g.sCn = 1;
    LAUNCH("dec_bwd:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  return MAPL_OK;
}
}  // namespace

extern "C" int mapl_decode_bwd(const mapl_codec_desc* desc, const void* dXhat, const void* payload,
                               const int32_t* ids, const float* U, const void* A_r, const void* B_r, const float* C,
                               void* dZ, float* dU, int accumulate_dU, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  return decode_bwd_impl(desc, dXhat, payload, ids, U, A_r, B_r, C, dZ, dU, accumulate_dU, ws, ws_bytes, stream,
                         nullptr);
}

namespace {
int check_gradq(const mapl_codec_desc* desc, int32_t Lg, int32_t Kg, int32_t gcode_dtype) {
  if (Lg < 1 || Lg > 8) return fail(MAPL_E_SHAPE, "gradient RVQ: need 1 <= Lg <= 8 (got %d)", Lg);
  if (Kg < 32 || Kg > 65536 || Kg % 32) return fail(MAPL_E_SHAPE, "gradient RVQ: need 32 <= Kg <= 65536, Kg %% 32 == 0");
  if (gcode_dtype == MAPL_U8) {
    if (Kg > 256) return fail(MAPL_E_RANGE, "Kg=%d does not fit MAPL_U8 codes", Kg);
  } else if (gcode_dtype != MAPL_U16) {
    return fail(MAPL_E_DTYPE, "gcode_dtype must be MAPL_U8 or MAPL_U16 (got %d)", gcode_dtype);
  }
  if (desc && desc->x_dtype == MAPL_BF16 && desc->r != 64 && desc->r != 128 && desc->r != 256)
    return fail(MAPL_E_UNSUPPORTED, "gradient RVQ on the bf16 path supports r in {64, 128, 256}");
  return MAPL_OK;
}
}  // namespace

extern "C" int mapl_decode_bwd_q(const mapl_codec_desc* desc, const void* dXhat, const void* payload,
                                 const int32_t* ids, const float* U, const void* A_r, const void* B_r, const float* C,
                                 int32_t Lg, int32_t Kg, int32_t gcode_dtype, const float* Cg, void* gcodes,
                                 float* dU, int accumulate_dU, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  int st = check_desc(desc);
  if (st) return st;
  if ((st = check_gradq(desc, Lg, Kg, gcode_dtype))) return st;
  GradQ q{Lg, Kg, gcode_dtype == MAPL_U8 ? 1 : 2, Cg, gcodes};
  return decode_bwd_impl(desc, dXhat, payload, ids, U, A_r, B_r, C, nullptr, dU, accumulate_dU, ws, ws_bytes,
                         stream, &q);
}

extern "C" size_t mapl_decode_bwd_q_workspace_bytes(const mapl_codec_desc* desc, int32_t Lg, int32_t Kg) {
  g_err.clear();
  if (check_desc(desc) != MAPL_OK) return 0;
  if (check_gradq(desc, Lg, Kg, Kg <= 256 ? MAPL_U8 : MAPL_U16) != MAPL_OK) return 0;
  GradQ q{Lg, Kg, Kg <= 256 ? 1 : 2, nullptr, nullptr};
  return layout(*desc, MAPL_CALL_DECODE_BWD, &q).total;
}

extern "C" int mapl_grad_dequantize(int64_t T, int64_t r, int32_t Lg, int32_t Kg, int32_t gcode_dtype,
                                    const void* gcodes, const float* Cg, int32_t out_dtype, void* dZ, void* stream) {
  g_err.clear();
  int st = check_gradq(nullptr, Lg, Kg, gcode_dtype);
  if (st) return st;
  if (T < 0 || T >= ((int64_t)1 << 31)) return fail(MAPL_E_SHAPE, "T=%lld out of range", (long long)T);
  if (r < 32 || r > 1024 || r % 32) return fail(MAPL_E_SHAPE, "r=%lld: need 32 <= r <= 1024, r %% 32 == 0", (long long)r);
  if (out_dtype != MAPL_BF16 && out_dtype != MAPL_F32) return fail(MAPL_E_DTYPE, "out_dtype must be MAPL_BF16 or MAPL_F32");
  const int cb = gcode_dtype == MAPL_U8 ? 1 : 2;
  const size_t nc = (size_t)T * Lg * cb, ng = (size_t)Lg * Kg * r * 4, no = (size_t)T * r * esize(out_dtype);
  st = check_ptrs({{gcodes, nc, "gcodes"}, {Cg, ng, "Cg"}, {dZ, no, "dZ"}}, {{dZ, no, "dZ"}},
                  {{gcodes, nc, "gcodes"}, {Cg, ng, "Cg"}});
  if (st) return st;
  if (T == 0) return MAPL_OK;
  hipStream_t s = (hipStream_t)stream;
  if (out_dtype == MAPL_F32) {
    LAUNCH("grad_dq:codes_sum_f32", launch_codes_sum_f32(gcodes, cb, Cg, (int)T, (int)r, Lg, Kg, (float*)dZ, s));
  } else {
    AssembleArgs a{};
    a.codes = gcodes; a.code_bytes = cb; a.C = Cg; a.L = Lg; a.K = Kg;
    a.T = (int)T; a.r = (int)r; a.ldo = r; a.out = (bf16_t*)dZ;
    LAUNCH("grad_dq:assemble", launch_assemble(a, s));
  }
  return MAPL_OK;
}

// ----------------------------------------------------------------- encode_bwd
extern "C" int mapl_encode_bwd(const mapl_codec_desc* desc, const void* dZ, const void* X, const int32_t* ids,
                               const float* U, const void* A_s, const void* B_s, void* dX, float* dU,
                               int accumulate_dU, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  int st = check_desc(desc);
  if (st) return st;
  const mapl_codec_desc& D = *desc;
  const int64_t T = D.T, d = D.d, r = D.r, k = D.k;
  const size_t xe = esize(D.x_dtype);
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  const bool need_anchor = amb && k > 0;
  st = check_ptrs({{dZ, (size_t)T * r * xe, "dZ"}, {X, (size_t)T * d * xe, "X"},
                   {ids, need_anchor ? (size_t)T * 4 : 0, "ids"}, {U, (size_t)d * r * 4, "U"},
                   {A_s, need_anchor ? (size_t)D.V * k * xe : 0, "A_s"},
                   {B_s, need_anchor ? (size_t)k * d * xe : 0, "B_s"}, {dX, (size_t)T * d * xe, "dX"},
                   {dU, (size_t)d * r * 4, "dU"}},
                  {{dX, (size_t)T * d * xe, "dX"}, {dU, (size_t)d * r * 4, "dU"}},
                  {{dZ, (size_t)T * r * xe, "dZ"}, {X, (size_t)T * d * xe, "X"}, {ids, (size_t)T * 4, "ids"},
                   {U, (size_t)d * r * 4, "U"}, {A_s, (size_t)D.V * k * xe, "A_s"},
                   {B_s, (size_t)k * b_cols(D) * xe, "B_s"}, {ws, ws_bytes, "workspace"}});
  if (st) return st;
  if (dX && dU) {
    const uintptr_t a0 = (uintptr_t)dX, a1 = a0 + T * d * xe, b0 = (uintptr_t)dU, b1 = b0 + d * r * 4;
    if (a0 < b1 && b0 < a1) return fail(MAPL_E_ALIAS, "output dX overlaps output dU");
  }
  const Layout Lo = layout(D, MAPL_CALL_ENCODE_BWD);
  if ((st = check_ws(ws, ws_bytes, Lo.total))) return st;
  hipStream_t s = (hipStream_t)stream;
  if (need_anchor && (st = run_id_check(ids, T, D.V, ws, Lo, s))) return st;
  if (T == 0) {
    if (!accumulate_dU) LAUNCH("enc_bwd:zero_bytes", launch_zero_bytes(dU, d * r * 4, s));
    return MAPL_OK;
  }

  if (D.x_dtype == MAPL_BF16) {
    // one launch: Ub = U~ and the gathered sender anchors a_s
    bf16_t* Ub = at<bf16_t>(ws, Lo.w2);
    bf16_t* ga = need_anchor ? at<bf16_t>(ws, Lo.ga) : nullptr;
    PrepJob jobs[2];
    int nj = 0;
    jobs[nj++] = prep_job_u(U, (int)d, (int)r, Ub, r, nullptr, 0);
    if (need_anchor) jobs[nj++] = prep_job_gather((const bf16_t*)A_s, (int)k, ids, (int)D.V, (int)T, ga);
    LAUNCH("enc_bwd:prep", launch_prep_batch(jobs, nj, s));
    TnArgs g{};
    g.A = (const bf16_t*)dZ; g.lda = r; g.Ka = (int)r;
    g.W = Ub; g.ldw = r;
    g.M = (int)T; g.N = (int)d;
    g.out = dX; g.ldo = d; g.out_f32 = 0;
    LAUNCH("enc_bwd:gemm_tn", launch_gemm_tn(g, s));
    WgradArgs w{};
    w.Pa = (const bf16_t*)X; w.ldp = d; w.Ma = (int)d;
    if (need_anchor) {
      w.Tg = ga; w.Mg = (int)k;
    }
    w.Q = (const bf16_t*)dZ; w.ldq = r;
    w.T = (int)T; w.N = (int)r; w.splits = Lo.sp.splits; w.tokens_per_split = Lo.sp.tps;
    w.part = at<float>(ws, Lo.part);
    const int64_t mao = wgrad_row_offset((int)d);
    const int64_t stride = (mao + w.Mg) * r;
    LAUNCH("enc_bwd:wgrad", launch_wgrad(w, s));
    if (need_anchor) {
      // dU = sum of the partials - B_s^T (a_s^T dZ); a_s^T dZ is summed first
      // from the anchor rows of the partials
      float* Wa = at<float>(ws, Lo.wsum);
      LAUNCH("enc_bwd:anchor_reduce", launch_reduce_splits(w.part + mao * r, w.splits, (int)k, (int)r, stride, Wa, 0, s));
      LAUNCH("enc_bwd:reduce_corr", launch_reduce_dU(w.part, w.splits, stride, (int)d, (int)r, dU, accumulate_dU,
                                                     (const bf16_t*)B_s, Wa, (int)k, s));
    } else {
      LAUNCH("enc_bwd:reduce", launch_reduce_splits(w.part, w.splits, (int)d, (int)r, stride, dU, accumulate_dU, s));
    }
    return MAPL_OK;
  }

  // ---------------- fp32 path
  {
    GemmF32Args g = gemm((int)T, (int)d, (int)r);
    g.A = dZ; g.sAm = r; g.sAk = 1;
    g.B = U; g.sBk = 1; g.sBn = r;
    g.C = dX; g.sCm = d; g.sCn = 1;
    LAUNCH("enc_bwd:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  {
    GemmF32Args g = gemm((int)d, (int)r, (int)T);
    g.A = X; g.sAm = 1; g.sAk = d;
    g.B = dZ; g.sBk = r; g.sBn = 1;
    if (accumulate_dU) { g.Cin = dU; g.sCinm = r; g.sCinn = 1; g.beta = 1.f; }
    g.C = dU; g.sCm = r; g.sCn = 1;
    LAUNCH("enc_bwd:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  if (need_anchor) {
    float* a = at<float>(ws, Lo.ga);
    float* Wm = at<float>(ws, Lo.wsum);
    LAUNCH("enc_bwd:gather_rows_f32", launch_gather_rows_f32((const float*)A_s, (int)k, ids, (int)D.V, (int)T, a, s));
    GemmF32Args g = gemm((int)k, (int)r, (int)T);
    g.A = a; g.sAm = 1; g.sAk = k;
    g.B = dZ; g.sBk = r; g.sBn = 1;
    g.C = Wm; g.sCm = r; g.sCn = 1;
    LAUNCH("enc_bwd:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
    GemmF32Args e = gemm((int)d, (int)r, (int)k);
    e.A = B_s; e.sAm = 1; e.sAk = d;
    e.B = Wm; e.sBk = r; e.sBn = 1;
    e.Cin = dU; e.sCinm = r; e.sCinn = 1; e.beta = 1.f;
    e.C = dU; e.sCm = r; e.sCn = 1;
    e.alpha = -1.f;
    LAUNCH("enc_bwd:gemm_f32", launch_gemm_f32(e, 0, 0, 0, s));
  }
  return MAPL_OK;
}

// ---------------------------------------------------------------- stiefel
extern "C" int mapl_stiefel_step(int64_t P, int64_t d, int64_t r, float* U, const float* G, float* M, float lr,
                                 float beta, int lmo_steps, int retract_steps, void* ws, size_t ws_bytes,
                                 void* stream) {
  g_err.clear();
  if (P < 1 || P > 65535 || d < 32 || r < 32 || r > d || r > 1024 || r % 32 || d % 32 || d > 65536)
    return fail(MAPL_E_SHAPE, "stiefel: need 1 <= P <= 65535, 32 <= r <= min(d,1024), d <= 65536, r and d multiples of 32");
  if (lmo_steps < 1 || lmo_steps > kPolarMaxSteps || retract_steps < 1 || retract_steps > kPolarMaxSteps)
    return fail(MAPL_E_SHAPE, "stiefel: 1 <= lmo_steps, retract_steps <= %d", kPolarMaxSteps);
  if (!(beta >= 0.f && beta < 1.f)) return fail(MAPL_E_RANGE, "stiefel: beta must lie in [0, 1)");
  if (!(lr >= 0.f && lr < 1.f)) return fail(MAPL_E_RANGE, "stiefel: lr must lie in [0, 1)");
  const size_t nb = (size_t)P * d * r * 4;
  int st = check_ptrs({{U, nb, "U"}, {G, nb, "G"}, {M, nb, "M"}}, {{U, nb, "U"}, {M, nb, "M"}},
                      {{G, nb, "G"}, {ws, ws_bytes, "workspace"}});
  if (st) return st;
  {
    const uintptr_t a0 = (uintptr_t)U, b0 = (uintptr_t)M;
    if (a0 < b0 + nb && b0 < a0 + nb) return fail(MAPL_E_ALIAS, "U overlaps M");
  }
  const size_t need = mapl_workspace_bytes(nullptr, MAPL_CALL_STIEFEL, P, d, r);
  if ((st = check_ws(ws, ws_bytes, need))) return st;
  hipStream_t s = (hipStream_t)stream;

  Carve c;
  float* S = at<float>(ws, c.take((size_t)P * r * r * 4));
  float* Qm = at<float>(ws, c.take((size_t)P * r * r * 4));
  float* X0 = at<float>(ws, c.take((size_t)P * d * r * 4));
  float* X1 = at<float>(ws, c.take((size_t)P * d * r * 4));
  float* partial = at<float>(ws, c.take((size_t)P * 2048 * 4));
  float* sc = at<float>(ws, c.take((size_t)P * 8 * 4));
  float* skp = gram_stream_k((int)P, (int)d, (int)r)
                   ? at<float>(ws, c.take(gemm_f32_sk_bytes((int)r, (int)d, (int)P)))
                   : nullptr;
  float* Q2 = at<float>(ws, c.take((size_t)P * r * r * 4));
  float* Tm = at<float>(ws, c.take((size_t)P * r * r * 4));
  float* Pq[2] = {at<float>(ws, c.take((size_t)P * r * r * 4)), at<float>(ws, c.take((size_t)P * r * r * 4))};
  float* scale = sc, *inv_nu = sc + P, *inv_nu2 = sc + 2 * P;
  const int64_t n = d * r, rr = r * r;

  // split: GEMM_SPLIT_F16 takes the products from fp16 pieces (hi.hi +
  // hi.lo + lo.hi) on the 16-bit matrix units, with fp32's accuracy for
  // operands below 255 (PolarExpress below keeps them there); Eq. 4 and the
  // Gram product of Y (any norm) run on the fp32 matrix units.
  // S = X^T X (X scaled by pre inside the split)
  auto gram = [&](const float* X, int split, const float* pre) {
    GemmF32Args g = gemm((int)r, (int)r, (int)d);
    g.split = split;
    g.pre_a = g.pre_b = pre;
    g.sym_upper = 1;  // X^T X: the tiles above the diagonal, mirrored
    g.batch = (int)P;
    g.A = X; g.sAm = 1; g.sAk = r; g.sAb = n;
    g.B = X; g.sBk = r; g.sBn = 1; g.sBb = n;
    g.C = S; g.sCm = r; g.sCn = 1; g.sCb = rr;
    g.sk_part = skp;  // split over two workgroups per CU where the upper tiles are fewer
    return launch_gemm_f32(g, 0, 0, 0, s);
  };
  // Qo = (a I + b S' + c S' S') / a with S' = sp S (sp: a per-projector
  // factor, or none); symmetric, like every r x r product of the iteration
  // below
  auto poly = [&](double a, double b, double cc, const float* sp, float* Qo) {
    GemmF32Args g = gemm((int)r, (int)r, (int)r);
    g.split = GEMM_SPLIT_F16;
    g.sym_upper = 1;
    g.pre_a = g.pre_b = sp;
    g.batch = (int)P;
    g.A = S; g.sAm = r; g.sAk = 1; g.sAb = rr;
    g.B = S; g.sBk = r; g.sBn = 1; g.sBb = rr;
    g.Cin = S; g.sCinm = r; g.sCinn = 1; g.sCinb = rr;
    g.C = Qo; g.sCm = r; g.sCn = 1; g.sCb = rr;
    g.alpha = (float)(cc / a); g.beta = (float)(b / a); g.diag = 1.f;
    g.beta_ptr = sp;
    return launch_gemm_f32(g, 0, 0, 0, s);
  };
  // Xo = alpha X' Bm with X' = pre X, or with Yin: Xo = Yin - lr alpha X' Bm
  // (the LMO's last product and Eq. 7's argument U - lr D in one launch)
  auto apply = [&](const float* X, const float* pre, const float* Bm, float* Xo, const float* Yin, double alpha) {
    GemmF32Args g = gemm((int)d, (int)r, (int)r);
    g.split = GEMM_SPLIT_F16;
    g.pre_a = pre;
    g.batch = (int)P;
    g.A = X; g.sAm = r; g.sAk = 1; g.sAb = n;
    g.B = Bm; g.sBk = r; g.sBn = 1; g.sBb = rr;
    g.C = Xo; g.sCm = r; g.sCn = 1; g.sCb = n;
    g.alpha = (float)alpha;
    if (Yin) {
      g.Cin = Yin; g.sCinm = r; g.sCinn = 1; g.sCinb = n; g.beta = 1.f;
      g.alpha = (float)(-lr * alpha);
    }
    return launch_gemm_f32(g, 0, 0, 0, s);
  };
  // Co = (A scaled by pre inside) B for r x r factors, fp16 split; sym: the
  // product is symmetric (upper tiles computed, mirrored)
  auto rmul = [&](float* Co, const float* Am, const float* Bm, const float* pre, bool sym, double alpha = 1.0) {
    GemmF32Args g = gemm((int)r, (int)r, (int)r);
    g.split = GEMM_SPLIT_F16;
    g.alpha = (float)alpha;
    g.pre_a = pre;
    g.sym_upper = sym ? 1 : 0;
    g.batch = (int)P;
    g.A = Am; g.sAm = r; g.sAk = 1; g.sAb = rr;
    g.B = Bm; g.sBk = r; g.sBn = 1; g.sBb = rr;
    g.C = Co; g.sCm = r; g.sCn = 1; g.sCb = rr;
    return launch_gemm_f32(g, 0, 0, 0, s);
  };

  // C1 = A1 Bm and C2 = A2 Bm in one launch (two symmetric r x r products sharing Bm)
  auto rmul2 = [&](float* C1, const float* A1, float* C2o, const float* A2m, const float* Bm) {
    GemmF32Args g = gemm((int)r, (int)r, (int)r);
    g.split = GEMM_SPLIT_F16;
    g.sym_upper = 1;
    g.batch = 2 * (int)P;
    g.bsplit = (int)P;
    g.A = A1; g.A2 = A2m; g.sAm = r; g.sAk = 1; g.sAb = rr;
    g.B = Bm; g.sBk = r; g.sBn = 1; g.sBb = rr;
    g.C = C1; g.C2 = C2o; g.sCm = r; g.sCn = 1; g.sCb = rr;
    return launch_gemm_f32(g, 0, 0, 0, s);
  };

  // Eq. 4: S = U^T G, sym, g_R = G - U sym(S)  -> X0
  {
    GemmF32Args g = gemm((int)r, (int)r, (int)d);
    g.batch = (int)P;
    g.A = U; g.sAm = 1; g.sAk = r; g.sAb = n;
    g.B = G; g.sBk = r; g.sBn = 1; g.sBb = n;
    g.C = S; g.sCm = r; g.sCn = 1; g.sCb = rr;
    LAUNCH("stiefel:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  LAUNCH("stiefel:symmetrize", launch_symmetrize(S, (int)P, (int)r, s));
  {
    GemmF32Args g = gemm((int)d, (int)r, (int)r);
    g.batch = (int)P;
    g.A = U; g.sAm = r; g.sAk = 1; g.sAb = n;
    g.B = S; g.sBk = r; g.sBn = 1; g.sBb = rr;
    g.Cin = G; g.sCinm = r; g.sCinn = 1; g.sCinb = n; g.beta = 1.f;
    g.C = X0; g.sCm = r; g.sCn = 1; g.sCb = n;
    g.alpha = -1.f;
    LAUNCH("stiefel:gemm_f32", launch_gemm_f32(g, 0, 0, 0, s));
  }
  // Eq. 5 and the LMO normalisation 1 / (||M||_F + 1e-7); the LMO is 0 for
  // a momentum at or below 2^-20 ||G||_F (under fp32 resolution of G)
  int nblk = (int)((n + 255) / 256);
  if (nblk > 1024) nblk = 1024;
  LAUNCH("stiefel:momentum", launch_momentum(M, X0, G, n, (int)P, beta, partial, nblk, s));
  LAUNCH("stiefel:fro_scale", launch_fro_scale(partial, nblk, (int)P, 1e-7f, 1.0f / 1048576.0f, scale, s));

  // PolarExpress (Eqs. 6 and 7) with the iterates carried in the r x r
  // space: for X_i = X_0 Q_0 ... Q_{i-1}, S_i = X_i^T X_i,
  // Q_i = a I + b S_i + c S_i^2, S_{i+1} = Q_i (S_i Q_i) and
  // P_{i+1} = P_i Q_i, and X_j = X_i P_j -- the same iterates, with r^3
  // products in place of each step's d r^2 Gram and apply products (the Q_i
  // are polynomials in S_i and commute with it).  Every product runs in the
  // fp16 split, whose operands must stay below 255, and the factors carry
  // Q~_i = Q_i / a_i, P~ = Q~_i ... Q~_{j-1}, with S_{i+1} = a_i^2 Q~_i (S_i Q~_i)
  // and X_j = (a_i ... a_{j-1}) X_i P~: X_0 has spectral norm <= 1
  // (M / (||M||_F + eps), Y / nu), both schedules keep every singular value
  // below 2.1 (so X, S and S Q~ stay below 5), and each quintic p has
  // |p(x)| <= a x on the values it meets, so Q~ and P~ have eigenvalues in
  // [-1, 1].  A segment runs while its a's multiply to at most kSegGrowth,
  // which keeps P~'s entries for the unit singular values above 2^-11 (the
  // fp16 split's full-precision range; the paper's schedules, 5 and 7
  // steps, are one segment each: 1043 and 116); a longer schedule forms
  // X_j = X_i P_j at a segment's end and starts the next from X_j's Gram
  // product.  On entry S holds X_0^T X_0 divided by spre (the first step's
  // products scale it by spre inside, null: 1); X_0 is Xs scaled by xpre
  // inside its one product.  X_K, or Yin - lr X_K, goes to out (null: the X
  // buffer not read last), and *written names the buffer.
  constexpr double kSegGrowth = 2048.0;
  float* bufs[2] = {X0, X1};
  auto other = [&](const float* p) { return p == bufs[0] ? bufs[1] : bufs[0]; };
  auto polar_rr = [&](const double (*coef)[3], int steps, const float* Xs, const float* xpre, const float* spre,
                      float* out, const float* Yin, float** written) -> int {
    const float* Xseg = Xs;
    for (int i = 0; i < steps;) {
      int j = i;
      double growth = 1.0;
      for (; j < steps && (j == i || growth * coef[j][0] <= kSegGrowth); ++j) growth *= coef[j][0];
      if (i > 0) LAUNCH("stiefel:pe_gram", gram(Xseg, GEMM_SPLIT_F16, nullptr));  // S_i = X_i^T X_i
      const float* Pprev = nullptr;
      int pq = 0;
      for (int k = i; k < j; ++k) {
        const double a = coef[k][0], b = coef[k][1], cc = coef[k][2];
        const float* sp = k == 0 ? spre : nullptr;
        float* Q = (k & 1) ? Q2 : Qm;
        LAUNCH("stiefel:pe_poly", poly(a, b, cc, sp, Q));  // Q~_k
        const bool pprod = k > i, supd = k + 1 < j;  // P~ <- P~ Q~_k; S_{k+1} = a^2 Q~_k (S_k Q~_k)
        // S_k, Q~_k and P~ are polynomials in the segment's first S, so they
        // commute and every product here is symmetric: each computes the
        // tiles on and above the diagonal and mirrors them
        if (pprod && supd)  // S_k Q~_k and P~ Q~_k share Q~_k: one launch (sp is null past step 0)
          LAUNCH("stiefel:pe_sq_p", rmul2(Tm, S, Pq[pq], Pprev, Q));
        else if (pprod)
          LAUNCH("stiefel:pe_p", rmul(Pq[pq], Pprev, Q, nullptr, true));
        else if (supd)
          LAUNCH("stiefel:pe_sq", rmul(Tm, S, Q, sp, true));
        if (pprod) {
          Pprev = Pq[pq];
          pq ^= 1;
        } else {
          Pprev = Q;  // P~ = Q~_i
        }
        if (supd) LAUNCH("stiefel:pe_s", rmul(S, Q, Tm, nullptr, true, a * a));  // S_{k+1} (symmetric)
      }
      float* Xo = j == steps && out ? out : other(Xseg);
      LAUNCH("stiefel:pe_apply",
             apply(Xseg, i == 0 ? xpre : nullptr, Pprev, Xo, j == steps ? Yin : nullptr, growth));
      Xseg = Xo;
      i = j;
    }
    if (written) *written = (float*)Xseg;
    return MAPL_OK;
  };

  // Eq. 6: D = PE(M / (||M||_F + eps)); the last product writes Y = U - lr D
  // (D itself is not kept)
  LAUNCH("stiefel:lmo_gram", gram(M, GEMM_SPLIT_F16, scale));
  float* Y = nullptr;
  if ((st = polar_rr(kLmoCoef, lmo_steps, M, scale, nullptr, nullptr, U, &Y))) return st;
  // Eq. 7: U = PE(Y / nu), nu^2 = max row sum |Y^T Y|: Y^T Y in fp32 (it fixes nu)
  LAUNCH("stiefel:gram", gram(Y, GEMM_SPLIT_NONE, nullptr));
  // (the momentum's norm partials are consumed by now; their buffer takes the row maxima)
  LAUNCH("stiefel:inf_norm_scales", launch_inf_norm_scales(S, (int)P, (int)r, partial, inv_nu, inv_nu2, s));
  if ((st = polar_rr(kRetractCoef, retract_steps, Y, inv_nu, inv_nu2, U, nullptr, nullptr))) return st;
  return MAPL_OK;
}

// ------------------------------------------------------ anchor-table gradient
namespace {
struct AnchorLayout {
  size_t total = 0, w = 0, bu = 0, g = 0, k0 = 0, v0 = 0, k1 = 0, v1 = 0, hist = 0, headp = 0, tailp = 0, hid = 0,
         hthru = 0, tid = 0;
  int kp = 0, K = 0, passes = 1, nsub = 0;
};

constexpr int64_t kAnchorMaxT = (int64_t)1 << 24;

int check_anchor_bwd(const mapl_codec_desc* desc, int side) {
  int st = check_desc(desc);
  if (st) return st;
  if (side != MAPL_SENDER && side != MAPL_RECEIVER) return fail(MAPL_E_SHAPE, "side must be MAPL_SENDER or MAPL_RECEIVER");
  if (desc->k < 1) return fail(MAPL_E_SHAPE, "anchor gradient needs k >= 1");
  if (desc->T > kAnchorMaxT) return fail(MAPL_E_SHAPE, "anchor gradient: T=%lld above 2^24", (long long)desc->T);
  return MAPL_OK;
}

AnchorLayout anchor_layout(const mapl_codec_desc& D, int side) {
  AnchorLayout Lo;
  Carve c;
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  const int64_t T = D.T;
  Lo.K = (int)((side == MAPL_RECEIVER && amb) ? D.d : D.r);  // width of the incoming gradient
  Lo.kp = (int)rup(D.k, 64);
  if (D.x_dtype == MAPL_BF16) Lo.w = c.take((size_t)Lo.kp * Lo.K * 2);
  else if (side == MAPL_SENDER && amb) Lo.bu = c.take((size_t)D.k * D.r * 4);
  Lo.g = c.take((size_t)T * Lo.kp * 4);
  Lo.k0 = c.take((size_t)T * 4);
  Lo.v0 = c.take((size_t)T * 4);
  Lo.k1 = c.take((size_t)T * 4);
  Lo.v1 = c.take((size_t)T * 4);
  Lo.hist = c.take((size_t)256 * radix_tiles((int)T) * 4);
  Lo.nsub = anchor_sub_chunks((int)T);
  Lo.headp = c.take((size_t)Lo.nsub * D.k * 4);
  Lo.tailp = c.take((size_t)Lo.nsub * D.k * 4);
  Lo.hid = c.take((size_t)Lo.nsub * 4);
  Lo.hthru = c.take((size_t)Lo.nsub * 4);
  Lo.tid = c.take((size_t)Lo.nsub * 4);
  int bits = 0;
  for (int64_t v = D.V - 1; v > 0; v >>= 1) ++bits;
  Lo.passes = bits > 8 ? (bits + 7) / 8 : 1;
  Lo.total = c.off;
  return Lo;
}
}  // namespace

extern "C" size_t mapl_anchor_bwd_workspace_bytes(const mapl_codec_desc* desc, int side) {
  g_err.clear();
  if (check_anchor_bwd(desc, side) != MAPL_OK) return 0;
  return anchor_layout(*desc, side).total;
}

extern "C" int mapl_anchor_bwd(const mapl_codec_desc* desc, int side, const void* dY, const int32_t* ids,
                               const float* U, const void* B, float* dA, int accumulate, void* ws, size_t ws_bytes,
                               void* stream) {
  g_err.clear();
  int st = check_anchor_bwd(desc, side);
  if (st) return st;
  const mapl_codec_desc& D = *desc;
  const int64_t T = D.T, d = D.d, r = D.r, k = D.k;
  const size_t xe = esize(D.x_dtype);
  const bool amb = D.anchor_space == MAPL_ANCHOR_AMBIENT;
  const bool need_u = side == MAPL_SENDER && amb;
  const AnchorLayout Lo = anchor_layout(D, side);
  const size_t ny = (size_t)T * Lo.K * xe, na = (size_t)D.V * k * 4;
  st = check_ptrs({{dY, ny, "dY"}, {ids, (size_t)T * 4, "ids"}, {U, need_u ? (size_t)d * r * 4 : 0, "U"},
                   {B, (size_t)k * b_cols(D) * xe, "B"}, {dA, na, "dA"}},
                  {{dA, na, "dA"}},
                  {{dY, ny, "dY"}, {ids, (size_t)T * 4, "ids"}, {U, need_u ? (size_t)d * r * 4 : 0, "U"},
                   {B, (size_t)k * b_cols(D) * xe, "B"}, {ws, ws_bytes, "workspace"}});
  if (st) return st;
  if ((st = check_ws(ws, ws_bytes, Lo.total))) return st;
  hipStream_t s = (hipStream_t)stream;
  if (!accumulate) LAUNCH("anchor_bwd:zero", launch_zero_bytes(dA, (int64_t)na, s));
  if (T == 0) return MAPL_OK;
  if (debug_ids()) {
    Layout tmp;
    tmp.flag = Lo.hid;  // the head-id slots are written later in the call
    if ((st = run_id_check(ids, T, D.V, ws, tmp, s))) return st;
  }
  float* g = at<float>(ws, Lo.g);
  // 1. per-token gradient rows g[t] (the sign of the sender's term is applied
  //    in the reduction): sender  dZ (B_s U)^T (ambient) or dZ B_s^T (coord),
  //    receiver dXhat B_r^T (ambient) or dZhat B_r^T (coord)
  if (D.x_dtype == MAPL_BF16) {
    bf16_t* W = at<bf16_t>(ws, Lo.w);
    if (need_u) {
      if (Lo.kp > k) LAUNCH("anchor_bwd:zero_w", launch_zero_bytes(W + k * r, (int64_t)(Lo.kp - k) * r * 2, s));
      PrepJob j = prep_job_small_gemm((const bf16_t*)B, d, U, r, 0, (int)k, (int)r, (int)d, 1.f, W, r, 0);
      j.dst_rows = 1;
      LAUNCH("anchor_bwd:prep", launch_prep_batch(&j, 1, s));
    } else {
      LAUNCH("anchor_bwd:prep", launch_pad_rows_bf16((const bf16_t*)B, (int)k, Lo.K, Lo.kp, W, s));
    }
    TnArgs gg{};
    gg.A = (const bf16_t*)dY; gg.lda = Lo.K; gg.Ka = Lo.K;
    gg.W = W; gg.ldw = Lo.K;
    gg.M = (int)T; gg.N = Lo.kp;
    gg.out = g; gg.ldo = Lo.kp; gg.out_f32 = 1;
    LAUNCH("anchor_bwd:gemm_tn", launch_gemm_tn(gg, s));
  } else {
    const float* Bk = (const float*)B;  // [k, K]
    if (need_u) {
      float* BU = at<float>(ws, Lo.bu);
      GemmF32Args e = gemm((int)k, (int)r, (int)d);
      e.A = B; e.sAm = d; e.sAk = 1;
      e.B = U; e.sBk = r; e.sBn = 1;
      e.C = BU; e.sCm = r; e.sCn = 1;
      LAUNCH("anchor_bwd:gemm_f32", launch_gemm_f32(e, 0, 0, 0, s));
      Bk = BU;
    }
    GemmF32Args e = gemm((int)T, (int)k, Lo.K);
    e.A = dY; e.sAm = Lo.K; e.sAk = 1;
    e.B = Bk; e.sBk = 1; e.sBn = Lo.K;
    e.C = g; e.sCm = Lo.kp; e.sCn = 1;
    LAUNCH("anchor_bwd:gemm_f32", launch_gemm_f32(e, 0, 0, 0, s));
  }
  // 2. tokens sorted by id (stable), 3. per-id sums in sorted order
  const int32_t *skey = nullptr, *sval = nullptr;
  LAUNCH("anchor_bwd:sort", launch_sort_ids(ids, (int)T, Lo.passes, at<int>(ws, Lo.hist), at<int32_t>(ws, Lo.k0),
                                            at<int32_t>(ws, Lo.v0), at<int32_t>(ws, Lo.k1), at<int32_t>(ws, Lo.v1),
                                            &skey, &sval, s));
  AnchorSegArgs a{};
  a.g = g; a.ldg = Lo.kp; a.k = (int)k;
  a.skey = skey; a.sval = sval; a.n = (int)T;
  a.dA = dA; a.V = (int)D.V; a.accumulate = accumulate ? 1 : 0; a.scale = side == MAPL_SENDER ? -1.f : 1.f;
  a.headp = at<float>(ws, Lo.headp); a.tailp = at<float>(ws, Lo.tailp);
  a.head_id = at<int32_t>(ws, Lo.hid); a.head_thru = at<int32_t>(ws, Lo.hthru); a.tail_id = at<int32_t>(ws, Lo.tid);
  a.nsub = Lo.nsub;
  LAUNCH("anchor_bwd:segsum", launch_anchor_segsum(a, s));
  return MAPL_OK;
}

// ------------------------------------------------------ codebook synchronisation
namespace {
int check_sync(int32_t L, int32_t K, int64_t r, int32_t n) {
  if (L < 1 || L > 8) return fail(MAPL_E_SHAPE, "codebook sync: need 1 <= L <= 8 (got %d)", L);
  if (K < 1 || K > 65536) return fail(MAPL_E_SHAPE, "codebook sync: need 1 <= K <= 65536 (got %d)", K);
  if (r < 4 || r > 1024 || r % 4) return fail(MAPL_E_SHAPE, "codebook sync: need 4 <= r <= 1024, r %% 4 == 0");
  if (n < 0 || n > K) return fail(MAPL_E_SHAPE, "codebook sync: need 0 <= n <= K (got n=%d)", n);
  return MAPL_OK;
}
}  // namespace

extern "C" int mapl_codebook_pack(int32_t L, int32_t K, int64_t r, const float* C, const int32_t* rows, int32_t n,
                                  float* buf, void* stream) {
  g_err.clear();
  int st = check_sync(L, K, r, n);
  if (st) return st;
  const size_t cb = (size_t)L * K * r * 4, bb = (size_t)L * n * r * 4, rb = (size_t)L * n * 4;
  st = check_ptrs({{C, cb, "C"}, {rows, rb, "rows"}, {buf, bb, "buf"}}, {{buf, bb, "buf"}},
                  {{C, cb, "C"}, {rows, rb, "rows"}});
  if (st) return st;
  hipStream_t s = (hipStream_t)stream;
  LAUNCH("sync:pack", launch_codebook_pack(C, rows, L, K, (int)r, n, buf, s));
  return MAPL_OK;
}

extern "C" int mapl_codebook_unpack(int32_t L, int32_t K, int64_t r, const float* buf, const int32_t* rows,
                                    int32_t n, float* C, void* stream) {
  g_err.clear();
  int st = check_sync(L, K, r, n);
  if (st) return st;
  const size_t cb = (size_t)L * K * r * 4, bb = (size_t)L * n * r * 4, rb = (size_t)L * n * 4;
  st = check_ptrs({{C, cb, "C"}, {rows, rb, "rows"}, {buf, bb, "buf"}}, {{C, cb, "C"}},
                  {{buf, bb, "buf"}, {rows, rb, "rows"}});
  if (st) return st;
  hipStream_t s = (hipStream_t)stream;
  LAUNCH("sync:unpack", launch_codebook_unpack(buf, rows, L, K, (int)r, n, C, s));
  return MAPL_OK;
}

// ------------------------------------------------------ allocation-free encode
// Scratch of mapl_encode_noalloc: a file-scope device array, one copy per GPU
// the library runs on, held until the process ends.  In host code the name
// `scratch` is only a stand-in for the symbol; its device address on each GPU
// comes from hipGetSymbolAddress, called once per device with that device
// current, and only that address is ever handed to kernels.
static __device__ __align__(256) unsigned char scratch[MAPL_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_for_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(MAPL_E_UNSUPPORTED, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(MAPL_E_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MAPL_OK;
}
}  // namespace

extern "C" int mapl_encode_noalloc(const mapl_codec_desc* desc, const void* X, const int32_t* ids, const float* U,
                                   const void* A_s, const void* B_s, const float* C, void* payload, void* stream) {
  g_err.clear();
  int st = check_desc(desc);
  if (st) return st;
  const size_t need = layout(*desc, MAPL_CALL_ENCODE).total;
  if (need > (size_t)MAPL_NOALLOC_SCRATCH_BYTES)
    return fail(MAPL_E_WORKSPACE,
                "mapl_encode_noalloc: this request needs %zu bytes of scratch, the static scratch holds %zu "
                "(use mapl_encode with a workspace)",
                need, (size_t)MAPL_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = scratch_for_current_device(&ws))) return st;
  return mapl_encode(desc, X, ids, U, A_s, B_s, C, payload, ws, (size_t)MAPL_NOALLOC_SCRATCH_BYTES, stream);
}

// ---------------------------------------------------------------- tracing API
extern "C" int mapl_profile(int enable) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof = enable != 0;
  g_prof_rvq = enable >= 2;
  return MAPL_OK;
}

extern "C" int mapl_profile_report(char* buf, size_t bytes) {
  std::vector<ProfRec> recs;
  long long rvq[kRvqStats];
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    recs.swap(g_prof_recs);
    for (int i = 0; i < kRvqStats; ++i) {
      rvq[i] = g_rvq_stats[i];
      g_rvq_stats[i] = 0;
    }
  }
  // one line per kernel name, in the order of first launch
  std::vector<std::string> order;
  std::map<std::string, std::pair<long, double>> agg;
  int st = MAPL_OK;
  for (const ProfRec& r : recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) {
      st = fail(MAPL_E_HIP, "profile: event query failed");
      continue;
    }
    auto it = agg.find(r.name);
    if (it == agg.end()) {
      order.push_back(r.name);
      it = agg.emplace(r.name, std::make_pair(0L, 0.0)).first;
    }
    it->second.first += 1;
    it->second.second += ms;
  }
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    for (const ProfRec& r : recs) {
      g_prof_pool.push_back(r.a);
      g_prof_pool.push_back(r.b);
    }
  }
  std::string outs;
  char line[256];
  for (const std::string& name : order) {
    const auto& v = agg[name];
    snprintf(line, sizeof line, "%s %ld %.6f\n", name.c_str(), v.first, v.second);
    outs += line;
  }
  if (rvq[4] > 0)
    for (int i = 0; i < kRvqStats; ++i) {
      snprintf(line, sizeof line, "%s %lld 0\n", kRvqStatNames[i], rvq[i]);
      outs += line;
    }
  if (buf && bytes) {
    const size_t n = outs.size() < bytes - 1 ? outs.size() : bytes - 1;
    memcpy(buf, outs.data(), n);
    buf[n] = 0;
    if (outs.size() >= bytes) return fail(MAPL_E_WORKSPACE, "profile report needs %zu bytes", outs.size() + 1);
  }
  return st;
}
