// Gradient of the anchor table (Sec. 3.2: E_small is trainable, Eq. 3).
// Every token contributes a gradient row g[t] (from the GEMM kernels) to the
// table row of its id; the rows are summed per id in a fixed order, so the
// result is reproducible bit for bit (no floating-point atomics):
//   1. a stable LSD radix sort of (id, token) pairs, 8-bit digits: per-tile
//      digit histograms, one exclusive scan, a stable scatter whose ranks
//      come from wave ballots;
//   2. a segmented sum over the sorted order in 64-position sub-chunks, one
//      wave each, walking its positions in order; a segment that crosses a
//      sub-chunk boundary leaves its pieces in per-sub-chunk slots;
//   3. a fix-up that adds those pieces in sub-chunk order.
// Zipf-distributed ids make a few rows very long (id 0 takes about a seventh
// of the tokens); the sub-chunk split keeps every wave's share at 64 rows.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int RS_THREADS = 256, RS_TILE = 2048, RS_ROUNDS = RS_TILE / RS_THREADS;
constexpr int SEG = 64, SEG_COLS = 8, SEG_BATCH = 8;  // positions per sub-chunk; k <= 512; rows in flight

// W[i][c] = B[i][c] for i < k, c < K, zero for the padding rows k <= i < kp.
__global__ void k_pad_rows_bf16(const bf16_t* __restrict__ B, int k, int K, int kp, bf16_t* __restrict__ W) {
  const int64_t n = (int64_t)kp * K;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / K);
    W[e] = i < k ? B[e] : (bf16_t)0;
  }
}

__global__ __launch_bounds__(RS_THREADS) void k_radix_hist(const int32_t* __restrict__ keys, int n, int shift,
                                                           int nb, int* __restrict__ hist) {
  __shared__ int h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int base = blockIdx.x * RS_TILE;
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const int i = base + j * RS_THREADS + threadIdx.x;
    if (i < n) atomicAdd(&h[((uint32_t)keys[i] >> shift) & 255u], 1);
  }
  __syncthreads();
  hist[threadIdx.x * nb + blockIdx.x] = h[threadIdx.x];
}

// Exclusive scan, in place, of m counts (digit-major: all tiles of digit 0,
// then digit 1, ...), by one block.
__global__ __launch_bounds__(1024) void k_radix_scan(int* __restrict__ hist, int m) {
  __shared__ int part[1024];
  const int tid = threadIdx.x;
  const int per = (m + 1023) / 1024;
  const int b0 = min(m, tid * per), b1 = min(m, b0 + per);
  int sum = 0;
  for (int i = b0; i < b1; ++i) sum += hist[i];
  part[tid] = sum;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int v = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int run = tid ? part[tid - 1] : 0;
  for (int i = b0; i < b1; ++i) {
    const int c = hist[i];
    hist[i] = run;
    run += c;
  }
}

// Stable scatter of one tile: keys are taken in rounds of 256 in input
// order; within a round, lanes of a wave with the same digit are ranked by
// ballots, waves in order, and rounds in order, so equal digits keep their
// input order.  vals == null stands for vals[i] = i.
__global__ __launch_bounds__(RS_THREADS) void k_radix_scatter(const int32_t* __restrict__ keys,
                                                              const int32_t* __restrict__ vals, int n, int shift,
                                                              int nb, const int* __restrict__ offs,
                                                              int32_t* __restrict__ keys_out,
                                                              int32_t* __restrict__ vals_out) {
  __shared__ int base[256];
  __shared__ int wcnt[4][256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  base[tid] = offs[tid * nb + blockIdx.x];
#pragma unroll
  for (int w = 0; w < 4; ++w) wcnt[w][tid] = 0;
  __syncthreads();
  const int b0 = blockIdx.x * RS_TILE;
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const int i = b0 + j * RS_THREADS + tid;
    const bool ok = i < n;
    const int key = ok ? keys[i] : 0;
    const int val = ok ? (vals ? vals[i] : i) : 0;
    const int dg = (int)(((uint32_t)key >> shift) & 255u);
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (dg >> b) & 1;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    const uint64_t lower = peers & ((1ull << lane) - 1ull);
    if (ok && lower == 0) wcnt[wave][dg] = __popcll(peers);
    __syncthreads();
    if (ok) {
      int pos = base[dg] + __popcll(lower);
      for (int w = 0; w < wave; ++w) pos += wcnt[w][dg];
      keys_out[pos] = key;
      vals_out[pos] = val;
    }
    __syncthreads();
    base[tid] += (wcnt[0][tid] + wcnt[1][tid]) + (wcnt[2][tid] + wcnt[3][tid]);
#pragma unroll
    for (int w = 0; w < 4; ++w) wcnt[w][tid] = 0;
    __syncthreads();
  }
}

__device__ __forceinline__ void seg_store(float* __restrict__ row, const float (&acc)[SEG_COLS], int k, int lane,
                                          float scale, int add) {
#pragma unroll
  for (int q = 0; q < SEG_COLS; ++q) {
    const int c = lane + 64 * q;
    if (c < k) row[c] = add ? row[c] + scale * acc[q] : scale * acc[q];
  }
}

// One wave per sub-chunk of 64 sorted positions: the rows of each segment
// (run of equal ids) are summed in sorted order; a segment wholly inside the
// sub-chunk is written to dA, a piece that continues from the previous
// sub-chunk goes to the head slot (flagged when it also continues into the
// next), a piece that starts here and continues goes to the tail slot.
__global__ __launch_bounds__(256) void k_seg_partial(AnchorSegArgs a) {
  const int lane = threadIdx.x & 63;
  const int s = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (s >= a.nsub) return;  // wave-uniform
  const int p0 = s * SEG, p1 = min(a.n, p0 + SEG);
  // -1 marks "no neighbour"; ids are non-negative (negative ones are never written)
  const int prev_id = p0 > 0 ? a.skey[p0 - 1] : -1;
  const int next_id = p1 < a.n ? a.skey[p1] : -1;
  if (lane == 0) {
    a.head_id[s] = -1;
    a.head_thru[s] = 0;
    a.tail_id[s] = -1;
  }
  float acc[SEG_COLS];
#pragma unroll
  for (int q = 0; q < SEG_COLS; ++q) acc[q] = 0.f;
  int pstart = p0;
  for (int pb = p0; pb < p1; pb += SEG_BATCH) {
    // the batch's ids, tokens and rows are requested before any is summed
    int id[SEG_BATCH], t[SEG_BATCH];
    float v[SEG_BATCH][SEG_COLS];
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      const int p = min(pb + u, p1 - 1);
      id[u] = a.skey[p];
      t[u] = a.sval[p];
    }
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      const float* gr = a.g + (int64_t)t[u] * a.ldg;
#pragma unroll
      for (int q = 0; q < SEG_COLS; ++q) {
        const int c = lane + 64 * q;
        v[u][q] = c < a.k ? gr[c] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      const int p = pb + u;
      if (p >= p1) break;
#pragma unroll
      for (int q = 0; q < SEG_COLS; ++q) acc[q] += v[u][q];
      const int nid = p + 1 < p1 ? (u + 1 < SEG_BATCH ? id[u + 1] : a.skey[p + 1]) : next_id;
      if (nid == id[u] && p + 1 < p1) continue;  // the segment goes on inside the sub-chunk
      const bool before = pstart == p0 && prev_id == id[u];
      const bool after = p + 1 == p1 && next_id == id[u];
      if (!before && !after) {
        if ((unsigned)id[u] < (unsigned)a.V)  // an id outside [0, V) is a caller error: skipped
          seg_store(a.dA + (int64_t)id[u] * a.k, acc, a.k, lane, a.scale, a.accumulate);
      } else if (before) {
        seg_store(a.headp + (int64_t)s * a.k, acc, a.k, lane, 1.f, 0);
        if (lane == 0) {
          a.head_id[s] = id[u];
          a.head_thru[s] = after ? 1 : 0;
        }
      } else {
        seg_store(a.tailp + (int64_t)s * a.k, acc, a.k, lane, 1.f, 0);
        if (lane == 0) a.tail_id[s] = id[u];
      }
#pragma unroll
      for (int q = 0; q < SEG_COLS; ++q) acc[q] = 0.f;
      pstart = p + 1;
    }
  }
}

// Segments that cross sub-chunk boundaries: the sub-chunk where one starts
// adds the head pieces of the following sub-chunks in order.
__global__ __launch_bounds__(256) void k_seg_fixup(AnchorSegArgs a) {
  const int lane = threadIdx.x & 63;
  const int s = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (s >= a.nsub) return;
  const int id = a.tail_id[s];
  if (id < 0 || id >= a.V) return;
  float acc[SEG_COLS];
#pragma unroll
  for (int q = 0; q < SEG_COLS; ++q) {
    const int c = lane + 64 * q;
    acc[q] = c < a.k ? a.tailp[(int64_t)s * a.k + c] : 0.f;
  }
  for (int s2 = s + 1; s2 < a.nsub; ++s2) {
#pragma unroll
    for (int q = 0; q < SEG_COLS; ++q) {
      const int c = lane + 64 * q;
      if (c < a.k) acc[q] += a.headp[(int64_t)s2 * a.k + c];
    }
    if (!a.head_thru[s2]) break;
  }
  seg_store(a.dA + (int64_t)id * a.k, acc, a.k, lane, a.scale, a.accumulate);
}

}  // namespace

hipError_t launch_pad_rows_bf16(const bf16_t* B, int k, int K, int kp, bf16_t* W, hipStream_t s) {
  const int64_t n = (int64_t)kp * K;
  if (n <= 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(k_pad_rows_bf16, dim3(blocks), dim3(256), 0, s, B, k, K, kp, W);
  return hipGetLastError();
}

int radix_tiles(int n) { return (n + RS_TILE - 1) / RS_TILE; }

hipError_t launch_sort_ids(const int32_t* ids, int n, int passes, int* hist, int32_t* k0, int32_t* v0, int32_t* k1,
                           int32_t* v1, const int32_t** skey, const int32_t** sval, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int nb = radix_tiles(n);
  const int32_t* kin = ids;
  const int32_t* vin = nullptr;
  int32_t* kb[2] = {k0, k1};
  int32_t* vb[2] = {v0, v1};
  for (int p = 0; p < passes; ++p) {
    hipLaunchKernelGGL(k_radix_hist, dim3(nb), dim3(RS_THREADS), 0, s, kin, n, 8 * p, nb, hist);
    hipLaunchKernelGGL(k_radix_scan, dim3(1), dim3(1024), 0, s, hist, 256 * nb);
    hipLaunchKernelGGL(k_radix_scatter, dim3(nb), dim3(RS_THREADS), 0, s, kin, vin, n, 8 * p, nb, hist, kb[p & 1],
                       vb[p & 1]);
    kin = kb[p & 1];
    vin = vb[p & 1];
  }
  *skey = kin;
  *sval = vin;
  return hipGetLastError();
}

hipError_t launch_anchor_segsum(const AnchorSegArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.k > 64 * SEG_COLS) return hipErrorInvalidValue;
  const int blocks = (a.nsub + 3) / 4;
  hipLaunchKernelGGL(k_seg_partial, dim3(blocks), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_seg_fixup, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

int anchor_sub_chunks(int n) { return (n + SEG - 1) / SEG; }

}  // namespace mapl
