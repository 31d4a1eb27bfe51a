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
//   3. a fix-up, one workgroup per segment that crosses sub-chunks, adding
//      its pieces in a fixed order (four interleaved wave sums, then the
//      waves in order).
// Zipf-distributed ids make a few rows very long (id 0 takes about a seventh
// of the tokens); the sub-chunk split keeps every wave's share at 64 rows.
#include "common.hpp"
#include "kernels.hpp"

namespace mapl {

namespace {

constexpr int RS_THREADS = 256, RS_TILE = 512, RS_ROUNDS = RS_TILE / RS_THREADS;
constexpr int SEG = 64;  // sorted positions per sub-chunk

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
// then digit 1, ...), by one block: chunks of 8192 counts move through LDS
// with coalesced loads and stores, each thread scans 8 consecutive counts,
// the 1024 thread sums are scanned in LDS, and a carry links the chunks.
__global__ __launch_bounds__(1024) void k_radix_scan(int* __restrict__ hist, int m) {
  constexpr int PER = 8, CH = 1024 * PER;
  __shared__ int buf[CH];
  __shared__ int part[1024];
  const int tid = threadIdx.x;
  int carry = 0;
  for (int base = 0; base < m; base += CH) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = base + j * 1024 + tid;
      buf[j * 1024 + tid] = i < m ? hist[i] : 0;
    }
    __syncthreads();
    int sum = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) sum += buf[tid * PER + j];
    part[tid] = sum;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
      const int v = tid >= o ? part[tid - o] : 0;
      __syncthreads();
      part[tid] += v;
      __syncthreads();
    }
    int run = carry + (tid ? part[tid - 1] : 0);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = buf[tid * PER + j];
      buf[tid * PER + j] = run;
      run += c;
    }
    const int total = part[1023];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = base + j * 1024 + tid;
      if (i < m) hist[i] = buf[j * 1024 + tid];
    }
    carry += total;
    __syncthreads();  // buf and part are reused by the next chunk
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

// row[c] (+)= scale acc[q] for the lane's columns c = lane + 64 q < k
template <int NC>
__device__ __forceinline__ void seg_store(float* __restrict__ row, const float (&acc)[NC], int k, int lane,
                                          float scale, int add) {
#pragma unroll
  for (int q = 0; q < NC; ++q) {
    const int c = lane + 64 * q;
    if (c < k) row[c] = add ? row[c] + scale * acc[q] : scale * acc[q];
  }
}

// One wave per sub-chunk of 64 sorted positions: the rows of each segment
// (run of equal ids) are summed in sorted order; a segment wholly inside the
// sub-chunk is written to dA, a piece that continues from the previous
// sub-chunk goes to the head slot (flagged when it also continues into the
// next), a piece that starts here and continues goes to the tail slot.
// NC columns per lane (k <= 64 NC); 64 / NC rows are requested at a time.
template <int NC>
__global__ __launch_bounds__(256) void k_seg_partial(AnchorSegArgs a) {
  constexpr int BR = 64 / NC;
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
  float acc[NC];
#pragma unroll
  for (int q = 0; q < NC; ++q) acc[q] = 0.f;
  int pstart = p0;
  for (int pb = p0; pb < p1; pb += BR) {
    // the batch's ids, tokens and rows are requested before any is summed
    int id[BR], t[BR];
    float v[BR][NC];
#pragma unroll
    for (int u = 0; u < BR; ++u) {
      const int p = min(pb + u, p1 - 1);
      id[u] = a.skey[p];
      t[u] = a.sval[p];
    }
#pragma unroll
    for (int u = 0; u < BR; ++u) {
      const float* gr = a.g + (int64_t)t[u] * a.ldg;
#pragma unroll
      for (int q = 0; q < NC; ++q) {
        const int c = lane + 64 * q;
        v[u][q] = c < a.k ? gr[c] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < BR; ++u) {
      const int p = pb + u;
      if (p >= p1) break;
#pragma unroll
      for (int q = 0; q < NC; ++q) acc[q] += v[u][q];
      const int nid = p + 1 < p1 ? (u + 1 < BR ? id[u + 1] : a.skey[p + 1]) : next_id;
      if (nid == id[u] && p + 1 < p1) continue;  // the segment goes on inside the sub-chunk
      const bool before = pstart == p0 && prev_id == id[u];
      const bool after = p + 1 == p1 && next_id == id[u];
      if (!before && !after) {
        if ((unsigned)id[u] < (unsigned)a.V)  // an id outside [0, V) is a caller error: skipped
          seg_store<NC>(a.dA + (int64_t)id[u] * a.k, acc, a.k, lane, a.scale, a.accumulate);
      } else if (before) {
        seg_store<NC>(a.headp + (int64_t)s * a.k, acc, a.k, lane, 1.f, 0);
        if (lane == 0) {
          a.head_id[s] = id[u];
          a.head_thru[s] = after ? 1 : 0;
        }
      } else {
        seg_store<NC>(a.tailp + (int64_t)s * a.k, acc, a.k, lane, 1.f, 0);
        if (lane == 0) a.tail_id[s] = id[u];
      }
#pragma unroll
      for (int q = 0; q < NC; ++q) acc[q] = 0.f;
      pstart = p + 1;
    }
  }
}

// Segments that cross sub-chunk boundaries, one workgroup per sub-chunk s
// whose tail piece starts one: its head pieces are those of sub-chunks
// s+1 .. e, e the first that does not continue further.  Wave w sums the
// pieces s+1+w, s+5+w, ... in order (eight requested at a time); the sum is
// tail + wave 0 + wave 1 + wave 2 + wave 3, a fixed order.
template <int NC>
__global__ __launch_bounds__(256) void k_seg_fixup(AnchorSegArgs a) {
  constexpr int FB = 8;
  __shared__ float part[4][64 * NC];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int s = blockIdx.x;
  const int id = a.tail_id[s];
  if (id < 0 || id >= a.V) return;  // workgroup-uniform
  // e: the first head piece after s that ends the segment (exists: a tail
  // piece continues into sub-chunk s + 1, and the last sub-chunk's head
  // piece never continues)
  int e = a.nsub - 1;
  for (int b = s + 1; b < a.nsub; b += 64) {
    const int i = b + lane;
    const uint64_t m = __ballot(i < a.nsub && a.head_thru[i] == 0);
    if (m) {
      e = b + __builtin_ctzll(m);
      break;
    }
  }
  float acc[NC];
#pragma unroll
  for (int q = 0; q < NC; ++q) acc[q] = 0.f;
  for (int b = s + 1 + wave; b <= e; b += 4 * FB) {
    float v[FB][NC];
#pragma unroll
    for (int u = 0; u < FB; ++u) {
      const int s2 = min(b + 4 * u, e);
#pragma unroll
      for (int q = 0; q < NC; ++q) {
        const int c = lane + 64 * q;
        v[u][q] = c < a.k ? a.headp[(int64_t)s2 * a.k + c] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < FB; ++u)
      if (b + 4 * u <= e) {
#pragma unroll
        for (int q = 0; q < NC; ++q) acc[q] += v[u][q];
      }
  }
#pragma unroll
  for (int q = 0; q < NC; ++q) part[wave][lane + 64 * q] = acc[q];
  __syncthreads();
  if (wave != 0) return;
  float tot[NC];
#pragma unroll
  for (int q = 0; q < NC; ++q) {
    const int c = lane + 64 * q;
    float x = c < a.k ? a.tailp[(int64_t)s * a.k + c] : 0.f;
    x += part[0][c];
    x += part[1][c];
    x += part[2][c];
    x += part[3][c];
    tot[q] = x;
  }
  seg_store<NC>(a.dA + (int64_t)id * a.k, tot, a.k, lane, a.scale, a.accumulate);
}

template <int NC>
void launch_segsum_nc(const AnchorSegArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_seg_partial<NC>, dim3((a.nsub + 3) / 4), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_seg_fixup<NC>, dim3(a.nsub), dim3(256), 0, s, a);
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
  if (a.k <= 64)
    launch_segsum_nc<1>(a, s);
  else if (a.k <= 128)
    launch_segsum_nc<2>(a, s);
  else if (a.k <= 256)
    launch_segsum_nc<4>(a, s);
  else if (a.k <= 512)
    launch_segsum_nc<8>(a, s);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

int anchor_sub_chunks(int n) { return (n + SEG - 1) / SEG; }

}  // namespace mapl
