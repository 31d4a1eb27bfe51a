// The memory-operation schedule of the short-K bf16 GEMM (k_gemm_tn_short):
// how its output stores are spread over a tile's k-steps and the vmcnt count
// of every stage wait.  Plain C++ (no device code), so the host-side tests can
// check the counts against a brute-force replay of the issue order.
//
// Issue order per wave: the prologue issues the W DMA of stages 0 .. D-1
// (WBLK blocks each); then every k-step q of a tile issues one W DMA block
// (stage s + D) and, after the stage wait that sits after k-step 2 of each
// stage, st(q) output row-segment stores (the previous tile's; the first
// tile's go to an out-of-range offset, so every tile issues the same
// operations).  vmcnt counts outstanding operations in issue order, so the
// wait for stage s + 1 in stage s is "at most wait_n(..) outstanding", the
// number issued after that stage's last DMA block.
#pragma once

namespace mapl {

template <int KS>
struct ShortPlan {
  static constexpr int KSTEP = 4;                 // 16-deep k-steps per 64-deep stage
  static constexpr int KST = KS * KSTEP;          // k-steps per tile
  static constexpr int D = KS < 4 ? KS : 4;       // W stages in flight ahead of the one consumed
  static constexpr int NSW = D + 1;               // W ring slots
  static constexpr int WBLK = 4;                  // 1 KiB DMA blocks per wave and stage
  static constexpr int NCH = 16;                  // row-segment stores per wave and tile
  // row-segment stores issued at the end of k-step q of a tile
  static constexpr int st(int q) { return (NCH * (q + 1)) / KST - (NCH * q) / KST; }
  static constexpr int st0(int q) { return (NCH * q) / KST; }  // first chunk stored at k-step q
  // operations issued after the last DMA block of stage s + 1 up to the wait
  // for it in stage s (s = stage ksi of the first tile, or of any later one)
  static constexpr int wait_n(int ksi, bool first) {
    const int s = (first ? 0 : KS) + ksi, y = s + 1;
    int n = 0, g0 = 0;
    if (y < D) {
      n += WBLK * (D - 1 - y);
    } else {
      const int gy = 4 * (y - D) + 3;
      n += st(gy % KST);
      g0 = gy + 1;
    }
    for (int gq = g0; gq < 4 * s + 2; ++gq) n += 1 + st(gq % KST);
    return n + 1;
  }
};

}  // namespace mapl
