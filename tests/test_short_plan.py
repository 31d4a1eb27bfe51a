"""The short-K GEMM's stage waits (k_gemm_tn_short): each is a fixed vmcnt
count, valid only if it equals the number of memory operations the wave
issues after the awaited stage's last DMA block.  The counts come from
csrc/short_plan.hpp (compiled here with the host compiler); they are checked
against a brute-force replay of the kernel's issue order for every K depth
the kernel takes (2 to 6 stages) and several tile counts, together with the
6-bit vmcnt limit and the 16 row-segment stores per tile."""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2606_05484_amd", "csrc")

PROG = r"""
#include <cstdio>
#include "short_plan.hpp"
template <int KS> void dump() {
  using P = mapl::ShortPlan<KS>;
  std::printf("KS %d KST %d D %d WBLK %d NCH %d\n", KS, P::KST, P::D, P::WBLK, P::NCH);
  std::printf("st");
  for (int q = 0; q < P::KST; ++q) std::printf(" %d", P::st(q));
  std::printf("\nst0");
  for (int q = 0; q < P::KST; ++q) std::printf(" %d", P::st0(q));
  std::printf("\nfirst");
  for (int k = 0; k < KS; ++k) std::printf(" %d", P::wait_n(k, true));
  std::printf("\nlater");
  for (int k = 0; k < KS; ++k) std::printf(" %d", P::wait_n(k, false));
  std::printf("\n");
}
int main() { dump<2>(); dump<3>(); dump<4>(); dump<5>(); dump<6>(); return 0; }
"""


def _plan():
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "p.cpp"), os.path.join(d, "p")
        open(src, "w").write(PROG)
        subprocess.run([cxx, "-std=c++17", "-O1", "-I", CSRC, src, "-o", exe], check=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.splitlines()
    plans = {}
    for i in range(0, len(out), 5):
        head = out[i].split()
        KS = int(head[1])
        vals = dict(zip(head[2::2], map(int, head[3::2])))
        vals["st"] = list(map(int, out[i + 1].split()[1:]))
        vals["st0"] = list(map(int, out[i + 2].split()[1:]))
        vals["first"] = list(map(int, out[i + 3].split()[1:]))
        vals["later"] = list(map(int, out[i + 4].split()[1:]))
        plans[KS] = vals
    return plans


def _replay(KS, p, ntiles):
    """The wave's memory operations in issue order; at each stage wait, the
    number issued after the awaited stage's last DMA block."""
    D, WB = p["D"], p["WBLK"]
    ops = []
    for s in range(D):  # prologue: W DMA of stages 0 .. D-1
        ops += [("dma", s)] * WB
    waits = []
    dstage, s = D, 0
    for t in range(ntiles):
        for ksi in range(KS):
            for kk in range(4):
                q = ksi * 4 + kk
                ops.append(("dma", dstage))  # one block of the stage D ahead
                if kk == 2:  # the wait for stage s + 1, then this k-step's stores
                    last = max(i for i, o in enumerate(ops) if o == ("dma", s + 1))
                    waits.append((t, ksi, len(ops) - 1 - last))
                ops += [("st", t)] * p["st"][q]
            dstage += 1
            s += 1
    return waits


def test_short_gemm_stage_waits_match_issue_order():
    plans = _plan()
    assert sorted(plans) == [2, 3, 4, 5, 6]
    for KS, p in plans.items():
        assert p["KST"] == 4 * KS and p["WBLK"] == 4 and 1 <= p["D"] <= min(KS, 4)
        # the 16 row-segment stores of a tile, in chunk order, at most two per k-step
        assert sum(p["st"]) == p["NCH"] == 16
        assert all(0 <= n <= 2 for n in p["st"])
        assert p["st0"] == [sum(p["st"][:q]) for q in range(p["KST"])]
        for ntiles in (1, 2, 3, 8):
            for t, ksi, n in _replay(KS, p, ntiles):
                want = p["first"][ksi] if t == 0 else p["later"][ksi]
                assert n == want, (KS, ntiles, t, ksi, n, want)
                assert n <= 63  # vmcnt is 6 bits wide


def test_replay_catches_a_miscount():
    """The replay is not vacuous: one store more in a k-step of the window
    before a wait changes the count it measures."""
    p = _plan()[6]
    base = _replay(6, p, 2)
    q2 = dict(p, st=list(p["st"]))
    q2["st"][15] += 1
    moved = _replay(6, q2, 2)
    assert base != moved
