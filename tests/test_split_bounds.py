"""The split products of the SPEL step, checked on the CPU.

Every PolarExpress product of the Stiefel step (Eqs. 6 and 7) takes fp16
pieces of its fp32 operands (y = 2^8 x, hi = fp16(y), lo = fp16(y - hi),
both round to nearest even, subnormals kept; hi.hi + hi.lo + lo.hi with fp32
accumulation).  Two facts carry that choice and are checked here:

  - the split keeps each operand to 2^-22 of its magnitude where
    |x| >= 2^-11, to an absolute 2^-33 below that, and has finite pieces for
    every |x| < 255;
  - the operands stay far inside that range: from X0 with spectral norm
    <= 1 (M / (||M||_F + eps) for the LMO, Y / nu for the retraction), both
    schedules keep the singular values below 2.1, so the iterates X, their
    Gram matrices S and S Q~ (Q~ = (a I + b S + c S^2) / a) have spectral
    norms, and so entries, below 5; every quintic has |p(x)| <= a x on the
    values it meets, so Q~ and any product of consecutive Q~'s (the r x r
    iteration's P~) have eigenvalues in [-1, 1].  The library's segments
    (consecutive a's multiplying to at most 2048) keep P~'s eigenvalue for
    a unit singular value at or above 2^-11.

The coefficients are the library's own tables (csrc/polar_coeffs.h,
compiled here with the host compiler)."""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2606_05484_amd", "csrc")


def _samples(rng, lo_exp, hi, n=200000):
    mag = np.exp2(rng.uniform(lo_exp, np.log2(hi), n))
    return (mag * rng.choice([-1.0, 1.0], n)).astype(np.float32)


def test_fp16_split_keeps_22_bits_and_stays_finite():
    rng = np.random.default_rng(1)
    x = np.concatenate([_samples(rng, -60, 254.99), np.float32([254.99, -254.99, 2.0 ** -11, 0.0])])
    y = x * np.float32(256.0)  # exact: a power of two
    with np.errstate(over="raise"):
        hi = y.astype(np.float16)
        lo = (y - hi.astype(np.float32)).astype(np.float16)
    assert np.isfinite(hi).all() and np.isfinite(lo).all()
    # y - hi is exact in fp32 (hi is y rounded to 11 bits)
    d = y.astype(np.float64) - hi.astype(np.float64)
    assert np.array_equal(d, (y - hi.astype(np.float32)).astype(np.float64))
    err = np.abs(d - lo.astype(np.float64)) / 256.0  # in units of x
    ax = np.abs(x.astype(np.float64))
    big = ax >= 2.0 ** -11
    assert np.all(err[big] <= 2.0 ** -22 * ax[big])
    assert np.all(err[~big] <= 2.0 ** -33)
    # typically the pieces hold the operand as well as fp32 itself
    assert np.median(err[big] / ax[big]) < 2.0 ** -24


def test_fp16_split_overflows_past_its_bound():
    """The bound is real: at 256 the high piece is no longer finite."""
    with np.errstate(over="ignore"):
        assert not np.isfinite((np.float32(256.0) * np.float32(256.0)).astype(np.float16))


PROG = r"""
#include <cstdio>
#include "polar_coeffs.h"
int main() {
  for (int i = 0; i < mapl::kPolarMaxSteps; ++i)
    std::printf("%.17g %.17g %.17g\n", mapl::kLmoCoef[i][0], mapl::kLmoCoef[i][1], mapl::kLmoCoef[i][2]);
  for (int i = 0; i < mapl::kPolarMaxSteps; ++i)
    std::printf("%.17g %.17g %.17g\n", mapl::kRetractCoef[i][0], mapl::kRetractCoef[i][1], mapl::kRetractCoef[i][2]);
  return 0;
}
"""


def _tables():
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    with tempfile.TemporaryDirectory() as tmp:
        src, exe = os.path.join(tmp, "c.cpp"), os.path.join(tmp, "c")
        open(src, "w").write(PROG)
        subprocess.run([cxx, "-std=c++17", "-I", CSRC, src, "-o", exe], check=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    rows = np.array([[float(v) for v in line.split()] for line in out.splitlines()])
    n = len(rows) // 2
    return {"lmo": rows[:n], "retraction": rows[n:]}


@pytest.mark.parametrize("schedule", ["lmo", "retraction"])
def test_polar_iterates_stay_bounded(schedule):
    coefs = _tables()[schedule]
    hi = 1.0  # spectral norm of X0
    worst, max_hi = 0.0, hi
    for a, b, c in coefs:
        x = np.linspace(0.0, hi, 200001)
        lam = x ** 2
        q = a + b * lam + c * lam ** 2  # eigenvalues of Q on S's spectrum [0, hi^2]
        assert np.abs(q).max() <= a * (1 + 1e-12)  # |p(x)| = x |q(x^2)| <= a x: Q~ = Q / a in [-1, 1]
        worst = max(worst, hi, hi ** 2, np.abs(lam * q / a).max())
        hi = np.abs(x * q).max()  # the next iterate's spectral norm bound
        max_hi = max(max_hi, hi)
    assert max_hi < 2.1 and worst < 5.0
    # the library's segments: consecutive a's multiply to at most 2048
    i = 0
    while i < len(coefs):
        j, g = i, 1.0
        while j < len(coefs) and (j == i or g * coefs[j][0] <= 2048.0):
            g *= coefs[j][0]
            j += 1
        assert g <= 2048.0
        i = j
