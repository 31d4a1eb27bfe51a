"""The split products of the SPEL step, checked on the CPU.

The Stiefel step takes its LMO products from bf16 pieces and its retraction
products from fp16 pieces of the fp32 operands (hi.hi + hi.lo + lo.hi with
fp32 accumulation).  Three facts carry those choices and are checked here:

  - the bf16 split keeps each operand to 2^-16 of its magnitude;
  - the fp16 split (y = 2^8 x, hi = fp16(y), lo = fp16(y - hi), both round
    to nearest even, subnormals kept) keeps each operand to 2^-22 of its
    magnitude where |x| >= 2^-11, to an absolute 2^-33 below that, and has
    finite pieces for every |x| < 255;
  - the retraction's operands stay far inside that range: the first
    PolarExpress quintic of the schedule maps [0, 1] into [0, 1.03], every
    later one maps [0, 1.03] into [0, 1.03], so with X0 = Y / nu (spectral
    norm <= 1) every iterate X, its Gram matrix S = X^T X and the polynomial
    a I + b S + c S^2 have spectral norms, and so entries, below 5.

The coefficients are the library's own table (csrc/polar_coeffs.h, compiled
here with the host compiler)."""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2606_05484_amd", "csrc")


def _bf16(x):
    """fp32 -> bf16 (round to nearest even), returned as fp32."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def _samples(rng, lo_exp, hi, n=200000):
    mag = np.exp2(rng.uniform(lo_exp, np.log2(hi), n))
    return (mag * rng.choice([-1.0, 1.0], n)).astype(np.float32)


def test_bf16_split_keeps_16_bits():
    rng = np.random.default_rng(0)
    x = _samples(rng, -100, 1e30)
    hi = _bf16(x)
    lo = _bf16(x - hi)
    err = np.abs(x.astype(np.float64) - hi.astype(np.float64) - lo.astype(np.float64))
    assert np.all(err <= 2.0 ** -16 * np.abs(x.astype(np.float64)))


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
    # the same operand in the bf16 split carries up to 2^-16: the fp16 split
    # is the one with fp32-class accuracy
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
    std::printf("%.17g %.17g %.17g\n", mapl::kRetractCoef[i][0], mapl::kRetractCoef[i][1], mapl::kRetractCoef[i][2]);
  return 0;
}
"""


def _retract_coefs():
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    with tempfile.TemporaryDirectory() as tmp:
        src, exe = os.path.join(tmp, "c.cpp"), os.path.join(tmp, "c")
        open(src, "w").write(PROG)
        subprocess.run([cxx, "-std=c++17", "-I", CSRC, src, "-o", exe], check=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    return np.array([[float(v) for v in line.split()] for line in out.splitlines()])


def _quintic(c, x):
    a, b, cc = c
    return a * x + b * x ** 3 + cc * x ** 5


def test_retraction_iterates_stay_bounded():
    coefs = _retract_coefs()
    x1 = np.linspace(0.0, 1.0, 200001)
    x3 = np.linspace(0.0, 1.03, 200001)
    bound = 1.03
    # the first step sees X0 = Y / nu, spectral norm <= 1
    assert _quintic(coefs[0], x1).min() >= 0.0 and _quintic(coefs[0], x1).max() <= bound
    for c in coefs[1:]:
        p = _quintic(c, x3)
        assert p.min() >= 0.0 and p.max() <= bound
    # an entry of a matrix is at most its spectral norm: X's is <= 1.03, the
    # symmetric S = X^T X has eigenvalues in [0, 1.03^2] (in [0, 1] at the
    # first step) and a I + b S + c S^2 has eigenvalues a + b l + c l^2 there
    lam1 = np.linspace(0.0, 1.0, 20001)
    lam = np.linspace(0.0, bound ** 2, 20001)
    q_max = max(np.abs(coefs[0][0] + coefs[0][1] * lam1 + coefs[0][2] * lam1 ** 2).max(),
                max(np.abs(a + b * lam + c * lam ** 2).max() for a, b, c in coefs[1:]))
    assert max(bound, bound ** 2, q_max) < 5.0 < 255.0
