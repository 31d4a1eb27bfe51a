"""Rounding helpers for the oracle (test infrastructure, see oracle/__init__).

The paper trains in bf16 (Sec. 4.1 and App. E).  Where a floating-point value
decides an integer (the RVQ argmin of Sec. 3.5) both sides must take that
decision from operands of the same precision, so the oracle rounds the
projector U (and the anchor factor B.U) to bf16 exactly where the bf16 codec
feeds them to its matrix units; every product and sum is then carried in
float64.

bf16 here is the IEEE-754 binary32 format truncated to its top 16 bits, with
round-to-nearest-even on the discarded 16 bits.
"""
import numpy as np


def to_f32(x):
    """float64 -> float32 with IEEE round-to-nearest-even (numpy's cast)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def f32_to_bf16_bits(x32):
    """float32 array -> uint16 bf16 bit patterns, round-to-nearest-even.

    NaN is kept quiet (payload forced non-zero); infinities pass through.
    """
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = (u + 0x7FFF + lsb) >> 16
    nan = np.isnan(np.asarray(x32, dtype=np.float32))
    out = rounded.astype(np.uint16)
    out[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return out


def bf16_bits_to_f64(bits):
    """uint16 bf16 bit patterns -> exact float64 values."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def round_bf16(x):
    """float64 -> nearest bf16 value (via float32, both steps RNE), as float64.

    This is the double rounding float64 -> fp32 -> bf16 that a kernel reading
    an fp32 master value into a bf16 operand performs.
    """
    return bf16_bits_to_f64(f32_to_bf16_bits(to_f32(x)))
