"""Greedy minimax odd-quintic schedule for PolarExpress (oracle side).

Test infrastructure (see oracle/__init__).  Sec. 3.3 (Eqs. 6-7) and the
hyper-parameter table of App. H name PolarExpress (Amsel et al., 2025) for
both the LMO direction (5 steps) and the retraction (7 steps) but print no
coefficients.  PolarExpress's published construction is: on the current
interval [l, u] that holds every singular value, choose the odd polynomial
p(x) = a x + b x^3 + c x^5 minimising max_{x in [l,u]} |1 - p(x)|; the image
of [l, u] under that p is [1 - E, 1 + E] where E is the minimax error, which
becomes the next interval.

This module derives that schedule in float64 with the Remez exchange
algorithm.  The HIP library carries its own table, produced by an independent
generator; a test compares the two.

Once the interval [l, u] is narrower than ``CONTACT_SWITCH`` (half-width
below 0.05) the minimax problem becomes ill-conditioned (the optimal error
is O(width^3) and the coefficients lose digits); from there on the schedule
uses the odd quintic with third-order contact at 1, fixed by p(1) = 1,
p'(1) = 0, p''(1) = 0, i.e. (a, b, c) = (15/8, -10/8, 3/8), which is
monotone and maps [1 - w, 1 + w] to within O(w^3) of 1.
"""
import numpy as np

CONTACT_SWITCH = 0.1


def _poly(coef, x):
    a, b, c = coef
    x2 = x * x
    return x * (a + x2 * (b + c * x2))


def _critical_points(coef, lo, hi):
    """Interior zeros of p'(x) = a + 3b x^2 + 5c x^4 inside (lo, hi)."""
    a, b, c = coef
    roots = np.roots([5.0 * c, 3.0 * b, a])  # in y = x^2
    pts = []
    for y in roots:
        if abs(y.imag) < 1e-12 * max(1.0, abs(y.real)) and y.real > 0:
            x = np.sqrt(y.real)
            if lo < x < hi:
                pts.append(x)
    return sorted(pts)


def minimax_quintic(lo, hi, iters=100, tol=1e-15):
    """Return (a, b, c, E) minimising max |1 - p| on [lo, hi] (Remez exchange).

    The optimum equioscillates at lo, two interior critical points and hi,
    with 1 - p(lo) = +E.
    """
    # Chebyshev-like initial reference on [lo, hi]
    t = np.cos(np.pi * np.arange(3, -1, -1) / 3.0)
    ref = lo + (hi - lo) * (t + 1.0) / 2.0
    sol = None
    for _ in range(iters):
        sgn = np.array([1.0, -1.0, 1.0, -1.0])
        # a x + b x^3 + c x^5 + sgn*E = 1
        M = np.stack([ref, ref ** 3, ref ** 5, sgn], axis=1)
        sol = np.linalg.solve(M, np.ones(4))
        coef = sol[:3]
        crit = _critical_points(coef, lo, hi)
        if len(crit) != 2:
            raise RuntimeError("Remez: expected two interior extrema on [%g, %g]" % (lo, hi))
        new_ref = np.array([lo, crit[0], crit[1], hi])
        if np.max(np.abs(new_ref - ref)) <= tol * hi:
            ref = new_ref
            break
        ref = new_ref
    # final solve on the converged reference
    sgn = np.array([1.0, -1.0, 1.0, -1.0])
    M = np.stack([ref, ref ** 3, ref ** 5, sgn], axis=1)
    sol = np.linalg.solve(M, np.ones(4))
    return float(sol[0]), float(sol[1]), float(sol[2]), float(abs(sol[3]))


def greedy_schedule(lo, steps, hi=1.0):
    """Greedy PolarExpress schedule: list of (a, b, c) for ``steps`` steps.

    Also returns the list of intervals [l_t, u_t] each step was designed for.
    """
    coefs, intervals = [], []
    l, u = float(lo), float(hi)
    for _ in range(steps):
        intervals.append((l, u))
        if u - l < CONTACT_SWITCH:
            a, b, c = 15.0 / 8.0, -10.0 / 8.0, 3.0 / 8.0
            coefs.append((a, b, c))
            # image of [l, u] under the contact polynomial
            xs = np.linspace(l, u, 65)
            ys = _poly((a, b, c), xs)
            l, u = float(ys.min()), float(ys.max())
            continue
        a, b, c, E = minimax_quintic(l, u)
        coefs.append((a, b, c))
        l, u = 1.0 - E, 1.0 + E
    return coefs, intervals


def compose(coefs, x):
    """Apply the scalar recursion x <- p_t(x) for every step (float64)."""
    y = np.asarray(x, dtype=np.float64)
    for cf in coefs:
        y = _poly(cf, y)
    return y
