"""Float64 oracle of the MAPL stage-boundary codec (test infrastructure).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use
this module (see oracle/__init__).  Every function is the plain definition
from the paper, computed in float64 with NumPy; nothing is blocked, fused or
reordered beyond what the equations state.

Notation (paper -> here):  X^{b_p} -> X [T,d];  A_p -> U [d,r];
E_p^small -> A [V,k];  P_p -> B ([k,d] for the ambient anchor of Eqs. 1-2,
[k,r] for the coordinate-space reading);  Z^{b_p} -> Z [T,r];  R residual
rounds -> L stages of K codewords, codebooks C [L,K,r].

Operand precision.  ``operand="bf16"`` states that the projector enters the
computation as bf16 (the paper trains in bf16, Sec. 4.1): U is replaced by
round_bf16(U) and, for the ambient anchor, the factor B.U by
round_bf16(B.round_bf16(U)).  Products and sums stay in float64.
``operand="exact"`` uses the given values unchanged (the fp32 path).
"""
import numpy as np

from .precision import round_bf16

AMBIENT = "ambient"
COORD = "coord"


def _projector(U, operand):
    U = np.asarray(U, dtype=np.float64)
    if operand == "bf16":
        return round_bf16(U)
    if operand == "exact":
        return U
    raise ValueError(operand)


def anchor(A, ids):
    """Row gather E_small[t_ids] (Sec. 3.2, Eqs. 1-3): a[t] = A[ids[t]]."""
    ids = np.asarray(ids)
    if ids.size and (ids.min() < 0 or ids.max() >= A.shape[0]):
        raise IndexError("token id out of range")
    return np.asarray(A, dtype=np.float64)[ids]


def project(X, ids, U, A_s, B_s, anchor_space=AMBIENT, operand="exact"):
    """Eq. 1: Z0 = (X - E_small[ids] P) A, before any quantisation.

    ambient: Z0 = (X - a B) U, written as X U - a (B U) (same quantity; the
             factor B U is what enters in bf16 when operand == "bf16").
    coord:   Z0 = X U - a B   (B is [k,r]: the anchor lives in coordinates).
    k == 0 (A_s is None) means no anchor.
    """
    X = np.asarray(X, dtype=np.float64)
    Uo = _projector(U, operand)
    Z0 = X @ Uo
    if A_s is not None and np.asarray(A_s).shape[1] > 0:
        a = anchor(A_s, ids)
        B = np.asarray(B_s, dtype=np.float64)
        if anchor_space == AMBIENT:
            BU = B @ Uo
            if operand == "bf16":
                BU = round_bf16(BU)
            Z0 = Z0 - a @ BU
        elif anchor_space == COORD:
            Z0 = Z0 - a @ B
        else:
            raise ValueError(anchor_space)
    return Z0


def sq_dist_direct(R, Cl):
    """||R_t - C_j||^2 by explicit differences ([T,K]); for tiny inputs."""
    diff = R[:, None, :] - Cl[None, :, :]
    return np.einsum("tkr,tkr->tk", diff, diff)


def sq_dist_expand(R, Cl):
    """||R_t||^2 - 2 R_t.C_j + ||C_j||^2 ([T,K]) in float64."""
    rn = np.einsum("tr,tr->t", R, R)
    cn = np.einsum("kr,kr->k", Cl, Cl)
    return rn[:, None] - 2.0 * (R @ Cl.T) + cn[None, :]


def rvq_encode(Z0, C, direct=False, chunk=4096):
    """Residual vector quantisation (Sec. 3.5): L rounds over codebooks C [L,K,r].

    Round l picks, for every token, the codeword nearest to the current
    residual (squared Euclidean distance; among equal distances the lowest
    index), then subtracts it from the residual.

    Returns (codes [T,L] int64, gap [T,L], resid_sq [T,L+1]) where
    gap[t,l] = (second-smallest - smallest distance) / max(||R_{l}||^2, 1e-300)
    measures how close round l was to a tie (||R_l||^2 is the distance to a
    zero codeword), and resid_sq[t,l] = ||R_l||^2 before round l (and after
    the last round in column L).
    """
    Z0 = np.asarray(Z0, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    T = Z0.shape[0]
    L, K, _ = C.shape
    R = Z0.copy()
    codes = np.zeros((T, L), dtype=np.int64)
    gap = np.zeros((T, L))
    resid_sq = np.zeros((T, L + 1))
    for l in range(L):
        resid_sq[:, l] = np.einsum("tr,tr->t", R, R)
        for t0 in range(0, T, chunk):
            t1 = min(T, t0 + chunk)
            Rc = R[t0:t1]
            s = sq_dist_direct(Rc, C[l]) if direct else sq_dist_expand(Rc, C[l])
            j = np.argmin(s, axis=1)  # first index among equal minima
            codes[t0:t1, l] = j
            if K > 1:
                part = np.partition(s, 1, axis=1)
                gap[t0:t1, l] = (part[:, 1] - part[:, 0]) / np.maximum(resid_sq[t0:t1, l], 1e-300)
            else:
                gap[t0:t1, l] = np.inf
        R = R - C[l][codes[:, l]]
    resid_sq[:, L] = np.einsum("tr,tr->t", R, R)
    return codes, gap, resid_sq


def rvq_decode(codes, C):
    """Progressive refinement of Sec. 3.5: Zhat = sum_l C_l[codes[:, l]]."""
    C = np.asarray(C, dtype=np.float64)
    codes = np.asarray(codes)
    Zh = np.zeros((codes.shape[0], C.shape[2]))
    for l in range(C.shape[0]):
        Zh += C[l][codes[:, l]]
    return Zh


def encode(X, ids, U, A_s, B_s, C=None, anchor_space=AMBIENT, operand="exact", direct=False, group_dim=0):
    """Sender side of Alg. 1: Eq. 1, then RVQ if codebooks are given.

    Returns Z0 [T,r] when C is None or has no rounds, else
    (codes, gap, resid_sq) from rvq_encode (group_dim 0: whole vectors) or
    grouped_rvq_encode.
    """
    Z0 = project(X, ids, U, A_s, B_s, anchor_space, operand)
    if C is None or np.asarray(C).shape[0] == 0:
        return Z0
    if group_dim:
        return grouped_rvq_encode(Z0, C, group_dim)
    return rvq_encode(Z0, C, direct=direct)


def coords(payload, C=None):
    """The receiver's coordinates Zhat: the payload itself, or the RVQ sum
    (whole-vector codes [T,L], or grouped codes [T,L,G] whose group size is
    r / G)."""
    if C is None or np.asarray(C).shape[0] == 0:
        return np.asarray(payload, dtype=np.float64)
    payload = np.asarray(payload)
    if payload.ndim == 3:
        return grouped_rvq_decode(payload, C, np.asarray(C).shape[2] // payload.shape[2])
    return rvq_decode(payload, C)


def decode(payload, ids, U, A_r, B_r, C=None, anchor_space=AMBIENT, operand="exact"):
    """Eq. 2 (receiver side of Alg. 1).

    ambient: Xhat = Zhat U^T + E_{p+1}[ids] P_{p+1}
    coord:   Xhat = (Zhat + a' B) U^T
    """
    Zh = coords(payload, C)
    Uo = _projector(U, operand)
    has_anchor = A_r is not None and np.asarray(A_r).shape[1] > 0
    if anchor_space == COORD and has_anchor:
        Zh = Zh + anchor(A_r, ids) @ np.asarray(B_r, dtype=np.float64)
    Xh = Zh @ Uo.T
    if anchor_space == AMBIENT and has_anchor:
        Xh = Xh + anchor(A_r, ids) @ np.asarray(B_r, dtype=np.float64)
    return Xh


def decode_bwd(dXhat, payload, ids, U, A_r, B_r, C=None, anchor_space=AMBIENT, operand="exact"):
    """Backward of Eq. 2 with respect to Zhat and U (Sec. 3.2, last sentence).

    dZhat = dXhat U                          (the r-dim gradient sent back)
    dU    = dXhat^T Zhat                      (ambient)
          = dXhat^T (Zhat + a' B)             (coord)
    """
    dXh = np.asarray(dXhat, dtype=np.float64)
    Uo = _projector(U, operand)
    Zh = coords(payload, C)
    if anchor_space == COORD and A_r is not None and np.asarray(A_r).shape[1] > 0:
        Zh = Zh + anchor(A_r, ids) @ np.asarray(B_r, dtype=np.float64)
    return dXh @ Uo, dXh.T @ Zh


def encode_bwd(dZ, X, ids, U, A_s, B_s, anchor_space=AMBIENT, operand="exact"):
    """Backward of Eq. 1 with the straight-through estimator across RVQ.

    dX = dZ U^T
    dU = (X - a B)^T dZ     (ambient)
       = X^T dZ             (coord: the anchor term does not involve U)
    """
    dZ = np.asarray(dZ, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    Uo = _projector(U, operand)
    dX = dZ @ Uo.T
    Xr = X
    if anchor_space == AMBIENT and A_s is not None and np.asarray(A_s).shape[1] > 0:
        Xr = X - anchor(A_s, ids) @ np.asarray(B_s, dtype=np.float64)
    return dX, Xr.T @ dZ


def grad_quantize(dXhat, U, Cg, operand="exact"):
    """Quantisation of the backward message (Sec. 3.5: the multi-codebook
    quantiser compresses the backward gradients as well as the forward
    activations).  The r-dim gradient that travels back across the boundary,
    dZhat = dXhat U (the backward of Eq. 2), is residual-vector-quantised
    over its own codebooks Cg [Lg,Kg,r] exactly as the activations are.
    Returns (codes, gap, resid_sq) as rvq_encode."""
    dZ0 = np.asarray(dXhat, dtype=np.float64) @ _projector(U, operand)
    return rvq_encode(dZ0, Cg)


def grad_dequantize(codes, Cg):
    """The sending stage's reconstruction of the quantised gradient:
    progressive refinement, sum_l Cg_l[codes[:, l]]."""
    return rvq_decode(codes, Cg)


def anchor_grad(dY, ids, U, B, V, side="sender", anchor_space=AMBIENT, operand="exact"):
    """Gradient of an anchor table E_small (trainable by Eq. 3), [V,k].

    Every token t contributes a row g[t] to the table row ids[t]:
      sender   (Eq. 1, dY = dZ, the gradient of the encoder's output):
               g = -dZ (B U)^T  (ambient; B U rounded to bf16 when the
               projector enters as bf16, as in project), g = -dZ B^T (coord)
      receiver (Eq. 2): g = dXhat B^T (ambient, dY = dXhat),
               g = dZhat B^T (coord, dY = dZhat = dXhat U)
    and dA[v] = sum of g[t] over the tokens with ids[t] == v.
    """
    dY = np.asarray(dY, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    if side == "sender":
        if anchor_space == AMBIENT:
            Uo = _projector(U, operand)
            BU = B @ Uo
            if operand == "bf16":
                BU = round_bf16(BU)
            g = -dY @ BU.T
        elif anchor_space == COORD:
            g = -dY @ B.T
        else:
            raise ValueError(anchor_space)
    elif side == "receiver":
        g = dY @ B.T
    else:
        raise ValueError(side)
    ids = np.asarray(ids)
    if ids.size and (ids.min() < 0 or ids.max() >= V):
        raise IndexError("token id out of range")
    dA = np.zeros((V, B.shape[0]))
    np.add.at(dA, ids, g)
    return dA


def grouped_rvq_encode(Z0, C, group_dim):
    """Residual vector quantisation with the coordinates decomposed into
    groups (Sec. 3.5; App. E: group dimension 2).  The r coordinates split
    into r / group_dim groups of group_dim consecutive coordinates; group i
    is quantised on its own, over the same group_dim columns of every
    codebook (the per-stage codebook C_p in R^{r x K} read as r / group_dim
    stacked codebooks of K group_dim-dimensional codewords), round after
    round as rvq_encode does for whole vectors.

    The near-tie measure of a group's round is its top-2 gap relative to the
    group's unquantised energy ||Z0_g||^2 (not to the round's own residual):
    two-coordinate groups shrink their residual by orders of magnitude per
    round, so late rounds decide on residuals whose size approaches the
    rounding of Z0 itself, and a gap is only meaningful against the scale at
    which Z0 was computed.

    Returns (codes [T,L,G], gap [T,L,G], resid_sq [T,L+1,G])."""
    Z0 = np.asarray(Z0, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    T, r = Z0.shape
    L = C.shape[0]
    G = r // group_dim
    codes = np.zeros((T, L, G), dtype=np.int64)
    gap = np.zeros((T, L, G))
    resid_sq = np.zeros((T, L + 1, G))
    for g in range(G):
        cols = slice(g * group_dim, (g + 1) * group_dim)
        codes[:, :, g], gap[:, :, g], resid_sq[:, :, g] = rvq_encode(Z0[:, cols], C[:, :, cols])
    # rvq_encode's gap is relative to each round's residual; rescale to ||Z0_g||^2
    gap = gap * resid_sq[:, :L, :] / np.maximum(resid_sq[:, :1, :], 1e-300)
    return codes, gap, resid_sq


def grouped_rvq_decode(codes, C, group_dim):
    """Zhat[:, group g] = sum_l C_l[codes[:, l, g], group g's columns]."""
    C = np.asarray(C, dtype=np.float64)
    codes = np.asarray(codes)
    T, L, G = codes.shape
    Zh = np.zeros((T, C.shape[2]))
    for g in range(G):
        cols = slice(g * group_dim, (g + 1) * group_dim)
        Zh[:, cols] = rvq_decode(codes[:, :, g], C[:, :, cols])
    return Zh
