"""Seeded synthetic inputs shaped like MAPL's stage-boundary workloads.

This module only draws random inputs; it holds none of the codec's or the
Stiefel step's arithmetic, and it is the one piece shared by the tests, the
benchmark and the oracle checks.  It depends on NumPy alone.

Workloads (boundary activations of the paper's LLaMA stages, App. E: d = 1024
for 150M, d = 2048 for 1B, vocabulary 32000, micro-batches of 4 x 2048 tokens):

  c1        T=512,   d=256,  r=32,  V=1024,  k=16,  L=2, K=64,   fp32
  c2_r{64,128,256,512}
            T=8192,  d=1024, r=.., V=32000, k=64,  L=0,         bf16
  c3        T=8192,  d=1024, r=128, V=32000, k=16,  L=4, K=256,  bf16, u8 codes
  c4        T=32768, d=2048, r=256, V=32000, k=128, L=2, K=1024, bf16, u16 codes
  c6        T=8192,  d=1024, r=256, V=32000, k=64,  L=2, K=256,  bf16, grouped RVQ
            (group dimension 2: u8 codes [T, 2, 128], 256 bytes per token)
  c5        16 projectors U_p [2048,512] fp32, G_p = 1e-3 N(0,1)

Recipe (PCG64 ``numpy.random.default_rng(seed)``, draws in this order):
  1. Q = QR(N(0,1)[d,d]) with columns sign-fixed so diag(R) > 0
  2. outlier channels: rng.choice(d, n_out, replace=False)
  3. X in chunks of 4096 tokens: Zc, Nc ~ N(0,1)[n,d] (Zc first);
     X = (Zc * s) Q^T + 0.1 Nc with s_i = i^-alpha (i = 1..d); outlier
     channels of X multiplied by 20.  Stored as fp32 (c1) or bf16 (RNE of
     the fp32 value).
  4. U = QR(N(0,1)[d,r]), sign-fixed, stored fp32
  5. A = 0.02 N(0,1)[V,k];  B = 0.02 N(0,1)[k,d] (ambient) or [k,r] (coord).
     anchor="orthonormal" instead draws A = a_scale N(0,1)[V,k] and B with
     orthonormal rows, B = Q^T for Q = QR(N(0,1)[cols,k]) sign-fixed (the
     frozen "random orthonormal" companion of Eq. 3 and the hyperparameter
     table): an anchor term as large as the activations themselves
  6. ids: finite Zipf(1.1), P(id = i) proportional to (i+1)^-1.1 on [0, V)
  7. codebooks C [L,K,r] fp32, C_l[0] = 0, other rows sigma_l N(0,1); sigma_l
     is 0.02 for c1 and the root-mean-square of the stored X for c3/c4 (the
     per-coordinate spread of an orthonormal projection of X onto a random
     r-subspace; with Gaussian codewords the zero codeword wins almost every
     token, so the residual keeps that spread at every stage)
  8. upstream gradient dXhat ~ N(0,1)[T,d] (same dtype as X)
  9. upstream gradient dZ ~ N(0,1)[T,r]
 10. Stiefel gradient G ~ gscale N(0,1)[d,r] (c1: gscale 1)
"""
import numpy as np

F32 = "f32"
BF16 = "bf16"

PRESETS = {
    "c1": dict(T=512, d=256, r=32, V=1024, k=16, L=2, K=64, dtype=F32, alpha=0.8, n_out=4,
               cb_sigma=0.02, gscale=1.0, lr=1e-2),
    "c3": dict(T=8192, d=1024, r=128, V=32000, k=16, L=4, K=256, dtype=BF16, alpha=0.8, n_out=4,
               cb_sigma=None, gscale=1.0, lr=1e-2),
    "c4": dict(T=32768, d=2048, r=256, V=32000, k=128, L=2, K=1024, dtype=BF16, alpha=0.7,
               n_out=16, cb_sigma=None, gscale=1.0, lr=1e-2),
}
# the paper's own VQ setting (App. E; Table 1's MAPL+VQ rows at 150M): r = 256,
# two-coordinate groups, K = 256, R = 2 rounds -> 256 bytes per token
PRESETS["c6"] = dict(T=8192, d=1024, r=256, V=32000, k=64, L=2, K=256, dtype=BF16, alpha=0.8, n_out=4,
                     cb_sigma=None, gscale=1.0, lr=1e-2, group_dim=2)
for _r in (64, 128, 256, 512):
    PRESETS["c2_r%d" % _r] = dict(T=8192, d=1024, r=_r, V=32000, k=64, L=0, K=0, dtype=BF16,
                                  alpha=0.8, n_out=4, cb_sigma=None, gscale=1.0, lr=1e-2)

SEEDS = {"c1": 1, "c2_r64": 2, "c2_r128": 2, "c2_r256": 2, "c2_r512": 2, "c3": 3, "c4": 4, "c5": 5, "c6": 6}

STIEFEL_PRESETS = {
    "c1": dict(P=1, d=256, r=32, gscale=1.0, lr=1e-2, beta=0.95, steps=1),
    "c5": dict(P=16, d=2048, r=512, gscale=1e-3, lr=1e-2, beta=0.95, steps=100),
}


def f32_to_bf16_bits(x):
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _sign_fixed_qr(rng, n, m):
    q, rr = np.linalg.qr(rng.standard_normal((n, m)))
    return q * np.sign(np.diag(rr))[None, :]


def zipf_ids(rng, V, T, exponent=1.1):
    p = (np.arange(V, dtype=np.float64) + 1.0) ** (-exponent)
    p /= p.sum()
    return rng.choice(V, size=T, p=p).astype(np.int32)


def _store(x32, dtype):
    return f32_to_bf16_bits(x32) if dtype == BF16 else np.ascontiguousarray(x32, dtype=np.float32)


def as_f64(arr, dtype):
    """Exact float64 values of a stored array (bf16 bits or fp32)."""
    if dtype == BF16:
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


def codec_inputs(name=None, seed=None, anchor_space="ambient", chunk=4096, anchor="gauss", a_scale=1.0,
                 **over):
    """Draw one codec workload.  Returns a dict of NumPy arrays plus sizes.

    Arrays with dtype "bf16" are uint16 bit patterns; "f32" arrays are float32.
    Keyword overrides replace preset fields (T, d, r, V, k, L, K, dtype, ...);
    rotate=False keeps the power-law spectrum on the coordinate axes instead
    of behind a random orthogonal Q (no d x d QR: for the widest d).
    """
    cfg = dict(PRESETS[name]) if name else {}
    cfg.update(over)
    if seed is None:
        seed = SEEDS.get(name, 0)
    T, d, r, V, k = (int(cfg[x]) for x in ("T", "d", "r", "V", "k"))
    L, K = int(cfg["L"]), int(cfg["K"])
    dt = cfg["dtype"]
    rng = np.random.default_rng(seed)
    rotate = bool(cfg.get("rotate", True))
    Q = _sign_fixed_qr(rng, d, d) if rotate else None
    out_ch = rng.choice(d, size=int(cfg["n_out"]), replace=False)
    s = np.arange(1, d + 1, dtype=np.float64) ** (-float(cfg["alpha"]))
    QsT = (Q * s[None, :]).T if rotate else None  # (Z * s) Q^T = Z (Q diag(s))^T
    X = np.empty((T, d), dtype=np.uint16 if dt == BF16 else np.float32)
    sq = 0.0
    for t0 in range(0, T, chunk):
        n = min(chunk, T - t0)
        Zc = rng.standard_normal((n, d))
        Nc = rng.standard_normal((n, d))
        Xc = (Zc @ QsT if rotate else Zc * s[None, :]) + 0.1 * Nc
        Xc[:, out_ch] *= 20.0
        Xc32 = Xc.astype(np.float32)
        X[t0:t0 + n] = _store(Xc32, dt)
        sq += float(np.square(as_f64(X[t0:t0 + n], dt)).sum())
    U = _sign_fixed_qr(rng, d, r).astype(np.float32)
    bdim = d if anchor_space == "ambient" else r
    if anchor == "gauss":
        A32 = (0.02 * rng.standard_normal((V, k))).astype(np.float32)
        B32 = (0.02 * rng.standard_normal((k, bdim))).astype(np.float32)
    elif anchor == "orthonormal":
        A32 = (a_scale * rng.standard_normal((V, k))).astype(np.float32)
        B32 = (_sign_fixed_qr(rng, bdim, k).T if k else np.zeros((0, bdim))).astype(np.float32)
    else:
        raise ValueError(anchor)
    ids = zipf_ids(rng, V, T)
    C = np.zeros((L, max(K, 0), r), dtype=np.float32)
    sigma = cfg.get("cb_sigma")
    if sigma is None:
        sigma = np.sqrt(sq / (T * d)) if T * d else 0.0
    for l in range(L):
        if K > 1:
            C[l, 1:] = (sigma * rng.standard_normal((K - 1, r))).astype(np.float32)
    dXhat = _store(rng.standard_normal((T, d)).astype(np.float32), dt)
    dZ = _store(rng.standard_normal((T, r)).astype(np.float32), dt)
    G = (float(cfg["gscale"]) * rng.standard_normal((d, r))).astype(np.float32)
    return dict(name=name, seed=seed, T=T, d=d, r=r, V=V, k=k, L=L, K=K, dtype=dt,
                anchor_space=anchor_space, X=X, U=U, A=_store(A32, dt), B=_store(B32, dt),
                ids=ids, C=C, dXhat=dXhat, dZ=dZ, G=G, cb_sigma=float(sigma),
                code_dtype=("u8" if K <= 256 else "u16"), lr=float(cfg.get("lr", 1e-2)), anchor=anchor,
                group_dim=int(cfg.get("group_dim", 0)))


def stiefel_inputs(name=None, seed=None, **over):
    """Draw a batch of projectors U [P,d,r] (QR of Gaussians, fp32), zero
    momentum, and the first gradient G [P,d,r] = gscale N(0,1)."""
    cfg = dict(STIEFEL_PRESETS[name]) if name else {}
    cfg.update(over)
    if seed is None:
        seed = SEEDS.get(name, 0) + 1000
    P, d, r = int(cfg["P"]), int(cfg["d"]), int(cfg["r"])
    rng = np.random.default_rng(seed)
    U = np.stack([_sign_fixed_qr(rng, d, r) for _ in range(P)]).astype(np.float32)
    G = (float(cfg["gscale"]) * rng.standard_normal((P, d, r))).astype(np.float32)
    return dict(name=name, seed=seed, P=P, d=d, r=r, U=U, G=G,
                M=np.zeros((P, d, r), dtype=np.float32), lr=float(cfg["lr"]),
                beta=float(cfg["beta"]), steps=int(cfg["steps"]), gscale=float(cfg["gscale"]),
                rng=rng)


def next_gradient(st):
    """Fresh gradient for the next step of a Stiefel trajectory."""
    rng = st["rng"]
    P, d, r = st["P"], st["d"], st["r"]
    return (st["gscale"] * rng.standard_normal((P, d, r))).astype(np.float32)
