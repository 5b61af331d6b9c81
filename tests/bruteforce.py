"""Exact-rational brute force of the paper's real-valued formulas.

Written from the equations of arXiv 2011.14504 Sec. 3 with Python Fractions,
on tiny tensors, independently of the oracle's integer formulation (no
exponents, shifts or integer codes: values are rationals throughout).  Used
to pin the oracle.
"""
import math
from fractions import Fraction as Fr


def delta(k):
    """Eq. 1: Delta(k) = 2^(1-k)."""
    return Fr(1, 2 ** (k - 1))


def clip(v, lo, hi):
    return max(lo, min(hi, v))


def UQ(x, k):
    """Eq. 2: Clip(Delta * floor(x / Delta + 1/2), -1 + Delta, 1 - Delta)."""
    d = delta(k)
    return clip(d * math.floor(x / d + Fr(1, 2)), -1 + d, 1 - d)


def pow2_scale(values):
    """Scale(x) (Eq. 3) read as the smallest power of two strictly above
    max|x|; None for an all-zero tensor."""
    M = max(abs(v) for v in values)
    if M == 0:
        return None
    S = Fr(1)
    while S <= M:
        S *= 2
    while S / 2 > M:
        S /= 2
    return S


def SQ(values, k):
    """Eq. 4: Scale(x) * UQ(x / Scale(x), k), one scale for the tensor."""
    S = pow2_scale(values)
    if S is None:
        return [Fr(0)] * len(values)
    return [S * UQ(v / S, k) for v in values]


def SQ_max(values, k):
    """Eq. 3-4 as printed: Scale(x) = max|x| exactly (not a power of two), so
    the largest element maps to x/Scale = 1 and is clipped to 1 - Delta.
    Used only to measure how far the power-of-two reading departs from it."""
    M = max(abs(v) for v in values)
    if M == 0:
        return [Fr(0)] * len(values)
    return [M * UQ(v / M, k) for v in values]


def RQ_probs(v, S, k):
    """Eq. 5-6 for one value scaled by S: returns {quantized value: prob}."""
    d = delta(k)
    y = v / S / d
    lo = math.floor(y)
    frac = y - lo
    out = {}
    for n, p in ((lo, 1 - frac), (lo + 1, frac)):
        if p == 0:
            continue
        val = S * clip(d * n, -1 + d, 1 - d)
        out[val] = out.get(val, 0) + p
    return out


def sgn(v):
    return (v > 0) - (v < 0)


def conv2d(x, w, stride, pad, dil):
    """Literal cross-correlation, zero padding. x[n][h][w][c], w[k][r][s][c]."""
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    K, R, S = len(w), len(w[0]), len(w[0][0])
    P = (H + 2 * pad - dil * (R - 1) - 1) // stride + 1
    Q = (W + 2 * pad - dil * (S - 1) - 1) // stride + 1
    out = [[[[0] * K for _ in range(Q)] for _ in range(P)] for _ in range(N)]
    for n in range(N):
        for p in range(P):
            for q in range(Q):
                for k in range(K):
                    s_ = 0
                    for r in range(R):
                        for s in range(S):
                            h = p * stride - pad + r * dil
                            ww = q * stride - pad + s * dil
                            if 0 <= h < H and 0 <= ww < W:
                                for c in range(C):
                                    s_ += x[n][h][ww][c] * w[k][r][s][c]
                    out[n][p][q][k] = s_
    return out


def l1bn_forward(xcols, gammas, betas, cfg):
    """Eq. 12-15 on per-channel columns of rational values.

    xcols[c] = list of the channel's m values.  gammas/betas are the already
    quantized gamma_q / beta_q values.  Readings: sigma from the quantized
    mean; eps = eps_code * 2^(2-k_sigma) with the denominator kept at least
    one sigma LSB; ReLU before Q_A; SQ with one scale per tensor.
    Returns dict with per-channel mu_q, sigma_q, den and per-element xhat_q,
    y (pre-ReLU), A (values)."""
    k_mu, k_sig, k_xh, k_A = cfg["k_mu"], cfg["k_sigma"], cfg["k_xhat"], cfg["k_A"]
    lsb_sig = 2 * delta(k_sig)
    res = dict(mu_q=[], sigma_q=[], den=[], xhat=[])
    for xs in xcols:
        m = len(xs)
        mu = sum(xs) / m                                   # Eq. 10
        mu_q = 2 * UQ(mu / 2, k_mu)                        # Eq. 14
        sigma = sum(abs(v - mu_q) for v in xs) / m         # Eq. 13 (reading: mu_q)
        sigma_q = 2 * UQ(sigma / 2, k_sig)                 # Eq. 14
        den = max(sigma_q + cfg["eps_code"] * lsb_sig, lsb_sig)
        res["mu_q"].append(mu_q)
        res["sigma_q"].append(sigma_q)
        res["den"].append(den)
        res["xhat"].append([(v - mu_q) / den for v in xs])  # Eq. 12
    flat = [v for col in res["xhat"] for v in col]
    flat_q = SQ(flat, k_xh)                                 # Eq. 14, Q_xhat
    m = len(xcols[0])
    xq = [flat_q[c * m:(c + 1) * m] for c in range(len(xcols))]
    y = [[gammas[c] * v + betas[c] for v in xq[c]] for c in range(len(xcols))]
    yr = [[max(v, 0) if cfg["relu"] else v for v in col] for col in y]
    flat_y = [v for col in yr for v in col]
    A = SQ(flat_y, k_A)                                     # Eq. 15
    res["xhat_q"] = xq
    res["y"] = y
    res["A"] = [A[c * m:(c + 1) * m] for c in range(len(xcols))]
    S = pow2_scale(flat)
    res["xhat_scale"] = S
    return res


def l1bn_backward(xcols, dAcols, gammas, betas, cfg):
    """Backward of L1BN (+ReLU) by the exact derivative of Eq. 12-13 with
    straight-through quantizers; E2 and E1 quantized by SQ (Eq. 16)."""
    fw = l1bn_forward(xcols, gammas, betas, cfg)
    Cn = len(xcols)
    m = len(xcols[0])
    delta_ = [[dAcols[c][i] if (not cfg["relu"] or fw["y"][c][i] > 0) else Fr(0)
               for i in range(m)] for c in range(Cn)]
    dbeta = [sum(col) for col in delta_]
    dgamma = [sum(delta_[c][i] * fw["xhat_q"][c][i] for i in range(m)) for c in range(Cn)]
    g = [gammas[c] * delta_[c][i] for c in range(Cn) for i in range(m)]
    E2f = SQ(g, cfg["k_E2"])
    E2 = [E2f[c * m:(c + 1) * m] for c in range(Cn)]
    dx = []
    for c in range(Cn):
        s = [sgn(v - fw["mu_q"][c]) for v in xcols[c]]
        mean_s = Fr(sum(s), m)
        mean_e = sum(E2[c]) / m
        mean_ex = sum(E2[c][i] * fw["xhat_q"][c][i] for i in range(m)) / m
        dx.append([(E2[c][i] - mean_e - mean_ex * (s[i] - mean_s)) / fw["den"][c]
                   for i in range(m)])
    flat = [v for col in dx for v in col]
    E1 = SQ(flat, cfg["k_E1"])
    return dict(dbeta=dbeta, dgamma=dgamma, dx_pre=dx,
                E1=[E1[c * m:(c + 1) * m] for c in range(Cn)])
