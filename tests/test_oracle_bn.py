"""Pins of the oracle's L1 batch normalization (Eq. 12-15) and its backward:
the hand-worked example, the exact-rational brute force of the real-valued
formulas, finite differences of Eq. 12-13, the zero-sum property of the
backward and the Gaussian L1/L2 deviation ratio."""
import json
import math
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

import bruteforce as bf
from paper_2011_14504_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))
CFG = dict(k_mu=16, k_sigma=16, k_xhat=16, k_gamma=8, k_beta=8, k_A=8, k_E1=8,
           k_E2=16, eps_code=0, relu=1)


def _cols(codes, e):
    """[M, C] codes -> per-channel lists of rational values."""
    a = np.asarray(codes).reshape(-1, np.asarray(codes).shape[-1])
    return [[Fr(int(v)) * Fr(2) ** e for v in a[:, c]] for c in range(a.shape[1])]


def test_l1bn_hand_example(orc):
    g = GOLD["l1bn_fwd"]
    x = np.array(g["x_codes"], np.int8).reshape(4, 1)
    r = orc.bn_fwd(x, g["x_exp"], [g["gamma_code"]], [g["beta_code"]], CFG)
    assert int(r["n_mu"][0]) == g["n_mu"] and int(r["n_sigma"][0]) == g["n_sigma"]
    assert r["b"] == g["b"]
    assert r["xhat"].ravel().tolist() == g["xhat_codes"]
    assert r["y"].ravel().tolist() == g["A_codes"] and r["y_exp"] == g["A_exp"]


def _bn_case(seed, M, C, x_exp, cfg, rand_affine=True, const_chan=False):
    x = synth.int_codes(seed, (M, C))
    if const_chan:
        x[:, 0] = 17
    if rand_affine:
        gq = synth.int_codes(seed + 1, (C,))
        bq = synth.int_codes(seed + 2, (C,))
    else:
        gq = np.full(C, 64, np.int8)
        bq = np.zeros(C, np.int8)
    return x, gq, bq


CASES = [
    dict(seed=1, M=6, C=3, x_exp=-7, cfg={}),
    dict(seed=2, M=5, C=2, x_exp=-2, cfg=dict(relu=0)),
    dict(seed=3, M=7, C=2, x_exp=-16, cfg=dict(eps_code=1)),
    dict(seed=4, M=4, C=3, x_exp=3, cfg=dict(k_E2=8)),
    dict(seed=5, M=8, C=2, x_exp=-9, cfg=dict(relu=0, k_E2=8), const_chan=True),
    dict(seed=6, M=3, C=4, x_exp=-20, cfg={}),
    dict(seed=7, M=9, C=1, x_exp=-7, cfg=dict(k_xhat=8, k_mu=8, k_sigma=8)),
    dict(seed=8, M=6, C=2, x_exp=-7, cfg={}, rand_affine=False),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c['seed']}")
def test_l1bn_fwd_vs_bruteforce(orc, case):
    cfg = dict(CFG, **case["cfg"])
    x, gq, bq = _bn_case(case["seed"], case["M"], case["C"], case["x_exp"], cfg,
                         case.get("rand_affine", True), case.get("const_chan", False))
    r = orc.bn_fwd(x, case["x_exp"], gq, bq, cfg)
    gam = [Fr(int(v)) * Fr(2) ** (2 - cfg["k_gamma"]) for v in gq]
    bet = [Fr(int(v)) * Fr(2) ** (2 - cfg["k_beta"]) for v in bq]
    ref = bf.l1bn_forward(_cols(x, case["x_exp"]), gam, bet, cfg)
    e_mu = 2 - cfg["k_mu"]
    assert [Fr(int(v)) * Fr(2) ** e_mu for v in r["n_mu"]] == ref["mu_q"]
    assert [Fr(int(v)) * Fr(2) ** (2 - cfg["k_sigma"]) for v in r["n_sigma"]] == ref["sigma_q"]
    e_xh = r["b"] - (cfg["k_xhat"] - 1)
    assert _cols(r["xhat"], e_xh) == ref["xhat_q"]
    assert _cols(r["y"], r["y_exp"]) == ref["A"]
    lim = 2 ** (cfg["k_A"] - 1) - 1
    assert r["y"].max() <= lim and r["y"].min() >= -lim


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c['seed']}")
def test_l1bn_bwd_vs_bruteforce(orc, case):
    cfg = dict(CFG, **case["cfg"])
    x, gq, bq = _bn_case(case["seed"], case["M"], case["C"], case["x_exp"], cfg,
                         case.get("rand_affine", True), case.get("const_chan", False))
    dA = synth.int_codes(case["seed"] + 50, x.shape)
    dA_exp = -20
    r = orc.bn_bwd(dA, dA_exp, x, case["x_exp"], gq, bq, cfg, want_pre=True)
    gam = [Fr(int(v)) * Fr(2) ** (2 - cfg["k_gamma"]) for v in gq]
    bet = [Fr(int(v)) * Fr(2) ** (2 - cfg["k_beta"]) for v in bq]
    ref = bf.l1bn_backward(_cols(x, case["x_exp"]), _cols(dA, dA_exp), gam, bet, cfg)
    assert [Fr(int(v)) * Fr(2) ** r["dbeta_exp"] for v in r["dbeta"]] == ref["dbeta"]
    assert [Fr(int(v)) * Fr(2) ** r["dgamma_exp"] for v in r["dgamma"]] == ref["dgamma"]
    assert _cols(r["dx"], r["dx_exp"]) == ref["E1"]
    pre = r["dx_pre"]
    for c in range(x.shape[1]):
        for i in range(x.shape[0]):
            assert abs(pre[i, c] - float(ref["dx_pre"][c][i])) <= 1e-12 * max(1e-300, abs(float(ref["dx_pre"][c][i]))) + 1e-300
    assert r["zero_sum_failures"] == 0


def _l1bn_float(x):
    mu = x.mean(axis=0)
    sig = np.abs(x - mu).mean(axis=0)
    return (x - mu) / sig


def test_l1bn_bwd_finite_differences(orc):
    # the oracle's dx before E1's quantizer against central differences of the
    # unquantized Eq. 12-13 (eps = 0); E2 exact (k_E2 = 16) and no ReLU, so the
    # upstream gradient is exactly gamma_q * dA.  The quantized statistics
    # (mu_q, sigma_q, xhat_q) leave a ~1e-4 relative gap; dropping the
    # mean-of-sign term of d sigma/dx would leave a gap of order 1e-1.
    M, C = 41, 3
    x_exp = -7
    x = synth.int_codes(61, (M, C))
    gq = np.array([64, -90, 37], np.int8)
    bq = np.zeros(C, np.int8)
    dA = synth.int_codes(62, (M, C))
    cfg = dict(CFG, relu=0)
    r = orc.bn_bwd(dA, -20, x, x_exp, gq, bq, cfg, want_pre=True)
    xf = x.astype(np.float64) * 2.0 ** x_exp
    gup = (gq.astype(np.float64) * 2.0 ** -6) * dA.astype(np.float64) * 2.0 ** -20
    mu = xf.mean(axis=0)
    assert np.all(np.abs(xf - mu) > 1e-9)      # no element at the kink of |x - mu|
    h = 1e-7
    fd = np.zeros_like(xf)
    for i in range(M):
        for c in range(C):
            xp = xf.copy(); xp[i, c] += h
            xm = xf.copy(); xm[i, c] -= h
            fd[i, c] = ((gup * _l1bn_float(xp)).sum() - (gup * _l1bn_float(xm)).sum()) / (2 * h)
    scale = np.abs(fd).max()
    err = np.abs(r["dx_pre"] - fd).max() / scale
    assert err < 2e-3, err
    # without the mean-of-sign term the derivative would be visibly different
    s = np.sign(xf - mu)
    xh = _l1bn_float(xf)
    sig = np.abs(xf - mu).mean(axis=0)
    no_sign_mean = (gup - gup.mean(0) - (gup * xh).mean(0) * s) / sig
    assert np.abs(no_sign_mean - fd).max() / scale > 20 * err


def test_l1bn_bwd_zero_sum_large(orc):
    x = synth.int_codes(71, (3000, 8))
    dA = synth.int_codes(72, (3000, 8))
    gq = synth.int_codes(73, (8,))
    bq = synth.int_codes(74, (8,))
    for kE2 in (8, 16):
        r = orc.bn_bwd(dA, -20, x, -7, gq, bq, dict(CFG, k_E2=kE2))
        assert r["zero_sum_failures"] == 0


def test_l1_deviation_ratio_gaussian(orc):
    # Sec. 1 relies on L1BN being equivalent to L2BN: for Gaussian data the
    # mean absolute deviation is sqrt(2/pi) times the standard deviation.
    M = 200000
    x = synth.gaussian_codes(81, (M, 1), std=20.0)
    r = orc.bn_fwd(x, -7, [64], [0], CFG)
    sigma_l1 = int(r["n_sigma"][0]) * 2.0 ** -14
    xf = x.astype(np.float64) * 2.0 ** -7
    ratio = sigma_l1 / xf.std()
    assert abs(ratio - math.sqrt(2 / math.pi)) < 5e-3


def test_l1bn_range_preconditions(orc):
    x = synth.int_codes(91, (4, 2))
    with pytest.raises(orc.OracleError):
        orc.bn_fwd(x, 17, [64, 64], [0, 0], CFG)
    with pytest.raises(orc.OracleError):
        orc.bn_fwd(x, -41, [64, 64], [0, 0], CFG)


# L1BN on the raw int32 sums of a convolution (the paper's literal dataflow:
# BN consumes the MAC output before any requantization, Sec. 3.2.2-3.2.3)
WIDE_CASES = [
    dict(seed=31, M=6, C=3, x_exp=-14, mag=1 << 20, cfg={}),
    dict(seed=32, M=5, C=2, x_exp=-20, mag=1 << 30, cfg=dict(relu=0)),
    dict(seed=33, M=7, C=2, x_exp=0, mag=1 << 30, cfg=dict(eps_code=3)),
    dict(seed=34, M=4, C=3, x_exp=-40, mag=1 << 12, cfg=dict(k_E2=8)),
    dict(seed=35, M=8, C=2, x_exp=-9, mag=3000, cfg=dict(relu=0, k_E2=8)),
]


def _wide_case(case):
    rng = synth.rng(case["seed"])
    m = case["mag"]
    x = rng.integers(-m, m + 1, size=(case["M"], case["C"])).astype(np.int32)
    x[0, 0] = m if case["seed"] % 2 else -m
    gq = synth.int_codes(case["seed"] + 1, (case["C"],))
    bq = synth.int_codes(case["seed"] + 2, (case["C"],))
    return x, gq, bq


@pytest.mark.parametrize("case", WIDE_CASES, ids=lambda c: f"seed{c['seed']}")
def test_l1bn_int32_input_vs_bruteforce(orc, case):
    cfg = dict(CFG, **case["cfg"])
    x, gq, bq = _wide_case(case)
    gam = [Fr(int(v)) * Fr(2) ** (2 - cfg["k_gamma"]) for v in gq]
    bet = [Fr(int(v)) * Fr(2) ** (2 - cfg["k_beta"]) for v in bq]
    r = orc.bn_fwd(x, case["x_exp"], gq, bq, cfg)
    ref = bf.l1bn_forward(_cols(x, case["x_exp"]), gam, bet, cfg)
    assert [Fr(int(v)) * Fr(2) ** (2 - cfg["k_mu"]) for v in r["n_mu"]] == ref["mu_q"]
    assert [Fr(int(v)) * Fr(2) ** (2 - cfg["k_sigma"]) for v in r["n_sigma"]] == ref["sigma_q"]
    assert _cols(r["xhat"], r["b"] - (cfg["k_xhat"] - 1)) == ref["xhat_q"]
    assert _cols(r["y"], r["y_exp"]) == ref["A"]
    dA = synth.int_codes(case["seed"] + 50, x.shape)
    rb = orc.bn_bwd(dA, -20, x, case["x_exp"], gq, bq, cfg)
    refb = bf.l1bn_backward(_cols(x, case["x_exp"]), _cols(dA, -20), gam, bet, cfg)
    assert [Fr(int(v)) * Fr(2) ** rb["dbeta_exp"] for v in rb["dbeta"]] == refb["dbeta"]
    assert [Fr(int(v)) * Fr(2) ** rb["dgamma_exp"] for v in rb["dgamma"]] == refb["dgamma"]
    assert _cols(rb["dx"], rb["dx_exp"]) == refb["E1"]
    assert rb["zero_sum_failures"] == 0


def test_l1bn_int32_input_equals_int8_path_on_8bit_codes(orc):
    """Codes that fit 8 bits give the same result through either input type."""
    x = synth.int_codes(41, (300, 8))
    gq = synth.int_codes(42, (8,))
    bq = synth.int_codes(43, (8,))
    dA = synth.int_codes(44, x.shape)
    a = orc.bn_fwd(x, -7, gq, bq, CFG)
    b = orc.bn_fwd(x.astype(np.int32), -7, gq, bq, CFG)
    for k in ("y", "n_mu", "n_sigma", "xhat"):
        assert np.array_equal(a[k], b[k]), k
    assert a["y_exp"] == b["y_exp"] and a["b"] == b["b"]
    ra = orc.bn_bwd(dA, -20, x, -7, gq, bq, CFG)
    rb = orc.bn_bwd(dA, -20, x.astype(np.int32), -7, gq, bq, CFG)
    for k in ("dx", "dgamma", "dbeta"):
        assert np.array_equal(ra[k], rb[k]), k
    assert ra["dx_exp"] == rb["dx_exp"]


def test_l1bn_int32_input_range(orc):
    x = synth.int_codes(91, (4, 2)).astype(np.int32) * 1000
    orc.bn_fwd(x, 0, [64, 64], [0, 0], CFG)
    with pytest.raises(orc.OracleError):
        orc.bn_fwd(x, 1, [64, 64], [0, 0], CFG)
    with pytest.raises(orc.OracleError):
        orc.bn_fwd(x, -41, [64, 64], [0, 0], CFG)


# Inference with the frozen state of a calibration forward (the paper gives
# no running-statistics rule; every quantizer keeps the calibration's step)
def test_requant_fixed_hand_examples(orc):
    a = np.array([1000, 1004, 1003, -1004, -1005, 5000, -5000, 0], np.int64)
    # step 2^3: 125, 125.5 -> 126 (half up), 125.375 -> 125, -125.5 -> -125, -125.625 -> -126, clip
    assert orc.requant_fixed(a, 0, 3).tolist() == [125, 126, 125, -125, -126, 127, -127, 0]
    assert orc.requant_fixed(np.array([3, -3], np.int64), -2, -4).tolist() == [12, -12]    # exact left shift


def test_bn_infer_on_the_calibration_batch_equals_training_forward(orc):
    for seed, cfg in ((61, {}), (62, dict(relu=0)), (63, dict(eps_code=2, k_xhat=12))):
        cfg = dict(CFG, **cfg)
        x = synth.int_codes(seed, (700, 12))
        gq = synth.int_codes(seed + 1, (12,))
        bq = synth.int_codes(seed + 2, (12,))
        fwd = orc.bn_fwd(x, -9, gq, bq, cfg)
        assert np.array_equal(orc.bn_infer(x, -9, gq, bq, orc.bn_state(fwd), cfg), fwd["y"])


def test_bn_infer_vs_bruteforce(orc):
    """A new batch through the frozen state, against Eq. 12-15 in Fractions
    with the calibration's mu_q, sigma_q and the fixed steps of Q_xhat, Q_A."""
    cfg = dict(CFG)
    cal = synth.int_codes(71, (9, 3))
    new = synth.int_codes(72, (7, 3)) // 2 + 40          # shifted: some codes clip
    gq = synth.int_codes(73, (3,))
    bq = synth.int_codes(74, (3,))
    st = orc.bn_state(orc.bn_fwd(cal, -5, gq, bq, cfg))
    got = orc.bn_infer(new, -5, gq, bq, st, cfg)
    lsb = Fr(2) ** (2 - cfg["k_sigma"])
    for c in range(3):
        mu = Fr(int(st["n_mu"][c])) * Fr(2) ** (2 - cfg["k_mu"])
        den = max(Fr(int(st["n_sigma"][c])) * lsb + cfg["eps_code"] * lsb, lsb)
        gam = Fr(int(gq[c])) * Fr(2) ** (2 - cfg["k_gamma"])
        bet = Fr(int(bq[c])) * Fr(2) ** (2 - cfg["k_beta"])
        Sx = Fr(2) ** st["b"]
        for i in range(new.shape[0]):
            xv = Fr(int(new[i, c])) * Fr(2) ** -5
            xq = Sx * bf.UQ((xv - mu) / den / Sx, cfg["k_xhat"])          # fixed step, clipped
            y = gam * xq + bet
            y = max(y, Fr(0)) if cfg["relu"] else y
            SA = Fr(2) ** (st["a_exp"] + cfg["k_A"] - 1)
            want = SA * bf.UQ(y / SA, cfg["k_A"])
            assert Fr(int(got[i, c])) * Fr(2) ** st["a_exp"] == want, (i, c)
