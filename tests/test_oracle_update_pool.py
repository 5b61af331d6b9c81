"""Pins of the oracle's weight/update quantizers (Eq. 7, 8, 19) and of the
max-pool glue."""
import json
import os
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import bruteforce as bf
from paper_2011_14504_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


@pytest.mark.parametrize("case", GOLD["q_w"], ids=lambda c: str(c["master"]))
def test_qw_hand_examples(orc, case):
    wq = orc.weight_quant(np.array([case["master"]], np.int32), case["k_U"], case["k_W"])
    assert int(wq[0]) == case["code"]


@pytest.mark.parametrize("case", GOLD["update"], ids=lambda c: str(c["master"]))
def test_update_hand_examples(orc, case):
    m, wq = orc.weight_update(np.array([case["master"]], np.int32), np.array([case["g"]], np.int8),
                              case["g_exp"], case["lr_shift"], -23, case["k_U"], case["k_W"])
    assert int(m[0]) == case["new_master"]
    assert int(wq[0]) == int(orc.weight_quant(m, case["k_U"], case["k_W"])[0])


def test_q_mu_hand_example(orc):
    c = GOLD["q_mu"][0]
    # Eq. 14: mu_q = 2 UQ(mu/2, k) -> code of UQ(mu/2)
    assert orc.uq_code(float(Fr(c["mu"])) / 2, c["k"]) == c["code"]


def test_update_vs_bruteforce(orc):
    rng = synth.rng(5)
    n = 500
    master = rng.integers(-(2 ** 23) + 1, 2 ** 23, size=n, dtype=np.int64).astype(np.int32)
    master[:5] = [2 ** 23 - 1, -(2 ** 23 - 1), 0, 65535, -32768]
    g = synth.int_codes(6, (n,))
    for g_exp, lr, mexp in [(-20, 10, -23), (-3, 4, -23), (-30, 0, -22), (5, 2, -23)]:
        m2, wq = orc.weight_update(master, g, g_exp, lr, mexp, 24, 8)
        d24 = bf.delta(24)
        for i in range(n):
            W = Fr(int(master[i])) * Fr(2) ** mexp
            G = Fr(int(g[i])) * Fr(2) ** g_exp
            fold = 2 if mexp == -22 else 1           # gamma/beta: 2 UQ(./2, k)
            dW = fold * bf.UQ(G * Fr(2) ** -lr / fold, 24)
            Wn = bf.clip(W - dW, -fold * (1 - d24), fold * (1 - d24))
            assert Fr(int(m2[i])) * Fr(2) ** mexp == Wn
            assert Fr(int(wq[i])) * Fr(2) ** (mexp + 16) == fold * bf.UQ(Wn / fold, 8)


def test_update_zero_gradient_is_identity(orc):
    master = synth.int_codes(7, (100,), -(2 ** 23) + 1, 2 ** 23 - 1, np.int32)
    m2, wq = orc.weight_update(master, np.zeros(100, np.int8), -5, 0)
    assert np.array_equal(m2, master)
    assert np.array_equal(wq, orc.weight_quant(master))


def test_master_init_eq7(orc):
    w = synth.he_normal(8, (64,), 27)
    m, e = orc.master_init(w, 24)
    assert e == -23
    assert [Fr(int(v)) * Fr(2) ** e for v in m] == [bf.UQ(Fr(float(v)), 24) for v in w]


@pytest.mark.parametrize("k,st,pad", [(2, 2, 0), (3, 2, 1), (3, 1, 1)])
def test_maxpool_fwd_vs_torch(orc, k, st, pad):
    x = synth.int_codes(9, (2, 9, 10, 5))
    y = orc.maxpool_fwd(x, k, st, pad)
    t = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    ref = F.max_pool2d(t, k, st, pad).permute(0, 2, 3, 1).numpy()
    assert np.array_equal(y.astype(np.float64), ref)


def test_maxpool_bwd_ties_and_conservation(orc):
    # window [[5, 5], [1, 5]]: the first maximum in row-major order takes the error
    x = np.array([5, 5, 1, 5], np.int8).reshape(1, 2, 2, 1)
    dy = np.array([9], np.int8).reshape(1, 1, 1, 1)
    dx, e = orc.maxpool_bwd(dy, -3, x, 2, 2, 0)
    assert [Fr(int(v)) * Fr(2) ** e for v in dx.ravel()] == [Fr(9, 8), 0, 0, 0]
    # overlapping windows: routed errors add up exactly, each one lands on a
    # window maximum, and the quantized result is SQ8 of the exact sums (Eq. 16)
    x = synth.int_codes(10, (1, 9, 9, 3))
    dy = synth.int_codes(11, (1, 5, 5, 3))
    raw = orc.maxpool_bwd_raw(dy, x, 3, 2, 1)
    assert int(raw.sum()) == int(dy.astype(np.int64).sum())
    y = orc.maxpool_fwd(x, 3, 2, 1)
    routed = set(zip(*np.nonzero(raw)))
    for n, h, w, c in routed:                   # only window maxima receive errors
        wins = [y[n, p, q, c] for p in range(5) for q in range(5)
                if 2 * p - 1 <= h <= 2 * p + 1 and 2 * q - 1 <= w <= 2 * q + 1]
        assert x[n, h, w, c] in wins
    dx, e = orc.maxpool_bwd(dy, -4, x, 3, 2, 1)
    assert [Fr(int(v)) * Fr(2) ** e for v in dx.ravel()] == \
        bf.SQ([Fr(int(v)) * Fr(2) ** -4 for v in raw.ravel()], 8)
