"""Pins of the oracle's quantizers (Eq. 1-6) against hand-worked values, the
exact-rational brute force of the paper's formulas, invariants and the Philox
known-answer vectors."""
import json
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

import bruteforce as bf
from paper_2011_14504_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


def _val(codes, e):
    return [Fr(int(c)) * Fr(2) ** e for c in np.ravel(codes)]


@pytest.mark.parametrize("case", GOLD["uq"], ids=lambda c: c["x"])
def test_uq_hand_examples(orc, case):
    x = float(Fr(case["x"]))
    assert orc.uq_code(x, case["k"]) == case["code"]
    # the same code through the tensor quantizer in UQ mode
    codes, e = orc.quantize_f32(np.array([x], np.float32), case["k"], "uq")
    assert int(codes[0]) == case["code"] and e == 1 - case["k"]


@pytest.mark.parametrize("case", GOLD["sq"], ids=lambda c: ",".join(c["x"]))
def test_sq_hand_examples(orc, case):
    x = np.array([float(Fr(v)) for v in case["x"]], np.float32)
    codes, e = orc.quantize_f32(x, case["k"], "sq")
    assert list(codes) == case["codes"] and e == case["exp"]


def test_delta8_matches_paper_step():
    # Sec. 3.1.2 quotes Delta(k_E = 8) ~ 0.008
    assert float(bf.delta(8)) == 0.0078125
    assert abs(float(bf.delta(8)) - 0.008) < 3e-4


def test_uq_exact_floor_edge(orc):
    # float32 0.49999997 (just below 1/2): x/Delta + 1/2 must floor to 0, not 1
    v = np.float32(0.49999997)
    assert float(v) < 0.5
    x = float(v) / 128.0
    assert orc.uq_code(x, 8) == 0
    assert orc.uq_code(-x, 8) == 0
    # exact midpoint rounds up
    assert orc.uq_code(0.5 / 128.0, 8) == 1
    assert orc.uq_code(-0.5 / 128.0, 8) == 0


def test_quantize_f32_vs_bruteforce(orc):
    for seed in range(20):
        x = synth.uniform_f32(seed, (37,), -3.0, 3.0) * np.float32(2.0 ** (seed % 7 - 3))
        for k in (4, 8, 16):
            codes, e = orc.quantize_f32(x, k, "sq")
            ref = bf.SQ([Fr(float(v)) for v in x], k)
            assert _val(codes, e) == ref
            codes, e = orc.quantize_f32(x, k, "uq")
            assert _val(codes, e) == [bf.UQ(Fr(float(v)), k) for v in x]


@pytest.mark.parametrize("k", [4, 8, 16])
def test_requant_sq_vs_bruteforce(orc, k):
    for seed in range(30):
        rng = synth.rng(1000 + seed)
        mag = int(rng.integers(0, 40))
        a = rng.integers(-(2 ** mag), 2 ** mag + 1, size=23, dtype=np.int64)
        if seed % 5 == 0:
            a[3] = 2 ** mag          # maximum exactly a power of two
        s = int(rng.integers(-30, 10))
        codes, e = orc.requant(a, s, k)
        assert _val(codes, e) == bf.SQ([Fr(int(v)) * Fr(2) ** s for v in a], k)
        lim = 2 ** (k - 1) - 1
        assert codes.max() <= lim and codes.min() >= -lim


def test_requant_zero_tensor(orc):
    codes, e = orc.requant(np.zeros(5, np.int64), -9, 8)
    assert not codes.any() and e == -9


def test_requant_identity_on_8bit_grid(orc):
    # a tensor already holding 8-bit codes at a power-of-two exponent keeps
    # its values exactly under SQ8 (the strictly-greater power-of-two scale)
    for seed in range(50):
        rng = synth.rng(2000 + seed)
        lim = int(rng.integers(1, 128))
        a = rng.integers(-lim, lim + 1, size=64, dtype=np.int64)
        a[0] = lim
        s = int(rng.integers(-25, 5))
        codes, e = orc.requant(a, s, 8)
        assert _val(codes, e) == _val(a, s)


def test_requant_idempotent(orc):
    for seed in range(30):
        rng = synth.rng(3000 + seed)
        a = rng.integers(-(2 ** 30), 2 ** 30, size=50, dtype=np.int64)
        c1, e1 = orc.requant(a, -14, 8)
        c2, e2 = orc.requant(c1, e1, 8)
        assert np.array_equal(c1, c2) and e1 == e2


def test_requant_monotone(orc):
    a = np.arange(-5000, 5001, 7, dtype=np.int64)
    codes, _ = orc.requant(a, 0, 8)
    assert np.all(np.diff(codes) >= 0)


def test_philox_known_answers(orc):
    # Random123 known-answer vectors for Philox4x32-10
    kat = [
        ([0, 0, 0, 0], [0, 0], [0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8]),
        ([0xffffffff] * 4, [0xffffffff] * 2, [0x408f276d, 0x41c83b0e, 0xa20bc7c6, 0x6d5451fd]),
        ([0x243f6a88, 0x85a308d3, 0x13198a2e, 0x03707344], [0xa4093822, 0x299f31d0],
         [0xd16cfe09, 0x94fdcceb, 0x5001e420, 0x24126ea1]),
    ]
    for ctr, key, out in kat:
        assert list(orc.philox4x32_10(ctr, key)) == out


def test_rq_support_and_determinism(orc):
    rng = synth.rng(77)
    a = rng.integers(-(2 ** 20), 2 ** 20, size=200, dtype=np.int64)
    codes, e = orc.requant(a, -3, 8, stochastic=True, seed=5, tensor_id=2, step=1)
    S = bf.pow2_scale([Fr(int(v)) for v in a]) * Fr(2) ** -3
    for c, v in zip(codes, a):
        support = bf.RQ_probs(Fr(int(v)) * Fr(2) ** -3, S, 8)
        assert Fr(int(c)) * Fr(2) ** e in support
    # same key -> same codes; different step -> different codes somewhere
    c2, _ = orc.requant(a, -3, 8, stochastic=True, seed=5, tensor_id=2, step=1)
    c3, _ = orc.requant(a, -3, 8, stochastic=True, seed=5, tensor_id=2, step=2)
    assert np.array_equal(codes, c2) and not np.array_equal(codes, c3)
    # values already on the 8-bit grid are never moved
    small = rng.integers(-127, 128, size=100, dtype=np.int64)
    c4, e4 = orc.requant(small, 0, 8, stochastic=True, seed=1)
    assert _val(c4, e4) == _val(small, 0)


def test_rq_unbiased(orc):
    # E[Round(x)] = x (Sec. 3.1.3): one value repeated at many indices
    n = 200000
    a = np.full(n, 1000, dtype=np.int64)
    a[0] = 4095                      # sets the scale: bitlen 12 -> r = 5
    codes, e = orc.requant(a, 0, 8, stochastic=True, seed=123, tensor_id=9)
    vals = codes[1:].astype(np.float64) * 2.0 ** e
    p = 1000 / 32 - np.floor(1000 / 32)
    sd = 32 * np.sqrt(p * (1 - p) / (n - 1))
    assert abs(vals.mean() - 1000) < 5 * sd


def test_gq1_gq2_same_codes(orc):
    rng = synth.rng(88)
    a = rng.integers(-(2 ** 25), 2 ** 25, size=300, dtype=np.int64)
    c1, e1 = orc.requant(a, -30, 8, stochastic=True, keep_scale=True, seed=3)
    c2, e2 = orc.requant(a, -30, 8, stochastic=True, keep_scale=False, seed=3)
    assert np.array_equal(c1, c2)
    assert e2 == -7 and e1 == -30 + (int(np.abs(a).max()).bit_length() - 7)
