"""Pins of the oracle's merges (residual add, error sums, concatenation,
global pooling and its broadcast) and of the float64 softmax cross-entropy
region, against hand-worked values, exact-rational brute force of the
definitions, adjoint identities and independent library routines (torch's
interpolate / cross_entropy / autograd in float64)."""
import json
import math
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

import bruteforce as bf
from paper_2011_14504_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


def _vals(codes, e):
    return [Fr(int(c)) * Fr(2) ** int(e) for c in np.ravel(codes)]


def _brute_sq(values, k=8):
    return bf.SQ(values, k)


# ---------------------------------------------------------------------------
# merges
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", GOLD["merge"], ids=lambda c: c["about"][:30])
def test_merge_hand_examples(orc, case):
    codes, e = orc.sum_requant([np.array(case["a"], np.int8), np.array(case["b"], np.int8)],
                               [case["a_exp"], case["b_exp"]], 8, relu=bool(case["relu"]))
    assert list(codes) == case["codes"] and e == case["exp"]


@pytest.mark.parametrize("seed", range(40))
def test_sum_requant_vs_brute_force(orc, seed):
    r = synth.rng(9000 + seed)
    n_in = int(r.integers(2, 6))
    shape = (2, 3, 2, 4)
    exps = [int(v) for v in r.integers(-30, -2, size=n_in)]
    mags = [int(v) for v in r.integers(1, 128, size=n_in)]
    ts = [r.integers(-m, m + 1, size=shape).astype(np.int8) for m in mags]
    relu = bool(seed % 2)
    codes, e = orc.sum_requant(ts, exps, 8, relu=relu)
    exact = [sum(Fr(int(t.ravel()[i])) * Fr(2) ** x for t, x in zip(ts, exps))
             for i in range(ts[0].size)]
    if relu:
        exact = [max(v, 0) for v in exact]
    assert _vals(codes, e) == _brute_sq(exact)
    assert np.abs(codes).max() <= 127


def test_sum_requant_broadcast_term(orc):
    # a [N,1,1,C] term (the backward of global pooling) adds to every position
    r = synth.rng(4)
    a = r.integers(-127, 128, size=(2, 3, 4, 5)).astype(np.int8)
    g = r.integers(-127, 128, size=(2, 1, 1, 5)).astype(np.int8)
    codes, e = orc.sum_requant([a, g], [-9, -13], 8)
    full = np.broadcast_to(g, a.shape)
    exact = [Fr(int(x)) * Fr(2) ** -9 + Fr(int(y)) * Fr(2) ** -13
             for x, y in zip(a.ravel(), full.ravel())]
    assert _vals(codes, e) == _brute_sq(exact)


def test_sum_with_zero_is_identity_on_values(orc):
    # adding an all-zero tensor changes no value of an 8-bit tensor
    a = synth.int_codes(5, (3, 7, 5, 8))
    z = np.zeros_like(a)
    codes, e = orc.sum_requant([a, z], [-5, -40], 8)
    assert _vals(codes, e) == _vals(a, -5)


def test_merge_gap_limit(orc):
    a = synth.int_codes(6, (4,))
    with pytest.raises(orc.OracleError):
        orc.sum_requant([a, a], [0, -(orc.MAX_GAP + 1)], 8)


def test_relu_mask_bwd(orc):
    r = synth.rng(17)
    a = r.integers(-127, 128, size=(2, 5, 5, 8)).astype(np.int8)
    b = r.integers(-127, 128, size=(2, 5, 5, 8)).astype(np.int8)
    a[0, 0, 0, :] = 0                       # exact zero sums: sgn 0, masked
    b[0, 0, 0, :] = 0
    b[1, 1, 1, 0], a[1, 1, 1, 0] = 2, -4    # 2*2^-8 - 4*2^-9 = 0 exactly
    dy = r.integers(-127, 128, size=a.shape).astype(np.int8)
    d = orc.relu_mask_bwd(dy, [a, b], [-9, -8])
    for i in range(a.size):
        s = Fr(int(a.ravel()[i]), 2 ** 9) + Fr(int(b.ravel()[i]), 2 ** 8)
        assert int(d.ravel()[i]) == (int(dy.ravel()[i]) if s > 0 else 0)
    assert d.ravel()[np.ravel_multi_index((1, 1, 1, 0), a.shape)] == 0


@pytest.mark.parametrize("case", GOLD["concat"], ids=lambda c: c["about"][:30])
def test_concat_hand_examples(orc, case):
    parts = [np.array(p, np.int8).reshape(1, 1, 1, -1) for p in case["parts"]]
    codes, e = orc.concat_requant(parts, case["exps"])
    assert list(np.ravel(codes)) == case["codes"] and e == case["exp"]


def test_concat_vs_brute_force_with_broadcast_part(orc):
    r = synth.rng(31)
    a = r.integers(-127, 128, size=(2, 4, 3, 5)).astype(np.int8)
    b = r.integers(-60, 61, size=(2, 4, 3, 3)).astype(np.int8)
    g = r.integers(-127, 128, size=(2, 1, 1, 2)).astype(np.int8)
    exps = [-8, -6, -11]
    codes, e = orc.concat_requant([a, b, g], exps, spatial=(4, 3))
    full = np.concatenate([a.astype(np.int64), b, np.broadcast_to(g, (2, 4, 3, 2))], axis=-1)
    ex = np.concatenate([np.full(a.shape, exps[0]), np.full(b.shape, exps[1]),
                         np.full((2, 4, 3, 2), exps[2])], axis=-1)
    exact = [Fr(int(v)) * Fr(2) ** int(x) for v, x in zip(full.ravel(), ex.ravel())]
    assert codes.shape == (2, 4, 3, 10)
    assert _vals(codes, e) == _brute_sq(exact)


def test_concat_equal_exponents_is_a_copy(orc):
    a = synth.int_codes(32, (1, 3, 3, 4))
    b = synth.int_codes(33, (1, 3, 3, 6))
    codes, e = orc.concat_requant([a, b], [-7, -7])
    assert e == -7 and np.array_equal(codes, np.concatenate([a, b], -1))
    parts = orc.concat_split(codes.astype(np.int8), [4, 6])
    assert np.array_equal(parts[0], a) and np.array_equal(parts[1], b)


@pytest.mark.parametrize("case", GOLD["gap"], ids=lambda c: c["about"][:30])
def test_gap_hand_examples(orc, case):
    x = np.array(case["x"], np.int8).reshape(1, case["H"], case["W"], 1)
    codes, e = orc.gap_fwd(x, case["x_exp"])
    assert int(codes.ravel()[0]) == case["code"] and e == case["exp"]


@pytest.mark.parametrize("shape", [(3, 8, 4, 6), (2, 6, 5, 3), (1, 3, 3, 4)], ids=str)
def test_gap_vs_torch_mean_and_brute_force(orc, shape):
    import torch
    x = synth.int_codes(40, shape)
    codes, e = orc.gap_fwd(x, -7)
    HW = shape[1] * shape[2]
    mean = torch.from_numpy(x.astype(np.float64)).mean(dim=(1, 2), keepdim=True)
    # the exact rational mean; torch's float64 mean agrees with it to rounding
    exact = [Fr(int(v), HW) * Fr(2) ** -7 for v in x.astype(np.int64).sum(axis=(1, 2)).ravel()]
    assert np.allclose([float(v) for v in exact], mean.numpy().ravel() * 2.0 ** -7, rtol=1e-15)
    assert codes.shape == (shape[0], 1, 1, shape[3])
    assert _vals(codes, e) == _brute_sq(exact)


def test_gap_all_zero(orc):
    codes, e = orc.gap_fwd(np.zeros((1, 6, 5, 2), np.int8), -7)
    assert not codes.any() and e == -7 - 5          # ceil(log2 30) = 5
    codes, e = orc.gap_fwd(np.zeros((1, 4, 8, 2), np.int8), -7)
    assert not codes.any() and e == -12


@pytest.mark.parametrize("hw", [(4, 8), (6, 5)], ids=str)
def test_gap_backward(orc, hw):
    # <mean(x), d> = <x, bcast(d / HW)>: the backward's value at every position
    # is d / HW, quantized by SQ8; for a power-of-two HW exactly (values kept)
    H, W = hw
    d = synth.int_codes(43, (2, 1, 1, 3))
    codes, e = orc.gap_bwd(d, -9, H, W)
    exact = [Fr(int(v), H * W) * Fr(2) ** -9 for v in d.ravel()]
    assert _vals(codes, e) == _brute_sq(exact)
    if (H * W) & (H * W - 1) == 0:
        assert _vals(codes, e) == exact
    x = synth.int_codes(42, (2, H, W, 3))
    lhs = sum(Fr(int(s), H * W) * Fr(int(v)) for s, v in
              zip(x.astype(np.int64).sum(axis=(1, 2)).ravel(), d.ravel()))
    rhs = sum(Fr(int(a)) * Fr(int(b), H * W) for a, b in
              zip(x.ravel(), np.broadcast_to(d, x.shape).ravel()))
    assert lhs == rhs


def test_bcast_backward_is_adjoint_of_broadcast(orc):
    # <bcast(u), v> = <u, sum_hw(v)> exactly, then Q_E on the sums
    u = synth.int_codes(44, (2, 1, 1, 5))
    v = synth.int_codes(45, (2, 6, 7, 5))
    codes, e = orc.bcast_bwd(v, -20)
    sums = v.astype(np.int64).sum(axis=(1, 2), keepdims=True)
    assert int((np.broadcast_to(u, v.shape).astype(np.int64) * v).sum()) == int((u * sums).sum())
    assert _vals(codes, e) == _brute_sq([Fr(int(s)) * Fr(2) ** -20 for s in sums.ravel()])


# ---------------------------------------------------------------------------
# float64 quantizer used at the float -> int crossing
# ---------------------------------------------------------------------------
def test_quantize_f64_exact_decisions(orc):
    below_half = math.nextafter(0.5, 0.0)          # 0.49999999999999994
    # scale fixed by the largest value (1.5 -> S = 2): v 2^6 for the others
    x = np.array([1.5, below_half / 64, 0.5 / 64, -0.5 / 64, -below_half / 64, 0.0])
    codes, e = orc.quantize_f64(x, 8)
    assert e == -6
    assert list(codes) == [96, 0, 1, 0, 0, 0]


@pytest.mark.parametrize("seed", range(10))
def test_quantize_f64_vs_brute_force(orc, seed):
    x = synth.rng(500 + seed).standard_normal(50) * 10.0 ** (seed - 5)
    codes, e = orc.quantize_f64(x, 8)
    assert _vals(codes, e) == _brute_sq([Fr(float(v)) for v in x])


# ---------------------------------------------------------------------------
# softmax cross-entropy region
# ---------------------------------------------------------------------------
def test_bilinear_matrix_properties(orc):
    A = orc.bilinear_matrix(32, 512)
    assert np.allclose(A.sum(axis=1), 1.0, rtol=0, atol=0)
    assert np.all(A * 32 == np.round(A * 32))          # weights are multiples of 1/32
    assert np.array_equal(orc.bilinear_matrix(7, 7), np.eye(7))


def test_softmax_ce_vs_torch_float64(orc):
    import torch
    import torch.nn.functional as F
    logits = synth.int_codes(60, (2, 4, 3, 11))
    labels = synth.labels(61, (2, 64, 48), 11)
    loss, grad = orc.softmax_ce(logits, -4, labels)
    x = torch.from_numpy(logits.astype(np.float64) * 2.0 ** -4).permute(0, 3, 1, 2)
    x.requires_grad_(True)
    up = F.interpolate(x, size=(64, 48), mode="bilinear", align_corners=False)
    ref = F.cross_entropy(up, torch.from_numpy(labels.astype(np.int64)))
    ref.backward()
    g = x.grad.permute(0, 2, 3, 1).numpy()
    assert abs(loss - ref.item()) <= 1e-13 * abs(ref.item())
    assert np.max(np.abs(grad - g)) <= 1e-13 * np.max(np.abs(g))


@pytest.mark.parametrize("case", GOLD["softmax_ce"], ids=lambda c: c["about"][:30])
def test_softmax_ce_equal_logits(orc, case):
    K = case["K"]
    logits = np.full((1, 2, 2, K), 17, np.int8)
    labels = synth.labels(62, (1, 32, 32), K)
    loss, grad = orc.softmax_ce(logits, -3, labels)
    assert abs(loss - float(case["loss"])) < 1e-14
    # per class, the gradient mass equals the upsampled gradient's: the
    # interpolation weights of each output pixel sum to one
    counts = np.bincount(labels.ravel(), minlength=K)
    P = labels.size
    mass = grad.sum(axis=(0, 1, 2))
    assert np.allclose(mass, (P / K - counts) / P, rtol=0, atol=1e-15)


def test_softmax_ce_gradient_sums_to_zero_over_classes(orc):
    logits = synth.int_codes(63, (1, 4, 4, 21))
    labels = synth.labels(64, (1, 64, 64), 21)
    _, grad = orc.softmax_ce(logits, -5, labels)
    assert np.max(np.abs(grad.sum(axis=-1))) < 1e-17


def test_mse_onehot_loss_and_error(orc):
    """The MSE loss against one-hot labels: the loss equals torch's float64
    mse_loss of the same values, its gradient torch's autograd, and the E1
    codes are SQ8 of the exact gradient 2 (y - t) / D (Fractions)."""
    import torch
    import bruteforce as bf
    from fractions import Fraction as Fr
    for (N, H, W, K, e) in ((1, 3, 4, 5, -3), (2, 5, 3, 7, 1), (1, 2, 2, 3, -9)):
        y = synth.int_codes(500 + K, (N, H, W, K))
        lab = synth.labels(600 + K, (N, H, W), K)
        loss, codes, ce = orc.mse_onehot(y, e, lab)
        yt = torch.tensor(y.astype(np.float64) * 2.0 ** e, requires_grad=True)
        t = torch.nn.functional.one_hot(torch.from_numpy(lab.astype(np.int64)), K).double()
        ref = torch.nn.functional.mse_loss(yt, t)
        ref.backward()
        assert abs(loss - ref.item()) <= 1e-12 * ref.item()
        D = y.size
        exact = [(Fr(int(v)) * Fr(2) ** e - int(k == l)) * Fr(2, D)
                 for v, k, l in zip(y.ravel(), np.tile(np.arange(K), N * H * W), np.repeat(lab.ravel(), K))]
        assert np.allclose([float(v) for v in exact], yt.grad.numpy().ravel(), rtol=1e-12, atol=0)
        q = bf.SQ(exact, 8)
        assert [Fr(int(c)) * Fr(2) ** ce for c in codes.ravel()] == q
