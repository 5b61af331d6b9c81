"""GPU parity of the merges (residual add, error sums, ReLU mask, concat and
its split, spatial sums) and of the float64 softmax cross-entropy region
against the CPU oracle: codes and exponents bit-exact, the float loss and
gradient within 1e-12 relative."""
import numpy as np
import pytest

from paper_2011_14504_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2011_14504_amd import iseg
    iseg.lib()
    return torch.device("cuda", 0)


def T(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def E(v, dev):
    import torch
    return torch.tensor([int(v)], dtype=torch.int32, device=dev)


def H(t):
    return t.cpu().numpy()


def ev(t):
    return int(t.item())


def _codes(seed, shape, mag=127):
    return synth.rng(seed).integers(-mag, mag + 1, size=shape).astype(np.int8)


# (shape, exps, relu, broadcast-second)
SUM_CASES = [
    ((2, 7, 5, 16), (-7, -6), True, False),        # residual add, vector path
    ((3, 9, 11, 64), (-5, -9), True, False),
    ((2, 4, 6, 20), (-7, -7), False, False),       # C % 16 != 0: scalar path
    ((1, 1, 1, 3), (-3, -12), True, False),        # tiny
    ((2, 8, 8, 32), (-20, -30), False, True),      # error sum with a pooled term
    ((4, 13, 3, 48), (-11, -11), False, False),
    ((2, 5, 6, 32), (-3, -40), True, False),       # gap 37: 64-bit sums
    ((1, 4, 4, 16), (-10, -31), False, False),     # gap 21: just past the int32 path
    ((1, 4, 4, 16), (-10, -30), True, False),      # gap 20: the widest int32 case
]


@pytest.mark.parametrize("case", SUM_CASES, ids=str)
def test_sum_requant(orc, dev, case):
    from paper_2011_14504_amd import iseg
    shape, exps, relu, bc = case
    a = _codes(1, shape)
    b = _codes(2, (shape[0], 1, 1, shape[3]) if bc else shape, 90)
    y, ye = iseg.sum_requant([T(a, dev), T(b, dev)], [E(exps[0], dev), E(exps[1], dev)], relu=relu,
                             bcast=[0, int(bc)])
    rc, re = orc.sum_requant([a, b], list(exps), 8, relu=relu)
    assert np.array_equal(H(y).astype(np.int64), rc) and ev(ye) == re


def test_sum_requant_many_inputs_and_exp_add(orc, dev):
    from paper_2011_14504_amd import iseg
    shape = (2, 6, 6, 32)
    ins = [_codes(10 + i, shape, 20 + 20 * i) for i in range(4)]
    g = _codes(20, (2, 1, 1, 32))
    exps = [-14, -13, -16, -15]
    y, ye = iseg.sum_requant([T(t, dev) for t in ins] + [T(g, dev)],
                             [E(e, dev) for e in exps] + [E(-12, dev)],
                             exp_add=[0, 0, 0, 0, -5], bcast=[0, 0, 0, 0, 1])
    rc, re = orc.sum_requant(ins + [g], exps + [-17], 8)
    assert np.array_equal(H(y).astype(np.int64), rc) and ev(ye) == re


def test_sum_requant_all_zero_and_gap_flag(orc, dev):
    import torch
    from paper_2011_14504_amd import iseg
    z = np.zeros((1, 4, 4, 16), np.int8)
    y, ye = iseg.sum_requant([T(z, dev), T(z, dev)], [E(-9, dev), E(-4, dev)], relu=True)
    assert not H(y).any() and ev(ye) == -9
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    a = _codes(3, (1, 4, 4, 16))
    iseg.sum_requant([T(a, dev), T(a, dev)], [E(0, dev), E(-60, dev)], status=st)
    assert ev(st) & iseg.ISEG_DEV_RANGE


@pytest.mark.parametrize("shape,exps", [((2, 9, 7, 64), (-8, -7)), ((1, 5, 3, 24), (-8, -7)),
                                        ((2, 6, 6, 32), (-2, -36))], ids=str)
def test_relu_mask_bwd(orc, dev, shape, exps):
    from paper_2011_14504_amd import iseg
    a = _codes(30, shape)
    b = _codes(31, shape)
    a[0, 0, :2, :] = 0
    b[0, 0, :2, :] = 0
    dy = _codes(32, shape)
    d = iseg.relu_mask_bwd(T(dy, dev), [T(a, dev), T(b, dev)], [E(exps[0], dev), E(exps[1], dev)])
    assert np.array_equal(H(d), orc.relu_mask_bwd(dy, [a, b], list(exps)))


@pytest.mark.parametrize("shape,exps,mexps", [((2, 9, 7, 64), (-8, -7), (-5, -30)),
                                               ((1, 5, 3, 24), (-8, -11), (-5, -5)),
                                               ((4, 16, 16, 256), (-30, -9), (-7, -3))], ids=str)
def test_sum_requant_relu_mask(orc, dev, shape, exps, mexps):
    """The fused sum + ReLU backward against the oracle's sum then mask."""
    from paper_2011_14504_amd import iseg
    e1, e2 = _codes(33, shape), _codes(34, shape)
    a, b = _codes(35, shape), _codes(36, shape)
    a[0, 0, :2, :] = 0
    b[0, 0, :2, :] = 0
    d, de = iseg.sum_requant_relu_mask([T(e1, dev), T(e2, dev)], [E(exps[0], dev), E(exps[1], dev)],
                                       [T(a, dev), T(b, dev)], [E(mexps[0], dev), E(mexps[1], dev)])
    s, se = orc.sum_requant([e1, e2], list(exps), 8, relu=False)
    assert ev(de) == se
    assert np.array_equal(H(d).astype(np.int64), orc.relu_mask_bwd(s, [a, b], list(mexps)).astype(np.int64))


CAT_CASES = [
    # part widths, exps, spatial of each part (None = full)
    ([256, 256, 256, 256, 256], [-4, -5, -4, -6, -3], [None, None, None, None, (1, 1)]),
    ([16, 32, 48], [-7, -7, -7], [None, None, None]),
    ([5, 11, 3], [-9, -6, -12], [None, (1, 1), None]),            # scalar path
]


@pytest.mark.parametrize("case", CAT_CASES, ids=lambda c: str(c[0]))
def test_concat_requant_and_split(orc, dev, case):
    from paper_2011_14504_amd import iseg
    widths, exps, sp = case
    N, Hh, W = 2, 6, 5
    parts = [_codes(40 + i, (N,) + (s if s else (Hh, W)) + (c,), 30 + 19 * i)
             for i, (c, s) in enumerate(zip(widths, sp))]
    y, ye = iseg.concat_requant([T(p, dev) for p in parts], [E(e, dev) for e in exps])
    rc, re = orc.concat_requant(parts, exps, spatial=(Hh, W))
    assert np.array_equal(H(y).astype(np.int64), rc) and ev(ye) == re
    dy = _codes(50, (N, Hh, W, sum(widths)))
    outs = iseg.concat_split(T(dy, dev), widths, skip=[s is not None for s in sp])
    ref = orc.concat_split(dy, widths)
    for o, r, s in zip(outs, ref, sp):
        if s is None:
            assert np.array_equal(H(o), r)
        else:
            assert o is None


@pytest.mark.parametrize("shape", [(8, 32, 32, 2048), (3, 4, 8, 20), (1, 16, 16, 256), (2, 6, 5, 64),
                                   (1, 3, 7, 9)], ids=str)
def test_gap_fwd_bwd(orc, dev, shape):
    from paper_2011_14504_amd import iseg
    x = _codes(60, shape)
    y, ye = iseg.gap_fwd(T(x, dev), E(-7, dev))
    rc, re = orc.gap_fwd(x, -7)
    assert np.array_equal(H(y).astype(np.int64), rc) and ev(ye) == re
    d = _codes(61, (shape[0], 1, 1, shape[3]))
    g, ge = iseg.gap_bwd(T(d, dev), E(-19, dev), shape[1], shape[2])
    rc, re = orc.gap_bwd(d, -19, shape[1], shape[2])
    assert np.array_equal(H(g).astype(np.int64), rc) and ev(ge) == re


def test_gap_all_zero(orc, dev):
    from paper_2011_14504_amd import iseg
    for shape in ((1, 6, 5, 16), (2, 4, 4, 8)):
        x = np.zeros(shape, np.int8)
        y, ye = iseg.gap_fwd(T(x, dev), E(-7, dev))
        rc, re = orc.gap_fwd(x, -7)
        assert not H(y).any() and ev(ye) == re


@pytest.mark.parametrize("c0,Cc,ldc", [(1024, 256, 1280), (0, 256, 1280), (3, 9, 17)], ids=str)
def test_spatial_sum_bcast_bwd(orc, dev, c0, Cc, ldc):
    from paper_2011_14504_amd import iseg
    dy = _codes(70, (2, 32, 32, ldc))
    y, ye = iseg.spatial_sum(T(dy, dev), E(-18, dev), 1, c0, Cc)
    rc, re = orc.bcast_bwd(dy[..., c0:c0 + Cc], -18)
    assert np.array_equal(H(y).astype(np.int64), rc) and ev(ye) == re


def test_spatial_sum_constant_zero(orc, dev):
    from paper_2011_14504_amd import iseg
    x = np.zeros((2, 4, 4, 8), np.int8)
    y, ye = iseg.spatial_sum(T(x, dev), E(-3, dev), 1)
    assert not H(y).any() and ev(ye) == -3


# (N, h, w, K, H, W, logit exponent)
CE_CASES = [
    (2, 4, 4, 21, 64, 64, -4),        # x16, VOC's class count
    (1, 8, 8, 150, 128, 128, -3),     # x16, ADE20K's class count
    (2, 3, 5, 7, 10, 13, -5),         # non-power-of-two ratios, ragged chunks
    (1, 2, 2, 64, 32, 32, -6),        # K exactly one wave
    (1, 4, 4, 200, 16, 16, -4),       # four classes per lane
]


@pytest.mark.parametrize("case", CE_CASES, ids=str)
def test_softmax_ce(orc, dev, case):
    from paper_2011_14504_amd import iseg
    N, h, w, K, Hh, W, le = case
    logits = _codes(80, (N, h, w, K))
    labels = synth.labels(81, (N, Hh, W), K)
    loss, grad, err, ee = iseg.softmax_ce(T(logits, dev), E(le, dev), T(labels, dev), want_grad=True)
    rl, rg = orc.softmax_ce(logits, le, labels)
    g = H(grad)
    assert abs(float(H(loss)[0]) - rl) <= 1e-12 * abs(rl)
    assert np.max(np.abs(g - rg)) <= 1e-12 * np.max(np.abs(rg))
    rc, re = orc.quantize_f64(rg, 8)
    assert ev(ee) == re
    mism = np.flatnonzero(H(err).astype(np.int64).ravel() != rc.ravel())
    if mism.size:
        # a disagreement is only acceptable within float64 noise of a rounding boundary
        v = rg.ravel()[mism] * 2.0 ** (7 - (re + 7))
        assert np.all(np.abs(np.abs(v - np.floor(v)) - 0.5) < 1e-9), mism
    assert mism.size == 0


def test_softmax_ce_label_range_flag(dev):
    import torch
    from paper_2011_14504_amd import iseg
    logits = _codes(82, (1, 2, 2, 5))
    labels = np.zeros((1, 8, 8), np.uint8)
    labels[0, 3, 3] = 9
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    iseg.softmax_ce(T(logits, dev), E(-4, dev), T(labels, dev), status=st)
    assert ev(st) & iseg.ISEG_DEV_RANGE
