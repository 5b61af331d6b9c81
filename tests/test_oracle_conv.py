"""Pins of the oracle's integer convolutions: float64 library convolutions
(exact on integer data), a literal 7-loop, the adjoint identity and the
dilation-as-zero-inserted-kernel identity."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import bruteforce as bf
from paper_2011_14504_amd import synth

# (N, H, W, C, K, R, S, stride, pad, dil)
SHAPES = [
    (1, 7, 7, 3, 4, 3, 3, 1, 1, 1),
    (2, 9, 8, 5, 3, 3, 3, 2, 1, 1),
    (1, 11, 11, 4, 2, 3, 3, 1, 2, 2),
    (1, 13, 12, 2, 3, 3, 3, 1, 3, 3),
    (2, 6, 6, 3, 5, 1, 1, 1, 0, 1),
    (1, 10, 10, 3, 2, 7, 7, 2, 3, 1),
    (1, 8, 9, 6, 4, 3, 3, 2, 0, 2),
]


def _geom(s):
    N, H, W, C, K, R, S, st, pad, d = s
    return (N, H, W, C, K, R, S, st, st, pad, pad, d, d)


def _inputs(s, seed):
    N, H, W, C, K, R, S, st, pad, d = s
    x = synth.int_codes(seed, (N, H, W, C))
    w = synth.int_codes(seed + 1, (K, R, S, C))
    return x, w


def _t(a):  # NHWC/KRSC int8 -> NCHW/KCRS float64
    return torch.from_numpy(a.astype(np.float64)).permute(0, 3, 1, 2).contiguous()


@pytest.mark.parametrize("s", SHAPES)
def test_conv_fwd_vs_torch(orc, s):
    x, w = _inputs(s, 11)
    g = _geom(s)
    acc = orc.conv_fwd_raw(x, w, g)
    ref = F.conv2d(_t(x), _t(w), stride=s[7], padding=s[8], dilation=s[9])
    assert np.array_equal(acc, ref.permute(0, 2, 3, 1).numpy().astype(np.int64))


@pytest.mark.parametrize("s", SHAPES)
def test_conv_bwd_vs_torch(orc, s):
    x, w = _inputs(s, 21)
    g = _geom(s)
    P, Q = orc.conv_out_hw(g)
    dy = synth.int_codes(99, (s[0], P, Q, s[4]))
    dx = orc.conv_bwd_data_raw(dy, w, g)
    dw = orc.conv_bwd_weight_raw(dy, x, g)
    ref_dx = torch.nn.grad.conv2d_input(_t(x).shape, _t(w), _t(dy), stride=s[7],
                                        padding=s[8], dilation=s[9])
    ref_dw = torch.nn.grad.conv2d_weight(_t(x), _t(w).shape, _t(dy), stride=s[7],
                                         padding=s[8], dilation=s[9])
    assert np.array_equal(dx, ref_dx.permute(0, 2, 3, 1).numpy().astype(np.int64))
    assert np.array_equal(dw, ref_dw.permute(0, 2, 3, 1).numpy().astype(np.int64))


def test_conv_fwd_vs_literal_loops(orc):
    s = (1, 5, 6, 2, 3, 3, 3, 2, 1, 2)
    x, w = _inputs(s, 5)
    acc = orc.conv_fwd_raw(x, w, _geom(s))
    ref = bf.conv2d(x.astype(int).tolist(), w.astype(int).tolist(), s[7], s[8], s[9])
    assert acc.tolist() == ref


@pytest.mark.parametrize("s", SHAPES)
def test_adjoint_identity(orc, s):
    # <conv(x, w), e> = <x, bwd_data(e, w)> = <w, bwd_weight(e, x)>, exactly
    x, w = _inputs(s, 31)
    g = _geom(s)
    P, Q = orc.conv_out_hw(g)
    e = synth.int_codes(32, (s[0], P, Q, s[4]))
    y = orc.conv_fwd_raw(x, w, g)
    a = int((y * e.astype(np.int64)).sum())
    b = int((x.astype(np.int64) * orc.conv_bwd_data_raw(e, w, g)).sum())
    c = int((w.astype(np.int64) * orc.conv_bwd_weight_raw(e, x, g)).sum())
    assert a == b == c


def test_dilation_is_zero_inserted_kernel(orc):
    N, H, W, C, K, R, d = 1, 15, 14, 3, 2, 3, 3
    x = synth.int_codes(41, (N, H, W, C))
    w = synth.int_codes(42, (K, R, R, C))
    Rd = d * (R - 1) + 1
    wz = np.zeros((K, Rd, Rd, C), np.int8)
    wz[:, ::d, ::d, :] = w
    a = orc.conv_fwd_raw(x, w, (N, H, W, C, K, R, R, 1, 1, 3, 3, d, d))
    b = orc.conv_fwd_raw(x, wz, (N, H, W, C, K, Rd, Rd, 1, 1, 3, 3, 1, 1))
    assert np.array_equal(a, b)


def test_conv_requant_composition(orc):
    # conv then SQ8 equals the brute-force SQ of the exact sums' values
    from fractions import Fraction as Fr
    s = SHAPES[0]
    x, w = _inputs(s, 51)
    codes, e = orc.conv_fwd(x, -7, w, -7, _geom(s))
    acc = orc.conv_fwd_raw(x, w, _geom(s))
    ref = bf.SQ([Fr(int(v)) * Fr(2) ** -14 for v in acc.ravel()], 8)
    assert [Fr(int(c)) * Fr(2) ** e for c in codes.ravel()] == ref


@pytest.mark.parametrize("geom", [(2, 19, 17, 32, 48, 3, 3, 2, 2, 2, 2, 2, 2),
                                  (1, 23, 21, 24, 40, 3, 3, 1, 1, 6, 6, 6, 6),
                                  (3, 16, 16, 64, 32, 1, 1, 2, 2, 0, 0, 1, 1)])
def test_library_conv_path_equals_loops(orc, geom):
    """The library path the oracle takes for large convolutions gives the
    same exact sums as its plain loops (forced on medium shapes here)."""
    rng = synth.rng(977)
    N, H, W, Cc, K, R, S = geom[:7]
    P, Q = orc.conv_out_hw(geom)
    x = rng.integers(-127, 128, (N, H, W, Cc)).astype(np.int8)
    w = rng.integers(-127, 128, (K, R, S, Cc)).astype(np.int8)
    dy = rng.integers(-127, 128, (N, P, Q, K)).astype(np.int8)
    saved = orc.LIBRARY_CONV_MACS
    try:
        orc.LIBRARY_CONV_MACS = 1 << 62
        loops = (orc.conv_fwd_raw(x, w, geom), orc.conv_bwd_data_raw(dy, w, geom),
                 orc.conv_bwd_weight_raw(dy, x, geom))
        orc.LIBRARY_CONV_MACS = 0
        lib_ = (orc.conv_fwd_raw(x, w, geom), orc.conv_bwd_data_raw(dy, w, geom),
                orc.conv_bwd_weight_raw(dy, x, geom))
    finally:
        orc.LIBRARY_CONV_MACS = saved
    for a, b in zip(loops, lib_):
        assert a.dtype == b.dtype == np.int64 and np.array_equal(a, b)
