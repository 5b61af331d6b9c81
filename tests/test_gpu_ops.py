"""GPU parity: every libiseg entry point against the CPU oracle, bit-exact on
codes and exponents, on seeded inputs that span several tiles and ragged
tails, plus the degenerate cases (all-zero tensors, a single element, padding
-only taps, constant BN channels)."""
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


# ---------------------------------------------------------------------------
# quantizers
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n", [1, 17, 4096 + 5, 300001])
@pytest.mark.parametrize("bits,mode", [(8, "sq"), (16, "sq"), (8, "uq"), (24, "uq")])
def test_quantize_f32(orc, dev, n, bits, mode):
    from paper_2011_14504_amd import iseg
    x = synth.uniform_f32(n + bits, (n,), -3.0, 3.0) * np.float32(2.0 ** (n % 5 - 2))
    if n > 4:
        x[3] = np.float32(0.5) / np.float32(2 ** (bits - 1))      # an exact tie
        x[4] = -x[3]
    codes, e = iseg.quantize(T(x, dev), bits, iseg.ISEG_Q_SQ if mode == "sq" else iseg.ISEG_Q_UQ)
    rc, re = orc.quantize_f32(x, bits, mode)
    assert np.array_equal(H(codes).astype(np.int64), rc) and ev(e) == re


def test_quantize_zero_tensor(orc, dev):
    from paper_2011_14504_amd import iseg
    x = np.zeros(1000, np.float32)
    codes, e = iseg.quantize(T(x, dev), 8)
    assert not H(codes).any() and ev(e) == -7


@pytest.mark.parametrize("dtype", [np.int32, np.int64])
@pytest.mark.parametrize("n", [1, 15, 16, 1000003])
@pytest.mark.parametrize("stochastic,keep", [(0, 1), (1, 1), (1, 0)])
def test_requant(orc, dev, dtype, n, stochastic, keep):
    from paper_2011_14504_amd import iseg
    mag = 30 if dtype == np.int32 else 50
    a = synth.rng(n + mag).integers(-(2 ** mag), 2 ** mag, size=n, dtype=np.int64).astype(dtype)
    codes, e = iseg.requant(T(a, dev), E(-11, dev), 8, stochastic=stochastic, keep_scale=keep,
                            seed=77, tensor_id=5, step=3)
    rc, re = orc.requant(a, -11, 8, stochastic=bool(stochastic), keep_scale=bool(keep), seed=77,
                         tensor_id=5, step=3)
    assert np.array_equal(H(codes).astype(np.int64), rc) and ev(e) == re


def test_requant_small_and_zero(orc, dev):
    from paper_2011_14504_amd import iseg
    for a in (np.zeros(37, np.int32), synth.int_codes(3, (999,), -20, 20, np.int32)):
        codes, e = iseg.requant(T(a, dev), E(-4, dev), 8)
        rc, re = orc.requant(a, -4, 8)
        assert np.array_equal(H(codes).astype(np.int64), rc) and ev(e) == re


# ---------------------------------------------------------------------------
# convolutions
# ---------------------------------------------------------------------------
# (N, H, W, C, K, R, stride, pad, dil)
CONV_SHAPES = [
    (1, 32, 32, 16, 16, 3, 1, 1, 1),      # single-conv workload
    (2, 23, 19, 3, 64, 3, 1, 1, 1),       # C = 3 stem, ragged
    (1, 37, 29, 64, 64, 3, 1, 1, 1),
    (2, 17, 18, 64, 128, 3, 2, 1, 1),     # stride 2
    (1, 20, 21, 32, 48, 3, 1, 2, 2),      # dilation 2
    (1, 26, 26, 16, 24, 3, 1, 6, 6),      # atrous, many padding-only taps
    (2, 14, 15, 64, 256, 1, 1, 0, 1),     # 1x1
    (1, 30, 30, 3, 64, 7, 2, 3, 1),       # 7x7/2 stem
    (1, 9, 11, 128, 130, 3, 1, 1, 1),     # K not a multiple of the tile
    (1, 5, 5, 20, 21, 1, 1, 0, 1),        # C % 16 != 0, K = 21
    (1, 21, 19, 64, 64, 3, 1, 2, 2),      # dilation 2 on the 64-channel paths
    (4, 9, 7, 64, 128, 3, 1, 1, 1),       # narrow rows: pixel runs wrap rows and images
    # direct-to-LDS implicit GEMM: two-pass codes for reductions <= 256
    # (1, 2, 3 steps of 64), int16 staging above (odd and even step counts)
    (1, 13, 11, 128, 64, 1, 1, 0, 1),
    (1, 12, 10, 192, 128, 1, 1, 0, 1),
    (2, 9, 10, 320, 64, 1, 1, 0, 1),
    (1, 18, 17, 128, 128, 3, 1, 6, 6),    # atrous 6: 18 steps, padding-only taps
    (1, 11, 13, 64, 128, 3, 1, 3, 3),     # dilation 3: 9 steps
    # 1x1 with a class count as K: backward-data pads K to a multiple of 64
    (2, 16, 16, 256, 150, 1, 1, 0, 1),
    (1, 9, 7, 128, 100, 1, 1, 0, 1),
    # strided 1x1 (projection shortcuts): backward-data on the output grid,
    # zeros interleaved (even and odd input sizes, stride 3)
    (2, 10, 12, 32, 64, 1, 2, 0, 1),
    (1, 9, 7, 64, 128, 1, 2, 0, 1),
    (1, 11, 10, 16, 32, 1, 3, 0, 1),
] + [
    # strided backward-data with few dy channels (K): the phase path (FCN's
    # upsampling adjoints at 21 classes among them)
    (1, 32, 32, 21, 21, 4, 2, 1, 1),
    (1, 24, 40, 21, 21, 16, 8, 4, 1),
    (2, 13, 11, 24, 10, 3, 2, 1, 1),
    (1, 9, 9, 40, 20, 1, 2, 0, 1),        # 1x1 stride 2: half the phases get no tap
    (1, 15, 17, 8, 33, 5, 3, 2, 1),
    (1, 10, 12, 9, 64, 3, 2, 1, 1),
]
PHASE_SHAPES = CONV_SHAPES[-6:]


def _geom(s):
    N, Hh, W, Cc, K, R, st, pad, d = s
    return (N, Hh, W, Cc, K, R, R, st, st, pad, pad, d, d)


@pytest.mark.parametrize("s", CONV_SHAPES, ids=str)
def test_conv_fwd(orc, dev, s):
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    x = synth.int_codes(11, (N, Hh, W, Cc))
    w = synth.int_codes(12, (K, R, R, Cc))
    raw, re = iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), st, pad, d,
                            out_mode=iseg.ISEG_OUT_RAW)
    ref = orc.conv_fwd_raw(x, w, _geom(s))
    assert np.array_equal(H(raw).astype(np.int64), ref) and ev(re) == -14
    y, ye = iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), st, pad, d)
    rc, rce = orc.requant(ref, -14, 8)
    assert np.array_equal(H(y).astype(np.int64), rc) and ev(ye) == rce


@pytest.mark.parametrize("s", CONV_SHAPES, ids=str)
def test_conv_bwd_data(orc, dev, s):
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    P, Q = orc.conv_out_hw(_geom(s))
    dy = synth.int_codes(21, (N, P, Q, K))
    w = synth.int_codes(22, (K, R, R, Cc))
    raw, re = iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc),
                                 st, pad, d, out_mode=iseg.ISEG_OUT_RAW)
    ref = orc.conv_bwd_data_raw(dy, w, _geom(s))
    assert np.array_equal(H(raw).astype(np.int64), ref) and ev(re) == -27
    dx, dxe = iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc),
                                 st, pad, d)
    rc, rce = orc.requant(ref, -27, 8)
    assert np.array_equal(H(dx).astype(np.int64), rc) and ev(dxe) == rce


@pytest.mark.parametrize("s", PHASE_SHAPES, ids=str)
def test_conv_bwd_data_phase_path(dev, s):
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    P = (Hh + 2 * pad - R) // st + 1
    Q = (W + 2 * pad - R) // st + 1
    dy = synth.int_codes(23, (N, P, Q, K))
    w = synth.int_codes(24, (K, R, R, Cc))
    iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc), st, pad, d)
    assert iseg.iseg_conv_last_plan() == "phase"
    assert iseg.wt_kind((N, Hh, W, Cc), w.shape, st, pad, d) == iseg.ISEG_WT_NONE


def _wt_layout(w, kind):
    """[K, R, S, C] -> [C, R*S, K] (taps reversed for the flipped kind): a plain
    permutation of the weight codes, the layout backward-data reads."""
    K, R, S, Cc = w.shape
    t = np.transpose(w.reshape(K, R * S, Cc), (2, 1, 0))
    return np.ascontiguousarray(t[:, ::-1, :] if kind == 2 else t)


@pytest.mark.parametrize("s", CONV_SHAPES, ids=str)
def test_conv_bwd_data_pretransposed(orc, dev, s):
    """Backward-data with a caller-transposed weight: the layout the plan asks
    for, the other layout (ignored, the library transposes itself) and none."""
    import torch
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    P, Q = orc.conv_out_hw(_geom(s))
    dy = synth.int_codes(23, (N, P, Q, K))
    w = synth.int_codes(24, (K, R, R, Cc))
    ref = orc.conv_bwd_data_raw(dy, w, _geom(s))
    rc, rce = orc.requant(ref, -27, 8)
    kind = iseg.wt_kind((N, Hh, W, Cc), w.shape, st, pad, d)
    if kind == iseg.ISEG_WT_NONE:
        # the phase path (strided, few dy channels) repacks w itself: a
        # caller's layout of either kind is ignored
        kind = iseg.ISEG_WT_CRSK
    assert kind in (iseg.ISEG_WT_CRSK, iseg.ISEG_WT_CRSK_FLIP)
    other = iseg.ISEG_WT_CRSK + iseg.ISEG_WT_CRSK_FLIP - kind
    for k in (kind, other):
        wt = T(_wt_layout(w, k), dev)
        for mode in (iseg.ISEG_OUT_RAW, iseg.ISEG_OUT_Q8):
            o, oe = iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc),
                                       st, pad, d, out_mode=mode, wt=wt, wt_kind=k)
            if mode == iseg.ISEG_OUT_RAW:
                assert np.array_equal(H(o).astype(np.int64), ref) and ev(oe) == -27
            else:
                assert np.array_equal(H(o).astype(np.int64), rc) and ev(oe) == rce
    # a weight whose layout does not match its stated kind must not be read
    # when the kind is the other one: garbage in the unused layout is harmless
    junk = torch.full((Cc * R * R * K,), 77, dtype=torch.int8, device=dev)
    o, oe = iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc),
                               st, pad, d, out_mode=iseg.ISEG_OUT_RAW, wt=junk, wt_kind=other)
    assert np.array_equal(H(o).astype(np.int64), ref)


def test_weight_transpose_multi(dev):
    """One launch transposes a table of weights of ragged sizes, both layouts,
    and leaves the bytes beyond each destination alone."""
    import torch
    from paper_2011_14504_amd import iseg
    shapes = [(16, 3, 3, 16), (130, 3, 3, 128), (21, 1, 1, 20), (64, 7, 7, 3), (256, 1, 1, 2048),
              (1, 1, 1, 1), (65, 3, 3, 67)]
    ents, ws, outs, kinds = [], [], [], []
    for i, (K, R, S, Cc) in enumerate(shapes):
        w = synth.int_codes(40 + i, (K, R, S, Cc))
        kind = iseg.ISEG_WT_CRSK_FLIP if i % 2 else iseg.ISEG_WT_CRSK
        wd = T(w, dev)
        buf = torch.full((w.size + 64,), 99, dtype=torch.int8, device=dev)
        ents.append((wd, buf[:w.size].view(w.shape), kind))
        ws.append(w)
        outs.append(buf)
        kinds.append(kind)
    tab, n, tiles = iseg.wt_table(ents, dev)
    iseg.iseg_weight_transpose_multi(tab, n, tiles)
    for w, buf, kind in zip(ws, outs, kinds):
        got = H(buf)
        assert np.array_equal(got[:w.size], _wt_layout(w, kind).reshape(-1))
        assert (got[w.size:] == 99).all()
    # a tile count beyond the table's sum launches idle blocks only
    iseg.iseg_weight_transpose_multi(tab, n, tiles + 37)
    for w, buf, kind in zip(ws, outs, kinds):
        got = H(buf)
        assert np.array_equal(got[:w.size], _wt_layout(w, kind).reshape(-1))
        assert (got[w.size:] == 99).all()


@pytest.mark.parametrize("s", CONV_SHAPES, ids=str)
def test_conv_bwd_weight(orc, dev, s):
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    P, Q = orc.conv_out_hw(_geom(s))
    dy = synth.int_codes(31, (N, P, Q, K))
    x = synth.int_codes(32, (N, Hh, W, Cc))
    raw, re = iseg.conv_bwd_weight(T(dy, dev), E(-20, dev), T(x, dev), E(-7, dev), (K, R, R, Cc),
                                   st, pad, d, g_mode=iseg.ISEG_G_RAW)
    ref = orc.conv_bwd_weight_raw(dy, x, _geom(s))
    assert np.array_equal(H(raw), ref) and ev(re) == -27
    for mode, keep in ((iseg.ISEG_G_KEEP, True), (iseg.ISEG_G_DROP, False)):
        g, ge = iseg.conv_bwd_weight(T(dy, dev), E(-20, dev), T(x, dev), E(-7, dev), (K, R, R, Cc),
                                     st, pad, d, g_mode=mode, seed=1450401, tensor_id=16, step=2)
        rc, rce = orc.requant(ref, -27, 8, stochastic=True, keep_scale=keep, seed=1450401,
                              tensor_id=16, step=2)
        assert np.array_equal(H(g).astype(np.int64), rc) and ev(ge) == rce


def test_conv_bwd_weight_long_reduction(orc, dev):
    # more output pixels than one int32 partial may hold (131008): the split
    # reduction must still be exact
    x = synth.int_codes(41, (3, 220, 220, 4))
    dy = synth.int_codes(42, (3, 220, 220, 4))
    from paper_2011_14504_amd import iseg
    raw, _ = iseg.conv_bwd_weight(T(dy, dev), E(0, dev), T(x, dev), E(0, dev), (4, 1, 1, 4),
                                  1, 0, 1, g_mode=iseg.ISEG_G_RAW)
    ref = orc.conv_bwd_weight_raw(dy, x, (3, 220, 220, 4, 4, 1, 1, 1, 1, 0, 0, 1, 1))
    assert np.array_equal(H(raw), ref)


# Reductions longer than one exact int32 sum may hold (C R S or K R S above
# 131071, e.g. FCN's fc6: 7x7 from 4096 channels): the channels are split into
# chunks whose int32 sums the quantizer adds in int64.  (pass, N, H, W, C, K,
# R, pad, codes): "max" makes every code 127 so the centre sums pass 2^31.
LONG_KRED_CASES = [
    ("fwd", 1, 7, 7, 2740, 32, 7, 3, "max"),       # 2 chunks, C % 16 != 0
    ("fwd", 1, 3, 3, 6000, 16, 7, 3, "rand"),      # 3 chunks
    ("fwd", 2, 6, 7, 2752, 64, 7, 3, "rand"),
    ("bwd", 1, 7, 7, 64, 4096, 7, 3, "max"),       # fc6's backward-data
    ("bwd", 2, 8, 6, 48, 4100, 7, 3, "rand"),      # K % 16 != 0
    ("bwd", 1, 4, 4, 512, 4096, 7, 3, "rand"),
    ("bwd", 2, 16, 16, 512, 4096, 7, 3, "rand"),    # fc6 at 512x512 input, batch 2
    ("fwd", 1, 7, 7, 2752, 64, 7, 3, "max"),
    ("bwd", 1, 7, 7, 40, 4100, 7, 3, "max"),
]


@pytest.mark.parametrize("case", LONG_KRED_CASES, ids=lambda c: "-".join(str(v) for v in c))
def test_conv_long_reduction_split(orc, dev, case):
    from paper_2011_14504_amd import iseg
    kind, N, Hh, W, Cc, K, R, pad, codes = case
    geom = (N, Hh, W, Cc, K, R, R, 1, 1, pad, pad, 1, 1)
    P, Q = orc.conv_out_hw(geom)
    a_shape = (N, Hh, W, Cc) if kind == "fwd" else (N, P, Q, K)
    if codes == "max":
        a = np.full(a_shape, 127, np.int8)
        w = np.full((K, R, R, Cc), 127, np.int8)
    else:
        a = synth.int_codes(51, a_shape)
        w = synth.int_codes(52, (K, R, R, Cc))
    print(f"[long-kred] {case}", flush=True)
    if kind == "fwd":
        ref = orc.conv_fwd_raw(a, w, geom)
        out, oe = iseg.conv_fwd(T(a, dev), E(-7, dev), T(w, dev), E(-6, dev), 1, pad, 1)
    else:
        ref = orc.conv_bwd_data_raw(a, w, geom)
        out, oe = iseg.conv_bwd_data(T(a, dev), E(-7, dev), T(w, dev), E(-6, dev), (N, Hh, W, Cc), 1, pad, 1)
    # channel multiples of 64: one implicit GEMM split over the reduction;
    # otherwise channel chunks gathered and run one by one
    ci, nout = (Cc, K) if kind == "fwd" else (K, Cc)
    want = "kred_dma_split" if ci % 64 == 0 and nout % 64 == 0 else "kred_split"
    assert iseg.iseg_conv_last_plan() == want
    if codes == "max":
        assert np.abs(ref).max() > 2 ** 31 - 1
    rc, rce = orc.requant(ref, -13, 8)
    assert np.array_equal(H(out).astype(np.int64), rc) and ev(oe) == rce
    # the raw sums of such a reduction need not fit int32: refused
    with pytest.raises(iseg.IsegError):
        if kind == "fwd":
            iseg.conv_fwd(T(a, dev), E(-7, dev), T(w, dev), E(-6, dev), 1, pad, 1, out_mode=iseg.ISEG_OUT_RAW)
        else:
            iseg.conv_bwd_data(T(a, dev), E(-7, dev), T(w, dev), E(-6, dev), (N, Hh, W, Cc), 1, pad, 1,
                               out_mode=iseg.ISEG_OUT_RAW)


# Full-size layer shapes of the DeepLabv3-ResNet50 step (batch 8, 512x512),
# one per kernel path the step takes: (pass, N, H, W, C, K, R, stride, pad,
# dil, the path iseg_conv_last_plan must report for the final codes).  Whole
# tensors are compared: the raw int32 sums with the oracle's exact sums (its
# library path: float64 convolutions, exact on these integers), the codes
# with the oracle's requant of those sums -- never of the GPU's own sums.
FULL_CASES = [
    ("fwd", 8, 32, 32, 2048, 256, 3, 1, 6, 6, "dma_split"),        # ASPP branches
    ("fwd", 8, 32, 32, 2048, 256, 3, 1, 18, 18, "dma_split"),
    ("fwd", 8, 32, 32, 1024, 2048, 1, 1, 0, 1, "dma_stage16"),     # layer4.0 projection
    ("fwd", 8, 128, 128, 64, 256, 1, 1, 0, 1, "gemm_short"),      # layer1 conv3
    ("fwd", 8, 64, 64, 128, 512, 1, 1, 0, 1, "conv_short"),       # layer2 conv3
    ("fwd", 8, 32, 32, 256, 1024, 1, 1, 0, 1, "dma_two_pass"),    # layer3 conv3
    ("data", 8, 64, 64, 512, 128, 1, 1, 0, 1, "conv_short"),      # layer2.{1-3}.conv1
    ("data", 8, 128, 128, 256, 64, 1, 1, 0, 1, "gemm_short"),     # layer1.{1,2}.conv1
    ("data", 8, 32, 32, 2048, 256, 3, 1, 6, 6, "dma_stage16"),    # ASPP branches
    ("data", 8, 32, 32, 2048, 256, 3, 1, 12, 12, "dma_stage16"),
    ("data", 8, 32, 32, 2048, 256, 3, 1, 18, 18, "dma_stage16"),
    ("data", 8, 64, 64, 512, 1024, 1, 2, 0, 1, "strided_1x1"),     # layer3.0 projection (strided)
]


@pytest.mark.parametrize("case", FULL_CASES, ids=lambda c: "-".join(str(v) for v in c))
def test_conv_full_size(orc, dev, case):
    from paper_2011_14504_amd import iseg
    which, plan, s = case[0], case[-1], case[1:-1]
    N, Hh, W, Cc, K, R, st, pad, d = s
    g = _geom(s)
    P, Q = orc.conv_out_hw(g)
    w = synth.int_codes(92, (K, R, R, Cc))
    print(f"[full-size conv] {which} {s}", flush=True)
    if which == "fwd":
        x = synth.int_codes(91, (N, Hh, W, Cc))
        ref = orc._library_conv("fwd", x, w, g)
        raw, _ = iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), st, pad, d,
                               out_mode=iseg.ISEG_OUT_RAW)
        y, ye = iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), st, pad, d)
    else:
        dy = synth.int_codes(93, (N, P, Q, K))
        ref = orc._library_conv("data", dy, w, g)
        raw, _ = iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc),
                                    st, pad, d, out_mode=iseg.ISEG_OUT_RAW)
        y, ye = iseg.conv_bwd_data(T(dy, dev), E(-20, dev), T(w, dev), E(-7, dev), (N, Hh, W, Cc),
                                   st, pad, d)
    took = iseg.iseg_conv_last_plan()
    print(f"  path {took}", flush=True)
    if plan is not None:
        assert took == plan, (took, plan)
    assert np.array_equal(H(raw).astype(np.int64), ref)
    rc, rce = orc.requant(ref, -14 if which == "fwd" else -27, 8)
    assert ev(ye) == rce and np.array_equal(H(y).astype(np.int64), rc)


@pytest.mark.parametrize("s", [(8, 32, 32, 2048, 256, 3, 1, 6, 6), (8, 64, 64, 128, 512, 1, 1, 0, 1),
                               (8, 128, 128, 64, 64, 3, 1, 1, 1), (8, 32, 32, 512, 512, 3, 1, 2, 2)],
                         ids=str)
def test_conv_bwd_weight_full_size(orc, dev, s):
    """Full-size weight gradients whose reduction is split over blocks: the
    whole raw int64 tensor against the oracle's exact sums, and Q_G (kept
    and dropped scale) against the oracle's requant of those sums."""
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    P, Q = orc.conv_out_hw(_geom(s))
    dy = synth.int_codes(94, (N, P, Q, K))
    x = synth.int_codes(95, (N, Hh, W, Cc))
    raw, re = iseg.conv_bwd_weight(T(dy, dev), E(-20, dev), T(x, dev), E(-7, dev), (K, R, R, Cc),
                                   st, pad, d, g_mode=iseg.ISEG_G_RAW)
    ref = orc._library_conv("weight", dy, x, _geom(s))
    assert np.array_equal(H(raw), ref) and ev(re) == -27
    for mode, keep in ((iseg.ISEG_G_KEEP, True), (iseg.ISEG_G_DROP, False)):
        g, ge = iseg.conv_bwd_weight(T(dy, dev), E(-20, dev), T(x, dev), E(-7, dev), (K, R, R, Cc),
                                     st, pad, d, g_mode=mode, seed=77, tensor_id=48, step=5)
        print(f"  wgrad path {iseg.iseg_conv_last_plan()}", flush=True)
        rc, rce = orc.requant(ref, -27, 8, stochastic=True, keep_scale=keep, seed=77,
                              tensor_id=48, step=5)
        assert np.array_equal(H(g).astype(np.int64), rc) and ev(ge) == rce


def test_conv_zero_input(orc, dev):
    from paper_2011_14504_amd import iseg
    x = np.zeros((1, 8, 8, 16), np.int8)
    w = synth.int_codes(5, (16, 3, 3, 16))
    y, ye = iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), 1, 1, 1)
    assert not H(y).any() and ev(ye) == -14


def test_conv_deterministic(dev):
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(51, (2, 40, 40, 64))
    dy = synth.int_codes(52, (2, 40, 40, 64))
    a, ae = iseg.conv_bwd_weight(T(dy, dev), E(-20, dev), T(x, dev), E(-7, dev), (64, 3, 3, 64),
                                 1, 1, 1, seed=9)
    b, be = iseg.conv_bwd_weight(T(dy, dev), E(-20, dev), T(x, dev), E(-7, dev), (64, 3, 3, 64),
                                 1, 1, 1, seed=9)
    assert np.array_equal(H(a), H(b)) and ev(ae) == ev(be)


# ---------------------------------------------------------------------------
# L1 batch normalization
# ---------------------------------------------------------------------------
BN_CASES = [
    dict(M=1024, C=16, x_exp=-9, cfg={}),
    dict(M=4099, C=64, x_exp=-7, cfg=dict(relu=0)),
    dict(M=777, C=128, x_exp=-14, cfg=dict(eps_code=1)),
    dict(M=300, C=256, x_exp=2, cfg=dict(k_E2=8)),
    dict(M=5, C=4, x_exp=-30, cfg={}),
    dict(M=2000, C=48, x_exp=-11, cfg=dict(k_E2=8, relu=0), const=True),
    dict(M=1500, C=20, x_exp=-7, cfg=dict(k_xhat=8, k_mu=8, k_sigma=8)),
    # the per-slice tails at scale: one slice of 256 blocks; 16 forward / 32
    # backward slices; C = 4 * 67, 67 four-channel slices (256 row groups in
    # each tail), both E2 paths
    dict(M=65536 + 37, C=64, x_exp=-8, cfg={}),
    dict(M=4096 + 3, C=2048, x_exp=-6, cfg=dict(relu=0)),
    dict(M=3001, C=268, x_exp=-10, cfg=dict(k_E2=8)),
    dict(M=3001, C=268, x_exp=-10, cfg={}),
    # rounding E2 (k_E2 < 15) at scale: its two streaming passes each end in
    # per-slice tails, one slice of 256 blocks / 32 slices / narrow E2
    dict(M=65536 + 37, C=64, x_exp=-8, cfg=dict(k_E2=8)),
    dict(M=4096 + 3, C=2048, x_exp=-6, cfg=dict(k_E2=12, relu=0)),
    dict(M=999, C=96, x_exp=-9, cfg=dict(k_E2=4)),
]


def _bn_inputs(i, case):
    x = synth.int_codes(100 + i, (case["M"], case["C"]))
    if case.get("const"):
        x[:, 1] = 17
        x[:, 2] = 0
    gq = synth.int_codes(200 + i, (case["C"],))
    bq = synth.int_codes(300 + i, (case["C"],))
    dA = synth.int_codes(400 + i, (case["M"], case["C"]))
    return x, gq, bq, dA


@pytest.mark.parametrize("i", range(len(BN_CASES)))
def test_bn_fwd(orc, dev, i):
    from paper_2011_14504_amd import iseg
    case = BN_CASES[i]
    x, gq, bq, _ = _bn_inputs(i, case)
    cfg = dict(orc.BN_DEFAULT, **case["cfg"])
    y, ye, saved = iseg.bn_fwd(T(x, dev), E(case["x_exp"], dev), T(gq, dev), T(bq, dev),
                               iseg.bn_cfg(**cfg))
    r = orc.bn_fwd(x, case["x_exp"], gq, bq, cfg)
    sv = iseg.bn_saved_view(saved, case["C"])
    assert np.array_equal(H(sv["n_mu"]), r["n_mu"])
    assert np.array_equal(H(sv["n_sigma"]), r["n_sigma"])
    assert int(H(sv["hdr"])[0]) == r["b"]
    xc = H(sv["xcode"])
    cols = np.arange(case["C"])[None, :]
    assert np.array_equal(xc[cols, x.astype(np.int64) + 128], r["xhat"])
    assert np.array_equal(H(y), r["y"]) and ev(ye) == r["y_exp"]


@pytest.mark.parametrize("i", range(len(BN_CASES)))
def test_bn_bwd(orc, dev, i):
    from paper_2011_14504_amd import iseg
    case = BN_CASES[i]
    x, gq, bq, dA = _bn_inputs(i, case)
    cfg = dict(orc.BN_DEFAULT, **case["cfg"])
    c = iseg.bn_cfg(**cfg)
    y, ye, saved = iseg.bn_fwd(T(x, dev), E(case["x_exp"], dev), T(gq, dev), T(bq, dev), c)
    dx, dxe, dg, db, dge, dbe = iseg.bn_bwd(T(dA, dev), E(-20, dev), T(x, dev), T(gq, dev), saved, c)
    r = orc.bn_bwd(dA, -20, x, case["x_exp"], gq, bq, cfg)
    assert np.array_equal(H(db), r["dbeta"]) and ev(dbe) == r["dbeta_exp"]
    assert np.array_equal(H(dg), r["dgamma"]) and ev(dge) == r["dgamma_exp"]
    assert np.array_equal(H(dx), r["dx"]) and ev(dxe) == r["dx_exp"]


def test_bn_repeated_calls_same_workspace(orc, dev):
    """Back-to-back calls of different shapes on one workspace: each call
    must leave the arrival counters at zero for the next."""
    from paper_2011_14504_amd import iseg
    refs = {}
    for rep in range(2):
        for i in (0, 3, 7, 9, 10, 11, 12, 13):
            case = BN_CASES[i]
            x, gq, bq, dA = _bn_inputs(i, case)
            cfg = dict(orc.BN_DEFAULT, **case["cfg"])
            c = iseg.bn_cfg(**cfg)
            y, ye, saved = iseg.bn_fwd(T(x, dev), E(case["x_exp"], dev), T(gq, dev), T(bq, dev), c)
            dx, dxe, dg, db, dge, dbe = iseg.bn_bwd(T(dA, dev), E(-20, dev), T(x, dev), T(gq, dev), saved, c)
            if i not in refs:
                refs[i] = (orc.bn_fwd(x, case["x_exp"], gq, bq, cfg),
                           orc.bn_bwd(dA, -20, x, case["x_exp"], gq, bq, cfg))
            r, rb = refs[i]
            assert np.array_equal(H(y), r["y"]) and ev(ye) == r["y_exp"], (rep, i)
            assert np.array_equal(H(dx), rb["dx"]) and ev(dxe) == rb["dx_exp"], (rep, i)
            assert np.array_equal(H(dg), rb["dgamma"]), (rep, i)


def test_bn_exponent_out_of_range_flags_status(dev):
    import torch
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(9, (64, 16))
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    iseg.bn_fwd(T(x, dev), E(30, dev), T(np.full(16, 64, np.int8), dev),
                T(np.zeros(16, np.int8), dev), status=st)
    assert ev(st) & iseg.ISEG_DEV_RANGE


# ---------------------------------------------------------------------------
# update, weight quantizer, max pooling
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("g_exp,lr,mexp", [(-20, 10, -23), (-3, 4, -23), (-30, 0, -22), (5, 2, -23)])
def test_weight_update(orc, dev, g_exp, lr, mexp):
    from paper_2011_14504_amd import iseg
    n = 100003
    master = synth.int_codes(61, (n,), -(2 ** 23) + 1, 2 ** 23 - 1, np.int32)
    g = synth.int_codes(62, (n,))
    m_t = T(master, dev)
    wq = iseg.weight_update(m_t, T(g, dev), E(g_exp, dev), lr, mexp)
    rm, rw = orc.weight_update(master, g, g_exp, lr, mexp)
    assert np.array_equal(H(m_t), rm) and np.array_equal(H(wq), rw)


def test_weight_quant_and_master_init(orc, dev):
    from paper_2011_14504_amd import iseg
    w = synth.he_normal(63, (64, 3, 3, 64), 576)
    m, me = iseg.quantize(T(w, dev), 24, iseg.ISEG_Q_UQ)
    rm, rme = orc.master_init(w)
    assert np.array_equal(H(m), rm) and ev(me) == rme == -23
    assert np.array_equal(H(iseg.weight_quant(m)), orc.weight_quant(rm))


@pytest.mark.parametrize("k,st,pad", [(2, 2, 0), (3, 2, 1), (3, 1, 1)])
def test_maxpool(orc, dev, k, st, pad):
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(71, (2, 29, 31, 24))
    x[0, :4, :4, :] = 5                       # ties
    y, ye = iseg.maxpool_fwd(T(x, dev), E(-6, dev), k, st, pad)
    assert np.array_equal(H(y), orc.maxpool_fwd(x, k, st, pad)) and ev(ye) == -6
    dy = synth.int_codes(72, H(y).shape)
    dx, dxe = iseg.maxpool_bwd(T(dy, dev), E(-20, dev), T(x, dev), k, st, pad)
    rc, rce = orc.maxpool_bwd(dy, -20, x, k, st, pad)
    assert np.array_equal(H(dx).astype(np.int64), rc) and ev(dxe) == rce


@pytest.mark.parametrize("shape,small", [((2, 29, 31, 32), False), ((1, 8, 8, 64), True),
                                         ((3, 16, 10, 16), False)])
def test_maxpool_2x2_window_path(orc, dev, shape, small):
    """2x2/2 windows with 16-channel vectors (per-window kernel), ragged H/W
    whose last row/column no window covers, ties, and an error tensor whose
    max is below 64 (negative requant shift)."""
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(73, shape)
    x[0, :4, :4, :] = -3                      # ties
    y, ye = iseg.maxpool_fwd(T(x, dev), E(-6, dev), 2, 2, 0)
    assert np.array_equal(H(y), orc.maxpool_fwd(x, 2, 2, 0))
    dy = synth.int_codes(74, H(y).shape)
    if small:
        dy = (dy // 8).astype(np.int8)
    dx, dxe = iseg.maxpool_bwd(T(dy, dev), E(-20, dev), T(x, dev), 2, 2, 0)
    rc, rce = orc.maxpool_bwd(dy, -20, x, 2, 2, 0)
    assert np.array_equal(H(dx).astype(np.int64), rc) and ev(dxe) == rce


@pytest.mark.parametrize("shape,k,st,pad", [((2, 64, 64, 64), 3, 2, 1), ((1, 29, 31, 16), 3, 2, 1),
                                            ((2, 17, 12, 32), 3, 1, 1), ((1, 23, 19, 48), 5, 3, 2),
                                            ((1, 9, 9, 16), 2, 1, 0)], ids=str)
def test_maxpool_overlapping_vector_path(orc, dev, shape, k, st, pad):
    """Overlapping windows with 16-channel vectors (per-window argmax taps and
    two gathers): the ResNet stem's 3x3/2 pad 1, stride 1, a 5x5/3 pad 2 and a
    2x2/1 case, with ties inside windows."""
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(75, shape)
    x[0, :5, :5, :] = 7                       # ties across overlapping windows
    y, ye = iseg.maxpool_fwd(T(x, dev), E(-6, dev), k, st, pad)
    assert np.array_equal(H(y), orc.maxpool_fwd(x, k, st, pad))
    dy = synth.int_codes(76, H(y).shape)
    dx, dxe = iseg.maxpool_bwd(T(dy, dev), E(-19, dev), T(x, dev), k, st, pad)
    rc, rce = orc.maxpool_bwd(dy, -19, x, k, st, pad)
    assert np.array_equal(H(dx).astype(np.int64), rc) and ev(dxe) == rce


def test_update_multi_matches_oracle(orc, dev):
    """One launch updating conv weights (quantized G) and L1BN gamma / beta (raw
    sums, Q_G first) equals the oracle's per-tensor Eq. 19 / Eq. 8."""
    import torch
    from paper_2011_14504_amd import iseg
    r = synth.rng(90)
    ents, ref = [], []
    for i, n in enumerate((64 * 9 * 64, 1000, 3)):
        m = r.integers(-(2 ** 23) + 1, 2 ** 23, size=n).astype(np.int32)
        g = r.integers(-127, 128, size=n).astype(np.int8)
        mt, gt = T(m, dev), T(g, dev)
        ents.append(dict(master=mt, w_q=torch.empty(n, dtype=torch.int8, device=dev), g=gt,
                         g_exp=E(-25 - i, dev), kind=iseg.ISEG_UPD_CODES, master_exp=-23))
        ref.append(orc.weight_update(m, g, -25 - i, 10, -23, 24, 8))
    for i, C in enumerate((64, 2048)):
        m = r.integers(-(2 ** 23) + 1, 2 ** 23, size=C).astype(np.int32)
        d = r.integers(-(2 ** 40), 2 ** 40, size=C).astype(np.int64)
        ents.append(dict(master=T(m, dev), w_q=torch.empty(C, dtype=torch.int8, device=dev), g=T(d, dev),
                         g_exp=E(-30, dev), kind=iseg.ISEG_UPD_RAW, master_exp=-22, tensor_id=17 + i,
                         g_q=torch.empty(C, dtype=torch.int8, device=dev), g_q_exp=E(0, dev)))
        gq, gqe = orc.requant(d, -30, 8, True, True, 55, 17 + i, 4)
        ref.append(orc.weight_update(m, gq, gqe, 10, -22, 24, 8) + (gq, gqe))
    table, n = iseg.update_table(ents, dev)
    iseg.iseg_update_multi(table, n, 8, 55, 4, 10, 24, 8)
    for e, rr in zip(ents, ref):
        assert np.array_equal(H(e["master"]), rr[0]) and np.array_equal(H(e["w_q"]), rr[1])
        if e["kind"] == iseg.ISEG_UPD_RAW:
            assert np.array_equal(H(e["g_q"]).astype(np.int64), rr[2]) and ev(e["g_q_exp"]) == rr[3]


def test_update_multi_per_tensor_width(orc, dev):
    """k_U = 16 with 4-bit conv weights and 8-bit gamma / beta in one launch
    (each descriptor's own k_w; 0 takes the call's k_W); an entry whose width
    is out of range is left untouched and flags ISEG_DEV_DESC."""
    import torch
    from paper_2011_14504_amd import iseg
    r = synth.rng(91)
    k_U = 16
    ents, ref = [], []
    for i, (n, kw) in enumerate(((3 * 3 * 64 * 32, 0), (777, 4), (33, 9))):
        m = r.integers(-(2 ** 15) + 1, 2 ** 15, size=n).astype(np.int32)
        g = r.integers(-127, 128, size=n).astype(np.int8)
        ents.append(dict(master=T(m, dev), w_q=torch.full((n,), 99, dtype=torch.int8, device=dev),
                         g=T(g, dev), g_exp=E(-18 - i, dev), kind=iseg.ISEG_UPD_CODES,
                         master_exp=1 - k_U, k_w=kw))
        ref.append(orc.weight_update(m, g, -18 - i, 6, 1 - k_U, k_U, 4) if kw != 9 else
                   (m, np.full(n, 99, np.int8)))
    C = 256
    m = r.integers(-(2 ** 15) + 1, 2 ** 15, size=C).astype(np.int32)
    d = r.integers(-(2 ** 30), 2 ** 30, size=C).astype(np.int64)
    ents.append(dict(master=T(m, dev), w_q=torch.empty(C, dtype=torch.int8, device=dev), g=T(d, dev),
                     g_exp=E(-28, dev), kind=iseg.ISEG_UPD_RAW, master_exp=2 - k_U, tensor_id=33,
                     g_q=torch.empty(C, dtype=torch.int8, device=dev), g_q_exp=E(0, dev), k_w=8))
    gq, gqe = orc.requant(d, -28, 8, True, True, 56, 33, 2)
    ref.append(orc.weight_update(m, gq, gqe, 6, 2 - k_U, k_U, 8))
    table, n = iseg.update_table(ents, dev)
    st = E(0, dev)
    iseg.iseg_update_multi(table, n, 8, 56, 2, 6, k_U, 4, st)
    for e, rr in zip(ents, ref):
        assert np.array_equal(H(e["master"]), rr[0]) and np.array_equal(H(e["w_q"]), rr[1])
    assert np.abs(H(ents[0]["w_q"]).astype(np.int64)).max() <= 7
    assert ev(st) == iseg.ISEG_DEV_DESC


@pytest.mark.parametrize("C,d_exp", [(64, -30), (128, -12), (2048, -40)])
def test_bn_param_update(orc, dev, C, d_exp):
    # Q_G (Eq. 17, stochastic) then Q_U (Eq. 19) of gamma/beta in one launch
    from paper_2011_14504_amd import iseg
    import torch
    rng = synth.rng(C)
    dg = rng.integers(-(2 ** 40), 2 ** 40, size=C, dtype=np.int64)
    db = rng.integers(-(2 ** 20), 2 ** 20, size=C, dtype=np.int64)
    gm = synth.int_codes(C + 1, (C,), -(2 ** 23) + 1, 2 ** 23 - 1, np.int32)
    bm = synth.int_codes(C + 2, (C,), -(2 ** 23) + 1, 2 ** 23 - 1, np.int32)
    gm_t, bm_t = T(gm, dev), T(bm, dev)
    gq = torch.empty(C, dtype=torch.int8, device=dev)
    bq = torch.empty(C, dtype=torch.int8, device=dev)
    Gg = torch.empty(C, dtype=torch.int8, device=dev)
    Gb = torch.empty(C, dtype=torch.int8, device=dev)
    Gge, Gbe = E(0, dev), E(0, dev)
    iseg.iseg_bn_param_update(T(dg, dev), E(d_exp, dev), T(db, dev), E(d_exp - 3, dev), 8, 99, 17,
                              18, 4, 10, -22, 24, 8, gm_t, bm_t, gq, bq, Gg, Gb, Gge, Gbe)
    for d, e, tid, m, m_t, q_t, G_t, Ge_t in ((dg, d_exp, 17, gm, gm_t, gq, Gg, Gge),
                                              (db, d_exp - 3, 18, bm, bm_t, bq, Gb, Gbe)):
        rc, re = orc.requant(d, e, 8, stochastic=True, keep_scale=True, seed=99, tensor_id=tid,
                             step=4)
        assert np.array_equal(H(G_t).astype(np.int64), rc) and ev(Ge_t) == re
        rm, rw = orc.weight_update(m, rc, re, 10, -22, 24, 8)
        assert np.array_equal(H(m_t), rm) and np.array_equal(H(q_t), rw)


# L1BN on the raw int32 sums of a convolution: magnitudes up to 2^30, input
# exponents across [-40, 0], a channel slice wider than one block (C > 256),
# ragged channel counts, constant and all-equal channels, long columns
BN32_CASES = [
    dict(M=1024, C=16, x_exp=-14, mag=1 << 20, cfg={}),
    dict(M=65536 + 37, C=64, x_exp=-13, mag=1 << 25, cfg=dict(relu=0)),
    dict(M=4096 + 3, C=2048, x_exp=-9, mag=1 << 18, cfg={}),
    dict(M=777, C=20, x_exp=-40, mag=1 << 12, cfg=dict(eps_code=3)),
    dict(M=300, C=264, x_exp=0, mag=1 << 30, cfg={}),
    dict(M=2000, C=48, x_exp=-11, mag=70000, cfg=dict(relu=0), const=True),
    dict(M=1500, C=20, x_exp=-12, mag=9000, cfg=dict(k_xhat=8, k_mu=8, k_sigma=8)),
    dict(M=5, C=4, x_exp=-20, mag=1 << 30, cfg={}),
]


def _bn32_inputs(i, case):
    rng = synth.rng(700 + i)
    m = case["mag"]
    x = rng.integers(-m, m + 1, size=(case["M"], case["C"])).astype(np.int32)
    if case.get("const"):
        x[:, 1] = 17
        x[:, 2] = 0
    gq = synth.int_codes(800 + i, (case["C"],))
    bq = synth.int_codes(900 + i, (case["C"],))
    dA = synth.int_codes(1000 + i, (case["M"], case["C"]))
    return x, gq, bq, dA


@pytest.mark.parametrize("i", range(len(BN32_CASES)))
def test_bn_int32_input_fwd_bwd(orc, dev, i):
    from paper_2011_14504_amd import iseg
    case = BN32_CASES[i]
    print(f"[bn int32] {case}", flush=True)
    x, gq, bq, dA = _bn32_inputs(i, case)
    cfg = dict(orc.BN_DEFAULT, **case["cfg"])
    c = iseg.bn_cfg(**cfg)
    st = torch_zeros_status(dev)
    y, ye, saved = iseg.bn_fwd(T(x, dev), E(case["x_exp"], dev), T(gq, dev), T(bq, dev), c, status=st)
    r = orc.bn_fwd(x, case["x_exp"], gq, bq, cfg)
    assert np.array_equal(H(y), r["y"]) and ev(ye) == r["y_exp"]
    dx, dxe, dg, db, dge, dbe = iseg.bn_bwd(T(dA, dev), E(-20, dev), T(x, dev), T(gq, dev), saved, c, status=st)
    rb = orc.bn_bwd(dA, -20, x, case["x_exp"], gq, bq, cfg)
    assert np.array_equal(H(dg), rb["dgamma"]) and np.array_equal(H(db), rb["dbeta"])
    assert ev(dge) == rb["dgamma_exp"] and ev(dbe) == rb["dbeta_exp"]
    assert np.array_equal(H(dx), rb["dx"]) and ev(dxe) == rb["dx_exp"]
    assert int(st.item()) == 0


def test_bn_int32_input_exponent_range(dev):
    from paper_2011_14504_amd import iseg
    x = (synth.int_codes(5, (256, 16)).astype(np.int32) * 1000)
    g = np.full(16, 64, np.int8)
    b = np.zeros(16, np.int8)
    for e, want in ((0, 0), (1, iseg.ISEG_DEV_RANGE), (-40, 0), (-41, iseg.ISEG_DEV_RANGE)):
        st = torch_zeros_status(dev)
        iseg.bn_fwd(T(x, dev), E(e, dev), T(g, dev), T(b, dev), status=st)
        assert int(st.item()) == want, e


def torch_zeros_status(dev):
    import torch
    return torch.zeros(1, dtype=torch.int32, device=dev)


# Inference with a calibration forward's frozen state: the A table on new
# codes, and conv + L1BN + ReLU + Q_A of one layer in one pass over the sums
@pytest.mark.parametrize("case", [dict(M=4099, C=64, x_exp=-9, cfg={}), dict(M=777, C=20, x_exp=-14, cfg=dict(relu=0)),
                                  dict(M=2048, C=2048, x_exp=-6, cfg=dict(eps_code=1))], ids=str)
def test_bn_infer_frozen_state(orc, dev, case):
    from paper_2011_14504_amd import iseg
    cfg = dict(orc.BN_DEFAULT, **case["cfg"])
    cal = synth.int_codes(1100, (case["M"], case["C"]))
    new = (synth.int_codes(1101, (case["M"], case["C"])).astype(np.int64) * 3 // 4 + 20).astype(np.int8)
    gq = synth.int_codes(1102, (case["C"],))
    bq = synth.int_codes(1103, (case["C"],))
    c = iseg.bn_cfg(**cfg)
    y, ye, saved = iseg.bn_fwd(T(cal, dev), E(case["x_exp"], dev), T(gq, dev), T(bq, dev), c)
    st = orc.bn_state(orc.bn_fwd(cal, case["x_exp"], gq, bq, cfg))
    for x, label in ((cal, "calibration batch"), (new, "new batch")):
        a, ae = iseg.bn_infer(T(x, dev), E(case["x_exp"], dev), saved)
        ref = orc.bn_infer(x, case["x_exp"], gq, bq, st, cfg)
        assert np.array_equal(H(a), ref) and ev(ae) == st["a_exp"], label
    assert np.array_equal(H(iseg.bn_infer(T(cal, dev), E(case["x_exp"], dev), saved)[0]), H(y))


@pytest.mark.parametrize("s", [(8, 32, 32, 64, 64, 3, 1, 1, 1), (8, 32, 32, 256, 64, 1, 1, 0, 1),
                               (2, 32, 32, 2048, 256, 3, 1, 6, 6), (1, 9, 7, 24, 36, 3, 2, 1, 1)], ids=str)
def test_conv_bn_infer(orc, dev, s):
    from paper_2011_14504_amd import iseg
    N, Hh, W, Cc, K, R, st, pad, d = s
    g = _geom(s)
    cfg = dict(orc.BN_DEFAULT)
    w = synth.int_codes(1200, (K, R, R, Cc)) // 4
    gq = synth.int_codes(1201, (K,))
    bq = synth.int_codes(1202, (K,))
    cal = synth.int_codes(1203, (N, Hh, W, Cc))
    new = synth.int_codes(1204, (N, Hh, W, Cc))
    # calibration: the training forward of the layer (conv -> SQ8 -> L1BN -> ReLU -> Q_A)
    z, ze = iseg.conv_fwd(T(cal, dev), E(-7, dev), T(w, dev), E(-7, dev), st, pad, d)
    y, ye, saved = iseg.bn_fwd(z, ze, T(gq, dev), T(bq, dev), iseg.bn_cfg(**cfg))
    zc, zce = orc.conv_fwd(cal, -7, w, -7, g)
    state = orc.bn_state(orc.bn_fwd(zc.astype(np.int8), zce, gq, bq, cfg))
    assert ev(ze) == zce
    for x in (cal, new):
        a, ae = iseg.conv_bn_infer(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), saved, st, pad, d)
        zz = orc.requant_fixed(orc.conv_fwd_raw(x, w, g), -14, zce, 8)
        ref = orc.bn_infer(zz, zce, gq, bq, state, cfg)
        assert np.array_equal(H(a), ref) and ev(ae) == state["a_exp"]


# Transposed convolutions of the FCN decoder (the adjoint of a conv): the
# forward is backward-data, the input error a forward conv, the weight
# gradient pairs the node's input with its output error; 21 classes
@pytest.mark.parametrize("s", [(2, 8, 8, 21, 21, 4, 2, 1), (1, 8, 8, 21, 21, 16, 8, 4), (2, 5, 7, 150, 150, 4, 2, 1),
                               (1, 6, 5, 12, 20, 3, 2, 1)], ids=str)
def test_transposed_conv(orc, dev, s):
    from paper_2011_14504_amd import iseg
    N, h, w, cin, cout, R, st, pad = s
    H = (h - 1) * st - 2 * pad + R
    W = (w - 1) * st - 2 * pad + R
    g = (N, H, W, cout, cin, R, R, st, st, pad, pad, 1, 1)      # the conv it is the adjoint of
    a = synth.int_codes(1400, (N, h, w, cin))
    wt = synth.int_codes(1401, (cin, R, R, cout))
    dz = synth.int_codes(1402, (N, H, W, cout))
    y, ye = iseg.conv_bwd_data(T(a, dev), E(-5, dev), T(wt, dev), E(-7, dev), (N, H, W, cout), st, pad, 1)
    ry, rye = orc.conv_bwd_data(a, -5, wt, -7, g)
    assert np.array_equal(H_(y), ry) and ev(ye) == rye
    e, ee = iseg.conv_fwd(T(dz, dev), E(-20, dev), T(wt, dev), E(-7, dev), st, pad, 1)
    re_, ree = orc.conv_fwd(dz, -20, wt, -7, g)
    assert np.array_equal(H_(e), re_) and ev(ee) == ree
    G, Ge = iseg.conv_bwd_weight(T(a, dev), E(-5, dev), T(dz, dev), E(-20, dev), (cin, R, R, cout), st, pad, 1,
                                 g_mode=iseg.ISEG_G_DROP, seed=9, tensor_id=32, step=1)
    rG, rGe = orc.conv_bwd_weight(a, -5, dz, -20, g, 8, False, 9, 32, 1)
    assert np.array_equal(H_(G), rG) and ev(Ge) == rGe


def H_(t):
    return t.cpu().numpy().astype(np.int64)


@pytest.mark.parametrize("shape", [(1, 6, 5, 3), (2, 64, 48, 21), (1, 128, 128, 150)], ids=str)
@pytest.mark.parametrize("y_exp", [-6, 1, -30])
def test_mse_onehot(orc, dev, shape, y_exp):
    from paper_2011_14504_amd import iseg
    N, Hh, W, K = shape
    y = synth.int_codes(1500 + K, shape)
    lab = synth.labels(1501 + K, (N, Hh, W), K)
    st = torch_zeros_status(dev)
    loss, e, ee = iseg.mse_onehot(T(y, dev), E(y_exp, dev), T(lab, dev), status=st)
    rl, rc, rce = orc.mse_onehot(y, y_exp, lab)
    assert int(st.item()) == 0
    assert abs(float(loss.item()) - rl) <= 1e-12 * rl
    assert np.array_equal(H_(e), rc) and ev(ee) == rce
