"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke
check.  This module holds no arithmetic of the method: it only draws random
numbers (numpy PCG64) with the shapes and value ranges of the workloads.

Recipe (stands in for PASCAL VOC 2012 / ADE20K, which are not available):
  * images, activations: int8 codes uniform on [-127, 127], exponent -7;
  * errors arriving at a layer output: int8 codes uniform on [-127, 127],
    exponent -20 (values up to ~1.2e-4, the 1e-5..1e-4 range the paper
    reports for errors in Sec. 3.1.2);
  * conv weights: float32 He-normal N(0, 2/fan_in) (MSRA initialisation,
    Sec. 3.2.1), turned into 24-bit master codes by the library's own Eq. 7
    quantizer on each side;
  * BN gamma/beta: gamma = 1, beta = 0 for benchmark runs; random int8 codes
    for parity runs;
  * labels: uint8 uniform over the class count.
Seeds: 1450400 + 100 * workload + ordinal.
"""
import numpy as np

SEED_BASE = 1450400
ACT_EXP = -7
ERR_EXP = -20


def seed_for(workload, ordinal):
    return SEED_BASE + 100 * int(workload) + int(ordinal)


def rng(seed):
    return np.random.Generator(np.random.PCG64(int(seed)))


def int_codes(seed, shape, lo=-127, hi=127, dtype=np.int8):
    """Integers uniform on [lo, hi]."""
    return rng(seed).integers(lo, hi + 1, size=shape, dtype=np.int64).astype(dtype)


def he_normal(seed, shape, fan_in):
    """float32 normal with standard deviation sqrt(2 / fan_in)."""
    std = np.sqrt(2.0 / float(fan_in))
    return (rng(seed).standard_normal(size=shape) * std).astype(np.float32)


def gaussian_codes(seed, shape, std, dtype=np.int8):
    """Rounded normal samples clipped to [-127, 127] (for BN statistics tests)."""
    v = np.rint(rng(seed).standard_normal(size=shape) * std)
    return np.clip(v, -127, 127).astype(dtype)


def labels(seed, shape, classes):
    return rng(seed).integers(0, classes, size=shape, dtype=np.int64).astype(np.uint8)


def uniform_f32(seed, shape, lo=-1.0, hi=1.0):
    return rng(seed).uniform(lo, hi, size=shape).astype(np.float32)


# ---------------------------------------------------------------------------
# workload shapes (shapes and seeds only)
# ---------------------------------------------------------------------------
# A layer is ("conv", C_in, C_out, R, stride, pad, dilation) -- each conv is
# followed by L1BN + ReLU -- or ("maxpool", k, stride, pad).

# Single 3x3 conv 16 -> 16, stride 1, pad 1, on a 1x32x32 map, then L1BN over
# 16 channels; the input gradient is computed too.
SINGLE_CONV = dict(id=1, name="single-conv3x3-16ch-32x32-n1", N=1, H=32, W=32, C=16,
                   input_grad=True,
                   layers=[("conv", 16, 16, 3, 1, 1, 1)])

# FCN-VGG16 encoder slice: conv1_1, conv1_2, maxpool 2x2/2, conv2_1, conv2_2,
# batch 8 of 3x224x224 images; no gradient is taken w.r.t. the image.
VGG16_BLOCKS12 = dict(id=2, name="fcn-vgg16-blocks1-2-n8-224", N=8, H=224, W=224, C=3,
                      input_grad=False,
                      layers=[("conv", 3, 64, 3, 1, 1, 1),
                              ("conv", 64, 64, 3, 1, 1, 1),
                              ("maxpool", 2, 2, 0),
                              ("conv", 64, 128, 3, 1, 1, 1),
                              ("conv", 128, 128, 3, 1, 1, 1)])

WORKLOADS = {1: SINGLE_CONV, 2: VGG16_BLOCKS12}


def workload_inputs(wl, N=None):
    """Seeded inputs of a workload: image/activation codes, float weights per
    conv (He-normal), and the error arriving at the last activation."""
    N = wl["N"] if N is None else N
    x = int_codes(seed_for(wl["id"], 0), (N, wl["H"], wl["W"], wl["C"]))
    weights = []
    Hh, W = wl["H"], wl["W"]
    ordinal = 1
    for layer in wl["layers"]:
        if layer[0] == "conv":
            _, cin, cout, R, st, pad, dil = layer
            weights.append(he_normal(seed_for(wl["id"], ordinal), (cout, R, R, cin), cin * R * R))
            ordinal += 1
            Hh = (Hh + 2 * pad - dil * (R - 1) - 1) // st + 1
            W = (W + 2 * pad - dil * (R - 1) - 1) // st + 1
            cl = cout
        else:
            _, k, st, pad = layer
            Hh = (Hh + 2 * pad - k) // st + 1
            W = (W + 2 * pad - k) // st + 1
    dy = int_codes(seed_for(wl["id"], 50), (N, Hh, W, cl))
    return dict(x=x, x_exp=ACT_EXP, weights=weights, dy=dy, dy_exp=ERR_EXP,
                seed=seed_for(wl["id"], 0))
