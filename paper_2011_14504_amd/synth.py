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
