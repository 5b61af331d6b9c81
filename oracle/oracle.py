"""Python face of the CPU oracle (ctypes over liboracle.so, numpy host arrays).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library or its binding.

Each function follows one step of the paper's quantized dataflow (arXiv
2011.14504, Sec. 3) and says which equation; the composition of a layer
(integer sum, then the quantizer) is written out here in the order the paper
applies it.  Quantized tensors are (codes, exponent) pairs: value = code*2^exp.
"""
import ctypes as C
import os

import numpy as np

from . import build as _build

_lib = None

# L1BN bit-widths, Sec. 5 implementation details (DeepLabv3 row):
# k_mu = k_sigma = k_xhat = 16, k_gamma = k_beta = 8, k_A = k_E1 = 8, k_E2 = 16.
BN_DEFAULT = dict(k_mu=16, k_sigma=16, k_xhat=16, k_gamma=8, k_beta=8,
                  k_A=8, k_E1=8, k_E2=16, eps_code=0, relu=1)
_BN_KEYS = ["k_mu", "k_sigma", "k_xhat", "k_gamma", "k_beta", "k_A", "k_E1",
            "k_E2", "eps_code", "relu"]


class OracleError(RuntimeError):
    pass


def lib():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
        L = C.CDLL(path)
        P = C.c_void_p
        i64, i32, u64, u32 = C.c_int64, C.c_int32, C.c_uint64, C.c_uint32
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_draw_u64.argtypes = [u64, u32, u32, u64]
        L.orc_draw_u64.restype = u64
        L.orc_uq_code_f64.argtypes = [C.c_double, C.c_int]
        L.orc_uq_code_f64.restype = i64
        L.orc_quantize_f32.argtypes = [P, i64, C.c_int, C.c_int, P, P]
        L.orc_quantize_f64.argtypes = [P, i64, C.c_int, C.c_int, P, P]
        L.orc_requant.argtypes = [P, i64, i32, C.c_int, C.c_int, C.c_int, u64, u32, u32, P, P]
        for f in ("orc_conv_fwd_raw", "orc_conv_bwd_data_raw", "orc_conv_bwd_weight_raw"):
            getattr(L, f).argtypes = [P, P, P, P]
            getattr(L, f).restype = None
        L.orc_bn_fwd.argtypes = [P, i32, i64, i64, P, P, P, P, P, P, P, P, P]
        L.orc_bn_bwd.argtypes = [P, i32, P, i32, i64, i64, P, P, P, P, P, P, P, P, P, P, P]
        L.orc_bn_fwd32.argtypes = L.orc_bn_fwd.argtypes
        L.orc_requant_fixed.argtypes = [P, i64, i32, i32, C.c_int, P]
        L.orc_bn_infer.argtypes = [P, i32, i64, i64, P, P, P, P, P, i32, i32, P]
        L.orc_bn_bwd32.argtypes = L.orc_bn_bwd.argtypes
        L.orc_weight_update.argtypes = [P, i64, P, i32, C.c_int, C.c_int, C.c_int, C.c_int, P]
        L.orc_weight_quant.argtypes = [P, i64, C.c_int, C.c_int, P]
        L.orc_maxpool_fwd.argtypes = [P, i64, i64, i64, i64, i64, i64, i64, P]
        L.orc_maxpool_fwd.restype = None
        L.orc_maxpool_bwd_raw.argtypes = [P, P, i64, i64, i64, i64, i64, i64, i64, P]
        L.orc_maxpool_bwd_raw.restype = None
        L.orc_num_threads.restype = C.c_int
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(C.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise OracleError(f"{what}: oracle returned {rc}")


def num_threads():
    return lib().orc_num_threads()


# --------------------------------------------------------------------------
# random numbers for stochastic rounding
# --------------------------------------------------------------------------
def philox4x32_10(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    o = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_p(c), _p(k), _p(o))
    return o


def draw_u64(seed, tensor_id, step, idx):
    return int(lib().orc_draw_u64(seed, tensor_id, step, idx))


# --------------------------------------------------------------------------
# quantizers (Sec. 3.1)
# --------------------------------------------------------------------------
def uq_code(x, k):
    """Eq. 2 on one real number (exact for float32/float64 input)."""
    return int(lib().orc_uq_code_f64(float(x), int(k)))


def quantize_f32(x, k, mode="sq"):
    """float32 tensor -> (int64 codes, exponent); mode 'uq' (Eq. 2) or 'sq' (Eq. 4)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.zeros(x.shape, dtype=np.int64)
    e = np.zeros(1, dtype=np.int32)
    rc = lib().orc_quantize_f32(_p(x), x.size, int(k), {"uq": 0, "sq": 1}[mode], _p(codes), _p(e))
    _check(rc, "quantize_f32")
    return codes, int(e[0])


def quantize_f64(x, k, mode="sq"):
    """float64 tensor -> (int64 codes, exponent), the same rules as quantize_f32."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    codes = np.zeros(x.shape, dtype=np.int64)
    e = np.zeros(1, dtype=np.int32)
    rc = lib().orc_quantize_f64(_p(x), x.size, int(k), {"uq": 0, "sq": 1}[mode], _p(codes), _p(e))
    _check(rc, "quantize_f64")
    return codes, int(e[0])


def requant(acc, in_exp, k, stochastic=False, keep_scale=True, seed=0, tensor_id=0, step=0):
    """SQ (Eq. 4) or RQ (Eq. 5-6) of an integer tensor -> (int64 codes, exponent).
    keep_scale=False drops the magnitude (Eq. 18)."""
    a = np.ascontiguousarray(acc, dtype=np.int64)
    codes = np.zeros(a.shape, dtype=np.int64)
    e = np.zeros(1, dtype=np.int32)
    rc = lib().orc_requant(_p(a), a.size, int(in_exp), int(k), int(bool(stochastic)),
                           int(bool(keep_scale)), int(seed), int(tensor_id), int(step),
                           _p(codes), _p(e))
    _check(rc, "requant")
    return codes, int(e[0])


# --------------------------------------------------------------------------
# convolutions
# --------------------------------------------------------------------------
def conv_out_hw(geom):
    N, H, W, Cc, K, R, S, sh, sw, ph, pw, dh, dw = geom
    P = (H + 2 * ph - dh * (R - 1) - 1) // sh + 1
    Q = (W + 2 * pw - dw * (S - 1) - 1) // sw + 1
    return P, Q


def _geom(geom):
    return np.asarray(geom, dtype=np.int64)


# Large convolutions take their exact sums from a library routine instead of
# the plain loops of the C file: torch's float64 CPU convolution (unfold and a
# dgemm, or its transpose) adds integer products, and every partial sum here
# stays below 2^53 (at most 2^22 pixels times 127^2), so each addition is
# exact whatever the order.  The C loops are pinned to the same routine on
# small shapes; this only saves time at the workloads' full sizes.
LIBRARY_CONV_MACS = 1 << 26


def _conv_macs(geom):
    N, H, W, Cc, K, R, S = geom[:7]
    P, Q = conv_out_hw(geom)
    return N * P * Q * K * R * S * Cc


def _nchw(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).permute(0, 3, 1, 2).contiguous()


def _nhwc_int(t):
    return t.permute(0, 2, 3, 1).contiguous().numpy().astype(np.int64)


def _library_conv(which, a, b, geom):
    import torch
    import torch.nn.functional as F
    N, H, W, Cc, K, R, S, sh, sw, ph, pw, dh, dw = [int(v) for v in geom]
    kw = dict(stride=(sh, sw), padding=(ph, pw), dilation=(dh, dw))
    with torch.no_grad():
        if which == "fwd":
            return _nhwc_int(F.conv2d(_nchw(a), _nchw(b), **kw))
        if which == "data":
            return _nhwc_int(torch.nn.grad.conv2d_input((N, Cc, H, W), _nchw(b), _nchw(a), **kw))
        dwt = torch.nn.grad.conv2d_weight(_nchw(b), (K, Cc, R, S), _nchw(a), **kw)
        return dwt.permute(0, 2, 3, 1).contiguous().numpy().astype(np.int64)


def conv_fwd_raw(x, w, geom):
    """Exact integer forward sums (NHWC x, KRSC w) -> int64 NPQK."""
    N, H, W, Cc, K, R, S = geom[:7]
    P, Q = conv_out_hw(geom)
    if _conv_macs(geom) >= LIBRARY_CONV_MACS:
        return _library_conv("fwd", x, w, geom)
    x = np.ascontiguousarray(x, dtype=np.int8)
    w = np.ascontiguousarray(w, dtype=np.int8)
    out = np.zeros((N, P, Q, K), dtype=np.int64)
    lib().orc_conv_fwd_raw(_p(x), _p(w), _p(_geom(geom)), _p(out))
    return out


def conv_bwd_data_raw(dy, w, geom):
    N, H, W, Cc = geom[:4]
    if _conv_macs(geom) >= LIBRARY_CONV_MACS:
        return _library_conv("data", dy, w, geom)
    dy = np.ascontiguousarray(dy, dtype=np.int8)
    w = np.ascontiguousarray(w, dtype=np.int8)
    out = np.zeros((N, H, W, Cc), dtype=np.int64)
    lib().orc_conv_bwd_data_raw(_p(dy), _p(w), _p(_geom(geom)), _p(out))
    return out


def conv_bwd_weight_raw(dy, x, geom):
    K, R, S, Cc = geom[4], geom[5], geom[6], geom[3]
    if _conv_macs(geom) >= LIBRARY_CONV_MACS:
        return _library_conv("weight", dy, x, geom)
    dy = np.ascontiguousarray(dy, dtype=np.int8)
    x = np.ascontiguousarray(x, dtype=np.int8)
    out = np.zeros((K, R, S, Cc), dtype=np.int64)
    lib().orc_conv_bwd_weight_raw(_p(dy), _p(x), _p(_geom(geom)), _p(out))
    return out


def conv_fwd(x, x_exp, w, w_exp, geom, k_A=8):
    """Conv forward then SQ to k_A bits (activation quantizer on the MAC output)."""
    acc = conv_fwd_raw(x, w, geom)
    return requant(acc, x_exp + w_exp, k_A)


def conv_bwd_data(dy, dy_exp, w, w_exp, geom, k_E1=8):
    """Backward-data sums then Q_E = SQ(., k_E1) (Eq. 16)."""
    acc = conv_bwd_data_raw(dy, w, geom)
    return requant(acc, dy_exp + w_exp, k_E1)


def conv_bwd_weight(dy, dy_exp, x, x_exp, geom, k_G=8, keep_scale=True, seed=0,
                    tensor_id=0, step=0):
    """Backward-weight sums then Q_G: stochastic RQ (Eq. 17, or Eq. 18 when
    keep_scale=False)."""
    acc = conv_bwd_weight_raw(dy, x, geom)
    return requant(acc, dy_exp + x_exp, k_G, stochastic=True, keep_scale=keep_scale,
                   seed=seed, tensor_id=tensor_id, step=step)


# --------------------------------------------------------------------------
# L1 batch normalization (Eq. 12-15) and its backward
# --------------------------------------------------------------------------
def _bn_cfg(cfg):
    d = dict(BN_DEFAULT)
    if cfg:
        d.update(cfg)
    return np.asarray([d[k] for k in _BN_KEYS], dtype=np.int32)


def bn_fwd(x, x_exp, gamma_q, beta_q, cfg=None):
    """x: int8 codes [..., C] (NHWC), or int32 raw conv sums (the wide input
    of the literal dataflow, Sec. 3.2.2-3.2.3).  Returns dict with A codes
    (int8), exponent, n_mu, n_sigma (per channel), b (exponent of Q_xhat's
    scale) and the per-element xhat codes."""
    wide = np.asarray(x).dtype == np.int32
    x = np.ascontiguousarray(x, dtype=np.int32 if wide else np.int8)
    Cc = x.shape[-1]
    M = x.size // Cc
    g = np.ascontiguousarray(gamma_q, dtype=np.int8)
    b = np.ascontiguousarray(beta_q, dtype=np.int8)
    out = np.zeros(x.shape, dtype=np.int8)
    e = np.zeros(1, dtype=np.int32)
    n_mu = np.zeros(Cc, dtype=np.int32)
    n_sig = np.zeros(Cc, dtype=np.int32)
    bx = np.zeros(1, dtype=np.int32)
    nxh = np.zeros(x.shape, dtype=np.int16)
    f = lib().orc_bn_fwd32 if wide else lib().orc_bn_fwd
    rc = f(_p(x), int(x_exp), M, Cc, _p(g), _p(b), _p(_bn_cfg(cfg)),
                          _p(out), _p(e), _p(n_mu), _p(n_sig), _p(bx), _p(nxh))
    _check(rc, "bn_fwd")
    return dict(y=out, y_exp=int(e[0]), n_mu=n_mu, n_sigma=n_sig, b=int(bx[0]), xhat=nxh)


def bn_bwd(dA, dA_exp, x, x_exp, gamma_q, beta_q, cfg=None, want_pre=False):
    """Backward of L1BN (+ReLU).  Returns dict with dx codes, exponent, raw
    dgamma/dbeta sums and their exponents; dx_pre (float64 value of dx before
    its quantizer) and the count of channels whose pre-quantizer dx does not
    sum to exactly zero.  x int8 codes or int32 raw sums, as in bn_fwd."""
    wide = np.asarray(x).dtype == np.int32
    x = np.ascontiguousarray(x, dtype=np.int32 if wide else np.int8)
    dA = np.ascontiguousarray(dA, dtype=np.int8)
    Cc = x.shape[-1]
    M = x.size // Cc
    g = np.ascontiguousarray(gamma_q, dtype=np.int8)
    b = np.ascontiguousarray(beta_q, dtype=np.int8)
    dx = np.zeros(x.shape, dtype=np.int8)
    e = np.zeros(1, dtype=np.int32)
    dg = np.zeros(Cc, dtype=np.int64)
    db = np.zeros(Cc, dtype=np.int64)
    dge = np.zeros(1, dtype=np.int32)
    dbe = np.zeros(1, dtype=np.int32)
    pre = np.zeros(x.shape, dtype=np.float64) if want_pre else None
    zf = np.zeros(1, dtype=np.int64)
    f = lib().orc_bn_bwd32 if wide else lib().orc_bn_bwd
    rc = f(_p(dA), int(dA_exp), _p(x), int(x_exp), M, Cc, _p(g), _p(b),
                          _p(_bn_cfg(cfg)), _p(dx), _p(e), _p(dg), _p(db), _p(dge), _p(dbe),
                          _p(pre) if want_pre else None, _p(zf))
    _check(rc, "bn_bwd")
    return dict(dx=dx, dx_exp=int(e[0]), dgamma=dg, dbeta=db, dgamma_exp=int(dge[0]),
                dbeta_exp=int(dbe[0]), dx_pre=pre, zero_sum_failures=int(zf[0]))


# --------------------------------------------------------------------------
# inference with frozen statistics and scales
# --------------------------------------------------------------------------
def requant_fixed(acc, acc_exp, out_exp, k=8):
    """Codes of the integer tensor acc 2^acc_exp on the fixed grid 2^out_exp:
    clamp(floor(acc 2^(acc_exp - out_exp) + 1/2)) to k bits."""
    a = np.ascontiguousarray(acc, dtype=np.int64)
    codes = np.zeros(a.shape, dtype=np.int64)
    rc = lib().orc_requant_fixed(_p(a), a.size, int(acc_exp), int(out_exp), int(k), _p(codes))
    _check(rc, "requant_fixed")
    return codes


def bn_state(fwd):
    """The inference state of a layer from a calibration forward's result
    (bn_fwd): per-channel n_mu, n_sigma, Q_xhat's exponent b and Q_A's exponent."""
    return dict(n_mu=np.asarray(fwd["n_mu"], np.int32), n_sigma=np.asarray(fwd["n_sigma"], np.int32),
                b=int(fwd["b"]), a_exp=int(fwd["y_exp"]))


def bn_infer(x, x_exp, gamma_q, beta_q, state, cfg=None):
    """L1BN (+ReLU) + Q_A of int8 codes with the frozen state of bn_state()."""
    x = np.ascontiguousarray(x, dtype=np.int8)
    Cc = x.shape[-1]
    M = x.size // Cc
    out = np.zeros(x.shape, dtype=np.int8)
    rc = lib().orc_bn_infer(_p(x), int(x_exp), M, Cc, _p(np.ascontiguousarray(gamma_q, dtype=np.int8)),
                            _p(np.ascontiguousarray(beta_q, dtype=np.int8)), _p(_bn_cfg(cfg)),
                            _p(state["n_mu"]), _p(state["n_sigma"]), int(state["b"]), int(state["a_exp"]),
                            _p(out))
    _check(rc, "bn_infer")
    return out


# --------------------------------------------------------------------------
# update (Eq. 19) and weight quantizer (Eq. 8)
# --------------------------------------------------------------------------
def weight_update(master, g_codes, g_exp, lr_shift, master_exp=-23, k_U=24, k_W=8):
    """Returns (new master codes int32, new W_q codes int8); master is not modified."""
    m = np.array(master, dtype=np.int32, copy=True).ravel()
    g = np.ascontiguousarray(g_codes, dtype=np.int8).ravel()
    wq = np.zeros(m.shape, dtype=np.int8)
    rc = lib().orc_weight_update(_p(m), m.size, _p(g), int(g_exp), int(lr_shift),
                                 int(master_exp), int(k_U), int(k_W), _p(wq))
    _check(rc, "weight_update")
    shape = np.shape(master)
    return m.reshape(shape), wq.reshape(shape)


def weight_quant(master, k_U=24, k_W=8):
    m = np.ascontiguousarray(master, dtype=np.int32)
    wq = np.zeros(m.shape, dtype=np.int8)
    rc = lib().orc_weight_quant(_p(m), m.size, int(k_U), int(k_W), _p(wq))
    _check(rc, "weight_quant")
    return wq


def master_init(w_float, k_U=24):
    """Eq. 7: W_m = UQ(W, k_U) -> int32 codes with exponent 1-k_U."""
    codes, e = quantize_f32(w_float, k_U, mode="uq")
    return codes.astype(np.int32), e


# --------------------------------------------------------------------------
# max pooling
# --------------------------------------------------------------------------
def maxpool_fwd(x, k, stride, pad):
    x = np.ascontiguousarray(x, dtype=np.int8)
    N, H, W, Cc = x.shape
    P = (H + 2 * pad - k) // stride + 1
    Q = (W + 2 * pad - k) // stride + 1
    y = np.zeros((N, P, Q, Cc), dtype=np.int8)
    lib().orc_maxpool_fwd(_p(x), N, H, W, Cc, k, stride, pad, _p(y))
    return y


def maxpool_bwd_raw(dy, x, k, stride, pad):
    """Routes each output error to its forward maximum; overlaps add exactly."""
    x = np.ascontiguousarray(x, dtype=np.int8)
    dy = np.ascontiguousarray(dy, dtype=np.int8)
    N, H, W, Cc = x.shape
    raw = np.zeros(x.shape, dtype=np.int64)
    lib().orc_maxpool_bwd_raw(_p(dy), _p(x), N, H, W, Cc, k, stride, pad, _p(raw))
    return raw


def maxpool_bwd(dy, dy_exp, x, k, stride, pad, k_E1=8):
    """Routed errors, then Q_E (Eq. 16)."""
    return requant(maxpool_bwd_raw(dy, x, k, stride, pad), dy_exp, k_E1)


# --------------------------------------------------------------------------
# merges of quantized tensors (residual add, ASPP concat, pooling branch)
# --------------------------------------------------------------------------
# A merge takes int8 tensors a_i with exponents e_i, forms the exact real
# result on the grid 2^min(e_i) and applies one quantizer to it: every tensor
# the dataflow carries is an 8-bit object with one scale (Sec. 3.1), so a sum
# or a concatenation of such objects is requantized as a new object (Eq. 4,
# or Eq. 16 for errors).  Exponent gaps above MAX_GAP are rejected so that the
# aligned terms stay far inside int64.
MAX_GAP = 48


def _align(tensors, exps):
    e0 = min(int(e) for e in exps)
    if max(int(e) for e in exps) - e0 > MAX_GAP:
        raise OracleError("merge: exponent gap above %d" % MAX_GAP)
    return [np.asarray(t, dtype=np.int64) * (np.int64(1) << np.int64(int(e) - e0))
            for t, e in zip(tensors, exps)], e0


def exact_sum(tensors, exps):
    """Exact sum of code tensors (value = code 2^e) on the grid 2^min(e);
    a [N,1,1,C] term is broadcast over the spatial axes."""
    terms, e0 = _align(tensors, exps)
    shape = np.broadcast_shapes(*[t.shape for t in terms])
    s = np.zeros(shape, dtype=np.int64)
    for t in terms:
        s = s + t
    return s, e0


def sum_requant(tensors, exps, k=8, relu=False):
    """SQ_k(ReLU?(sum_i a_i 2^e_i)): residual add (with the ReLU that follows
    it) and the sum of the errors a tensor receives from several consumers."""
    s, e0 = exact_sum(tensors, exps)
    if relu:
        s = np.maximum(s, 0)
    return requant(s, e0, k)


def relu_mask_bwd(dy, tensors, exps):
    """Backward of ReLU(sum_i a_i 2^e_i): dy where the exact sum is > 0, else 0
    (the values stay on dy's grid, so dy's exponent is kept)."""
    s, _ = exact_sum(tensors, exps)
    return np.where(s > 0, np.asarray(dy, dtype=np.int64), 0).astype(np.int8)


def concat_requant(tensors, exps, spatial=None, k=8):
    """SQ_k of the channel concatenation of a_i 2^e_i (one object, one scale).
    A [N,1,1,C] part is broadcast to `spatial` = (H, W) first."""
    terms, e0 = _align(tensors, exps)
    if spatial is not None:
        terms = [np.broadcast_to(t, t.shape[:1] + tuple(spatial) + t.shape[3:]) for t in terms]
    return requant(np.concatenate(terms, axis=-1), e0, k)


def concat_split(dy, widths):
    """Backward of a concatenation: the channel slices of dy, dy's exponent."""
    out, c0 = [], 0
    for w in widths:
        out.append(np.ascontiguousarray(dy[..., c0:c0 + w]))
        c0 += w
    return out


def mean_requant(sums, exp, divisor, k=8):
    """SQ_k of the rationals sums * 2^exp / divisor (Eq. 4 with the
    power-of-two Scale): b = the smallest integer with max|value| < 2^b,
    code = floor(value 2^(k-1-b) + 1/2) decided exactly, exponent b + 1 - k.
    All-zero sums keep exponent exp - ceil(log2 divisor).  For a power-of-two
    divisor this is SQ of the integer tensor `sums` on the grid 2^(exp - t)."""
    s = [int(v) for v in np.ravel(sums)]
    D = int(divisor)
    M = max((abs(v) for v in s), default=0)
    if M == 0:
        return np.zeros(np.shape(sums), np.int64), exp - (D - 1).bit_length()
    u = 0                     # smallest u with M < D 2^u
    while not (M < D * 2 ** u if u >= 0 else M * 2 ** -u < D):
        u += 1
    while (M < D * 2 ** (u - 1) if u - 1 >= 0 else M * 2 ** (1 - u) < D):
        u -= 1
    sh = k - 1 - u
    lim = 2 ** (k - 1) - 1
    codes = []
    for v in s:
        num, den = (v * 2 ** sh, D) if sh >= 0 else (v, D * 2 ** -sh)
        c = (2 * num + den) // (2 * den)          # floor(num/den + 1/2)
        codes.append(max(-lim, min(lim, c)))
    return np.array(codes, np.int64).reshape(np.shape(sums)), exp + u + 1 - k


def gap_fwd(x, x_exp, k=8):
    """Global average pooling over H x W: the exact mean sum / (H W) of the
    codes at exponent x_exp, then SQ_k -> [N,1,1,C]."""
    N, H, W, Cc = x.shape
    s = np.asarray(x, dtype=np.int64).sum(axis=(1, 2), keepdims=True)
    return mean_requant(s, x_exp, H * W, k)


def gap_bwd(dy, dy_exp, H, W, k=8):
    """Backward of the mean: every input position receives dy / (H W); Q_E =
    SQ_k of that [N,1,1,C] value, broadcast over H x W by the consumer (for a
    power-of-two H W the values are kept exactly)."""
    return mean_requant(np.asarray(dy, dtype=np.int64), dy_exp, H * W, k)


def bcast_bwd(dy, dy_exp, k=8):
    """Backward of broadcasting a [N,1,1,C] tensor over H x W: the exact
    spatial sum of the error, then Q_E = SQ_k (Eq. 16)."""
    s = np.asarray(dy, dtype=np.int64).sum(axis=(1, 2), keepdims=True)
    return requant(s, dy_exp, k)


# --------------------------------------------------------------------------
# float region of the segmentation loss (float64)
# --------------------------------------------------------------------------
def bilinear_matrix(n_in, n_out):
    """[n_out, n_in] matrix of 1-D linear interpolation with half-pixel
    centres (source coordinate (o + 1/2) n_in / n_out - 1/2, clamped at 0;
    the upper neighbour clamped at n_in - 1)."""
    A = np.zeros((n_out, n_in), dtype=np.float64)
    for o in range(n_out):
        src = (o + 0.5) * n_in / n_out - 0.5
        if src < 0:
            src = 0.0
        i0 = int(np.floor(src))
        i1 = min(i0 + 1, n_in - 1)
        lam = src - i0
        A[o, i0] += 1.0 - lam
        A[o, i1] += lam
    return A


def mse_onehot(y, y_exp, labels, k=8):
    """MSE loss of the network output against one-hot labels (the FCN8s
    loss): L = mean over the N H W K elements of (y - t)^2, t = [k ==
    label], in float64; and E1 = SQ_k of its gradient 2 (y - t) / (N H W K)
    (Eq. 4 / 16), decided exactly: with g = min(y_exp, 0) every y - t is an
    integer V on the grid 2^g, and the gradient is V 2^(g+1) / (N H W K).
    Returns (loss, codes, exponent)."""
    y = np.asarray(y, dtype=np.int64)
    N, H, W, K = y.shape
    lab = np.asarray(labels, dtype=np.int64)
    if lab.shape != (N, H, W) or lab.min(initial=0) < 0 or lab.max(initial=0) >= K:
        raise OracleError("mse_onehot: labels must be [N, H, W] in [0, K)")
    g = min(int(y_exp), 0)
    t = (np.arange(K)[None, None, None, :] == lab[..., None]).astype(np.int64)
    V = y * (1 << (int(y_exp) - g)) - t * (1 << (-g))
    D = N * H * W * K
    loss = float((V.astype(np.float64) ** 2).sum()) * 2.0 ** (2 * g) / D
    codes, e = mean_requant(V, g + 1, D, k)
    return loss, codes, e


LOGIT_EXP_MIN, LOGIT_EXP_MAX = -1000, 0


def softmax_ce(logits, logit_exp, labels):
    """Pixel-wise softmax cross-entropy of the bilinearly upsampled logits.
    logits: int codes [N,h,w,K] with exponent logit_exp; labels [N,H,W] in
    [0, K).  Returns (mean loss, d loss / d logits as float64 [N,h,w,K]).
    The region's domain is logit_exp in [-1000, 0] (|logit| < 128); outside
    it the call is rejected, as the GPU flags it."""
    if not (LOGIT_EXP_MIN <= int(logit_exp) <= LOGIT_EXP_MAX):
        raise OracleError("softmax_ce: logit exponent %d outside [%d, %d]"
                          % (int(logit_exp), LOGIT_EXP_MIN, LOGIT_EXP_MAX))
    N, h, w, K = logits.shape
    _, H, W = labels.shape
    Ay, Ax = bilinear_matrix(h, H), bilinear_matrix(w, W)
    x = np.asarray(logits, dtype=np.float64) * 2.0 ** logit_exp
    loss = 0.0
    grad = np.zeros((N, h, w, K), dtype=np.float64)
    P = N * H * W
    for n in range(N):
        up = np.einsum("yi,ijk,xj->yxk", Ay, x[n], Ax, optimize=True)   # [H, W, K]
        m = up.max(axis=-1, keepdims=True)
        z = np.exp(up - m)
        s = z.sum(axis=-1, keepdims=True)
        lab = labels[n].astype(np.int64)
        logp = (up - m - np.log(s))
        loss -= np.take_along_axis(logp, lab[..., None], axis=-1).sum()
        g = z / s
        np.put_along_axis(g, lab[..., None], np.take_along_axis(g, lab[..., None], -1) - 1.0, -1)
        g /= P
        grad[n] = np.einsum("yi,yxk,xj->ijk", Ay, g, Ax, optimize=True)
    return loss / P, grad
