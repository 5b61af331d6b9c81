"""Python binding of libiseg.so (ctypes).

The `iseg_*` functions here carry the C ABI's names and arguments one to one:
they only turn torch tensors into device pointers, pass the current HIP
stream, and raise on a non-zero status.  Every computation runs in the HIP
kernels; there is no fallback.  The helpers below them (conv_fwd, bn_fwd, ...)
allocate outputs and workspaces with torch and call those entry points.

A quantized tensor is a pair (codes, exp): integer codes and a 1-element int32
device tensor holding the power-of-two exponent (value = code * 2^exp).
"""
import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libiseg.so")

ISEG_OK, ISEG_ERR_ARG, ISEG_ERR_SHAPE, ISEG_ERR_UNSUPPORTED, ISEG_ERR_WORKSPACE, ISEG_ERR_DEVICE = range(6)
ISEG_DEV_RANGE, ISEG_DEV_NONFINITE, ISEG_DEV_DESC = 1, 4, 8
ISEG_I8, ISEG_I16, ISEG_I32, ISEG_I64 = range(4)
ISEG_Q_UQ, ISEG_Q_SQ = 0, 1
ISEG_OUT_Q8, ISEG_OUT_RAW = 0, 1
ISEG_G_KEEP, ISEG_G_DROP, ISEG_G_RAW = 0, 1, 2
(ISEG_KID_NONE, ISEG_KID_CONV_FWD, ISEG_KID_CONV_BWD_DATA, ISEG_KID_CONV_WGRAD, ISEG_KID_REQUANT,
 ISEG_KID_BN_FWD_APPLY, ISEG_KID_BN_BWD_APPLY, ISEG_KID_BN_FWD_STATS1, ISEG_KID_BN_FWD_STATS2,
 ISEG_KID_BN_BWD_STATS, ISEG_KID_MAXPOOL_BWD) = range(11)

_ERRS = {1: "ISEG_ERR_ARG", 2: "ISEG_ERR_SHAPE", 3: "ISEG_ERR_UNSUPPORTED",
         4: "ISEG_ERR_WORKSPACE", 5: "ISEG_ERR_DEVICE"}


class IsegError(RuntimeError):
    pass


class ConvGeom(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("N", "H", "W", "C", "K", "R", "S")] + \
               [(n, C.c_int32) for n in ("stride_h", "stride_w", "pad_h", "pad_w", "dil_h", "dil_w")]


class UpdateDesc(C.Structure):
    _fields_ = [("master", C.c_void_p), ("w_q", C.c_void_p), ("g", C.c_void_p), ("g_exp", C.c_void_p),
                ("g_q", C.c_void_p), ("g_q_exp", C.c_void_p), ("n", C.c_int64), ("kind", C.c_int32),
                ("master_exp", C.c_int32), ("tensor_id", C.c_uint32), ("k_w", C.c_int32)]


ISEG_UPD_CODES, ISEG_UPD_RAW = 0, 1


class WtDesc(C.Structure):
    _fields_ = [("w", C.c_void_p), ("wt", C.c_void_p), ("K", C.c_int32), ("RS", C.c_int32), ("C", C.c_int32),
                ("kind", C.c_int32), ("tile_begin", C.c_int64)]


ISEG_WT_NONE, ISEG_WT_CRSK, ISEG_WT_CRSK_FLIP = 0, 1, 2


class BnCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("k_mu", "k_sigma", "k_xhat", "k_gamma", "k_beta",
                                         "k_A", "k_E1", "k_E2", "eps_code", "relu")]


BN_DEFAULT = dict(k_mu=16, k_sigma=16, k_xhat=16, k_gamma=8, k_beta=8, k_A=8, k_E1=8, k_E2=16,
                  eps_code=0, relu=1)

_lib = None
_P, _I64, _I32, _U64, _U32, _SZ = C.c_void_p, C.c_int64, C.c_int32, C.c_uint64, C.c_uint32, C.c_size_t

_SIGS = {
    "iseg_quantize_ws": ([_I64], _SZ),
    "iseg_quantize": ([_P, _I64, _I32, _I32, _I32, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_requant_ws": ([_I64], _SZ),
    "iseg_requant": ([_P, _I32, _I64, _P, _I32, _I32, _I32, _U64, _U32, _U32, _I32, _P, _P, _P, _SZ,
                      _P, _P], C.c_int),
    "iseg_conv_fwd_ws": ([_P, _I32], _SZ),
    "iseg_conv_fwd": ([_P, _P, _P, _P, _P, _I32, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_conv_bwd_data_ws": ([_P, _I32], _SZ),
    "iseg_conv_bwd_data": ([_P, _P, _P, _P, _P, _I32, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_conv_bwd_data_t": ([_P, _P, _P, _P, _P, _I32, _P, _I32, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_conv_bwd_data_wt_kind": ([_P], C.c_int32),
    "iseg_weight_transpose_multi": ([_P, _I32, _I64, _P], C.c_int),
    "iseg_conv_bwd_weight_ws": ([_P, _I32], _SZ),
    "iseg_conv_bwd_weight": ([_P, _P, _P, _P, _P, _I32, _I32, _U64, _U32, _U32, _P, _P, _P, _SZ,
                              _P, _P], C.c_int),
    "iseg_bn_saved_bytes": ([_I64], _SZ),
    "iseg_bn_fwd_ws": ([_I64, _I64], _SZ),
    "iseg_bn_fwd": ([_P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_bn_fwd_noalloc_max_bytes": ([], _SZ),
    "iseg_bn_fwd_noalloc": ([_P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P], C.c_int),
    "iseg_bn_bwd_ws": ([_I64, _I64], _SZ),
    "iseg_bn_infer": ([_P, _P, _I64, _I64, _P, _P, _P, _P, _P], C.c_int),
    "iseg_conv_bn_infer_ws": ([_P], _SZ),
    "iseg_conv_bn_infer": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_bn_i32_saved_bytes": ([_I64], _SZ),
    "iseg_bn_fwd_i32_ws": ([_I64, _I64], _SZ),
    "iseg_bn_fwd_i32": ([_P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_bn_bwd_i32_ws": ([_I64, _I64], _SZ),
    "iseg_bn_bwd_i32": ([_P, _P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P],
                        C.c_int),
    "iseg_bn_bwd": ([_P, _P, _P, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P],
                    C.c_int),
    "iseg_weight_update": ([_P, _I64, _P, _P, _I32, _I32, _I32, _I32, _P, _P, _P], C.c_int),
    "iseg_weight_quant": ([_P, _I64, _I32, _I32, _P, _P], C.c_int),
    "iseg_maxpool_fwd": ([_P, _P, _I64, _I64, _I64, _I64, _I32, _I32, _I32, _P, _P, _P], C.c_int),
    "iseg_maxpool_bwd_ws": ([_I64, _I64, _I64, _I64], _SZ),
    "iseg_maxpool_bwd": ([_P, _P, _P, _I64, _I64, _I64, _I64, _I32, _I32, _I32, _I32, _P, _P, _P,
                          _SZ, _P, _P], C.c_int),
    "iseg_bn_param_update": ([_P, _P, _P, _P, _I64, _I32, _U64, _U32, _U32, _U32, _I32, _I32, _I32,
                              _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P], C.c_int),
    "iseg_sum_requant_ws": ([_I64, _I64, _I64], _SZ),
    "iseg_sum_requant": ([_I32, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _I32, _P, _P, _P, _SZ, _P, _P],
                         C.c_int),
    "iseg_relu_mask_bwd": ([_P, _I32, _P, _P, _P, _I64, _I64, _P, _P, _P], C.c_int),
    "iseg_sum_requant_relu_mask": ([_I32, _P, _P, _P, _I64, _I64, _I64, _I32, _I32, _P, _P, _P, _P, _P, _SZ,
                                    _P, _P], C.c_int),
    "iseg_concat_requant_ws": ([_I32], _SZ),
    "iseg_concat_requant": ([_I32, _P, _P, _P, _P, _I64, _I64, _I32, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_concat_split": ([_P, _I64, _I32, _P, _P, _P], C.c_int),
    "iseg_spatial_sum_ws": ([_I64, _I64, _I64], _SZ),
    "iseg_spatial_sum": ([_P, _P, _I64, _I64, _I64, _I64, _I64, _I64, _I32, _P, _P, _P, _SZ, _P, _P],
                         C.c_int),
    "iseg_softmax_ce_ws": ([_I64, _I64, _I64, _I64, _I64, _I64], _SZ),
    "iseg_softmax_ce": ([_P, _P, _P, _I64, _I64, _I64, _I64, _I64, _I64, _I32, _P, _P, _P, _P, _P, _SZ,
                         _P, _P], C.c_int),
    "iseg_mse_onehot_ws": ([_I64], _SZ),
    "iseg_mse_onehot": ([_P, _P, _P, _I64, _I64, _I64, _I64, _I32, _P, _P, _P, _P, _SZ, _P, _P], C.c_int),
    "iseg_update_multi": ([_P, _I32, _I32, _U64, _U32, _I32, _I32, _I32, _P, _P], C.c_int),
    "iseg_philox4x32_10": ([_P, _P, _P], None),
    "iseg_profile_arm": ([_I32, _P, _P], C.c_int),
    "iseg_conv_last_plan": ([], C.c_char_p),
    "iseg_status_read": ([_P, _P, _P], C.c_int),
    "iseg_status_clear": ([_P, _P], C.c_int),
    "iseg_check_codes": ([_P, _I64, _I32, _P, _P], C.c_int),
    "iseg_version": ([], C.c_char_p),
    "iseg_tape_create": ([], _P),
    "iseg_tape_destroy": ([_P], None),
    "iseg_tape_entry": ([C.c_char_p], C.c_int),
    "iseg_tape_entry_nargs": ([C.c_int], C.c_int),
    "iseg_tape_add_call": ([_P, C.c_int, _P, C.c_int, _P, _SZ, _P, C.c_int, _I32, _I64], C.c_int),
    "iseg_tape_add_record": ([_P, _I32, _P], C.c_int),
    "iseg_tape_add_wait": ([_P, _P, _I32], C.c_int),
    "iseg_tape_arm_count": ([_P], C.c_int),
    "iseg_tape_set_arm_events": ([_P, _P, _I32], C.c_int),
    "iseg_tape_run": ([_P, _U32, _P], C.c_int),
    "iseg_tape_size": ([_P], _I64),
}


def lib():
    """Load libiseg.so; raises if it has not been built (no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libiseg.so not built at {LIB_PATH}; run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    if _REC is not None:
        return _REC.lib
    return _lib


def _ptr(t):
    if t is None:
        return None
    if _REC is not None:
        _REC.keep.append(t)          # a recorded call's buffer stays allocated
    return C.c_void_p(t.data_ptr())


_raw_stream = torch._C._cuda_getCurrentRawStream if hasattr(torch._C, "_cuda_getCurrentRawStream") else None
_raw_device = torch._C._cuda_getDevice if hasattr(torch._C, "_cuda_getDevice") else torch.cuda.current_device


def _stream_handle(dev_index=None):
    """Raw handle of the current stream of a device (the current device by
    default): the launch path asks for it on every call, so it bypasses the
    Stream object construction of torch.cuda.current_stream()."""
    if dev_index is None:
        dev_index = _raw_device()
    if _raw_stream is not None:
        return _raw_stream(dev_index)
    return torch.cuda.current_stream(dev_index).cuda_stream


def _stream():
    return C.c_void_p(_stream_handle())


def _check(rc, name):
    if rc != ISEG_OK:
        raise IsegError(f"{name} returned {_ERRS.get(rc, rc)}")


def _ws_tuple(ws):
    return (_ptr(ws), C.c_size_t(ws.numel() if ws is not None else 0))


# --------------------------------------------------------------------------
# entry points, one to one with include/iseg.h
# --------------------------------------------------------------------------
def iseg_quantize(x, bits, mode, out_dtype, out, out_exp, ws, status=None):
    rc = lib().iseg_quantize(_ptr(x), x.numel(), bits, mode, out_dtype, _ptr(out), _ptr(out_exp),
                             *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_quantize")


def iseg_requant(inp, in_dtype, in_exp, bits, stochastic, keep_scale, seed, tensor_id, step,
                 out_dtype, out, out_exp, ws, status=None):
    rc = lib().iseg_requant(_ptr(inp), in_dtype, inp.numel(), _ptr(in_exp), bits, stochastic,
                            keep_scale, seed, tensor_id, step, out_dtype, _ptr(out), _ptr(out_exp),
                            *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_requant")


def iseg_conv_fwd(x, x_exp, w, w_exp, geom, out_mode, y, y_exp, ws, status=None):
    rc = lib().iseg_conv_fwd(_ptr(x), _ptr(x_exp), _ptr(w), _ptr(w_exp), C.byref(geom), out_mode,
                             _ptr(y), _ptr(y_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_conv_fwd")


def iseg_conv_bwd_data(dy, dy_exp, w, w_exp, geom, out_mode, dx, dx_exp, ws, status=None):
    rc = lib().iseg_conv_bwd_data(_ptr(dy), _ptr(dy_exp), _ptr(w), _ptr(w_exp), C.byref(geom),
                                  out_mode, _ptr(dx), _ptr(dx_exp), *_ws_tuple(ws), _ptr(status),
                                  _stream())
    _check(rc, "iseg_conv_bwd_data")


def iseg_conv_bwd_data_t(dy, dy_exp, w, w_exp, wt, wt_kind, geom, out_mode, dx, dx_exp, ws, status=None):
    rc = lib().iseg_conv_bwd_data_t(_ptr(dy), _ptr(dy_exp), _ptr(w), _ptr(w_exp), _ptr(wt), wt_kind,
                                    C.byref(geom), out_mode, _ptr(dx), _ptr(dx_exp), *_ws_tuple(ws),
                                    _ptr(status), _stream())
    _check(rc, "iseg_conv_bwd_data_t")


def iseg_conv_bwd_data_wt_kind(geom):
    return int(lib().iseg_conv_bwd_data_wt_kind(C.byref(geom)))


def iseg_weight_transpose_multi(table, n, total_tiles):
    rc = lib().iseg_weight_transpose_multi(_ptr(table), n, total_tiles, _stream())
    _check(rc, "iseg_weight_transpose_multi")


def iseg_conv_bwd_weight(dy, dy_exp, x, x_exp, geom, g_mode, bits, seed, tensor_id, step, dw,
                         dw_exp, ws, status=None):
    rc = lib().iseg_conv_bwd_weight(_ptr(dy), _ptr(dy_exp), _ptr(x), _ptr(x_exp), C.byref(geom),
                                    g_mode, bits, seed, tensor_id, step, _ptr(dw), _ptr(dw_exp),
                                    *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_conv_bwd_weight")


def iseg_bn_fwd(x, x_exp, M, Cc, gamma_q, beta_q, cfg, y, y_exp, saved, ws, status=None):
    rc = lib().iseg_bn_fwd(_ptr(x), _ptr(x_exp), M, Cc, _ptr(gamma_q), _ptr(beta_q), C.byref(cfg),
                           _ptr(y), _ptr(y_exp), _ptr(saved), *_ws_tuple(ws), _ptr(status),
                           _stream())
    _check(rc, "iseg_bn_fwd")


def iseg_bn_infer(z, z_exp, M, Cc, saved, a, a_exp, status=None):
    rc = lib().iseg_bn_infer(_ptr(z), _ptr(z_exp), M, Cc, _ptr(saved), _ptr(a), _ptr(a_exp), _ptr(status),
                             _stream())
    _check(rc, "iseg_bn_infer")


def iseg_conv_bn_infer(x, x_exp, w, w_exp, geom, saved, a, a_exp, ws, status=None):
    rc = lib().iseg_conv_bn_infer(_ptr(x), _ptr(x_exp), _ptr(w), _ptr(w_exp), C.byref(geom), _ptr(saved),
                                  _ptr(a), _ptr(a_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_conv_bn_infer")


def bn_infer(z, z_exp, saved, status=None):
    """A codes of int8 codes z through a calibration forward's frozen state."""
    Cc = z.shape[-1]
    a = torch.empty_like(z)
    e = _out_exp(z.device)
    iseg_bn_infer(z, z_exp, z.numel() // Cc, Cc, saved, a, e, status)
    return a, e


def conv_bn_infer(x, x_exp, w, w_exp, saved, stride=1, pad=0, dil=1, status=None):
    """Conv + L1BN + ReLU? + Q_A of one layer with a calibration's frozen state."""
    N, H, W, Cc = x.shape
    K, R, S, _ = w.shape
    g = geom(N, H, W, Cc, K, R, S, stride, pad, dil)
    P, Q = conv_out_hw(g)
    a = torch.empty((N, P, Q, K), dtype=torch.int8, device=x.device)
    e = _out_exp(x.device)
    ws = workspace(x.device).get(lib().iseg_conv_bn_infer_ws(C.byref(g)))
    iseg_conv_bn_infer(x, x_exp, w, w_exp, g, saved, a, e, ws, status)
    return a, e


def iseg_bn_fwd_i32(x, x_exp, M, Cc, gamma_q, beta_q, cfg, y, y_exp, saved, ws, status=None):
    rc = lib().iseg_bn_fwd_i32(_ptr(x), _ptr(x_exp), M, Cc, _ptr(gamma_q), _ptr(beta_q), C.byref(cfg),
                               _ptr(y), _ptr(y_exp), _ptr(saved), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_bn_fwd_i32")


def iseg_bn_bwd_i32(dy, dy_exp, x, M, Cc, gamma_q, cfg, saved, dx, dx_exp, dgamma, dbeta, dgamma_exp,
                    dbeta_exp, ws, status=None):
    rc = lib().iseg_bn_bwd_i32(_ptr(dy), _ptr(dy_exp), _ptr(x), M, Cc, _ptr(gamma_q), C.byref(cfg),
                               _ptr(saved), _ptr(dx), _ptr(dx_exp), _ptr(dgamma), _ptr(dbeta),
                               _ptr(dgamma_exp), _ptr(dbeta_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_bn_bwd_i32")


def iseg_bn_fwd_noalloc(x, x_exp, M, Cc, gamma_q, beta_q, cfg, y, y_exp, saved, status=None):
    rc = lib().iseg_bn_fwd_noalloc(_ptr(x), _ptr(x_exp), M, Cc, _ptr(gamma_q), _ptr(beta_q), C.byref(cfg),
                                   _ptr(y), _ptr(y_exp), _ptr(saved), _ptr(status), _stream())
    _check(rc, "iseg_bn_fwd_noalloc")


def iseg_bn_bwd(dy, dy_exp, x, M, Cc, gamma_q, cfg, saved, dx, dx_exp, dgamma, dbeta, dgamma_exp,
                dbeta_exp, ws, status=None):
    rc = lib().iseg_bn_bwd(_ptr(dy), _ptr(dy_exp), _ptr(x), M, Cc, _ptr(gamma_q), C.byref(cfg),
                           _ptr(saved), _ptr(dx), _ptr(dx_exp), _ptr(dgamma), _ptr(dbeta),
                           _ptr(dgamma_exp), _ptr(dbeta_exp), *_ws_tuple(ws), _ptr(status),
                           _stream())
    _check(rc, "iseg_bn_bwd")


def iseg_weight_update(master, g, g_exp, lr_shift, master_exp, k_U, k_W, w_q, status=None):
    rc = lib().iseg_weight_update(_ptr(master), master.numel(), _ptr(g), _ptr(g_exp), lr_shift,
                                  master_exp, k_U, k_W, _ptr(w_q), _ptr(status), _stream())
    _check(rc, "iseg_weight_update")


def iseg_bn_param_update(dgamma, dgamma_exp, dbeta, dbeta_exp, bits, seed, tid_gamma, tid_beta, step,
                         lr_shift, master_exp, k_U, k_W, gamma_m, beta_m, gamma_q, beta_q,
                         g_gamma=None, g_beta=None, g_gamma_exp=None, g_beta_exp=None, status=None):
    rc = lib().iseg_bn_param_update(_ptr(dgamma), _ptr(dgamma_exp), _ptr(dbeta), _ptr(dbeta_exp),
                                    dgamma.numel(), bits, seed, tid_gamma, tid_beta, step, lr_shift,
                                    master_exp, k_U, k_W, _ptr(gamma_m), _ptr(beta_m), _ptr(gamma_q),
                                    _ptr(beta_q), _ptr(g_gamma), _ptr(g_beta), _ptr(g_gamma_exp),
                                    _ptr(g_beta_exp), _ptr(status), _stream())
    _check(rc, "iseg_bn_param_update")


def iseg_update_multi(descs, n_desc, bits, seed, step, lr_shift, k_U, k_W, status=None):
    rc = lib().iseg_update_multi(_ptr(descs), n_desc, bits, seed, step, lr_shift, k_U, k_W, _ptr(status),
                                 _stream())
    _check(rc, "iseg_update_multi")


def iseg_weight_quant(master, k_U, k_W, w_q):
    rc = lib().iseg_weight_quant(_ptr(master), master.numel(), k_U, k_W, _ptr(w_q), _stream())
    _check(rc, "iseg_weight_quant")


def iseg_maxpool_fwd(x, x_exp, k, stride, pad, y, y_exp):
    N, H, W, Cc = x.shape
    rc = lib().iseg_maxpool_fwd(_ptr(x), _ptr(x_exp), N, H, W, Cc, k, stride, pad, _ptr(y),
                                _ptr(y_exp), _stream())
    _check(rc, "iseg_maxpool_fwd")


def iseg_maxpool_bwd(dy, dy_exp, x, k, stride, pad, bits, dx, dx_exp, ws, status=None):
    N, H, W, Cc = x.shape
    rc = lib().iseg_maxpool_bwd(_ptr(dy), _ptr(dy_exp), _ptr(x), N, H, W, Cc, k, stride, pad, bits,
                                _ptr(dx), _ptr(dx_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_maxpool_bwd")


def _ptr_array(ts):
    if _REC is not None:
        _REC.keep.extend(t for t in ts if t is not None)
    return (C.c_void_p * len(ts))(*[None if t is None else t.data_ptr() for t in ts])


def _i32_array(v):
    return (C.c_int32 * len(v))(*[int(x) for x in v])


def _i64_array(v):
    return (C.c_int64 * len(v))(*[int(x) for x in v])


def iseg_sum_requant(ins, in_exps, exp_add, bcast, N, HW, Cc, relu, bits, out, out_exp, ws,
                     status=None):
    n = len(ins)
    rc = lib().iseg_sum_requant(n, _ptr_array(ins), _ptr_array(in_exps),
                                _i32_array(exp_add or [0] * n), _i32_array(bcast or [0] * n),
                                N, HW, Cc, relu, bits, _ptr(out), _ptr(out_exp), *_ws_tuple(ws),
                                _ptr(status), _stream())
    _check(rc, "iseg_sum_requant")


def iseg_sum_requant_relu_mask(ins, in_exps, exp_add, N, HW, Cc, bits, masks, mask_exps, out, out_exp, ws,
                               status=None):
    n = len(ins)
    rc = lib().iseg_sum_requant_relu_mask(n, _ptr_array(ins), _ptr_array(in_exps), _i32_array(exp_add or [0] * n),
                                          N, HW, Cc, bits, len(masks), _ptr_array(masks), _ptr_array(mask_exps),
                                          _ptr(out), _ptr(out_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_sum_requant_relu_mask")


def iseg_relu_mask_bwd(dy, ins, in_exps, exp_add, Cc, dx, status=None):
    n = len(ins)
    rc = lib().iseg_relu_mask_bwd(_ptr(dy), n, _ptr_array(ins), _ptr_array(in_exps),
                                  _i32_array(exp_add or [0] * n), dy.numel(), Cc, _ptr(dx),
                                  _ptr(status), _stream())
    _check(rc, "iseg_relu_mask_bwd")


def iseg_concat_requant(ins, in_exps, widths, bcast, N, HW, bits, out, out_exp, ws, status=None):
    n = len(ins)
    rc = lib().iseg_concat_requant(n, _ptr_array(ins), _ptr_array(in_exps), _i64_array(widths),
                                   _i32_array(bcast or [0] * n), N, HW, bits, _ptr(out),
                                   _ptr(out_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_concat_requant")


def iseg_concat_split(dy, rows, widths, outs):
    rc = lib().iseg_concat_split(_ptr(dy), rows, len(widths), _i64_array(widths), _ptr_array(outs),
                                 _stream())
    _check(rc, "iseg_concat_split")


def iseg_spatial_sum(x, x_exp, N, HW, ldc, c0, Cc, divisor, bits, out, out_exp, ws, status=None):
    rc = lib().iseg_spatial_sum(_ptr(x), _ptr(x_exp), N, HW, ldc, c0, Cc, divisor, bits, _ptr(out),
                                _ptr(out_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_spatial_sum")


def iseg_softmax_ce(logits, logit_exp, labels, N, h, w, K, H, W, bits, loss, grad, err, err_exp,
                    ws, status=None):
    rc = lib().iseg_softmax_ce(_ptr(logits), _ptr(logit_exp), _ptr(labels), N, h, w, K, H, W, bits,
                               _ptr(loss), _ptr(grad), _ptr(err), _ptr(err_exp), *_ws_tuple(ws),
                               _ptr(status), _stream())
    _check(rc, "iseg_softmax_ce")


def iseg_mse_onehot(y, y_exp, labels, bits, loss, err, err_exp, ws, status=None):
    N, H, W, K = y.shape
    rc = lib().iseg_mse_onehot(_ptr(y), _ptr(y_exp), _ptr(labels), N, H, W, K, bits, _ptr(loss), _ptr(err),
                               _ptr(err_exp), *_ws_tuple(ws), _ptr(status), _stream())
    _check(rc, "iseg_mse_onehot")


def mse_onehot(y, y_exp, labels, bits=8, status=None):
    """(loss, E1 codes, exponent) of the MSE loss against one-hot labels."""
    loss = torch.empty(1, dtype=torch.float64, device=y.device)     # written whole by the kernel
    err = torch.empty_like(y)
    e = _out_exp(y.device)
    ws = workspace(y.device).get(lib().iseg_mse_onehot_ws(y.numel()))
    iseg_mse_onehot(y, y_exp, labels, bits, loss, err, e, ws, status)
    return loss, err, e


def iseg_philox4x32_10(ctr, key):
    c = (C.c_uint32 * 4)(*ctr)
    k = (C.c_uint32 * 2)(*key)
    o = (C.c_uint32 * 4)()
    lib().iseg_philox4x32_10(c, k, o)
    return list(o)


def iseg_conv_last_plan():
    return lib().iseg_conv_last_plan().decode()


def iseg_status_read(status):
    v = C.c_int32(0)
    _check(lib().iseg_status_read(_ptr(status), C.byref(v), _stream()), "iseg_status_read")
    return v.value


def iseg_status_clear(status):
    _check(lib().iseg_status_clear(_ptr(status), _stream()), "iseg_status_clear")


def iseg_check_codes(x, bits, status):
    _check(lib().iseg_check_codes(_ptr(x), x.numel(), bits, _ptr(status), _stream()), "iseg_check_codes")


def iseg_version():
    return lib().iseg_version().decode()


def iseg_profile_arm(kernel_id, start_event, stop_event):
    _check(lib().iseg_profile_arm(kernel_id, start_event, stop_event), "iseg_profile_arm")


# --------------------------------------------------------------------------
# in-place kernel timing (HIP events recorded around one kernel launch)
# --------------------------------------------------------------------------
_hip = None


def _hiprt():
    global _hip
    if _hip is None:
        h = C.CDLL("libamdhip64.so")
        h.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        h.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        h.hipEventSynchronize.argtypes = [C.c_void_p]
        h.hipEventDestroy.argtypes = [C.c_void_p]
        _hip = h
    return _hip


class KernelTimer:
    """Times every launch of one or more kernel families whose layer key
    matches, with a pair of HIP events that the library records around the
    launch on its own stream (iseg_profile_arm).  Families timed together
    must be separate entry-point calls (one arming is held at a time)."""

    def __init__(self, kernel_id, layer_match=None):
        self.kids = set(kernel_id) if isinstance(kernel_id, (tuple, list, set)) else {kernel_id}
        self.kid = next(iter(self.kids))
        self.match = tuple(layer_match) if layer_match is not None else None
        self.pairs = []                  # (start, stop, kernel id, layer key)
        self.free = []                   # created events not in use

    def wants(self, kid, key):
        return kid in self.kids and (self.match is None or tuple(key) == self.match)

    def _event(self):
        if self.free:
            return self.free.pop()
        e = C.c_void_p()
        if _hiprt().hipEventCreate(C.byref(e)):
            raise IsegError("hipEventCreate failed")
        return e

    def arm(self, kid=None, key=None):
        a, b = self._event(), self._event()
        kid = self.kid if kid is None else kid
        self.pairs.append((a, b, kid, tuple(key) if key is not None else None))
        iseg_profile_arm(kid, a, b)

    def reset(self):
        """Forget the timed launches and keep their events for the next ones
        (an untimed pass with the timer installed creates the events a timed
        region then reuses, keeping event creation out of it)."""
        h = _hiprt()
        for a, b, _, _ in self.pairs:
            h.hipEventSynchronize(b)
            self.free += [a, b]
        self.pairs = []

    def launches(self):
        """[(kernel id, layer key, ms)] of every timed launch."""
        h = _hiprt()
        out = []
        for a, b, kid, key in self.pairs:
            h.hipEventSynchronize(b)
            ms = C.c_float()
            if h.hipEventElapsedTime(C.byref(ms), a, b) == 0:
                out.append((kid, key, ms.value))
        return out

    def times_ms(self):
        return [t for _, _, t in self.launches()]

    def mean_ms(self):
        t = self.times_ms()
        return sum(t) / len(t) if t else None

    def count(self):
        return len(self.pairs)

    def close(self):
        h = _hiprt()
        for a, b, _, _ in self.pairs:
            h.hipEventDestroy(a)
            h.hipEventDestroy(b)
        for e in self.free:
            h.hipEventDestroy(e)
        self.pairs, self.free = [], []


_TIMER = None


def set_kernel_timer(timer):
    """Install (or remove, with None) the timer consulted by the helpers below."""
    global _TIMER
    if timer is None:
        iseg_profile_arm(ISEG_KID_NONE, None, None)
    _TIMER = timer


def _maybe_arm(kid, key):
    if _TIMER is not None and _TIMER.wants(kid, key):
        _TIMER.arm(kid, key)


# --------------------------------------------------------------------------
# workspace and helpers (allocation with torch; compute in the entry points)
# --------------------------------------------------------------------------
class Workspace:
    """A growable device scratch buffer shared by consecutive calls on one
    stream (stream order keeps the uses apart); each stream has its own.
    `zeroed` buffers start at zero (the BN workspace, whose arrival counters
    every call leaves at zero)."""

    def __init__(self, device="cuda", zeroed=False):
        self.device = device
        self.zeroed = zeroed
        self.buf = None

    def get(self, nbytes):
        nbytes = max(int(nbytes), 256)
        if self.buf is None or self.buf.numel() < nbytes:
            alloc = torch.zeros if self.zeroed else torch.empty
            self.buf = alloc(nbytes, dtype=torch.uint8, device=self.device)
        return self.buf[:nbytes]


_WS = {}


def workspace(device, bn=False):
    """The workspace of the current stream; L1BN (int8 input) has one of its own."""
    d = device if isinstance(device, torch.device) else torch.device(device)
    if d.type == "cuda":
        idx = d.index if d.index is not None else _raw_device()
        key = (idx, _stream_handle(idx), bn)
    else:
        idx, key = None, (str(d), 0, bn)
    ws = _WS.get(key)
    if ws is None:
        ws = _WS[key] = Workspace(torch.device("cuda", idx) if d.type == "cuda" else d, zeroed=bn)
    return ws


# --------------------------------------------------------------------------
# step tape: the calls of one step recorded, then replayed from native code
# --------------------------------------------------------------------------
_REC = None

# parameter index of the step counter (stochastic rounding, Eq. 5-6)
_STEP_ARG = {"iseg_conv_bwd_weight": 9, "iseg_update_multi": 4, "iseg_bn_param_update": 9, "iseg_requant": 9}
_U64_MASK = (1 << 64) - 1


def iseg_tape_create():
    return C.c_void_p(lib().iseg_tape_create())


def iseg_tape_destroy(h):
    lib().iseg_tape_destroy(h)


def iseg_tape_entry(name):
    return int(lib().iseg_tape_entry(name.encode()))


def iseg_tape_entry_nargs(entry):
    return int(lib().iseg_tape_entry_nargs(entry))


def iseg_tape_add_call(h, entry, words, blob, blob_words, step_word, step_base):
    w = (C.c_uint64 * max(len(words), 1))(*words)
    bw = (C.c_int32 * max(len(blob_words), 1))(*blob_words)
    b = (C.c_char * max(len(blob), 1)).from_buffer_copy(bytes(blob) or b"\0")
    _check(lib().iseg_tape_add_call(h, entry, w, len(words), b, len(blob), bw, len(blob_words), step_word,
                                    step_base), "iseg_tape_add_call")


def iseg_tape_add_record(h, slot, stream_handle):
    _check(lib().iseg_tape_add_record(h, slot, C.c_void_p(stream_handle)), "iseg_tape_add_record")


def iseg_tape_add_wait(h, stream_handle, slot):
    _check(lib().iseg_tape_add_wait(h, C.c_void_p(stream_handle), slot), "iseg_tape_add_wait")


def iseg_tape_arm_count(h):
    return int(lib().iseg_tape_arm_count(h))


def iseg_tape_set_arm_events(h, events, runs):
    """events: (start, stop) pairs of hipEvent_t handles, runs x armed calls of them."""
    flat = (C.c_void_p * max(len(events) * 2, 1))(*[e for pair in events for e in pair])
    _check(lib().iseg_tape_set_arm_events(h, flat, runs), "iseg_tape_set_arm_events")


def iseg_tape_run(h, step):
    failed = C.c_int64(-1)
    rc = lib().iseg_tape_run(h, int(step) & 0xFFFFFFFF, C.byref(failed))
    if rc != ISEG_OK:
        raise IsegError(f"iseg_tape_run: operation {failed.value} returned {_ERRS.get(rc, rc)}")


def iseg_tape_size(h):
    return int(lib().iseg_tape_size(h))


class _RecLib:
    """The library as seen while a tape records: each call of a tape entry
    point runs, then is appended to the tape."""

    def __init__(self, tape):
        self._tape = tape

    def __getattr__(self, name):
        f = getattr(_lib, name)
        if not name.startswith("iseg_") or name.startswith("iseg_tape_") or name not in self._tape.entries:
            return f
        tape = self._tape

        def call(*args):
            rc = f(*args)
            if rc == ISEG_OK:
                tape.add_call(name, args)
            return rc
        return call


class Tape:
    """One training step's library calls and stream orderings, recorded while
    the step runs inside `with tape:` (every call of a tape entry point made
    then is appended after it returns ISEG_OK), replayed from native code by
    run(step).  Keeps every buffer the recorded calls use allocated; the
    caller keeps the streams alive and replays with the same stream setup.""" 

    def __init__(self, step):
        L = lib()
        self.h = iseg_tape_create()
        if not self.h.value:
            raise IsegError("iseg_tape_create failed")
        self.step = int(step)
        self.keep = []
        self.slots = 0
        self.arms = []
        self.entries = {n: L.iseg_tape_entry(n.encode()) for n in _SIGS if n.startswith("iseg_")}
        self.entries = {n: e for n, e in self.entries.items() if e >= 0}
        self.lib = _RecLib(self)

    def __enter__(self):
        global _REC
        if _REC is not None:
            raise IsegError("a tape is already recording")
        _REC = self
        return self

    def __exit__(self, *exc):
        global _REC
        _REC = None
        return False

    def add_call(self, name, args):
        argtypes = getattr(_lib, name).argtypes
        words, blob, blob_words = [], bytearray(), []
        for i, a in enumerate(args):
            if a is None:
                words.append(0)
            elif isinstance(a, C.c_void_p):
                words.append(a.value or 0)
            elif type(a).__name__ == "CArgObject" or isinstance(a, C.Array):
                obj = a._obj if type(a).__name__ == "CArgObject" else a
                blob_words.append(i)
                words.append(len(blob))
                blob += C.string_at(C.addressof(obj), C.sizeof(obj))
                blob += bytes(-len(blob) % 8)
            elif isinstance(a, C._SimpleCData):
                words.append(int(a.value) & _U64_MASK)
            elif isinstance(a, int):
                words.append(a & _U64_MASK)
            else:
                raise IsegError(f"{name}: argument {i} of type {type(a).__name__} cannot be recorded")
            if argtypes[i] is not _P and isinstance(a, C.c_void_p):
                raise IsegError(f"{name}: argument {i} is a pointer where an integer is declared")
        sw = _STEP_ARG.get(name, -1)
        base = int(args[sw].value if isinstance(args[sw], C._SimpleCData) else args[sw]) - self.step if sw >= 0 else 0
        if name == "iseg_profile_arm":
            self.arms.append(int(args[0]))
        iseg_tape_add_call(self.h, self.entries[name], words, blob, blob_words, sw, base)

    def new_slot(self):
        self.slots += 1
        return self.slots - 1

    def add_record(self, slot, stream_handle):
        iseg_tape_add_record(self.h, slot, stream_handle)

    def add_wait(self, stream_handle, slot):
        iseg_tape_add_wait(self.h, stream_handle, slot)

    def set_arm_events(self, events, runs):
        """events: runs x (armed calls) (start, stop) pairs of hipEvent_t handles."""
        iseg_tape_set_arm_events(self.h, events, runs)

    def size(self):
        return iseg_tape_size(self.h)

    def run(self, step):
        iseg_tape_run(self.h, step)

    def close(self):
        if self.h is not None and self.h.value:
            iseg_tape_destroy(self.h)
        self.h = None
        self.keep = []

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _out_exp(device):
    """Exponent slot for a kernel to write (no initialization kernel)."""
    return torch.empty(1, dtype=torch.int32, device=device)


def new_exp(device="cuda", value=0):
    return torch.full((1,), int(value), dtype=torch.int32, device=device)


def geom(N, H, W, Cc, K, R, S, stride=1, pad=0, dil=1):
    st = stride if isinstance(stride, (tuple, list)) else (stride, stride)
    pd = pad if isinstance(pad, (tuple, list)) else (pad, pad)
    dl = dil if isinstance(dil, (tuple, list)) else (dil, dil)
    return ConvGeom(N, H, W, Cc, K, R, S, st[0], st[1], pd[0], pd[1], dl[0], dl[1])


def conv_out_hw(g):
    P = (g.H + 2 * g.pad_h - g.dil_h * (g.R - 1) - 1) // g.stride_h + 1
    Q = (g.W + 2 * g.pad_w - g.dil_w * (g.S - 1) - 1) // g.stride_w + 1
    return P, Q


def bn_cfg(**kw):
    d = dict(BN_DEFAULT)
    d.update(kw)
    return BnCfg(*[d[k] for k in ("k_mu", "k_sigma", "k_xhat", "k_gamma", "k_beta", "k_A", "k_E1",
                                  "k_E2", "eps_code", "relu")])


def quantize(x, bits, mode=ISEG_Q_SQ, status=None, out_dtype=None):
    """Codes in the narrowest of int8 / int16 / int32 that holds `bits`, or in
    out_dtype (a torch integer dtype at least that wide)."""
    w = 8 if bits <= 8 else 16 if bits <= 16 else 32
    if out_dtype is not None:
        w = {torch.int8: 8, torch.int16: 16, torch.int32: 32}[out_dtype]
        if (w == 8 and bits > 8) or (w == 16 and bits > 16):
            raise ValueError("out_dtype too narrow for bits")
    dt = {8: (torch.int8, ISEG_I8), 16: (torch.int16, ISEG_I16), 32: (torch.int32, ISEG_I32)}[w]
    out = torch.empty(x.shape, dtype=dt[0], device=x.device)
    e = _out_exp(x.device)
    ws = workspace(x.device).get(lib().iseg_quantize_ws(x.numel()))
    iseg_quantize(x.contiguous(), bits, mode, dt[1], out, e, ws, status)
    return out, e


def requant(acc, acc_exp, bits=8, stochastic=False, keep_scale=True, seed=0, tensor_id=0, step=0,
            status=None):
    in_dt = {torch.int32: ISEG_I32, torch.int64: ISEG_I64}[acc.dtype]
    od, odt = (torch.int8, ISEG_I8) if bits <= 8 else (torch.int16, ISEG_I16)
    out = torch.empty(acc.shape, dtype=od, device=acc.device)
    e = _out_exp(acc.device)
    ws = workspace(acc.device).get(lib().iseg_requant_ws(acc.numel()))
    iseg_requant(acc.contiguous(), in_dt, acc_exp, bits, int(stochastic), int(keep_scale), seed,
                 tensor_id, step, odt, out, e, ws, status)
    return out, e


def conv_fwd(x, x_exp, w, w_exp, stride=1, pad=0, dil=1, out_mode=ISEG_OUT_Q8, status=None):
    N, H, W, Cc = x.shape
    K, R, S, _ = w.shape
    g = geom(N, H, W, Cc, K, R, S, stride, pad, dil)
    P, Q = conv_out_hw(g)
    y = torch.empty((N, P, Q, K), dtype=torch.int8 if out_mode == ISEG_OUT_Q8 else torch.int32,
                    device=x.device)
    e = _out_exp(x.device)
    ws = workspace(x.device).get(lib().iseg_conv_fwd_ws(C.byref(g), out_mode))
    _maybe_arm(ISEG_KID_CONV_FWD, (N, H, W, Cc, K, R, g.stride_h, g.pad_h, g.dil_h))
    iseg_conv_fwd(x, x_exp, w, w_exp, g, out_mode, y, e, ws, status)
    return y, e


def conv_bwd_data(dy, dy_exp, w, w_exp, x_shape, stride=1, pad=0, dil=1, out_mode=ISEG_OUT_Q8,
                  status=None, wt=None, wt_kind=ISEG_WT_NONE):
    N, H, W, Cc = x_shape
    K, R, S, _ = w.shape
    g = geom(N, H, W, Cc, K, R, S, stride, pad, dil)
    dx = torch.empty((N, H, W, Cc), dtype=torch.int8 if out_mode == ISEG_OUT_Q8 else torch.int32,
                     device=dy.device)
    e = _out_exp(dy.device)
    ws = workspace(dy.device).get(lib().iseg_conv_bwd_data_ws(C.byref(g), out_mode))
    _maybe_arm(ISEG_KID_CONV_BWD_DATA, (N, H, W, Cc, K, R, g.stride_h, g.pad_h, g.dil_h))
    if wt is None:
        iseg_conv_bwd_data(dy, dy_exp, w, w_exp, g, out_mode, dx, e, ws, status)
    else:
        iseg_conv_bwd_data_t(dy, dy_exp, w, w_exp, wt, wt_kind, g, out_mode, dx, e, ws, status)
    return dx, e


def conv_bwd_weight(dy, dy_exp, x, x_exp, w_shape, stride=1, pad=0, dil=1, g_mode=ISEG_G_KEEP,
                    bits=8, seed=0, tensor_id=0, step=0, status=None, out=None):
    N, H, W, Cc = x.shape
    K, R, S, _ = w_shape
    g = geom(N, H, W, Cc, K, R, S, stride, pad, dil)
    if out is None:
        dw = torch.empty((K, R, S, Cc), dtype=torch.int64 if g_mode == ISEG_G_RAW else torch.int8,
                         device=x.device)
        e = _out_exp(x.device)
    else:
        dw, e = out
    ws = workspace(x.device).get(lib().iseg_conv_bwd_weight_ws(C.byref(g), g_mode))
    _maybe_arm(ISEG_KID_CONV_WGRAD, (N, H, W, Cc, K, R, g.stride_h, g.pad_h, g.dil_h))
    iseg_conv_bwd_weight(dy, dy_exp, x, x_exp, g, g_mode, bits, seed, tensor_id, step, dw, e, ws,
                         status)
    return dw, e


def bn_fwd(x, x_exp, gamma_q, beta_q, cfg=None, saved=None, status=None):
    """L1BN forward of int8 codes, or of int32 raw conv sums (the wide input)."""
    Cc = x.shape[-1]
    M = x.numel() // Cc
    cfg = cfg or bn_cfg()
    if x.dtype == torch.int32:
        y = torch.empty(x.shape, dtype=torch.int8, device=x.device)
        e = _out_exp(x.device)
        if saved is None:
            saved = torch.empty(lib().iseg_bn_i32_saved_bytes(Cc), dtype=torch.uint8, device=x.device)
        ws = workspace(x.device).get(lib().iseg_bn_fwd_i32_ws(M, Cc))
        iseg_bn_fwd_i32(x, x_exp, M, Cc, gamma_q, beta_q, cfg, y, e, saved, ws, status)
        return y, e, saved
    y = torch.empty_like(x)
    e = _out_exp(x.device)
    if saved is None:
        saved = torch.empty(lib().iseg_bn_saved_bytes(Cc), dtype=torch.uint8, device=x.device)
    ws = workspace(x.device, bn=True).get(lib().iseg_bn_fwd_ws(M, Cc))
    for kid in (ISEG_KID_BN_FWD_APPLY, ISEG_KID_BN_FWD_STATS1, ISEG_KID_BN_FWD_STATS2):
        _maybe_arm(kid, (M, Cc))
    iseg_bn_fwd(x, x_exp, M, Cc, gamma_q, beta_q, cfg, y, e, saved, ws, status)
    return y, e, saved


def bn_bwd(dy, dy_exp, x, gamma_q, saved, cfg=None, status=None, dgb_out=None):
    Cc = x.shape[-1]
    M = x.numel() // Cc
    cfg = cfg or bn_cfg()
    dx = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    e = _out_exp(x.device)
    if dgb_out is None:
        dg = torch.empty(Cc, dtype=torch.int64, device=x.device)
        db = torch.empty(Cc, dtype=torch.int64, device=x.device)
        dge, dbe = _out_exp(x.device), _out_exp(x.device)
    else:
        dg, db, dge, dbe = dgb_out
    if x.dtype == torch.int32:
        ws = workspace(x.device).get(lib().iseg_bn_bwd_i32_ws(M, Cc))
        iseg_bn_bwd_i32(dy, dy_exp, x, M, Cc, gamma_q, cfg, saved, dx, e, dg, db, dge, dbe, ws, status)
        return dx, e, dg, db, dge, dbe
    ws = workspace(x.device, bn=True).get(lib().iseg_bn_bwd_ws(M, Cc))
    for kid in (ISEG_KID_BN_BWD_APPLY, ISEG_KID_BN_BWD_STATS):
        _maybe_arm(kid, (M, Cc))
    iseg_bn_bwd(dy, dy_exp, x, M, Cc, gamma_q, cfg, saved, dx, e, dg, db, dge, dbe, ws, status)
    return dx, e, dg, db, dge, dbe


def bn_saved_view(saved, Cc):
    """Named views of the saved-state buffer (layout of iseg.h)."""
    def al(v):
        return (v + 255) // 256 * 256
    off = 256
    out = {"hdr": saved[:64].view(torch.int32)}
    for name in ("n_mu", "n_sigma", "den", "qmin", "qmax", "t0", "p0", "mlo", "mhi"):
        out[name] = saved[off:off + 4 * Cc].view(torch.int32)
        off += al(4 * Cc)
    out["xcode"] = saved[off:off + 512 * Cc].view(torch.int16).view(Cc, 256)
    off += al(512 * Cc)
    out["flags"] = saved[off:off + 256 * Cc].view(Cc, 256)
    off += al(256 * Cc)
    out["acode"] = saved[off:off + 256 * Cc].view(torch.int8).view(Cc, 256)
    off += al(256 * Cc)
    out["bwd_entry"] = saved[off:off + 1024 * Cc].view(torch.int32).view(Cc, 256)
    return out


def weight_update(master, g, g_exp, lr_shift, master_exp=-23, k_U=24, k_W=8, w_q=None, status=None):
    if w_q is None:
        w_q = torch.empty(master.shape, dtype=torch.int8, device=master.device)
    iseg_weight_update(master, g, g_exp, lr_shift, master_exp, k_U, k_W, w_q, status)
    return w_q


def weight_quant(master, k_U=24, k_W=8):
    w_q = torch.empty(master.shape, dtype=torch.int8, device=master.device)
    iseg_weight_quant(master, k_U, k_W, w_q)
    return w_q


def maxpool_fwd(x, x_exp, k, stride, pad=0):
    N, H, W, Cc = x.shape
    P = (H + 2 * pad - k) // stride + 1
    Q = (W + 2 * pad - k) // stride + 1
    y = torch.empty((N, P, Q, Cc), dtype=torch.int8, device=x.device)
    e = _out_exp(x.device)
    iseg_maxpool_fwd(x, x_exp, k, stride, pad, y, e)
    return y, e


def maxpool_bwd(dy, dy_exp, x, k, stride, pad=0, bits=8, status=None):
    N, H, W, Cc = x.shape
    dx = torch.empty_like(x)
    e = _out_exp(x.device)
    ws = workspace(x.device).get(lib().iseg_maxpool_bwd_ws(N, H, W, Cc))
    _maybe_arm(ISEG_KID_MAXPOOL_BWD, (N, H, W, Cc))
    iseg_maxpool_bwd(dy, dy_exp, x, k, stride, pad, bits, dx, e, ws, status)
    return dx, e


def sum_requant(ins, in_exps, relu=False, exp_add=None, bcast=None, bits=8, status=None):
    """SQ(ReLU?(sum of the inputs)); the first input fixes the shape [N,H,W,C]
    (a broadcast input is [N,1,1,C])."""
    ref = next(t for t, b in zip(ins, bcast or [0] * len(ins)) if not b)
    N, H, W, Cc = ref.shape
    out = torch.empty_like(ref)
    e = _out_exp(ref.device)
    ws = workspace(ref.device).get(lib().iseg_sum_requant_ws(N, H * W, Cc))
    iseg_sum_requant(ins, in_exps, exp_add, bcast, N, H * W, Cc, int(relu), bits, out, e, ws, status)
    return out, e


def sum_requant_relu_mask(ins, in_exps, masks, mask_exps, exp_add=None, bits=8, status=None):
    """sum_requant (no ReLU, no broadcast) followed by relu_mask_bwd with the
    mask inputs, in one call: (codes, exponent)."""
    N, H, W, Cc = ins[0].shape
    out = torch.empty_like(ins[0])
    e = _out_exp(ins[0].device)
    ws = workspace(ins[0].device).get(lib().iseg_sum_requant_ws(N, H * W, Cc))
    iseg_sum_requant_relu_mask(ins, in_exps, exp_add, N, H * W, Cc, bits, masks, mask_exps, out, e, ws, status)
    return out, e


def relu_mask_bwd(dy, ins, in_exps, status=None):
    dx = torch.empty_like(dy)
    iseg_relu_mask_bwd(dy, ins, in_exps, None, dy.shape[-1], dx, status)
    return dx


def concat_requant(ins, in_exps, bits=8, status=None):
    """Channel concatenation of [N,H,W,C_i] tensors (a [N,1,1,C_i] part is
    broadcast to H x W), SQ to `bits`."""
    N = ins[0].shape[0]
    H = max(t.shape[1] for t in ins)
    W = max(t.shape[2] for t in ins)
    widths = [t.shape[3] for t in ins]
    bc = [int(tuple(t.shape[1:3]) != (H, W)) for t in ins]
    out = torch.empty((N, H, W, sum(widths)), dtype=torch.int8, device=ins[0].device)
    e = _out_exp(ins[0].device)
    ws = workspace(ins[0].device).get(lib().iseg_concat_requant_ws(len(ins)))
    iseg_concat_requant(ins, in_exps, widths, bc, N, H * W, bits, out, e, ws, status)
    return out, e


def concat_split(dy, widths, skip=None):
    """Channel slices of dy (None where skip[i])."""
    N, H, W, _ = dy.shape
    outs = [None if (skip and skip[i]) else
            torch.empty((N, H, W, c), dtype=torch.int8, device=dy.device)
            for i, c in enumerate(widths)]
    iseg_concat_split(dy, N * H * W, widths, outs)
    return outs


def spatial_sum(x, x_exp, divisor=1, c0=0, Cc=None, bits=8, status=None):
    """SQ(sum over H x W of channels [c0, c0 + Cc) / divisor) -> [N,1,1,Cc]."""
    N, H, W, ldc = x.shape
    Cc = ldc - c0 if Cc is None else Cc
    out = torch.empty((N, 1, 1, Cc), dtype=torch.int8, device=x.device)
    e = _out_exp(x.device)
    ws = workspace(x.device).get(lib().iseg_spatial_sum_ws(N, H * W, Cc))
    iseg_spatial_sum(x, x_exp, N, H * W, ldc, c0, Cc, divisor, bits, out, e, ws, status)
    return out, e


def gap_fwd(x, x_exp, bits=8, status=None):
    """Global average pooling over H x W -> [N,1,1,C] (SQ of the exact mean)."""
    return spatial_sum(x, x_exp, x.shape[1] * x.shape[2], bits=bits, status=status)


def gap_bwd(dy, dy_exp, H, W, bits=8, status=None):
    """Backward of the mean over H x W: SQ(dy / (H W)), [N,1,1,C], to be
    broadcast over H x W by the consumer."""
    return spatial_sum(dy, dy_exp, H * W, bits=bits, status=status)


def softmax_ce(logits, logit_exp, labels, bits=8, want_grad=False, status=None):
    """Loss (device double), optional float64 gradient, and E1 = SQ(gradient)."""
    N, h, w, K = logits.shape
    _, H, W = labels.shape
    dev = logits.device
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    grad = torch.empty((N, h, w, K), dtype=torch.float64, device=dev) if want_grad else None
    err = torch.empty((N, h, w, K), dtype=torch.int8, device=dev)
    e = _out_exp(dev)
    ws = workspace(dev).get(lib().iseg_softmax_ce_ws(N, h, w, K, H, W))
    iseg_softmax_ce(logits, logit_exp, labels, N, h, w, K, H, W, bits, loss, grad, err, e, ws, status)
    return loss, grad, err, e


def wt_kind(x_shape, w_shape, stride=1, pad=0, dil=1):
    """Transposed-weight layout the backward-data of this conv uses."""
    N, H, W, Cc = x_shape
    K, R, S, _ = w_shape
    return iseg_conv_bwd_data_wt_kind(geom(N, H, W, Cc, K, R, S, stride, pad, dil))


def wt_table(entries, device):
    """Device array of iseg_wt_desc for iseg_weight_transpose_multi.  entries:
    (w [K,R,S,C] int8, wt same size, kind); returns (table, n, total_tiles)."""
    n = len(entries)
    host = (WtDesc * max(n, 1))()
    tiles = 0
    for i, (w, wt, kind) in enumerate(entries):
        K, R, S, Cc = w.shape
        d = host[i]
        d.w, d.wt = w.data_ptr(), wt.data_ptr()
        d.K, d.RS, d.C, d.kind = K, R * S, Cc, kind
        d.tile_begin = tiles
        tiles += ((Cc + 63) // 64) * ((K + 63) // 64) * R * S
    raw = torch.frombuffer(bytearray(bytes(host)), dtype=torch.uint8)
    return raw.to(device), n, tiles


def update_table(entries, device):
    """Device array of iseg_update_desc for iseg_update_multi.  entries: dicts
    with master, w_q, g, g_exp, kind, master_exp and, for ISEG_UPD_RAW,
    tensor_id, g_q, g_q_exp (torch tensors; their storage must stay alive);
    optional k_w, the tensor's own Q_W width (0 = the call's k_W)."""
    n = len(entries)
    host = (UpdateDesc * max(n, 1))()
    for i, e in enumerate(entries):
        d = host[i]
        d.master = e["master"].data_ptr()
        d.w_q = e["w_q"].data_ptr()
        d.g = e["g"].data_ptr()
        d.g_exp = e["g_exp"].data_ptr()
        d.g_q = e["g_q"].data_ptr() if e.get("g_q") is not None else None
        d.g_q_exp = e["g_q_exp"].data_ptr() if e.get("g_q_exp") is not None else None
        d.n = e["master"].numel()
        d.kind = e["kind"]
        d.master_exp = e["master_exp"]
        d.tensor_id = e.get("tensor_id", 0)
        d.k_w = e.get("k_w", 0)
    raw = torch.frombuffer(bytearray(bytes(host)), dtype=torch.uint8)
    return raw.to(device), n
