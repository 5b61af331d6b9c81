"""CPU checks of the C ABI: the library loads, exports every function the
header declares, validates arguments on the host before touching a device,
and its host-side Philox matches the published known-answer vectors."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "iseg.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(iseg_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2011_14504_amd import iseg
    return iseg.lib()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n


def test_binding_covers_every_declared_symbol():
    from paper_2011_14504_amd import iseg
    for n in _declared():
        assert n in iseg._SIGS, n
        assert callable(getattr(iseg, n, None)) or n.endswith("_ws") or n.endswith("_bytes"), n


def test_philox_known_answers(lib):
    from paper_2011_14504_amd import iseg
    assert iseg.iseg_philox4x32_10([0, 0, 0, 0], [0, 0]) == \
        [0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8]
    assert iseg.iseg_philox4x32_10([0xffffffff] * 4, [0xffffffff] * 2) == \
        [0x408f276d, 0x41c83b0e, 0xa20bc7c6, 0x6d5451fd]


def test_host_validation_without_device(lib):
    from paper_2011_14504_amd import iseg
    bad = iseg.geom(1, 2, 2, 3, 4, 5, 5, 1, 0, 1)        # kernel larger than the padded input
    assert lib.iseg_conv_fwd(None, None, None, None, C.byref(bad), 0, None, None, None, 0, None,
                             None) == iseg.ISEG_ERR_SHAPE
    g = iseg.geom(1, 8, 8, 16, 16, 3, 3, 1, 1, 1)
    assert lib.iseg_conv_fwd(None, None, None, None, C.byref(g), 7, None, None, None, 0, None,
                             None) == iseg.ISEG_ERR_ARG
    one = C.c_void_p(1)
    # raw int32 sums of a reduction longer than 131071 products: refused; final
    # codes split it into at most 8 channel chunks, refused beyond that
    big = iseg.geom(1, 8, 8, 20000, 16, 3, 3, 1, 1, 1)
    assert lib.iseg_conv_fwd(one, one, one, one, C.byref(big), iseg.ISEG_OUT_RAW, one, one, one, 1 << 40, None,
                             None) == iseg.ISEG_ERR_UNSUPPORTED
    huge = iseg.geom(1, 8, 8, 120000, 16, 3, 3, 1, 1, 1)
    assert lib.iseg_conv_fwd(one, one, one, one, C.byref(huge), iseg.ISEG_OUT_Q8, one, one, one, 1 << 40, None,
                             None) == iseg.ISEG_ERR_UNSUPPORTED
    assert lib.iseg_conv_bwd_data(one, one, one, one, C.byref(iseg.geom(1, 8, 8, 16, 120000, 3, 3, 1, 1, 1)),
                                  iseg.ISEG_OUT_Q8, one, one, one, 1 << 40, None, None) == iseg.ISEG_ERR_UNSUPPORTED
    assert lib.iseg_conv_fwd_ws(C.byref(huge), iseg.ISEG_OUT_Q8) == 0
    assert lib.iseg_conv_fwd_ws(C.byref(big), iseg.ISEG_OUT_Q8) > 0
    assert lib.iseg_conv_fwd(one, one, one, one, C.byref(g), 0, one, one, one, 16, None,
                             None) == iseg.ISEG_ERR_WORKSPACE
    cfg = iseg.bn_cfg(k_A=9)
    assert lib.iseg_bn_fwd(one, one, 10, 16, one, one, C.byref(cfg), one, one, one, one, 1 << 30,
                           None, None) == iseg.ISEG_ERR_ARG
    assert lib.iseg_bn_fwd(one, one, 10, 3, one, one, C.byref(iseg.bn_cfg()), one, one, one, one,
                           1 << 30, None, None) == iseg.ISEG_ERR_SHAPE
    assert lib.iseg_requant(one, 7, 10, one, 8, 0, 1, 0, 0, 0, 0, one, one, one, 256, None,
                            None) == iseg.ISEG_ERR_ARG
    assert lib.iseg_weight_update(one, 10, one, one, 10, -23, 40, 8, one, None, None) == \
        iseg.ISEG_ERR_ARG
    assert lib.iseg_profile_arm(99, None, None) == iseg.ISEG_ERR_ARG


def test_workspace_queries(lib):
    from paper_2011_14504_amd import iseg
    g = iseg.geom(8, 224, 224, 64, 64, 3, 3, 1, 1, 1)
    assert lib.iseg_conv_fwd_ws(C.byref(g), iseg.ISEG_OUT_Q8) >= 8 * 224 * 224 * 64 * 4
    assert lib.iseg_conv_fwd_ws(C.byref(g), iseg.ISEG_OUT_RAW) <= 4096
    assert lib.iseg_conv_bwd_weight_ws(C.byref(g), 0) >= 64 * 9 * 64 * 8
    assert lib.iseg_bn_saved_bytes(64) > 64 * 1024
    assert lib.iseg_bn_fwd_ws(401408, 64) > 0 and lib.iseg_bn_bwd_ws(401408, 64) > 0
    assert lib.iseg_bn_fwd_ws(10, 3) == 0


def test_transposed_weight_host_checks(lib):
    from paper_2011_14504_amd import iseg
    g = iseg.geom(1, 8, 8, 16, 16, 3, 3, 1, 1, 1)
    assert lib.iseg_conv_bwd_data_t(None, None, None, None, None, 7, C.byref(g), 0, None, None, None,
                                    0, None, None) == iseg.ISEG_ERR_ARG
    bad = iseg.geom(1, 2, 2, 3, 4, 5, 5, 1, 0, 1)
    assert lib.iseg_conv_bwd_data_wt_kind(C.byref(bad)) == iseg.ISEG_WT_NONE
    assert lib.iseg_conv_bwd_data_wt_kind(C.byref(g)) in (iseg.ISEG_WT_CRSK, iseg.ISEG_WT_CRSK_FLIP)
    s2 = iseg.geom(1, 16, 16, 64, 128, 3, 3, 2, 1, 1)     # stride 2: only the implicit GEMM reads it
    assert lib.iseg_conv_bwd_data_wt_kind(C.byref(s2)) == iseg.ISEG_WT_CRSK
    assert lib.iseg_weight_transpose_multi(None, 0, 0, None) == iseg.ISEG_OK
    assert lib.iseg_weight_transpose_multi(None, -1, 1, None) == iseg.ISEG_ERR_ARG
    assert lib.iseg_weight_transpose_multi(None, 1, 0, None) == iseg.ISEG_ERR_ARG


def test_tape_entries_match_the_binding():
    """The step tape resolves every call a training step makes, each with the
    parameter count of its declaration in the binding."""
    from paper_2011_14504_amd import iseg
    L = iseg.lib()
    step_calls = ["iseg_conv_fwd", "iseg_conv_bwd_data", "iseg_conv_bwd_data_t", "iseg_conv_bwd_weight",
                  "iseg_weight_transpose_multi", "iseg_bn_fwd", "iseg_bn_bwd", "iseg_bn_fwd_i32",
                  "iseg_bn_bwd_i32", "iseg_update_multi", "iseg_maxpool_fwd", "iseg_maxpool_bwd",
                  "iseg_sum_requant", "iseg_relu_mask_bwd", "iseg_sum_requant_relu_mask", "iseg_concat_requant", "iseg_concat_split",
                  "iseg_spatial_sum", "iseg_softmax_ce", "iseg_mse_onehot", "iseg_profile_arm"]
    for name in step_calls:
        assert L.iseg_tape_entry(name.encode()) >= 0, name
    n = 0
    for name, (args, res) in iseg._SIGS.items():
        e = L.iseg_tape_entry(name.encode())
        if e >= 0:
            assert L.iseg_tape_entry_nargs(e) == len(args), name
            n += 1
    assert n >= len(step_calls)
    assert L.iseg_tape_entry(b"iseg_nonexistent") == -1
