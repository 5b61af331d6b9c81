"""The device status word: every range condition the kernels detect is forced
from crafted inputs (the kernels take their documented fallback and exit
normally), read back through iseg_status_read, and cleared by
iseg_status_clear; and the kernel path an entry point reports."""
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


def _status(dev):
    import torch
    return torch.zeros(1, dtype=torch.int32, device=dev)


def T(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def E(v, dev):
    import torch
    return torch.tensor([int(v)], dtype=torch.int32, device=dev)


def test_status_read_and_clear(dev):
    import torch
    from paper_2011_14504_amd import iseg
    st = torch.full((1,), 5, dtype=torch.int32, device=dev)
    assert iseg.iseg_status_read(st) == 5
    iseg.iseg_status_clear(st)
    assert iseg.iseg_status_read(st) == 0


@pytest.mark.parametrize("n", [16, 4096 + 7, 1 << 20])
def test_check_codes(dev, n):
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(3, (n,))
    st = _status(dev)
    iseg.iseg_check_codes(T(x, dev), 8, st)
    assert iseg.iseg_status_read(st) == 0
    for pos in (0, n - 1, n // 2):
        y = x.copy()
        y[pos] = -128
        st = _status(dev)
        iseg.iseg_check_codes(T(y, dev), 8, st)
        assert iseg.iseg_status_read(st) == iseg.ISEG_DEV_RANGE, pos
    # a 4-bit tensor holding an 8-bit code
    z = np.clip(x, -7, 7).astype(np.int8)
    st = _status(dev)
    iseg.iseg_check_codes(T(z, dev), 4, st)
    assert iseg.iseg_status_read(st) == 0
    z[n // 3] = 8
    iseg.iseg_check_codes(T(z, dev), 4, st)
    assert iseg.iseg_status_read(st) == iseg.ISEG_DEV_RANGE


def test_softmax_logit_exponent_outside_domain(orc, dev):
    """|logit| must stay below 128 (exponent <= 0): at the bound the region
    matches the oracle; above it the status is set, the codes are zero and
    the loss is NaN, and the oracle rejects the call."""
    from paper_2011_14504_amd import iseg
    logits = synth.int_codes(11, (1, 4, 4, 21))
    labels = synth.labels(12, (1, 64, 64), 21)
    st = _status(dev)
    loss, _, e, ee = iseg.softmax_ce(T(logits, dev), E(0, dev), T(labels, dev), status=st)
    assert iseg.iseg_status_read(st) == 0
    ref, grad = orc.softmax_ce(logits, 0, labels)
    assert abs(float(loss.item()) - ref) <= 1e-12 * abs(ref)
    for bad in (1, 40, -1001):
        st = _status(dev)
        loss, _, e, ee = iseg.softmax_ce(T(logits, dev), E(bad, dev), T(labels, dev), status=st)
        assert iseg.iseg_status_read(st) == iseg.ISEG_DEV_RANGE, bad
        assert not e.cpu().numpy().any() and np.isnan(float(loss.item()))
        with pytest.raises(orc.OracleError):
            orc.softmax_ce(logits, bad, labels)


def test_softmax_bad_label(dev):
    from paper_2011_14504_amd import iseg
    logits = synth.int_codes(11, (1, 4, 4, 21))
    labels = synth.labels(12, (1, 64, 64), 21)
    labels[0, 5, 7] = 21
    st = _status(dev)
    iseg.softmax_ce(T(logits, dev), E(-3, dev), T(labels, dev), status=st)
    assert iseg.iseg_status_read(st) == iseg.ISEG_DEV_RANGE


def test_bn_input_exponent_out_of_range(dev):
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(21, (256, 16))
    g = np.full(16, 64, np.int8)
    b = np.zeros(16, np.int8)
    for e, want in ((16, 0), (17, iseg.ISEG_DEV_RANGE), (-40, 0), (-41, iseg.ISEG_DEV_RANGE)):
        st = _status(dev)
        iseg.bn_fwd(T(x, dev), E(e, dev), T(g, dev), T(b, dev), status=st)
        assert iseg.iseg_status_read(st) == want, e


def test_merge_exponent_gap(dev):
    from paper_2011_14504_amd import iseg
    a = synth.int_codes(31, (2, 8, 8, 32))
    b = synth.int_codes(32, (2, 8, 8, 32))
    for gap, want in ((48, 0), (49, iseg.ISEG_DEV_RANGE)):
        st = _status(dev)
        iseg.sum_requant([T(a, dev), T(b, dev)], [E(-10, dev), E(-10 - gap, dev)], status=st)
        assert iseg.iseg_status_read(st) == want, gap


def test_conv_last_plan_reports_the_path(dev):
    from paper_2011_14504_amd import iseg
    x = synth.int_codes(41, (1, 10, 9, 3))
    w = synth.int_codes(42, (64, 7, 7, 3))
    iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), 2, 3, 1)
    assert iseg.iseg_conv_last_plan() == "stem"
    x = synth.int_codes(43, (1, 6, 5, 64))
    w = synth.int_codes(44, (64, 3, 3, 64))
    iseg.conv_fwd(T(x, dev), E(-7, dev), T(w, dev), E(-7, dev), 1, 1, 1)
    assert iseg.iseg_conv_last_plan() not in ("none", "stem")
