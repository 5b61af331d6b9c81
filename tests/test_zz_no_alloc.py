"""iseg_bn_fwd_noalloc (workspace in a static device array) against
iseg_bn_fwd with a caller workspace: outputs, exponents and the saved state
bit-identical, over two calls in a row (the second on a smaller input, so
stale contents of the static array from the first call would show), and
shapes beyond the array rejected on the host."""
import ctypes as C

import numpy as np
import pytest

from paper_2011_14504_amd import synth

pytestmark = pytest.mark.gpu


def _run_pair(iseg, torch, dev, M, Cc, relu, seed):
    x = torch.from_numpy(synth.int_codes(seed, (M, Cc))).to(dev)
    g = torch.from_numpy(synth.int_codes(seed + 1, (Cc,))).to(dev)
    b = torch.from_numpy(synth.int_codes(seed + 2, (Cc,))).to(dev)
    xe = torch.tensor([-9], dtype=torch.int32, device=dev)
    cfg = iseg.bn_cfg(**dict(iseg.BN_DEFAULT, relu=relu))
    nsv = iseg.lib().iseg_bn_saved_bytes(Cc)
    outs = []
    for noalloc in (False, True):
        y = torch.zeros((M, Cc), dtype=torch.int8, device=dev)
        ye = torch.zeros(1, dtype=torch.int32, device=dev)
        sv = torch.zeros(nsv, dtype=torch.uint8, device=dev)
        st = torch.zeros(1, dtype=torch.int32, device=dev)
        if noalloc:
            iseg.iseg_bn_fwd_noalloc(x, xe, M, Cc, g, b, cfg, y, ye, sv, st)
        else:
            # the workspace starts with arrival counters that must be zero
            ws = torch.zeros(iseg.lib().iseg_bn_fwd_ws(M, Cc), dtype=torch.uint8, device=dev)
            iseg.iseg_bn_fwd(x, xe, M, Cc, g, b, cfg, y, ye, sv, ws, st)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        outs.append((y.cpu().numpy(), int(ye.item()), sv.cpu().numpy()))
    (y0, e0, s0), (y1, e1, s1) = outs
    assert np.array_equal(y0, y1) and e0 == e1 and np.array_equal(s0, s1)
    assert np.abs(y0.astype(np.int64)).max() > 0


def test_bn_fwd_noalloc_matches_bn_fwd():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2011_14504_amd import iseg
    dev = torch.device("cuda", 0)
    # two calls in a row, the second smaller, then a shape with more channels
    _run_pair(iseg, torch, dev, 8 * 64 * 64, 256, 1, 501)
    _run_pair(iseg, torch, dev, 1000, 64, 0, 502)
    _run_pair(iseg, torch, dev, 8 * 32 * 32, 2048, 1, 503)


def test_bn_fwd_noalloc_rejects_shapes_beyond_the_array():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2011_14504_amd import iseg
    L = iseg.lib()
    M, Cc = 1024, 65536
    assert L.iseg_bn_fwd_ws(M, Cc) > L.iseg_bn_fwd_noalloc_max_bytes()
    dev = torch.device("cuda", 0)
    x = torch.zeros((M, Cc), dtype=torch.int8, device=dev)
    g = torch.zeros(Cc, dtype=torch.int8, device=dev)
    xe = torch.zeros(1, dtype=torch.int32, device=dev)
    cfg = iseg.bn_cfg(**iseg.BN_DEFAULT)
    sv = torch.zeros(L.iseg_bn_saved_bytes(Cc), dtype=torch.uint8, device=dev)
    rc = L.iseg_bn_fwd_noalloc(iseg._ptr(x), iseg._ptr(xe), M, Cc, iseg._ptr(g), iseg._ptr(g), C.byref(cfg),
                               iseg._ptr(x), iseg._ptr(xe), iseg._ptr(sv), None, iseg._stream())
    assert rc == iseg.ISEG_ERR_WORKSPACE
