"""GPU parity of whole training steps (forward, backward, update) against the
oracle's composition of the same steps: every activation, error, gradient
code, exponent and the updated masters, bit-exact."""
import numpy as np
import pytest

from paper_2011_14504_amd import synth

pytestmark = pytest.mark.gpu


def _cmp(g, o, what):
    a = g.cpu().numpy() if hasattr(g, "cpu") else np.asarray(g)
    assert np.array_equal(a.astype(np.int64), np.asarray(o).astype(np.int64)), what


def _ev(t):
    return int(t.item())


def _run_both(wl, N, steps=1):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from oracle.model import OracleNet
    from paper_2011_14504_amd.model import IntNet
    inp = synth.workload_inputs(wl, N)
    gnet = IntNet(wl, inp, "cuda:0")
    onet = OracleNet(wl, inp)
    for s in range(steps):
        grec = gnet.step()
        orec = onet.step()
        torch.cuda.synchronize()
        for i, (g, o) in enumerate(zip(grec, orec)):
            tag = f"step {s} layer {i} ({g['kind']})"
            _cmp(g["a_out"], o["a_out"], tag + " activation")
            assert _ev(g["a_out_exp"]) == o["a_out_exp"], tag
            if g["kind"] == "conv":
                _cmp(g["z"], o["z"], tag + " conv output")
                assert _ev(g["z_exp"]) == o["z_exp"], tag
                for k in ("dz", "G", "Gg", "Gb", "dgamma", "dbeta"):
                    _cmp(g[k], o[k], tag + " " + k)
                for k in ("dz_exp", "G_exp", "Gg_exp", "Gb_exp"):
                    assert _ev(g[k]) == o[k], tag + " " + k
            if "e_in" in o:
                _cmp(g["e_in"], o["e_in"], tag + " input error")
                assert _ev(g["e_in_exp"]) == o["e_in_exp"], tag
        for gl, ol in zip(gnet.convs, onet.convs):
            for k in ("w_m", "g_m", "b_m", "w_q", "g_q", "b_q"):
                _cmp(gl[k], ol[k], f"step {s} {k}")


def test_single_conv_two_steps():
    _run_both(synth.SINGLE_CONV, None, steps=2)


def test_vgg16_blocks12_one_image():
    # full 224x224 resolution, one image: every tile and ragged tail of the
    # real layer shapes, compared element by element
    _run_both(synth.VGG16_BLOCKS12, 1)
