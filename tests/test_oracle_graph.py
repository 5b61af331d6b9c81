"""The oracle's composition of whole training steps over the workload graphs
(residual stages, the ASPP head, the DeepLabv3-ResNet50 step), at small
spatial sizes: every tensor stays in its code range, errors reach every node,
and the merged errors agree with the pinned merge on the contributions."""
import numpy as np
import pytest

from paper_2011_14504_amd import synth


def _run(wl):
    from oracle.model import OracleNet
    inp = synth.workload_inputs(wl)
    net = OracleNet(wl, inp)
    rec = net.step()
    return net, rec


@pytest.mark.parametrize("wl", [synth.scaled(synth.RESNET50_CONV2X, 1, 10, 9),
                                synth.scaled(synth.ASPP_HEAD, 1, 8, 8),
                                synth.scaled(synth.DEEPLABV3_R50, 1, 32, 32)],
                         ids=["resnet-stage", "aspp", "deeplabv3"])
def test_graph_step_ranges(wl):
    net, rec = _run(wl)
    shapes = synth.node_shapes(wl)
    for nd in wl["nodes"]:
        r = rec[nd["name"]]
        assert tuple(r["a_out"].shape) == shapes[nd["name"]]
        assert np.abs(r["a_out"].astype(np.int64)).max() <= 127
        assert "e_out" in r, nd["name"]
        assert tuple(r["e_out"].shape) == shapes[nd["name"]]
        if nd["kind"] == "conv":
            assert np.abs(r["G"].astype(np.int64)).max() <= 127
    if wl["input_grad"]:
        assert rec["input"]["e_out"].shape == shapes["input"]
    if wl["loss"] == "softmax_ce":
        assert np.isfinite(net.loss) and net.loss > 0


def test_residual_block_input_error_is_merge_of_both_paths():
    from oracle import oracle as O
    wl = synth.scaled(synth.RESNET50_CONV2X, 1, 6, 7)
    net, rec = _run(wl)
    # block 1 has an identity shortcut: the error at its input (block 0's
    # output) is SQ8 of conv1's backward-data result plus the masked error
    add = rec["conv2_x.1.out"]
    c1 = rec["conv2_x.1.conv1"]
    e, ee = O.sum_requant([c1["e_in"], add["e_in"]], [c1["e_in_exp"], add["e_in_exp"]], 8)
    out0 = rec["conv2_x.0.out"]
    assert np.array_equal(out0["e_out"], e.astype(np.int8)) and out0["e_out_exp"] == ee
