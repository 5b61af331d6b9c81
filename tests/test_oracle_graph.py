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


def _sq_ok(vals, codes, exp, k, m):
    """SQ_k of exact values (Eq. 4 with the power-of-two scale): the scale
    2^(exp+k-1) is the smallest power of two strictly above m, the maximum
    magnitude of the whole tensor (vals may be a part of it), every
    code is within [-(2^(k-1)-1), 2^(k-1)-1] and within half a step of its
    value (a clamped code at the top of the range within one step)."""
    from fractions import Fraction
    step = Fraction(2) ** exp
    top = 2 ** (k - 1) - 1
    if m == 0:
        return all(c == 0 for c in codes)
    if not (Fraction(2) ** (exp + k - 2) <= m < Fraction(2) ** (exp + k - 1)):
        return False
    for v, c in zip(vals, codes):
        if abs(c) > top:
            return False
        err = abs(c * step - v)
        if err > step / 2 and not (abs(c) == top and err <= step):
            return False
    return True


@pytest.mark.parametrize("wl", [synth.scaled(synth.RESNET50_CONV2X, 1, 6, 7),
                                synth.scaled(synth.ASPP_HEAD, 1, 5, 4)],
                         ids=["resnet-stage", "aspp"])
def test_low_bit_widths(wl):
    """Table 1's last DeepLab row (k_W = k_A = 4, k_E2 = 8) with k_U = 16:
    weights, masters and every activation a conv reads hold codes of their
    width, a conv feeding BN keeps 8-bit outputs, errors stay 8-bit, and the
    merges are SQ_4 of their exact results."""
    from fractions import Fraction
    from oracle.model import OracleNet
    k_W, k_A, k_U = 4, 4, 16
    inp = synth.workload_inputs(wl)
    net = OracleNet(wl, inp, bn_cfg={"k_A": k_A, "k_E2": 8}, k_W=k_W, k_U=k_U)
    for ci, nd in enumerate(n for n in wl["nodes"] if n["kind"] == "conv"):
        # Eq. 7 then Eq. 8 from the float weights: two roundings, each at most
        # half its step
        wf = inp["weights"][ci].astype(np.float64)
        wq = net.convs[nd["name"]]["w_q"].astype(np.float64) * 2.0 ** (1 - k_W)
        assert np.abs(wq - np.clip(wf, -1 + 2.0 ** (1 - k_W), 1)).max() <= 2.0 ** -k_W + 2.0 ** -k_U
    rec = net.step()
    top_a = 2 ** (k_A - 1) - 1
    for nd in wl["nodes"]:
        r = rec[nd["name"]]
        a = np.abs(r["a_out"].astype(np.int64)).max()
        reads = nd["kind"] in ("add", "concat", "gap") or (nd["kind"] == "conv")
        if reads:
            assert a <= top_a, nd["name"]
        if nd["kind"] == "conv" and nd["bn"]:
            # Eq. 8's fixed step 2^(1-k_W) can zero a whole tensor of small
            # weights (MSRA-scaled 3x3x2048 ones stay below half of 2^-3)
            zm = np.abs(r["z"].astype(np.int64)).max()
            assert zm == 0 or 64 <= zm <= 127, nd["name"]
        e = np.abs(r["e_out"].astype(np.int64)).max()
        assert e == 0 or 64 <= e <= 127, nd["name"]
        if nd["kind"] == "add":
            s = [max(Fraction(int(x)) * Fraction(2) ** r["a_in_exp"]
                     + Fraction(int(y)) * Fraction(2) ** r["b_in_exp"], 0) if nd["relu"]
                 else Fraction(int(x)) * Fraction(2) ** r["a_in_exp"]
                 + Fraction(int(y)) * Fraction(2) ** r["b_in_exp"]
                 for x, y in zip(r["a_in"].ravel()[:4096], r["b_in"].ravel()[:4096])]
            # the scale is the whole tensor's: check it on the full maximum,
            # the codes on the first elements
            full = (r["a_in"].astype(np.int64) * 2.0 ** r["a_in_exp"]
                    + r["b_in"].astype(np.int64) * 2.0 ** r["b_in_exp"])
            if nd["relu"]:
                full = np.maximum(full, 0)
            m = Fraction(float(np.abs(full).max()))
            codes = [int(c) for c in r["a_out"].ravel()[:4096]]
            assert _sq_ok(s, codes, r["a_out_exp"], k_A, m), nd["name"]
    for nd, _ in [(n, None) for n in wl["nodes"] if n["kind"] == "conv"]:
        L = net.convs[nd["name"]]
        assert np.abs(L["w_m"].astype(np.int64)).max() <= 2 ** (k_U - 1) - 1
        assert np.abs(L["w_q"].astype(np.int64)).max() <= 2 ** (k_W - 1) - 1
        # Eq. 8 after the update: W_q within half a k_W step of the master
        d = L["w_q"].astype(np.float64) * 2.0 ** (1 - k_W) - L["w_m"].astype(np.float64) * 2.0 ** (1 - k_U)
        assert np.abs(d).max() <= 2.0 ** -k_W
        for q in ("g_q", "b_q"):
            assert np.abs(L[q].astype(np.int64)).max() <= 127


def test_no_bn_gq2_step():
    """The no-BN network with GQ2 (Eq. 18): one step's gradient codes equal
    GQ1's (the same stochastic RQ; only the exponent differs, 1 - k_G), ReLU
    convs output non-negative k_A-bit codes, and their backward passes the
    error exactly where the 8-bit conv output is positive."""
    from oracle.model import OracleNet
    wl = synth.without_bn(synth.scaled(synth.RESNET50_CONV2X, 1, 6, 7))
    inp = synth.workload_inputs(wl)
    r1 = OracleNet(wl, inp, gq=1).step()
    r2 = OracleNet(wl, inp, gq=2).step()
    for nd in wl["nodes"]:
        a, b = r1[nd["name"]], r2[nd["name"]]
        if nd["kind"] != "conv":
            continue
        # the forward is the same; G codes agree, exponents follow Eq. 17 / 18
        assert np.array_equal(a["a_out"], b["a_out"])
        if np.array_equal(a["dz"], b["dz"]) and a["dz_exp"] == b["dz_exp"]:
            assert np.array_equal(a["G"], b["G"]), nd["name"]
        assert b["G_exp"] == 1 - 8
        if nd["relu"]:
            assert a["a_out"].min() >= 0 and a["a_out"].max() <= 127
            z = a["z"].astype(np.int64)
            e = a["e_out"].astype(np.int64)
            assert np.array_equal(a["dz"].astype(np.int64), np.where(z > 0, e, 0)), nd["name"]
            assert a["dz_exp"] == a["e_out_exp"]
