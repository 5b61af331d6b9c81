"""The oracle's composition of whole training steps, pinned by an independent
exact-rational brute force (tests/bruteforce_step.py): forward order, the
routing of errors to both branches of a residual block and their merge, the
inputs of every weight gradient, the Philox keys of Q_G, and the update of
every master.  The brute force shares no code with the oracle; it is written
from Eq. 2-8 and 12-19 with Fractions.  Every activation, error, gradient
code, exponent and updated master of OracleNet.step() must equal it."""
import numpy as np
import pytest

from paper_2011_14504_amd import synth
import bruteforce_step as B


def _same(codes, exp, vals, vexp, what, check_exp=True):
    got = B.values(np.asarray(codes).astype(np.int64), exp)
    assert got.shape == vals.shape, what
    assert all(g == v for g, v in zip(got.ravel(), vals.ravel())), what
    if check_exp and vexp is not None:
        assert exp == vexp, (what, exp, vexp)


def _compare_node(o, b, name):
    for key in ("z", "a_out", "e_out", "dz", "G", "e_in", "Gg", "Gb"):
        if key in b:
            assert key in o, (name, key)
            _same(o[key], o[key + "_exp"], b[key], b[key + "_exp"], f"{name} {key}")
    for key in ("dgamma", "dbeta"):
        if key in b:
            _same(o[key], o[key + "_exp"], np.array(b[key], dtype=object), None, f"{name} {key}")


def _compare_params(onet, bnet, k_U, k_W, cfg):
    for name, L in bnet.L.items():
        O = onet.convs[name]
        _same(O["w_m"], 1 - k_U, L["w_m"], None, f"{name} w_m")
        _same(O["w_q"], 1 - k_W, bnet.w_q(name), None, f"{name} w_q")
        if L["nd"]["bn"]:
            g, b = bnet.gamma_beta(name)
            _same(O["g_m"], 2 - k_U, np.array(L["g_m"], dtype=object), None, f"{name} g_m")
            _same(O["b_m"], 2 - k_U, np.array(L["b_m"], dtype=object), None, f"{name} b_m")
            _same(O["g_q"], 2 - cfg["k_gamma"], np.array(g, dtype=object), None, f"{name} g_q")
            _same(O["b_q"], 2 - cfg["k_beta"], np.array(b, dtype=object), None, f"{name} b_q")


def test_python_philox_known_answers():
    # Random123 known-answer vectors for Philox4x32-10
    assert B.philox4x32_10([0, 0, 0, 0], [0, 0]) == [0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8]
    assert B.philox4x32_10([0xffffffff] * 4, [0xffffffff] * 2) == \
        [0x408f276d, 0x41c83b0e, 0xa20bc7c6, 0x6d5451fd]
    assert B.philox4x32_10([0x243f6a88, 0x85a308d3, 0x13198a2e, 0x03707344],
                           [0xa4093822, 0x299f31d0]) == [0xd16cfe09, 0x94fdcceb, 0x5001e420, 0x24126ea1]


def test_bruteforce_conv_adjoints():
    """The brute force's own conv, data gradient and weight gradient satisfy
    <conv(x, w), dy> = <x, dgrad(dy, w)> = <w, wgrad(dy, x)> exactly."""
    from fractions import Fraction as Fr
    rng = synth.rng(4242)
    for (N, H, W, C, K, R, st, pad, dil) in [(1, 7, 6, 3, 4, 3, 2, 1, 1), (2, 5, 5, 2, 3, 3, 1, 2, 2),
                                            (1, 6, 4, 3, 2, 1, 2, 0, 1)]:
        x = B.values(rng.integers(-127, 128, (N, H, W, C)), -3)
        w = B.values(rng.integers(-127, 128, (K, R, R, C)), -7)
        y = B.conv(x, w, st, pad, dil)
        dy = B.values(rng.integers(-127, 128, y.shape), -5)
        lhs = sum((a * b for a, b in zip(y.ravel(), dy.ravel())), Fr(0))
        dx = B.conv_data_grad(dy, w, H, W, st, pad, dil)
        assert lhs == sum((a * b for a, b in zip(x.ravel(), dx.ravel())), Fr(0))
        dw = B.conv_weight_grad(dy, x, R, st, pad, dil)
        assert lhs == sum((a * b for a, b in zip(w.ravel(), dw.ravel())), Fr(0))


def test_single_conv_two_steps_match_bruteforce():
    """Workload 1 at its full size (1x32x32, 16 -> 16 channels, 3x3): two
    steps, so the second one runs with updated W, gamma, beta and step 1 of
    the Philox counter."""
    from oracle.model import OracleNet
    wl = synth.SINGLE_CONV
    inp = synth.workload_inputs(wl)
    onet = OracleNet(wl, inp)
    bnet = B.Net(wl, inp, dict(onet.cfg))
    for s in range(2):
        orec = onet.step()
        brec = B.single_conv_step(bnet, inp["x"], inp["x_exp"], inp["dy"], inp["dy_exp"])
        _compare_node(orec["conv"], brec["conv"], f"step {s} conv")
        _compare_params(onet, bnet, 24, 8, onet.cfg)


TINY_STAGE = dict(id=3, name="tiny-stage-8ch-7x6", N=1, H=7, W=6, C=8, input_grad=True, loss="given",
                  nodes=synth.res_stage("s", "input", 8, 4, 16, 2, stride=2)[0])


@pytest.mark.parametrize("variant", ["bn", "bn-w4a4-e2-8", "no-bn-gq2", "bn-raw", "bn-raw-w4a4"])
def test_residual_stage_two_steps_match_bruteforce(variant):
    """Two bottlenecks (the first strided, with a projection shortcut; the
    second with the identity) on a 1x7x6x8 input with the input gradient:
    every tensor of two training steps against the brute force.  Variants:
    the 8-bit DeepLab setting; W4A4 with E2 at 8 bits (Table 1); the network
    without BN and Eq. 18's gradient quantizer; L1BN on the raw MAC sums (the
    literal dataflow), at 8 and 4 bits."""
    from oracle.model import OracleNet
    wl = TINY_STAGE
    kw = {}
    if variant == "bn-w4a4-e2-8":
        kw = dict(k_W=4, k_U=16, bn_cfg={"k_A": 4, "k_E2": 8})
    if variant == "no-bn-gq2":
        wl = synth.without_bn(wl)
        kw = dict(gq=2)
    if variant == "bn-raw":
        kw = dict(bn_input="raw")
    if variant == "bn-raw-w4a4":
        kw = dict(k_W=4, k_U=16, bn_cfg={"k_A": 4}, bn_input="raw")
    inp = synth.workload_inputs(wl)
    # random gamma / beta would need another draw; the update moves them off 1 / 0
    onet = OracleNet(wl, inp, **kw)
    bnet = B.Net(wl, inp, dict(onet.cfg), k_W=kw.get("k_W", 8), k_U=kw.get("k_U", 24),
                 gq=kw.get("gq", 1), bn_input=kw.get("bn_input", "q8"))
    for s in range(2):
        orec = onet.step()
        brec = B.stage_step(bnet, inp["x"], inp["x_exp"], inp["dy"], inp["dy_exp"], "s", 2)
        for nd in wl["nodes"]:
            _compare_node(orec[nd["name"]], brec[nd["name"]], f"step {s} {nd['name']}")
        _same(orec["input"]["e_out"], orec["input"]["e_out_exp"], brec["input"]["e_out"],
              brec["input"]["e_out_exp"], f"step {s} input error")
        _compare_params(onet, bnet, kw.get("k_U", 24), kw.get("k_W", 8), onet.cfg)


def test_max_exact_scale_deviation_single_conv():
    """How far the power-of-two Scale departs from Eq. 3's literal max|x|, at
    every SQ of one step of workload 1 (the same pre-quantizer values fed to
    both readings).  Both stay within a step of the exact value; the counts
    of elements whose quantized value differs are printed (recorded with the
    readings of the paper)."""
    from fractions import Fraction as Fr
    import bruteforce as bf
    wl = synth.SINGLE_CONV
    inp = synth.workload_inputs(wl)
    from oracle import oracle as O
    seen = []
    orig = B.SQ

    def spy(arr, k):
        seen.append((arr, k))
        return orig(arr, k)

    B.SQ = spy
    try:
        bnet = B.Net(wl, inp, dict(O.BN_DEFAULT))
        B.single_conv_step(bnet, inp["x"], inp["x_exp"], inp["dy"], inp["dy_exp"])
    finally:
        B.SQ = orig
    report = []
    for arr, k in seen:
        flat = list(arr.ravel())
        M = max(abs(v) for v in flat)
        if M == 0:
            continue
        p2 = bf.SQ(flat, k)
        mx = bf.SQ_max(flat, k)
        S2 = bf.pow2_scale(flat)
        step2, stepm = S2 * bf.delta(k), M * bf.delta(k)
        differ = sum(1 for a, b in zip(p2, mx) if a != b)
        for v, a, b in zip(flat, p2, mx):
            assert abs(a - v) <= step2 / 2 and abs(b - v) <= stepm
        mean_dev = sum((abs(a - b) for a, b in zip(p2, mx)), Fr(0)) / len(flat) / stepm
        report.append((k, len(flat), differ, float(S2 / M), float(mean_dev)))
    print("\n[max-exact vs power-of-two] (k, elements, differing, S_pow2/max, mean |diff| in "
          "max-scale steps):")
    for r in report:
        print("  ", r)
    assert len(report) >= 4


def test_bn_on_raw_sums_against_the_requantized_reading():
    """How far L1BN on the raw MAC sums (the literal dataflow) moves the codes
    from the default reading (BN on the SQ8 conv output), one step of
    workload 1 and of a ResNet-50 stage at 28x28: the share of activation
    codes A that differ after each BN, and of the input-error codes.  The
    counts are printed (recorded with the readings of the paper)."""
    from oracle.model import OracleNet
    rows = []
    for wl in (synth.SINGLE_CONV, synth.scaled(synth.RESNET50_CONV2X, 1, 28, 28)):
        inp = synth.workload_inputs(wl)
        ra = OracleNet(wl, inp).step()
        rb = OracleNet(wl, inp, bn_input="raw").step()
        for nd in wl["nodes"]:
            if nd["kind"] != "conv" or not nd["bn"]:
                continue
            a, b = ra[nd["name"]], rb[nd["name"]]
            va = a["a_out"].astype(np.float64) * 2.0 ** a["a_out_exp"]
            vb = b["a_out"].astype(np.float64) * 2.0 ** b["a_out_exp"]
            step = 2.0 ** max(a["a_out_exp"], b["a_out_exp"])
            rows.append((wl["name"][:14], nd["name"], va.size, int((va != vb).sum()),
                         float(np.abs(va - vb).max() / step), a["a_out_exp"] - b["a_out_exp"]))
        ea, eb = ra["input"]["e_out"], rb["input"]["e_out"]
        rows.append((wl["name"][:14], "input error", ea.size,
                     int((ea.astype(np.int64) * 2.0 ** ra["input"]["e_out_exp"]
                          != eb.astype(np.int64) * 2.0 ** rb["input"]["e_out_exp"]).sum()), None, None))
    print("\n[BN on raw sums vs on SQ8 codes] (workload, tensor, elements, values differing, "
          "max |diff| in steps, exponent difference):")
    for r in rows:
        print("  ", r)
    # a BN whose conv reads the (shared) input differs only through the
    # rounding of that conv's output: a minority of codes, by at most two
    # steps; deeper layers also inherit the differences of their inputs
    first = {("single-conv3x3", "conv"), ("resnet50-conv2", "conv2_x.0.proj"),
             ("resnet50-conv2", "conv2_x.0.conv1")}
    for r in rows:
        if (r[0], r[1]) in first:
            assert r[3] < 0.5 * r[2] and r[4] <= 2.0, r


def test_inference_on_the_calibration_batch_equals_training_forward():
    """With the frozen state of a calibration forward, inference on the same
    batch gives the training forward's activations at every layer (the
    fixed-step quantizers then coincide with the data-dependent ones)."""
    from oracle.model import OracleNet
    wl = synth.scaled(synth.VGG16_BLOCKS12, 1, 40, 36)
    inp = synth.workload_inputs(wl)
    net = OracleNet(wl, inp)
    rec = net.forward()
    inf = net.infer(rec, inp["x"], inp["x_exp"])
    for nd in wl["nodes"]:
        codes, e = inf[nd["name"]]
        assert np.array_equal(codes, rec[nd["name"]]["a_out"]) and e == rec[nd["name"]]["a_out_exp"], nd["name"]


TINY_DECODER = dict(id=6, name="tiny-fcn-decoder", N=1, H=6, W=6, C=4, input_grad=False, loss="mse",
                    classes=3, gq=2,
                    nodes=[synth.conv("c1", "input", 4, 6, 3, 2, 1, bn=False),
                           synth.conv("s1", "c1", 6, 3, 1, bn=False, relu=False),
                           synth.deconv("up", "s1", 3, 3, 4, 2, 1),
                           synth.conv("s0", "input", 4, 3, 1, bn=False, relu=False),
                           synth.add("fuse", "up", "s0")])


def test_decoder_two_steps_match_bruteforce():
    """A transposed conv initialised as bilinear upsampling, a score fusion
    without ReLU, the MSE loss and Eq. 18's gradients: two steps of OracleNet
    against the brute force, every tensor and master."""
    from oracle.model import OracleNet
    wl = TINY_DECODER
    inp = synth.workload_inputs(wl)
    onet = OracleNet(wl, inp, gq=2)
    bnet = B.Net(wl, inp, dict(onet.cfg), gq=2)
    for s in range(2):
        orec = onet.step()
        brec, bloss = B.decoder_step(bnet, inp["x"], inp["x_exp"], inp["labels"], 3)
        for nd in wl["nodes"]:
            _compare_node(orec[nd["name"]], brec[nd["name"]], f"step {s} {nd['name']}")
        assert abs(onet.loss - float(bloss)) <= 1e-12 * float(bloss)
        _compare_params(onet, bnet, 24, 8, onet.cfg)
