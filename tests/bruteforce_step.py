"""Exact-rational brute force of whole training steps (test infrastructure).

Rebuilds one training step of small networks straight from the paper's
real-valued formulas (arXiv 2011.14504, Sec. 3), independently of the oracle
and of its graph interpreter: tensors are arrays of Python Fractions, every
quantizer is the equation applied to those values, and each network's
forward, backward and update are written out by hand in the order of the
dataflow (Fig. 4 forward, Fig. 5 backward), not interpreted from a graph.

Readings taken (the same ones the rest of the build takes, restated here so
that a misreading in the oracle's composition shows up as a mismatch):
  * Scale(x) is the smallest power of two strictly above max|x| (Eq. 3-4);
  * a conv output is SQ8 of the exact MAC result (Eq. 15 before BN), or with
    bn_input="raw" the exact MAC result itself when BN follows; with BN,
    A = SQ_kA(ReLU?(L1BN(Z))) (Eq. 12-15); without BN, A = SQ_kA(ReLU?(Z)),
    whose backward passes the error where Z > 0;
  * a residual add is SQ_kA(ReLU(a + b)); its backward passes the error where
    a + b > 0 to both inputs unchanged;
  * a tensor read by several nodes receives SQ8 of the exact sum of the errors
    they send back (Eq. 16); one consumer's error passes unchanged;
  * G = conv of the error with the input, then Q_G: Eq. 5-6 stochastic
    rounding with U the Philox4x32-10 draw of the element (key (seed,
    16 l + object), counter (index, step)) over 2^64, keeping Scale(G)
    (Eq. 17) or dropping it (Eq. 18); dgamma, dbeta keep their scale;
  * Eq. 19 then Eq. 8 on the masters, lr = 2^-lr_shift; gamma and beta carry
    Eq. 14's fixed x2 fold in their masters and updates.
Convolution sums are formed exactly on integer grids (numpy int64 tap loops
written here; every value of a quantized tensor is an integer multiple of one
power of two), everything else in Fractions.
"""
import math
from fractions import Fraction as Fr

import numpy as np

import bruteforce as bf

MASK32 = 0xFFFFFFFF


# ---------------------------------------------------------------------------
# Philox4x32-10 (Salmon et al., SC'11), written from the published definition
# ---------------------------------------------------------------------------
def philox4x32_10(ctr, key):
    m0, m1 = 0xD2511F53, 0xCD9E8D57
    w0, w1 = 0x9E3779B9, 0xBB67AE85
    c0, c1, c2, c3 = ctr
    k0, k1 = key
    for _ in range(10):
        p0, p1 = m0 * c0, m1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0) & MASK32, p1 & MASK32, \
                         ((p0 >> 32) ^ c3 ^ k1) & MASK32, p0 & MASK32
        k0, k1 = (k0 + w0) & MASK32, (k1 + w1) & MASK32
    return [c0, c1, c2, c3]


def uniform(seed, tensor_id, step, idx):
    """U in [0, 1) of Eq. 5-6 for one element: the 64-bit draw over 2^64."""
    w = philox4x32_10([idx & MASK32, idx >> 32, step, 0], [seed & MASK32, tensor_id])
    return Fr(w[0] | (w[1] << 32), 1 << 64)


# ---------------------------------------------------------------------------
# tensors of rationals
# ---------------------------------------------------------------------------
def values(codes, exp):
    """Object array of Fractions code * 2^exp."""
    s = Fr(2) ** int(exp)
    a = np.empty(np.shape(codes), dtype=object)
    for i, c in zip(np.ndindex(a.shape), np.ravel(codes)):
        a[i] = Fr(int(c)) * s
    return a


def SQ(arr, k):
    """Eq. 4 on a whole tensor: (values, exponent of the step S Delta), the
    exponent None for an all-zero tensor."""
    flat = list(arr.ravel())
    S = bf.pow2_scale(flat)
    if S is None:
        return np.full(arr.shape, Fr(0), dtype=object), None
    q = np.array([S * bf.UQ(v / S, k) for v in flat], dtype=object).reshape(arr.shape)
    return q, int(math.log2(S * bf.delta(k)))


def RQ(arr, k, keep_scale, seed, tensor_id, step):
    """Eq. 5-6 (Eq. 17 with the scale kept, Eq. 18 without) of a tensor whose
    elements are indexed in C order."""
    flat = list(arr.ravel())
    S = bf.pow2_scale(flat)
    d = bf.delta(k)
    if S is None:
        return np.full(arr.shape, Fr(0), dtype=object), (None if keep_scale else 1 - k)
    out = []
    for idx, v in enumerate(flat):
        y = v / S / d
        n = math.floor(y)
        if uniform(seed, tensor_id, step, idx) < y - n:
            n += 1
        q = bf.clip(d * n, -1 + d, 1 - d)
        out.append(S * q if keep_scale else q)
    e = int(math.log2(S * d)) if keep_scale else 1 - k
    return np.array(out, dtype=object).reshape(arr.shape), e


def relu(arr):
    return np.vectorize(lambda v: max(v, Fr(0)), otypes=[object])(arr)


def positive(arr):
    return np.vectorize(lambda v: v > 0, otypes=[bool])(arr)


def masked(arr, mask):
    return np.where(mask, arr, Fr(0))


def _grid(arr):
    """(int64 array, D) with arr == ints / D exactly (D a power of two)."""
    D = max((v.denominator for v in arr.ravel()), default=1)
    assert D & (D - 1) == 0
    ints = np.array([int(v * D) for v in arr.ravel()], dtype=np.int64).reshape(arr.shape)
    assert np.abs(ints).max(initial=0) < 2 ** 31
    return ints, D


def _from_ints(ints, D):
    out = np.empty(ints.shape, dtype=object)
    for i in np.ndindex(ints.shape):
        out[i] = Fr(int(ints[i]), D)
    return out


def _padded(x, pad):
    N, H, W, C = x.shape
    xp = np.zeros((N, H + 2 * pad, W + 2 * pad, C), dtype=np.int64)
    xp[:, pad:pad + H, pad:pad + W] = x
    return xp


def _out_hw(H, W, R, st, pad, dil):
    return (H + 2 * pad - dil * (R - 1) - 1) // st + 1, (W + 2 * pad - dil * (R - 1) - 1) // st + 1


def conv(x, w, st, pad, dil):
    """Cross-correlation with zero padding of rational tensors x [N,H,W,C] and
    w [K,R,S,C]: one integer matrix product per tap."""
    xi, dx = _grid(x)
    wi, dw = _grid(w)
    N, H, W, C = xi.shape
    K, R, S, _ = wi.shape
    P, Q = _out_hw(H, W, R, st, pad, dil)
    xp = _padded(xi, pad)
    out = np.zeros((N, P, Q, K), dtype=np.int64)
    for r in range(R):
        for s in range(S):
            patch = xp[:, r * dil: r * dil + st * (P - 1) + 1: st, s * dil: s * dil + st * (Q - 1) + 1: st]
            out += patch @ wi[:, r, s, :].T
    return _from_ints(out, dx * dw)


def conv_data_grad(dy, w, H, W, st, pad, dil):
    """Gradient of conv w.r.t. its input: every output term sends dy * w back
    to the input position it read (the transpose of conv, written as that
    scatter)."""
    gi, dg = _grid(dy)
    wi, dw = _grid(w)
    N, P, Q, K = gi.shape
    _, R, S, C = wi.shape
    xp = np.zeros((N, H + 2 * pad, W + 2 * pad, C), dtype=np.int64)
    for r in range(R):
        for s in range(S):
            xp[:, r * dil: r * dil + st * (P - 1) + 1: st,
               s * dil: s * dil + st * (Q - 1) + 1: st] += gi @ wi[:, r, s, :]
    return _from_ints(xp[:, pad:pad + H, pad:pad + W], dg * dw)


def conv_weight_grad(dy, x, R, st, pad, dil):
    """Gradient of conv w.r.t. its weights: G[k,r,s,c] = sum over output
    positions of dy times the input value that tap read."""
    gi, dg = _grid(dy)
    xi, dx = _grid(x)
    N, P, Q, K = gi.shape
    C = xi.shape[3]
    xp = _padded(xi, pad)
    G = np.zeros((K, R, R, C), dtype=np.int64)
    for r in range(R):
        for s in range(R):
            patch = xp[:, r * dil: r * dil + st * (P - 1) + 1: st, s * dil: s * dil + st * (Q - 1) + 1: st]
            G[:, r, s, :] = gi.reshape(-1, K).T @ patch.reshape(-1, C)
    return _from_ints(G, dg * dx)


# ---------------------------------------------------------------------------
# layers
# ---------------------------------------------------------------------------
def channels(arr):
    """Per-channel columns of an NHWC tensor (the L1BN batch of each channel)."""
    C = arr.shape[-1]
    flat = arr.reshape(-1, C)
    return [list(flat[:, c]) for c in range(C)]


def from_channels(cols, shape):
    out = np.empty(shape, dtype=object)
    flat = out.reshape(-1, shape[-1])
    for c, col in enumerate(cols):
        flat[:, c] = col
    return out


def bn_forward(z, gamma, beta, cfg):
    """L1BN (Eq. 12-14) + ReLU? + Q_A (Eq. 15): A values and exponent."""
    f = bf.l1bn_forward(channels(z), gamma, beta, cfg)
    y = from_channels(f["y"], z.shape)
    return SQ(relu(y) if cfg["relu"] else y, cfg["k_A"])


def bn_backward(z, dA, gamma, beta, cfg):
    """Exact derivative of Eq. 12-13 with straight-through quantizers:
    E1 (values, exponent) and the raw dgamma, dbeta per channel."""
    b = bf.l1bn_backward(channels(z), channels(dA), gamma, beta, cfg)
    pre = from_channels(b["dx_pre"], z.shape)
    e1, e1_exp = SQ(pre, cfg["k_E1"])
    return e1, e1_exp, b["dgamma"], b["dbeta"]


def fold_quant(master, k):
    """Eq. 14: 2 UQ(v/2, k) of gamma / beta."""
    return [2 * bf.UQ(v / 2, k) for v in master]


class Net:
    """Parameters of a network: per conv layer, the float weights turned
    into masters by Eq. 7, W_q by Eq. 8, and gamma = 1, beta = 0 masters."""

    def __init__(self, wl, inputs, cfg, k_W=8, k_U=24, lr_shift=10, gq=1, bn_input="q8"):
        self.cfg, self.k_W, self.k_U, self.lr, self.gq = cfg, k_W, k_U, Fr(1, 2 ** lr_shift), gq
        # "raw": L1BN reads the exact MAC output instead of its SQ8 codes
        self.bn_raw = bn_input == "raw"
        self.seed = inputs["seed"]
        self.L = {}
        convs = [nd for nd in wl["nodes"] if nd["kind"] == "conv"]
        for i, nd in enumerate(convs):
            wf = inputs["weights"][i]
            w_m = np.array([bf.UQ(Fr(float(v)), k_U) for v in wf.ravel()],
                           dtype=object).reshape(wf.shape)                     # Eq. 7
            self.L[nd["name"]] = dict(l=i + 1, nd=nd, w_m=w_m, g_m=[Fr(1)] * nd["cout"],
                                      b_m=[Fr(0)] * nd["cout"])
        self.step_no = 0

    def w_q(self, name):
        w = self.L[name]["w_m"]
        return np.array([bf.UQ(v, self.k_W) for v in w.ravel()], dtype=object).reshape(w.shape)  # Eq. 8

    def gamma_beta(self, name):
        L = self.L[name]
        return fold_quant(L["g_m"], self.cfg["k_gamma"]), fold_quant(L["b_m"], self.cfg["k_beta"])

    # --- one conv node ------------------------------------------------------
    def conv_forward(self, name, a):
        """Z = SQ8(conv(A, W_q)) (Eq. 15 on the MAC output) and A' of the
        node: with BN, Q_A(ReLU?(L1BN(Z))); without, Q_A(ReLU?(Z))."""
        nd = self.L[name]["nd"]
        if nd.get("transposed"):
            # the adjoint of the conv whose input has this node's output shape
            H = (a.shape[1] - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
            W = (a.shape[2] - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
            acc = conv_data_grad(a, self.w_q(name), H, W, nd["stride"], nd["pad"], nd["dil"])
        else:
            acc = conv(a, self.w_q(name), nd["stride"], nd["pad"], nd["dil"])
        if self.bn_raw and nd["bn"]:
            z, z_exp = acc, None          # the MAC output itself (exponent not compared)
        else:
            z, z_exp = SQ(acc, 8)
        cfg = dict(self.cfg, relu=int(nd["relu"]))
        if nd["bn"]:
            g, b = self.gamma_beta(name)
            out, out_exp = bn_forward(z, g, b, cfg)
        elif nd["relu"] or cfg["k_A"] < 8:
            out, out_exp = SQ(relu(z) if nd["relu"] else z, cfg["k_A"])
        else:
            out, out_exp = z, z_exp
        return dict(a_in=a, z=z, z_exp=z_exp, a_out=out, a_out_exp=out_exp)

    def conv_backward(self, name, r, e, e_exp, want_input):
        """L1BN backward (or the ReLU mask), then G = Q_G(dz * x) and the
        error at the input E1 = Q_E(dz * w) (Eq. 16-18)."""
        L = self.L[name]
        nd, l, step = L["nd"], L["l"], self.step_no
        cfg = dict(self.cfg, relu=int(nd["relu"]))
        if nd["bn"]:
            g, b = self.gamma_beta(name)
            dz, dz_exp, dgam, dbet = bn_backward(r["z"], e, g, b, cfg)
            r["dgamma"], r["dbeta"] = dgam, dbet
            r["Gg"], r["Gg_exp"] = RQ(np.array(dgam, dtype=object), 8, True, self.seed, 16 * l + 1, step)
            r["Gb"], r["Gb_exp"] = RQ(np.array(dbet, dtype=object), 8, True, self.seed, 16 * l + 2, step)
        elif nd["relu"]:
            dz, dz_exp = masked(e, positive(r["z"])), e_exp
        else:
            dz, dz_exp = e, e_exp
        r["dz"], r["dz_exp"] = dz, dz_exp
        if nd.get("transposed"):
            # the adjoint conv reads dz and writes this node's input: its weight
            # gradient pairs the node's input with dz, its forward gives E1
            Gsum = conv_weight_grad(r["a_in"], dz, nd["R"], nd["stride"], nd["pad"], nd["dil"])
            r["G"], r["G_exp"] = RQ(Gsum, 8, self.gq == 1, self.seed, 16 * l, step)
            if want_input:
                r["e_in"], r["e_in_exp"] = SQ(conv(dz, self.w_q(name), nd["stride"], nd["pad"], nd["dil"]), 8)
            return r
        Gsum = conv_weight_grad(dz, r["a_in"], nd["R"], nd["stride"], nd["pad"], nd["dil"])
        r["G"], r["G_exp"] = RQ(Gsum, 8, self.gq == 1, self.seed, 16 * l, step)
        if want_input:
            H, W = r["a_in"].shape[1:3]
            r["e_in"], r["e_in_exp"] = SQ(conv_data_grad(dz, self.w_q(name), H, W, nd["stride"],
                                                         nd["pad"], nd["dil"]), 8)
        return r

    # --- Eq. 19, then Eq. 8 / 14 ----------------------------------------------
    def update(self, recs):
        d = bf.delta(self.k_U)
        for name, L in self.L.items():
            r = recs[name]
            step = [bf.UQ(v * self.lr, self.k_U) for v in r["G"].ravel()]
            L["w_m"] = np.array([bf.clip(m - s, -1 + d, 1 - d) for m, s in zip(L["w_m"].ravel(), step)],
                                dtype=object).reshape(L["w_m"].shape)
            if L["nd"]["bn"]:
                for key, gkey in (("g_m", "Gg"), ("b_m", "Gb")):
                    L[key] = [2 * bf.clip(m / 2 - bf.UQ(gv * self.lr / 2, self.k_U), -1 + d, 1 - d)
                              for m, gv in zip(L[key], r[gkey].ravel())]
        self.step_no += 1


def merge(parts):
    """The error of a tensor several nodes read: SQ8 of the exact sum of what
    they send back (Eq. 16); a single contribution passes unchanged."""
    if len(parts) == 1:
        return parts[0]
    total = parts[0][0]
    for p in parts[1:]:
        total = total + p[0]
    return SQ(total, 8)


# ---------------------------------------------------------------------------
# networks, written out by hand
# ---------------------------------------------------------------------------
def single_conv_step(net, x, x_exp, dy, dy_exp):
    """Workload 1: conv -> L1BN -> ReLU -> Q_A, the error dy given at A; the
    input gradient is taken."""
    a = values(x, x_exp)
    r = net.conv_forward("conv", a)
    e = values(dy, dy_exp)
    r["e_out"], r["e_out_exp"] = e, dy_exp
    net.conv_backward("conv", r, e, dy_exp, True)
    recs = {"conv": r}
    net.update(recs)
    return recs


def bottleneck_forward(net, p, a, a_exp, proj):
    """A ResNet v1.5 bottleneck: conv1 -> conv2 -> conv3 (its BN without
    ReLU), the shortcut (a projection conv with BN and no ReLU, or the input
    itself), then A = Q_A(ReLU(conv3 + shortcut))."""
    recs = {}
    r1 = net.conv_forward(p + ".conv1", a)
    r2 = net.conv_forward(p + ".conv2", r1["a_out"])
    r3 = net.conv_forward(p + ".conv3", r2["a_out"])
    recs[p + ".conv1"], recs[p + ".conv2"], recs[p + ".conv3"] = r1, r2, r3
    if proj:
        rp = net.conv_forward(p + ".proj", a)
        recs[p + ".proj"] = rp
        sc, sc_exp = rp["a_out"], rp["a_out_exp"]
    else:
        sc, sc_exp = a, a_exp
    s = r3["a_out"] + sc
    out, out_exp = SQ(relu(s), net.cfg["k_A"])
    recs[p + ".out"] = dict(sum=s, a_out=out, a_out_exp=out_exp)
    return recs, out, out_exp


def bottleneck_backward(net, p, recs, e, e_exp, proj, want_input):
    """Returns the errors the block sends to its input: from conv1 and from
    the shortcut (the projection's E1, or the masked error itself)."""
    ro = recs[p + ".out"]
    ro["e_out"], ro["e_out_exp"] = e, e_exp
    d = masked(e, positive(ro["sum"]))           # ReLU after the add
    ro["e_in"], ro["e_in_exp"] = d, e_exp
    to_input = []
    # conv3 <- d, conv2 <- conv3's E1, conv1 <- conv2's E1
    r3, r2, r1 = recs[p + ".conv3"], recs[p + ".conv2"], recs[p + ".conv1"]
    r3["e_out"], r3["e_out_exp"] = d, e_exp
    net.conv_backward(p + ".conv3", r3, d, e_exp, True)
    r2["e_out"], r2["e_out_exp"] = r3["e_in"], r3["e_in_exp"]
    net.conv_backward(p + ".conv2", r2, r3["e_in"], r3["e_in_exp"], True)
    r1["e_out"], r1["e_out_exp"] = r2["e_in"], r2["e_in_exp"]
    net.conv_backward(p + ".conv1", r1, r2["e_in"], r2["e_in_exp"], want_input)
    if want_input:
        to_input.append((r1["e_in"], r1["e_in_exp"]))
    if proj:
        rp = recs[p + ".proj"]
        rp["e_out"], rp["e_out_exp"] = d, e_exp
        net.conv_backward(p + ".proj", rp, d, e_exp, want_input)
        if want_input:
            to_input.append((rp["e_in"], rp["e_in_exp"]))
    elif want_input:
        to_input.append((d, e_exp))
    return to_input


def stage_step(net, x, x_exp, dy, dy_exp, prefix, blocks):
    """A residual stage of `blocks` bottlenecks (the first with a projection)
    with the error dy given at its output and the input gradient taken."""
    a, a_exp = values(x, x_exp), x_exp
    recs, outs = {}, []
    for b in range(blocks):
        rb, a, a_exp = bottleneck_forward(net, f"{prefix}.{b}", a, a_exp, b == 0)
        recs.update(rb)
        outs.append((a, a_exp))
    e, e_exp = values(dy, dy_exp), dy_exp
    for b in reversed(range(blocks)):
        parts = bottleneck_backward(net, f"{prefix}.{b}", recs, e, e_exp, b == 0, True)
        e, e_exp = merge(parts)
    recs["input"] = dict(e_out=e, e_out_exp=e_exp)
    net.update({k: v for k, v in recs.items() if k in net.L})
    return recs


def mse_error(y, labels, classes):
    """The MSE loss of y against one-hot labels, mean over every element, and
    E1 = SQ8 of its gradient 2 (y - t) / (number of elements)."""
    t = np.zeros(y.shape, dtype=object)
    for idx in np.ndindex(labels.shape):
        for k in range(classes):
            t[idx + (k,)] = Fr(int(labels[idx] == k))
    D = y.size
    diff = y - t
    loss = sum((v * v for v in diff.ravel()), Fr(0)) / D
    return loss, SQ(diff * Fr(2, D), 8)


def decoder_step(net, x, x_exp, labels, classes):
    """A tiny FCN-style decoder: c1 = ReLU conv 3x3 stride 2 (no BN), s1 = 1x1
    score conv on c1, up = transposed conv x2 (4x4, stride 2, pad 1) of s1,
    s0 = 1x1 score conv on the input, fuse = Q_A(up + s0) without ReLU; the
    MSE loss on fuse; no input gradient."""
    a = values(x, x_exp)
    recs = {}
    recs["c1"] = net.conv_forward("c1", a)
    recs["s1"] = net.conv_forward("s1", recs["c1"]["a_out"])
    recs["up"] = net.conv_forward("up", recs["s1"]["a_out"])
    recs["s0"] = net.conv_forward("s0", a)
    s = recs["up"]["a_out"] + recs["s0"]["a_out"]
    out, out_exp = SQ(s, net.cfg["k_A"])
    recs["fuse"] = dict(a_out=out, a_out_exp=out_exp)
    loss, (e, e_exp) = mse_error(out, labels, classes)
    recs["fuse"].update(e_out=e, e_out_exp=e_exp, e_in=e, e_in_exp=e_exp)
    # the sum passes its error to both inputs unchanged
    for name in ("up", "s0"):
        recs[name]["e_out"], recs[name]["e_out_exp"] = e, e_exp
    net.conv_backward("s0", recs["s0"], e, e_exp, False)
    net.conv_backward("up", recs["up"], e, e_exp, True)
    recs["s1"]["e_out"], recs["s1"]["e_out_exp"] = recs["up"]["e_in"], recs["up"]["e_in_exp"]
    net.conv_backward("s1", recs["s1"], recs["up"]["e_in"], recs["up"]["e_in_exp"], True)
    recs["c1"]["e_out"], recs["c1"]["e_out_exp"] = recs["s1"]["e_in"], recs["s1"]["e_in_exp"]
    net.conv_backward("c1", recs["c1"], recs["s1"]["e_in"], recs["s1"]["e_in_exp"], False)
    net.update({k: v for k, v in recs.items() if k in net.L})
    return recs, loss
