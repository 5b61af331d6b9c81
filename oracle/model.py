"""Oracle of one integer training step of a workload graph (TEST
INFRASTRUCTURE ONLY), composed from the oracle's functions in the order of the
paper's dataflow (Sec. 3):

  forward   W_q = Q_W(W_m) (Eq. 8); Z = SQ8(conv(A, W_q)) (Eq. 15); with BN
            A' = Q_A(ReLU?(L1BN(Z))) (Eq. 12-15); max pooling keeps codes;
            residual add, concatenation and global pooling are SQ8 of the
            exact result
  loss      given int8 error at the output, or the float64 softmax
            cross-entropy of the bilinearly upsampled logits whose gradient
            is quantized by SQ8 (the error E1 at the logits)
  backward  nodes in reverse order; the error of a tensor read by several
            nodes is SQ8 of the exact sum of what they send back (Eq. 16);
            L1BN backward -> G = Q_G(sum dy x) (Eq. 17, stochastic), E1 =
            Q_E(sum dy w) (Eq. 16), Q_G of the raw dgamma / dbeta sums
  update    Eq. 19 on the k_U-bit masters (lr = 2^-lr_shift), then Eq. 8

Bit widths (Table 1's rows): k_W for conv weights (W = code 2^(1-k_W)), k_U
for the masters (Eq. 7, 19), k_gamma / k_beta of the BN configuration for the
BN parameters, and k_A for every activation a conv reads: Q_A of the BN
output, the output of a conv without BN, and the forward merges (residual
add, concatenation, global pooling).  A conv feeding BN keeps its output at 8
bits (BN's input), max pooling keeps codes, and errors and gradients stay at
8 bits (k_E1 = k_G = 8 in every row of Table 1).

Stochastic rounding keys: workload seed, step, tensor id 16*l + {0,1,2} for
W, gamma, beta of the l-th conv (l = 1, 2, ... in node order).
"""
import numpy as np

from . import oracle as O

class OracleNet:
    def __init__(self, wl, inputs, lr_shift=10, bn_cfg=None, k_W=8, k_U=24, gq=1, bn_input="q8"):
        self.wl = wl
        # L1BN reads a conv's SQ8 codes ("q8"), or its raw int32 sums ("raw",
        # the literal dataflow of Sec. 3.2.2-3.2.3: BN on the MAC output)
        self.bn_raw = bn_input == "raw"
        self.gq = gq                              # 1: Eq. 17 keeps Scale(G); 2: Eq. 18 drops it
        self.lr_shift = lr_shift
        self.k_W, self.k_U = k_W, k_U
        self.seed = inputs["seed"]
        self.cfg = dict(O.BN_DEFAULT, **(bn_cfg or {}))
        self.step_no = 0
        self.x, self.x_exp = inputs["x"], inputs["x_exp"]
        self.dy, self.dy_exp = inputs.get("dy"), inputs.get("dy_exp")
        self.labels = inputs.get("labels")
        self.k_A = self.cfg["k_A"]
        self.w_exp = 1 - k_W                      # Eq. 8: UQ to k_W bits
        self.convs = {}
        ci = 0
        for nd in wl["nodes"]:
            if nd["kind"] != "conv":
                continue
            w_m, e = O.master_init(inputs["weights"][ci], k_U)   # Eq. 7
            ci += 1
            cout = nd["cout"]
            g_m = np.full(cout, 1 << (k_U - 2), np.int32)           # gamma = 1 at 2^(2-k_U)
            b_m = np.zeros(cout, np.int32)
            self.convs[nd["name"]] = dict(l=ci, w_m=w_m, g_m=g_m, b_m=b_m,
                                          w_q=O.weight_quant(w_m, k_U, k_W),
                                          g_q=O.weight_quant(g_m, k_U, self.cfg["k_gamma"]),
                                          b_q=O.weight_quant(b_m, k_U, self.cfg["k_beta"]))
        self.loss = None

    def _bn_cfg(self, nd):
        return dict(self.cfg, relu=int(nd["relu"]))

    @staticmethod
    def _tgeom(a_shape, nd):
        """Geometry of the conv a transposed-conv node is the adjoint of: its
        input has the node's output shape, its output the node's input shape."""
        N, h, w, cin = a_shape
        H = (h - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
        W = (w - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
        return (N, H, W, nd["cout"], cin, nd["R"], nd["R"], nd["stride"], nd["stride"], nd["pad"],
                nd["pad"], nd["dil"], nd["dil"])

    @staticmethod
    def _geom(a_shape, nd):
        N, H, W, C = a_shape
        return (N, H, W, C, nd["cout"], nd["R"], nd["R"], nd["stride"], nd["stride"], nd["pad"],
                nd["pad"], nd["dil"], nd["dil"])

    # ------------------------------------------------------------------
    def forward(self):
        act = {"input": (self.x, self.x_exp)}
        rec = {}
        for nd in self.wl["nodes"]:
            k, name = nd["kind"], nd["name"]
            a, ae = act[nd["src"][0]]
            r = dict(kind=k, a_in=a, a_in_exp=ae)
            if k == "conv":
                L = self.convs[name]
                if nd.get("transposed"):
                    # the adjoint of the conv whose input has this node's output shape
                    z, ze = O.conv_bwd_data(a, ae, L["w_q"], self.w_exp, self._tgeom(a.shape, nd))
                    z = z.astype(np.int8)
                elif self.bn_raw and nd["bn"]:
                    # |sum| < 2^31 (the reduction bound), so int32 holds it
                    z, ze = O.conv_fwd_raw(a, L["w_q"], self._geom(a.shape, nd)).astype(np.int32), ae + self.w_exp
                else:
                    z, ze = O.conv_fwd(a, ae, L["w_q"], self.w_exp, self._geom(a.shape, nd))
                    z = z.astype(np.int8)
                r.update(z=z, z_exp=ze)
                if nd["bn"]:
                    b = O.bn_fwd(z, ze, L["g_q"], L["b_q"], self._bn_cfg(nd))
                    y, ye = b["y"], b["y_exp"]
                    r["bn_state"] = O.bn_state(b)
                elif nd["relu"] or self.k_A < 8:
                    # without BN: A = Q_A(ReLU?(Z)) on the 8-bit conv output
                    y, ye = O.sum_requant([z], [ze], self.k_A, relu=nd["relu"])
                    y = y.astype(np.int8)
                else:
                    y, ye = z, ze
            elif k == "maxpool":
                y, ye = O.maxpool_fwd(a, nd["k"], nd["stride"], nd["pad"]), ae
            elif k == "add":
                b_, be = act[nd["src"][1]]
                y, ye = O.sum_requant([a, b_], [ae, be], self.k_A, relu=nd["relu"])
                y = y.astype(np.int8)
                r.update(b_in=b_, b_in_exp=be)
            elif k == "gap":
                y, ye = O.gap_fwd(a, ae, self.k_A)
                y = y.astype(np.int8)
            elif k == "concat":
                parts = [act[s] for s in nd["src"]]
                H = max(p[0].shape[1] for p in parts)
                W = max(p[0].shape[2] for p in parts)
                y, ye = O.concat_requant([p[0] for p in parts], [p[1] for p in parts], (H, W),
                                         self.k_A)
                y = y.astype(np.int8)
                r.update(widths=[p[0].shape[3] for p in parts],
                         bcast=[p[0].shape[1:3] != (H, W) for p in parts])
            else:
                raise ValueError(k)
            r.update(a_out=y, a_out_exp=ye)
            rec[name] = r
            act[name] = (y, ye)
        return rec

    # ------------------------------------------------------------------
    def loss_error(self, rec):
        """The error arriving at the output node, and the loss if any."""
        out = rec[self.wl["nodes"][-1]["name"]]
        if self.wl["loss"] == "given":
            return self.dy, self.dy_exp
        if self.wl["loss"] == "mse":
            loss, e, ee = O.mse_onehot(out["a_out"], out["a_out_exp"], self.labels)
            self.loss = loss
            return e.astype(np.int8), ee
        loss, grad = O.softmax_ce(out["a_out"], out["a_out_exp"], self.labels)
        e, ee = O.quantize_f64(grad, 8)
        self.loss, self.loss_grad = loss, grad
        return e.astype(np.int8), ee

    def backward(self, rec):
        contrib = {}

        def send(name, codes, exp):
            contrib.setdefault(name, []).append((codes, exp))

        def merged(name):
            parts = contrib.pop(name)
            if len(parts) == 1:
                return parts[0]
            e, ee = O.sum_requant([p[0] for p in parts], [p[1] for p in parts], 8)
            return e.astype(np.int8), ee

        e, ee = self.loss_error(rec)
        send(self.wl["nodes"][-1]["name"], e, ee)
        want_input = self.wl["input_grad"]
        grads = []
        for nd in reversed(self.wl["nodes"]):
            k, name = nd["kind"], nd["name"]
            r = rec[name]
            e, ee = merged(name)
            r.update(e_out=e, e_out_exp=ee)
            src = nd["src"][0]
            need_in = src != "input" or want_input
            if k == "conv":
                L = self.convs[name]
                if nd["bn"]:
                    b = O.bn_bwd(e, ee, r["z"], r["z_exp"], L["g_q"], L["b_q"], self._bn_cfg(nd))
                    dz, dze = b["dx"], b["dx_exp"]
                    l = L["l"]
                    Gg, Gge = O.requant(b["dgamma"], b["dgamma_exp"], 8, True, True, self.seed,
                                        16 * l + 1, self.step_no)
                    Gb, Gbe = O.requant(b["dbeta"], b["dbeta_exp"], 8, True, True, self.seed,
                                        16 * l + 2, self.step_no)
                    r.update(dgamma=b["dgamma"], dbeta=b["dbeta"], dgamma_exp=b["dgamma_exp"],
                             dbeta_exp=b["dbeta_exp"], Gg=Gg, Gg_exp=Gge, Gb=Gb, Gb_exp=Gbe)
                elif nd["relu"]:
                    dz, dze = O.relu_mask_bwd(e, [r["z"]], [r["z_exp"]]), ee
                else:
                    dz, dze = e, ee
                if nd.get("transposed"):
                    # the adjoint conv's weight gradient pairs this node's input
                    # (the conv's output side) with dz (its input side); the
                    # input error is that conv's forward of dz
                    geom = self._tgeom(r["a_in"].shape, nd)
                    G, Ge = O.conv_bwd_weight(r["a_in"], r["a_in_exp"], dz, dze, geom, 8, self.gq == 1,
                                              self.seed, 16 * L["l"], self.step_no)
                else:
                    geom = self._geom(r["a_in"].shape, nd)
                    G, Ge = O.conv_bwd_weight(dz, dze, r["a_in"], r["a_in_exp"], geom, 8, self.gq == 1,
                                              self.seed, 16 * L["l"], self.step_no)
                r.update(dz=dz, dz_exp=dze, G=G, G_exp=Ge)
                grads.append((nd, r))
                if need_in and nd.get("transposed"):
                    ei, eie = O.conv_fwd(dz, dze, L["w_q"], self.w_exp, geom)
                    ei = ei.astype(np.int8)
                    r.update(e_in=ei, e_in_exp=eie)
                    send(src, ei, eie)
                elif need_in:
                    ei, eie = O.conv_bwd_data(dz, dze, L["w_q"], self.w_exp, geom)
                    ei = ei.astype(np.int8)
                    r.update(e_in=ei, e_in_exp=eie)
                    send(src, ei, eie)
            elif k == "maxpool":
                if need_in:
                    ei, eie = O.maxpool_bwd(e, ee, r["a_in"], nd["k"], nd["stride"], nd["pad"])
                    ei = ei.astype(np.int8)
                    r.update(e_in=ei, e_in_exp=eie)
                    send(src, ei, eie)
            elif k == "add":
                d = (O.relu_mask_bwd(e, [r["a_in"], r["b_in"]], [r["a_in_exp"], r["b_in_exp"]])
                     if nd["relu"] else e)
                r.update(e_in=d, e_in_exp=ee)
                for s in nd["src"]:
                    if s != "input" or want_input:
                        send(s, d, ee)
            elif k == "gap":
                if need_in:
                    H, W = r["a_in"].shape[1:3]
                    eg, ege = O.gap_bwd(e, ee, H, W)
                    r.update(e_in=eg.astype(np.int8), e_in_exp=ege)
                    send(src, eg.astype(np.int8), ege)
            elif k == "concat":
                parts = O.concat_split(e, r["widths"])
                for s, p, bc in zip(nd["src"], parts, r["bcast"]):
                    if bc:
                        pe, pee = O.bcast_bwd(p, ee)
                        send(s, pe.astype(np.int8), pee)
                    else:
                        send(s, p, ee)
        if want_input:
            e, ee = merged("input")
            rec["input"] = dict(kind="input", e_out=e, e_out_exp=ee)
        return grads

    def update(self, grads):
        k_U, k_W, cf = self.k_U, self.k_W, self.cfg
        for nd, r in grads:
            L = self.convs[nd["name"]]
            L["w_m"], L["w_q"] = O.weight_update(L["w_m"], r["G"], r["G_exp"], self.lr_shift,
                                                 1 - k_U, k_U, k_W)
            if nd["bn"]:
                L["g_m"], L["g_q"] = O.weight_update(L["g_m"], r["Gg"], r["Gg_exp"], self.lr_shift,
                                                     2 - k_U, k_U, cf["k_gamma"])
                L["b_m"], L["b_q"] = O.weight_update(L["b_m"], r["Gb"], r["Gb_exp"], self.lr_shift,
                                                     2 - k_U, k_U, cf["k_beta"])

    def infer(self, calib, x, x_exp):
        """Forward of a chain of conv + L1BN (+ReLU) layers and max pooling in
        inference with the frozen state of a calibration forward `calib` (the
        record forward() returned): each conv's sums go to the calibration's
        Z grid (a fixed-step quantizer), then L1BN + ReLU + Q_A with the
        calibration's statistics and steps.  Returns {node: (codes, exp)}."""
        act = {"input": (x, x_exp)}
        out = {}
        for nd in self.wl["nodes"]:
            a, ae = act[nd["src"][0]]
            if nd["kind"] == "conv":
                if not nd["bn"]:
                    raise ValueError("inference covers conv layers with L1BN")
                L, c = self.convs[nd["name"]], calib[nd["name"]]
                sums = O.conv_fwd_raw(a, L["w_q"], self._geom(a.shape, nd))
                z = O.requant_fixed(sums, ae + self.w_exp, c["z_exp"], 8)
                y = O.bn_infer(z, c["z_exp"], L["g_q"], L["b_q"], c["bn_state"], self._bn_cfg(nd))
                res = (y, c["bn_state"]["a_exp"])
            elif nd["kind"] == "maxpool":
                res = (O.maxpool_fwd(a, nd["k"], nd["stride"], nd["pad"]), ae)
            else:
                raise ValueError("inference covers chains of conv layers and max pooling")
            out[nd["name"]] = res
            act[nd["name"]] = res
        return out

    def step(self):
        rec = self.forward()
        grads = self.backward(rec)
        self.update(grads)
        self.step_no += 1
        return rec
