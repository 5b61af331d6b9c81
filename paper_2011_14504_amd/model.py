"""One integer training step of a conv / L1BN / ReLU / max-pool stack on the
GPU, built from the libiseg entry points (Sec. 3 dataflow of arXiv
2011.14504).

Forward, per conv layer l:  W_q = Q_W(W_m) (Eq. 8);  Z = SQ8(conv(A, W_q))
(Eq. 15 on the MAC output);  A' = L1BN + ReLU + Q_A (Eq. 12-15).
Backward, in reverse:  L1BN backward (E2, Eq. 16) -> G = Q_G(conv_bwd_weight)
(Eq. 17, stochastic) and E1 = Q_E(conv_bwd_data) (Eq. 16); the raw dgamma /
dbeta sums go through Q_G too.  Update, after the backward:  Eq. 19 on the
24-bit masters of W, gamma and beta (learning rate 2^-lr_shift), then Q_W.

Stochastic rounding keys: seed of the workload, step counter, tensor id
16*l + {0: W, 1: gamma, 2: beta} for conv layer l = 1, 2, ...
"""
import torch

from . import iseg

K_U, K_W = 24, 8
W_MASTER_EXP = 1 - K_U          # -23
GB_MASTER_EXP = 2 - K_U         # -22: gamma/beta quantizers carry the x2 fold


class IntNet:
    def __init__(self, wl, inputs, device="cuda", lr_shift=10, bn_cfg=None):
        self.wl = wl
        self.dev = torch.device(device)
        self.lr_shift = lr_shift
        self.seed = inputs["seed"]
        self.cfg = bn_cfg or iseg.bn_cfg()
        self.step_no = 0
        self.x = torch.from_numpy(inputs["x"]).to(self.dev)
        self.x_exp = iseg.new_exp(self.dev, inputs["x_exp"])
        self.dy = torch.from_numpy(inputs["dy"]).to(self.dev)
        self.dy_exp = iseg.new_exp(self.dev, inputs["dy_exp"])
        self.w_exp = iseg.new_exp(self.dev, W_MASTER_EXP + K_U - K_W)
        self.convs = []
        wi = 0
        for layer in wl["layers"]:
            if layer[0] != "conv":
                continue
            _, cin, cout, R, st, pad, dil = layer
            wf = torch.from_numpy(inputs["weights"][wi]).to(self.dev)
            wi += 1
            master, mexp = iseg.quantize(wf, K_U, iseg.ISEG_Q_UQ)          # Eq. 7
            assert int(mexp.item()) == W_MASTER_EXP
            g_m = torch.full((cout,), 1 << (-GB_MASTER_EXP), dtype=torch.int32, device=self.dev)
            b_m = torch.zeros(cout, dtype=torch.int32, device=self.dev)
            self.convs.append(dict(
                cin=cin, cout=cout, R=R, st=st, pad=pad, dil=dil,
                w_m=master, g_m=g_m, b_m=b_m,
                w_q=iseg.weight_quant(master, K_U, K_W),
                g_q=iseg.weight_quant(g_m, K_U, K_W),
                b_q=iseg.weight_quant(b_m, K_U, K_W)))

    # -------------------------------------------------------------------
    def forward(self):
        a, ae = self.x, self.x_exp
        rec = []
        ci = 0
        for layer in self.wl["layers"]:
            if layer[0] == "conv":
                L = self.convs[ci]
                ci += 1
                z, ze = iseg.conv_fwd(a, ae, L["w_q"], self.w_exp, L["st"], L["pad"], L["dil"])
                y, ye, saved = iseg.bn_fwd(z, ze, L["g_q"], L["b_q"], self.cfg)
                rec.append(dict(kind="conv", L=L, a_in=a, a_in_exp=ae, z=z, z_exp=ze,
                                saved=saved, a_out=y, a_out_exp=ye))
                a, ae = y, ye
            else:
                _, k, st, pad = layer
                y, ye = iseg.maxpool_fwd(a, ae, k, st, pad)
                rec.append(dict(kind="pool", k=k, st=st, pad=pad, a_in=a, a_out=y, a_out_exp=ye))
                a, ae = y, ye
        return rec

    def backward(self, rec):
        e, ee = self.dy, self.dy_exp
        grads = []
        nconv = len(self.convs)
        li = nconv
        for i in range(len(rec) - 1, -1, -1):
            r = rec[i]
            if r["kind"] == "pool":
                e, ee = iseg.maxpool_bwd(e, ee, r["a_in"], r["k"], r["st"], r["pad"])
                r["e_in"], r["e_in_exp"] = e, ee
                continue
            L = r["L"]
            dz, dze, dg, db, dge, dbe = iseg.bn_bwd(e, ee, r["z"], L["g_q"], r["saved"], self.cfg)
            G, Ge = iseg.conv_bwd_weight(dz, dze, r["a_in"], r["a_in_exp"], L["w_q"].shape,
                                         L["st"], L["pad"], L["dil"], iseg.ISEG_G_KEEP, 8,
                                         self.seed, 16 * li, self.step_no)
            r.update(dz=dz, dz_exp=dze, dgamma=dg, dbeta=db, dgamma_exp=dge, dbeta_exp=dbe,
                     G=G, G_exp=Ge, li=li)
            grads.append(r)
            if li > 1 or self.wl["input_grad"]:
                e, ee = iseg.conv_bwd_data(dz, dze, L["w_q"], self.w_exp, r["a_in"].shape,
                                           L["st"], L["pad"], L["dil"])
                r["e_in"], r["e_in_exp"] = e, ee
            li -= 1
        return grads

    def update(self, grads):
        for r in grads:
            L, li = r["L"], r["li"]
            iseg.weight_update(L["w_m"], r["G"], r["G_exp"], self.lr_shift, W_MASTER_EXP, K_U, K_W,
                               L["w_q"])
            C = L["cout"]
            r["Gg"] = torch.empty(C, dtype=torch.int8, device=self.dev)
            r["Gb"] = torch.empty(C, dtype=torch.int8, device=self.dev)
            r["Gg_exp"], r["Gb_exp"] = iseg._out_exp(self.dev), iseg._out_exp(self.dev)
            iseg.iseg_bn_param_update(r["dgamma"], r["dgamma_exp"], r["dbeta"], r["dbeta_exp"], 8,
                                      self.seed, 16 * li + 1, 16 * li + 2, self.step_no,
                                      self.lr_shift, GB_MASTER_EXP, K_U, K_W, L["g_m"], L["b_m"],
                                      L["g_q"], L["b_q"], r["Gg"], r["Gb"], r["Gg_exp"],
                                      r["Gb_exp"])

    def step(self):
        rec = self.forward()
        grads = self.backward(rec)
        self.update(grads)
        self.step_no += 1
        return rec
