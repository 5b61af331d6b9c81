"""Oracle of one integer training step of a conv / L1BN / ReLU / max-pool
stack (TEST INFRASTRUCTURE ONLY), composed from the oracle's functions in the
order of the paper's dataflow (Sec. 3):

  forward   W_q = Q_W(W_m) (Eq. 8); Z = SQ8(conv(A, W_q)) (Eq. 15);
            A' = Q_A(ReLU(L1BN(Z))) (Eq. 12-15); max pooling keeps codes
  backward  L1BN backward -> G = Q_G(sum dy x) (Eq. 17, stochastic),
            E1 = Q_E(sum dy w) (Eq. 16), Q_G of the raw dgamma / dbeta sums
  update    Eq. 19 on the 24-bit masters (lr = 2^-lr_shift), then Eq. 8

Stochastic rounding keys: workload seed, step, tensor id 16*l + {0,1,2} for
W, gamma, beta of conv layer l = 1, 2, ...
"""
import numpy as np

from . import oracle as O

K_U, K_W = 24, 8


class OracleNet:
    def __init__(self, wl, inputs, lr_shift=10, bn_cfg=None):
        self.wl = wl
        self.lr_shift = lr_shift
        self.seed = inputs["seed"]
        self.cfg = dict(O.BN_DEFAULT, **(bn_cfg or {}))
        self.step_no = 0
        self.x, self.x_exp = inputs["x"], inputs["x_exp"]
        self.dy, self.dy_exp = inputs["dy"], inputs["dy_exp"]
        self.w_exp = 1 - K_U + K_U - K_W          # -7
        self.convs = []
        wi = 0
        for layer in wl["layers"]:
            if layer[0] != "conv":
                continue
            _, cin, cout, R, st, pad, dil = layer
            w_m, e = O.master_init(inputs["weights"][wi], K_U)   # Eq. 7
            wi += 1
            g_m = np.full(cout, 1 << (K_U - 2), np.int32)           # gamma = 1 at 2^-22
            b_m = np.zeros(cout, np.int32)
            self.convs.append(dict(cin=cin, cout=cout, R=R, st=st, pad=pad, dil=dil,
                                   w_m=w_m, g_m=g_m, b_m=b_m,
                                   w_q=O.weight_quant(w_m, K_U, K_W),
                                   g_q=O.weight_quant(g_m, K_U, K_W),
                                   b_q=O.weight_quant(b_m, K_U, K_W)))

    @staticmethod
    def _geom(a_shape, L):
        N, H, W, C = a_shape
        return (N, H, W, C, L["cout"], L["R"], L["R"], L["st"], L["st"], L["pad"], L["pad"],
                L["dil"], L["dil"])

    def forward(self):
        a, ae = self.x, self.x_exp
        rec = []
        ci = 0
        for layer in self.wl["layers"]:
            if layer[0] == "conv":
                L = self.convs[ci]
                ci += 1
                z, ze = O.conv_fwd(a, ae, L["w_q"], self.w_exp, self._geom(a.shape, L))
                z = z.astype(np.int8)
                r = O.bn_fwd(z, ze, L["g_q"], L["b_q"], self.cfg)
                rec.append(dict(kind="conv", L=L, a_in=a, a_in_exp=ae, z=z, z_exp=ze,
                                a_out=r["y"], a_out_exp=r["y_exp"], bn=r))
                a, ae = r["y"], r["y_exp"]
            else:
                _, k, st, pad = layer
                y = O.maxpool_fwd(a, k, st, pad)
                rec.append(dict(kind="pool", k=k, st=st, pad=pad, a_in=a, a_out=y, a_out_exp=ae))
                a = y
        return rec

    def backward(self, rec):
        e, ee = self.dy, self.dy_exp
        grads = []
        li = len(self.convs)
        for r in reversed(rec):
            if r["kind"] == "pool":
                e, ee = O.maxpool_bwd(e, ee, r["a_in"], r["k"], r["st"], r["pad"])
                e = e.astype(np.int8)
                r["e_in"], r["e_in_exp"] = e, ee
                continue
            L = r["L"]
            b = O.bn_bwd(e, ee, r["z"], r["z_exp"], L["g_q"], L["b_q"], self.cfg)
            dz, dze = b["dx"], b["dx_exp"]
            geom = self._geom(r["a_in"].shape, L)
            G, Ge = O.conv_bwd_weight(dz, dze, r["a_in"], r["a_in_exp"], geom, 8, True, self.seed,
                                      16 * li, self.step_no)
            Gg, Gge = O.requant(b["dgamma"], b["dgamma_exp"], 8, True, True, self.seed, 16 * li + 1,
                                self.step_no)
            Gb, Gbe = O.requant(b["dbeta"], b["dbeta_exp"], 8, True, True, self.seed, 16 * li + 2,
                                self.step_no)
            r.update(dz=dz, dz_exp=dze, dgamma=b["dgamma"], dbeta=b["dbeta"], G=G, G_exp=Ge,
                     Gg=Gg, Gg_exp=Gge, Gb=Gb, Gb_exp=Gbe)
            grads.append((L, G, Ge, Gg, Gge, Gb, Gbe))
            if li > 1 or self.wl["input_grad"]:
                e, ee = O.conv_bwd_data(dz, dze, L["w_q"], self.w_exp, geom)
                e = e.astype(np.int8)
                r["e_in"], r["e_in_exp"] = e, ee
            li -= 1
        return grads

    def update(self, grads):
        for (L, G, Ge, Gg, Gge, Gb, Gbe) in grads:
            L["w_m"], L["w_q"] = O.weight_update(L["w_m"], G, Ge, self.lr_shift, 1 - K_U, K_U, K_W)
            L["g_m"], L["g_q"] = O.weight_update(L["g_m"], Gg, Gge, self.lr_shift, 2 - K_U, K_U, K_W)
            L["b_m"], L["b_q"] = O.weight_update(L["b_m"], Gb, Gbe, self.lr_shift, 2 - K_U, K_U, K_W)

    def step(self):
        rec = self.forward()
        grads = self.backward(rec)
        self.update(grads)
        self.step_no += 1
        return rec
