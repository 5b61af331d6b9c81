"""One integer training step of a workload graph on the GPU, built from the
libiseg entry points (Sec. 3 dataflow of arXiv 2011.14504).

Forward, in node order:  conv: W_q = Q_W(W_m) (Eq. 8), Z = SQ8(conv(A, W_q))
(Eq. 15 on the MAC output), then with BN A' = Q_A(ReLU?(L1BN(Z))) (Eq. 12-15);
max pooling keeps codes; residual add (+ReLU), concatenation and global
average pooling are SQ8 of their exact result.
Loss:  a given int8 error at the output, or the float64 softmax cross-entropy
of the bilinearly upsampled logits, whose gradient is quantized to E1.
Backward, in reverse node order:  the error of a tensor read by several nodes
is SQ8 of the exact sum of their contributions (Eq. 16); L1BN backward (E2) ->
G = Q_G(conv_bwd_weight) (Eq. 17, stochastic) and E1 = Q_E(conv_bwd_data);
the raw dgamma / dbeta sums go through Q_G too.
Update, after the backward:  Eq. 19 on the k_U-bit masters of W, gamma and
beta (learning rate 2^-lr_shift), then Q_W.

Bit widths (Table 1's rows): k_W for conv weights, k_U for the masters,
k_gamma / k_beta of the BN configuration for the BN parameters (their own
width in the update table), k_A for every activation a conv reads (Q_A of the
BN output, Q_A(ReLU?(Z)) after a conv without BN, the forward merges).  Every
conv output Z is 8 bits; errors and gradients stay at 8 bits.  gq selects
Q_G: Eq. 17 keeps Scale(G) (GQ1), Eq. 18 drops it (GQ2).  Codes of
fewer than 8 bits run through the same int8 kernels.

Stochastic rounding keys: seed of the workload, step counter, tensor id
16*l + {0: W, 1: gamma, 2: beta} for the l-th conv (l = 1, 2, ... in node
order).
"""
import torch

from . import iseg

class IntNet:
    def __init__(self, wl, inputs, device="cuda", lr_shift=10, bn_cfg=None, k_W=8, k_U=24, gq=1,
                 bn_input="q8", branch_streams=2, replay_from=None):
        if not (2 <= k_W <= 8 and 9 <= k_U <= 31 and gq in (1, 2)):
            raise ValueError("k_W must be in [2, 8], k_U in [9, 31], gq 1 or 2")
        if bn_input not in ("q8", "raw"):
            raise ValueError("bn_input is 'q8' (BN on the SQ8 conv output) or 'raw' (on the int32 sums)")
        # where L1BN reads a conv's output: its SQ8 codes, or the raw int32
        # sums (the literal dataflow, Sec. 3.2.2-3.2.3)
        self.bn_raw = bn_input == "raw"
        self.wl = wl
        # weight-gradient quantizer: GQ1 (Eq. 17, the DeepLab setting) keeps
        # Scale(G); GQ2 (Eq. 18, the FCN setting) drops it
        self.g_mode = iseg.ISEG_G_KEEP if gq == 1 else iseg.ISEG_G_DROP
        self.k_W, self.k_U = k_W, k_U
        self.w_master_exp = 1 - k_U             # Eq. 7
        self.gb_master_exp = 2 - k_U            # gamma/beta quantizers carry the x2 fold
        self.dev = torch.device(device)
        self.lr_shift = lr_shift
        self.seed = inputs["seed"]
        self.cfg = dict(iseg.BN_DEFAULT, **(bn_cfg or {}))
        if self.bn_raw and self.cfg["k_E2"] < 15:
            raise ValueError("L1BN on the raw sums supports the exact E2 (k_E2 >= 15) only")
        self._cfgs = {r: iseg.bn_cfg(**dict(self.cfg, relu=r)) for r in (0, 1)}
        self.k_A = self.cfg["k_A"]
        self.step_no = 0
        # backward-weight runs on a second stream (default priority): each
        # conv's weight gradient only needs its dz and input, so it overlaps
        # the backward-data / L1BN / merge chain of the layers below
        self.side = torch.cuda.Stream(device=self.dev) if self.dev.type == "cuda" else None
        # branches of the graph (a projection shortcut, the ASPP branches) run
        # on streams of their own (default priority) so that their
        # latency-bound kernels overlap the other branch; forward and
        # backward of a node use the same stream.  Two branch streams: with
        # the caller's stream and the side stream that is one hardware queue
        # each at HIP's default of four per process (a fifth stream would
        # share a queue, and serialize, with another)
        nb = branch_streams if self.side is not None else 0
        self.branch = [torch.cuda.Stream(device=self.dev) for _ in range(nb)]
        self.node_stream = self._plan_streams(wl["nodes"], nb)
        # nodes with a reader on another stream (an event marks their output)
        self.cross = {src for nd in wl["nodes"] for src in nd["src"]
                      if src != "input" and self.node_stream[src] != self.node_stream[nd["name"]]}
        # nodes whose backward sends errors to a source on another stream (the
        # input's error is merged on the caller's stream)
        self.bwd_cross = {nd["name"] for nd in wl["nodes"] for src in nd["src"]
                          if self.node_stream[src] != self.node_stream[nd["name"]]}
        # one sticky device status word for every call of the step (range
        # violations the kernels detect: merge exponent gaps, BN exponents out
        # of range, bad labels, logits outside the loss region's domain)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.dev)
        self.x = torch.from_numpy(inputs["x"]).to(self.dev)
        self.x_exp = iseg.new_exp(self.dev, inputs["x_exp"])
        # the input codes come from outside the library: check their range once
        iseg.iseg_check_codes(self.x, 8, self.status)
        self.dy = self.labels = None
        if wl["loss"] == "given":
            self.dy = torch.from_numpy(inputs["dy"]).to(self.dev)
            self.dy_exp = iseg.new_exp(self.dev, inputs["dy_exp"])
        else:
            self.labels = torch.from_numpy(inputs["labels"]).to(self.dev)
        self.w_exp = iseg.new_exp(self.dev, 1 - k_W)                         # Eq. 8
        self.convs = {}
        ci = 0
        for nd in wl["nodes"]:
            if nd["kind"] != "conv":
                continue
            wf = torch.from_numpy(inputs["weights"][ci]).to(self.dev)
            ci += 1
            master, mexp = iseg.quantize(wf, k_U, iseg.ISEG_Q_UQ, out_dtype=torch.int32)   # Eq. 7
            assert int(mexp.item()) == self.w_master_exp
            cout = nd["cout"]
            g_m = torch.full((cout,), 1 << (-self.gb_master_exp), dtype=torch.int32, device=self.dev)
            b_m = torch.zeros(cout, dtype=torch.int32, device=self.dev)
            L = dict(l=ci, w_m=master, g_m=g_m, b_m=b_m,
                     w_q=iseg.weight_quant(master, k_U, k_W),
                     g_q=iseg.weight_quant(g_m, k_U, self.cfg["k_gamma"]),
                     b_q=iseg.weight_quant(b_m, k_U, self.cfg["k_beta"]),
                     # gradient buffers, written every step (fixed addresses for the update table)
                     G=torch.empty(master.shape, dtype=torch.int8, device=self.dev),
                     G_exp=iseg._out_exp(self.dev))
            if nd["bn"]:
                L.update(dg=torch.empty(cout, dtype=torch.int64, device=self.dev),
                         db=torch.empty(cout, dtype=torch.int64, device=self.dev),
                         dg_exp=iseg._out_exp(self.dev), db_exp=iseg._out_exp(self.dev),
                         Gg=torch.empty(cout, dtype=torch.int8, device=self.dev),
                         Gb=torch.empty(cout, dtype=torch.int8, device=self.dev),
                         Gg_exp=iseg._out_exp(self.dev), Gb_exp=iseg._out_exp(self.dev))
            self.convs[nd["name"]] = L
        self._build_update_table()
        self.wt_tab = None
        self.loss = None
        # step replay: step number `replay_from` runs and is recorded into a
        # tape (every library call and stream ordering, the step counter of
        # the stochastic rounding as a parameter); later steps replay the tape
        # from native code and return that step's record, whose tensors each
        # replay rewrites
        self.replay_from = replay_from if self.side is not None else None
        self.tape = None
        self._tape_rec = None
        self._tape_out = None

    def _build_update_table(self):
        """Every parameter tensor of the network for one iseg_update_multi launch."""
        ents = []
        for nd in self.wl["nodes"]:
            if nd["kind"] != "conv":
                continue
            L = self.convs[nd["name"]]
            ents.append(dict(master=L["w_m"], w_q=L["w_q"], g=L["G"], g_exp=L["G_exp"],
                             kind=iseg.ISEG_UPD_CODES, master_exp=self.w_master_exp))
            if nd["bn"]:
                for m, q, g, ge, gq, gqe, t, kw in (
                        ("g_m", "g_q", "dg", "dg_exp", "Gg", "Gg_exp", 1, self.cfg["k_gamma"]),
                        ("b_m", "b_q", "db", "db_exp", "Gb", "Gb_exp", 2, self.cfg["k_beta"])):
                    ents.append(dict(master=L[m], w_q=L[q], g=L[g], g_exp=L[ge], g_q=L[gq],
                                     g_q_exp=L[gqe], kind=iseg.ISEG_UPD_RAW,
                                     master_exp=self.gb_master_exp, tensor_id=16 * L["l"] + t,
                                     k_w=kw))
        self.upd_table, self.upd_n = iseg.update_table(ents, self.dev)

    def _build_wt_table(self, rec):
        """Transposed copy of every weight whose backward-data runs, in the
        layout that conv's backward-data plan reads ([C, RS, K], taps reversed
        for the stride-1 plans); written by one launch after each update."""
        ents = []
        for nd in self.wl["nodes"]:
            if nd["kind"] != "conv" or (nd["src"][0] == "input" and not self.wl["input_grad"]):
                continue
            L = self.convs[nd["name"]]
            # a transposed conv runs backward-data in its forward, on the
            # geometry of the conv it is the adjoint of
            xs = rec[nd["name"]]["a_out"].shape if nd.get("transposed") else rec[nd["name"]]["a_in"].shape
            L["wt_kind"] = iseg.wt_kind(xs, L["w_q"].shape, nd["stride"], nd["pad"], nd["dil"])
            if L["wt_kind"] == iseg.ISEG_WT_NONE:
                continue    # a reduction split over channel chunks reads w itself
            L["w_t"] = torch.empty_like(L["w_q"])
            ents.append((L["w_q"], L["w_t"], L["wt_kind"]))
        self.wt_tab, self.wt_n, self.wt_tiles = iseg.wt_table(ents, self.dev)

    def _transpose_weights(self):
        iseg.iseg_weight_transpose_multi(self.wt_tab, self.wt_n, self.wt_tiles)

    @staticmethod
    def _plan_streams(nodes, nbranch):
        """Stream index of every node (0: the caller's current stream, k >= 1:
        branch stream k).  A one-input node that is not the last one-input
        reader (in node order) of its input opens a branch on the next branch
        stream (round robin); a one-input node otherwise continues its input's
        stream; a node with several inputs (a merge) runs on the stream of its
        input that comes last."""
        order = {nd["name"]: i for i, nd in enumerate(nodes)}
        order["input"] = -1
        readers = {}
        for nd in nodes:
            if len(nd["src"]) == 1:
                readers.setdefault(nd["src"][0], []).append(nd["name"])
        st, nxt = {"input": 0}, 0
        for nd in nodes:
            src = nd["src"]
            if len(src) > 1:
                st[nd["name"]] = st[max(src, key=lambda n: order[n])]
            elif nbranch and readers[src[0]][-1] != nd["name"]:
                nxt = nxt % nbranch + 1
                st[nd["name"]] = nxt
            else:
                st[nd["name"]] = st[src[0]]
        return st

    def _streams(self):
        if self.side is None:
            return [None]
        return [torch.cuda.current_stream(self.dev)] + self.branch

    # stream orderings go through these so that a recording tape sees them
    def _record(self, stream):
        ev = stream.record_event()
        slot = None
        if self._tape_rec is not None:
            slot = self._tape_rec.new_slot()
            self._tape_rec.add_record(slot, stream.cuda_stream)
        return ev, slot

    def _wait(self, stream, tok):
        stream.wait_event(tok[0])
        if self._tape_rec is not None:
            self._tape_rec.add_wait(stream.cuda_stream, tok[1])

    def _join(self, stream, other):
        """stream waits for the work enqueued on other so far"""
        self._wait(stream, self._record(other))

    @staticmethod
    def _on(stream, idx, fn):
        """fn() with `stream` current (the caller's stream needs no switch)"""
        if idx == 0:
            return fn()
        with torch.cuda.stream(stream):
            return fn()

    # -------------------------------------------------------------------
    def forward(self):
        act = {"input": (self.x, self.x_exp)}
        rec = {}
        streams = self._streams()
        for b in self.branch:
            self._join(b, streams[0])
        ready = {}
        for nd in self.wl["nodes"]:
            si = self.node_stream[nd["name"]]
            for src in nd["src"]:
                if src != "input" and self.node_stream[src] != si:   # the input is ready before the branches start
                    self._wait(streams[si], ready[src])
                    for t in act[src]:
                        t.record_stream(streams[si])
            rec[nd["name"]], act[nd["name"]] = self._on(streams[si], si, lambda: self._fwd_node(nd, act))
            if nd["name"] in self.cross:
                ready[nd["name"]] = self._record(streams[si])
        for b in self.branch:
            self._join(streams[0], b)
        return rec

    def _fwd_node(self, nd, act):
        k, name = nd["kind"], nd["name"]
        a, ae = act[nd["src"][0]]
        r = dict(kind=k, a_in=a, a_in_exp=ae)
        if k == "conv":
            L = self.convs[name]
            raw = self.bn_raw and nd["bn"]
            if nd.get("transposed"):
                # the adjoint of the conv whose input has this node's output shape
                N, h, w, _ = a.shape
                H = (h - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
                W = (w - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
                z, ze = iseg.conv_bwd_data(a, ae, L["w_q"], self.w_exp, (N, H, W, nd["cout"]), nd["stride"],
                                           nd["pad"], nd["dil"], wt=L.get("w_t"), wt_kind=L.get("wt_kind", 0),
                                           status=self.status)
            else:
                z, ze = iseg.conv_fwd(a, ae, L["w_q"], self.w_exp, nd["stride"], nd["pad"], nd["dil"],
                                      out_mode=iseg.ISEG_OUT_RAW if raw else iseg.ISEG_OUT_Q8,
                                      status=self.status)
            r.update(z=z, z_exp=ze)
            if nd["bn"]:
                y, ye, saved = iseg.bn_fwd(z, ze, L["g_q"], L["b_q"], self._cfgs[int(nd["relu"])],
                                           status=self.status)
                r["saved"] = saved
            elif nd["relu"] or self.k_A < 8:
                # without BN: A = Q_A(ReLU?(Z)) on the 8-bit conv output
                y, ye = iseg.sum_requant([z], [ze], relu=nd["relu"], bits=self.k_A, status=self.status)
            else:
                y, ye = z, ze
        elif k == "maxpool":
            y, ye = iseg.maxpool_fwd(a, ae, nd["k"], nd["stride"], nd["pad"])
        elif k == "add":
            b, be = act[nd["src"][1]]
            y, ye = iseg.sum_requant([a, b], [ae, be], relu=nd["relu"], bits=self.k_A,
                                      status=self.status)
            r.update(b_in=b, b_in_exp=be)
        elif k == "gap":
            y, ye = iseg.gap_fwd(a, ae, bits=self.k_A, status=self.status)
        elif k == "concat":
            parts = [act[s] for s in nd["src"]]
            y, ye = iseg.concat_requant([p[0] for p in parts], [p[1] for p in parts], bits=self.k_A,
                                         status=self.status)
            H, W = y.shape[1], y.shape[2]
            r.update(widths=[p[0].shape[3] for p in parts],
                     bcast=[tuple(p[0].shape[1:3]) != (H, W) for p in parts])
        else:
            raise ValueError(k)
        r.update(a_out=y, a_out_exp=ye)
        return r, (y, ye)

    def loss_error(self, rec):
        out = rec[self.wl["nodes"][-1]["name"]]
        if self.wl["loss"] == "given":
            return self.dy, self.dy_exp
        if self.wl["loss"] == "mse":
            loss, e, ee = iseg.mse_onehot(out["a_out"], out["a_out_exp"], self.labels, status=self.status)
            self.loss = loss
            return e, ee
        loss, grad, e, ee = iseg.softmax_ce(out["a_out"], out["a_out_exp"], self.labels, status=self.status)
        self.loss = loss
        return e, ee

    def backward(self, rec):
        contrib = {}
        streams = self._streams()
        for b in self.branch:
            self._join(b, streams[0])
        done = {}           # node -> event after its backward, when a source runs on another stream
        sender = ["loss"]

        def send(name, codes, exp, exp_add=0, bcast=0):
            contrib.setdefault(name, []).append((codes, exp, exp_add, bcast, sender[0]))

        def merged(name, si, mask=None):
            # the summed error of a tensor; with mask (a residual add's inputs
            # and exponents) a sum of several parts also goes through the add's
            # ReLU backward in the same call (third result True)
            parts = contrib.pop(name)
            for p in parts:
                if p[4] in done and self._stream_of(p[4]) != si:
                    self._wait(streams[si], done[p[4]])
                    for t in p[:2]:
                        t.record_stream(streams[si])
            if len(parts) == 1 and not parts[0][2] and not parts[0][3]:
                return parts[0][0], parts[0][1], False
            if mask is not None and not any(p[3] for p in parts):
                d, de = iseg.sum_requant_relu_mask([p[0] for p in parts], [p[1] for p in parts], mask[0], mask[1],
                                                   exp_add=[p[2] for p in parts], status=self.status)
                return d, de, True
            e, ee = iseg.sum_requant([p[0] for p in parts], [p[1] for p in parts],
                                     exp_add=[p[2] for p in parts], bcast=[p[3] for p in parts],
                                     status=self.status)
            return e, ee, False

        if self.wt_tab is None:
            self._build_wt_table(rec)
            self._transpose_weights()
        e, ee = self.loss_error(rec)
        send(self.wl["nodes"][-1]["name"], e, ee)
        if self.node_stream[self.wl["nodes"][-1]["name"]] != 0:
            done["loss"] = self._record(streams[0])
        grads = []
        for nd in reversed(self.wl["nodes"]):
            si = self.node_stream[nd["name"]]
            sender[0] = nd["name"]
            self._on(streams[si], si, lambda: self._bwd_node(nd, rec, merged, send, grads, si))
            if nd["name"] in self.bwd_cross:
                done[nd["name"]] = self._record(streams[si])
        if self.wl["input_grad"]:
            e, ee, _ = merged("input", 0)
            rec["input"] = dict(kind="input", e_out=e, e_out_exp=ee)
        for b in self.branch:
            self._join(streams[0], b)
        if self.side is not None:
            self._join(streams[0], self.side)
        return grads

    def _stream_of(self, name):
        return 0 if name == "loss" else self.node_stream[name]

    def _bwd_node(self, nd, rec, merged, send, grads, si):
        k, name = nd["kind"], nd["name"]
        want_input = self.wl["input_grad"]
        r = rec[name]
        mask = ([r["a_in"], r["b_in"]], [r["a_in_exp"], r["b_in_exp"]]) if k == "add" and nd["relu"] else None
        e, ee, masked = merged(name, si, mask)
        r.update(e_out=e, e_out_exp=ee, e_out_masked=masked)
        src = nd["src"][0]
        need_in = src != "input" or want_input
        if k == "conv":
            L = self.convs[name]
            if nd["bn"]:
                dz, dze, dg, db, dge, dbe = iseg.bn_bwd(e, ee, r["z"], L["g_q"], r["saved"],
                                                        self._cfgs[int(nd["relu"])],
                                                        status=self.status, dgb_out=(L["dg"], L["db"], L["dg_exp"],
                                                                 L["db_exp"]))
                r.update(dgamma=dg, dbeta=db, dgamma_exp=dge, dbeta_exp=dbe)
            elif nd["relu"]:
                dz, dze = iseg.relu_mask_bwd(e, [r["z"]], [r["z_exp"]], status=self.status), ee
            else:
                dz, dze = e, ee
            G, Ge = self._wgrad(nd, L, r, dz, dze)
            r.update(dz=dz, dz_exp=dze, G=G, G_exp=Ge)
            grads.append((nd, r))
            if need_in and nd.get("transposed"):
                # the input error of a transposed conv is the forward of the
                # conv it is the adjoint of
                ei, eie = iseg.conv_fwd(dz, dze, L["w_q"], self.w_exp, nd["stride"], nd["pad"], nd["dil"],
                                        status=self.status)
                r.update(e_in=ei, e_in_exp=eie)
                send(src, ei, eie)
            elif need_in:
                ei, eie = iseg.conv_bwd_data(dz, dze, L["w_q"], self.w_exp, r["a_in"].shape,
                                             nd["stride"], nd["pad"], nd["dil"], wt=L.get("w_t"),
                                             wt_kind=L["wt_kind"], status=self.status)
                r.update(e_in=ei, e_in_exp=eie)
                send(src, ei, eie)
        elif k == "maxpool":
            if need_in:
                ei, eie = iseg.maxpool_bwd(e, ee, r["a_in"], nd["k"], nd["stride"], nd["pad"],
                                           status=self.status)
                r.update(e_in=ei, e_in_exp=eie)
                send(src, ei, eie)
        elif k == "add":
            d = (iseg.relu_mask_bwd(e, [r["a_in"], r["b_in"]], [r["a_in_exp"], r["b_in_exp"]],
                                    status=self.status) if nd["relu"] and not masked else e)
            r.update(e_in=d, e_in_exp=ee)
            for s in nd["src"]:
                if s != "input" or want_input:
                    send(s, d, ee)
        elif k == "gap":
            if need_in:
                H, W = r["a_in"].shape[1:3]
                eg, ege = iseg.gap_bwd(e, ee, H, W, status=self.status)
                r.update(e_in=eg, e_in_exp=ege)
                send(src, eg, ege, bcast=1)
        elif k == "concat":
            parts = iseg.concat_split(e, r["widths"], skip=r["bcast"])
            c0 = 0
            for s, p, wdt, bc in zip(nd["src"], parts, r["widths"], r["bcast"]):
                if bc:
                    pe, pee = iseg.spatial_sum(e, ee, 1, c0, wdt, status=self.status)
                    send(s, pe, pee)
                else:
                    send(s, p, ee)
                c0 += wdt

    def _wgrad(self, nd, L, r, dz, dze):
        """Q_G(backward-weight) of one conv (Eq. 17), on the side stream once
        dz is ready; its inputs are marked as in use there."""
        if nd.get("transposed"):
            # the adjoint conv reads dz and writes this node's input: its
            # weight gradient pairs the node's input (as the error) with dz
            args = (r["a_in"], r["a_in_exp"], dz, dze, L["w_q"].shape, nd["stride"], nd["pad"], nd["dil"],
                    self.g_mode, 8, self.seed, 16 * L["l"], self.step_no)
        else:
            args = (dz, dze, r["a_in"], r["a_in_exp"], L["w_q"].shape, nd["stride"], nd["pad"], nd["dil"],
                    self.g_mode, 8, self.seed, 16 * L["l"], self.step_no)
        if self.side is None:
            return iseg.conv_bwd_weight(*args, out=(L["G"], L["G_exp"]), status=self.status)
        ready = self._record(torch.cuda.current_stream(self.dev))
        with torch.cuda.stream(self.side):
            self._wait(self.side, ready)
            G, Ge = iseg.conv_bwd_weight(*args, out=(L["G"], L["G_exp"]), status=self.status)
        for t in (dz, dze, r["a_in"], r["a_in_exp"]):
            t.record_stream(self.side)
        return G, Ge

    def update(self, grads):
        """Q_G of gamma / beta, Eq. 19 and Q_W for every parameter: one launch."""
        iseg.iseg_update_multi(self.upd_table, self.upd_n, 8, self.seed, self.step_no, self.lr_shift,
                               self.k_U, self.k_W, status=self.status)
        if self.wt_tab is not None:
            self._transpose_weights()
        for nd, r in grads:
            if nd["bn"]:
                L = self.convs[nd["name"]]
                r.update(Gg=L["Gg"], Gb=L["Gb"], Gg_exp=L["Gg_exp"], Gb_exp=L["Gb_exp"])

    def infer(self, calib, x, x_exp):
        """Forward of a chain of conv + L1BN (+ReLU) layers and max pooling in
        inference with the frozen state that a calibration forward `calib`
        (the record forward() returned) saved: one iseg_conv_bn_infer per conv
        layer.  Returns {node: (codes, exp)}."""
        act = {"input": (x, x_exp)}
        out = {}
        for nd in self.wl["nodes"]:
            a, ae = act[nd["src"][0]]
            if nd["kind"] == "conv":
                if not nd["bn"] or self.bn_raw:
                    raise ValueError("inference covers conv layers with L1BN on their 8-bit outputs")
                L = self.convs[nd["name"]]
                res = iseg.conv_bn_infer(a, ae, L["w_q"], self.w_exp, calib[nd["name"]]["saved"], nd["stride"],
                                         nd["pad"], nd["dil"], status=self.status)
            elif nd["kind"] == "maxpool":
                res = iseg.maxpool_fwd(a, ae, nd["k"], nd["stride"], nd["pad"])
            else:
                raise ValueError("inference covers chains of conv layers and max pooling")
            out[nd["name"]] = res
            act[nd["name"]] = res
        return out

    def read_status(self):
        """The sticky status word after the work enqueued so far (waits for
        the current stream): 0, or ISEG_DEV_* bits."""
        return iseg.iseg_status_read(self.status)

    def step(self, eager=False):
        """One training step; with a recorded tape a replay unless `eager`."""
        if self.tape is not None and not eager:
            self.tape.run(self.step_no)
            self.step_no += 1
            return self._tape_out
        if self.replay_from is not None and self.tape is None and self.step_no >= self.replay_from:
            tape = iseg.Tape(self.step_no)
            self._tape_rec = tape
            try:
                with tape:
                    rec = self._step()
            finally:
                self._tape_rec = None
            self.tape, self._tape_out = tape, rec
            return rec
        return self._step()

    def _step(self):
        rec = self.forward()
        grads = self.backward(rec)
        self.update(grads)
        self.step_no += 1
        return rec
