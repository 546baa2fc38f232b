"""Oracle composition of one NITI training step (Algorithm 1) -- test
infrastructure only.

Tensors are NCHW / KCRS numpy arrays; a fully-connected layer after
convolutions reads its input flattened in (c, h, w) order.  Layer specs:
  ("fc",   n_in, n_out, relu)
  ("conv", c_in, c_out, ksize, stride, pad, relu)
  ("pool",)
Per step: forward with s_y = s_x + s_w + bp and ReLU on the accumulators
(reading R5); integer loss gradient; then, last layer first, the input
error from the weights before their update, rounded with target 7 and
masked by the ReLU of the layer below (after the 2x2 pooling routing when a
pooling layer sits between), and the weight gradient rounded to mu bits and
subtracted (Section 3.3).  The first layer's input error is not formed.
"""
from __future__ import annotations

import numpy as np

import oracle as O


class OracleNet:
    def __init__(self, specs, in_shape, batch, weights, w_exps, mu=5, mode=O.PSR):
        """in_shape = (c, h, w); weights KCRS (conv) or [out][in] (fc)."""
        self.specs = list(specs)
        self.batch = batch
        self.mu = mu
        self.mode = mode
        self.w = [np.array(w, dtype=np.int8, copy=True) for w in weights]
        self.s_w = list(w_exps)
        self.layers = []
        c, h, w = in_shape
        for sp in self.specs:
            L = {"spec": sp, "in": (c, h, w)}
            if sp[0] == "conv":
                _, cin, cout, k, st, pd, relu = sp
                d = O.conv_desc(batch, cin, h, w, cout, k, k, st, pd)
                P, Q = O.conv_out_hw(d)
                L.update(kind="conv", desc=d, relu=relu)
                c, h, w = cout, P, Q
            elif sp[0] == "fc":
                _, nin, nout, relu = sp
                L.update(kind="fc", relu=relu, nin=nin, nout=nout,
                         desc=O.conv_desc(batch, nin, 1, 1, nout, 1, 1, 1, 0))
                c, h, w = nout, 1, 1
            else:
                L.update(kind="pool")
                h, w = h // 2, w // 2
            L["out"] = (c, h, w)
            self.layers.append(L)
        self.history = []

    def step(self, x, s_x, labels):
        B = self.batch
        a, s_a = x, s_x
        wi = 0
        rec = {"fwd": [], "s": []}
        # forward
        for L in self.layers:
            L["x"] = a
            if L["kind"] == "conv":
                L["wi"] = wi
                y, _, st = O.conv_fwd(L["desc"], a, self.w[wi], relu=L["relu"], mode=self.mode)
                s_a, _ = O.out_exponent(s_a, self.s_w[wi], st["bp"])
                wi += 1
            elif L["kind"] == "fc":
                L["wi"] = wi
                y, _, st = O.gemm_fwd(a.reshape(B, -1), self.w[wi], relu=L["relu"], mode=self.mode)
                y = y.reshape(B, L["nout"], 1, 1)
                s_a, _ = O.out_exponent(s_a, self.s_w[wi], st["bp"])
                wi += 1
            else:
                y, idx = O.maxpool2_fwd(a)
                L["idx"] = idx
            L["y"] = y
            rec["fwd"].append(y)
            rec["s"].append(s_a)
            a = y
        logits = a.reshape(B, -1)
        err, _, _ = O.int_ce_loss_grad(logits, s_a, labels, mode=self.mode)
        # backward
        e = err.reshape(self.layers[-1]["y"].shape)
        for i in range(len(self.layers) - 1, -1, -1):
            L = self.layers[i]
            below = self.layers[i - 1] if i > 0 else None
            relu_below = below is not None and below["kind"] in ("conv", "fc") and below["relu"]
            if L["kind"] == "pool":
                e_in = O.maxpool2_bwd(e, L["idx"], L["x"].shape)
                if relu_below:
                    O.relu_mask(e_in, below["y"])
                e = e_in
                continue
            wi = L["wi"]
            if L["kind"] == "conv":
                d, xv, ev = L["desc"], L["x"], e
                wv = self.w[wi]
            else:
                d = L["desc"]
                xv = L["x"].reshape(B, L["nin"], 1, 1)
                ev = e.reshape(B, L["nout"], 1, 1)
                wv = self.w[wi].reshape(L["nout"], L["nin"], 1, 1)
            e_in = None
            if i > 0:
                e_in, _, _ = O.conv_bwd_data(d, ev, wv, mode=self.mode,
                                             relu_src=(L["x"].reshape(xv.shape) if relu_below else None))
                e_in = e_in.reshape(L["x"].shape)
            w_new, _, _ = O.conv_bwd_weight(d, xv, ev, wv, mu=self.mu, mode=self.mode)
            self.w[wi] = w_new.reshape(self.w[wi].shape)
            e = e_in
        rec["err"] = err
        self.history.append(rec)
        return logits, s_a
