"""Oracle composition of one NITI training step (Algorithm 1) -- test
infrastructure only.

Tensors are NCHW / KCRS numpy arrays; a fully-connected layer after
convolutions reads its input flattened in (h, w, c) order (the order the
activations are stored in by the library, so its weights are the same
arrays on both sides).  Layer specs:
  ("fc",   n_in, n_out, relu)
  ("conv", c_in, c_out, ksize, stride, pad, relu)
  ("pool",)
  ("dropout", drop256)      dropout with probability drop256/256 (drop256 =
                            128: kept values doubled through the exponent)
Per step: forward with s_y = s_x + s_w + bp and ReLU on the accumulators
(reading R5); integer loss gradient; then, last layer first, the input
error from the weights before their update, rounded with target 7 and
masked by the ReLU of the layer below (after the 2x2 pooling routing or the
dropout mask when one sits between), and the weight gradient rounded to
mu bits and subtracted (Section 3.3).  The first layer's input error is not
formed.  `mode` rounds activations and errors, `grad_mode` the weight
gradients; stochastic draws use seed sr_seed + block (blocks numbered like
the library network's statistics blocks: three per weighted layer --
forward, back-propagation, weight gradient -- then the loss) and the step
index as call count; dropout draws use (drop_seed, step index).
"""
from __future__ import annotations

import numpy as np

import oracle as O


def _hwc_flat(a):
    """[n][c][h][w] -> [n][h*w*c] in (h, w, c) order."""
    a = np.asarray(a)
    if a.ndim == 4:
        return np.ascontiguousarray(a.transpose(0, 2, 3, 1)).reshape(a.shape[0], -1)
    return a.reshape(a.shape[0], -1)


def _from_hwc_flat(v, shape):
    """Inverse of _hwc_flat for a tensor of NCHW shape."""
    if len(shape) == 4:
        n, c, h, w = shape
        return np.ascontiguousarray(np.asarray(v).reshape(n, h, w, c).transpose(0, 3, 1, 2))
    return np.asarray(v).reshape(shape)


class OracleNet:
    def __init__(self, specs, in_shape, batch, weights, w_exps, mu=5, mode=O.PSR, grad_mode=None, sr_seed=0,
                 drop_seed=0):
        """in_shape = (c, h, w); weights KCRS (conv) or [out][in] (fc)."""
        self.specs = list(specs)
        self.batch = batch
        self.mu = mu
        self.mode = mode
        self.grad_mode = mode if grad_mode is None else grad_mode
        self.sr_seed = sr_seed
        self.drop_seed = drop_seed
        self.t = 0
        self.w = [np.array(w, dtype=np.int8, copy=True) for w in weights]
        self.s_w = list(w_exps)
        self.layers = []
        c, h, w = in_shape
        nw = 0
        for sp in self.specs:
            L = {"spec": sp, "in": (c, h, w)}
            if sp[0] == "conv":
                _, cin, cout, k, st, pd, relu = sp
                d = O.conv_desc(batch, cin, h, w, cout, k, k, st, pd)
                P, Q = O.conv_out_hw(d)
                L.update(kind="conv", desc=d, relu=relu, block=3 * nw)
                c, h, w = cout, P, Q
                nw += 1
            elif sp[0] == "fc":
                _, nin, nout, relu = sp
                L.update(kind="fc", relu=relu, nin=nin, nout=nout, block=3 * nw,
                         desc=O.conv_desc(batch, nin, 1, 1, nout, 1, 1, 1, 0))
                c, h, w = nout, 1, 1
                nw += 1
            elif sp[0] == "pool":
                L.update(kind="pool")
                h, w = h // 2, w // 2
            else:
                L.update(kind="dropout", drop256=sp[1])
            L["out"] = (c, h, w)
            self.layers.append(L)
        self.loss_block = 3 * nw
        self.history = []

    def _key(self, block):
        return {"sr_seed": self.sr_seed + block, "sr_call": self.t}

    def step(self, x, s_x, labels, mu=None):
        B = self.batch
        mu = self.mu if mu is None else mu
        a, s_a = x, s_x
        wi = 0
        rec = {"fwd": [], "s": []}
        # forward
        for L in self.layers:
            L["x"] = a
            if L["kind"] == "conv":
                L["wi"] = wi
                y, _, st = O.conv_fwd(L["desc"], a, self.w[wi], relu=L["relu"], mode=self.mode,
                                      **self._key(L["block"]))
                s_a, _ = O.out_exponent(s_a, self.s_w[wi], st["bp"])
                wi += 1
            elif L["kind"] == "fc":
                L["wi"] = wi
                y, _, st = O.gemm_fwd(_hwc_flat(a), self.w[wi], relu=L["relu"], mode=self.mode,
                                      **self._key(L["block"]))
                y = y.reshape(B, L["nout"], 1, 1)
                s_a, _ = O.out_exponent(s_a, self.s_w[wi], st["bp"])
                wi += 1
            elif L["kind"] == "pool":
                y, idx = O.maxpool2_fwd(a)
                L["idx"] = idx
            else:
                y, keep = O.dropout_fwd(a, self.drop_seed, self.t, L["drop256"])
                L["keep"] = keep
                s_a = max(-128, min(127, s_a + (1 if L["drop256"] == 128 else 0)))
            L["y"] = y
            rec["fwd"].append(y)
            rec["s"].append(s_a)
            a = y
        logits = a.reshape(B, -1)
        err, _, _ = O.int_ce_loss_grad(logits, s_a, labels, mode=self.mode, **self._key(self.loss_block))
        # backward
        e = err.reshape(self.layers[-1]["y"].shape)
        for i in range(len(self.layers) - 1, -1, -1):
            L = self.layers[i]
            below = self.layers[i - 1] if i > 0 else None
            relu_below = below is not None and below["kind"] in ("conv", "fc") and below["relu"]
            if L["kind"] in ("pool", "dropout"):
                if L["kind"] == "pool":
                    e_in = O.maxpool2_bwd(e, L["idx"], L["x"].shape)
                else:
                    e_in = O.dropout_bwd(e, L["keep"])
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
                xv = _hwc_flat(L["x"]).reshape(B, L["nin"], 1, 1)
                ev = e.reshape(B, L["nout"], 1, 1)
                wv = self.w[wi].reshape(L["nout"], L["nin"], 1, 1)
            e_in = None
            if i > 0:
                src = xv if relu_below else None
                e_in, _, _ = O.conv_bwd_data(d, ev, wv, mode=self.mode, relu_src=src, **self._key(L["block"] + 1))
                e_in = e_in if L["kind"] == "conv" else _from_hwc_flat(e_in.reshape(B, -1), L["x"].shape)
            w_new, _, _ = O.conv_bwd_weight(d, xv, ev, wv, mu=mu, mode=self.grad_mode, **self._key(L["block"] + 2))
            self.w[wi] = w_new.reshape(self.w[wi].shape)
            e = e_in
        rec["err"] = err
        self.history.append(rec)
        self.t += 1
        return logits, s_a
