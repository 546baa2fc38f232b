"""Integer networks trained with the NITI step (Algorithm 1), run through the
C ABI.  Every arithmetic step is a libniti call on the current HIP stream;
this module only owns device buffers and call order.

A network is a list of layer specs:
  ("fc",   n_in, n_out, relu)
  ("conv", c_in, c_out, ksize, stride, pad, relu)
  ("pool",)                                  2x2 stride-2 max pooling
  ("dropout", drop256)                       dropout with probability drop256/256;
                                             drop256 = 128 doubles the kept values
                                             through the exponent (inverted dropout)
Activations are NHWC int8 with one int8 exponent per tensor; a fully-
connected layer after convolutions reads the NHWC tensor flattened in
(h, w, c) order.  One training step (Algorithm 1):
  forward: y = round(layer(x)) with s_y = s_x + s_w + bp, ReLU on the int32
           accumulators where the spec asks;
  loss:    integer cross-entropy gradient of the logits (Section 3.5);
  backward, last layer first: the error of the layer input is computed with
           the weights before their update (the backward ReLU mask of the
           layer below is fused into that call), then the weight gradient is
           formed, shifted to mu bits and subtracted from the weights
           (Section 3.3).  The first layer's input error is not needed.
Rounding: `mode` for activations and errors, `grad_mode` for the weight
gradients (the paper's experiments round a and e to nearest and g with
pseudo stochastic rounding, Section 4.3); `mu` may change from step to step
(the schedule 5 -> 4 -> 3 of Section 4.3).  Stochastic rounding draws are
keyed by each stats block's seed (sr_seed + block index) and call count;
dropout draws by (drop_seed, step index, element).
"""
from __future__ import annotations

import numpy as np

from . import niti


def _i8(v):
    import torch
    return torch.tensor([int(v)], dtype=torch.int8, device="cuda")


_SIDE = None


def side_stream():
    """The second stream of IntNet steps, one per process: streams beyond the
    device's few hardware queues share queues and then order each other's
    work, so the networks of a process share this one."""
    global _SIDE
    if _SIDE is None:
        import torch
        _SIDE = torch.cuda.Stream()
    return _SIDE


class IntNet:
    def __init__(self, specs, in_shape, batch, weights, w_exps, mu=5, mode=niti.PSR, grad_mode=None, sr_seed=0,
                 drop_seed=0, streams=2):
        """in_shape = (h, w, c) of the NHWC input (c a multiple of 4 for convs);
        weights: list of int8 numpy arrays (KRSC for conv, [out][in] for fc),
        one per weighted layer; w_exps: their static exponents.  streams=2:
        the weight gradients and updates run on a second stream beside the
        back-propagation (each after the back-propagation that reads the same
        weights), and the caller's stream waits for them at the end of the
        step; streams=1: every call on the caller's stream, in the order of
        Algorithm 1.  Results are the same either way."""
        import torch
        self.specs = list(specs)
        self.batch = batch
        self.mu = mu
        self.mode = mode
        self.grad_mode = mode if grad_mode is None else grad_mode
        self.drop_seed = drop_seed
        self.t = 0
        self.layers = []
        h, w, c = in_shape
        wi = 0
        nstats = 0
        for sp in self.specs:
            L = {"spec": sp, "in_shape": (h, w, c)}
            if sp[0] == "conv":
                _, cin, cout, k, st, pd, relu = sp
                assert cin == c, (sp, c)
                d = niti.ConvDesc.make(batch, h, w, c, cout, k, k, st, pd)
                L.update(kind="conv", desc=d, relu=relu)
                h, w, c = d.p, d.q, cout
            elif sp[0] == "fc":
                _, nin, nout, relu = sp
                assert nin == h * w * c, (sp, (h, w, c))
                d = niti.ConvDesc.make(batch, 1, 1, nin, nout, 1, 1, 1, 0)
                L.update(kind="fc", desc=d, relu=relu, nin=nin, nout=nout)
                h, w, c = 1, 1, nout
            elif sp[0] == "pool":
                L.update(kind="pool")
                h, w = h // 2, w // 2
            elif sp[0] == "dropout":
                L.update(kind="dropout", drop256=sp[1])
            else:
                raise ValueError(sp)
            L["out_shape"] = (h, w, c)
            if L["kind"] in ("conv", "fc"):
                arr = np.ascontiguousarray(weights[wi])
                L["w"] = torch.from_numpy(arr).cuda()
                L["s_w"] = _i8(w_exps[wi])
                L["stats"] = nstats       # fwd, bwd_data, bwd_weight
                nstats += 3
                wi += 1
            self.layers.append(L)
        assert wi == len(weights)
        self.stats = niti.new_stats(nstats + 1)
        self.loss_stats = nstats
        for i in range(nstats + 1):
            niti.set_sr_seed(self.stats, sr_seed + i, index=i)
        # buffers
        for L in self.layers:
            oh, ow, oc = L["out_shape"]
            L["y"] = torch.empty((batch, oh, ow, oc), dtype=torch.int8, device="cuda")
            L["s_y"] = _i8(0)
            L["e_in"] = torch.empty((batch,) + tuple(L["in_shape"]), dtype=torch.int8, device="cuda")
            if L["kind"] == "pool":
                L["idx"] = torch.empty_like(L["y"], dtype=torch.uint8)
            if L["kind"] == "dropout":
                L["keep"] = torch.empty_like(L["y"], dtype=torch.uint8)
        ws = 0
        for L in self.layers:
            if L["kind"] in ("conv", "fc"):
                ws = max(ws, niti.workspace_bytes(niti.OP_CONV_FWD, L["desc"]),
                         niti.workspace_bytes(niti.OP_CONV_BWD_DATA, L["desc"]),
                         niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, L["desc"]))
        n_cls = self.layers[-1]["out_shape"][2]
        ws = max(ws, niti.workspace_bytes(niti.OP_INT_CE_LOSS, None, batch, n_cls))
        self.ws = niti.new_workspace(ws)
        self.err = torch.empty((batch, n_cls), dtype=torch.int8, device="cuda")
        assert streams in (1, 2)
        self.two = streams == 2
        if self.two:
            self.sB = side_stream()
            self.ws_b = niti.new_workspace(ws)
            from .stream_event import StreamEvent
            self.ev_upd = StreamEvent()
            self.ev_bwd = [StreamEvent() for _ in range(wi)]

    # -------------------------------------------------------------- forward
    def forward(self, x, s_x):
        a, s_a = x, s_x
        for L in self.layers:
            k = L["kind"]
            if k == "conv":
                niti.conv_fwd(L["desc"], a, L["w"], L["y"], self.stats, s_a, L["s_w"], L["s_y"],
                              relu=L["relu"], mode=self.mode, stats_index=L["stats"], ws=self.ws)
            elif k == "fc":
                niti.gemm_fwd(a.view(self.batch, L["nin"]), L["w"], L["y"].view(self.batch, L["nout"]),
                              self.stats, s_a, L["s_w"], L["s_y"], 7, L["relu"], self.mode,
                              stats_index=L["stats"])
            elif k == "pool":
                niti.maxpool2_fwd(a, L["y"], L["idx"])
                L["s_y"] = s_a
            else:
                niti.dropout_fwd(a, L["y"], L["keep"], self.drop_seed, self.t, L["drop256"], s_a, L["s_y"],
                                 1 if L["drop256"] == 128 else 0)
            L["x"] = a
            a, s_a = L["y"], L["s_y"]
        return a, s_a

    # -------------------------------------------------------------- backward
    def backward(self, err, mu):
        import torch
        e = err.view(self.layers[-1]["y"].shape)
        cur = torch.cuda.current_stream()
        nw = sum(1 for L in self.layers if L["kind"] in ("conv", "fc"))
        for i in range(len(self.layers) - 1, -1, -1):
            L = self.layers[i]
            k = L["kind"]
            below = self.layers[i - 1] if i > 0 else None
            need_e_in = i > 0
            # ReLU mask of the layer whose output is this layer's input
            mask = None
            if below is not None and below["kind"] in ("conv", "fc") and below["relu"]:
                mask = L["x"]
            if k in ("pool", "dropout"):
                if k == "pool":
                    niti.maxpool2_bwd(e, L["idx"], L["e_in"])
                else:
                    niti.dropout_bwd(e, L["keep"], L["e_in"])
                if below is not None and below["kind"] in ("conv", "fc") and below["relu"]:
                    niti.relu_mask(L["e_in"], below["y"])
                e = L["e_in"]
                continue
            d = L["desc"]
            if k == "conv":
                x_v, e_v, ein_v, m_v = L["x"], e, L["e_in"], mask
            else:
                B = self.batch
                x_v = L["x"].reshape(B, 1, 1, L["nin"])
                e_v = e.reshape(B, 1, 1, L["nout"])
                ein_v = L["e_in"].view(B, 1, 1, L["nin"])
                m_v = mask.reshape(B, 1, 1, L["nin"]) if mask is not None else None
            w_v = L["w"] if k == "conv" else L["w"].view(L["nout"], 1, 1, L["nin"])
            if need_e_in:
                niti.conv_bwd_data(d, e_v, w_v, ein_v, self.stats, self.ws, relu_src=m_v, mode=self.mode,
                                   stats_index=L["stats"] + 1)
            if self.two:
                # after the back-propagation that reads w (issued above on this
                # stream) and everything that produced this layer's error
                nw -= 1
                niti.stream_record(self.ev_bwd[nw], cur)
                niti.stream_wait(self.sB, self.ev_bwd[nw])
                with torch.cuda.stream(self.sB):
                    niti.conv_bwd_weight(d, x_v, e_v, w_v, self.stats, self.ws_b, mu=mu, mode=self.grad_mode,
                                         stats_index=L["stats"] + 2)
            else:
                niti.conv_bwd_weight(d, x_v, e_v, w_v, self.stats, self.ws, mu=mu, mode=self.grad_mode,
                                     stats_index=L["stats"] + 2)
            e = L["e_in"]
        if self.two:
            niti.stream_record(self.ev_upd, self.sB)

    def step(self, x, s_x, labels, mu=None):
        """One training step; returns (logits, s_logits) of the forward pass.
        mu: this step's update width (default: the net's)."""
        logits, s_l = self.forward(x, s_x)
        n_cls = logits.shape[-1]
        niti.int_ce_loss_grad(logits.view(self.batch, n_cls), s_l, labels, self.err, self.stats, self.ws,
                              mode=self.mode, stats_index=self.loss_stats)
        self.backward(self.err, self.mu if mu is None else mu)
        if self.two:
            import torch
            niti.stream_wait(torch.cuda.current_stream(), self.ev_upd)   # the updates, before anything after
        self.t += 1
        return logits, s_l

    def weights(self):
        return [L["w"] for L in self.layers if L["kind"] in ("conv", "fc")]


def mu_schedule(epoch, steps=((0, 5), (100, 4), (150, 3))):
    """m_u of an epoch under the schedule of Section 4.3 (Tables 3 and 4):
    5 bits, 4 from epoch 100, 3 from epoch 150."""
    mu = steps[0][1]
    for start, m in steps:
        if epoch >= start:
            mu = m
    return mu


# ------------------------------------------------------------------ workloads
MLP_784 = [("fc", 784, 256, True), ("fc", 256, 128, True), ("fc", 128, 10, False)]

# The paper's own networks (Section 4, Tables 5 and 6), on inputs with the
# datasets' shapes.  The kernels need channel counts that are multiples of 4,
# so an image's channels are padded with zeros (MNIST 1 -> 4, CIFAR10 3 -> 4)
# and LeNet-5's six first-layer filters with two filters held at zero (their
# outputs, errors and gradients stay zero, so the network is unchanged).
LENET5 = [("conv", 4, 8, 5, 1, 2, True), ("pool",), ("conv", 8, 16, 5, 1, 0, True), ("pool",),
          ("fc", 400, 120, True), ("fc", 120, 84, True), ("fc", 84, 10, False)]
LENET5_REAL = {"image_channels": 1, "zero_filters": {0: (6, 8)}}


def vgg_small(depth):
    """VGG-small-7/8/9 of Table 5 on 32x32 inputs: 3x3 convolutions
    128-128(-128), pool, 256-256(-256), pool, 512-512, pool, dropout, FC 10."""
    assert depth in (7, 8, 9)
    c1 = [128, 128] + ([128] if depth >= 8 else [])
    c2 = [256, 256] + ([256] if depth >= 9 else [])
    specs, cin = [], 4
    for block in (c1, c2, [512, 512]):
        for cout in block:
            specs.append(("conv", cin, cout, 3, 1, 1, True))
            cin = cout
        specs.append(("pool",))
    specs += [("dropout", 128), ("fc", 512 * 4 * 4, 10, False)]
    return specs

VGG_32 = [("conv", 4, 64, 3, 1, 1, True), ("conv", 64, 64, 3, 1, 1, True), ("pool",),
          ("conv", 64, 128, 3, 1, 1, True), ("conv", 128, 128, 3, 1, 1, True), ("pool",),
          ("conv", 128, 256, 3, 1, 1, True), ("conv", 256, 256, 3, 1, 1, True), ("pool",),
          ("fc", 4096, 10, False)]

# ResNet-18 at 224x224: each distinct layer shape with its multiplicity in
# the network (name, c_in, c_out, ksize, stride, pad, input size, count).
RESNET18_LAYERS = [
    ("stem7x7s2", 4, 64, 7, 2, 3, 224, 1),
    ("l1_3x3", 64, 64, 3, 1, 1, 56, 4),
    ("l2_3x3s2", 64, 128, 3, 2, 1, 56, 1),
    ("l2_1x1s2", 64, 128, 1, 2, 0, 56, 1),
    ("l2_3x3", 128, 128, 3, 1, 1, 28, 3),
    ("l3_3x3s2", 128, 256, 3, 2, 1, 28, 1),
    ("l3_1x1s2", 128, 256, 1, 2, 0, 28, 1),
    ("l3_3x3", 256, 256, 3, 1, 1, 14, 3),
    ("l4_3x3s2", 256, 512, 3, 2, 1, 14, 1),
    ("l4_1x1s2", 256, 512, 1, 2, 0, 14, 1),
    ("l4_3x3", 512, 512, 3, 1, 1, 7, 3),
]
RESNET18_FC = (512, 1000)

# AlexNet on 224x224 ImageNet-shaped inputs (the network of the paper's
# Table 6, 62.38M parameters: no channel groups): the contraction layers as
# (name, c_in, c_out, ksize, stride, pad, input size).  Its 3x3 stride-2
# overlapping max pools sit between them (55 -> 27 -> 13 -> 6); the image's
# three channels are padded to 4.
ALEXNET_LAYERS = [
    ("conv1_11x11s4", 4, 96, 11, 4, 2, 224),
    ("conv2_5x5", 96, 256, 5, 1, 2, 27),
    ("conv3_3x3", 256, 384, 3, 1, 1, 13),
    ("conv4_3x3", 384, 384, 3, 1, 1, 13),
    ("conv5_3x3", 384, 256, 3, 1, 1, 13),
]
ALEXNET_FC = [("fc6", 256 * 6 * 6, 4096), ("fc7", 4096, 4096), ("fc8", 4096, 1000)]


# ------------------------------------------------------------------ synthetic set-up
def synthetic_weights(specs, in_channels, cfg, image_channels=None, first_id=10, zero_filters=None):
    """Seeded U[-127,127] weights in the library's layouts for a layer list:
    KRSC for convolutions (channels past image_channels of the first layer
    zero), [out][in] for fully-connected layers with the input read in
    (h, w, c) order; plus the static exponents (He-uniform style, from the
    real fan-in).  zero_filters maps a convolution's index among the weighted
    layers to a range [lo, hi) of its output filters held at zero, together
    with the same input channels of the convolution after it.  Returns
    (weights as numpy arrays, exponents)."""
    from . import inputs as I
    zero_filters = zero_filters or {}
    ws, exps = [], []
    wi = 0
    for sp in specs:
        if sp[0] == "conv":
            _, cin, cout, k = sp[:4]
            w = I.weights(I.base_seed(cfg, first_id + wi), (cout, k, k, cin))
            real = cin
            if wi == 0 and image_channels is not None and image_channels < cin:
                w[..., image_channels:] = 0
                real = image_channels
            if wi in zero_filters:
                lo, hi = zero_filters[wi]
                w[lo:hi] = 0
            if wi - 1 in zero_filters:
                lo, hi = zero_filters[wi - 1]
                w[..., lo:hi] = 0
                real = cin - (hi - lo)
            ws.append(w)
            exps.append(I.weight_exponent(real * k * k))
            wi += 1
        elif sp[0] == "fc":
            ws.append(I.weights(I.base_seed(cfg, first_id + wi), (sp[2], sp[1])))
            exps.append(I.weight_exponent(sp[1]))
            wi += 1
    return ws, exps


def contraction_macs(specs, in_shape, batch, image_channels=None):
    """Multiply-accumulates of one training step of a layer list (forward,
    back-propagation of every layer but the first, weight gradient), counted
    on the real channel count of the image layer."""
    h, w, c = in_shape
    macs = 0
    first = True
    for sp in specs:
        if sp[0] == "conv":
            _, cin, cout, k, st, pd = sp[:6]
            p = (h + 2 * pd - k) // st + 1
            q = (w + 2 * pd - k) // st + 1
            real = image_channels if (first and image_channels) else cin
            m = batch * p * q * cout * real * k * k
            macs += m * (2 if first else 3)
            h, w, c = p, q, cout
            first = False
        elif sp[0] == "fc":
            m = batch * sp[1] * sp[2]
            macs += m * (2 if first else 3)
            h, w, c = 1, 1, sp[2]
            first = False
        else:
            h, w = h // 2, w // 2
    return macs
