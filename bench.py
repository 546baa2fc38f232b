#!/usr/bin/env python3
"""Throughput of the NITI integer-training hot path on one MI355X.

Default workload: the ResNet-18-shaped int8 layer set at 224x224, batch 128
(7x7/2 stem, 3x3 stages at 56/28/14/7 with 64..512 channels, the 1x1/2
downsample convolutions, the 512->1000 head).  One step runs, for every
layer of the network (20 convolutions and the head, each with its own
weights): the forward contraction with fused ReLU / block exponent / pseudo
stochastic rounding, the error back-propagation with fused rounding and
backward ReLU mask (not for the stem, whose input error is not needed), and
the weight gradient with the discrete mu=5 update; the head also runs the
integer cross-entropy gradient.  Inputs are seeded synthetic int8 tensors
resident in device memory before timing starts.

Printed: one JSON line.  value = algorithmic int8 tera-operations per second
of the whole step (2 ops per multiply-accumulate of each contraction,
counted on the unpadded channel count); roofline = the contraction kernel
with the most time in the step, timed live with HIP events on its launch
stream; c4_layers = every layer's forward, back-propagation and weight
gradient + update against its own bound (int8 MFMA or HBM); passes = the
split-sum, update and loss passes in GB/s; c1-c3 = the other training
workloads (fully-connected layer, MLP, VGG-style CNN) in microseconds per
step; c5 = the fused GEMM + exponent + rounding sweep over M, N, K in
{4096, 8192, 16384}; table7_context = the paper's GPU conv shapes, with its
RTX 3090 figures beside them; cpu_baseline = the CPU oracle on a bounded
sample of the layer set.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "int8 TOPS of fused NITI conv/GEMM+round (fwd/bwd/wgrad), % of int8 MFMA peak"
PEAK_INT8_TOPS = 5000.0       # MI355X dense int8 MFMA
PEAK_HBM_GBS = 8000.0


def _stream_event():
    from paper_2009_13108_amd.stream_event import StreamEvent
    return StreamEvent()


def conv_macs(n, c, h, w, k, r, s, st, pd):
    p = (h + 2 * pd - r) // st + 1
    q = (w + 2 * pd - s) // st + 1
    return n * p * q * k * c * r * s


# ----------------------------------------------------------------------------
class ResNetStep:
    """Buffers and call sequence of one training step over the layer set."""

    def __init__(self, batch=128, seed_cfg=4, mu=5, a_tail=1):
        import torch
        from paper_2009_13108_amd import inputs as I
        from paper_2009_13108_amd import model as M
        from paper_2009_13108_amd import niti

        self.niti = niti
        self.batch = batch
        self.mu = mu
        dev = "cuda"
        self.layers = []
        nst = 0
        ws = 0
        for li, (name, cin, cout, k, st, pd, hw, count) in enumerate(M.RESNET18_LAYERS):
            d = niti.ConvDesc.make(batch, hw, hw, cin, cout, k, k, st, pd)
            x = I.activations(I.base_seed(seed_cfg, 100 + li), (batch, hw, hw, cin), device=dev)
            c_real = cin
            if name.startswith("stem"):
                x[..., 3:] = 0          # 3 image channels, zero-padded to 4
                c_real = 3
                # The input batch is stored with its zero border (as a data
                # loader can write it), so that the image layer's descriptor
                # has no padding and the library reads the image in place;
                # the outputs and the work are those of the padded 224 x 224
                # convolution.
                hb = hw + 2 * pd
                xb = torch.zeros((batch, hb, hb, cin), dtype=torch.int8, device=dev)
                xb[:, pd:pd + hw, pd:pd + hw] = x
                x = xb
                d = niti.ConvDesc.make(batch, hb, hb, cin, cout, k, k, st, 0)
            dy = I.errors8(I.base_seed(seed_cfg, 200 + li), d.y_shape(), device=dev)
            ws_ = []
            for cpy in range(count):
                w = I.weights(I.base_seed(seed_cfg, 1000 + 10 * li + cpy), d.w_shape(), device=dev)
                if name.startswith("stem"):
                    w[..., 3:] = 0
                ws_.append(w)
            L = {"name": name, "desc": d, "x": x, "dy": dy, "w": ws_, "count": count,
                 "y": torch.empty(d.y_shape(), dtype=torch.int8, device=dev),
                 "dx": torch.empty(d.x_shape(), dtype=torch.int8, device=dev),
                 "stats": nst, "bwd_data": not name.startswith("stem"),
                 "packed": [niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, d)) for _ in range(count)],
                 "macs": conv_macs(batch, c_real, hw, hw, cout, k, k, st, pd)}
            nst += 3 * count
            ws = max(ws, niti.workspace_bytes(niti.OP_CONV_FWD, d),
                     niti.workspace_bytes(niti.OP_CONV_BWD_DATA, d),
                     niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, d))
            self.layers.append(L)
        fin, fout = M.RESNET18_FC
        self.fc_desc = niti.ConvDesc.make(batch, 1, 1, fin, fout, 1, 1, 1, 0)
        self.feat = I.activations(I.base_seed(seed_cfg, 300), (batch, fin), device=dev)
        self.wfc = I.weights(I.base_seed(seed_cfg, 301), (fout, fin), device=dev)
        self.labels = I.labels(I.base_seed(seed_cfg, 302), batch, fout, device=dev)
        self.logits = torch.empty((batch, fout), dtype=torch.int8, device=dev)
        self.err = torch.empty((batch, fout), dtype=torch.int8, device=dev)
        self.dfeat = torch.empty((batch, fin), dtype=torch.int8, device=dev)
        self.s_feat = torch.tensor([-9], dtype=torch.int8, device=dev)
        self.s_wfc = torch.tensor([-11], dtype=torch.int8, device=dev)
        self.s_logits = torch.zeros(1, dtype=torch.int8, device=dev)
        self.fc_packed = niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, self.fc_desc))
        self.fc_stats = nst
        nst += 4
        self.fc_macs = batch * fin * fout
        ws = max(ws, niti.workspace_bytes(niti.OP_CONV_BWD_DATA, self.fc_desc),
                 niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, self.fc_desc),
                 niti.workspace_bytes(niti.OP_INT_CE_LOSS, None, batch, fout))
        self.ws = niti.new_workspace(ws)       # stream A: forward, back-propagation, loss
        self.ws_b = niti.new_workspace(ws)     # stream B: weight gradients
        self.stats = niti.new_stats(nst)
        # Two streams, as in a training step: A runs the forward pass and the
        # back-propagation chain; B runs each layer's weight gradient + update
        # as soon as that layer's back-propagation is enqueued, overlapping the
        # next layer's back-propagation (the image layer's, which has no
        # back-propagation, runs on A after the chain).  B's update of w(l) follows A's
        # back-propagation of layer l (which reads w(l)), and the next step's
        # forward pass follows all of B's updates from its second layer on (the
        # image layer's filter is updated on A).
        self.sA = torch.cuda.Stream()
        self.sB = torch.cuda.Stream()
        self.ev_bwd = [_stream_event() for _ in range(sum(L["count"] for L in self.layers) + 1)]
        self.ev_fwd = [_stream_event() for _ in range(8)]
        self.ev_upd = _stream_event()
        self.ev_pack = _stream_event()
        self.ev_tail = _stream_event()
        self.ev_upd.record(self.sB)
        self.ev_tail.record(self.sA)
        # The weight gradients of the last a_tail layers before the image
        # layer run on stream A, after their back-propagation: A is idle
        # there, while B still works through the earlier layers' gradients
        # (one layer measured ~1% faster than none, two or three).
        self.a_tail = a_tail
        self.fam_ops = {"igemm": 0, "wgrad": 0}
        for L in self.layers:
            self.fam_ops["igemm"] += 2 * L["macs"] * L["count"] * (2 if L["bwd_data"] else 1)
            self.fam_ops["wgrad"] += 2 * L["macs"] * L["count"]
        self.fam_ops["igemm"] += 2 * 2 * self.fc_macs
        self.fam_ops["wgrad"] += 2 * self.fc_macs
        self.ops_per_step = self.fam_ops["igemm"] + self.fam_ops["wgrad"]
        # algorithmic bytes (operands, output, mask) per step, per family
        self.fam_bytes = {"igemm": 0, "wgrad": 0}
        for L in self.layers:
            d = L["desc"]
            xb = d.n * d.h * d.w * d.c
            yb = d.n * d.p * d.q * d.k
            wb = d.k * d.r * d.s * d.c
            self.fam_bytes["igemm"] += L["count"] * (xb + wb + yb)                              # x, w -> y
            if L["bwd_data"]:
                self.fam_bytes["igemm"] += L["count"] * (yb + wb + xb + xb)                     # dy, w, mask -> dx
            self.fam_bytes["wgrad"] += L["count"] * (xb + yb + 4 * wb)                         # x, dy -> g32
        self.fam_bytes["igemm"] += 2 * (batch * fin + fout * fin + batch * fout) + batch * fin  # head fwd, bwd
        self.fam_bytes["wgrad"] += batch * fin + batch * fout + 4 * fin * fout
        self.fam_calls = {"igemm": 0, "wgrad": 0}
        for L in self.layers:
            self.fam_calls["igemm"] += L["count"] * (2 if L["bwd_data"] else 1)
            self.fam_calls["wgrad"] += L["count"]
        self.fam_calls["igemm"] += 2
        self.fam_calls["wgrad"] += 1

    def step(self, plan=None):
        """Enqueue one step: forward and back-propagation on stream A
        (self.sA), weight gradients on stream B (self.sB).  plan: a list that
        receives the step as replayable operations -- the library calls of each
        stream segment, marshalled once (niti.recording), and the event record
        and wait operations between the streams; step_prepared() replays it."""
        import torch
        from contextlib import nullcontext
        niti = self.niti
        A, B = self.sA, self.sB
        Bsz = self.batch
        fin, fout = self.fc_desc.c, self.fc_desc.k
        s = self.fc_stats
        fd = self.fc_desc

        def seg(stream, fn):
            with torch.cuda.stream(stream), (niti.recording() if plan is not None else nullcontext()) as calls:
                fn()
            if plan is not None:
                plan.append(("calls", calls))

        def rec(ev, stream):
            ev.record(stream)
            if plan is not None:
                plan.append(("rec", ev, stream))

        def wait(stream, ev):
            ev.wait(stream)
            if plan is not None:
                plan.append(("wait", stream, ev))

        def conv_fwd(L, c, ws):
            niti.conv_fwd(L["desc"], L["x"], L["w"][c], L["y"], self.stats, relu=True,
                          stats_index=L["stats"] + 3 * c, ws=ws)

        def head():
            niti.gemm_fwd(self.feat, self.wfc, self.logits, self.stats, self.s_feat, self.s_wfc, self.s_logits, 7,
                          False, stats_index=s)
            niti.int_ce_loss_grad(self.logits, self.s_logits, self.labels, self.err, self.stats, self.ws,
                                  stats_index=s + 1)
            niti.conv_bwd_data_packed(fd, self.err.view(Bsz, 1, 1, fout), self.fc_packed,
                                      self.dfeat.view(Bsz, 1, 1, fin), self.stats,
                                      relu_src=self.feat.view(Bsz, 1, 1, fin), stats_index=s + 2)

        # (layer, copy) of the layers with a back-propagation, last first;
        # the final a_tail of them take their weight gradient on A.
        bwd = [(L, c) for L in reversed(self.layers) if L["bwd_data"] for c in reversed(range(L["count"]))]
        on_a = set((id(L), c) for L, c in bwd[len(bwd) - self.a_tail:]) if self.a_tail > 0 else set()
        pos = {(id(L), c): i for i, (L, c) in enumerate(bwd)}

        def pack_filters(tail):
            for L in self.layers:
                if L["bwd_data"]:
                    for c in range(L["count"]):
                        if ((id(L), c) in on_a) == tail:
                            niti.conv_pack_bwd_data(L["desc"], L["w"][c], L["packed"][c])
            if not tail:
                niti.conv_pack_bwd_data(fd, self.wfc.view(fout, 1, 1, fin), self.fc_packed)

        # The filters rearranged for the back-propagation, on stream B (in
        # order after the previous step's updates, and nearly idle in the
        # forward pass); A waits for them before the back-propagation.  The
        # filters that A updated last step are packed after A's updates.
        seg(B, lambda: pack_filters(False))
        if on_a:
            wait(B, self.ev_tail)
            seg(B, lambda: pack_filters(True))
        rec(self.ev_pack, B)
        # Forward.  A downsampling block's 1x1 projection reads the block input,
        # as its first 3x3 convolution does, and its output is needed only when
        # the block's two branches are added, before the next block: it runs on
        # stream B (idle in the forward pass) beside the two 3x3 convolutions.
        blk = 0
        pending = None
        upd_waited = False
        for L in self.layers:
            if L["bwd_data"] and not upd_waited:
                # The image layer's filter is updated on A itself, so its
                # forward overlaps B's last weight updates; every later layer
                # waits for them.
                wait(A, self.ev_upd)
                upd_waited = True
            if L["name"].endswith("_1x1s2"):
                seg(B, lambda: conv_fwd(L, 0, self.ws_b))
                pending = self.ev_fwd[2 * blk + 1]
                rec(pending, B)
                blk += 1
                continue
            for c in range(L["count"]):
                if L["name"].endswith("3x3s2"):
                    rec(self.ev_fwd[2 * blk], A)      # the block input is ready
                    wait(B, self.ev_fwd[2 * blk])
                if pending is not None and c == 1:
                    wait(A, pending)                  # both branches done before the next block
                    pending = None
                seg(A, lambda: conv_fwd(L, c, self.ws))
        wait(A, self.ev_pack)
        seg(A, head)
        ev = 0
        rec(self.ev_bwd[ev], A)
        wait(B, self.ev_bwd[ev])
        seg(B, lambda: niti.conv_bwd_weight(fd, self.feat.view(Bsz, 1, 1, fin), self.err.view(Bsz, 1, 1, fout),
                                            self.wfc.view(fout, 1, 1, fin), self.stats, self.ws_b, mu=self.mu,
                                            stats_index=s + 3))
        # B waits, before layer l's weight gradient, for the event after the
        # A call that produced dy(l) (the back-propagation of layer l + 1, or
        # the head): the back-propagation of layer l itself reads the packed
        # copy of w(l), not w(l), so the update need not wait for it.
        waited = ev
        for L in reversed(self.layers):
            d = L["desc"]
            for c in reversed(range(L["count"])):
                w = L["w"][c]
                s0 = L["stats"] + 3 * c
                if not L["bwd_data"]:
                    # The image layer has no back-propagation: stream A,
                    # idle from here on, takes its weight gradient, which
                    # then overlaps B's remaining queue instead of ending it.
                    seg(A, lambda: niti.conv_bwd_weight(d, L["x"], L["dy"], w, self.stats, self.ws, mu=self.mu,
                                                        stats_index=s0 + 2))
                    continue
                if (id(L), c) not in on_a:
                    if waited != ev:
                        wait(B, self.ev_bwd[ev])
                        waited = ev
                    seg(B, lambda: niti.conv_bwd_weight(d, L["x"], L["dy"], w, self.stats, self.ws_b, mu=self.mu,
                                                        stats_index=s0 + 2))
                pk = L["packed"][c]
                seg(A, lambda: niti.conv_bwd_data_packed(d, L["dy"], pk, L["dx"], self.stats,
                                                         relu_src=L["x"], stats_index=s0 + 1))
                nb = pos[(id(L), c)] + 1
                if nb < len(bwd) and (id(bwd[nb][0]), bwd[nb][1]) not in on_a:
                    ev += 1                         # dy of the next layer, for its weight gradient on B
                    rec(self.ev_bwd[ev], A)
                if (id(L), c) in on_a:
                    seg(A, lambda: niti.conv_bwd_weight(d, L["x"], L["dy"], w, self.stats, self.ws, mu=self.mu,
                                                        stats_index=s0 + 2))
        rec(self.ev_upd, B)
        if on_a:
            rec(self.ev_tail, A)

    def prepare(self):
        """Run one step and keep it as a plan for step_prepared()."""
        self.plan = []
        self.step(plan=self.plan)

    def step_prepared(self):
        """Replay the plan recorded by prepare(): the same calls and events."""
        replay = self.niti.replay
        for op in self.plan:
            if op[0] == "calls":
                replay(op[1])
            elif op[0] == "rec":
                op[1].record(op[2])
            else:
                op[2].wait(op[1])

    def serial_plan(self):
        """The step's calls one after another on the current stream, as a
        list of (layer, pass, ops, algorithmic bytes, call); contraction calls
        launch exactly one main kernel each (pass fwd / dgrad / wgrad), the
        loss none.  Algorithmic bytes: int8 operands read once and the int8
        output written once (+ the ReLU source read by the back-propagation;
        the weight read and written by the update)."""
        niti = self.niti
        Bsz = self.batch
        fin, fout = self.fc_desc.c, self.fc_desc.k
        s = self.fc_stats
        fd = self.fc_desc
        plan = []
        for L in self.layers:
            d = L["desc"]
            xb, yb = d.n * d.h * d.w * d.c, d.n * d.p * d.q * d.k
            wb = d.k * d.r * d.s * d.c
            for c in range(L["count"]):
                plan.append((L["name"], "fwd", 2 * L["macs"], xb + wb + yb,
                             lambda L=L, c=c: niti.conv_fwd(L["desc"], L["x"], L["w"][c], L["y"], self.stats,
                                                            relu=True, stats_index=L["stats"] + 3 * c, ws=self.ws)))
        plan.append(("fc", "fwd", 2 * self.fc_macs, Bsz * fin + fout * fin + Bsz * fout,
                     lambda: niti.gemm_fwd(self.feat, self.wfc, self.logits, self.stats, self.s_feat, self.s_wfc,
                                           self.s_logits, 7, False, stats_index=s)))
        plan.append(("fc", "loss", 0, 2 * Bsz * fout,
                     lambda: niti.int_ce_loss_grad(self.logits, self.s_logits, self.labels, self.err, self.stats,
                                                   self.ws, stats_index=s + 1)))
        plan.append(("fc", "dgrad", 2 * self.fc_macs, Bsz * fout + fout * fin + 2 * Bsz * fin,
                     lambda: niti.conv_bwd_data(fd, self.err.view(Bsz, 1, 1, fout), self.wfc.view(fout, 1, 1, fin),
                                                self.dfeat.view(Bsz, 1, 1, fin), self.stats, self.ws,
                                                relu_src=self.feat.view(Bsz, 1, 1, fin), stats_index=s + 2)))
        plan.append(("fc", "wgrad", 2 * self.fc_macs, Bsz * fin + Bsz * fout + 2 * fout * fin,
                     lambda: niti.conv_bwd_weight(fd, self.feat.view(Bsz, 1, 1, fin), self.err.view(Bsz, 1, 1, fout),
                                                  self.wfc.view(fout, 1, 1, fin), self.stats, self.ws, mu=self.mu,
                                                  stats_index=s + 3)))
        for L in reversed(self.layers):
            d = L["desc"]
            xb, yb = d.n * d.h * d.w * d.c, d.n * d.p * d.q * d.k
            wb = d.k * d.r * d.s * d.c
            for c in reversed(range(L["count"])):
                s0 = L["stats"] + 3 * c
                if L["bwd_data"]:
                    plan.append((L["name"], "dgrad", 2 * L["macs"], yb + wb + 2 * xb,
                                 lambda L=L, c=c, s0=s0: niti.conv_bwd_data(L["desc"], L["dy"], L["w"][c], L["dx"],
                                                                            self.stats, self.ws, relu_src=L["x"],
                                                                            stats_index=s0 + 1)))
                plan.append((L["name"], "wgrad", 2 * L["macs"], xb + yb + 2 * wb,
                             lambda L=L, c=c, s0=s0: niti.conv_bwd_weight(L["desc"], L["x"], L["dy"], L["w"][c],
                                                                          self.stats, self.ws, mu=self.mu,
                                                                          stats_index=s0 + 2)))
        return plan

    def step_serial(self):
        """The same calls, all on the current stream, one after another (for
        per-call kernel durations without overlap)."""
        if not hasattr(self, "_serial"):
            self._serial = self.serial_plan()
        for entry in self._serial:
            entry[-1]()

    def misses(self):
        st = self.niti.read_stats(self.stats)
        return sum(x["misses"] for x in st), sum(x["calls"] for x in st)

    def miss_table(self):
        """{layer/pass: misses} for stats blocks that missed at least once."""
        st = self.niti.read_stats(self.stats)
        out = {}
        for L in self.layers:
            for c in range(L["count"]):
                for k, name in enumerate(("fwd", "bwd_data", "bwd_weight")):
                    m = st[L["stats"] + 3 * c + k]["misses"]
                    if m:
                        out["%s#%d/%s" % (L["name"], c, name)] = m
        for k, name in enumerate(("fwd", "loss", "bwd_data", "bwd_weight")):
            m = st[self.fc_stats + k]["misses"]
            if m:
                out["fc/%s" % name] = m
        return out


# ----------------------------------------------------------------------------
def _bound(ops, nbytes):
    """The roofline bound of a pass: (name, microseconds at that bound)."""
    t_mfma = ops / (PEAK_INT8_TOPS * 1e12) * 1e6
    t_hbm = nbytes / (PEAK_HBM_GBS * 1e9) * 1e6
    return ("mfma", t_mfma) if t_mfma >= t_hbm else ("hbm", t_hbm)


def _spin():
    """Let the host queue run ahead of the GPU, so that no timing event
    waits on the host."""
    import torch
    torch.cuda.synchronize()
    try:
        torch.cuda._sleep(int(0.05 * 2.4e9))
    except Exception:
        pass


def measure_serial(job, steps):
    """`steps` serial steps with the library's timing records on.  Records
    come in enqueue order; every plan entry opens with one record of family
    IGEMM (forward, back-propagation), WGRAD (weight gradient) or LOSS, and
    the KERNEL / SUM / UPDATE records that follow belong to it."""
    import collections
    import torch
    niti = job.niti
    plan = job.serial_plan()
    job._serial = plan
    _spin()
    niti.timing_enable(True)
    for _ in range(steps):
        job.step_serial()
    niti.timing_enable(False)
    torch.cuda.synchronize()
    recs = niti.timing_records()
    lead = {niti.TIMING_IGEMM, niti.TIMING_WGRAD, niti.TIMING_LOSS}
    calls = []
    for fam, name, ms in recs:
        if fam in lead:
            calls.append({"fam": fam, "ms": ms, "kernel": None, "kernel_ms": 0.0, "sum": None, "update_ms": 0.0})
        elif fam == niti.TIMING_KERNEL:
            calls[-1]["kernel"], calls[-1]["kernel_ms"] = name, ms
        elif fam == niti.TIMING_SUM:
            calls[-1]["sum"] = (name, ms)
        elif fam == niti.TIMING_UPDATE:
            calls[-1]["update_ms"] = ms
    assert len(calls) == steps * len(plan), (len(calls), steps, len(plan))
    kern = collections.OrderedDict()
    fam = {"igemm": [0, 0.0, 0], "wgrad": [0, 0.0, 0]}
    layer = collections.OrderedDict()
    passes = {"split_sum": [0.0, 0, 0], "update": [0.0, 0, 0], "loss": [0.0, 0, 0]}
    for i, c in enumerate(calls):
        lname, pss, ops, nbytes, _ = plan[i % len(plan)]
        if pss == "loss":
            passes["loss"][0] += c["ms"]
            passes["loss"][1] += 1
            passes["loss"][2] += job.batch * job.fc_desc.k * (1 + 16 + 16 + 1) + 4 * job.batch
            call_ms = c["ms"]
        else:
            k = kern.setdefault(c["kernel"], [0, 0.0, 0, 0])
            k[0] += 1
            k[1] += c["kernel_ms"]
            k[2] += ops
            k[3] += nbytes
            f = fam["wgrad" if pss == "wgrad" else "igemm"]
            f[0] += 1
            f[1] += c["ms"]
            f[2] += ops
            call_ms = c["ms"]
            if pss == "wgrad":
                d = job.fc_desc if lname == "fc" else [L for L in job.layers if L["name"] == lname][0]["desc"]
                nw = d.k * d.r * d.s * d.c
                sname, sms = c["sum"]
                splits = int(sname.split("<")[1].rstrip(">"))
                passes["split_sum"][0] += sms
                passes["split_sum"][1] += 1
                passes["split_sum"][2] += 4 * nw * splits + (4 * nw if splits > 1 else 0)
                passes["update"][0] += c["update_ms"]
                passes["update"][1] += 1
                passes["update"][2] += 6 * nw
                call_ms += sms + c["update_ms"]
        e = layer.setdefault((lname, pss), [0, 0.0, ops, nbytes])
        e[0] += 1
        e[1] += call_ms
    return {"kernels": kern, "families": fam, "layers": layer, "passes": passes}


def c4_layer_table(ser):
    out = []
    for (lname, pss), (n, ms, ops, nbytes) in ser["layers"].items():
        us = ms * 1e3 / n
        bname, t_bound = _bound(ops, nbytes)
        rec = {"layer": lname, "pass": pss, "us": round(us, 2), "bound": bname,
               "frac_of_bound": round(t_bound / us, 4)}
        if ops:
            rec["tops"] = round(ops / (us * 1e-6) / 1e12, 1)
        out.append(rec)
    return out


def c5_sweep(reps=5, sizes=(4096, 8192, 16384), dists=("u127", "u15")):
    """The fused GEMM + block maximum + Algorithm 3 rounding (one
    niti_gemm_fwd call: main kernel and finishing launch) on every (M, N, K)
    in sizes^3, int8 operands U[-127,127] and U[-15,15].  A cold call (no
    binary-point guess yet: the output is rounded twice) is timed apart from
    the median of `reps` steady calls."""
    import torch
    from paper_2009_13108_amd import inputs as I
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    big = max(sizes)
    out = []
    C = torch.empty(big * big, dtype=torch.int8, device="cuda")
    for di, dist in enumerate(dists):
        gen = I.weights if dist == "u127" else I.errors5
        A = gen(I.base_seed(5, 1 + 10 * di), (big * big,), device="cuda")
        B = gen(I.base_seed(5, 2 + 10 * di), (big * big,), device="cuda")
        for M in sizes:
            for N in sizes:
                for K in sizes:
                    a, b, c = A[:M * K].view(M, K), B[:N * K].view(N, K), C[:M * N].view(M, N)
                    stats = niti.new_stats()
                    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * (reps + 1))]
                    torch.cuda.synchronize()
                    for r in range(reps + 1):
                        ev[2 * r].record()
                        niti.gemm_fwd(a, b, c, stats)
                        ev[2 * r + 1].record()
                    torch.cuda.synchronize()
                    t = [ev[2 * r].elapsed_time(ev[2 * r + 1]) for r in range(reps + 1)]
                    steady = sorted(t[1:])[reps // 2]
                    tops = 2.0 * M * N * K / (steady * 1e-3) / 1e12
                    st = niti.read_stats(stats)[0]
                    out.append({"M": M, "N": N, "K": K, "dist": dist, "ms": round(steady, 4),
                                "cold_ms": round(t[0], 4), "tops": round(tops, 1),
                                "frac": round(tops / PEAK_INT8_TOPS, 4), "misses": st["misses"]})
        del A, B
    return out


def _replay_time(calls, reps):
    import torch
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    for _ in range(2):
        niti.replay(calls)
    _spin()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        niti.replay(calls)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def small_configs(reps=50):
    """Configs 1-3 as whole steps, each step's library calls marshalled once
    and replayed (so that the host does not pace the GPU).
      c1: fully-connected 784->128, batch 32: forward, back-propagation of
          5-bit errors, weight gradient + update;
      c2: MLP 784-256-128-10, batch 256: input quantisation, forward, loss,
          backward (Algorithm 1);
      c3: VGG-style CNN on 32x32x3, batch 256, the same."""
    import torch
    from paper_2009_13108_amd import inputs as I
    from paper_2009_13108_amd import model as M
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    res = {}
    # c1
    B, K, N = 32, 784, 128
    x = I.activations(I.base_seed(1, 1), (B, K), device="cuda")
    w = I.weights(I.base_seed(1, 2), (N, K), device="cuda")
    e = I.errors5(I.base_seed(1, 3), (B, N), device="cuda")
    gd = niti.ConvDesc.make(B, 1, 1, K, N, 1, 1, 1, 0)
    stats = niti.new_stats(3)
    y = torch.empty((B, N), dtype=torch.int8, device="cuda")
    dx = torch.empty((B, 1, 1, K), dtype=torch.int8, device="cuda")
    ws = niti.new_workspace(max(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, gd),
                                niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, gd)))
    s_x, s_w, s_y = (torch.tensor([v], dtype=torch.int8, device="cuda") for v in (-7, -7, 0))
    with niti.recording() as calls:
        niti.gemm_fwd(x, w, y, stats, s_x, s_w, s_y, stats_index=0)
        niti.conv_bwd_data(gd, e.view(B, 1, 1, N), w.view(N, 1, 1, K), dx, stats, ws, stats_index=1)
        niti.conv_bwd_weight(gd, x.view(B, 1, 1, K), e.view(B, 1, 1, N), w.view(N, 1, 1, K), stats, ws, mu=5,
                             stats_index=2)
    ms = _replay_time(calls, reps)
    ops = 3 * 2 * B * K * N
    res["c1"] = {"workload": "fc784x128_b32", "us_per_step": round(ms * 1e3, 2),
                 "tops": round(ops / (ms * 1e-3) / 1e12, 3), "ops_per_step": ops}
    # c2, c3
    for key, specs, hwc, img_c, batch, cfg, name in (
            ("c2", M.MLP_784, (28, 28, 1), 1, 256, 2, "mlp784_256_128_10_b256"),
            ("c3", M.VGG_32, (32, 32, 4), 3, 256, 3, "vgg32_64_64_128_128_256_256_fc10_b256")):
        ws_, exps = M.synthetic_weights(specs, hwc[2], cfg, image_channels=img_c if hwc[2] != img_c else None)
        net = M.IntNet(specs, hwc, batch, ws_, exps)
        px = I.pixels(I.base_seed(cfg, 1), (batch, img_c, hwc[0], hwc[1]), device="cuda")
        lab = I.labels(I.base_seed(cfg, 2), batch, 10, device="cuda")
        xq = torch.empty((batch,) + hwc, dtype=torch.int8, device="cuda")
        s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")
        with niti.recording() as calls:
            niti.quantize_u8(px, xq)
            net.step(xq, s0, lab)
        ms = _replay_time(calls, reps if key != "c3" else 10)
        ops = 2 * M.contraction_macs(specs, hwc, batch, img_c if hwc[2] != img_c else None)
        res[key] = {"workload": name, "us_per_step": round(ms * 1e3, 2),
                    "tops": round(ops / (ms * 1e-3) / 1e12, 3), "ops_per_step": ops}
    return res


def paper_nets(reps=10, batch=256):
    """The paper's own networks (Section 4, Tables 5) as whole training
    steps at batch 256 on synthetic inputs of the datasets' shapes (input
    quantisation, forward, integer loss, backward and update; dropout before
    VGG-small's classifier), each step's calls marshalled once and replayed."""
    import torch
    from paper_2009_13108_amd import inputs as I
    from paper_2009_13108_amd import model as M
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    res = {}
    nets = [("lenet5", M.LENET5, 28, 1, M.LENET5_REAL["zero_filters"])]
    nets += [("vgg_small%d" % dd, M.vgg_small(dd), 32, 3, None) for dd in (7, 8, 9)]
    for i, (name, specs, hw, img_c, zf) in enumerate(nets):
        cfg = 40 + i
        ws_, exps = M.synthetic_weights(specs, 4, cfg, image_channels=img_c, zero_filters=zf)
        net = M.IntNet(specs, (hw, hw, 4), batch, ws_, exps, drop_seed=cfg)
        px = I.pixels(I.base_seed(cfg, 1), (batch, img_c, hw, hw), device="cuda")
        lab = I.labels(I.base_seed(cfg, 2), batch, 10, device="cuda")
        xq = torch.empty((batch, hw, hw, 4), dtype=torch.int8, device="cuda")
        s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")
        with niti.recording() as calls:
            niti.quantize_u8(px, xq)
            net.step(xq, s0, lab)
        ms = _replay_time(calls, reps)
        ops = 2 * M.contraction_macs(specs, (hw, hw, 4), batch, img_c)
        res[name] = {"batch": batch, "input": "%dx%dx%d" % (hw, hw, img_c), "us_per_step": round(ms * 1e3, 2),
                     "tops": round(ops / (ms * 1e-3) / 1e12, 1), "ops_per_step": ops}
        del net, calls
    return res


def alexnet_layers(reps=5, batch=128):
    """AlexNet's contraction shapes (Table 6's network) at batch 128: per
    layer the forward (exponent + rounding + ReLU fused), the
    back-propagation (rounding and ReLU mask fused; not formed for the first
    layer) and the weight gradient with its update."""
    import torch
    from paper_2009_13108_amd import inputs as I
    from paper_2009_13108_amd import model as M
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    out = []
    shapes = [(n, ci, co, k, st, pd, hw) for (n, ci, co, k, st, pd, hw) in M.ALEXNET_LAYERS]
    shapes += [(n, fi, fo, 1, 1, 0, 1) for (n, fi, fo) in M.ALEXNET_FC]
    for li, (name, cin, cout, k, st, pd, hw) in enumerate(shapes):
        d = niti.ConvDesc.make(batch, hw, hw, cin, cout, k, k, st, pd)
        x = I.activations(I.base_seed(8, 100 + li), d.x_shape(), device="cuda")
        w = I.weights(I.base_seed(8, 200 + li), d.w_shape(), device="cuda")
        c_real = cin
        if li == 0:
            x[..., 3:] = 0
            w[..., 3:] = 0
            c_real = 3
        dy = I.errors8(I.base_seed(8, 300 + li), d.y_shape(), device="cuda")
        y = torch.empty(d.y_shape(), dtype=torch.int8, device="cuda")
        dx = torch.empty(d.x_shape(), dtype=torch.int8, device="cuda")
        stats = niti.new_stats(3)
        ws = niti.new_workspace(max(niti.workspace_bytes(op, d) for op in (1, 2, 3)))
        passes = {"fwd": lambda: niti.conv_fwd(d, x, w, y, stats, relu=True, ws=ws, stats_index=0),
                  "bwd_data": lambda: niti.conv_bwd_data(d, dy, w, dx, stats, ws, relu_src=x, stats_index=1),
                  "bwd_weight+update": lambda: niti.conv_bwd_weight(d, x, dy, w, stats, ws, mu=5, stats_index=2)}
        if li == 0:
            del passes["bwd_data"]
        macs = conv_macs(batch, c_real, hw, hw, cout, k, k, st, pd)
        for pss, fn in passes.items():
            with niti.recording() as calls:
                fn()
            ms = _replay_time(calls, reps)
            tops = 2 * macs / (ms * 1e-3) / 1e12
            out.append({"layer": name, "pass": pss, "us": round(ms * 1e3, 2), "tops": round(tops, 1),
                        "frac": round(tops / PEAK_INT8_TOPS, 4)})
        del x, w, dy, y, dx, ws
    return out


def launch_overhead_us(reps=50):
    """Average time between a HIP event pair around one empty launch (the
    int8 MFMA loop with no iterations, one workgroup) on the current stream,
    queued behind other work: what an event-timed kernel duration holds
    besides the kernel itself."""
    import torch
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    out = torch.empty(1024 * 256, dtype=torch.int32, device="cuda")
    niti.mfma_loop(0, 1, out)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    # a few milliseconds of matrix work first, so that the pairs below are
    # queued before the GPU reaches them and time the GPU, not the host
    niti.mfma_loop(8192, 1024, out)
    for a, b in ev:
        a.record()
        niti.mfma_loop(0, 1, out)
        b.record()
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in ev) * 1e3 / reps


def mfma_loop_rate(iters=4096, per_cu=4, reps=5):
    """The int8 MFMA loop (register operands, no memory traffic) over
    256 x per_cu workgroups: the rate matrix work sustains on this device."""
    import torch
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    wg = 256 * per_cu
    out = torch.empty(wg * 256, dtype=torch.int32, device="cuda")
    niti.mfma_loop(16, wg, out)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        niti.mfma_loop(iters, wg, out)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = sorted(times)[len(times) // 2]
    ops = wg * 4 * iters * 8 * 65536
    tops = ops / (ms * 1e-3) / 1e12
    return {"workgroups": wg, "iters": iters, "us": round(ms * 1e3, 1), "tops": round(tops, 1),
            "frac": round(tops / PEAK_INT8_TOPS, 4)}


# RTX 3090 int8 times (ms) the paper's Table 7 reports for these shapes: context only.
TABLE7_PAPER_3090_MS = {"a": {224: 3.928, 112: 1.006, 56: 0.289, 28: 0.089, 14: 0.038},
                        "e": {224: 4.731, 112: 1.269, 56: 0.453, 28: 0.185, 14: 0.117},
                        "g": {224: 122.301, 112: 27.327, 56: 6.911, 28: 1.074, 14: 0.272}}


def table7(reps=5):
    """The paper's GPU shapes (batch 64, 64 -> 128 channels, 3x3, stride 1,
    pad 1; inputs 224 ... 14): a = forward (fused exponent and rounding),
    e = error back-propagation (fused), g = weight gradient + update."""
    import torch
    from paper_2009_13108_amd import inputs as I
    niti = __import__("paper_2009_13108_amd.niti", fromlist=["niti"])
    out = []
    for hw in (224, 112, 56, 28, 14):
        d = niti.ConvDesc.make(64, hw, hw, 64, 128, 3, 3, 1, 1)
        x = I.activations(I.base_seed(7, 1), d.x_shape(), device="cuda")
        w = I.weights(I.base_seed(7, 2), d.w_shape(), device="cuda")
        dy = I.errors8(I.base_seed(7, 3), d.y_shape(), device="cuda")
        y = torch.empty(d.y_shape(), dtype=torch.int8, device="cuda")
        dx = torch.empty(d.x_shape(), dtype=torch.int8, device="cuda")
        stats = niti.new_stats(3)
        ws = niti.new_workspace(max(niti.workspace_bytes(op, d) for op in (1, 2, 3)))
        passes = {"a": lambda: niti.conv_fwd(d, x, w, y, stats, relu=True, ws=ws, stats_index=0),
                  "e": lambda: niti.conv_bwd_data(d, dy, w, dx, stats, ws, relu_src=x, stats_index=1),
                  "g": lambda: niti.conv_bwd_weight(d, x, dy, w, stats, ws, mu=5, stats_index=2)}
        macs = 64 * hw * hw * 128 * 64 * 9
        for k, fn in passes.items():
            with niti.recording() as calls:
                fn()
            ms = _replay_time(calls, reps)
            out.append({"input": hw, "pass": k, "ms": round(ms, 4),
                        "tops": round(2 * macs / (ms * 1e-3) / 1e12, 1),
                        "paper_rtx3090_int8_ms": TABLE7_PAPER_3090_MS[k][hw]})
        del x, dy, y, dx, ws
    return out


# ----------------------------------------------------------------------------
def cpu_baseline(batch=2):
    """The oracle on the same layer set at a small batch: one step of
    forward, error back-propagation and weight gradient + update per distinct
    layer shape (each once), plus the head and the loss."""
    import numpy as np

    import oracle
    from paper_2009_13108_amd import inputs as I
    from paper_2009_13108_amd import model as M

    ops = 0
    t0 = time.time()
    for li, (name, cin, cout, k, st, pd, hw, count) in enumerate(M.RESNET18_LAYERS):
        c = 3 if name.startswith("stem") else cin
        d = oracle.conv_desc(batch, c, hw, hw, cout, k, k, st, pd)
        P, Q = oracle.conv_out_hw(d)
        x = I.activations(I.base_seed(4, 100 + li), (batch, c, hw, hw))
        dy = I.errors8(I.base_seed(4, 200 + li), (batch, cout, P, Q))
        w = I.weights(I.base_seed(4, 1000 + 10 * li), (cout, c, k, k))
        macs = conv_macs(batch, c, hw, hw, cout, k, k, st, pd)
        oracle.conv_fwd(d, x, w, relu=True)
        ops += 2 * macs
        if not name.startswith("stem"):
            oracle.conv_bwd_data(d, dy, w, relu_src=x)
            ops += 2 * macs
        oracle.conv_bwd_weight(d, x, dy, w, mu=5)
        ops += 2 * macs
    fin, fout = M.RESNET18_FC
    feat = I.activations(I.base_seed(4, 300), (batch, fin))
    wfc = I.weights(I.base_seed(4, 301), (fout, fin))
    lab = I.labels(I.base_seed(4, 302), batch, fout)
    logits, _, _ = oracle.gemm_fwd(feat, wfc)
    err, _, _ = oracle.int_ce_loss_grad(logits, -9, lab)
    fd = oracle.conv_desc(batch, fin, 1, 1, fout, 1, 1, 1, 0)
    oracle.conv_bwd_data(fd, err.reshape(batch, fout, 1, 1), wfc.reshape(fout, fin, 1, 1))
    oracle.conv_bwd_weight(fd, feat.reshape(batch, fin, 1, 1), err.reshape(batch, fout, 1, 1),
                           wfc.reshape(fout, fin, 1, 1))
    ops += 3 * 2 * batch * fin * fout
    dt = time.time() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": ops / dt / 1e12, "unit": "TOPS", "cores": cores, "kind": "oracle",
            "sample": "ResNet-18 layer set at 224x224, batch %d, each distinct layer shape once "
                      "(fwd+bwd_data+bwd_weight/update) plus the 512->1000 head and loss; %.2f GOP in %.1f s"
                      % (batch, ops / 1e9, dt)}


# ----------------------------------------------------------------------------
TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "resnet18_b128_traffic.md")


def kernel_sources_digest():
    """sha256 over the library's kernel sources (name and bytes, sorted)."""
    import glob
    import hashlib
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2009_13108_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of a kernel from the committed counter summary, or
    None when the kernel sources changed since the counters were taken."""
    try:
        vals = {}
        with open(TRAFFIC_FILE) as f:
            for line in f:
                k, _, v = line.partition(":")
                vals[k.strip()] = v.strip()
        if vals.get("kernel_sources_sha256") != kernel_sources_digest():
            return None
        return int(vals["%s_hbm_bytes_per_launch" % kernel])
    except (OSError, KeyError, ValueError):
        return None


def kernel_label(profiler_name):
    """The library's label for a profiler kernel name: the kernel's own name
    and its template arguments, without namespaces, spaces or the argument
    list (niti::(anonymous namespace)::igemm_dma_main<128, 128, 4, 4, 2, 1>(...)
    -> igemm_dma_main<128,128,4,4,2,1>)."""
    import re
    n = profiler_name.replace("(anonymous namespace)::", "").replace("void ", "")
    n = re.sub(r"^niti::", "", n)
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
    return n[:cut].replace(" ", "")


def summarize_kernel_trace(path):
    """Per-kernel durations from a rocprofv3 kernel-trace CSV
    (--kernel-trace --output-format csv), labelled as the library labels its
    timing records: all launches, and the launches on the default stream
    (stream 0: the serial pass whose per-kernel times the bench line's
    roofline uses; the timed steps run on two other streams, where kernels
    overlap)."""
    import collections
    import csv

    per = collections.OrderedDict()
    ser = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        if "niti::" not in r["Kernel_Name"]:
            continue
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        lab = kernel_label(r["Kernel_Name"])
        per.setdefault(lab, []).append(dur)
        if r.get("Stream_Id", "0") == "0":
            ser[lab].append(dur)
    print("%-44s %7s %11s %9s %11s %11s" % ("kernel", "calls", "total_us", "avg_us", "serial_n", "serial_avg"))
    for name, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        sv = ser.get(name, [])
        print("%-44s %7d %11.1f %9.2f %11d %11s" % (name[:44], len(v), sum(v), sum(v) / len(v), len(sv),
                                                     "%.2f" % (sum(sv) / len(sv)) if sv else "-"))


def summarize_counters(path):
    """Per-kernel averages of a rocprofv3 --pmc counter CSV (e.g. FETCH_SIZE
    or WRITE_SIZE in KiB per dispatch), labelled as above, plus the plain
    copy kernel used for calibration.  When the run collected
    GRBM_GUI_ACTIVE with SQ_VALU_MFMA_BUSY_CYCLES (and optionally
    SQ_INSTS_VALU_MFMA_MOPS_I8), also per kernel: the shader clock
    (GRBM_GUI_ACTIVE is summed over the 8 XCDs, so cycles = value / 8, over
    the dispatch's duration), the matrix cores' busy fraction (busy cycles
    over 1024 SIMDs x cycles) and the int8 rate (MOPS_I8 counts units of
    512 operations)."""
    import collections
    import csv

    per = collections.defaultdict(lambda: collections.defaultdict(float))
    disp = collections.defaultdict(dict)
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"]
        lab = kernel_label(name) if "niti::" in name else name[:60]
        per[r["Counter_Name"]][lab] += float(r["Counter_Value"])
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 if "End_Timestamp" in r else 0.0
        disp[lab][r["Dispatch_Id"]] = dur
    for cname, vals in per.items():
        for lab, v in sorted(vals.items(), key=lambda kv: -kv[1]):
            n = len(disp[lab])
            print("%s %-60s launches %6d per launch %14.1f" % (cname, lab, n, v / n))
    grbm, busy = per.get("GRBM_GUI_ACTIVE"), per.get("SQ_VALU_MFMA_BUSY_CYCLES")
    if not grbm or not busy:
        return
    mops = per.get("SQ_INSTS_VALU_MFMA_MOPS_I8", {})
    print()
    print("%-48s %7s %9s %6s %7s %8s" % ("kernel", "calls", "avg_us", "GHz", "mfma%", "int8TOPS"))
    rows = []
    for lab in grbm:
        n = len(disp[lab])
        us = sum(disp[lab].values()) / n
        cyc = grbm[lab] / 8.0 / n
        if cyc <= 0 or us <= 0:
            continue
        util = busy.get(lab, 0.0) / n / (cyc * 1024.0)
        tops = mops.get(lab, 0.0) * 512.0 / n / (us * 1e-6) / 1e12
        rows.append((us * n, lab, n, us, cyc / us / 1e3, 100.0 * util, tops))
    for _, lab, n, us, ghz, util, tops in sorted(rows, reverse=True):
        print("%-48s %7d %9.2f %6.2f %7.1f %8.1f" % (lab[:48], n, us, ghz, util, tops))


def copy_calibration(nbytes, pattern="contiguous"):
    """A plain device copy of nbytes (torch's copy kernel), five times: the
    reference for scaling FETCH_SIZE / WRITE_SIZE to bytes.  pattern:
      contiguous  read nbytes, write nbytes;
      strided128  read the first 128 bytes of every 256-byte row of a
                  2 * nbytes buffer (whole 128-byte lines, every other one),
                  write them contiguously: nbytes each way;
      strided64   read the first 64 bytes of every 128-byte row (half lines),
                  write them contiguously: nbytes of data each way."""
    import torch
    if pattern == "contiguous":
        a = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
        src = a
    else:
        w = 128 if pattern == "strided128" else 64
        a = torch.empty(2 * nbytes, dtype=torch.uint8, device="cuda").fill_(1)
        src = a.view(nbytes // w, 2 * w)[:, :w]
    b = torch.empty(src.shape, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    for _ in range(5):
        b.copy_(src)
    torch.cuda.synchronize()
    print("copied %d bytes x5 (%s)" % (nbytes, pattern), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-batch", type=int, default=64)
    ap.add_argument("--no-configs", action="store_true",
                    help="skip configs 1-3, the config-5 GEMM sweep, the Table 7 shapes, the paper networks and the AlexNet layers")
    ap.add_argument("--only", choices=("c5", "small", "table7", "paper_nets", "alexnet", "mfma_loop"),
                    help="run only the config-5 sweep, configs 1-3 or the Table 7 shapes and print their JSON "
                         "(for profiling one workload)")
    ap.add_argument("--c5-sizes", default="4096,8192,16384", help="sizes of the --only c5 sweep")
    ap.add_argument("--no-prepared", action="store_true",
                    help="enqueue every call through the checked binding instead of replaying prepared calls")
    ap.add_argument("--kernel-trace", metavar="CSV",
                    help="summarize a rocprofv3 kernel-trace CSV of a bench run and exit (no GPU)")
    ap.add_argument("--counters", metavar="CSV",
                    help="summarize a rocprofv3 --pmc counter CSV per kernel family and exit (no GPU)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="run only a plain device copy of this many bytes (counter calibration)")
    ap.add_argument("--copy-pattern", choices=("contiguous", "strided128", "strided64"), default="contiguous",
                    help="access pattern of the --copy-bytes copy")
    args = ap.parse_args()
    if args.kernel_trace:
        summarize_kernel_trace(args.kernel_trace)
        return
    if args.counters:
        summarize_counters(args.counters)
        return
    if args.copy_bytes:
        copy_calibration(args.copy_bytes, args.copy_pattern)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.only:
        if args.only == "c5":
            res = c5_sweep(sizes=tuple(int(v) for v in args.c5_sizes.split(",")))
        elif args.only == "small":
            res = small_configs()
        elif args.only == "paper_nets":
            res = paper_nets()
        elif args.only == "alexnet":
            res = alexnet_layers()
        elif args.only == "mfma_loop":
            res = mfma_loop_rate()
        else:
            res = table7()
        print(json.dumps({"only": args.only, "result": res}), flush=True)
        return
    print("[bench] building inputs", file=sys.stderr, flush=True)
    job = ResNetStep(batch=args.batch)
    torch.cuda.synchronize()
    print("[bench] warmup %d" % args.warmup, file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        job.step()
    torch.cuda.synchronize()
    m0, c0 = job.misses()

    # headline: K whole steps between two events.  Default: the step's calls
    # are marshalled once (prepare) and replayed each step, so the host's
    # Python argument checks do not pace the GPU; --no-prepared enqueues
    # every call through the checked binding.
    prepared = not args.no_prepared
    if prepared:
        job.prepare()
        torch.cuda.synchronize()
        m0, c0 = job.misses()
    print("[bench] timing %d steps" % args.steps, file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(job.sA)   # steps start on stream A; A waits for B's last updates before e1
    h0 = time.perf_counter()
    for _ in range(args.steps):
        if prepared:
            job.step_prepared()
        else:
            job.step()
    host_ms = (time.perf_counter() - h0) * 1e3 / args.steps
    job.ev_upd.wait(job.sA)
    e1.record(job.sA)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    m1, c1 = job.misses()

    # Kernel-level timing: the same steps again, serialized on one stream (so
    # that no other call's kernels share the GPU while a call is timed), with
    # the library's own HIP events recorded on the launch stream around each
    # contraction's main kernel, each call's kernels, and the sum, update and
    # loss passes.
    ser = measure_serial(job, args.steps)
    kern = ser["kernels"]
    top = max(kern, key=lambda k: kern[k][1])
    n_top, ms_top, ops_top, bytes_top = kern[top]
    achieved = ops_top / (ms_top * 1e-3) / 1e12
    value = job.ops_per_step / (ms * 1e-3) / 1e12
    fam = ser["families"]

    # the matrix cores' sustained int8 rate with no memory traffic (context
    # for the roofline fraction, which stays against the published peak)
    loop = mfma_loop_rate()
    overhead = launch_overhead_us()

    extra = {}
    if not args.no_configs:
        print("[bench] configs 1-3", file=sys.stderr, flush=True)
        extra.update(small_configs())
        print("[bench] config 5 GEMM sweep", file=sys.stderr, flush=True)
        extra["c5"] = c5_sweep()
        print("[bench] paper Table 7 shapes", file=sys.stderr, flush=True)
        extra["table7_context"] = table7()
        print("[bench] paper networks", file=sys.stderr, flush=True)
        extra["paper_nets"] = paper_nets()
        print("[bench] AlexNet layer shapes", file=sys.stderr, flush=True)
        extra["alexnet_layers"] = alexnet_layers()

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle, batch %d)" % args.cpu_batch, file=sys.stderr, flush=True)
        cpu = cpu_baseline(args.cpu_batch)

    passes = {}
    for k, (pms, n, nbytes) in ser["passes"].items():
        if n:
            passes[k] = {"calls_per_step": n // args.steps, "us_per_call": round(pms * 1e3 / n, 2),
                         "gbs": round(nbytes / (pms * 1e-3) / 1e9, 1),
                         "frac_of_hbm": round(nbytes / (pms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    c5 = extra.get("c5", [])
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "host_enqueue_ms_per_step": round(host_ms, 4),
        "execution": "two streams (forward + back-propagation; weight gradients), "
                     + ("prepared calls" if prepared else "checked calls"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "resnet18_layers_224_b%d: 20 conv layers (7x7/2 stem, 3x3 at 56/28/14/7, "
                               "1x1/2 downsample) + 512->1000 head; fwd+bwd_data+bwd_weight/update per layer, "
                               "integer CE loss" % args.batch,
                   "batch": args.batch, "image": 224, "mu": 5, "rounding": "pseudo-stochastic",
                   "parallelism": "single GPU"},
        "pct_of_int8_mfma_peak": round(100.0 * value / PEAK_INT8_TOPS, 2),
        "ops_per_step": job.ops_per_step,
        "hint": {"misses_timed": m1 - m0, "calls_timed": c1 - c0, "misses_by_call": job.miss_table()},
        "roofline": {"bound": "mfma", "kernel": top, "achieved": round(achieved, 3), "peak": PEAK_INT8_TOPS,
                     "unit": "TOPS", "frac": round(achieved / PEAK_INT8_TOPS, 4),
                     "traffic": measured_traffic(top),
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "launches_per_step": n_top // args.steps,
                     "avg_us": round(ms_top * 1e3 / n_top, 2),
                     "event_launch_overhead_us": round(overhead, 2),
                     "avg_us_less_launch_overhead": round(ms_top * 1e3 / n_top - overhead, 2),
                     "algorithmic_ops_per_launch": ops_top // n_top,
                     "algorithmic_bytes_per_launch": bytes_top // n_top,
                     "kernels": {k: {"launches_per_step": v[0] // args.steps, "avg_us": round(v[1] * 1e3 / v[0], 2),
                                     "tops": round(v[2] / (v[1] * 1e-3) / 1e12, 1)}
                                 for k, v in sorted(kern.items(), key=lambda kv: -kv[1][1])},
                     "family_tops": {f: round(v[2] / (v[1] * 1e-3) / 1e12, 1) for f, v in fam.items()},
                     "family_ms_per_step": {f: round(v[1] / args.steps, 4) for f, v in fam.items()}},
        "passes": passes,
        "c4_layers": c4_layer_table(ser),
        "mfma_loop": loop,
        "cpu_baseline": cpu,
    }
    for k in ("c1", "c2", "c3"):
        if k in extra:
            out[k] = extra[k]
    if c5:
        out["c5"] = c5
        big = [r for r in c5 if r["M"] == r["N"] == r["K"]]
        out["c5_square_frac"] = {"%s_%d" % (r["dist"], r["M"]): r["frac"] for r in big}
        out["c5_best_frac"] = max(r["frac"] for r in c5)
    for k in ("table7_context", "paper_nets", "alexnet_layers"):
        if k in extra:
            out[k] = extra[k]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
