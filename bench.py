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
counted on the unpadded channel count); roofline = the dominant kernel
family timed live with HIP events on its stream; cpu_baseline = the CPU
oracle on a bounded sample of the same layer set.
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


def conv_macs(n, c, h, w, k, r, s, st, pd):
    p = (h + 2 * pd - r) // st + 1
    q = (w + 2 * pd - s) // st + 1
    return n * p * q * k * c * r * s


# ----------------------------------------------------------------------------
class ResNetStep:
    """Buffers and call sequence of one training step over the layer set."""

    def __init__(self, batch=128, seed_cfg=4, mu=5):
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
        self.ev_bwd = [torch.cuda.Event() for _ in range(sum(L["count"] for L in self.layers) + 1)]
        self.ev_fwd = [torch.cuda.Event() for _ in range(8)]
        self.ev_upd = torch.cuda.Event()
        self.ev_pack = torch.cuda.Event()
        self.ev_upd.record(self.sB)
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
            stream.wait_event(ev)
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

        def pack_filters():
            for L in self.layers:
                if L["bwd_data"]:
                    for c in range(L["count"]):
                        niti.conv_pack_bwd_data(L["desc"], L["w"][c], L["packed"][c])
            niti.conv_pack_bwd_data(fd, self.wfc.view(fout, 1, 1, fin), self.fc_packed)

        # The filters rearranged for the back-propagation, on stream B (in
        # order after the previous step's updates, and nearly idle in the
        # forward pass); A waits for them before the back-propagation.
        seg(B, pack_filters)
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
                pk = L["packed"][c]
                seg(A, lambda: niti.conv_bwd_data_packed(d, L["dy"], pk, L["dx"], self.stats,
                                                         relu_src=L["x"], stats_index=s0 + 1))
                ev += 1
                rec(self.ev_bwd[ev], A)
                wait(B, self.ev_bwd[ev])
                seg(B, lambda: niti.conv_bwd_weight(d, L["x"], L["dy"], w, self.stats, self.ws_b, mu=self.mu,
                                                    stats_index=s0 + 2))
        rec(self.ev_upd, B)

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
                op[1].wait_event(op[2])

    def step_serial(self):
        """The same calls, all on the current stream, one after another (for
        per-call kernel durations without overlap)."""
        niti = self.niti
        Bsz = self.batch
        fin, fout = self.fc_desc.c, self.fc_desc.k
        s = self.fc_stats
        fd = self.fc_desc
        for L in self.layers:
            for c in range(L["count"]):
                niti.conv_fwd(L["desc"], L["x"], L["w"][c], L["y"], self.stats, relu=True,
                              stats_index=L["stats"] + 3 * c, ws=self.ws)
        niti.gemm_fwd(self.feat, self.wfc, self.logits, self.stats, self.s_feat, self.s_wfc, self.s_logits, 7, False,
                      stats_index=s)
        niti.int_ce_loss_grad(self.logits, self.s_logits, self.labels, self.err, self.stats, self.ws,
                              stats_index=s + 1)
        niti.conv_bwd_data(fd, self.err.view(Bsz, 1, 1, fout), self.wfc.view(fout, 1, 1, fin),
                           self.dfeat.view(Bsz, 1, 1, fin), self.stats, self.ws,
                           relu_src=self.feat.view(Bsz, 1, 1, fin), stats_index=s + 2)
        niti.conv_bwd_weight(fd, self.feat.view(Bsz, 1, 1, fin), self.err.view(Bsz, 1, 1, fout),
                             self.wfc.view(fout, 1, 1, fin), self.stats, self.ws, mu=self.mu, stats_index=s + 3)
        for L in reversed(self.layers):
            d = L["desc"]
            for c in reversed(range(L["count"])):
                w = L["w"][c]
                s0 = L["stats"] + 3 * c
                if L["bwd_data"]:
                    niti.conv_bwd_data(d, L["dy"], w, L["dx"], self.stats, self.ws, relu_src=L["x"],
                                       stats_index=s0 + 1)
                niti.conv_bwd_weight(d, L["x"], L["dy"], w, self.stats, self.ws, mu=self.mu, stats_index=s0 + 2)

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


def measured_traffic(family):
    """HBM bytes per call of a family from the committed counter summary, or
    None when the kernel sources changed since the counters were taken."""
    try:
        vals = {}
        with open(TRAFFIC_FILE) as f:
            for line in f:
                k, _, v = line.partition(":")
                vals[k.strip()] = v.strip()
        if vals.get("kernel_sources_sha256") != kernel_sources_digest():
            return None
        return int(vals["%s_hbm_bytes_per_call" % family])
    except (OSError, KeyError, ValueError):
        return None


def summarize_kernel_trace(path):
    """Per-kernel and per-family durations from a rocprofv3 kernel-trace CSV
    (--kernel-trace --output-format csv), grouped the way the library's timing
    hooks group them: igemm = implicit-GEMM kernels and their finishing
    launches, wgrad = weight-gradient contraction kernels."""
    import collections
    import csv
    import re

    rows = list(csv.DictReader(open(path)))
    per = collections.OrderedDict()
    for r in rows:
        name = re.sub(r"\(.*", "", r["Kernel_Name"].replace("(anonymous namespace)::", "")).replace("void ", "")
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        per.setdefault(name, []).append(dur)
    print("%-58s %7s %11s %9s" % ("kernel", "calls", "total_us", "avg_us"))
    for name, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        if "niti::" in name:
            print("%-58s %7d %11.1f %9.2f" % (name[:58], len(v), sum(v), sum(v) / len(v)))
    fam = {"igemm": (r"niti::igemm_(dma_|wres_)?(main|fixup)<", r"niti::igemm_(dma_|wres_)?main<"),
           "wgrad": (r"niti::wgrad_\w*kernel<", r"niti::wgrad_\w*kernel<")}
    for f, (member, counter) in fam.items():
        tot = sum(sum(v) for n, v in per.items() if re.search(member, n))
        calls = sum(len(v) for n, v in per.items() if re.search(counter, n))
        if calls:
            print("family %-6s calls %6d  total %11.1f us  per call %8.2f us" % (f, calls, tot, tot / calls))


def summarize_counters(path):
    """Per-family sums of a rocprofv3 --pmc counter CSV (one counter per run,
    e.g. FETCH_SIZE or WRITE_SIZE in KiB per dispatch): total over the
    family's kernels divided by its calls, plus the calibration copy."""
    import collections
    import csv
    import re

    per = collections.defaultdict(lambda: collections.defaultdict(float))
    disp = collections.defaultdict(set)
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"]
        per[r["Counter_Name"]][name] += float(r["Counter_Value"])
        disp[name].add(r["Dispatch_Id"])
    calls = {n: len(d) for n, d in disp.items()}
    fam = {"igemm": (r"niti::\(anonymous namespace\)::igemm_(dma_|wres_)?(main|fixup)<", r"igemm_(dma_|wres_)?main<"),
           "wgrad": (r"niti::\(anonymous namespace\)::wgrad_\w*kernel<", r"wgrad_\w*kernel<")}
    for cname, vals in per.items():
        for f, (member, counter) in fam.items():
            tot = sum(v for n, v in vals.items() if re.search(member, n))
            n = sum(c for k, c in calls.items() if re.search(counter, k))
            if n:
                print("%s family %-6s calls %6d  per call %12.1f KiB" % (cname, f, n, tot / n))
        cp = [(n, v) for n, v in vals.items() if "copy" in n.lower() or "elementwise" in n.lower()]
        for n, v in cp:
            print("%s copy-like kernel %s... calls %d per call %.1f KiB" % (cname, n[:60], calls[n], v / max(1, calls[n])))


def copy_calibration(nbytes):
    """A plain device copy of nbytes (torch's copy kernel), five times: the
    reference for scaling FETCH_SIZE / WRITE_SIZE to bytes."""
    import torch
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print("copied %d bytes x5" % nbytes, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-batch", type=int, default=64)
    ap.add_argument("--layers", action="store_true", help="per-layer timing table on stderr")
    ap.add_argument("--no-prepared", action="store_true",
                    help="enqueue every call through the checked binding instead of replaying prepared calls")
    ap.add_argument("--kernel-trace", metavar="CSV",
                    help="summarize a rocprofv3 kernel-trace CSV of a bench run and exit (no GPU)")
    ap.add_argument("--counters", metavar="CSV",
                    help="summarize a rocprofv3 --pmc counter CSV per kernel family and exit (no GPU)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="run only a plain device copy of this many bytes (counter calibration)")
    args = ap.parse_args()
    if args.kernel_trace:
        summarize_kernel_trace(args.kernel_trace)
        return
    if args.counters:
        summarize_counters(args.counters)
        return
    if args.copy_bytes:
        copy_calibration(args.copy_bytes)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
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
    job.sA.wait_event(job.ev_upd)
    e1.record(job.sA)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    m1, c1 = job.misses()

    # roofline: the same steps again, with the library's own HIP events
    # recorded on the launch stream around every contraction launch.  A spin
    # kernel first lets the host queue run ahead, so that no event waits on
    # the host.
    # (serialized on one stream, so that no other call's kernels share the GPU
    # while a call is timed)
    torch.cuda.synchronize()
    try:
        torch.cuda._sleep(int(0.05 * 2.4e9))
    except Exception:
        pass
    niti = job.niti
    niti.timing_enable(True)
    for _ in range(args.steps):
        job.step_serial()
    niti.timing_enable(False)
    torch.cuda.synchronize()
    fams = {"igemm": niti.timing_read(niti.TIMING_IGEMM), "wgrad": niti.timing_read(niti.TIMING_WGRAD)}
    for f, (_, n) in fams.items():
        assert n == args.steps * job.fam_calls[f], (f, n)
    fam = max(fams, key=lambda f: fams[f][0])
    per_call_ms = fams[fam][0] / fams[fam][1]
    ops_per_call = job.fam_ops[fam] / job.fam_calls[fam]
    achieved = ops_per_call / (per_call_ms * 1e-3) / 1e12
    value = job.ops_per_step / (ms * 1e-3) / 1e12

    if args.layers:
        report_layers(job)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle, batch %d)" % args.cpu_batch, file=sys.stderr, flush=True)
        cpu = cpu_baseline(args.cpu_batch)

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
        "roofline": {"bound": "mfma", "kernel": fam, "achieved": round(achieved, 3), "peak": PEAK_INT8_TOPS,
                     "unit": "TOPS", "frac": round(achieved / PEAK_INT8_TOPS, 4),
                     "traffic": measured_traffic(fam),
                     "traffic_unit": "HBM bytes per call (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "algorithmic_bytes_per_call": job.fam_bytes[fam] // job.fam_calls[fam],
                     "per_call_ms": round(per_call_ms, 5), "calls_per_step": job.fam_calls[fam],
                     "family_ms_per_step": {f: round(v[0] / args.steps, 4) for f, v in fams.items()},
                     "family_tops": {f: round(job.fam_ops[f] * args.steps / (v[0] * 1e-3) / 1e12, 2)
                                     for f, v in fams.items()}},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def report_layers(job, reps=5):
    """Per-layer pass times (stderr), for the design notes."""
    import torch
    niti = job.niti
    print("%-12s %10s %10s %10s %8s %8s %8s" % ("layer", "fwd_us", "dgrad_us", "wgrad_us", "fwdTOPS",
                                                 "dgTOPS", "wgTOPS"), file=sys.stderr)
    for L in job.layers:
        d, w, s0 = L["desc"], L["w"][0], L["stats"]
        calls = [lambda: niti.conv_fwd(d, L["x"], w, L["y"], job.stats, relu=True, stats_index=s0, ws=job.ws),
                 (lambda: niti.conv_bwd_data(d, L["dy"], w, L["dx"], job.stats, job.ws, relu_src=L["x"],
                                             stats_index=s0 + 1)) if L["bwd_data"] else None,
                 lambda: niti.conv_bwd_weight(d, L["x"], L["dy"], w, job.stats, job.ws, mu=job.mu,
                                              stats_index=s0 + 2)]
        us = []
        for fn in calls:
            if fn is None:
                us.append(float("nan"))
                continue
            fn()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            us.append(a.elapsed_time(b) * 1e3 / reps)
        tops = [2 * L["macs"] / (u * 1e-6) / 1e12 if u == u else float("nan") for u in us]
        print("%-12s %10.1f %10.1f %10.1f %8.1f %8.1f %8.1f" % ((L["name"],) + tuple(us) + tuple(tops)),
              file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
