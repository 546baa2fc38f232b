"""Whole NITI training steps (Algorithm 1) on the GPU against the oracle's
composition, several steps in a row, byte for byte: logits, their exponent,
and every layer's weights after each step.

Workloads: one fully-connected layer 784->128 (batch 32, 5-bit errors); the
integer MLP 784-256-128-10 on 28x28 synthetic images (batch 256); the
VGG-style CNN on 32x32x3 synthetic images (reduced batch here; the full
batch is checked against stored digests in test_gpu_fullsize).
"""
import numpy as np
import pytest

import oracle
from oracle.model import OracleNet
from paper_2009_13108_amd import inputs as I
from paper_2009_13108_amd import model as M
from paper_2009_13108_amd import niti
from helpers import dev, host, kcrs, krsc, nchw, nhwc, pad_channels, say

pytestmark = pytest.mark.gpu


def _i8(v):
    import torch
    return torch.tensor([int(v)], dtype=torch.int8, device="cuda")


def test_config1_fc_layer_fwd_bwd_update():
    import torch
    say("config1 fc 784->128 b32")
    B, K, N = 32, 784, 128
    x = I.activations(I.base_seed(1, 1), (B, K))
    w = I.weights(I.base_seed(1, 2), (N, K))
    e = I.errors5(I.base_seed(1, 3), (B, N))
    y_o, _, st_f = oracle.gemm_fwd(x, w)
    d = oracle.conv_desc(B, K, 1, 1, N, 1, 1, 1, 0)
    dx_o, _, st_d = oracle.conv_bwd_data(d, e.reshape(B, N, 1, 1), w.reshape(N, K, 1, 1))
    w_o, g_o, st_w = oracle.conv_bwd_weight(d, x.reshape(B, K, 1, 1), e.reshape(B, N, 1, 1),
                                            w.reshape(N, K, 1, 1), mu=5)
    gd = niti.ConvDesc.make(B, 1, 1, K, N, 1, 1, 1, 0)
    stats = niti.new_stats(3)
    xd, wd, ed = dev(x), dev(w), dev(e)
    y = torch.empty((B, N), dtype=torch.int8, device="cuda")
    sy = _i8(0)
    niti.gemm_fwd(xd, wd, y, stats, _i8(-7), _i8(-7), sy, stats_index=0)
    dx = torch.empty((B, 1, 1, K), dtype=torch.int8, device="cuda")
    ws = niti.new_workspace(max(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, gd),
                                niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, gd)))
    niti.conv_bwd_data(gd, ed.view(B, 1, 1, N), wd.view(N, 1, 1, K), dx, stats, ws, stats_index=1)
    g32 = torch.empty((N, 1, 1, K), dtype=torch.int32, device="cuda")
    niti.conv_bwd_weight(gd, xd.view(B, 1, 1, K), ed.view(B, 1, 1, N), wd.view(N, 1, 1, K), stats,
                         g32_out=g32, mu=5, stats_index=2)
    torch.cuda.synchronize()
    st = niti.read_stats(stats)
    assert (host(y) == y_o).all() and int(host(sy)[0]) == -14 + st_f["bp"]
    assert (host(dx).reshape(B, K) == dx_o.reshape(B, K)).all()
    assert (host(g32).reshape(N, K) == g_o.reshape(N, K)).all()
    assert (host(wd) == w_o.reshape(N, K)).all()
    for g, o in zip(st, (st_f, st_d, st_w)):
        assert g["max_abs"] == o["max_abs"] and g["bp"] == o["bp"]


def _mlp_setup(batch, cfg=2):
    px = I.pixels(I.base_seed(cfg, 1), (batch, 1, 28, 28))
    labels = I.labels(I.base_seed(cfg, 2), batch, 10)
    ws, exps = [], []
    for i, sp in enumerate(M.MLP_784):
        ws.append(I.weights(I.base_seed(cfg, 10 + i), (sp[2], sp[1])))
        exps.append(I.weight_exponent(sp[1]))
    return px, labels, ws, exps


@pytest.mark.parametrize("batch,steps", [(256, 3), (5, 2)])
def test_config2_mlp_training_steps(batch, steps):
    import torch
    say("config2 mlp", batch, steps)
    px, labels, ws, exps = _mlp_setup(batch)
    onet = OracleNet(M.MLP_784, (1, 28, 28), batch, ws, exps)
    gnet = M.IntNet(M.MLP_784, (28, 28, 1), batch, ws, exps)
    x_o = oracle.quantize_u8(px)
    x_g = torch.empty((batch, 28, 28, 1), dtype=torch.int8, device="cuda")
    niti.quantize_u8(dev(px), x_g)
    lab = dev(labels)
    s0 = _i8(-7)
    for step in range(steps):
        lo, so = onet.step(x_o, -7, labels)
        lg, sg = gnet.step(x_g, s0, lab)
        torch.cuda.synchronize()
        assert (host(lg).reshape(batch, -1) == lo).all(), "logits step %d" % step
        assert int(host(sg)[0]) == so, "exponent step %d" % step
        for li, (wg, wo) in enumerate(zip(gnet.weights(), onet.w)):
            assert (host(wg) == wo).all(), "weights layer %d step %d" % (li, step)


def _vgg_setup(batch, cfg=3):
    px = I.pixels(I.base_seed(cfg, 1), (batch, 3, 32, 32))
    labels = I.labels(I.base_seed(cfg, 2), batch, 10)
    w_orc, w_gpu, exps = [], [], []
    wi = 0
    c_prev, hw = 3, 32
    for sp in M.VGG_32:
        if sp[0] == "conv":
            cin = 3 if wi == 0 else sp[1]
            w = I.weights(I.base_seed(cfg, 10 + wi), (sp[2], cin, sp[3], sp[3]))
            w_orc.append(w)
            w_gpu.append(krsc(pad_channels(w, sp[1])))
            exps.append(I.weight_exponent(cin * sp[3] * sp[3]))
            c_prev = sp[2]
            wi += 1
        elif sp[0] == "pool":
            hw //= 2
        else:
            w = I.weights(I.base_seed(cfg, 10 + wi), (sp[2], sp[1]))  # drawn as [out][(c,h,w)]
            w_hwc = np.ascontiguousarray(w.reshape(sp[2], c_prev, hw, hw).transpose(0, 2, 3, 1).reshape(sp[2], -1))
            w_orc.append(w_hwc)         # both sides read the flattened input in (h, w, c) order
            w_gpu.append(w_hwc.copy())
            exps.append(I.weight_exponent(sp[1]))
            wi += 1
    return px, labels, w_orc, w_gpu, exps


def _vgg_orc_specs():
    specs = list(M.VGG_32)
    specs[0] = ("conv", 3) + specs[0][2:]
    return specs


@pytest.mark.parametrize("batch,steps", [(8, 2), (3, 1)])
def test_config3_vgg_training_steps(batch, steps):
    import torch
    say("config3 vgg", batch, steps)
    px, labels, w_orc, w_gpu, exps = _vgg_setup(batch)
    onet = OracleNet(_vgg_orc_specs(), (3, 32, 32), batch, w_orc, exps)
    gnet = M.IntNet(M.VGG_32, (32, 32, 4), batch, w_gpu, exps)
    x_o = oracle.quantize_u8(px)
    x_g = torch.empty((batch, 32, 32, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(dev(px), x_g)
    lab = dev(labels)
    s0 = _i8(-7)
    for step in range(steps):
        lo, so = onet.step(x_o, -7, labels)
        lg, sg = gnet.step(x_g, s0, lab)
        torch.cuda.synchronize()
        assert (host(lg).reshape(batch, -1) == lo).all(), "logits step %d" % step
        assert int(host(sg)[0]) == so
        gw = [host(t) for t in gnet.weights()]
        for li in range(6):
            assert (kcrs(gw[li])[:, :w_orc[li].shape[1]] == onet.w[li]).all(), "conv %d step %d" % (li, step)
        assert (kcrs(gw[0])[:, 3] == 0).all()
        assert (gw[6] == onet.w[6]).all(), "fc step %d" % step


def test_graph_replay_matches_eager():
    """A training step captured as a HIP graph and replayed matches eager
    steps call for call: two nets start from the same weights; each round
    runs one eager step on one and one replay on the other (with eager work
    and synchronizations between replays), then compares weights and logits."""
    import torch
    batch = 8
    say("graph replay vgg", batch)
    px, labels, w_orc, w_gpu, exps = _vgg_setup(batch)
    eager = M.IntNet(M.VGG_32, (32, 32, 4), batch, [w.copy() for w in w_gpu], exps, streams=1)
    graphed = M.IntNet(M.VGG_32, (32, 32, 4), batch, [w.copy() for w in w_gpu], exps, streams=1)
    x = torch.empty((batch, 32, 32, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(dev(px), x)
    lab = dev(labels)
    s0 = _i8(-7)
    # one eager step on both (first calls set up kernel attributes and guesses)
    eager.step(x, s0, lab)
    graphed.step(x, s0, lab)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=cap):
        lg, sg = graphed.step(x, s0, lab)
    torch.cuda.synchronize()
    for rnd in range(3):
        le, se = eager.step(x, s0, lab)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert (host(lg) == host(le)).all(), "logits round %d" % rnd
        assert int(host(sg)[0]) == int(host(se)[0])
        for a, b in zip(graphed.weights(), eager.weights()):
            assert (host(a) == host(b)).all(), "weights round %d" % rnd
