"""Full-size parity: the configurations at their real sizes, in the launch
configuration bench.py times, against oracle digests.

The digests in tests/golden/fullsize_*.json were written by
tests/golden/make_fullsize.py, which calls only the oracle and the input
generator.  Here the same inputs are regenerated on the device (the torch
path of the generator gives the same bytes as its numpy path,
tests/test_inputs.py), the library computes each result through its C ABI,
and the SHA-256 of the whole result must equal the oracle's.  Every call is
made twice: once with a fresh statistics block (no usable guess of the
rounding shift) and once reusing it (the guess path).
"""
import hashlib
import json
import os

import numpy as np
import pytest

from paper_2009_13108_amd import inputs as I
from paper_2009_13108_amd import model as M
from paper_2009_13108_amd import niti
from helpers import say

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    path = os.path.join(GOLD, name)
    if not os.path.exists(path):
        pytest.skip("%s not generated" % name)
    with open(path) as f:
        return json.load(f)["cases"]


def sha(t):
    return hashlib.sha256(t.detach().contiguous().cpu().numpy().tobytes()).hexdigest()


def _stats_ok(g, rec):
    return all(int(g[k]) == int(rec[k]) for k in ("max_abs", "b", "bp"))


# ---------------------------------------------------------------- config 5
def _c5_cases():
    path = os.path.join(GOLD, "fullsize_c5.json")
    if not os.path.exists(path):
        return []
    with open(path) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("rec", _c5_cases(), ids=lambda r: "%dx%dx%d-%s" % (r["M"], r["N"], r["K"], r["dist"]))
def test_gemm_sweep_fullsize(rec):
    import torch
    M_, N_, K_, dist = rec["M"], rec["N"], rec["K"], rec["dist"]
    say("c5 gemm", M_, N_, K_, dist)
    gen = I.weights if dist == "w" else I.errors5
    off = 0 if dist == "w" else 10
    A = gen(I.base_seed(5, 1 + off), (M_, K_), device="cuda")
    B = gen(I.base_seed(5, 2 + off), (N_, K_), device="cuda")
    C = torch.empty((M_, N_), dtype=torch.int8, device="cuda")
    stats = niti.new_stats()
    for rep in range(2):
        niti.gemm_fwd(A, B, C, stats)
        torch.cuda.synchronize()
        g = niti.read_stats(stats)[0]
        assert _stats_ok(g, rec), (rep, g, rec)
        assert sha(C) == rec["sha256"], "rep %d" % rep
    del A, B, C
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- config 4
def _c4_layer_cases():
    path = os.path.join(GOLD, "fullsize_c4.json")
    if not os.path.exists(path):
        return []
    with open(path) as f:
        return [c for c in json.load(f)["cases"] if c["layer"] != "fc"]


@pytest.mark.parametrize("rec", _c4_layer_cases(), ids=lambda r: r["layer"])
def test_resnet18_layer_fullsize(rec):
    import torch
    li = rec["li"]
    name, cin, cout, k, st, pd, hw, count = M.RESNET18_LAYERS[li]
    say("c4 layer", name)
    B = 128
    d = niti.ConvDesc.make(B, hw, hw, cin, cout, k, k, st, pd)
    x = I.activations(I.base_seed(4, 100 + li), d.x_shape(), device="cuda")
    dy = I.errors8(I.base_seed(4, 200 + li), d.y_shape(), device="cuda")
    w0 = I.weights(I.base_seed(4, 1000 + 10 * li), d.w_shape(), device="cuda")
    if name.startswith("stem"):
        x[..., 3:] = 0
        w0[..., 3:] = 0
    stats = niti.new_stats(3)
    y = torch.empty(d.y_shape(), dtype=torch.int8, device="cuda")
    dx = torch.empty(d.x_shape(), dtype=torch.int8, device="cuda")
    g32 = torch.empty(d.w_shape(), dtype=torch.int32, device="cuda")
    ws = niti.new_workspace(max(niti.workspace_bytes(niti.OP_CONV_FWD, d),
                                niti.workspace_bytes(niti.OP_CONV_BWD_DATA, d),
                                niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, d)))
    for rep in range(2):
        niti.conv_fwd(d, x, w0, y, stats, relu=True, stats_index=0, ws=ws)
        if "bwd_data" in rec:
            niti.conv_bwd_data(d, dy, w0, dx, stats, ws, relu_src=x, stats_index=1)
        w = w0.clone()
        niti.conv_bwd_weight(d, x, dy, w, stats, ws, g32_out=g32, mu=5, stats_index=2)
        torch.cuda.synchronize()
        g = niti.read_stats(stats)
        assert _stats_ok(g[0], rec["fwd"]) and sha(y) == rec["fwd"]["sha256"], ("fwd", rep)
        if "bwd_data" in rec:
            assert _stats_ok(g[1], rec["bwd_data"]) and sha(dx) == rec["bwd_data"]["sha256"], ("dgrad", rep)
        assert sha(g32) == rec["bwd_weight"]["sha256_g32"], ("g32", rep)
        assert _stats_ok(g[2], rec["bwd_weight"]) and sha(w) == rec["bwd_weight"]["sha256_w"], ("update", rep)


def test_resnet18_bordered_image_layer_fullsize():
    """The image layer as bench.py runs it: the batch stored with its 3-pixel
    zero border (230 x 230) and a descriptor without padding, read in place.
    The forward output and the weight gradient and update must be the
    oracle's digests of the padded 224 x 224 layer."""
    import torch
    recs = [c for c in _c4_layer_cases() if c["layer"].startswith("stem")]
    if not recs:
        pytest.skip("fullsize_c4.json not generated")
    rec = recs[0]
    li = rec["li"]
    name, cin, cout, k, st, pd, hw, count = M.RESNET18_LAYERS[li]
    say("c4 bordered image layer", name)
    B = 128
    dp = niti.ConvDesc.make(B, hw, hw, cin, cout, k, k, st, pd)
    x = I.activations(I.base_seed(4, 100 + li), dp.x_shape(), device="cuda")
    dy = I.errors8(I.base_seed(4, 200 + li), dp.y_shape(), device="cuda")
    w = I.weights(I.base_seed(4, 1000 + 10 * li), dp.w_shape(), device="cuda")
    x[..., 3:] = 0
    w[..., 3:] = 0
    hb = hw + 2 * pd
    xb = torch.zeros((B, hb, hb, cin), dtype=torch.int8, device="cuda")
    xb[:, pd:pd + hw, pd:pd + hw] = x
    del x
    d = niti.ConvDesc.make(B, hb, hb, cin, cout, k, k, st, 0)
    assert d.y_shape() == dp.y_shape()
    stats = niti.new_stats(3)
    y = torch.empty(d.y_shape(), dtype=torch.int8, device="cuda")
    g32 = torch.empty(d.w_shape(), dtype=torch.int32, device="cuda")
    ws = niti.new_workspace(max(niti.workspace_bytes(niti.OP_CONV_FWD, d),
                                niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, d)))
    niti.conv_fwd(d, xb, w, y, stats, relu=True, stats_index=0, ws=ws)
    niti.conv_bwd_weight(d, xb, dy, w, stats, ws, g32_out=g32, mu=5, stats_index=2)
    torch.cuda.synchronize()
    g = niti.read_stats(stats)
    assert _stats_ok(g[0], rec["fwd"]) and sha(y) == rec["fwd"]["sha256"]
    assert sha(g32) == rec["bwd_weight"]["sha256_g32"]
    assert _stats_ok(g[2], rec["bwd_weight"]) and sha(w) == rec["bwd_weight"]["sha256_w"]


def test_resnet18_head_and_loss_fullsize():
    import torch
    cases = [c for c in _load("fullsize_c4.json") if c["layer"] == "fc"]
    rec = cases[0]
    say("c4 head")
    B = 128
    fin, fout = M.RESNET18_FC
    feat = I.activations(I.base_seed(4, 300), (B, fin), device="cuda")
    wfc0 = I.weights(I.base_seed(4, 301), (fout, fin), device="cuda")
    lab = I.labels(I.base_seed(4, 302), B, fout, device="cuda")
    i8 = lambda v: torch.tensor([v], dtype=torch.int8, device="cuda")
    s_feat, s_w, s_log = i8(-9), i8(-11), i8(0)
    logits = torch.empty((B, fout), dtype=torch.int8, device="cuda")
    err = torch.empty_like(logits)
    dfeat = torch.empty((B, fin), dtype=torch.int8, device="cuda")
    g32 = torch.empty((fout, fin), dtype=torch.int32, device="cuda")
    fd = niti.ConvDesc.make(B, 1, 1, fin, fout, 1, 1, 1, 0)
    ws = niti.new_workspace(max(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, fd),
                                niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, fd),
                                niti.workspace_bytes(niti.OP_INT_CE_LOSS, None, B, fout)))
    stats = niti.new_stats(4)
    for rep in range(2):
        niti.gemm_fwd(feat, wfc0, logits, stats, s_feat, s_w, s_log, stats_index=0)
        niti.int_ce_loss_grad(logits, s_log, lab, err, stats, ws, stats_index=1)
        niti.conv_bwd_data(fd, err.view(B, 1, 1, fout), wfc0.view(fout, 1, 1, fin), dfeat.view(B, 1, 1, fin),
                           stats, ws, relu_src=feat.view(B, 1, 1, fin), stats_index=2)
        w = wfc0.clone()
        niti.conv_bwd_weight(fd, feat.view(B, 1, 1, fin), err.view(B, 1, 1, fout), w.view(fout, 1, 1, fin), stats,
                             ws, g32_out=g32.view(fout, 1, 1, fin), mu=5, stats_index=3)
        torch.cuda.synchronize()
        g = niti.read_stats(stats)
        assert int(s_log.cpu()[0]) == rec["s_logits"]
        assert _stats_ok(g[0], rec["fwd"]) and sha(logits) == rec["fwd"]["sha256"]
        assert _stats_ok(g[1], rec["loss"]) and sha(err) == rec["loss"]["sha256"]
        assert _stats_ok(g[2], rec["bwd_data"]) and sha(dfeat) == rec["bwd_data"]["sha256"]
        assert sha(g32) == rec["bwd_weight"]["sha256_g32"]
        assert _stats_ok(g[3], rec["bwd_weight"]) and sha(w) == rec["bwd_weight"]["sha256_w"]


# ---------------------------------------------------------------- config 3
def test_vgg_full_batch_step():
    import torch
    path = os.path.join(GOLD, "fullsize_c3.json")
    if not os.path.exists(path):
        pytest.skip("fullsize_c3.json not generated")
    rec = json.load(open(path))["cases"]
    say("c3 vgg batch", rec["batch"])
    batch = rec["batch"]
    px = I.pixels(I.base_seed(3, 1), (batch, 3, 32, 32), device="cuda")
    labels = I.labels(I.base_seed(3, 2), batch, 10, device="cuda")
    w_gpu, exps = [], []
    wi, c_prev, hw = 0, 3, 32
    for sp in M.VGG_32:
        if sp[0] == "conv":
            cin = 3 if wi == 0 else sp[1]
            w = I.weights(I.base_seed(3, 10 + wi), (sp[2], cin, sp[3], sp[3]))
            if wi == 0:
                w = np.concatenate([w, np.zeros((sp[2], 1, sp[3], sp[3]), np.int8)], axis=1)
            w_gpu.append(np.ascontiguousarray(w.transpose(0, 2, 3, 1)))
            exps.append(I.weight_exponent(cin * sp[3] * sp[3]))
            c_prev = sp[2]
            wi += 1
        elif sp[0] == "pool":
            hw //= 2
        else:
            w = I.weights(I.base_seed(3, 10 + wi), (sp[2], sp[1]))
            w_gpu.append(np.ascontiguousarray(
                w.reshape(sp[2], c_prev, hw, hw).transpose(0, 2, 3, 1).reshape(sp[2], -1)))
            exps.append(I.weight_exponent(sp[1]))
            wi += 1
    net = M.IntNet(M.VGG_32, (32, 32, 4), batch, w_gpu, exps)
    x = torch.empty((batch, 32, 32, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(px, x)
    s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")
    logits, s = net.step(x, s0, labels)
    torch.cuda.synchronize()
    assert sha(logits.reshape(batch, -1)) == rec["logits_sha256"]
    assert int(s.cpu()[0]) == rec["s_logits"]
    for li, w in enumerate(net.weights()):
        assert sha(w) == rec["weights_sha256"][li], "layer %d" % li


NETS = [("lenet5", M.LENET5, 28, 1, M.LENET5_REAL["zero_filters"])]
NETS += [("vgg_small%d" % d, M.vgg_small(d), 32, 3, None) for d in (7, 8, 9)]


@pytest.mark.parametrize("net", NETS, ids=[n[0] for n in NETS])
def test_paper_network_full_batch_steps(net):
    """LeNet-5 and VGG-small-7/8/9 (Section 4, Table 5) trained at batch 256
    exactly as bench.py times them (same seeds and rounding; dropout on in
    VGG-small): every step's logits and exponent, and every layer's weights
    after the last step, against the oracle's digests."""
    import torch
    name, specs, hw, img_c, zf = net
    recs = [r for r in _load("fullsize_nets.json") if r["net"] == name]
    if not recs:
        pytest.skip("no digest for %s" % name)
    rec = recs[0]
    batch, cfg = rec["batch"], rec["seed"]
    say("paper net full batch", name, batch, len(rec["steps"]))
    ws, exps = M.synthetic_weights(specs, 4, cfg, image_channels=img_c, zero_filters=zf)
    gnet = M.IntNet(specs, (hw, hw, 4), batch, ws, exps, drop_seed=cfg)
    px = I.pixels(I.base_seed(cfg, 1), (batch, img_c, hw, hw), device="cuda")
    lab = I.labels(I.base_seed(cfg, 2), batch, 10, device="cuda")
    x = torch.empty((batch, hw, hw, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(px, x)
    s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")
    for i, want in enumerate(rec["steps"]):
        lg, s = gnet.step(x, s0, lab)
        torch.cuda.synchronize()
        assert sha(lg.reshape(batch, -1)) == want["logits_sha256"], "logits step %d" % i
        assert int(s.cpu()[0]) == want["s_logits"], "exponent step %d" % i
    for li, w in enumerate(gnet.weights()):
        assert sha(w) == rec["weights_sha256"][li], "weights layer %d" % li
