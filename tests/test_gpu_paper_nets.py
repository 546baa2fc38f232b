"""The paper's own networks (Section 4, Tables 5 and 6) trained step by step
on the GPU against the oracle's composition, byte for byte: LeNet-5 on
28x28x1 inputs and VGG-small-7/8/9 (with dropout before the classifier) on
32x32x3 inputs, synthetic images and labels of the datasets' shapes.  Cases
cover the paper's default rounding (a, e: nearest; g: pseudo stochastic),
the m_u schedule 5 -> 4 -> 3, pseudo stochastic rounding everywhere and
stochastic rounding for the gradients.  Image channels are padded with zeros
to 4 on both sides (and LeNet-5's six first filters to eight, two held at
zero), so that the stochastic draws, keyed by storage offset, agree."""
import numpy as np
import pytest

import oracle
from oracle.model import OracleNet
from paper_2009_13108_amd import inputs as I
from paper_2009_13108_amd import model as M
from paper_2009_13108_amd import niti
from helpers import dev, host, kcrs, nchw, nhwc, say

pytestmark = pytest.mark.gpu


def _orc_specs(specs):
    return [("conv",) + tuple(sp[1:]) if sp[0] == "conv" else sp for sp in specs]


def _setup(specs, hw, img_c, batch, cfg):
    """Seeded pixels, labels and weights of a network in both layouts."""
    px = I.pixels(I.base_seed(cfg, 1), (batch, img_c, hw, hw))
    labels = I.labels(I.base_seed(cfg, 2), batch, 10)
    zf = M.LENET5_REAL["zero_filters"] if specs is M.LENET5 else None
    w_gpu, exps = M.synthetic_weights(specs, 4, cfg, image_channels=img_c, zero_filters=zf)
    w_orc = [kcrs(w) if w.ndim == 4 else w.copy() for w in w_gpu]
    x_orc = np.zeros((batch, 4, hw, hw), np.int8)
    x_orc[:, :img_c] = oracle.quantize_u8(px)
    return px, labels, w_gpu, w_orc, exps, x_orc


CASES = [
    # name, specs, image size, image channels, batch, steps (mu per step), mode, grad mode
    ("lenet5_psr", M.LENET5, 28, 1, 16, (3, 3), oracle.PSR, oracle.PSR),
    ("lenet5_paper_rounding", M.LENET5, 28, 1, 16, (3, 3, 3), oracle.RTN, oracle.PSR),
    ("lenet5_sr_g", M.LENET5, 28, 1, 8, (3, 3), oracle.RTN, oracle.SR),
    ("vgg_small7_psr", M.vgg_small(7), 32, 3, 4, (5, 5), oracle.PSR, oracle.PSR),
    ("vgg_small7_schedule", M.vgg_small(7), 32, 3, 4, (5, 4, 3), oracle.RTN, oracle.PSR),
    ("vgg_small7_sr", M.vgg_small(7), 32, 3, 2, (5, 4), oracle.SR, oracle.SR),
    ("vgg_small8", M.vgg_small(8), 32, 3, 2, (5,), oracle.RTN, oracle.PSR),
    ("vgg_small9", M.vgg_small(9), 32, 3, 2, (5,), oracle.RTN, oracle.PSR),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_paper_network_training_steps(case):
    import torch
    name, specs, hw, img_c, batch, mus, mode, gmode = case
    say("paper net", name, batch, mus)
    cfg = 20 + CASES.index(case)
    px, labels, w_gpu, w_orc, exps, x_orc = _setup(specs, hw, img_c, batch, cfg)
    seed, dseed = 1000 + cfg, 2000 + cfg
    onet = OracleNet(_orc_specs(specs), (4, hw, hw), batch, w_orc, exps, mode=mode, grad_mode=gmode, sr_seed=seed,
                     drop_seed=dseed)
    gnet = M.IntNet(specs, (hw, hw, 4), batch, w_gpu, exps, mode=mode, grad_mode=gmode, sr_seed=seed,
                    drop_seed=dseed)
    x_g = torch.empty((batch, hw, hw, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(dev(px), x_g)
    assert (nchw(host(x_g)) == x_orc).all()
    lab = dev(labels)
    s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")
    w0 = [w.copy() for w in w_gpu]
    for step, mu in enumerate(mus):
        lo, so = onet.step(x_orc, -7, labels, mu=mu)
        lg, sg = gnet.step(x_g, s0, lab, mu=mu)
        torch.cuda.synchronize()
        assert (host(lg).reshape(batch, -1) == lo).all(), "logits step %d" % step
        assert int(host(sg)[0]) == so, "exponent step %d" % step
        for li, (wg, wo) in enumerate(zip(gnet.weights(), onet.w)):
            got = host(wg)
            assert ((kcrs(got) if got.ndim == 4 else got) == wo).all(), "weights layer %d step %d" % (li, step)
    moved = [not (host(a) == b).all() for a, b in zip(gnet.weights(), w0)]
    assert any(moved)
    if specs is M.LENET5:
        got = [host(w) for w in gnet.weights()]
        assert not got[0][6:].any() and not got[1][..., 6:].any()    # the padding filters stay zero


@pytest.mark.parametrize("name", ["lenet5", "vgg_small7"])
def test_two_streams_equal_one_stream(name):
    """The step with the weight gradients on a second stream leaves exactly
    the logits, exponents and weights of the single-stream step (every
    call in Algorithm 1's order), step after step."""
    import torch
    specs, hw, img_c, batch = (M.LENET5, 28, 1, 16) if name == "lenet5" else (M.vgg_small(7), 32, 3, 8)
    say("streams", name, batch)
    px, labels, w_gpu, _, exps, _ = _setup(specs, hw, img_c, batch, 70)
    nets = [M.IntNet(specs, (hw, hw, 4), batch, [w.copy() for w in w_gpu], exps, drop_seed=5, streams=k)
            for k in (1, 2)]
    x = torch.empty((batch, hw, hw, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(dev(px), x)
    lab = dev(labels)
    s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")
    for step in range(3):
        out = [net.step(x, s0, lab) for net in nets]
        torch.cuda.synchronize()
        assert (host(out[0][0]) == host(out[1][0])).all(), "logits step %d" % step
        assert int(host(out[0][1])[0]) == int(host(out[1][1])[0])
        for a, b in zip(nets[0].weights(), nets[1].weights()):
            assert (host(a) == host(b)).all(), "weights step %d" % step


ALEX = [(n, ci, co, k, st, pd, hw, 2) for (n, ci, co, k, st, pd, hw) in M.ALEXNET_LAYERS]
ALEX += [(n, fi, fo, 1, 1, 0, 1, 4) for (n, fi, fo) in M.ALEXNET_FC]


@pytest.mark.parametrize("layer", ALEX, ids=[a[0] for a in ALEX])
def test_alexnet_layer_shapes(layer):
    """AlexNet's contraction shapes (Table 6's network), each layer's three
    contractions with their fused epilogues, element by element and with the
    statistics, at a small batch; weights and errors with the first layer's
    padding channel held at zero."""
    import torch
    from helpers import krsc, same_stats
    name, cin, cout, k, st, pd, hw, n = layer
    say("alexnet", name, n)
    seed = 300 + 10 * ALEX.index(layer)
    d = oracle.conv_desc(n, cin, hw, hw, cout, k, k, st, pd)
    P, Q = oracle.conv_out_hw(d)
    x = I.activations(seed + 1, (n, cin, hw, hw))
    wt = I.weights(seed + 2, (cout, cin, k, k))
    dy = I.errors8(seed + 3, (n, cout, P, Q))
    if cin == 4:
        x[:, 3:] = 0
        wt[:, 3:] = 0
    gd = niti.ConvDesc.make(n, hw, hw, cin, cout, k, k, st, pd)
    ws = niti.new_workspace(max(niti.workspace_bytes(op, gd) for op in (1, 2, 3)))
    stats = niti.new_stats(3)
    xs, wd, dyd = dev(nhwc(x)), dev(krsc(wt)), dev(nhwc(dy))
    # forward
    y_o, _, st_f = oracle.conv_fwd(d, x, wt, relu=True)
    y = torch.empty(gd.y_shape(), dtype=torch.int8, device="cuda")
    niti.conv_fwd(gd, xs, wd, y, stats, relu=True, ws=ws, stats_index=0)
    # back-propagation, masked by the ReLU of the layer below (not formed
    # for the stride-4 first layer: the library rejects it)
    dx = torch.empty(gd.x_shape(), dtype=torch.int8, device="cuda")
    if st > 2:
        with pytest.raises(niti.NitiError) as ei:
            niti.conv_bwd_data(gd, dyd, wd, dx, stats, ws, relu_src=xs, stats_index=1)
        assert ei.value.status == -3
    else:
        dx_o, _, st_d = oracle.conv_bwd_data(d, dy, wt, relu_src=x)
        niti.conv_bwd_data(gd, dyd, wd, dx, stats, ws, relu_src=xs, stats_index=1)
    # weight gradient and update
    w_o, g_o, st_w = oracle.conv_bwd_weight(d, x, dy, wt, mu=5)
    g32 = torch.empty(gd.w_shape(), dtype=torch.int32, device="cuda")
    niti.conv_bwd_weight(gd, xs, dyd, wd, stats, ws, g32_out=g32, mu=5, stats_index=2)
    torch.cuda.synchronize()
    g = niti.read_stats(stats)
    assert (nchw(host(y)) == y_o).all() and same_stats(g[0], st_f)
    if st <= 2:
        assert (nchw(host(dx)) == dx_o).all() and same_stats(g[1], st_d)
    assert (kcrs(host(g32)) == g_o).all()
    assert (kcrs(host(wd)) == w_o).all() and same_stats(g[2], st_w)


FIT_CASES = [
    # name, specs, image size, image channels, m_u, steps, training accuracy required after them
    ("lenet5", M.LENET5, 28, 1, 3, 200, 0.95),
    ("vgg_small7", M.vgg_small(7), 32, 3, 5, 150, 0.75),
]


@pytest.mark.parametrize("case", FIT_CASES, ids=[c[0] for c in FIT_CASES])
def test_integer_training_fits_a_fixed_batch(case):
    """The method learns: the library alone (integer forward, loss,
    back-propagation and update; nearest rounding for activations and
    errors, pseudo stochastic for gradients, as in the paper's experiments;
    dropout on in VGG-small) trained on one fixed batch of 256 synthetic
    images with random labels drives the training accuracy (argmax of the
    int8 logits) from chance to near memorisation.  Every result is an
    integer, so the run is deterministic."""
    import torch
    name, specs, hw, img_c, mu, steps, need = case
    say("fit", name, steps)
    batch = 256
    zf = M.LENET5_REAL["zero_filters"] if specs is M.LENET5 else None
    ws, exps = M.synthetic_weights(specs, 4, 60, image_channels=img_c, zero_filters=zf)
    net = M.IntNet(specs, (hw, hw, 4), batch, ws, exps, mode=niti.RTN, grad_mode=niti.PSR, drop_seed=3)
    px = I.pixels(I.base_seed(61, 1), (batch, img_c, hw, hw), device="cuda")
    lab = I.labels(I.base_seed(61, 2), batch, 10, device="cuda")
    x = torch.empty((batch, hw, hw, 4), dtype=torch.int8, device="cuda")
    niti.quantize_u8(px, x)
    s0 = torch.tensor([-7], dtype=torch.int8, device="cuda")

    def accuracy(lg):
        return (lg.view(batch, -1).float().argmax(1) == lab.long()).float().mean().item()

    lg, _ = net.step(x, s0, lab, mu=mu)
    torch.cuda.synchronize()
    first = accuracy(lg)
    for _ in range(steps - 1):
        lg, _ = net.step(x, s0, lab, mu=mu)
    torch.cuda.synchronize()
    last = accuracy(lg)
    say("fit", name, "accuracy", first, "->", last)
    assert first < 0.2 and last >= need, (first, last)
