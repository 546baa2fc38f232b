"""GPU parity of the cases the main parity file does not reach: round to
nearest through every rounding site (forward, back-propagation, weight
update, loss), and int32 accumulators that wrap (exact sums beyond 2^31,
kept mod 2^32 by the method's int32 accumulation)."""
import numpy as np
import pytest

import oracle
from paper_2009_13108_amd import inputs as I
from paper_2009_13108_amd import niti
from helpers import dev, host, kcrs, krsc, nchw, nhwc, say, same_stats

pytestmark = pytest.mark.gpu


def _i8(v):
    import torch
    return torch.tensor([v], dtype=torch.int8, device="cuda")


RTN_CONV_CASES = [
    # n, c, h, w, k, r, s, stride, pad, relu
    (2, 64, 14, 14, 64, 3, 3, 1, 1, True),      # weight-resident forward
    (5, 64, 13, 11, 64, 3, 3, 1, 1, False),
    (1, 4, 32, 32, 64, 7, 7, 2, 3, True),       # image layer: padded copy, windows
    (2, 12, 9, 9, 16, 3, 3, 1, 1, True),
    (2, 128, 13, 13, 256, 3, 3, 2, 1, True),    # ring (DMA) kernel, strided classes
    (2, 256, 7, 7, 256, 3, 3, 1, 1, False),
    (2, 64, 14, 14, 128, 1, 1, 2, 0, True),     # strided 1x1
    (4, 128, 7, 7, 130, 3, 3, 1, 1, False),     # general kernel
    (128, 512, 1, 1, 1000, 1, 1, 1, 0, True),   # classifier head
]


def _conv_inputs(case, seed):
    n, c, h, w, k, r, s, st, pd, relu = case
    d = oracle.conv_desc(n, c, h, w, k, r, s, st, pd)
    P, Q = oracle.conv_out_hw(d)
    x = I.activations(seed + 1, (n, c, h, w))
    wt = I.weights(seed + 2, (k, c, r, s))
    dy = I.errors8(seed + 3, (n, k, P, Q))
    gd = niti.ConvDesc.make(n, h, w, c, k, r, s, st, pd)
    return d, gd, x, wt, dy


@pytest.mark.parametrize("case", RTN_CONV_CASES)
def test_conv_passes_round_to_nearest(case):
    import torch
    say("rtn conv", case)
    RTN = oracle.RTN
    d, gd, x, wt, dy = _conv_inputs(case, 9000 + case[1] + 3 * case[4])
    relu = case[-1]
    stats = niti.new_stats(3)
    # forward (twice: the second call runs on the speculated shift)
    exp_y, _, st = oracle.conv_fwd(d, x, wt, relu=relu, mode=RTN)
    y = torch.empty(gd.y_shape(), dtype=torch.int8, device="cuda")
    nws = niti.workspace_bytes(niti.OP_CONV_FWD, gd)
    ws = niti.new_workspace(nws) if nws else None
    for rep in range(2):
        niti.conv_fwd(gd, dev(nhwc(x)), dev(krsc(wt)), y, stats, relu=relu, mode=niti.RTN, ws=ws, stats_index=0)
        torch.cuda.synchronize()
        assert (nchw(host(y)) == exp_y).all(), rep
        assert same_stats(niti.read_stats(stats)[0], st)
    # back-propagation with the backward ReLU mask
    relu_src = I.weights(9100 + case[1], (d.n, d.c, d.h, d.w))
    exp_dx, _, st = oracle.conv_bwd_data(d, dy, wt, mode=RTN, relu_src=relu_src)
    dx = torch.empty(gd.x_shape(), dtype=torch.int8, device="cuda")
    wsd = niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, gd))
    for rep in range(2):
        niti.conv_bwd_data(gd, dev(nhwc(dy)), dev(krsc(wt)), dx, stats, wsd, relu_src=dev(nhwc(relu_src)),
                           mode=niti.RTN, stats_index=1)
        torch.cuda.synchronize()
        assert (nchw(host(dx)) == exp_dx).all(), rep
        assert same_stats(niti.read_stats(stats)[1], st)
    # weight gradient and update
    for mu in (5, 2):
        exp_w, exp_g, st = oracle.conv_bwd_weight(d, x, dy, wt, mu=mu, mode=RTN)
        w_dev = dev(krsc(wt))
        g32 = torch.empty(gd.w_shape(), dtype=torch.int32, device="cuda")
        wsw = niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, gd))
        niti.conv_bwd_weight(gd, dev(nhwc(x)), dev(nhwc(dy)), w_dev, stats, wsw, g32_out=g32, mu=mu,
                             mode=niti.RTN, stats_index=2)
        torch.cuda.synchronize()
        assert (kcrs(host(g32)) == exp_g).all()
        assert (kcrs(host(w_dev)) == exp_w).all(), mu
        assert same_stats(niti.read_stats(stats)[2], st)


@pytest.mark.parametrize("n,mu", [(1, 5), (1003, 6), (36864, 3), (4194309, 1)])
def test_sgd_update_round_to_nearest(n, mu):
    import torch
    say("rtn sgd_update", n, mu)
    w = I.weights(7100 + n, (n,))
    g32 = I.uniform_int(7200 + n, (n,), -(1 << 26), 1 << 26, dtype=np.int32)
    exp_w, st = oracle.sgd_update(w, g32, mu, oracle.RTN)
    wd = dev(w)
    stats = niti.new_stats()
    niti.sgd_update(wd, dev(g32), stats, mu, mode=niti.RTN)
    torch.cuda.synchronize()
    assert (host(wd) == exp_w).all() and same_stats(niti.read_stats(stats)[0], st)


# ---------------------------------------------------------------- int32 wrap
def _wrap_operands(M, N, K, seed):
    """+-127 operands whose exact dot products spread over +-K 127^2, so
    that many of them leave the int32 range (K 127^2 > 2^31)."""
    rng = np.random.default_rng(seed)
    A = np.full((M, K), 127, np.int8)
    B = np.full((N, K), 127, np.int8)
    for m in range(M):
        A[m, :int(rng.integers(0, K // 2))] = -127
    for j in range(N):
        B[j, K - int(rng.integers(0, K // 2)):] = -127
    return A, B


@pytest.mark.parametrize("M,N,relu", [(48, 40, False), (48, 40, True), (1100, 64, False), (1500, 300, True)])
def test_gemm_accumulator_wraps_mod_2_32(M, N, relu):
    import torch
    K = 140000
    say("gemm wrap", M, N, K, relu)
    A, B = _wrap_operands(M, N, K, 5000 + M + N)
    S = oracle.gemm_nt_exact(A, B, block_rows=64)
    assert np.abs(S).max() >= 2 ** 31                  # the case really wraps
    exp_out, acc, st = oracle.finish(S, relu, 7, oracle.PSR, K)
    assert st["flags"] & oracle.FLAG_ACC_WRAP and st["flags"] & oracle.FLAG_ACC_BOUND
    C = torch.empty((M, N), dtype=torch.int8, device="cuda")
    stats = niti.new_stats()
    for rep in range(2):
        niti.gemm_fwd(dev(A), dev(B), C, stats, relu=relu)
        torch.cuda.synchronize()
        assert (host(C) == exp_out).all(), rep
        assert same_stats(niti.read_stats(stats)[0], st)


@pytest.mark.parametrize("case", [
    # n, c, h, w, k, r, s, stride, pad: npix >= 2^17, sums beyond 2^31
    (140000, 64, 1, 1, 64, 1, 1, 1, 0),         # fully-connected weight gradient over 140000 samples
    (33, 64, 64, 64, 64, 3, 3, 1, 1),           # 3x3 over 135168 pixels
])
def test_weight_gradient_wraps_mod_2_32(case):
    import torch
    say("wgrad wrap", case)
    n, c, h, w, k, r, s, stride, pd = case
    d = oracle.conv_desc(n, c, h, w, k, r, s, stride, pd)
    P, Q = oracle.conv_out_hw(d)
    assert n * P * Q >= oracle.ACC_BOUND_LEN
    # x = 127 everywhere except a few negative channels; dy = +-127 by output channel
    x = np.full((n, c, h, w), 127, np.int8)
    x[:, ::7] = -127
    dy = np.full((n, k, P, Q), 127, np.int8)
    dy[:, 1::3] = -127
    dy[: n // 3, 2::5] = 5
    wt = I.weights(5100, (k, c, r, s))
    exp_w, exp_g, st = oracle.conv_bwd_weight(d, x, dy, wt, mu=5)
    assert st["flags"] & oracle.FLAG_ACC_WRAP          # some exact sum left the int32 range
    gd = niti.ConvDesc.make(n, h, w, c, k, r, s, stride, pd)
    w_dev = dev(krsc(wt))
    g32 = torch.empty(gd.w_shape(), dtype=torch.int32, device="cuda")
    stats = niti.new_stats()
    ws = niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, gd))
    niti.conv_bwd_weight(gd, dev(nhwc(x)), dev(nhwc(dy)), w_dev, stats, ws, g32_out=g32, mu=5)
    torch.cuda.synchronize()
    assert (kcrs(host(g32)) == exp_g).all()
    assert (kcrs(host(w_dev)) == exp_w).all()
    assert same_stats(niti.read_stats(stats)[0], st)


# ---------------------------------------------------------------- stochastic rounding
SR_SEED = 0x5EED0F5A17
SR_CONV_CASES = [
    (2, 64, 14, 14, 64, 3, 3, 1, 1, True),
    (1, 4, 16, 16, 32, 7, 7, 2, 3, True),       # few channels (general kernel over the unpadded input)
    (2, 128, 13, 13, 256, 3, 3, 2, 1, False),   # strided back-propagation classes
    (2, 64, 14, 14, 128, 1, 1, 2, 0, True),     # strided 1x1 (tapless classes)
    (16, 512, 1, 1, 1000, 1, 1, 1, 0, True),    # classifier head
]


@pytest.mark.parametrize("case", SR_CONV_CASES)
def test_conv_passes_stochastic_rounding(case):
    """Two calls in a row on each stats block (call index 0, then 1: new
    draws, and the second call runs on the speculated shift)."""
    import torch
    say("sr conv", case)
    SR = oracle.SR
    d, gd, x, wt, dy = _conv_inputs(case, 9500 + case[1] + case[4])
    relu = case[-1]
    stats = niti.new_stats(3)
    niti.set_sr_seed(stats, SR_SEED)
    y = torch.empty(gd.y_shape(), dtype=torch.int8, device="cuda")
    nws = niti.workspace_bytes(niti.OP_CONV_FWD, gd)
    ws = niti.new_workspace(nws) if nws else None
    relu_src = I.weights(9600 + case[1], (d.n, d.c, d.h, d.w))
    dx = torch.empty(gd.x_shape(), dtype=torch.int8, device="cuda")
    wsd = niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_DATA, gd))
    wsw = niti.new_workspace(niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, gd))
    for call in range(2):
        exp_y, _, st = oracle.conv_fwd(d, x, wt, relu=relu, mode=SR, sr_seed=SR_SEED, sr_call=call)
        niti.conv_fwd(gd, dev(nhwc(x)), dev(krsc(wt)), y, stats, relu=relu, mode=niti.SR, ws=ws, stats_index=0)
        torch.cuda.synchronize()
        assert (nchw(host(y)) == exp_y).all(), call
        assert same_stats(niti.read_stats(stats)[0], st)
        exp_dx, _, st = oracle.conv_bwd_data(d, dy, wt, mode=SR, relu_src=relu_src, sr_seed=SR_SEED, sr_call=call)
        niti.conv_bwd_data(gd, dev(nhwc(dy)), dev(krsc(wt)), dx, stats, wsd, relu_src=dev(nhwc(relu_src)),
                           mode=niti.SR, stats_index=1)
        torch.cuda.synchronize()
        assert (nchw(host(dx)) == exp_dx).all(), call
        assert same_stats(niti.read_stats(stats)[1], st)
        exp_w, exp_g, st = oracle.conv_bwd_weight(d, x, dy, wt, mu=4, mode=SR, sr_seed=SR_SEED, sr_call=call)
        w_dev = dev(krsc(wt))
        niti.conv_bwd_weight(gd, dev(nhwc(x)), dev(nhwc(dy)), w_dev, stats, wsw, mu=4, mode=niti.SR, stats_index=2)
        torch.cuda.synchronize()
        assert (kcrs(host(w_dev)) == exp_w).all(), call
        assert same_stats(niti.read_stats(stats)[2], st)


@pytest.mark.parametrize("M,N,K,relu", [(300, 200, 784, True), (2000, 300, 512, False), (128, 1000, 512, False)])
def test_gemm_stochastic_rounding(M, N, K, relu):
    import torch
    say("sr gemm", M, N, K)
    A = I.activations(9700 + M, (M, K)); B = I.weights(9701 + N, (N, K))
    C = torch.empty((M, N), dtype=torch.int8, device="cuda")
    stats = niti.new_stats()
    niti.set_sr_seed(stats, SR_SEED + M)
    for call in range(2):
        exp, _, st = oracle.gemm_fwd(A, B, relu=relu, mode=oracle.SR, sr_seed=SR_SEED + M, sr_call=call)
        niti.gemm_fwd(dev(A), dev(B), C, stats, relu=relu, mode=niti.SR)
        torch.cuda.synchronize()
        assert (host(C) == exp).all(), call
        assert same_stats(niti.read_stats(stats)[0], st)


@pytest.mark.parametrize("n,mu", [(1, 5), (1003, 3), (4194309, 5)])
def test_sgd_update_and_round_stochastic(n, mu):
    import torch
    say("sr update/round", n, mu)
    w = I.weights(9800 + n, (n,))
    g32 = I.uniform_int(9801 + n, (n,), -(1 << 26), 1 << 26, dtype=np.int32)
    stats = niti.new_stats(3)
    niti.set_sr_seed(stats, 99)
    wd = dev(w)
    for call in range(2):
        exp_w, st = oracle.sgd_update(w if call == 0 else exp_prev, g32, mu, oracle.SR, sr_seed=99, sr_call=call)
        niti.sgd_update(wd, dev(g32), stats, mu, mode=niti.SR, stats_index=0)
        torch.cuda.synchronize()
        assert (host(wd) == exp_w).all(), call
        assert same_stats(niti.read_stats(stats)[0], st)
        exp_prev = exp_w
    # rounding with a derived binary point (counts calls), then a fixed one (does not)
    y = torch.empty(n, dtype=torch.int8, device="cuda")
    exp, st = oracle.shift_round(g32, 7, oracle.SR, sr_seed=99, sr_call=0)
    niti.round_psr(dev(g32), y, -1, 7, stats, mode=niti.SR, stats_index=1)
    torch.cuda.synchronize()
    assert (host(y) == exp).all() and same_stats(niti.read_stats(stats)[1], st)
    niti.round_psr(dev(g32), y, 9, 7, stats, mode=niti.SR, stats_index=1)
    torch.cuda.synchronize()
    assert (host(y) == oracle.round_fixed(g32, 9, oracle.SR, sr_seed=99, sr_call=1)).all()


@pytest.mark.parametrize("s_a", [-60, -30, -9, -3, 4])
def test_loss_stochastic_rounding(s_a):
    import torch
    say("sr loss", s_a)
    B, N = 64, 1000
    logits = I.weights(9900 - s_a, (B, N)); labels = I.labels(9901, B, N)
    err = torch.empty((B, N), dtype=torch.int8, device="cuda")
    stats = niti.new_stats()
    niti.set_sr_seed(stats, 7)
    ws = niti.new_workspace(niti.workspace_bytes(niti.OP_INT_CE_LOSS, None, B, N))
    for call in range(2):
        exp, _, st = oracle.int_ce_loss_grad(logits, s_a, labels, mode=oracle.SR, sr_seed=7, sr_call=call)
        niti.int_ce_loss_grad(dev(logits), _i8(s_a), dev(labels), err, stats, ws, mode=niti.SR)
        torch.cuda.synchronize()
        assert (host(err) == exp).all(), call
        assert same_stats(niti.read_stats(stats)[0], st)
