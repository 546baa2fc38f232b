"""Pins of the CPU oracle to facts other than its own code.

Each test ties one oracle function to something fixed independently of it:
values worked by hand from the paper's algorithms (``tests/golden``), closed
forms, invariants the rounding scheme must satisfy, library routines that
compute the same mathematical object (torch float64 convolutions, numpy
matmul -- exact here because every partial sum is an integer far below
2^53), and adjoint identities that any correct forward / backward pair obeys.
None of this needs a GPU.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2009_13108_amd import inputs as I

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ------------------------------------------------------------------ PSR (Alg. 3)
def test_psr_worked_examples():
    g = _gold("psr_examples.json")
    for c in g["cases"]:
        assert oracle.psr(c["x"], c["bp"]) == c["out"], c


def test_shift_round_worked_blocks():
    g = _gold("psr_examples.json")
    for c in g["blocks"]:
        out, st = oracle.shift_round(np.array(c["acc"], np.int32), c["target"])
        assert st["b"] == c["b"] and st["bp"] == c["bp"]
        assert out.tolist() == c["out"]


def test_bitlen_closed_form():
    # Section 3.2: effective bitwidth = bits needed for the largest magnitude;
    # Python's int.bit_length is the library routine for exactly that.
    for m in [0, 1, 2, 3, 127, 128, 255, 256, 2 ** 31 - 1, 2 ** 31, 2 ** 32 - 1,
              2 ** 62, 2 ** 63 - 1, 2 ** 63]:
        assert oracle.bitlen(m) == int(m).bit_length()


@pytest.mark.parametrize("bp", list(range(0, 13)))
def test_psr_outputs_are_floor_or_floor_plus_one(bp):
    xs = np.arange(0, 1 << min(bp + 7, 18))
    for x in xs[:: max(1, len(xs) // 4000)]:
        x = int(x)
        r = oracle.psr(x, bp)
        q = x >> bp
        assert r in (min(q, 127), min(q + 1, 127))
        assert oracle.psr(-x, bp) == -r                       # odd symmetry
        if bp and (x & ((1 << bp) - 1)) == 0:
            assert r == min(q, 127)                           # no fraction -> exact


def test_psr_identity_and_truncation():
    for x in range(-300, 301):
        assert oracle.psr(x, 0) == max(-127, min(127, x))     # bp = 0: nothing to round
        q = min(abs(x) >> 1, 127)                             # bp = 1: fraction is dropped
        assert oracle.psr(x, 1) == (q if x >= 0 else -q)


@pytest.mark.parametrize("bp", [2, 4, 6, 8, 10])
def test_psr_conditional_mean_is_top_half(bp):
    # Over all values of the lower half of the fraction (the pseudo random
    # draw), the mean result is q + top/2^h exactly: the scheme is unbiased
    # with respect to the truncated fraction (Section 3.4).
    h = bp // 2
    for q in (0, 5, 100):
        for top in range(0, 1 << h, max(1, (1 << h) // 8)):
            tot = Fraction(0)
            for low in range(1 << h):
                x = (q << bp) | (top << h) | low
                tot += oracle.psr(x, bp)
            assert tot / (1 << h) == q + Fraction(top, 1 << h)


@pytest.mark.parametrize("bp", [3, 5, 7, 9])
def test_psr_odd_bp_ignores_lowest_bit(bp):
    for x in range(0, 1 << (bp + 6), 7):
        assert oracle.psr(x, bp) == oracle.psr(x ^ 1, bp)


@pytest.mark.parametrize("bp", [2, 4, 8])
def test_psr_total_bias_closed_form(bp):
    # Uniform fraction: mean(PSR) - mean(x / 2^bp) = -(2^h - 1) / 2^(2h+1).
    h = bp // 2
    q = 3
    xs = range(q << bp, (q + 1) << bp)
    got = Fraction(sum(oracle.psr(x, bp) for x in xs), 1 << bp)
    exact = Fraction(sum(xs), 1 << bp) / (1 << bp)
    assert got - exact == -Fraction((1 << h) - 1, 1 << (2 * h + 1))


def test_psr_histogram_of_draws_near_uniform():
    # The lower half of the fraction acts as the random number; on
    # accumulator-like values its histogram is near uniform (Fig. 3's claim).
    acc = I.uniform_int(11, (200000,), -(1 << 20), 1 << 20, dtype=np.int64)
    bp, h = 14, 7
    low = (np.abs(acc) & ((1 << bp) - 1)) & ((1 << h) - 1)
    hist = np.bincount(low, minlength=1 << h) / low.size
    assert np.abs(hist * (1 << h) - 1).max() < 0.1


def test_rtn_half_away_from_zero():
    for x in range(-2000, 2000, 3):
        for bp in range(0, 6):
            exp = int(math.copysign(math.floor(abs(x) / (1 << bp) + 0.5), x)) if x else 0
            assert oracle.rtn(x, bp) == max(-127, min(127, exp))


def test_shift_round_uses_int8_range():
    for seed in range(5):
        acc = I.uniform_int(seed, (4096,), -(1 << 27), 1 << 27, dtype=np.int32)
        out, st = oracle.shift_round(acc, 7)
        mx = int(np.abs(acc.astype(np.int64)).max())
        assert st["max_abs"] == mx and st["b"] == mx.bit_length()
        assert st["bp"] == max(0, mx.bit_length() - 7)
        assert np.abs(out.astype(int)).max() >= 64       # top bit of int8 in use
        assert np.abs(out.astype(int)).max() <= 127
        # every output within one step of the exact quotient
        quo = np.abs(acc.astype(np.int64)) / (1 << st["bp"])
        assert (np.abs(np.abs(out.astype(np.int64)) - quo) < 1.0 + 1e-9).all()


def test_exponent_arithmetic():
    # Algorithm 2: s_q = s_q32 + bp, with s_q32 = s_a + s_w (Section 3.1).
    assert oracle.out_exponent(-7, -8, 5) == (-10, 0)
    assert oracle.out_exponent(-128, -1, 0) == (-128, oracle.FLAG_EXP_RANGE)
    assert oracle.out_exponent(120, 10, 0) == (127, oracle.FLAG_EXP_RANGE)


def test_int32_min_block():
    acc = np.array([-(2 ** 31), 5, -7], np.int32)
    out, st = oracle.shift_round(acc, 7)
    assert st["max_abs"] == 2 ** 31 and st["b"] == 32 and st["bp"] == 25
    assert out.tolist() == [-64, 0, 0]


# ------------------------------------------------------------------ contractions
def _torch():
    torch = pytest.importorskip("torch")
    return torch


def test_gemm_matches_numpy_matmul():
    for (M, N, K) in [(1, 1, 1), (7, 5, 3), (33, 17, 65), (64, 128, 784)]:
        A = I.weights(M * 7 + K, (M, K))
        B = I.weights(N * 3 + K, (N, K))
        S = oracle.gemm_nt_raw(A, B)
        assert (S == A.astype(np.int64) @ B.astype(np.int64).T).all()
        rows = np.array([0, M - 1, M // 2]); cols = np.array([N - 1, 0, N // 2])
        assert (oracle.gemm_nt_pick(A, B, rows, cols) == S[rows, cols]).all()


def test_gemm_exact_large_route_matches_int64_loops():
    # the float64 route used for the large GEMM digests equals the int64 loops
    for (M, N, K) in [(300, 257, 4096), (64, 3000, 16384), (1, 1, 16384)]:
        A = I.weights(M + K, (M, K)); B = I.weights(N + 2 * K, (N, K))
        assert (oracle.gemm_nt_exact(A, B, block_rows=100) == oracle.gemm_nt_raw(A, B)).all()
    A = np.full((2, 16384), -127, np.int8)
    assert (oracle.gemm_nt_exact(A, A) == 16384 * 127 * 127).all()


def test_gemm_all_ones_and_overflow_flag():
    K = 140000                          # 140000 * 127^2 > 2^31
    A = np.full((1, K), 127, np.int8)
    out, acc, st = oracle.gemm_fwd(A, A)
    assert acc[0, 0] == np.int32(np.uint32((K * 127 * 127) % (1 << 32)).view(np.int32))
    assert st["flags"] == oracle.FLAG_ACC_BOUND | oracle.FLAG_ACC_WRAP
    # a long reduction that stays in range: the static bound only
    _, acc, st = oracle.gemm_fwd(np.ones((1, K), np.int8), np.ones((1, K), np.int8))
    assert acc[0, 0] == K and st["flags"] == oracle.FLAG_ACC_BOUND
    ones = np.ones((2, 100), np.int8)
    _, acc, st = oracle.gemm_fwd(ones, ones)
    assert (acc == 100).all() and st["flags"] == 0


def test_accumulator_bound_covers_every_wrap():
    """Below 2^17 products no int8 sum can leave the int32 range (each product
    is at most 2^14 in magnitude: (-128)^2), at 2^17 one can."""
    n = oracle.ACC_BOUND_LEN
    assert (n - 1) * 128 * 128 < 2 ** 31 <= n * 128 * 128
    A = np.full((1, n), -128, np.int8)
    _, acc, st = oracle.gemm_fwd(A, A)
    assert st["flags"] == oracle.FLAG_ACC_BOUND | oracle.FLAG_ACC_WRAP and acc[0, 0] == -2 ** 31
    _, acc, st = oracle.gemm_fwd(A[:, 1:], A[:, 1:])
    assert st["flags"] == 0 and acc[0, 0] == 2 ** 31 - 2 ** 14


CONV_CASES = [
    # n, c, h, w, k, r, s, stride, pad
    (1, 1, 5, 5, 1, 3, 3, 1, 1),
    (2, 3, 7, 6, 4, 3, 3, 1, 1),
    (2, 5, 9, 9, 3, 3, 3, 2, 1),
    (1, 3, 11, 11, 2, 7, 7, 2, 3),
    (2, 4, 8, 8, 5, 1, 1, 2, 0),
    (1, 2, 6, 7, 3, 1, 1, 1, 0),
    (3, 2, 5, 5, 2, 3, 3, 1, 0),
    (1, 3, 6, 6, 2, 2, 3, 2, 2),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_three_passes_match_torch_float64(case):
    torch = _torch()
    n, c, h, w, k, r, s, st, pd = case
    d = oracle.conv_desc(n, c, h, w, k, r, s, st, pd)
    P, Q = oracle.conv_out_hw(d)
    x = I.activations(1 + n + c, (n, c, h, w))
    wt = I.weights(2 + k, (k, c, r, s))
    dy = I.errors8(3 + h, (n, k, P, Q))
    F = torch.nn.functional
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    wtt = torch.tensor(wt, dtype=torch.float64, requires_grad=True)
    y = F.conv2d(xt, wtt, stride=st, padding=pd)
    y.backward(torch.tensor(dy, dtype=torch.float64))
    assert (oracle.conv_fwd_raw(d, x, wt) == y.detach().numpy().astype(np.int64)).all()
    assert (oracle.conv_bwd_data_raw(d, dy, wt) == xt.grad.numpy().astype(np.int64)).all()
    assert (oracle.conv_bwd_weight_raw(d, x, dy) == wtt.grad.numpy().astype(np.int64)).all()


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_adjoint_identities(case):
    # <conv(x,w), dy> = <x, bwd_data(dy,w)> = <w, bwd_weight(x,dy)>, exactly.
    n, c, h, w, k, r, s, st, pd = case
    d = oracle.conv_desc(n, c, h, w, k, r, s, st, pd)
    P, Q = oracle.conv_out_hw(d)
    x = I.weights(10 + c, (n, c, h, w))
    wt = I.weights(20 + k, (k, c, r, s))
    dy = I.weights(30 + h, (n, k, P, Q))
    a = int((oracle.conv_fwd_raw(d, x, wt) * dy.astype(np.int64)).sum())
    b = int((oracle.conv_bwd_data_raw(d, dy, wt) * x.astype(np.int64)).sum())
    g = int((oracle.conv_bwd_weight_raw(d, x, dy) * wt.astype(np.int64)).sum())
    assert a == b == g


def test_conv_identity_kernel_and_fc_equivalence():
    x = I.activations(5, (2, 4, 6, 6))
    w = np.zeros((4, 4, 3, 3), np.int8)
    for i in range(4):
        w[i, i, 1, 1] = 1
    d = oracle.conv_desc(2, 4, 6, 6, 4, 3, 3, 1, 1)
    assert (oracle.conv_fwd_raw(d, x, w) == x).all()
    # a 1x1 convolution on 1x1 maps is the fully-connected layer
    A = I.activations(6, (5, 12))
    W = I.weights(7, (3, 12))
    d1 = oracle.conv_desc(5, 12, 1, 1, 3, 1, 1, 1, 0)
    assert (oracle.conv_fwd_raw(d1, A.reshape(5, 12, 1, 1), W.reshape(3, 12, 1, 1)).reshape(5, 3)
            == oracle.gemm_nt_raw(A, W)).all()


def test_conv_fwd_one_matches_full():
    d = oracle.conv_desc(2, 3, 9, 9, 4, 3, 3, 2, 1)
    x = I.activations(8, (2, 3, 9, 9)); w = I.weights(9, (4, 3, 3, 3))
    y = oracle.conv_fwd_raw(d, x, w)
    for (n, k, p, q) in [(0, 0, 0, 0), (1, 3, 4, 4), (1, 2, 0, 3)]:
        assert oracle.conv_fwd_one(d, x, w, n, k, p, q) == y[n, k, p, q]


def test_forward_relu_before_exponent():
    S = np.array([[-1000, 300, 5]], np.int64)
    out, acc, st = oracle.finish(S, relu=True, target=7)
    assert acc.tolist() == [[0, 300, 5]] and st["b"] == 9 and st["bp"] == 2
    out2, _, st2 = oracle.finish(S, relu=False, target=7)
    assert st2["b"] == 10


# ------------------------------------------------------------------ update (Sec 3.3)
def test_update_zero_gradient_keeps_weights():
    w = I.weights(1, (50,))
    w2, st = oracle.sgd_update(w, np.zeros(50, np.int32), 5)
    assert (w2 == w).all() and st["b"] == 0 and st["bp"] == 0


@pytest.mark.parametrize("mu", [1, 2, 3, 4, 5])
def test_update_single_power_of_two(mu):
    for k in range(mu, 30):
        g = np.zeros(9, np.int32); g[4] = 1 << k; g[2] = -(1 << k)
        w = np.zeros(9, np.int8)
        w2, st = oracle.sgd_update(w, g, mu)
        assert w2[4] == -(1 << (mu - 1)) and w2[2] == (1 << (mu - 1))
        assert st["bp"] == k + 1 - mu


def test_update_saturates_and_moves_against_gradient():
    w = np.array([127, -127, 0, 100], np.int8)
    g = np.array([-(1 << 20), 1 << 20, 1 << 19, 1 << 20], np.int32)
    w2, st = oracle.sgd_update(w, g, 5)
    assert w2.tolist() == [127, -127, -8, 84]  # g = [-16, 16, 8, 16]


def test_update_step_bounded_by_mu():
    w = I.weights(3, (10000,))
    g = I.uniform_int(4, (10000,), -(1 << 24), 1 << 24, dtype=np.int32)
    for mu in (1, 3, 5):
        w2, _ = oracle.sgd_update(w, g, mu)
        step = np.abs(w2.astype(int) - w.astype(int))
        assert step.max() <= (1 << mu)
        moved = (w2 != w)
        assert (np.sign(w.astype(int) - w2.astype(int))[moved] == np.sign(g[moved])).all()


# ------------------------------------------------------------------ loss (Sec 3.5)
def test_loss_worked_examples():
    g = _gold("loss_examples.json")
    for c in g["cases"]:
        err, e32, st = oracle.int_ce_loss_grad(np.array(c["logits"], np.int8), c["s_a"],
                                               np.array(c["labels"], np.int32))
        assert e32.tolist() == c["e32"], c["why"]
        assert st["bp"] == c["bp"]
        assert err.tolist() == c["err"]


@pytest.mark.parametrize("s_a", [-6, -5, -3, -1, 0, 2, 7, 14, 15, 16, 40, 127])
def test_loss_base2_branch_tracks_exp(s_a):
    # Non-label entries are t_i = 2^xtilde: powers of two in [1, 2^10]; the
    # largest logit gets 2^10; each row sums to zero (sum t - C = 0); and the
    # integer exponent xhat stays within one of log2(e) a 2^s_a.
    logits = I.weights(300 + s_a, (64, 10))
    labels = I.labels(5, 64, 10)
    _, e32, _ = oracle.int_ce_loss_grad(logits, s_a, labels)
    for b in range(64):
        row = e32[b]
        assert int(row.sum()) == 0
        others = [int(v) for i, v in enumerate(row) if i != labels[b]]
        assert all(1 <= v <= 1024 and (v & (v - 1)) == 0 for v in others)
        a = logits[b].astype(np.int64)
        am = int(np.argmax(a))
        if am != labels[b]:
            assert row[am] == 1024
        if s_a < 15:
            x = float(a.max()) * math.log2(math.e) * 2.0 ** s_a
            xhat = math.floor(47274 * int(a.max()) / 2.0 ** (15 - s_a))
            assert abs(xhat - x) < 1 + 1e-5 * abs(x)


@pytest.mark.parametrize("s_a", [-7, -8, -10, -13, -16, -22])
def test_loss_taylor_branch_tracks_exp(s_a):
    logits = I.weights(300 - s_a, (32, 10))
    labels = I.labels(6, 32, 10)
    _, e32, st = oracle.int_ce_loss_grad(logits, s_a, labels)
    assert st["flags"] == 0
    scale = 2.0 ** (1 - 2 * s_a)
    for b in range(32):
        row = e32[b]
        assert int(row.sum()) == 0
        for i in range(10):
            if i == labels[b]:
                continue
            x = float(logits[b, i]) * 2.0 ** s_a
            # second-order Taylor error is at most |x|^3 e^|x| / 6
            assert abs(row[i] / scale - math.exp(x)) <= abs(x) ** 3 * math.exp(abs(x)) / 6 + 1e-12


def test_loss_gradient_signs():
    for s_a in (-9, -4, 3):
        logits = I.weights(7, (16, 100)); labels = I.labels(8, 16, 100)
        err, e32, _ = oracle.int_ce_loss_grad(logits, s_a, labels)
        for b in range(16):
            assert e32[b, labels[b]] < 0 and (np.delete(e32[b], labels[b]) > 0).all()
            assert err[b, labels[b]] <= 0 and (np.delete(err[b], labels[b]) >= 0).all()


def _literal_loss(logits, s_a, labels, mode=oracle.PSR):
    """Section 3.5 in unbounded Python integers (tests/alg1_bigint.py, which
    shares nothing with the oracle): (err, pre-rounding values, max, bp)."""
    import alg1_bigint as R
    rows = []
    for a, y in zip(logits.tolist(), labels.tolist()):
        t = R.loss_terms(a, s_a)
        c = sum(t)
        t[y] -= c
        rows.append(t)
    flat = [v for r in rows for v in r]
    err, bp = R.shift_and_round(flat, 7, R.PSR if mode == oracle.PSR else R.RTN)
    return np.array(err, np.int8).reshape(logits.shape), rows, max(abs(v) for v in flat), bp


def _loss_logits(kind, seed, B, N):
    if kind == "uniform":
        return I.weights(seed, (B, N))
    if kind == "5bit":
        return I.errors5(seed, (B, N))
    lg = np.full((B, N), 127, np.int8)
    if kind == "edge":
        lg[:, ::3] = -127
    elif kind == "min":
        lg[:, ::2] = -128
    return lg


@pytest.mark.parametrize("s_a", [-7, -8, -15, -22, -23, -24, -31, -40, -54])
@pytest.mark.parametrize("N,B,kind", [(1, 3, "uniform"), (2, 4, "uniform"), (10, 8, "uniform"),
                                      (1000, 2, "edge"), (1000, 2, "5bit"), (4097, 1, "min")])
def test_loss_taylor_exact_against_bigint(s_a, N, B, kind):
    """The Taylor branch is evaluated exactly for -54 <= s_a <= -7: every
    pre-rounding value, the block b and bp, and the int8 error equal the
    literal formula in unbounded integers; max_abs is the maximum shifted
    right by 2 (-22 - s_a) bits below s_a = -22."""
    logits = _loss_logits(kind, 700 + N + B, B, N)
    labels = I.labels(701 + N, B, N)
    for mode in (oracle.PSR, oracle.RTN):
        err, e, st = oracle.int_ce_loss_grad(logits, s_a, labels, mode=mode)
        ref_err, rows, mx, bp = _literal_loss(logits, s_a, labels, mode)
        assert [[int(v) for v in r] for r in e] == rows
        assert st["flags"] == 0 and st["bp"] == bp and st["b"] == mx.bit_length()
        assert st["max_abs"] == mx >> (2 * (-22 - s_a) if s_a < -22 else 0)
        assert (err == ref_err).all()


@pytest.mark.parametrize("s_a", [-55, -64, -100, -128])
@pytest.mark.parametrize("N,B,kind", [(10, 8, "uniform"), (100, 4, "edge"), (1000, 2, "edge"),
                                      (1000, 2, "5bit"), (4097, 1, "min")])
def test_loss_below_hold_equals_literal(s_a, N, B, kind):
    """Below s_a = -54 the oracle evaluates s_a = -54 and flags it; its int8
    error equals the literal formula at the true s_a (the rounded result no
    longer depends on s_a there)."""
    logits = _loss_logits(kind, 900 + N + B, B, N)
    labels = I.labels(901 + N, B, N)
    err, _, st = oracle.int_ce_loss_grad(logits, s_a, labels)
    ref_err, _, _, _ = _literal_loss(logits, s_a, labels)
    assert st["flags"] & oracle.FLAG_LOSS_SA
    assert (err == ref_err).all()


def test_loss_hold_at_22_would_be_wrong():
    """The reason the Taylor branch is wide: s_a = -23 gives a different
    int8 error than s_a = -22 for a 1000-class row of extreme logits."""
    logits = _loss_logits("edge", 1000 + 4 + 2, 4, 1000)
    labels = I.labels(1000 + 4, 4, 1000)
    e22, _, _ = oracle.int_ce_loss_grad(logits, -22, labels)
    e23, _, _ = oracle.int_ce_loss_grad(logits, -23, labels)
    ref23, _, _, _ = _literal_loss(logits, -23, labels)
    assert (e23 == ref23).all() and not (e23 == e22).all()


def test_loss_constant_is_log2e():
    # the printed constant 47274 is floor(log2(e) * 2^15)
    assert math.floor(math.log2(math.e) * 2 ** 15) == 47274


# ------------------------------------------------------------------ glue
def test_maxpool_matches_numpy():
    x = I.weights(3, (2, 3, 6, 8))
    y, idx = oracle.maxpool2_fwd(x)
    win = x.reshape(2, 3, 3, 2, 4, 2).transpose(0, 1, 2, 4, 3, 5).reshape(2, 3, 3, 4, 4)
    assert (y == win.max(-1)).all()
    assert (idx == win.argmax(-1)).all()       # numpy argmax picks the first maximum
    dy = I.weights(4, y.shape)
    dx = oracle.maxpool2_bwd(dy, idx, x.shape)
    assert int(dx.astype(np.int64).sum()) == int(dy.astype(np.int64).sum())
    assert ((dx != 0).sum() <= (dy != 0).sum())


def test_relu_mask_and_quantize():
    e = np.array([5, -3, 7, 9], np.int8); a = np.array([1, 0, -2, 127], np.int8)
    assert oracle.relu_mask(e, a).tolist() == [5, 0, 0, 9]
    px = np.arange(256, dtype=np.uint8)
    assert (oracle.quantize_u8(px) == (np.arange(256) // 2)).all()


# ------------------------------------------------------------------ stochastic rounding (Sec 3.4, Rs)
def test_sr_generator_is_splitmix64():
    """The draws are the SplitMix64 stream: seed 0 gives the reference
    implementation's first outputs, and the counter advances by one per
    element and by 2^40 per call."""
    assert [oracle.sr_draw(0, 0, i) for i in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                                          0x06C45D188009454F]
    assert oracle.sr_draw(0, 1, 0) == oracle.sr_draw(0, 0, 1 << 40)
    assert oracle.sr_draw(5, 0, 0) != oracle.sr_draw(6, 0, 0)


@pytest.mark.parametrize("bp", [1, 2, 3, 5, 8, 11])
def test_sr_expectation_is_exact_over_all_draws(bp):
    """Rs rounds up with probability f / 2^bp: over the 2^bp equally likely
    values of the draw's top bits the outputs sum to exactly x (no clamp)."""
    for x in (0, 1, 3, 1000, (1 << bp) - 1, 100 << bp, (127 << bp) - 1):
        if (x >> bp) >= 127:
            continue
        for sign in (1, -1):
            tot = sum(oracle.sr(sign * x, bp, r << (64 - bp)) for r in range(1 << bp))
            assert tot == sign * x, (x, bp)


def test_sr_is_unbiased_with_the_generator():
    """With the generator's draws, the mean rounded value of many equal
    inputs is x / 2^bp within a few standard errors (Section 3.4: zero
    rounding bias)."""
    x, bp, n = 1003, 5, 40000
    out, _ = oracle.shift_round(np.full(n, x, np.int32), 7, oracle.SR, sr_seed=77)
    # the block exponent of 1003 is b = 10, bp = 3 for target 7
    assert int(np.abs(out).max()) <= (x >> 3) + 1
    mean = out.astype(np.float64).mean()
    p = (x & 7) / 8
    assert abs(mean - x / 8) < 5 * math.sqrt(p * (1 - p) / n)
    r = oracle.round_fixed(np.full(n, -x, np.int32), bp, oracle.SR, sr_seed=3, sr_call=2)
    p = (x & 31) / 32
    assert abs(r.astype(np.float64).mean() + x / 32) < 5 * math.sqrt(p * (1 - p) / n)


def test_sr_tensor_rounding_uses_the_keyed_draws():
    v = I.uniform_int(11, (3000,), -(1 << 20), 1 << 20, dtype=np.int32)
    out, st = oracle.shift_round(v, 7, oracle.SR, sr_seed=12345, sr_call=9)
    bp = st["bp"]
    exp = [oracle.sr(int(a), bp, oracle.sr_draw(12345, 9, i)) for i, a in enumerate(v[:300])]
    assert out[:300].tolist() == exp
    out2, _ = oracle.shift_round(v, 7, oracle.SR, sr_seed=12345, sr_call=10)
    assert (out2 != out).any()                          # another call, other draws
    assert (np.abs(out2.astype(int) - out.astype(int)) <= 1).all()


def test_sr_update_and_conv_follow_storage_order():
    """The update's draws are keyed by the KRSC position of each weight."""
    d = oracle.conv_desc(2, 4, 5, 5, 3, 3, 3, 1, 1)
    x = I.activations(1, (2, 4, 5, 5)); dy = I.errors8(2, (2, 3, 5, 5)); w = I.weights(3, (3, 4, 3, 3))
    w2, g32, st = oracle.conv_bwd_weight(d, x, dy, w, mu=5, mode=oracle.SR, sr_seed=1, sr_call=4)
    bp = st["bp"]
    krsc = np.ascontiguousarray(g32.transpose(0, 2, 3, 1)).reshape(-1)
    wk = np.ascontiguousarray(w.transpose(0, 2, 3, 1)).reshape(-1)
    exp = [max(-127, min(127, int(wk[i]) - oracle.sr(int(krsc[i]), bp, oracle.sr_draw(1, 4, i))))
           for i in range(krsc.size)]
    assert np.ascontiguousarray(w2.transpose(0, 2, 3, 1)).reshape(-1).tolist() == exp
