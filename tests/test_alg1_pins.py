"""Pins of the oracle's whole-step composition (oracle.model.OracleNet,
Algorithm 1) against an independent pure-Python big-integer statement of
the same step (tests/alg1_bigint.py, which imports nothing from the oracle).

Tiny networks, a few samples, two consecutive steps: the logits, their
exponent and every weight tensor after each step must agree exactly.  The
cases cover both branches of the integer loss (Section 3.5), both rounding
modes, several update widths m_u, a ReLU'd layer below a fully-connected
layer, a pooling layer between a ReLU'd convolution and a fully-connected
layer (error routing, then the mask of the convolution below), and a strided
convolution."""
import numpy as np
import pytest

import oracle
from oracle.model import OracleNet
from paper_2009_13108_amd import inputs as I

import alg1_bigint as R

FC_NET = [("fc", 6, 5, True), ("fc", 5, 4, False)]
CONV_NET = [("conv", 2, 3, 3, 1, 1, True), ("pool",), ("fc", 12, 4, False)]
DEEP_NET = [("conv", 1, 2, 3, 2, 1, True), ("conv", 2, 3, 3, 1, 1, True), ("pool",), ("fc", 12, 3, True),
            ("fc", 3, 2, False)]

CASES = [
    # name, specs, input (c, h, w), batch, weight exponents, mu, mode, pixel range
    ("fc_psr", FC_NET, (6, 1, 1), 3, (-7, -7), 5, oracle.PSR, 127),
    ("fc_rtn_mu3", FC_NET, (6, 1, 1), 3, (-7, -7), 3, oracle.RTN, 127),
    ("fc_taylor", FC_NET, (6, 1, 1), 2, (-12, -12), 5, oracle.PSR, 127),
    ("fc_taylor_rtn", FC_NET, (6, 1, 1), 2, (-12, -13), 2, oracle.RTN, 127),
    ("conv_pool_fc", CONV_NET, (2, 4, 4), 2, (-7, -7), 5, oracle.PSR, 127),
    ("conv_pool_fc_taylor", CONV_NET, (2, 4, 4), 2, (-9, -11), 4, oracle.PSR, 127),
    ("conv_pool_fc_rtn", CONV_NET, (2, 4, 4), 3, (-6, -8), 1, oracle.RTN, 127),
    ("deep_strided", DEEP_NET, (1, 8, 8), 2, (-7, -7, -7, -7), 5, oracle.PSR, 127),
    ("deep_small_pixels", DEEP_NET, (1, 8, 8), 2, (-5, -6, -7, -8), 5, oracle.PSR, 3),
]


def _init(specs, in_shape, batch, seed, pix):
    c, h, w = in_shape
    ws = []
    for sp in specs:
        if sp[0] == "conv":
            _, cin, cout, k, _, _, _ = sp
            ws.append(I.weights(seed + len(ws), (cout, cin, k, k)))
        elif sp[0] == "fc":
            ws.append(I.weights(seed + len(ws), (sp[2], sp[1])))
    x = (I.activations(seed + 50, (batch, c, h, w)).astype(np.int16) % (pix + 1)).astype(np.int8)
    ncls = [sp for sp in specs if sp[0] == "fc"][-1][2]
    return ws, x, ncls


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_oracle_step_matches_bigint_algorithm1(case):
    name, specs, in_shape, batch, wexp, mu, mode, pix = case
    seed = 3100 + 17 * CASES.index(case)
    ws, x, ncls = _init(specs, in_shape, batch, seed, pix)
    net = OracleNet(specs, in_shape, batch, ws, wexp, mu=mu, mode=mode)
    ref_w = [w.tolist() for w in ws]
    s_logits = []
    for step in range(2):
        labels = I.labels(seed + 60 + step, batch, ncls)
        lo, so = net.step(x, -7, labels)
        lr, sr = R.train_step(specs, ref_w, list(wexp), x.tolist(), -7, [int(v) for v in labels], mu=mu,
                              mode=mode)
        assert so == sr, (step, so, sr)
        assert np.array_equal(np.asarray(lo).reshape(batch, -1), np.array(lr).reshape(batch, -1)), step
        for li, (wo, wr) in enumerate(zip(net.w, ref_w)):
            assert np.array_equal(wo, np.array(wr, dtype=np.int8)), (step, li)
        s_logits.append(so)
    # the weights moved (the step is not vacuous)
    assert any(not np.array_equal(a, b) for a, b in zip(net.w, ws))


def test_cases_cover_both_loss_branches():
    """The exponents of the cases above put the logits in both loss cases."""
    seen = set()
    for case in CASES:
        name, specs, in_shape, batch, wexp, mu, mode, pix = case
        seed = 3100 + 17 * CASES.index(case)
        ws, x, ncls = _init(specs, in_shape, batch, seed, pix)
        net = OracleNet(specs, in_shape, batch, ws, wexp, mu=mu, mode=mode)
        _, s = net.step(x, -7, I.labels(seed + 60, batch, ncls))
        seen.add("taylor" if s <= -7 else "base2")
    assert seen == {"taylor", "base2"}


def test_reference_rounding_matches_worked_examples():
    """The big-integer reference's rounding agrees with the hand-derived
    Algorithm 3 examples, so the two statements start from the same facts."""
    import json
    import os
    ex = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "psr_examples.json")))
    for e in ex["cases"]:
        assert R.psr(e["x"], e["bp"]) == e["out"], e
