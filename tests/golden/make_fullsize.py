#!/usr/bin/env python3
"""Digests of the oracle's results at the workloads' full sizes.

Calls only ``oracle`` and the seeded input generator.  For every case it
stores the SHA-256 of the int8 (or int32) result bytes in the library's
layout (NHWC / KRSC / row-major) together with the block statistics, so the
GPU tests can compare whole full-size outputs without running the oracle.

    python tests/golden/make_fullsize.py c5      # GEMM sweep, 27 shapes x 2 ranges
    python tests/golden/make_fullsize.py c4      # ResNet-18 layer set, batch 128
    python tests/golden/make_fullsize.py c3      # VGG-style CNN, batch 256, one step
    python tests/golden/make_fullsize.py nets    # LeNet-5, VGG-small-7/8/9, batch 256, 1-3 steps
    python tests/golden/make_fullsize.py nets vgg_small8,vgg_small9   # only those (others kept)

Writes tests/golden/fullsize_<config>.json.
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle.model import OracleNet  # noqa: E402
from paper_2009_13108_amd import inputs as I  # noqa: E402

SIZES = (4096, 8192, 16384)


def sha(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def nhwc(a):
    return np.ascontiguousarray(np.asarray(a).transpose(0, 2, 3, 1))


def nchw(a):
    return np.ascontiguousarray(np.asarray(a).transpose(0, 3, 1, 2))


def pad_c(a_nchw, c):
    a = np.asarray(a_nchw)
    if a.shape[1] == c:
        return a
    z = np.zeros((a.shape[0], c - a.shape[1]) + a.shape[2:], a.dtype)
    return np.concatenate([a, z], axis=1)


def stats(st):
    return {k: int(st[k]) for k in ("max_abs", "b", "bp")}


# ---------------------------------------------------------------- config 5
def gemm_operands(M, N, K, dist):
    gen = I.weights if dist == "w" else I.errors5
    off = 0 if dist == "w" else 10
    return gen(I.base_seed(5, 1 + off), (M, K)), gen(I.base_seed(5, 2 + off), (N, K))


def make_c5(only=None):
    out = []
    for dist in ("w", "e5"):
        for M in SIZES:
            for N in SIZES:
                for K in SIZES:
                    if only and (M, N, K) not in only:
                        continue
                    t0 = time.time()
                    A, B = gemm_operands(M, N, K, dist)
                    S = oracle.gemm_nt_exact(A, B)
                    y, _, st = oracle.finish(S, False, 7)
                    rec = {"M": M, "N": N, "K": K, "dist": dist, "sha256": sha(y), **stats(st)}
                    out.append(rec)
                    print(rec, "%.1fs" % (time.time() - t0), flush=True)
                    del S, y
    return out


# ---------------------------------------------------------------- config 4
def resnet_layer_inputs(li, name, cin, cout, k, st, pd, hw, batch=128):
    """The bench's tensors for layer li (copy 0), in the library's layouts."""
    p = (hw + 2 * pd - k) // st + 1
    x = I.activations(I.base_seed(4, 100 + li), (batch, hw, hw, cin))
    dy = I.errors8(I.base_seed(4, 200 + li), (batch, p, p, cout))
    w = I.weights(I.base_seed(4, 1000 + 10 * li), (cout, k, k, cin))
    if name.startswith("stem"):
        x[..., 3:] = 0
        w[..., 3:] = 0
    return x, dy, w


def make_c4(batch=128):
    from paper_2009_13108_amd import model as M
    out = []
    for li, (name, cin, cout, k, st, pd, hw, count) in enumerate(M.RESNET18_LAYERS):
        t0 = time.time()
        x, dy, w = resnet_layer_inputs(li, name, cin, cout, k, st, pd, hw, batch)
        creal = 3 if name.startswith("stem") else cin
        d = oracle.conv_desc(batch, creal, hw, hw, cout, k, k, st, pd)
        xo, wo, dyo = nchw(x)[:, :creal], nchw(w)[:, :creal], nchw(dy)
        rec = {"layer": name, "li": li}
        y, _, s1 = oracle.conv_fwd(d, xo, wo, relu=True)
        rec["fwd"] = {"sha256": sha(nhwc(y)), **stats(s1)}
        if not name.startswith("stem"):
            dx, _, s2 = oracle.conv_bwd_data(d, dyo, wo, relu_src=xo)
            rec["bwd_data"] = {"sha256": sha(nhwc(dx)), **stats(s2)}
        w2, g32, s3 = oracle.conv_bwd_weight(d, xo, dyo, wo, mu=5)
        rec["bwd_weight"] = {"sha256_w": sha(nhwc(pad_c(w2, cin))),
                             "sha256_g32": sha(nhwc(pad_c(g32, cin))),
                             **stats(s3)}
        out.append(rec)
        print(rec, "%.1fs" % (time.time() - t0), flush=True)
    # the 512 -> 1000 head and the loss
    fin, fout = M.RESNET18_FC
    feat = I.activations(I.base_seed(4, 300), (batch, fin))
    wfc = I.weights(I.base_seed(4, 301), (fout, fin))
    lab = I.labels(I.base_seed(4, 302), batch, fout)
    logits, _, s1 = oracle.gemm_fwd(feat, wfc)
    s_log, _ = oracle.out_exponent(-9, -11, s1["bp"])
    err, _, s2 = oracle.int_ce_loss_grad(logits, s_log, lab)
    fd = oracle.conv_desc(batch, fin, 1, 1, fout, 1, 1, 1, 0)
    dfeat, _, s3 = oracle.conv_bwd_data(fd, err.reshape(batch, fout, 1, 1), wfc.reshape(fout, fin, 1, 1),
                                        relu_src=feat.reshape(batch, fin, 1, 1))
    w2, g32, s4 = oracle.conv_bwd_weight(fd, feat.reshape(batch, fin, 1, 1), err.reshape(batch, fout, 1, 1),
                                         wfc.reshape(fout, fin, 1, 1), mu=5)
    out.append({"layer": "fc", "s_logits": int(s_log),
                "fwd": {"sha256": sha(logits), **stats(s1)},
                "loss": {"sha256": sha(err), **stats(s2)},
                "bwd_data": {"sha256": sha(dfeat.reshape(batch, fin)), **stats(s3)},
                "bwd_weight": {"sha256_w": sha(w2.reshape(fout, fin)),
                               "sha256_g32": sha(g32.reshape(fout, fin).astype(np.int32)), **stats(s4)}})
    print(out[-1], flush=True)
    return out


# ---------------------------------------------------------------- config 3
def make_c3(batch=256):
    from paper_2009_13108_amd import model as M
    px = I.pixels(I.base_seed(3, 1), (batch, 3, 32, 32))
    labels = I.labels(I.base_seed(3, 2), batch, 10)
    w_orc, exps = [], []
    wi = 0
    specs = []
    for sp in M.VGG_32:
        if sp[0] == "conv":
            cin = 3 if wi == 0 else sp[1]
            w_orc.append(I.weights(I.base_seed(3, 10 + wi), (sp[2], cin, sp[3], sp[3])))
            exps.append(I.weight_exponent(cin * sp[3] * sp[3]))
            specs.append(("conv", cin) + tuple(sp[2:]))
            wi += 1
        elif sp[0] == "fc":
            # drawn as [out][(c, h, w)], stored as [out][(h, w, c)]: the order the
            # oracle network flattens its input in
            w = I.weights(I.base_seed(3, 10 + wi), (sp[2], sp[1]))
            w_orc.append(np.ascontiguousarray(w.reshape(sp[2], 256, 4, 4).transpose(0, 2, 3, 1).reshape(sp[2], -1)))
            exps.append(I.weight_exponent(sp[1]))
            specs.append(sp)
            wi += 1
        else:
            specs.append(sp)
    net = OracleNet(specs, (3, 32, 32), batch, w_orc, exps)
    t0 = time.time()
    logits, s = net.step(oracle.quantize_u8(px), -7, labels)
    rec = {"batch": batch, "steps": 1, "logits_sha256": sha(logits), "s_logits": int(s),
           "weights_sha256": []}
    for li, w in enumerate(net.w):
        if w.ndim == 4:      # conv: KCRS -> KRSC, channels padded to 4 for the image layer
            rec["weights_sha256"].append(sha(nhwc(pad_c(w, 4 if li == 0 else w.shape[1]))))
        else:                # fc: [out][(h,w,c)], the library's order
            rec["weights_sha256"].append(sha(w))
    print(rec, "%.1fs" % (time.time() - t0), flush=True)
    return rec


# ------------------------------------------------- the paper's networks
def net_weights(specs, cfg, image_channels, zero_filters):
    """The benchmark's seeded weights of a layer list in the oracle's layouts
    (KCRS, [out][in] with the input in (h, w, c) order) and their static
    exponents: the first layer's channels past the image's, and the filters
    in zero_filters (with the same input channels of the next convolution),
    held at zero; exponents from the real fan-in."""
    ws, exps = [], []
    wi = 0
    for sp in specs:
        if sp[0] == "conv":
            _, cin, cout, k = sp[:4]
            w = I.weights(I.base_seed(cfg, 10 + wi), (cout, k, k, cin))
            real = cin
            if wi == 0 and image_channels < cin:
                w[..., image_channels:] = 0
                real = image_channels
            if wi in zero_filters:
                lo, hi = zero_filters[wi]
                w[lo:hi] = 0
            if wi - 1 in zero_filters:
                lo, hi = zero_filters[wi - 1]
                w[..., lo:hi] = 0
                real = cin - (hi - lo)
            ws.append(nchw(w))
            exps.append(I.weight_exponent(real * k * k))
            wi += 1
        elif sp[0] == "fc":
            ws.append(I.weights(I.base_seed(cfg, 10 + wi), (sp[2], sp[1])))
            exps.append(I.weight_exponent(sp[1]))
            wi += 1
    return ws, exps


def make_nets(only=None, batch=256):
    """LeNet-5 (28x28x1) and VGG-small-7/8/9 (32x32x3, dropout) as the
    benchmark builds them: seeds 40 to 43, pseudo stochastic rounding everywhere,
    m_u = 5, dropout seed = the seed; image channels padded with zeros to 4.
    Per step the logits digest and exponent; after the last step every
    layer's weights (KRSC / [out][in])."""
    from paper_2009_13108_amd import model as M
    nets = [("lenet5", M.LENET5, 28, 1, {0: (6, 8)}, 40, 3), ("vgg_small7", M.vgg_small(7), 32, 3, {}, 41, 2),
            ("vgg_small8", M.vgg_small(8), 32, 3, {}, 42, 1), ("vgg_small9", M.vgg_small(9), 32, 3, {}, 43, 1)]
    out = []
    for name, specs, hw, img_c, zf, cfg, steps in nets:
        if only and name not in only:
            continue
        t0 = time.time()
        w, exps = net_weights(specs, cfg, img_c, zf)
        px = I.pixels(I.base_seed(cfg, 1), (batch, img_c, hw, hw))
        labels = I.labels(I.base_seed(cfg, 2), batch, 10)
        x = np.zeros((batch, 4, hw, hw), np.int8)
        x[:, :img_c] = oracle.quantize_u8(px)
        ospecs = [("conv",) + tuple(sp[1:]) if sp[0] == "conv" else sp for sp in specs]
        net = OracleNet(ospecs, (4, hw, hw), batch, w, exps, mu=5, mode=oracle.PSR, grad_mode=oracle.PSR,
                        sr_seed=0, drop_seed=cfg)
        rec = {"net": name, "batch": batch, "seed": cfg, "steps": []}
        for _ in range(steps):
            logits, s = net.step(x, -7, labels)
            rec["steps"].append({"logits_sha256": sha(logits), "s_logits": int(s)})
        rec["weights_sha256"] = [sha(nhwc(v)) if v.ndim == 4 else sha(v) for v in net.w]
        out.append(rec)
        print(rec, "%.1fs" % (time.time() - t0), flush=True)
    return out


def main():
    which = sys.argv[1]
    fn = {"c5": make_c5, "c4": make_c4, "c3": make_c3, "nets": make_nets}[which]
    path = os.path.join(HERE, "fullsize_%s.json" % which)
    if which == "nets" and len(sys.argv) > 2:
        # only the named networks; the others' cases already in the file are kept
        only = sys.argv[2].split(",")
        res = fn(only)
        if os.path.exists(path):
            with open(path) as f:
                kept = [c for c in json.load(f)["cases"] if c["net"] not in only]
            res = kept + res
    else:
        res = fn()
    with open(path, "w") as f:
        json.dump({"source": "oracle (tests/golden/make_fullsize.py %s)" % which, "cases": res}, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
