"""A second, independent statement of one NITI training step (Algorithm 1),
in plain Python integers, for tiny networks only.

It pins the oracle's layer composition: it imports nothing from ``oracle``
and shares no helper with it.  Tensors are nested lists (activations
[n][c][h][w], filters [k][c][r][s], fully-connected weights [out][in]).
Every sum is an exact Python integer; the int32 accumulator of the method
is that sum reduced mod 2^32 (no test here comes near the bound).

Readings of the points the paper leaves open are the ones the design notes
list: B(V) counts magnitude bits (R1); a rounded magnitude is held at 127
(R2); the update saturates to [-127, 127] (R4); forward ReLU acts on the
int32 sums before the block maximum, backward ReLU zeroes the rounded int8
error where the stored activation is not positive (R5); the loss offset is
p = max(xhat) - 10 (R6) with the constant 47274 (R7) and a flooring shift
(R8); the Taylor branch of the loss is evaluated exactly (R9); 2x2 pooling
routes an error to the first maximum of its window in row-major order
(S10); a fully-connected layer after a convolution reads its input
flattened in (h, w, c) order.  Stochastic rounding (Section 3.4's Rs) and
dropout draw from SplitMix64 (Steele, Lea and Flood 2014), written out here
from its definition, keyed by (seed, call, storage offset): offsets follow
the library's storage order (NHWC activations and errors, KRSC filters,
row-major matrices); seeds are sr_seed + statistics block (three blocks per
weighted layer -- forward, back-propagation, weight gradient -- then the
loss) and the call is the step index.
"""
from __future__ import annotations

PSR = 0
RTN = 1
SR = 2
M64 = (1 << 64) - 1


def splitmix(seed, call, index):
    """Output number call * 2^40 + index + 1 of the SplitMix64 stream."""
    z = (seed + ((call << 40) + index + 1) * 0x9E3779B97F4A7C15) & M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


# --------------------------------------------------------------- rounding
def wrap32(v: int) -> int:
    """The int32 the method accumulates in: v mod 2^32, two's complement."""
    v &= 0xFFFFFFFF
    return v - (1 << 32) if v >= (1 << 31) else v


def bits(m: int) -> int:
    """Effective bitwidth of a magnitude (Section 3.2)."""
    n = 0
    while m:
        n += 1
        m >>= 1
    return n


def psr(v: int, bp: int) -> int:
    """Algorithm 3: integer part of |v| above the binary point, fraction
    below it; odd bp drops the fraction's lowest bit; the upper half of the
    fraction is compared with the lower half; the sign of v is put back."""
    mag = -v if v < 0 else v
    if bp == 0:
        q = mag
    else:
        q = mag // (2 ** bp)
        f = mag % (2 ** bp)
        width = bp
        if width % 2 == 1:
            f = f // 2
            width -= 1
        half = width // 2
        top, low = f // (2 ** half), f % (2 ** half)
        if top > low:
            q += 1
    q = min(q, 127)
    return -q if v < 0 else q


def rtn(v: int, bp: int) -> int:
    """Round to nearest on the magnitude, ties away from zero."""
    mag = -v if v < 0 else v
    q = (mag + (2 ** (bp - 1) if bp > 0 else 0)) // (2 ** bp)
    q = min(q, 127)
    return -q if v < 0 else q


def sr(v: int, bp: int, draw: int) -> int:
    """Rs: up with probability f / 2^bp -- here when the draw's top bp bits
    are below the fraction f."""
    mag = -v if v < 0 else v
    q, f = mag >> bp, mag & ((1 << bp) - 1)
    if bp and (draw >> (64 - bp)) < f:
        q += 1
    q = min(q, 127)
    return -q if v < 0 else q


def shift_and_round(values, target, mode, key=None, offsets=None):
    """Algorithm 2 over a flat list: bp = max(0, B(max|v|) - target), every
    value rounded with that one bp.  key = (seed, call) and offsets (storage
    offset of each value, default its position) for stochastic rounding.
    Returns (rounded, bp)."""
    mx = max((abs(v) for v in values), default=0)
    bp = max(0, bits(mx) - target)
    if mode == SR:
        offs = offsets if offsets is not None else range(len(values))
        return [sr(v, bp, splitmix(key[0], key[1], o)) for v, o in zip(values, offs)], bp
    r = psr if mode == PSR else rtn
    return [r(v, bp) for v in values], bp


def nhwc_offsets(shape):
    """Storage offsets, in NHWC order, of the elements of an [n][c][h][w]
    tensor listed in (n, c, h, w) order (also KRSC offsets of a KCRS filter)."""
    n_, c_, h_, w_ = shape
    return [((n * h_ + h) * w_ + w) * c_ + c
            for n in range(n_) for c in range(c_) for h in range(h_) for w in range(w_)]


def hwc_row(sample):
    """A [c][h][w] sample flattened in (h, w, c) order."""
    c_, h_, w_ = shape_of(sample)
    return [sample[c][h][w] for h in range(h_) for w in range(w_) for c in range(c_)]


# --------------------------------------------------------------- tensors
def zeros(*shape):
    if len(shape) == 1:
        return [0] * shape[0]
    return [zeros(*shape[1:]) for _ in range(shape[0])]


def flat(t):
    if isinstance(t, list):
        out = []
        for e in t:
            out.extend(flat(e))
        return out
    return [t]


def shaped(values, shape):
    it = iter(values)

    def build(dims):
        if len(dims) == 1:
            return [next(it) for _ in range(dims[0])]
        return [build(dims[1:]) for _ in range(dims[0])]
    return build(list(shape))


def shape_of(t):
    s = []
    while isinstance(t, list):
        s.append(len(t))
        t = t[0]
    return tuple(s)


# --------------------------------------------------------------- layers
def conv_sums(x, w, stride, pad):
    """Exact sums of the forward convolution, by its definition."""
    N, C, H, W = shape_of(x)
    K, C2, R, S = shape_of(w)
    assert C2 == C
    P = (H + 2 * pad - R) // stride + 1
    Q = (W + 2 * pad - S) // stride + 1
    y = zeros(N, K, P, Q)
    for n in range(N):
        for k in range(K):
            for p in range(P):
                for q in range(Q):
                    s = 0
                    for c in range(C):
                        for r in range(R):
                            for t in range(S):
                                hh, ww = p * stride - pad + r, q * stride - pad + t
                                if 0 <= hh < H and 0 <= ww < W:
                                    s += w[k][c][r][t] * x[n][c][hh][ww]
                    y[n][k][p][q] = s
    return y


def conv_back_sums(e, w, x_shape, stride, pad):
    """e(l-1) = w (x) e(l): every forward product w[k][c][r][s] x[...] sends
    w[k][c][r][s] e[n][k][p][q] back to the input position it read
    (written as a scatter over forward positions)."""
    N, C, H, W = x_shape
    K, _, R, S = shape_of(w)
    _, _, P, Q = shape_of(e)
    dx = zeros(N, C, H, W)
    for n in range(N):
        for k in range(K):
            for p in range(P):
                for q in range(Q):
                    ev = e[n][k][p][q]
                    for c in range(C):
                        for r in range(R):
                            for t in range(S):
                                hh, ww = p * stride - pad + r, q * stride - pad + t
                                if 0 <= hh < H and 0 <= ww < W:
                                    dx[n][c][hh][ww] += w[k][c][r][t] * ev
    return dx


def conv_grad_sums(x, e, w_shape, stride, pad):
    """g = a(l-1) (x) e(l): each forward product's error times its input,
    gathered onto the filter tap it used (scatter over forward positions)."""
    N, C, H, W = shape_of(x)
    K, _, R, S = w_shape
    _, _, P, Q = shape_of(e)
    g = zeros(K, C, R, S)
    for n in range(N):
        for k in range(K):
            for p in range(P):
                for q in range(Q):
                    ev = e[n][k][p][q]
                    if ev == 0:
                        continue
                    for c in range(C):
                        for r in range(R):
                            for t in range(S):
                                hh, ww = p * stride - pad + r, q * stride - pad + t
                                if 0 <= hh < H and 0 <= ww < W:
                                    g[k][c][r][t] += ev * x[n][c][hh][ww]
    return g


def fc_sums(x, w):
    """x [n][in], w [out][in] -> [n][out] exact sums."""
    return [[sum(a * b for a, b in zip(row, wr)) for wr in w] for row in x]


def pool_fwd(x):
    N, C, H, W = shape_of(x)
    y = zeros(N, C, H // 2, W // 2)
    arg = zeros(N, C, H // 2, W // 2)
    for n in range(N):
        for c in range(C):
            for i in range(H // 2):
                for j in range(W // 2):
                    best, pos = None, 0
                    for t, (di, dj) in enumerate(((0, 0), (0, 1), (1, 0), (1, 1))):
                        v = x[n][c][2 * i + di][2 * j + dj]
                        if best is None or v > best:
                            best, pos = v, t
                    y[n][c][i][j] = best
                    arg[n][c][i][j] = pos
    return y, arg


def pool_bwd(e, arg, x_shape):
    dx = zeros(*x_shape)
    N, C, H2, W2 = shape_of(e)
    for n in range(N):
        for c in range(C):
            for i in range(H2):
                for j in range(W2):
                    t = arg[n][c][i][j]
                    dx[n][c][2 * i + t // 2][2 * j + t % 2] = e[n][c][i][j]
    return dx


# --------------------------------------------------------------- loss
def loss_terms(a, s_a):
    """Unnormalised exponentials t_i of one sample (Section 3.5)."""
    if s_a <= -7:
        # second-order Taylor series of 2^(x ln2)... scaled by 2^(1-2 s_a):
        # (1 + a 2^s_a + a^2 2^(2 s_a) / 2) * 2^(1 - 2 s_a), exact
        u = -s_a
        return [2 ** (1 + 2 * u) + ai * 2 ** (1 + u) + ai * ai for ai in a]
    xh = []
    for ai in a:
        prod = 47274 * ai
        xh.append(prod >> (15 - s_a) if s_a <= 15 else prod << (s_a - 15))
    p = max(xh) - 10
    return [2 ** max(0, v - p) for v in xh]


def loss_grad(logits, s_a, labels, mode, key=None):
    """e_i = t_i - [i = y] sum(t), then one block exponent over the batch,
    rounded with target 7."""
    e32 = []
    for a, y in zip(logits, labels):
        t = loss_terms(a, s_a)
        c = sum(t)
        row = list(t)
        row[y] -= c
        e32.append(row)
    vals, _ = shift_and_round(flat(e32), 7, mode, key)
    return shaped(vals, (len(logits), len(logits[0])))


# --------------------------------------------------------------- the step
def train_step(specs, weights, w_exps, x, s_x, labels, mu=5, mode=PSR, grad_mode=None, t=0, sr_seed=0,
               drop_seed=0):
    """One step of Algorithm 1 over a layer list like the oracle's:
    ("conv", cin, cout, k, stride, pad, relu), ("fc", nin, nout, relu),
    ("pool",), ("dropout", drop256).  weights are updated in place; t is the
    step index (the call count of every statistics block).  Returns
    (logits, s_logits)."""
    grad_mode = mode if grad_mode is None else grad_mode
    acts = []        # the input of each layer
    outs = []        # the int8 output of each layer
    args = {}
    a, s = x, s_x
    wi = 0
    widx = {}
    block = {}
    for i, sp in enumerate(specs):
        acts.append(a)
        if sp[0] == "conv":
            _, _, _, _, st, pd, relu = sp
            block[i] = 3 * wi
            sums = conv_sums(a, weights[wi], st, pd)
            shp = shape_of(sums)
            v = [wrap32(t_) for t_ in flat(sums)]
            if relu:
                v = [max(0, t_) for t_ in v]
            r, bp = shift_and_round(v, 7, mode, (sr_seed + block[i], t), nhwc_offsets(shp))
            a, s = shaped(r, shp), s + w_exps[wi] + bp
            widx[i] = wi
            wi += 1
        elif sp[0] == "fc":
            _, nin, nout, relu = sp
            block[i] = 3 * wi
            rows = [hwc_row(sample) if isinstance(sample[0], list) else list(sample) for sample in a]
            v = [wrap32(t_) for t_ in flat(fc_sums(rows, weights[wi]))]
            if relu:
                v = [max(0, t_) for t_ in v]
            r, bp = shift_and_round(v, 7, mode, (sr_seed + block[i], t))
            a, s = shaped(r, (len(rows), nout)), s + w_exps[wi] + bp
            widx[i] = wi
            wi += 1
        elif sp[0] == "pool":
            a, args[i] = pool_fwd(a)
        else:
            shp = shape_of(a)
            offs = nhwc_offsets(shp) if len(shp) == 4 else list(range(len(flat(a))))
            keep = [1 if (splitmix(drop_seed, t, o) >> 56) >= sp[1] else 0 for o in offs]
            args[i] = keep
            a = shaped([v * k for v, k in zip(flat(a), keep)], shp)
            s = s + (1 if sp[1] == 128 else 0)
        outs.append(a)
    logits, s_logits = a, s
    e = loss_grad(logits, s_logits, labels, mode, (sr_seed + 3 * wi, t))
    for i in range(len(specs) - 1, -1, -1):
        sp = specs[i]
        below = specs[i - 1] if i > 0 else None
        mask_src = acts[i] if below is not None and below[0] in ("conv", "fc") and below[-1] else None
        if sp[0] in ("pool", "dropout"):
            if sp[0] == "pool":
                e = pool_bwd(e, args[i], shape_of(acts[i]))
            else:
                e = shaped([v * k for v, k in zip(flat(e), args[i])], shape_of(e))
            if mask_src is not None:
                e = shaped([0 if m <= 0 else v for v, m in zip(flat(e), flat(mask_src))], shape_of(e))
            continue
        w = weights[widx[i]]
        key_b, key_g = (sr_seed + block[i] + 1, t), (sr_seed + block[i] + 2, t)
        if sp[0] == "conv":
            _, _, _, _, st, pd, _ = sp
            g_sums = conv_grad_sums(acts[i], e, shape_of(w), st, pd)
            g_offs = nhwc_offsets(shape_of(w))
            back = conv_back_sums(e, w, shape_of(acts[i]), st, pd) if i > 0 else None
            back_offs = nhwc_offsets(shape_of(acts[i])) if back is not None else None
        else:
            volume = isinstance(acts[i][0][0], list)
            rows = [hwc_row(sample) if volume else list(sample) for sample in acts[i]]
            g_sums = [[sum(e[n][o] * rows[n][j] for n in range(len(rows))) for j in range(len(rows[0]))]
                      for o in range(len(w))]
            g_offs = None
            back = None
            if i > 0:
                back_rows = [[sum(w[o][j] * e[n][o] for o in range(len(w))) for j in range(len(rows[0]))]
                             for n in range(len(rows))]
                back = back_rows            # [n][hwc]: storage order already
                back_offs = None
        e_next = None
        if back is not None:
            r, _ = shift_and_round([wrap32(t_) for t_ in flat(back)], 7, mode, key_b, back_offs)
            if sp[0] == "fc" and isinstance(acts[i][0][0], list):
                # back to [n][c][h][w] from (n, h, w, c) order
                n_, c_, h_, w_ = shape_of(acts[i])
                r = [r[((n * h_ + h) * w_ + ww) * c_ + c]
                     for n in range(n_) for c in range(c_) for h in range(h_) for ww in range(w_)]
            if mask_src is not None:
                r = [0 if m <= 0 else v for v, m in zip(r, flat(mask_src))]
            e_next = shaped(r, shape_of(acts[i]))
        g, _ = shift_and_round([wrap32(t_) for t_ in flat(g_sums)], mu, grad_mode, key_g, g_offs)
        new_w = [max(-127, min(127, wv - gv)) for wv, gv in zip(flat(w), g)]
        weights[widx[i]] = shaped(new_w, shape_of(w))
        e = e_next
    return logits, s_logits
