"""NITI CPU oracle -- test infrastructure only.

Plain, exact (int64) restatement of the integer-only training method of
"Training Integer Neural Networks Using Integer-only Arithmetic" (NITI,
arXiv 2009.13108).  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package.  It shares no code
with the HIP library and never imports it.

Every function takes and returns numpy arrays.  Activation/error tensors are
NCHW and weights KCRS here (the HIP library's NHWC/KRSC tensors are permuted
by the callers).  The arithmetic lives in ``niti_oracle.c``; this module only
marshals arguments, except for the layer compositions in ``oracle.model``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "niti_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

FLAG_ACC_BOUND = 1    # reduction of 2^17 or more products: int32 sums may wrap
FLAG_EXP_RANGE = 2
FLAG_LOSS_SA = 4
FLAG_ACC_WRAP = 16    # oracle only: an exact sum left the int32 range
ACC_BOUND_LEN = 1 << 17

PSR = 0
RTN = 1
SR = 2


def build(force: bool = False) -> str:
    """Compile ``niti_oracle.c`` into ``liboracle.so`` (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c99",
             "-Wall", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class Stats(ctypes.Structure):
    _fields_ = [("max_abs", ctypes.c_uint64), ("b", ctypes.c_int32),
                ("bp", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("s_out", ctypes.c_int32)]

    def as_dict(self):
        return {"max_abs": int(self.max_abs), "b": int(self.b), "bp": int(self.bp),
                "flags": int(self.flags)}


class Conv(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("n", "c", "h", "w", "k", "r", "s", "sh", "sw", "ph", "pw")]


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            P = ctypes.c_void_p
            I64 = ctypes.c_int64
            I = ctypes.c_int
            U64 = ctypes.c_uint64
            U32 = ctypes.c_uint32
            sig = {
                "orc_bitlen": (I, [ctypes.c_uint64]),
                "orc_psr": (I64, [I64, I]),
                "orc_rtn": (I64, [I64, I]),
                "orc_sr": (I64, [I64, I, U64]),
                "orc_sr_draw": (U64, [U64, U32, U64]),
                "orc_shift_round_i64": (I, [P, I64, I, I, P, P, U64, U32, P]),
                "orc_shift_round_i32": (I, [P, I64, I, I, P, P, U64, U32, P]),
                "orc_round_fixed_i32": (None, [P, I64, I, I, P, U64, U32]),
                "orc_out_exponent": (I, [I, I, I, P]),
                "orc_gemm_nt_raw": (None, [P, P, I64, I64, I64, P]),
                "orc_gemm_nt_pick": (None, [P, P, I64, P, P, I64, P]),
                "orc_conv_fwd_raw": (None, [P, P, P, P]),
                "orc_conv_bwd_data_raw": (None, [P, P, P, P]),
                "orc_conv_bwd_weight_raw": (None, [P, P, P, P]),
                "orc_conv_fwd_one": (I64, [P, P, P, I64, I64, I64, I64]),
                "orc_finish_i64": (None, [P, I64, I, I, I, P, P, P, I64, U64, U32, P]),
                "orc_sgd_update": (None, [P, P, I64, I, I, P, U64, U32]),
                "orc_loss_t_case": (I, [I]),
                "orc_int_ce_loss_grad": (None, [P, I, P, I64, I64, I, P, P, P, P, U64, U32]),
                "orc_relu_mask": (None, [P, P, I64]),
                "orc_maxpool2_fwd": (None, [P, I64, I64, I64, I64, P, P]),
                "orc_maxpool2_bwd": (None, [P, P, I64, I64, I64, I64, P]),
                "orc_quantize_u8": (None, [P, I64, P]),
                "orc_dropout_fwd": (None, [P, P, I64, U64, U32, I, P, P]),
                "orc_dropout_bwd": (None, [P, P, I64, P]),
            }
            for name, (res, args) in sig.items():
                f = getattr(lib, name)
                f.restype = res
                f.argtypes = args
            _lib = lib
    return _lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- scalars
def bitlen(m: int) -> int:
    """Effective bitwidth of a magnitude (Section 3.2)."""
    return _load().orc_bitlen(int(m))


def psr(v: int, bp: int) -> int:
    """Pseudo stochastic rounding of one value (Algorithm 3)."""
    return _load().orc_psr(int(v), int(bp))


def rtn(v: int, bp: int) -> int:
    return _load().orc_rtn(int(v), int(bp))


def out_exponent(s_a: int, s_w: int, bp: int):
    """Output block exponent s_a + s_w + bp (Algorithm 2) and range flag."""
    fl = ctypes.c_int32(0)
    s = _load().orc_out_exponent(int(s_a), int(s_w), int(bp), ctypes.byref(fl))
    return s, fl.value


def loss_case(s_a: int) -> int:
    return _load().orc_loss_t_case(int(s_a))


# ---------------------------------------------------------------- rounding
def sr(v: int, bp: int, draw: int) -> int:
    """Stochastic rounding of one value with a given 64-bit draw (Section 3.4)."""
    return _load().orc_sr(int(v), int(bp), int(draw) & 0xFFFFFFFFFFFFFFFF)


def sr_draw(seed: int, call: int, index: int) -> int:
    """The 64-bit draw of element `index` in call `call` (SplitMix64 stream)."""
    return int(_load().orc_sr_draw(int(seed) & 0xFFFFFFFFFFFFFFFF, int(call), int(index)))


def nhwc_index(shape):
    """Storage offsets in NHWC order of the elements of an NCHW tensor (the
    stochastic draws are keyed by the library's storage order); for a KCRS
    filter the same map gives KRSC offsets."""
    n, c, h, w = shape
    i = np.arange(n * h * w * c, dtype=np.int64).reshape(n, h, w, c)
    return np.ascontiguousarray(i.transpose(0, 3, 1, 2))


def _idx_ptr(idx):
    if idx is None:
        return None, None
    a = np.ascontiguousarray(idx, dtype=np.int64)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def shift_round(v, target: int, mode: int = PSR, sr_seed: int = 0, sr_call: int = 0):
    """Block exponent + rounding of a whole tensor (Algorithms 1-3).

    ``v`` is int32 (accumulators) or int64 (loss values).  Returns
    (int8 array of v's shape, stats dict)."""
    v = np.asarray(v)
    st = Stats()
    out = np.empty(v.shape, np.int8)
    seed = int(sr_seed) & 0xFFFFFFFFFFFFFFFF
    if v.dtype == np.int64:
        vc, pv = _c(v, np.int64)
        _load().orc_shift_round_i64(pv, vc.size, int(target), int(mode), _ptr(out), ctypes.byref(st),
                                    seed, int(sr_call), None)
    else:
        vc, pv = _c(v, np.int32)
        _load().orc_shift_round_i32(pv, vc.size, int(target), int(mode), _ptr(out), ctypes.byref(st),
                                    seed, int(sr_call), None)
    return out, st.as_dict()


def round_fixed(v, bp: int, mode: int = PSR, sr_seed: int = 0, sr_call: int = 0):
    """Round an int32 tensor with a given binary point."""
    vc, pv = _c(v, np.int32)
    out = np.empty(vc.shape, np.int8)
    _load().orc_round_fixed_i32(pv, vc.size, int(bp), int(mode), _ptr(out),
                                int(sr_seed) & 0xFFFFFFFFFFFFFFFF, int(sr_call))
    return out


# ---------------------------------------------------------------- contractions
def gemm_nt_raw(A, B):
    """Exact S = A @ B.T in int64 (A: M x K, B: N x K int8)."""
    A, pa = _c(A, np.int8)
    B, pb = _c(B, np.int8)
    M, K = A.shape
    N, K2 = B.shape
    assert K == K2
    S = np.empty((M, N), np.int64)
    _load().orc_gemm_nt_raw(pa, pb, M, N, K, _ptr(S))
    return S


def gemm_nt_exact(A, B, block_rows=2048):
    """Exact S = A @ B.T for large int8 matrices through a float64 matmul.

    Every product is an integer of magnitude <= 127^2 and every partial sum
    an integer of magnitude <= K * 127^2 < 2^53, so float64 arithmetic (with
    or without fused multiply-add, in any summation order) is exact.  Rows
    are processed in blocks to bound memory."""
    A = np.ascontiguousarray(A, dtype=np.int8)
    B = np.ascontiguousarray(B, dtype=np.int8)
    M, K = A.shape
    N, K2 = B.shape
    assert K == K2 and K * 127 * 127 < 2 ** 53
    Bf = B.astype(np.float64).T.copy()
    S = np.empty((M, N), np.int64)
    for r in range(0, M, block_rows):
        S[r:r + block_rows] = (A[r:r + block_rows].astype(np.float64) @ Bf).astype(np.int64)
    return S


def gemm_nt_pick(A, B, rows, cols):
    """Exact sums S[rows[i], cols[i]] only."""
    A, pa = _c(A, np.int8)
    B, pb = _c(B, np.int8)
    rows, pr = _c(rows, np.int64)
    cols, pc = _c(cols, np.int64)
    S = np.empty(rows.shape, np.int64)
    _load().orc_gemm_nt_pick(pa, pb, A.shape[1], pr, pc, rows.size, _ptr(S))
    return S


def conv_desc(n, c, h, w, k, r, s, stride=1, pad=0):
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    return Conv(n, c, h, w, k, r, s, sh, sw, ph, pw)


def conv_out_hw(d: Conv):
    return ((d.h + 2 * d.ph - d.r) // d.sh + 1, (d.w + 2 * d.pw - d.s) // d.sw + 1)


def conv_fwd_raw(d: Conv, x, w):
    """Exact forward convolution sums, NCHW x KCRS -> NKPQ (int64)."""
    P, Q = conv_out_hw(d)
    x, px = _c(x, np.int8)
    w, pw = _c(w, np.int8)
    assert x.shape == (d.n, d.c, d.h, d.w) and w.shape == (d.k, d.c, d.r, d.s)
    y = np.empty((d.n, d.k, P, Q), np.int64)
    _load().orc_conv_fwd_raw(ctypes.byref(d), px, pw, _ptr(y))
    return y


def conv_bwd_data_raw(d: Conv, dy, w):
    """Exact error back-propagation sums NKPQ x KCRS -> NCHW (int64)."""
    P, Q = conv_out_hw(d)
    dy, pdy = _c(dy, np.int8)
    w, pw = _c(w, np.int8)
    assert dy.shape == (d.n, d.k, P, Q) and w.shape == (d.k, d.c, d.r, d.s)
    dx = np.empty((d.n, d.c, d.h, d.w), np.int64)
    _load().orc_conv_bwd_data_raw(ctypes.byref(d), pdy, pw, _ptr(dx))
    return dx


def conv_bwd_weight_raw(d: Conv, x, dy):
    """Exact weight-gradient sums NCHW x NKPQ -> KCRS (int64)."""
    P, Q = conv_out_hw(d)
    x, px = _c(x, np.int8)
    dy, pdy = _c(dy, np.int8)
    assert x.shape == (d.n, d.c, d.h, d.w) and dy.shape == (d.n, d.k, P, Q)
    g = np.empty((d.k, d.c, d.r, d.s), np.int64)
    _load().orc_conv_bwd_weight_raw(ctypes.byref(d), px, pdy, _ptr(g))
    return g


def conv_fwd_one(d: Conv, x, w, n, k, p, q):
    x, px = _c(x, np.int8)
    w, pw = _c(w, np.int8)
    return _load().orc_conv_fwd_one(ctypes.byref(d), px, pw, n, k, p, q)


# ---------------------------------------------------------------- composites
def finish(S, relu: bool, target: int, mode: int = PSR, red_len: int = 0, sr_seed: int = 0, sr_call: int = 0,
           sr_index=None):
    """Exact sums -> int32 accumulators -> (ReLU) -> block exponent -> int8.
    red_len: products per sum (FLAG_ACC_BOUND when >= 2^17); sr_index: the
    storage-order offset of each element for stochastic draws (default: its
    position in S).

    Returns (int8 out, int32 accumulators, stats dict)."""
    S, ps = _c(S, np.int64)
    out = np.empty(S.shape, np.int8)
    acc = np.empty(S.shape, np.int32)
    st = Stats()
    idx, pidx = _idx_ptr(sr_index)
    _load().orc_finish_i64(ps, S.size, int(bool(relu)), int(target), int(mode),
                           _ptr(out), _ptr(acc), ctypes.byref(st), int(red_len),
                           int(sr_seed) & 0xFFFFFFFFFFFFFFFF, int(sr_call), pidx)
    return out, acc, st.as_dict()


def gemm_fwd(A, B, relu=False, mode=PSR, target=7, sr_seed=0, sr_call=0):
    """Fully-connected / plain GEMM forward step: int8 A (M x K), B (N x K)."""
    return finish(gemm_nt_raw(A, B), relu, target, mode, np.shape(A)[1], sr_seed, sr_call)


def conv_fwd(d, x, w, relu=False, mode=PSR, target=7, sr_seed=0, sr_call=0):
    P, Q = conv_out_hw(d)
    idx = nhwc_index((d.n, d.k, P, Q)) if mode == SR else None
    return finish(conv_fwd_raw(d, x, w), relu, target, mode, d.c * d.r * d.s, sr_seed, sr_call, idx)


def conv_bwd_data(d, dy, w, mode=PSR, relu_src=None, target=7, sr_seed=0, sr_call=0):
    """Error back-propagation step; the optional ReLU mask (reading R5) is
    applied to the rounded int8 error and does not move its exponent."""
    idx = nhwc_index((d.n, d.c, d.h, d.w)) if mode == SR else None
    out, acc, st = finish(conv_bwd_data_raw(d, dy, w), False, target, mode, d.k * d.r * d.s, sr_seed, sr_call,
                          idx)
    if relu_src is not None:
        relu_mask(out, relu_src)
    return out, acc, st


def sgd_update(w, g32, mu: int = 5, mode: int = PSR, sr_seed: int = 0, sr_call: int = 0):
    """Discrete weight update (Section 3.3).  Returns (new w, stats).  The
    stochastic draws are keyed by the flat position in w and g32."""
    w = np.array(w, dtype=np.int8, copy=True, order="C")
    g32, pg = _c(g32, np.int32)
    assert w.size == g32.size
    st = Stats()
    _load().orc_sgd_update(_ptr(w), pg, w.size, int(mu), int(mode), ctypes.byref(st),
                           int(sr_seed) & 0xFFFFFFFFFFFFFFFF, int(sr_call))
    return w, st.as_dict()


def conv_bwd_weight(d, x, dy, w, mu: int = 5, mode: int = PSR, sr_seed: int = 0, sr_call: int = 0):
    """Weight gradient + discrete update.  Returns (new w, g32, stats).  In
    SR mode the draws follow the filter's KRSC storage order."""
    S = conv_bwd_weight_raw(d, x, dy)
    P, Q = conv_out_hw(d)
    fl = np.zeros(1, np.int32)
    g32 = wrap32(S, fl)
    if mode == SR:
        # update in the KRSC order the draws are keyed by, then back to KCRS
        perm = (0, 2, 3, 1)
        w2k, st = sgd_update(np.ascontiguousarray(np.asarray(w).transpose(perm)),
                             np.ascontiguousarray(g32.transpose(perm)), mu, mode, sr_seed, sr_call)
        w2 = np.ascontiguousarray(w2k.transpose(0, 3, 1, 2))
    else:
        w2, st = sgd_update(w, g32, mu, mode)
    st["flags"] |= int(fl[0]) | (FLAG_ACC_BOUND if d.n * P * Q >= ACC_BOUND_LEN else 0)
    return w2, g32, st


def wrap32(S, flags_out=None):
    """int64 exact sums -> int32 two's complement accumulators."""
    S = np.asarray(S, np.int64)
    if flags_out is not None and S.size and (S.max() >= 2 ** 31 or S.min() < -2 ** 31):
        flags_out[0] |= FLAG_ACC_WRAP
    return S.astype(np.uint64).astype(np.uint32).view(np.int32).reshape(S.shape)


def int_ce_loss_grad(logits, s_a: int, labels, mode: int = PSR, sr_seed: int = 0, sr_call: int = 0):
    """Integer cross-entropy gradient (Section 3.5).

    Returns (int8 err [B x N], pre-rounding values, stats dict).  The
    pre-rounding values are an int64 array when they all fit 64 bits, else an
    object array of Python integers (the Taylor branch below s_a = -22)."""
    logits, pl = _c(logits, np.int8)
    labels, plab = _c(labels, np.int32)
    B, N = logits.shape
    assert labels.shape == (B,) and (labels >= 0).all() and (labels < N).all()
    err = np.empty((B, N), np.int8)
    hi = np.empty((B, N), np.int64)
    lo = np.empty((B, N), np.uint64)
    st = Stats()
    _load().orc_int_ce_loss_grad(pl, int(s_a), plab, B, N, int(mode), _ptr(err),
                                 _ptr(hi), _ptr(lo), ctypes.byref(st),
                                 int(sr_seed) & 0xFFFFFFFFFFFFFFFF, int(sr_call))
    lo_signed = lo.view(np.int64)
    fits = ((hi == 0) & (lo_signed >= 0)) | ((hi == -1) & (lo_signed < 0))
    if fits.all():
        e = lo_signed.copy()
    else:
        e = np.empty((B, N), dtype=object)
        for idx in np.ndindex(B, N):
            e[idx] = (int(hi[idx]) << 64) + int(lo[idx])
    return err, e, st.as_dict()


def relu_mask(e, a):
    """In place: e[a <= 0] = 0 (int8 error, int8 stored activation)."""
    assert e.flags["C_CONTIGUOUS"] and e.dtype == np.int8
    a, pa = _c(a, np.int8)
    assert a.size == e.size
    _load().orc_relu_mask(_ptr(e), pa, e.size)
    return e


def maxpool2_fwd(x):
    x, px = _c(x, np.int8)
    n, c, h, w = x.shape
    y = np.empty((n, c, h // 2, w // 2), np.int8)
    idx = np.empty(y.shape, np.uint8)
    _load().orc_maxpool2_fwd(px, n, c, h, w, _ptr(y), _ptr(idx))
    return y, idx


def maxpool2_bwd(dy, idx, shape):
    dy, pdy = _c(dy, np.int8)
    idx, pidx = _c(idx, np.uint8)
    n, c, h, w = shape
    dx = np.empty(shape, np.int8)
    _load().orc_maxpool2_bwd(pdy, pidx, n, c, h, w, _ptr(dx))
    return dx


def quantize_u8(px):
    px, pp = _c(px, np.uint8)
    q = np.empty(px.shape, np.int8)
    _load().orc_quantize_u8(pp, px.size, _ptr(q))
    return q


def dropout_fwd(x, seed: int, call: int, drop256: int = 128, nhwc=True):
    """Dropout of an NCHW tensor (draws keyed by NHWC storage offsets when
    nhwc, else by flat position).  Returns (y, keep)."""
    x, px = _c(x, np.int8)
    idx = nhwc_index(x.shape) if (nhwc and x.ndim == 4) else None
    idx, pidx = _idx_ptr(idx)
    y = np.empty(x.shape, np.int8)
    keep = np.empty(x.shape, np.uint8)
    _load().orc_dropout_fwd(px, pidx, x.size, int(seed) & 0xFFFFFFFFFFFFFFFF, int(call), int(drop256),
                            _ptr(y), _ptr(keep))
    return y, keep


def dropout_bwd(dy, keep):
    dy, pdy = _c(dy, np.int8)
    keep, pk = _c(keep, np.uint8)
    dx = np.empty(dy.shape, np.int8)
    _load().orc_dropout_bwd(pdy, pk, dy.size, _ptr(dx))
    return dx
