"""ctypes binding of libniti.so (the C ABI in include/niti.h).

Argument marshalling only: every function checks tensor dtypes, devices and
contiguity, derives the sizes the C call needs and calls it on torch's
current HIP stream.  All arithmetic runs in the library's HIP kernels; if
the library has not been built this module raises instead of computing
anything another way.
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libniti.so")

PSR = 0
RTN = 1
SR = 2

FLAG_ACC_BOUND = 1
FLAG_EXP_RANGE = 2
FLAG_LOSS_SA = 4
FLAG_HINT_MISS = 8

OP_GEMM_FWD = 0
OP_CONV_FWD = 1
OP_CONV_BWD_DATA = 2
OP_CONV_BWD_WEIGHT = 3
OP_INT_CE_LOSS = 4

STATS_BYTES = 128
STATS_DTYPE = np.dtype([
    ("max_abs", "<u8"), ("b", "<i4"), ("bp", "<i4"), ("flags", "<i4"), ("s_out", "<i4"),
    ("bp_hint", "<i4"), ("calls", "<u4"), ("misses", "<u4"), ("reserved0", "<u4"),
    ("acc_max", "<u8", (2,)), ("wflags", "<u4", (2,)), ("cur", "<i4"), ("hint_used", "<i4"),
    ("sr_seed", "<u8"), ("sr_call", "<u4"), ("reserved", "<u4", (11,)),
])
assert STATS_DTYPE.itemsize == STATS_BYTES


class NitiError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__("%s: %s (status %d)" % (what, status_str(status), status))
        self.status = status


class ConvDesc(ctypes.Structure):
    """niti_conv_desc: NHWC input [n][h][w][c], KRSC filter [k][r][s][c]."""
    _fields_ = [("n", ctypes.c_int64), ("h", ctypes.c_int64), ("w", ctypes.c_int64),
                ("c", ctypes.c_int64), ("k", ctypes.c_int64), ("r", ctypes.c_int64),
                ("s", ctypes.c_int64), ("stride_h", ctypes.c_int32), ("stride_w", ctypes.c_int32),
                ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32)]

    @classmethod
    def make(cls, n, h, w, c, k, r, s, stride=1, pad=0):
        return cls(n, h, w, c, k, r, s, stride, stride, pad, pad)

    @property
    def p(self):
        return (self.h + 2 * self.pad_h - self.r) // self.stride_h + 1

    @property
    def q(self):
        return (self.w + 2 * self.pad_w - self.s) // self.stride_w + 1

    def x_shape(self):
        return (self.n, self.h, self.w, self.c)

    def w_shape(self):
        return (self.k, self.r, self.s, self.c)

    def y_shape(self):
        return (self.n, self.p, self.q, self.k)


_lock = threading.Lock()
_lib = None

EXPORTS = [
    "niti_gemm_fwd", "niti_conv_fwd", "niti_conv_bwd_data", "niti_conv_pack_bwd_data",
    "niti_conv_bwd_data_packed", "niti_conv_bwd_weight", "niti_conv_bwd_weight_noalloc",
    "niti_round_psr", "niti_int_ce_loss_grad", "niti_sgd_update", "niti_workspace_bytes",
    "niti_status_str", "niti_quantize_u8", "niti_maxpool2_fwd", "niti_maxpool2_bwd",
    "niti_relu_mask", "niti_dropout_fwd", "niti_dropout_bwd", "niti_stats_bytes", "niti_timing_enable", "niti_timing_read", "niti_timing_record",
    "niti_mfma_loop",
]

TIMING_IGEMM = 0
TIMING_WGRAD = 1
TIMING_KERNEL = 2
TIMING_SUM = 3
TIMING_UPDATE = 4
TIMING_LOSS = 5


def lib():
    """Load libniti.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError("libniti.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
            L = ctypes.CDLL(LIB_PATH)
            P, I64, I, Z = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
            sig = {
                "niti_gemm_fwd": [P, P, P, I64, I64, I64, P, P, P, I, I, I, P, P],
                "niti_conv_fwd": [P, P, P, P, P, P, P, I, I, P, P, Z, P],
                "niti_conv_bwd_data": [P, P, P, P, P, I, P, P, Z, P],
                "niti_conv_pack_bwd_data": [P, P, P, Z, P],
                "niti_conv_bwd_data_packed": [P, P, P, P, P, I, P, Z, P],
                "niti_conv_bwd_weight": [P, P, P, P, P, I, I, P, P, Z, P],
                "niti_conv_bwd_weight_noalloc": [P, P, P, P, P, I, I, P, P],
                "niti_round_psr": [P, P, I64, I, I, I, P, P, P, P],
                "niti_int_ce_loss_grad": [P, P, P, P, I64, I64, I, P, P, Z, P],
                "niti_sgd_update": [P, P, I64, I, I, P, P],
                "niti_quantize_u8": [P, P, I64, I64, I64, I64, I64, P],
                "niti_maxpool2_fwd": [P, P, P, I64, I64, I64, I64, P],
                "niti_maxpool2_bwd": [P, P, P, I64, I64, I64, I64, P],
                "niti_relu_mask": [P, P, I64, P],
                "niti_dropout_fwd": [P, P, P, I64, ctypes.c_uint64, ctypes.c_uint32, I, P, P, I, P],
                "niti_dropout_bwd": [P, P, P, I64, P],
                "niti_timing_enable": [I],
                "niti_timing_read": [I, P, P],
                "niti_timing_record": [I64, P, P, P],
                "niti_mfma_loop": [I64, I64, P, P],
            }
            for name, args in sig.items():
                f = getattr(L, name)
                f.argtypes = args
                f.restype = ctypes.c_int
            L.niti_workspace_bytes.argtypes = [I, P, I64, I64, I64]
            L.niti_workspace_bytes.restype = Z
            L.niti_status_str.argtypes = [I]
            L.niti_status_str.restype = ctypes.c_char_p
            L.niti_stats_bytes.argtypes = []
            L.niti_stats_bytes.restype = Z
            assert L.niti_stats_bytes() == STATS_BYTES
            _lib = L
    return _lib


def status_str(s: int) -> str:
    return lib().niti_status_str(int(s)).decode()


def timing_enable(on: bool):
    """Start (clearing earlier records) or stop the library's kernel timing."""
    _check(lib().niti_timing_enable(int(bool(on))), "niti_timing_enable")


def timing_read(family: int):
    """(summed milliseconds, calls) of a timing family; waits for its events."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().niti_timing_read(int(family), ctypes.byref(ms), ctypes.byref(n)), "niti_timing_read")
    return ms.value, n.value


def mfma_loop(iters, workgroups, out, stream=None):
    """Matrix-core rate check: workgroups x 4 waves x iters x 8 int8 MFMAs
    of 65536 operations; out is an int32 device tensor of at least
    workgroups * 256 elements."""
    torch = _torch()
    _dev(out, torch.int32, "out")
    if out.numel() < workgroups * 256:
        raise ValueError("mfma_loop: out too small")
    _run("niti_mfma_loop", int(iters), int(workgroups), _ptr(out), _stream(stream))


def timing_records():
    """Every timing record in enqueue order: (family, label, milliseconds)."""
    out = []
    fam = ctypes.c_int(0)
    name = ctypes.c_char_p()
    ms = ctypes.c_double(0.0)
    i = 0
    while True:
        st = lib().niti_timing_record(i, ctypes.byref(fam), ctypes.byref(name), ctypes.byref(ms))
        if st == -6:
            return out
        _check(st, "niti_timing_record")
        out.append((fam.value, name.value.decode(), ms.value))
        i += 1


# ------------------------------------------------------------------ helpers
def _torch():
    import torch
    return torch


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _dev(t, dtype, what):
    torch = _torch()
    if t is None:
        return
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a device tensor" % what)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (what, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(st, what):
    if st != 0:
        raise NitiError(st, what)


# Prepared calls: while a recorder list is set, every entry point appends
# (function, marshalled arguments, name) after checking its arguments and
# running.  replay() reissues such a list without the Python-side checks,
# for callers that enqueue the same calls (same tensors, streams, stats)
# every step.
_recorder = None


def _run(name, *args):
    f = getattr(lib(), name)
    if _recorder is not None:
        _recorder.append((f, args, name))
    _check(f(*args), name)


class recording:
    """with niti.recording() as calls: ... -> calls lists the entry-point calls made."""

    def __enter__(self):
        global _recorder
        self.calls = []
        _recorder = self.calls
        return self.calls

    def __exit__(self, *exc):
        global _recorder
        _recorder = None
        return False


def _kept(fn):
    """A recorded non-library operation: runs fn and reports success."""
    def run():
        fn()
        return 0
    return run


def stream_record(event, stream):
    """Record an event (torch.cuda.Event or stream_event.StreamEvent) on a
    stream, to order work across streams; kept in an active recording, so
    that replay() issues it again in place."""
    event.record(stream)
    if _recorder is not None:
        _recorder.append((_kept(lambda: event.record(stream)), (), "event record"))


def stream_wait(stream, event):
    """Make a stream wait for an event's last record; kept in an active
    recording like stream_record."""
    event.wait(stream)
    if _recorder is not None:
        _recorder.append((_kept(lambda: event.wait(stream)), (), "event wait"))


def replay(calls):
    """Reissue recorded calls (see recording); raises on the first error."""
    for f, args, name in calls:
        st = f(*args)
        if st != 0:
            raise NitiError(st, name)


def _stats_ptr(stats, index=0):
    torch = _torch()
    _dev(stats, torch.uint8, "stats")
    if stats.numel() < STATS_BYTES * (index + 1):
        raise ValueError("stats tensor too small")
    return ctypes.c_void_p(stats.data_ptr() + STATS_BYTES * index)


def new_stats(count: int = 1, device="cuda"):
    """Zero-filled niti_stats blocks (count x 128 bytes of device memory)."""
    torch = _torch()
    return torch.zeros((count, STATS_BYTES), dtype=torch.uint8, device=device)


def set_sr_seed(stats, seed: int, index=None):
    """Write the stochastic-rounding seed into stats blocks (all, or one)."""
    torch = _torch()
    val = int(seed) & 0xFFFFFFFFFFFFFFFF
    if val >= 1 << 63:
        val -= 1 << 64
    v = torch.tensor([val], dtype=torch.int64).view(torch.uint8).to(stats.device)
    off = STATS_DTYPE.fields["sr_seed"][1]
    rows = stats.view(-1, STATS_BYTES)
    if index is None:
        rows[:, off:off + 8] = v
    else:
        rows[index, off:off + 8] = v


def read_stats(stats):
    """Copy stats blocks to the host: list of dicts."""
    raw = stats.detach().reshape(-1, STATS_BYTES).cpu().numpy().copy()
    recs = raw.view(STATS_DTYPE).reshape(-1)
    out = []
    for r in recs:
        out.append({k: (int(r[k]) if r[k].shape == () else [int(v) for v in r[k]])
                    for k in STATS_DTYPE.names if not k.startswith("reserved")})
    return out


def workspace_bytes(op: int, desc: ConvDesc | None = None, M: int = 0, N: int = 0, K: int = 0) -> int:
    return int(lib().niti_workspace_bytes(int(op), ctypes.byref(desc) if desc is not None else None,
                                          int(M), int(N), int(K)))


def new_workspace(nbytes: int, device="cuda"):
    torch = _torch()
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _exp3(a, b, c, what):
    torch = _torch()
    given = [t is not None for t in (a, b, c)]
    if any(given) and not all(given):
        raise ValueError("%s: give all three exponents or none" % what)
    for t in (a, b, c):
        _dev(t, torch.int8, "exponent")


# ------------------------------------------------------------------ C ABI
def gemm_fwd(A, B, C, stats, s_a=None, s_b=None, s_c=None, target_bits=7, relu=False, mode=PSR,
             stats_index=0, stream=None):
    """C[M][N] = round(A[M][K] B[N][K]^T) (niti_gemm_fwd)."""
    torch = _torch()
    _dev(A, torch.int8, "A"); _dev(B, torch.int8, "B"); _dev(C, torch.int8, "C")
    M, K = A.shape
    N, K2 = B.shape
    if K2 != K or tuple(C.shape) != (M, N):
        raise ValueError("gemm_fwd: shapes %s %s %s" % (tuple(A.shape), tuple(B.shape), tuple(C.shape)))
    _exp3(s_a, s_b, s_c, "gemm_fwd")
    _run("niti_gemm_fwd", _ptr(A), _ptr(B), _ptr(C), M, N, K, _ptr(s_a), _ptr(s_b), _ptr(s_c),
                               int(target_bits), int(bool(relu)), int(mode),
                               _stats_ptr(stats, stats_index), _stream(stream))


def _conv_check(d: ConvDesc, **tensors):
    torch = _torch()
    shapes = {"x": d.x_shape(), "w": d.w_shape(), "y": d.y_shape(), "dy": d.y_shape(),
              "dx": d.x_shape(), "relu_src": d.x_shape()}
    for name, t in tensors.items():
        if t is None:
            continue
        _dev(t, torch.int8, name)
        if tuple(t.shape) != tuple(shapes[name]):
            raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), shapes[name]))


def conv_fwd(d: ConvDesc, x, w, y, stats, s_x=None, s_w=None, s_y=None, relu=False, mode=PSR,
             stats_index=0, ws=None, stream=None):
    """Forward convolution; ws is needed when workspace_bytes(OP_CONV_FWD, d) > 0."""
    torch = _torch()
    _conv_check(d, x=x, w=w, y=y)
    _exp3(s_x, s_w, s_y, "conv_fwd")
    if ws is not None:
        _dev(ws, torch.uint8, "ws")
    _run("niti_conv_fwd", ctypes.byref(d), _ptr(x), _ptr(w), _ptr(y), _ptr(s_x), _ptr(s_w),
                               _ptr(s_y), int(bool(relu)), int(mode), _stats_ptr(stats, stats_index),
                               _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream))


def conv_bwd_data(d: ConvDesc, dy, w, dx, stats, ws, relu_src=None, mode=PSR, stats_index=0, stream=None):
    torch = _torch()
    _conv_check(d, dy=dy, w=w, dx=dx, relu_src=relu_src)
    _dev(ws, torch.uint8, "ws")
    _run("niti_conv_bwd_data", ctypes.byref(d), _ptr(dy), _ptr(w), _ptr(dx), _ptr(relu_src), int(mode),
                                    _stats_ptr(stats, stats_index), _ptr(ws), ws.numel(), _stream(stream))


def conv_pack_bwd_data(d: ConvDesc, w, packed, stream=None):
    torch = _torch()
    _conv_check(d, w=w)
    _dev(packed, torch.uint8, "packed")
    _run("niti_conv_pack_bwd_data", ctypes.byref(d), _ptr(w), _ptr(packed), packed.numel(), _stream(stream))


def conv_bwd_data_packed(d: ConvDesc, dy, packed, dx, stats, relu_src=None, mode=PSR, stats_index=0, stream=None):
    torch = _torch()
    _conv_check(d, dy=dy, dx=dx, relu_src=relu_src)
    _dev(packed, torch.uint8, "packed")
    _run("niti_conv_bwd_data_packed", ctypes.byref(d), _ptr(dy), _ptr(packed), _ptr(dx), _ptr(relu_src), int(mode),
         _stats_ptr(stats, stats_index), packed.numel(), _stream(stream))


def conv_bwd_weight(d: ConvDesc, x, dy, w, stats, ws=None, g32_out=None, mu=5, mode=PSR, stats_index=0,
                    stream=None):
    torch = _torch()
    _conv_check(d, x=x, dy=dy, w=w)
    if g32_out is not None:
        _dev(g32_out, torch.int32, "g32_out")
        if tuple(g32_out.shape) != tuple(d.w_shape()):
            raise ValueError("g32_out shape")
    if ws is not None:
        _dev(ws, torch.uint8, "ws")
    _run("niti_conv_bwd_weight", ctypes.byref(d), _ptr(x), _ptr(dy), _ptr(w), _ptr(g32_out), int(mu),
                                      int(mode), _stats_ptr(stats, stats_index), _ptr(ws),
                                      ws.numel() if ws is not None else 0, _stream(stream))


NOALLOC_SCRATCH_BYTES = 64 << 20


def conv_bwd_weight_noalloc(d: ConvDesc, x, dy, w, stats, g32_out=None, mu=5, mode=PSR, stats_index=0,
                            stream=None):
    """conv_bwd_weight with the library's fixed per-GPU scratch array in place of a workspace."""
    torch = _torch()
    _conv_check(d, x=x, dy=dy, w=w)
    if g32_out is not None:
        _dev(g32_out, torch.int32, "g32_out")
        if tuple(g32_out.shape) != tuple(d.w_shape()):
            raise ValueError("g32_out shape")
    _run("niti_conv_bwd_weight_noalloc", ctypes.byref(d), _ptr(x), _ptr(dy), _ptr(w), _ptr(g32_out), int(mu),
         int(mode), _stats_ptr(stats, stats_index), _stream(stream))


def round_psr(x, y, bp=-1, target_bits=7, stats=None, s_in=None, s_out=None, mode=PSR, stats_index=0,
              stream=None):
    torch = _torch()
    _dev(x, torch.int32, "x"); _dev(y, torch.int8, "y")
    if x.numel() != y.numel():
        raise ValueError("round_psr: sizes differ")
    _dev(s_in, torch.int8, "s_in"); _dev(s_out, torch.int8, "s_out")
    sp = _stats_ptr(stats, stats_index) if stats is not None else None
    _run("niti_round_psr", _ptr(x), _ptr(y), x.numel(), int(bp), int(target_bits), int(mode),
                                _ptr(s_in), _ptr(s_out), sp, _stream(stream))


def int_ce_loss_grad(logits, s_logits, labels, err, stats, ws, mode=PSR, stats_index=0, stream=None):
    torch = _torch()
    _dev(logits, torch.int8, "logits"); _dev(s_logits, torch.int8, "s_logits")
    _dev(labels, torch.int32, "labels"); _dev(err, torch.int8, "err"); _dev(ws, torch.uint8, "ws")
    B, N = logits.shape
    if tuple(err.shape) != (B, N) or tuple(labels.shape) != (B,):
        raise ValueError("int_ce_loss_grad: shapes")
    _run("niti_int_ce_loss_grad", _ptr(logits), _ptr(s_logits), _ptr(labels), _ptr(err), B, N,
                                       int(mode), _stats_ptr(stats, stats_index), _ptr(ws), ws.numel(),
                                       _stream(stream))


def sgd_update(w, g32, stats, mu=5, mode=PSR, stats_index=0, stream=None):
    torch = _torch()
    _dev(w, torch.int8, "w"); _dev(g32, torch.int32, "g32")
    if w.numel() != g32.numel():
        raise ValueError("sgd_update: sizes differ")
    _run("niti_sgd_update", _ptr(w), _ptr(g32), w.numel(), int(mu), int(mode),
                                 _stats_ptr(stats, stats_index), _stream(stream))


# ------------------------------------------------------------------ glue
def quantize_u8(px, x, stream=None):
    """px uint8 NCHW [n][c][h][w] -> x int8 NHWC [n][h][w][c_pad]."""
    torch = _torch()
    _dev(px, torch.uint8, "px"); _dev(x, torch.int8, "x")
    n, c, h, w = px.shape
    if tuple(x.shape[:3]) != (n, h, w) or x.shape[3] < c:
        raise ValueError("quantize_u8: shapes")
    _run("niti_quantize_u8", _ptr(px), _ptr(x), n, c, h, w, x.shape[3], _stream(stream))


def maxpool2_fwd(x, y, idx, stream=None):
    torch = _torch()
    _dev(x, torch.int8, "x"); _dev(y, torch.int8, "y"); _dev(idx, torch.uint8, "idx")
    n, h, w, c = x.shape
    if tuple(y.shape) != (n, h // 2, w // 2, c) or tuple(idx.shape) != tuple(y.shape):
        raise ValueError("maxpool2_fwd: shapes")
    _run("niti_maxpool2_fwd", _ptr(x), _ptr(y), _ptr(idx), n, h, w, c, _stream(stream))


def maxpool2_bwd(dy, idx, dx, stream=None):
    torch = _torch()
    _dev(dy, torch.int8, "dy"); _dev(idx, torch.uint8, "idx"); _dev(dx, torch.int8, "dx")
    n, h, w, c = dx.shape
    if tuple(dy.shape) != (n, h // 2, w // 2, c) or tuple(idx.shape) != tuple(dy.shape):
        raise ValueError("maxpool2_bwd: shapes")
    _run("niti_maxpool2_bwd", _ptr(dy), _ptr(idx), _ptr(dx), n, h, w, c, _stream(stream))


def relu_mask(e, a, stream=None):
    torch = _torch()
    _dev(e, torch.int8, "e"); _dev(a, torch.int8, "a")
    if e.numel() != a.numel():
        raise ValueError("relu_mask: sizes differ")
    _run("niti_relu_mask", _ptr(e), _ptr(a), e.numel(), _stream(stream))


def dropout_fwd(x, y, keep, seed: int, call: int, drop256: int = 128, s_x=None, s_y=None, exp_add: int = 0,
                stream=None):
    """y = x where the draw keeps the element (probability 1 - drop256/256),
    else 0; *s_y = *s_x + exp_add when the exponents are given."""
    torch = _torch()
    _dev(x, torch.int8, "x"); _dev(y, torch.int8, "y"); _dev(keep, torch.uint8, "keep")
    _dev(s_x, torch.int8, "s_x"); _dev(s_y, torch.int8, "s_y")
    if not (x.numel() == y.numel() == keep.numel()):
        raise ValueError("dropout_fwd: sizes differ")
    _run("niti_dropout_fwd", _ptr(x), _ptr(y), _ptr(keep), x.numel(), int(seed) & 0xFFFFFFFFFFFFFFFF, int(call),
         int(drop256), _ptr(s_x), _ptr(s_y), int(exp_add), _stream(stream))


def dropout_bwd(dy, keep, dx, stream=None):
    torch = _torch()
    _dev(dy, torch.int8, "dy"); _dev(keep, torch.uint8, "keep"); _dev(dx, torch.int8, "dx")
    if not (dy.numel() == dx.numel() == keep.numel()):
        raise ValueError("dropout_bwd: sizes differ")
    _run("niti_dropout_bwd", _ptr(dy), _ptr(keep), _ptr(dx), dy.numel(), _stream(stream))
