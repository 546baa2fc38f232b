"""Shared test plumbing: layout permutations between the oracle's NCHW/KCRS
tensors and the library's NHWC/KRSC tensors, device transfer, and a printout
of each GPU case before it runs (so a failing run names its case)."""
import sys

import numpy as np


def nhwc(x_nchw):
    return np.ascontiguousarray(np.asarray(x_nchw).transpose(0, 2, 3, 1))


def nchw(x_nhwc):
    return np.ascontiguousarray(np.asarray(x_nhwc).transpose(0, 3, 1, 2))


krsc = nhwc   # KCRS -> KRSC is the same permutation
kcrs = nchw


def pad_channels(x_nchw, c_to):
    """Zero channels appended to an NCHW/KCRS tensor (dim 1)."""
    x = np.asarray(x_nchw)
    if x.shape[1] == c_to:
        return x
    pad = np.zeros((x.shape[0], c_to - x.shape[1]) + x.shape[2:], x.dtype)
    return np.concatenate([x, pad], axis=1)


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def say(*args):
    print("[case]", *args, flush=True)
    sys.stdout.flush()


FLAG_HINT_MISS = 8   # library only: the speculated shift was wrong (timing, not a result)
FLAG_ACC_WRAP = 16   # oracle only: an exact sum actually left the int32 range
FLAG_ACC_BOUND = 1   # both: reduction of 2^17 or more products


def same_flags(gpu_flags, orc_flags):
    """Library flags equal the oracle's except for the library's speculation
    bit and the oracle's observed-wrap bit; every observed wrap lies under
    the static accumulator bound the library reports."""
    g, o = int(gpu_flags), int(orc_flags)
    if o & FLAG_ACC_WRAP and not g & FLAG_ACC_BOUND:
        return False
    return (g & ~FLAG_HINT_MISS) == (o & ~FLAG_ACC_WRAP)


def same_stats(gpu, orc, keys=("max_abs", "b", "bp", "flags")):
    for k in keys:
        if k == "flags":
            if not same_flags(gpu[k], orc[k]):
                return False
        elif int(gpu[k]) != int(orc[k]):
            return False
    return True
