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


def same_stats(gpu, orc, keys=("max_abs", "b", "bp")):
    return all(int(gpu[k]) == int(orc[k]) for k in keys)
