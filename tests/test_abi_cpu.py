"""The C ABI library loads without a GPU, exports every symbol its header
declares, and rejects bad arguments on the host before launching anything."""
import ctypes
import os
import re

import pytest

from paper_2009_13108_amd import niti

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "niti.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(niti_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_seven_hot_path_calls():
    names = declared_functions()
    for n in ["niti_gemm_fwd", "niti_conv_fwd", "niti_conv_bwd_data", "niti_conv_bwd_weight",
              "niti_round_psr", "niti_int_ce_loss_grad", "niti_sgd_update"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    L = niti.lib()
    for n in declared_functions():
        assert hasattr(L, n), n
    assert set(declared_functions()) == set(niti.EXPORTS)


def test_stats_layout_matches_header():
    assert niti.lib().niti_stats_bytes() == 128 == niti.STATS_DTYPE.itemsize


def test_status_strings():
    for s in range(0, -7, -1):
        assert isinstance(niti.status_str(s), str) and niti.status_str(s)


def test_workspace_sizes():
    d = niti.ConvDesc.make(2, 8, 8, 64, 128, 3, 3, 1, 1)
    assert niti.workspace_bytes(niti.OP_CONV_BWD_DATA, d) >= 128 * 9 * 64
    assert niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, d) >= 128 * 9 * 64 * 4
    assert niti.workspace_bytes(niti.OP_INT_CE_LOSS, None, 128, 1000) >= 128 * 1000 * 8
    assert niti.workspace_bytes(niti.OP_CONV_FWD, d) == 0


FAKE = ctypes.c_void_p(0x100000)   # never dereferenced: every call below fails validation


def test_gemm_rejects_on_host():
    L = niti.lib()
    S = FAKE
    assert L.niti_gemm_fwd(None, FAKE, FAKE, 4, 4, 4, None, None, None, 7, 0, 0, S, None) == -1
    assert L.niti_gemm_fwd(FAKE, FAKE, None, 4, 4, 0, None, None, None, 7, 0, 0, S, None) == -1
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 0, 4, 4, None, None, None, 7, 0, 0, S, None) == -2
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 4, 4, -1, None, None, None, 7, 0, 0, S, None) == -2
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 4, 4, 4, None, None, None, 0, 0, 0, S, None) == -6
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 4, 4, 4, None, None, None, 7, 0, 5, S, None) == -6
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 4, 4, 4, FAKE, None, None, 7, 0, 0, S, None) == -1
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 4, 4, 4, None, None, None, 7, 0, 0, None, None) == -1
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 1 << 20, 1 << 20, 4, None, None, None, 7, 0, 0, S, None) == -3
    # an operand of exactly 2^31 bytes (A: 2^27 x 16) is past the 32-bit offsets
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 1 << 27, 16, 16, None, None, None, 7, 0, 0, S, None) == -3
    assert L.niti_gemm_fwd(FAKE, FAKE, FAKE, 16, 1 << 27, 16, None, None, None, 7, 0, 0, S, None) == -3


def test_conv_rejects_on_host():
    L = niti.lib()
    d = niti.ConvDesc.make(2, 8, 8, 3, 16, 3, 3, 1, 1)           # c % 4 != 0
    assert L.niti_conv_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, None, None, None, 0, 0, FAKE, None, 0, None) == -3
    d = niti.ConvDesc.make(2, 32, 32, 4, 16, 3, 3, 9, 1)         # stride 9
    assert L.niti_conv_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, None, None, None, 0, 0, FAKE, None, 0, None) == -3
    assert L.niti_conv_bwd_weight(ctypes.byref(d), FAKE, FAKE, FAKE, None, 5, 0, FAKE, FAKE, 1 << 20, None) == -3
    d = niti.ConvDesc.make(2, 8, 8, 4, 16, 3, 3, 3, 1)           # stride 3: no back-propagation
    assert L.niti_workspace_bytes(niti.OP_CONV_BWD_DATA, ctypes.byref(d), 0, 0, 0) == 0
    assert L.niti_conv_bwd_data(ctypes.byref(d), FAKE, FAKE, FAKE, None, 0, FAKE, FAKE, 1 << 20, None) == -3
    assert L.niti_conv_pack_bwd_data(ctypes.byref(d), FAKE, FAKE, 1 << 20, None) == -3
    assert L.niti_conv_bwd_data_packed(ctypes.byref(d), FAKE, FAKE, FAKE, None, 0, FAKE, 1 << 20, None) == -3
    assert L.niti_workspace_bytes(niti.OP_CONV_FWD, ctypes.byref(d), 0, 0, 0) > 0   # few channels: window copy
    d = niti.ConvDesc.make(2, 2, 2, 4, 16, 5, 5, 1, 0)           # filter larger than padded input
    assert L.niti_conv_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, None, None, None, 0, 0, FAKE, None, 0, None) == -2
    d = niti.ConvDesc.make(2, 8, 8, 4, 16, 3, 3, 1, 1)
    assert L.niti_conv_fwd(None, FAKE, FAKE, FAKE, None, None, None, 0, 0, FAKE, None, 0, None) == -1
    assert L.niti_conv_bwd_data(ctypes.byref(d), FAKE, FAKE, FAKE, None, 0, FAKE, None, 0, None) == -4
    assert L.niti_conv_bwd_data(ctypes.byref(d), FAKE, FAKE, FAKE, None, 0, FAKE, FAKE, 16, None) == -4
    assert L.niti_conv_bwd_weight(ctypes.byref(d), FAKE, FAKE, FAKE, None, 5, 0, FAKE, None, 0, None) == -4
    assert L.niti_conv_bwd_weight(ctypes.byref(d), FAKE, FAKE, FAKE, None, 0, 0, FAKE, FAKE, 1 << 20, None) == -6
    assert L.niti_conv_bwd_weight(ctypes.byref(d), FAKE, FAKE, FAKE, None, 9, 0, FAKE, FAKE, 1 << 20, None) == -6


def test_other_calls_reject_on_host():
    L = niti.lib()
    assert L.niti_round_psr(FAKE, FAKE, -1, 3, 7, 0, None, None, None, None) == -2
    assert L.niti_round_psr(FAKE, FAKE, 10, -1, 7, 0, None, None, None, None) == -1   # derive needs stats
    assert L.niti_round_psr(FAKE, FAKE, 10, 32, 7, 0, None, None, None, None) == -6
    assert L.niti_round_psr(FAKE, FAKE, 10, 3, 7, 0, FAKE, None, None, None) == -1
    assert L.niti_int_ce_loss_grad(FAKE, FAKE, FAKE, FAKE, 4, 10, 0, FAKE, None, 0, None) == -4
    assert L.niti_int_ce_loss_grad(FAKE, FAKE, FAKE, FAKE, 4, 100000, 0, FAKE, FAKE, 1 << 30, None) == -6
    assert L.niti_int_ce_loss_grad(FAKE, None, FAKE, FAKE, 4, 10, 0, FAKE, FAKE, 1 << 20, None) == -1
    assert L.niti_sgd_update(FAKE, FAKE, 10, 0, 0, FAKE, None) == -6
    assert L.niti_sgd_update(FAKE, FAKE, 10, 5, 0, None, None) == -1
    assert L.niti_maxpool2_fwd(FAKE, FAKE, FAKE, 1, 3, 4, 4, None) == -2
    assert L.niti_quantize_u8(FAKE, FAKE, 1, 3, 4, 4, 2, None) == -2
    assert L.niti_relu_mask(FAKE, FAKE, -4, None) == -2
    # dropout: size, missing buffers, one exponent pointer without the other, rate and exponent step ranges
    assert L.niti_dropout_fwd(FAKE, FAKE, FAKE, -1, 0, 0, 128, None, None, 1, None) == -2
    assert L.niti_dropout_fwd(None, FAKE, FAKE, 16, 0, 0, 128, None, None, 1, None) == -1
    assert L.niti_dropout_fwd(FAKE, FAKE, FAKE, 16, 0, 0, 128, FAKE, None, 1, None) == -1
    assert L.niti_dropout_fwd(FAKE, FAKE, FAKE, 16, 0, 0, 257, None, None, 1, None) == -6
    assert L.niti_dropout_fwd(FAKE, FAKE, FAKE, 16, 0, 0, -1, None, None, 1, None) == -6
    assert L.niti_dropout_fwd(FAKE, FAKE, FAKE, 16, 0, 0, 128, FAKE, FAKE, 9, None) == -6
    assert L.niti_dropout_bwd(FAKE, FAKE, FAKE, -1, None) == -2
    assert L.niti_dropout_bwd(FAKE, None, FAKE, 16, None) == -1
    # the matrix-core rate check
    assert L.niti_mfma_loop(16, 4, None, None) == -1
    assert L.niti_mfma_loop(-1, 4, FAKE, None) == -2
    assert L.niti_mfma_loop(16, 0, FAKE, None) == -2
    assert L.niti_mfma_loop(16, (1 << 20) + 1, FAKE, None) == -2


def test_conv_fwd_workspace_rules():
    """Few-channel layers need a forward workspace; wide ones need none."""
    L = niti.lib()
    stem = niti.ConvDesc.make(128, 224, 224, 4, 64, 7, 7, 2, 3)
    need = niti.workspace_bytes(niti.OP_CONV_FWD, stem)
    # padded 230x230 image copy plus 64 filters of 7 rows x 32 bytes (rounded to 256 bytes)
    assert need == 128 * 230 * 230 * 4 + 64 * 256
    assert L.niti_conv_fwd(ctypes.byref(stem), FAKE, FAKE, FAKE, None, None, None, 0, 0, FAKE,
                           None, 0, None) == -4
    assert L.niti_conv_fwd(ctypes.byref(stem), FAKE, FAKE, FAKE, None, None, None, 0, 0, FAKE,
                           FAKE, need - 1, None) == -4
    wide = niti.ConvDesc.make(8, 14, 14, 64, 64, 3, 3, 1, 1)
    assert niti.workspace_bytes(niti.OP_CONV_FWD, wide) == 0
    # the weight-gradient workspace of a few-channel layer also holds the padded copy
    assert niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, stem) > 128 * 230 * 230 * 4


def test_misaligned_pointers_rejected():
    L = niti.lib()
    odd = ctypes.c_void_p(0x100008)
    S = FAKE
    assert L.niti_gemm_fwd(odd, FAKE, FAKE, 4, 4, 16, None, None, None, 7, 0, 0, S, None) == -6
    d = niti.ConvDesc.make(2, 8, 8, 64, 16, 3, 3, 1, 1)
    assert L.niti_conv_fwd(ctypes.byref(d), FAKE, FAKE, odd, None, None, None, 0, 0, FAKE,
                           None, 0, None) == -6
    assert L.niti_sgd_update(FAKE, odd, 16, 5, 0, S, None) == -6


def test_noalloc_weight_gradient_rejects_on_host():
    """The workspace-free weight gradient checks its arguments and the size
    of its fixed scratch array before it touches any device."""
    L = niti.lib()
    big = niti.ConvDesc.make(256, 224, 224, 4, 64, 7, 7, 2, 3)       # ~88 MiB of temporary memory
    assert niti.workspace_bytes(niti.OP_CONV_BWD_WEIGHT, big) > niti.NOALLOC_SCRATCH_BYTES
    assert L.niti_conv_bwd_weight_noalloc(ctypes.byref(big), FAKE, FAKE, FAKE, None, 5, 0, FAKE, None) == -4
    d = niti.ConvDesc.make(2, 8, 8, 64, 16, 3, 3, 1, 1)
    assert L.niti_conv_bwd_weight_noalloc(None, FAKE, FAKE, FAKE, None, 5, 0, FAKE, None) == -1
    assert L.niti_conv_bwd_weight_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, None, 5, 0, None, None) == -1
    assert L.niti_conv_bwd_weight_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, None, 9, 0, FAKE, None) == -6
    odd = niti.ConvDesc.make(2, 8, 8, 3, 16, 3, 3, 1, 1)
    assert L.niti_conv_bwd_weight_noalloc(ctypes.byref(odd), FAKE, FAKE, FAKE, None, 5, 0, FAKE, None) == -3
