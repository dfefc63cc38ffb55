"""The C ABI loads, exports every entry point include/lw.h declares, and
rejects bad arguments with the documented codes before any HIP call (these
tests run without a GPU: no call here reaches a launch)."""
import ctypes
import os
import re

import pytest

import golden_io
from paper_2605_20706_amd import binding
from paper_2605_20706_amd.layout import F16, Q4_0, Q4_K, Q8_0

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LW_OK, LW_EINVAL, LW_EFMT, LW_ESHAPE, LW_EALIGN = 0, -1, -2, -3, -4
FMT = {"f16": F16, "q8_0": Q8_0, "q4_0": Q4_0, "q4_k": Q4_K}

# Fake, never dereferenced addresses: every call below fails validation first.
A256 = 0x7F0000000000
A16 = A256 + 16


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("liblw.so not built")
    return binding.library()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "lw.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lw_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(binding.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_weight_bytes_matches_hand_sizes(lib):
    for name, n, _, _, total in golden_io.plane_sizes():
        assert lib.lw_weight_bytes(FMT[name], n) == total


def test_weight_bytes_errors(lib):
    assert lib.lw_weight_bytes(7, 256) == LW_EFMT
    assert lib.lw_weight_bytes(Q4_0, -256) == LW_EINVAL
    assert lib.lw_weight_bytes(Q4_0, 100) == LW_ESHAPE
    assert lib.lw_weight_bytes(Q4_0, (1 << 40) + 256) == LW_EINVAL
    assert lib.lw_weight_bytes(Q4_0, 0) == 0


def mv(lib, fmt=Q4_0, W=A256, x=A16, y=A16, M=4, K=256, n_tok=1):
    return lib.lw_matvec(fmt, W, x, y, M, K, n_tok, None)


def test_matvec_error_order(lib):
    assert mv(lib, fmt=4, W=None) == LW_EFMT          # format first
    assert mv(lib, fmt=-1) == LW_EFMT
    assert mv(lib, W=None) == LW_EINVAL
    assert mv(lib, x=None) == LW_EINVAL
    assert mv(lib, y=None) == LW_EINVAL
    assert mv(lib, M=0) == LW_EINVAL
    assert mv(lib, K=0) == LW_EINVAL
    assert mv(lib, n_tok=0) == LW_EINVAL
    assert mv(lib, M=-3) == LW_EINVAL
    assert mv(lib, M=(1 << 31) + 1) == LW_EINVAL
    assert mv(lib, M=1 << 30, K=1 << 12) == LW_EINVAL  # M*K > 2^40
    assert mv(lib, K=255, W=A256 + 1) == LW_ESHAPE     # shape before alignment
    assert mv(lib, K=32) == LW_ESHAPE
    assert mv(lib, K=256 + 32) == LW_ESHAPE
    assert mv(lib, W=A256 + 128) == LW_EALIGN
    assert mv(lib, x=A16 + 4) == LW_EALIGN
    assert mv(lib, y=A16 + 8) == LW_EALIGN


def test_dequant_errors(lib):
    assert lib.lw_dequant(9, A256, A16, 256) == LW_EFMT
    assert lib.lw_dequant(Q4_K, None, A16, 256) == LW_EINVAL
    assert lib.lw_dequant(Q4_K, A256, None, 256) == LW_EINVAL
    assert lib.lw_dequant(Q4_K, A256, A16, -256) == LW_EINVAL
    assert lib.lw_dequant(Q4_K, A256, A16, 100) == LW_ESHAPE
    assert lib.lw_dequant(Q4_K, A256 + 16, A16, 256) == LW_EALIGN
    assert lib.lw_dequant(Q4_K, A256, A16 + 4, 256) == LW_EALIGN
    assert lib.lw_dequant(Q4_K, A256, A16, 0) == LW_OK  # no-op, no launch


def test_strerror(lib):
    for code in (0, -1, -2, -3, -4, -5, 12345):
        s = lib.lw_strerror(code)
        assert isinstance(s, bytes) and len(s) > 3


def test_binding_fails_loudly_without_gpu_tensors(lib):
    torch = pytest.importorskip("torch")
    W = torch.zeros(1024, dtype=torch.uint8)
    x = torch.zeros(256, dtype=torch.float32)
    with pytest.raises(ValueError):
        binding.matvec(Q4_0, W, x, 4, 256)
    with pytest.raises(ValueError):
        binding.dequant(Q4_0, W, 256)
