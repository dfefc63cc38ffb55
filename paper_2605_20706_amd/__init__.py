"""Fused dequantize x matrix-vector product for MI355X (gfx950).

The compute path is the HIP library ``liblw.so`` built from ``csrc/`` (C ABI
declared in ``include/lw.h``); ``binding`` marshals torch device tensors into
it. There is no CPU fallback: every call fails loudly if the library is not
built or no GPU is present.

``layout`` (byte placement of quantized fields) and ``synth`` (seeded
synthetic inputs) import no compiled code.
"""
from .layout import F16, Q8_0, Q4_0, Q4_K, FORMATS, FORMAT_NAMES  # noqa: F401

LW_OK, LW_EINVAL, LW_EFMT, LW_ESHAPE, LW_EALIGN, LW_EHIP = 0, -1, -2, -3, -4, -5
GEMV_MAX_TOK = 8


def __getattr__(name):
    # The binding (and with it the HIP library) is loaded on first use only.
    if name in ("matvec", "dequant", "weight_bytes", "strerror", "LwError", "library", "raw"):
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
