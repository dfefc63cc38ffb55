"""ctypes binding of the lw C ABI (``include/lw.h``): argument marshalling only.

Every computation runs in the HIP kernels of ``liblw.so``. torch is used for
device memory and streams: tensors pass their device pointers, and the
current torch stream is passed to ``lw_matvec``. If the library is not built,
or the tensors are not on a GPU, calls raise; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblw.so")

LW_OK = 0
EXPORTS = ("lw_matvec", "lw_matvec_multi", "lw_dequant", "lw_weight_bytes", "lw_strerror", "lw_kernel_name",
           "lw_kernel_name_multi", "lw_launch_count", "lw_launch_count_multi", "lw_attn_decode",
           "lw_attn_workspace_bytes", "lw_attn_decode_noalloc", "lw_matvec_ws", "lw_matvec_workspace_bytes",
           "lw_kernel_name_ws", "lw_launch_count_ws", "lw_attn_kernel_name")
LW_MULTI_MAX = 4


class LwError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__("%s: %s (%d)" % (where, _strerror(code), code))


_lib = None


def library() -> ctypes.CDLL:
    """Load liblw.so (built in-tree by ``python -m paper_2605_20706_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("liblw.so is not built (%s); run python -m paper_2605_20706_amd.build"
                               % LIB_PATH)
        # torch ships its own HIP runtime under the same soname as the one
        # liblw.so links; whichever is loaded first serves both. Loading
        # torch first keeps torch on its own runtime (loaded second, it would
        # bind to the system one and may find no device).
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        lib = ctypes.CDLL(LIB_PATH)
        i64 = ctypes.c_int64
        vp = ctypes.c_void_p
        lib.lw_matvec.argtypes = [ctypes.c_int, vp, vp, vp, i64, i64, i64, vp]
        lib.lw_matvec.restype = ctypes.c_int
        lib.lw_matvec_multi.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                        ctypes.POINTER(i64), vp, i64, i64, vp]
        lib.lw_matvec_multi.restype = ctypes.c_int
        lib.lw_dequant.argtypes = [ctypes.c_int, vp, vp, i64]
        lib.lw_dequant.restype = ctypes.c_int
        lib.lw_weight_bytes.argtypes = [ctypes.c_int, i64]
        lib.lw_weight_bytes.restype = i64
        lib.lw_strerror.argtypes = [ctypes.c_int]
        lib.lw_strerror.restype = ctypes.c_char_p
        lib.lw_kernel_name.argtypes = [ctypes.c_int, i64, i64, i64]
        lib.lw_kernel_name.restype = ctypes.c_char_p
        lib.lw_kernel_name_multi.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(i64), i64, i64]
        lib.lw_kernel_name_multi.restype = ctypes.c_char_p
        lib.lw_launch_count.argtypes = [ctypes.c_int, i64, i64, i64]
        lib.lw_launch_count.restype = i64
        lib.lw_launch_count_multi.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(i64), i64, i64]
        lib.lw_launch_count_multi.restype = i64
        lib.lw_attn_decode.argtypes = [ctypes.c_int, vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_float, vp, i64, vp]
        lib.lw_attn_decode.restype = ctypes.c_int
        lib.lw_attn_workspace_bytes.argtypes = [ctypes.c_int, i64, i64, i64, i64]
        lib.lw_attn_workspace_bytes.restype = i64
        lib.lw_attn_kernel_name.argtypes = [ctypes.c_int, i64, i64, i64, i64]
        lib.lw_attn_kernel_name.restype = ctypes.c_char_p
        lib.lw_attn_decode_noalloc.argtypes = [ctypes.c_int, vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_float, vp]
        lib.lw_attn_decode_noalloc.restype = ctypes.c_int
        lib.lw_matvec_ws.argtypes = [ctypes.c_int, vp, vp, vp, i64, i64, i64, vp, i64, vp]
        lib.lw_matvec_ws.restype = ctypes.c_int
        lib.lw_matvec_workspace_bytes.argtypes = [ctypes.c_int, i64, i64, i64]
        lib.lw_matvec_workspace_bytes.restype = i64
        lib.lw_kernel_name_ws.argtypes = [ctypes.c_int, i64, i64, i64]
        lib.lw_kernel_name_ws.restype = ctypes.c_char_p
        lib.lw_launch_count_ws.argtypes = [ctypes.c_int, i64, i64, i64]
        lib.lw_launch_count_ws.restype = i64
        _lib = lib
    return _lib


def raw():
    """The ctypes functions themselves (pointers as ints), for ABI-level use."""
    return library()


def _strerror(code: int) -> str:
    return library().lw_strerror(code).decode()


def strerror(code: int) -> str:
    return _strerror(code)


def weight_bytes(fmt: int, n: int) -> int:
    v = library().lw_weight_bytes(fmt, n)
    if v < 0:
        raise LwError(v, "lw_weight_bytes")
    return v


def kernel_name(fmt: int, M: int, K: int, n_tok: int):
    """Name (template part) of the kernel lw_matvec launches for these sizes,
    or None when lw_matvec would reject them. Host-only."""
    v = library().lw_kernel_name(fmt, M, K, n_tok)
    return None if v is None else v.decode()


def kernel_name_multi(fmt: int, Ms, K: int, n_tok: int):
    """Name of the kernel lw_matvec_multi launches for matrices of Ms rows
    sharing x (the fused launch's, else the first matrix's), or None."""
    ma = (ctypes.c_int64 * len(Ms))(*Ms)
    v = library().lw_kernel_name_multi(fmt, len(Ms), ma, K, n_tok)
    return None if v is None else v.decode()


def launch_count(fmt: int, M: int, K: int, n_tok: int) -> int:
    """Kernel launches lw_matvec makes for these sizes (host-only)."""
    v = library().lw_launch_count(fmt, M, K, n_tok)
    if v < 0:
        raise LwError(v, "lw_launch_count")
    return v


def launch_count_multi(fmt: int, Ms, K: int, n_tok: int) -> int:
    """Kernel launches lw_matvec_multi makes for matrices of Ms rows (host-only)."""
    ma = (ctypes.c_int64 * len(Ms))(*Ms)
    v = library().lw_launch_count_multi(fmt, len(Ms), ma, K, n_tok)
    if v < 0:
        raise LwError(v, "lw_launch_count_multi")
    return v


def kernel_name_ws(fmt: int, M: int, K: int, n_tok: int):
    """kernel_name for lw_matvec_ws with a large enough workspace."""
    v = library().lw_kernel_name_ws(fmt, M, K, n_tok)
    return None if v is None else v.decode()


def launch_count_ws(fmt: int, M: int, K: int, n_tok: int) -> int:
    """launch_count for lw_matvec_ws with a large enough workspace."""
    v = library().lw_launch_count_ws(fmt, M, K, n_tok)
    if v < 0:
        raise LwError(v, "lw_launch_count_ws")
    return v


def matvec_workspace_bytes(fmt: int, M: int, K: int, n_tok: int) -> int:
    """Workspace bytes lw_matvec_ws needs for these sizes (0: none)."""
    v = library().lw_matvec_workspace_bytes(fmt, M, K, n_tok)
    if v < 0:
        raise LwError(v, "lw_matvec_workspace_bytes")
    return v


def _check_gpu(t, name):
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def matvec(fmt: int, W, x, M: int, K: int, y=None, stream=None):
    """y[n_tok, M] = dequant(W)[M, K] @ x[n_tok, K]^T on the GPU.

    W: uint8 GPU tensor with the packed weights (lw layout); x: float32 GPU
    tensor [K] or [n_tok, K]; y: optional float32 output [n_tok, M].
    stream: a torch.cuda.Stream (default: the current stream)."""
    import torch

    _check_gpu(W, "W")
    _check_gpu(x, "x")
    if x.dtype != torch.float32:
        raise ValueError("x must be float32")
    x2 = x.reshape(1, -1) if x.dim() == 1 else x
    if x2.dim() != 2 or x2.shape[1] != K:
        raise ValueError("x must be [n_tok, K] with K = %d" % K)
    n_tok = x2.shape[0]
    if y is None:
        y = torch.empty((n_tok, M), dtype=torch.float32, device=x.device)
    _check_gpu(y, "y")
    if y.dtype != torch.float32 or y.numel() != n_tok * M:
        raise ValueError("y must be float32 with n_tok*M elements")
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    rc = library().lw_matvec(fmt, W.data_ptr(), x2.data_ptr(), y.data_ptr(), M, K, n_tok,
                             ctypes.c_void_p(stream.cuda_stream))
    if rc != LW_OK:
        raise LwError(rc, "lw_matvec")
    return y


def matvec_ws(fmt: int, W, x, M: int, K: int, y=None, workspace=None, stream=None):
    """matvec through lw_matvec_ws: the same product, with a workspace (a
    uint8 GPU tensor, allocated here when not given) for the paths that
    need one."""
    import torch

    _check_gpu(W, "W")
    _check_gpu(x, "x")
    if x.dtype != torch.float32:
        raise ValueError("x must be float32")
    x2 = x.reshape(1, -1) if x.dim() == 1 else x
    if x2.dim() != 2 or x2.shape[1] != K:
        raise ValueError("x must be [n_tok, K] with K = %d" % K)
    n_tok = x2.shape[0]
    if y is None:
        y = torch.empty((n_tok, M), dtype=torch.float32, device=x.device)
    _check_gpu(y, "y")
    if y.dtype != torch.float32 or y.numel() != n_tok * M:
        raise ValueError("y must be float32 with n_tok*M elements")
    nb = matvec_workspace_bytes(fmt, M, K, n_tok)
    if workspace is None and nb > 0:
        workspace = torch.empty(nb, dtype=torch.uint8, device=x.device)
    if workspace is not None:
        _check_gpu(workspace, "workspace")
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    rc = library().lw_matvec_ws(fmt, W.data_ptr(), x2.data_ptr(), y.data_ptr(), M, K, n_tok,
                                None if workspace is None else workspace.data_ptr(),
                                0 if workspace is None else workspace.numel(), ctypes.c_void_p(stream.cuda_stream))
    if rc != LW_OK:
        raise LwError(rc, "lw_matvec_ws")
    return y


def multi_args(Ws, ys, Ms):
    """ctypes arrays (W pointers, y pointers, row counts) for lw_matvec_multi
    from integer device addresses."""
    n = len(Ws)
    vp = ctypes.c_void_p
    return ((vp * n)(*[vp(w) for w in Ws]), (vp * n)(*[vp(v) for v in ys]),
            (ctypes.c_int64 * n)(*Ms))


def matvec_multi(fmt: int, Ws, x, Ms, K: int, ys=None, stream=None):
    """[y_i[n_tok, M_i] = dequant(W_i) @ x^T for each i], as one lw_matvec_multi
    call: matrices that share the activations x (float32 [K] or [n_tok, K]).
    Ws: uint8 GPU tensors (lw layout); ys: optional float32 outputs."""
    import torch

    x2 = x.reshape(1, -1) if x.dim() == 1 else x
    _check_gpu(x2, "x")
    if x2.dtype != torch.float32 or x2.dim() != 2 or x2.shape[1] != K:
        raise ValueError("x must be float32 [n_tok, K] with K = %d" % K)
    n_tok = x2.shape[0]
    if len(Ws) != len(Ms):
        raise ValueError("one row count per matrix")
    for i, W in enumerate(Ws):
        _check_gpu(W, "W[%d]" % i)
    if ys is None:
        ys = [torch.empty((n_tok, m), dtype=torch.float32, device=x.device) for m in Ms]
    for i, (v, m) in enumerate(zip(ys, Ms)):
        _check_gpu(v, "y[%d]" % i)
        if v.dtype != torch.float32 or v.numel() != n_tok * m:
            raise ValueError("y[%d] must be float32 with n_tok*M elements" % i)
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    wa, ya, ma = multi_args([W.data_ptr() for W in Ws], [v.data_ptr() for v in ys], list(Ms))
    rc = library().lw_matvec_multi(fmt, len(Ws), wa, ya, ma, x2.data_ptr(), K, n_tok,
                                   ctypes.c_void_p(stream.cuda_stream))
    if rc != LW_OK:
        raise LwError(rc, "lw_matvec_multi")
    return ys


def dequant(fmt: int, W, n: int, out=None):
    """float32[n] = dequant(W) on the GPU (null stream)."""
    import torch

    _check_gpu(W, "W")
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device=W.device)
    _check_gpu(out, "out")
    if out.dtype != torch.float32 or out.numel() != n:
        raise ValueError("out must be float32[n]")
    rc = library().lw_dequant(fmt, W.data_ptr(), out.data_ptr(), n)
    if rc != LW_OK:
        raise LwError(rc, "lw_dequant")
    return out


def attn_workspace_bytes(fmt: int, n_heads: int, n_kv_heads: int, head_dim: int, kv_len: int) -> int:
    v = library().lw_attn_workspace_bytes(fmt, n_heads, n_kv_heads, head_dim, kv_len)
    if v < 0:
        raise LwError(v, "lw_attn_workspace_bytes")
    return v


def attn_kernel_name(fmt: int, n_heads: int, n_kv_heads: int, head_dim: int, kv_len: int):
    """The first kernel lw_attn_decode launches for these sizes (None when
    they fail its checks)."""
    v = library().lw_attn_kernel_name(fmt, n_heads, n_kv_heads, head_dim, kv_len)
    return None if v is None else v.decode()


def attn_decode(fmt: int, q, K, V, n_heads: int, n_kv_heads: int, head_dim: int, kv_len: int, scale: float,
                out=None, workspace=None, stream=None):
    """out[n_heads, head_dim] = attention of one query token over the KV cache
    (K, V: uint8 GPU tensors in the packed layout, head-major). The
    workspace (a uint8 GPU tensor) is allocated here when not given."""
    import torch

    _check_gpu(q, "q")
    _check_gpu(K, "K")
    _check_gpu(V, "V")
    if q.dtype != torch.float32 or q.numel() != n_heads * head_dim:
        raise ValueError("q must be float32 [n_heads, head_dim]")
    if out is None:
        out = torch.empty((n_heads, head_dim), dtype=torch.float32, device=q.device)
    _check_gpu(out, "out")
    nb = attn_workspace_bytes(fmt, n_heads, n_kv_heads, head_dim, kv_len)
    if workspace is None:
        workspace = torch.empty(max(nb, 16), dtype=torch.uint8, device=q.device)
    _check_gpu(workspace, "workspace")
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    rc = library().lw_attn_decode(fmt, q.data_ptr(), K.data_ptr(), V.data_ptr(), out.data_ptr(), n_heads, n_kv_heads,
                                  head_dim, kv_len, float(scale), workspace.data_ptr(), workspace.numel(),
                                  ctypes.c_void_p(stream.cuda_stream))
    if rc != LW_OK:
        raise LwError(rc, "lw_attn_decode")
    return out
