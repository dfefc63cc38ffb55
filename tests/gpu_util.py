"""Helpers for the GPU parity tests: upload numpy inputs, call the library
through its binding, bring results back."""
import numpy as np


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def to_gpu(a):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def gpu_dequant(fmt, W, n):
    from paper_2605_20706_amd import binding
    torch = torch_cuda()
    out = binding.dequant(fmt, to_gpu(W), n)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def gpu_matvec(fmt, W, x, M, K, Wg=None):
    from paper_2605_20706_amd import binding
    torch = torch_cuda()
    Wg = to_gpu(W) if Wg is None else Wg
    y = binding.matvec(fmt, Wg, to_gpu(np.atleast_2d(x)), M, K)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def same_bits_or_both_zero(a, b):
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    eq = (a.view(np.uint32) == b.view(np.uint32)) | ((a == 0) & (b == 0))
    return eq | (np.isnan(a) & np.isnan(b))
