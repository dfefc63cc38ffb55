"""lw_attn_decode_noalloc (the allocation-free variant of lw_attn_decode,
partials in the library's fixed per-GPU array) against lw_attn_decode with a
caller workspace, through the C ABI: two calls in a row, the second smaller,
each bit for bit the workspace call's output and within the oracle's bound;
and a call needing more than the array's 2 MiB is refused before any launch."""
import ctypes

import numpy as np
import pytest

from gpu_util import to_gpu
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import Q4_0, Q8_0

pytestmark = pytest.mark.gpu

LW_EINVAL = -1


def make(fmt, n_kv, L, D, seed):
    return synth.pack_fields(fmt, synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(seed), 1.0))


def test_noalloc_matches_workspace_call(oracle_mod):
    import torch
    lib = binding.library()
    stream = torch.cuda.current_stream()
    for fmt, H, n_kv, D, L, seed in [(Q8_0, 32, 8, 128, 4096, 1), (Q4_0, 16, 4, 64, 700, 2)]:
        Kc, Vc = make(fmt, n_kv, L, D, seed), make(fmt, n_kv, L, D, seed + 50)
        q = np.random.default_rng(seed).standard_normal((H, D)).astype(np.float32)
        qg, Kg, Vg = to_gpu(q), to_gpu(Kc), to_gpu(Vc)
        o1 = torch.full((H, D), float("nan"), device="cuda")
        o2 = torch.full((H, D), float("nan"), device="cuda")
        nb = binding.attn_workspace_bytes(fmt, H, n_kv, D, L)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        s = ctypes.c_void_p(stream.cuda_stream)
        scale = ctypes.c_float(1 / np.sqrt(D))
        print("noalloc fmt=%d H=%d n_kv=%d D=%d L=%d" % (fmt, H, n_kv, D, L), flush=True)
        rc = lib.lw_attn_decode(fmt, qg.data_ptr(), Kg.data_ptr(), Vg.data_ptr(), o1.data_ptr(), H, n_kv, D, L, scale,
                                ws.data_ptr(), nb, s)
        assert rc == 0
        rc = lib.lw_attn_decode_noalloc(fmt, qg.data_ptr(), Kg.data_ptr(), Vg.data_ptr(), o2.data_ptr(), H, n_kv, D,
                                        L, scale, s)
        assert rc == 0
        torch.cuda.synchronize()
        a, b = o1.cpu().numpy(), o2.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), (fmt, L)
        ref, A, T = oracle_mod.attn_decode(fmt, q, Kc, Vc, H, n_kv, D, L, 1 / np.sqrt(D))
        assert (np.abs(b - ref) <= 2.0 ** -12 * (1 + T)[:, None] * A).all(), (fmt, L)


def test_noalloc_refuses_beyond_its_array():
    lib = binding.library()
    # 4088 heads over 511 key/value heads of 128 at 4096 positions: one split of 4088 x 130 floats,
    # above the array's 2 MiB; refused by the size check, before any pointer is used or kernel launched
    assert binding.attn_workspace_bytes(Q8_0, 4088, 511, 128, 4096) > 2 << 20
    A256, A16 = 0x7F0000000000, 0x7F0000000010
    rc = lib.lw_attn_decode_noalloc(Q8_0, A16, A256, A256, A16, 4088, 511, 128, 4096, ctypes.c_float(0.1), None)
    assert rc == LW_EINVAL
