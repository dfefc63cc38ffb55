"""The C ABI loads, exports every entry point include/lw.h declares, and
rejects bad arguments with the documented codes before any HIP call (these
tests run without a GPU: no call here reaches a launch)."""
import ctypes
import os
import re

import pytest

import golden_io
from paper_2605_20706_amd import binding, layout
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LW_OK, LW_EINVAL, LW_EFMT, LW_ESHAPE, LW_EALIGN = 0, -1, -2, -3, -4
FMT = {"f16": F16, "q8_0": Q8_0, "q4_0": Q4_0, "q4_k": Q4_K, "q4_1": Q4_1, "q1_0": Q1_0}

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


def test_exports_only_the_c_abi(lib):
    """Only the C ABI is exported (hidden visibility): no symbol of a host
    program can stand in for one of the library's internal functions (such as
    the kernel-name query flag the launchers consult)."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    names = {l.split()[-1] for l in out.splitlines() if l.strip() and l.split()[-2] in ("T", "W", "D", "B")}
    names = {n for n in names if not n.startswith("__hip_cuid")}
    assert names == set(binding.EXPORTS), sorted(names)


def test_weight_bytes_matches_hand_sizes(lib):
    for name, n, _, _, total in golden_io.plane_sizes():
        assert lib.lw_weight_bytes(FMT[name], n) == total
    for name, n, _, _, _, total in golden_io.plane_sizes4():
        assert lib.lw_weight_bytes(layout.FORMATS[name], n) == total


def test_weight_bytes_errors(lib):
    assert lib.lw_weight_bytes(12, 256) == LW_EFMT
    assert lib.lw_weight_bytes(Q4_0, -256) == LW_EINVAL
    assert lib.lw_weight_bytes(Q4_0, 100) == LW_ESHAPE
    assert lib.lw_weight_bytes(Q4_0, (1 << 40) + 256) == LW_EINVAL
    assert lib.lw_weight_bytes(Q4_0, 0) == 0


def mv(lib, fmt=Q4_0, W=A256, x=A16, y=A16, M=4, K=256, n_tok=1):
    return lib.lw_matvec(fmt, W, x, y, M, K, n_tok, None)


def test_matvec_error_order(lib):
    assert mv(lib, fmt=12, W=None) == LW_EFMT          # format first
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


def mvm(lib, fmt=Q4_0, Ws=(A256, A256 + 4096), ys=(A16, A16 + 4096), Ms=(4, 8), x=A16, K=256, n_tok=1, n=None):
    n = len(Ws) if n is None else n
    wa, ya, ma = binding.multi_args(list(Ws), list(ys), list(Ms))
    return lib.lw_matvec_multi(fmt, n, wa, ya, ma, x, K, n_tok, None)


def test_matvec_multi_error_order(lib):
    """lw_matvec_multi checks as lw_matvec does, over all matrices, in the same
    order (no call here reaches a launch)."""
    assert mvm(lib, fmt=12, x=None) == LW_EFMT
    assert mvm(lib, x=None) == LW_EINVAL
    assert mvm(lib, n=0) == LW_EINVAL
    assert mvm(lib, n=binding.LW_MULTI_MAX + 1) == LW_EINVAL
    assert lib.lw_matvec_multi(Q4_0, 2, None, None, None, A16, 256, 1, None) == LW_EINVAL
    assert mvm(lib, Ws=(A256, 0)) == LW_EINVAL
    assert mvm(lib, ys=(0, A16)) == LW_EINVAL
    assert mvm(lib, Ms=(4, 0)) == LW_EINVAL
    assert mvm(lib, Ms=(0, 4), K=300) == LW_EINVAL                      # sizes before shape
    assert mvm(lib, K=300, Ws=(A256 + 1, A256)) == LW_ESHAPE            # shape before alignment
    assert mvm(lib, Ws=(A256, A256 + 128)) == LW_EALIGN
    assert mvm(lib, ys=(A16, A16 + 4)) == LW_EALIGN
    assert mvm(lib, x=A16 + 8) == LW_EALIGN


def test_kernel_name_multi(lib):
    """One token: one fused launch of the single-token kernel over all rows
    (last template parameter: a table of 2 or 4 segments); 3 to 8 tokens of a
    4-bit format: one few-token launch where that kernel takes the summed rows;
    otherwise the first matrix's lw_matvec kernel; None where lw_matvec_multi
    would reject the sizes."""
    assert binding.kernel_name_multi(Q4_K, [14336, 14336], 4096, 1) == "gemv1r_kernel<%d, 1, 2, 1, 8, 2, 2>" % Q4_K
    assert binding.kernel_name_multi(F16, [8192, 8192], 2048, 1) == "gemv1_kernel<%d, 1, 4, 8, 2>" % F16
    assert binding.kernel_name_multi(Q4_K, [3000, 3000, 2048], 4096, 1) == "gemv1_kernel<%d, 1, 2, 8, 4>" % Q4_K
    assert binding.kernel_name_multi(Q4_K, [4096, 4096, 2048], 4096, 1) == "gemv1r_kernel<%d, 1, 2, 1, 8, 2, 4>" % Q4_K
    assert binding.kernel_name_multi(Q4_0, [14336, 14336], 4096, 4) == "fewtok_kernel<%d, 1, 2>" % Q4_0
    assert binding.kernel_name_multi(Q4_K, [3000, 3000, 2048], 4096, 8) == "fewtok_kernel<%d, 1, 4>" % Q4_K
    for args in [(Q4_0, [14336, 14336], 4096, 2), (Q4_0, [14336, 14336], 4096, 9), (Q4_0, [8192, 8192], 2048, 4),
                 (F16, [8192, 8192], 2048, 4), (Q8_0, [14336, 14336], 4096, 4)]:
        assert binding.kernel_name_multi(*args) == binding.kernel_name(args[0], args[1][0], args[2], args[3]), args
    assert binding.kernel_name_multi(Q4_0, [100], 2304, 1) == binding.kernel_name(Q4_0, 100, 2304, 1)
    assert binding.kernel_name_multi(Q4_0, [100, 0], 2304, 1) is None
    assert binding.kernel_name_multi(Q4_0, [100, 4], 300, 1) is None
    assert binding.kernel_name_multi(Q4_0, [1] * (binding.LW_MULTI_MAX + 1), 256, 1) is None


def test_dequant_errors(lib):
    assert lib.lw_dequant(12, A256, A16, 256) == LW_EFMT
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


def test_kernel_name_rejects_what_matvec_rejects(lib):
    assert binding.kernel_name(12, 4, 256, 1) is None           # format
    assert binding.kernel_name(Q4_0, 0, 256, 1) is None        # sizes
    assert binding.kernel_name(Q4_0, 4, 256, 0) is None
    assert binding.kernel_name(Q4_0, 4, 300, 1) is None        # shape
    assert binding.kernel_name(Q4_0, 4, 256, 1) is not None


def test_kernel_selection_table(lib):
    """The kernels the workloads' shapes select (no launch: a host-only query).
    One token: the register-activation kernel when K is a whole number of
    2048-element chunks and its table has the shape, else the LDS-activation
    kernel; two tokens over the 4-bit formats: the register kernel; 3..8
    tokens over the 4-bit formats: the matrix-core kernel with the
    activations in LDS for matrices with at least two 16-row tiles per
    workgroup (and K >= 4096 for Q4_0), else the pair-step matrix-core kernel;
    9..16 the few-token one with two MFMAs per block; more: the tiled
    matrix-core kernel. The formats without the pair-step kernel
    (Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4) take the first matrix-core kernel
    for 2..8 tokens at every shape and the tiled kernel beyond."""
    from paper_2605_20706_amd import synth

    def kind(fmt, M, K, nt):
        return binding.kernel_name(fmt, M, K, nt).split("<")[0]

    for key, wl in synth.WORKLOADS.items():
        for m in wl.matrices:
            for nt in (1, 2, 4, 8, 12, 512):
                name = binding.kernel_name(wl.fmt, m.M, m.K, nt)
                assert name and re.fullmatch(r"\w+_kernel<\d+(, \d+)*>", name), (key, m, nt, name)
                assert name.startswith(("gemv", "multitok", "fewtok", "skinny", "gemm")), name
    # shapes the swept table names (profiles/sweep_select.json): see test_selection_table_matches_sweep;
    # the built-in rules elsewhere
    assert kind(Q4_K, 14336, 4096, 1) == "gemv1r_kernel"      # 8B gate: 2 chunks, many rows
    assert kind(Q4_K, 4096, 14336, 1) == "gemv1r_kernel"      # 8B down: 7 chunks split over 7 waves
    assert kind(Q4_K, 6144, 4096, 1) == "gemv1_kernel"        # 8B qkv: too few rows per wave
    assert kind(Q4_0, 100, 2304, 1) == "gemv1_kernel"         # K not whole chunks
    assert kind(Q4_0, 14336, 4096, 2) == "gemv1r_kernel"
    assert kind(Q4_K, 128256, 4096, 8) == "fewtok_kernel"       # lm_head: two tiles per wave
    assert kind(Q4_0, 8192, 2048, 4) == "multitok_pk_kernel"    # 1B gate Q4_0: K below 4096
    assert kind(Q4_K, 14336, 4096, 9) == "multitok_kernel"
    assert kind(Q4_0, 14336, 4096, 512) == "gemm32_kernel"
    assert kind(Q8_0, 14336, 4096, 512) == "gemm_kernel"
    assert kind(F16, 2048, 2048, 1) == "gemv1_kernel"
    assert kind(Q8_0, 2048, 2048, 12) == "skinny_kernel"
    assert kind(F16, 2048, 2048, 20) == "gemv_kernel"
    for fmt in (Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, 11):            # one token: the LDS kernel
        assert kind(fmt, 14336, 4096, 1) == "gemv1_kernel"
    for fmt in (Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, 11):            # 2..8 tokens: the few-token matrix-core kernel
        for nt in (2, 4, 8):
            assert kind(fmt, 14336, 4096, nt) == "fewtok_kernel"
        assert kind(fmt, 100, 2304, 4) == "fewtok_kernel"     # one tile, K split over the waves
        assert kind(fmt, 4096, 14336, 8) == "fewtok_kernel"   # the 8B down projection
    for fmt in (Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, 11):            # from 9 tokens: the tiled matrix cores
        assert kind(fmt, 14336, 4096, 12) == "gemm32_kernel"
        assert kind(fmt, 14336, 4096, 512) == "gemm32_kernel"


def test_ceiling_library_exports_and_checks():
    """libceiling.so (the benchmark's streaming-ceiling kernels) exports what
    include/lw_ceiling.h declares and rejects bad arguments before any HIP
    call."""
    path = os.path.join(ROOT, "paper_2605_20706_amd", "libceiling.so")
    if not os.path.exists(path):
        pytest.skip("libceiling.so not built")
    src = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "lw_ceiling.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(lw_[a-z_]+)\s*\(", src)))
    assert names == ["lw_ceiling_read", "lw_ceiling_write"]
    lib = ctypes.CDLL(path)
    lib.lw_ceiling_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    lib.lw_ceiling_write.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    assert lib.lw_ceiling_read(None, 16, A16, None) == -1
    assert lib.lw_ceiling_read(A256, 16, None, None) == -1
    assert lib.lw_ceiling_read(A256, 24, A16, None) == -1
    assert lib.lw_ceiling_read(A256 + 8, 16, A16, None) == -1
    assert lib.lw_ceiling_write(A256, 0, None) == -1
    assert lib.lw_ceiling_write(A256 + 4, 16, None) == -1


def test_edge_cases_cover_every_kernel_family(lib):
    """The GPU edge-case table (zero rows, zero scales, Eq. (1)-encoded
    weights, activations scaled by 2^+-60) reaches every kernel family the
    library selects."""
    import test_gpu_edges as e
    seen = set()
    for fmt in e.FMTS:
        for M, K, nt in e.EDGE_SHAPES:
            seen.add(binding.kernel_name(fmt, M, K, nt).split("<")[0])
        for Ms, K, nt in e.EDGE_MULTI:
            seen.add(binding.kernel_name_multi(fmt, list(Ms), K, nt).split("<")[0])
    families = {"gemv_kernel", "gemv1_kernel", "gemv1r_kernel", "fewtok_kernel", "multitok_kernel",
                "multitok_pk_kernel", "skinny_kernel", "gemm_kernel", "gemm32_kernel"}
    assert families <= seen, families - seen


def test_launch_count(lib):
    """lw_launch_count / lw_launch_count_multi: the kernel launches a call
    makes (a prefill K split adds the fill kernel; f16 token blocks plus a
    remainder are two launches), and the size errors of the calls they
    describe."""
    assert binding.launch_count(Q4_K, 14336, 4096, 1) == 1
    assert binding.launch_count(Q4_0, 4096, 14336, 512) == 2      # 8B down: K split over a zeroed y
    assert binding.launch_count(Q4_0, 14336, 4096, 512) == 1
    assert binding.launch_count(F16, 2048, 2048, 17) == 2         # two blocks of 8, then one token
    assert binding.launch_count(F16, 2048, 2048, 16) == 1
    assert binding.launch_count(Q1_0, 2048, 2048, 512) == 2       # tiled: K split over a zeroed y
    assert binding.launch_count(F16, 2048, 2048, 512) == 1        # 64 blocks of 8 in one launch
    assert binding.launch_count_multi(Q4_K, [14336, 14336], 4096, 1) == 1   # fused gate + up
    assert binding.launch_count_multi(Q4_K, [14336, 14336], 4096, 2) == 2   # one per matrix
    assert binding.launch_count_multi(Q4_0, [14336, 14336], 4096, 4) == 1
    assert binding.launch_count_multi(Q5_K, [14336, 14336], 4096, 2) == 1   # no register kernel: fused
    assert binding.launch_count_multi(Q1_0, [6144, 6144], 2048, 2) == 2     # the register kernel per matrix
    assert binding.launch_count_multi(Q1_0, [6144, 6144], 2048, 4) == 1
    f = lib.lw_launch_count
    assert f(12, 4, 256, 1) == LW_EFMT
    assert f(Q4_0, 0, 256, 1) == LW_EINVAL
    assert f(Q4_0, 4, 300, 1) == LW_ESHAPE
    g = lib.lw_launch_count_multi
    Ms = (ctypes.c_int64 * 2)(4, 8)
    assert g(Q4_0, 0, Ms, 256, 1) == LW_EINVAL
    assert g(Q4_0, 2, None, 256, 1) == LW_EINVAL
    assert g(12, 2, Ms, 256, 1) == LW_EFMT
    assert g(Q4_0, 2, Ms, 300, 1) == LW_ESHAPE


def test_forced_candidates_name_their_kernels(lib, monkeypatch):
    """LW_FORCE_CFG selects each candidate where it takes the shape (the
    kernel name shows its configuration) and falls back to the built-in
    choice where it does not."""
    seen = {}
    for cand, K, nt, M in [(10, 2048, 1, 3001), (11, 2048, 1, 3001), (12, 2048, 1, 3001), (13, 4096, 1, 3001),
                           (14, 4096, 1, 3001), (15, 4096, 1, 3001), (16, 4096, 1, 3001), (17, 4096, 1, 3001),
                           (18, 14336, 1, 3001), (19, 14336, 1, 3001), (20, 14336, 1, 3001),
                           (21, 2048, 2, 2500), (22, 4096, 2, 2500), (23, 8192, 2, 2500), (24, 14336, 2, 2500),
                           (25, 4096, 2, 2500)]:
        monkeypatch.setenv("LW_FORCE_CFG", str(cand))
        name = binding.kernel_name(Q4_K, M, K, nt)
        assert name.startswith("gemv1r_kernel<3, %d, " % nt), (cand, name)
        seen[cand] = name
    assert len(set(seen.values())) == len(seen)  # every candidate a distinct configuration
    monkeypatch.setenv("LW_FORCE_CFG", "1")
    assert binding.kernel_name(Q4_K, 14336, 4096, 1).startswith("gemv1_kernel<")
    monkeypatch.setenv("LW_FORCE_CFG", "30")
    assert binding.kernel_name(Q4_0, 8200, 4096, 4).startswith("fewtok_kernel<")
    monkeypatch.setenv("LW_FORCE_CFG", "31")
    assert binding.kernel_name(Q4_0, 8200, 4096, 4).startswith("multitok")
    monkeypatch.setenv("LW_FORCE_CFG", "32")
    assert binding.kernel_name(Q4_0, 8200, 4096, 12).startswith("gemm32_kernel<")
    # a 2-chunk candidate on a 1-chunk shape: the built-in rule for one chunk
    monkeypatch.setenv("LW_FORCE_CFG", "13")
    assert binding.kernel_name(Q4_K, 3001, 2048, 1) == "gemv1r_kernel<3, 1, 1, 1, 8, 2, 1>"


def test_selection_table_matches_sweep(lib):
    """The compiled table is the one the committed sweep generates, and every
    swept shape selects the sweep's fastest candidate."""
    import json
    from paper_2605_20706_amd import gen_select
    with open(gen_select.OUT) as fh:
        assert fh.read() == gen_select.render(gen_select.entries())
    if not os.path.exists(gen_select.SWEEP):
        pytest.skip("no sweep results committed")
    with open(gen_select.SWEEP) as fh:
        sweep = json.load(fh)
    for sh in sweep["shapes"]:
        res = [r for r in sh["results"] if r.get("us") is not None]
        best = min(res, key=lambda r: r["us"])
        Ms = sh.get("Ms", [sh["M"]])
        if len(Ms) > 1:
            name = binding.kernel_name_multi(sh["fmt"], Ms, sh["K"], sh["n_tok"])
        else:
            name = binding.kernel_name(sh["fmt"], sh["M"], sh["K"], sh["n_tok"])
        assert name == best["kernel"], (sh["fmt"], sh["M"], sh["K"], sh["n_tok"], name, best)


def test_attn_errors_and_workspace(lib):
    """lw_attn_decode's checks in the documented order, and the workspace
    size (heads x splits x (head_dim + 2) floats)."""
    f = lib.lw_attn_decode

    def call(fmt=Q8_0, q=A16, K=A256, V=A256, out=A16, H=32, kv=8, D=128, L=2048, scale=0.088, ws=A16, wsb=1 << 30):
        return f(fmt, q, K, V, out, H, kv, D, L, scale, ws, wsb, None)
    assert call(fmt=Q4_K) == LW_EFMT                      # a super-block format: rows of 128 hold no block
    assert call(fmt=12, q=None) == LW_EFMT
    assert call(q=None) == LW_EINVAL
    assert call(ws=None) == LW_EINVAL
    assert call(H=12) == LW_EINVAL                         # 12 heads over 8
    assert call(H=96, kv=8) == LW_EINVAL                   # group of 12
    assert call(D=96) == LW_EINVAL
    assert call(L=0) == LW_EINVAL
    assert call(scale=float("inf")) == LW_EINVAL
    assert call(wsb=16) == LW_EINVAL                       # workspace too small
    assert call(kv=1, H=1, D=64, L=3) == LW_ESHAPE         # 192 elements
    assert call(K=A256 + 16) == LW_EALIGN
    assert call(out=A16 + 4) == LW_EALIGN
    wb = binding.attn_workspace_bytes(Q8_0, 32, 8, 128, 2048)
    assert wb > 0 and wb % (32 * 130 * 4) == 0
    assert binding.attn_workspace_bytes(Q8_0, 32, 8, 128, 1) == 32 * 130 * 4   # one split
    assert lib.lw_attn_workspace_bytes(Q4_K, 32, 8, 128, 16) == LW_EFMT


def test_attn_kernel_routing(lib):
    """f16, Q8_0 and Q4_0 caches take the matrix-core score kernel when the
    split leaves more than 64 positions per workgroup (32 heads over 8:
    32 splits from 2048 positions on), the other formats the vector kernel."""
    name = binding.attn_kernel_name
    assert name(Q8_0, 32, 8, 128, 1000) == "attn_split_kernel<1, 128, 4>"     # 16 splits of 63
    assert name(Q8_0, 32, 8, 128, 2048) == "attn_split_kernel<1, 128, 4>"     # 32 splits of 64
    assert name(Q8_0, 32, 8, 128, 2080) == "attn_mf_kernel<1, 128, 4>"        # 32 splits of 65
    assert name(F16, 64, 8, 64, 32768) == "attn_mf_kernel<0, 64, 8>"
    assert name(Q4_0, 8, 8, 128, 8192) == "attn_mf_kernel<2, 128, 1>"
    assert name(Q4_1, 32, 8, 128, 32768) == "attn_split_kernel<4, 128, 4>"
    assert name(MXFP4, 32, 8, 128, 32768) == "attn_split_kernel<11, 128, 4>"
    assert name(Q4_K, 32, 8, 128, 32768) is None
    assert name(Q8_0, 12, 8, 128, 2048) is None


def _ws_bytes(M, K, n_tok, ks):
    """The fp4 path's workspace: four e2m3 pieces (24 bytes of codes and one
    scale byte per 32 activations each) of n_tok rounded up to 64 tokens, and
    with ks > 1 K splits their float32 partial results [ks][n_tok][M]; each
    part rounded up to 256 bytes."""
    ntp = -(-n_tok // 64) * 64
    nb = K // 32
    r256 = lambda v: -(-v // 256) * 256
    return r256(nb * 4 * ntp * 24) + r256(nb * 4 * ntp) + (r256(4 * ks * n_tok * M) if ks > 1 else 0)


def test_matvec_workspace_bytes(lib):
    f = lib.lw_matvec_workspace_bytes
    # K splits planned for 256 compute units (512 x 64 tiles): 28 x 8 tiles
    # fill the chip unsplit; 8 x 8 tiles take 4 splits of 14 super-blocks; a
    # K of one super-block cannot split; 1 x 2 tiles take the most splits
    # that keep 4 super-blocks each (2)
    for M, K, n_tok, ks in [(14336, 4096, 512, 1), (4096, 14336, 512, 4), (41, 256, 17, 1), (1, 2048, 65, 2)]:
        assert f(layout.MXFP4, M, K, n_tok) == _ws_bytes(M, K, n_tok, ks), (M, K, n_tok)
    # every other call takes a path without a workspace
    for fmt in (F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K):
        assert f(fmt, 4096, 4096, 512) == 0
    for n_tok in (1, 2, 8, 16):
        assert f(layout.MXFP4, 4096, 4096, n_tok) == 0
    assert f(12, 64, 256, 512) == LW_EFMT
    assert f(layout.MXFP4, 0, 256, 512) == LW_EINVAL
    assert f(layout.MXFP4, 64, 300, 512) == LW_ESHAPE


def test_matvec_ws_error_order(lib):
    f = lib.lw_matvec_ws
    MX = layout.MXFP4
    need = _ws_bytes(64, 256, 64, 1)
    assert f(12, A256, A16, A16, 64, 256, 64, A256, need, None) == LW_EFMT
    assert f(MX, None, A16, A16, 64, 256, 64, A256, need, None) == LW_EINVAL
    assert f(MX, A256, A16, A16, 0, 256, 64, A256, need, None) == LW_EINVAL
    assert f(MX, A256, A16, A16, 64, 300, 64, A256, need, None) == LW_ESHAPE
    # the workspace: needed and missing or too small, then its alignment
    assert f(MX, A256, A16, A16, 64, 256, 64, None, need, None) == LW_EINVAL
    assert f(MX, A256, A16, A16, 64, 256, 64, A256, need - 1, None) == LW_EINVAL
    assert f(MX, A256, A16, A16, 64, 256, 64, A16, need, None) == LW_EALIGN
    assert f(MX, A16, A16, A16, 64, 256, 64, A256, need, None) == LW_EALIGN
    assert f(MX, A256, A16 + 4, A16, 64, 256, 64, A256, need, None) == LW_EALIGN


def test_kernel_name_and_launch_count_ws(lib):
    MX = layout.MXFP4
    # mxfp4 from 17 tokens: the split kernel and the fp4 matrix-core kernel
    # (plus the kernel that sums the partial results where K is split)
    for M, K, n_tok in [(14336, 4096, 512), (300, 1024, 17), (1100, 4352, 100)]:
        assert binding.kernel_name_ws(MX, M, K, n_tok).startswith("fp4mm_kernel<")
        assert binding.launch_count_ws(MX, M, K, n_tok) in (2, 3)
        assert binding.kernel_name(MX, M, K, n_tok) != binding.kernel_name_ws(MX, M, K, n_tok)
    assert binding.launch_count_ws(MX, 14336, 4096, 512) == 2
    assert binding.launch_count_ws(MX, 4096, 14336, 512) == 3
    # elsewhere lw_matvec_ws is lw_matvec
    for fmt, n_tok in [(Q4_0, 512), (MX, 16), (MX, 1), (F16, 100), (Q4_K, 4)]:
        assert binding.kernel_name_ws(fmt, 4096, 4096, n_tok) == binding.kernel_name(fmt, 4096, 4096, n_tok)
        assert binding.launch_count_ws(fmt, 4096, 4096, n_tok) == binding.launch_count(fmt, 4096, 4096, n_tok)
    assert lib.lw_kernel_name_ws(12, 64, 256, 512) is None
    assert lib.lw_launch_count_ws(MX, 64, 300, 512) == LW_ESHAPE
