"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/sinkhorn.h declares, and rejects invalid arguments on
the host before anything is launched."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_1907_01729_amd as sk
from paper_1907_01729_amd import _binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sinkhorn.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SK_API\s+[\w\s\*]+?\b(sinkhorn_\w+)\s*\(", text)))


def test_header_declares_the_abi():
    assert declared_functions() == sorted(_binding.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = sk.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", sk.library_path()], capture_output=True, text=True,
                         check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if l.strip()}
    for name in declared_functions():
        assert name in exported, name
    # nothing else of the library's own leaks into the dynamic symbol table
    assert not [s for s in exported if s.startswith("_ZN2sk")]


def test_library_reads_no_environment():
    """No environment variable changes what the library computes: it imports
    no getenv (kernel choices for tests go through sinkhorn_forward_select)."""
    out = subprocess.run(["nm", "-D", "--undefined-only", sk.library_path()], capture_output=True, text=True,
                         check=True).stdout
    imported = {l.split()[-1].split("@")[0] for l in out.splitlines() if l.strip()}
    assert not imported & {"getenv", "secure_getenv", "__secure_getenv"}


def test_forward_select_rejects_unknown_selector():
    lib = sk.load_library()
    p = _binding.problem(4, 10, 10, 0, 0.1, 10)
    v = None
    for sel in (-1, 5, 1 << 20):
        assert lib.sinkhorn_forward_select(ctypes.byref(p), sel, v, v, v, v, v, v, v, v, v, 0, None) == -7
    # a valid selector goes on to the ordinary checks
    assert lib.sinkhorn_forward_select(ctypes.byref(p), 2, v, v, v, v, v, v, v, v, v, 0, None) == -1
    assert lib.sinkhorn_forward_select(ctypes.byref(_binding.problem(4, 10, 10, 0, 0.0, 10)), 1, v, v, v, v, v, v,
                                       v, v, v, 0, None) == -3
    with pytest.raises(ValueError):
        sk.sinkhorn_forward_select("fast", None, None, None, 0.1, 10)


def test_status_strings():
    for code in range(-7, 1):
        assert sk.sinkhorn_status_string(code)
    assert "lambda" in sk.sinkhorn_status_string(-3)
    assert sk.sinkhorn_status_string(-99) == "unknown status"


def test_regime_and_workspace_queries():
    assert sk.sinkhorn_regime(4, 10, 10, 0) == 1
    assert sk.sinkhorn_regime(1024, 100, 100, 0) == 1
    assert sk.sinkhorn_regime(4, 128, 128, 1) == 1
    assert sk.sinkhorn_regime(4, 129, 10, 0) == 2
    assert sk.sinkhorn_regime(4, 10, 10, 0, lam=0.0) == 0
    assert sk.sinkhorn_workspace_bytes(4, 10, 10, 0, 0.1, 100) == 0
    assert sk.sinkhorn_workspace_bytes(256, 784, 784, 0, 0.01, 300) > 0
    # rows wider than 4096 take the two-pass sweep of the tiled regime
    assert sk.sinkhorn_regime(4, 200, 4097, 0) == 2
    assert sk.sinkhorn_regime(4, 3, 100000, 1) == 2
    assert sk.sinkhorn_workspace_bytes(4, 200, 4097, 0, 0.1, 10) >= 4 * 4 * 4352  # column potentials, padded
    # the tiled regime runs a batch above one grid dimension (65535) in chunks
    # that share the workspace of one chunk
    assert sk.sinkhorn_regime(65536, 130, 130, 0) == 2
    assert sk.sinkhorn_regime(1 << 20, 130, 8, 1) == 2
    chunk = sk.sinkhorn_workspace_bytes(65535, 130, 130, 0, 0.1, 10)
    assert sk.sinkhorn_workspace_bytes(65536, 130, 130, 0, 0.1, 10) == chunk
    assert sk.sinkhorn_workspace_bytes(200000, 130, 130, 0, 0.1, 10) == chunk
    assert sk.sinkhorn_sharp_workspace_bytes(200000, 130, 8, 0) == sk.sinkhorn_sharp_workspace_bytes(65535, 130, 8, 0)
    assert (sk.sinkhorn_points_workspace_bytes(70000, 130, 8, 1, 3, 0.1, 10)
            == sk.sinkhorn_points_workspace_bytes(65535, 130, 8, 1, 3, 0.1, 10))
    assert sk.sinkhorn_regime(1 << 20, 8, 8, 0) == 1  # the resident regime has no such limit
    assert sk.sinkhorn_workspace_bytes(-1, 784, 784, 0, 0.01, 300) == 0


def _fwd(p, ptr=None, ws=0):
    lib = sk.load_library()
    v = ctypes.c_void_p(ptr) if ptr else None
    return lib.sinkhorn_forward(ctypes.byref(p), v, v, v, v, v, v, v, v, v, ctypes.c_size_t(ws), None)


def _bwd(p, ptr=None):
    lib = sk.load_library()
    v = ctypes.c_void_p(ptr) if ptr else None
    return lib.sinkhorn_backward(ctypes.byref(p), v, v, v, v, v, v, v, v, None, None)


@pytest.mark.parametrize("args,code", [
    ((4, 0, 10, 0, 0.1, 10), -2),
    ((4, 10, 0, 0, 0.1, 10), -2),
    ((-1, 10, 10, 0, 0.1, 10), -2),
    ((4, 10, 10, 2, 0.1, 10), -2),
    ((4, 10, 10, 0, 0.0, 10), -3),
    ((4, 10, 10, 0, -1.0, 10), -3),
    ((4, 10, 10, 0, float("inf"), 10), -3),
    ((4, 10, 10, 0, float("nan"), 10), -3),
    ((4, 10, 10, 0, 0.1, -1), -4),
])
def test_invalid_problems_rejected_on_host(args, code):
    p = _binding.problem(*args)
    assert _fwd(p) == code
    if code != -4:  # backward ignores n_iter
        assert _bwd(p) == code


def test_invalid_tol_and_null_pointers():
    assert _fwd(_binding.problem(4, 10, 10, 0, 0.1, 10, float("nan"))) == -4
    assert _fwd(_binding.problem(4, 10, 10, 0, 0.1, 10)) == -1
    assert _bwd(_binding.problem(4, 10, 10, 0, 0.1, 10)) == -1
    lib = sk.load_library()
    assert lib.sinkhorn_forward(None, None, None, None, None, None, None, None, None, None, 0, None) == -1
    # B == 0 is a no-op that succeeds without touching any pointer
    assert _fwd(_binding.problem(0, 10, 10, 0, 0.1, 10)) == 0


def test_workspace_too_small_rejected_before_launch():
    p = _binding.problem(8, 784, 784, 0, 0.01, 10)
    need = sk.sinkhorn_workspace_bytes(8, 784, 784, 0, 0.01, 10)
    assert need > 0
    # non-NULL (never dereferenced) pointers so that only the size check fires
    assert _fwd(p, ptr=0x1000, ws=need - 1) == -5


def _fwd_points(p, D, ptr=None, ws=0):
    lib = sk.load_library()
    v = ctypes.c_void_p(ptr) if ptr else None
    return lib.sinkhorn_forward_points(ctypes.byref(p), D, v, v, v, v, v, v, v, v, v, v, ctypes.c_size_t(ws), None)


def _bwd_points(p, D, ptr=None):
    lib = sk.load_library()
    v = ctypes.c_void_p(ptr) if ptr else None
    return lib.sinkhorn_backward_points(ctypes.byref(p), D, v, v, v, v, v, v, v, v, v, None, None, None)


def test_points_rejections_on_host():
    p = _binding.problem(4, 300, 500, 1, 0.1, 10)
    for D in (0, -1, 17):
        assert _fwd_points(p, D) == -2
        assert _bwd_points(p, D) == -2
        assert sk.sinkhorn_points_workspace_bytes(4, 300, 500, 1, D, 0.1, 10) == 0
    assert _fwd_points(p, 3) == -1
    assert _bwd_points(p, 3) == -1
    assert _fwd_points(_binding.problem(4, 300, 500, 1, 0.0, 10), 3) == -3
    assert _fwd_points(_binding.problem(0, 300, 500, 1, 0.1, 10), 3) == 0
    need = sk.sinkhorn_points_workspace_bytes(4, 300, 500, 1, 3, 0.1, 10)
    assert need > 0
    assert _fwd_points(p, 3, ptr=0x1000, ws=need - 1) == -5


def test_points_workspace_sizes():
    # on-the-fly sweep (per-sample clouds, tiled shape, D <= 3, d2 <= 2048): no cost matrix in the workspace
    on_the_fly = sk.sinkhorn_points_workspace_bytes(32, 1024, 2048, 1, 3, 0.05, 100)
    assert 0 < on_the_fly < 32 * 1024 * 2048 * 4
    # everything else holds the cost matrix written out, then the forward's own workspace
    cost = 32 * 1024 * 2048 * 4
    assert sk.sinkhorn_points_workspace_bytes(32, 1024, 2048, 1, 4, 0.05, 100) >= cost
    assert sk.sinkhorn_points_workspace_bytes(32, 100, 100, 1, 3, 0.05, 100) >= 32 * 100 * 100 * 4
    assert sk.sinkhorn_points_workspace_bytes(32, 1024, 2100, 1, 3, 0.05, 100) >= 32 * 1024 * 2100 * 4
    shared = sk.sinkhorn_points_workspace_bytes(32, 784, 784, 0, 2, 0.01, 100)
    assert shared >= 784 * 784 * 4 + sk.sinkhorn_workspace_bytes(32, 784, 784, 0, 0.01, 100)


def test_sharp_rejections_on_host():
    lib = sk.load_library()
    v = None

    def call(p, max_cg=10, tol=1e-6, ws=0, ptr=None):
        a = ctypes.c_void_p(ptr) if ptr else None
        return lib.sinkhorn_backward_sharp(ctypes.byref(p), a, a, a, a, a, a, a, a, max_cg, ctypes.c_float(tol),
                                           None, a, ctypes.c_size_t(ws), None)
    # rows wider than 4096 take the two-pass products: a workspace, then pointers
    wide = sk.sinkhorn_sharp_workspace_bytes(4, 200, 4097, 0)
    assert wide > 0
    assert call(_binding.problem(4, 200, 4097, 0, 0.1, 0), ws=wide - 1, ptr=0x1000) == -5
    assert call(_binding.problem(4, 200, 4097, 0, 0.1, 0), ws=wide) == -1
    assert call(_binding.problem(4, 0, 4097, 0, 0.1, 0)) == -2
    assert call(_binding.problem(4, 10, 10, 0, 0.0, 0)) == -3
    assert call(_binding.problem(4, 10, 10, 0, 0.1, 0), max_cg=0) == -4
    assert call(_binding.problem(4, 10, 10, 0, 0.1, 0), tol=float("nan")) == -4
    assert call(_binding.problem(4, 10, 10, 0, 0.1, 0)) == -1
    assert call(_binding.problem(0, 10, 10, 0, 0.1, 0)) == 0
    # larger supports need a workspace; resident ones none
    assert sk.sinkhorn_sharp_workspace_bytes(4, 128, 128, 0) == 0
    need = sk.sinkhorn_sharp_workspace_bytes(4, 129, 10, 0)
    assert need > 0
    assert sk.sinkhorn_sharp_workspace_bytes(256, 784, 784, 0) > 0
    assert sk.sinkhorn_sharp_workspace_bytes(4, 0, 4097, 0) == 0  # invalid problem
    assert call(_binding.problem(4, 129, 10, 0, 0.1, 0), ws=need - 1, ptr=0x1000) == -5
    assert call(_binding.problem(4, 129, 10, 0, 0.1, 0), ws=need) == -1  # then the pointers are checked


def test_describe_names_the_dispatch():
    d = sk.sinkhorn_describe
    label = d(1024, 100, 100, 0, 0.05, 200)
    assert label.startswith("resident: sk_resident_sym_kernel<13>") and "in place" in label
    assert "sk_resident_log_kernel<13>" in d(1024, 100, 100, 0, 0.05, 200, select="log")
    assert "sk_resident_gen_kernel<13>" in d(1024, 100, 100, 0, 0.05, 200, select="nosym")
    assert "left unsolved" in d(1024, 100, 100, 0, 0.05, 200, select="plain")
    wide_res = d(8, 120, 120, 1, 0.1, 10)
    assert "sk_resident_gen_kernel<16>" in wide_res and "second launch" in wide_res
    assert "sk_resident_log_kernel<2>" in d(4, 10, 10, 0, 0.1, 0)  # n_iter = 0
    grid = d(64, 4096, 4096, 0, 1e-3, 500, 1e-6)
    assert "sk_tiled_sweep_shared<64, 8, 4, 1>" in grid and "32 row blocks of 128 rows" in grid
    assert "running list" in grid and "running list" not in d(64, 4096, 4096, 0, 1e-3, 500, 1e-6, select="nocompact")
    assert f"workspace {sk.sinkhorn_workspace_bytes(64, 4096, 4096, 0, 1e-3, 500, 1e-6)} bytes" in grid
    assert "sk_tiled_sweep_shared<13, 8, 8, 4>" in d(256, 784, 784, 0, 0.01, 300)
    clouds = d(32, 1024, 2048, 1, 0.05, 100)
    assert "sk_tiled_sweep_stream<8>" in clouds and "folded" in clouds
    assert "sk_tiled_sweep<4>" in d(2, 300, 200, 0, 0.1, 10)  # a shared cost with B < 4
    assert "sk_wide_rows" in d(4, 200, 5000, 0, 0.1, 10)
    assert "2 chunks" in d(70000, 130, 8, 1, 0.1, 10)
    assert d(0, 10, 10, 0, 0.1, 10).startswith("nothing")


def test_describe_truncates_and_rejects():
    lib = sk.load_library()
    p = _binding.problem(64, 4096, 4096, 0, 1e-3, 500)
    n = lib.sinkhorn_describe(ctypes.byref(p), 0, None, 0)
    assert n > 40
    buf = ctypes.create_string_buffer(b"x" * 32)
    assert lib.sinkhorn_describe(ctypes.byref(p), 0, buf, 16) == n  # snprintf semantics
    assert len(buf.value) == 15 and buf.raw[16:32] == b"x" * 16
    assert lib.sinkhorn_describe(ctypes.byref(p), 9, None, 0) == -7
    assert lib.sinkhorn_describe(ctypes.byref(_binding.problem(4, 0, 10, 0, 0.1, 10)), 0, None, 0) == -2
    assert lib.sinkhorn_describe(ctypes.byref(p), 0, None, 8) == -1
    with pytest.raises(_binding.SinkhornError):
        sk.sinkhorn_describe(4, 10, 10, 0, lam=0.0)


def test_warm_start_rejections_on_host():
    lib = sk.load_library()
    v = None

    def call(p, ptr=None, ws=0):
        a = ctypes.c_void_p(ptr) if ptr else None
        return lib.sinkhorn_forward_warm(ctypes.byref(p), a, a, a, a, a, a, a, a, a, a, ctypes.c_size_t(ws), None)
    assert call(_binding.problem(4, 10, 10, 0, 0.1, 10)) == -1  # alpha0 and the arrays are NULL
    assert call(_binding.problem(0, 10, 10, 0, 0.1, 10)) == 0   # empty batch
    assert call(_binding.problem(4, 10, 10, 0, 0.0, 10)) == -3
    assert call(_binding.problem(4, 10, 10, 0, 0.1, -2)) == -4
    need = sk.sinkhorn_workspace_bytes(8, 784, 784, 0, 0.01, 10)
    assert call(_binding.problem(8, 784, 784, 0, 0.01, 10), ptr=0x1000, ws=need - 1) == -5
