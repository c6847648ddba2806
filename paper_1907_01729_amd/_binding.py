"""ctypes binding of include/sinkhorn.h (argument marshalling only)."""
from __future__ import annotations

import contextlib
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsinkhorn_hip.so")
_lib = None

SK_STATUS = {
    0: "SK_OK",
    -1: "SK_ERR_NULLPTR",
    -2: "SK_ERR_SHAPE",
    -3: "SK_ERR_LAMBDA",
    -4: "SK_ERR_ITERS",
    -5: "SK_ERR_WORKSPACE",
    -6: "SK_ERR_HIP",
    -7: "SK_ERR_ARG",
}

# Selector values of sinkhorn_forward_select (sk_select in include/sinkhorn.h).
SK_SELECT = {"default": 0, "log": 1, "plain": 2, "nosym": 3, "nocompact": 4}

EXPORTED = (
    "sinkhorn_workspace_bytes",
    "sinkhorn_forward",
    "sinkhorn_forward_select",
    "sinkhorn_forward_noalloc",
    "sinkhorn_backward",
    "sinkhorn_status_string",
    "sinkhorn_regime",
    "sinkhorn_points_workspace_bytes",
    "sinkhorn_forward_points",
    "sinkhorn_backward_points",
    "sinkhorn_backward_sharp",
    "sinkhorn_sharp_workspace_bytes",
    "sinkhorn_describe",
    "sinkhorn_forward_warm",
)


class SinkhornError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {SK_STATUS.get(status, status)} ({sinkhorn_status_string(status)})")


class SkProblem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32),
        ("d1", ctypes.c_int32),
        ("d2", ctypes.c_int32),
        ("c_batched", ctypes.c_int32),
        ("lam", ctypes.c_float),
        ("n_iter", ctypes.c_int32),
        ("tol", ctypes.c_float),
    ]


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libsinkhorn_hip.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build it with `python paper_1907_01729_amd/build.py` "
            "(or __graft_entry__.build()); there is no CPU fallback")
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    PP = ctypes.POINTER(SkProblem)
    lib.sinkhorn_workspace_bytes.argtypes = [PP]
    lib.sinkhorn_workspace_bytes.restype = ctypes.c_size_t
    lib.sinkhorn_forward.argtypes = [PP, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sinkhorn_forward.restype = ctypes.c_int
    lib.sinkhorn_forward_select.argtypes = [PP, ctypes.c_int32, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sinkhorn_forward_select.restype = ctypes.c_int
    lib.sinkhorn_forward_noalloc.argtypes = [PP, P, P, P, P, P, P, P, P, P]
    lib.sinkhorn_forward_noalloc.restype = ctypes.c_int
    lib.sinkhorn_backward.argtypes = [PP, P, P, P, P, P, P, P, P, P, P]
    lib.sinkhorn_backward.restype = ctypes.c_int
    lib.sinkhorn_status_string.argtypes = [ctypes.c_int]
    lib.sinkhorn_status_string.restype = ctypes.c_char_p
    lib.sinkhorn_regime.argtypes = [PP]
    lib.sinkhorn_regime.restype = ctypes.c_int32
    I = ctypes.c_int32
    lib.sinkhorn_points_workspace_bytes.argtypes = [PP, I]
    lib.sinkhorn_points_workspace_bytes.restype = ctypes.c_size_t
    lib.sinkhorn_forward_points.argtypes = [PP, I, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sinkhorn_forward_points.restype = ctypes.c_int
    lib.sinkhorn_backward_points.argtypes = [PP, I, P, P, P, P, P, P, P, P, P, P, P, P]
    lib.sinkhorn_backward_points.restype = ctypes.c_int
    lib.sinkhorn_backward_sharp.argtypes = [PP, P, P, P, P, P, P, P, P, I, ctypes.c_float, P, P, ctypes.c_size_t, P]
    lib.sinkhorn_backward_sharp.restype = ctypes.c_int
    lib.sinkhorn_sharp_workspace_bytes.argtypes = [PP]
    lib.sinkhorn_sharp_workspace_bytes.restype = ctypes.c_size_t
    lib.sinkhorn_forward_warm.argtypes = [PP, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.sinkhorn_forward_warm.restype = ctypes.c_int
    lib.sinkhorn_describe.argtypes = [PP, I, ctypes.c_char_p, ctypes.c_size_t]
    lib.sinkhorn_describe.restype = ctypes.c_int32
    _lib = lib
    return lib


def problem(B, d1, d2, c_batched, lam, n_iter, tol=0.0) -> SkProblem:
    return SkProblem(int(B), int(d1), int(d2), int(c_batched), float(lam), int(n_iter), float(tol))


def sinkhorn_status_string(status: int) -> str:
    return load_library().sinkhorn_status_string(int(status)).decode()


def sinkhorn_workspace_bytes(B, d1, d2, c_batched, lam, n_iter, tol=0.0) -> int:
    p = problem(B, d1, d2, c_batched, lam, n_iter, tol)
    return int(load_library().sinkhorn_workspace_bytes(ctypes.byref(p)))


def sinkhorn_regime(B, d1, d2, c_batched, lam=1.0, n_iter=1, tol=0.0) -> int:
    p = problem(B, d1, d2, c_batched, lam, n_iter, tol)
    return int(load_library().sinkhorn_regime(ctypes.byref(p)))


def sinkhorn_describe(B, d1, d2, c_batched=0, lam=1.0, n_iter=1, tol=0.0, select="default") -> str:
    """The kernels and launch shape a forward takes for this problem (one line;
    nothing is launched).  Raises SinkhornError for an invalid problem."""
    if select not in SK_SELECT:
        raise ValueError(f"select must be one of {sorted(SK_SELECT)}, got {select!r}")
    lib = load_library()
    p = problem(B, d1, d2, c_batched, lam, n_iter, tol)
    n = int(lib.sinkhorn_describe(ctypes.byref(p), SK_SELECT[select], None, 0))
    if n < 0:
        raise SinkhornError(n, "sinkhorn_describe")
    buf = ctypes.create_string_buffer(n + 1)
    lib.sinkhorn_describe(ctypes.byref(p), SK_SELECT[select], buf, n + 1)
    return buf.value.decode()


def _dev(t: torch.Tensor, name: str, dtype=torch.float32) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _shapes(mu, nu, C):
    if mu.dim() != 2 or nu.dim() != 2 or mu.shape[0] != nu.shape[0]:
        raise ValueError(f"mu must be [B,d1] and nu [B,d2], got {tuple(mu.shape)} {tuple(nu.shape)}")
    B, d1 = mu.shape
    d2 = nu.shape[1]
    if C.dim() == 2:
        C = C.unsqueeze(0)
    if C.dim() != 3 or tuple(C.shape[1:]) != (d1, d2) or C.shape[0] not in (1, B):
        raise ValueError(f"C must be [d1,d2], [1,d1,d2] or [B,d1,d2], got {tuple(C.shape)}")
    c_batched = int(C.shape[0] == B and B != 1)
    return B, d1, d2, c_batched


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(device, stream=None):
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _on(stream):
    """Context in which outputs and the workspace are allocated: the stream the
    library will run on, so that PyTorch's caching allocator orders their reuse
    after the library's kernels (a temporary workspace is freed on return,
    while the kernels may still be using it)."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def _forward(select, mu, nu, C, lam, n_iter, tol, stream, workspace, alpha0=None):
    lib = load_library()
    _dev(mu, "mu"), _dev(nu, "nu"), _dev(C, "C")
    B, d1, d2, cb = _shapes(mu, nu, C)
    if alpha0 is not None:
        _dev(alpha0, "alpha0")
        if tuple(alpha0.shape) != (B, d1):
            raise ValueError(f"alpha0 must be [B, d1] = [{B}, {d1}], got {tuple(alpha0.shape)}")
    p = problem(B, d1, d2, cb, lam, n_iter, tol)
    dev = mu.device
    f = dict(device=dev, dtype=torch.float32)
    with _on(stream):
        alpha = torch.empty((B, d1), **f)
        beta = torch.empty((B, d2), **f)
        loss = torch.empty((B,), **f)
        merr = torch.empty((B,), **f)
        iters = torch.empty((B,), device=dev, dtype=torch.int32)
        need = int(lib.sinkhorn_workspace_bytes(ctypes.byref(p)))
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty((max(need, 1),), device=dev, dtype=torch.uint8)
    if alpha0 is not None:
        st = lib.sinkhorn_forward_warm(ctypes.byref(p), _ptr(alpha0), _ptr(mu), _ptr(nu), _ptr(C), _ptr(alpha),
                                       _ptr(beta), _ptr(loss), _ptr(merr), _ptr(iters), _ptr(workspace),
                                       ctypes.c_size_t(workspace.numel()), _stream(dev, stream))
        if st != 0:
            raise SinkhornError(st, "sinkhorn_forward_warm")
        return dict(alpha=alpha, beta=beta, loss=loss, marg_err=merr, iters=iters)
    st = lib.sinkhorn_forward_select(ctypes.byref(p), int(select), _ptr(mu), _ptr(nu), _ptr(C), _ptr(alpha),
                                     _ptr(beta), _ptr(loss), _ptr(merr), _ptr(iters), _ptr(workspace),
                                     ctypes.c_size_t(workspace.numel()), _stream(dev, stream))
    if st != 0:
        raise SinkhornError(st, "sinkhorn_forward" if select == 0 else "sinkhorn_forward_select")
    return dict(alpha=alpha, beta=beta, loss=loss, marg_err=merr, iters=iters)


def sinkhorn_forward(mu, nu, C, lam, n_iter, tol=0.0, stream=None, workspace=None, alpha0=None):
    """Run the forward on the GPU.

    mu [B,d1], nu [B,d2], C [d1,d2] | [1,d1,d2] | [B,d1,d2]: float32 CUDA tensors.
    alpha0 [B,d1] (optional): warm start from these row log-scalings (e.g. the
    alpha of an earlier forward: n more iterations continue it), through
    sinkhorn_forward_warm.
    Returns dict(alpha [B,d1], beta [B,d2], loss [B], marg_err [B], iters [B] int32).
    """
    return _forward(0, mu, nu, C, lam, n_iter, tol, stream, workspace, alpha0)


# Size of the library's fixed scratch array (SINKHORN_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 32 << 20


def sinkhorn_forward_noalloc(mu, nu, C, lam, n_iter, tol=0.0, stream=None, out=None):
    """Forward through the entry point that allocates nothing: its scratch is
    the library's fixed per-GPU array.  out (optional) = dict of preallocated
    outputs (alpha, beta, loss, marg_err, iters), else they are allocated here."""
    lib = load_library()
    _dev(mu, "mu"), _dev(nu, "nu"), _dev(C, "C")
    B, d1, d2, cb = _shapes(mu, nu, C)
    p = problem(B, d1, d2, cb, lam, n_iter, tol)
    dev = mu.device
    if out is None:
        f = dict(device=dev, dtype=torch.float32)
        with _on(stream):
            out = dict(alpha=torch.empty((B, d1), **f), beta=torch.empty((B, d2), **f), loss=torch.empty((B,), **f),
                       marg_err=torch.empty((B,), **f), iters=torch.empty((B,), device=dev, dtype=torch.int32))
    st = lib.sinkhorn_forward_noalloc(ctypes.byref(p), _ptr(mu), _ptr(nu), _ptr(C), _ptr(out["alpha"]),
                                      _ptr(out["beta"]), _ptr(out["loss"]), _ptr(out["marg_err"]),
                                      _ptr(out["iters"]), _stream(dev, stream))
    if st != 0:
        raise SinkhornError(st, "sinkhorn_forward_noalloc")
    return out


def sinkhorn_forward_select(select, mu, nu, C, lam, n_iter, tol=0.0, stream=None, workspace=None):
    """Diagnostic forward with pinned kernels: select is one of "default",
    "log", "plain", "nosym", "nocompact" (see sk_select in sinkhorn.h)."""
    if select not in SK_SELECT:
        raise ValueError(f"select must be one of {sorted(SK_SELECT)}, got {select!r}")
    return _forward(SK_SELECT[select], mu, nu, C, lam, n_iter, tol, stream, workspace)


def sinkhorn_backward(grad_loss, mu, nu, C, lam, alpha, beta, grad_C=False, stream=None):
    """Multiplier gradient (Section 2) on the GPU: dict(grad_mu, grad_nu[, grad_C])."""
    lib = load_library()
    for t, n in ((grad_loss, "grad_loss"), (mu, "mu"), (nu, "nu"), (C, "C"), (alpha, "alpha"), (beta, "beta")):
        _dev(t, n)
    B, d1, d2, cb = _shapes(mu, nu, C)
    p = problem(B, d1, d2, cb, lam, 0, 0.0)
    dev = mu.device
    f = dict(device=dev, dtype=torch.float32)
    with _on(stream):
        gmu = torch.empty((B, d1), **f)
        gnu = torch.empty((B, d2), **f)
        gC = torch.empty(((B if cb else 1), d1, d2), **f) if grad_C else None
    st = lib.sinkhorn_backward(ctypes.byref(p), _ptr(grad_loss), _ptr(mu), _ptr(nu), _ptr(C), _ptr(alpha),
                               _ptr(beta), _ptr(gmu), _ptr(gnu), _ptr(gC), _stream(dev, stream))
    if st != 0:
        raise SinkhornError(st, "sinkhorn_backward")
    out = dict(grad_mu=gmu, grad_nu=gnu)
    if grad_C:
        out["grad_C"] = gC
    return out


def _point_shapes(mu, nu, X, Y):
    if mu.dim() != 2 or nu.dim() != 2 or mu.shape[0] != nu.shape[0]:
        raise ValueError(f"mu must be [B,d1] and nu [B,d2], got {tuple(mu.shape)} {tuple(nu.shape)}")
    B, d1 = mu.shape
    d2 = nu.shape[1]
    if X.dim() == 2:
        X = X.unsqueeze(0)
    if Y.dim() == 2:
        Y = Y.unsqueeze(0)
    if X.dim() != 3 or Y.dim() != 3 or X.shape[0] != Y.shape[0] or X.shape[2] != Y.shape[2]:
        raise ValueError(f"X must be [(B,)d1,D] and Y [(B,)d2,D], got {tuple(X.shape)} {tuple(Y.shape)}")
    if X.shape[1] != d1 or Y.shape[1] != d2 or X.shape[0] not in (1, B):
        raise ValueError(f"X/Y shapes {tuple(X.shape)} {tuple(Y.shape)} do not match mu/nu")
    c_batched = int(X.shape[0] == B and B != 1)
    return B, d1, d2, c_batched, int(X.shape[2])


def sinkhorn_points_workspace_bytes(B, d1, d2, c_batched, D, lam, n_iter, tol=0.0) -> int:
    p = problem(B, d1, d2, c_batched, lam, n_iter, tol)
    return int(load_library().sinkhorn_points_workspace_bytes(ctypes.byref(p), int(D)))


def sinkhorn_forward_points(mu, nu, X, Y, lam, n_iter, tol=0.0, stream=None, workspace=None):
    """Forward with the cost C_ij = |X_i - Y_j|^2 given by point clouds.

    X [d1,D] | [1,d1,D] | [B,d1,D], Y [d2,D] | [1,d2,D] | [B,d2,D] (shared or per-sample clouds).
    Returns the same dict as sinkhorn_forward.
    """
    lib = load_library()
    for t, n in ((mu, "mu"), (nu, "nu"), (X, "X"), (Y, "Y")):
        _dev(t, n)
    B, d1, d2, cb, D = _point_shapes(mu, nu, X, Y)
    p = problem(B, d1, d2, cb, lam, n_iter, tol)
    dev = mu.device
    f = dict(device=dev, dtype=torch.float32)
    with _on(stream):
        alpha = torch.empty((B, d1), **f)
        beta = torch.empty((B, d2), **f)
        loss = torch.empty((B,), **f)
        merr = torch.empty((B,), **f)
        iters = torch.empty((B,), device=dev, dtype=torch.int32)
        need = int(lib.sinkhorn_points_workspace_bytes(ctypes.byref(p), D))
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty((max(need, 1),), device=dev, dtype=torch.uint8)
    st = lib.sinkhorn_forward_points(ctypes.byref(p), D, _ptr(mu), _ptr(nu), _ptr(X), _ptr(Y), _ptr(alpha),
                                     _ptr(beta), _ptr(loss), _ptr(merr), _ptr(iters), _ptr(workspace),
                                     ctypes.c_size_t(workspace.numel()), _stream(dev, stream))
    if st != 0:
        raise SinkhornError(st, "sinkhorn_forward_points")
    return dict(alpha=alpha, beta=beta, loss=loss, marg_err=merr, iters=iters)


def sinkhorn_backward_points(grad_loss, mu, nu, X, Y, lam, alpha, beta, grad_points=False, stream=None):
    """Multiplier gradient for point clouds: dict(grad_mu, grad_nu[, grad_X, grad_Y])."""
    lib = load_library()
    for t, n in ((grad_loss, "grad_loss"), (mu, "mu"), (nu, "nu"), (X, "X"), (Y, "Y"), (alpha, "alpha"),
                 (beta, "beta")):
        _dev(t, n)
    B, d1, d2, cb, D = _point_shapes(mu, nu, X, Y)
    p = problem(B, d1, d2, cb, lam, 0, 0.0)
    dev = mu.device
    f = dict(device=dev, dtype=torch.float32)
    with _on(stream):
        gmu = torch.empty((B, d1), **f)
        gnu = torch.empty((B, d2), **f)
        gX = torch.empty(X.shape, **f) if grad_points else None
        gY = torch.empty(Y.shape, **f) if grad_points else None
    st = lib.sinkhorn_backward_points(ctypes.byref(p), D, _ptr(grad_loss), _ptr(mu), _ptr(nu), _ptr(X), _ptr(Y),
                                      _ptr(alpha), _ptr(beta), _ptr(gmu), _ptr(gnu), _ptr(gX), _ptr(gY),
                                      _stream(dev, stream))
    if st != 0:
        raise SinkhornError(st, "sinkhorn_backward_points")
    out = dict(grad_mu=gmu, grad_nu=gnu)
    if grad_points:
        out["grad_X"] = gX
        out["grad_Y"] = gY
    return out


def sinkhorn_sharp_workspace_bytes(B, d1, d2, c_batched, lam=1.0) -> int:
    p = problem(B, d1, d2, c_batched, lam, 0, 0.0)
    return int(load_library().sinkhorn_sharp_workspace_bytes(ctypes.byref(p)))


def sinkhorn_backward_sharp(grad_loss, mu, nu, C, lam, alpha, beta, max_cg=200, cg_tol=1e-6, stream=None,
                            workspace=None):
    """Gradient of the sharp loss E^0 itself (implicit differentiation of the
    plan, conjugate gradients per problem): dict(grad_mu, grad_nu, cg_iters)."""
    lib = load_library()
    for t, n in ((grad_loss, "grad_loss"), (mu, "mu"), (nu, "nu"), (C, "C"), (alpha, "alpha"), (beta, "beta")):
        _dev(t, n)
    B, d1, d2, cb = _shapes(mu, nu, C)
    p = problem(B, d1, d2, cb, lam, 0, 0.0)
    dev = mu.device
    f = dict(device=dev, dtype=torch.float32)
    with _on(stream):
        gmu = torch.empty((B, d1), **f)
        gnu = torch.empty((B, d2), **f)
        its = torch.empty((B,), device=dev, dtype=torch.int32)
        need = int(lib.sinkhorn_sharp_workspace_bytes(ctypes.byref(p)))
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty((max(need, 1),), device=dev, dtype=torch.uint8)
    st = lib.sinkhorn_backward_sharp(ctypes.byref(p), _ptr(grad_loss), _ptr(mu), _ptr(nu), _ptr(C), _ptr(alpha),
                                     _ptr(beta), _ptr(gmu), _ptr(gnu), int(max_cg), ctypes.c_float(cg_tol),
                                     _ptr(its), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
                                     _stream(dev, stream))
    if st != 0:
        raise SinkhornError(st, "sinkhorn_backward_sharp")
    return dict(grad_mu=gmu, grad_nu=gnu, cg_iters=its)
