"""ctypes binding of libflashdiff.so: argument marshalling only.

Every function here has the name of the C entry point it wraps and passes
torch tensors' device pointers straight through; all arithmetic happens in
the library's HIP kernels.  PyTorch provides device memory (outputs and the
workspace) and the current HIP stream.  There is no fallback: if the library
is missing, or a call fails, an exception is raised.

The library must be loaded after ``import torch`` so that it binds to the
HIP runtime torch has already loaded (both carry the same soname).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch  # noqa: F401  (load torch's HIP runtime first)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflashdiff.so")

FD_OK = 0
STATUS = {
    0: "FD_OK", 1: "FD_ERR_INVALID_ARG", 2: "FD_ERR_UNSUPPORTED", 3: "FD_ERR_WORKSPACE",
    4: "FD_ERR_HIP", 5: "FD_ERR_NOT_CONVERGED", 6: "FD_ERR_PERRON_WALL",
}
FD_F32, FD_BF16 = 0, 1
FD_OP_KERNEL_MATMUL, FD_OP_DEGREE, FD_OP_BLOCK_LANCZOS, FD_OP_CONTINUATION = 0, 1, 2, 3
FD_OP_BETA_FLOW = 4
FD_OP_DEGREE_DYADIC = 5
FLOW_EXIT = {0: "bracket", 1: "wall", 2: "budget", 3: "range"}

EXPORTS = (
    "fd_lanczos_default_opts", "fd_workspace_size", "fd_kernel_matmul", "fd_degree",
    "fd_block_lanczos", "fd_continuation", "fd_last_error", "fd_status_string",
    "fd_profile_enable", "fd_profile_read", "fd_flow_default_opts", "fd_beta_flow",
    "fd_beta_flow_cascade", "fd_degree_dyadic", "fd_kernel_matmul_noalloc",
    "fd_kernel_matmul_noalloc_limit",
)
FD_KERNEL_PRODUCT, FD_KERNEL_ROWSUM = 0, 1


class FdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status
        self.msg = msg


class LanczosOpts(ctypes.Structure):
    _fields_ = [("tol", ctypes.c_double), ("max_restarts", ctypes.c_int32),
                ("max_basis_blocks", ctypes.c_int32), ("keep", ctypes.c_int32),
                ("max_matvecs", ctypes.c_int32), ("verbose", ctypes.c_int32),
                ("seed", ctypes.c_uint64)]


class LanczosInfo(ctypes.Structure):
    _fields_ = [("restarts", ctypes.c_int32), ("block_matvecs", ctypes.c_int32),
                ("nconv", ctypes.c_int32), ("wall", ctypes.c_int32),
                ("gap_perron", ctypes.c_double), ("s_off", ctypes.c_double),
                ("max_residual", ctypes.c_double), ("seconds", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


class FlowOpts(ctypes.Structure):
    _fields_ = [("beta_start", ctypes.c_double), ("eta", ctypes.c_double),
                ("kappa", ctypes.c_double), ("p", ctypes.c_double),
                ("max_probes", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class FlowProbe(ctypes.Structure):
    _fields_ = [("beta", ctypes.c_double), ("s_off", ctypes.c_double),
                ("gap_perron", ctypes.c_double), ("v_bias", ctypes.c_double),
                ("v_mach", ctypes.c_double), ("n_eff", ctypes.c_double),
                ("v_stat", ctypes.c_double), ("v_total", ctypes.c_double),
                ("d_hat", ctypes.c_double), ("seconds", ctypes.c_double),
                ("role", ctypes.c_int32), ("admissible", ctypes.c_int32),
                ("status", ctypes.c_int32), ("block_matvecs", ctypes.c_int32),
                ("nconv", ctypes.c_int32), ("level", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "reserved"}


_c_i64 = ctypes.c_int64
_c_p = ctypes.c_void_p
_LIB = None


def load(path: str = LIB_PATH):
    """Load the library (once) and declare the signatures."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise FdError(2, f"{path} is not built; run __graft_entry__.build() or "
                         "python -m paper_2609_38198_amd.build")
    lib = ctypes.CDLL(path)
    lib.fd_lanczos_default_opts.argtypes = [ctypes.POINTER(LanczosOpts)]
    lib.fd_lanczos_default_opts.restype = None
    lib.fd_workspace_size.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64, _c_i64,
                                      ctypes.POINTER(LanczosOpts)]
    lib.fd_workspace_size.restype = ctypes.c_size_t
    lib.fd_kernel_matmul.argtypes = [_c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64, ctypes.c_int,
                                     ctypes.c_float, _c_p, _c_p, _c_p, _c_i64, _c_i64, _c_p,
                                     _c_i64, _c_p, ctypes.c_size_t, _c_p]
    lib.fd_kernel_matmul.restype = ctypes.c_int
    lib.fd_kernel_matmul_noalloc.argtypes = [_c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64,
                                             ctypes.c_int, ctypes.c_float, _c_p, _c_p, _c_p,
                                             _c_i64, _c_i64, _c_p, _c_i64, _c_p]
    lib.fd_kernel_matmul_noalloc.restype = ctypes.c_int
    lib.fd_kernel_matmul_noalloc_limit.argtypes = []
    lib.fd_kernel_matmul_noalloc_limit.restype = ctypes.c_size_t
    lib.fd_degree.argtypes = [_c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_float,
                              ctypes.c_float, _c_p, _c_p, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]
    lib.fd_degree.restype = ctypes.c_int
    lib.fd_degree_dyadic.argtypes = [_c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_float,
                                     ctypes.c_int32, ctypes.c_float, _c_p, _c_p, _c_p, _c_p, _c_p,
                                     ctypes.c_size_t, _c_p]
    lib.fd_degree_dyadic.restype = ctypes.c_int
    lib.fd_block_lanczos.argtypes = [
        _c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_float, ctypes.c_float, _c_i64, _c_i64,
        _c_p, _c_i64, _c_i64, ctypes.c_int32, ctypes.POINTER(LanczosOpts), _c_p, _c_p, _c_p, _c_p,
        ctypes.POINTER(LanczosInfo), _c_p, ctypes.c_size_t, _c_p]
    lib.fd_block_lanczos.restype = ctypes.c_int
    lib.fd_continuation.argtypes = [
        _c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_float, _c_p, _c_p, _c_i64, _c_i64,
        _c_i64, _c_p, _c_i64, _c_i64, ctypes.POINTER(LanczosOpts), _c_p, _c_p, _c_p,
        ctypes.POINTER(LanczosInfo), ctypes.c_int32, _c_p, _c_p, ctypes.c_size_t, _c_p]
    lib.fd_continuation.restype = ctypes.c_int
    lib.fd_flow_default_opts.argtypes = [ctypes.POINTER(FlowOpts)]
    lib.fd_flow_default_opts.restype = None
    lib.fd_beta_flow.argtypes = [
        _c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_float, _c_i64, _c_i64,
        ctypes.POINTER(FlowOpts), ctypes.POINTER(LanczosOpts), ctypes.POINTER(FlowProbe),
        ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
        ctypes.POINTER(ctypes.c_int32), _c_p, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]
    lib.fd_beta_flow.restype = ctypes.c_int
    lib.fd_beta_flow_cascade.argtypes = [
        ctypes.POINTER(_c_p), ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int64),
        ctypes.c_int32, _c_i64, _c_i64, ctypes.c_float, _c_i64, _c_i64,
        ctypes.POINTER(FlowOpts), ctypes.POINTER(LanczosOpts), ctypes.POINTER(FlowProbe),
        ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
        ctypes.POINTER(ctypes.c_int32), _c_p, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]
    lib.fd_beta_flow_cascade.restype = ctypes.c_int
    lib.fd_last_error.argtypes = []
    lib.fd_last_error.restype = ctypes.c_char_p
    lib.fd_status_string.argtypes = [ctypes.c_int]
    lib.fd_status_string.restype = ctypes.c_char_p
    lib.fd_profile_enable.argtypes = [ctypes.c_int32]
    lib.fd_profile_enable.restype = None
    lib.fd_profile_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int64)]
    lib.fd_profile_read.restype = ctypes.c_int
    _LIB = lib
    return lib


def _check(status: int, allow=(FD_OK,)) -> int:
    if status not in allow:
        raise FdError(status, load().fd_last_error().decode())
    return status


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dtype_code(X: torch.Tensor) -> int:
    if X.dtype == torch.float32:
        return FD_F32
    if X.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return FD_BF16
    raise TypeError(f"X must be float32 or bfloat16, got {X.dtype}")


def _check_dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("all tensors must live on the GPU")


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 256-byte aligned blocks
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def fd_profile_enable(on: bool = True) -> None:
    load().fd_profile_enable(int(bool(on)))


def fd_profile_read(kind: int) -> "tuple[float, int]":
    """(summed kernel milliseconds, timed launches) of one kernel kind; clears it."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(load().fd_profile_read(kind, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def default_opts(**kw) -> LanczosOpts:
    o = LanczosOpts()
    load().fd_lanczos_default_opts(ctypes.byref(o))
    for k, v in kw.items():
        if not hasattr(o, k):
            raise AttributeError(k)
        setattr(o, k, v)
    return o


def fd_workspace_size(op: int, Nr: int, Nc: int, D: int, b: int = 1, k: int = 1,
                      opts: Optional[LanczosOpts] = None) -> int:
    return int(load().fd_workspace_size(op, Nr, Nc, D, b, k,
                                        None if opts is None else ctypes.byref(opts)))


def fd_kernel_matmul(Xr: torch.Tensor, Xc: Optional[torch.Tensor], beta: float, V: torch.Tensor,
                     sl: Optional[torch.Tensor] = None, sr: Optional[torch.Tensor] = None,
                     Y: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Y = diag(sl) K(Xr, Xc) diag(sr) V (Xc = None: the square product on Xr)."""
    lib = load()
    if Xc is None:
        Xc = Xr
    _check_dev(Xr, Xc, V, sl, sr, Y)
    if Xr.dim() != 2 or Xc.dim() != 2 or Xr.shape[1] != Xc.shape[1]:
        raise ValueError("Xr and Xc must be N x D with the same D")
    if Xr.stride(1) != 1 or Xc.stride(1) != 1 or Xr.stride(0) != Xc.stride(0):
        raise ValueError("Xr and Xc must be row-major with the same leading dimension")
    V2 = V.unsqueeze(1) if V.dim() == 1 else V
    if V2.dtype != torch.float32 or V2.stride(1) != 1:
        raise ValueError("V must be float32 row-major")
    Nr, D = Xr.shape
    Nc = Xc.shape[0]
    b = V2.shape[1]
    if V2.shape[0] != Nc:
        raise ValueError("V must have Nc rows")
    if Y is None:
        Y = torch.empty((Nr, b), dtype=torch.float32, device=Xr.device)
    Y2 = Y.unsqueeze(1) if Y.dim() == 1 else Y
    for t, n in ((sl, Nr), (sr, Nc)):
        if t is not None and (t.dtype != torch.float32 or t.numel() != n or not t.is_contiguous()):
            raise ValueError("sl / sr must be contiguous float32 vectors of matching length")
    need = fd_workspace_size(FD_OP_KERNEL_MATMUL, Nr, Nc, D, b)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, Xr.device)
    _check(lib.fd_kernel_matmul(_ptr(Xr), Nr, _ptr(Xc), Nc, D, Xr.stride(0), _dtype_code(Xr),
                                float(beta), _ptr(sl), _ptr(sr), _ptr(V2), b, V2.stride(0),
                                _ptr(Y2), Y2.stride(0), _ptr(ws), ws.numel(),
                                _stream(Xr.device)))
    return Y


def fd_kernel_matmul_noalloc(Xr: torch.Tensor, Xc: Optional[torch.Tensor], beta: float,
                             V: torch.Tensor, Y: torch.Tensor,
                             sl: Optional[torch.Tensor] = None,
                             sr: Optional[torch.Tensor] = None) -> torch.Tensor:
    """fd_kernel_matmul into a caller-provided Y, using the library's built-in
    scratch instead of a workspace (the call allocates nothing)."""
    lib = load()
    if Xc is None:
        Xc = Xr
    _check_dev(Xr, Xc, V, sl, sr, Y)
    if Xr.dim() != 2 or Xc.dim() != 2 or Xr.shape[1] != Xc.shape[1]:
        raise ValueError("Xr and Xc must be N x D with the same D")
    if Xr.stride(1) != 1 or Xc.stride(1) != 1 or Xr.stride(0) != Xc.stride(0):
        raise ValueError("Xr and Xc must be row-major with the same leading dimension")
    if V.dim() != 2 or Y.dim() != 2 or V.stride(1) != 1 or Y.stride(1) != 1:
        raise ValueError("V and Y must be row-major N x b")
    if V.dtype != torch.float32 or Y.dtype != torch.float32:
        raise ValueError("V and Y must be float32")
    Nr, D = Xr.shape
    Nc, b = Xc.shape[0], V.shape[1]
    if V.shape[0] != Nc or Y.shape[0] != Nr or Y.shape[1] != b:
        raise ValueError("V must be Nc x b and Y Nr x b")
    for t, n in ((sl, Nr), (sr, Nc)):
        if t is not None and (t.dtype != torch.float32 or t.numel() != n or not t.is_contiguous()):
            raise ValueError("sl / sr must be contiguous float32 vectors of matching length")
    _check(lib.fd_kernel_matmul_noalloc(_ptr(Xr), Nr, _ptr(Xc), Nc, D, Xr.stride(0),
                                        _dtype_code(Xr), float(beta), _ptr(sl), _ptr(sr),
                                        _ptr(V), b, V.stride(0), _ptr(Y), Y.stride(0),
                                        _stream(Xr.device)))
    return Y


def fd_kernel_matmul_noalloc_limit() -> int:
    return int(load().fd_kernel_matmul_noalloc_limit())


@dataclass
class Degree:
    q: torch.Tensor
    d: torch.Tensor
    s: torch.Tensor
    s_off: torch.Tensor   # one float64 on the device


def fd_degree(X: torch.Tensor, beta: float, alpha: float = 0.5,
              ws: Optional[torch.Tensor] = None) -> Degree:
    """q = K 1, d = w (K w) with w = q^-alpha, s = w d^-1/2, S_off = sum(q) - N."""
    lib = load()
    _check_dev(X)
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be row-major N x D")
    N, D = X.shape
    dev = X.device
    q = torch.empty(N, dtype=torch.float32, device=dev)
    d = torch.empty_like(q)
    s = torch.empty_like(q)
    s_off = torch.empty(1, dtype=torch.float64, device=dev)
    need = fd_workspace_size(FD_OP_DEGREE, N, N, D)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(lib.fd_degree(_ptr(X), _dtype_code(X), N, D, X.stride(0), float(beta), float(alpha),
                         _ptr(q), _ptr(d), _ptr(s), _ptr(s_off), _ptr(ws), ws.numel(),
                         _stream(dev)))
    return Degree(q, d, s, s_off)


def fd_degree_dyadic(X: torch.Tensor, beta0: float, nbeta: int, alpha: float = 0.5,
                     ws: Optional[torch.Tensor] = None) -> Degree:
    """fd_degree at beta0 * 2^l for l < nbeta: q, d, s are nbeta x N, s_off nbeta."""
    lib = load()
    _check_dev(X)
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be row-major N x D")
    N, D = X.shape
    dev = X.device
    q = torch.empty((nbeta, N), dtype=torch.float32, device=dev)
    d = torch.empty_like(q)
    s = torch.empty_like(q)
    s_off = torch.empty(nbeta, dtype=torch.float64, device=dev)
    need = fd_workspace_size(FD_OP_DEGREE_DYADIC, N, N, D)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(lib.fd_degree_dyadic(_ptr(X), _dtype_code(X), N, D, X.stride(0), float(beta0),
                                int(nbeta), float(alpha), _ptr(q), _ptr(d), _ptr(s),
                                _ptr(s_off), _ptr(ws), ws.numel(), _stream(dev)))
    return Degree(q, d, s, s_off)


@dataclass
class Eigen:
    evals: "list[float]"
    evecs: torch.Tensor
    psi: Optional[torch.Tensor]
    residuals: "list[float]"
    info: dict
    status: int


def fd_block_lanczos(X: torch.Tensor, beta: float, k: int, b: int, alpha: float = 0.5,
                     V0: Optional[torch.Tensor] = None, warm_is_psi: bool = True,
                     opts: Optional[LanczosOpts] = None, want_psi: bool = True,
                     ws: Optional[torch.Tensor] = None, allow_not_converged: bool = False) -> Eigen:
    """Top-k eigenpairs of M = diag(s) K diag(s) (Perron pair included)."""
    lib = load()
    _check_dev(X, V0)
    N, D = X.shape
    dev = X.device
    o = opts if opts is not None else default_opts()
    evals = (ctypes.c_double * k)()
    res = (ctypes.c_double * k)()
    info = LanczosInfo()
    evecs = torch.empty((N, k), dtype=torch.float32, device=dev)
    psi = torch.empty((N, k), dtype=torch.float32, device=dev) if want_psi else None
    k0 = 0 if V0 is None else V0.shape[1]
    ldv0 = 0 if V0 is None else V0.stride(0)
    need = fd_workspace_size(FD_OP_BLOCK_LANCZOS, N, N, D, b, k, o)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    allow = (FD_OK, 5) if allow_not_converged else (FD_OK,)
    st = _check(lib.fd_block_lanczos(_ptr(X), _dtype_code(X), N, D, X.stride(0), float(beta),
                                     float(alpha), b, k, _ptr(V0), k0, ldv0, int(warm_is_psi),
                                     ctypes.byref(o), evals, _ptr(evecs), _ptr(psi), res,
                                     ctypes.byref(info), _ptr(ws), ws.numel(), _stream(dev)),
                allow)
    return Eigen(list(evals), evecs, psi, list(res), info.as_dict(), st)


@dataclass
class Ladder:
    evals: "list[list[float]]"
    evecs: torch.Tensor
    psi: Optional[torch.Tensor]
    info: "list[dict]"
    steps_done: int
    status: int


def fd_continuation(X: torch.Tensor, n_steps: Sequence[int], beta_steps: Sequence[float], k: int,
                    b: int, alpha: float = 0.5, V0: Optional[torch.Tensor] = None,
                    opts: Optional[LanczosOpts] = None, stop_at_wall: bool = False,
                    want_psi: bool = True, ws: Optional[torch.Tensor] = None,
                    allow=(FD_OK,)) -> Ladder:
    """Warm-started ladder over prefixes X[:n_t] and bandwidths beta_t."""
    lib = load()
    _check_dev(X, V0)
    N, D = X.shape
    dev = X.device
    T = len(n_steps)
    if T != len(beta_steps) or T == 0:
        raise ValueError("n_steps and beta_steps must have the same non-zero length")
    o = opts if opts is not None else default_opts()
    ns = (ctypes.c_int64 * T)(*[int(n) for n in n_steps])
    bs = (ctypes.c_float * T)(*[float(x) for x in beta_steps])
    evals = (ctypes.c_double * (T * k))()
    infos = (LanczosInfo * T)()
    nlast = int(n_steps[-1])
    evecs = torch.empty((nlast, k), dtype=torch.float32, device=dev)
    psi = torch.empty((nlast, k), dtype=torch.float32, device=dev) if want_psi else None
    done = ctypes.c_int64(0)
    k0 = 0 if V0 is None else V0.shape[1]
    ldv0 = 0 if V0 is None else V0.stride(0)
    need = fd_workspace_size(FD_OP_CONTINUATION, max(int(n) for n in n_steps), T, D, b, k, o)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    st = _check(lib.fd_continuation(_ptr(X), _dtype_code(X), N, D, X.stride(0), float(alpha), ns, bs,
                                    T, b, k, _ptr(V0), k0, ldv0, ctypes.byref(o), evals,
                                    _ptr(evecs), _ptr(psi), infos, int(stop_at_wall),
                                    ctypes.byref(done), _ptr(ws), ws.numel(), _stream(dev)),
                allow)
    ev = [[evals[t * k + i] for i in range(k)] for t in range(T)]
    return Ladder(ev, evecs, psi, [infos[t].as_dict() for t in range(T)], done.value, st)


def flow_default_opts(**kw) -> FlowOpts:
    o = FlowOpts()
    load().fd_flow_default_opts(ctypes.byref(o))
    for key, v in kw.items():
        setattr(o, key, v)
    return o


@dataclass
class Flow:
    probes: list       # per-probe records (dicts), in the order run
    beta_x: float      # achieved bandwidth
    reason: str        # "bracket", "wall", "budget" or "range"
    evals: list
    evecs: torch.Tensor
    psi: Optional[torch.Tensor]
    status: int


def fd_beta_flow(X: torch.Tensor, k: int, b: int, alpha: float = 0.5,
                 fopts: Optional[FlowOpts] = None, opts: Optional[LanczosOpts] = None,
                 want_psi: bool = True, ws: Optional[torch.Tensor] = None,
                 allow=(FD_OK,)) -> Flow:
    """Bandwidth selection by the beta-function flow; eigenpairs at beta_x."""
    lib = load()
    _check_dev(X)
    N, D = X.shape
    dev = X.device
    fo = fopts if fopts is not None else flow_default_opts()
    o = opts if opts is not None else default_opts()
    cap = int(fo.max_probes) + 2
    recs = (FlowProbe * cap)()
    nrec = ctypes.c_int64(0)
    bx = ctypes.c_double(0.0)
    why = ctypes.c_int32(0)
    evals = (ctypes.c_double * k)()
    evecs = torch.empty((N, k), dtype=torch.float32, device=dev)
    psi = torch.empty((N, k), dtype=torch.float32, device=dev) if want_psi else None
    need = fd_workspace_size(FD_OP_BETA_FLOW, N, N, D, b, k, o)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    st = _check(lib.fd_beta_flow(_ptr(X), _dtype_code(X), N, D, X.stride(0), float(alpha), b, k,
                                 ctypes.byref(fo), ctypes.byref(o), recs, ctypes.byref(nrec),
                                 ctypes.byref(bx), ctypes.byref(why), evals, _ptr(evecs),
                                 _ptr(psi), _ptr(ws), ws.numel(), _stream(dev)), allow)
    return Flow([recs[i].as_dict() for i in range(nrec.value)], bx.value,
                FLOW_EXIT.get(why.value, str(why.value)), [evals[i] for i in range(k)], evecs,
                psi, st)


def fd_beta_flow_cascade(Xs: Sequence[torch.Tensor], k: int, b: int, alpha: float = 0.5,
                         fopts: Optional[FlowOpts] = None, opts: Optional[LanczosOpts] = None,
                         want_psi: bool = True, ws: Optional[torch.Tensor] = None,
                         allow=(FD_OK,)) -> Flow:
    """Precision cascade of the flow: the same points in each dtype of Xs, lowest first."""
    lib = load()
    Xs = list(Xs)
    if not 1 <= len(Xs) <= 4:
        raise ValueError("the cascade takes 1 to 4 levels")
    for X in Xs:
        _check_dev(X)
        if X.dim() != 2 or X.stride(1) != 1 or X.shape != Xs[0].shape:
            raise ValueError("every level must be the same row-major N x D points")
    N, D = Xs[0].shape
    dev = Xs[0].device
    fo = fopts if fopts is not None else flow_default_opts()
    o = opts if opts is not None else default_opts()
    cap = len(Xs) * (int(fo.max_probes) + 2)
    recs = (FlowProbe * cap)()
    nrec = ctypes.c_int64(0)
    bx = ctypes.c_double(0.0)
    why = ctypes.c_int32(0)
    evals = (ctypes.c_double * k)()
    evecs = torch.empty((N, k), dtype=torch.float32, device=dev)
    psi = torch.empty((N, k), dtype=torch.float32, device=dev) if want_psi else None
    need = fd_workspace_size(FD_OP_BETA_FLOW, N, N, D, b, k, o)
    if need == 0:
        raise FdError(1, "unsupported sizes")
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    ptrs = (_c_p * len(Xs))(*[X.data_ptr() for X in Xs])
    codes = (ctypes.c_int * len(Xs))(*[_dtype_code(X) for X in Xs])
    lds = (ctypes.c_int64 * len(Xs))(*[X.stride(0) for X in Xs])
    st = _check(lib.fd_beta_flow_cascade(ptrs, codes, lds, len(Xs), N, D, float(alpha), b, k,
                                         ctypes.byref(fo), ctypes.byref(o), recs,
                                         ctypes.byref(nrec), ctypes.byref(bx), ctypes.byref(why),
                                         evals, _ptr(evecs), _ptr(psi), _ptr(ws), ws.numel(),
                                         _stream(dev)), allow)
    return Flow([recs[i].as_dict() for i in range(nrec.value)], bx.value,
                FLOW_EXIT.get(why.value, str(why.value)), [evals[i] for i in range(k)], evecs,
                psi, st)
