"""ctypes marshalling for the C ABI of ``libbhtsne.so`` (argument passing only).

Tensors must be contiguous CUDA (HIP) tensors of the documented dtypes; their
data pointers and the current torch stream are handed to the library.  There
is no fallback: when the shared library is missing the import of a function
fails loudly.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = os.path.join(_HERE, "lib", "libbhtsne.so")

BHTSNE_OK, BHTSNE_EINVAL, BHTSNE_EWORKSPACE, BHTSNE_ENONFINITE, BHTSNE_EDEVICE = 0, -1, -2, -3, -4
BHTSNE_EINPUT, BHTSNE_ECAPACITY = -5, -6
ORDER_MORTON, ORDER_BFS, ORDER_AUTO = 0, 1, 2  # point orders of a layout (bhtsne_layout_build_ordered)
PHASES = ("bbox_morton", "sort", "tree", "repulsive", "attractive", "update")


class BhtsneError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


class _Csr(C.Structure):
    _fields_ = [("n", C.c_int64), ("nnz", C.c_int64), ("row_ptr", C.c_void_p),
                ("col", C.c_void_p), ("val", C.c_void_p)]


class _Layout(C.Structure):
    _fields_ = [("n", C.c_int64), ("nnz", C.c_int64), ("mem", C.c_void_p), ("bytes", C.c_size_t),
                ("tiles", C.c_int64), ("items", C.c_int64), ("entries", C.c_int64), ("windows", C.c_int64),
                ("segments", C.c_int64), ("order", C.c_int64), ("magic", C.c_uint64)]


class _Stats(C.Structure):
    _fields_ = [("Z", C.c_double), ("interactions", C.c_int64), ("nodes", C.c_int64),
                ("bbox", C.c_double * 4), ("r_span", C.c_double), ("device_flags", C.c_uint32),
                ("max_depth", C.c_int32)]


class _Timing(C.Structure):
    _fields_ = [("ms", C.c_double * 6), ("count", C.c_int64 * 6)]


_lib = None


def library_path() -> str:
    return _LIB


def load_library():
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        raise ImportError(f"{_LIB} is missing: build it with paper_2212_11506_amd/build.py")
    lib = C.CDLL(_LIB)
    vp, i64, f32, f64p = C.c_void_p, C.c_int64, C.c_float, C.POINTER(C.c_double)
    sigs = {
        "bhtsne_workspace_size": (C.c_size_t, [i64, i64]),
        "bhtsne_gradient": (C.c_int, [vp, C.POINTER(_Csr), f32, f32, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_step": (C.c_int, [vp, C.POINTER(_Csr), f32, f32, f32, f32, f32, vp, vp, vp, f64p, vp,
                                  C.c_size_t, vp]),
        "bhtsne_get_stats": (C.c_int, [vp, C.POINTER(_Stats), vp]),
        "bhtsne_layout_size": (C.c_size_t, [i64, i64]),
        "bhtsne_layout_build": (C.c_int, [C.POINTER(_Csr), vp, vp, C.c_size_t, C.POINTER(_Layout), vp,
                                          C.c_size_t, vp]),
        "bhtsne_layout_build_ordered": (C.c_int, [C.POINTER(_Csr), vp, C.c_int, vp, C.c_size_t, C.POINTER(_Layout),
                                                  vp, C.c_size_t, vp]),
        "bhtsne_gradient_layout": (C.c_int, [vp, C.POINTER(_Layout), f32, f32, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_step_layout": (C.c_int, [vp, C.POINTER(_Layout), f32, f32, f32, f32, f32, vp, vp, vp, f64p, vp,
                                         C.c_size_t, vp]),
        "bhtsne_status_string": (C.c_char_p, [C.c_int]),
        "bhtsne_timing_enable": (C.c_int, [C.c_int]),
        "bhtsne_timing_phases": (C.c_int, [C.c_uint32]),
        "bhtsne_z_exact": (C.c_int, [vp, i64, C.POINTER(C.c_double), vp, C.c_size_t, vp]),
        "bhtsne_kl": (C.c_int, [vp, C.POINTER(_Csr), C.c_double, C.POINTER(C.c_double), vp, C.c_size_t, vp]),
        "bhtsne_timing_read": (C.c_int, [C.POINTER(_Timing), C.c_int]),
        "bhtsne_affinities_workspace_size": (C.c_size_t, [i64, C.c_int32]),
        "bhtsne_workspace_size_f64": (C.c_size_t, [i64, i64]),
        "bhtsne_gradient_f64": (C.c_int, [vp, C.POINTER(_Csr), C.c_double, C.c_double, vp, f64p, vp, C.c_size_t,
                                          vp]),
        "bhtsne_step_f64": (C.c_int, [vp, C.POINTER(_Csr), C.c_double, C.c_double, C.c_double, C.c_double,
                                      C.c_double, vp, vp, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_affinities": (C.c_int, [vp, vp, i64, C.c_int32, C.c_double, vp, vp, vp, i64,
                                        C.POINTER(C.c_int64), vp, vp, C.c_size_t, vp]),
        "bhtsne_noalloc_max_bytes": (C.c_size_t, []),
        "bhtsne_step_noalloc": (C.c_int, [vp, C.POINTER(_Csr), f32, f32, f32, f32, f32, vp, vp, vp, f64p, vp]),
        "bhtsne_layout_size_f64": (C.c_size_t, [i64, i64]),
        "bhtsne_layout_build_f64": (C.c_int, [C.POINTER(_Csr), vp, vp, C.c_size_t, C.POINTER(_Layout), vp,
                                              C.c_size_t, vp]),
        "bhtsne_gradient_layout_f64": (C.c_int, [vp, C.POINTER(_Layout), C.c_double, C.c_double, vp, f64p, vp,
                                                 C.c_size_t, vp]),
        "bhtsne_step_layout_f64": (C.c_int, [vp, C.POINTER(_Layout), C.c_double, C.c_double, C.c_double,
                                             C.c_double, C.c_double, vp, vp, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_workspace_size_3d": (C.c_size_t, [i64, i64]),
        "bhtsne_gradient_3d": (C.c_int, [vp, C.POINTER(_Csr), f32, f32, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_step_3d": (C.c_int, [vp, C.POINTER(_Csr), f32, f32, f32, f32, f32, vp, vp, vp, f64p, vp,
                                     C.c_size_t, vp]),
        "bhtsne_layout_size_3d": (C.c_size_t, [i64, i64]),
        "bhtsne_layout_build_3d": (C.c_int, [C.POINTER(_Csr), vp, vp, C.c_size_t, C.POINTER(_Layout), vp,
                                             C.c_size_t, vp]),
        "bhtsne_gradient_layout_3d": (C.c_int, [vp, C.POINTER(_Layout), f32, f32, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_step_layout_3d": (C.c_int, [vp, C.POINTER(_Layout), f32, f32, f32, f32, f32, vp, vp, vp, f64p, vp,
                                            C.c_size_t, vp]),
        "bhtsne_debug_sort_3d": (C.c_int, [vp, i64, vp, vp, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_debug_tree_3d": (C.c_int, [vp, i64, f32, C.POINTER(C.c_int64), vp, vp, vp, vp, vp, vp, vp, vp,
                                           C.c_size_t, vp]),
        "bhtsne_debug_sort": (C.c_int, [vp, i64, vp, vp, vp, f64p, vp, C.c_size_t, vp]),
        "bhtsne_debug_tree": (C.c_int, [vp, i64, f32, C.POINTER(C.c_int64), vp, vp, vp, vp, vp, vp, vp,
                                        C.c_size_t, vp]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().bhtsne_status_string(int(status)).decode()


def _check(rc: int, where: str):
    if rc != BHTSNE_OK:
        raise BhtsneError(rc, where)


def _ptr(t: Optional[torch.Tensor], dtype=None, where="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{where} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{where} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{where} must be {dtype}, got {t.dtype}")
    return C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


class Csr:
    """Device CSR matrix P (int64 row_ptr, int32 col, float32 val)."""

    def __init__(self, row_ptr: torch.Tensor, col: torch.Tensor, val: torch.Tensor):
        self.row_ptr, self.col, self.val = row_ptr, col, val
        self.n = int(row_ptr.numel()) - 1
        self.nnz = int(col.numel())
        self._s = _Csr(self.n, self.nnz, _ptr(row_ptr, torch.int64, "row_ptr").value,
                       _ptr(col, torch.int32, "col").value if self.nnz else None,
                       _ptr(val, torch.float32, "val").value if self.nnz else None)

    @classmethod
    def from_numpy(cls, row_ptr, col, val, device="cuda"):
        return cls(torch.as_tensor(row_ptr, dtype=torch.int64).to(device),
                   torch.as_tensor(col, dtype=torch.int32).to(device),
                   torch.as_tensor(val, dtype=torch.float32).to(device))

    @property
    def struct(self):
        return C.byref(self._s)


class CsrF64(Csr):
    """Device CSR matrix P with fp64 values, for the fp64 variant (same
    struct layout as Csr: bhtsne_csr_f64)."""

    def __init__(self, row_ptr: torch.Tensor, col: torch.Tensor, val: torch.Tensor):
        self.row_ptr, self.col, self.val = row_ptr, col, val
        self.n = int(row_ptr.numel()) - 1
        self.nnz = int(col.numel())
        self._s = _Csr(self.n, self.nnz, _ptr(row_ptr, torch.int64, "row_ptr").value,
                       _ptr(col, torch.int32, "col").value if self.nnz else None,
                       _ptr(val, torch.float64, "val").value if self.nnz else None)

    @classmethod
    def from_numpy(cls, row_ptr, col, val, device="cuda"):
        return cls(torch.as_tensor(row_ptr, dtype=torch.int64).to(device),
                   torch.as_tensor(col, dtype=torch.int32).to(device),
                   torch.as_tensor(val, dtype=torch.float64).to(device))


def workspace_size_f64(n: int, nnz: int) -> int:
    return int(load_library().bhtsne_workspace_size_f64(int(n), int(nnz)))


def gradient_f64(Y: torch.Tensor, P: "CsrF64", theta: float, exaggeration: float = 1.0,
                 grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                 return_z: bool = True):
    """bhtsne_gradient_f64: returns (grad fp64, Z or None)."""
    lib = load_library()
    if not isinstance(P, (CsrF64, LayoutF64)):
        raise TypeError("gradient_f64 takes P as a CsrF64 or a LayoutF64")
    if grad is None:
        grad = torch.empty_like(Y)
    ws = workspace if workspace is not None else torch.empty(workspace_size_f64(P.n, P.nnz), dtype=torch.uint8,
                                                             device=Y.device)
    z = C.c_double(0.0)
    fn = lib.bhtsne_gradient_layout_f64 if isinstance(P, LayoutF64) else lib.bhtsne_gradient_f64
    rc = fn(_ptr(Y, torch.float64, "Y"), P.struct, float(theta), float(exaggeration),
            _ptr(grad, torch.float64, "grad"), C.byref(z) if return_z else None,
            _ptr(ws, None, "workspace"), ws.numel(), _stream())
    _check(rc, fn.__name__)
    return grad, (z.value if return_z else None)


def step_f64(Y: torch.Tensor, P: "CsrF64", theta: float, exaggeration: float, learning_rate: float,
             momentum: float, min_gain: float, update: torch.Tensor, gains: torch.Tensor,
             grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
             return_z: bool = False):
    """bhtsne_step_f64: one fp64 iteration in place on Y, update and gains."""
    lib = load_library()
    if not isinstance(P, (CsrF64, LayoutF64)):
        raise TypeError("step_f64 takes P as a CsrF64 or a LayoutF64")
    ws = workspace if workspace is not None else torch.empty(workspace_size_f64(P.n, P.nnz), dtype=torch.uint8,
                                                             device=Y.device)
    z = C.c_double(0.0)
    fn = lib.bhtsne_step_layout_f64 if isinstance(P, LayoutF64) else lib.bhtsne_step_f64
    rc = fn(_ptr(Y, torch.float64, "Y"), P.struct, float(theta), float(exaggeration),
            float(learning_rate), float(momentum), float(min_gain),
            _ptr(update, torch.float64, "update"), _ptr(gains, torch.float64, "gains"),
            _ptr(grad, torch.float64, "grad"), C.byref(z) if return_z else None,
            _ptr(ws, None, "workspace"), ws.numel(), _stream())
    _check(rc, fn.__name__)
    return z.value if return_z else None


def workspace_size(n: int, nnz: int) -> int:
    return int(load_library().bhtsne_workspace_size(int(n), int(nnz)))


def _workspace(n, nnz, ws):
    need = workspace_size(n, nnz)
    if need == 0:
        raise BhtsneError(BHTSNE_EINVAL, "workspace_size")
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    return ws, need


class Layout:
    """A locality layout of P (relabelled copy in device memory) for the *_layout calls.
    order: None (bhtsne_layout_build, the automatic choice) or one of
    ORDER_MORTON, ORDER_BFS, ORDER_AUTO (bhtsne_layout_build_ordered)."""

    def __init__(self, P: Csr, Y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                 order: Optional[int] = None):
        lib = load_library()
        self.n, self.nnz = P.n, P.nnz
        need = int(lib.bhtsne_layout_size(P.n, P.nnz))
        if need == 0:
            raise BhtsneError(BHTSNE_EINVAL, "bhtsne_layout_size")
        self.mem = torch.empty(need, dtype=torch.uint8, device="cuda")
        ws, _ = _workspace(P.n, P.nnz, workspace)
        self._s = _Layout()
        if order is None:
            rc = lib.bhtsne_layout_build(P.struct, _ptr(Y, torch.float32, "Y"), _ptr(self.mem), need,
                                         C.byref(self._s), _ptr(ws), ws.numel(), _stream())
            _check(rc, "bhtsne_layout_build")
        else:
            rc = lib.bhtsne_layout_build_ordered(P.struct, _ptr(Y, torch.float32, "Y"), int(order), _ptr(self.mem),
                                                 need, C.byref(self._s), _ptr(ws), ws.numel(), _stream())
            _check(rc, "bhtsne_layout_build_ordered")

    @property
    def order(self) -> int:
        """ORDER_MORTON or ORDER_BFS: the point order the copy was built in."""
        return int(self._s.order)

    @property
    def tiles(self) -> int:
        return int(self._s.tiles)

    @property
    def items(self) -> int:
        return int(self._s.items)

    @property
    def entries(self) -> int:
        return int(self._s.entries)

    @property
    def windows(self) -> int:
        return int(self._s.windows)

    @property
    def segments(self) -> int:
        return int(self._s.segments)

    @property
    def struct(self):
        return C.byref(self._s)


class LayoutF64(Layout):
    """A locality layout of an fp64 P (CsrF64) for the fp64 variant's calls:
    relabelled rows with fp64 values, then the sliced copy over 8192-point
    windows or, without tile locality, windowed segments."""

    def __init__(self, P: "CsrF64", Y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
        lib = load_library()
        if not isinstance(P, CsrF64):
            raise TypeError("LayoutF64 takes P as a CsrF64")
        self.n, self.nnz = P.n, P.nnz
        need = int(lib.bhtsne_layout_size_f64(P.n, P.nnz))
        if need == 0:
            raise BhtsneError(BHTSNE_EINVAL, "bhtsne_layout_size_f64")
        self.mem = torch.empty(need, dtype=torch.uint8, device="cuda")
        ws = workspace if workspace is not None else torch.empty(workspace_size_f64(P.n, P.nnz), dtype=torch.uint8,
                                                                 device="cuda")
        self._s = _Layout()
        rc = lib.bhtsne_layout_build_f64(P.struct, _ptr(Y, torch.float64, "Y"), _ptr(self.mem), need,
                                         C.byref(self._s), _ptr(ws), ws.numel(), _stream())
        _check(rc, "bhtsne_layout_build_f64")


def layout_size(n: int, nnz: int) -> int:
    return int(load_library().bhtsne_layout_size(int(n), int(nnz)))


def gradient(Y: torch.Tensor, P, theta: float, exaggeration: float = 1.0,
             grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
             return_z: bool = True):
    """bhtsne_gradient (P a Csr) or bhtsne_gradient_layout (P a Layout): returns (grad, Z or None)."""
    lib = load_library()
    if grad is None:
        grad = torch.empty_like(Y)
    ws, _ = _workspace(P.n, P.nnz, workspace)
    z = C.c_double(0.0)
    fn = lib.bhtsne_gradient_layout if isinstance(P, Layout) else lib.bhtsne_gradient
    rc = fn(_ptr(Y, torch.float32, "Y"), P.struct, float(theta), float(exaggeration),
                             _ptr(grad, torch.float32, "grad"), C.byref(z) if return_z else None,
                             _ptr(ws, None, "workspace"), ws.numel(), _stream())
    _check(rc, fn.__name__)
    return grad, (z.value if return_z else None)


def z_exact(Y: torch.Tensor, workspace: Optional[torch.Tensor] = None) -> float:
    """bhtsne_z_exact: the exact normaliser over all ordered pairs i != j."""
    lib = load_library()
    n = Y.shape[0]
    ws, _ = _workspace(n, 0, workspace)
    z = C.c_double(0.0)
    _check(lib.bhtsne_z_exact(_ptr(Y, torch.float32, "Y"), n, C.byref(z), _ptr(ws, None, "workspace"),
                              ws.numel(), _stream()), "bhtsne_z_exact")
    return z.value


def kl(Y: torch.Tensor, P: "Csr", Z: float, workspace: Optional[torch.Tensor] = None) -> float:
    """bhtsne_kl: KL(P || Q) over P's stored entries for the given normaliser Z."""
    lib = load_library()
    if not isinstance(P, Csr):
        raise TypeError("kl takes P as a Csr")
    ws, _ = _workspace(P.n, 0, workspace)
    out = C.c_double(0.0)
    _check(lib.bhtsne_kl(_ptr(Y, torch.float32, "Y"), P.struct, float(Z), C.byref(out),
                         _ptr(ws, None, "workspace"), ws.numel(), _stream()), "bhtsne_kl")
    return out.value


def affinities_workspace_size(n: int, k: int) -> int:
    return int(load_library().bhtsne_affinities_workspace_size(int(n), int(k)))


def affinities(knn_idx: torch.Tensor, knn_dist: torch.Tensor, perplexity: float,
               workspace: Optional[torch.Tensor] = None, capacity: Optional[int] = None,
               sigma2: bool = False):
    """bhtsne_affinities: the symmetric P of k-nearest-neighbour lists
    (knn_idx int32 [n, k], knn_dist float32 [n, k]) at the given perplexity.
    Returns (Csr, sigma^2 fp64 [n] or None).  Output arrays hold `capacity`
    entries (default 2 n k, the most P can have) and are trimmed to nnz."""
    lib = load_library()
    n, k = int(knn_idx.shape[0]), int(knn_idx.shape[1])
    if tuple(knn_dist.shape) != (n, k):
        raise ValueError("knn_idx and knn_dist must have the same shape")
    need = affinities_workspace_size(n, k)
    if need == 0:
        raise BhtsneError(BHTSNE_EINVAL, "bhtsne_affinities_workspace_size")
    ws = workspace if workspace is not None else torch.empty(need, dtype=torch.uint8, device=knn_idx.device)
    cap = 2 * n * k if capacity is None else int(capacity)
    dev = knn_idx.device
    row_ptr = torch.empty(n + 1, dtype=torch.int64, device=dev)
    col = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    val = torch.empty(max(cap, 1), dtype=torch.float32, device=dev)
    s2 = torch.empty(n, dtype=torch.float64, device=dev) if sigma2 else None
    nnz = C.c_int64(0)
    rc = lib.bhtsne_affinities(_ptr(knn_idx, torch.int32, "knn_idx"), _ptr(knn_dist, torch.float32, "knn_dist"),
                               n, k, float(perplexity), _ptr(row_ptr, torch.int64, "row_ptr"),
                               _ptr(col, torch.int32, "col"), _ptr(val, torch.float32, "val"), cap,
                               C.byref(nnz), _ptr(s2, torch.float64, "sigma2"), _ptr(ws, None, "workspace"),
                               ws.numel(), _stream())
    if rc == BHTSNE_ECAPACITY:
        raise BhtsneError(rc, f"bhtsne_affinities (needs {nnz.value} entries)")
    _check(rc, "bhtsne_affinities")
    m = nnz.value
    return Csr(row_ptr, col[:m], val[:m]), s2


def step(Y: torch.Tensor, P, theta: float, exaggeration: float, learning_rate: float,
         momentum: float, min_gain: float, update: torch.Tensor, gains: torch.Tensor,
         grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
         return_z: bool = False):
    """bhtsne_step (P a Csr) or bhtsne_step_layout (P a Layout): Y, update and gains are
    updated in place; returns Z or None."""
    lib = load_library()
    ws, _ = _workspace(P.n, P.nnz, workspace)
    z = C.c_double(0.0)
    fn = lib.bhtsne_step_layout if isinstance(P, Layout) else lib.bhtsne_step
    rc = fn(_ptr(Y, torch.float32, "Y"), P.struct, float(theta), float(exaggeration),
                         float(learning_rate), float(momentum), float(min_gain),
                         _ptr(update, torch.float32, "update"), _ptr(gains, torch.float32, "gains"),
                         _ptr(grad, torch.float32, "grad"), C.byref(z) if return_z else None,
                         _ptr(ws, None, "workspace"), ws.numel(), _stream())
    _check(rc, fn.__name__)
    return z.value if return_z else None


def noalloc_max_bytes() -> int:
    return int(load_library().bhtsne_noalloc_max_bytes())


def step_noalloc(Y: torch.Tensor, P: "Csr", theta: float, exaggeration: float, learning_rate: float,
                 momentum: float, min_gain: float, update: torch.Tensor, gains: torch.Tensor,
                 grad: Optional[torch.Tensor] = None, return_z: bool = False):
    """bhtsne_step_noalloc: bhtsne_step on the library's fixed scratch array
    (no workspace, nothing allocated); Y, update and gains change in place."""
    lib = load_library()
    if not isinstance(P, Csr):
        raise TypeError("step_noalloc takes P as a Csr")
    z = C.c_double(0.0)
    rc = lib.bhtsne_step_noalloc(_ptr(Y, torch.float32, "Y"), P.struct, float(theta), float(exaggeration),
                                 float(learning_rate), float(momentum), float(min_gain),
                                 _ptr(update, torch.float32, "update"), _ptr(gains, torch.float32, "gains"),
                                 _ptr(grad, torch.float32, "grad"), C.byref(z) if return_z else None, _stream())
    _check(rc, "bhtsne_step_noalloc")
    return z.value if return_z else None


def get_stats(workspace: torch.Tensor, check: bool = True) -> dict:
    lib = load_library()
    s = _Stats()
    rc = lib.bhtsne_get_stats(_ptr(workspace, None, "workspace"), C.byref(s), _stream())
    if check:
        _check(rc, "bhtsne_get_stats")
    return {"Z": s.Z, "interactions": s.interactions, "nodes": s.nodes, "bbox": list(s.bbox),
            "r_span": s.r_span, "device_flags": s.device_flags, "max_depth": s.max_depth, "status": rc}


def timing_enable(on: bool = True):
    _check(load_library().bhtsne_timing_enable(1 if on else 0), "bhtsne_timing_enable")


def timing_phases(names=None):
    """Phases that record events while timing is on (None: all of them)."""
    mask = (1 << len(PHASES)) - 1 if names is None else sum(1 << PHASES.index(p) for p in set(names))
    _check(load_library().bhtsne_timing_phases(mask), "bhtsne_timing_phases")


def timing_read(reset: bool = True) -> dict:
    t = _Timing()
    _check(load_library().bhtsne_timing_read(C.byref(t), 1 if reset else 0), "bhtsne_timing_read")
    return {name: (t.ms[k], t.count[k]) for k, name in enumerate(PHASES)}


def debug_sort(Y: torch.Tensor, workspace: Optional[torch.Tensor] = None):
    """(codes, sorted_codes, perm, params[10]) as tensors / list."""
    lib = load_library()
    n = Y.shape[0]
    ws, _ = _workspace(n, 0, workspace)
    codes = torch.empty(n, dtype=torch.int64, device=Y.device)
    scodes = torch.empty(n, dtype=torch.int64, device=Y.device)
    perm = torch.empty(n, dtype=torch.int32, device=Y.device)
    params = (C.c_double * 10)()
    rc = lib.bhtsne_debug_sort(_ptr(Y, torch.float32, "Y"), n, _ptr(codes), _ptr(scodes), _ptr(perm),
                               params, _ptr(ws), ws.numel(), _stream())
    _check(rc, "bhtsne_debug_sort")
    return codes, scodes, perm, list(params)


def debug_tree(Y: torch.Tensor, theta: float = 0.5, workspace: Optional[torch.Tensor] = None) -> dict:
    """Tree arrays (pre-order) truncated to the node count, on the device."""
    lib = load_library()
    n = Y.shape[0]
    ws, _ = _workspace(n, 0, workspace)
    dev = Y.device
    level = torch.empty(2 * n, dtype=torch.uint8, device=dev)
    kind = torch.empty(2 * n, dtype=torch.uint8, device=dev)
    begin = torch.empty(2 * n, dtype=torch.int32, device=dev)
    end = torch.empty(2 * n, dtype=torch.int32, device=dev)
    summ = torch.empty((2 * n, 4), dtype=torch.float32, device=dev)
    meta = torch.empty(2 * n, dtype=torch.int32, device=dev)
    nn = C.c_int64(0)
    rc = lib.bhtsne_debug_tree(_ptr(Y, torch.float32, "Y"), n, float(theta), C.byref(nn), _ptr(level),
                               _ptr(kind), _ptr(begin), _ptr(end), _ptr(summ), _ptr(meta), _ptr(ws),
                               ws.numel(), _stream())
    _check(rc, "bhtsne_debug_tree")
    k = nn.value
    return {"nodes": k, "level": level[:k], "kind": kind[:k], "begin": begin[:k], "end": end[:k],
            "summary": summ[:k], "meta": meta[:k]}


# ---------------------------------------------------------------- 3-D embeddings
def workspace_size_3d(n: int, nnz: int) -> int:
    return int(load_library().bhtsne_workspace_size_3d(int(n), int(nnz)))


def _workspace_3d(n, nnz, ws):
    need = workspace_size_3d(n, nnz)
    if need == 0:
        raise BhtsneError(BHTSNE_EINVAL, "workspace_size_3d")
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    return ws


def _check_3d(Y):
    if Y.dim() != 2 or Y.shape[1] != 3:
        raise ValueError("a 3-D embedding is an n x 3 tensor")


class Layout3(Layout):
    """A locality layout of P for 3-D embeddings (bhtsne_layout_build_3d): the
    relabelled rows and their sliced copy over 8192-point windows of 3-D
    points.  With tiles == 0 (no tile locality) the 3-D calls refuse it and
    the plain Csr serves."""

    def __init__(self, P: Csr, Y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
        lib = load_library()
        if Y is not None:
            _check_3d(Y)
        self.n, self.nnz = P.n, P.nnz
        need = int(lib.bhtsne_layout_size_3d(P.n, P.nnz))
        if need == 0:
            raise BhtsneError(BHTSNE_EINVAL, "bhtsne_layout_size_3d")
        self.mem = torch.empty(need, dtype=torch.uint8, device="cuda")
        ws = _workspace_3d(P.n, P.nnz, workspace)
        self._s = _Layout()
        rc = lib.bhtsne_layout_build_3d(P.struct, _ptr(Y, torch.float32, "Y"), _ptr(self.mem), need,
                                        C.byref(self._s), _ptr(ws), ws.numel(), _stream())
        _check(rc, "bhtsne_layout_build_3d")


def layout_size_3d(n: int, nnz: int) -> int:
    return int(load_library().bhtsne_layout_size_3d(int(n), int(nnz)))


def gradient_3d(Y: torch.Tensor, P: "Csr", theta: float, exaggeration: float = 1.0,
                grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                return_z: bool = True):
    """bhtsne_gradient_3d (P a Csr) or bhtsne_gradient_layout_3d (P a Layout3):
    returns (grad n x 3, Z or None)."""
    lib = load_library()
    _check_3d(Y)
    if isinstance(P, Layout) and not isinstance(P, Layout3):
        raise TypeError("gradient_3d takes P as a Csr or a Layout3")
    if grad is None:
        grad = torch.empty_like(Y)
    ws = _workspace_3d(P.n, P.nnz, workspace)
    z = C.c_double(0.0)
    fn = lib.bhtsne_gradient_layout_3d if isinstance(P, Layout3) else lib.bhtsne_gradient_3d
    rc = fn(_ptr(Y, torch.float32, "Y"), P.struct, float(theta), float(exaggeration),
            _ptr(grad, torch.float32, "grad"), C.byref(z) if return_z else None,
            _ptr(ws, None, "workspace"), ws.numel(), _stream())
    _check(rc, fn.__name__)
    return grad, (z.value if return_z else None)


def step_3d(Y: torch.Tensor, P: "Csr", theta: float, exaggeration: float, learning_rate: float,
            momentum: float, min_gain: float, update: torch.Tensor, gains: torch.Tensor,
            grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
            return_z: bool = False):
    """bhtsne_step_3d (P a Csr) or bhtsne_step_layout_3d (P a Layout3): one
    iteration in place on Y, update and gains (n x 3)."""
    lib = load_library()
    _check_3d(Y)
    if isinstance(P, Layout) and not isinstance(P, Layout3):
        raise TypeError("step_3d takes P as a Csr or a Layout3")
    ws = _workspace_3d(P.n, P.nnz, workspace)
    z = C.c_double(0.0)
    fn = lib.bhtsne_step_layout_3d if isinstance(P, Layout3) else lib.bhtsne_step_3d
    rc = fn(_ptr(Y, torch.float32, "Y"), P.struct, float(theta), float(exaggeration),
            float(learning_rate), float(momentum), float(min_gain),
            _ptr(update, torch.float32, "update"), _ptr(gains, torch.float32, "gains"),
            _ptr(grad, torch.float32, "grad"), C.byref(z) if return_z else None,
            _ptr(ws, None, "workspace"), ws.numel(), _stream())
    _check(rc, fn.__name__)
    return z.value if return_z else None


def debug_sort_3d(Y: torch.Tensor, workspace: Optional[torch.Tensor] = None):
    """(codes, sorted_codes, perm, params[14]) of a 3-D embedding."""
    lib = load_library()
    _check_3d(Y)
    n = Y.shape[0]
    ws = _workspace_3d(n, 0, workspace)
    codes = torch.empty(n, dtype=torch.int64, device=Y.device)
    scodes = torch.empty(n, dtype=torch.int64, device=Y.device)
    perm = torch.empty(n, dtype=torch.int32, device=Y.device)
    params = (C.c_double * 14)()
    rc = lib.bhtsne_debug_sort_3d(_ptr(Y, torch.float32, "Y"), n, _ptr(codes), _ptr(scodes), _ptr(perm),
                                  params, _ptr(ws), ws.numel(), _stream())
    _check(rc, "bhtsne_debug_sort_3d")
    return codes, scodes, perm, list(params)


def debug_tree_3d(Y: torch.Tensor, theta: float = 0.5, workspace: Optional[torch.Tensor] = None) -> dict:
    """Octree arrays (pre-order) truncated to the node count, on the device."""
    lib = load_library()
    _check_3d(Y)
    n = Y.shape[0]
    ws = _workspace_3d(n, 0, workspace)
    dev = Y.device
    level = torch.empty(2 * n, dtype=torch.uint8, device=dev)
    kind = torch.empty(2 * n, dtype=torch.uint8, device=dev)
    begin = torch.empty(2 * n, dtype=torch.int32, device=dev)
    end = torch.empty(2 * n, dtype=torch.int32, device=dev)
    summ = torch.empty((2 * n, 4), dtype=torch.float32, device=dev)
    thr = torch.empty(2 * n, dtype=torch.float32, device=dev)
    meta = torch.empty(2 * n, dtype=torch.int32, device=dev)
    nn = C.c_int64(0)
    rc = lib.bhtsne_debug_tree_3d(_ptr(Y, torch.float32, "Y"), n, float(theta), C.byref(nn), _ptr(level),
                                  _ptr(kind), _ptr(begin), _ptr(end), _ptr(summ), _ptr(thr), _ptr(meta),
                                  _ptr(ws), ws.numel(), _stream())
    _check(rc, "bhtsne_debug_tree_3d")
    k = nn.value
    return {"nodes": k, "level": level[:k], "kind": kind[:k], "begin": begin[:k], "end": end[:k],
            "summary": summ[:k], "threshold": thr[:k], "meta": meta[:k]}
