"""Python face of the fp64 CPU oracle (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this package.  The GPU library never touches it.  The functions take
numpy arrays, promote float32 embeddings to float64 exactly and call the C
implementation in ``bhtsne_oracle.c`` (built by ``oracle/build.py``).
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

INTERNAL, BUCKET, SINGLE = 0, 1, 2

_d = C.POINTER(C.c_double)
_u64 = C.POINTER(C.c_uint64)
_u32 = C.POINTER(C.c_uint32)
_i64 = C.POINTER(C.c_int64)
_i32 = C.POINTER(C.c_int32)
_u8 = C.POINTER(C.c_uint8)
_f = C.POINTER(C.c_float)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = C.CDLL(_LIB_PATH)
    sig = {
        "orc_bbox": (None, [_d, C.c_int64, _d]),
        "orc_interleave": (C.c_uint64, [C.c_uint32, C.c_uint32]),
        "orc_morton": (None, [_d, C.c_int64, _u64, _u32, _d]),
        "orc_sort": (None, [_u64, C.c_int64, _u64, _u32]),
        "orc_tree": (C.c_int64, [_u64, C.c_int64, _u8, _u8, _u32, _u32, _i32]),
        "orc_state_build": (C.c_void_p, [_d, C.c_int64]),
        "orc_state_free": (None, [C.c_void_p]),
        "orc_state_nodes": (C.c_int64, [C.c_void_p]),
        "orc_state_export": (None, [C.c_void_p, _d, _d, _u64, _u64, _u32, _u8, _u8, _u32, _u32,
                                    _i32, _d, _u32]),
        "orc_state_repulsive": (None, [C.c_void_p, C.c_double, _i64, C.c_int64, _d, _d, _i64]),
        "orc_attractive": (None, [_d, _i64, _i32, _f, _i64, C.c_int64, _d]),
        "orc_sum": (C.c_double, [_d, C.c_int64]),
        "orc_gradient": (None, [_d, C.c_int64, _i64, _i32, _f, C.c_double, C.c_double, _d, _d]),
        "orc_update": (None, [_d, _d, _d, _d, C.c_int64, C.c_double, C.c_double, C.c_double]),
        "orc_step": (None, [_d, C.c_int64, _i64, _i32, _f, C.c_double, C.c_double, C.c_double,
                            C.c_double, C.c_double, _d, _d, _d, _d]),
        "orc_z_exact": (C.c_double, [_d, C.c_int64]),
        "orc_kl": (C.c_double, [_d, C.c_int64, _i64, _i32, _f, C.c_double]),
        "orc_threads": (C.c_int, []),
        "orc_set_threads": (None, [C.c_int]),
        "orc_step_timed": (None, [_d, C.c_int64, _i64, _i32, _f, C.c_double, C.c_double, C.c_double,
                                  C.c_double, C.c_double, _d, _d, _d, _d]),
        # three-dimensional embeddings
        "orc3_bbox": (None, [_d, C.c_int64, _d]),
        "orc3_interleave": (C.c_uint64, [C.c_uint32, C.c_uint32, C.c_uint32]),
        "orc3_morton": (None, [_d, C.c_int64, _u64, _u32, _d]),
        "orc3_tree": (C.c_int64, [_u64, C.c_int64, _u8, _u8, _u32, _u32, _i32]),
        "orc3_state_build": (C.c_void_p, [_d, C.c_int64]),
        "orc3_state_free": (None, [C.c_void_p]),
        "orc3_state_nodes": (C.c_int64, [C.c_void_p]),
        "orc3_state_export": (None, [C.c_void_p, _d, _d, _u64, _u64, _u32, _u8, _u8, _u32, _u32,
                                     _i32, _d, _u32]),
        "orc3_state_repulsive": (None, [C.c_void_p, C.c_double, _i64, C.c_int64, _d, _d, _i64]),
        "orc3_attractive": (None, [_d, _i64, _i32, _f, _i64, C.c_int64, _d]),
        "orc3_gradient": (None, [_d, C.c_int64, _i64, _i32, _f, C.c_double, C.c_double, _d, _d]),
        "orc3_step": (None, [_d, C.c_int64, _i64, _i32, _f, C.c_double, C.c_double, C.c_double,
                             C.c_double, C.c_double, _d, _d, _d, _d]),
        "orc3_z_exact": (C.c_double, [_d, C.c_int64]),
        "orc3_kl": (C.c_double, [_d, C.c_int64, _i64, _i32, _f, C.c_double]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _p(a, t):
    return a.ctypes.data_as(t) if a is not None else None


def _y64(Y) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(Y), dtype=np.float64).reshape(-1, 2)


def _csr(row_ptr, col, val):
    return (np.ascontiguousarray(row_ptr, dtype=np.int64), np.ascontiguousarray(col, dtype=np.int32),
            np.ascontiguousarray(val, dtype=np.float32))


def threads() -> int:
    return int(_load().orc_threads())


def bbox(Y) -> np.ndarray:
    """[min_x, max_x, min_y, max_y, cent_x, cent_y, r_span]."""
    y = _y64(Y)
    out = np.empty(7)
    _load().orc_bbox(_p(y, _d), y.shape[0], _p(out, _d))
    return out


def interleave(m0: int, m1: int) -> int:
    return int(_load().orc_interleave(m0, m1))


def morton(Y):
    """(codes u64[n], grid u32[n,2], [y_root_x, y_root_y, scale])."""
    y = _y64(Y)
    n = y.shape[0]
    codes = np.empty(n, np.uint64)
    grid = np.empty((n, 2), np.uint32)
    yrs = np.empty(3)
    _load().orc_morton(_p(y, _d), n, _p(codes, _u64), _p(grid, _u32), _p(yrs, _d))
    return codes, grid, yrs


def sort_codes(codes):
    codes = np.ascontiguousarray(codes, dtype=np.uint64)
    n = codes.size
    s = np.empty(n, np.uint64)
    perm = np.empty(n, np.uint32)
    _load().orc_sort(_p(codes, _u64), n, _p(s, _u64), _p(perm, _u32))
    return s, perm


@dataclass
class Tree:
    """Canonical compressed quadtree, nodes in (begin, level) order."""
    box: np.ndarray
    yrs: np.ndarray
    codes: np.ndarray
    sorted_codes: np.ndarray
    perm: np.ndarray
    level: np.ndarray
    kind: np.ndarray
    begin: np.ndarray
    end: np.ndarray
    parent: np.ndarray
    com: np.ndarray
    count: np.ndarray

    @property
    def nodes(self) -> int:
        return int(self.level.size)


class State:
    """Oracle tree state of one embedding; frees its C memory on close()."""

    def __init__(self, Y):
        self._y = _y64(Y)
        self.n = self._y.shape[0]
        if self.n < 2:
            raise ValueError("need at least two points")
        self._h = _load().orc_state_build(_p(self._y, _d), self.n)

    def close(self):
        if self._h:
            _load().orc_state_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def tree(self) -> Tree:
        lib = _load()
        nn = int(lib.orc_state_nodes(self._h))
        n = self.n
        t = Tree(np.empty(7), np.empty(3), np.empty(n, np.uint64), np.empty(n, np.uint64),
                 np.empty(n, np.uint32), np.empty(nn, np.uint8), np.empty(nn, np.uint8),
                 np.empty(nn, np.uint32), np.empty(nn, np.uint32), np.empty(nn, np.int32),
                 np.empty((nn, 2)), np.empty(nn, np.uint32))
        lib.orc_state_export(self._h, _p(t.box, _d), _p(t.yrs, _d), _p(t.codes, _u64),
                             _p(t.sorted_codes, _u64), _p(t.perm, _u32), _p(t.level, _u8),
                             _p(t.kind, _u8), _p(t.begin, _u32), _p(t.end, _u32),
                             _p(t.parent, _i32), _p(t.com, _d), _p(t.count, _u32))
        return t

    def repulsive(self, theta: float, points=None):
        """(F_rep [k,2] positive-sign sums, Z_i [k], interactions [k]) for the given
        original indices (all points when None)."""
        pts = None if points is None else np.ascontiguousarray(points, dtype=np.int64)
        k = self.n if pts is None else pts.size
        frep = np.empty((k, 2))
        zi = np.empty(k)
        inter = np.empty(k, np.int64)
        _load().orc_state_repulsive(self._h, float(theta), _p(pts, _i64), k, _p(frep, _d),
                                    _p(zi, _d), _p(inter, _i64))
        return frep, zi, inter


def tree(Y) -> Tree:
    with State(Y) as s:
        return s.tree()


def attractive(Y, row_ptr, col, val, rows=None) -> np.ndarray:
    y = _y64(Y)
    rp, c, v = _csr(row_ptr, col, val)
    r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    k = y.shape[0] if r is None else r.size
    out = np.empty((k, 2))
    _load().orc_attractive(_p(y, _d), _p(rp, _i64), _p(c, _i32), _p(v, _f), _p(r, _i64), k,
                           _p(out, _d))
    return out


def ordered_sum(x) -> float:
    x = np.ascontiguousarray(x, dtype=np.float64)
    return float(_load().orc_sum(_p(x, _d), x.size))


def gradient(Y, row_ptr, col, val, theta: float, exaggeration: float = 1.0):
    """(grad [n,2], Z, interactions, nodes) of one BH gradient."""
    y = _y64(Y)
    rp, c, v = _csr(row_ptr, col, val)
    g = np.empty_like(y)
    st = np.empty(3)
    _load().orc_gradient(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f),
                         float(theta), float(exaggeration), _p(g, _d), _p(st, _d))
    return g, float(st[0]), int(st[1]), int(st[2])


def update(y, u, gains, g, eta, mu, min_gain=0.01):
    """In-place gains/momentum update on float64 arrays."""
    for a in (y, u, gains, g):
        assert a.dtype == np.float64 and a.flags.c_contiguous
    _load().orc_update(_p(y, _d), _p(u, _d), _p(gains, _d), _p(g, _d), y.size, float(eta),
                       float(mu), float(min_gain))


def step(y, u, gains, row_ptr, col, val, theta, exaggeration, learning_rate, momentum,
         min_gain=0.01):
    """One full iteration on fp64 state arrays (modified in place); returns
    (grad, Z, interactions, nodes)."""
    for a in (y, u, gains):
        assert a.dtype == np.float64 and a.flags.c_contiguous
    rp, c, v = _csr(row_ptr, col, val)
    g = np.empty_like(y)
    st = np.empty(3)
    _load().orc_step(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f), float(theta),
                     float(exaggeration), float(learning_rate), float(momentum), float(min_gain),
                     _p(u, _d), _p(gains, _d), _p(g, _d), _p(st, _d))
    return g, float(st[0]), int(st[1]), int(st[2])


STEP_PHASES = ("tree", "summarization", "attractive", "repulsive", "update")


def set_threads(t: int):
    """Threads of the oracle's OpenMP loops (results do not depend on it)."""
    _load().orc_set_threads(int(t))


def step_timed(y, u, gains, row_ptr, col, val, theta, exaggeration, learning_rate, momentum,
               min_gain=0.01):
    """oracle.step with the wall time of each of the paper's steps: returns
    (Z, interactions, nodes, {phase: ms})."""
    for a in (y, u, gains):
        assert a.dtype == np.float64 and a.flags.c_contiguous
    rp, c, v = _csr(row_ptr, col, val)
    st = np.empty(3)
    ms = np.empty(5)
    _load().orc_step_timed(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f), float(theta),
                           float(exaggeration), float(learning_rate), float(momentum), float(min_gain),
                           _p(u, _d), _p(gains, _d), _p(st, _d), _p(ms, _d))
    return float(st[0]), int(st[1]), int(st[2]), dict(zip(STEP_PHASES, ms.tolist()))


def z_exact(Y) -> float:
    y = _y64(Y)
    return float(_load().orc_z_exact(_p(y, _d), y.shape[0]))


def kl(Y, row_ptr, col, val, Z=None) -> float:
    """KL(P||Q) over the stored entries of P; Z defaults to the exact O(n^2) sum."""
    y = _y64(Y)
    rp, c, v = _csr(row_ptr, col, val)
    if Z is None:
        Z = z_exact(y)
    return float(_load().orc_kl(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f),
                                float(Z)))


# ---------------------------------------------------------------- 3-D embeddings
def _y3(Y) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(Y), dtype=np.float64).reshape(-1, 3)


def bbox3(Y) -> np.ndarray:
    """[min_x, max_x, min_y, max_y, min_z, max_z, cent_x, cent_y, cent_z, r_span]."""
    y = _y3(Y)
    out = np.empty(10)
    _load().orc3_bbox(_p(y, _d), y.shape[0], _p(out, _d))
    return out


def interleave3(m0: int, m1: int, m2: int) -> int:
    return int(_load().orc3_interleave(m0, m1, m2))


def morton3(Y):
    """(codes u64[n], grid u32[n,3], [y_root_x, y_root_y, y_root_z, scale])."""
    y = _y3(Y)
    n = y.shape[0]
    codes = np.empty(n, np.uint64)
    grid = np.empty((n, 3), np.uint32)
    yrs = np.empty(4)
    _load().orc3_morton(_p(y, _d), n, _p(codes, _u64), _p(grid, _u32), _p(yrs, _d))
    return codes, grid, yrs


class State3:
    """Oracle octree state of one 3-D embedding; frees its C memory on close()."""

    def __init__(self, Y):
        self._y = _y3(Y)
        self.n = self._y.shape[0]
        if self.n < 2:
            raise ValueError("need at least two points")
        self._h = _load().orc3_state_build(_p(self._y, _d), self.n)

    def close(self):
        if self._h:
            _load().orc3_state_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def tree(self) -> Tree:
        """The canonical compressed octree (box has 10 entries, yrs 4, com 3 columns)."""
        lib = _load()
        nn = int(lib.orc3_state_nodes(self._h))
        n = self.n
        t = Tree(np.empty(10), np.empty(4), np.empty(n, np.uint64), np.empty(n, np.uint64),
                 np.empty(n, np.uint32), np.empty(nn, np.uint8), np.empty(nn, np.uint8),
                 np.empty(nn, np.uint32), np.empty(nn, np.uint32), np.empty(nn, np.int32),
                 np.empty((nn, 3)), np.empty(nn, np.uint32))
        lib.orc3_state_export(self._h, _p(t.box, _d), _p(t.yrs, _d), _p(t.codes, _u64),
                              _p(t.sorted_codes, _u64), _p(t.perm, _u32), _p(t.level, _u8),
                              _p(t.kind, _u8), _p(t.begin, _u32), _p(t.end, _u32),
                              _p(t.parent, _i32), _p(t.com, _d), _p(t.count, _u32))
        return t

    def repulsive(self, theta: float, points=None):
        """(F_rep [k,3], Z_i [k], interactions [k]) for the given original indices."""
        pts = None if points is None else np.ascontiguousarray(points, dtype=np.int64)
        k = self.n if pts is None else pts.size
        frep = np.empty((k, 3))
        zi = np.empty(k)
        inter = np.empty(k, np.int64)
        _load().orc3_state_repulsive(self._h, float(theta), _p(pts, _i64), k, _p(frep, _d),
                                     _p(zi, _d), _p(inter, _i64))
        return frep, zi, inter


def tree3(Y) -> Tree:
    with State3(Y) as s:
        return s.tree()


def attractive3(Y, row_ptr, col, val, rows=None) -> np.ndarray:
    y = _y3(Y)
    rp, c, v = _csr(row_ptr, col, val)
    r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    k = y.shape[0] if r is None else r.size
    out = np.empty((k, 3))
    _load().orc3_attractive(_p(y, _d), _p(rp, _i64), _p(c, _i32), _p(v, _f), _p(r, _i64), k,
                            _p(out, _d))
    return out


def gradient3(Y, row_ptr, col, val, theta: float, exaggeration: float = 1.0):
    """(grad [n,3], Z, interactions, nodes) of one BH gradient of a 3-D embedding."""
    y = _y3(Y)
    rp, c, v = _csr(row_ptr, col, val)
    g = np.empty_like(y)
    st = np.empty(3)
    _load().orc3_gradient(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f),
                          float(theta), float(exaggeration), _p(g, _d), _p(st, _d))
    return g, float(st[0]), int(st[1]), int(st[2])


def step3(y, u, gains, row_ptr, col, val, theta, exaggeration, learning_rate, momentum,
          min_gain=0.01):
    """One 3-D iteration on fp64 state arrays (n x 3, modified in place)."""
    for a in (y, u, gains):
        assert a.dtype == np.float64 and a.flags.c_contiguous and a.shape[-1] == 3
    rp, c, v = _csr(row_ptr, col, val)
    g = np.empty_like(y)
    st = np.empty(3)
    _load().orc3_step(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f), float(theta),
                      float(exaggeration), float(learning_rate), float(momentum), float(min_gain),
                      _p(u, _d), _p(gains, _d), _p(g, _d), _p(st, _d))
    return g, float(st[0]), int(st[1]), int(st[2])


def z_exact3(Y) -> float:
    y = _y3(Y)
    return float(_load().orc3_z_exact(_p(y, _d), y.shape[0]))


def kl3(Y, row_ptr, col, val, Z=None) -> float:
    y = _y3(Y)
    rp, c, v = _csr(row_ptr, col, val)
    if Z is None:
        Z = z_exact3(y)
    return float(_load().orc3_kl(_p(y, _d), y.shape[0], _p(rp, _i64), _p(c, _i32), _p(v, _f),
                                 float(Z)))
