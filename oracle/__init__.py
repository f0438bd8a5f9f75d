"""CAGQ CPU oracle -- test infrastructure only.

ctypes wrapper over ``libcagq_oracle.so`` (plain single-threaded C99 built
from ``cagq_oracle.c`` with gcc). Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the HIP library never
does. Arrays are numpy, host memory, row-major.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# CAGQ_ORACLE_LIB selects another build of the same source (the sanitizer
# run in sanitize.sh); the default is the in-tree build
LIB_PATH = os.environ.get("CAGQ_ORACLE_LIB") or os.path.join(_HERE, "libcagq_oracle.so")
SRC_PATH = os.path.join(_HERE, "cagq_oracle.c")

CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/libcagq_oracle.so``."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        subprocess.run(["gcc", *CFLAGS, SRC_PATH, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


class Grid(C.Structure):
    _fields_ = [("origin", C.c_float * 3), ("voxel_size", C.c_float * 3),
                ("dims", C.c_int32 * 3), ("n_v", C.c_int32), ("radius", C.c_int32)]


class _Table(C.Structure):
    _fields_ = [("B", C.c_int32), ("N", C.c_int32), ("g", Grid),
                ("nvox", C.c_void_p), ("vox_lin", C.c_void_p), ("vox_count", C.c_void_p),
                ("vox_off", C.c_void_p), ("pt_list", C.c_void_p)]


_lib = None

QUERY_MODES = {"cube": 0, "knn": 1, "knn_ring": 2}


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=False)
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        L.orc_splitmix64.restype = C.c_uint64
        L.orc_splitmix64.argtypes = [C.c_uint64]
        L.orc_voxelize.argtypes = [P, C.c_int64, C.POINTER(Grid), P]
        L.orc_build_table.argtypes = [P, C.c_int32, C.c_int32, C.POINTER(Grid), P, P, P, P, P]
        L.orc_sample_rvs.argtypes = [C.POINTER(_Table), C.c_int32, C.c_uint64, P, P]
        L.orc_sample_cas.argtypes = [C.POINTER(_Table), C.c_int32, C.c_uint32, P, P, P, P]
        L.orc_sample_cas_swap.argtypes = [C.POINTER(_Table), C.c_int32, C.c_uint64, C.c_uint32, P, P, P, P]
        L.orc_query.argtypes = [C.POINTER(_Table), P, P, P, P, C.c_int32, C.c_int32,
                                C.c_int32, C.c_uint64, P, P, P, P, P, P]
        L.orc_query_points.argtypes = [C.POINTER(_Table), P, P, C.c_int32, C.c_int32, C.c_int32, C.c_uint64,
                                       P, P, P, P, P]
        L.orc_context_list.argtypes = [C.POINTER(_Table), P, C.c_int32, P, P, C.c_int64]
        L.orc_sample_points.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_uint64, P]
        L.orc_ball_query.argtypes = [P, C.c_int32, C.c_int32, P, C.c_int32, C.c_int32, C.c_float, P, P]
        L.orc_coverage.argtypes = [C.POINTER(_Table), P, P, P, C.c_int32, C.c_int32, P]
        for f in ("orc_voxelize", "orc_build_table", "orc_sample_rvs", "orc_sample_cas", "orc_sample_cas_swap",
                  "orc_query", "orc_query_points", "orc_context_list", "orc_sample_points", "orc_ball_query",
                  "orc_coverage"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} returned {rc}")


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def make_grid(origin, voxel_size, dims, n_v, radius) -> Grid:
    g = Grid()
    for a in range(3):
        g.origin[a] = float(origin[a])
        g.voxel_size[a] = float(voxel_size[a])
        g.dims[a] = int(dims[a])
    g.n_v = int(n_v)
    g.radius = int(radius)
    return g


def grid_from_spec(spec) -> Grid:
    return make_grid(spec.origin, spec.voxel_size, spec.dims, spec.n_v, spec.radius)


def splitmix64(x: int) -> int:
    return int(lib().orc_splitmix64(C.c_uint64(x & 0xFFFFFFFFFFFFFFFF)))


def voxelize(points: np.ndarray, grid: Grid) -> np.ndarray:
    P = np.ascontiguousarray(points, dtype=np.float32).reshape(-1, 3)
    lin = np.empty(P.shape[0], dtype=np.uint32)
    _check(lib().orc_voxelize(_ptr(P), P.shape[0], C.byref(grid), _ptr(lin)), "orc_voxelize")
    return lin.reshape(points.shape[:-1])


class Table:
    """Occupied-voxel table of a batch [B, N, 3] (Appendix D, step 1)."""

    def __init__(self, points: np.ndarray, grid: Grid):
        P = np.ascontiguousarray(points, dtype=np.float32)
        assert P.ndim == 3 and P.shape[2] == 3
        B, N = P.shape[:2]
        self.B, self.N, self.grid, self.points = B, N, grid, P
        self.nvox = np.zeros(B, np.int32)
        self.vox_lin = np.zeros((B, N), np.uint32)
        self.vox_count = np.zeros((B, N), np.uint32)
        self.vox_off = np.zeros((B, N + 1), np.uint32)
        self.pt_list = np.zeros((B, N), np.uint32)
        _check(lib().orc_build_table(_ptr(P), B, N, C.byref(grid), _ptr(self.nvox),
                                     _ptr(self.vox_lin), _ptr(self.vox_count),
                                     _ptr(self.vox_off), _ptr(self.pt_list)), "orc_build_table")
        self._t = _Table(B, N, grid, _ptr(self.nvox), _ptr(self.vox_lin), _ptr(self.vox_count),
                         _ptr(self.vox_off), _ptr(self.pt_list))

    def sample_rvs(self, M: int, seed: int):
        cl = np.zeros((self.B, M), np.int32)
        mv = np.zeros(self.B, np.int32)
        _check(lib().orc_sample_rvs(C.byref(self._t), M, C.c_uint64(seed), _ptr(cl), _ptr(mv)),
               "orc_sample_rvs")
        return cl, mv

    def sample_cas(self, M: int, beta_q16: int = 0):
        """Returns (center_lin ascending, m_valid, pick_lin in pick order, pick_score)."""
        cl = np.zeros((self.B, M), np.int32)
        mv = np.zeros(self.B, np.int32)
        pl = np.zeros((self.B, M), np.int32)
        ps = np.zeros((self.B, M), np.int64)
        _check(lib().orc_sample_cas(C.byref(self._t), M, C.c_uint32(beta_q16), _ptr(cl), _ptr(mv),
                                    _ptr(pl), _ptr(ps)), "orc_sample_cas")
        return cl, mv, pl, ps

    def sample_cas_swap(self, M: int, seed: int, beta_q16: int = 0):
        """The paper's challenger / incumbent CAS from the RVS choice.
        Returns (center_lin ascending, m_valid, decision [B][N], n_swaps [B]);
        decision[b, t] is the slot challenge t went to, >= 0 when accepted,
        -(slot + 1) when refused; entries past the last challenge are 0."""
        cl = np.zeros((self.B, M), np.int32)
        mv = np.zeros(self.B, np.int32)
        dec = np.zeros((self.B, self.N), np.int32)
        ns = np.zeros(self.B, np.int32)
        _check(lib().orc_sample_cas_swap(C.byref(self._t), M, C.c_uint64(seed), C.c_uint32(beta_q16),
                                         _ptr(cl), _ptr(mv), _ptr(dec), _ptr(ns)), "orc_sample_cas_swap")
        return cl, mv, dec, ns

    def sample(self, M: int, mode: str, seed: int, beta_q16: int = 0):
        if mode == "rvs":
            return self.sample_rvs(M, seed)
        if mode == "cas_swap":
            cl, mv, _, _ = self.sample_cas_swap(M, seed, beta_q16)
            return cl, mv
        cl, mv, _, _ = self.sample_cas(M, beta_q16)
        return cl, mv

    def query(self, center_lin: np.ndarray, m_valid: np.ndarray, K: int, mode: str,
              seed: int, weights: Optional[np.ndarray] = None,
              points: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
        P = self.points if points is None else np.ascontiguousarray(points, np.float32)
        B, M = center_lin.shape
        cl = np.ascontiguousarray(center_lin, np.int32)
        mv = np.ascontiguousarray(m_valid, np.int32)
        W = None if weights is None else np.ascontiguousarray(weights, np.uint32)
        out = dict(
            node_idx=np.zeros((B, M, K), np.int32),
            node_xyz=np.zeros((B, M, K, 3), np.float32),
            n_valid=np.zeros((B, M), np.int32),
            center_xyz=np.zeros((B, M, 3), np.float32),
            center_w=np.zeros((B, M), np.uint32),
            ctx_count=np.zeros((B, M), np.int32),
        )
        m = QUERY_MODES[mode]
        _check(lib().orc_query(C.byref(self._t), _ptr(P), _ptr(W), _ptr(cl), _ptr(mv), M, K, m,
                               C.c_uint64(seed), _ptr(out["node_idx"]), _ptr(out["node_xyz"]),
                               _ptr(out["n_valid"]), _ptr(out["center_xyz"]), _ptr(out["center_w"]),
                               _ptr(out["ctx_count"])), "orc_query")
        return out

    def query_points(self, centers: np.ndarray, K: int, mode: str, seed: int,
                     points: Optional[np.ndarray] = None, allow_nonfinite: bool = False) -> Dict[str, np.ndarray]:
        """Upsampling query: K nodes around given center points [B][M][3]."""
        P = self.points if points is None else np.ascontiguousarray(points, np.float32)
        Q = np.ascontiguousarray(centers, np.float32)
        B, M = Q.shape[:2]
        out = dict(
            node_idx=np.zeros((B, M, K), np.int32),
            node_xyz=np.zeros((B, M, K, 3), np.float32),
            n_valid=np.zeros((B, M), np.int32),
            ctx_count=np.zeros((B, M), np.int32),
            center_lin=np.zeros((B, M), np.int32),
        )
        m = QUERY_MODES[mode]
        rc = lib().orc_query_points(C.byref(self._t), _ptr(P), _ptr(Q), M, K, m, C.c_uint64(seed),
                                    _ptr(out["node_idx"]), _ptr(out["node_xyz"]), _ptr(out["n_valid"]),
                                    _ptr(out["ctx_count"]), _ptr(out["center_lin"]))
        if not (allow_nonfinite and rc == -4):
            _check(rc, "orc_query_points")
        return out

    def context_list(self, center_lin: np.ndarray):
        """Context lists of center voxels [B][M]: (ctx_off [B*M+1] int64,
        ctx_idx [total] int32)."""
        cl = np.ascontiguousarray(center_lin, np.int32)
        B, M = cl.shape
        off = np.zeros(B * M + 1, np.int64)
        _check(lib().orc_context_list(C.byref(self._t), _ptr(cl), M, _ptr(off), None, 0), "orc_context_list")
        idx = np.zeros(max(int(off[-1]), 1), np.int32)
        _check(lib().orc_context_list(C.byref(self._t), _ptr(cl), M, _ptr(off), _ptr(idx), int(off[-1])),
               "orc_context_list")
        return off, idx[: int(off[-1])]

    def coverage(self, node_idx: np.ndarray, n_valid: np.ndarray, points: Optional[np.ndarray] = None) -> np.ndarray:
        """Occupied voxels [B] holding a valid node point (Sec. 4)."""
        P = self.points if points is None else np.ascontiguousarray(points, np.float32)
        ni = np.ascontiguousarray(node_idx, np.int32)
        nv = np.ascontiguousarray(n_valid, np.int32)
        B, M, K = ni.shape
        out = np.zeros(B, np.int32)
        _check(lib().orc_coverage(C.byref(self._t), _ptr(P), _ptr(ni), _ptr(nv), M, K, _ptr(out)), "orc_coverage")
        return out


SAMPLE_POINT_MODES = {"rps": 0, "fps": 1}


def sample_points(points: np.ndarray, M: int, mode: str, seed: int = 0) -> np.ndarray:
    """Random / Farthest Point Sampling: center point indices [B][M]."""
    P = np.ascontiguousarray(points, np.float32)
    B, N = P.shape[:2]
    out = np.zeros((B, M), np.int32)
    _check(lib().orc_sample_points(_ptr(P), B, N, M, SAMPLE_POINT_MODES[mode], C.c_uint64(seed), _ptr(out)),
           "orc_sample_points")
    return out


def ball_query(points: np.ndarray, center_idx: np.ndarray, K: int, radius2: float):
    """Ball Query: (node_idx [B][M][K], n_valid [B][M])."""
    P = np.ascontiguousarray(points, np.float32)
    ci = np.ascontiguousarray(center_idx, np.int32)
    B, N = P.shape[:2]
    M = ci.shape[1]
    ni = np.zeros((B, M, K), np.int32)
    nv = np.zeros((B, M), np.int32)
    _check(lib().orc_ball_query(_ptr(P), B, N, _ptr(ci), M, K, C.c_float(radius2), _ptr(ni), _ptr(nv)),
           "orc_ball_query")
    return ni, nv


def run_layer(points: np.ndarray, layer, weights: Optional[np.ndarray] = None):
    """One CAGQ layer: table, centers, query. Returns (table, centers, m_valid, query dict)."""
    t = Table(points, grid_from_spec(layer.grid))
    cl, mv = t.sample(layer.M, layer.sample, layer.seed)
    q = t.query(cl, mv, layer.K, layer.query, layer.seed, weights=weights)
    return t, cl, mv, q
