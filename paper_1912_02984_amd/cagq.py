"""Python binding of the gfx950 CAGQ library (``libcagq.so``).

Argument marshalling only: every step of the path runs in the library's HIP
kernels. Tensors are torch CUDA (HIP) tensors; the library enqueues on the
current torch stream. The names mirror the C ABI in ``include/cagq.h``:
``build_grid``, ``sample_centers``, ``query_context``, ``get_device_status``.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Dict, Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcagq.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_GRID_TOO_LARGE = -2
ERR_WORKSPACE_TOO_SMALL = -3
ERR_NONFINITE_INPUT = -4
ERR_CAPACITY = -5
ERR_HIP = -6
ERR_CENTER_NOT_OCCUPIED = -7

SAMPLE = {"rvs": 0, "cas": 1, "cas_swap": 2}
QUERY = {"cube": 0, "knn": 1, "knn_ring": 2}
MAX_K = 128
MAX_NV = 64
MAX_RADIUS = 3


class GridDesc(C.Structure):
    _fields_ = [("origin", C.c_float * 3), ("voxel_size", C.c_float * 3),
                ("dims", C.c_int32 * 3), ("n_v", C.c_int32), ("radius", C.c_int32)]


class LayoutC(C.Structure):
    _fields_ = [("total_bytes", C.c_size_t), ("nvox", C.c_size_t), ("vox_lin", C.c_size_t),
                ("vox_count", C.c_size_t), ("vox_off", C.c_size_t), ("pt_list", C.c_size_t)]


class GridC(C.Structure):
    _fields_ = [("B", C.c_int32), ("N", C.c_int32), ("desc", GridDesc), ("points", C.c_void_p),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t)]


class CagqError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {status_string(code)} ({code})")
        self.code = code


_lib = None


def lib() -> C.CDLL:
    """Load ``libcagq.so``; raises if the library has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_1912_02984_amd.build")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        F3, I3 = C.c_float * 3, C.c_int32 * 3
        L.cagq_desc_from_voxel_size.argtypes = [C.POINTER(F3), C.POINTER(F3), C.POINTER(F3), C.c_int32,
                                                C.c_int32, C.POINTER(GridDesc)]
        L.cagq_desc_from_dims.argtypes = [C.POINTER(F3), C.POINTER(F3), C.POINTER(I3), C.c_int32, C.c_int32,
                                          C.POINTER(GridDesc)]
        L.cagq_workspace_layout.argtypes = [C.c_int32, C.c_int32, C.POINTER(GridDesc), C.POINTER(LayoutC)]
        L.cagq_build_grid_static.argtypes = [P, C.c_int32, C.c_int32, C.POINTER(GridDesc), P, C.POINTER(GridC)]
        L.cagq_build_grid.argtypes = [P, C.c_int32, C.c_int32, C.POINTER(GridDesc), P, C.c_size_t, P,
                                      C.POINTER(GridC)]
        L.cagq_sample_centers.argtypes = [C.POINTER(GridC), C.c_int32, C.c_int32, C.c_uint64, C.c_uint32,
                                          P, P, P]
        L.cagq_query_context.argtypes = [C.POINTER(GridC), P, P, C.c_int32, C.c_int32, C.c_int32,
                                         C.c_uint64, P, P, P, P, P, P, P]
        L.cagq_query_points.argtypes = [C.POINTER(GridC), P, C.c_int32, C.c_int32, C.c_int32, C.c_uint64,
                                        P, P, P, P, P, P]
        L.cagq_context_offsets.argtypes = [C.POINTER(GridC), P, C.c_int32, P, P]
        L.cagq_context_list.argtypes = [C.POINTER(GridC), P, C.c_int32, P, P, C.c_int64, P]
        L.cagq_sample_points.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_uint64, P, P]
        L.cagq_ball_query.argtypes = [P, C.c_int32, C.c_int32, P, C.c_int32, C.c_int32, C.c_float, P, P, P]
        L.cagq_coverage.argtypes = [C.POINTER(GridC), P, P, C.c_int32, C.c_int32, P, P]
        L.cagq_get_device_status.argtypes = [C.POINTER(GridC), P]
        L.cagq_status_string.argtypes = [C.c_int]
        L.cagq_status_string.restype = C.c_char_p
        for f in ("cagq_desc_from_voxel_size", "cagq_desc_from_dims", "cagq_workspace_layout", "cagq_build_grid", "cagq_build_grid_static", "cagq_sample_centers",
                  "cagq_query_context", "cagq_query_points", "cagq_context_offsets", "cagq_context_list",
                  "cagq_sample_points", "cagq_ball_query", "cagq_coverage", "cagq_get_device_status"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().cagq_status_string(int(code)).decode()


def _check(rc: int, what: str):
    if rc != OK:
        raise CagqError(rc, what)


def make_desc(origin: Sequence[float], voxel_size: Sequence[float], dims: Sequence[int],
              n_v: int, radius: int = 1) -> GridDesc:
    d = GridDesc()
    for a in range(3):
        d.origin[a] = float(origin[a])
        d.voxel_size[a] = float(voxel_size[a])
        d.dims[a] = int(dims[a])
    d.n_v = int(n_v)
    d.radius = int(radius)
    return d


def desc_from_voxel_size(lo: Sequence[float], hi: Sequence[float], voxel_size: Sequence[float], n_v: int,
                         radius: int = 1) -> GridDesc:
    """GridDesc of the smallest grid at origin ``lo`` with the given voxel
    size whose voxels hold every point of the box [lo, hi] without clamping."""
    F3 = C.c_float * 3
    d = GridDesc()
    _check(lib().cagq_desc_from_voxel_size(C.byref(F3(*lo)), C.byref(F3(*hi)), C.byref(F3(*voxel_size)),
                                           int(n_v), int(radius), C.byref(d)), "cagq_desc_from_voxel_size")
    return d


def desc_from_dims(lo: Sequence[float], hi: Sequence[float], dims: Sequence[int], n_v: int,
                   radius: int = 1) -> GridDesc:
    """GridDesc at origin ``lo`` with ``dims`` voxels per axis spanning [lo, hi]."""
    F3, I3 = C.c_float * 3, C.c_int32 * 3
    d = GridDesc()
    _check(lib().cagq_desc_from_dims(C.byref(F3(*lo)), C.byref(F3(*hi)), C.byref(I3(*dims)),
                                     int(n_v), int(radius), C.byref(d)), "cagq_desc_from_dims")
    return d


def desc_from_spec(spec) -> GridDesc:
    """GridDesc from an object with origin, voxel_size, dims, n_v, radius."""
    return make_desc(spec.origin, spec.voxel_size, spec.dims, spec.n_v, spec.radius)


def workspace_layout(B: int, N: int, desc: GridDesc) -> LayoutC:
    out = LayoutC()
    _check(lib().cagq_workspace_layout(B, N, C.byref(desc), C.byref(out)), "cagq_workspace_layout")
    return out


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream_ptr(stream: Optional[torch.cuda.Stream] = None):
    """The HIP stream to launch on: ``stream``, else torch's current stream
    (read as a raw handle: building a Stream object per call costs ~3 us)."""
    if stream is not None:
        return C.c_void_p(stream.cuda_stream)
    if _raw_stream is not None and _cur_device is not None:
        return C.c_void_p(_raw_stream(_cur_device()))
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _need(t: torch.Tensor, dtype, shape, name: str):
    if not t.is_cuda or t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)} on the GPU, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


STATIC_WORKSPACE_BYTES = 64 << 20  # CAGQ_STATIC_WORKSPACE_BYTES


@dataclass
class Grid:
    """A built grid: the C record plus the tensors it borrows (workspace is
    None for a grid in the library's own array, cagq_build_grid_static)."""
    rec: GridC
    points: torch.Tensor
    workspace: Optional[torch.Tensor]
    layout: LayoutC

    @property
    def B(self) -> int:
        return self.rec.B

    @property
    def N(self) -> int:
        return self.rec.N

    def _view(self, off: int, count: int, dtype, ws: torch.Tensor) -> torch.Tensor:
        nbytes = count * torch.tensor([], dtype=dtype).element_size()
        return ws[off:off + nbytes].view(dtype)

    def _exposed(self) -> torch.Tensor:
        """The workspace bytes up to the end of the exposed arrays: the
        tensor itself, or a copy out of the library's array."""
        if self.workspace is not None:
            return self.workspace
        L = self.layout
        n = L.pt_list + 4 * self.B * self.N
        out = torch.empty(n, dtype=torch.uint8, device=self.points.device)
        torch.cuda.current_stream().synchronize()
        _check(0 if _hip().hipMemcpy(C.c_void_p(out.data_ptr()), C.c_void_p(self.rec.workspace), C.c_size_t(n),
                                     3) == 0 else ERR_HIP, "hipMemcpy")  # 3: device to device
        return out

    def table(self) -> Dict[str, torch.Tensor]:
        """Views of the occupied-voxel table inside the workspace (uint32 as int32)."""
        B, N, L = self.B, self.N, self.layout
        ws = self._exposed()
        return dict(
            nvox=self._view(L.nvox, B, torch.int32, ws),
            vox_lin=self._view(L.vox_lin, B * N, torch.int32, ws).view(B, N),
            vox_count=self._view(L.vox_count, B * N, torch.int32, ws).view(B, N),
            vox_off=self._view(L.vox_off, B * (N + 1), torch.int32, ws).view(B, N + 1),
            pt_list=self._view(L.pt_list, B * N, torch.int32, ws).view(B, N),
        )


_hip_lib = None


def _hip() -> C.CDLL:
    """The HIP runtime torch has loaded (for copies out of the library's own array)."""
    global _hip_lib
    if _hip_lib is None:
        _hip_lib = C.CDLL("libamdhip64.so")
        _hip_lib.hipMemcpy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]
        _hip_lib.hipMemcpy.restype = C.c_int
    return _hip_lib


def build_grid(points: torch.Tensor, desc: GridDesc, workspace: Optional[torch.Tensor] = None,
               stream: Optional[torch.cuda.Stream] = None) -> Grid:
    """Voxelize and index a batch ``points`` float32 [B, N, 3] (cagq_build_grid)."""
    if points.dim() != 3 or points.shape[2] != 3:
        raise ValueError("points must be [B, N, 3]")
    B, N = int(points.shape[0]), int(points.shape[1])
    _need(points, torch.float32, (B, N, 3), "points")
    lay = workspace_layout(B, N, desc)
    if workspace is None:
        workspace = torch.empty(lay.total_bytes, dtype=torch.uint8, device=points.device)
    rec = GridC()
    _check(lib().cagq_build_grid(_ptr(points), B, N, C.byref(desc), _ptr(workspace), workspace.numel(),
                                 _stream_ptr(stream), C.byref(rec)), "cagq_build_grid")
    return Grid(rec, points, workspace, lay)


def build_grid_static(points: torch.Tensor, desc: GridDesc, stream: Optional[torch.cuda.Stream] = None) -> Grid:
    """cagq_build_grid into the library's own array (cagq_build_grid_static):
    no workspace, no allocation by the call. A later static build on the same
    GPU overwrites the grid."""
    if points.dim() != 3 or points.shape[2] != 3:
        raise ValueError("points must be [B, N, 3]")
    B, N = int(points.shape[0]), int(points.shape[1])
    _need(points, torch.float32, (B, N, 3), "points")
    lay = workspace_layout(B, N, desc)
    rec = GridC()
    _check(lib().cagq_build_grid_static(_ptr(points), B, N, C.byref(desc), _stream_ptr(stream), C.byref(rec)),
           "cagq_build_grid_static")
    return Grid(rec, points, None, lay)


def sample_centers(grid: Grid, M: int, mode: str, seed: int, beta_q16: int = 0,
                   center_lin: Optional[torch.Tensor] = None, m_valid: Optional[torch.Tensor] = None,
                   stream: Optional[torch.cuda.Stream] = None):
    """M center voxels per cloud by RVS, CAS (greedy) or CAS with the paper's
    challenger / incumbent swaps (cagq_sample_centers; mode "rvs", "cas" or
    "cas_swap")."""
    dev = grid.points.device
    if center_lin is None:
        center_lin = torch.empty((grid.B, M), dtype=torch.int32, device=dev)
    if m_valid is None:
        m_valid = torch.empty((grid.B,), dtype=torch.int32, device=dev)
    _need(center_lin, torch.int32, (grid.B, M), "center_lin")
    _need(m_valid, torch.int32, (grid.B,), "m_valid")
    _check(lib().cagq_sample_centers(C.byref(grid.rec), M, SAMPLE[mode], C.c_uint64(seed & (2**64 - 1)),
                                     C.c_uint32(beta_q16), _ptr(center_lin), _ptr(m_valid),
                                     _stream_ptr(stream)), "cagq_sample_centers")
    return center_lin, m_valid


def alloc_query_outputs(B: int, M: int, K: int, device, want_xyz: bool = True,
                        want_ctx: bool = True) -> Dict[str, torch.Tensor]:
    return dict(
        node_idx=torch.empty((B, M, K), dtype=torch.int32, device=device),
        node_xyz=torch.empty((B, M, K, 3), dtype=torch.float32, device=device) if want_xyz else None,
        n_valid=torch.empty((B, M), dtype=torch.int32, device=device),
        center_xyz=torch.empty((B, M, 3), dtype=torch.float32, device=device),
        center_w=torch.empty((B, M), dtype=torch.int32, device=device),
        ctx_count=torch.empty((B, M), dtype=torch.int32, device=device) if want_ctx else None,
    )


def query_context(grid: Grid, center_lin: torch.Tensor, K: int, mode: str, seed: int,
                  weights: Optional[torch.Tensor] = None, out: Optional[Dict[str, torch.Tensor]] = None,
                  want_xyz: bool = True, want_ctx: bool = True,
                  stream: Optional[torch.cuda.Stream] = None) -> Dict[str, torch.Tensor]:
    """K node points and the group center per center voxel (cagq_query_context).

    ``weights`` int32/uint32-valued [B, N] or None (all 1). ``center_w`` holds
    uint32 values in an int32 tensor.
    """
    B, M = int(center_lin.shape[0]), int(center_lin.shape[1])
    _need(center_lin, torch.int32, (B, M), "center_lin")
    if weights is not None:
        _need(weights, torch.int32, (grid.B, grid.N), "weights")
    if out is None:
        out = alloc_query_outputs(B, M, K, grid.points.device, want_xyz, want_ctx)
    _check(lib().cagq_query_context(
        C.byref(grid.rec), _ptr(weights), _ptr(center_lin), M, K, QUERY[mode], C.c_uint64(seed & (2**64 - 1)),
        _ptr(out["node_idx"]), _ptr(out.get("node_xyz")), _ptr(out["n_valid"]), _ptr(out["center_xyz"]),
        _ptr(out["center_w"]), _ptr(out.get("ctx_count")), _stream_ptr(stream)), "cagq_query_context")
    return out


def query_points(grid: Grid, centers: torch.Tensor, K: int, mode: str, seed: int,
                 out: Optional[Dict[str, torch.Tensor]] = None, want_xyz: bool = True,
                 stream: Optional[torch.cuda.Stream] = None) -> Dict[str, torch.Tensor]:
    """Upsampling query: K node points around given center points [B, M, 3]
    (cagq_query_points). Also returns ctx_count and each center's voxel lin."""
    B, M = int(centers.shape[0]), int(centers.shape[1])
    _need(centers, torch.float32, (B, M, 3), "centers")
    dev = grid.points.device
    if out is None:
        out = dict(
            node_idx=torch.empty((B, M, K), dtype=torch.int32, device=dev),
            node_xyz=torch.empty((B, M, K, 3), dtype=torch.float32, device=dev) if want_xyz else None,
            n_valid=torch.empty((B, M), dtype=torch.int32, device=dev),
            ctx_count=torch.empty((B, M), dtype=torch.int32, device=dev),
            center_lin=torch.empty((B, M), dtype=torch.int32, device=dev),
        )
    _check(lib().cagq_query_points(
        C.byref(grid.rec), _ptr(centers), M, K, QUERY[mode], C.c_uint64(seed & (2**64 - 1)),
        _ptr(out["node_idx"]), _ptr(out.get("node_xyz")), _ptr(out["n_valid"]), _ptr(out.get("ctx_count")),
        _ptr(out.get("center_lin")), _stream_ptr(stream)), "cagq_query_points")
    return out


def context_offsets(grid: Grid, center_lin: torch.Tensor, out: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """CSR offsets [B*M + 1] (int64) of the centers' context lists."""
    B, M = int(center_lin.shape[0]), int(center_lin.shape[1])
    _need(center_lin, torch.int32, (B, M), "center_lin")
    if out is None:
        out = torch.empty(B * M + 1, dtype=torch.int64, device=grid.points.device)
    _need(out, torch.int64, (B * M + 1,), "ctx_off")
    _check(lib().cagq_context_offsets(C.byref(grid.rec), _ptr(center_lin), M, _ptr(out), _stream_ptr(stream)),
           "cagq_context_offsets")
    return out


def context_list(grid: Grid, center_lin: torch.Tensor, ctx_off: torch.Tensor,
                 out: Optional[torch.Tensor] = None, capacity: Optional[int] = None,
                 stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """The context lists (int32 point indices) laid out by ``ctx_off``. Without
    ``out`` the total is read back from ``ctx_off`` to size it."""
    B, M = int(center_lin.shape[0]), int(center_lin.shape[1])
    _need(center_lin, torch.int32, (B, M), "center_lin")
    _need(ctx_off, torch.int64, (B * M + 1,), "ctx_off")
    if out is None:
        total = int(ctx_off[-1].item())
        out = torch.empty(max(total, 1), dtype=torch.int32, device=grid.points.device)
        capacity = total
    if capacity is None:
        capacity = int(out.numel())
    _check(lib().cagq_context_list(C.byref(grid.rec), _ptr(center_lin), M, _ptr(ctx_off), _ptr(out),
                                   int(capacity), _stream_ptr(stream)), "cagq_context_list")
    return out


POINTS = {"rps": 0, "fps": 1}


def sample_points(points: torch.Tensor, M: int, mode: str, seed: int = 0, out: Optional[torch.Tensor] = None,
                  stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Random / Farthest Point Sampling (comparison methods): [B, M] point indices."""
    B, N = int(points.shape[0]), int(points.shape[1])
    _need(points, torch.float32, (B, N, 3), "points")
    if out is None:
        out = torch.empty((B, M), dtype=torch.int32, device=points.device)
    _check(lib().cagq_sample_points(_ptr(points), B, N, M, POINTS[mode], C.c_uint64(seed & (2**64 - 1)), _ptr(out),
                                    _stream_ptr(stream)), "cagq_sample_points")
    return out


def ball_query(points: torch.Tensor, center_idx: torch.Tensor, K: int, radius2: float,
               out: Optional[Dict[str, torch.Tensor]] = None,
               stream: Optional[torch.cuda.Stream] = None) -> Dict[str, torch.Tensor]:
    """Ball Query (comparison method): the first K points within the radius."""
    B, N = int(points.shape[0]), int(points.shape[1])
    M = int(center_idx.shape[1])
    _need(points, torch.float32, (B, N, 3), "points")
    _need(center_idx, torch.int32, (B, M), "center_idx")
    if out is None:
        out = dict(node_idx=torch.empty((B, M, K), dtype=torch.int32, device=points.device),
                   n_valid=torch.empty((B, M), dtype=torch.int32, device=points.device))
    _check(lib().cagq_ball_query(_ptr(points), B, N, _ptr(center_idx), M, K, C.c_float(radius2),
                                 _ptr(out["node_idx"]), _ptr(out["n_valid"]), _stream_ptr(stream)),
           "cagq_ball_query")
    return out


def coverage(grid: Grid, node_idx: torch.Tensor, n_valid: torch.Tensor, out: Optional[torch.Tensor] = None,
             stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Occupied voxels [B] holding a valid node point (divide by nvox for the metric)."""
    B, M, K = (int(x) for x in node_idx.shape)
    _need(node_idx, torch.int32, (B, M, K), "node_idx")
    _need(n_valid, torch.int32, (B, M), "n_valid")
    if out is None:
        out = torch.empty(B, dtype=torch.int32, device=node_idx.device)
    _check(lib().cagq_coverage(C.byref(grid.rec), _ptr(node_idx), _ptr(n_valid), M, K, _ptr(out),
                               _stream_ptr(stream)), "cagq_coverage")
    return out


def get_device_status(grid: Grid, stream: Optional[torch.cuda.Stream] = None) -> int:
    """Synchronises the stream; first device-side error since the grid was built."""
    return int(lib().cagq_get_device_status(C.byref(grid.rec), _stream_ptr(stream)))


def run_layer(points: torch.Tensor, layer, weights: Optional[torch.Tensor] = None,
              workspace: Optional[torch.Tensor] = None):
    """One CAGQ layer (build, sample, query) for a LayerSpec-like object.

    Returns (grid, center_lin, m_valid, query outputs)."""
    g = build_grid(points, desc_from_spec(layer.grid), workspace)
    cl, mv = sample_centers(g, layer.M, layer.sample, layer.seed)
    q = query_context(g, cl, layer.K, layer.query, layer.seed, weights=weights)
    return g, cl, mv, q
