"""Independent reference computations that pin the oracle (tests only).

Nothing here imports the oracle or the HIP library. Each helper re-derives a
piece of CAGQ from a textbook routine (numpy unique / argsort / lexsort,
brute-force enumeration) rather than from the oracle's code path.
"""
from __future__ import annotations

import itertools
from typing import Dict, List, Sequence, Tuple

import numpy as np

MASK64 = (1 << 64) - 1


def py_splitmix64_next(state: int) -> Tuple[int, int]:
    """One step of the splitmix64 generator: (new_state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return state, z ^ (z >> 31)


def py_sm64(x: int) -> int:
    """The generator's output for state x (mix of x + golden gamma)."""
    return py_splitmix64_next(x & MASK64)[1]


def py_chain(seed: int, tag: int, *fields: int) -> int:
    h = py_sm64(seed ^ tag)
    for a in fields:
        h = py_sm64(h ^ (int(a) & MASK64))
    return h


def grid_coords_f64(points: np.ndarray, origin, size, dims) -> np.ndarray:
    """Voxel coordinates in exact-ish fp64 (valid away from voxel faces)."""
    t = (points.astype(np.float64) - np.asarray(origin, np.float64)) / np.asarray(size, np.float64)
    g = np.floor(t)
    return np.clip(g, 0, np.asarray(dims) - 1).astype(np.int64)


def lin_of(g: np.ndarray, dims) -> np.ndarray:
    return g[..., 0] + dims[0] * (g[..., 1] + dims[1] * g[..., 2])


def table_numpy(lin: np.ndarray, n_v: int) -> Dict[str, np.ndarray]:
    """Occupied-voxel table of one cloud from np.unique and a stable argsort."""
    vox, counts = np.unique(lin, return_counts=True)
    order = np.argsort(lin, kind="stable")          # by voxel, then by point index
    stored = np.minimum(counts, n_v)
    off = np.concatenate([[0], np.cumsum(stored)])
    starts = np.concatenate([[0], np.cumsum(counts)])
    lists = np.concatenate([order[starts[s]:starts[s] + stored[s]] for s in range(len(vox))])
    return dict(vox_lin=vox, vox_count=counts, vox_off=off, pt_list=lists)


def decode(lin: int, dims) -> Tuple[int, int, int]:
    return lin % dims[0], (lin // dims[0]) % dims[1], lin // (dims[0] * dims[1])


def neighbourhood_sets(vox_lin: Sequence[int], dims, r: int) -> List[List[int]]:
    """pi(v) as lists of indices into vox_lin, by brute force over all pairs."""
    coords = np.array([decode(int(l), dims) for l in vox_lin]).reshape(-1, 3)
    out = []
    for i in range(len(vox_lin)):
        d = np.abs(coords - coords[i]).max(axis=1)
        out.append(list(np.nonzero(d <= r)[0]))
    return out


def cas_scores_bruteforce(nbr: List[List[int]], C: np.ndarray, lam: int, beta_q16: int) -> np.ndarray:
    s = np.empty(len(nbr), dtype=object)
    for v, vs in enumerate(nbr):
        U = sum(1 for V in vs if C[V] == 0)
        s[v] = 65536 * lam * U - beta_q16 * int(sum(int(C[V]) for V in vs))
    return s


def coverage(nbr: List[List[int]], chosen: Sequence[int]) -> int:
    cov = set()
    for v in chosen:
        cov.update(nbr[v])
    return len(cov)


def exhaustive_best_coverage(nbr: List[List[int]], M: int) -> int:
    best = 0
    for comb in itertools.combinations(range(len(nbr)), M):
        best = max(best, coverage(nbr, comb))
    return best
