"""The CPU oracle against what the paper and the mathematics fix.

Each test pins one oracle function to something other than itself: published
generator outputs, textbook routines (numpy unique / argsort / lexsort),
brute force on small inputs, exhaustive optima, closed forms and statistics.
"""
import math
import os

import numpy as np
import pytest

import oracle
from paper_1912_02984_amd import workloads as W
from tests import pins

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _grid(origin=(0, 0, 0), size=(0.25, 0.25, 0.25), dims=(8, 8, 8), n_v=4, r=1):
    return oracle.make_grid(origin, size, dims, n_v, r)


# ---------------------------------------------------------------- splitmix64

def test_splitmix64_published_outputs():
    """The hash chain's primitive reproduces the generator's published outputs."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "splitmix64.txt")) if l.strip() and l[0] != "#"]
    assert len(rows) == 4
    for seed, idx, out in rows:
        state = int(seed)
        # the idx-th output of a generator seeded with `state` is sm64(state + (idx-1)*gamma)
        x = (state + (int(idx) - 1) * 0x9E3779B97F4A7C15) & pins.MASK64
        assert oracle.splitmix64(x) == int(out, 16)
        st, o = state, None
        for _ in range(int(idx)):
            st, o = pins.py_splitmix64_next(st)
        assert o == int(out, 16)


def test_splitmix64_matches_python_generator_on_random_inputs():
    rng = np.random.default_rng(7)
    for x in rng.integers(0, 2**63, size=200, dtype=np.int64):
        x = int(x) * 2 + 1
        assert oracle.splitmix64(x) == pins.py_sm64(x)


# ---------------------------------------------------------------- voxelize

def test_voxelize_hand_placed_points():
    """Exact voxel faces, clamping outside the grid, x-fastest linear order."""
    g = _grid(dims=(8, 4, 2))
    P = np.array([
        [0.0, 0.0, 0.0],        # corner -> voxel (0,0,0)
        [0.25, 0.0, 0.0],       # exactly on the face x=1 -> g_x = 1
        [0.2499999, 0.0, 0.0],  # just below the face -> 0
        [1.999, 0.99, 0.49],    # last voxel (7,3,1)
        [2.0, 1.0, 0.5],        # exactly dims*size -> clamped to (7,3,1)
        [-5.0, -0.0, -1e-30],   # negative -> clamped to 0
        [1e30, 0.5, 0.3],       # far outside -> clamped to D-1 on x
        [0.75, 0.5, 0.25],      # (3,2,1)
    ], np.float32)
    lin = oracle.voxelize(P, g)
    expect = [(0, 0, 0), (1, 0, 0), (0, 0, 0), (7, 3, 1), (7, 3, 1), (0, 0, 0), (7, 2, 1), (3, 2, 1)]
    assert [int(l) for l in lin] == [x + 8 * (y + 4 * z) for x, y, z in expect]


def test_voxelize_divide_is_correctly_rounded():
    """(p - o) / s is one correctly rounded fp32 divide: with s = 0.1f and
    p = 1.3f the exact quotient is 12.9999993..., so g = 12 (a reciprocal
    multiply would round to 13)."""
    g = oracle.make_grid((0, 0, 0), (0.1, 0.1, 0.1), (40, 40, 40), 4, 1)
    xs = np.array([1.3, 2.1, 2.6], np.float32)
    P = np.stack([xs, np.zeros(3, np.float32), np.zeros(3, np.float32)], 1)
    exact = np.floor(xs.astype(np.float64) / np.float64(np.float32(0.1)))
    assert list(exact) == [12, 20, 25]
    assert list(oracle.voxelize(P, g)) == [12, 20, 25]


def test_voxelize_nonfinite_is_an_error():
    g = _grid()
    with pytest.raises(oracle.OracleError, match="-4"):
        oracle.voxelize(np.array([[0.1, np.nan, 0.1]], np.float32), g)
    with pytest.raises(oracle.OracleError, match="-4"):
        oracle.voxelize(np.array([[np.inf, 0.1, 0.1]], np.float32), g)


def test_voxelize_agrees_with_fp64_floor_away_from_faces():
    """Away from voxel faces the fp32 index equals the exact floor((p - o) / s)."""
    w = W.get_workload("room")
    P = w.points(B=1)[0]
    gs = w.layers[0].grid
    lin = oracle.voxelize(P, oracle.grid_from_spec(gs))
    t = (P.astype(np.float64) - np.array(gs.origin)) / np.array(gs.voxel_size)
    far = np.all(np.abs(t - np.round(t)) > 1e-4, axis=1)
    assert far.mean() > 0.99
    g = pins.grid_coords_f64(P, gs.origin, gs.voxel_size, gs.dims)
    assert np.array_equal(lin[far], pins.lin_of(g, gs.dims)[far])


# ---------------------------------------------------------------- table

@pytest.mark.parametrize("name", ["tiny", "object", "room"])
def test_table_matches_numpy_unique_and_stable_argsort(name):
    w = W.get_workload(name)
    P = w.points()
    gs = w.layers[0].grid
    # a tighter cap than the workload's so that the cap binds somewhere
    for n_v in (gs.n_v, 2):
        grid = oracle.make_grid(gs.origin, gs.voxel_size, gs.dims, n_v, gs.radius)
        t = oracle.Table(P, grid)
        lin = oracle.voxelize(P, grid)
        for b in range(min(t.B, 4)):
            ref = pins.table_numpy(lin[b], n_v)
            nv = t.nvox[b]
            assert nv == len(ref["vox_lin"])
            assert np.array_equal(t.vox_lin[b, :nv], ref["vox_lin"])
            assert np.array_equal(t.vox_count[b, :nv], ref["vox_count"])
            assert int(t.vox_count[b, :nv].sum()) == t.N          # every point in one voxel
            assert np.array_equal(t.vox_off[b, :nv + 1], ref["vox_off"])
            S = t.vox_off[b, nv]
            assert np.array_equal(t.pt_list[b, :S], ref["pt_list"])


def test_table_all_points_in_one_voxel():
    P = np.full((1, 100, 3), 0.1, np.float32)
    t = oracle.Table(P, _grid(n_v=5))
    assert t.nvox[0] == 1 and t.vox_count[0, 0] == 100
    assert list(t.pt_list[0, :5]) == [0, 1, 2, 3, 4]


# ---------------------------------------------------------------- RVS

def test_rvs_is_the_m_smallest_keys_in_slot_order():
    w = W.get_workload("object")
    P = w.points()[:3]
    L = w.layers[0]
    t = oracle.Table(P, oracle.grid_from_spec(L.grid))
    for M, seed in ((128, 42), (5, 9), (10_000, 3)):
        cl, mv = t.sample_rvs(M, seed)
        for b in range(t.B):
            nv = int(t.nvox[b])
            keys = [((pins.py_chain(seed, 1, b, s) >> 32) << 32) | s for s in range(nv)]
            m = min(M, nv)
            assert mv[b] == m
            chosen = sorted(k & 0xFFFFFFFF for k in sorted(keys)[:m])
            expect = [int(t.vox_lin[b, s]) for s in chosen]
            assert list(cl[b, :m]) == expect
            assert all(cl[b, j] == cl[b, j % m] for j in range(m, M))


def test_rvs_equal_inclusion_probability():
    """Every occupied voxel is picked with the same probability (Sec. 3.2)."""
    P = W.uniform_cube(1, 300, 5)
    t = oracle.Table(P, oracle.make_grid((0, 0, 0), (0.25,) * 3, (4, 4, 4), 8, 1))
    nv = int(t.nvox[0])
    M, trials = 16, 3000
    hits = np.zeros(nv)
    for seed in range(trials):
        cl, _ = t.sample_rvs(M, seed)
        hits[np.searchsorted(t.vox_lin[0, :nv], cl[0])] += 1
    expect = trials * M / nv
    chi2 = ((hits - expect) ** 2 / expect).sum()
    # chi-square with nv-1 dof; 99.9th percentile is below dof + 4.5*sqrt(2 dof)
    assert chi2 < (nv - 1) + 4.5 * math.sqrt(2 * (nv - 1)), chi2


# ---------------------------------------------------------------- CAS

def _small_table(seed, npts=60, dims=(6, 6, 3), n_v=4):
    rng = np.random.default_rng(seed)
    P = (rng.random((1, npts, 3)) * np.array(dims) * 0.25).astype(np.float32)
    return oracle.Table(P, oracle.make_grid((0, 0, 0), (0.25,) * 3, dims, n_v, 1))


@pytest.mark.parametrize("beta_q16", [0, 65536 // 4, 3 * 65536])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_cas_every_step_is_the_bruteforce_argmax(seed, beta_q16):
    t = _small_table(seed)
    nv = int(t.nvox[0])
    vl = [int(x) for x in t.vox_lin[0, :nv]]
    nbr = pins.neighbourhood_sets(vl, t.grid.dims, 1)
    M = min(25, nv)
    cl, mv, pick_lin, pick_score = t.sample_cas(M, beta_q16)
    C = np.zeros(nv, np.int64)
    picked = set()
    for step in range(M):
        scores = pins.cas_scores_bruteforce(nbr, C, 27, beta_q16)
        cand = [v for v in range(nv) if v not in picked]
        best = max(scores[v] for v in cand)
        v = min(v for v in cand if scores[v] == best)          # ties -> lowest lin
        assert pick_lin[0, step] == vl[v]
        assert pick_score[0, step] == best
        picked.add(v)
        for V in nbr[v]:
            C[V] += 1
    assert list(cl[0, :M]) == sorted(pick_lin[0, :M])


def test_cas_monotone_scores_and_exact_coverage_gain():
    """beta = 0: pick scores never rise and each pick covers exactly U(pick) new voxels."""
    w = W.get_workload("object")
    t = oracle.Table(w.points()[:2], oracle.grid_from_spec(w.layers[0].grid))
    M = 300
    cl, mv, pick_lin, pick_score = t.sample_cas(M)
    for b in range(t.B):
        nv = int(t.nvox[b])
        vl = [int(x) for x in t.vox_lin[b, :nv]]
        index = {l: i for i, l in enumerate(vl)}
        nbr = pins.neighbourhood_sets(vl, t.grid.dims, 1)
        covered = set()
        prev = None
        for j in range(M):
            s = int(pick_score[b, j])
            if prev is not None:
                assert s <= prev
            prev = s
            new = set(nbr[index[int(pick_lin[b, j])]]) - covered
            assert s == 65536 * 27 * len(new)
            covered |= new


@pytest.mark.parametrize("seed", range(6))
def test_cas_against_exhaustive_optimum(seed):
    """Greedy max-coverage: equal to OPT at M = 1 and >= (1-(1-1/M)^M) OPT
    (Nemhauser, Wolsey, Fisher 1978) on <= 64 occupied voxels."""
    t = _small_table(100 + seed, npts=18, dims=(5, 5, 2))
    nv = int(t.nvox[0])
    assert nv <= 64
    vl = [int(x) for x in t.vox_lin[0, :nv]]
    index = {l: i for i, l in enumerate(vl)}
    nbr = pins.neighbourhood_sets(vl, t.grid.dims, 1)
    for M in (1, 2, 3):
        cl, mv, _, _ = t.sample_cas(M)
        got = pins.coverage(nbr, [index[int(l)] for l in cl[0, :M]])
        opt = pins.exhaustive_best_coverage(nbr, M)
        if M == 1:
            assert got == opt
        assert got >= (1 - (1 - 1 / M) ** M) * opt - 1e-9
        assert got <= opt


def test_cas_disjoint_neighbourhoods_pick_lowest_lin():
    """All neighbourhoods disjoint and equal: every score ties, so CAS returns
    the M lowest linear ids."""
    pts = []
    for x in range(0, 12, 3):
        for y in range(0, 12, 3):
            pts.append([(x + 0.5) * 0.25, (y + 0.5) * 0.25, 0.1])
    P = np.array([pts], np.float32)
    t = oracle.Table(P, oracle.make_grid((0, 0, 0), (0.25,) * 3, (12, 12, 1), 4, 1))
    cl, mv, _, ps = t.sample_cas(5)
    assert list(cl[0]) == sorted(t.vox_lin[0, :t.nvox[0]])[:5]
    assert np.all(ps[0] == 65536 * 27 * 1)


def test_cas_takes_everything_when_m_exceeds_occupancy():
    t = _small_table(3, npts=10)
    nv = int(t.nvox[0])
    cl, mv, _, _ = t.sample_cas(nv + 7)
    assert mv[0] == nv
    assert list(cl[0, :nv]) == list(t.vox_lin[0, :nv])
    assert all(cl[0, j] == cl[0, j % nv] for j in range(nv, nv + 7))


# ---------------------------------------------------------------- CAS, the paper's swap procedure

def _replay_swaps(t, b, M, seed, dec):
    """Incumbent slots after every challenge, replaying the oracle's
    decisions from its RVS choice: a list of (accepted, incumbent voxel
    indices) per challenge."""
    nv = int(t.nvox[b])
    vl = [int(x) for x in t.vox_lin[b, :nv]]
    index = {l: i for i, l in enumerate(vl)}
    rvs, mv = t.sample_rvs(M, seed)
    m = int(mv[b])
    inc = [index[int(l)] for l in rvs[b, :m]]
    initial = set(inc)
    challengers = [v for v in range(nv) if v not in initial]
    states = []
    for tch, v in enumerate(challengers):
        d = int(dec[b, tch])
        j = d if d >= 0 else -d - 1
        # the slot draw, from an independent hash: hi32(h(seed, 3, b, t)) mod m
        assert j == (pins.py_chain(seed, 3, b, tch) >> 32) % m
        if d >= 0:
            inc[j] = v
        states.append((d >= 0, list(inc)))
    return vl, inc, states


@pytest.mark.parametrize("seed", [0, 5, 9])
def test_cas_swap_decisions_replay_and_coverage_grows(seed):
    """beta = 0 (Sec. 3.2): every accepted replacement strictly enlarges the
    covered occupied space, recomputed from scratch from the replayed
    incumbent sets; refusals leave it unchanged; the replay ends at the
    emitted centers."""
    w = W.get_workload("object")
    L = w.layers[0]
    t = oracle.Table(w.points()[:3], oracle.grid_from_spec(L.grid))
    M = 200
    cl, mv, dec, ns = t.sample_cas_swap(M, seed)
    total = 0
    for b in range(t.B):
        vl, inc, states = _replay_swaps(t, b, M, seed, dec)
        nbr = pins.neighbourhood_sets(vl, t.grid.dims, 1)
        rvs, _ = t.sample_rvs(M, seed)
        index = {l: i for i, l in enumerate(vl)}
        prev = pins.coverage(nbr, [index[int(l)] for l in rvs[b, :mv[b]]])
        swaps = 0
        for accepted, cur in states:
            cov = pins.coverage(nbr, cur)
            if accepted:
                assert cov > prev
                swaps += 1
            else:
                assert cov == prev
            prev = cov
        assert swaps == ns[b]
        assert sorted(vl[v] for v in inc) == list(cl[b, :mv[b]])
        total += swaps
    assert total > 0


def test_cas_swap_hand_worked_row():
    """Occupied voxels x = 0, 2, 3, 4 of one grid row, r = 1, M = 1. From
    Eqs. 2-3 by hand: starting at x = 0, challenger 2 has H_add = 2 (x = 2,
    3 uncovered) against H_rmv = 1 and replaces it, after which 3 and 4
    gain 1 against 2; starting at 2, 3 or 4 no challenger wins. So the
    result is 2, 2, 3, 4 for a start at 0, 2, 3, 4."""
    pts = [[(x + 0.5) * 0.25, 0.1, 0.1] for x in (0, 2, 3, 4)]
    P = np.array([pts], np.float32)
    t = oracle.Table(P, oracle.make_grid((0, 0, 0), (0.25,) * 3, (8, 1, 1), 4, 1))
    expect = {0: 2, 2: 2, 3: 3, 4: 4}
    seen = set()
    for seed in range(40):
        rvs, _ = t.sample_rvs(1, seed)
        cl, mv, dec, ns = t.sample_cas_swap(1, seed)
        start = int(rvs[0, 0])
        assert int(cl[0, 0]) == expect[start]
        assert ns[0] == (1 if start == 0 else 0)
        seen.add(start)
    assert 0 in seen  # the swapping case was exercised


def test_cas_swap_never_swaps_isolated_voxels():
    """pi(v) = {v} for every voxel: H_add = 1 = H_rmv, so no challenger wins
    and the result is the RVS choice."""
    pts = [[(x + 0.5) * 0.25, (y + 0.5) * 0.25, 0.1] for x in range(0, 16, 2) for y in range(0, 16, 2)]
    P = np.array([pts], np.float32)
    t = oracle.Table(P, oracle.make_grid((0, 0, 0), (0.25,) * 3, (16, 16, 1), 4, 1))
    for seed in range(3):
        cl, mv, dec, ns = t.sample_cas_swap(10, seed)
        rvs, _ = t.sample_rvs(10, seed)
        assert ns[0] == 0
        assert np.array_equal(cl, rvs)


def test_cas_swap_takes_everything_when_m_exceeds_occupancy():
    t = _small_table(3, npts=10)
    nv = int(t.nvox[0])
    cl, mv, dec, ns = t.sample_cas_swap(nv + 5, 1)
    assert mv[0] == nv and ns[0] == 0
    assert list(cl[0, :nv]) == list(t.vox_lin[0, :nv])


# ---------------------------------------------------------------- query

def _context_bruteforce(P, lin, tb, center_lin, dims, r):
    """Stored points of every occupied voxel within Chebyshev distance r."""
    gc = np.array(pins.decode(center_lin, dims))
    stored = tb["pt_list"]
    g = np.stack([lin % dims[0], (lin // dims[0]) % dims[1], lin // (dims[0] * dims[1])], -1)
    near = np.abs(g - gc).max(axis=1) <= r
    keep = np.zeros(len(lin), bool)
    keep[stored] = True
    return np.nonzero(near & keep)[0]


@pytest.mark.parametrize("n_v", [32, 3])
def test_knn_matches_bruteforce_over_the_context(n_v):
    w = W.get_workload("room")
    P = w.points(B=1)
    gs = w.layers[0].grid
    grid = oracle.make_grid(gs.origin, gs.voxel_size, gs.dims, n_v, 1)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(200, 11)
    K = 16
    q = t.query(cl, mv, K, "knn", 0)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, n_v)
    o, s, dims = np.float32(gs.origin), np.float32(gs.voxel_size), gs.dims
    for j in range(200):
        ctx = _context_bruteforce(P[0], lin, tb, int(cl[0, j]), dims, 1)
        assert q["ctx_count"][0, j] == len(ctx)
        g = np.array(pins.decode(int(cl[0, j]), dims), np.float32)
        c = o + (g + np.float32(0.5)) * s                   # voxel center, fp32
        d = P[0, ctx] - c
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        order = np.lexsort((ctx, d2.view(np.uint32)))
        n = min(K, len(ctx))
        assert q["n_valid"][0, j] == n
        assert list(q["node_idx"][0, j, :n]) == list(ctx[order[:n]])
        assert np.all(q["node_idx"][0, j, n:] == q["node_idx"][0, j, 0])
        assert np.array_equal(q["node_xyz"][0, j].view(np.uint32), P[0, q["node_idx"][0, j]].view(np.uint32))


def test_knn_bruteforce_on_a_non_cubic_grid():
    """Unequal dims and voxel sizes per axis exercise the x-fastest decode."""
    P = W.uniform_cube(1, 600, 31) * np.array([0.7, 0.5, 0.8], np.float32)
    dims, size = (7, 5, 4), (0.1, 0.1, 0.2)
    grid = oracle.make_grid((0, 0, 0), size, dims, 6, 1)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(60, 2)
    K = 12
    q = t.query(cl, mv, K, "knn", 0)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, 6)
    for j in range(60):
        ctx = _context_bruteforce(P[0], lin, tb, int(cl[0, j]), dims, 1)
        g = np.array(pins.decode(int(cl[0, j]), dims), np.float32)
        c = np.zeros(3, np.float32) + (g + np.float32(0.5)) * np.array(size, np.float32)
        d = P[0, ctx] - c
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        order = np.lexsort((ctx, d2.view(np.uint32)))
        n = min(K, len(ctx))
        assert list(q["node_idx"][0, j, :n]) == list(ctx[order[:n]])


def test_knn_equals_global_knn_when_the_neighbourhood_suffices():
    """No cap binding and the K-th distance well inside the (2r+1)^3 block:
    CAGQ k-NN is the ordinary k-NN over all N points (textbook brute force)."""
    P = W.uniform_cube(1, 4000, 21)
    size = 0.1
    grid = oracle.make_grid((0, 0, 0), (size,) * 3, (10, 10, 10), 64, 1)
    t = oracle.Table(P, grid)
    assert t.vox_count.max() <= 64
    cl, mv = t.sample_rvs(300, 4)
    K = 8
    q = t.query(cl, mv, K, "knn", 0)
    checked = 0
    for j in range(300):
        g = np.array(pins.decode(int(cl[0, j]), (10, 10, 10)))
        c = (g + 0.5) * size
        d = np.sqrt(((P[0].astype(np.float64) - c) ** 2).sum(1))
        order = np.argsort(d, kind="stable")
        if d[order[K - 1]] < 1.5 * size - 1e-3 and d[order[K]] - d[order[K - 1]] > 1e-5:
            assert set(q["node_idx"][0, j]) == set(order[:K])
            checked += 1
    assert checked > 100


def test_cube_query_is_a_random_subset_of_the_context():
    w = W.get_workload("room")
    P = w.points(B=1)
    gs = w.layers[0].grid
    grid = oracle.grid_from_spec(gs)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(300, 5)
    K = 8
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, gs.n_v)
    q = t.query(cl, mv, K, "cube", 77)
    for j in range(300):
        ctx = set(_context_bruteforce(P[0], lin, tb, int(cl[0, j]), gs.dims, 1))
        n = min(K, len(ctx))
        got = list(q["node_idx"][0, j, :n])
        assert q["n_valid"][0, j] == n and len(set(got)) == n and set(got) <= ctx
        if len(ctx) <= K:
            assert set(got) == ctx
        key = [pins.py_chain(77, 2, 0, int(cl[0, j]), i) >> 32 for i in got]
        assert key == sorted(key)


def test_cube_query_inclusion_frequency():
    """Each context point is kept with probability K / c (uniform subset)."""
    P = W.uniform_cube(1, 400, 8)
    grid = oracle.make_grid((0, 0, 0), (0.5,) * 3, (2, 2, 2), 64, 1)
    t = oracle.Table(P, grid)
    cl = np.array([[int(t.vox_lin[0, 0])]], np.int32)
    K, trials = 10, 2000
    hits = np.zeros(400)
    c = None
    for seed in range(trials):
        q = t.query(cl, np.array([1], np.int32), K, "cube", seed)
        c = int(q["ctx_count"][0, 0])
        hits[q["node_idx"][0, 0]] += 1
    ctx = hits > 0
    assert ctx.sum() == c
    p = K / c
    expect = trials * p
    z = (hits[ctx] - expect) / math.sqrt(trials * p * (1 - p))
    assert np.abs(z).max() < 5.0


def test_center_closed_forms():
    grid = oracle.make_grid((0, 0, 0), (4.0,) * 3, (1, 1, 1), 8, 1)
    # one node, weight 1: the center is that point
    P = np.array([[[1.25, 2.5, 3.75]]], np.float32)
    t = oracle.Table(P, grid)
    cl = np.array([[0]], np.int32)
    q = t.query(cl, np.array([1], np.int32), 4, "knn", 0)
    assert np.array_equal(q["center_xyz"][0, 0], P[0, 0]) and q["center_w"][0, 0] == 1
    # two nodes: the correctly rounded midpoint
    P = np.array([[[1.0, 0.1, 3.0], [1.0000001, 0.3, 2.9]]], np.float32)
    t = oracle.Table(P, grid)
    q = t.query(cl, np.array([1], np.int32), 4, "knn", 0)
    mid = ((P[0, 0].astype(np.float64) + P[0, 1]) / 2).astype(np.float32)
    assert np.array_equal(q["center_xyz"][0, 0], mid)
    # weights: w_c is the integer sum, the center the weighted mean
    w = np.array([[3, 5]], np.uint32)
    q = t.query(cl, np.array([1], np.int32), 4, "knn", 0, weights=w)
    assert q["center_w"][0, 0] == 8
    ref = (3 * P[0, 0].astype(np.float64) + 5 * P[0, 1]) / 8
    assert np.allclose(q["center_xyz"][0, 0], ref, rtol=2e-7, atol=0)


def test_center_follows_the_pairwise_order():
    """x = [1, 2^-24, 2^-24, 2^-24] (in node order): pairwise gives
    (1 + 2^-24) + (2^-24 + 2^-24) = 1 + 2^-23, a left-to-right sum gives 1."""
    e = 2.0 ** -24
    # node order is the k-NN order; y places the points at increasing distance
    # from the voxel center (2, 2, 2) while x carries the test values
    P = np.array([[[1.0, 2.0, 2.0], [e, 2.0, 2.0], [e, 2.2, 2.0], [e, 2.4, 2.0]]], np.float32)
    grid = oracle.make_grid((0, 0, 0), (4.0,) * 3, (1, 1, 1), 8, 1)
    t = oracle.Table(P, grid)
    q = t.query(np.array([[0]], np.int32), np.array([1], np.int32), 4, "knn", 0)
    assert list(q["node_idx"][0, 0]) == [0, 1, 2, 3]
    assert q["center_xyz"][0, 0, 0] == np.float32((1 + 2 * e) / 4)


def test_center_error_bound_on_a_workload():
    """|chi_c - exact weighted mean| <= (ceil(log2 n) + 1) * 2^-24 * max|p| (pairwise sum + divide)."""
    w = W.get_workload("room")
    P = w.points(B=2)
    L = w.layers[0]
    t, cl, mv, q = oracle.run_layer(P, L)
    for b in range(2):
        idx = q["node_idx"][b]
        n = q["n_valid"][b]
        for j in range(0, L.M, 7):
            pts = P[b, idx[j, :n[j]]].astype(np.float64)
            exact = pts.mean(0)
            bound = (math.ceil(math.log2(max(n[j], 2))) + 1) * 2.0 ** -24 * np.abs(pts).max()
            assert np.all(np.abs(q["center_xyz"][b, j] - exact) <= bound)
            lo, hi = pts.min(0), pts.max(0)
            assert np.all(q["center_xyz"][b, j] >= np.nextafter(lo.astype(np.float32), -np.inf))
            assert np.all(q["center_xyz"][b, j] <= np.nextafter(hi.astype(np.float32), np.inf))


def test_query_rejects_unoccupied_center():
    t = _small_table(0)
    occupied = set(int(x) for x in t.vox_lin[0, :t.nvox[0]])
    empty = next(l for l in range(6 * 6 * 3) if l not in occupied)
    with pytest.raises(oracle.OracleError, match="-7"):
        t.query(np.array([[empty]], np.int32), np.array([1], np.int32), 4, "cube", 0)


# ---------------------------------------------------------------- upsampling query

def _upsampling_centers(P, gs, n, seed):
    """Center points of three kinds: points of the cloud, uniform points in
    the grid's box, and points just outside it (clamped onto border voxels)."""
    rng = np.random.default_rng(seed)
    lo = np.asarray(gs.origin, np.float64)
    hi = lo + np.asarray(gs.voxel_size, np.float64) * np.asarray(gs.dims)
    own = P[rng.integers(0, P.shape[0], n // 3)]
    box = rng.uniform(lo, hi, (n // 3, 3))
    out = rng.uniform(lo - 0.3, hi + 0.3, (n - 2 * (n // 3), 3))
    return np.concatenate([own, box, out]).astype(np.float32)


@pytest.mark.parametrize("n_v", [32, 3])
def test_query_points_knn_matches_bruteforce(n_v):
    """Sec. 3.1 upsampling: the nodes of a given center point are its K
    nearest stored points of the block around the voxel it falls in, the
    distance measured from the point itself (numpy lexsort on (i, d^2) in
    the same fp32 order); an empty block gives n = 0 and -1 everywhere."""
    w = W.get_workload("room")
    P = w.points(B=1)
    gs = w.layers[0].grid
    grid = oracle.make_grid(gs.origin, gs.voxel_size, gs.dims, n_v, 1)
    t = oracle.Table(P, grid)
    Q = _upsampling_centers(P[0], gs, 300, 3)[None]
    K = 16
    q = t.query_points(Q, K, "knn", 0)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, n_v)
    qlin = oracle.voxelize(Q, grid)[0]
    empty = 0
    for j in range(Q.shape[1]):
        assert q["center_lin"][0, j] == qlin[j]
        ctx = _context_bruteforce(P[0], lin, tb, int(qlin[j]), gs.dims, 1)
        assert q["ctx_count"][0, j] == len(ctx)
        d = P[0, ctx] - Q[0, j]
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        order = np.lexsort((ctx, d2.view(np.uint32)))
        n = min(K, len(ctx))
        assert q["n_valid"][0, j] == n
        if n == 0:
            empty += 1
            assert np.all(q["node_idx"][0, j] == -1) and np.all(q["node_xyz"][0, j] == 0)
            continue
        assert list(q["node_idx"][0, j, :n]) == list(ctx[order[:n]])
        assert np.all(q["node_idx"][0, j, n:] == q["node_idx"][0, j, 0])
        assert np.array_equal(q["node_xyz"][0, j].view(np.uint32), P[0, q["node_idx"][0, j]].view(np.uint32))
    assert 0 < empty < Q.shape[1] // 2


def test_query_points_equals_global_knn_when_the_block_suffices():
    """The block around a center point reaches at least r voxel edges past
    it on every side: when the K-th nearest of all N points is closer than
    that and the cap never binds, the upsampling k-NN is the ordinary k-NN."""
    P = W.uniform_cube(1, 4000, 23)
    size = 0.1
    grid = oracle.make_grid((0, 0, 0), (size,) * 3, (10, 10, 10), 64, 1)
    t = oracle.Table(P, grid)
    assert t.vox_count.max() <= 64
    Q = np.random.default_rng(8).random((1, 300, 3)).astype(np.float32)
    K = 8
    q = t.query_points(Q, K, "knn", 0)
    checked = 0
    for j in range(300):
        d = np.sqrt(((P[0].astype(np.float64) - Q[0, j]) ** 2).sum(1))
        order = np.argsort(d, kind="stable")
        if d[order[K - 1]] < size - 1e-3 and d[order[K]] - d[order[K - 1]] > 1e-5:
            assert set(q["node_idx"][0, j]) == set(order[:K])
            checked += 1
    assert checked > 100


def test_query_points_cube_is_a_subset_of_the_block_and_depends_on_the_voxel():
    """Cube Query around a given point: distinct context points, the whole
    context when c <= K; two points in one voxel get the same nodes."""
    w = W.get_workload("room")
    P = w.points(B=1)
    gs = w.layers[0].grid
    grid = oracle.grid_from_spec(gs)
    t = oracle.Table(P, grid)
    Q = _upsampling_centers(P[0], gs, 200, 4)[None]
    Q2 = Q.copy()
    # a second point in the same voxel: the lower corner's side of the first
    g = pins.grid_coords_f64(Q[0], gs.origin, gs.voxel_size, gs.dims)
    inner = np.all((Q[0] - gs.origin) / gs.voxel_size - g > 0.05, axis=1) & np.all(
        (Q[0] - gs.origin) / gs.voxel_size - g < 0.95, axis=1)
    Q2[0, inner] = (np.asarray(gs.origin) + (g[inner] + 0.5) * np.asarray(gs.voxel_size)).astype(np.float32)
    K = 8
    a = t.query_points(Q, K, "cube", 5)
    b = t.query_points(Q2, K, "cube", 5)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, gs.n_v)
    for j in range(200):
        ctx = set(_context_bruteforce(P[0], lin, tb, int(a["center_lin"][0, j]), gs.dims, 1))
        n = min(K, len(ctx))
        got = list(a["node_idx"][0, j, :n])
        assert len(set(got)) == n and set(got) <= ctx
        if len(ctx) <= K:
            assert set(got) == ctx
        if inner[j]:
            assert b["center_lin"][0, j] == a["center_lin"][0, j]
            assert list(b["node_idx"][0, j]) == list(a["node_idx"][0, j])


def test_query_points_nonfinite_center_is_an_error():
    t = _small_table(0)
    Q = np.array([[[np.nan, 0.1, 0.1]]], np.float32)
    with pytest.raises(oracle.OracleError, match="-4"):
        t.query_points(Q, 4, "knn", 0)
    q = t.query_points(Q, 4, "knn", 0, allow_nonfinite=True)
    assert q["center_lin"][0, 0] % t.grid.dims[0] == 0


# ---------------------------------------------------------------- context lists

@pytest.mark.parametrize("n_v", [32, 3])
def test_context_list_matches_block_enumeration(n_v):
    """Sec. 3.3 grid context pooling reads every context point: per center,
    the stored points of the occupied voxels of the block, ordered by
    (voxel lin, point index) -- a numpy enumeration over all points -- and
    concatenated with CSR offsets over the batch. Unoccupied center voxels
    have a context too."""
    w = W.get_workload("room")
    P = w.points(B=2)
    gs = w.layers[0].grid
    grid = oracle.make_grid(gs.origin, gs.voxel_size, gs.dims, n_v, 1)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(120, 6)
    rng = np.random.default_rng(1)
    V = int(np.prod(gs.dims))
    cl = np.concatenate([cl, rng.integers(0, V, (2, 40)).astype(np.int32)], axis=1)
    off, idx = t.context_list(cl)
    assert off[0] == 0 and np.all(np.diff(off) >= 0) and off[-1] == len(idx)
    M = cl.shape[1]
    for b in range(2):
        lin = oracle.voxelize(P[b], grid)
        tb = pins.table_numpy(lin, n_v)
        for j in range(M):
            ctx = _context_bruteforce(P[b], lin, tb, int(cl[b, j]), gs.dims, 1)
            ctx = ctx[np.lexsort((ctx, lin[ctx]))]
            k = b * M + j
            assert list(idx[off[k]:off[k + 1]]) == list(ctx)


def test_context_list_counts_equal_the_query_context_counts():
    w = W.get_workload("object")
    L = w.layers[0]
    t = oracle.Table(w.points()[:4], oracle.grid_from_spec(L.grid))
    cl, mv = t.sample_rvs(L.M, 2)
    q = t.query(cl, mv, L.K, "knn", 0)
    off, _ = t.context_list(cl)
    assert np.array_equal(np.diff(off).reshape(cl.shape), q["ctx_count"])


def test_context_list_rejects_a_lin_outside_the_grid():
    t = _small_table(0)
    with pytest.raises(oracle.OracleError, match="-7"):
        t.context_list(np.array([[6 * 6 * 3]], np.int32))


# ---------------------------------------------------------------- level-wise k-NN (Appendix D)

def _ring_table():
    """Voxels of edge 1, center voxel (2,2,2). Points by index: 0 E in
    (2,3,2), 1 A at the center voxel's far corner, 2 C just past its +x face,
    3 B inside it, 4 D just past its -x face. Distances from the voxel center
    (2.5,2.5,2.5): A 0.779, B 0.4, C 0.55, D 0.6, E 1.1."""
    P = np.array([[[2.5, 3.6, 2.5], [2.95, 2.95, 2.95], [3.05, 2.5, 2.5], [2.5, 2.5, 2.9],
                   [1.9, 2.5, 2.5]]], np.float32)
    t = oracle.Table(P, oracle.make_grid((0, 0, 0), (1, 1, 1), (5, 5, 5), 8, 1))
    return t, np.array([[2 + 5 * (2 + 5 * 2)]], np.int32), np.array([1], np.int32)


@pytest.mark.parametrize("K,nodes", [
    (1, [3]),                # level 0 holds 2 > K: its nearest, B
    (2, [1, 3]),             # level 0 fits exactly: appended as gathered (A, B)
    (3, [1, 3, 2]),          # then the nearest of level 1: C
    (5, [1, 3, 4, 2, 0]),    # level 1 fits: gathered by voxel lin (D, C, E)
    (6, [1, 3, 4, 2, 0, 1]),  # c = 5 < K: slots past n repeat slot 0
])
def test_knn_ring_hand_worked(K, nodes):
    """The level-wise k-NN of Appendix D, worked by hand on five points.
    K = 2 shows the paper's early-exit claim failing: C (0.55) is nearer
    than A (0.78), yet the whole of level 0 is taken first."""
    t, cl, mv = _ring_table()
    q = t.query(cl, mv, K, "knn_ring", 0)
    assert list(q["node_idx"][0, 0]) == nodes
    assert q["n_valid"][0, 0] == min(K, 5)
    exact = t.query(cl, mv, K, "knn", 0)
    if K == 2:
        assert list(exact["node_idx"][0, 0]) == [3, 2]


def test_knn_ring_is_the_center_voxels_knn_when_it_holds_k_points():
    """When the center voxel stores at least K points, level 0 alone is
    searched: the result is the ordinary K nearest of its stored points."""
    rng = np.random.default_rng(2)
    P = (rng.random((1, 3000, 3)) * np.float32(0.5)).astype(np.float32)
    grid = oracle.make_grid((0, 0, 0), (0.125,) * 3, (4, 4, 4), 64, 1)
    t = oracle.Table(P, grid)
    nv = int(t.nvox[0])
    cl = t.vox_lin[:, :nv].astype(np.int32)
    K = 16
    q = t.query(cl, np.array([nv], np.int32), K, "knn_ring", 0)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, 64)
    checked = 0
    for j in range(nv):
        s = int(np.searchsorted(tb["vox_lin"], cl[0, j]))
        own = tb["pt_list"][tb["vox_off"][s]:tb["vox_off"][s + 1]]
        if len(own) < K:
            continue
        g = np.array(pins.decode(int(cl[0, j]), (4, 4, 4)), np.float32)
        c = (g + np.float32(0.5)) * np.float32(0.125)
        d = P[0, own] - c
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        order = np.lexsort((own, d2.view(np.uint32)))
        assert list(q["node_idx"][0, j]) == list(own[order[:K]])
        checked += 1
    assert checked >= 4


def test_knn_ring_takes_the_whole_context_in_level_order_when_it_fits():
    """c <= K: every context point, levels ascending, each level in gathering
    order (voxel lin, then point index) -- a numpy sort of the block."""
    w = W.get_workload("room")
    P = w.points(B=1)
    gs = w.layers[0].grid
    grid = oracle.make_grid(gs.origin, gs.voxel_size, gs.dims, 4, 2)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(300, 3)
    K = 64
    q = t.query(cl, mv, K, "knn_ring", 0)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, 4)
    g_all = np.stack([lin % gs.dims[0], (lin // gs.dims[0]) % gs.dims[1], lin // (gs.dims[0] * gs.dims[1])], -1)
    checked = 0
    for j in range(300):
        ctx = _context_bruteforce(P[0], lin, tb, int(cl[0, j]), gs.dims, 2)
        if len(ctx) > K:
            continue
        gc = np.array(pins.decode(int(cl[0, j]), gs.dims))
        level = np.abs(g_all[ctx] - gc).max(axis=1)
        order = np.lexsort((ctx, lin[ctx], level))
        assert list(q["node_idx"][0, j, :len(ctx)]) == list(ctx[order])
        checked += 1
    assert checked > 50


def test_knn_ring_levels_before_the_last_are_whole_and_the_last_is_nearest_first():
    """On a workload: the chosen nodes take every point of the levels before
    the last level used, and from that level the nearest by (d^2, index)."""
    w = W.get_workload("room")
    P = w.points(B=1)
    gs = w.layers[0].grid
    grid = oracle.grid_from_spec(gs)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(400, 9)
    K = 32
    q = t.query(cl, mv, K, "knn_ring", 0)
    lin = oracle.voxelize(P, grid)[0]
    tb = pins.table_numpy(lin, gs.n_v)
    g_all = np.stack([lin % gs.dims[0], (lin // gs.dims[0]) % gs.dims[1], lin // (gs.dims[0] * gs.dims[1])], -1)
    o, s = np.float32(gs.origin), np.float32(gs.voxel_size)
    partial = 0
    for j in range(400):
        ctx = _context_bruteforce(P[0], lin, tb, int(cl[0, j]), gs.dims, 1)
        gc = np.array(pins.decode(int(cl[0, j]), gs.dims))
        level = np.abs(g_all[ctx] - gc).max(axis=1)
        n = int(q["n_valid"][0, j])
        got = q["node_idx"][0, j, :n]
        assert n == min(K, len(ctx)) and len(set(got)) == n and set(got) <= set(ctx)
        lv = dict(zip(ctx, level))
        last = max(lv[i] for i in got)
        for i, l in zip(ctx, level):
            if l < last:
                assert i in set(got)
        inlast = ctx[level == last]
        if len(inlast) > sum(1 for i in got if lv[i] == last):
            partial += 1
            c = o + (gc.astype(np.float32) + np.float32(0.5)) * s
            d = P[0, inlast] - c
            d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
            take = sum(1 for i in got if lv[i] == last)
            best = inlast[np.lexsort((inlast, d2.view(np.uint32)))[:take]]
            assert list(got[n - take:]) == list(best)
    assert partial > 20


# ---------------------------------------------------------------- comparison methods and coverage (Sec. 4)

def test_rps_is_the_m_smallest_keys_in_index_order():
    P = W.uniform_cube(2, 700, 3)
    c = oracle.sample_points(P, 90, "rps", 17)
    for b in range(2):
        keys = [((pins.py_chain(17, 4, b, i) >> 32) << 32) | i for i in range(700)]
        assert list(c[b]) == sorted(int(k & 0xFFFFFFFF) for k in sorted(keys)[:90])


def _fps_numpy(P, M):
    """Farthest point sampling in numpy fp32, from point 0."""
    d = np.full(P.shape[0], np.inf, np.float32)
    out, cur = [], 0
    for _ in range(M):
        out.append(cur)
        v = P - P[cur]
        d2 = (v[:, 0] * v[:, 0] + v[:, 1] * v[:, 1]) + v[:, 2] * v[:, 2]
        d = np.minimum(d, d2)
        cur = int(np.argmax(d))  # first maximum: ties to the lowest index
    return out


def test_fps_matches_numpy_farthest_point_sampling():
    P = W.uniform_cube(2, 600, 8)
    P[1, 100:140] = P[1, 0]  # duplicates: ties and zero distances
    c = oracle.sample_points(P, 120, "fps", 0)
    for b in range(2):
        assert list(c[b]) == _fps_numpy(P[b], 120)


def test_fps_picks_are_farthest_and_spread_shrinks():
    """Each pick maximises the distance to the chosen set, so the sequence of
    pick distances never increases (Gonzalez's 2-approximation property)."""
    P = W.get_workload("object").points()[:1]
    c = oracle.sample_points(P, 64, "fps", 0)[0]
    X = P[0].astype(np.float64)
    prev = np.inf
    for j in range(1, 64):
        dj = np.min(((X[c[:j]] - X[c[j]]) ** 2).sum(1))
        dall = np.min(((X[c[:j], None, :] - X[None, :, :]) ** 2).sum(-1), axis=0).max()
        assert dj <= prev + 1e-9 and abs(dj - dall) <= 1e-6 * max(1.0, dall)
        prev = dj


def test_ball_query_is_the_first_k_inside_the_radius():
    P = W.get_workload("room").points(B=1)
    c = oracle.sample_points(P, 200, "rps", 1)
    r2 = np.float32(0.186) ** 2
    K = 16
    ni, nv = oracle.ball_query(P, c, K, float(r2))
    for j in range(200):
        v = P[0] - P[0, c[0, j]]
        d2 = (v[:, 0] * v[:, 0] + v[:, 1] * v[:, 1]) + v[:, 2] * v[:, 2]
        inside = np.nonzero(d2 < r2)[0][:K]
        n = len(inside)
        assert nv[0, j] == n >= 1
        assert list(ni[0, j, :n]) == list(inside) and np.all(ni[0, j, n:] == inside[0])


def test_coverage_is_the_share_of_occupied_voxels_holding_a_node():
    w = W.get_workload("room")
    P = w.points(B=2)
    grid = oracle.grid_from_spec(w.layers[0].grid)
    t = oracle.Table(P, grid)
    cl, mv = t.sample_rvs(300, 2)
    q = t.query(cl, mv, 16, "cube", 2)
    cov = t.coverage(q["node_idx"], q["n_valid"])
    lin = oracle.voxelize(P, grid)
    for b in range(2):
        nodes = np.concatenate([q["node_idx"][b, j, :q["n_valid"][b, j]] for j in range(300)])
        assert cov[b] == len(np.unique(lin[b, nodes]))
        assert t.nvox[b] == len(np.unique(lin[b]))


@pytest.mark.parametrize("name", ["object", "room"])
def test_cas_covers_more_than_rvs(name):
    """Sec. 4: CAS leads the occupied-space coverage (beta = 0), as in every
    row of the paper's latency/coverage tables."""
    w = W.get_workload(name)
    L = w.layers[0]
    P = w.points()[:4]
    t = oracle.Table(P, oracle.grid_from_spec(L.grid))
    M = max(8, int(t.nvox.min()) // 8)
    cas, mc, _, _ = t.sample_cas(M)
    rvs, mr = t.sample_rvs(M, 3)
    a = t.query(cas, mc, L.K, "cube", 0)
    b = t.query(rvs, mr, L.K, "cube", 0)
    assert np.all(t.coverage(a["node_idx"], a["n_valid"]) > t.coverage(b["node_idx"], b["n_valid"]))
