"""HIP path vs the CPU oracle, element by element, bit-exact.

Every integer output (slots, counts, offsets, lists, centers, node indices,
counts of valid nodes, weights) must be equal; every float output (node
coordinates, group centers) must have the same bit pattern. Inputs are the
seeded synthetic workloads at their full sizes plus hand-built edge cases.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1912_02984_amd import cagq
from paper_1912_02984_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _np(t):
    return t.detach().cpu().numpy()


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


def assert_table(g, ot, where=""):
    tb = {k: _np(v) for k, v in g.table().items()}
    assert np.array_equal(tb["nvox"], ot.nvox), where
    for b in range(ot.B):
        nv = int(ot.nvox[b])
        S = int(ot.vox_off[b, nv])
        assert np.array_equal(_bits(tb["vox_lin"][b, :nv]), ot.vox_lin[b, :nv]), (where, b)
        assert np.array_equal(_bits(tb["vox_count"][b, :nv]), ot.vox_count[b, :nv]), (where, b)
        assert np.array_equal(_bits(tb["vox_off"][b, :nv + 1]), ot.vox_off[b, :nv + 1]), (where, b)
        assert np.array_equal(_bits(tb["pt_list"][b, :S]), ot.pt_list[b, :S]), (where, b)


def assert_query(qg, qo, where=""):
    assert np.array_equal(_np(qg["node_idx"]), qo["node_idx"]), where
    assert np.array_equal(_np(qg["n_valid"]), qo["n_valid"]), where
    assert np.array_equal(_bits(_np(qg["center_w"])), qo["center_w"]), where
    assert np.array_equal(_bits(_np(qg["center_xyz"])), _bits(qo["center_xyz"])), where
    if qg.get("node_xyz") is not None:
        assert np.array_equal(_bits(_np(qg["node_xyz"])), _bits(qo["node_xyz"])), where
    if qg.get("ctx_count") is not None:
        assert np.array_equal(_np(qg["ctx_count"]), qo["ctx_count"]), where


def run_both(P, grid_spec, M, K, sample, query, seed, weights=None, beta_q16=0, where=""):
    """One layer on both sides from the same float32 input; checks every output."""
    P = np.ascontiguousarray(P, np.float32)
    ot = oracle.Table(P, oracle.grid_from_spec(grid_spec))
    if sample == "rvs":
        ocl, omv = ot.sample_rvs(M, seed)
    elif sample == "cas_swap":
        ocl, omv, _, _ = ot.sample_cas_swap(M, seed, beta_q16)
    else:
        ocl, omv, _, _ = ot.sample_cas(M, beta_q16)
    qo = ot.query(ocl, omv, K, query, seed, weights=weights)

    Pt = torch.from_numpy(P).to(DEV)
    Wt = None if weights is None else torch.from_numpy(weights.astype(np.uint32).view(np.int32)).to(DEV)
    g = cagq.build_grid(Pt, cagq.desc_from_spec(grid_spec))
    cl, mv = cagq.sample_centers(g, M, sample, seed, beta_q16)
    qg = cagq.query_context(g, cl, K, query, seed, weights=Wt)
    assert cagq.get_device_status(g) == 0, where
    assert_table(g, ot, where)
    assert np.array_equal(_np(mv), omv), where
    assert np.array_equal(_np(cl), ocl), where
    assert_query(qg, qo, where)
    return qo


@pytest.mark.parametrize("sample", ["rvs", "cas"])
@pytest.mark.parametrize("query", ["cube", "knn"])
def test_tiny_all_modes(sample, query):
    w = W.get_workload("tiny")
    L = w.layers[0]
    run_both(w.points(), L.grid, L.M, L.K, sample, query, L.seed, where=f"tiny {sample} {query}")


@pytest.mark.parametrize("name", ["tiny", "object", "room", "bigroom/cas-knn", "bigroom/rvs-cube", "lidar"])
def test_workload_full_size(name):
    """Every layer of the workload at its full size, chained through the
    centers and weights each side produced."""
    w = W.get_workload(name)
    P = w.points()
    weights = None
    for li, L in enumerate(w.layers):
        print(f"[parity] {name} layer {li}: B={P.shape[0]} N={P.shape[1]} M={L.M} K={L.K} "
              f"{L.sample}+{L.query}", flush=True)
        qo = run_both(P, L.grid, L.M, L.K, L.sample, L.query, L.seed, weights=weights,
                      where=f"{name} L{li}")
        P, weights = qo["center_xyz"], qo["center_w"]


def _spec(origin, size, dims, n_v, r=1):
    return W.GridSpec(tuple(origin), tuple(size), tuple(dims), n_v, r)


@pytest.mark.parametrize("N", [5000, 12000])
def test_capped_and_big_voxels(N):
    """Voxels holding up to a few hundred points: the cap keeps the lowest
    indices, through both the per-point ranking and the wave selection, in
    the one-workgroup build (5000 points) and the brick build (12000: one
    brick of 12000 points per cloud, built by six parts that meet in
    memory)."""
    rng = np.random.default_rng(5)
    B = 3
    P = rng.random((B, N, 3), dtype=np.float32)
    # a third of each cloud crowds into three voxels
    P[:, : N // 3] = (np.float32(0.01) + rng.random((B, N // 3, 3), dtype=np.float32) * np.float32(0.02))
    P[:, N // 3: N // 3 + 200] = np.float32(0.55)
    spec = _spec((0, 0, 0), (0.125,) * 3, (8, 8, 8), 16)
    for n_v in (1, 4, 16, 64):
        s = _spec((0, 0, 0), (0.125,) * 3, (8, 8, 8), n_v)
        run_both(P, s, 40, 32, "rvs", "knn", 3, where=f"n_v={n_v}")
    run_both(P, spec, 12, 64, "cas", "cube", 9, where="cas")


@pytest.mark.parametrize("case", ["brick-capacity", "ragged-bricks", "wide-bricks", "scan-launch",
                                  "grid-too-large-for-bricks"])
def test_brick_build_edges(case):
    """The brick build of larger clouds: bricks of 2048 consecutive voxels
    holding exactly the 2048 points one work item takes and one more (then
    split into two parts that meet in memory), voxels of more than 64 points
    in both, a last brick cut short by the grid; 1280 bricks per cloud (the
    scatter tiles scan the bricks' totals in two passes); clouds whose tiles
    times bricks exceed 2^16 (the histogram columns are scanned by a launch
    of their own), with a brick of 3000 points and tiles holding points of
    two clouds; and a grid with more bricks than the build holds, which
    takes the seven-kernel build."""
    rng = np.random.default_rng(11)
    if case == "brick-capacity":
        # 64 x 32 voxels per z-slice: brick q is slice z = q
        B, N, dims, n_v = 2, 10000, (64, 32, 64), 16
        P = rng.random((B, N, 3), dtype=np.float32) * np.float32([6.4, 3.2, 6.4])
        P[:, 4197:, 2] = np.float32(0.3) + rng.random((B, N - 4197), dtype=np.float32) * np.float32(6.0)
        P[:, :1948, 2] = np.float32(0.05)                 # brick 0: 1948 spread points
        P[:, 1948:2048] = np.float32([0.33, 0.47, 0.05])  # and 100 in one voxel: 2048
        P[:, 2048:3997, 2] = np.float32(0.15)             # brick 1: 1949 spread points
        P[:, 3997:4097] = np.float32([0.33, 0.47, 0.15])  # and 100 in one voxel: 2049
        P[:, 4097:4197] = np.float32([0.33, 0.47, 0.25])  # 100 in one voxel of brick 2
        P = P[:, rng.permutation(N)]
        spec = _spec((0, 0, 0), (0.1,) * 3, dims, n_v)
    elif case == "ragged-bricks":
        B, N, dims, n_v = 3, 9000, (70, 33, 50), 8
        P = rng.random((B, N, 3), dtype=np.float32) * np.float32([7.0, 3.3, 5.0])
        P[:, :300] = np.float32([6.95, 3.25, 4.95])      # the grid's last voxel
        spec = _spec((0, 0, 0), (0.1,) * 3, dims, n_v)
    elif case == "wide-bricks":
        B, N, dims, n_v = 1, 20000, (256, 256, 40), 8
        P = rng.random((B, N, 3), dtype=np.float32) * np.float32([2.56, 2.56, 0.4])
        spec = _spec((0, 0, 0), (0.01,) * 3, dims, n_v)
    elif case == "scan-launch":
        # (ceil(N / 4096) + 1) * Q = 26 * 2560 > 2^16
        B, N, dims, n_v = 2, 100000, (256, 256, 80), 8
        P = rng.random((B, N, 3), dtype=np.float32) * np.float32([2.56, 2.56, 0.8])
        # brick 0 (x < 2.56, y < 0.08, z < 0.01): 3000 points, two work items
        P[:, :3000] = rng.random((B, 3000, 3), dtype=np.float32) * np.float32([2.55, 0.079, 0.0099])
        P = P[:, rng.permutation(N)]
        spec = _spec((0, 0, 0), (0.01,) * 3, dims, n_v)
    else:
        B, N, dims, n_v = 2, 9000, (512, 512, 128), 4
        P = rng.random((B, N, 3), dtype=np.float32) * np.float32([5.12, 5.12, 1.28])
        P[:, :500] = np.float32([0.001, 0.001, 0.001])
        spec = _spec((0, 0, 0), (0.01,) * 3, dims, n_v)
    print(f"[parity] brick build {case}: B={B} N={N} dims={dims} n_v={n_v}", flush=True)
    run_both(P, spec, 300, 32, "rvs", "knn", 4, where=case)
    run_both(P, spec, 300, 16, "rvs", "cube", 5, where=case + " cube")


def test_all_points_in_one_voxel():
    P = np.full((2, 777, 3), 0.3, np.float32)
    P[1] += np.linspace(0, 0.01, 777, dtype=np.float32)[:, None]
    run_both(P, _spec((0, 0, 0), (1.0,) * 3, (4, 4, 4), 64), 5, 64, "rvs", "knn", 1, where="one voxel")
    run_both(P, _spec((0, 0, 0), (1.0,) * 3, (4, 4, 4), 3), 5, 8, "cas", "cube", 1, where="one voxel cas")


@pytest.mark.parametrize("nvox", [1023, 1024, 1025, 2048, 3072])
def test_slot_count_at_scan_tile_edges(nvox):
    """Occupied-voxel counts on both sides of the scan tile size."""
    rng = np.random.default_rng(nvox)
    dims = (64, 64, 4)
    lin = rng.choice(64 * 64 * 4, size=nvox, replace=False)
    g = np.stack([lin % 64, (lin // 64) % 64, lin // 4096], 1).astype(np.float32)
    P = ((g + np.float32(0.5)) * np.float32(0.1))[None]
    extra = P[:, rng.integers(0, nvox, size=500)] + np.float32(0.01)
    P = np.concatenate([P, extra], axis=1)[:, rng.permutation(nvox + 500)]
    run_both(P, _spec((0, 0, 0), (0.1,) * 3, dims, 4), 300, 16, "rvs", "cube", 2, where=f"nvox={nvox}")


def test_ragged_batch_and_clamping():
    """B*N not a multiple of the block size; points outside the grid and on
    voxel faces are clamped, not dropped."""
    rng = np.random.default_rng(11)
    B, N = 3, 1001
    P = (rng.random((B, N, 3), dtype=np.float32) * np.float32(3.0) - np.float32(1.0))
    P[0, :50] = np.float32(0.25) * rng.integers(0, 5, size=(50, 3)).astype(np.float32)  # exact faces
    spec = _spec((0, 0, 0), (0.25,) * 3, (4, 5, 6), 8)
    run_both(P, spec, 17, 8, "rvs", "knn", 4, where="ragged rvs")
    run_both(P, spec, 17, 8, "cas", "knn", 4, where="ragged cas")


def test_more_centers_than_occupied_voxels():
    rng = np.random.default_rng(2)
    P = rng.random((2, 50, 3), dtype=np.float32) * np.float32(0.5)
    spec = _spec((0, 0, 0), (0.25,) * 3, (2, 2, 2), 8)
    run_both(P, spec, 20, 16, "rvs", "knn", 7, where="M>nvox rvs")
    run_both(P, spec, 20, 16, "cas", "cube", 7, where="M>nvox cas")


@pytest.mark.parametrize("K", [1, 2, 16, 17, 24, 31, 32, 33, 64, 65, 96, 128])
def test_node_counts(K):
    w = W.get_workload("room")
    L = w.layers[0]
    P = w.points(B=2)
    run_both(P, L.grid, 256, K, "rvs", "knn", 5, where=f"K={K} knn")
    run_both(P, L.grid, 256, K, "rvs", "cube", 5, where=f"K={K} cube")


@pytest.mark.parametrize("r", [2, 3])
def test_wider_neighbourhoods(r):
    w = W.get_workload("room")
    L = w.layers[0]
    spec = _spec(L.grid.origin, L.grid.voxel_size, L.grid.dims, 16, r)
    P = w.points(B=2)
    run_both(P, spec, 300, 32, "rvs", "knn", 8, where=f"r={r} knn")
    run_both(P, spec, 300, 32, "rvs", "cube", 8, where=f"r={r} cube")
    if r == 2:
        run_both(P, spec, 300, 32, "cas", "knn", 8, where=f"r={r} cas")


@pytest.mark.parametrize("N,dims", [(1024, (10, 10, 10)), (1025, (40, 40, 20)), (700, (48, 48, 24)),
                                    (4096, (96, 96, 40)), (4097, (32, 32, 16)), (3000, (16, 16, 16)),
                                    (4096, (12, 12, 12)), (8192, (16, 16, 16))])
def test_cas_single_workgroup_limits(N, dims):
    """CAS with beta = 0 runs in one workgroup per cloud up to N = 4096 and in
    the many-kernel rounds (with neighbour lists for r = 1) beyond: clouds on
    both sides of the limit, small ones, one whose every voxel is chosen (M >= nvox, so
    the best unpicked key ends at 0), and dense grids whose voxels have full
    neighbour lists, with r = 1 and r = 2."""
    rng = np.random.default_rng(N + dims[2])
    P = rng.random((2, N, 3), dtype=np.float32) * np.float32(0.999)
    P[1, : N // 2] *= np.float32(0.3)  # a denser half in the second cloud
    spec = _spec((0, 0, 0), tuple(1.0 / d for d in dims), dims, 8)
    M = 5000 if dims == (16, 16, 16) and N in (3000, 8192) else 1500  # M above the occupied voxels
    run_both(P, spec, M, 8, "cas", "knn", 0, where=f"N={N} dims={dims}")
    if dims in ((16, 16, 16), (12, 12, 12), (10, 10, 10), (48, 48, 24)):
        spec2 = _spec((0, 0, 0), tuple(1.0 / d for d in dims), dims, 8, 2)
        run_both(P, spec2, 700, 8, "cas", "knn", 0, where=f"N={N} dims={dims} r=2")


@pytest.mark.parametrize("name", ["tiny", "object", "room"])
def test_cas_swap_workloads(name):
    """The paper's challenger / incumbent CAS on the small workloads, each
    layer fed by the previous one's centers."""
    w = W.get_workload(name)
    P = w.points()[:4]
    wts = None
    for li, L in enumerate(w.layers):
        qo = run_both(P, L.grid, L.M, L.K, "cas_swap", L.query, L.seed, weights=wts, where=f"{name} L{li}")
        P, wts = qo["center_xyz"], qo["center_w"]


@pytest.mark.parametrize("r,beta_q16", [(1, 65536 // 4), (2, 0), (3, 0)])
def test_cas_swap_radius_and_penalty(r, beta_q16):
    rng = np.random.default_rng(r)
    P = rng.random((2, 1500, 3), dtype=np.float32) * np.float32(0.999)
    spec = _spec((0, 0, 0), (1 / 16,) * 3, (16, 16, 16), 8, r)
    run_both(P, spec, 100, 8, "cas_swap", "cube", 11, beta_q16=beta_q16, where=f"r={r} beta={beta_q16}")


@pytest.mark.parametrize("beta_q16", [0, 65536 // 4])
def test_cas_swap_at_bench_size(beta_q16):
    """CAS-P where the bench times it: one full indoor scene of 81920 points,
    M = 8192, r = 1 (about 125 KB of one workgroup's LDS), with and without
    the over-coverage penalty."""
    w = W.get_workload("bigroom/cas-knn")
    L = w.layers[0]
    print(f"[parity] cas_swap N=81920 M={L.M} beta={beta_q16}", flush=True)
    run_both(w.points(B=1), L.grid, L.M, L.K, "cas_swap", "knn", L.seed, beta_q16=beta_q16,
             where=f"cas_swap bench size beta={beta_q16}")


@pytest.mark.parametrize("r,beta_q16,M", [(1, 65536 // 4, 2048), (2, 0, 2048), (2, 0, 20000),
                                           (2, 3 * 65536 // 4, 2048)])
def test_cas_on_large_clouds_with_penalty_or_radius_two(r, beta_q16, M):
    """CAS on 81920-point scenes where neither the single workgroup nor the
    list rounds apply (beta > 0, or r = 2): the row-scan rounds and the
    many-block selection of the pick keys. With beta = 0 the pick keys take
    few values, so the selection's threshold digit holds thousands of ties
    (more than its LDS holds at M = 20000: the keys are read again)."""
    w = W.get_workload("bigroom/cas-knn")
    L = w.layers[0]
    spec = _spec(L.grid.origin, L.grid.voxel_size, L.grid.dims, L.grid.n_v, r)
    print(f"[parity] cas N=81920 r={r} beta={beta_q16} M={M}", flush=True)
    run_both(w.points(B=2), spec, M, 16, "cas", "cube", 5, beta_q16=beta_q16, where=f"r={r} beta={beta_q16} M={M}")


@pytest.mark.parametrize("M", [1, 2, 4095, 4096, 4097, 30000, 60000])
def test_rvs_many_block_selection_bounds(M):
    """The many-block RVS selection (clouds of 16384 points or more) at every
    kind of bound: one center, the block size and its neighbours, most of
    the occupied voxels, and more centers than occupied voxels."""
    w = W.get_workload("bigroom/rvs-cube")
    L = w.layers[0]
    run_both(w.points(B=2), L.grid, M, 8, "rvs", "cube", 11 + M, where=f"M={M}")


@pytest.mark.parametrize("B,N,dims,M", [(1, 600000, (128, 128, 64), 250000),
                                        (2, 300000, (100, 100, 50), 90000),
                                        (3, 40000, (64, 64, 32), 20000)])
def test_rvs_many_block_selection_large_clouds(B, N, dims, M):
    """The many-block RVS select on larger and more clouds than the indoor
    scenes: m = 250K of ~457K occupied voxels (a bound digit holding many
    keys), 90K of ~226K in each of two clouds, 20K of ~34K in each of
    three."""
    rng = np.random.default_rng(N + M)
    P = rng.random((B, N, 3), dtype=np.float32) * np.float32(0.999)
    spec = _spec((0, 0, 0), tuple(1.0 / d for d in dims), dims, 4)
    print(f"[parity] rvs many-block B={B} N={N} M={M}", flush=True)
    run_both(P, spec, M, 4, "rvs", "cube", 17, where=f"B={B} N={N} M={M}")


def test_rvs_many_block_selection_dense_cloud():
    """A dense cloud (about 140K of 262K voxels occupied): M from one center
    to beyond the occupied voxels."""
    rng = np.random.default_rng(31)
    P = rng.random((1, 200000, 3), dtype=np.float32)
    spec = _spec((0, 0, 0), (1 / 64,) * 3, (64, 64, 64), 4)
    for M in (1, 100000, 150000, 262143, 262144, 262145):
        run_both(P, spec, M, 4, "rvs", "cube", M, where=f"dense M={M}")


def test_back_to_back_cas_calls():
    """Two CAS calls in a row from one thread, each on its own stream and
    workspace, without waiting in between: the first (81920 points, M = 8192)
    returns while some of its rounds may still be queued, the second (M = 4)
    must neither be paced by them nor stopped early. Both against the
    oracle."""
    w = W.get_workload("bigroom/cas-knn")
    L = w.layers[0]
    P = w.points(B=2)
    ot = oracle.Table(P, oracle.grid_from_spec(L.grid))
    Pt = torch.from_numpy(P).to(DEV)
    desc = cagq.desc_from_spec(L.grid)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(3):
        with torch.cuda.stream(s1):
            g1 = cagq.build_grid(Pt, desc)
            cl1, mv1 = cagq.sample_centers(g1, L.M, "cas", 0)
        with torch.cuda.stream(s2):
            g2 = cagq.build_grid(Pt, desc)
            cl2, mv2 = cagq.sample_centers(g2, 4, "cas", 0)
        assert cagq.get_device_status(g1, s1) == 0 and cagq.get_device_status(g2, s2) == 0
        for M, cl, mv in ((L.M, cl1, mv1), (4, cl2, mv2)):
            ocl, omv, _, _ = ot.sample_cas(M)
            assert np.array_equal(_np(cl), ocl), (rep, M)
            assert np.array_equal(_np(mv), omv), (rep, M)


def test_cas_swap_more_centers_than_voxels_and_capacity():
    rng = np.random.default_rng(4)
    P = rng.random((2, 60, 3), dtype=np.float32) * np.float32(0.5)
    spec = _spec((0, 0, 0), (0.25,) * 3, (2, 2, 2), 8)
    run_both(P, spec, 20, 8, "cas_swap", "knn", 3, where="M>nvox")
    # a cloud too large for one workgroup's state is refused before anything runs
    big = torch.zeros((1, 200000, 3), device=DEV)
    g = cagq.build_grid(big, cagq.desc_from_spec(_spec((0, 0, 0), (1.0,) * 3, (4, 4, 4), 8)))
    with pytest.raises(cagq.CagqError) as ei:
        cagq.sample_centers(g, 40000, "cas_swap", 0)
    assert ei.value.code == cagq.ERR_CAPACITY


@pytest.mark.parametrize("name", ["object", "room"])
@pytest.mark.parametrize("beta_q16", [1, 65536 // 4, 3 * 65536])
def test_cas_with_overcoverage_penalty(name, beta_q16):
    """beta > 0 on small clouds (the two-kernel rounds over occupancy rows)
    and on 8192-point clouds (the one-kernel rounds on neighbour lists, whose
    key lowering then also subtracts beta per raised count, and the radix
    selection instead of the U histogram)."""
    w = W.get_workload(name)
    L = w.layers[0]
    run_both(w.points()[:2 if name == "room" else 4], L.grid, L.M, L.K, "cas", "knn", 0, beta_q16=beta_q16,
             where=f"{name} beta={beta_q16}")


def test_weighted_centers():
    w = W.get_workload("room")
    L = w.layers[0]
    P = w.points(B=2)
    wts = np.random.default_rng(3).integers(1, 1000, size=P.shape[:2]).astype(np.uint32)
    run_both(P, L.grid, 512, 32, "rvs", "knn", 1, weights=wts, where="weights knn")
    run_both(P, L.grid, 512, 32, "rvs", "cube", 1, weights=wts, where="weights cube")


def _workload_outputs(w, Pt):
    """Every layer of a workload on the GPU, chained through centers and
    weights: the valid part of each table and every sample / query output."""
    res, pts, wts = [], Pt, None
    for L in w.layers:
        g = cagq.build_grid(pts, cagq.desc_from_spec(L.grid))
        cl, mv = cagq.sample_centers(g, L.M, L.sample, L.seed)
        q = cagq.query_context(g, cl, L.K, L.query, L.seed, weights=wts)
        assert cagq.get_device_status(g) == 0
        tb = {k: _np(v) for k, v in g.table().items()}
        res.append(tb["nvox"])
        for b in range(pts.shape[0]):  # entries past nvox / the stored total are unspecified
            nv = int(tb["nvox"][b])
            S = int(tb["vox_off"][b, nv])
            res += [tb["vox_lin"][b, :nv], tb["vox_count"][b, :nv], tb["vox_off"][b, :nv + 1],
                    tb["pt_list"][b, :S]]
        res += [_np(cl), _np(mv)] + [_np(v).copy() for v in q.values() if v is not None]
        pts, wts = q["center_xyz"], q["center_w"]
    return res


@pytest.mark.parametrize("name", ["tiny", "object", "room", "bigroom/cas-knn", "bigroom/rvs-cube", "lidar"])
def test_repeat_runs_are_identical(name):
    """Atomic arrival order never reaches an output: every workload ten times
    at two batch sizes (different grids of blocks, and for the indoor layers
    both the one-workgroup and the many-block build and CAS), each run
    bitwise equal to the first."""
    w = W.get_workload(name)
    for B in sorted({1, min(w.B, 3)}):
        Pt = torch.from_numpy(w.points(B=B)).to(DEV)
        print(f"[determinism] {name} B={B}", flush=True)
        first = _workload_outputs(w, Pt)
        for rep in range(1, 10):
            again = _workload_outputs(w, Pt)
            for i, (a, b) in enumerate(zip(first, again)):
                assert np.array_equal(a, b), (name, B, rep, i)


def test_nonfinite_input_is_reported():
    P = np.random.default_rng(0).random((1, 100, 3), dtype=np.float32)
    P[0, 17, 1] = np.nan
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.make_desc((0, 0, 0), (0.25,) * 3, (4, 4, 4), 8, 1))
    assert cagq.get_device_status(g) == cagq.ERR_NONFINITE_INPUT
    # the oracle reports the same condition
    with pytest.raises(oracle.OracleError, match="-4"):
        oracle.Table(P, oracle.make_grid((0, 0, 0), (0.25,) * 3, (4, 4, 4), 8, 1))


@pytest.mark.parametrize("N", [100, 12000])
def test_build_error_of_a_later_cloud_and_its_clearing(N):
    """A non-finite coordinate in cloud 2 of 3 is reported whichever build
    runs (100 points: the one-workgroup build, which keeps each cloud's code
    in a word of its own; 12000: the brick build), and a build of finite
    points into the same workspace reports none."""
    rng = np.random.default_rng(N)
    P = rng.random((3, N, 3), dtype=np.float32)
    P[2, N // 2, 0] = np.float32(np.inf)
    desc = cagq.make_desc((0, 0, 0), (0.25,) * 3, (4, 4, 4), 8, 1)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), desc)
    assert cagq.get_device_status(g) == cagq.ERR_NONFINITE_INPUT
    P[2, N // 2, 0] = np.float32(0.5)
    g2 = cagq.build_grid(torch.from_numpy(P).to(DEV), desc, workspace=g.workspace)
    assert cagq.get_device_status(g2) == 0
    cl, mv = cagq.sample_centers(g2, 8, "rvs", 1)
    assert cagq.get_device_status(g2) == 0


def test_unoccupied_center_is_reported():
    P = np.random.default_rng(0).random((1, 20, 3), dtype=np.float32) * np.float32(0.2)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.make_desc((0, 0, 0), (0.25,) * 3, (4, 4, 4), 8, 1))
    assert cagq.get_device_status(g) == 0
    cl = torch.tensor([[0, 63]], dtype=torch.int32, device=DEV)  # voxel 63 is empty
    q = cagq.query_context(g, cl, 4, "knn", 0)
    assert cagq.get_device_status(g) == cagq.ERR_CENTER_NOT_OCCUPIED
    assert int(q["n_valid"][0, 0]) > 0 and int(q["n_valid"][0, 1]) == 0
    assert torch.all(q["node_idx"][0, 1] == 0) and torch.all(q["center_xyz"][0, 1] == 0)


# ---------------------------------------------------------------- upsampling query and context lists

def run_up(P, grid_spec, Q, K, mode, seed, where="", context=True):
    """Upsampling query (and the context lists of the centers' voxels) on
    both sides: grid on P [B,N,3], given centers Q [B,M,3]."""
    P = np.ascontiguousarray(P, np.float32)
    Q = np.ascontiguousarray(Q, np.float32)
    ot = oracle.Table(P, oracle.grid_from_spec(grid_spec))
    qo = ot.query_points(Q, K, mode, seed)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.desc_from_spec(grid_spec))
    qg = cagq.query_points(g, torch.from_numpy(Q).to(DEV), K, mode, seed)
    assert cagq.get_device_status(g) == 0, where
    for k in ("node_idx", "n_valid", "ctx_count", "center_lin"):
        assert np.array_equal(_np(qg[k]), qo[k]), (where, k)
    assert np.array_equal(_bits(_np(qg["node_xyz"])), _bits(qo["node_xyz"])), where
    if context:
        assert_context(g, ot, qg["center_lin"], where)
    return qo


def assert_context(g, ot, center_lin, where=""):
    off_o, idx_o = ot.context_list(_np(center_lin))
    off = cagq.context_offsets(g, center_lin)
    idx = cagq.context_list(g, center_lin, off)
    assert cagq.get_device_status(g) == 0, where
    assert np.array_equal(_np(off), off_o), where
    assert np.array_equal(_np(idx)[: len(idx_o)], idx_o), where


@pytest.mark.parametrize("name", ["object", "room", "bigroom/cas-knn"])
def test_query_points_workloads(name):
    """The upsampling step of a segmentation network: the grid holds the
    centers of layer 1, and every input point of layer 0 is a center whose
    nodes are queried among them (K of the layer, both query modes)."""
    w = W.get_workload(name)
    P = w.points()
    # a one-layer workload queries its centers on the same grid
    L0, L1 = w.layers[0], w.layers[min(1, len(w.layers) - 1)]
    t, cl, mv, q = oracle.run_layer(P, L0)
    coarse = q["center_xyz"]
    for mode in ("knn", "cube"):
        print(f"[parity] upsampling {name} {mode}: B={P.shape[0]} N={coarse.shape[1]} M={P.shape[1]} K={L1.K}",
              flush=True)
        run_up(coarse, L1.grid, P, L1.K, mode, 7, where=f"{name} {mode}", context=(mode == "knn"))


@pytest.mark.parametrize("r", [1, 2, 3])
@pytest.mark.parametrize("K", [1, 16, 17, 32, 33, 64, 65, 128])
def test_query_points_radius_and_node_counts(r, K):
    """Centers of three kinds (cloud points, points in the box, points
    outside it, clamped): contexts from empty to a few hundred points."""
    rng = np.random.default_rng(10 * r + K)
    B, N, M = 2, 3000, 1111
    # the points fill [0, 0.7)^3 of the grid's unit box, densest near 0
    P = (rng.random((B, N, 3), dtype=np.float32) ** 2 * np.float32(0.7)).astype(np.float32)
    Q = np.concatenate([P[:, :300], rng.random((B, 500, 3), dtype=np.float32),
                        (rng.random((B, M - 800, 3), dtype=np.float32) * np.float32(1.6) - np.float32(0.3))], 1)
    spec = _spec((0, 0, 0), (0.05,) * 3, (20, 20, 20), 8, r)
    qo = run_up(P, spec, Q, K, "knn", 1, where=f"r={r} K={K}")
    assert (qo["n_valid"] == 0).any() and (qo["ctx_count"] > 64).any()
    run_up(P, spec, Q, K, "cube", 2, where=f"cube r={r} K={K}", context=False)


def test_query_points_nonfinite_center_is_reported():
    rng = np.random.default_rng(3)
    P = rng.random((1, 500, 3), dtype=np.float32)
    Q = rng.random((1, 40, 3), dtype=np.float32)
    Q[0, 5, 2] = np.inf
    Q[0, 9, 0] = np.nan
    spec = _spec((0, 0, 0), (0.1,) * 3, (10, 10, 10), 8)
    ot = oracle.Table(P, oracle.grid_from_spec(spec))
    qo = ot.query_points(Q, 8, "knn", 0, allow_nonfinite=True)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.desc_from_spec(spec))
    qg = cagq.query_points(g, torch.from_numpy(Q).to(DEV), 8, "knn", 0)
    assert cagq.get_device_status(g) == cagq.ERR_NONFINITE_INPUT
    for k in ("node_idx", "n_valid", "ctx_count", "center_lin"):
        assert np.array_equal(_np(qg[k]), qo[k]), k


@pytest.mark.parametrize("name", ["tiny", "object", "room", "bigroom/cas-knn", "lidar"])
def test_context_lists_of_sampled_centers(name):
    """The context lists of each workload's layer-1 centers, at full size."""
    w = W.get_workload(name)
    P = w.points()
    L = w.layers[0]
    print(f"[parity] context lists {name}: B={P.shape[0]} N={P.shape[1]} M={L.M}", flush=True)
    ot = oracle.Table(P, oracle.grid_from_spec(L.grid))
    ocl, _ = ot.sample_rvs(L.M, L.seed)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.desc_from_spec(L.grid))
    cl, _ = cagq.sample_centers(g, L.M, "rvs", L.seed)
    assert np.array_equal(_np(cl), ocl)
    assert_context(g, ot, cl, name)


@pytest.mark.parametrize("BM", [1, 1023, 1024, 1025, 3073])
def test_context_offsets_at_scan_tile_edges(BM):
    """Center counts on both sides of the offsets scan's tile size, with
    unoccupied center voxels and repeated centers."""
    rng = np.random.default_rng(BM)
    P = rng.random((1, 4000, 3), dtype=np.float32)
    spec = _spec((0, 0, 0), (0.05,) * 3, (20, 20, 20), 4)
    cl = rng.integers(0, 8000, (1, BM)).astype(np.int32)
    ot = oracle.Table(P, oracle.grid_from_spec(spec))
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.desc_from_spec(spec))
    assert_context(g, ot, torch.from_numpy(cl).to(DEV), f"BM={BM}")


def test_context_list_capacity_and_outside_lin():
    rng = np.random.default_rng(4)
    P = rng.random((2, 2000, 3), dtype=np.float32)
    spec = _spec((0, 0, 0), (0.1,) * 3, (10, 10, 10), 8)
    ot = oracle.Table(P, oracle.grid_from_spec(spec))
    cl = rng.integers(0, 1000, (2, 50)).astype(np.int32)
    off_o, idx_o = ot.context_list(cl)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.desc_from_spec(spec))
    clt = torch.from_numpy(cl).to(DEV)
    off = cagq.context_offsets(g, clt)
    cap = len(idx_o) // 2
    out = torch.full((len(idx_o),), -9, dtype=torch.int32, device=DEV)
    cagq.context_list(g, clt, off, out=out, capacity=cap)
    assert cagq.get_device_status(g) == cagq.ERR_CAPACITY
    got = _np(out)
    assert np.array_equal(got[:cap], idx_o[:cap]) and np.all(got[cap:] == -9)
    # a lin outside the grid: empty context, reported
    g2 = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.desc_from_spec(spec))
    bad = clt.clone()
    bad[1, 7] = 1000
    off2 = cagq.context_offsets(g2, bad)
    assert cagq.get_device_status(g2) == cagq.ERR_CENTER_NOT_OCCUPIED
    o2 = _np(off2)
    assert o2[57 + 1] == o2[57]
    with pytest.raises(oracle.OracleError, match="-7"):
        ot.context_list(_np(bad))


# ---------------------------------------------------------------- level-wise k-NN (Appendix D)

@pytest.mark.parametrize("name", ["tiny", "object", "room", "bigroom/cas-knn", "lidar"])
def test_knn_ring_workloads(name):
    """Layer 1 of each workload with the level-wise k-NN, at full size."""
    w = W.get_workload(name)
    P = w.points()
    L = w.layers[0]
    print(f"[parity] knn_ring {name}: B={P.shape[0]} N={P.shape[1]} M={L.M} K={L.K} r={L.grid.radius}", flush=True)
    run_both(P, L.grid, L.M, L.K, L.sample, "knn_ring", L.seed, where=f"{name} ring")


@pytest.mark.parametrize("r", [1, 2, 3])
@pytest.mark.parametrize("K", [1, 5, 32, 64, 65, 96, 128])
def test_knn_ring_radius_and_node_counts(r, K):
    """Levels cut at every position: clustered points with small and large
    voxel populations, n_v binding, weights."""
    rng = np.random.default_rng(100 * r + K)
    B, N = 2, 4000
    P = (rng.random((B, N, 3), dtype=np.float32) ** 3).astype(np.float32)
    spec = _spec((0, 0, 0), (0.05,) * 3, (20, 20, 20), 16, r)
    wts = rng.integers(1, 9, (B, N)).astype(np.uint32)
    run_both(P, spec, 300, K, "rvs", "knn_ring", 4, weights=wts, where=f"ring r={r} K={K}")


def test_knn_ring_hand_worked_on_gpu():
    """The five-point example worked by hand for the oracle's pins."""
    P = np.array([[[2.5, 3.6, 2.5], [2.95, 2.95, 2.95], [3.05, 2.5, 2.5], [2.5, 2.5, 2.9],
                   [1.9, 2.5, 2.5]]], np.float32)
    g = cagq.build_grid(torch.from_numpy(P).to(DEV), cagq.make_desc((0, 0, 0), (1, 1, 1), (5, 5, 5), 8, 1))
    cl = torch.tensor([[62]], dtype=torch.int32, device=DEV)
    for K, nodes in [(1, [3]), (2, [1, 3]), (3, [1, 3, 2]), (5, [1, 3, 4, 2, 0]), (6, [1, 3, 4, 2, 0, 1])]:
        q = cagq.query_context(g, cl, K, "knn_ring", 0)
        assert _np(q["node_idx"])[0, 0].tolist() == nodes, K
    assert cagq.get_device_status(g) == 0


@pytest.mark.parametrize("r", [1, 2])
def test_query_points_knn_ring(r):
    rng = np.random.default_rng(r)
    P = (rng.random((2, 3000, 3), dtype=np.float32) ** 2 * np.float32(0.7)).astype(np.float32)
    Q = rng.random((2, 900, 3), dtype=np.float32)
    spec = _spec((0, 0, 0), (0.05,) * 3, (20, 20, 20), 8, r)
    run_up(P, spec, Q, 16, "knn_ring", 0, where=f"up ring r={r}", context=False)


# ---------------------------------------------------------------- comparison methods and coverage (Sec. 4)

@pytest.mark.parametrize("B,N,M", [(1, 1, 1), (2, 1000, 1000), (3, 5000, 77), (2, 70000, 8192), (1, 81920, 1)])
def test_rps_matches_oracle(B, N, M):
    P = W.uniform_cube(B, N, N % 97)
    c = cagq.sample_points(torch.from_numpy(P).to(DEV), M, "rps", 5)
    assert np.array_equal(_np(c), oracle.sample_points(P, M, "rps", 5))


@pytest.mark.parametrize("B,N,M", [(1, 1, 1), (2, 1000, 1000), (2, 3000, 500), (1, 20000, 300), (2, 81920, 2048)])
def test_fps_matches_oracle(B, N, M):
    rng = np.random.default_rng(N)
    P = rng.random((B, N, 3), dtype=np.float32)
    P[:, N // 2:N // 2 + min(50, N // 2)] = P[:, :1]  # duplicate points: ties and zero distances
    print(f"[parity] fps B={B} N={N} M={M}", flush=True)
    c = cagq.sample_points(torch.from_numpy(P).to(DEV), M, "fps")
    assert np.array_equal(_np(c), oracle.sample_points(P, M, "fps"))


@pytest.mark.parametrize("K", [1, 16, 64])
def test_ball_query_matches_oracle(K):
    w = W.get_workload("room")
    P = w.points()
    c = oracle.sample_points(P, 500, "rps", 3)
    c[0, :5] = [-1, P.shape[1], 0, 1, 2]  # out-of-range centers get nothing
    r2 = float(np.float32(0.186) ** 2)
    q = cagq.ball_query(torch.from_numpy(P).to(DEV), torch.from_numpy(c).to(DEV), K, r2)
    ni_o, nv_o = oracle.ball_query(P, np.where((c >= 0) & (c < P.shape[1]), c, 0), K, r2)
    ni_o[0, :2], nv_o[0, :2] = -1, 0
    assert np.array_equal(_np(q["node_idx"]), ni_o)
    assert np.array_equal(_np(q["n_valid"]), nv_o)


@pytest.mark.parametrize("name", ["room", "bigroom/cas-knn"])
def test_coverage_matches_oracle(name):
    """Coverage of CAGQ nodes and of RPS + Ball Query nodes, on the layer-1 grid."""
    w = W.get_workload(name)
    P = w.points()
    L = w.layers[0]
    ot = oracle.Table(P, oracle.grid_from_spec(L.grid))
    Pt = torch.from_numpy(P).to(DEV)
    g = cagq.build_grid(Pt, cagq.desc_from_spec(L.grid))
    cl, mv = cagq.sample_centers(g, L.M, "rvs", 1)
    q = cagq.query_context(g, cl, L.K, "cube", 1)
    cov = cagq.coverage(g, q["node_idx"], q["n_valid"])
    assert np.array_equal(_np(cov), ot.coverage(_np(q["node_idx"]), _np(q["n_valid"])))
    c = cagq.sample_points(Pt, L.M, "rps", 1)
    bq = cagq.ball_query(Pt, c, L.K, float(np.float32(0.1) ** 2))
    cov2 = cagq.coverage(g, bq["node_idx"], bq["n_valid"])
    assert np.array_equal(_np(cov2), ot.coverage(_np(bq["node_idx"]), _np(bq["n_valid"])))
    assert cagq.get_device_status(g) == 0


@pytest.mark.parametrize("r", [1, 2, 3])
@pytest.mark.parametrize("K", [17, 32])
def test_sixteen_lane_query_with_large_contexts(r, K):
    """Contexts from empty to several hundred points in one block of 16
    centers (the query sorts the block's centers by context size), weights,
    K between 17 and 32: several chunks merged into two result registers."""
    rng = np.random.default_rng(7 * r + K)
    B, N = 2, 6000
    P = (rng.random((B, N, 3), dtype=np.float32) ** 4).astype(np.float32)
    spec = _spec((0, 0, 0), (0.04,) * 3, (25, 25, 25), 32, r)
    wts = rng.integers(1, 50, (B, N)).astype(np.uint32)
    for q in ("knn", "cube"):
        qo = run_both(P, spec, 333, K, "rvs", q, 3, weights=wts, where=f"r={r} K={K} {q}")
    assert qo["ctx_count"].max() > 64 and qo["ctx_count"].min() < 16


@pytest.mark.parametrize("r", [1, 2, 3])
@pytest.mark.parametrize("K", [65, 96, 128])
def test_two_register_query_with_large_contexts(r, K):
    """64 < K <= 128 (a whole wave per center, ranks 64..127 in a second
    register): contexts from a handful of points to a few thousand, so that
    some chunks are merged into both registers, others leave the second one
    empty; weights; every mode."""
    rng = np.random.default_rng(11 * r + K)
    B, N = 2, 6000
    P = (rng.random((B, N, 3), dtype=np.float32) ** 4).astype(np.float32)
    spec = _spec((0, 0, 0), (0.04,) * 3, (25, 25, 25), 64, r)
    wts = rng.integers(1, 50, (B, N)).astype(np.uint32)
    for q in ("knn", "cube", "knn_ring"):
        qo = run_both(P, spec, 333, K, "rvs", q, 3, weights=wts, where=f"r={r} K={K} {q}")
        assert qo["ctx_count"].max() > 2 * K and qo["ctx_count"].min() < 64
    assert (qo["n_valid"] == K).any() and (qo["n_valid"] < 64).any()


def test_paper_latency_conditions_with_k128():
    """The paper's latency tables sweep K up to 128 (Sec. 4; Appendix F):
    N = 81920 and N = 8192 with M = 1024 and K = 128, both samplers and both
    queries, on the synthetic indoor scene."""
    w = W.get_workload("bigroom/rvs-cube")
    L = w.layers[0]
    P = w.points(B=1)
    for (sample, query) in (("rvs", "cube"), ("cas", "knn"), ("rvs", "knn"), ("cas", "cube")):
        print(f"[parity] K=128 N=81920 M=1024 {sample}+{query}", flush=True)
        run_both(P, L.grid, 1024, 128, sample, query, L.seed, where=f"K=128 {sample}+{query}")
    r = W.get_workload("room")
    run_both(r.points(B=1), r.layers[0].grid, 1024, 128, "cas", "knn", 3, where="K=128 N=8192")


# ---------------------------------------------------------------- HIP graph replay

def _rvs_plan(w, B, dev):
    plan, n = [], w.N
    for L in w.layers:
        desc = cagq.desc_from_spec(L.grid)
        lay = cagq.workspace_layout(B, n, desc)
        plan.append((L, desc, torch.empty(lay.total_bytes, dtype=torch.uint8, device=dev),
                     cagq.alloc_query_outputs(B, L.M, L.K, dev), torch.empty((B, L.M), dtype=torch.int32, device=dev),
                     torch.empty((B,), dtype=torch.int32, device=dev)))
        n = L.M
    return plan


def _run_plan(P, plan, first=0):
    pts, wts = (P, None) if first == 0 else (plan[first - 1][3]["center_xyz"], plan[first - 1][3]["center_w"])
    for (L, desc, ws, out, cl, mv) in plan[first:]:
        g = cagq.build_grid(pts, desc, ws)
        cagq.sample_centers(g, L.M, L.sample, L.seed, center_lin=cl, m_valid=mv)
        cagq.query_context(g, cl, L.K, L.query, L.seed, weights=wts, out=out)
        pts, wts = out["center_xyz"], out["center_w"]


def _snapshot(plan):
    return [(_np(cl).copy(), _np(mv).copy(), {k: _np(v).copy() for k, v in out.items() if v is not None})
            for (L, desc, ws, out, cl, mv) in plan]


def test_graph_replay_of_the_rvs_cube_path():
    """The four RVS + Cube Query layers of the indoor scenes, captured once in
    a HIP graph (all kernels, no memory-set nodes) and replayed three times,
    with eager runs of the same path on other inputs and synchronizations in
    between: every replay equals the eager result bit for bit, and layer 1
    equals the oracle."""
    w = W.get_workload("bigroom/rvs-cube")
    B = 4
    P_np = w.points(B=B)
    P = torch.from_numpy(P_np).to(DEV)
    plan = _rvs_plan(w, B, DEV)
    _run_plan(P, plan)
    torch.cuda.synchronize()
    ref = _snapshot(plan)
    # layer 1 against the oracle
    L = w.layers[0]
    ot = oracle.Table(P_np, oracle.grid_from_spec(L.grid))
    ocl, omv = ot.sample_rvs(L.M, L.seed)
    assert np.array_equal(ref[0][0], ocl)
    qo = ot.query(ocl, omv, L.K, L.query, L.seed)
    assert np.array_equal(ref[0][2]["node_idx"], qo["node_idx"])
    assert np.array_equal(_bits(ref[0][2]["center_xyz"]), _bits(qo["center_xyz"]))

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        _run_plan(P, plan)
    torch.cuda.synchronize()
    other = _rvs_plan(w, B, DEV)
    P2 = (P * 0.5).contiguous()
    for rep in range(3):
        for (L, desc, ws, out, cl, mv) in plan:  # scribble over the outputs first
            cl.fill_(-5)
            for v in out.values():
                if v is not None:
                    v.fill_(7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(plan)
        for li, ((a_cl, a_mv, a_out), (b_cl, b_mv, b_out)) in enumerate(zip(ref, got)):
            assert np.array_equal(a_cl, b_cl) and np.array_equal(a_mv, b_mv), (rep, li)
            for k in a_out:
                assert np.array_equal(_bits(a_out[k]), _bits(b_out[k])), (rep, li, k)
        _run_plan(P2, other)  # the program's own eager work between replays
        torch.cuda.synchronize()


def test_two_stream_overlapped_step_matches_oracle():
    """The bench's step: RVS+Cube replayed from a graph on one stream while
    CAS+k-NN runs eagerly (its large layers paced from the host) on another;
    every layer of both variants against the oracle, three steps in a row."""
    B = 2
    dev = torch.device(DEV)
    w_cas, w_rvs = W.get_workload("bigroom/cas-knn"), W.get_workload("bigroom/rvs-cube")
    P_np = w_cas.points(B=B)
    P = torch.from_numpy(P_np).to(dev)
    plan_cas, plan_rvs = _rvs_plan(w_cas, B, dev), _rvs_plan(w_rvs, B, dev)
    s_cas, s_rvs = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s_rvs):
        _run_plan(P, plan_rvs)
    torch.cuda.synchronize()
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr, stream=s_rvs):
        _run_plan(P, plan_rvs)
    torch.cuda.synchronize()
    expect = {}
    for w in (w_cas, w_rvs):
        pts, wts, layers = P_np, None, []
        for L in w.layers:
            _, ocl, omv, q = oracle.run_layer(pts, L, weights=wts)
            layers.append((ocl, omv, q))
            pts, wts = q["center_xyz"], q["center_w"]
        expect[w.name] = layers
    for step in range(3):
        for plan in (plan_cas, plan_rvs):  # clobber the outputs of the previous step
            for (L, desc, ws, out, cl, mv) in plan:
                cl.fill_(-5)
                for v in out.values():
                    if v is not None:
                        v.fill_(7)
        torch.cuda.synchronize()
        main = torch.cuda.current_stream()
        s_cas.wait_stream(main)
        s_rvs.wait_stream(main)
        with torch.cuda.stream(s_rvs):
            gr.replay()
        with torch.cuda.stream(s_cas):
            _run_plan(P, plan_cas)
        torch.cuda.synchronize()
        for w, plan in ((w_cas, plan_cas), (w_rvs, plan_rvs)):
            for li, ((L, desc, ws, out, cl, mv), (ocl, omv, q)) in enumerate(zip(plan, expect[w.name])):
                where = f"step {step} {w.name} layer {li + 1}"
                assert np.array_equal(_np(cl), ocl), where
                assert np.array_equal(_np(mv), omv), where
                for k, v in out.items():
                    if v is not None:
                        assert np.array_equal(_bits(_np(v)), _bits(q[k])), (where, k)


def test_graph_replay_of_the_single_workgroup_cas_layers():
    """Layers 3-4 of the CAS + k-NN indoor path (2048 and 512 points per
    cloud: single-workgroup CAS, no host round trips), captured in a HIP graph
    after eager layers 1-2 and replayed three times with eager work and
    synchronizations between: every replay equals the eager result bit for
    bit, and layer 3's centers equal the oracle's CAS on layer 2's output."""
    w = W.get_workload("bigroom/cas-knn")
    B = 4
    P = torch.from_numpy(w.points(B=B)).to(DEV)
    plan = _rvs_plan(w, B, DEV)
    _run_plan(P, plan)
    torch.cuda.synchronize()
    ref = _snapshot(plan)
    L3 = w.layers[2]
    ot = oracle.Table(_np(plan[1][3]["center_xyz"]).copy(), oracle.grid_from_spec(L3.grid))
    ocl, omv, _, _ = ot.sample_cas(L3.M)
    assert np.array_equal(ref[2][0], ocl) and np.array_equal(ref[2][1], omv)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        _run_plan(P, plan, first=2)
    torch.cuda.synchronize()
    other = _rvs_plan(w, B, DEV)
    P2 = (P * 0.5).contiguous()
    for rep in range(3):
        for (L, desc, ws, out, cl, mv) in plan[2:]:  # scribble over the outputs first
            cl.fill_(-5)
            for v in out.values():
                if v is not None:
                    v.fill_(7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(plan)
        for li in (2, 3):
            (a_cl, a_mv, a_out), (b_cl, b_mv, b_out) = ref[li], got[li]
            assert np.array_equal(a_cl, b_cl) and np.array_equal(a_mv, b_mv), (rep, li)
            for k in a_out:
                assert np.array_equal(_bits(a_out[k]), _bits(b_out[k])), (rep, li, k)
        _run_plan(P2, other)  # the program's own eager work between replays
        torch.cuda.synchronize()
