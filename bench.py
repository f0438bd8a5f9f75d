"""CAGQ throughput on one MI355X.

A step is one pass of the whole CAGQ hot path over one batch: B = 4 synthetic
indoor scenes of 81920 points, four downsampling layers (voxel sizes 0.05 /
0.1 / 0.2 / 0.4 m, M = 8192 / 2048 / 512 / 128, K = 32, n_v = 32), run once
with Coverage-Aware Sampling + k-NN and once with Random Voxel Sampling +
Cube Query; the two variants are independent and run on two streams. Each
layer builds the grid, samples the centers and queries the nodes; layer l+1
consumes the centers and weights of layer l. Inputs are resident in HBM
before timing starts; workspaces and outputs are allocated once, outside the
timed region.

Prints one JSON line: points/s over the step, ms per step, a roofline entry
for the layer-1 query kernel (algorithmic bytes per launch over its HIP-event
duration on the launch stream) and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
COPY_PROBE_BYTES = 1 << 30  # the calibration copy reads and writes this many bytes
SLEEP_CYCLES = 1_000_000  # about 0.4 ms of the GPU clock before each bracketed launch
QUERY_REPS = 10  # layer-1 query launches between the roofline's events
ROOF_PASSES = 3  # variant passes that time them
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_query_bigroom_b4_traffic.md")
QUERY_SOURCES = ("paper_1912_02984_amd/csrc/cagq_query.hip", "paper_1912_02984_amd/csrc/cagq_internal.h")
QUERY_NAMES = {"0": "k_query<cube>", "1": "k_query<knn>"}
WORKLOAD = "bigroom"
VARIANTS = ("bigroom/cas-knn", "bigroom/rvs-cube")
METRIC = "CAGQ points/sec & ms/batch at 81920 pts; achieved HBM GB/s vs MI355X peak"


def query_alg_bytes(M_total: int, K: int, S_total: int) -> int:
    """Algorithmic bytes of one query launch: the stored points' coordinates
    read once (12 B each, S of them), per center its outputs (node_idx and
    node_xyz, 16 B per node) and 28 B of center id, center_xyz, center_w and
    n_valid."""
    return 12 * S_total + M_total * (16 * K + 28)


def query_reread_bytes(M_total: int, K: int, ctx_total: int) -> int:
    """The same launch counting every context point of every center (16 B:
    coordinates and index), so overlapping neighbourhoods are read again."""
    return M_total * (16 * K + 28) + 16 * ctx_total


def layer_alg_bytes(N_total: int, S_total: int, nvox_total: int, M_total: int, K: int, weights: bool) -> int:
    """Algorithmic bytes of a whole layer (voxelize, table, sampling, query):
    points read (12 B, plus 4 B of weight), lists and voxel records written
    and read (8 B per stored point, 24 B per occupied voxel), the stored
    points' coordinates read by the query (12 B), the nodes (16 B) and the
    centers (28 B)."""
    return (12 + (4 if weights else 0)) * N_total + 20 * S_total + 24 * nvox_total + M_total * (16 * K + 28)


def query_source_hash() -> str:
    h = hashlib.sha256()
    for rel in QUERY_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic() -> dict:
    """Per-launch HBM bytes of the layer-1 query kernels from the committed
    counter summary; empty unless it was taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            txt = f.read()
    except OSError:
        return {}
    m = re.search(r"kernel source sha256\[:16\]: `([0-9a-f]+)`", txt)
    if not m or m.group(1) != query_source_hash():
        return {}
    return {k: int(v) for k, v in re.findall(r"^\| `(k_query<\w+>)` \|(?:[^|]*\|){3} (\d+) \|", txt, re.M)}


def _short(name: str) -> str:
    m = re.search(r"(k_\w+)<(\d)(?:, \d+)*>", name)
    if m and m.group(1) == "k_query":
        return QUERY_NAMES[m.group(2)]
    m = re.search(r"(k_\w+(?:<[^>(]*>)?)\(", name)
    return m.group(1) if m else name[:40]


def summarize_stats(stats_csv: str, command: str) -> str:
    """Markdown table of a rocprofv3 --stats kernel summary, and, when the
    run's kernel trace sits beside it, the query launches by grid size."""
    rows = list(csv.DictReader(open(stats_csv)))
    out = ["| Kernel | Calls | Total (us) | Avg (us) | Min (us) | Max (us) | % |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e3:.1f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                   f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    trace_csv = stats_csv.replace("_kernel_stats.csv", "_kernel_trace.csv")
    if trace_csv != stats_csv and os.path.exists(trace_csv):
        by = {}
        for r in csv.DictReader(open(trace_csv)):
            if "k_query" not in r["Kernel_Name"]:
                continue
            blocks = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]))
            d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            by.setdefault((_short(r["Kernel_Name"]), blocks), []).append(d)
        out += ["", "Query launches by grid size (from the kernel trace of the same run):", "",
                "| Kernel | Blocks | Launches | Avg (us) | Min (us) |", "|---|---|---|---|---|"]
        for (name, blocks), ds in sorted(by.items(), key=lambda kv: (kv[0][0], -kv[0][1])):
            out.append(f"| {name} | {blocks} | {len(ds)} | {sum(ds) / len(ds):.2f} | {min(ds):.2f} |")
    return "\n".join([f"Command: `{command}`", ""] + out) + "\n"


def summarize_counters(csv_path: str) -> str:
    """Per kernel, the dispatches and the average of every counter per
    dispatch, from a rocprofv3 --pmc counter collection."""
    rows = list(csv.DictReader(open(csv_path)))
    sums, disp, names = {}, {}, []
    for r in rows:
        m = re.search(r"(k_\w+(?:<[^>]*>)?|at::native::\w+|__amd_\w+)", r["Kernel_Name"])
        k = m.group(1) if m else r["Kernel_Name"][:40]
        c = r["Counter_Name"]
        if c not in names:
            names.append(c)
        sums.setdefault(k, {}).setdefault(c, 0.0)
        sums[k][c] += float(r["Counter_Value"])
        disp.setdefault(k, set()).add(r["Dispatch_Id"])
    out = ["| Kernel | Dispatches | " + " | ".join(names) + " |", "|---|---|" + "---|" * len(names)]
    for k in sorted(sums, key=lambda k: -sums[k].get(names[0], 0.0) / len(disp[k])):
        n = len(disp[k])
        out.append(f"| {k} | {n} | " + " | ".join(f"{sums[k].get(c, 0.0) / n:.1f}" for c in names) + " |")
    return "\n".join(out) + "\n"


LAYER_FILE = os.path.join(ROOT, "profiles", "cagq_layer1_bigroom_b4.md")
LAYER_SOURCES = "paper_1912_02984_amd/csrc"


def layer_source_hash() -> str:
    """Hash of every HIP source and header of the library."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, LAYER_SOURCES)
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def load_layer_profile() -> dict:
    """Per variant: summed kernel time (us), HBM bytes and launches of one
    layer-1 pass from the committed profile; empty unless it was taken on
    the current library sources."""
    try:
        with open(LAYER_FILE) as f:
            txt = f.read()
    except OSError:
        return {}
    m = re.search(r"library source sha256\[:16\]: `([0-9a-f]+)`", txt)
    if not m or m.group(1) != layer_source_hash():
        return {}
    out = {}
    for v, us, by, n in re.findall(r"^layer1 (\S+): kernel_us=([0-9.]+) bytes=(\d+) launches=(\d+)$", txt, re.M):
        out[v] = {"us": float(us), "bytes": int(by), "launches": int(n)}
    return out


def summarize_layer(variant: str, fetch_csv: str, write_csv: str, trace_csv: str, passes: int) -> str:
    """One variant's layer-1 kernels from a --layer1-passes run: per kernel
    the launches per pass, the average duration (kernel trace) and the HBM
    bytes per launch (FETCH_SIZE and WRITE_SIZE, each scaled by what it reads
    for the calibration copy); then their sums over one pass. The warm-up
    pass (the first 1/(passes+1) of the dispatches) is left out."""
    def cagq_rows(rows, key):
        rows = sorted((r for r in rows if "cagq::" in r["Kernel_Name"]), key=lambda r: int(r[key]))
        return rows[len(rows) // (passes + 1):]

    def load(path, counter):
        return [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
    fr, wr = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")

    def copy_kib(rows):  # the largest torch kernel of the run is the calibration copy
        return max(float(r["Counter_Value"]) for r in rows if "at::native" in r["Kernel_Name"])
    cf, cw = copy_kib(fr), copy_kib(wr)
    sf, sw = COPY_PROBE_BYTES / (cf * 1024), COPY_PROBE_BYTES / (cw * 1024)
    fr, wr = cagq_rows(fr, "Dispatch_Id"), cagq_rows(wr, "Dispatch_Id")
    tr = cagq_rows(list(csv.DictReader(open(trace_csv))), "Start_Timestamp")
    per = {}
    for r in tr:
        e = per.setdefault(_short(r["Kernel_Name"]), {"n": 0, "us": 0.0, "f": 0.0, "w": 0.0})
        e["n"] += 1
        e["us"] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    for rows, k in ((fr, "f"), (wr, "w")):
        for r in rows:
            per.setdefault(_short(r["Kernel_Name"]), {"n": 0, "us": 0.0, "f": 0.0, "w": 0.0})[k] += \
                float(r["Counter_Value"])
    lines = [f"### {variant}", "",
             f"Calibration: the {COPY_PROBE_BYTES >> 20} MiB copy reads FETCH_SIZE {cf:.0f} KiB (scale {sf:.4f}) and "
             f"WRITE_SIZE {cw:.0f} KiB (scale {sw:.4f}).", "",
             "| Kernel | Launches per pass | Avg (us) | FETCH_SIZE (KiB) per launch | WRITE_SIZE (KiB) per launch "
             "| HBM bytes per pass |", "|---|---|---|---|---|---|"]
    tot_us = tot_b = tot_n = 0.0
    for k, e in sorted(per.items(), key=lambda kv: -kv[1]["us"]):
        n = max(e["n"], 1)
        b = (e["f"] * sf + e["w"] * sw) * 1024 / passes
        tot_us += e["us"] / passes
        tot_b += b
        tot_n += e["n"] / passes
        lines.append(f"| {k} | {e['n'] / passes:.1f} | {e['us'] / n:.2f} | {e['f'] / n:.1f} | {e['w'] / n:.1f} "
                     f"| {int(round(b))} |")
    lines.append(f"| **one layer-1 pass** | {tot_n:.1f} | {tot_us:.2f} (sum) | | | {int(round(tot_b))} |")
    lines += ["", f"layer1 {variant}: kernel_us={tot_us:.2f} bytes={int(round(tot_b))} launches={int(round(tot_n))}", "",
              f"library source sha256[:16]: `{layer_source_hash()}` ({LAYER_SOURCES}/*.hip, *.h)", ""]
    return "\n".join(lines) + "\n"


def summarize_traffic(fetch_csv: str, write_csv: str) -> str:
    """HBM bytes per launch of the layer-1 query kernels from a FETCH_SIZE
    and a WRITE_SIZE pass, each scaled by what the same counter reads for
    the calibration copy (COPY_PROBE_BYTES read and written)."""
    def load(path, counter):
        return [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
    fr, wr = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")

    def copy_kib(rows):  # the largest torch kernel of the run is the calibration copy
        return max(float(r["Counter_Value"]) for r in rows if "at::native" in r["Kernel_Name"])
    cf, cw = copy_kib(fr), copy_kib(wr)
    sf, sw = COPY_PROBE_BYTES / (cf * 1024), COPY_PROBE_BYTES / (cw * 1024)

    def layer1(rows, mode):
        q = [r for r in rows if re.search(rf"k_query(?:_r2)?<{mode}, \d+(?:, \d+)?(?:, false)?>", r["Kernel_Name"])]
        g = max(int(r["Grid_Size"]) for r in q)
        return [float(r["Counter_Value"]) for r in q if int(r["Grid_Size"]) == g]
    lines = [f"Calibration: a {COPY_PROBE_BYTES >> 20} MiB fp32 copy kernel reads FETCH_SIZE {cf:.0f} KiB "
             f"(scale {sf:.4f}) and WRITE_SIZE {cw:.0f} KiB (scale {sw:.4f}).", "",
             "| Kernel | Dispatches | FETCH_SIZE (KiB) | WRITE_SIZE (KiB) | HBM bytes per launch |",
             "|---|---|---|---|---|"]
    for mode, name in QUERY_NAMES.items():
        f, w = layer1(fr, mode), layer1(wr, mode)
        fk, wk = float(np.mean(f)), float(np.mean(w))
        lines.append(f"| `{name}` | {len(f)} | {fk:.1f} | {wk:.1f} | {int(round(fk * 1024 * sf + wk * 1024 * sw))} |")
    lines += ["", f"kernel source sha256[:16]: `{query_source_hash()}` "
                  f"({' + '.join(QUERY_SOURCES)})"]
    return "\n".join(lines) + "\n"


def measure_cas_swap(P, P_np, B: int, N: int, L, with_oracle: bool, reps: int = 3) -> dict:
    """The paper's challenger / incumbent CAS (a sequential procedure, so
    latency-bound: reported in ms and challenges per second) on the layer-1
    grid of the bench batch, with the oracle on one scene beside it."""
    import torch
    from paper_1912_02984_amd import cagq
    desc = cagq.desc_from_spec(L.grid)
    g = cagq.build_grid(P, desc)
    cl, mv = cagq.sample_centers(g, L.M, "cas_swap", L.seed)
    torch.cuda.synchronize()
    nvox = g.table()["nvox"].cpu().numpy()
    challenges = int(sum(int(n) - min(L.M, int(n)) for n in nvox))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        cagq.sample_centers(g, L.M, "cas_swap", L.seed, center_lin=cl, m_valid=mv)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    status = cagq.get_device_status(g)
    row = {"workload": f"layer 1 of the bench batch: B={B} x {N} pts, M={L.M}, r={L.grid.radius}",
           "ms": round(ms, 3), "challenges": challenges,
           "challenges_per_s": round(challenges / (ms / 1e3), 1), "bound": "latency (sequential challenges)",
           "device_status": status}
    if with_oracle:
        import oracle
        t0 = time.perf_counter()
        ot = oracle.Table(P_np[:1], oracle.grid_from_spec(L.grid))
        ocl, omv, _, _ = ot.sample_cas_swap(L.M, L.seed)
        dt = time.perf_counter() - t0
        ch1 = int(ot.nvox[0]) - min(L.M, int(ot.nvox[0]))
        row["oracle"] = {"ms": round(dt * 1e3, 2), "challenges": ch1, "challenges_per_s": round(ch1 / dt, 1),
                         "cores": 1, "sample": "1 of the scenes, table build included"}
        same = (status == 0 and np.array_equal(cl[:1].cpu().numpy(), ocl)
                and np.array_equal(mv[:1].cpu().numpy(), omv))
        row["parity"] = {"checked": "scene 0: center_lin and m_valid of the timed call vs the oracle, "
                                    "and the device status", "bit_exact": bool(same)}
    return row


def _timed(fn, reps: int):
    """Average ms of fn() over reps calls, each bracketed by HIP events on the
    current stream after a bounded GPU-side delay (so the host has enqueued
    the calls before the GPU reaches the start event)."""
    import torch
    fn()
    torch.cuda.synchronize()
    pairs = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SLEEP_CYCLES)
        e0.record()
        fn()
        e1.record()
        pairs.append((e0, e1))
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in pairs) / reps


def measure_upsampling(P, P_np, B: int, N: int, wl, with_oracle: bool, reps: int = 20) -> dict:
    """The upsampling query (centers given: the N input points of each scene)
    against the grid of the layer-1 centers, with the layer-2 grid spec and K,
    and the context lists of the layer-1 centers on the layer-1 grid."""
    import torch
    from paper_1912_02984_amd import cagq
    L0, L1 = wl.layers[0], wl.layers[1]
    # the coarse points: the layer-1 group centers of the same batch
    g0 = cagq.build_grid(P, cagq.desc_from_spec(L0.grid))
    cl0, _ = cagq.sample_centers(g0, L0.M, L0.sample, L0.seed)
    q0 = cagq.query_context(g0, cl0, L0.K, L0.query, L0.seed)
    coarse = q0["center_xyz"].contiguous()
    g1 = cagq.build_grid(coarse, cagq.desc_from_spec(L1.grid))
    out = cagq.query_points(g1, P, L1.K, "knn", 1)
    ms = _timed(lambda: cagq.query_points(g1, P, L1.K, "knn", 1, out=out), reps)
    ctx = int(out["ctx_count"].sum().item())
    M = B * N
    # algorithmic bytes: center xyz in; per node index and xyz out; n_valid,
    # ctx_count and lin out; the context points' xyz + index (16 B each)
    alg = M * (12 + 16 * L1.K + 12) + 16 * ctx
    up = {"workload": f"B={B} x {N} centers (the input points) on the grid of the {L0.M} layer-1 centers, "
                      f"{tuple(L1.grid.dims)} voxels of {L1.grid.voxel_size[0]:.2f} m, K={L1.K}, k-NN",
          "ms": round(ms, 4), "centers_per_s": round(M / (ms / 1e3), 1),
          "roofline": {"bound": "hbm", "achieved": round(alg / (ms / 1e3) / 1e9, 1), "peak": 8000.0,
                       "unit": "GB/s", "frac": round(alg / (ms / 1e3) / 1e9 / 8000.0, 4), "traffic": None}}
    # context lists of the layer-1 centers
    off = cagq.context_offsets(g0, cl0)
    idx = cagq.context_list(g0, cl0, off)
    total = int(off[-1].item())

    def ctx_once():
        cagq.context_offsets(g0, cl0, out=off)
        cagq.context_list(g0, cl0, off, out=idx, capacity=total)
    ms_c = _timed(ctx_once, reps)
    alg_c = 8 * total + B * L0.M * (4 + 8)
    cx = {"workload": f"B={B} x {L0.M} layer-1 centers, {tuple(L0.grid.dims)} voxels, r={L0.grid.radius}: "
                      f"{total} context entries",
          "ms": round(ms_c, 4), "entries_per_s": round(total / (ms_c / 1e3), 1),
          "roofline": {"bound": "hbm", "achieved": round(alg_c / (ms_c / 1e3) / 1e9, 1), "peak": 8000.0,
                       "unit": "GB/s", "frac": round(alg_c / (ms_c / 1e3) / 1e9 / 8000.0, 4), "traffic": None}}
    if with_oracle:
        import oracle
        t0 = time.perf_counter()
        ot0 = oracle.Table(P_np[:1], oracle.grid_from_spec(L0.grid))
        ocl, omv = ot0.sample(L0.M, L0.sample, L0.seed)
        oq = ot0.query(ocl, omv, L0.K, L0.query, L0.seed)
        t1 = time.perf_counter()
        ot1 = oracle.Table(oq["center_xyz"], oracle.grid_from_spec(L1.grid))
        ot1.query_points(P_np[:1], L1.K, "knn", 1)
        t2 = time.perf_counter()
        _, oidx = ot0.context_list(ocl)
        t3 = time.perf_counter()
        up["oracle"] = {"ms": round((t2 - t1) * 1e3, 2), "centers_per_s": round(N / (t2 - t1), 1), "cores": 1,
                        "sample": "1 of the scenes, coarse table build included"}
        cx["oracle"] = {"ms": round((t3 - t2) * 1e3, 2), "entries_per_s": round(len(oidx) / (t3 - t2), 1),
                        "cores": 1, "sample": "1 of the scenes"}
    return {"query_points": up, "context_list": cx}


def measure_knn_ring(P, P_np, B: int, N: int, wl, with_oracle: bool, reps: int = 20) -> dict:
    """The level-wise k-NN of Appendix D against the exact context k-NN on the
    layer-1 centers of the bench batch: time per launch, and how far its nodes
    are from the exact ones (recall, centers with the same node set, and the
    ratio of the K-th node distance from the voxel center)."""
    import torch
    from paper_1912_02984_amd import cagq
    L = wl.layers[0]
    g = cagq.build_grid(P, cagq.desc_from_spec(L.grid))
    cl, _ = cagq.sample_centers(g, L.M, L.sample, L.seed)
    ex = cagq.query_context(g, cl, L.K, "knn", L.seed)
    rg = cagq.query_context(g, cl, L.K, "knn_ring", L.seed)
    ms_ex = _timed(lambda: cagq.query_context(g, cl, L.K, "knn", L.seed, out=ex), reps)
    ms_rg = _timed(lambda: cagq.query_context(g, cl, L.K, "knn_ring", L.seed, out=rg), reps)
    # K-th node distance from the center voxel's center (float64)
    dims = torch.tensor(L.grid.dims, device=P.device, dtype=torch.int64)
    lin = cl.long()
    gxyz = torch.stack([lin % dims[0], (lin // dims[0]) % dims[1], lin // (dims[0] * dims[1])], -1).double()
    q = torch.tensor(L.grid.origin, device=P.device, dtype=torch.float64) + (gxyz + 0.5) * torch.tensor(
        L.grid.voxel_size, device=P.device, dtype=torch.float64)

    def deviation(exact, ring, K):
        full = exact["n_valid"] == K
        a, b_ = ring["node_idx"].long(), exact["node_idx"].long()
        hit = (a[..., :, None] == b_[..., None, :]).any(-1).sum(-1).float()

        def kth(out):
            return (out["node_xyz"].double() - q[..., None, :]).norm(dim=-1).max(-1).values

        ratio = kth(ring)[full] / kth(exact)[full].clamp_min(1e-12)
        return {"K": K, "centers_with_K_nodes": int(full.sum().item()),
                "recall_vs_exact": round((hit[full] / K).mean().item(), 5),
                "same_node_set": round((hit[full] == K).float().mean().item(), 5),
                "kth_distance_ratio_mean": round(ratio.mean().item(), 5),
                "kth_distance_ratio_max": round(ratio.max().item(), 5)}

    dev = [deviation(ex, rg, L.K)]
    k2 = max(1, L.K // 4)
    dev.append(deviation(cagq.query_context(g, cl, k2, "knn", L.seed),
                         cagq.query_context(g, cl, k2, "knn_ring", L.seed), k2))
    row = {"workload": f"layer 1 of the bench batch: B={B} x {L.M} centers, K={L.K}, r={L.grid.radius}",
           "ms": round(ms_rg, 4), "ms_exact": round(ms_ex, 4), "deviation": dev}
    if with_oracle:
        import oracle
        ot = oracle.Table(P_np[:1], oracle.grid_from_spec(L.grid))
        ocl = np.ascontiguousarray(cl[:1].cpu().numpy())
        omv = np.full(1, min(L.M, int(ot.nvox[0])), np.int32)
        t0 = time.perf_counter()
        ot.query(ocl, omv, L.K, "knn_ring", L.seed)
        t1 = time.perf_counter()
        row["oracle"] = {"ms": round((t1 - t0) * 1e3, 2), "cores": 1, "sample": "the centers of 1 of the scenes"}
    return row


def measure_coverage(P, B: int, N: int, wl, reps: int = 3) -> dict:
    """Sec. 4's comparison on the layer-1 shape of the bench batch: latency of
    the whole data structuring (sampling + query; CAGQ includes its grid
    build) and the occupied-space coverage of the nodes, for RPS / FPS with
    Ball Query (radius giving the ball the cube's volume) and for RVS / CAS
    with Cube Query and k-NN. Coverage is the mean over the clouds of the
    occupied voxels holding a node over all occupied voxels."""
    import math
    import torch
    from paper_1912_02984_amd import cagq
    L = wl.layers[0]
    desc = cagq.desc_from_spec(L.grid)
    g = cagq.build_grid(P, desc)
    nvox = g.table()["nvox"].double()
    edge = (2 * L.grid.radius + 1) * L.grid.voxel_size[0]
    radius = edge * (3.0 / (4.0 * math.pi)) ** (1.0 / 3.0)
    r2 = float(np.float32(radius) ** 2)
    rows = {}

    def cagq_run(sample, query):
        gg = cagq.build_grid(P, desc)
        cl, _ = cagq.sample_centers(gg, L.M, sample, L.seed)
        return cagq.query_context(gg, cl, L.K, query, L.seed)

    def base_run(sample, query):
        c = cagq.sample_points(P, L.M, sample, L.seed)
        return cagq.ball_query(P, c, L.K, r2)

    for name, fn in [("RPS+Ball", lambda: base_run("rps", "ball")), ("FPS+Ball", lambda: base_run("fps", "ball")),
                     ("RVS+Cube", lambda: cagq_run("rvs", "cube")), ("CAS+Cube", lambda: cagq_run("cas", "cube")),
                     ("RVS+kNN", lambda: cagq_run("rvs", "knn")), ("CAS+kNN", lambda: cagq_run("cas", "knn"))]:
        ms = _timed(fn, reps)
        out = fn()
        cov = cagq.coverage(g, out["node_idx"], out["n_valid"]).double() / nvox
        rows[name] = {"ms": round(ms, 3), "coverage": round(cov.mean().item(), 4)}
    return {"workload": f"B={B} x {N} points, M={L.M}, K={L.K}, {tuple(L.grid.dims)} voxels of "
                        f"{L.grid.voxel_size[0]:.2f} m, r={L.grid.radius}; ball radius {radius:.4f} m",
            "methods": rows}


CONFIGS = ("tiny", "object", "room", "bigroom/cas-knn", "bigroom/rvs-cube", "lidar")


def _host_info() -> dict:
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count()}


class _OneCore:
    """Pins this process to one core of those it may use (the oracle is
    single-threaded; pinning keeps it on one core while it is timed)."""

    def __init__(self):
        self.saved = None
        self.where = "no core (affinity unavailable)"

    def __enter__(self):
        if hasattr(os, "sched_getaffinity"):
            self.saved = os.sched_getaffinity(0)
            core = max(self.saved)
            os.sched_setaffinity(0, {core})
            self.where = f"core {core}"
        return self

    def __exit__(self, *exc):
        if self.saved is not None:
            os.sched_setaffinity(0, self.saved)


def measure_configs(dev, with_oracle: bool, reps: int = 50, reps_big: int = 20) -> dict:
    """Every workload config, each layer chained as in the parity tests:
    median and interquartile range of the whole pass (build + sample + query
    of every layer) between two events after a GPU-side delay, the median of
    each call bracketed on its own (which adds the events' overhead), a
    replay of the pass captured in a HIP graph where no layer waits on the
    host, points/s, and algorithmic bytes per pass (per cloud and layer:
    12N (+4N with weights) + 20S + 24|O_v| + 16MK + 28M, S the stored points)
    over the median time. The oracle runs the same pass on one core."""
    import torch
    from paper_1912_02984_amd import cagq
    from paper_1912_02984_amd import workloads as W

    def ev():
        return torch.cuda.Event(enable_timing=True)

    out_all = {}
    for name in CONFIGS:
        w = W.get_workload(name)
        P_np = w.points()
        B, N = P_np.shape[0], P_np.shape[1]
        P = torch.from_numpy(P_np).to(dev)
        plan, n = [], N
        for L in w.layers:
            desc = cagq.desc_from_spec(L.grid)
            lay = cagq.workspace_layout(B, n, desc)
            plan.append((L, desc, torch.empty(lay.total_bytes, dtype=torch.uint8, device=dev),
                         cagq.alloc_query_outputs(B, L.M, L.K, dev), torch.empty((B, L.M), dtype=torch.int32, device=dev),
                         torch.empty((B,), dtype=torch.int32, device=dev)))
            n = L.M
        grids = []

        def run(marks=None):
            grids.clear()
            pts, wts = P, None
            for (L, desc, ws, out, cl, mv) in plan:
                g = cagq.build_grid(pts, desc, ws)
                if marks is not None:
                    marks.append(ev()); marks[-1].record()
                cagq.sample_centers(g, L.M, L.sample, L.seed, center_lin=cl, m_valid=mv)
                if marks is not None:
                    marks.append(ev()); marks[-1].record()
                cagq.query_context(g, cl, L.K, L.query, L.seed, weights=wts, out=out)
                if marks is not None:
                    marks.append(ev()); marks[-1].record()
                grids.append(g)
                pts, wts = out["center_xyz"], out["center_w"]

        for _ in range(5):
            run()
        torch.cuda.synchronize()
        nrep = reps_big if N * B > 1_000_000 else reps
        pairs = []
        for _ in range(nrep):
            a, b = ev(), ev()
            torch.cuda._sleep(SLEEP_CYCLES)
            a.record()
            run()
            b.record()
            pairs.append((a, b))
        torch.cuda.synchronize()
        tot = np.array([a.elapsed_time(b) for a, b in pairs])
        # per call, each bracketed by events
        calls = []
        for _ in range(max(5, nrep // 4)):
            marks = [ev()]
            torch.cuda._sleep(SLEEP_CYCLES)
            marks[0].record()
            run(marks)
            calls.append(marks)
        torch.cuda.synchronize()
        d = np.array([[m[i].elapsed_time(m[i + 1]) for i in range(len(m) - 1)] for m in calls])
        med = np.median(d, axis=0)
        layers = []
        alg = 0
        for li, (L, desc, ws, out, cl, mv) in enumerate(plan):
            tb = grids[li].table()
            nv = tb["nvox"].cpu().numpy().astype(np.int64)
            S = np.array([int(tb["vox_off"][b_, int(nv[b_])]) for b_ in range(B)], np.int64)
            n_in = N if li == 0 else plan[li - 1][0].M
            per = 12 * n_in + (4 * n_in if li > 0 else 0) + 20 * S + 24 * nv + 16 * L.M * L.K + 28 * L.M
            alg += int(per.sum())
            layers.append({"sample": L.sample, "query": L.query, "M": L.M, "K": L.K,
                           "build_ms": round(float(med[3 * li]), 4), "sample_ms": round(float(med[3 * li + 1]), 4),
                           "query_ms": round(float(med[3 * li + 2]), 4)})
            if L.sample == "cas":  # greedy picks (one per step) over the sampling time
                steps = int(mv.sum().item())
                layers[-1]["cas_steps"] = steps
                layers[-1]["cas_steps_per_s"] = round(steps / (float(med[3 * li + 1]) / 1e3), 1)
        t_med = float(np.median(tot))
        row = {"B": B, "N": N, "layers": layers, "ms_median": round(t_med, 4),
               "ms_iqr": [round(float(np.percentile(tot, 25)), 4), round(float(np.percentile(tot, 75)), 4)],
               "reps": nrep, "points_per_s": round(B * N / (t_med / 1e3), 1), "alg_bytes": alg,
               "alg_gbs": round(alg / (t_med / 1e3) / 1e9, 1)}
        # a HIP graph of the pass, where nothing in it waits on the host
        host_rounds = any(L.sample == "cas" and n_l > 4096
                          for L, n_l in zip(w.layers, [N] + [L.M for L in w.layers[:-1]]))
        if not host_rounds:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=side):
                run()
            torch.cuda.synchronize()
            pairs = []
            for _ in range(nrep):
                a, b = ev(), ev()
                torch.cuda._sleep(SLEEP_CYCLES)
                a.record()
                gr.replay()
                b.record()
                pairs.append((a, b))
            torch.cuda.synchronize()
            row["graph_ms_median"] = round(float(np.median([a.elapsed_time(b) for a, b in pairs])), 4)
            del gr
        if with_oracle and name not in ("bigroom/cas-knn", "bigroom/rvs-cube"):
            import oracle
            times = []
            with _OneCore():
                for _ in range(3 if B * N <= 100_000 else 1):
                    t0 = time.perf_counter()
                    pts, wts = P_np, None
                    for L in w.layers:
                        _, ocl, omv, oq = oracle.run_layer(pts, L, weights=wts)
                        pts, wts = oq["center_xyz"], oq["center_w"]
                    times.append(time.perf_counter() - t0)
            row["oracle_ms"] = round(float(np.median(times)) * 1e3, 2)
            row["oracle_cores"] = 1
        out_all[name] = row
        del plan, grids
        torch.cuda.synchronize()
    return out_all


def profile_workload(name: str, passes: int, dev) -> None:
    """Every layer of one workload config, chained as in the parity tests,
    passes times after a warm-up pass (for kernel traces and counters of one
    config alone)."""
    import torch
    from paper_1912_02984_amd import cagq
    from paper_1912_02984_amd import workloads as W
    w = W.get_workload(name)
    P = torch.from_numpy(w.points()).to(dev)
    B = P.shape[0]
    plan, n = [], w.N
    for L in w.layers:
        desc = cagq.desc_from_spec(L.grid)
        lay = cagq.workspace_layout(B, n, desc)
        plan.append((L, desc, torch.empty(lay.total_bytes, dtype=torch.uint8, device=dev),
                     cagq.alloc_query_outputs(B, L.M, L.K, dev)))
        n = L.M

    def run():
        pts, wts = P, None
        for (L, desc, ws, out) in plan:
            g = cagq.build_grid(pts, desc, ws)
            cl, _ = cagq.sample_centers(g, L.M, L.sample, L.seed)
            cagq.query_context(g, cl, L.K, L.query, L.seed, weights=wts, out=out)
            pts, wts = out["center_xyz"], out["center_w"]
    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(passes):
        run()
    e1.record()
    torch.cuda.synchronize()
    print(json.dumps({"workload": name, "passes": passes, "ms_per_pass": round(e0.elapsed_time(e1) / passes, 4)}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=4)
    ap.add_argument("--variants", default="both", choices=["both", "cas-knn", "rvs-cube"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum oracle time to accumulate for the CPU baseline")
    ap.add_argument("--rvs-after-layer", type=int, default=2,
                    help="a step issues RVS+cube once CAS+kNN has enqueued this layer's sampling (0-3)")
    ap.add_argument("--no-graph", action="store_true",
                    help="issue every kernel one by one instead of replaying the captured graphs of the layers that do not wait on the host")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the timing of every workload config")
    ap.add_argument("--no-next", action="store_true",
                    help="skip the measurement of the rows beyond the hot path")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run one fp32 copy kernel of known size first (counter calibration)")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("STATS_CSV", "COMMAND"),
                    help="print a markdown table of a rocprofv3 kernel summary and exit")
    ap.add_argument("--summarize-counters", metavar="COUNTER_CSV",
                    help="print a markdown table of a rocprofv3 --pmc collection per kernel and exit")
    ap.add_argument("--layer1-passes", type=int, default=0,
                    help="profiling mode: run only layer 1 (build + sample + query) of the selected variants "
                         "this many times after one warm-up pass, then exit (for the counter and trace runs "
                         "behind the layer roofline)")
    ap.add_argument("--profile-workload", metavar="NAME",
                    help="profiling mode: run every layer of one workload config (tiny, object, room, "
                         "bigroom/cas-knn, bigroom/rvs-cube, lidar) --layer1-passes times (default 10) after "
                         "one warm-up pass, then exit")
    ap.add_argument("--summarize-layer", nargs=5, metavar=("VARIANT", "FETCH_CSV", "WRITE_CSV", "TRACE_CSV", "PASSES"),
                    help="per-kernel time and HBM bytes of a --layer1-passes run, and their sums per pass")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the query kernels' HBM bytes from two counter passes and exit")
    args = ap.parse_args()
    if args.summarize_stats:
        print(summarize_stats(*args.summarize_stats), end="")
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters), end="")
        return
    if args.summarize_traffic:
        print(summarize_traffic(*args.summarize_traffic), end="")
        return
    if args.summarize_layer:
        v, f, w_, t, n = args.summarize_layer
        print(summarize_layer(v, f, w_, t, int(n)), end="")
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the CAGQ path here is single-GPU; see the sharding notes in the design document)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1912_02984_amd import cagq
    from paper_1912_02984_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.profile_workload:
        profile_workload(args.profile_workload, args.layer1_passes or 10, dev)
        return
    variants = VARIANTS if args.variants == "both" else (f"bigroom/{args.variants}",)
    wls = [W.get_workload(v) for v in variants]
    B = args.batch
    N = wls[0].N
    P_np = wls[0].points(B=B)
    P = torch.from_numpy(P_np).to(dev)

    # per variant, per layer: workspace and outputs, allocated once
    plans = []
    for w in wls:
        layers = []
        n = N
        for L in w.layers:
            desc = cagq.desc_from_spec(L.grid)
            lay = cagq.workspace_layout(B, n, desc)
            ws = torch.empty(lay.total_bytes, dtype=torch.uint8, device=dev)
            out = cagq.alloc_query_outputs(B, L.M, L.K, dev)
            cl = torch.empty((B, L.M), dtype=torch.int32, device=dev)
            mv = torch.empty((B,), dtype=torch.int32, device=dev)
            layers.append((L, desc, ws, out, cl, mv))
            n = L.M
        plans.append((w, layers))

    # the two variants are independent: each runs on its own stream (default
    # priority) and a step ends when both have finished
    streams = [torch.cuda.Stream() for _ in plans]
    q_events = []  # (variant, start, end) around layer-1 query launches

    grids_of = {}  # variant -> the grid records of its last pass, by layer

    def run_variant(plan, record=False, hook=None, hook_layer=-1, first=0, last=None, query_before=False,
                    query_last=True):
        """Layers [first, last) of a variant; a later layer reads the
        previous layer's outputs, which stay at fixed addresses. With
        query_before, the query of layer first - 1 comes first (its grid and
        centers are already in place); without query_last, the last layer
        stops after its sampling."""
        w, layers = plan
        if query_before and first > 0:
            Lq, _, _, outq, clq, _ = layers[first - 1]
            wq = layers[first - 2][3]["center_w"] if first >= 2 else None
            cagq.query_context(grids_of[w.name][first - 1], clq, Lq.K, Lq.query, Lq.seed, weights=wq, out=outq)
        if first == 0:
            pts, wts = P, None
        else:
            prev = layers[first - 1][3]
            pts, wts = prev["center_xyz"], prev["center_w"]
        end = len(layers) if last is None else last
        for li in range(first, end):
            L, desc, ws, out, cl, mv = layers[li]
            g = cagq.build_grid(pts, desc, ws)
            grids_of.setdefault(w.name, {})[li] = g
            cagq.sample_centers(g, L.M, L.sample, L.seed, center_lin=cl, m_valid=mv)
            if li == hook_layer and hook is not None:
                hook()
            if not query_last and li == end - 1:
                break
            if record and li == 0:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                # a bounded GPU-side delay first: the host enqueues the start
                # event, QUERY_REPS identical launches and the end event while
                # the stream is still busy, so the events bracket the kernels
                # alone, back to back, and not the host's time to issue them
                torch.cuda._sleep(SLEEP_CYCLES)
                e0.record()
                for _ in range(QUERY_REPS - 1):
                    cagq.query_context(g, cl, L.K, L.query, L.seed, weights=wts, out=out)
            cagq.query_context(g, cl, L.K, L.query, L.seed, weights=wts, out=out)
            if record and li == 0:
                e1.record()
                q_events.append((w.name, e0, e1))
            pts, wts = out["center_xyz"], out["center_w"]

    if args.layer1_passes:
        if args.copy_probe:
            src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            torch.mul(src, 1.0, out=dst)
            torch.cuda.synchronize()
            del src, dst
        sizes = {}
        for plan in plans:
            run_variant(plan, last=1)  # warm-up (not counted by the summaries, which take the last passes)
            torch.cuda.synchronize()
            for _ in range(args.layer1_passes):
                run_variant(plan, last=1)
            torch.cuda.synchronize()
            tb = grids_of[plan[0].name][0].table()
            nv = tb["nvox"].cpu().numpy().astype(np.int64)
            sizes[plan[0].name] = {"nvox": int(nv.sum()),
                                   "S": int(sum(int(tb["vox_off"][b, int(nv[b])]) for b in range(B)))}
        print(json.dumps({"layer1_passes": args.layer1_passes, "sizes": sizes}), flush=True)
        return

    def host_layers(w):
        """Leading layers whose sampling waits on the host: CAS outside the
        single-workgroup kernel (more than 4096 points or r > 2) issues its
        rounds from the host until every cloud is done."""
        n, k = N, 0
        for li, L in enumerate(w.layers):
            if L.sample == "cas" and not (n <= 4096 and L.grid.radius in (1, 2)):
                k = li + 1
            n = L.M
        return k

    # The layers after the last one that waits on the host only enqueue
    # kernels, so they are captured once in a HIP graph (kernel launches only)
    # and a step replays it: one launch from the host instead of ~10 per layer
    # (all of RVS+cube; layers 3-4 of CAS+kNN)
    graphs = {}
    if not args.no_graph:
        for i, (w, layers) in enumerate(plans):
            t = host_layers(w)
            if t >= len(layers):
                continue
            with torch.cuda.stream(streams[i]):
                run_variant(plans[i])  # eager once, outside the capture
            torch.cuda.synchronize()
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=streams[i]):
                # the query of the last layer that waits on the host goes
                # into the graph too: one launch fewer from the host between
                # that layer's rounds and the graph
                run_variant(plans[i], first=t, query_before=True)
            torch.cuda.synchronize()
            graphs[i] = (t, gr)

    def run_planned(i, hook=None, hook_layer=-1):
        """A variant as a step runs it: its host-driven layers eagerly, the
        rest from its graph."""
        t, gr = graphs.get(i, (len(plans[i][1]), None))
        run_variant(plans[i], hook=hook, hook_layer=hook_layer, last=t, query_last=gr is None)
        if gr is not None:
            gr.replay()
            if hook is not None and hook_layer >= t:
                hook()

    def step():
        main = torch.cuda.current_stream()
        start = torch.cuda.Event()
        start.record(main)
        for st in streams:
            st.wait_event(start)
        # CAS+kNN waits on the host for the rounds of its two large layers.
        # RVS+cube only enqueues; it is issued from inside CAS+kNN once a
        # layer's sampling is enqueued (by default the third layer's, which
        # comes with the graph of the last two: their single-workgroup CAS
        # holds four CUs for ~0.25 ms and RVS+cube's kernels fill the others,
        # where beside the large layers' rounds they delay each round's
        # launches)
        cas = [i for i in range(len(plans)) if plans[i][0].layers[0].sample != "rvs"]
        rvs = [i for i in range(len(plans)) if plans[i][0].layers[0].sample == "rvs"]

        def issue_rvs():
            for i in rvs:
                with torch.cuda.stream(streams[i]):
                    run_planned(i)

        if cas:
            with torch.cuda.stream(streams[cas[0]]):
                run_planned(cas[0], hook=issue_rvs, hook_layer=args.rvs_after_layer)
        else:
            issue_rvs()
        for st in streams:
            main.wait_stream(st)

    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t_ev0 = torch.cuda.Event(enable_timing=True)
    t_ev1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t_ev0.record()
    for _ in range(args.steps):
        step()
    t_ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t_ev0.elapsed_time(t_ev1) / args.steps
    points_per_s = B * N / (ms_step / 1e3)
    # what the timed steps left in the outputs: scene 0 of every layer of both
    # variants, checked against the oracle in the CPU leg below
    timed_out = {w.name: [(cl[0].cpu().numpy(), mv[:1].cpu().numpy(),
                           {k: v[0].cpu().numpy() for k, v in out.items() if v is not None})
                          for (L, desc, ws, out, cl, mv) in layers] for w, layers in plans}

    # per-variant times, one variant at a time on the default stream
    variant_ms = {}
    reps = max(5, args.steps // 2)
    for plan in plans:
        run_variant(plan)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            run_variant(plan)
        e1.record()
        torch.cuda.synchronize()
        variant_ms[plan[0].name] = e0.elapsed_time(e1) / reps
    # then passes whose layer-1 query runs QUERY_REPS times between events:
    # the roofline entry
    for plan in plans:
        for _ in range(ROOF_PASSES):
            run_variant(plan, record=True)
    torch.cuda.synchronize()

    # layer 1 of each variant as a whole (build + sample + query), between
    # events after a GPU-side delay
    l_events = []
    for plan in plans:
        for _ in range(ROOF_PASSES):
            a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(SLEEP_CYCLES)
            a.record()
            run_variant(plan, last=1)
            b_.record()
            l_events.append((plan[0].name, a, b_))
    torch.cuda.synchronize()

    # roofline of the layer-1 query kernel and of the whole layer, per variant
    roof, layer_roof = {}, {}
    layer_prof = load_layer_profile()
    for w, layers in plans:
        L, desc, ws, out, cl, mv = layers[0]
        tb = grids_of[w.name][0].table()
        nv = tb["nvox"].cpu().numpy().astype(np.int64)
        S_total = int(sum(int(tb["vox_off"][b, int(nv[b])]) for b in range(B)))
        durs = [a.elapsed_time(b) / QUERY_REPS for name, a, b in q_events if name == w.name]
        t_ms = float(np.mean(durs))
        ctx_total = int(out["ctx_count"].sum().item())
        alg = query_alg_bytes(B * L.M, L.K, S_total)
        reread = query_reread_bytes(B * L.M, L.K, ctx_total)
        gbs = alg / (t_ms / 1e3) / 1e9
        roof[w.name] = dict(kernel=f"k_query<{L.query}>", us=t_ms * 1e3, alg_bytes=alg, achieved_gbs=gbs,
                            S=S_total, ctx_total=ctx_total, reread_bytes=reread,
                            reread_gbs=reread / (t_ms / 1e3) / 1e9)
        l_ms = float(np.mean([a.elapsed_time(b) for name, a, b in l_events if name == w.name]))
        l_alg = layer_alg_bytes(B * N, S_total, int(nv.sum()), B * L.M, L.K, weights=False)
        ent = {"us": round(l_ms * 1e3, 2), "alg_bytes": l_alg,
               "achieved_gbs": round(l_alg / (l_ms / 1e3) / 1e9, 1),
               "frac": round(l_alg / (l_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
               "nvox": int(nv.sum()), "S": S_total}
        lp = layer_prof.get(w.name)
        if lp:  # kernel time and counter bytes of the same layer from the committed profile
            ent.update({"kernel_us_sum": lp["us"], "alg_gbs_over_kernel_sum": round(l_alg / lp["us"] / 1e3, 1),
                        "frac_over_kernel_sum": round(l_alg / lp["us"] / 1e3 / HBM_PEAK_GBS, 4),
                        "traffic": lp["bytes"], "traffic_gbs_over_kernel_sum": round(lp["bytes"] / lp["us"] / 1e3, 1),
                        "launches": lp["launches"]})
        layer_roof[w.name] = ent
    dom = max(roof.values(), key=lambda r: r["us"])
    traffic = load_traffic().get(dom["kernel"])
    # what a plain streaming copy reaches on this GPU, for context: a 1 GiB
    # fp32 copy (read + write), timed like the query
    src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    cps = []
    for _ in range(3):
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SLEEP_CYCLES)
        a.record()
        dst.copy_(src)
        b_.record()
        cps.append((a, b_))
    torch.cuda.synchronize()
    copy_gbs = 2 * COPY_PROBE_BYTES / (min(a.elapsed_time(b_) for a, b_ in cps) / 1e3) / 1e9
    del src, dst
    roofline = {"bound": "hbm", "achieved": round(dom["achieved_gbs"], 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(dom["achieved_gbs"] / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": dom["kernel"], "launch_us": round(dom["us"], 2), "alg_bytes": dom["alg_bytes"],
                "copy_gbs": round(copy_gbs, 1),
                "per_variant": {k: {kk: (round(vv, 3) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                                for k, v in roof.items()},
                "layer": layer_roof}

    # rows beyond the hot path, measured on the layer-1 grid of the same batch
    next_rows = None
    if not args.no_next:
        next_rows = {"cas_swap": measure_cas_swap(P, P_np, B, N, wls[0].layers[0], with_oracle=not args.no_cpu_baseline)}
        next_rows.update(measure_upsampling(P, P_np, B, N, wls[0], with_oracle=not args.no_cpu_baseline))
        next_rows["knn_ring"] = measure_knn_ring(P, P_np, B, N, wls[0], with_oracle=not args.no_cpu_baseline)
        next_rows["coverage"] = measure_coverage(P, B, N, wls[0])

    # every workload config (the C4 step above is the headline)
    configs = None
    if not args.no_configs:
        configs = measure_configs(dev, with_oracle=not args.no_cpu_baseline)
        configs["host"] = _host_info()

    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle
        pin = _OneCore()
        pin.__enter__()
        t0 = time.perf_counter()
        done = 0
        mismatch = []
        while True:
            for w in wls:
                pts, wts = P_np[:1], None
                for li, L in enumerate(w.layers):
                    _, ocl, omv, q = oracle.run_layer(pts, L, weights=wts)
                    if done == 0:  # the timed step's scene 0, element by element (floats as bits)
                        gcl, gmv, gq = timed_out[w.name][li]
                        same = np.array_equal(gcl, ocl[0]) and np.array_equal(gmv, omv)
                        for k, v in gq.items():
                            o = q[k][0]
                            same = same and np.array_equal(np.ascontiguousarray(v).view(np.uint32),
                                                           np.ascontiguousarray(o).view(np.uint32))
                        if not same:
                            mismatch.append(f"{w.name} layer {li + 1}")
                    pts, wts = q["center_xyz"], q["center_w"]
            done += 1
            if time.perf_counter() - t0 >= args.cpu_seconds or done >= 32:
                break
        dt = time.perf_counter() - t0
        pin.__exit__(None, None, None)
        cpu = {"value": round(done * N / dt, 1), "unit": "points/s", "cores": 1, "kind": "oracle",
               "sample": f"{done} pass(es) of the same hot path (all layers, "
                         f"{'both variants' if len(wls) == 2 else variants[0]}) over 1 of the {B} scenes, "
                         f"single-threaded C oracle pinned to {pin.where}, {dt:.1f} s",
               **_host_info()}
        parity = {"checked": "the timed step's outputs for scene 0, every layer of "
                             f"{' and '.join(w.name for w in wls)}, vs the oracle's timed pass",
                  "bit_exact": not mismatch, "mismatch": mismatch}

    line = {
        "metric": METRIC,
        "value": round(points_per_s, 1),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"indoor scenes B={B} x {N} pts, 4 layers "
                               f"(M=8192/2048/512/128, K=32, n_v=32), "
                               + (" and ".join(v.split('/')[1] for v in variants)),
                   "global_batch": B, "points_per_scene": N},
        "variant_ms": {k: round(v, 4) for k, v in variant_ms.items()},
        "wall_s": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity": parity,
        "next_rows": next_rows,
        "configs": configs,
    }
    print(json.dumps(line), flush=True)
    if parity is not None and not parity["bit_exact"]:
        print(f"bench.py: the timed step differs from the oracle: {parity['mismatch']}", file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
