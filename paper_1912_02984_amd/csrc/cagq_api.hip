// C ABI of the gfx950 CAGQ library (declared in include/cagq.h): argument
// validation on the host, workspace layout, and the launch sequence of each
// step. Every argument error is returned before anything is enqueued.
#include <math.h>
#include <string.h>

#include <mutex>

#include <vector>

#include "cagq_internal.h"

namespace cagq {

// The workspace of cagq_build_grid_static: one array per GPU, resident from
// the library's load until the process ends. Host code never uses the
// array's name as an address (on the host it is only a stand-in for the
// symbol): its device address comes from hipGetSymbolAddress, once per
// device.
constexpr size_t kStaticScratchBytes = CAGQ_STATIC_WORKSPACE_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;

// The device address of the current device's array, or null on failure.
static void* static_scratch() {
    static std::mutex mu;
    static void* ptr[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        ptr[dev] = p;
    }
    return ptr[dev];
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static int check_desc(const cagq_grid_desc* d) {
    if (!d) return CAGQ_ERR_INVALID_ARG;
    int64_t v = 1;
    for (int a = 0; a < 3; ++a) {
        if (d->dims[a] < 1) return CAGQ_ERR_INVALID_ARG;
        if (!(d->voxel_size[a] > 0.0f) || !isfinite(d->voxel_size[a])) return CAGQ_ERR_INVALID_ARG;
        if (!isfinite(d->origin[a])) return CAGQ_ERR_INVALID_ARG;
        v *= d->dims[a];
        if (v > 2147483647LL) return CAGQ_ERR_GRID_TOO_LARGE;
    }
    if (d->n_v < 1 || d->n_v > CAGQ_MAX_NV) return CAGQ_ERR_INVALID_ARG;
    if (d->radius < 1 || d->radius > CAGQ_MAX_RADIUS) return CAGQ_ERR_INVALID_ARG;
    return CAGQ_OK;
}

bool make_layout(int32_t B, int32_t N, const cagq_grid_desc* d, Layout* L) {
    if (B < 1 || N < 1 || (int64_t)B * N > 2147483647LL) return false;
    memset(L, 0, sizeof(*L));
    L->B = B;
    L->N = N;
    L->V = (int64_t)d->dims[0] * d->dims[1] * d->dims[2];
    L->W = (L->V + 63) / 64;
    L->tiles_w = (L->W + kRankTile - 1) / kRankTile;
    L->tiles_s = ((int64_t)N + kScanTile - 1) / kScanTile;
    L->big_cap = (int64_t)B * N / (kBigVoxel + 1) + 1;
    const size_t BN = (size_t)B * N;
    L->Q = (int32_t)((L->W + kBrickW - 1) / kBrickW);
    L->T = (int32_t)(((int64_t)B * N + kSortTile - 1) / kSortTile);
    // the histogram matrix (B * Q by T entries) stays within 2^24 entries
    L->bricks = (int64_t)B * L->Q <= kMaxBricks && (int64_t)B * L->Q * L->T <= (int64_t(1) << 24);
    // a cloud's points span at most ceil(N / kSortTile) + 1 tiles
    L->tile_scan = L->bricks && ((int64_t)(N + kSortTile - 1) / kSortTile + 1) * L->Q <= kTileScanCap;
    const size_t BQ = L->bricks ? (size_t)B * L->Q : 0;
    const size_t hist_n = BQ * (size_t)L->T;
    L->items_max = L->bricks ? (int64_t)BQ + ((int64_t)BN + kBrickCap - 1) / kBrickCap : 0;
    L->heavy_max = L->bricks ? (int64_t)BN / (kBrickCap + 1) : 0;
    const size_t H = (size_t)L->heavy_max;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align256(off + bytes);
        return o;
    };
    L->nvox = take(4 * (size_t)B);
    L->vox_lin = take(4 * BN);
    L->vox_count = take(4 * BN);
    L->vox_off = take(4 * (size_t)B * (N + 1));
    L->pt_list = take(4 * BN);
    L->status = take(4 * kStSlots);
    L->berr = take(4 * (size_t)B);
    L->sel_ghist = take(4 * (size_t)B * kSelBins);
    L->sel_cnt = take(4 * (size_t)B);
    L->clear_small = off;
    L->desc_h = take(8 * ((BQ + 63) / 64));
    L->hdone = take(4 * (L->bricks ? (size_t)BN / (kBrickCap + 1) : 0));
    L->clear_brick = off;
    // the occupancy bytes and rank descriptors serve the many-kernel build of
    // grids too large for the bricks only
    L->desc_w = take(L->bricks ? 0 : 8 * (size_t)B * L->tiles_w);
    L->desc_s = take(8 * (size_t)B * L->tiles_s);
    L->bytemap = take(L->bricks ? 0 : 64 * (size_t)B * L->W);
    L->clear_end = off;
    L->bitmap = take(8 * (size_t)B * L->W);
    L->word_rank = take(4 * (size_t)B * L->W);
    L->pt_slot = take(4 * BN);
    L->pt_pos = take(4 * BN);
    L->hist = take(4 * hist_n);
    L->bstart = take(4 * BQ);
    L->brick_hb = take(4 * BQ);
    L->item_extra = take(8 * ((size_t)L->items_max - BQ));
    L->agg = take(8 * BQ);
    L->hlist = take(4 * H);
    L->hebase = take(4 * H);
    L->pcnt = take(4 * ((size_t)L->items_max - BQ) * kBrickV);

    L->hfo = take(4 * H * (kBrickV + 1));
    L->hso = take(4 * H * kBrickV);
    L->hpre = take(8 * H);
    L->sorted = take(L->bricks ? 16 * BN : 0);
    L->full_off = take(L->bricks ? 0 : 4 * (size_t)B * (N + 1));
    L->bucket = take(4 * BN);
    L->pt4 = take(16 * BN);
    L->big = take(L->bricks ? 0 : 4 * (size_t)L->big_cap);
    L->cas_cover = take(4 * BN);
    L->cas_key = take(8 * BN);
    L->cas_pick = take(8 * BN);
    L->cas_round = take(4 * BN);
    L->cas_blocker = take(4 * BN);
    L->cas_dirty = take(4 * BN);
    L->cas_ctl = take(CasCtl::bytes(B));
    L->has_nbr16 = N <= kCasLdsMaxN && d->radius <= 2;
    L->has_nbr32 = N > kCasLdsMaxN && d->radius == 1;
    L->cas_nbr = take(L->has_nbr16 ? 2 * BN * (size_t)nbr_stride(d->radius) : 0);
    L->cas_nbr32 = take(L->has_nbr32 ? 4 * BN * (size_t)kNbr32Stride : 0);
    L->sel_thr = take(8 * (size_t)B);
    const size_t sel_chunks = ((size_t)N + kSelChunk - 1) / kSelChunk;
    L->sel_keys = take(4 * (size_t)B * sel_chunks * kSelChunk);
    L->sel_bins = take(4 * (size_t)B * sel_chunks * kSelBins);
    L->sel_base = take(4 * (size_t)B * sel_chunks);
    L->sel_take = take(4 * (size_t)B * sel_chunks);
    L->cov_mark = take((BN + 15) / 16 * 16);
    L->total = off;
    return true;
}

static int grid_layout(const cagq_grid* g, Layout* L) {
    if (!g || !g->points || !g->workspace) return CAGQ_ERR_INVALID_ARG;
    int rc = check_desc(&g->desc);
    if (rc != CAGQ_OK) return rc;
    if (!make_layout(g->B, g->N, &g->desc, L)) return CAGQ_ERR_INVALID_ARG;
    if (g->workspace_bytes < L->total) return CAGQ_ERR_WORKSPACE_TOO_SMALL;
    return CAGQ_OK;
}

}  // namespace cagq

using namespace cagq;

extern "C" {

// The box [lo, hi] must be finite and not inverted on any axis.
static int check_box(const float* lo, const float* hi) {
    if (!lo || !hi) return CAGQ_ERR_INVALID_ARG;
    for (int a = 0; a < 3; ++a)
        if (!isfinite(lo[a]) || !isfinite(hi[a]) || !(lo[a] <= hi[a])) return CAGQ_ERR_INVALID_ARG;
    return CAGQ_OK;
}

int cagq_desc_from_voxel_size(const float lo[3], const float hi[3], const float vs[3], int32_t n_v, int32_t radius,
                              cagq_grid_desc* out) {
    int rc = check_box(lo, hi);
    if (rc != CAGQ_OK) return rc;
    if (!vs || !out) return CAGQ_ERR_INVALID_ARG;
    cagq_grid_desc d;
    for (int a = 0; a < 3; ++a) {
        if (!(vs[a] > 0.0f) || !isfinite(vs[a])) return CAGQ_ERR_INVALID_ARG;
        // the voxelize rule applied to hi: one rounded subtract, one
        // correctly rounded divide (the host compiler keeps fp32 here)
        const volatile float diff = hi[a] - lo[a];
        const volatile float t = diff / vs[a];
        const float f = floorf(t);
        if (!isfinite(t) || f >= 2147483647.0f) return CAGQ_ERR_GRID_TOO_LARGE;
        d.origin[a] = lo[a];
        d.voxel_size[a] = vs[a];
        d.dims[a] = (int32_t)f + 1;
    }
    d.n_v = n_v;
    d.radius = radius;
    rc = check_desc(&d);
    if (rc == CAGQ_OK) *out = d;
    return rc;
}

int cagq_desc_from_dims(const float lo[3], const float hi[3], const int32_t dims[3], int32_t n_v, int32_t radius,
                        cagq_grid_desc* out) {
    int rc = check_box(lo, hi);
    if (rc != CAGQ_OK) return rc;
    if (!dims || !out) return CAGQ_ERR_INVALID_ARG;
    cagq_grid_desc d;
    for (int a = 0; a < 3; ++a) {
        if (dims[a] < 1) return CAGQ_ERR_INVALID_ARG;
        const volatile float diff = hi[a] - lo[a];
        const volatile float s = diff / (float)dims[a];
        d.origin[a] = lo[a];
        d.voxel_size[a] = diff == 0.0f ? 1.0f : s;
        d.dims[a] = dims[a];
    }
    d.n_v = n_v;
    d.radius = radius;
    rc = check_desc(&d);
    if (rc == CAGQ_OK) *out = d;
    return rc;
}

int cagq_workspace_layout(int32_t B, int32_t N, const cagq_grid_desc* desc, cagq_layout* out) {
    if (!out) return CAGQ_ERR_INVALID_ARG;
    int rc = check_desc(desc);
    if (rc != CAGQ_OK) return rc;
    Layout L;
    if (!make_layout(B, N, desc, &L)) return CAGQ_ERR_INVALID_ARG;
    out->total_bytes = L.total;
    out->nvox = L.nvox;
    out->vox_lin = L.vox_lin;
    out->vox_count = L.vox_count;
    out->vox_off = L.vox_off;
    out->pt_list = L.pt_list;
    return CAGQ_OK;
}

int cagq_build_grid(const float* points, int32_t B, int32_t N, const cagq_grid_desc* desc,
                    void* workspace, size_t workspace_bytes, void* stream, cagq_grid* out) {
    if (!points || !workspace || !out) return CAGQ_ERR_INVALID_ARG;
    if (((uintptr_t)workspace & 255u) != 0) return CAGQ_ERR_INVALID_ARG;
    int rc = check_desc(desc);
    if (rc != CAGQ_OK) return rc;
    Layout L;
    if (!make_layout(B, N, desc, &L)) return CAGQ_ERR_INVALID_ARG;
    if (workspace_bytes < L.total) return CAGQ_ERR_WORKSPACE_TOO_SMALL;
    out->B = B;
    out->N = N;
    out->desc = *desc;
    out->points = points;
    out->workspace = workspace;
    out->workspace_bytes = workspace_bytes;
    hipError_t e = launch_build(points, L, *desc, workspace, (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_build_grid_static(const float* points, int32_t B, int32_t N, const cagq_grid_desc* desc, void* stream,
                           cagq_grid* out) {
    if (!points || !out) return CAGQ_ERR_INVALID_ARG;
    int rc = check_desc(desc);
    if (rc != CAGQ_OK) return rc;
    Layout L;
    if (!make_layout(B, N, desc, &L)) return CAGQ_ERR_INVALID_ARG;
    if (L.total > kStaticScratchBytes) return CAGQ_ERR_WORKSPACE_TOO_SMALL;
    void* ws = static_scratch();
    if (!ws) return CAGQ_ERR_HIP;
    out->B = B;
    out->N = N;
    out->desc = *desc;
    out->points = points;
    out->workspace = ws;
    out->workspace_bytes = kStaticScratchBytes;
    hipError_t e = launch_build(points, L, *desc, ws, (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_sample_centers(const cagq_grid* g, int32_t M, int32_t mode, uint64_t seed, uint32_t beta_q16,
                        int32_t* center_lin, int32_t* m_valid, void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (M < 1 || (int64_t)g->B * M > 2147483647LL || !center_lin || !m_valid) return CAGQ_ERR_INVALID_ARG;
    if (mode == CAGQ_SAMPLE_RVS) {
        hipError_t e = launch_select(L, g->workspace, M, 0, seed, center_lin, m_valid, (hipStream_t)stream);
        return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
    }
    if (mode == CAGQ_SAMPLE_CAS_SWAP) {  // 64-bit comparisons: no range limit on beta
        if (!cas_swap_fits(L, g->desc, M)) return CAGQ_ERR_CAPACITY;
        hipError_t e = launch_cas_swap(L, g->desc, g->workspace, M, seed, beta_q16, center_lin, m_valid,
                                       (hipStream_t)stream);
        return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
    }
    if (mode != CAGQ_SAMPLE_CAS) return CAGQ_ERR_INVALID_ARG;
    const int64_t side = 2 * (int64_t)g->desc.radius + 1;
    const int64_t lam = side * side * side;
    if ((65536LL + (int64_t)beta_q16) * lam * lam >= 2147483648LL) return CAGQ_ERR_INVALID_ARG;
    if (cas_lds_fits(L, g->desc, beta_q16)) {
        hipError_t e = launch_cas_lds(L, g->desc, g->workspace, M, center_lin, m_valid, (hipStream_t)stream);
        return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
    }
    int status = CAGQ_OK;
    hipError_t e = run_cas(L, g->desc, g->workspace, M, beta_q16, (hipStream_t)stream, &status);
    if (e != hipSuccess) return CAGQ_ERR_HIP;
    if (status != CAGQ_OK) return status;
    e = launch_select_cas(L, g->desc, g->workspace, M, beta_q16, center_lin, m_valid, (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_query_context(const cagq_grid* g, const uint32_t* weights, const int32_t* center_lin, int32_t M,
                       int32_t K, int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                       int32_t* n_valid, float* center_xyz, uint32_t* center_w, int32_t* ctx_count,
                       void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (M < 1 || (int64_t)g->B * M > 2147483647LL) return CAGQ_ERR_INVALID_ARG;
    if (K < 1 || K > CAGQ_MAX_K) return CAGQ_ERR_INVALID_ARG;
    if (mode != CAGQ_QUERY_CUBE && mode != CAGQ_QUERY_KNN && mode != CAGQ_QUERY_KNN_RING) return CAGQ_ERR_INVALID_ARG;
    if (!center_lin || !node_idx || !n_valid || !center_xyz || !center_w) return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_query(L, g->desc, g->points, g->workspace, weights, center_lin, M, K, mode, seed,
                                node_idx, node_xyz, n_valid, center_xyz, center_w, ctx_count,
                                (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_query_points(const cagq_grid* g, const float* centers, int32_t M, int32_t K, int32_t mode, uint64_t seed,
                      int32_t* node_idx, float* node_xyz, int32_t* n_valid, int32_t* ctx_count,
                      int32_t* center_lin, void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (M < 1 || (int64_t)g->B * M > 2147483647LL) return CAGQ_ERR_INVALID_ARG;
    if (K < 1 || K > CAGQ_MAX_K) return CAGQ_ERR_INVALID_ARG;
    if (mode != CAGQ_QUERY_CUBE && mode != CAGQ_QUERY_KNN && mode != CAGQ_QUERY_KNN_RING) return CAGQ_ERR_INVALID_ARG;
    if (!centers || !node_idx || !n_valid) return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_query_points(L, g->desc, g->workspace, centers, M, K, mode, seed, node_idx, node_xyz,
                                       n_valid, ctx_count, center_lin, (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_context_offsets(const cagq_grid* g, const int32_t* center_lin, int32_t M, int64_t* ctx_off,
                         void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (M < 1 || (int64_t)g->B * M > 2147483647LL) return CAGQ_ERR_INVALID_ARG;
    if (!center_lin || !ctx_off) return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_context_offsets(L, g->desc, g->workspace, center_lin, M, ctx_off, (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_context_list(const cagq_grid* g, const int32_t* center_lin, int32_t M, const int64_t* ctx_off,
                      int32_t* ctx_idx, int64_t capacity, void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (M < 1 || (int64_t)g->B * M > 2147483647LL) return CAGQ_ERR_INVALID_ARG;
    if (!center_lin || !ctx_off || capacity < 0 || (capacity > 0 && !ctx_idx)) return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_context_list(L, g->desc, g->workspace, center_lin, M, ctx_off, ctx_idx, capacity,
                                       (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_sample_points(const float* points, int32_t B, int32_t N, int32_t M, int32_t mode, uint64_t seed,
                       int32_t* center_idx, void* stream) {
    if (!points || !center_idx || B < 1 || N < 1 || (int64_t)B * N > 2147483647LL) return CAGQ_ERR_INVALID_ARG;
    if (M < 1 || M > N || (mode != CAGQ_POINTS_RPS && mode != CAGQ_POINTS_FPS)) return CAGQ_ERR_INVALID_ARG;
    if (mode == CAGQ_POINTS_FPS && N > kFpsMaxN) return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_sample_points(points, B, N, M, mode, seed, center_idx, (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_ball_query(const float* points, int32_t B, int32_t N, const int32_t* center_idx, int32_t M, int32_t K,
                    float radius2, int32_t* node_idx, int32_t* n_valid, void* stream) {
    if (!points || !center_idx || !node_idx || !n_valid) return CAGQ_ERR_INVALID_ARG;
    if (B < 1 || N < 1 || (int64_t)B * N > 2147483647LL || M < 1 || (int64_t)B * M > 2147483647LL)
        return CAGQ_ERR_INVALID_ARG;
    if (K < 1 || (int64_t)B * M * K > 2147483647LL || !(radius2 >= 0.0f) || radius2 == __builtin_inff())
        return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_ball_query(points, B, N, center_idx, M, K, radius2, node_idx, n_valid,
                                     (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_coverage(const cagq_grid* g, const int32_t* node_idx, const int32_t* n_valid, int32_t M, int32_t K,
                  int32_t* covered, void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (!node_idx || !n_valid || !covered || M < 1 || K < 1) return CAGQ_ERR_INVALID_ARG;
    if ((int64_t)g->B * M * K > 2147483647LL) return CAGQ_ERR_INVALID_ARG;
    hipError_t e = launch_coverage(L, g->desc, g->points, g->workspace, node_idx, n_valid, M, K, covered,
                                   (hipStream_t)stream);
    return e == hipSuccess ? CAGQ_OK : CAGQ_ERR_HIP;
}

int cagq_get_device_status(const cagq_grid* g, void* stream) {
    Layout L;
    int rc = grid_layout(g, &L);
    if (rc != CAGQ_OK) return rc;
    if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return CAGQ_ERR_HIP;
    // the build's per-cloud codes come first in the pipeline (only the
    // one-workgroup build writes them; every build leaves them at zero otherwise)
    std::vector<int> berr((size_t)L.B);
    if (hipMemcpy(berr.data(), at<int>(g->workspace, L.berr), sizeof(int) * (size_t)L.B, hipMemcpyDeviceToHost) !=
        hipSuccess)
        return CAGQ_ERR_HIP;
    for (int e : berr)
        if (e != 0) return e;
    int st = 0;
    if (hipMemcpy(&st, at<int>(g->workspace, L.status), sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
        return CAGQ_ERR_HIP;
    return st;
}

const char* cagq_status_string(int status) {
    switch (status) {
        case CAGQ_OK: return "ok";
        case CAGQ_ERR_INVALID_ARG: return "invalid argument";
        case CAGQ_ERR_GRID_TOO_LARGE: return "grid has more than 2^31-1 voxels";
        case CAGQ_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
        case CAGQ_ERR_NONFINITE_INPUT: return "non-finite input coordinate";
        case CAGQ_ERR_CAPACITY: return "internal capacity exceeded";
        case CAGQ_ERR_HIP: return "HIP runtime error";
        case CAGQ_ERR_CENTER_NOT_OCCUPIED: return "query center voxel is not occupied";
        default: return "unknown status";
    }
}

}  // extern "C"
