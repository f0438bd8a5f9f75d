// Voxelization and the occupied-voxel index (Appendix D, CAGQ general
// procedure, step 1; Sec. 3.2 "voxelize the input space ... map each point to
// a voxel index ... store up to n_v points in each voxel").
//
// Design (gfx950): the set O_v of non-empty voxels is an occupancy bitmap
// with one bit per grid voxel; a voxel's slot is its rank (popcount of the
// bits before it), which is a minimal, order-preserving hash of the linear
// voxel id to a compact slot. Points mark a byte per voxel with plain stores
// (no atomics); a single-pass decoupled look-back scan packs the bytes into
// bitmap words and ranks them; counts come from one atomic per point,
// offsets from a second look-back scan over the slots. Per-voxel lists hold
// the n_v lowest point indices in ascending order, independent of the
// arrival order the atomics produce: small voxels rank each point against
// the voxel's bucket, large voxels are reduced by a wavefront bitonic
// selection.
#include "cagq_internal.h"

namespace cagq {

namespace {

struct GridArgs {
    float o[3];
    float s[3];
    int32_t D[3];
};

GridArgs grid_args(const cagq_grid_desc& d) {
    GridArgs g;
    for (int a = 0; a < 3; ++a) {
        g.o[a] = d.origin[a];
        g.s[a] = d.voxel_size[a];
        g.D[a] = d.dims[a];
    }
    return g;
}

__global__ void k_clear(uint4* __restrict__ p, size_t n16) {
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// One lane per point: linear voxel id, occupancy byte.
__global__ __launch_bounds__(256) void k_mark(const float* __restrict__ P, int32_t N, int32_t BN,
                                              GridArgs g, int64_t W, uint32_t* __restrict__ pt_lin,
                                              uint8_t* __restrict__ bytemap, int* __restrict__ status) {
    int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    if (gid >= BN) return;
    int32_t b = gid / N;
    const float* p = P + (size_t)gid * 3;
    float c[3] = {p[0], p[1], p[2]};
    uint32_t gg[3];
    bool bad = false;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        if (!isfinite(c[a])) {
            bad = true;
            gg[a] = 0;
        } else {
            gg[a] = (uint32_t)axis_index(c[a], g.o[a], g.s[a], g.D[a]);
        }
    }
    uint32_t lin = gg[0] + (uint32_t)g.D[0] * (gg[1] + (uint32_t)g.D[1] * gg[2]);
    pt_lin[gid] = lin;
    // every point of a voxel stores the same byte: no atomic is needed
    bytemap[(size_t)b * W * 64 + lin] = 1;
    if (bad) raise_error(status, CAGQ_ERR_NONFINITE_INPUT);
}

// 64 occupancy bytes (each 0 or 1) to one occupancy word: byte j -> bit j.
// Multiplying 4 such bytes by 0x01020408 moves byte k to bit 24 + k with no
// other term reaching bits 24..31.
__device__ __forceinline__ uint64_t pack_bytes(const uint4* __restrict__ p) {
    uint64_t r = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint4 v = p[q];
        const uint32_t a[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) r |= (uint64_t)((a[k] * 0x01020408u) >> 24) << (16 * q + 4 * k);
    }
    return r;
}

// Occupancy words from the bytes, and their ranks: word_rank[w] = occupied
// voxels before word w. Also lists every occupied voxel's linear id at its
// slot and clears its count.
__global__ __launch_bounds__(kScanThreads) void k_rank(
    const uint8_t* __restrict__ bytemap, uint64_t* __restrict__ bitmap, int64_t W, int64_t tiles_w, int32_t N,
    uint32_t* __restrict__ word_rank, uint32_t* __restrict__ vox_lin, uint32_t* __restrict__ vox_count,
    int32_t* __restrict__ nvox, uint64_t* __restrict__ desc_w, int* __restrict__ status) {
    __shared__ uint32_t s_ticket;
    __shared__ uint64_t s_wave[kScanThreads / kWave];
    __shared__ uint64_t s_prefix;
    if (threadIdx.x == 0) s_ticket = atomicAdd((unsigned*)&status[kStTicketRank], 1u);
    __syncthreads();
    const uint32_t t = s_ticket;
    const int32_t b = (int32_t)(t / tiles_w);
    const int64_t tile = (int64_t)(t % tiles_w);
    const uint4* bytes = reinterpret_cast<const uint4*>(bytemap + (size_t)b * W * 64);
    uint64_t* bm = bitmap + (size_t)b * W;
    const int64_t w0 = tile * kRankTile + (int64_t)threadIdx.x * kRankItems;
    uint64_t words[kRankItems];
    uint32_t cnt = 0;
#pragma unroll
    for (int i = 0; i < kRankItems; ++i) {
        int64_t w = w0 + i;
        words[i] = w < W ? pack_bytes(bytes + (size_t)w * 4) : 0ull;
        if (w < W) bm[w] = words[i];
        cnt += (uint32_t)__popcll(words[i]);
    }
    uint64_t total;
    uint64_t excl = block_excl_scan(cnt, s_wave, &total);
    uint64_t prefix = tile_lookback(desc_w + (size_t)b * tiles_w, tile, total, &s_prefix);
    uint32_t r = (uint32_t)(prefix + excl);
    uint32_t* wr = word_rank + (size_t)b * W;
    uint32_t* vl = vox_lin + (size_t)b * N;
    uint32_t* vc = vox_count + (size_t)b * N;
#pragma unroll
    for (int i = 0; i < kRankItems; ++i) {
        int64_t w = w0 + i;
        if (w >= W) break;
        wr[w] = r;
        uint64_t m = words[i];
        while (m) {
            int bit = __ffsll((unsigned long long)m) - 1;
            vl[r] = (uint32_t)(w * 64 + bit);
            vc[r] = 0u;
            ++r;
            m &= m - 1;
        }
    }
    if (tile == tiles_w - 1 && threadIdx.x == 0) nvox[b] = (int32_t)(prefix + total);
}

// One lane per point: slot (rank of its voxel) and arrival position.
__global__ __launch_bounds__(256) void k_count(int32_t BN, int32_t N, int64_t W,
                                               const uint64_t* __restrict__ bitmap,
                                               const uint32_t* __restrict__ word_rank,
                                               uint32_t* __restrict__ pt_slot, uint32_t* __restrict__ pt_pos,
                                               uint32_t* __restrict__ vox_count) {
    const int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    const bool active = gid < BN;  // a prefix of the wave
    const int32_t b = active ? gid / N : 0;
    const uint32_t lin = active ? pt_slot[gid] : 0u;
    const uint32_t slot = active ? (uint32_t)slot_of(bitmap + (size_t)b * W, word_rank + (size_t)b * W, lin) : 0u;
    // Adjacent lanes with the same voxel (runs of one voxel's points, as in
    // a scan-ordered cloud) take their arrival positions with one atomic per
    // run: the positions within a voxel are a permutation either way.
    const size_t gs = (size_t)b * N + slot;
    const int lane = lane_id();
    const uint64_t prev = shfl_up64((uint64_t)gs, 1);
    const bool head = active && (lane == 0 || prev != (uint64_t)gs);
    const uint64_t heads = __ballot(head);
    const uint32_t n_act = (uint32_t)__popcll(__ballot(active));
    const uint64_t upto = lane == kWave - 1 ? ~0ull : ((2ull << lane) - 1);  // lanes <= this one
    const int h = active ? 63 - __clzll(heads & upto) : lane;  // the head of this lane's run
    uint32_t pos0 = 0;
    if (head) {
        const uint64_t next = heads & ~upto;
        const uint32_t end = next ? (uint32_t)(__ffsll((unsigned long long)next) - 1) : n_act;
        pos0 = atomicAdd(&vox_count[gs], end - (uint32_t)lane);
    }
    pos0 = (uint32_t)__shfl((int)pos0, h, kWave);
    if (!active) return;
    pt_slot[gid] = slot;
    pt_pos[gid] = pos0 + (uint32_t)(lane - h);
}

// Offsets: vox_off = exclusive prefix of min(count, n_v), full_off = exclusive
// prefix of count, over the slots [0, nvox[b]) of each cloud; entry nvox[b]
// holds the totals. Both are scanned at once, packed as (full << 31) | stored.
__global__ __launch_bounds__(kScanThreads) void k_offsets(
    int32_t N, int64_t tiles_s, uint32_t n_v, const int32_t* __restrict__ nvox,
    const uint32_t* __restrict__ vox_count, uint32_t* __restrict__ vox_off, uint32_t* __restrict__ full_off,
    uint64_t* __restrict__ desc_s, int* __restrict__ status, uint32_t* __restrict__ big, int64_t big_cap) {
    __shared__ uint32_t s_ticket;
    __shared__ uint64_t s_wave[kScanThreads / kWave];
    __shared__ uint64_t s_prefix;
    if (threadIdx.x == 0) s_ticket = atomicAdd((unsigned*)&status[kStTicketOff], 1u);
    __syncthreads();
    const uint32_t t = s_ticket;
    const int32_t b = (int32_t)(t / tiles_s);
    const int64_t tile = (int64_t)(t % tiles_s);
    const int64_t nv = nvox[b];
    if (tile * kScanTile >= nv) return;  // no slot here; later tiles never wait on this one
    const int64_t s0 = tile * kScanTile + (int64_t)threadIdx.x * kScanItems;
    const uint32_t* vc = vox_count + (size_t)b * N;
    uint32_t cnt[kScanItems];
    uint64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        int64_t s = s0 + i;
        cnt[i] = s < nv ? vc[s] : 0u;
        uint32_t st = cnt[i] < n_v ? cnt[i] : n_v;
        sum += ((uint64_t)cnt[i] << 31) | st;
        if (cnt[i] > kBigVoxel) {
            uint32_t k = atomicAdd((unsigned*)&status[kStBigCount], 1u);
            if ((int64_t)k < big_cap) big[k] = (uint32_t)((size_t)b * N + s);
        }
    }
    uint64_t total;
    uint64_t excl = block_excl_scan(sum, s_wave, &total);
    uint64_t run = tile_lookback(desc_s + (size_t)b * tiles_s, tile, total, &s_prefix) + excl;
    uint32_t* vo = vox_off + (size_t)b * (N + 1);
    uint32_t* fo = full_off + (size_t)b * (N + 1);
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        int64_t s = s0 + i;
        if (s > nv) break;
        vo[s] = (uint32_t)(run & 0x7FFFFFFFu);
        fo[s] = (uint32_t)(run >> 31);
        if (s < nv) {
            uint32_t st = cnt[i] < n_v ? cnt[i] : n_v;
            run += ((uint64_t)cnt[i] << 31) | st;
        }
    }
    // the slot nvox sits in the next tile when nvox is a multiple of the tile size
    if (threadIdx.x == 0 && nv == (tile + 1) * kScanTile) {
        uint64_t end = s_prefix + total;
        vo[nv] = (uint32_t)(end & 0x7FFFFFFFu);
        fo[nv] = (uint32_t)(end >> 31);
    }
}

// One lane per point: its index into the bucket of its slot.
__global__ __launch_bounds__(256) void k_scatter(int32_t BN, int32_t N, const uint32_t* __restrict__ pt_slot,
                                                 const uint32_t* __restrict__ pt_pos,
                                                 const uint32_t* __restrict__ full_off,
                                                 uint32_t* __restrict__ bucket) {
    int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    if (gid >= BN) return;
    int32_t b = gid / N;
    uint32_t slot = pt_slot[gid];
    bucket[(size_t)b * N + full_off[(size_t)b * (N + 1) + slot] + pt_pos[gid]] = (uint32_t)(gid - b * N);
}

// Stored lists. Blocks [0, part_a): one lane per point of a voxel with at
// most kBigVoxel points -- its rank among the voxel's indices places it.
// Blocks [part_a, grid): one wave per larger voxel -- the n_v smallest
// indices by bitonic selection in 64-key chunks.
__global__ __launch_bounds__(256) void k_finalize(
    const float* __restrict__ P, int32_t BN, int32_t N, uint32_t n_v, int32_t part_a,
    const uint32_t* __restrict__ pt_slot, const uint32_t* __restrict__ vox_count,
    const uint32_t* __restrict__ vox_off, const uint32_t* __restrict__ full_off,
    const uint32_t* __restrict__ bucket, const uint32_t* __restrict__ big, int64_t big_cap,
    const int* __restrict__ status, uint32_t* __restrict__ pt_list, float4* __restrict__ pt4) {
    if ((int32_t)blockIdx.x < part_a) {
        int32_t gid = (int32_t)xcd_block(blockIdx.x, (uint32_t)part_a) * blockDim.x + threadIdx.x;
        if (gid >= BN) return;
        int32_t b = gid / N;
        uint32_t i = (uint32_t)(gid - b * N);
        uint32_t slot = pt_slot[gid];
        size_t sg = (size_t)b * N + slot;
        uint32_t cnt = vox_count[sg];
        if (cnt > kBigVoxel) return;
        const uint32_t* bk = bucket + (size_t)b * N + full_off[(size_t)b * (N + 1) + slot];
        uint32_t rank = 0;
        for (uint32_t j = 0; j < cnt; ++j) rank += bk[j] < i ? 1u : 0u;
        if (rank < n_v) {
            size_t dst = (size_t)b * N + vox_off[(size_t)b * (N + 1) + slot] + rank;
            const float* p = P + (size_t)gid * 3;
            pt_list[dst] = i;
            pt4[dst] = make_float4(p[0], p[1], p[2], __uint_as_float(i));
        }
        return;
    }
    const int lane = lane_id();
    const int32_t nbig = (int64_t)status[kStBigCount] < big_cap ? status[kStBigCount] : (int32_t)big_cap;
    const int32_t wpb = blockDim.x / kWave;
    const int32_t nwaves = (gridDim.x - part_a) * wpb;
    for (int32_t v = (blockIdx.x - part_a) * wpb + threadIdx.x / kWave; v < nbig; v += nwaves) {
        uint32_t g = big[v];
        int32_t b = (int32_t)(g / (uint32_t)N);
        uint32_t s = g - (uint32_t)b * N;
        uint32_t cnt = vox_count[g];
        const uint32_t* bk = bucket + (size_t)b * N + full_off[(size_t)b * (N + 1) + s];
        uint64_t best = ~0ull, kth = ~0ull;
        uint64_t k_n = (uint32_t)lane < cnt ? (uint64_t)bk[lane] : ~0ull;  // loaded a chunk ahead
        for (uint32_t c0 = 0; c0 < cnt; c0 += kWave) {
            uint64_t k = k_n;
            k_n = (c0 + kWave + lane < cnt) ? (uint64_t)bk[c0 + kWave + lane] : ~0ull;
            // an index above the n_v-th lowest so far is never kept; a chunk
            // left without any is not sorted
            k = k < kth ? k : ~0ull;
            if (c0 != 0 && !__ballot(k != ~0ull)) continue;
            k = wave_sort64(k);
            best = c0 == 0 ? k : wave_merge_low64(best, k);
            kth = shfl64(best, (int)n_v - 1);
        }
        if ((uint32_t)lane < n_v) {
            uint32_t i = (uint32_t)best;
            size_t dst = (size_t)b * N + vox_off[(size_t)b * (N + 1) + s] + lane;
            const float* p = P + ((size_t)b * N + i) * 3;
            pt_list[dst] = i;
            pt4[dst] = make_float4(p[0], p[1], p[2], __uint_as_float(i));
        }
    }
}

// ---- larger clouds: sort the points into bricks, then build each brick.
// A brick is a run of kBrickV consecutive linear voxel ids (kBrickW occupancy
// words) of one cloud; the batch holds B * Q of them. The points are grouped
// by brick with a counting sort: a histogram per tile of points (one row per
// tile), a scan of each brick's column and of the bricks' totals (by each
// scatter tile itself, or by a launch of its own when a tile would read too
// many entries), a scatter that carries each point's coordinates and index. Then one workgroup per
// brick marks its occupancy words in LDS, ranks its occupied voxels by
// popcount, counts their points, and places the n_v lowest point indices of
// every voxel. The occupied and stored counts of the cloud's earlier bricks
// come from a look-back. Every output is written once, the work is
// proportional to the points and the occupied voxels, and no global atomic
// is taken per point.
constexpr int kSortT = 1024;                    // threads per sort tile
constexpr int kSortIPT = kSortTile / kSortT;    // points per thread
constexpr int kHGroup = 64;                     // bricks per block of the column scan
constexpr int kBrickIPT = kBrickCap / kBrickT;  // points per thread, kept in registers
constexpr int kBrickWaves = kBrickT / kWave;
static_assert(2 * kBrickCap + 1 >= kBrickV, "a heavy part counts every voxel of its brick in LDS");
static_assert(kBrickCap <= kBrickV, "a brick of one part has at most kBrickCap occupied voxels");
static_assert(kBrickW <= kWave, "a brick's occupancy words are scanned by one wave");

// Linear voxel id of a point; `bad` is set for a non-finite coordinate (its
// axis index is then 0).
__device__ __forceinline__ uint32_t voxel_lin(float x, float y, float z, const GridArgs& g, bool& bad) {
    const float c[3] = {x, y, z};
    uint32_t gg[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        if (!isfinite(c[a])) {
            bad = true;
            gg[a] = 0;
        } else {
            gg[a] = (uint32_t)axis_index(c[a], g.o[a], g.s[a], g.D[a]);
        }
    }
    return gg[0] + (uint32_t)g.D[0] * (gg[1] + (uint32_t)g.D[1] * gg[2]);
}

// Row t of the histogram: points of tile t in each brick of the batch (with
// `own`, only the entries of the bricks of the clouds the tile holds points
// of, which are the only ones read then). The blocks also zero the control
// words [clr, clr + n16) (status, tickets, descriptors) that the later
// kernels use.
__global__ __launch_bounds__(kSortT) void k_bhist(const float* __restrict__ P, int32_t N, int32_t BN, GridArgs g,
                                                  int32_t Q, int32_t BQ, int32_t T, bool own,
                                                  uint32_t* __restrict__ hist, uint4* __restrict__ clr, int64_t n16) {
    __shared__ uint32_t s_h[kMaxBricks];
    const int tid = threadIdx.x;
    const int32_t t = (int32_t)blockIdx.x;
    const int32_t p0 = t * kSortTile, p1 = p0 + kSortTile < BN ? p0 + kSortTile : BN;
    const int32_t e0 = own ? (p0 / N) * Q : 0, e1 = own ? ((p1 - 1) / N + 1) * Q : BQ;
    for (int32_t i = e0 + tid; i < e1; i += kSortT) s_h[i] = 0u;
    for (int64_t i = (int64_t)t * kSortT + tid; i < n16; i += (int64_t)T * kSortT) clr[i] = make_uint4(0u, 0u, 0u, 0u);
    // the points' coordinates first, all loads in flight together (a load
    // under the bounds test would be waited for before the next is issued)
    float c[kSortIPT][3];
#pragma unroll
    for (int k = 0; k < kSortIPT; ++k) {
        const int32_t gid = p0 + k * kSortT + tid;
        const float* p = P + (size_t)(gid < BN ? gid : 0) * 3;
#pragma unroll
        for (int a = 0; a < 3; ++a) c[k][a] = p[a];
    }
    lds_barrier();
#pragma unroll
    for (int k = 0; k < kSortIPT; ++k) {
        const int32_t gid = p0 + k * kSortT + tid;
        if (gid >= BN) break;
        bool bad = false;
        const uint32_t lin = voxel_lin(c[k][0], c[k][1], c[k][2], g, bad);
        atomicAdd(&s_h[(gid / N) * Q + (int32_t)(lin / kBrickV)], 1u);
    }
    lds_barrier();
    uint32_t* row = hist + (size_t)t * BQ;
    for (int32_t i = e0 + tid; i < e1; i += kSortT) row[i] = s_h[i];
}

// Sorted positions and work items: bstart[g] = points of the bricks before g
// (bricks in cloud-major order), and entry (t, g) of the histogram becomes
// the first position of tile t's points in brick g. Work item g < B * Q is
// brick g (its first kBrickCap points); a brick of more than kBrickCap points
// (heavy) has one more item per further kBrickCap points, listed in
// item_extra as (part << 32 | g), and heavy bricks are numbered in hlist. A
// block takes kHGroup bricks (one per lane) and splits the tiles over its
// waves; the blocks' totals are chained by a look-back.
__global__ __launch_bounds__(kScanThreads) void k_hscan(uint32_t* __restrict__ hist, int32_t BQ, int32_t T,
                                                        uint32_t* __restrict__ bstart, int32_t* __restrict__ brick_hb,
                                                        uint64_t* __restrict__ item_extra,
                                                        uint32_t* __restrict__ hlist, uint32_t* __restrict__ hebase,
                                                        uint64_t* __restrict__ desc,
                                                        int* __restrict__ status) {
    constexpr int kW = kScanThreads / kWave;
    __shared__ uint32_t s_ticket;
    __shared__ uint32_t s_part[kW][kHGroup];
    __shared__ uint32_t s_bex[kHGroup];
    __shared__ uint64_t s_prefix;
    if (threadIdx.x == 0) s_ticket = atomicAdd((unsigned*)&status[kStTicketHist], 1u);
    __syncthreads();
    const int32_t grp = (int32_t)s_ticket;
    const int lane = lane_id(), wv = threadIdx.x / kWave;
    const int32_t g = grp * kHGroup + lane;
    const bool valid = g < BQ;
    const int32_t tc = (T + kW - 1) / kW;
    const int32_t t0 = wv * tc, t1 = t0 + tc < T ? t0 + tc : T;
    // the column's first kHKeep entries stay in registers for the rewrite
    constexpr int kHKeep = 16;
    uint32_t col[kHKeep];
    uint32_t sum = 0;
    if (valid) {
#pragma unroll
        for (int j = 0; j < kHKeep; ++j) {
            col[j] = t0 + j < t1 ? hist[(size_t)(t0 + j) * BQ + g] : 0u;
            sum += col[j];
        }
        for (int32_t t = t0 + kHKeep; t < t1; ++t) sum += hist[(size_t)t * BQ + g];
    }
    s_part[wv][lane] = sum;
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
        const uint32_t x = s_part[w][lane];
        pre += w < wv ? x : 0u;
        tot += x;
    }
    // (extra parts << 32 | points), scanned over the bricks
    const uint32_t parts = !valid ? 0u : (tot > (uint32_t)kBrickCap ? (tot + kBrickCap - 1) / kBrickCap : 1u);
    uint64_t gtot = 0, ex = 0;
    if (wv == 0) {
        const uint64_t x = ((uint64_t)(parts ? parts - 1 : 0u) << 32) | tot;
        const uint64_t incl = wave_incl_scan<uint64_t>(x);
        ex = incl - x;
        s_bex[lane] = (uint32_t)ex;
        gtot = shfl64(incl, kWave - 1);
    }
    const uint64_t P0 = tile_lookback(desc, grp, gtot, &s_prefix);
    if (!valid) return;
    const uint32_t base = (uint32_t)P0 + s_bex[lane];
    if (wv == 0) {
        const uint32_t ebase = (uint32_t)((P0 + ex) >> 32);
        bstart[g] = base;
        for (uint32_t k = 1; k < parts; ++k) item_extra[ebase + k - 1] = ((uint64_t)k << 32) | (uint32_t)g;
        int32_t hb = -1;
        if (parts > 1) {
            hb = (int32_t)atomicAdd((unsigned*)&status[kStHeavy], 1u);
            hlist[hb] = (uint32_t)g;
            hebase[hb] = ebase;
        }
        brick_hb[g] = hb;
        if (g == BQ - 1) status[kStItems] = (int)(ebase + parts - 1);
    }
    uint32_t run = base + pre;
#pragma unroll
    for (int j = 0; j < kHKeep; ++j) {
        if (t0 + j < t1) hist[(size_t)(t0 + j) * BQ + g] = run;
        run += col[j];
    }
    for (int32_t t = t0 + kHKeep; t < t1; ++t) {
        const size_t e = (size_t)t * BQ + g;
        const uint32_t x = hist[e];
        hist[e] = run;
        run += x;
    }
}

// Exclusive scan of one value per thread of a kSortT block; *total receives
// the block sum. Every thread of the block calls it.
__device__ __forceinline__ uint32_t sort_excl_scan(uint32_t v, uint32_t* s_wave, uint32_t* total) {
    const uint32_t incl = wave_incl_scan<uint32_t>(v);
    const int wv = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wave[wv] = incl;
    lds_barrier();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kSortT / kWave; ++i) {
        const uint32_t x = s_wave[i];
        off += i < wv ? x : 0u;
        tot += x;
    }
    lds_barrier();
    *total = tot;
    return off + incl - v;
}

// The first sorted position of tile t's points in each brick of the clouds
// it holds points of, into s_o (indexed by brick): per brick, the column of
// the histogram over the cloud's tiles gives the points of the tiles before
// t and the brick's total, and an exclusive scan of the totals over the
// cloud's bricks (clouds hold N sorted positions each) gives the brick's
// first position. The cloud's first tile also writes those (bstart) and
// lists the bricks of more than kBrickCap points (heavy): one more work item
// per further kBrickCap points in item_extra as (part << 32 | brick),
// numbered in hlist and counted in the status words.
__device__ __forceinline__ void tile_columns(int32_t t, int32_t N, int32_t BN, int32_t Q, int32_t BQ,
                                             const uint32_t* __restrict__ hist, uint32_t* s_o, uint32_t* s_wave,
                                             uint32_t* __restrict__ bstart, int32_t* __restrict__ brick_hb,
                                             uint64_t* __restrict__ item_extra, uint32_t* __restrict__ hlist,
                                             uint32_t* __restrict__ hebase, int* __restrict__ status) {
    constexpr int kU = 32;  // column loads in flight per thread (a cloud of up to 126976 points: all of them)
    const int tid = threadIdx.x;
    const int32_t p0 = t * kSortTile, p1 = p0 + kSortTile < BN ? p0 + kSortTile : BN;
    for (int32_t b = p0 / N; b <= (p1 - 1) / N; ++b) {
        const int32_t tf = (int32_t)((int64_t)b * N / kSortTile);
        const int32_t tl = (int32_t)((((int64_t)b + 1) * N - 1) / kSortTile);
        uint32_t carry = (uint32_t)b * (uint32_t)N;
        for (int32_t q0 = 0; q0 < Q; q0 += kSortT) {
            const int32_t q = q0 + tid;
            const size_t col = (size_t)b * Q + (q < Q ? q : 0);
            uint32_t pre = 0, tot = 0;
            for (int32_t t0 = tf; t0 <= tl; t0 += kU) {
                uint32_t x[kU];
#pragma unroll
                for (int u = 0; u < kU; ++u) x[u] = hist[(size_t)(t0 + u <= tl ? t0 + u : tl) * BQ + col];
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    const uint32_t v = t0 + u <= tl ? x[u] : 0u;
                    tot += v;
                    pre += t0 + u < t ? v : 0u;
                }
            }
            if (q >= Q) tot = 0;
            uint32_t sum;
            const uint32_t start = carry + sort_excl_scan(tot, s_wave, &sum);
            carry += sum;
            if (q >= Q) continue;
            const int32_t gg = b * Q + q;
            s_o[gg] = start + pre;
            if (t != tf) continue;
            bstart[gg] = start;
            int32_t hb = -1;
            if (tot > (uint32_t)kBrickCap) {
                const uint32_t parts = (tot + kBrickCap - 1) / kBrickCap;
                hb = atomicAdd(&status[kStHeavy], 1);
                const uint32_t eb = (uint32_t)atomicAdd(&status[kStItems], (int)(parts - 1));
                hlist[hb] = (uint32_t)gg;
                hebase[hb] = eb;
                for (uint32_t k = 1; k < parts; ++k) item_extra[eb + k - 1] = ((uint64_t)k << 32) | (uint32_t)gg;
            }
            brick_hb[gg] = hb;
        }
    }
}

// One lane per point: (x, y, z, index) at the next free position of its
// brick within the tile's range. With SCAN the tile finds its ranges from
// the histogram columns itself (tile_columns); otherwise k_hscan has
// rewritten row t of the histogram into them.
template <bool SCAN>
__global__ __launch_bounds__(kSortT) void k_bscatter(const float* __restrict__ P, int32_t N, int32_t BN, GridArgs g,
                                                     int32_t Q, int32_t BQ, const uint32_t* __restrict__ hist,
                                                     float4* __restrict__ sorted, uint32_t* __restrict__ bstart,
                                                     int32_t* __restrict__ brick_hb, uint64_t* __restrict__ item_extra,
                                                     uint32_t* __restrict__ hlist, uint32_t* __restrict__ hebase,
                                                     int* __restrict__ status) {
    __shared__ uint32_t s_o[kMaxBricks];
    __shared__ uint32_t s_wave[kSortT / kWave];
    const int tid = threadIdx.x;
    const int32_t t = (int32_t)blockIdx.x;
    // the points' coordinates first, all loads in flight together
    float c[kSortIPT][3];
#pragma unroll
    for (int k = 0; k < kSortIPT; ++k) {
        const int32_t gid = t * kSortTile + k * kSortT + tid;
        const float* p = P + (size_t)(gid < BN ? gid : 0) * 3;
#pragma unroll
        for (int a = 0; a < 3; ++a) c[k][a] = p[a];
    }
    if constexpr (SCAN) {
        tile_columns(t, N, BN, Q, BQ, hist, s_o, s_wave, bstart, brick_hb, item_extra, hlist, hebase, status);
    } else {
        const uint32_t* row = hist + (size_t)t * BQ;
        for (int32_t i = tid; i < BQ; i += kSortT) s_o[i] = row[i];
    }
    lds_barrier();
    bool bad = false;
#pragma unroll
    for (int k = 0; k < kSortIPT; ++k) {
        const int32_t gid = t * kSortTile + k * kSortT + tid;
        if (gid >= BN) break;
        const float x = c[k][0], y = c[k][1], z = c[k][2];
        const uint32_t lin = voxel_lin(x, y, z, g, bad);
        const int32_t b = gid / N;
        const uint32_t pos = atomicAdd(&s_o[b * Q + (int32_t)(lin / kBrickV)], 1u);
        sorted[pos] = make_float4(x, y, z, __uint_as_float((uint32_t)(gid - b * N)));
    }
    if (bad) raise_error(status, CAGQ_ERR_NONFINITE_INPUT);
}

struct BrickArgs {
    const float* P;
    int32_t N, BN, Q, BQ;
    int64_t W;
    uint32_t n_v;
    GridArgs g;
    const uint32_t* bstart;
    const int32_t* brick_hb;
    const uint64_t* item_extra;
    const uint32_t* hlist;
    const float4* sorted;
    uint64_t* bitmap;
    uint32_t* word_rank;
    uint32_t* vox_lin;
    uint32_t* vox_count;
    int32_t* nvox;
    uint32_t* vox_off;
    uint32_t* pt_list;
    float4* pt4;
    uint64_t* agg;      // per brick: occupied voxels << 31 | stored points
    uint32_t* bucket;   // point indices of heavy bricks, grouped by voxel
    const uint32_t* hebase; // per heavy brick: its first item in item_extra
    uint32_t* pcnt;     // per further part of a heavy brick and voxel: the brick's points in the parts before it
    uint32_t* hfo;      // per heavy brick and voxel: exclusive prefix of the points (kBrickV + 1)
    uint32_t* hso;      // per heavy brick and voxel: exclusive prefix of min(points, n_v)
    uint64_t* hpre;     // per heavy brick: the aggregate of the cloud's bricks before it
    uint32_t* hdone;    // per heavy brick: its parts that have grouped their points
    int* status;
};

// Occupancy words of a brick and their exclusive ranks.
struct WordLds {
    uint64_t word[kBrickW];
    uint32_t wocc[kBrickW];
    uint32_t nocc;
};

__device__ __forceinline__ uint32_t brick_rank(const WordLds& s, uint32_t v) {
    return s.wocc[v >> 6] + (uint32_t)__popcll(s.word[v >> 6] & ((1ull << (v & 63)) - 1));
}

// Exclusive ranks of the occupancy words (one wave): sets s.wocc and s.nocc.
__device__ __forceinline__ void brick_word_scan(WordLds& s) {
    const int tid = threadIdx.x;
    if (tid < kWave) {
        const uint32_t o = tid < kBrickW ? (uint32_t)__popcll(s.word[tid]) : 0u;
        const uint32_t oi = wave_incl_scan<uint32_t>(o);
        if (tid < kBrickW) s.wocc[tid] = oi - o;
        if (tid == kWave - 1) s.nocc = oi;
    }
}

// Sum and exclusive scan of one value per thread over a brick block; the
// waves meet at an LDS-only barrier (their global stores are not waited for).
__device__ __forceinline__ uint64_t block_sum64(uint64_t v, uint64_t* s_wave) {
    v = wave_sum<uint64_t>(v);
    if (lane_id() == 0) s_wave[threadIdx.x / kWave] = v;
    lds_barrier();
    uint64_t t = 0;
#pragma unroll
    for (int i = 0; i < kBrickWaves; ++i) t += s_wave[i];
    return t;
}

__device__ __forceinline__ uint64_t brick_excl_scan(uint64_t v, uint64_t* s_wave, uint64_t* total) {
    const uint64_t incl = wave_incl_scan<uint64_t>(v);
    const int wv = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wave[wv] = incl;
    lds_barrier();
    uint64_t off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kBrickWaves; ++i) {
        const uint64_t x = s_wave[i];
        off += i < wv ? x : 0ull;
        tot += x;
    }
    *total = tot;
    return off + incl - v;
}

// The work item of a block: brick g = blockIdx.x (its first kBrickCap
// points), or a further part of a heavy brick.
struct BrickItem {
    int32_t g, b, q;
    uint32_t start, cnt;  // the brick's sorted range
    uint32_t p0, n;       // the part's sorted range
    uint32_t part, parts;
    bool heavy;
};

__device__ __forceinline__ bool brick_id(const BrickArgs& a, BrickItem& it) {
    const uint32_t u = blockIdx.x;
    it.part = 0;
    if (u < (uint32_t)a.BQ) {
        it.g = (int32_t)u;
    } else {
        if (u - (uint32_t)a.BQ >= (uint32_t)a.status[kStItems]) return false;
        const uint64_t x = a.item_extra[u - a.BQ];
        it.g = (int32_t)(uint32_t)x;
        it.part = (uint32_t)(x >> 32);
    }
    it.b = it.g / a.Q;
    it.q = it.g - it.b * a.Q;
    return true;
}

__device__ __forceinline__ void brick_range(const BrickArgs& a, BrickItem& it) {
    it.start = a.bstart[it.g];
    const uint32_t end = it.g + 1 < a.BQ ? a.bstart[it.g + 1] : (uint32_t)a.BN;
    it.cnt = end - it.start;
    it.heavy = it.cnt > (uint32_t)kBrickCap;
    it.parts = it.heavy ? (it.cnt + kBrickCap - 1) / kBrickCap : 1u;
    it.p0 = it.start + it.part * (uint32_t)kBrickCap;
    it.n = end - it.p0 < (uint32_t)kBrickCap ? end - it.p0 : (uint32_t)kBrickCap;
}

__device__ __forceinline__ bool brick_item(const BrickArgs& a, BrickItem& it) {
    if (!brick_id(a, it)) return false;
    brick_range(a, it);
    return true;
}

// Voxel (within the brick) of each of the part's points; with MARK, also its
// occupancy bit in s.word (zeroed and published by the caller's barrier).
template <bool MARK>
__device__ __forceinline__ void brick_voxels(const BrickArgs& a, WordLds& s, const BrickItem& it,
                                             uint32_t (&v)[kBrickIPT], uint32_t (&idx)[kBrickIPT]) {
    const uint32_t vbase = (uint32_t)it.q * kBrickV;
    // every point's load first, so that they are in flight together (a load
    // used under its bounds test would be waited for before the next)
    float4 ee[kBrickIPT];
#pragma unroll
    for (int k = 0; k < kBrickIPT; ++k) {
        const uint32_t i = threadIdx.x + k * kBrickT;
        if (i < it.n) ee[k] = a.sorted[it.p0 + i];
    }
#pragma unroll
    for (int k = 0; k < kBrickIPT; ++k) {
        const uint32_t i = threadIdx.x + k * kBrickT;
        v[k] = 0u;
        idx[k] = 0u;
        if (i < it.n) {
            const float4 e = ee[k];
            bool bad = false;
            v[k] = voxel_lin(e.x, e.y, e.z, a.g, bad) - vbase;
            idx[k] = __float_as_uint(e.w);
            if (MARK) atomicOr(reinterpret_cast<unsigned long long*>(&s.word[v[k] >> 6]), 1ull << (v[k] & 63));
        }
    }
}

struct CountLds {
    WordLds w;
    uint32_t cnt[kBrickV];  // per occupied voxel (by rank), or per voxel for a heavy brick
    uint64_t wave[kScanThreads / kWave];
};

// Pass 1 over the bricks: per brick its occupancy words (final) and its
// aggregate (occupied voxels, stored points). A heavy brick is counted by the
// block of its first part, which streams the parts in turn and writes, per
// part and voxel, the brick's points in the parts before it (the second pass
// places each part's points after them), then the per-voxel prefixes and the
// voxels of more than kBigVoxel points. The blocks of further parts have
// nothing to do here.
__global__ __launch_bounds__(kBrickT) void k_brick_count(BrickArgs a) {
    __shared__ CountLds s;
    BrickItem it;
    if (!brick_item(a, it) || it.part != 0) return;
    const int tid = threadIdx.x;
    const size_t wbase = (size_t)it.b * a.W + (size_t)it.q * kBrickW;
    const int64_t wlim = a.W - (int64_t)it.q * kBrickW;  // words of this brick inside the grid
    if (it.cnt == 0) {
        if (tid < kBrickW && tid < wlim) a.bitmap[wbase + tid] = 0ull;
        if (tid == 0) a.agg[it.g] = 0ull;
        return;
    }
    if (tid < kBrickW) s.w.word[tid] = 0ull;
    if (it.heavy)
        for (int j = tid; j < kBrickV; j += kBrickT) s.cnt[j] = 0u;
    lds_barrier();
    uint32_t v[kBrickIPT], idx[kBrickIPT];
    if (!it.heavy) {
        brick_voxels<true>(a, s.w, it, v, idx);
        lds_barrier();
        brick_word_scan(s.w);
        lds_barrier();
        const uint32_t n_occ = s.w.nocc;
        for (uint32_t j = tid; j < n_occ; j += kBrickT) s.cnt[j] = 0u;
        lds_barrier();
#pragma unroll
        for (int k = 0; k < kBrickIPT; ++k)
            if (threadIdx.x + k * kBrickT < it.n) atomicAdd(&s.cnt[brick_rank(s.w, v[k])], 1u);
        lds_barrier();
        uint64_t st = 0;
        for (uint32_t j = tid; j < n_occ; j += kBrickT) st += s.cnt[j] < a.n_v ? s.cnt[j] : a.n_v;
        st = block_sum64(st, s.wave);
        if (tid < kBrickW && tid < wlim) a.bitmap[wbase + tid] = s.w.word[tid];
        if (tid == 0) a.agg[it.g] = ((uint64_t)n_occ << 31) | st;
        return;
    }
    // a heavy brick: its parts in turn; before each, the counts so far are that part's row
    const int32_t hb = a.brick_hb[it.g];
    const uint32_t eb = a.hebase[hb];
    for (uint32_t p = 0; p < it.parts; ++p) {
        BrickItem pt = it;
        pt.part = p;
        pt.p0 = it.start + p * (uint32_t)kBrickCap;
        pt.n = it.start + it.cnt - pt.p0 < (uint32_t)kBrickCap ? it.start + it.cnt - pt.p0 : (uint32_t)kBrickCap;
        brick_voxels<true>(a, s.w, pt, v, idx);
        if (p != 0) {
            uint32_t* row = a.pcnt + (size_t)(eb + p - 1) * kBrickV;
            for (int j = tid; j < kBrickV; j += kBrickT) row[j] = s.cnt[j];
        }
        lds_barrier();
#pragma unroll
        for (int k = 0; k < kBrickIPT; ++k)
            if (threadIdx.x + k * kBrickT < pt.n) atomicAdd(&s.cnt[v[k]], 1u);
        lds_barrier();
    }
    brick_word_scan(s.w);
    if (tid < kBrickW && tid < wlim) a.bitmap[wbase + tid] = s.w.word[tid];
    constexpr int kPer = kBrickV / kBrickT;
    uint32_t c[kPer];
    uint64_t sum = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        c[j] = s.cnt[tid * kPer + j];
        sum += ((uint64_t)c[j] << 32) | (c[j] < a.n_v ? c[j] : a.n_v);
    }
    uint64_t total;
    uint64_t pos = brick_excl_scan(sum, s.wave, &total);
    uint32_t* fo = a.hfo + (size_t)hb * (kBrickV + 1);
    uint32_t* so = a.hso + (size_t)hb * kBrickV;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const uint32_t vv = tid * kPer + j;
        fo[vv] = (uint32_t)(pos >> 32);
        so[vv] = (uint32_t)pos;
        pos += ((uint64_t)c[j] << 32) | (c[j] < a.n_v ? c[j] : a.n_v);
    }
    if (tid == 0) {
        fo[kBrickV] = it.cnt;
        a.agg[it.g] = ((uint64_t)s.w.nocc << 31) | (uint32_t)total;
    }
}

// The n_v smallest of the cnt indices at p (in memory), sorted ascending over
// the wave's lanes: 64-key chunks, four loaded at a time, each sorted by a
// bitonic network and merged into the best so far; a chunk without an index
// below the n_v-th best is skipped.
__device__ __forceinline__ uint64_t wave_select_lowest(const uint32_t* p, uint32_t cnt, uint32_t n_v) {
    const int lane = lane_id();
    uint64_t best = ~0ull, kth = ~0ull;
    for (uint32_t c0 = 0; c0 < cnt; c0 += 4 * kWave) {
        uint64_t key[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t i = c0 + j * kWave + lane;
            key[j] = i < cnt ? (uint64_t)p[i] : ~0ull;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (c0 + j * kWave >= cnt) break;
            uint64_t k = key[j] < kth ? key[j] : ~0ull;
            const bool first = c0 == 0 && j == 0;
            if (!first && !__ballot(k != ~0ull)) continue;
            k = wave_sort64(k);
            best = first ? k : wave_merge_low64(best, k);
            kth = shfl64(best, (int)n_v - 1);
        }
    }
    return best;
}

struct BuildLds {
    WordLds w;
    uint64_t bigm[kBrickW];         // bit r: occupied voxel r holds more than kBigVoxel points
    union {
        struct {
            uint32_t va[kBrickCap + 1]; // per occupied voxel: count, then (stored prefix << 16 | point prefix)
            uint32_t idx[kBrickCap];    // point indices grouped by voxel (arrival order)
        } one;                          // a brick of one part
        uint32_t arr[kBrickV];          // a part of a heavy brick: its arrivals per voxel
    } u;
    uint64_t wave[kScanThreads / kWave];
    uint32_t ticket;
};

// Pass 2 over the bricks: slots, offsets and stored lists. The aggregates of
// the cloud's earlier bricks are summed directly (every one is final). A
// brick of one part does everything in LDS; a part of a heavy brick groups
// its points by voxel in `bucket`, and the last of its parts to finish then
// selects the brick's lists from there.
__global__ __launch_bounds__(kBrickT) void k_brick(BrickArgs a) {
    __shared__ BuildLds s;
    BrickItem it;
    if (!brick_id(a, it)) return;
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wv = tid / kWave;
    // the cloud's bricks before this one (loads issued with the range's,
    // four per thread at a time)
    uint64_t pre = 0;
    const uint64_t* ag = a.agg + (size_t)it.b * a.Q;
    for (int32_t j0 = 0; j0 < it.q; j0 += 4 * kBrickT) {
        uint64_t x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int32_t j = j0 + u * kBrickT + tid;
            x[u] = j < it.q ? ag[j] : 0ull;
        }
        pre += (x[0] + x[1]) + (x[2] + x[3]);
    }
    const uint64_t my = ag[it.q];
    brick_range(a, it);
    const uint32_t vbase = (uint32_t)it.q * kBrickV;
    const size_t pb = (size_t)it.b * a.N;
    const size_t wbase = (size_t)it.b * a.W + (size_t)it.q * kBrickW;
    const int64_t wlim = a.W - (int64_t)it.q * kBrickW;
    uint32_t* vo = a.vox_off + (size_t)it.b * (a.N + 1);
    if (tid < kBrickW) {
        s.w.word[tid] = it.heavy ? (tid < wlim ? a.bitmap[wbase + tid] : 0ull) : 0ull;
        s.bigm[tid] = 0ull;
    }
    pre = block_sum64(pre, s.wave);  // its barrier also publishes the words
    const uint32_t p_occ = (uint32_t)(pre >> 31), p_st = (uint32_t)(pre & 0x7FFFFFFFu);
    if (it.cnt == 0) {
        if (tid < kBrickW && tid < wlim) a.word_rank[wbase + tid] = p_occ;
        if (it.q == a.Q - 1 && tid == 0) {
            a.nvox[it.b] = (int32_t)p_occ;
            vo[p_occ] = p_st;
        }
        return;
    }
    uint32_t v[kBrickIPT], idx[kBrickIPT];
    if (it.heavy) brick_voxels<false>(a, s.w, it, v, idx);
    else brick_voxels<true>(a, s.w, it, v, idx);
    lds_barrier();
    brick_word_scan(s.w);
    lds_barrier();
    const uint32_t n_occ = (uint32_t)(my >> 31);
    if (it.part == 0) {
        if (tid < kBrickW && tid < wlim) a.word_rank[wbase + tid] = p_occ + s.w.wocc[tid];
        if (it.q == a.Q - 1 && tid == 0) {
            a.nvox[it.b] = (int32_t)(p_occ + n_occ);
            vo[p_occ + n_occ] = p_st + (uint32_t)(my & 0x7FFFFFFFu);
        }
        if (it.heavy && tid == 0) a.hpre[a.brick_hb[it.g]] = pre;
    }
    if (it.heavy) {
        // a point's position within its voxel: the voxel's points in the
        // parts before this one, then its arrival in this part
        const int32_t hb = a.brick_hb[it.g];
        const uint32_t* before = it.part == 0 ? nullptr : a.pcnt + (size_t)(a.hebase[hb] + it.part - 1) * kBrickV;
        const uint32_t* fo = a.hfo + (size_t)hb * (kBrickV + 1);
        const uint32_t* so = a.hso + (size_t)hb * kBrickV;
        for (int j = tid; j < kBrickV; j += kBrickT) s.u.arr[j] = 0u;
        lds_barrier();
        // every point's loads first, then the stores
        uint32_t bf[kBrickIPT], f0s[kBrickIPT], f1s[kBrickIPT], sos[kBrickIPT];
#pragma unroll
        for (int k = 0; k < kBrickIPT; ++k) {
            const bool in = threadIdx.x + k * kBrickT < it.n;
            bf[k] = in && before ? before[v[k]] : 0u;
            f0s[k] = in ? fo[v[k]] : 0u;
            f1s[k] = in ? fo[v[k] + 1] : 0u;
            sos[k] = in ? so[v[k]] : 0u;
        }
#pragma unroll
        for (int k = 0; k < kBrickIPT; ++k) {
            if (threadIdx.x + k * kBrickT >= it.n) break;
            const uint32_t ps = bf[k] + atomicAdd(&s.u.arr[v[k]], 1u);
            const uint32_t f0 = f0s[k];
            a.bucket[it.start + f0 + ps] = idx[k];
            if (ps == 0) {
                const uint32_t slot = p_occ + brick_rank(s.w, v[k]);
                a.vox_lin[pb + slot] = vbase + v[k];
                a.vox_count[pb + slot] = f1s[k] - f0;
                vo[slot] = p_st + sos[k];
            }
        }
        // the last part to finish selects the brick's stored lists: a point
        // of a voxel of at most kBigVoxel points by its rank (one lane per
        // point), a larger voxel by one wave's bitonic selection
        __threadfence();
        __syncthreads();
        if (tid == 0) s.ticket = atomicAdd(&a.hdone[hb], 1u);
        __syncthreads();
        if (s.ticket != it.parts - 1) return;
        __threadfence();
        const uint32_t* bk = a.bucket + it.start;
        for (uint32_t i = tid; i < it.cnt; i += kBrickT) {
            const float4 e = a.sorted[it.start + i];
            bool bad = false;
            const uint32_t vv = voxel_lin(e.x, e.y, e.z, a.g, bad) - vbase;
            const uint32_t f0 = fo[vv], c = fo[vv + 1] - f0;
            if (c > kBigVoxel) continue;
            const uint32_t id = __float_as_uint(e.w);
            uint32_t rank = 0;
            for (uint32_t j = 0; j < c; ++j) rank += bk[f0 + j] < id ? 1u : 0u;
            if (rank < a.n_v) {
                const size_t dst = pb + p_st + so[vv] + rank;
                a.pt_list[dst] = id;
                a.pt4[dst] = e;
            }
        }
        for (uint32_t ch = tid / kWave; ch < (uint32_t)kBrickV / kWave; ch += kBrickWaves) {
            const uint32_t f0v = fo[ch * kWave + lane], cv = fo[ch * kWave + lane + 1] - f0v;
            const uint32_t sov = so[ch * kWave + lane];
            for (uint64_t m = __ballot(cv > kBigVoxel); m; m &= m - 1) {
                const int l = __ffsll((unsigned long long)m) - 1;
                const uint32_t f0 = (uint32_t)__shfl((int)f0v, l, kWave);
                const uint32_t cnt = (uint32_t)__shfl((int)cv, l, kWave);
                const uint32_t sl = (uint32_t)__shfl((int)sov, l, kWave);
                const uint64_t best = wave_select_lowest(bk + f0, cnt, a.n_v);
                if ((uint32_t)lane < a.n_v) {
                    const uint32_t i = (uint32_t)best;
                    const size_t dst = pb + p_st + sl + lane;
                    const float* p = a.P + (pb + i) * 3;
                    a.pt_list[dst] = i;
                    a.pt4[dst] = make_float4(p[0], p[1], p[2], __uint_as_float(i));
                }
            }
        }
        return;
    }
    // a brick of one part: counts per occupied voxel, arrival positions
    uint32_t* va = s.u.one.va;  // n_occ + 1 entries
    for (uint32_t j = tid; j <= n_occ; j += kBrickT) va[j] = 0u;
    lds_barrier();
    uint32_t r[kBrickIPT], pos[kBrickIPT];
#pragma unroll
    for (int k = 0; k < kBrickIPT; ++k) {
        r[k] = 0u;
        pos[k] = 0u;
        if (threadIdx.x + k * kBrickT < it.n) {
            r[k] = brick_rank(s.w, v[k]);
            pos[k] = atomicAdd(&va[r[k]], 1u);
        }
    }
    lds_barrier();
    // the points' coordinates, loaded again for the stored lists (issued here
    // so that the scan and grouping below hide their latency)
    float4 e[kBrickIPT];
#pragma unroll
    for (int k = 0; k < kBrickIPT; ++k)
        if (threadIdx.x + k * kBrickT < it.n) e[k] = a.sorted[it.p0 + threadIdx.x + k * kBrickT];
    // exclusive prefixes of (count, stored) over the occupied voxels, packed
    // as stored << 16 | count (both at most kBrickCap)
    const uint32_t per = (n_occ + kBrickT - 1) / kBrickT;
    const uint32_t r0 = (uint32_t)tid * per;
    uint32_t sum = 0;
    for (uint32_t j = 0; j < per; ++j) {
        if (r0 + j >= n_occ) break;
        const uint32_t c = va[r0 + j];
        sum += ((c < a.n_v ? c : a.n_v) << 16) | c;
    }
    uint64_t total;
    uint32_t run = (uint32_t)brick_excl_scan(sum, s.wave, &total);
    for (uint32_t j = 0; j < per; ++j) {
        const uint32_t rr = r0 + j;
        if (rr >= n_occ) break;
        const uint32_t c = va[rr];
        va[rr] = run;
        if (c > kBigVoxel) atomicOr(reinterpret_cast<unsigned long long*>(&s.bigm[rr >> 6]), 1ull << (rr & 63));
        run += ((c < a.n_v ? c : a.n_v) << 16) | c;
    }
    if (tid == 0) va[n_occ] = it.cnt;
    lds_barrier();
    // the points grouped by voxel; the first arrival in a voxel writes its slot
#pragma unroll
    for (int k = 0; k < kBrickIPT; ++k) {
        if (threadIdx.x + k * kBrickT >= it.n) break;
        const uint32_t o = va[r[k]], f0 = o & 0xFFFFu;
        s.u.one.idx[f0 + pos[k]] = idx[k];
        if (pos[k] == 0) {
            const uint32_t slot = p_occ + r[k];
            a.vox_lin[pb + slot] = vbase + v[k];
            a.vox_count[pb + slot] = (va[r[k] + 1] & 0xFFFFu) - f0;
            vo[slot] = p_st + (o >> 16);
        }
    }
    lds_barrier();
    // stored lists: a point of a voxel of at most kBigVoxel points by its rank
#pragma unroll
    for (int k = 0; k < kBrickIPT; ++k) {
        if (threadIdx.x + k * kBrickT >= it.n) break;
        const uint32_t o = va[r[k]], f0 = o & 0xFFFFu, c = (va[r[k] + 1] & 0xFFFFu) - f0;
        if (c > kBigVoxel) continue;
        uint32_t rank = 0;
        for (uint32_t j = 0; j < c; ++j) rank += s.u.one.idx[f0 + j] < idx[k] ? 1u : 0u;
        if (rank < a.n_v) {
            const size_t dst = pb + p_st + (o >> 16) + rank;
            a.pt_list[dst] = idx[k];
            a.pt4[dst] = e[k];
        }
    }
    // larger voxels: one wave each, the n_v smallest indices by bitonic selection
    for (int j = wv; j < kBrickW; j += kBrickWaves) {
        for (uint64_t m = s.bigm[j]; m; m &= m - 1) {
            const uint32_t rr = (uint32_t)j * kWave + (uint32_t)(__ffsll((unsigned long long)m) - 1);
            const uint32_t o = va[rr], f0 = o & 0xFFFFu, c = (va[rr + 1] & 0xFFFFu) - f0;
            uint64_t best = ~0ull, kth = ~0ull;
            for (uint32_t c0 = 0; c0 < c; c0 += kWave) {
                uint64_t key = (c0 + lane < c) ? (uint64_t)s.u.one.idx[f0 + c0 + lane] : ~0ull;
                // an index above the n_v-th lowest so far is never kept
                key = key < kth ? key : ~0ull;
                if (c0 != 0 && !__ballot(key != ~0ull)) continue;
                key = wave_sort64(key);
                best = c0 == 0 ? key : wave_merge_low64(best, key);
                kth = shfl64(best, (int)a.n_v - 1);
            }
            if ((uint32_t)lane < a.n_v) {
                const uint32_t i = (uint32_t)best;
                const size_t dst = pb + p_st + (o >> 16) + lane;
                const float* p = a.P + (pb + i) * 3;
                a.pt_list[dst] = i;
                a.pt4[dst] = make_float4(p[0], p[1], p[2], __uint_as_float(i));
            }
        }
    }
}

// ---- small clouds: the whole build in one workgroup per cloud.
// For clouds of at most kSmallN points whose grid has at most kSmallW
// occupancy words, every step above runs in one 1024-thread workgroup with
// the bitmap, the ranks, the counts and offsets and the buckets in LDS, so
// the seven launches (and their dependent round trips to memory) become one.
// The outputs are those of the steps above, bit for bit: the same bitmap,
// ranks, slots and linear ids, counts and offsets, and per voxel the n_v
// lowest point indices in ascending order (ranked against the voxel's
// bucket, or selected by a wave for voxels of more than kBigVoxel points).
// The threads exchange data through LDS only, so the barriers do not wait for
// the global stores of the steps before them.
constexpr int kSmallT = 1024;
constexpr int kSmallPts = 8;   // points per thread
constexpr int kSmallWd = 4;    // occupancy words per thread
constexpr int32_t kSmallN = kSmallT * kSmallPts;
constexpr int64_t kSmallW = kSmallT * kSmallWd;
constexpr int kSmallBig = kSmallN / (kBigVoxel + 1) + 1;  // voxels of more than kBigVoxel points

// Exclusive scan of one value per thread over the kSmallT threads.
__device__ __forceinline__ uint64_t small_excl_scan(uint64_t v, uint64_t* s_wave, uint64_t* total) {
    const uint64_t incl = wave_incl_scan<uint64_t>(v);
    const int wv = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wave[wv] = incl;
    lds_barrier();
    uint64_t off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kSmallT / kWave; ++i) {
        const uint64_t x = s_wave[i];
        off += i < wv ? x : 0ull;
        tot += x;
    }
    *total = tot;
    lds_barrier();
    return off + incl - v;
}

size_t small_lds_bytes(int32_t N, int64_t W) { return (size_t)12 * W + (size_t)4 * (2 * (size_t)N + 1); }

__global__ __launch_bounds__(kSmallT) void k_build_small(
    const float* __restrict__ P, int32_t N, GridArgs g, int64_t W, uint32_t n_v, uint32_t* __restrict__ pt_slot,
    uint64_t* __restrict__ bitmap, uint32_t* __restrict__ word_rank, uint32_t* __restrict__ vox_lin,
    uint32_t* __restrict__ vox_count, int32_t* __restrict__ nvox, uint32_t* __restrict__ vox_off,
    uint32_t* __restrict__ pt_list, float4* __restrict__ pt4, int* __restrict__ status, int* __restrict__ berr) {
    extern __shared__ __align__(16) unsigned char lds[];
    uint64_t* s_bm = reinterpret_cast<uint64_t*>(lds);   // [W] occupancy words
    uint32_t* s_wr = reinterpret_cast<uint32_t*>(s_bm + W);  // [W] ranks
    uint32_t* s_off = s_wr + W;  // [N + 1] counts, then (full offset << 16) | stored offset
    uint32_t* s_bk = s_off + N + 1;  // [N] point indices grouped by slot (arrival order)
    __shared__ uint64_t s_wave[kSmallT / kWave];
    __shared__ uint32_t s_big[kSmallBig];
    __shared__ uint32_t s_nbig, s_bad;
    const int32_t b = blockIdx.x;
    const int tid = threadIdx.x;
    const size_t pb = (size_t)b * N;

    // the status words start at zero for the kernels after this one (this
    // kernel writes none: its errors go to the cloud's own word)
    if (b == 0 && tid < kStSlots) status[tid] = 0;
    for (int64_t w = tid; w < W; w += kSmallT) s_bm[w] = 0ull;
    for (int32_t i = tid; i <= N; i += kSmallT) s_off[i] = 0u;
    if (tid == 0) {
        s_nbig = 0;
        s_bad = 0;
    }
    lds_barrier();

    // voxelize: linear id, occupancy bit (every point's coordinates are
    // loaded first, so that their loads are in flight together)
    float pc[kSmallPts][3];
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        const float* p = P + (pb + (i < N ? i : 0)) * 3;
#pragma unroll
        for (int a = 0; a < 3; ++a) pc[k][a] = p[a];
    }
    uint32_t lin[kSmallPts];
    bool bad = false;
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        lin[k] = 0;
        if (i >= N) continue;
        uint32_t gg[3];
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            if (!isfinite(pc[k][a])) {
                bad = true;
                gg[a] = 0;
            } else {
                gg[a] = (uint32_t)axis_index(pc[k][a], g.o[a], g.s[a], g.D[a]);
            }
        }
        lin[k] = gg[0] + (uint32_t)g.D[0] * (gg[1] + (uint32_t)g.D[1] * gg[2]);
        atomicOr(reinterpret_cast<unsigned long long*>(&s_bm[lin[k] >> 6]), 1ull << (lin[k] & 63));
    }
    if (bad) s_bad = 1;
    lds_barrier();
    if (tid == 0) berr[b] = s_bad ? CAGQ_ERR_NONFINITE_INPUT : 0;

    // ranks of the words
    uint64_t wd[kSmallWd];
    uint32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < kSmallWd; ++j) {
        const int64_t w = (int64_t)tid * kSmallWd + j;
        wd[j] = w < W ? s_bm[w] : 0ull;
        cnt += (uint32_t)__popcll(wd[j]);
    }
    uint64_t total;
    uint32_t r = (uint32_t)small_excl_scan(cnt, s_wave, &total);
    const uint32_t nv = (uint32_t)total;
#pragma unroll
    for (int j = 0; j < kSmallWd; ++j) {
        const int64_t w = (int64_t)tid * kSmallWd + j;
        if (w >= W) break;
        s_wr[w] = r;
        bitmap[(size_t)b * W + w] = wd[j];
        word_rank[(size_t)b * W + w] = r;
        r += (uint32_t)__popcll(wd[j]);
    }
    if (tid == 0) nvox[b] = (int32_t)nv;
    lds_barrier();

    // slot and arrival position of every point, packed as slot << 16 | position;
    // the first arrival in a voxel puts its linear id at its slot of s_bk
    // (free until the buckets), for the coalesced writes after the offsets
    uint32_t sp[kSmallPts];
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        sp[k] = 0;
        if (i >= N) continue;
        const uint32_t w = lin[k] >> 6;
        const uint32_t sl = s_wr[w] + (uint32_t)__popcll(s_bm[w] & ((1ull << (lin[k] & 63)) - 1));
        const uint32_t pos = atomicAdd(&s_off[sl], 1u);
        sp[k] = (sl << 16) | pos;
        pt_slot[pb + i] = sl;
        if (pos == 0) s_bk[sl] = lin[k];
    }
    lds_barrier();

    // offsets: (full << 31) | stored, scanned over the slots [0, nv)
    uint32_t c8[kSmallPts];
    uint64_t sum = 0;
#pragma unroll
    for (int j = 0; j < kSmallPts; ++j) {
        const uint32_t sl = (uint32_t)tid * kSmallPts + j;
        c8[j] = sl < nv ? s_off[sl] : 0u;
        sum += ((uint64_t)c8[j] << 31) | (c8[j] < n_v ? c8[j] : n_v);
    }
    uint64_t run = small_excl_scan(sum, s_wave, &total);
    uint32_t* vo = vox_off + (size_t)b * (N + 1);
#pragma unroll
    for (int j = 0; j < kSmallPts; ++j) {
        const uint32_t sl = (uint32_t)tid * kSmallPts + j;
        if (sl >= nv) break;
        const uint32_t full = (uint32_t)(run >> 31), stored = (uint32_t)(run & 0x7FFFFFFFu);
        s_off[sl] = (full << 16) | stored;
        if (c8[j] > kBigVoxel) s_big[atomicAdd(&s_nbig, 1u)] = sl;
        run += ((uint64_t)c8[j] << 31) | (c8[j] < n_v ? c8[j] : n_v);
    }
    if (tid == 0) {
        vo[nv] = (uint32_t)(total & 0x7FFFFFFFu);
        s_off[nv] = ((uint32_t)(total >> 31) << 16) | (uint32_t)(total & 0x7FFFFFFFu);
    }
    lds_barrier();
    // offsets, counts and linear ids, each slot's from LDS: consecutive
    // threads store consecutive slots
    for (uint32_t sl = (uint32_t)tid; sl < nv; sl += kSmallT) {
        const uint32_t o0 = s_off[sl], o1 = s_off[sl + 1];
        vo[sl] = o0 & 0xFFFFu;
        vox_count[pb + sl] = (o1 >> 16) - (o0 >> 16);
        vox_lin[pb + sl] = s_bk[sl];
    }
    lds_barrier();  // s_bk is read above and filled below

    // buckets
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        if (i < N) s_bk[(s_off[sp[k] >> 16] >> 16) + (sp[k] & 0xFFFFu)] = (uint32_t)i;
    }
    lds_barrier();

    // stored lists: a point of a voxel of at most kBigVoxel points by its rank
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        if (i >= N) continue;
        const uint32_t o0 = s_off[sp[k] >> 16], o1 = s_off[(sp[k] >> 16) + 1];
        const uint32_t f0 = o0 >> 16, cnt_v = (o1 >> 16) - f0;
        if (cnt_v > kBigVoxel) continue;
        uint32_t rank = 0;
        for (uint32_t j = 0; j < cnt_v; ++j) rank += s_bk[f0 + j] < (uint32_t)i ? 1u : 0u;
        if (rank < n_v) {
            const size_t dst = pb + (o0 & 0xFFFFu) + rank;
            const float* p = P + (pb + i) * 3;
            pt_list[dst] = (uint32_t)i;
            pt4[dst] = make_float4(p[0], p[1], p[2], __uint_as_float((uint32_t)i));
        }
    }
    // larger voxels: one wave each, the n_v smallest indices by bitonic selection
    const int lane = lane_id();
    for (uint32_t v = (uint32_t)(tid / kWave); v < s_nbig; v += kSmallT / kWave) {
        const uint32_t sl = s_big[v];
        const uint32_t o0 = s_off[sl], f0 = o0 >> 16, cnt_v = (s_off[sl + 1] >> 16) - f0;
        uint64_t best = ~0ull, kth = ~0ull;
        for (uint32_t c0 = 0; c0 < cnt_v; c0 += kWave) {
            uint64_t key = (c0 + lane < cnt_v) ? (uint64_t)s_bk[f0 + c0 + lane] : ~0ull;
            // an index above the n_v-th lowest so far is never kept
            key = key < kth ? key : ~0ull;
            if (c0 != 0 && !__ballot(key != ~0ull)) continue;
            key = wave_sort64(key);
            best = c0 == 0 ? key : wave_merge_low64(best, key);
            kth = shfl64(best, (int)n_v - 1);
        }
        if ((uint32_t)lane < n_v) {
            const uint32_t i = (uint32_t)best;
            const size_t dst = pb + (o0 & 0xFFFFu) + lane;
            const float* p = P + (pb + i) * 3;
            pt_list[dst] = i;
            pt4[dst] = make_float4(p[0], p[1], p[2], __uint_as_float(i));
        }
    }
}

// Dynamic LDS a workgroup of k_build_small may take on the current device, or -1.
int64_t small_lds_avail() {
    static int64_t avail[64];  // per device, 0 until known
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return -1;
    if (avail[dev] == 0) {
        int max_sh = 0;
        hipFuncAttributes fa{};
        if (hipDeviceGetAttribute(&max_sh, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
            hipFuncGetAttributes(&fa, (const void*)k_build_small) != hipSuccess)
            return -1;
        avail[dev] = (int64_t)max_sh - (int64_t)fa.sharedSizeBytes;
    }
    return avail[dev];
}

}  // namespace

hipError_t launch_build(const float* points, const Layout& L, const cagq_grid_desc& d, void* ws,
                        hipStream_t s) {
    const int32_t B = L.B, N = L.N, BN = B * N;
    const GridArgs g = grid_args(d);
    int* status = at<int>(ws, L.status);
    if (N <= kSmallN && L.W <= kSmallW && (int64_t)small_lds_bytes(N, L.W) <= small_lds_avail()) {
        // no clearing launch: the build zeroes the status words itself and
        // writes each cloud's error code (the selection's histogram serves
        // clouds of at least 16384 points only, the scan descriptors and
        // occupancy bytes other builds)
        const size_t bytes = small_lds_bytes(N, L.W);
        hipError_t e = hipFuncSetAttribute((const void*)k_build_small, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)bytes);
        if (e != hipSuccess) return e;
        k_build_small<<<B, kSmallT, bytes, s>>>(points, N, g, L.W, (uint32_t)d.n_v, at<uint32_t>(ws, L.pt_slot),
                                                at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
                                                at<uint32_t>(ws, L.vox_lin), at<uint32_t>(ws, L.vox_count),
                                                at<int32_t>(ws, L.nvox), at<uint32_t>(ws, L.vox_off),
                                                at<uint32_t>(ws, L.pt_list), at<float4>(ws, L.pt4), status,
                                                at<int>(ws, L.berr));
        return hipGetLastError();
    }
    if (L.bricks) {
        const int32_t BQ = B * L.Q;
        uint32_t* hist = at<uint32_t>(ws, L.hist);
        int* status_w = at<int>(ws, L.status);
        k_bhist<<<(unsigned)L.T, kSortT, 0, s>>>(points, N, BN, g, L.Q, BQ, L.T, L.tile_scan, hist,
                                                 at<uint4>(ws, L.status), (int64_t)(L.clear_brick - L.status) / 16);
        if (!L.tile_scan)
            k_hscan<<<(unsigned)((BQ + kHGroup - 1) / kHGroup), kScanThreads, 0, s>>>(
                hist, BQ, L.T, at<uint32_t>(ws, L.bstart), at<int32_t>(ws, L.brick_hb), at<uint64_t>(ws, L.item_extra),
                at<uint32_t>(ws, L.hlist), at<uint32_t>(ws, L.hebase), at<uint64_t>(ws, L.desc_h), status_w);
        (L.tile_scan ? k_bscatter<true> : k_bscatter<false>)<<<(unsigned)L.T, kSortT, 0, s>>>(
            points, N, BN, g, L.Q, BQ, hist, at<float4>(ws, L.sorted), at<uint32_t>(ws, L.bstart),
            at<int32_t>(ws, L.brick_hb), at<uint64_t>(ws, L.item_extra), at<uint32_t>(ws, L.hlist),
            at<uint32_t>(ws, L.hebase), status_w);
        BrickArgs a;
        a.P = points;
        a.N = N;
        a.BN = BN;
        a.Q = L.Q;
        a.BQ = BQ;
        a.W = L.W;
        a.n_v = (uint32_t)d.n_v;
        a.g = g;
        a.bstart = at<uint32_t>(ws, L.bstart);
        a.brick_hb = at<int32_t>(ws, L.brick_hb);
        a.item_extra = at<uint64_t>(ws, L.item_extra);
        a.hlist = at<uint32_t>(ws, L.hlist);
        a.sorted = at<float4>(ws, L.sorted);
        a.bitmap = at<uint64_t>(ws, L.bitmap);
        a.word_rank = at<uint32_t>(ws, L.word_rank);
        a.vox_lin = at<uint32_t>(ws, L.vox_lin);
        a.vox_count = at<uint32_t>(ws, L.vox_count);
        a.nvox = at<int32_t>(ws, L.nvox);
        a.vox_off = at<uint32_t>(ws, L.vox_off);
        a.pt_list = at<uint32_t>(ws, L.pt_list);
        a.pt4 = at<float4>(ws, L.pt4);
        a.agg = at<uint64_t>(ws, L.agg);
        a.bucket = at<uint32_t>(ws, L.bucket);
        a.hebase = at<uint32_t>(ws, L.hebase);
        a.pcnt = at<uint32_t>(ws, L.pcnt);
        a.hdone = at<uint32_t>(ws, L.hdone);
        a.hfo = at<uint32_t>(ws, L.hfo);
        a.hso = at<uint32_t>(ws, L.hso);
        a.hpre = at<uint64_t>(ws, L.hpre);
        a.status = status_w;
        k_brick_count<<<(unsigned)L.items_max, kBrickT, 0, s>>>(a);
        k_brick<<<(unsigned)L.items_max, kBrickT, 0, s>>>(a);
        return hipGetLastError();
    }
    size_t n16 = (L.clear_end - L.status) / 16;
    int cb = (int)((n16 + 255) / 256);
    if (cb > 4096) cb = 4096;
    k_clear<<<cb, 256, 0, s>>>(at<uint4>(ws, L.status), n16);
    const int pb = (BN + 255) / 256;
    k_mark<<<pb, 256, 0, s>>>(points, N, BN, g, L.W, at<uint32_t>(ws, L.pt_slot), at<uint8_t>(ws, L.bytemap),
                              status);
    k_rank<<<(unsigned)(B * L.tiles_w), kScanThreads, 0, s>>>(
        at<uint8_t>(ws, L.bytemap), at<uint64_t>(ws, L.bitmap), L.W, L.tiles_w, N, at<uint32_t>(ws, L.word_rank),
        at<uint32_t>(ws, L.vox_lin), at<uint32_t>(ws, L.vox_count), at<int32_t>(ws, L.nvox),
        at<uint64_t>(ws, L.desc_w), status);
    k_count<<<pb, 256, 0, s>>>(BN, N, L.W, at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
                               at<uint32_t>(ws, L.pt_slot), at<uint32_t>(ws, L.pt_pos),
                               at<uint32_t>(ws, L.vox_count));
    k_offsets<<<(unsigned)(B * L.tiles_s), kScanThreads, 0, s>>>(
        N, L.tiles_s, (uint32_t)d.n_v, at<int32_t>(ws, L.nvox), at<uint32_t>(ws, L.vox_count),
        at<uint32_t>(ws, L.vox_off), at<uint32_t>(ws, L.full_off), at<uint64_t>(ws, L.desc_s), status,
        at<uint32_t>(ws, L.big), L.big_cap);
    k_scatter<<<pb, 256, 0, s>>>(BN, N, at<uint32_t>(ws, L.pt_slot), at<uint32_t>(ws, L.pt_pos),
                                 at<uint32_t>(ws, L.full_off), at<uint32_t>(ws, L.bucket));
    int64_t bigb = (L.big_cap + 3) / 4;
    if (bigb > 1024) bigb = 1024;
    if (bigb < 1) bigb = 1;
    k_finalize<<<(unsigned)(pb + bigb), 256, 0, s>>>(
        points, BN, N, (uint32_t)d.n_v, pb, at<uint32_t>(ws, L.pt_slot), at<uint32_t>(ws, L.vox_count),
        at<uint32_t>(ws, L.vox_off), at<uint32_t>(ws, L.full_off), at<uint32_t>(ws, L.bucket),
        at<uint32_t>(ws, L.big), L.big_cap, status, at<uint32_t>(ws, L.pt_list), at<float4>(ws, L.pt4));
    return hipGetLastError();
}

}  // namespace cagq
