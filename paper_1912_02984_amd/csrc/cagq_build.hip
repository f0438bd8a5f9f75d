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
    uint32_t* __restrict__ pt_list, float4* __restrict__ pt4, int* __restrict__ status) {
    extern __shared__ __align__(16) unsigned char lds[];
    uint64_t* s_bm = reinterpret_cast<uint64_t*>(lds);   // [W] occupancy words
    uint32_t* s_wr = reinterpret_cast<uint32_t*>(s_bm + W);  // [W] ranks
    uint32_t* s_off = s_wr + W;  // [N + 1] counts, then (full offset << 16) | stored offset
    uint32_t* s_bk = s_off + N + 1;  // [N] point indices grouped by slot (arrival order)
    __shared__ uint64_t s_wave[kSmallT / kWave];
    __shared__ uint32_t s_big[kSmallBig];
    __shared__ uint32_t s_nbig;
    const int32_t b = blockIdx.x;
    const int tid = threadIdx.x;
    const size_t pb = (size_t)b * N;

    for (int64_t w = tid; w < W; w += kSmallT) s_bm[w] = 0ull;
    for (int32_t i = tid; i <= N; i += kSmallT) s_off[i] = 0u;
    if (tid == 0) s_nbig = 0;
    lds_barrier();

    // voxelize: linear id, occupancy bit
    uint32_t lin[kSmallPts];
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        lin[k] = 0;
        if (i >= N) continue;
        const float* p = P + (pb + i) * 3;
        const float c[3] = {p[0], p[1], p[2]};
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
        lin[k] = gg[0] + (uint32_t)g.D[0] * (gg[1] + (uint32_t)g.D[1] * gg[2]);
        atomicOr(reinterpret_cast<unsigned long long*>(&s_bm[lin[k] >> 6]), 1ull << (lin[k] & 63));
        if (bad) raise_error(status, CAGQ_ERR_NONFINITE_INPUT);
    }
    lds_barrier();

    // ranks of the words; the linear id of every occupied voxel at its slot
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
        for (uint64_t m = wd[j]; m; m &= m - 1) vox_lin[pb + r++] = (uint32_t)(w * 64 + __ffsll((unsigned long long)m) - 1);
    }
    if (tid == 0) nvox[b] = (int32_t)nv;
    lds_barrier();

    // slot and arrival position of every point, packed as slot << 16 | position
    uint32_t sp[kSmallPts];
#pragma unroll
    for (int k = 0; k < kSmallPts; ++k) {
        const int32_t i = tid + k * kSmallT;
        sp[k] = 0;
        if (i >= N) continue;
        const uint32_t w = lin[k] >> 6;
        const uint32_t sl = s_wr[w] + (uint32_t)__popcll(s_bm[w] & ((1ull << (lin[k] & 63)) - 1));
        sp[k] = (sl << 16) | atomicAdd(&s_off[sl], 1u);
        pt_slot[pb + i] = sl;
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
        vo[sl] = stored;
        vox_count[pb + sl] = c8[j];
        s_off[sl] = (full << 16) | stored;
        if (c8[j] > kBigVoxel) s_big[atomicAdd(&s_nbig, 1u)] = sl;
        run += ((uint64_t)c8[j] << 31) | (c8[j] < n_v ? c8[j] : n_v);
    }
    if (tid == 0) {
        vo[nv] = (uint32_t)(total & 0x7FFFFFFFu);
        s_off[nv] = ((uint32_t)(total >> 31) << 16) | (uint32_t)(total & 0x7FFFFFFFu);
    }
    lds_barrier();

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
        // the status words and the selection's histogram only: the small
        // build uses no scan descriptors or occupancy bytes
        k_clear<<<(unsigned)((L.clear_small - L.status + 4095) / 4096), 256, 0, s>>>(
            at<uint4>(ws, L.status), (L.clear_small - L.status) / 16);
        const size_t bytes = small_lds_bytes(N, L.W);
        hipError_t e = hipFuncSetAttribute((const void*)k_build_small, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)bytes);
        if (e != hipSuccess) return e;
        k_build_small<<<B, kSmallT, bytes, s>>>(points, N, g, L.W, (uint32_t)d.n_v, at<uint32_t>(ws, L.pt_slot),
                                                at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
                                                at<uint32_t>(ws, L.vox_lin), at<uint32_t>(ws, L.vox_count),
                                                at<int32_t>(ws, L.nvox), at<uint32_t>(ws, L.vox_off),
                                                at<uint32_t>(ws, L.pt_list), at<float4>(ws, L.pt4), status);
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
