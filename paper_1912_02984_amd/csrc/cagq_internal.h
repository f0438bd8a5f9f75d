// Internal declarations of the gfx950 CAGQ library: workspace layout,
// device helpers shared by the build, sampling and query kernels, and the
// host-side launch functions the C ABI (cagq_api.hip) sequences.
//
// Everything here is HIP for gfx950 only (64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cagq.h"

namespace cagq {

constexpr int kWave = 64;
constexpr int kScanThreads = 256;       // threads per scan tile
constexpr int kScanItems = 4;           // items per thread in a scan tile
constexpr int kScanTile = kScanThreads * kScanItems;
constexpr int kRankItems = 1;           // occupancy words per thread of the rank scan
constexpr int kRankTile = kScanThreads * kRankItems;
constexpr uint32_t kBigVoxel = 64;      // voxels holding more points use the wave selector
constexpr int kSelBins = 2048;          // bins of the 11-bit digits of the many-block select
constexpr int kSelChunk = 4096;         // slots per chunk of the many-block select
constexpr int kBrickW = 32;             // occupancy words per brick of the brick build
constexpr int kBrickV = kBrickW * 64;   // voxels per brick (a run of consecutive linear ids)
constexpr int32_t kMaxBricks = 8192;    // bricks over the batch the brick build's histograms hold
constexpr int kSortTile = 4096;         // points per tile of the brick histogram and scatter
constexpr int kBrickT = 256;            // threads per brick work item
constexpr int kBrickCap = 2048;         // points per brick work item (heavier bricks are split)
constexpr int64_t kTileScanCap = 1 << 16;  // histogram entries a scatter tile may sum (tiles of a cloud x Q)

// Status word slots (int32 each) at the start of the workspace's control block.
enum StatusSlot {
    kStError = 0,      // first device-side error code (0 = none)
    kStTicketRank = 1, // tile tickets of the occupancy-rank scan
    kStTicketOff = 2,  // tile tickets of the offsets scan
    kStBigCount = 3,   // number of voxels with more than kBigVoxel points
    kStTicketSel = 4,  // tile tickets of the center compaction scan
    kStTicketCtx = 5,  // tile tickets of the context-offsets scan
    kStTicketHist = 6, // tile tickets of the brick-histogram scan
    kStItems = 7,      // brick build: work items (bricks and parts of heavy bricks)
    kStHeavy = 8,      // brick build: bricks of more than kBrickCap points
    kStSlots = 16
};

// Byte offsets of every array in the caller's workspace. Exposed arrays first
// (their offsets are also published through cagq_layout), then internal ones.
struct Layout {
    int32_t B, N;
    int64_t V;            // voxels per grid
    int64_t W;            // 64-bit occupancy words per cloud
    int64_t tiles_w;      // rank-scan tiles (kRankTile words) over the words of one cloud
    int64_t tiles_s;      // scan tiles over the slots of one cloud
    int64_t big_cap;      // capacity of the big-voxel list
    int32_t Q;            // bricks per cloud (kBrickW words each)
    int32_t T;            // point tiles (kSortTile points) over the batch
    bool bricks;          // the brick build's arrays are present (B * Q <= kMaxBricks)
    bool tile_scan;       // brick build: each scatter tile sums its clouds' histogram columns itself
                          // (at most kTileScanCap entries per tile); otherwise a scan launch does
    int64_t items_max;    // brick build: bound on the work items, B * Q + ceil(B * N / kBrickCap)
                          // (the bricks, then the further parts of heavy bricks)
    int64_t heavy_max;    // brick build: bound on the heavy bricks, B * N / (kBrickCap + 1)
    size_t total;
    // exposed
    size_t nvox, vox_lin, vox_count, vox_off, pt_list;
    // internal
    size_t status;        // int32[kStSlots]
    size_t berr;          // int32[B] per cloud: the one-workgroup build's error code (0 = none)
    size_t desc_h;        // u64 [blocks of the column scan] scan descriptors (brick totals)
    size_t clear_brick;   // [status, clear_brick) is zeroed by the brick build (status, tickets,
                          // descriptors, hdone)
    size_t desc_w;        // u64 [B][tiles_w] scan descriptors (occupancy ranks)
    size_t desc_s;        // u64 [B][tiles_s] scan descriptors (offsets)
    size_t bytemap;       // u8  [B][64 W] one byte per voxel, 1 when a point lies in it
    size_t bitmap;        // u64 [B][W] occupancy bits, bit (lin & 63) of word lin >> 6
    size_t word_rank;     // u32 [B][W] occupied voxels before word w (the slot of its first bit)
    size_t pt_slot;       // u32 [B][N] per point: linear id, then slot
    size_t pt_pos;        // u32 [B][N] per point: arrival position inside its voxel
    size_t hist;          // u32 [T][B*Q] points of tile t in brick g, then the first sorted position of them
    size_t bstart;        // u32 [B*Q] first sorted position of each brick
    size_t brick_hb;      // i32 [B*Q] index of a heavy brick in hlist, else -1
    size_t item_extra;    // u64 [items_max - B*Q] further parts of heavy bricks: part << 32 | brick
    size_t agg;           // u64 [B*Q] occupied voxels << 31 | stored points of each brick
    size_t hlist;         // u32 [heavy_max] the heavy bricks
    size_t hebase;        // u32 [heavy_max] first item_extra entry of each heavy brick
    size_t pcnt;          // u32 [items_max - B*Q][kBrickV] per further part of a heavy brick and voxel:
                          // the brick's points in the parts before it
    size_t hdone;         // u32 [heavy_max] parts of each heavy brick that have grouped their points
    size_t hfo;           // u32 [heavy_max][kBrickV + 1] their exclusive prefix
    size_t hso;           // u32 [heavy_max][kBrickV] exclusive prefix of min(points, n_v)
    size_t hpre;          // u64 [heavy_max] aggregate of the bricks before each heavy brick
    size_t sorted;        // float4 [B*N] x, y, z, bits(index) grouped by brick
    size_t full_off;      // u32 [B][N+1] exclusive prefix of the full counts
    size_t bucket;        // u32 [B][N] every point index grouped by slot (arrival order); in the
                          // brick build, those of bricks too large for LDS, at their sorted position
    size_t pt4;           // float4 [B][N] stored points grouped by slot: x, y, z, bits(index)
    size_t big;           // u32 [big_cap] global slot ids (b*N + s) of big voxels
    size_t cas_cover;     // u32 [B][N] CAS: centers whose neighbourhood holds the voxel
    size_t cas_key;       // u64 [B][N] CAS: key of an unpicked voxel in the current round
    size_t cas_pick;      // u64 [B][N] CAS: key at pick time (0 = unpicked)
    size_t cas_round;     // u32 [B][N] CAS: round that picked the voxel + 1 (0 = unpicked)
    size_t cas_blocker;   // i32 [B][N] CAS: a neighbour whose key beat the voxel's (-1 = none)
    size_t cas_dirty;     // u32 [B][N] CAS: round whose scoring must recompute the voxel
    size_t cas_ctl;       // CAS control block, see CasCtl
    size_t cas_nbr;       // u16 [B][N][nbr_stride(r)] CAS neighbour lists of small clouds (see below)
    size_t cas_nbr32;     // u32 [B][N][kNbr32Stride] CAS neighbour lists of larger clouds, r = 1
    bool has_nbr16, has_nbr32;
    size_t sel_thr;       // u64 [B] selection threshold, see sel_pack
    size_t sel_ghist;     // u32 [B][kSelBins] top-11-bit histogram of the many-block select (zero between selections)
    size_t sel_cnt;       // u32 [B] block tickets of the many-block select (zero between selections)
    size_t sel_keys;      // u32 [B][chunks][4096] top halves of the select keys, each chunk sorted by its top 11 bits
    size_t sel_bins;      // u32 [B][chunks][kSelBins] end of each 11-bit bin in its sorted chunk
    size_t sel_base;      // u32 [B][chunks] first output position of each chunk's chosen slots
    size_t sel_take;      // u32 [B][chunks] ties at the bound each chunk takes
    size_t clear_small;   // [status, clear_small) is zeroed by every build
    size_t cov_mark;      // u8  [B][N] coverage metric: 1 when the slot holds a node point
    size_t clear_end;     // [status, clear_end) is zeroed at the start of every build
};

// CAS control block, placed at Layout::cas_ctl: per round buffer (a round
// writes one, reads the previous one and clears the next) and cloud,
// kCasParts partial maxima / counts (spreading the atomics of one round over
// several addresses), then per cloud a done flag, then the number of clouds
// done, then the number of clouds done, then per cloud kCasParts partial
// histograms of the picks' uncovered counts U (rounds on lists with beta = 0):
// u64 gpart[3][B][kCasParts]; u32 cpart[3][B][kCasParts]; u32 done[B];
// u32 ndone; u32 uhist[B][kCasParts][kCasUBins].
constexpr int kCasParts = 128;
constexpr int kCasBufs = 3;
constexpr int kCasUBins = 32;  // U <= 27 with r = 1
struct CasCtl {
    static size_t bytes(int B) {
        return (size_t)B * (kCasBufs * kCasParts * 12 + 4 + 4 * kCasParts * kCasUBins) + 64;
    }
};

// Neighbour lists of the single-workgroup CAS (clouds of at most kCasLdsMaxN
// points, r <= 2): per slot a header of 8 u16 (entries within Chebyshev r,
// entries within 2r, 6 unused) and then the slots of the occupied voxels
// within distance 2r, those within r (the slot itself included) first.
constexpr int32_t kCasLdsMaxN = 4096;
__host__ __device__ constexpr int nbr_stride(int r) {
    return 8 + (((4 * r + 1) * (4 * r + 1) * (4 * r + 1) + 7) & ~7);
}

// The same lists with u32 entries behind a 4-entry header, for clouds of
// more than kCasLdsMaxN points with r = 1 (at most 125 entries).
constexpr int kNbr32Stride = 4 + 128;

bool make_layout(int32_t B, int32_t N, const cagq_grid_desc* d, Layout* L);

template <typename T>
__host__ __device__ inline T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// ------------------------------------------------------------------ device helpers

// splitmix64 output function (Steele, Lea, Flood, OOPSLA 2014): the state
// x is advanced by the golden gamma, then mixed by two xor-shift-multiplies.
__device__ __forceinline__ uint64_t sm64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    int lo = __shfl((int)(uint32_t)v, src, kWave);
    int hi = __shfl((int)(uint32_t)(v >> 32), src, kWave);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int m) {
    int lo = __shfl_xor((int)(uint32_t)v, m, kWave);
    int hi = __shfl_xor((int)(uint32_t)(v >> 32), m, kWave);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ uint64_t shfl_up64(uint64_t v, int d) {
    int lo = __shfl_up((int)(uint32_t)v, d, kWave);
    int hi = __shfl_up((int)(uint32_t)(v >> 32), d, kWave);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// Lane i of a 16-lane row reads lane i - N of the row; lanes below N read 0.
template <int N>
__device__ __forceinline__ uint32_t dpp_row_shr(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 + N, 0xF, 0xF, false);
}

// Sum and maximum over the wave, the same in every lane: an inclusive scan
// within each 16-lane row by DPP row shifts, then the four rows' last lanes
// read as scalars (no LDS permutes). Every lane of the wave must be active.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
    v += dpp_row_shr<1>(v);
    v += dpp_row_shr<2>(v);
    v += dpp_row_shr<4>(v);
    v += dpp_row_shr<8>(v);
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 15) + (uint32_t)__builtin_amdgcn_readlane((int)v, 31) +
           (uint32_t)__builtin_amdgcn_readlane((int)v, 47) + (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Inclusive prefix sum over the wave by DPP alone: within each 16-lane row
// by row shifts, then row 0's total into rows 1 and 3 (row_bcast:15, lane
// 15 of each even row into the next row) and rows 0-1's into rows 2 and 3
// (row_bcast:31). Every lane of the wave must be active.
__device__ __forceinline__ uint32_t wave_incl_sum_u32(uint32_t v) {
    v += dpp_row_shr<1>(v);
    v += dpp_row_shr<2>(v);
    v += dpp_row_shr<4>(v);
    v += dpp_row_shr<8>(v);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
    return v;
}

template <int N>
__device__ __forceinline__ uint64_t dpp_row_shr64(uint64_t v) {
    return ((uint64_t)dpp_row_shr<N>((uint32_t)(v >> 32)) << 32) | dpp_row_shr<N>((uint32_t)v);
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    uint64_t o = dpp_row_shr64<1>(v);
    v = o > v ? o : v;
    o = dpp_row_shr64<2>(v);
    v = o > v ? o : v;
    o = dpp_row_shr64<4>(v);
    v = o > v ? o : v;
    o = dpp_row_shr64<8>(v);
    v = o > v ? o : v;
    uint64_t m = 0;
#pragma unroll
    for (int r = 15; r < kWave; r += 16) {
        const uint64_t x = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), r) << 32) |
                           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, r);
        m = x > m ? x : m;
    }
    return m;
}

template <int C, int RM>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
    return ((uint64_t)(uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), C, RM, 0xF, false) << 32) |
           (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, C, RM, 0xF, false);
}

// Inclusive prefix sum across the 64 lanes of a wave, by DPP as
// wave_incl_sum_u32 (64-bit values move as two halves). Every lane of the
// wave must be active.
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
    static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit values");
    if constexpr (sizeof(T) == 4) {
        return (T)wave_incl_sum_u32((uint32_t)v);
    } else {
        uint64_t x = (uint64_t)v;
        x += dpp64<0x111, 0xF>(x);
        x += dpp64<0x112, 0xF>(x);
        x += dpp64<0x114, 0xF>(x);
        x += dpp64<0x118, 0xF>(x);
        x += dpp64<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
        x += dpp64<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
        return (T)x;
    }
}

// Sum over the wave, in every lane (the inclusive sum's last lane).
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
    const T incl = wave_incl_scan<T>(v);
    if constexpr (sizeof(T) == 4) {
        return (T)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)incl, kWave - 1);
    } else {
        return (T)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)incl >> 32), kWave - 1)
                    << 32) |
                   (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)incl, kWave - 1));
    }
}

__device__ __forceinline__ uint64_t wave_max64(uint64_t v) { return wave_max_u64(v); }

// Ascending bitonic sort of one 64-bit key per lane over the whole wave.
__device__ __forceinline__ uint64_t wave_sort64(uint64_t v) {
    const int lane = lane_id();
#pragma unroll
    for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            uint64_t o = shfl_xor64(v, j);
            bool asc = (lane & k) == 0;
            bool low = (lane & j) == 0;
            uint64_t mn = o < v ? o : v, mx = o < v ? v : o;
            v = (asc == low) ? mn : mx;
        }
    }
    return v;
}

// `best` and `add` each sorted ascending over the wave: returns the 64
// smallest keys of their union, sorted ascending.
__device__ __forceinline__ uint64_t wave_merge_low64(uint64_t best, uint64_t add) {
    const int lane = lane_id();
    uint64_t rev = shfl64(add, kWave - 1 - lane);
    uint64_t v = rev < best ? rev : best;     // bitonic: the 64 smallest of the union
#pragma unroll
    for (int j = kWave >> 1; j > 0; j >>= 1) {
        uint64_t o = shfl_xor64(v, j);
        bool low = (lane & j) == 0;
        uint64_t mn = o < v ? o : v, mx = o < v ? v : o;
        v = low ? mn : mx;
    }
    return v;
}

// Agent-scope atomics for the cross-workgroup scan descriptors (the 8 XCDs
// have separate L2s, so these must reach the coherent level). Relaxed: a
// descriptor carries its value and status in one word, and no tile reads
// another tile's other output within the kernel, so no ordering with other
// memory is needed (an agent-scope release or acquire would also write back
// or invalidate the XCD's L2 at every descriptor).
__device__ __forceinline__ uint64_t ld_desc(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_desc(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A workgroup barrier that orders LDS accesses only: the global stores issued
// before it are not waited for (__syncthreads also waits for those, a full
// memory round trip). For kernels whose threads exchange data through LDS
// alone.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ void raise_error(int* status, int code) {
    atomicCAS(status + kStError, 0, code);
}

// Tile descriptors of the look-back scans: status in bits 62-63 (1 = the
// tile's own aggregate, 2 = inclusive prefix), value in bits 0-61.
constexpr uint64_t kDescAgg = 1ull << 62;
constexpr uint64_t kDescInc = 2ull << 62;
constexpr uint64_t kDescVal = (1ull << 62) - 1;

// Exclusive prefix of `agg` over the tiles before `tile` in one segment;
// desc(t) is the address of tile t's descriptor. Every thread of the block
// calls it; wave 0 publishes and looks back. Tiles are numbered by a ticket
// taken at block start, so every predecessor has started and will publish:
// the spin always ends.
template <typename F>
__device__ inline uint64_t tile_lookback_at(F desc, int64_t tile, uint64_t agg, uint64_t* s_out) {
    if (threadIdx.x < kWave) {
        const int lane = lane_id();
        uint64_t excl = 0;
        if (tile == 0) {
            if (lane == 0) st_desc(desc(0), kDescInc | agg);
        } else {
            if (lane == 0) st_desc(desc(tile), kDescAgg | agg);
            int64_t base = tile - 1;
            while (true) {
                int64_t idx = base - lane;
                uint64_t d = kDescInc;  // before the first tile: an inclusive zero
                if (idx >= 0) {
                    do {
                        d = ld_desc(desc(idx));
                    } while ((d >> 62) == 0);
                }
                uint64_t inc = __ballot((d >> 62) == 2);
                if (inc) {
                    int first = __ffsll((unsigned long long)inc) - 1;
                    excl += wave_sum<uint64_t>(lane <= first ? (d & kDescVal) : 0ull);
                    break;
                }
                excl += wave_sum<uint64_t>(d & kDescVal);
                base -= kWave;
            }
            if (lane == 0) st_desc(desc(tile), kDescInc | (excl + agg));
        }
        if (lane == 0) *s_out = excl;
    }
    __syncthreads();
    return *s_out;
}

// The same over a contiguous descriptor array.
__device__ inline uint64_t tile_lookback(uint64_t* desc, int64_t tile, uint64_t agg, uint64_t* s_out) {
    return tile_lookback_at([desc](int64_t t) { return desc + t; }, tile, agg, s_out);
}

// Exclusive scan of one 64-bit value per thread across a kScanThreads block;
// *total receives the block sum.
__device__ inline uint64_t block_excl_scan(uint64_t v, uint64_t* s_wave, uint64_t* total) {
    uint64_t incl = wave_incl_scan<uint64_t>(v);
    const int wv = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wave[wv] = incl;
    __syncthreads();
    uint64_t off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kScanThreads / kWave; ++i) {
        uint64_t x = s_wave[i];
        if (i < wv) off += x;
        tot += x;
    }
    *total = tot;
    return off + incl - v;
}

// Block id remapped so that consecutive logical blocks share an XCD (blocks
// are dispatched to the 8 XCDs round-robin; each XCD has its own L2).
__device__ __forceinline__ uint32_t xcd_block(uint32_t bid, uint32_t nblocks) {
    const uint32_t nx = 8;
    uint32_t q = nblocks / nx, rem = nblocks % nx;
    uint32_t x = bid % nx, i = bid / nx;
    return x < rem ? x * (q + 1) + i : rem * (q + 1) + (x - rem) * q + i;
}

// CAS key of a voxel of score `score` and linear id `lin`: (score, -lin) as
// one unsigned 64-bit word, the score offset by 2^31.
__device__ __forceinline__ uint64_t cas_key(int64_t score, uint32_t lin) {
    return ((uint64_t)(score + 2147483648ll) << 32) | (uint64_t)(0xFFFFFFFFu - lin);
}

// Slot of the occupied voxel `lin` of a cloud (the number of occupied voxels
// with a smaller linear id), or -1 when it is empty.
__device__ __forceinline__ int32_t slot_of(const uint64_t* bm, const uint32_t* wr, uint32_t lin) {
    uint64_t w = bm[lin >> 6];
    uint64_t bit = 1ull << (lin & 63);
    if (!(w & bit)) return -1;
    return (int32_t)(wr[lin >> 6] + __popcll(w & (bit - 1)));
}

// clamp(floor((p - o) / s), 0, D - 1): one rounded subtract, one correctly
// rounded divide, an exact floor and an exact clamp.
__device__ __forceinline__ int32_t axis_index(float p, float o, float s, int32_t D) {
    float diff = p - o;
    float t = diff / s;
    float f = floorf(t);
    if (f < 0.0f) return 0;
    if (f >= 2147483648.0f) return D - 1;
    int32_t gi = (int32_t)f;
    return gi > D - 1 ? D - 1 : gi;
}

struct GridDims {
    int32_t D[3];
};

// One grid-row segment of a cloud's occupancy: the slot of the first occupied
// voxel at or after the segment's start, and bit j set when voxel x - h + j
// of the segment is occupied (clear outside the grid).
struct GridRow {
    uint32_t first;
    uint32_t mask;
};

// The segment x' in [x - h, x + h] of grid row (yy, zz), h <= 15. Branch-free:
// rows outside the grid are clamped into it for the loads and get an empty
// mask, and the second word is always loaded (the same word unless the
// segment crosses a word boundary), so the loads of many rows are in flight
// together.
__device__ __forceinline__ GridRow load_row(const uint64_t* __restrict__ bm, const uint32_t* __restrict__ wr,
                                            const GridDims& g, int32_t x, int32_t yy, int32_t zz, int32_t h) {
    const bool inside = yy >= 0 && yy < g.D[1] && zz >= 0 && zz < g.D[2];
    const int32_t yc = yy < 0 ? 0 : (yy >= g.D[1] ? g.D[1] - 1 : yy);
    const int32_t zc = zz < 0 ? 0 : (zz >= g.D[2] ? g.D[2] - 1 : zz);
    const int32_t xs = x - h;
    const int32_t lo_x = xs < 0 ? 0 : xs;
    const int32_t hi_x = x + h > g.D[0] - 1 ? g.D[0] - 1 : x + h;
    const uint32_t base = (uint32_t)g.D[0] * ((uint32_t)yc + (uint32_t)g.D[1] * (uint32_t)zc);
    const uint32_t lo = base + (uint32_t)lo_x, hi = base + (uint32_t)hi_x;
    const uint32_t w0 = lo >> 6, o = lo & 63;
    // the word's rank is loaded with the words (its address does not depend
    // on them), so that the row costs one load latency
    const uint32_t rk = wr[w0];
    const uint64_t a = bm[w0];
    const uint64_t c = bm[hi >> 6];
    // when both ends share a word, the bits shifted in from c lie above the segment
    const uint64_t bits = (a >> o) | (o ? c << (64 - o) : 0ull);
    GridRow r;
    r.mask = inside ? (uint32_t)(bits & ((1ull << (hi_x - lo_x + 1)) - 1)) << (lo_x - xs) : 0u;
    r.first = rk + (uint32_t)__popcll(a & ((1ull << o) - 1));
    return r;
}

// NR rows (yy[i], zz[i]) around the same x at once, as load_row each: all
// their loads are issued before any is used, so that the rows cost one load
// latency together instead of one each.
template <int NR>
__device__ __forceinline__ void load_rows(const uint64_t* __restrict__ bm, const uint32_t* __restrict__ wr,
                                          const GridDims& g, int32_t x, const int32_t (&yy)[NR],
                                          const int32_t (&zz)[NR], int32_t h, GridRow (&out)[NR]) {
    const int32_t xs = x - h;
    const int32_t lo_x = xs < 0 ? 0 : xs;
    const int32_t hi_x = x + h > g.D[0] - 1 ? g.D[0] - 1 : x + h;
    uint32_t rk[NR], o[NR];
    uint64_t a[NR], c[NR];
#pragma unroll
    for (int i = 0; i < NR; ++i) {
        const int32_t yc = yy[i] < 0 ? 0 : (yy[i] >= g.D[1] ? g.D[1] - 1 : yy[i]);
        const int32_t zc = zz[i] < 0 ? 0 : (zz[i] >= g.D[2] ? g.D[2] - 1 : zz[i]);
        const uint32_t base = (uint32_t)g.D[0] * ((uint32_t)yc + (uint32_t)g.D[1] * (uint32_t)zc);
        const uint32_t lo = base + (uint32_t)lo_x, hi = base + (uint32_t)hi_x;
        o[i] = lo & 63;
        rk[i] = wr[lo >> 6];
        a[i] = bm[lo >> 6];
        c[i] = bm[hi >> 6];
    }
#pragma unroll
    for (int i = 0; i < NR; ++i) {
        const bool inside = yy[i] >= 0 && yy[i] < g.D[1] && zz[i] >= 0 && zz[i] < g.D[2];
        const uint64_t bits = (a[i] >> o[i]) | (o[i] ? c[i] << (64 - o[i]) : 0ull);
        out[i].mask = inside ? (uint32_t)(bits & ((1ull << (hi_x - lo_x + 1)) - 1)) << (lo_x - xs) : 0u;
        out[i].first = rk[i] + (uint32_t)__popcll(a[i] & ((1ull << o[i]) - 1));
    }
}

__device__ __forceinline__ void decode_lin(uint32_t lin, const GridDims& g, int32_t& x, int32_t& y, int32_t& z) {
    x = (int32_t)(lin % (uint32_t)g.D[0]);
    y = (int32_t)((lin / (uint32_t)g.D[0]) % (uint32_t)g.D[1]);
    z = (int32_t)(lin / ((uint32_t)g.D[0] * (uint32_t)g.D[1]));
}

// Calls f(slot) for every occupied voxel within Chebyshev distance `rad` of
// grid cell (x, y, z), in ascending linear id, one occupancy word per grid
// row segment; stops early (returning false) when f returns false.
template <typename F>
__device__ __forceinline__ bool for_each_neighbour(const uint64_t* __restrict__ bm,
                                                   const uint32_t* __restrict__ wr, const int32_t* D,
                                                   int32_t x, int32_t y, int32_t z, int32_t rad, F f) {
    const int32_t x0 = x - rad < 0 ? 0 : x - rad;
    const int32_t x1 = x + rad > D[0] - 1 ? D[0] - 1 : x + rad;
    const int32_t z0 = z - rad < 0 ? 0 : z - rad, z1 = z + rad > D[2] - 1 ? D[2] - 1 : z + rad;
    const int32_t y0 = y - rad < 0 ? 0 : y - rad, y1 = y + rad > D[1] - 1 ? D[1] - 1 : y + rad;
    for (int32_t zz = z0; zz <= z1; ++zz) {
        for (int32_t yy = y0; yy <= y1; ++yy) {
            const uint32_t base = (uint32_t)D[0] * ((uint32_t)yy + (uint32_t)D[1] * (uint32_t)zz);
            const uint32_t l0 = base + (uint32_t)x0, l1 = base + (uint32_t)x1;
            for (uint32_t w = l0 >> 6; w <= (l1 >> 6); ++w) {
                const uint64_t bits = bm[w];
                const uint32_t lo = w == (l0 >> 6) ? (l0 & 63) : 0u;
                const uint32_t hi = w == (l1 >> 6) ? (l1 & 63) : 63u;
                const uint64_t upto = hi == 63 ? ~0ull : ((1ull << (hi + 1)) - 1);
                uint64_t m = bits & upto & ~((1ull << lo) - 1);
                if (!m) continue;
                const uint32_t rb = wr[w];
                while (m) {
                    const int bit = __ffsll((unsigned long long)m) - 1;
                    if (!f(rb + (uint32_t)__popcll(bits & ((1ull << bit) - 1)))) return false;
                    m &= m - 1;
                }
            }
        }
    }
    return true;
}

// ------------------------------------------------------------------ host launchers

// Build: voxelize, occupancy bitmap, slots, counts, offsets, capped lists.
hipError_t launch_build(const float* points, const Layout& L, const cagq_grid_desc& d,
                        void* ws, hipStream_t s);

// Selects, per cloud, the m = min(M, nvox) slots with the smallest key and
// writes their linear ids in ascending slot order (cyclic padding to M).
// key_mode 0: RVS keys from `seed`; key_mode 1: CAS pick keys (largest first).
hipError_t launch_select(const Layout& L, void* ws, int32_t M, int key_mode, uint64_t seed,
                         int32_t* center_lin, int32_t* m_valid, hipStream_t s);

// The selection after run_cas: the m largest pick keys. Rounds on lists with
// beta = 0 kept a histogram of the picks' U, which gives the bound at once;
// otherwise the radix select of launch_select.
hipError_t launch_select_cas(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, uint32_t beta_q16,
                             int32_t* center_lin, int32_t* m_valid, hipStream_t s);

// The paper's challenger / incumbent CAS: RVS incumbents, then one
// workgroup per cloud walks the challengers.
bool cas_swap_fits(const Layout& L, const cagq_grid_desc& d, int32_t M);
hipError_t launch_cas_swap(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, uint64_t seed,
                           uint32_t beta_q16, int32_t* center_lin, int32_t* m_valid, hipStream_t s);

// The words the CAS rounds on lists start from: per slot zero coverage,
// pick, pick round and rescoring round and no blocker; the control block's
// partial slots, done flags and U histogram at zero; and the scan state of
// the selection's compaction after the rounds.
struct CasClear {
    uint32_t* cover;
    uint64_t* pick;
    uint32_t* round;
    int32_t* blocker;
    uint32_t* dirty;
    uint64_t* gpart;
    uint32_t* cpart;
    uint32_t* done;
    uint32_t* ndone;
    uint32_t* uhist;
    int32_t nparts;  // entries of gpart and of cpart
    int32_t nhist;   // entries of uhist
    uint64_t* desc;  // the compaction's tile descriptors
    int32_t ndesc;
    int* ticket;     // the compaction's tile ticket
};

// Writes the CAS neighbour lists of the grid in whichever format the layout
// holds (has_nbr16 or has_nbr32). With u32 lists and `key` given, also sets
// each occupied voxel's round-0 key, cas_key(unit * entries within r, lin),
// and with `clr` given clears the rounds' state (a launch of its own before).
hipError_t launch_cas_nbr(const Layout& L, const cagq_grid_desc& d, void* ws, hipStream_t s,
                          uint64_t* key = nullptr, int64_t unit = 0, const CasClear* clr = nullptr);

// Greedy coverage-aware sampling (rounds of neighbourhood maxima).
hipError_t run_cas(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M,
                   uint32_t beta_q16, hipStream_t s, int* status_out);

// The same greedy for small clouds with beta = 0: one workgroup per cloud
// holds every round's state in LDS and also selects and emits the centers.
bool cas_lds_fits(const Layout& L, const cagq_grid_desc& d, uint32_t beta_q16);
hipError_t launch_cas_lds(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, int32_t* center_lin,
                          int32_t* m_valid, hipStream_t s);

// Context lists (Sec. 3.3, grid context pooling): CSR offsets over the batch
// of every center's context count, then the lists themselves.
hipError_t launch_context_offsets(const Layout& L, const cagq_grid_desc& d, void* ws, const int32_t* center_lin,
                                  int32_t M, int64_t* ctx_off, hipStream_t s);
hipError_t launch_context_list(const Layout& L, const cagq_grid_desc& d, void* ws, const int32_t* center_lin,
                               int32_t M, const int64_t* ctx_off, int32_t* ctx_idx, int64_t capacity,
                               hipStream_t s);

// Comparison methods of Sec. 4 and the coverage metric.
hipError_t launch_sample_points(const float* points, int32_t B, int32_t N, int32_t M, int32_t mode, uint64_t seed,
                                int32_t* center_idx, hipStream_t s);
hipError_t launch_ball_query(const float* points, int32_t B, int32_t N, const int32_t* center_idx, int32_t M,
                             int32_t K, float radius2, int32_t* node_idx, int32_t* n_valid, hipStream_t s);
hipError_t launch_coverage(const Layout& L, const cagq_grid_desc& d, const float* points, void* ws,
                           const int32_t* node_idx, const int32_t* n_valid, int32_t M, int32_t K, int32_t* covered,
                           hipStream_t s);
constexpr int32_t kFpsMaxN = 80 * 1024;  // points per cloud Farthest Point Sampling keeps in registers

// Upsampling query around given center points [B][M][3] (Sec. 3.1).
hipError_t launch_query_points(const Layout& L, const cagq_grid_desc& d, void* ws, const float* centers, int32_t M,
                               int32_t K, int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                               int32_t* n_valid, int32_t* ctx_count, int32_t* center_lin, hipStream_t s);

hipError_t launch_query(const Layout& L, const cagq_grid_desc& d, const float* points, void* ws,
                        const uint32_t* weights, const int32_t* center_lin, int32_t M, int32_t K,
                        int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                        int32_t* n_valid, float* center_xyz, uint32_t* center_w,
                        int32_t* ctx_count, hipStream_t s);

}  // namespace cagq
