// Node points querying and group centers (Sec. 3.2 "Node points querying";
// Appendix D, general procedure, step 3; Appendix E, Eqs. 7-8).
//
// One group of G lanes (G = 16, 32 or 64, G >= K; a whole wave with two
// result registers per lane for 64 < K <= 128) per center voxel v, 64/G
// centers per wavefront:
//   1. the group's lanes probe the (2r+1)^3 voxels of pi(v) in the occupancy
//      bitmap and compact the occupied ones (slot start, running context
//      count) into LDS -- the context is the concatenation of their stored
//      lists, c points;
//   2. context points are streamed G at a time from the slot-ordered copy of
//      the stored points (one 16-byte load gives x, y, z and the index); each
//      lane forms a 64-bit key, (hi32(h(seed,2,b,lin(v),i)) << 32) | i for
//      Cube Query or (bits(d^2) << 32) | i for k-NN, d measured from the
//      center of v;
//   3. a bitonic sort of the chunk across the group is merged into the
//      running G smallest keys (each key carries its position in the copy);
//      lanes 0..min(K, c)-1 end up holding the node points in key order;
//   4. node coordinates are bit copies re-read from the copy; w_c is the
//      integer sum of the node weights and chi_c the pairwise fp32 sum of
//      w_k * p_k (shuffle-down tree: stride 1, 2, 4, ...) divided by w_c.
//
// The level-wise k-NN (Appendix D, "CAGQ k-NN": levels 0..r of pi(v), a
// level that fits in what is left of K taken whole as gathered, otherwise its
// nearest points) probes the block level by level, so that the context is
// compacted level-major and the levels' cumulative counts fall out of the
// probe. With L* the first level whose cumulative count reaches K, only the
// entries up to the end of L* are streamed; entry e gets the key e (gathering
// order) before L*'s first entry, or throughout when L* fits exactly, and
// (1 << 62) | (bits(d^2) << 31) | i inside a level L* that does not fit: the
// K smallest keys are the procedure's nodes, in its order.
//
// The upsampling variant (Sec. 3.1: centers arrive through long-range
// connections, only their nodes are queried) takes center points instead:
// v is the voxel a point falls in (it need not be occupied), k-NN distances
// are measured from the point itself, an empty context gives index -1, and
// no group center is formed.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kQueryThreads = 256;

// Division by a divisor d that is the same for the whole launch, for
// dividends below 2^31: floor(n / d) = (n * m) >> (31 + l) with
// l = ceil(log2 d) and m = ceil(2^(31+l) / d) < 2^32 (Granlund and
// Montgomery, "Division by invariant integers using multiplication", 1994).
struct Magic {
    uint32_t m, sh;
};

Magic make_magic(uint32_t d) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    const uint64_t p = 1ull << (31 + l);
    return Magic{(uint32_t)((p + d - 1) / d), 31 + l};
}

__device__ __forceinline__ uint32_t udiv(uint32_t n, const Magic& g) {
    return (uint32_t)(((uint64_t)n * g.m) >> g.sh);
}

constexpr int kRing = CAGQ_QUERY_KNN_RING;  // the level-wise k-NN mode

// The voxels of the (2R+1)^3 block, R = 3, level by level (Chebyshev distance
// 0, 1, 2, 3), each level in ascending (dz, dy, dx); packed (dx+3) |
// (dy+3) << 4 | (dz+3) << 8. The first (2r+1)^3 entries are the block of
// radius r in the same order.
struct Shells {
    uint32_t v[343];
};

constexpr Shells make_shells() {
    Shells t{};
    int n = 0;
    for (int lev = 0; lev <= 3; ++lev)
        for (int dz = -lev; dz <= lev; ++dz)
            for (int dy = -lev; dy <= lev; ++dy)
                for (int dx = -lev; dx <= lev; ++dx) {
                    const int ax = dx < 0 ? -dx : dx, ay = dy < 0 ? -dy : dy, az = dz < 0 ? -dz : dz;
                    const int m = ax > ay ? (ax > az ? ax : az) : (ay > az ? ay : az);
                    if (m == lev) t.v[n++] = (uint32_t)(dx + 3) | (uint32_t)(dy + 3) << 4 | (uint32_t)(dz + 3) << 8;
                }
    return t;
}

__constant__ Shells kShells = make_shells();

struct QGrid {
    float o[3];
    float s[3];
    int32_t D[3];
    Magic d0, d01, mm;  // division by D_x, by D_x * D_y and by M
};

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Value of lane `lane ^ j` (j a power of two below 64, known at compile time
// once unrolled): DPP moves within rows of 16 lanes for j <= 8 (quad
// permutes for 1 and 2, both row shifts for 4, a row rotate for 8), a
// swizzle for 16 and a permute for 32. None of them touches LDS memory.
__device__ __forceinline__ uint32_t xlane(uint32_t v, int j) {
    switch (j) {
        case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, true);  // quad_perm 1,0,3,2
        case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, true);  // quad_perm 2,3,0,1
        case 4: {
            const uint32_t up = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x104, 0xF, 0xF, true);  // row_shl:4
            const uint32_t dn = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x114, 0xF, 0xF, true);  // row_shr:4
            return (threadIdx.x & 4) ? dn : up;
        }
        case 8: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, true);  // row_ror:8
        case 16: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);  // xor 16 within 32 lanes
        default: return (uint32_t)__shfl_xor((int)v, j, kWave);
    }
}

__device__ __forceinline__ float xlanef(float v, int j) { return __uint_as_float(xlane(__float_as_uint(v), j)); }

__device__ __forceinline__ uint64_t xlane64(uint64_t v, int j) {
    return ((uint64_t)xlane((uint32_t)(v >> 32), j) << 32) | xlane((uint32_t)v, j);
}

// One 12-byte store of a node's coordinates (a single dwordx3 store: the
// group's nodes land as one contiguous run).
__device__ __forceinline__ void store_xyz(float* p, float x, float y, float z) {
    typedef float f3 __attribute__((ext_vector_type(3)));
    f3 v;
    v.x = x;
    v.y = y;
    v.z = z;
    __builtin_nontemporal_store(v, reinterpret_cast<f3*>(p));
}

// Value of lane `first` (0 or G-1) of this lane's group of G, by lane reads.
template <int G>
__device__ __forceinline__ uint32_t gbcast(uint32_t v, int first) {
    const int lane = lane_id();
    uint32_t r = 0;
#pragma unroll
    for (int g0 = 0; g0 < kWave; g0 += G) {
        const uint32_t x = (uint32_t)__builtin_amdgcn_readlane((int)v, g0 + first);
        r = (lane >= g0 && lane < g0 + G) ? x : r;
    }
    return r;
}

template <int G>
__device__ __forceinline__ uint64_t gshfl64(uint64_t v, int src) {
    int lo = __shfl((int)(uint32_t)v, src, G);
    int hi = __shfl((int)(uint32_t)(v >> 32), src, G);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

template <int G>
__device__ __forceinline__ uint32_t gscan_incl(uint32_t v, int lg) {
#pragma unroll
    for (int d = 1; d < G; d <<= 1) {
        uint32_t o = (uint32_t)__shfl_up((int)v, d, G);
        if (lg >= d) v += o;
    }
    return v;
}

// Compare-exchange of (key, payload) with the partner lane lg ^ j: this lane
// keeps the smaller key when keep_min, else the larger.
__device__ __forceinline__ void gcx(uint64_t& k, uint32_t& p, int j, bool keep_min) {
    const uint64_t ok = xlane64(k, j);
    const uint32_t op = xlane(p, j);
    // keys are distinct but for the ~0 fillers, which may trade places freely
    const bool take = (ok < k) == keep_min;
    if (take) {
        k = ok;
        p = op;
    }
}

// Ascending bitonic sort of one (key, payload) per lane across the group,
// given that only lanes below `top` (a power of two, the same for the whole
// wave) hold keys other than ~0: the merge levels above `top` change nothing
// and are skipped.
template <int G>
__device__ __forceinline__ void gsort(uint64_t& k, uint32_t& p, int lg, uint32_t top) {
#pragma unroll
    for (int s = 2; s <= G; s <<= 1) {
        if ((uint32_t)s > top && s > 2) break;
#pragma unroll
        for (int j = s >> 1; j > 0; j >>= 1) {
            const bool asc = (lg & s) == 0;
            const bool low = (lg & j) == 0;
            gcx(k, p, j, asc == low);
        }
    }
}

// `bk` and `ak` each sorted ascending across the group: bk receives the G
// smallest of their union, sorted ascending.
template <int G>
__device__ __forceinline__ void gmerge_low(uint64_t& bk, uint32_t& bp, uint64_t ak, uint32_t ap, int lg) {
    const uint64_t rk = gshfl64<G>(ak, G - 1 - lg);
    const uint32_t rp = (uint32_t)__shfl((int)ap, G - 1 - lg, G);
    if (rk < bk) {  // bitonic: the G smallest of the union
        bk = rk;
        bp = rp;
    }
#pragma unroll
    for (int j = G >> 1; j > 0; j >>= 1) gcx(bk, bp, j, (lg & j) == 0);
}

// `bk` and `b1` sorted ascending across the group with every key of bk below
// every key of b1 (ranks 0..G-1 and G..2G-1 of the keys seen so far), and a
// chunk `ak` sorted ascending: bk and b1 receive ranks 0..2G-1 of the union.
// The G smallest of b1 and the chunk hold every key of rank below 2G that
// is not in bk; bk and those are then split by a bitonic merge.
template <int G>
__device__ __forceinline__ void gmerge_low2(uint64_t& bk, uint32_t& bp, uint64_t& b1k, uint32_t& b1p, uint64_t ak,
                                            uint32_t ap, int lg) {
    gmerge_low<G>(b1k, b1p, ak, ap, lg);
    const uint64_t rk = gshfl64<G>(b1k, G - 1 - lg);
    const uint32_t rp = (uint32_t)__shfl((int)b1p, G - 1 - lg, G);
    const bool sw = rk < bk;
    b1k = sw ? bk : rk;
    b1p = sw ? bp : rp;
    bk = sw ? rk : bk;
    bp = sw ? rp : bp;
#pragma unroll
    for (int j = G >> 1; j > 0; j >>= 1) {
        gcx(bk, bp, j, (lg & j) == 0);
        gcx(b1k, b1p, j, (lg & j) == 0);
    }
}

// NR result registers per lane: NR = 1 keeps ranks 0..G-1 (K <= G), NR = 2
// (G = 64) also ranks 64..127 in a second register (64 < K <= 128).
// DEFER: the second pass of a query whose 16-lane kernel left its largest
// contexts (n_valid marked -1) to one wave each (G = 64); every other
// center's wave returns at once. D: chunks whose points are loaded ahead.
template <int MODE, int G, int RAD, bool UP, int NR, bool DEFER = false, int D = 1>
__global__ __launch_bounds__(kQueryThreads) void k_query(
    const uint32_t* __restrict__ Wt, int32_t N, int32_t M, int32_t K, int32_t total, QGrid g,
    int64_t W, const uint64_t* __restrict__ bitmap, const uint32_t* __restrict__ word_rank,
    const uint32_t* __restrict__ vox_off, const float4* __restrict__ pt4, const int32_t* __restrict__ center_lin,
    const float* __restrict__ center_pts, uint64_t seed, int32_t* __restrict__ node_idx,
    float* __restrict__ node_xyz, int32_t* __restrict__ n_valid, float* __restrict__ center_xyz,
    uint32_t* __restrict__ center_w, int32_t* __restrict__ ctx_count, int32_t* __restrict__ lin_out,
    int* __restrict__ status) {
    extern __shared__ uint32_t smem[];
    constexpr int GPB = kQueryThreads / G;  // groups per block
    constexpr int rad = RAD, side = 2 * RAD + 1, nnb = side * side * side;
    const int lane = lane_id();
    const int lg = lane & (G - 1);
    const int gb = threadIdx.x / G;  // group within the block
    uint32_t* s_pre = smem + (size_t)gb * (2 * nnb + 1);
    uint32_t* s_st = s_pre + nnb + 1;
    // the deferred pass spreads neighbouring (similarly long) contexts over
    // the XCDs round-robin; the others keep neighbours on one XCD's L2
    const uint32_t blk = DEFER ? blockIdx.x : xcd_block(blockIdx.x, gridDim.x);
    const int32_t cid = (int32_t)blk * GPB + gb;
    // every group runs to the end (the group- and wave-wide steps need all
    // lanes); a group past the end works on center 0 and writes nothing
    const bool live = cid < total;
    if constexpr (DEFER) {
        static_assert(G == kWave, "one center per wave");
        if (!live || n_valid[cid] != -1) return;  // the whole wave: no block-wide step follows
    }
    const int32_t c_id = live ? cid : 0;
    const int32_t b = (int32_t)udiv((uint32_t)c_id, g.mm);
    const size_t cK = (size_t)c_id * K;
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    const uint32_t* vo = vox_off + (size_t)b * (N + 1);
    const float4* p4 = pt4 + (size_t)b * N;
    bool in_grid = true;
    uint32_t lin;
    int32_t gx, gy, gz;
    float px = 0.f, py = 0.f, pz = 0.f;  // the given center point (upsampling)
    if constexpr (UP) {
        px = center_pts[(size_t)c_id * 3 + 0];
        py = center_pts[(size_t)c_id * 3 + 1];
        pz = center_pts[(size_t)c_id * 3 + 2];
        const bool bad = !isfinite(px) || !isfinite(py) || !isfinite(pz);
        gx = isfinite(px) ? axis_index(px, g.o[0], g.s[0], g.D[0]) : 0;
        gy = isfinite(py) ? axis_index(py, g.o[1], g.s[1], g.D[1]) : 0;
        gz = isfinite(pz) ? axis_index(pz, g.o[2], g.s[2], g.D[2]) : 0;
        lin = (uint32_t)gx + (uint32_t)g.D[0] * ((uint32_t)gy + (uint32_t)g.D[1] * (uint32_t)gz);
        if (live && bad && lg == 0) raise_error(status, CAGQ_ERR_NONFINITE_INPUT);
    } else {
        const int32_t lin_s = center_lin[c_id];
        const int64_t V = (int64_t)g.D[0] * g.D[1] * g.D[2];
        in_grid = lin_s >= 0 && (int64_t)lin_s < V;
        lin = in_grid ? (uint32_t)lin_s : 0u;
        const uint32_t zq = udiv(lin, g.d01);
        const uint32_t rem = lin - zq * (uint32_t)g.D[0] * (uint32_t)g.D[1];
        const uint32_t yq = udiv(rem, g.d0);
        gx = (int32_t)(rem - yq * (uint32_t)g.D[0]), gy = (int32_t)yq, gz = (int32_t)zq;
    }

    // 1. occupied voxels of pi(v), compacted in ascending linear id; the
    // center voxel is one of them (q = nnb / 2), so its own check costs
    // nothing extra
    uint32_t nocc = 0, c = 0;
    uint32_t cum[RAD + 1];  // level-wise mode: context points of levels 0..l
    bool occupied = false;
    const int gshift = lane & ~(G - 1);
    const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
    for (int q0 = 0; q0 < nnb; q0 += G) {
        const int q = q0 + lg;
        bool occ = false;
        uint32_t st = 0, cnt = 0;
        if (in_grid && q < nnb) {
            int32_t x, y, z;
            if (MODE == kRing) {
                const uint32_t o = kShells.v[q];
                x = gx + (int32_t)(o & 15u) - 3;
                y = gy + (int32_t)((o >> 4) & 15u) - 3;
                z = gz + (int32_t)(o >> 8) - 3;
            } else {
                x = gx + q % side - rad;
                y = gy + (q / side) % side - rad;
                z = gz + q / (side * side) - rad;
            }
            if (x >= 0 && y >= 0 && z >= 0 && x < g.D[0] && y < g.D[1] && z < g.D[2]) {
                const uint32_t nl = (uint32_t)x + (uint32_t)g.D[0] * ((uint32_t)y + (uint32_t)g.D[1] * (uint32_t)z);
                const int32_t sl = slot_of(bm, wr, nl);
                if (sl >= 0) {
                    st = vo[sl];
                    cnt = vo[sl + 1] - st;
                    occ = true;
                }
            }
        }
        const uint64_t mask = (__ballot(occ) >> gshift) & gmask;
        constexpr int qc = MODE == kRing ? 0 : nnb / 2;  // the center voxel's probe index
        if (qc >= q0 && qc < q0 + G) occupied = (mask >> (qc - q0)) & 1ull;
        const uint32_t pos = nocc + (uint32_t)__popcll(mask & ((1ull << lg) - 1));
        const uint32_t incl = gscan_incl<G>(cnt, lg);
        if (occ) {
            s_st[pos] = st;
            s_pre[pos] = c + incl - cnt;
        }
        if (MODE == kRing) {
            // level l ends at probe index (2l+1)^3 - 1
#pragma unroll
            for (int l = 0; l <= RAD; ++l) {
                const int last = (2 * l + 1) * (2 * l + 1) * (2 * l + 1) - 1;
                if (last >= q0 && last < q0 + G) cum[l] = c + (uint32_t)__shfl((int)incl, last - q0, G);
            }
        }
        c += gbcast<G>(incl, G - 1);
        nocc += (uint32_t)__popcll(mask);
    }
    // a sampled center that is not occupied has an empty context and gets
    // zeros (an upsampling center's voxel may be empty)
    if (!UP) {
        if (live && !occupied && lg == 0) raise_error(status, CAGQ_ERR_CENTER_NOT_OCCUPIED);
        if (!occupied) {
            nocc = 0;
            c = 0;
        }
    }
    if (lg == 0) s_pre[nocc] = c;
    wave_lds_sync();

    // 2-3. keys of the context points, G smallest kept sorted across the group
    uint64_t hc = 0;
    float qx = 0.f, qy = 0.f, qz = 0.f;
    if (MODE == CAGQ_QUERY_CUBE) {
        hc = sm64(sm64(sm64(seed ^ 2ull) ^ (uint64_t)b) ^ (uint64_t)lin);
    } else if (UP) {
        qx = px;
        qy = py;
        qz = pz;
    } else {
        qx = g.o[0] + ((float)gx + 0.5f) * g.s[0];
        qy = g.o[1] + ((float)gy + 0.5f) * g.s[1];
        qz = g.o[2] + ((float)gz + 0.5f) * g.s[2];
    }
    // the entries streamed: all c, or in the level-wise mode those up to the
    // end of L*, the first level whose cumulative count reaches K; `base` is
    // where L* starts, `part` whether L* is cut
    uint32_t cs = c, base = 0;
    bool part = false;
    if (MODE == kRing && c >= (uint32_t)K) {
        int ls = RAD;
#pragma unroll
        for (int l = RAD - 1; l >= 0; --l)
            if (cum[l] >= (uint32_t)K) ls = l;
        cs = cum[ls];
        base = 0;
#pragma unroll
        for (int l = 0; l < RAD; ++l)
            if (l + 1 == ls) base = cum[l];
        part = cs > (uint32_t)K;
    }
    static_assert(NR == 1 || (NR == 2 && G == kWave), "two result registers need a whole wave");
    uint64_t bk = ~0ull, b1k = ~0ull;
    uint32_t bp = 0, b1p = 0;
    // the chunk loop runs the same number of times for every group of the wave
    uint32_t cmax = cs;
#pragma unroll
    for (int d = G; d < kWave; d <<= 1) {
        const uint32_t o = xlane(cmax, d);
        cmax = o > cmax ? o : cmax;
    }
    cmax = (uint32_t)__builtin_amdgcn_readfirstlane((int)cmax);  // the same in every lane
    // a context of at most G points is one chunk: its points and weights stay
    // in the lanes that loaded them, and the sort carries the lane (entry)
    // instead of the position in the copy
    const bool one = cs <= (uint32_t)G;
    // the sort levels that matter: up to the smallest power of two >= cmax
    uint32_t top = 2;
    while (top < cmax && top < (uint32_t)G) top <<= 1;
    float4 v0 = make_float4(0.f, 0.f, 0.f, 0.f);
    uint32_t w0 = 1u;
    // position in the copy of context entry e: the compacted voxel holding it
    auto locate = [&](uint32_t e) {
        uint32_t lo = 0, hi = nocc - 1;
        while (lo < hi) {
            const uint32_t mid = (lo + hi + 1) >> 1;
            if (s_pre[mid] <= e) lo = mid; else hi = mid - 1;
        }
        return s_st[lo] + (e - s_pre[lo]);
    };
    if constexpr (DEFER) {
        // A long context, one wave: the keys below the K-th best so far are
        // gathered in an LDS buffer of 64 and sorted and merged only when it
        // is full (at the end, what is left). The chunk's positions come from
        // a walk over the compacted voxels that the whole wave shares: the
        // voxel holding the chunk's first entry, and the voxel starts inside
        // the chunk as one 64-bit mask (every compacted voxel holds at least
        // one point, so at most 64 of them start inside a chunk).
        static_assert(G == kWave, "one center per wave");
        uint64_t* cbk = reinterpret_cast<uint64_t*>(smem + ((GPB * (2 * nnb + 1) + 1) & ~1)) + gb * kWave;
        uint32_t* cbp = reinterpret_cast<uint32_t*>(cbk + (GPB - gb) * kWave) + gb * kWave;
        uint32_t wv = 0;  // the compacted voxel holding the walk's next chunk start
        auto walk = [&](uint32_t c0) {
            const uint32_t j = wv + 1 + (uint32_t)lg;
            const uint32_t bj = j < nocc ? s_pre[j] - c0 : 65u;  // >= 1: voxel j starts after c0
            uint64_t mk = bj < 64 ? (1ull << bj) : 0ull;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) mk |= shfl_xor64(mk, d);
            const uint32_t v = wv + (uint32_t)__popcll(mk & ((2ull << lg) - 1));
            wv += (uint32_t)__popcll(mk) + (__ballot(bj == 64) ? 1u : 0u);
            return s_st[v] + (c0 + (uint32_t)lg - s_pre[v]);
        };
        uint32_t pq[D];
        float4 vq[D];
#pragma unroll
        for (int d = 0; d < D; ++d) {
            pq[d] = walk((uint32_t)(d * G));
            vq[d] = make_float4(0.f, 0.f, 0.f, 0.f);
            if ((uint32_t)(d * G + lg) < cs) vq[d] = p4[pq[d]];
        }
        uint64_t kth = ~0ull;
        uint32_t fill = 0;
        auto flush = [&]() {
            uint64_t key = (uint32_t)lg < fill ? cbk[lg] : ~0ull;
            uint32_t pos = (uint32_t)lg < fill ? cbp[lg] : 0u;
            gsort<G>(key, pos, lg, (uint32_t)G);
            if (NR == 1)
                gmerge_low<G>(bk, bp, key, pos, lg);
            else
                gmerge_low2<G>(bk, bp, b1k, b1p, key, pos, lg);
            kth = NR == 1 ? gshfl64<G>(bk, K - 1) : gshfl64<G>(b1k, K - 1 - G);
            fill = 0;
        };
        for (uint32_t e0 = 0; e0 < cmax; e0 += G) {
            const uint32_t e = e0 + lg;
            const uint32_t pos = pq[0];
            const float4 v = vq[0];
#pragma unroll
            for (int d = 0; d + 1 < D; ++d) {
                pq[d] = pq[d + 1];
                vq[d] = vq[d + 1];
            }
            if (e0 + D * G < cs) {  // the wave's next chunk to load
                pq[D - 1] = walk(e0 + D * G);
                if (e + D * G < cs) vq[D - 1] = p4[pq[D - 1]];
            }
            uint64_t key = ~0ull;
            if (e < cs) {
                const uint32_t i = __float_as_uint(v.w);
                if (MODE == CAGQ_QUERY_CUBE) {
                    key = (sm64(hc ^ (uint64_t)i) & 0xFFFFFFFF00000000ull) | i;
                } else {
                    const float dx = v.x - qx, dy = v.y - qy, dz = v.z - qz;
                    const float xx = dx * dx, yy = dy * dy, zz = dz * dz;
                    const float sxy = xx + yy;
                    const float d2 = sxy + zz;
                    key = ((uint64_t)__float_as_uint(d2) << 32) | i;
                }
                key = key < kth ? key : ~0ull;
            }
            const uint64_t m = __ballot(key != ~0ull);
            const uint32_t nc = (uint32_t)__popcll(m);
            if (fill + nc > (uint32_t)kWave) {
                flush();
                wave_lds_sync();
                // the new keys against the new K-th best
                key = key < kth ? key : ~0ull;
            }
            const uint64_t m2 = __ballot(key != ~0ull);
            if (key != ~0ull) {
                const uint32_t at_ = fill + (uint32_t)__popcll(m2 & ((1ull << lg) - 1));
                cbk[at_] = key;
                cbp[at_] = pos;
            }
            fill += (uint32_t)__popcll(m2);
            wave_lds_sync();
        }
        if (fill) flush();
    } else {
    // each chunk's points are loaded D chunks ahead, so that a long
    // context's loads overlap the sort and merge of the chunks before
    uint32_t pq[D];
    float4 vq[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
        const uint32_t e = (uint32_t)(d * G + lg);
        pq[d] = 0;
        vq[d] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (e < cs) {
            pq[d] = locate(e);
            vq[d] = p4[pq[d]];
        }
    }
    uint64_t kth = ~0ull;
    for (uint32_t e0 = 0; e0 < cmax; e0 += G) {
        const uint32_t e = e0 + lg;
        uint64_t key = ~0ull;
        uint32_t pos = pq[0];
        const float4 v = vq[0];
#pragma unroll
        for (int d = 0; d + 1 < D; ++d) {
            pq[d] = pq[d + 1];
            vq[d] = vq[d + 1];
        }
        if (e + D * G < cs) {
            pq[D - 1] = locate(e + D * G);
            vq[D - 1] = p4[pq[D - 1]];
        }
        if (e < cs) {
            const uint32_t i = __float_as_uint(v.w);
            if (one) {
                v0 = v;
                if (Wt) w0 = Wt[(size_t)b * N + i];
                pos = e;
            }
            if (MODE == CAGQ_QUERY_CUBE) {
                key = (sm64(hc ^ (uint64_t)i) & 0xFFFFFFFF00000000ull) | i;
            } else {
                const float dx = v.x - qx, dy = v.y - qy, dz = v.z - qz;
                const float xx = dx * dx, yy = dy * dy, zz = dz * dz;
                const float sxy = xx + yy;
                const float d2 = sxy + zz;
                if (MODE == kRing)
                    key = (part && e >= base) ? (1ull << 62) | ((uint64_t)__float_as_uint(d2) << 31) | i
                                              : (uint64_t)e;
                else
                    key = ((uint64_t)__float_as_uint(d2) << 32) | i;
            }
        } else {
            pos = 0;
        }
        // a key above the K-th best so far can never be kept (keys are
        // distinct); a chunk left without keys anywhere in the wave changes
        // nothing and is not sorted
        if (e0 != 0) {
            key = key < kth ? key : ~0ull;
            if (!__ballot(key != ~0ull)) continue;
        }
        gsort<G>(key, pos, lg, top);
        if (e0 == 0) {
            bk = key;
            bp = pos;
        } else if (NR == 1) {
            gmerge_low<G>(bk, bp, key, pos, lg);
        } else {
            gmerge_low2<G>(bk, bp, b1k, b1p, key, pos, lg);
        }
        // the K-th best key so far (a filler, ~0, while fewer than K are held)
        kth = NR == 1 ? gshfl64<G>(bk, K - 1) : gshfl64<G>(b1k, K - 1 - G);
    }
    }

    // 4. outputs (an empty context gives n = 0 and zeros): node slot k is
    // lane k of the first register or lane k - G of the second; slots k >= n
    // repeat slot 0
    const uint32_t n = c < (uint32_t)K ? c : (uint32_t)K;
    const uint64_t k0 = ((uint64_t)gbcast<G>((uint32_t)(bk >> 32), 0) << 32) | gbcast<G>((uint32_t)bk, 0);
    const uint32_t p0 = gbcast<G>(bp, 0);
    float tx = 0.f, ty = 0.f, tz = 0.f, ux = 0.f, uy = 0.f, uz = 0.f;
    uint32_t wsum = 0;
#pragma unroll
    for (int h = 0; h < NR; ++h) {
        const uint32_t k = (uint32_t)(h * G + lg);
        const bool own = k < n;
        const uint64_t mine = own ? (h ? b1k : bk) : k0;
        const uint32_t mpos = own ? (h ? b1p : bp) : p0;
        // the node's point index is the key's low half, except in the
        // level-wise mode, whose keys order by position: there it comes with
        // the point
        uint32_t idx = n ? (uint32_t)mine : 0u;
        // a one-chunk context reads node point and weight from the lane
        // holding them; a longer one reads them again
        const int from = one ? (int)mpos : 0;
        float x = __shfl(v0.x, from, G), y = __shfl(v0.y, from, G), z = __shfl(v0.z, from, G);
        uint32_t w = (uint32_t)__shfl((int)w0, from, G);
        if (MODE == kRing) idx = (uint32_t)__shfl((int)__float_as_uint(v0.w), from, G);
        if (!one) {
            const float4 pv = p4[mpos];
            x = pv.x;
            y = pv.y;
            z = pv.z;
            if (MODE == kRing) idx = __float_as_uint(pv.w);
            w = Wt ? Wt[(size_t)b * N + idx] : 1u;
        }
        if (!n) {
            x = y = z = 0.0f;
            w = 1u;
            idx = 0u;
        }
        if (live && k < (uint32_t)K) {
            node_idx[cK + k] = UP ? (n ? (int32_t)idx : -1) : (int32_t)idx;
            if (node_xyz) {
                store_xyz(node_xyz + (cK + k) * 3, x, y, z);
            }
        }
        const float wf = (float)w;
        if (h == 0) {
            tx = wf * x, ty = wf * y, tz = wf * z;
        } else {
            ux = wf * x, uy = wf * y, uz = wf * z;
        }
        wsum += own ? w : 0u;
    }
    if (UP) {
        if (live && lg == 0) {
            n_valid[cid] = (int32_t)n;
            if (ctx_count) ctx_count[cid] = (int32_t)c;
            if (lin_out) lin_out[cid] = (int32_t)lin;
        }
        return;
    }
    // n <= top, or n > G = top with two registers: the levels at and above
    // `top` add nothing
    uint32_t wc = wsum;
#pragma unroll
    for (int d = 1; d < G; d <<= 1)
        if ((uint32_t)d < top) wc += xlane(wc, d);
#pragma unroll
    for (int h = 1; h < G; h <<= 1) {
        if ((uint32_t)h >= top) break;
        // the lanes that add (multiples of 2h) read lane + h = lane ^ h
        const bool lead = (lg & (2 * h - 1)) == 0;
        const float ox = xlanef(tx, h);
        const float oy = xlanef(ty, h);
        const float oz = xlanef(tz, h);
        if (lead && (uint32_t)(lg + h) < n) {
            tx = tx + ox;
            ty = ty + oy;
            tz = tz + oz;
        }
        if (NR == 2 && cmax > (uint32_t)G) {
            const float px = xlanef(ux, h), py = xlanef(uy, h), pz = xlanef(uz, h);
            if (lead && (uint32_t)(G + lg + h) < n) {
                ux = ux + px;
                uy = uy + py;
                uz = uz + pz;
            }
        }
    }
    if (NR == 2 && n > (uint32_t)G) {  // stride G: node G into node 0 (lane 0)
        tx = tx + ux;
        ty = ty + uy;
        tz = tz + uz;
    }
    // lanes 0, 1, 2 of the group each divide one of lane 0's sums
    const float sx = __uint_as_float((uint32_t)__builtin_amdgcn_mov_dpp((int)__float_as_uint(tx), 0x00, 0xF, 0xF, true));
    const float sy = __uint_as_float((uint32_t)__builtin_amdgcn_mov_dpp((int)__float_as_uint(ty), 0x00, 0xF, 0xF, true));
    const float sz = __uint_as_float((uint32_t)__builtin_amdgcn_mov_dpp((int)__float_as_uint(tz), 0x00, 0xF, 0xF, true));
    const uint32_t sw = (uint32_t)__builtin_amdgcn_mov_dpp((int)wc, 0x00, 0xF, 0xF, true);  // quad_perm 0,0,0,0
    if (live && lg < 3) {
        const float num = lg == 0 ? sx : (lg == 1 ? sy : sz);
        center_xyz[(size_t)cid * 3 + lg] = n ? num / (float)sw : 0.0f;
    }
    if (live && lg == 0) {
        center_w[cid] = wc;
        n_valid[cid] = (int32_t)n;
        if (ctx_count) ctx_count[cid] = (int32_t)c;
    }
}

// Value of lane 15 - l within the 16-lane row (DPP row_mirror).
__device__ __forceinline__ uint32_t mirror(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, true);
}

__device__ __forceinline__ uint64_t mirror64(uint64_t v) {
    return ((uint64_t)mirror((uint32_t)(v >> 32)) << 32) | mirror((uint32_t)v);
}

// Value of lane L of this lane's 16-lane row (DPP row_share).
template <int L>
__device__ __forceinline__ uint32_t row_lane(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x150 + L, 0xF, 0xF, true);
}

// Value of lane 0 of this lane's 16-lane row.
__device__ __forceinline__ uint32_t row0(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x150, 0xF, 0xF, true);  // row_share:0
}

// Bitonic half-cleaners j = 8, 4, 2, 1 over a 16-lane row: a bitonic
// sequence ends ascending.
__device__ __forceinline__ void clean16(uint64_t& k, uint32_t& p, int lg) {
#pragma unroll
    for (int j = 8; j > 0; j >>= 1) gcx(k, p, j, (lg & j) == 0);
}

// Sampled centers with 16 < K <= 32, Cube Query or k-NN: 16 lanes per center
// (four per wave), two result registers per lane, ranks 0..15 in `b0` and
// 16..31 in `b1`.
//   1. Each group probes the (2r+1)^2 grid rows of its center's block, one
//      lane per row: a row segment of the block holds consecutive slots,
//      whose stored points are contiguous in the slot-ordered copy, so the
//      context is (2r+1)^2 ranges (some empty). Their starts and prefix
//      counts go to LDS, with the center's facts (lin, cloud, reference
//      point, context size).
//   2. The block's 16 centers are ranked by context size and group g takes
//      the center of rank g, so each wave works on four centers of similar
//      size and its chunk loop and sort depth follow them.
//   3. Chunks of 16 entries are sorted across the group; the first is the
//      running best, each later one is merged in: the 16 smallest of b1 and
//      the chunk (elementwise minimum against the chunk reversed, then
//      half-cleaners), then b0 and that merged the same way into the new b0
//      (smaller half) and b1 (larger half).
//   4. Node slot k is b0 lane k or b1 lane k - 16; slots k >= n repeat slot 0.
//      The center's pairwise sum runs strides 1..8 inside each half, then
//      node 16 into node 0 -- the order of the single-register tree.
constexpr int32_t kRankMin = 8192;  // centers of a launch above which k_query_r2 ranks a block's centers

template <int MODE, int RAD, bool UP>
__global__ __launch_bounds__(kQueryThreads) void k_query_r2(
    const uint32_t* __restrict__ Wt, int32_t N, int32_t M, int32_t K, int32_t total, QGrid g,
    int64_t W, const uint64_t* __restrict__ bitmap, const uint32_t* __restrict__ word_rank,
    const uint32_t* __restrict__ vox_off, const float4* __restrict__ pt4, const int32_t* __restrict__ center_lin,
    const float* __restrict__ center_pts, uint64_t seed, int32_t* __restrict__ node_idx,
    float* __restrict__ node_xyz, int32_t* __restrict__ n_valid, float* __restrict__ center_xyz,
    uint32_t* __restrict__ center_w, int32_t* __restrict__ ctx_count, int32_t* __restrict__ lin_out,
    int* __restrict__ status, uint32_t defer) {
    constexpr int G = 16, GPB = kQueryThreads / G;
    constexpr int S = 2 * RAD + 1, NR = S * S;
    __shared__ uint32_t s_st[GPB][NR];
    __shared__ uint32_t s_pre[GPB][NR + 1];
    __shared__ uint32_t s_c[GPB], s_lin[GPB], s_b[GPB];
    __shared__ float s_q[GPB][3];
    __shared__ uint32_t s_src[GPB];
    __shared__ uint32_t s_def[GPB];
    const int lane = lane_id();
    const int lg = lane & (G - 1);
    const int gb = threadIdx.x / G;
    const uint32_t blk = xcd_block(blockIdx.x, gridDim.x);

    // 1. this group's own center
    {
        const int32_t cid = (int32_t)blk * GPB + gb;
        const bool live = cid < total;
        const int32_t c_id = live ? cid : 0;
        const int32_t b = (int32_t)udiv((uint32_t)c_id, g.mm);
        const uint64_t* bm = bitmap + (size_t)b * W;
        const uint32_t* wr = word_rank + (size_t)b * W;
        const uint32_t* vo = vox_off + (size_t)b * (N + 1);
        bool in_grid = true;
        uint32_t lin;
        int32_t gx, gy, gz;
        float qx, qy, qz;
        if constexpr (UP) {
            qx = center_pts[(size_t)c_id * 3 + 0];
            qy = center_pts[(size_t)c_id * 3 + 1];
            qz = center_pts[(size_t)c_id * 3 + 2];
            const bool bad = !isfinite(qx) || !isfinite(qy) || !isfinite(qz);
            gx = isfinite(qx) ? axis_index(qx, g.o[0], g.s[0], g.D[0]) : 0;
            gy = isfinite(qy) ? axis_index(qy, g.o[1], g.s[1], g.D[1]) : 0;
            gz = isfinite(qz) ? axis_index(qz, g.o[2], g.s[2], g.D[2]) : 0;
            lin = (uint32_t)gx + (uint32_t)g.D[0] * ((uint32_t)gy + (uint32_t)g.D[1] * (uint32_t)gz);
            if (live && bad && lg == 0) raise_error(status, CAGQ_ERR_NONFINITE_INPUT);
        } else {
            const int32_t lin_s = center_lin[c_id];
            const int64_t V = (int64_t)g.D[0] * g.D[1] * g.D[2];
            in_grid = lin_s >= 0 && (int64_t)lin_s < V;
            lin = in_grid ? (uint32_t)lin_s : 0u;
            const uint32_t zq = udiv(lin, g.d01);
            const uint32_t rem = lin - zq * (uint32_t)g.D[0] * (uint32_t)g.D[1];
            const uint32_t yq = udiv(rem, g.d0);
            gx = (int32_t)(rem - yq * (uint32_t)g.D[0]), gy = (int32_t)yq, gz = (int32_t)zq;
            qx = g.o[0] + ((float)gx + 0.5f) * g.s[0];
            qy = g.o[1] + ((float)gy + 0.5f) * g.s[1];
            qz = g.o[2] + ((float)gz + 0.5f) * g.s[2];
        }
        // the block's rows: each a range [st, st + len) of the copy
        GridDims gd;
        gd.D[0] = g.D[0], gd.D[1] = g.D[1], gd.D[2] = g.D[2];
        uint32_t c = 0;
        bool occupied = false;
#pragma unroll
        for (int q0 = 0; q0 < NR; q0 += G) {
            const int q = q0 + lg;
            uint32_t st = 0, len = 0, mask = 0;
            if (q < NR) {
                const GridRow r = load_row(bm, wr, gd, gx, gy + q % S - RAD, gz + q / S - RAD, RAD);
                mask = in_grid ? r.mask : 0u;
                st = vo[r.first];
                len = mask ? vo[r.first + (uint32_t)__popc(mask)] - st : 0u;
            }
            static_assert(G == 16, "a group is a 16-lane row");
            if (NR / 2 >= q0 && NR / 2 < q0 + G) occupied = (row_lane<(NR / 2) % G>(mask) >> RAD) & 1;
            // inclusive scan of the lengths across the row of 16 lanes
            uint32_t incl = len;
            incl += dpp_row_shr<1>(incl);
            incl += dpp_row_shr<2>(incl);
            incl += dpp_row_shr<4>(incl);
            incl += dpp_row_shr<8>(incl);
            if (q < NR) {
                s_st[gb][q] = st;
                s_pre[gb][q] = c + incl - len;
            }
            c += row_lane<G - 1>(incl);
        }
        // a sampled center that is not occupied has an empty context and
        // gets zeros (an upsampling center's voxel may be empty)
        if (!UP) {
            if (live && !occupied && lg == 0) raise_error(status, CAGQ_ERR_CENTER_NOT_OCCUPIED);
            if (!occupied) c = 0;
        }
        // a context above `defer` points is left to the one-wave-per-center
        // pass: here it counts as empty, and its n_valid is marked -1
        const bool def = live && c > defer;
        if (lg == 0) {
            s_pre[gb][NR] = c;
            s_def[gb] = def ? 1u : 0u;
            s_c[gb] = live && !def ? c : 0u;
            s_lin[gb] = lin;
            s_b[gb] = (uint32_t)b;
            s_q[gb][0] = qx, s_q[gb][1] = qy, s_q[gb][2] = qz;
        }
    }
    // 2. in a launch of more than kRankMin centers, the block's centers by
    // context size (ties by group): group g takes the center of rank g, so
    // that a wave's four centers are alike. A smaller launch skips the
    // block's two barriers: each group goes on with its own center, whose
    // rows its own wave has put in LDS.
    int src = gb;
    if (total > kRankMin) {
        __syncthreads();
        if (lg == 0) {
            const uint32_t mine = s_c[gb];
            uint32_t r = 0;
#pragma unroll
            for (int h = 0; h < GPB; ++h) {
                const uint32_t o = s_c[h];
                r += (o < mine || (o == mine && h < gb)) ? 1u : 0u;
            }
            s_src[r] = (uint32_t)gb;
        }
        __syncthreads();
        src = (int)s_src[gb];
    } else {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    const int32_t cid = (int32_t)blk * GPB + src;
    if (s_def[src] && lg == 0) n_valid[cid] = -1;
    const bool live = cid < total && !s_def[src];
    const uint32_t c = s_c[src];
    const uint32_t lin = s_lin[src];
    const int32_t b = (int32_t)s_b[src];
    const float qx = s_q[src][0], qy = s_q[src][1], qz = s_q[src][2];
    const uint32_t* s_pr = s_pre[src];
    const uint32_t* s_sr = s_st[src];
    const float4* p4 = pt4 + (size_t)b * N;
    const size_t cK = (size_t)(live ? cid : 0) * K;

    // 3. keys, sorted 16 at a time and merged into the best 32
    uint64_t hc = 0;
    if (MODE == CAGQ_QUERY_CUBE) hc = sm64(sm64(sm64(seed ^ 2ull) ^ (uint64_t)b) ^ (uint64_t)lin);
    uint32_t cmax = c;
#pragma unroll
    for (int d = G; d < kWave; d <<= 1) {
        const uint32_t o = xlane(cmax, d);
        cmax = o > cmax ? o : cmax;
    }
    cmax = (uint32_t)__builtin_amdgcn_readfirstlane((int)cmax);
    const bool one = c <= (uint32_t)G;
    uint32_t top = 2;
    while (top < cmax && top < (uint32_t)G) top <<= 1;
    uint64_t b0k = ~0ull, b1k = ~0ull;
    uint32_t b0p = 0, b1p = 0;
    float4 v0 = make_float4(0.f, 0.f, 0.f, 0.f);
    uint32_t w0 = 1u;
    // position in the copy of context entry e: the last row range starting
    // at or before it
    auto locate = [&](uint32_t e) {
        uint32_t lo = 0, hi = NR - 1;
        while (lo < hi) {
            const uint32_t mid = (lo + hi + 1) >> 1;
            if (s_pr[mid] <= e) lo = mid; else hi = mid - 1;
        }
        return s_sr[lo] + (e - s_pr[lo]);
    };
    // each chunk's points are loaded one chunk ahead, so that a long
    // context's loads overlap the previous chunk's sort and merge
    uint32_t pos_n = 0;
    float4 v_n = make_float4(0.f, 0.f, 0.f, 0.f);
    uint64_t kth = ~0ull;
    if ((uint32_t)lg < c) {
        pos_n = locate((uint32_t)lg);
        v_n = p4[pos_n];
    }
    for (uint32_t e0 = 0; e0 < cmax; e0 += G) {
        const uint32_t e = e0 + lg;
        uint64_t key = ~0ull;
        uint32_t pos = pos_n;
        const float4 v = v_n;
        if (e + G < c) {
            pos_n = locate(e + G);
            v_n = p4[pos_n];
        }
        if (e < c) {
            const uint32_t i = __float_as_uint(v.w);
            if (one) {
                v0 = v;
                if (Wt) w0 = Wt[(size_t)b * N + i];
                pos = (uint32_t)lg;
            }
            if (MODE == CAGQ_QUERY_CUBE) {
                key = (sm64(hc ^ (uint64_t)i) & 0xFFFFFFFF00000000ull) | i;
            } else {
                const float dx = v.x - qx, dy = v.y - qy, dz = v.z - qz;
                const float xx = dx * dx, yy = dy * dy, zz = dz * dz;
                const float sxy = xx + yy;
                const float d2 = sxy + zz;
                key = ((uint64_t)__float_as_uint(d2) << 32) | i;
            }
        } else {
            pos = 0;
        }
        // a key above the K-th best so far can never be kept (keys are
        // distinct); a chunk left without keys anywhere in the wave changes
        // nothing and is not sorted
        if (e0 != 0) {
            key = key < kth ? key : ~0ull;
            if (!__ballot(key != ~0ull)) continue;
        }
        gsort<G>(key, pos, lg, e0 == 0 ? top : (uint32_t)G);
        if (e0 == 0) {
            b0k = key;
            b0p = pos;
        } else {
            // the 16 smallest of b1 and the chunk
            uint64_t rk = mirror64(key);
            uint32_t rp = mirror(pos);
            if (rk < b1k) {
                b1k = rk;
                b1p = rp;
            }
            clean16(b1k, b1p, lg);
            // b0 and those: smaller half to b0, larger to b1
            rk = mirror64(b1k);
            rp = mirror(b1p);
            const bool sw = rk < b0k;
            b1k = sw ? b0k : rk;
            b1p = sw ? b0p : rp;
            b0k = sw ? rk : b0k;
            b0p = sw ? rp : b0p;
            clean16(b0k, b0p, lg);
            clean16(b1k, b1p, lg);
        }
        // the K-th best key so far, rank K-1 in b1 (~0 while fewer than K are held)
        kth = gshfl64<G>(b1k, K - 1 - G);
    }

    // 4. outputs (an empty context gives n = 0)
    const uint32_t n = c < (uint32_t)K ? c : (uint32_t)K;
    uint32_t nmax = n;
#pragma unroll
    for (int d = G; d < kWave; d <<= 1) {
        const uint32_t o = xlane(nmax, d);
        nmax = o > nmax ? o : nmax;
    }
    nmax = (uint32_t)__builtin_amdgcn_readfirstlane((int)nmax);
    const uint64_t s0k = ((uint64_t)row0((uint32_t)(b0k >> 32)) << 32) | row0((uint32_t)b0k);
    const uint32_t s0p = row0(b0p);
    float tx = 0.f, ty = 0.f, tz = 0.f, ux = 0.f, uy = 0.f, uz = 0.f;
    uint32_t wsum = 0;
    // slot lg (from b0) and slot 16 + lg (from b1, written only when K > 16 + lg)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t k = (uint32_t)(h * G + lg);
        const bool own = k < n;
        const uint64_t mk = own ? (h ? b1k : b0k) : s0k;
        const uint32_t mp = own ? (h ? b1p : b0p) : s0p;
        const uint32_t idx = n ? (uint32_t)mk : 0u;
        const int from = one ? (int)mp : 0;
        float x = __shfl(v0.x, from, G), y = __shfl(v0.y, from, G), z = __shfl(v0.z, from, G);
        uint32_t w = (uint32_t)__shfl((int)w0, from, G);
        if (!one) {
            const float4 pv = p4[mp];
            x = pv.x;
            y = pv.y;
            z = pv.z;
            if (!UP) w = Wt ? Wt[(size_t)b * N + idx] : 1u;
        }
        if (!n) {
            x = y = z = 0.0f;
            w = 1u;
        }
        if (live && k < (uint32_t)K) {
            node_idx[cK + k] = UP ? (n ? (int32_t)idx : -1) : (int32_t)idx;
            if (node_xyz) {
                store_xyz(node_xyz + (cK + k) * 3, x, y, z);
            }
        }
        if (!UP) {
            const float wf = (float)w;
            if (h == 0) {
                tx = wf * x, ty = wf * y, tz = wf * z;
            } else {
                ux = wf * x, uy = wf * y, uz = wf * z;
            }
            wsum += own ? w : 0u;
        }
    }
    if (UP) {
        if (live && lg == 0) {
            n_valid[cid] = (int32_t)n;
            if (ctx_count) ctx_count[cid] = (int32_t)c;
            if (lin_out) lin_out[cid] = (int32_t)lin;
        }
        return;
    }
    uint32_t wc = wsum;
#pragma unroll
    for (int d = 1; d < G; d <<= 1) wc += xlane(wc, d);
    // strides 1..8 inside each half (only as far as the wave's largest n
    // reaches), then node 16 into node 0
#pragma unroll
    for (int hh = 1; hh < G; hh <<= 1) {
        if ((uint32_t)hh >= nmax) break;
        const bool lead = (lg & (2 * hh - 1)) == 0;
        const float ox = xlanef(tx, hh), oy = xlanef(ty, hh), oz = xlanef(tz, hh);
        if (lead && (uint32_t)(lg + hh) < n) {
            tx = tx + ox;
            ty = ty + oy;
            tz = tz + oz;
        }
        if (nmax > (uint32_t)G) {
            const float px = xlanef(ux, hh), py = xlanef(uy, hh), pz = xlanef(uz, hh);
            if (lead && (uint32_t)(G + lg + hh) < n) {
                ux = ux + px;
                uy = uy + py;
                uz = uz + pz;
            }
        }
    }
    if (n > (uint32_t)G) {  // lane 0 holds nodes 0 and 16
        tx = tx + ux;
        ty = ty + uy;
        tz = tz + uz;
    }
    // lanes 0, 1, 2 of the group each divide one of lane 0's sums
    const float sx = __uint_as_float(row0(__float_as_uint(tx)));
    const float sy = __uint_as_float(row0(__float_as_uint(ty)));
    const float sz = __uint_as_float(row0(__float_as_uint(tz)));
    if (live && lg < 3) {
        const float num = lg == 0 ? sx : (lg == 1 ? sy : sz);
        center_xyz[(size_t)cid * 3 + lg] = n ? num / (float)wc : 0.0f;
    }
    if (live && lg == 0) {
        center_w[cid] = wc;
        n_valid[cid] = (int32_t)n;
        if (ctx_count) ctx_count[cid] = (int32_t)c;
    }
}

// The pointers of one query launch.
struct QueryIO {
    const uint32_t* weights;
    const int32_t* center_lin;
    const float* center_pts;
    int32_t* node_idx;
    float* node_xyz;
    int32_t* n_valid;
    float* center_xyz;
    uint32_t* center_w;
    int32_t* ctx_count;
    int32_t* lin_out;
};

template <int MODE, int G, int RAD, bool UP, int NR, bool DEFER = false, int D = 1>
void launch_g(const Layout& L, const QGrid& g, void* ws, const QueryIO& io, int32_t M, int32_t K, uint64_t seed,
              hipStream_t s) {
    constexpr int GPB = kQueryThreads / G;
    const int32_t total = L.B * M;
    const unsigned blocks = (unsigned)((total + GPB - 1) / GPB);
    constexpr int side = 2 * RAD + 1;
    // the groups' compacted voxels; with DEFER also each group's candidate
    // buffer (64 keys and positions), 8-byte aligned after them
    const size_t lds = (((size_t)GPB * (2 * side * side * side + 1) + 1) & ~(size_t)1) * sizeof(uint32_t) +
                       (DEFER ? (size_t)GPB * kWave * (sizeof(uint64_t) + sizeof(uint32_t)) : 0);
    k_query<MODE, G, RAD, UP, NR, DEFER, D><<<blocks, kQueryThreads, lds, s>>>(
        io.weights, L.N, M, K, total, g, L.W, at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
        at<uint32_t>(ws, L.vox_off), at<float4>(ws, L.pt4), io.center_lin, io.center_pts, seed, io.node_idx,
        io.node_xyz, io.n_valid, io.center_xyz, io.center_w, io.ctx_count, io.lin_out, at<int>(ws, L.status));
}

template <int MODE, int G, bool UP, int NR = 1>
void launch_r(const Layout& L, const QGrid& g, int32_t rad, void* ws, const QueryIO& io, int32_t M, int32_t K,
              uint64_t seed, hipStream_t s) {
    if (rad == 1)
        launch_g<MODE, G, 1, UP, NR>(L, g, ws, io, M, K, seed, s);
    else if (rad == 2)
        launch_g<MODE, G, 2, UP, NR>(L, g, ws, io, M, K, seed, s);
    else
        launch_g<MODE, G, 3, UP, NR>(L, g, ws, io, M, K, seed, s);
}

// Contexts of more points than this go to one wave each when the grid can
// hold contexts of more than kBigGrid points ((2r+1)^3 n_v): a 16-lane group
// works through a long context chunk after chunk, one load latency each.
constexpr uint32_t kDefer = 128;
constexpr int64_t kBigGrid = 1024;

template <int MODE, int RAD, bool UP>
void launch_r2(const Layout& L, const QGrid& g, void* ws, const QueryIO& io, int32_t M, int32_t K, uint64_t seed,
               int32_t n_v, hipStream_t s) {
    constexpr int GPB = kQueryThreads / 16;
    const int32_t total = L.B * M;
    const unsigned blocks = (unsigned)((total + GPB - 1) / GPB);
    constexpr int64_t side = 2 * RAD + 1;
    const bool big = side * side * side * (int64_t)n_v > kBigGrid;
    k_query_r2<MODE, RAD, UP><<<blocks, kQueryThreads, 0, s>>>(
        io.weights, L.N, M, K, total, g, L.W, at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
        at<uint32_t>(ws, L.vox_off), at<float4>(ws, L.pt4), io.center_lin, io.center_pts, seed, io.node_idx,
        io.node_xyz, io.n_valid, io.center_xyz, io.center_w, io.ctx_count, io.lin_out, at<int>(ws, L.status),
        big ? kDefer : 0xFFFFFFFFu);
    if (big) launch_g<MODE, 64, RAD, UP, 1, true, 6>(L, g, ws, io, M, K, seed, s);
}

template <int MODE, bool UP>
void launch_mode(const Layout& L, const QGrid& g, int32_t rad, int32_t n_v, void* ws, const QueryIO& io, int32_t M,
                 int32_t K, uint64_t seed, hipStream_t s) {
    if (MODE != kRing && K > 16 && K <= 32) {
        // 16 lanes and two result registers per center
        if (rad == 1)
            launch_r2<MODE, 1, UP>(L, g, ws, io, M, K, seed, n_v, s);
        else if (rad == 2)
            launch_r2<MODE, 2, UP>(L, g, ws, io, M, K, seed, n_v, s);
        else
            launch_r2<MODE, 3, UP>(L, g, ws, io, M, K, seed, n_v, s);
        return;
    }
    if (K <= 16)
        launch_r<MODE, 16, UP>(L, g, rad, ws, io, M, K, seed, s);
    else if (K <= 32)
        launch_r<MODE, 32, UP>(L, g, rad, ws, io, M, K, seed, s);
    else if (K <= 64)
        launch_r<MODE, 64, UP>(L, g, rad, ws, io, M, K, seed, s);
    else
        launch_r<MODE, 64, UP, 2>(L, g, rad, ws, io, M, K, seed, s);
}

QGrid make_qgrid(const cagq_grid_desc& d, int32_t M) {
    QGrid g;
    for (int a = 0; a < 3; ++a) {
        g.o[a] = d.origin[a];
        g.s[a] = d.voxel_size[a];
        g.D[a] = d.dims[a];
    }
    g.d0 = make_magic((uint32_t)d.dims[0]);
    g.d01 = make_magic((uint32_t)d.dims[0] * (uint32_t)d.dims[1]);
    g.mm = make_magic((uint32_t)M);
    return g;
}

}  // namespace

hipError_t launch_query(const Layout& L, const cagq_grid_desc& d, const float* points, void* ws,
                        const uint32_t* weights, const int32_t* center_lin, int32_t M, int32_t K,
                        int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                        int32_t* n_valid, float* center_xyz, uint32_t* center_w, int32_t* ctx_count,
                        hipStream_t s) {
    (void)points;  // node coordinates are bit copies read from the slot-ordered copy
    const QGrid g = make_qgrid(d, M);
    const QueryIO io{weights, center_lin, nullptr, node_idx, node_xyz, n_valid, center_xyz, center_w, ctx_count,
                     nullptr};
    if (mode == CAGQ_QUERY_CUBE)
        launch_mode<CAGQ_QUERY_CUBE, false>(L, g, d.radius, d.n_v, ws, io, M, K, seed, s);
    else if (mode == CAGQ_QUERY_KNN)
        launch_mode<CAGQ_QUERY_KNN, false>(L, g, d.radius, d.n_v, ws, io, M, K, seed, s);
    else
        launch_mode<kRing, false>(L, g, d.radius, d.n_v, ws, io, M, K, seed, s);
    return hipGetLastError();
}

hipError_t launch_query_points(const Layout& L, const cagq_grid_desc& d, void* ws, const float* centers, int32_t M,
                               int32_t K, int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                               int32_t* n_valid, int32_t* ctx_count, int32_t* center_lin, hipStream_t s) {
    const QGrid g = make_qgrid(d, M);
    const QueryIO io{nullptr, nullptr, centers, node_idx, node_xyz, n_valid, nullptr, nullptr, ctx_count,
                     center_lin};
    if (mode == CAGQ_QUERY_CUBE)
        launch_mode<CAGQ_QUERY_CUBE, true>(L, g, d.radius, d.n_v, ws, io, M, K, seed, s);
    else if (mode == CAGQ_QUERY_KNN)
        launch_mode<CAGQ_QUERY_KNN, true>(L, g, d.radius, d.n_v, ws, io, M, K, seed, s);
    else
        launch_mode<kRing, true>(L, g, d.radius, d.n_v, ws, io, M, K, seed, s);
    return hipGetLastError();
}

}  // namespace cagq
