// Coverage-Aware Sampling, the paper's own challenger / incumbent procedure
// (Sec. 3.2, Eqs. 2-3): start from M random incumbents (the RVS choice with
// the same seed, in slots 0..m-1 in ascending linear id); every other
// occupied voxel, in ascending linear id, challenges incumbent slot
// hi32(h(seed, 3, b, t)) mod m (t counts the challenges) and replaces it when
//   H_add = sum_{V in pi(C)} delta(C_V) - beta * C_V / lambda      (Eq. 2)
//   H_rmv = sum_{V in pi(I)} delta(C_V - 1)                         (Eq. 3)
// satisfy H_add > H_rmv, both scaled by 2^16 * lambda to integers; C_V counts
// the incumbents whose neighbourhood holds V. A replaced incumbent does not
// challenge again. The final incumbents are emitted in ascending linear id.
//
// The procedure is sequential, but most challenges leave the state alone
// (about one in eight is accepted on the indoor scenes), so one wave per
// cloud decides 64 challenges at a time, one per lane, speculatively:
// * every lane loads the grid rows of pi(C) and pi(I) for its challenge once
//   and evaluates both heuristics against the current coverage counts;
// * a sweep walks the accepted lanes in challenge order; an accepted lane
//   marks every later lane whose footprint it may touch (same incumbent slot,
//   or any pair of C/I centers within Chebyshev distance 2r, the condition
//   for two r-neighbourhoods to meet) as stale; the sweep ends at the first
//   stale lane, and every lane before it is decided exactly as the sequential
//   procedure decides it;
// * the accepted lanes of the sweep touch pairwise disjoint voxels, so they
//   update the counts together; the stale lanes evaluate again (from the
//   counts in LDS; a lane whose incumbent was replaced reloads its rows);
//   the next sweep starts at the first of them.
// The coverage counts (8 bits for r <= 2, 16 for r = 3), the incumbents'
// linear ids and the bits of the initial set live in LDS.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr size_t kSwapLdsLimit = 160000;  // bytes a gfx950 workgroup may hold
constexpr size_t kSwapLdsStatic = 256;     // bound on the kernel's own __shared__ variables

struct Occ {
    const uint64_t* bm;
    const uint32_t* wr;
    GridDims g;
};

// The (2r+1)^2 grid-row segments of half-width r around V, which hold pi(V).
// For r <= 2 they are loaded once and kept in registers; for r = 3 (49 rows)
// only V is kept and every use loads the rows again.
template <int RAD>
struct Hood {
    static constexpr int S = 2 * RAD + 1;
    static constexpr bool kKeep = RAD <= 2;
    GridRow row[kKeep ? S * S : 1];
    int32_t x, y, z;
    bool live;

    __device__ __forceinline__ void load(const Occ& o, int32_t x_, int32_t y_, int32_t z_, bool live_) {
        x = x_, y = y_, z = z_, live = live_;
        if constexpr (kKeep) {
#pragma unroll
            for (int q = 0; q < S * S; ++q) row[q] = fetch(o, q);
        }
    }
    __device__ __forceinline__ GridRow fetch(const Occ& o, int q) const {
        GridRow r = load_row(o.bm, o.wr, o.g, x, y + q % S - RAD, z + q / S - RAD, RAD);
        if (!live) r.mask = 0u;
        return r;
    }
    __device__ __forceinline__ GridRow get(const Occ& o, int q) const {
        if constexpr (kKeep)
            return row[q];
        else
            return fetch(o, q);
    }
};

// f(q) for every row q of a window: unrolled when the rows sit in registers.
template <int RAD, typename F>
__device__ __forceinline__ void for_rows(F f) {
    constexpr int S = 2 * RAD + 1;
    if constexpr (Hood<RAD>::kKeep) {
#pragma unroll
        for (int q = 0; q < S * S; ++q) f(q);
    } else {
#pragma unroll 1
        for (int q = 0; q < S * S; ++q) f(q);
    }
}

// Over the occupied voxels of a neighbourhood: how many have coverage 0, how
// many coverage 1, and the coverage sum. Every position of a row is read and
// the unoccupied ones are masked out, so the reads are in flight together
// (such a read lands on a slot <= nvox, inside the counts' buffer).
template <int RAD, typename CT>
__device__ __forceinline__ void tally(const CT* cov, const Occ& o, const Hood<RAD>& h, uint32_t& n0, uint32_t& n1,
                                      uint32_t& sum) {
    constexpr int S = 2 * RAD + 1;
    for_rows<RAD>([&](int q) {
        const GridRow r = h.get(o, q);
#pragma unroll
        for (int k = 0; k < S; ++k) {
            const uint32_t on = (r.mask >> k) & 1u;
            const uint32_t c = cov[r.first + (uint32_t)__popc(r.mask & ((1u << k) - 1))];
            n0 += on & (c == 0 ? 1u : 0u);
            n1 += on & (c == 1 ? 1u : 0u);
            sum += on ? c : 0u;
        }
    });
}

// Adds +1 or -1 to the coverage count of every occupied voxel of a
// neighbourhood: word-wide LDS adds of the shifted unit (a count stays in
// 0..(2r+1)^3, so no carry or borrow crosses into the next count).
template <int RAD, typename CT>
__device__ __forceinline__ void cover(uint32_t* cov_w, const Occ& o, const Hood<RAD>& h, bool add) {
    constexpr uint32_t kPer = 4 / sizeof(CT);
    for_rows<RAD>([&](int q) {
        const GridRow r = h.get(o, q);
        for (uint32_t m = r.mask, sl = r.first; m; m &= m - 1, ++sl) {
            const uint32_t unit = 1u << (8 * sizeof(CT) * (sl % kPer));
            if (add)
                atomicAdd(&cov_w[sl / kPer], unit);
            else
                atomicSub(&cov_w[sl / kPer], unit);
        }
    });
}

__device__ __forceinline__ bool near(int32_t ax, int32_t ay, int32_t az, int32_t bx, int32_t by, int32_t bz,
                                     int32_t d) {
    return abs(ax - bx) <= d && abs(ay - by) <= d && abs(az - bz) <= d;
}

template <int RAD, typename CT>
__global__ __launch_bounds__(kWave) void k_cas_swap(int32_t N, int64_t W, GridDims g, int32_t M, uint64_t seed,
                                                    uint32_t beta_q16, const int32_t* __restrict__ nvox,
                                                    const uint32_t* __restrict__ vox_lin,
                                                    const uint64_t* __restrict__ bitmap,
                                                    const uint32_t* __restrict__ word_rank,
                                                    int32_t* __restrict__ center_lin,
                                                    const int32_t* __restrict__ m_valid) {
    constexpr int S = 2 * RAD + 1;
    constexpr int64_t lam = (int64_t)S * S * S;
    constexpr uint32_t kPer = 4 / sizeof(CT);  // counts per 32-bit LDS word
    extern __shared__ __align__(16) unsigned char lds[];
    __shared__ uint32_t stage[kWave];  // the slots of the next challengers
    const int32_t b = blockIdx.x;
    const int lane = lane_id();
    const int32_t nv = nvox[b];
    const int32_t m = m_valid[b];
    if (m <= 0) return;
    uint32_t* inc = reinterpret_cast<uint32_t*>(lds);             // incumbent slot j -> linear id
    uint32_t* bits = inc + M;                                      // initial set, one bit per slot
    CT* cov = reinterpret_cast<CT*>(bits + (N + 31) / 32);         // incumbents covering the voxel
    uint32_t* cov_w = reinterpret_cast<uint32_t*>(cov);
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    const Occ o{bm, wr, g};
    const uint32_t* vl = vox_lin + (size_t)b * N;
    int32_t* out = center_lin + (size_t)b * M;

    for (int32_t w = lane; w < (nv + 31) / 32; w += kWave) bits[w] = 0u;
    for (int32_t w = lane; w < (int32_t)((nv + kPer - 1) / kPer); w += kWave) cov_w[w] = 0u;
    __syncthreads();
    // the RVS incumbents: their linear ids and their bits
    for (int32_t j = lane; j < m; j += kWave) {
        const uint32_t lin = (uint32_t)out[j];
        const int32_t sl = slot_of(bm, wr, lin);
        inc[j] = lin;
        atomicOr(&bits[sl >> 5], 1u << (sl & 31));
    }
    __syncthreads();
    // initial coverage: every incumbent adds 1 over its neighbourhood
    for (int32_t j0 = 0; j0 < m; j0 += kWave) {
        const int32_t j = j0 + lane;
        int32_t x, y, z;
        decode_lin(j < m ? inc[j] : 0u, g, x, y, z);
        Hood<RAD> h;
        h.load(o, x, y, z, j < m);
        cover<RAD, CT>(cov_w, o, h, true);
    }
    __syncthreads();

    const uint64_t hb = sm64(sm64(seed ^ 3ull) ^ (uint64_t)b);
    const int32_t T = nv - m;  // every voxel outside the initial set challenges once
    int32_t t0 = 0, sc = 0;    // challenges decided, slot cursor
    while (t0 < T) {
        // the next (up to) 64 challengers, in ascending slot order
        int32_t filled = 0;
        while (filled < kWave && sc < nv) {
            const int32_t sv = sc + lane;
            const bool ch = sv < nv && !((bits[sv >> 5] >> (sv & 31)) & 1u);
            const uint64_t bal = __ballot(ch);
            const int32_t rank = (int32_t)__popcll(bal & ((1ull << lane) - 1));
            const int32_t need = kWave - filled;
            if (ch && rank < need) stage[filled + rank] = (uint32_t)sv;
            const int32_t cnt = (int32_t)__popcll(bal);
            if (cnt <= need) {
                sc = sc + kWave < nv ? sc + kWave : nv;
                filled += cnt;
            } else {
                sc += __ffsll((unsigned long long)__ballot(ch && rank == need - 1));
                filled = kWave;
            }
        }
        __syncthreads();
        const int32_t nb = filled;
        if (nb == 0) break;  // unreachable: the initial set holds exactly m slots
        const bool live = lane < nb;
        const uint32_t clin = live ? vl[stage[lane]] : 0u;
        const int32_t t = t0 + lane;
        const uint32_t j = live ? (uint32_t)((sm64(hb ^ (uint64_t)t) >> 32) % (uint64_t)m) : 0u;
        int32_t cx, cy, cz, ix = 0, iy = 0, iz = 0;
        decode_lin(clin, g, cx, cy, cz);
        Hood<RAD> hc, hi;
        hc.load(o, cx, cy, cz, live);
        uint32_t ilin = 0;
        bool reload = live, stale = live, acc = false;
        int32_t cur = 0;
        while (cur < nb) {
            if (reload) {
                ilin = inc[j];
                decode_lin(ilin, g, ix, iy, iz);
                hi.load(o, ix, iy, iz, true);
                reload = false;
            }
            if (stale) {
                uint32_t c0 = 0, c1 = 0, cs = 0, r0 = 0, r1 = 0, rs = 0;
                tally<RAD, CT>(cov, o, hc, c0, c1, cs);
                tally<RAD, CT>(cov, o, hi, r0, r1, rs);
                const int64_t h_add = 65536LL * lam * (int64_t)c0 - (int64_t)beta_q16 * (int64_t)cs;
                const int64_t h_rmv = 65536LL * lam * (int64_t)r1;
                acc = h_add > h_rmv;
                stale = false;
            }
            // walk the accepted lanes from cur on, in challenge order
            uint64_t A = __ballot(acc && live) & (~0ull << cur);
            int32_t stop = nb;
            bool commit = false;
            while (A) {
                const int a = __ffsll((unsigned long long)A) - 1;
                if (a >= stop) break;
                A &= A - 1;
                commit = commit || lane == a;
                const int32_t ax = __builtin_amdgcn_readlane(cx, a), ay = __builtin_amdgcn_readlane(cy, a),
                              az = __builtin_amdgcn_readlane(cz, a);
                const int32_t bx = __builtin_amdgcn_readlane(ix, a), by = __builtin_amdgcn_readlane(iy, a),
                              bz = __builtin_amdgcn_readlane(iz, a);
                const uint32_t ja = (uint32_t)__builtin_amdgcn_readlane((int)j, a);
                const bool after = live && lane > a;
                const bool same = after && j == ja;
                const bool touch = same || (after && (near(cx, cy, cz, ax, ay, az, 2 * RAD) ||
                                                      near(cx, cy, cz, bx, by, bz, 2 * RAD) ||
                                                      near(ix, iy, iz, ax, ay, az, 2 * RAD) ||
                                                      near(ix, iy, iz, bx, by, bz, 2 * RAD)));
                reload = reload || same;
                stale = stale || touch;
                const uint64_t tm = __ballot(touch);
                if (tm) {
                    const int32_t f = __ffsll((unsigned long long)tm) - 1;
                    stop = f < stop ? f : stop;
                }
            }
            // the sweep's accepted swaps touch disjoint voxels and slots
            if (commit) {
                cover<RAD, CT>(cov_w, o, hi, false);
                cover<RAD, CT>(cov_w, o, hc, true);
                inc[j] = clin;
                acc = false;
            }
            __syncthreads();
            cur = stop;
        }
        t0 += nb;
    }

    // the final incumbents in ascending linear id: their bits, then an
    // ordered pass over the slots; position p < m also fills p + m, ...
    for (int32_t w = lane; w < (nv + 31) / 32; w += kWave) bits[w] = 0u;
    __syncthreads();
    for (int32_t j = lane; j < m; j += kWave) {
        const int32_t sl = slot_of(bm, wr, inc[j]);
        atomicOr(&bits[sl >> 5], 1u << (sl & 31));
    }
    __syncthreads();
    uint32_t base = 0;
    for (int32_t s0 = 0; s0 < nv; s0 += kWave) {
        const int32_t s = s0 + lane;
        const bool chosen = s < nv && ((bits[s >> 5] >> (s & 31)) & 1u);
        const uint64_t bal = __ballot(chosen);
        if (chosen) {
            const uint32_t pos = base + (uint32_t)__popcll(bal & ((1ull << lane) - 1));
            for (int32_t k = (int32_t)pos; k < M; k += m) out[k] = (int32_t)vl[s];
        }
        base += (uint32_t)__popcll(bal);
    }
}

size_t swap_lds_bytes(int32_t N, int32_t M, int rad) {
    const size_t cbytes = rad <= 2 ? 1 : 2;
    return 4 * (size_t)M + 4 * (size_t)((N + 31) / 32) + cbytes * (size_t)N + 16;
}

}  // namespace

bool cas_swap_fits(const Layout& L, const cagq_grid_desc& d, int32_t M) {
    return swap_lds_bytes(L.N, M, d.radius) + kSwapLdsStatic <= kSwapLdsLimit;
}

hipError_t launch_cas_swap(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, uint64_t seed,
                           uint32_t beta_q16, int32_t* center_lin, int32_t* m_valid, hipStream_t s) {
    // the incumbents start as the RVS choice
    hipError_t e = launch_select(L, ws, M, 0, seed, center_lin, m_valid, s);
    if (e != hipSuccess) return e;
    GridDims g;
    for (int a = 0; a < 3; ++a) g.D[a] = d.dims[a];
    const size_t bytes = swap_lds_bytes(L.N, M, d.radius);
    auto go = [&](auto kern) {
        hipError_t r = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (r != hipSuccess) return r;
        kern<<<L.B, kWave, bytes, s>>>(L.N, L.W, g, M, seed, beta_q16, at<int32_t>(ws, L.nvox),
                                       at<uint32_t>(ws, L.vox_lin), at<uint64_t>(ws, L.bitmap),
                                       at<uint32_t>(ws, L.word_rank), center_lin, m_valid);
        return hipGetLastError();
    };
    switch (d.radius) {
        case 1: return go(k_cas_swap<1, uint8_t>);
        case 2: return go(k_cas_swap<2, uint8_t>);
        default: return go(k_cas_swap<3, uint16_t>);
    }
}

}  // namespace cagq
