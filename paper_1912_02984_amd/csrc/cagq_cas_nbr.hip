// Neighbour lists for Coverage-Aware Sampling (Sec. 3.2, Eqs. 1-2): every
// round of the greedy walks, for some voxels, the occupied voxels within
// Chebyshev distance r (the coverage term of a score) or 2r (the voxels a
// pick competes with and the voxels whose score it changes). One thread per
// occupied voxel writes these slots once per grid, so that the rounds need
// no geometry: first those within r (the voxel itself included), then those
// at distance r+1..2r, each group in ascending (dz, dy, dx) order.
//
// Two formats: u16 entries behind an 8-entry header for clouds of at most
// kCasLdsMaxN points (r <= 2), u32 entries behind a 4-entry header for
// larger clouds with r = 1. Header entry 0 is the number within r, entry 1
// the number within 2r.
#include <algorithm>
#include <type_traits>

#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kNbrThreads = 64;  // one wave per block: small clouds spread over every CU

// The u32 lists of large clouds gather their entries 4 at a time and store
// each group with one 16-byte store: a lane's list is one run of whole
// groups behind the 16-byte header, instead of a 4-byte store per entry
// across the lanes' far-apart lists (layer 1 of the indoor scenes: 53 ->
// 40 us). Unused entries of the last group hold whatever the group held
// (readers look at the first n entries only). The u16 lists of small clouds
// keep one store per entry, which measured faster there.
template <typename E>
struct Direct {
    E* out;
    __device__ __forceinline__ void push(uint32_t v) { *out++ = (E)v; }
    __device__ __forceinline__ void flush() {}
};

template <typename E>
struct Group16 {
    static constexpr int kPer = 16 / (int)sizeof(E);
    static constexpr int kBits = 8 * (int)sizeof(E);
    uint64_t lo = 0, hi = 0;  // the entries so far, the latest in the top bits
    int k = 0;                // entries held
    E* out;                   // where the next whole group goes
    __device__ __forceinline__ void push(uint32_t v) {
        lo = (lo >> kBits) | (hi << (64 - kBits));
        hi = (hi >> kBits) | ((uint64_t)v << (64 - kBits));
        if (++k == kPer) {
            *reinterpret_cast<uint4*>(out) = make_uint4((uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi,
                                                        (uint32_t)(hi >> 32));
            out += kPer;
            k = 0;
        }
    }
    __device__ __forceinline__ void flush() {
        if (k == 0) return;
        // k entries sit in the top k slots: move them to the bottom
        const int sh = (kPer - k) * kBits;  // 0 < sh < 128
        uint64_t l = lo, h = hi;
        if (sh >= 64) {
            l = h >> (sh - 64);
            h = 0;
        } else {
            l = (l >> sh) | (h << (64 - sh));
            h = h >> sh;
        }
        *reinterpret_cast<uint4*>(out) = make_uint4((uint32_t)l, (uint32_t)(l >> 32), (uint32_t)h,
                                                    (uint32_t)(h >> 32));
    }
};

// E: entry type, ST: entries per voxel (header included), HDR: header entries.
template <int RAD, typename E, int ST, int HDR>
__global__ __launch_bounds__(kNbrThreads) void k_cas_nbr(int32_t B, int32_t N, int64_t W, GridDims g,
                                                         const int32_t* __restrict__ nvox,
                                                         const uint32_t* __restrict__ vox_lin,
                                                         const uint64_t* __restrict__ bitmap,
                                                         const uint32_t* __restrict__ word_rank, E* __restrict__ nbr,
                                                         uint64_t* __restrict__ key, int64_t unit, CasClear clr,
                                                         bool clear) {
    constexpr int H = 2 * RAD, S2 = 2 * H + 1;
    const int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    if (clear) {  // the rounds' starting state (the grid covers the control block too)
        if (gid < B * N) {
            clr.cover[gid] = 0;
            clr.pick[gid] = 0;
            clr.round[gid] = 0;
            clr.blocker[gid] = -1;
            clr.dirty[gid] = 0;
        }
        if (gid < clr.nparts) {
            clr.gpart[gid] = 0;
            clr.cpart[gid] = 0;
        }
        if (gid < B) clr.done[gid] = 0;
        if (gid < clr.nhist) clr.uhist[gid] = 0;
        if (gid < clr.ndesc) clr.desc[gid] = 0;
        if (gid == 0) {
            *clr.ndone = 0;
            *clr.ticket = 0;
        }
    }
    if (gid >= B * N) return;
    const int32_t b = gid / N, s = gid - b * N;
    if (s >= nvox[b]) return;
    int32_t x, y, z;
    const uint32_t lin = vox_lin[gid];
    decode_lin(lin, g, x, y, z);
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    E* out = nbr + (size_t)gid * ST;
    static_assert(HDR * sizeof(E) == 16 && (ST * sizeof(E)) % 16 == 0, "16-byte header and list stride");
    std::conditional_t<sizeof(E) == 4, Group16<E>, Direct<E>> grp;
    grp.out = out + HDR;
    uint32_t n = HDR;
    // bits H-RAD..H+RAD of a row of half-width H are the voxels within r in x
    constexpr uint32_t kInner = ((1u << (2 * RAD + 1)) - 1) << (H - RAD);
    if constexpr (RAD == 1) {
        // the 25 rows of the window, a plane of 5 at a time
        GridRow rows[S2 * S2];
#pragma unroll
        for (int pl = 0; pl < S2; ++pl) {
            int32_t yy[S2], zz[S2];
            GridRow rp[S2];
#pragma unroll
            for (int i = 0; i < S2; ++i) {
                yy[i] = y + i - H;
                zz[i] = z + pl - H;
            }
            load_rows<S2>(bm, wr, g, x, yy, zz, H, rp);
#pragma unroll
            for (int i = 0; i < S2; ++i) rows[pl * S2 + i] = rp[i];
        }
#pragma unroll
        for (int j = 0; j < S2 * S2; ++j) {
            const int dy = j % S2 - H, dz = j / S2 - H;
            if (dy < -RAD || dy > RAD || dz < -RAD || dz > RAD) continue;
            for (uint32_t m = rows[j].mask & kInner; m; m &= m - 1) {
                const uint32_t q = (uint32_t)__ffs(m) - 1;
                grp.push(rows[j].first + (uint32_t)__popc(rows[j].mask & ((1u << q) - 1)));
                ++n;
            }
        }
        const uint32_t n_r = n - HDR;
#pragma unroll
        for (int j = 0; j < S2 * S2; ++j) {
            const int dy = j % S2 - H, dz = j / S2 - H;
            const bool inner = dy >= -RAD && dy <= RAD && dz >= -RAD && dz <= RAD;
            for (uint32_t m = rows[j].mask & (inner ? ~kInner : ~0u); m; m &= m - 1) {
                const uint32_t q = (uint32_t)__ffs(m) - 1;
                grp.push(rows[j].first + (uint32_t)__popc(rows[j].mask & ((1u << q) - 1)));
                ++n;
            }
        }
        grp.flush();
        out[0] = (E)n_r;
        out[1] = (E)(n - HDR);
        if (key) key[gid] = cas_key(unit * (int64_t)n_r, lin);
    } else {
        // one plane of rows at a time, the window within r first
        for (int dz = -RAD; dz <= RAD; ++dz) {
            GridRow rows[2 * RAD + 1];
#pragma unroll
            for (int j = 0; j < 2 * RAD + 1; ++j) rows[j] = load_row(bm, wr, g, x, y + j - RAD, z + dz, RAD);
#pragma unroll
            for (int j = 0; j < 2 * RAD + 1; ++j)
                for (uint32_t sl = rows[j].first, m = rows[j].mask; m; m &= m - 1, ++sl) {
                    grp.push(sl);
                    ++n;
                }
        }
        const uint32_t n_r = n - HDR;
        for (int dz = -H; dz <= H; ++dz) {
            GridRow rows[S2];
#pragma unroll
            for (int j = 0; j < S2; ++j) rows[j] = load_row(bm, wr, g, x, y + j - H, z + dz, H);
#pragma unroll
            for (int j = 0; j < S2; ++j) {
                const int dy = j - H;
                const bool inner = dy >= -RAD && dy <= RAD && dz >= -RAD && dz <= RAD;
                for (uint32_t m = rows[j].mask & (inner ? ~kInner : ~0u); m; m &= m - 1) {
                    const uint32_t q = (uint32_t)__ffs(m) - 1;
                    grp.push(rows[j].first + (uint32_t)__popc(rows[j].mask & ((1u << q) - 1)));
                    ++n;
                }
            }
        }
        grp.flush();
        out[0] = (E)n_r;
        out[1] = (E)(n - HDR);
    }
}

}  // namespace

hipError_t launch_cas_nbr(const Layout& L, const cagq_grid_desc& d, void* ws, hipStream_t s, uint64_t* key,
                          int64_t unit, const CasClear* clr) {
    GridDims g;
    for (int a = 0; a < 3; ++a) g.D[a] = d.dims[a];
    int64_t lanes = (int64_t)L.B * L.N;
    if (clr) lanes = std::max<int64_t>({lanes, clr->nparts, clr->nhist, clr->ndesc});
    const unsigned blocks = (unsigned)((lanes + kNbrThreads - 1) / kNbrThreads);
    const CasClear none{};
    const CasClear c = clr ? *clr : none;
    const int32_t* nvox = at<int32_t>(ws, L.nvox);
    const uint32_t* vox_lin = at<uint32_t>(ws, L.vox_lin);
    const uint64_t* bitmap = at<uint64_t>(ws, L.bitmap);
    const uint32_t* word_rank = at<uint32_t>(ws, L.word_rank);
    if (L.has_nbr32 && d.radius == 1) {
        k_cas_nbr<1, uint32_t, kNbr32Stride, 4><<<blocks, kNbrThreads, 0, s>>>(
            L.B, L.N, L.W, g, nvox, vox_lin, bitmap, word_rank, at<uint32_t>(ws, L.cas_nbr32), key, unit, c,
            clr != nullptr);
    } else if (L.has_nbr16 && d.radius == 1) {
        k_cas_nbr<1, uint16_t, nbr_stride(1), 8><<<blocks, kNbrThreads, 0, s>>>(
            L.B, L.N, L.W, g, nvox, vox_lin, bitmap, word_rank, at<uint16_t>(ws, L.cas_nbr), nullptr, 0, c, false);
    } else if (L.has_nbr16 && d.radius == 2) {
        k_cas_nbr<2, uint16_t, nbr_stride(2), 8><<<blocks, kNbrThreads, 0, s>>>(
            L.B, L.N, L.W, g, nvox, vox_lin, bitmap, word_rank, at<uint16_t>(ws, L.cas_nbr), nullptr, 0, c, false);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace cagq
