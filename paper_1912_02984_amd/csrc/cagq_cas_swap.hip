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
// The procedure is sequential: one workgroup of one wave per cloud walks the
// challengers. Per challenge the wave reads the grid rows of pi(C) and pi(I)
// from the occupancy bitmap, one row per lane, and reduces the two
// heuristics; an accepted swap subtracts 1 over pi(I), then adds 1 over
// pi(C). The coverage counts (8 bits for r <= 2, 16 for r = 3), the
// incumbent slots and the bits of the initial set live in LDS.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr size_t kSwapLdsLimit = 160000;  // bytes a gfx950 workgroup may hold
constexpr size_t kSwapLdsStatic = 256;     // bound on the kernel's own __shared__ variables

struct Dims {
    int32_t D[3];
};

struct Row {
    uint32_t first;  // slot of the first occupied voxel at or after the segment's start
    uint32_t mask;   // bit j: voxel x - h + j occupied (0 outside the grid)
};

// Occupancy of the grid-row segment x' in [x - h, x + h] at (yy, zz) (an empty
// mask outside the grid).
__device__ __forceinline__ Row grid_row(const uint64_t* __restrict__ bm, const uint32_t* __restrict__ wr,
                                        const Dims& g, int32_t x, int32_t yy, int32_t zz, int32_t h) {
    Row r{0u, 0u};
    if (yy < 0 || yy >= g.D[1] || zz < 0 || zz >= g.D[2]) return r;
    const int32_t xs = x - h;
    const int32_t lo_x = xs < 0 ? 0 : xs;
    const int32_t hi_x = x + h > g.D[0] - 1 ? g.D[0] - 1 : x + h;
    const uint32_t base = (uint32_t)g.D[0] * ((uint32_t)yy + (uint32_t)g.D[1] * (uint32_t)zz);
    const uint32_t lo = base + (uint32_t)lo_x, hi = base + (uint32_t)hi_x;
    const uint32_t w0 = lo >> 6, o = lo & 63;
    const uint64_t a = bm[w0];
    uint64_t bits = a >> o;
    if ((hi >> 6) != w0) bits |= bm[w0 + 1] << (64 - o);  // o > 0 here
    r.mask = (uint32_t)(bits & ((1ull << (hi - lo + 1)) - 1)) << (lo_x - xs);
    r.first = wr[w0] + (uint32_t)__popcll(a & ((1ull << o) - 1));
    return r;
}

__device__ __forceinline__ void decode3(uint32_t lin, const Dims& g, int32_t& x, int32_t& y, int32_t& z) {
    x = (int32_t)(lin % (uint32_t)g.D[0]);
    y = (int32_t)((lin / (uint32_t)g.D[0]) % (uint32_t)g.D[1]);
    z = (int32_t)(lin / ((uint32_t)g.D[0] * (uint32_t)g.D[1]));
}

__device__ __forceinline__ int64_t wsum64(int64_t v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) v += (int64_t)shfl_xor64((uint64_t)v, d);
    return v;
}

// Adds `delta` to the coverage count of every occupied voxel within r of lin
// (one grid row per lane, as many passes as rows). Every lane must call it.
template <int RAD, typename CT>
__device__ __forceinline__ void cover_add(CT* cov, const uint64_t* bm, const uint32_t* wr, const Dims& g,
                                          uint32_t lin, int delta) {
    constexpr int S = 2 * RAD + 1;
    int32_t x, y, z;
    decode3(lin, g, x, y, z);
    for (int j0 = 0; j0 < S * S; j0 += kWave) {
        const int j = j0 + lane_id();
        if (j < S * S) {
            const Row r = grid_row(bm, wr, g, x, y + j % S - RAD, z + j / S - RAD, RAD);
            for (uint32_t m = r.mask, sl = r.first; m; m &= m - 1, ++sl) cov[sl] = (CT)((int)cov[sl] + delta);
        }
    }
}

template <int RAD, typename CT>
__global__ __launch_bounds__(kWave) void k_cas_swap(int32_t N, int64_t W, Dims g, int32_t M, uint64_t seed,
                                                    uint32_t beta_q16, const int32_t* __restrict__ nvox,
                                                    const uint32_t* __restrict__ vox_lin,
                                                    const uint64_t* __restrict__ bitmap,
                                                    const uint32_t* __restrict__ word_rank,
                                                    int32_t* __restrict__ center_lin,
                                                    const int32_t* __restrict__ m_valid) {
    constexpr int S = 2 * RAD + 1;
    constexpr int64_t lam = (int64_t)S * S * S;
    constexpr int NR = (2 * S * S + kWave - 1) / kWave;  // row passes for pi(C) and pi(I)
    extern __shared__ __align__(16) unsigned char lds[];
    const int32_t b = blockIdx.x;
    const int lane = lane_id();
    const int32_t nv = nvox[b];
    const int32_t m = m_valid[b];
    if (m <= 0) return;
    uint32_t* inc = reinterpret_cast<uint32_t*>(lds);             // incumbent slot j -> linear id
    uint32_t* bits = inc + M;                                      // initial set, one bit per slot
    CT* cov = reinterpret_cast<CT*>(bits + (N + 31) / 32);         // incumbents covering the voxel
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    const uint32_t* vl = vox_lin + (size_t)b * N;
    int32_t* out = center_lin + (size_t)b * M;

    for (int32_t w = lane; w < (nv + 31) / 32; w += kWave) bits[w] = 0u;
    __syncthreads();
    // the RVS incumbents: their linear ids and their bits
    for (int32_t j = lane; j < m; j += kWave) {
        const uint32_t lin = (uint32_t)out[j];
        const int32_t sl = slot_of(bm, wr, lin);
        inc[j] = lin;
        atomicOr(&bits[sl >> 5], 1u << (sl & 31));
    }
    __syncthreads();
    // initial coverage: each voxel counts the incumbents within distance r
    for (int32_t s0 = 0; s0 < nv; s0 += kWave) {
        const int32_t sv = s0 + lane;
        if (sv < nv) {
            int32_t x, y, z;
            decode3(vl[sv], g, x, y, z);
            uint32_t c = 0;
            for (int j = 0; j < S * S; ++j) {
                const Row r = grid_row(bm, wr, g, x, y + j % S - RAD, z + j / S - RAD, RAD);
                for (uint32_t mm = r.mask, sl = r.first; mm; mm &= mm - 1, ++sl) c += (bits[sl >> 5] >> (sl & 31)) & 1u;
            }
            cov[sv] = (CT)c;
        }
    }
    __syncthreads();

    const uint64_t hb = sm64(sm64(seed ^ 3ull) ^ (uint64_t)b);
    uint64_t t = 0;
    for (int32_t s0 = 0; s0 < nv; s0 += kWave) {
        // the linear ids of the next 64 slots, and which of them challenge
        const int32_t sv = s0 + lane;
        const uint32_t lins = sv < nv ? vl[sv] : 0u;
        const bool ch = sv < nv && !((bits[sv >> 5] >> (sv & 31)) & 1u);
        uint64_t chal = __ballot(ch);
        while (chal) {
            const int k = __ffsll((unsigned long long)chal) - 1;
            chal &= chal - 1;
            const uint32_t j = (uint32_t)((sm64(hb ^ t) >> 32) % (uint64_t)m);
            ++t;
            const uint32_t lc = (uint32_t)__shfl((int)lins, k, kWave), li = inc[j];
            int32_t cx, cy, cz, ix, iy, iz;
            decode3(lc, g, cx, cy, cz);
            decode3(li, g, ix, iy, iz);
            // lanes [0, S*S) read the rows of pi(C), lanes [S*S, 2*S*S) those of pi(I)
            int64_t unc = 0, csum = 0, single = 0;
#pragma unroll
            for (int p = 0; p < NR; ++p) {
                const int q = p * kWave + lane;
                if (q < 2 * S * S) {
                    const bool chl = q < S * S;
                    const int jj = chl ? q : q - S * S;
                    const Row r = chl ? grid_row(bm, wr, g, cx, cy + jj % S - RAD, cz + jj / S - RAD, RAD)
                                      : grid_row(bm, wr, g, ix, iy + jj % S - RAD, iz + jj / S - RAD, RAD);
                    for (uint32_t mm = r.mask, sl = r.first; mm; mm &= mm - 1, ++sl) {
                        const uint32_t c = cov[sl];
                        if (chl) {
                            unc += c == 0 ? 1 : 0;
                            csum += c;
                        } else {
                            single += c == 1 ? 1 : 0;
                        }
                    }
                }
            }
            unc = wsum64(unc);
            csum = wsum64(csum);
            single = wsum64(single);
            const int64_t h_add = 65536LL * lam * unc - (int64_t)beta_q16 * csum;
            const int64_t h_rmv = 65536LL * lam * single;
            if (h_add > h_rmv) {
                cover_add<RAD>(cov, bm, wr, g, li, -1);
                cover_add<RAD>(cov, bm, wr, g, lc, +1);
                if (lane == 0) inc[j] = lc;
            }
            __syncthreads();
        }
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
    Dims g;
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
