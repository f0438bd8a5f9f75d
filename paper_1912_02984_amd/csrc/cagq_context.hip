// Context lists for grid context pooling (Sec. 3.3: the context feature of a
// group is pooled over all of its context points, which CAGQ has already
// associated with the center voxel). The context of center voxel v is the
// stored points of the occupied voxels of pi(v), voxels in ascending linear
// id, each voxel's stored points ascending; v itself need not be occupied.
//
// A row segment of the (2r+1)^3 block holds consecutive slots, and the
// stored points are grouped by slot, so the context of one grid row is one
// contiguous range of the stored list: the block is (2r+1)^2 ranges.
//   k_ctx_clear      resets the scan's tile descriptors and ticket;
//   k_ctx_count      per center the context count c (range lengths from the
//                    offsets array), and a decoupled look-back scan over the
//                    batch that writes the CSR offsets. A tile's descriptor
//                    lives in the offsets array itself, at the tile's last
//                    output, whose final value it holds (flag bits aside);
//   k_ctx_unflag     clears the flag bits of those entries;
//   k_ctx_fill       one group of 16 lanes per center copies its ranges.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kFillG = 16;  // lanes per center in the fill
constexpr int kFillThreads = 256;

// Offsets position holding the descriptor of tile t (its last output).
__device__ __forceinline__ int64_t desc_pos(int64_t t, int64_t total) {
    const int64_t e = (t + 1) * kScanTile;
    return e < total ? e : total;
}

__global__ void k_ctx_clear(uint64_t* __restrict__ off, int64_t total, int64_t tiles, int* __restrict__ status) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < tiles) off[desc_pos(t, total)] = 0ull;
    if (t == 0) {
        off[0] = 0ull;
        status[kStTicketCtx] = 0;
    }
}

// Voxel coordinates of center j, or false when its lin is outside the grid.
__device__ __forceinline__ bool center_voxel(const int32_t* center_lin, int64_t j, const GridDims& g, int32_t& x,
                                             int32_t& y, int32_t& z) {
    const int32_t l = center_lin[j];
    const int64_t V = (int64_t)g.D[0] * g.D[1] * g.D[2];
    if (l < 0 || (int64_t)l >= V) return false;
    decode_lin((uint32_t)l, g, x, y, z);
    return true;
}

template <int RAD>
__global__ __launch_bounds__(kScanThreads) void k_ctx_count(int32_t N, int32_t M, int64_t total, int64_t W,
                                                            GridDims g, const uint64_t* __restrict__ bitmap,
                                                            const uint32_t* __restrict__ word_rank,
                                                            const uint32_t* __restrict__ vox_off,
                                                            const int32_t* __restrict__ center_lin,
                                                            uint64_t* __restrict__ off, int* __restrict__ status) {
    constexpr int S = 2 * RAD + 1;
    __shared__ uint32_t s_ticket;
    __shared__ uint64_t s_wave[kScanThreads / kWave];
    __shared__ uint64_t s_prefix;
    if (threadIdx.x == 0) s_ticket = atomicAdd((unsigned*)&status[kStTicketCtx], 1u);
    __syncthreads();
    const int64_t tile = s_ticket;
    const int64_t j0 = tile * kScanTile + (int64_t)threadIdx.x * kScanItems;
    uint32_t cnt[kScanItems];
    uint64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int64_t j = j0 + i;
        cnt[i] = 0;
        int32_t x, y, z;
        if (j < total && !center_voxel(center_lin, j, g, x, y, z)) raise_error(status, CAGQ_ERR_CENTER_NOT_OCCUPIED);
        else if (j < total) {
            const int32_t b = (int32_t)(j / M);
            const uint64_t* bm = bitmap + (size_t)b * W;
            const uint32_t* wr = word_rank + (size_t)b * W;
            const uint32_t* vo = vox_off + (size_t)b * (N + 1);
#pragma unroll
            for (int q = 0; q < S * S; ++q) {
                const GridRow r = load_row(bm, wr, g, x, y + q % S - RAD, z + q / S - RAD, RAD);
                cnt[i] += vo[r.first + (uint32_t)__popc(r.mask)] - vo[r.first];
            }
        }
        sum += cnt[i];
    }
    uint64_t agg;
    const uint64_t excl = block_excl_scan(sum, s_wave, &agg);
    const uint64_t base = tile_lookback_at([off, total](int64_t t) { return off + desc_pos(t, total); }, tile, agg,
                                           &s_prefix);
    uint64_t run = base + excl;
    const int64_t dpos = desc_pos(tile, total);
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int64_t j = j0 + i;
        run += cnt[i];
        // the tile's last output is its descriptor, published by the look-back
        if (j < total && j + 1 != dpos) off[j + 1] = run;
    }
}

__global__ void k_ctx_unflag(uint64_t* __restrict__ off, int64_t total, int64_t tiles) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < tiles) off[desc_pos(t, total)] &= kDescVal;
}

template <int RAD>
__global__ __launch_bounds__(kFillThreads) void k_ctx_fill(int32_t N, int32_t M, int64_t total, int64_t W,
                                                           GridDims g, const uint64_t* __restrict__ bitmap,
                                                           const uint32_t* __restrict__ word_rank,
                                                           const uint32_t* __restrict__ vox_off,
                                                           const uint32_t* __restrict__ pt_list,
                                                           const int32_t* __restrict__ center_lin,
                                                           const int64_t* __restrict__ off,
                                                           int32_t* __restrict__ ctx_idx, int64_t capacity,
                                                           int* __restrict__ status) {
    constexpr int S = 2 * RAD + 1;
    constexpr int GPB = kFillThreads / kFillG;
    __shared__ uint32_t s_pre[GPB][kFillG + 1];
    __shared__ uint32_t s_st[GPB][kFillG];
    const int gb = threadIdx.x / kFillG, lg = threadIdx.x & (kFillG - 1);
    const int64_t j = (int64_t)xcd_block(blockIdx.x, gridDim.x) * GPB + gb;
    // whole groups leave together: the group steps below need every lane
    if (j >= total) return;
    int32_t x, y, z;
    if (!center_voxel(center_lin, j, g, x, y, z)) return;  // an empty context
    const int32_t b = (int32_t)(j / M);
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    const uint32_t* vo = vox_off + (size_t)b * (N + 1);
    const uint32_t* pl = pt_list + (size_t)b * N;
    int64_t dst = off[j];
    bool over = false;
    for (int q0 = 0; q0 < S * S; q0 += kFillG) {
        const int q = q0 + lg;
        uint32_t st = 0, len = 0;
        if (q < S * S) {
            const GridRow r = load_row(bm, wr, g, x, y + q % S - RAD, z + q / S - RAD, RAD);
            st = vo[r.first];
            len = vo[r.first + (uint32_t)__popc(r.mask)] - st;
        }
        // inclusive scan of the range lengths across the group
        uint32_t incl = len;
#pragma unroll
        for (int d = 1; d < kFillG; d <<= 1) {
            const uint32_t o = (uint32_t)__shfl_up((int)incl, d, kFillG);
            if (lg >= d) incl += o;
        }
        s_pre[gb][lg] = incl - len;
        s_st[gb][lg] = st;
        const uint32_t tot = (uint32_t)__shfl((int)incl, kFillG - 1, kFillG);
        if (lg == kFillG - 1) s_pre[gb][kFillG] = tot;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        for (uint32_t e = (uint32_t)lg; e < tot; e += kFillG) {
            // the last range starting at or before e (empty ranges share starts)
            uint32_t lo = 0, hi = kFillG - 1;
            while (lo < hi) {
                const uint32_t mid = (lo + hi + 1) >> 1;
                if (s_pre[gb][mid] <= e) lo = mid; else hi = mid - 1;
            }
            const int64_t k = dst + (int64_t)e;
            if (k < capacity)
                ctx_idx[k] = (int32_t)pl[s_st[gb][lo] + (e - s_pre[gb][lo])];
            else
                over = true;
        }
        dst += tot;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (over) raise_error(status, CAGQ_ERR_CAPACITY);
}

}  // namespace

hipError_t launch_context_offsets(const Layout& L, const cagq_grid_desc& d, void* ws, const int32_t* center_lin,
                                  int32_t M, int64_t* ctx_off, hipStream_t s) {
    GridDims g;
    for (int a = 0; a < 3; ++a) g.D[a] = d.dims[a];
    const int64_t total = (int64_t)L.B * M;
    const int64_t tiles = (total + kScanTile - 1) / kScanTile;
    uint64_t* off = reinterpret_cast<uint64_t*>(ctx_off);
    int* status = at<int>(ws, L.status);
    k_ctx_clear<<<(unsigned)((tiles + 255) / 256), 256, 0, s>>>(off, total, tiles, status);
    auto go = [&](auto kern) {
        kern<<<(unsigned)tiles, kScanThreads, 0, s>>>(L.N, M, total, L.W, g, at<uint64_t>(ws, L.bitmap),
                                                      at<uint32_t>(ws, L.word_rank), at<uint32_t>(ws, L.vox_off),
                                                      center_lin, off, status);
    };
    if (d.radius == 1)
        go(k_ctx_count<1>);
    else if (d.radius == 2)
        go(k_ctx_count<2>);
    else
        go(k_ctx_count<3>);
    k_ctx_unflag<<<(unsigned)((tiles + 255) / 256), 256, 0, s>>>(off, total, tiles);
    return hipGetLastError();
}

hipError_t launch_context_list(const Layout& L, const cagq_grid_desc& d, void* ws, const int32_t* center_lin,
                               int32_t M, const int64_t* ctx_off, int32_t* ctx_idx, int64_t capacity,
                               hipStream_t s) {
    GridDims g;
    for (int a = 0; a < 3; ++a) g.D[a] = d.dims[a];
    const int64_t total = (int64_t)L.B * M;
    constexpr int GPB = kFillThreads / kFillG;
    const unsigned blocks = (unsigned)((total + GPB - 1) / GPB);
    auto go = [&](auto kern) {
        kern<<<blocks, kFillThreads, 0, s>>>(L.N, M, total, L.W, g, at<uint64_t>(ws, L.bitmap),
                                             at<uint32_t>(ws, L.word_rank), at<uint32_t>(ws, L.vox_off),
                                             at<uint32_t>(ws, L.pt_list), center_lin, ctx_off, ctx_idx, capacity,
                                             at<int>(ws, L.status));
    };
    if (d.radius == 1)
        go(k_ctx_fill<1>);
    else if (d.radius == 2)
        go(k_ctx_fill<2>);
    else
        go(k_ctx_fill<3>);
    return hipGetLastError();
}

}  // namespace cagq
