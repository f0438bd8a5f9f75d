// Node points querying and group centers (Sec. 3.2 "Node points querying";
// Appendix D, general procedure, step 3; Appendix E, Eqs. 7-8).
//
// One group of G lanes (G = 16, 32 or 64, G >= K) per center voxel v, 64/G
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
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kQueryThreads = 256;

struct QGrid {
    float o[3];
    float s[3];
    int32_t D[3];
};

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int G>
__device__ __forceinline__ uint64_t gshfl64(uint64_t v, int src) {
    int lo = __shfl((int)(uint32_t)v, src, G);
    int hi = __shfl((int)(uint32_t)(v >> 32), src, G);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

template <int G>
__device__ __forceinline__ uint64_t gxor64(uint64_t v, int m) {
    int lo = __shfl_xor((int)(uint32_t)v, m, G);
    int hi = __shfl_xor((int)(uint32_t)(v >> 32), m, G);
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

template <int G>
__device__ __forceinline__ uint32_t gsum(uint32_t v) {
#pragma unroll
    for (int d = 1; d < G; d <<= 1) v += (uint32_t)__shfl_xor((int)v, d, G);
    return v;
}

// Compare-exchange of (key, payload) with the partner lane lg ^ j: this lane
// keeps the smaller key when keep_min, else the larger.
template <int G>
__device__ __forceinline__ void gcx(uint64_t& k, uint32_t& p, int j, bool keep_min) {
    const uint64_t ok = gxor64<G>(k, j);
    const uint32_t op = (uint32_t)__shfl_xor((int)p, j, G);
    const bool take = keep_min ? (ok < k) : (ok > k);
    if (take) {
        k = ok;
        p = op;
    }
}

// Ascending bitonic sort of one (key, payload) per lane across the group.
template <int G>
__device__ __forceinline__ void gsort(uint64_t& k, uint32_t& p, int lg) {
#pragma unroll
    for (int s = 2; s <= G; s <<= 1) {
#pragma unroll
        for (int j = s >> 1; j > 0; j >>= 1) {
            const bool asc = (lg & s) == 0;
            const bool low = (lg & j) == 0;
            gcx<G>(k, p, j, asc == low);
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
    for (int j = G >> 1; j > 0; j >>= 1) gcx<G>(bk, bp, j, (lg & j) == 0);
}

template <int MODE, int G>
__global__ __launch_bounds__(kQueryThreads) void k_query(
    const uint32_t* __restrict__ Wt, int32_t N, int32_t M, int32_t K, int32_t total, QGrid g, int32_t rad,
    int64_t W, const uint64_t* __restrict__ bitmap, const uint32_t* __restrict__ word_rank,
    const uint32_t* __restrict__ vox_off, const float4* __restrict__ pt4, const int32_t* __restrict__ center_lin,
    uint64_t seed, int32_t* __restrict__ node_idx, float* __restrict__ node_xyz, int32_t* __restrict__ n_valid,
    float* __restrict__ center_xyz, uint32_t* __restrict__ center_w, int32_t* __restrict__ ctx_count,
    int* __restrict__ status) {
    extern __shared__ uint32_t smem[];
    constexpr int GPB = kQueryThreads / G;  // groups per block
    const int side = 2 * rad + 1;
    const int nnb = side * side * side;
    const int lane = lane_id();
    const int lg = lane & (G - 1);
    const int gb = threadIdx.x / G;  // group within the block
    uint32_t* s_pre = smem + (size_t)gb * (2 * nnb + 1);
    uint32_t* s_st = s_pre + nnb + 1;
    const uint32_t blk = xcd_block(blockIdx.x, gridDim.x);
    const int32_t cid = (int32_t)blk * GPB + gb;
    // every group runs to the end (the group- and wave-wide steps need all
    // lanes); a group past the end works on center 0 and writes nothing
    const bool live = cid < total;
    const int32_t c_id = live ? cid : 0;
    const int32_t b = c_id / M;
    const size_t cK = (size_t)c_id * K;
    const int32_t lin_s = center_lin[c_id];
    const int64_t V = (int64_t)g.D[0] * g.D[1] * g.D[2];
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    const uint32_t* vo = vox_off + (size_t)b * (N + 1);
    const float4* p4 = pt4 + (size_t)b * N;
    // an unoccupied center has an empty context and gets zeros
    const bool occupied = lin_s >= 0 && (int64_t)lin_s < V && slot_of(bm, wr, (uint32_t)lin_s) >= 0;
    if (live && !occupied && lg == 0) raise_error(status, CAGQ_ERR_CENTER_NOT_OCCUPIED);
    const uint32_t lin = occupied ? (uint32_t)lin_s : 0u;
    const int32_t gx = (int32_t)(lin % (uint32_t)g.D[0]);
    const int32_t gy = (int32_t)((lin / (uint32_t)g.D[0]) % (uint32_t)g.D[1]);
    const int32_t gz = (int32_t)(lin / ((uint32_t)g.D[0] * (uint32_t)g.D[1]));

    // 1. occupied voxels of pi(v), compacted in ascending linear id
    uint32_t nocc = 0, c = 0;
    const int gshift = lane & ~(G - 1);
    const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
    for (int q0 = 0; q0 < nnb; q0 += G) {
        const int q = q0 + lg;
        bool occ = false;
        uint32_t st = 0, cnt = 0;
        if (occupied && q < nnb) {
            const int32_t x = gx + q % side - rad;
            const int32_t y = gy + (q / side) % side - rad;
            const int32_t z = gz + q / (side * side) - rad;
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
        const uint32_t pos = nocc + (uint32_t)__popcll(mask & ((1ull << lg) - 1));
        const uint32_t incl = gscan_incl<G>(cnt, lg);
        if (occ) {
            s_st[pos] = st;
            s_pre[pos] = c + incl - cnt;
        }
        c += (uint32_t)__shfl((int)incl, G - 1, G);
        nocc += (uint32_t)__popcll(mask);
    }
    if (lg == 0) s_pre[nocc] = c;
    wave_lds_sync();

    // 2-3. keys of the context points, G smallest kept sorted across the group
    uint64_t hc = 0;
    float qx = 0.f, qy = 0.f, qz = 0.f;
    if (MODE == CAGQ_QUERY_CUBE) {
        hc = sm64(sm64(sm64(seed ^ 2ull) ^ (uint64_t)b) ^ (uint64_t)lin);
    } else {
        qx = g.o[0] + ((float)gx + 0.5f) * g.s[0];
        qy = g.o[1] + ((float)gy + 0.5f) * g.s[1];
        qz = g.o[2] + ((float)gz + 0.5f) * g.s[2];
    }
    uint64_t bk = ~0ull;
    uint32_t bp = 0;
    // the chunk loop runs the same number of times for every group of the wave
    uint32_t cmax = c;
#pragma unroll
    for (int d = G; d < kWave; d <<= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)cmax, d, kWave);
        cmax = o > cmax ? o : cmax;
    }
    for (uint32_t e0 = 0; e0 < cmax; e0 += G) {
        const uint32_t e = e0 + lg;
        uint64_t key = ~0ull;
        uint32_t pos = 0;
        if (e < c) {
            // the compacted voxel holding context entry e
            uint32_t lo = 0, hi = nocc - 1;
            while (lo < hi) {
                const uint32_t mid = (lo + hi + 1) >> 1;
                if (s_pre[mid] <= e) lo = mid; else hi = mid - 1;
            }
            pos = s_st[lo] + (e - s_pre[lo]);
            const float4 v = p4[pos];
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
        }
        gsort<G>(key, pos, lg);
        if (e0 == 0) {
            bk = key;
            bp = pos;
        } else {
            gmerge_low<G>(bk, bp, key, pos, lg);
        }
    }

    // 4. outputs (an empty context gives n = 0 and zeros)
    const uint32_t n = c < (uint32_t)K ? c : (uint32_t)K;
    const int src = (uint32_t)lg < n ? lg : 0;
    const uint64_t mine = gshfl64<G>(bk, src);
    const uint32_t mpos = (uint32_t)__shfl((int)bp, src, G);
    const uint32_t idx = n ? (uint32_t)mine : 0u;
    const float4 pv = n ? p4[mpos] : make_float4(0.f, 0.f, 0.f, 0.f);
    const float x = pv.x, y = pv.y, z = pv.z;
    if (live && lg < K) {
        node_idx[cK + lg] = (int32_t)idx;
        if (node_xyz) {
            node_xyz[(cK + lg) * 3 + 0] = x;
            node_xyz[(cK + lg) * 3 + 1] = y;
            node_xyz[(cK + lg) * 3 + 2] = z;
        }
    }
    const bool valid = (uint32_t)lg < n;
    const uint32_t w = (Wt && n) ? Wt[(size_t)b * N + idx] : 1u;
    const uint32_t wc = gsum<G>(valid ? w : 0u);
    const float wf = (float)w;
    float tx = wf * x, ty = wf * y, tz = wf * z;
#pragma unroll
    for (int h = 1; h < G; h <<= 1) {
        const float ox = __shfl_down(tx, h, G);
        const float oy = __shfl_down(ty, h, G);
        const float oz = __shfl_down(tz, h, G);
        if ((lg & (2 * h - 1)) == 0 && (uint32_t)(lg + h) < n) {
            tx = tx + ox;
            ty = ty + oy;
            tz = tz + oz;
        }
    }
    if (live && lg == 0) {
        const float wcf = (float)wc;
        center_xyz[(size_t)cid * 3 + 0] = n ? tx / wcf : 0.0f;
        center_xyz[(size_t)cid * 3 + 1] = n ? ty / wcf : 0.0f;
        center_xyz[(size_t)cid * 3 + 2] = n ? tz / wcf : 0.0f;
        center_w[cid] = wc;
        n_valid[cid] = (int32_t)n;
        if (ctx_count) ctx_count[cid] = (int32_t)c;
    }
}

template <int MODE, int G>
void launch_g(const Layout& L, const QGrid& g, int32_t rad, void* ws, const uint32_t* weights,
              const int32_t* center_lin, int32_t M, int32_t K, uint64_t seed, int32_t* node_idx, float* node_xyz,
              int32_t* n_valid, float* center_xyz, uint32_t* center_w, int32_t* ctx_count, hipStream_t s) {
    constexpr int GPB = kQueryThreads / G;
    const int32_t total = L.B * M;
    const unsigned blocks = (unsigned)((total + GPB - 1) / GPB);
    const int side = 2 * rad + 1;
    const size_t lds = (size_t)GPB * (2 * side * side * side + 1) * sizeof(uint32_t);
    k_query<MODE, G><<<blocks, kQueryThreads, lds, s>>>(
        weights, L.N, M, K, total, g, rad, L.W, at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
        at<uint32_t>(ws, L.vox_off), at<float4>(ws, L.pt4), center_lin, seed, node_idx, node_xyz, n_valid,
        center_xyz, center_w, ctx_count, at<int>(ws, L.status));
}

template <int MODE>
void launch_mode(const Layout& L, const QGrid& g, int32_t rad, void* ws, const uint32_t* weights,
                 const int32_t* center_lin, int32_t M, int32_t K, uint64_t seed, int32_t* node_idx,
                 float* node_xyz, int32_t* n_valid, float* center_xyz, uint32_t* center_w, int32_t* ctx_count,
                 hipStream_t s) {
    if (K <= 16)
        launch_g<MODE, 16>(L, g, rad, ws, weights, center_lin, M, K, seed, node_idx, node_xyz, n_valid,
                           center_xyz, center_w, ctx_count, s);
    else if (K <= 32)
        launch_g<MODE, 32>(L, g, rad, ws, weights, center_lin, M, K, seed, node_idx, node_xyz, n_valid,
                           center_xyz, center_w, ctx_count, s);
    else
        launch_g<MODE, 64>(L, g, rad, ws, weights, center_lin, M, K, seed, node_idx, node_xyz, n_valid,
                           center_xyz, center_w, ctx_count, s);
}

}  // namespace

hipError_t launch_query(const Layout& L, const cagq_grid_desc& d, const float* points, void* ws,
                        const uint32_t* weights, const int32_t* center_lin, int32_t M, int32_t K,
                        int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                        int32_t* n_valid, float* center_xyz, uint32_t* center_w, int32_t* ctx_count,
                        hipStream_t s) {
    (void)points;  // node coordinates are bit copies read from the slot-ordered copy
    QGrid g;
    for (int a = 0; a < 3; ++a) {
        g.o[a] = d.origin[a];
        g.s[a] = d.voxel_size[a];
        g.D[a] = d.dims[a];
    }
    if (mode == CAGQ_QUERY_CUBE)
        launch_mode<CAGQ_QUERY_CUBE>(L, g, d.radius, ws, weights, center_lin, M, K, seed, node_idx, node_xyz,
                                     n_valid, center_xyz, center_w, ctx_count, s);
    else
        launch_mode<CAGQ_QUERY_KNN>(L, g, d.radius, ws, weights, center_lin, M, K, seed, node_idx, node_xyz,
                                    n_valid, center_xyz, center_w, ctx_count, s);
    return hipGetLastError();
}

}  // namespace cagq
