// Node points querying and group centers (Sec. 3.2 "Node points querying";
// Appendix D, general procedure, step 3; Appendix E, Eqs. 7-8).
//
// One 64-lane wavefront per center voxel v:
//   1. the lanes probe the (2r+1)^3 voxels of pi(v) in the occupancy bitmap
//      and compact the occupied ones (slot start, running context count) into
//      LDS -- the context is the concatenation of their stored lists, c points;
//   2. context points are streamed 64 at a time from the slot-ordered copy of
//      the stored points (one 16-byte load gives x, y, z and the index); each
//      lane forms a 64-bit key, (hi32(h(seed,2,b,lin(v),i)) << 32) | i for
//      Cube Query or (bits(d^2) << 32) | i for k-NN, d measured from the
//      center of v;
//   3. a wavefront bitonic sort of the chunk is merged into the running 64
//      smallest keys; lanes 0..min(K, c)-1 end up holding the node points in
//      ascending key order;
//   4. node coordinates are bit copies of the input; w_c is the integer sum of
//      the node weights and chi_c the pairwise fp32 sum of w_k * p_k (a
//      shuffle-down tree: stride 1, 2, 4, ...) divided by w_c.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kQueryThreads = 256;
constexpr int kQueryWaves = kQueryThreads / kWave;
constexpr int kMaxNb = (2 * CAGQ_MAX_RADIUS + 1) * (2 * CAGQ_MAX_RADIUS + 1) * (2 * CAGQ_MAX_RADIUS + 1);

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

template <int MODE>
__global__ __launch_bounds__(kQueryThreads) void k_query(
    const float* __restrict__ P, const uint32_t* __restrict__ Wt, int32_t N, int32_t M, int32_t K,
    int32_t total, QGrid g, int32_t rad, int64_t W, const uint64_t* __restrict__ bitmap,
    const uint32_t* __restrict__ word_rank, const uint32_t* __restrict__ vox_off,
    const float4* __restrict__ pt4, const int32_t* __restrict__ center_lin, uint64_t seed,
    int32_t* __restrict__ node_idx, float* __restrict__ node_xyz, int32_t* __restrict__ n_valid,
    float* __restrict__ center_xyz, uint32_t* __restrict__ center_w, int32_t* __restrict__ ctx_count,
    int* __restrict__ status) {
    __shared__ uint32_t s_pre[kQueryWaves][kMaxNb + 1];
    __shared__ uint32_t s_st[kQueryWaves][kMaxNb];
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const uint32_t blk = xcd_block(blockIdx.x, gridDim.x);
    const int32_t cid = (int32_t)blk * kQueryWaves + wv;
    if (cid >= total) return;
    const int32_t b = cid / M;
    const size_t cK = (size_t)cid * K;
    const int32_t lin_s = center_lin[cid];
    const int64_t V = (int64_t)g.D[0] * g.D[1] * g.D[2];
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    const uint32_t* vo = vox_off + (size_t)b * (N + 1);
    const float4* p4 = pt4 + (size_t)b * N;
    const float* Pb = P + (size_t)b * N * 3;

    if (lin_s < 0 || (int64_t)lin_s >= V || slot_of(bm, wr, (uint32_t)lin_s) < 0) {
        if (lane == 0) raise_error(status, CAGQ_ERR_CENTER_NOT_OCCUPIED);
        if (lane < K) {
            node_idx[cK + lane] = 0;
            if (node_xyz) {
                node_xyz[(cK + lane) * 3 + 0] = 0.0f;
                node_xyz[(cK + lane) * 3 + 1] = 0.0f;
                node_xyz[(cK + lane) * 3 + 2] = 0.0f;
            }
        }
        if (lane < 3) center_xyz[(size_t)cid * 3 + lane] = 0.0f;
        if (lane == 0) {
            n_valid[cid] = 0;
            center_w[cid] = 0;
            if (ctx_count) ctx_count[cid] = 0;
        }
        return;
    }
    const uint32_t lin = (uint32_t)lin_s;
    const int32_t gx = (int32_t)(lin % (uint32_t)g.D[0]);
    const int32_t gy = (int32_t)((lin / (uint32_t)g.D[0]) % (uint32_t)g.D[1]);
    const int32_t gz = (int32_t)(lin / ((uint32_t)g.D[0] * (uint32_t)g.D[1]));

    // 1. occupied voxels of pi(v), compacted in ascending linear id
    const int32_t side = 2 * rad + 1;
    const int32_t nnb = side * side * side;
    uint32_t nocc = 0, c = 0;
    for (int32_t q0 = 0; q0 < nnb; q0 += kWave) {
        const int32_t q = q0 + lane;
        bool occ = false;
        uint32_t st = 0, cnt = 0;
        if (q < nnb) {
            int32_t x = gx + q % side - rad;
            int32_t y = gy + (q / side) % side - rad;
            int32_t z = gz + q / (side * side) - rad;
            if (x >= 0 && y >= 0 && z >= 0 && x < g.D[0] && y < g.D[1] && z < g.D[2]) {
                uint32_t nl = (uint32_t)x + (uint32_t)g.D[0] * ((uint32_t)y + (uint32_t)g.D[1] * (uint32_t)z);
                int32_t sl = slot_of(bm, wr, nl);
                if (sl >= 0) {
                    st = vo[sl];
                    cnt = vo[sl + 1] - st;
                    occ = true;
                }
            }
        }
        const uint64_t mask = __ballot(occ);
        const uint32_t pos = nocc + (uint32_t)__popcll(mask & ((1ull << lane) - 1));
        const uint32_t incl = wave_incl_scan<uint32_t>(cnt);
        if (occ) {
            s_st[wv][pos] = st;
            s_pre[wv][pos] = c + incl - cnt;
        }
        c += (uint32_t)__shfl((int)incl, kWave - 1, kWave);
        nocc += (uint32_t)__popcll(mask);
    }
    if (lane == 0) s_pre[wv][nocc] = c;
    wave_lds_sync();

    // 2-3. keys of the context points, 64 smallest kept sorted across the lanes
    uint64_t hc = 0;
    float qx = 0.f, qy = 0.f, qz = 0.f;
    if (MODE == CAGQ_QUERY_CUBE) {
        hc = sm64(sm64(sm64(seed ^ 2ull) ^ (uint64_t)b) ^ (uint64_t)lin);
    } else {
        qx = g.o[0] + ((float)gx + 0.5f) * g.s[0];
        qy = g.o[1] + ((float)gy + 0.5f) * g.s[1];
        qz = g.o[2] + ((float)gz + 0.5f) * g.s[2];
    }
    uint64_t best = ~0ull;
    for (uint32_t e0 = 0; e0 < c; e0 += kWave) {
        const uint32_t e = e0 + lane;
        uint64_t key = ~0ull;
        if (e < c) {
            // the compacted voxel holding context entry e
            uint32_t lo = 0, hi = nocc - 1;
            while (lo < hi) {
                uint32_t mid = (lo + hi + 1) >> 1;
                if (s_pre[wv][mid] <= e) lo = mid; else hi = mid - 1;
            }
            const float4 v = p4[s_st[wv][lo] + (e - s_pre[wv][lo])];
            const uint32_t i = __float_as_uint(v.w);
            if (MODE == CAGQ_QUERY_CUBE) {
                key = (sm64(hc ^ (uint64_t)i) & 0xFFFFFFFF00000000ull) | i;
            } else {
                float dx = v.x - qx, dy = v.y - qy, dz = v.z - qz;
                float xx = dx * dx, yy = dy * dy, zz = dz * dz;
                float sxy = xx + yy;
                float d2 = sxy + zz;
                key = ((uint64_t)__float_as_uint(d2) << 32) | i;
            }
        }
        key = wave_sort64(key);
        best = e0 == 0 ? key : wave_merge_low64(best, key);
    }

    // 4. outputs
    const uint32_t n = c < (uint32_t)K ? c : (uint32_t)K;
    const uint64_t mine = shfl64(best, (uint32_t)lane < n ? lane : 0);
    const uint32_t idx = (uint32_t)mine;
    const float* p = Pb + (size_t)idx * 3;
    const float x = p[0], y = p[1], z = p[2];
    if (lane < K) {
        node_idx[cK + lane] = (int32_t)idx;
        if (node_xyz) {
            node_xyz[(cK + lane) * 3 + 0] = x;
            node_xyz[(cK + lane) * 3 + 1] = y;
            node_xyz[(cK + lane) * 3 + 2] = z;
        }
    }
    const bool valid = (uint32_t)lane < n;
    const uint32_t w = Wt ? Wt[(size_t)b * N + idx] : 1u;
    const uint32_t wc = wave_sum<uint32_t>(valid ? w : 0u);
    const float wf = (float)w;
    float tx = wf * x, ty = wf * y, tz = wf * z;
#pragma unroll
    for (int h = 1; h < kWave; h <<= 1) {
        float ox = __shfl_down(tx, h, kWave);
        float oy = __shfl_down(ty, h, kWave);
        float oz = __shfl_down(tz, h, kWave);
        if ((lane & (2 * h - 1)) == 0 && (uint32_t)(lane + h) < n) {
            tx = tx + ox;
            ty = ty + oy;
            tz = tz + oz;
        }
    }
    if (lane == 0) {
        const float wcf = (float)wc;
        center_xyz[(size_t)cid * 3 + 0] = tx / wcf;
        center_xyz[(size_t)cid * 3 + 1] = ty / wcf;
        center_xyz[(size_t)cid * 3 + 2] = tz / wcf;
        center_w[cid] = wc;
        n_valid[cid] = (int32_t)n;
        if (ctx_count) ctx_count[cid] = (int32_t)c;
    }
}

}  // namespace

hipError_t launch_query(const Layout& L, const cagq_grid_desc& d, const float* points, void* ws,
                        const uint32_t* weights, const int32_t* center_lin, int32_t M, int32_t K,
                        int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz,
                        int32_t* n_valid, float* center_xyz, uint32_t* center_w, int32_t* ctx_count,
                        hipStream_t s) {
    QGrid g;
    for (int a = 0; a < 3; ++a) {
        g.o[a] = d.origin[a];
        g.s[a] = d.voxel_size[a];
        g.D[a] = d.dims[a];
    }
    const int32_t total = L.B * M;
    const unsigned blocks = (unsigned)((total + kQueryWaves - 1) / kQueryWaves);
    auto args = [&](auto kern) {
        kern<<<blocks, kQueryThreads, 0, s>>>(points, weights, L.N, M, K, total, g, d.radius, L.W,
                                              at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
                                              at<uint32_t>(ws, L.vox_off), at<float4>(ws, L.pt4), center_lin,
                                              seed, node_idx, node_xyz, n_valid, center_xyz, center_w,
                                              ctx_count, at<int>(ws, L.status));
    };
    if (mode == CAGQ_QUERY_CUBE) args(k_query<CAGQ_QUERY_CUBE>);
    else args(k_query<CAGQ_QUERY_KNN>);
    return hipGetLastError();
}

}  // namespace cagq
