// The comparison methods CAGQ is measured against (Sec. 4, the latency and
// coverage tables), and the occupied-space coverage metric. None of this is
// CAGQ itself:
//   Random Point Sampling   the M points of smallest key
//                           (hi32(h(seed, 4, b, i)) << 32) | i, in ascending
//                           index: one 1024-thread workgroup per cloud finds
//                           the bound by a 4-pass 8-bit radix select over the
//                           keys' top halves, then compacts in index order;
//   Farthest Point Sampling from point 0, each next center the point with the
//                           largest d^2 to its nearest chosen center (ties to
//                           the lowest index): one 1024-thread workgroup per
//                           cloud keeps every point's distance in registers
//                           and reduces (d^2, -index) to the next center;
//   Ball Query              the first K points in index order with
//                           d^2 < R^2 among all N: one wave per center scans
//                           64 points at a time and stops at K;
//   coverage                occupied voxels holding at least one node point,
//                           marked per slot (each point's slot is kept by
//                           the grid build), then counted per cloud.
// d^2 = (dx*dx + dy*dy) + dz*dz in fp32, each operation rounded.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kSelThreads = 1024;

__device__ __forceinline__ float dist2(const float* a, float bx, float by, float bz) {
    const float dx = a[0] - bx, dy = a[1] - by, dz = a[2] - bz;
    const float xx = dx * dx, yy = dy * dy, zz = dz * dz;
    const float s = xx + yy;
    return s + zz;
}

// ------------------------------------------------------------------ RPS

__global__ __launch_bounds__(kSelThreads) void k_rps(int32_t N, int32_t M, uint64_t seed,
                                                     int32_t* __restrict__ center_idx) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_prefix, s_need;
    __shared__ uint32_t s_wave[kSelThreads / kWave];
    const int32_t b = blockIdx.x;
    const int tid = threadIdx.x;
    const uint64_t hb = sm64(sm64(seed ^ 4ull) ^ (uint64_t)b);
    // radix select of the bound T on the keys' top halves, most significant
    // digit first: `need` keys with top half equal to T are taken
    uint32_t prefix = 0, need = (uint32_t)M;
    for (int pass = 0; pass < 4; ++pass) {
        const int sh = 24 - 8 * pass;
        const uint32_t hmask = pass == 0 ? 0u : ~0u << (sh + 8);
        for (int i = tid; i < 256; i += kSelThreads) hist[i] = 0;
        __syncthreads();
        for (int32_t i = tid; i < N; i += kSelThreads) {
            const uint32_t k = (uint32_t)(sm64(hb ^ (uint64_t)i) >> 32);
            if ((k & hmask) == prefix) atomicAdd(&hist[(k >> sh) & 255u], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            uint32_t acc = 0, d = 0;
            while (acc + hist[d] < need) acc += hist[d++];
            s_prefix = prefix | (d << sh);
            s_need = need - acc;
        }
        __syncthreads();
        prefix = s_prefix;
        need = s_need;
        __syncthreads();
    }
    // ordered compaction: keys below T, and the first `need` equal to T
    uint32_t base = 0, eq_base = 0;
    int32_t* out = center_idx + (size_t)b * M;
    const int lane = lane_id(), wv = tid / kWave;
    for (int32_t i0 = 0; i0 < N; i0 += kSelThreads) {
        const int32_t i = i0 + tid;
        const uint32_t k = i < N ? (uint32_t)(sm64(hb ^ (uint64_t)i) >> 32) : ~0u;
        const bool eq = i < N && k == prefix;
        // rank of this equal key among the equal keys so far
        const uint64_t eb = __ballot(eq);
        if (lane == 0) s_wave[wv] = (uint32_t)__popcll(eb);
        __syncthreads();
        uint32_t eoff = eq_base, etot = 0;
        for (int w = 0; w < kSelThreads / kWave; ++w) {
            if (w < wv) eoff += s_wave[w];
            etot += s_wave[w];
        }
        eoff += (uint32_t)__popcll(eb & ((1ull << lane) - 1));
        __syncthreads();
        const bool take = i < N && (k < prefix || (eq && eoff < need));
        const uint64_t tb = __ballot(take);
        if (lane == 0) s_wave[wv] = (uint32_t)__popcll(tb);
        __syncthreads();
        uint32_t off = base, tot = 0;
        for (int w = 0; w < kSelThreads / kWave; ++w) {
            if (w < wv) off += s_wave[w];
            tot += s_wave[w];
        }
        off += (uint32_t)__popcll(tb & ((1ull << lane) - 1));
        if (take) out[off] = i;
        base += tot;
        eq_base += etot;
        __syncthreads();
    }
}

// ------------------------------------------------------------------ FPS

template <int PER>
__global__ __launch_bounds__(kSelThreads) void k_fps(const float* __restrict__ points, int32_t N, int32_t M,
                                                     int32_t* __restrict__ center_idx) {
    __shared__ uint64_t s_best[kSelThreads / kWave];
    __shared__ int32_t s_cur;
    const int32_t b = blockIdx.x;
    const int tid = threadIdx.x, lane = lane_id(), wv = tid / kWave;
    const float* P = points + (size_t)b * N * 3;
    int32_t* out = center_idx + (size_t)b * M;
    float dmin[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) dmin[k] = __builtin_inff();
    // the cloud as a raw buffer: point tid + k * 1024 sits at the thread's
    // byte offset plus a constant, so no per-point address stays live
    // across the iterations (loads past the buffer's end read 0)
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)P, (short)0, N * 12, 0x00020000);
    const int vo = tid * 12;
    int32_t cur = 0;
    for (int32_t j = 0; j < M; ++j) {
        if (tid == 0) out[j] = cur;
        const float cx = P[(size_t)cur * 3 + 0], cy = P[(size_t)cur * 3 + 1], cz = P[(size_t)cur * 3 + 2];
        // this thread's farthest point (its indices ascend with k, so a
        // strict comparison keeps the lowest index of a tie)
        float bd = -1.0f;
        int32_t bi = 0;
#pragma unroll
        for (int k0 = 0; k0 < PER; k0 += 4) {
#pragma unroll
            for (int k = k0; k < k0 + 4 && k < PER; ++k) {
                const int32_t i = tid + k * kSelThreads;
                // one 12-byte load per point
                const auto v = __builtin_amdgcn_raw_buffer_load_b96(rs, vo, k * kSelThreads * 12, 0);
                const float px = __uint_as_float(v[0]), py = __uint_as_float(v[1]), pz = __uint_as_float(v[2]);
                if (i < N) {
                    const float dx = px - cx, dy = py - cy, dz = pz - cz;
                    const float xx = dx * dx, yy = dy * dy, zz = dz * dz;
                    const float sxy = xx + yy;
                    const float d = sxy + zz;
                    dmin[k] = d < dmin[k] ? d : dmin[k];
                    if (dmin[k] > bd) {
                        bd = dmin[k];
                        bi = i;
                    }
                }
            }
            // a few points' loads in flight at a time keep the distances in
            // registers
            __builtin_amdgcn_sched_barrier(0);
        }
        // (bits(d^2) << 32) | ~i: the largest is the farthest point, ties to
        // the lowest index (d^2 >= 0, so its bits order as the value)
        uint64_t best = bd < 0.0f ? 0ull : ((uint64_t)__float_as_uint(bd) << 32) | (uint32_t)~(uint32_t)bi;
        best = wave_max64(best);
        if (lane == 0) s_best[wv] = best;
        __syncthreads();
        if (tid < kWave) {
            uint64_t v = tid < kSelThreads / kWave ? s_best[tid] : 0ull;
            v = wave_max64(v);
            if (tid == 0) s_cur = (int32_t)~(uint32_t)v;
        }
        __syncthreads();
        cur = s_cur;
    }
}

// ------------------------------------------------------------------ Ball Query

constexpr int kBallThreads = 256;

__global__ __launch_bounds__(kBallThreads) void k_ball(const float* __restrict__ points, int32_t N, int32_t M,
                                                       int32_t total, const int32_t* __restrict__ center_idx,
                                                       int32_t K, float r2, int32_t* __restrict__ node_idx,
                                                       int32_t* __restrict__ n_valid) {
    const int lane = lane_id();
    const int32_t cid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * (kBallThreads / kWave) + threadIdx.x / kWave;
    if (cid >= total) return;  // whole waves leave together
    const int32_t b = cid / M;
    const float* P = points + (size_t)b * N * 3;
    int32_t* out = node_idx + (size_t)cid * K;
    const int32_t ci = center_idx[cid];
    int32_t n = 0, first = -1;
    if (ci >= 0 && ci < N) {
        const float cx = P[(size_t)ci * 3 + 0], cy = P[(size_t)ci * 3 + 1], cz = P[(size_t)ci * 3 + 2];
        for (int32_t i0 = 0; i0 < N && n < K; i0 += kWave) {
            const int32_t i = i0 + lane;
            const bool in = i < N && dist2(P + (size_t)i * 3, cx, cy, cz) < r2;
            const uint64_t bal = __ballot(in);
            const int32_t pos = n + (int32_t)__popcll(bal & ((1ull << lane) - 1));
            if (in && pos < K) out[pos] = i;
            if (bal && first < 0) first = i0 + (__ffsll((unsigned long long)bal) - 1);
            n += (int32_t)__popcll(bal);
        }
    }
    n = n < K ? n : K;
    for (int32_t k = n + lane; k < K; k += kWave) out[k] = first;  // -1 when nothing is inside
    if (lane == 0) n_valid[cid] = n;
}

// ------------------------------------------------------------------ coverage

__global__ void k_cov_clear(uint4* __restrict__ p, size_t n16) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

struct CovGrid {
    float o[3], s[3];
    int32_t D[3];
    int64_t W;
};

// Every valid node point stores 1 into the byte of its voxel's slot (the same
// value from every writer: no atomic needed). The slot comes from the point's
// coordinates by the voxelization rule and the occupancy words.
__global__ __launch_bounds__(256) void k_cov_mark(const float* __restrict__ P, int32_t N, int32_t M, int32_t K,
                                                  int64_t total, CovGrid g, const int32_t* __restrict__ node_idx,
                                                  const int32_t* __restrict__ n_valid,
                                                  const uint64_t* __restrict__ bitmap,
                                                  const uint32_t* __restrict__ word_rank, uint8_t* __restrict__ mark) {
    const int64_t t = (int64_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    if (t >= total) return;
    const int64_t cj = t / K;
    const int32_t k = (int32_t)(t - cj * K);
    if (k >= n_valid[cj]) return;
    const int32_t i = node_idx[t];
    if (i < 0 || i >= N) return;
    const int32_t b = (int32_t)(cj / M);
    const float* p = P + ((size_t)b * N + i) * 3;
    uint32_t gg[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        const float c = p[a];
        gg[a] = isfinite(c) ? (uint32_t)axis_index(c, g.o[a], g.s[a], g.D[a]) : 0u;
    }
    const uint32_t lin = gg[0] + (uint32_t)g.D[0] * (gg[1] + (uint32_t)g.D[1] * gg[2]);
    const int32_t slot = slot_of(bitmap + (size_t)b * g.W, word_rank + (size_t)b * g.W, lin);
    if (slot >= 0) mark[(size_t)b * N + slot] = 1;
}

__global__ __launch_bounds__(1024) void k_cov_count(int32_t N, const int32_t* __restrict__ nvox,
                                                    const uint8_t* __restrict__ mark, int32_t* __restrict__ covered) {
    __shared__ uint32_t s_wave[1024 / kWave];
    const int32_t b = blockIdx.x;
    const int32_t nv = nvox[b];
    const uint8_t* m = mark + (size_t)b * N;
    uint32_t c = 0;
    for (int32_t s = threadIdx.x; s < nv; s += blockDim.x) c += m[s];
    c = wave_sum<uint32_t>(c);
    if (lane_id() == 0) s_wave[threadIdx.x / kWave] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int w = 0; w < 1024 / kWave; ++w) t += s_wave[w];
        covered[b] = (int32_t)t;
    }
}

}  // namespace

hipError_t launch_sample_points(const float* points, int32_t B, int32_t N, int32_t M, int32_t mode, uint64_t seed,
                                int32_t* center_idx, hipStream_t s) {
    if (mode == 0) {
        k_rps<<<B, kSelThreads, 0, s>>>(N, M, seed, center_idx);
    } else {
        const int32_t per = (N + kSelThreads - 1) / kSelThreads;
        if (per <= 4)
            k_fps<4><<<B, kSelThreads, 0, s>>>(points, N, M, center_idx);
        else if (per <= 16)
            k_fps<16><<<B, kSelThreads, 0, s>>>(points, N, M, center_idx);
        else if (per <= 40)
            k_fps<40><<<B, kSelThreads, 0, s>>>(points, N, M, center_idx);
        else
            k_fps<80><<<B, kSelThreads, 0, s>>>(points, N, M, center_idx);
    }
    return hipGetLastError();
}

hipError_t launch_ball_query(const float* points, int32_t B, int32_t N, const int32_t* center_idx, int32_t M,
                             int32_t K, float radius2, int32_t* node_idx, int32_t* n_valid, hipStream_t s) {
    const int32_t total = B * M;
    constexpr int WPB = kBallThreads / kWave;
    k_ball<<<(unsigned)((total + WPB - 1) / WPB), kBallThreads, 0, s>>>(points, N, M, total, center_idx, K, radius2,
                                                                        node_idx, n_valid);
    return hipGetLastError();
}

hipError_t launch_coverage(const Layout& L, const cagq_grid_desc& d, const float* points, void* ws,
                           const int32_t* node_idx, const int32_t* n_valid, int32_t M, int32_t K, int32_t* covered,
                           hipStream_t s) {
    const size_t BN = (size_t)L.B * L.N;
    uint8_t* mark = at<uint8_t>(ws, L.cov_mark);
    const size_t n16 = (BN + 15) / 16;
    k_cov_clear<<<(unsigned)((n16 + 255) / 256 < 2048 ? (n16 + 255) / 256 : 2048), 256, 0, s>>>(
        reinterpret_cast<uint4*>(mark), n16);
    const int64_t total = (int64_t)L.B * M * K;
    CovGrid g;
    for (int a = 0; a < 3; ++a) {
        g.o[a] = d.origin[a];
        g.s[a] = d.voxel_size[a];
        g.D[a] = d.dims[a];
    }
    g.W = L.W;
    k_cov_mark<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(points, L.N, M, K, total, g, node_idx, n_valid,
                                                               at<uint64_t>(ws, L.bitmap),
                                                               at<uint32_t>(ws, L.word_rank), mark);
    k_cov_count<<<L.B, 1024, 0, s>>>(L.N, at<int32_t>(ws, L.nvox), mark, covered);
    return hipGetLastError();
}

}  // namespace cagq
