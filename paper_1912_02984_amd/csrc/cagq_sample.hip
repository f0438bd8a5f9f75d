// Center voxel sampling (Sec. 3.2 "center voxels sampling"; Appendix D,
// general procedure, step 2).
//
// RVS: every occupied voxel is equally likely. Slot s of cloud b gets the
// key (hi32(h(seed, 1, b, s)) << 32) | s with h the splitmix64 chain; the
// m = min(M, |O_v|) smallest keys win. One workgroup per cloud finds the m-th
// smallest key by an 8-bit radix select in LDS and writes the winners in slot
// (= ascending linear id) order.
//
// CAS (Eqs. 1-2, greedy reading): the sequential greedy repeatedly picks the
// unpicked voxel of largest score 2^16*lambda*#{V in pi(v): C_V = 0} -
// beta_q16 * sum_{V in pi(v)} C_V, ties to the lowest linear id. With
// beta >= 0 no score ever rises, and a pick only changes the scores of voxels
// within Chebyshev distance 2r of it. Hence a voxel whose key (score, -lin)
// beats every unpicked voxel within distance 2r is picked by the sequential
// greedy with that very key, and all such voxels of a round can be applied
// at once (their neighbourhoods are disjoint). Rounds repeat until the picks
// whose key exceeds the best unpicked key number at least m: those are the
// sequential greedy's first picks, and the m largest keys among them are
// its first m picks. They are emitted in ascending linear id.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kSelThreads = 1024;

struct CasPtrs {
    uint64_t* gmax;   // [2][B] best key among unpicked voxels, per round parity
    uint32_t* count;  // [2][B] picks whose key beats that best, per round parity
    uint32_t* done;   // [B]
};

CasPtrs cas_ptrs(const Layout& L, void* ws) {
    char* base = static_cast<char*>(ws) + L.cas_ctl;
    CasPtrs c;
    c.gmax = reinterpret_cast<uint64_t*>(base);
    c.count = reinterpret_cast<uint32_t*>(base + (size_t)16 * L.B);
    c.done = reinterpret_cast<uint32_t*>(base + (size_t)24 * L.B);
    return c;
}

__device__ __forceinline__ uint64_t select_key(int key_mode, uint64_t hb, int32_t s,
                                               const uint64_t* __restrict__ pick) {
    if (key_mode == 0) {
        uint64_t h = sm64(hb ^ (uint64_t)(uint32_t)s);
        return (h & 0xFFFFFFFF00000000ull) | (uint32_t)s;
    }
    return ~pick[s];  // largest pick key first; unpicked voxels (0) last
}

__global__ __launch_bounds__(kSelThreads) void k_select(int32_t N, const int32_t* __restrict__ nvox,
                                                        const uint32_t* __restrict__ vox_lin, int32_t M,
                                                        int key_mode, uint64_t seed,
                                                        const uint64_t* __restrict__ cas_pick,
                                                        int32_t* __restrict__ center_lin,
                                                        int32_t* __restrict__ m_valid) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_digit, s_below, s_cnt;
    __shared__ uint32_t s_wave[kSelThreads / kWave];
    const int32_t b = blockIdx.x;
    const int32_t nv = nvox[b];
    const int32_t m = M < nv ? M : nv;
    const uint64_t hb = sm64(sm64(seed ^ 1ull) ^ (uint64_t)b);
    const uint64_t* pick = cas_pick ? cas_pick + (size_t)b * N : nullptr;
    const int tid = threadIdx.x;

    // radix select of the m-th smallest key T
    uint64_t prefix = 0, mask = 0, T = 0;
    uint32_t need = (uint32_t)m;
    bool exact = true;
    for (int shift = 56; shift >= 0; shift -= 8) {
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        for (int32_t s = tid; s < nv; s += kSelThreads) {
            uint64_t k = select_key(key_mode, hb, s, pick);
            if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1u);
        }
        __syncthreads();
        if (tid < kWave) {
            // the digit whose cumulative count first reaches `need`
            uint32_t h4[4], sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h4[j] = hist[tid * 4 + j];
                sum += h4[j];
            }
            uint32_t incl = wave_incl_scan<uint32_t>(sum);
            uint32_t run = incl - sum;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (run < need && run + h4[j] >= need) {
                    s_digit = (uint32_t)(tid * 4 + j);
                    s_below = run;
                    s_cnt = h4[j];
                }
                run += h4[j];
            }
        }
        __syncthreads();
        const uint32_t digit = s_digit, below = s_below, cnt = s_cnt;
        __syncthreads();
        prefix |= (uint64_t)digit << shift;
        mask |= 255ull << shift;
        need -= below;
        if (cnt == need) {  // every key under this prefix is among the m smallest
            T = prefix | ~mask;
            exact = false;
            break;
        }
    }
    if (exact) T = prefix;

    // ordered compaction of {s : key(s) <= T}
    const int32_t chunk = (nv + kSelThreads - 1) / kSelThreads;
    const int32_t s_begin = tid * chunk;
    const int32_t s_end = min(nv, s_begin + chunk);
    uint32_t mine = 0;
    for (int32_t s = s_begin; s < s_end; ++s) mine += select_key(key_mode, hb, s, pick) <= T ? 1u : 0u;
    uint32_t incl = wave_incl_scan<uint32_t>(mine);
    const int wv = tid / kWave;
    if (lane_id() == kWave - 1) s_wave[wv] = incl;
    __syncthreads();
    uint32_t pos = incl - mine;
    for (int i = 0; i < wv; ++i) pos += s_wave[i];
    int32_t* out = center_lin + (size_t)b * M;
    const uint32_t* vl = vox_lin + (size_t)b * N;
    for (int32_t s = s_begin; s < s_end; ++s)
        if (select_key(key_mode, hb, s, pick) <= T && pos < (uint32_t)m) out[pos++] = (int32_t)vl[s];
    __syncthreads();
    for (int32_t j = m + tid; j < M; j += kSelThreads) out[j] = out[j % m];
    if (tid == 0) m_valid[b] = m;
}

struct GridDims {
    int32_t D[3];
};

__device__ __forceinline__ void decode(uint32_t lin, const GridDims& g, int32_t* x, int32_t* y, int32_t* z) {
    *x = (int32_t)(lin % (uint32_t)g.D[0]);
    *y = (int32_t)((lin / (uint32_t)g.D[0]) % (uint32_t)g.D[1]);
    *z = (int32_t)(lin / ((uint32_t)g.D[0] * (uint32_t)g.D[1]));
}

__global__ void k_cas_init(int32_t BN, int32_t B, uint32_t* __restrict__ cover, uint64_t* __restrict__ pick,
                           uint32_t* __restrict__ round, CasPtrs ctl) {
    int32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    if (gid < BN) {
        cover[gid] = 0;
        pick[gid] = 0;
        round[gid] = 0;
    }
    if (gid < B) {
        ctl.gmax[gid] = 0;
        ctl.gmax[B + gid] = 0;
        ctl.count[gid] = 0;
        ctl.count[B + gid] = 0;
        ctl.done[gid] = 0;
    }
}

// Round R, phase 1: key of every unpicked voxel and their maximum per cloud.
__global__ __launch_bounds__(256) void k_cas_score(
    int32_t R, int32_t B, int32_t N, int64_t W, GridDims g, int32_t rad, int64_t lam, uint32_t beta_q16,
    int32_t M, const int32_t* __restrict__ nvox, const uint32_t* __restrict__ vox_lin,
    const uint64_t* __restrict__ bitmap, const uint32_t* __restrict__ word_rank,
    const uint32_t* __restrict__ cover, const uint64_t* __restrict__ pick, uint64_t* __restrict__ key,
    CasPtrs ctl) {
    // no early exit: every lane takes part in the wave reduction at the end
    const int32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    const bool in_range = gid < B * N;
    const int32_t b = in_range ? gid / N : B - 1, s = in_range ? gid - b * N : N;
    bool active = in_range && ctl.done[b] == 0;
    const int32_t nv = nvox[b];
    if (active && R > 0) {
        const uint32_t m = (uint32_t)(M < nv ? M : nv);
        if (ctl.count[((R - 1) & 1) * B + b] >= m) {
            if (s == 0) ctl.done[b] = 1;
            active = false;
        }
    }
    if (active && s == 0) ctl.count[(R & 1) * B + b] = 0;
    uint64_t k = 0;
    if (active && s < nv && pick[gid] == 0) {
        const uint64_t* bm = bitmap + (size_t)b * W;
        const uint32_t* wr = word_rank + (size_t)b * W;
        const uint32_t* cv = cover + (size_t)b * N;
        const uint32_t lin = vox_lin[gid];
        int32_t x, y, z;
        decode(lin, g, &x, &y, &z);
        int64_t U = 0, cs = 0;
        for (int32_t dz = -rad; dz <= rad; ++dz) {
            int32_t zz = z + dz;
            if (zz < 0 || zz >= g.D[2]) continue;
            for (int32_t dy = -rad; dy <= rad; ++dy) {
                int32_t yy = y + dy;
                if (yy < 0 || yy >= g.D[1]) continue;
                for (int32_t dx = -rad; dx <= rad; ++dx) {
                    int32_t xx = x + dx;
                    if (xx < 0 || xx >= g.D[0]) continue;
                    uint32_t nl = (uint32_t)xx + (uint32_t)g.D[0] * ((uint32_t)yy + (uint32_t)g.D[1] * (uint32_t)zz);
                    int32_t sl = slot_of(bm, wr, nl);
                    if (sl < 0) continue;
                    uint32_t c = cv[sl];
                    U += c == 0 ? 1 : 0;
                    cs += c;
                }
            }
        }
        int64_t score = 65536ll * lam * U - (int64_t)beta_q16 * cs;
        k = ((uint64_t)(score + 2147483648ll) << 32) | (uint64_t)(0xFFFFFFFFu - lin);
        key[gid] = k;
    }
    // per-cloud maximum: reduce over the lanes of this wave that share the cloud
    const int32_t b0 = __shfl(b, 0, kWave), b1 = __shfl(b, kWave - 1, kWave);
    if (b0 == b1) {
        uint64_t mx = wave_max64(k);
        if (lane_id() == 0 && mx) atomicMax((unsigned long long*)&ctl.gmax[(R & 1) * B + b], mx);
    } else if (k) {
        atomicMax((unsigned long long*)&ctl.gmax[(R & 1) * B + b], k);
    }
}

// Round R, phase 2: voxels whose key beats every voxel unpicked at the round's
// start within distance 2r are picked; coverage counts of their neighbourhoods
// rise by one. Also counts earlier picks whose key beats this round's best.
__global__ __launch_bounds__(256) void k_cas_pick(
    int32_t R, int32_t B, int32_t N, int64_t W, GridDims g, int32_t rad, const int32_t* __restrict__ nvox,
    const uint32_t* __restrict__ vox_lin, const uint64_t* __restrict__ bitmap,
    const uint32_t* __restrict__ word_rank, uint32_t* __restrict__ cover, uint64_t* __restrict__ pick,
    uint32_t* __restrict__ round, const uint64_t* __restrict__ key, CasPtrs ctl) {
    // no early exit: every lane takes part in the wave reduction at the end
    const int32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    const bool in_range = gid < B * N;
    const int32_t b = in_range ? gid / N : B - 1, s = in_range ? gid - b * N : N;
    const bool active = in_range && ctl.done[b] == 0;
    if (active && s == 0) ctl.gmax[((R + 1) & 1) * B + b] = 0;
    const int32_t nv = nvox[b];
    uint32_t above = 0;
    if (active && s < nv) {
        const uint64_t G = ctl.gmax[(R & 1) * B + b];
        const uint64_t pk = pick[gid];
        if (pk != 0) {
            above = pk > G ? 1u : 0u;
        } else {
            const uint64_t* bm = bitmap + (size_t)b * W;
            const uint32_t* wr = word_rank + (size_t)b * W;
            const uint64_t* ky = key + (size_t)b * N;
            const uint32_t* rd = round + (size_t)b * N;
            const uint64_t my = key[gid];
            const uint32_t lin = vox_lin[gid];
            int32_t x, y, z;
            decode(lin, g, &x, &y, &z);
            const int32_t r2 = 2 * rad;
            bool best = true;
            for (int32_t dz = -r2; dz <= r2 && best; ++dz) {
                int32_t zz = z + dz;
                if (zz < 0 || zz >= g.D[2]) continue;
                for (int32_t dy = -r2; dy <= r2 && best; ++dy) {
                    int32_t yy = y + dy;
                    if (yy < 0 || yy >= g.D[1]) continue;
                    for (int32_t dx = -r2; dx <= r2; ++dx) {
                        int32_t xx = x + dx;
                        if (xx < 0 || xx >= g.D[0] || (dx == 0 && dy == 0 && dz == 0)) continue;
                        uint32_t nl = (uint32_t)xx + (uint32_t)g.D[0] * ((uint32_t)yy + (uint32_t)g.D[1] * (uint32_t)zz);
                        int32_t sl = slot_of(bm, wr, nl);
                        if (sl < 0) continue;
                        uint32_t rr = rd[sl];
                        // unpicked at the round's start: never picked, or picked in this round
                        if ((rr == 0 || rr == (uint32_t)R + 1) && ky[sl] > my) {
                            best = false;
                            break;
                        }
                    }
                }
            }
            if (best) {
                round[gid] = (uint32_t)R + 1;
                pick[gid] = my;
                uint32_t* cv = cover + (size_t)b * N;
                for (int32_t dz = -rad; dz <= rad; ++dz) {
                    int32_t zz = z + dz;
                    if (zz < 0 || zz >= g.D[2]) continue;
                    for (int32_t dy = -rad; dy <= rad; ++dy) {
                        int32_t yy = y + dy;
                        if (yy < 0 || yy >= g.D[1]) continue;
                        for (int32_t dx = -rad; dx <= rad; ++dx) {
                            int32_t xx = x + dx;
                            if (xx < 0 || xx >= g.D[0]) continue;
                            uint32_t nl = (uint32_t)xx + (uint32_t)g.D[0] * ((uint32_t)yy + (uint32_t)g.D[1] * (uint32_t)zz);
                            int32_t sl = slot_of(bm, wr, nl);
                            if (sl >= 0) atomicAdd(&cv[sl], 1u);
                        }
                    }
                }
            }
        }
    }
    const int32_t b0 = __shfl(b, 0, kWave), b1 = __shfl(b, kWave - 1, kWave);
    if (b0 == b1) {
        uint32_t tot = wave_sum<uint32_t>(above);
        if (lane_id() == 0 && tot) atomicAdd(&ctl.count[(R & 1) * B + b], tot);
    } else if (above) {
        atomicAdd(&ctl.count[(R & 1) * B + b], above);
    }
}

}  // namespace

hipError_t launch_select(const Layout& L, void* ws, int32_t M, int key_mode, uint64_t seed,
                         int32_t* center_lin, int32_t* m_valid, hipStream_t s) {
    k_select<<<L.B, kSelThreads, 0, s>>>(L.N, at<int32_t>(ws, L.nvox), at<uint32_t>(ws, L.vox_lin), M, key_mode,
                                         seed, key_mode ? at<uint64_t>(ws, L.cas_pick) : nullptr, center_lin,
                                         m_valid);
    return hipGetLastError();
}

hipError_t run_cas(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, uint32_t beta_q16,
                   hipStream_t s, int* status_out) {
    *status_out = CAGQ_OK;
    const int32_t B = L.B, N = L.N, BN = B * N;
    const int pb = (BN + 255) / 256;
    CasPtrs ctl = cas_ptrs(L, ws);
    GridDims g;
    for (int a = 0; a < 3; ++a) g.D[a] = d.dims[a];
    const int32_t rad = d.radius;
    const int64_t side = 2 * rad + 1;
    const int64_t lam = side * side * side;
    k_cas_init<<<pb, 256, 0, s>>>(BN, B, at<uint32_t>(ws, L.cas_cover), at<uint64_t>(ws, L.cas_pick),
                                  at<uint32_t>(ws, L.cas_round), ctl);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // every round picks at least the best unpicked voxel, so min(M, N) + 2
    // rounds always suffice (the last one only records that the cloud is done)
    const int64_t max_rounds = (int64_t)(M < N ? M : N) + 2;
    uint32_t done_h[64];
    const int check_every = 8;
    int64_t R = 0;
    bool all_done = false;
    while (!all_done) {
        for (int i = 0; i < check_every; ++i, ++R) {
            k_cas_score<<<pb, 256, 0, s>>>((int32_t)R, B, N, L.W, g, rad, lam, beta_q16, M,
                                           at<int32_t>(ws, L.nvox), at<uint32_t>(ws, L.vox_lin),
                                           at<uint64_t>(ws, L.bitmap), at<uint32_t>(ws, L.word_rank),
                                           at<uint32_t>(ws, L.cas_cover), at<uint64_t>(ws, L.cas_pick),
                                           at<uint64_t>(ws, L.cas_key), ctl);
            k_cas_pick<<<pb, 256, 0, s>>>((int32_t)R, B, N, L.W, g, rad, at<int32_t>(ws, L.nvox),
                                          at<uint32_t>(ws, L.vox_lin), at<uint64_t>(ws, L.bitmap),
                                          at<uint32_t>(ws, L.word_rank), at<uint32_t>(ws, L.cas_cover),
                                          at<uint64_t>(ws, L.cas_pick), at<uint32_t>(ws, L.cas_round),
                                          at<uint64_t>(ws, L.cas_key), ctl);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        all_done = true;
        for (int32_t b0 = 0; b0 < B && all_done; b0 += 64) {
            int32_t nb = B - b0 < 64 ? B - b0 : 64;
            e = hipMemcpyAsync(done_h, ctl.done + b0, sizeof(uint32_t) * nb, hipMemcpyDeviceToHost, s);
            if (e != hipSuccess) return e;
            e = hipStreamSynchronize(s);
            if (e != hipSuccess) return e;
            for (int32_t i = 0; i < nb; ++i) all_done = all_done && done_h[i] != 0;
        }
        if (!all_done && R > max_rounds) {
            *status_out = CAGQ_ERR_CAPACITY;
            return hipSuccess;
        }
    }
    return hipSuccess;
}

}  // namespace cagq
