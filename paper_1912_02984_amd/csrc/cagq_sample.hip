// Center voxel sampling (Sec. 3.2 "center voxels sampling"; Appendix D,
// general procedure, step 2).
//
// RVS: every occupied voxel is equally likely. Slot s of cloud b gets the
// key (hi32(h(seed, 1, b, s)) << 32) | s with h the splitmix64 chain; the
// m = min(M, |O_v|) smallest keys win. The low half of every select key (the
// slot, or the linear id for CAS) rises with the slot, so the m smallest
// keys are those whose top half is below a bound T, plus the first `need`
// slots whose top half equals T. A radix select over the top halves finds T
// and `need` (one workgroup per cloud in LDS, or one histogram kernel per
// digit for large clouds); a look-back compaction over the slots, counting
// keys below T and keys equal to T, then writes the winners in slot (=
// ascending linear id) order.
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
//
// With neighbour lists (r = 1, clouds above the single-workgroup size) a
// round is one kernel: each pick lowers the keys its coverage changes, so
// no voxel is rescored (k_cas_round). Without lists a round is a scoring
// kernel that recomputes the keys near the last picks from the occupancy
// rows and a picking kernel (k_cas_score, k_cas_pick).
#include <algorithm>
#include <chrono>

#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kSelThreads = 1024;
constexpr int32_t kSelManyBlockMin = 16384;  // clouds of this many points use the many-block select (measured: below it one workgroup per cloud is faster)

struct CasPtrs {
    uint64_t* gpart;  // [kCasBufs][B][kCasParts] partial maxima of the unpicked keys, per round buffer
    uint32_t* cpart;  // [kCasBufs][B][kCasParts] partial counts of picks above a maximum
    uint32_t* done;   // [B]
    uint32_t* ndone;  // clouds done
    uint32_t* uhist;  // [B][kCasParts][kCasUBins] picks per uncovered count U (lists, beta = 0)
    uint64_t* host;       // pinned host words (or null), each tagged with the call's epoch in
                          // the top half: [0] = (epoch, 1) once every cloud is done,
                          // [1] = (epoch, the round being run: all earlier rounds have finished)
    uint64_t epoch;       // this call's tag, shifted into the top half
};

CasPtrs cas_ptrs(const Layout& L, void* ws) {
    char* base = static_cast<char*>(ws) + L.cas_ctl;
    const size_t parts = (size_t)kCasBufs * L.B * kCasParts;
    CasPtrs c;
    c.gpart = reinterpret_cast<uint64_t*>(base);
    c.cpart = reinterpret_cast<uint32_t*>(base + parts * 8);
    c.done = reinterpret_cast<uint32_t*>(base + parts * 12);
    c.ndone = c.done + L.B;
    c.uhist = c.ndone + 1;
    c.host = nullptr;
    c.epoch = 0;
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

// Per-cloud selection result: top halves below `bound` (<= 2^32) are
// chosen, and of those equal to `bound` the first `need` in slot order.
__device__ __forceinline__ uint64_t sel_pack(uint64_t bound, uint32_t need) {
    return ((uint64_t)need << 33) | bound;
}

// One workgroup per cloud: the bound and tie count of the m = min(M, |O_v|)
// smallest keys by an 8-bit radix select over their top halves. Unpicked CAS
// voxels (key ~0) are never among the m smallest and are not counted. Also
// clears the scan state of the compaction that follows.
__global__ __launch_bounds__(kSelThreads) void k_sel_threshold(
    int32_t N, int64_t tiles_s, const int32_t* __restrict__ nvox, int32_t M, int key_mode, uint64_t seed,
    const uint64_t* __restrict__ cas_pick, uint64_t* __restrict__ thr, int32_t* __restrict__ m_valid,
    uint64_t* __restrict__ desc_s, int* __restrict__ status) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_digit, s_below, s_cnt;
    constexpr int U = 4;  // keys per thread per sweep, loaded together
    const int32_t b = blockIdx.x;
    const int32_t nv = nvox[b];
    const int32_t m = M < nv ? M : nv;
    const uint64_t hb = sm64(sm64(seed ^ 1ull) ^ (uint64_t)b);
    const uint64_t* pick = cas_pick ? cas_pick + (size_t)b * N : nullptr;
    const int tid = threadIdx.x;
    const int lane = lane_id();
    for (int64_t t = tid; t < tiles_s; t += kSelThreads) desc_s[(size_t)b * tiles_s + t] = 0;
    if (b == 0 && tid == 0) status[kStTicketSel] = 0;

    uint64_t prefix = 0, mask = 0, bound = 0;
    uint32_t need = (uint32_t)m;
    bool exact = true;
    for (int shift = 56; shift >= 32; shift -= 8) {
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        for (int32_t s0 = 0; s0 < nv; s0 += kSelThreads * U) {
            uint64_t k[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t s = s0 + u * kSelThreads + tid;
                k[u] = s < nv ? select_key(key_mode, hb, s, pick) : 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t s = s0 + u * kSelThreads + tid;
                const bool act = s < nv && (k[u] & mask) == prefix && (key_mode == 0 || k[u] != ~0ull);
                const uint32_t d = (uint32_t)(k[u] >> shift) & 255u;
                // one atomic for the wave when all its counted keys share a digit
                const uint64_t am = __ballot(act);
                if (am) {
                    const int leader = __ffsll((unsigned long long)am) - 1;
                    const uint32_t d0 = (uint32_t)__shfl((int)d, leader, kWave);
                    if (__ballot(act && d == d0) == am) {
                        if (lane == leader) atomicAdd(&hist[d0], (uint32_t)__popcll(am));
                    } else if (act) {
                        atomicAdd(&hist[d], 1u);
                    }
                }
            }
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
            const uint32_t incl = wave_incl_scan<uint32_t>(sum);
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
            bound = ((prefix | ~mask) >> 32) + 1;
            need = 0;
            exact = false;
            break;
        }
    }
    if (exact) bound = prefix >> 32;
    if (tid == 0) {
        thr[b] = sel_pack(bound, need);
        m_valid[b] = m;
    }
}

// Bound and tie count of the m largest CAS pick keys from the picks' U
// (beta = 0: a pick key is (unit * U + 2^31, ~lin), so the m largest are the
// picks with U > U* and, of those with U = U*, the lowest slots, U* being the
// largest U with at least m picks at or above it), as the select key's
// packed bound (the select key is the pick key's complement). Cloud b's
// kCasParts partial histograms are summed by 8 threads per bin, 16 partials
// each, loaded together; the result goes to *out. Every thread of a
// kScanThreads block calls it.
__device__ __forceinline__ void cas_u_bound(const uint32_t* __restrict__ uhist, int32_t b, uint32_t m, int64_t unit,
                                            uint32_t* s_h, uint64_t* out) {
    constexpr int kPer = kCasParts / 8;
    static_assert(8 * kCasUBins <= kScanThreads && kCasParts % 8 == 0, "8 threads per bin");
    const int tid = threadIdx.x;
    if (tid < kCasUBins) s_h[tid] = 0;
    __syncthreads();
    if (tid < 8 * kCasUBins) {
        const int bin = tid % kCasUBins, g = tid / kCasUBins;
        const uint32_t* h0 = uhist + ((size_t)b * kCasParts + (size_t)g * kPer) * kCasUBins + bin;
        uint32_t x[kPer], h = 0;
#pragma unroll
        for (int i = 0; i < kPer; ++i) x[i] = h0[(size_t)i * kCasUBins];
#pragma unroll
        for (int i = 0; i < kPer; ++i) h += x[i];
        if (h) atomicAdd(&s_h[bin], h);
    }
    __syncthreads();
    // the first wave: lane l holds U = kCasUBins - 1 - l (from the top), an
    // inclusive scan of the counts, and the first lane whose running count
    // reaches m gives U* and the ties taken there (no picks at all: 0, 0)
    static_assert(kCasUBins <= kWave, "one bin per lane");
    if (tid < kWave) {
        const int u = kCasUBins - 1 - tid;
        const uint32_t hu = tid < kCasUBins ? s_h[u] : 0u;
        const uint32_t incl = wave_incl_sum_u32(hu);
        const uint64_t hit = __ballot(m > 0 && tid < kCasUBins && incl >= m);
        if (!hit) {
            if (tid == 0) *out = sel_pack(0, 0);
        } else if (tid == __ffsll((unsigned long long)hit) - 1) {
            const uint64_t bound = 0xFFFFFFFFull - (uint64_t)(unit * u + 2147483648ll);
            *out = sel_pack(bound, m - (incl - hu));
        }
    }
}

// Ordered compaction of the chosen slots: tile of kScanTile slots per block,
// look-back scan over the packed pair (keys below the bound << 31 | keys at
// the bound). Slot s chosen at position p < m writes its linear id to every
// j = p, p + m, p + 2m, ... < M (the cyclic padding). The bound comes from
// thr, or with `uhist` (CAS on lists, beta = 0) from the picks' U histogram,
// when the first tile of each cloud also writes thr and m_valid.
__global__ __launch_bounds__(kScanThreads) void k_sel_emit(
    int32_t N, int64_t tiles_s, const int32_t* __restrict__ nvox, const uint32_t* __restrict__ vox_lin,
    int32_t M, int key_mode, uint64_t seed, const uint64_t* __restrict__ cas_pick,
    uint64_t* __restrict__ thr, int32_t* __restrict__ center_lin, uint64_t* __restrict__ desc_s,
    int* __restrict__ status, const uint32_t* __restrict__ uhist, int64_t unit, int32_t* __restrict__ m_valid) {
    __shared__ uint32_t s_ticket;
    __shared__ uint64_t s_wave[kScanThreads / kWave];
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_h[kCasUBins];
    __shared__ uint64_t s_thr;
    if (threadIdx.x == 0) s_ticket = atomicAdd((unsigned*)&status[kStTicketSel], 1u);
    __syncthreads();
    const uint32_t t = s_ticket;
    const int32_t b = (int32_t)(t / tiles_s);
    const int64_t tile = (int64_t)(t % tiles_s);
    const int32_t s0 = (int32_t)(tile * kScanTile) + (int32_t)threadIdx.x * kScanItems;
    // the slots' picks and linear ids are loaded at once, beside the bound's
    // inputs (from indices clamped into the cloud's row; used below nv only)
    uint64_t pk[kScanItems];
    uint32_t ln[kScanItems];
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const size_t at = (size_t)b * N + (size_t)(s0 + i < N ? s0 + i : N - 1);
        pk[i] = cas_pick ? cas_pick[at] : 0ull;
        ln[i] = vox_lin[at];
    }
    const int32_t nv = nvox[b];
    const int32_t m = M < nv ? M : nv;
    if (uhist && tile == 0 && threadIdx.x == 0 && m <= 0) {
        thr[b] = sel_pack(0, 0);
        m_valid[b] = 0;
    }
    if (tile * kScanTile >= nv) return;  // later tiles never wait on this one
    uint64_t packed;
    if (uhist) {
        cas_u_bound(uhist, b, (uint32_t)m, unit, s_h, &s_thr);
        __syncthreads();
        packed = s_thr;
        if (tile == 0 && threadIdx.x == 0) {
            thr[b] = packed;
            m_valid[b] = m;
        }
    } else {
        packed = thr[b];
    }
    const uint64_t bound = packed & ((1ull << 33) - 1);
    const uint32_t need = (uint32_t)(packed >> 33);
    const uint64_t hb = sm64(sm64(seed ^ 1ull) ^ (uint64_t)b);
    bool lt[kScanItems], eq[kScanItems];
    uint64_t cnt = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int32_t s = s0 + i;
        const uint64_t k = s < nv ? (key_mode == 0 ? select_key(0, hb, s, nullptr) : ~pk[i]) : ~0ull;
        const uint64_t top = k >> 32;
        const bool counted = s < nv && (key_mode == 0 || k != ~0ull);
        lt[i] = counted && top < bound;
        eq[i] = counted && top == bound;
        cnt += lt[i] ? (1ull << 31) : (eq[i] ? 1ull : 0ull);
    }
    uint64_t total;
    const uint64_t excl = block_excl_scan(cnt, s_wave, &total);
    uint64_t before = tile_lookback(desc_s + (size_t)b * tiles_s, tile, total, &s_prefix) + excl;
    int32_t* out = center_lin + (size_t)b * M;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const uint32_t nlt = (uint32_t)(before >> 31), neq = (uint32_t)(before & 0x7FFFFFFFull);
        if (lt[i] || (eq[i] && neq < need)) {
            const uint32_t pos = nlt + (neq < need ? neq : need);
            if (pos < (uint32_t)m) {
                const int32_t l = (int32_t)ln[i];
                for (int64_t j = (int64_t)pos; j < M; j += m) out[j] = l;
            }
        }
        before += lt[i] ? (1ull << 31) : (eq[i] ? 1ull : 0ull);
    }
}

// ---- many-block selection (large clouds): two launches.
// k_sel_pick splits each cloud's slots into chunks of kPickSlots. Per chunk
// it computes the select keys, counts the top 11 bits of their top halves
// into the cloud's histogram and, in LDS, counting-sorts the top halves by
// those 11 bits: the sorted chunk and the end of each bin go to memory. The
// last block of each cloud to finish (by a ticket) reads the histogram,
// finds the digit whose cumulative count reaches m,
// gathers the keys of that digit from every chunk's bin and resolves them
// exactly by a radix select over their next 11 and 10 bits (in LDS when
// they fit, else reading them again per digit). It then writes each chunk's
// first output position and share of the ties at the bound, and leaves the
// histogram and the ticket at zero for the next selection (the build zeroes
// them first).
// k_sel_emit_chunks then writes every chunk's chosen slots in slot order.
constexpr int kPickThreads = 1024;
constexpr int kPickItems = 4;
constexpr int kPickSlots = kPickThreads * kPickItems;  // slots per chunk (kSelChunk)
constexpr int kPickBlocks = 1024;                       // at most this many blocks per cloud
constexpr int kCandCap = 4096;                          // candidate keys held in LDS
static_assert(kPickSlots == kSelChunk && kCandCap <= kPickSlots && 2 * kPickThreads == kSelBins, "select sizes");

// Exclusive scan of one value per thread of a kPickThreads block.
__device__ __forceinline__ uint32_t pick_excl_scan(uint32_t v, uint32_t* s_wave, uint32_t* total) {
    const uint32_t incl = wave_incl_scan<uint32_t>(v);
    const int wv = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wave[wv] = incl;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kPickThreads / kWave; ++i) {
        const uint32_t x = s_wave[i];
        off += i < wv ? x : 0u;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return off + incl - v;
}

// Over the histogram h of `bins` (1024 or 2048) bins in LDS: the bin where
// the cumulative count first reaches `need`, the count before it and its
// own count, returned to every thread (out[] keeps its previous content
// when the total is below `need`). Every thread of the block calls it.
__device__ __forceinline__ void pick_find(const uint32_t* h, int bins, uint32_t need, uint32_t* s_find,
                                          uint32_t* s_wave, uint32_t (&out)[3]) {
    const int per = bins / kPickThreads;
    const int tid = threadIdx.x;
    const uint32_t v0 = h[tid * per], v1 = per > 1 ? h[tid * per + 1] : 0u;
    uint32_t tot;
    uint32_t run = pick_excl_scan(v0 + v1, s_wave, &tot);
    if (run < need && run + v0 >= need) {
        s_find[0] = (uint32_t)(tid * per);
        s_find[1] = run;
        s_find[2] = v0;
    }
    run += v0;
    if (per > 1 && run < need && run + v1 >= need) {
        s_find[0] = (uint32_t)(tid * per + 1);
        s_find[1] = run;
        s_find[2] = v1;
    }
    __syncthreads();
    if (tot >= need) {
        out[0] = s_find[0];
        out[1] = s_find[1];
        out[2] = s_find[2];
    }
    __syncthreads();
}

__global__ __launch_bounds__(kPickThreads) void k_sel_pick(
    int32_t N, const int32_t* __restrict__ nvox, int32_t M, int key_mode, uint64_t seed,
    const uint64_t* __restrict__ cas_pick, uint32_t* __restrict__ sorted, uint32_t* __restrict__ bin_end,
    uint32_t* __restrict__ ghist, uint32_t* __restrict__ gcnt, uint64_t* __restrict__ thr,
    int32_t* __restrict__ m_valid, uint32_t* __restrict__ sel_base, uint32_t* __restrict__ sel_take) {
    __shared__ uint32_t lh[kSelBins];     // histogram, then the bins' cursors
    __shared__ uint32_t sk[kPickSlots];   // the chunk's sorted top halves; later the candidates
    __shared__ uint32_t sp[kPickThreads]; // the last block: candidates before each chunk of a group
    __shared__ uint32_t ss[kPickThreads]; //                 and where its bin starts
    __shared__ uint32_t s_wave[kPickThreads / kWave];
    __shared__ uint32_t s_find[3];
    __shared__ uint32_t s_last;
    const int32_t b = blockIdx.y;
    const int32_t nblk = gridDim.x;
    const int tid = threadIdx.x;
    const int32_t nv = nvox[b];
    const uint32_t m = (uint32_t)(M < nv ? M : nv);
    const int32_t nchunk = (N + kPickSlots - 1) / kPickSlots;
    uint32_t* srt = sorted + (size_t)b * nchunk * kPickSlots;
    uint32_t* be = bin_end + (size_t)b * nchunk * kSelBins;
    // an unpicked CAS voxel (key ~0) is never chosen and is not counted: its
    // top half 2^32-1 is no picked key's
    auto counted = [&](uint32_t top) { return key_mode == 0 || top != 0xFFFFFFFFu; };
    const uint64_t hb = sm64(sm64(seed ^ 1ull) ^ (uint64_t)b);
    const uint64_t* pick = cas_pick ? cas_pick + (size_t)b * N : nullptr;
    for (int32_t c = blockIdx.x; c < nchunk; c += nblk) {
        for (int i = tid; i < kSelBins; i += kPickThreads) lh[i] = 0;
        __syncthreads();
        uint32_t top[kPickItems];
        bool cnt_it[kPickItems];
#pragma unroll
        for (int u = 0; u < kPickItems; ++u) {
            const int32_t sl = c * kPickSlots + u * kPickThreads + tid;
            top[u] = sl < nv ? (uint32_t)(select_key(key_mode, hb, sl, pick) >> 32) : 0u;
            cnt_it[u] = sl < nv && counted(top[u]);
            if (cnt_it[u]) atomicAdd(&lh[top[u] >> 21], 1u);
        }
        __syncthreads();
        // the cloud's histogram, and this chunk's bins: ends in memory,
        // starts as cursors in LDS
        const uint32_t h0 = lh[2 * tid], h1 = lh[2 * tid + 1];
        if (h0) atomicAdd(&ghist[(size_t)b * kSelBins + 2 * tid], h0);
        if (h1) atomicAdd(&ghist[(size_t)b * kSelBins + 2 * tid + 1], h1);
        uint32_t tot;
        const uint32_t ex = pick_excl_scan(h0 + h1, s_wave, &tot);
        be[(size_t)c * kSelBins + 2 * tid] = ex + h0;
        be[(size_t)c * kSelBins + 2 * tid + 1] = ex + h0 + h1;
        lh[2 * tid] = ex;
        lh[2 * tid + 1] = ex + h0;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kPickItems; ++u)
            if (cnt_it[u]) sk[atomicAdd(&lh[top[u] >> 21], 1u)] = top[u];
        __syncthreads();
        for (uint32_t i = tid; i < tot; i += kPickThreads) srt[(size_t)c * kPickSlots + i] = sk[i];
        __syncthreads();
    }
    // publish, then the last block of the cloud takes over. The barrier
    // orders every wave's stores before thread 0's agent-scope fence (one
    // L2 write-back per block, not per wave); the last block's fence, again
    // by one thread before a barrier, makes the other blocks' stores visible
    // to all its waves (they share the CU's caches)
    __syncthreads();
    if (tid == 0) {
        __threadfence();
        s_last = atomicAdd(&gcnt[b], 1u) == (uint32_t)(nblk - 1) ? 1u : 0u;
        if (s_last) __threadfence();
    }
    __syncthreads();
    if (!s_last) return;
    for (int i = tid; i < kSelBins; i += kPickThreads)
        lh[i] = __hip_atomic_load(&ghist[(size_t)b * kSelBins + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    uint32_t f[3] = {kSelBins - 1, 0u, 0u};
    pick_find(lh, kSelBins, m, s_find, s_wave, f);
    const uint32_t dig = f[0];
    uint32_t prefix = dig << 21, pmask = 0xFFE00000u;
    uint32_t need = m - f[1];
    const uint32_t cnt = f[2];
    uint64_t bound = 0;
    bool done = false;
    if (cnt == need) {  // every key under this prefix is among the m smallest
        bound = (uint64_t)(prefix | ~pmask) + 1;
        need = 0;
        done = true;
    }
    // Calls visit(i, key) for the keys of bin `dig` of every chunk, i
    // counting them from 0: chunks 1024 at a time, their bins' counts
    // scanned, each key found by a binary search over the scan.
    auto gather = [&](auto visit) {
        uint32_t base = 0;
        for (int32_t c0 = 0; c0 < nchunk; c0 += kPickThreads) {
            const int32_t c = c0 + tid;
            uint32_t st = 0, n = 0;
            if (c < nchunk) {
                const uint32_t* e = be + (size_t)c * kSelBins;
                st = dig ? e[dig - 1] : 0u;
                n = e[dig] - st;
            }
            uint32_t tot;
            const uint32_t pre = pick_excl_scan(n, s_wave, &tot);
            sp[tid] = pre;
            ss[tid] = (uint32_t)c * kPickSlots + st;
            __syncthreads();
            const int32_t nc = nchunk - c0 < kPickThreads ? nchunk - c0 : kPickThreads;
            for (uint32_t i = tid; i < tot; i += kPickThreads) {
                int32_t lo = 0, hi = nc - 1;
                while (lo < hi) {
                    const int32_t mid = (lo + hi + 1) >> 1;
                    if (sp[mid] <= i) lo = mid; else hi = mid - 1;
                }
                visit(base + i, srt[ss[lo] + (i - sp[lo])]);
            }
            base += tot;
            __syncthreads();
        }
    };
    // the keys of the digit into LDS when they fit, in chunk order (with at
    // most 1024 chunks the scan of the last group stays in LDS too)
    const bool in_lds = cnt <= (uint32_t)kCandCap;
    if (in_lds) {
        gather([&](uint32_t i, uint32_t key) {
            if (i < (uint32_t)kCandCap) sk[i] = key;  // exactly cnt of them
        });
        __syncthreads();
    }
    // digits of bits 10..20 and 0..9 among the keys under the prefix
    for (int q = 0; q < 2 && !done; ++q) {
        const int shift = q == 0 ? 10 : 0, width = q == 0 ? 11 : 10;
        const uint32_t dmask = (1u << width) - 1;
        for (int i = tid; i < kSelBins; i += kPickThreads) lh[i] = 0;
        __syncthreads();
        auto count = [&](uint32_t, uint32_t key) {
            if ((key & pmask) == prefix) atomicAdd(&lh[(key >> shift) & dmask], 1u);
        };
        if (in_lds) {
            for (uint32_t i = tid; i < cnt; i += kPickThreads) count(i, sk[i]);
        } else {  // too many for LDS: read them again
            gather(count);
        }
        __syncthreads();
        f[0] = dmask;
        f[1] = 0;
        f[2] = 0;
        pick_find(lh, 1 << width, need, s_find, s_wave, f);
        prefix |= f[0] << shift;
        pmask |= dmask << shift;
        need -= f[1];
        if (f[2] == need) {
            bound = (uint64_t)(prefix | ~pmask) + 1;
            need = 0;
            done = true;
        }
    }
    if (!done) bound = prefix;  // every bit fixed: ties at the bound go by slot
    // Per chunk, in chunk order: the keys below the bound (its bins below
    // `dig`, and those of bin `dig` below the bound) and the ties at it, of
    // which the chunk takes what is left of `need`; the chunk's first output
    // position is the number chosen in the chunks before it.
    uint32_t run_eq = 0, run_base = 0;
    for (int32_t c0 = 0; c0 < nchunk; c0 += kPickThreads) {
        const int32_t c = c0 + tid;
        uint32_t lt = 0, eq = 0;
        if (in_lds && nchunk <= kPickThreads) {  // the chunk's start and keys from the gather, in LDS
            if (c < nchunk) {
                const uint32_t p0 = sp[c], p1 = c + 1 < nchunk ? sp[c + 1] : cnt;
                lt = ss[c] - (uint32_t)c * kPickSlots;
                for (uint32_t i = p0; i < p1; ++i) {
                    const uint32_t top = sk[i];
                    lt += (uint64_t)top < bound ? 1u : 0u;
                    eq += (uint64_t)top == bound ? 1u : 0u;
                }
            }
        } else if (c < nchunk) {
            const uint32_t* e = be + (size_t)c * kSelBins;
            const uint32_t st = dig ? e[dig - 1] : 0u, en = e[dig];
            lt = st;
            for (uint32_t i = st; i < en; ++i) {
                const uint32_t top = srt[(size_t)c * kPickSlots + i];
                lt += (uint64_t)top < bound ? 1u : 0u;
                eq += (uint64_t)top == bound ? 1u : 0u;
            }
        }
        uint32_t tot_eq, tot_ch;
        const uint32_t eq_pre = run_eq + pick_excl_scan(eq, s_wave, &tot_eq);
        const uint32_t take = need > eq_pre ? (need - eq_pre < eq ? need - eq_pre : eq) : 0u;
        const uint32_t base = run_base + pick_excl_scan(lt + take, s_wave, &tot_ch);
        if (c < nchunk) {
            sel_base[(size_t)b * nchunk + c] = base;
            sel_take[(size_t)b * nchunk + c] = take;
        }
        run_eq += tot_eq;
        run_base += tot_ch;
    }
    if (tid == 0) {
        thr[b] = sel_pack(bound, need);
        m_valid[b] = (int32_t)m;
        gcnt[b] = 0;
    }
    for (int i = tid; i < kSelBins; i += kPickThreads) ghist[(size_t)b * kSelBins + i] = 0;
}

// The chosen slots of one chunk (block (c, b)), in slot order: a slot is
// chosen when its key's top half is below the bound, or equal to it and
// among the first `take` such slots of the chunk. Its output position is the
// chunk's base plus the chosen slots before it in the chunk (one block scan
// of the packed counts below / at the bound); it writes its linear id there
// and at every m-th entry after it (the cyclic padding).
__global__ __launch_bounds__(kPickThreads) void k_sel_emit_chunks(
    int32_t N, const int32_t* __restrict__ nvox, const uint32_t* __restrict__ vox_lin, int32_t M, int key_mode,
    uint64_t seed, const uint64_t* __restrict__ cas_pick, const uint64_t* __restrict__ thr,
    const uint32_t* __restrict__ sel_base, const uint32_t* __restrict__ sel_take, int32_t* __restrict__ center_lin) {
    __shared__ uint32_t s_wave[kPickThreads / kWave];
    const int32_t c = blockIdx.x, b = blockIdx.y, nchunk = gridDim.x;
    const int32_t s0 = c * kPickSlots + (int32_t)threadIdx.x * kPickItems;
    // the slots' picks and linear ids are loaded at once, beside the bound
    // (from indices clamped into the cloud's row; used below nv only)
    uint64_t pk[kPickItems];
    uint32_t ln[kPickItems];
#pragma unroll
    for (int u = 0; u < kPickItems; ++u) {
        const size_t at = (size_t)b * N + (size_t)(s0 + u < N ? s0 + u : N - 1);
        pk[u] = cas_pick ? cas_pick[at] : 0ull;
        ln[u] = vox_lin[at];
    }
    const int32_t nv = nvox[b];
    const int32_t m = M < nv ? M : nv;
    const uint64_t bound = thr[b] & ((1ull << 33) - 1);
    const uint32_t base = sel_base[(size_t)b * nchunk + c], take = sel_take[(size_t)b * nchunk + c];
    const uint64_t hb = sm64(sm64(seed ^ 1ull) ^ (uint64_t)b);
    bool lt[kPickItems], eq[kPickItems];
    uint32_t packed = 0;
#pragma unroll
    for (int u = 0; u < kPickItems; ++u) {
        const int32_t sl = s0 + u;
        const uint64_t top = sl < nv ? (key_mode == 0 ? select_key(0, hb, sl, nullptr) : ~pk[u]) >> 32 : 0xFFFFFFFFull;
        const bool counted = sl < nv && (key_mode == 0 || top != 0xFFFFFFFFull);
        lt[u] = counted && top < bound;
        eq[u] = counted && top == bound;
        packed += lt[u] ? (1u << 16) : (eq[u] ? 1u : 0u);
    }
    uint32_t tot;
    uint32_t run = pick_excl_scan(packed, s_wave, &tot);
    int32_t* out = center_lin + (size_t)b * M;
#pragma unroll
    for (int u = 0; u < kPickItems; ++u) {
        const uint32_t nlt = run >> 16, neq = run & 0xFFFFu;
        if (lt[u] || (eq[u] && neq < take)) {
            const uint32_t pos = base + nlt + (neq < take ? neq : take);
            if (pos < (uint32_t)m) {
                const int32_t l = (int32_t)ln[u];
                for (int64_t j = (int64_t)pos; j < M; j += m) out[j] = l;
            }
        }
        run += lt[u] ? (1u << 16) : (eq[u] ? 1u : 0u);
    }
}

// Slot of bit j of a row, or `self` when bit j is clear (a harmless address).
__device__ __forceinline__ uint32_t row_slot_or(const GridRow& r, int j, uint32_t self) {
    return ((r.mask >> j) & 1u) ? r.first + (uint32_t)__popc(r.mask & ((1u << j) - 1)) : self;
}

__device__ __forceinline__ uint32_t row_slot(const GridRow& r, int j) {
    return r.first + (uint32_t)__popc(r.mask & ((1u << j) - 1));
}

// Component j (0..3) of a 16-byte group of u32 list entries.
__device__ __forceinline__ uint32_t u4(const uint4& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

// Reduction of the kCasParts partials of the cloud `b` of each lane. Every
// lane of the wave must call it.
__device__ __forceinline__ uint64_t parts_max(const uint64_t* __restrict__ part, int32_t b) {
    static_assert(kCasParts % kWave == 0, "partials per lane");
    const int32_t b0 = __shfl(b, 0, kWave), b1 = __shfl(b, kWave - 1, kWave);
    if (b0 == b1) {
        uint64_t v = 0;
#pragma unroll
        for (int i = 0; i < kCasParts / kWave; ++i) {
            const uint64_t o = part[(size_t)b0 * kCasParts + i * kWave + lane_id()];
            v = o > v ? o : v;
        }
        return wave_max_u64(v);
    }
    uint64_t v = 0;
    for (int i = 0; i < kCasParts; ++i) {
        uint64_t o = part[(size_t)b * kCasParts + i];
        v = o > v ? o : v;
    }
    return v;
}

__device__ __forceinline__ uint32_t parts_sum(const uint32_t* __restrict__ part, int32_t b) {
    const int32_t b0 = __shfl(b, 0, kWave), b1 = __shfl(b, kWave - 1, kWave);
    if (b0 == b1) {
        uint32_t v = 0;
#pragma unroll
        for (int i = 0; i < kCasParts / kWave; ++i) v += part[(size_t)b0 * kCasParts + i * kWave + lane_id()];
        return wave_sum_u32(v);
    }
    uint32_t v = 0;
    for (int i = 0; i < kCasParts; ++i) v += part[(size_t)b * kCasParts + i];
    return v;
}

// Partial slot a wave accumulates into.
__device__ __forceinline__ int part_slot() {
    return (int)((blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave) & (kCasParts - 1));
}

struct CasState {
    uint32_t* cover;    // centers whose neighbourhood holds the voxel (C_V)
    uint64_t* key;      // current key of an unpicked voxel
    uint64_t* pick;     // key at pick time, 0 = unpicked
    uint32_t* round;    // round that picked the voxel + 1, 0 = unpicked
    int32_t* blocker;   // a neighbour whose key beat the voxel's last time, -1 = none
    uint32_t* dirty;    // round whose scoring must recompute the voxel's key (row-scan rounds)
};

// Clears the state and the control block for the row-scan rounds (with
// lists, the neighbour-list kernel clears them and sets the round-0 keys).
__global__ void k_cas_init(int32_t BN, int32_t B, CasState st, CasPtrs ctl) {
    int32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    if (gid < BN) {
        st.cover[gid] = 0;
        st.pick[gid] = 0;
        st.round[gid] = 0;
        st.blocker[gid] = -1;
        st.dirty[gid] = 0;
    }
    if (gid < kCasBufs * B * kCasParts) {
        ctl.gpart[gid] = 0;
        ctl.cpart[gid] = 0;
    }
    if (gid < B) ctl.done[gid] = 0;
    if (gid < B * kCasParts * kCasUBins) ctl.uhist[gid] = 0;
    if (gid == 0) *ctl.ndone = 0;
}

// Round R, phase 1: the key of every unpicked voxel (recomputed in round 0
// and wherever a pick of round R-1 came within distance 2r) and their
// maximum per cloud. Also retires a cloud once round R-1 found enough picks
// above the best unpicked key.
template <int RAD>
__global__ __launch_bounds__(256) void k_cas_score(
    int32_t R, int32_t B, int32_t N, int64_t W, GridDims g, int64_t lam, uint32_t beta_q16, int32_t M,
    const int32_t* __restrict__ nvox, const uint32_t* __restrict__ vox_lin, const uint64_t* __restrict__ bitmap,
    const uint32_t* __restrict__ word_rank, CasState st, CasPtrs ctl) {
    // no early exit: every lane takes part in the wave reductions
    const int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    const bool in_range = gid < B * N;
    const int32_t b = in_range ? gid / N : B - 1, s = in_range ? gid - b * N : N;
    // the voxel's own state is loaded up front, together with the cloud's,
    // so that the chain of dependent loads stays short (from a valid index
    // for every lane: a load under the range test would be waited for alone)
    const size_t gc = in_range ? (size_t)gid : 0;
    const uint32_t rnd0_ = st.round[gc], dty0_ = st.dirty[gc], lin0_ = vox_lin[gc];
    const uint64_t key0_ = st.key[gc];
    const uint32_t rnd0 = in_range ? rnd0_ : 0u;
    const uint32_t dty0 = in_range ? dty0_ : 0u;
    const uint64_t key0 = in_range ? key0_ : 0ull;
    const uint32_t lin0 = in_range ? lin0_ : 0u;
    bool active = in_range && ctl.done[b] == 0;
    if (ctl.host && blockIdx.x == 0 && threadIdx.x == 0)  // progress for the host's round issue
        __hip_atomic_store(ctl.host + 1, ctl.epoch | (uint32_t)R, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const int32_t nv = nvox[b];
    const uint32_t prev = R > 0 ? parts_sum(ctl.cpart + (size_t)((R - 1) & 1) * B * kCasParts, b) : 0u;
    if (active && R > 0 && prev >= (uint32_t)(M < nv ? M : nv)) {
        if (s == 0) {
            ctl.done[b] = 1;
            // the last cloud to finish tells the host, without a copy on the stream
            if (atomicAdd(ctl.ndone, 1u) + 1 == (uint32_t)B && ctl.host)
                __hip_atomic_store(ctl.host, ctl.epoch | 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        active = false;
    }
    if (active)  // this round's pick counts start from zero
        for (int32_t i = s; i < kCasParts; i += N) ctl.cpart[((size_t)(R & 1) * B + b) * kCasParts + i] = 0;
    uint64_t k = 0;
    const uint32_t rnd = active && s < nv ? rnd0 : 0u;
    // a voxel picked in the previous round stops competing: its key becomes 0
    if (active && s < nv && rnd != 0 && rnd == (uint32_t)R) st.key[gid] = 0;
    if (active && s < nv && rnd == 0) {
        if (R == 0 || dty0 == (uint32_t)R) {
            const uint32_t* cv = st.cover + (size_t)b * N;
            const uint32_t lin = lin0;
            int64_t U = 0, cs = 0;
            const uint64_t* bm = bitmap + (size_t)b * W;
            const uint32_t* wr = word_rank + (size_t)b * W;
            int32_t x, y, z;
            decode_lin(lin, g, x, y, z);
            constexpr int S = 2 * RAD + 1;
            GridRow rows[S * S];
#pragma unroll
            for (int j = 0; j < S * S; ++j)
                rows[j] = load_row(bm, wr, g, x, y + j % S - RAD, z + j / S - RAD, RAD);
            // every coverage count of the window loaded at once, then masked
            uint32_t c[S * S * S];
#pragma unroll
            for (int j = 0; j < S * S; ++j)
#pragma unroll
                for (int q = 0; q < S; ++q) c[j * S + q] = cv[row_slot_or(rows[j], q, (uint32_t)s)];
#pragma unroll
            for (int j = 0; j < S * S; ++j)
#pragma unroll
                for (int q = 0; q < S; ++q) {
                    const bool occ = (rows[j].mask >> q) & 1u;
                    const uint32_t cc = occ ? c[j * S + q] : 0u;
                    U += (occ && cc == 0) ? 1 : 0;
                    cs += cc;
                }
            k = cas_key(65536ll * lam * U - (int64_t)beta_q16 * cs, lin);
            st.key[gid] = k;
        } else {
            k = key0;
        }
    }
    // per-cloud maximum into one of the partial slots
    uint64_t* gp = ctl.gpart + (size_t)(R & 1) * B * kCasParts;
    const int32_t b0 = __shfl(b, 0, kWave), b1 = __shfl(b, kWave - 1, kWave);
    if (b0 == b1) {
        const uint64_t mx = wave_max64(k);
        if (lane_id() == 0 && mx) atomicMax((unsigned long long*)&gp[(size_t)b * kCasParts + part_slot()], mx);
    } else if (k) {
        atomicMax((unsigned long long*)&gp[(size_t)b * kCasParts + part_slot()], k);
    }
}

// Round R, phase 2: a voxel whose key beats that of every voxel unpicked at
// the round's start within distance 2r is picked: the coverage counts of its
// neighbourhood rise by one and the voxels within 2r are marked for
// rescoring. A voxel first re-checks the neighbour that beat it last time
// and scans its 2r-neighbourhood, one z-plane at a time, only when that one
// no longer does. Also counts earlier picks whose key beats this round's
// best unpicked key.
template <int RAD>
__global__ __launch_bounds__(256) void k_cas_pick(
    int32_t R, int32_t B, int32_t N, int64_t W, GridDims g, const int32_t* __restrict__ nvox,
    const uint32_t* __restrict__ vox_lin, const uint64_t* __restrict__ bitmap,
    const uint32_t* __restrict__ word_rank, CasState st, CasPtrs ctl) {
    constexpr int H = 2 * RAD;      // half-width of the competition window
    constexpr int S2 = 2 * H + 1;
    // no early exit: every lane takes part in the wave-wide steps
    const int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    const bool in_range = gid < B * N;
    const int32_t b = in_range ? gid / N : B - 1, s = in_range ? gid - b * N : N;
    // the voxel's own state is loaded up front, together with the cloud's
    const uint64_t pk0 = in_range ? st.pick[gid] : 0ull;
    const uint64_t my0 = in_range ? st.key[gid] : 0ull;
    const int32_t bl0 = in_range ? st.blocker[gid] : -1;
    const bool active = in_range && ctl.done[b] == 0;
    const uint64_t G = parts_max(ctl.gpart + (size_t)(R & 1) * B * kCasParts, b);
    if (active)  // next round's maxima start from zero
        for (int32_t i = s; i < kCasParts; i += N) ctl.gpart[((size_t)((R + 1) & 1) * B + b) * kCasParts + i] = 0;
    const int32_t nv = nvox[b];
    const uint32_t cur = (uint32_t)R + 1;
    const size_t cb = (size_t)b * N;
    const uint64_t* bm = bitmap + (size_t)b * W;
    const uint32_t* wr = word_rank + (size_t)b * W;
    uint32_t above = 0;
    bool winner = false;
    int32_t x = 0, y = 0, z = 0;
    if (active && s < nv) {
        const uint64_t pk = pk0;
        if (pk != 0) {
            above = pk > G ? 1u : 0u;
        } else {
            // competitors are the voxels unpicked at the round's start: earlier
            // picks have key 0 (set by this round's scoring), this round's keep theirs
            const uint64_t* ky = st.key + cb;
            const uint64_t my = my0;
            const int32_t bl = bl0;
            const bool beaten = bl >= 0 && ky[bl] > my;
            if (!beaten) {
                int32_t found = -1;
                decode_lin(vox_lin[gid], g, x, y, z);
                // planes in the order dz = 0, -1, +1, -2, +2, ...; per plane all
                // row descriptors, then all keys are loaded before comparing (a
                // clear bit loads the voxel's own key, which never beats it)
                for (int p = 0; p < S2 && found < 0; ++p) {
                    const int32_t dz = (p & 1) ? -((p + 1) >> 1) : (p >> 1);
                    GridRow rows[S2];
#pragma unroll
                    for (int j = 0; j < S2; ++j) rows[j] = load_row(bm, wr, g, x, y + j - H, z + dz, H);
                    uint32_t sl[S2 * S2];
                    uint64_t kk[S2 * S2];
#pragma unroll
                    for (int i = 0; i < S2 * S2; ++i) sl[i] = row_slot_or(rows[i / S2], i % S2, (uint32_t)s);
#pragma unroll
                    for (int i = 0; i < S2 * S2; ++i) kk[i] = ky[sl[i]];
#pragma unroll
                    for (int i = 0; i < S2 * S2; ++i)
                        if (found < 0 && kk[i] > my) found = (int32_t)sl[i];
                }
                if (found >= 0) {
                    st.blocker[gid] = found;
                } else {
                    winner = true;
                    st.round[gid] = cur;
                    st.pick[gid] = my;
                }
            }
        }
    }
    // Marks of the winners: rescoring flags within 2r, coverage counts
    // within r. Winners of a round are more than 2r apart, so their
    // r-neighbourhoods are disjoint and no count is raised twice in a round:
    // plain read-modify-write is exact. The whole wave marks each winner's
    // window, one grid row per lane.
    uint64_t wins = __ballot(winner);
    while (wins) {
        const int wl = __ffsll((unsigned long long)wins) - 1;
        wins &= wins - 1;
        const int32_t wb = __shfl(b, wl, kWave);
        uint32_t* cv = st.cover + (size_t)wb * N;
        uint32_t* dt = st.dirty + (size_t)wb * N;
        {
            const int32_t wx = __shfl(x, wl, kWave), wy = __shfl(y, wl, kWave), wz = __shfl(z, wl, kWave);
            const uint64_t* wbm = bitmap + (size_t)wb * W;
            const uint32_t* wwr = word_rank + (size_t)wb * W;
            for (int j = lane_id(); j < S2 * S2; j += kWave) {
                const int dy = j % S2 - H, dz = j / S2 - H;
                const GridRow r = load_row(wbm, wwr, g, wx, wy + dy, wz + dz, H);
                const bool inner = dy >= -RAD && dy <= RAD && dz >= -RAD && dz <= RAD;
#pragma unroll
                for (int q = 0; q < S2; ++q) {
                    if ((r.mask >> q) & 1u) {
                        const uint32_t sl = row_slot(r, q);
                        dt[sl] = cur;
                        if (inner && q - H >= -RAD && q - H <= RAD) cv[sl] = cv[sl] + 1u;
                    }
                }
            }
        }
    }
    uint32_t* cp = ctl.cpart + (size_t)(R & 1) * B * kCasParts;
    const int32_t b0 = __shfl(b, 0, kWave), b1 = __shfl(b, kWave - 1, kWave);
    if (b0 == b1) {
        const uint32_t tot = wave_sum<uint32_t>(above);
        if (lane_id() == 0 && tot) atomicAdd(&cp[(size_t)b * kCasParts + part_slot()], tot);
    } else if (above) {
        atomicAdd(&cp[(size_t)b * kCasParts + part_slot()], above);
    }
}

// The lane of the wave that owns pair p0 + lane_id(), lane L owning the pairs
// [incl - n, incl) of its own incl and n (lanes in order, ranges possibly
// empty): a range that starts inside the window marks its start with L + 1
// in the wave's LDS row, an unsigned max-scan across the lanes (DPP) carries
// each mark forward, and the window's first pair goes to the first lane whose
// range ends past it (one ballot). One LDS round trip and six DPP steps, where
// a binary search over the lanes takes six dependent permutes. Every lane of
// the wave must call it; pairs at or past the wave's total get the last range.
__device__ __forceinline__ int window_owner(uint32_t incl, uint32_t n, uint32_t p0, uint32_t* s_mark) {
    const int lane = lane_id();
    s_mark[lane] = 0u;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint32_t st = incl - n;
    if (n != 0 && st >= p0 && st - p0 < (uint32_t)kWave) s_mark[st - p0] = (uint32_t)lane + 1u;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    uint32_t v = s_mark[lane];
    const uint64_t past = __ballot(incl > p0);
    const uint32_t first = past ? (uint32_t)__ffsll((unsigned long long)past) : (uint32_t)kWave;  // lane + 1
    if (lane == 0) v = v > first ? v : first;
    uint32_t o;
    o = dpp_row_shr<1>(v);
    v = o > v ? o : v;
    o = dpp_row_shr<2>(v);
    v = o > v ? o : v;
    o = dpp_row_shr<4>(v);
    v = o > v ? o : v;
    o = dpp_row_shr<8>(v);
    v = o > v ? o : v;
    o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
    v = o > v ? o : v;
    o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
    v = o > v ? o : v;
    return (int)v - 1;
}

// The first of entries 16c..16c+15 of a list of n2 entries (held in q) that
// is a competitor and whose key beats `my`, or -1. Positions past the list's
// end read the voxel's own slot `self`, whose key never beats its own.
__device__ __forceinline__ int32_t beats(const uint4 (&q)[4], uint32_t c, uint32_t n2, uint32_t self, uint64_t my,
                                         uint32_t cur, const uint64_t* __restrict__ ky,
                                         const uint32_t* __restrict__ rd) {
    uint32_t sl[16], rr[16];
    uint64_t kk[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) sl[j] = 16 * c + j < n2 ? u4(q[j / 4], j % 4) : self;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        kk[j] = ky[sl[j]];
        rr[j] = rd[sl[j]];
    }
    // every entry is tested, without short cuts (which the compiler turns
    // into loads issued one at a time), the first from the end to the front
    int32_t found = -1;
#pragma unroll
    for (int j = 15; j >= 0; --j) {
        const bool bt = (kk[j] > my) & ((rr[j] == 0u) | (rr[j] == cur));
        found = bt ? (int32_t)sl[j] : found;
    }
    return found;
}

// One round of CAS on neighbour lists (r = 1), in one kernel: the keys stay
// exact without rescoring. A winner raises the coverage count of every voxel
// u within r of it, and the score of every voxel v within r of such a u
// falls by beta_q16 (its coverage sum rose by one), and by 2^16 * lambda
// more when u was uncovered (v lost an uncovered neighbour): the winner
// subtracts that from v's key with an atomic add, so every key equals the
// score formula on the current counts once the round's kernel has ended.
//
// Keys fall while other lanes of the same round read them, which keeps the
// round exact:
// * a voxel's key is lowered only by winners within distance 2r of it;
// * two winners within 2r of each other cannot happen: of such pairs take
//   the winner z of largest key. Any winner near z read z's key below its
//   own, hence below z's, so a winner near z had lowered it before, after
//   reading it below its own key in turn, and so on backwards in time
//   through finitely many winners: a contradiction. So a winner's own key is
//   exact, and it keeps that key for the whole round (it is never lowered);
// * for a winner w and a voxel u within 2r of it, take the winner x near u
//   with key below w's that read u first. It read u lowered only by winners
//   with keys above w's, and still below its own key. So u's key, with every
//   winner above w applied, is below w's, and stays below: w is picked by
//   the sequential greedy, after those winners, with its very key.
// A voxel picked in an earlier round keeps its key in the array; competitors
// tell it apart by its pick round. The round's best unpicked key (read at the
// round's start) bounds every later pick, so round R counts the picks above
// round R-1's bound and round R+1 retires the cloud: the stopping rule of the
// two-kernel rounds, one round later.
constexpr int kRoundThreads = 64;  // one wave per block: the blocks spread over every CU
constexpr int kRoundEnt = 28;      // list entries a possible winner keeps in LDS
__global__ __launch_bounds__(kRoundThreads) __attribute__((amdgpu_waves_per_eu(5))) void k_cas_round(int32_t R, int32_t B, int32_t N, int64_t unit, uint32_t beta_q16,
                                                   int32_t M, const int32_t* __restrict__ nvox,
                                                   const uint32_t* __restrict__ nbr, CasState st, CasPtrs ctl) {
    // no early exit: every lane takes part in the wave-wide steps
    const int32_t gid = (int32_t)xcd_block(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    const bool in_range = gid < B * N;
    const int32_t b = in_range ? gid / N : B - 1, s = in_range ? gid - b * N : N;
    // Everything the round's first decisions need is loaded at once: the
    // voxel's own state, the cloud's done flag and size, and the previous
    // round's partials (no kernel of this round writes them), from valid
    // indices for every lane (a load under a test would be waited for
    // alone); then the blocker's key and pick round, together.
    const size_t gc = in_range ? (size_t)gid : 0;
    const uint32_t rnd0_ = st.round[gc];
    const uint64_t pk0_ = st.pick[gc], my0_ = st.key[gc];
    const int32_t bl0_ = st.blocker[gc];
    const uint32_t done0 = ctl.done[b];
    const int32_t nv = nvox[b];
    const size_t part = (size_t)B * kCasParts;
    const int32_t b0 = __builtin_amdgcn_readlane(b, 0), b1 = __builtin_amdgcn_readlane(b, kWave - 1);
    const bool one_cloud = b0 == b1;  // the wave's lanes all in one cloud: each lane reduces two partials
    static_assert(kCasParts == 2 * kWave, "two partials per lane");
    uint32_t cp0 = 0, cp1 = 0;
    uint64_t gp0 = 0, gp1 = 0;
    if (R > 0 && one_cloud) {
        const size_t pp = (size_t)((R - 1) % kCasBufs) * part + (size_t)b0 * kCasParts + lane_id();
        cp0 = ctl.cpart[pp];
        cp1 = ctl.cpart[pp + kWave];
        gp0 = ctl.gpart[pp];
        gp1 = ctl.gpart[pp + kWave];
    }
    const size_t cb = (size_t)b * N;
    const int32_t blc = bl0_ >= 0 && bl0_ < N ? bl0_ : 0;
    const uint64_t kb_ = st.key[cb + blc];
    const uint32_t rb_ = st.round[cb + blc];
    const uint32_t rnd0 = in_range ? rnd0_ : 0u;
    const uint64_t pk0 = in_range ? pk0_ : 0ull;
    const uint64_t my0 = in_range ? my0_ : 0ull;
    const int32_t bl0 = in_range ? bl0_ : -1;
    bool active = in_range && done0 == 0;
    if (ctl.host && blockIdx.x == 0 && threadIdx.x == 0)  // progress for the host's round issue
        __hip_atomic_store(ctl.host + 1, ctl.epoch | (uint32_t)R, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const uint32_t prev = R == 0 ? 0u
                          : one_cloud ? wave_sum_u32(cp0 + cp1)
                                      : parts_sum(ctl.cpart + (size_t)((R - 1) % kCasBufs) * part, b);
    if (active && prev >= (uint32_t)(M < nv ? M : nv)) {
        if (s == 0) {
            ctl.done[b] = 1;
            // the last cloud to finish tells the host, without a copy on the stream
            if (atomicAdd(ctl.ndone, 1u) + 1 == (uint32_t)B && ctl.host)
                __hip_atomic_store(ctl.host, ctl.epoch | 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        active = false;
    }
    if (active)  // the next round's partials start from zero
        for (int32_t i = s; i < kCasParts; i += N) {
            const size_t o = (size_t)((R + 1) % kCasBufs) * part + (size_t)b * kCasParts + i;
            ctl.gpart[o] = 0;
            ctl.cpart[o] = 0;
        }
    const uint64_t G = R == 0 ? ~0ull
                       : one_cloud ? wave_max_u64(gp0 > gp1 ? gp0 : gp1)
                                   : parts_max(ctl.gpart + (size_t)((R - 1) % kCasBufs) * part, b);
    const uint32_t cur = (uint32_t)R + 1;
    uint64_t k = 0;
    uint32_t above = 0;
    bool winner = false;
    // A voxel unpicked at the round's start is beaten when its blocker
    // still beats it, or else when an entry of its 2r-list does; the
    // competitors are the voxels unpicked at the round's start or picked in
    // this round (their keys stay in the array, their pick round tells them
    // apart). Each lane checks its blocker and its list's first 16 entries;
    // longer lists not yet decided are then scanned by the whole wave, one
    // (voxel, 16 entries) pair per lane, so that no lane walks a long list
    // alone.
    const uint64_t* ky = st.key + cb;
    const uint32_t* rd = st.round + cb;
    const uint4* el = reinterpret_cast<const uint4*>(nbr + (size_t)(in_range ? gid : 0) * kNbr32Stride);
    int32_t found = -2;  // -2: not competing, -1: no entry beats it so far
    uint32_t n2 = 0, n_r = 0;
    // a possible winner's list entries that can be within r (those come
    // first: at most 27), kept for the wave's coverage pass below
    __shared__ uint32_t s_ent[kRoundThreads][kRoundEnt];
    if (active && s < nv) {
        if (rnd0 != 0) {
            above = pk0 > G ? 1u : 0u;
        } else {
            k = my0;
            bool beaten = false;
            if (bl0 >= 0) beaten = kb_ > my0 && (rb_ == 0 || rb_ == cur);
            // the list (which does not fit in the caches) is read only by a
            // voxel its blocker no longer beats: after the first rounds most
            // voxels stay blocked
            if (!beaten) {
                const uint4 h = el[0];
                uint4 q[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) q[j] = el[1 + j];
                n2 = h.y;
                n_r = h.x;
                found = beats(q, 0, n2, (uint32_t)s, my0, cur, ky, rd);
                if (found == -1) {
                    uint4* se = reinterpret_cast<uint4*>(s_ent[threadIdx.x]);
#pragma unroll
                    for (int j = 0; j < 4; ++j) se[j] = q[j];
                }
            }
        }
    }
    const uint32_t nrest = found == -1 && n2 > 16 ? (n2 - 1) / 16 : 0u;  // chunks 1.. still to scan
    const uint32_t sincl = wave_incl_sum_u32(nrest);
    const uint32_t stot = (uint32_t)__builtin_amdgcn_readlane((int)sincl, kWave - 1);
    __shared__ uint32_t s_mark[kRoundThreads];  // window_owner's row (the block is one wave)
    if (stot) {
        __shared__ int32_t s_found[kRoundThreads];
        const int wbase = threadIdx.x & ~(kWave - 1);
        s_found[threadIdx.x] = -1;
        for (uint32_t p0 = 0; p0 < stot; p0 += kWave) {
            const uint32_t p = p0 + (uint32_t)lane_id();
            const int owner = window_owner(sincl, nrest, p0, s_mark);
            const uint32_t o_incl = (uint32_t)__shfl((int)sincl, owner, kWave);
            const uint32_t o_n = (uint32_t)__shfl((int)nrest, owner, kWave);
            const uint32_t o_n2 = (uint32_t)__shfl((int)n2, owner, kWave);
            const int32_t o_gid = __shfl(gid, owner, kWave);
            const int32_t o_b = __shfl(b, owner, kWave);
            const uint64_t o_my = shfl64(my0, owner);
            if (p < stot) {
                const uint32_t c = 1 + p - (o_incl - o_n);
                const size_t ob = (size_t)o_b * N;
                const uint4* e = reinterpret_cast<const uint4*>(nbr + (size_t)o_gid * kNbr32Stride);
                uint4 q[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) q[j] = e[1 + 4 * c + j];
                if (c == 1) {  // entries 16..27, which can be within r
                    uint4* se = reinterpret_cast<uint4*>(s_ent[wbase + owner] + 16);
#pragma unroll
                    for (int j = 0; j < 3; ++j) se[j] = q[j];
                }
                const int32_t f = beats(q, c, o_n2, (uint32_t)((size_t)o_gid - ob), o_my, cur, st.key + ob,
                                        st.round + ob);
                if (f >= 0) s_found[wbase + owner] = f;  // any beating entry will do
            }
        }
        if (nrest) found = s_found[threadIdx.x];
    }
    if (found >= 0) {
        st.blocker[gid] = found;
    } else if (found == -1) {
        winner = true;
        st.round[gid] = cur;
        st.pick[gid] = my0;
        if (beta_q16 == 0) {  // the score is unit * U: the pick's U, for the selection
            const uint32_t u = (uint32_t)(((int64_t)(my0 >> 32) - 2147483648ll) / unit);
            atomicAdd(&ctl.uhist[((size_t)b * kCasParts + part_slot()) * kCasUBins + u], 1u);
        }
    }
    // The winners' coverage counts and key updates, by the whole wave over
    // all (winner, u) pairs with u within r of the winner, 64 at a time (u
    // from the winner's entries in LDS). Winners are more than 2r apart, so no
    // count is raised twice in a round: a plain read-modify-write is exact.
    // A lane loads u's count and u's list within r together, and when u was
    // uncovered (or beta > 0) lowers the keys on that list.
    const uint32_t nrw = winner ? n_r : 0u;
    const uint32_t incl = wave_incl_sum_u32(nrw);
    const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1);
    const int wb = threadIdx.x & ~(kWave - 1);
    for (uint32_t p0 = 0; p0 < total; p0 += kWave) {
        const uint32_t p = p0 + (uint32_t)lane_id();
        const int owner = window_owner(incl, nrw, p0, s_mark);
        const uint32_t o_incl = (uint32_t)__shfl((int)incl, owner, kWave);
        const uint32_t o_nr = (uint32_t)__shfl((int)nrw, owner, kWave);
        const int32_t o_gid = __shfl(gid, owner, kWave);
        const int32_t o_b = __shfl(b, owner, kWave);
        if (p < total) {
            const uint32_t j = p - (o_incl - o_nr);
            const size_t ob = (size_t)o_b * N;
            const uint32_t u = s_ent[wb + owner][j];
            uint32_t* cv = st.cover + ob;
            const uint4* lu = reinterpret_cast<const uint4*>(nbr + (ob + u) * kNbr32Stride);
            uint4 lq[8];  // header and entries 0..27 (a list within r holds at most 27)
#pragma unroll
            for (int i = 0; i < 8; ++i) lq[i] = lu[i];
            const uint32_t c = cv[u];
            cv[u] = c + 1u;
            const int64_t d = (c == 0 ? unit : 0) + (int64_t)beta_q16;
            if (d != 0) {
                // the score field (the key's upper word) falls by d: a 32-bit
                // add to that word changes the key exactly as the 64-bit add
                // of -d << 32 would, and 64-bit loads of the key still see it
                // whole (the lower word never changes)
                const uint32_t dec = (uint32_t)(-d);
                uint32_t* kw = reinterpret_cast<uint32_t*>(st.key + ob) + 1;
                const uint32_t o_s = (uint32_t)((size_t)o_gid - ob);
                const uint32_t n_ru = lq[0].x;
#pragma unroll
                for (int i = 0; i < 28; ++i) {
                    const uint32_t v = u4(lq[1 + i / 4], i % 4);
                    if ((uint32_t)i < n_ru && v != o_s) atomicAdd(kw + 2 * (size_t)v, dec);
                }
            }
        }
    }
    // per-cloud maximum of the unpicked keys and count of picks above the
    // previous round's maximum, into this round's partial slots
    const size_t mine = (size_t)(R % kCasBufs) * part;
    if (one_cloud) {
        const uint64_t mx = wave_max_u64(k);
        const uint32_t tot = wave_sum_u32(above);
        if (lane_id() == 0 && mx) atomicMax((unsigned long long*)&ctl.gpart[mine + (size_t)b * kCasParts + part_slot()], mx);
        if (lane_id() == 0 && tot) atomicAdd(&ctl.cpart[mine + (size_t)b * kCasParts + part_slot()], tot);
    } else {
        if (k) atomicMax((unsigned long long*)&ctl.gpart[mine + (size_t)b * kCasParts + part_slot()], k);
        if (above) atomicAdd(&ctl.cpart[mine + (size_t)b * kCasParts + part_slot()], above);
    }
}


// A small pinned host buffer per calling thread for polling the progress of
// the rounds without stalling the stream. Allocated on first use, kept for
// the life of the process. Every call takes a new epoch, and its kernels
// tag each word they write with it: a round still queued from an earlier
// call of the thread (whose words it may overwrite) is told apart and
// ignored.
struct PollBuffer {
    uint64_t* words;
    uint32_t epoch;
};

PollBuffer* poll_buffer() {
    thread_local PollBuffer pb{nullptr, 0u};
    if (!pb.words) {
        void* p = nullptr;
        if (hipHostMalloc(&p, 64, hipHostMallocDefault) != hipSuccess) return nullptr;
        pb.words = static_cast<uint64_t*>(p);
    }
    return &pb;
}

}  // namespace

hipError_t launch_select(const Layout& L, void* ws, int32_t M, int key_mode, uint64_t seed,
                         int32_t* center_lin, int32_t* m_valid, hipStream_t s) {
    const uint64_t* pick = key_mode ? at<uint64_t>(ws, L.cas_pick) : nullptr;
    const int32_t* nvox = at<int32_t>(ws, L.nvox);
    uint64_t* thr = at<uint64_t>(ws, L.sel_thr);
    uint64_t* desc_s = at<uint64_t>(ws, L.desc_s);
    int* status = at<int>(ws, L.status);
    if (L.N >= kSelManyBlockMin) {
        // large clouds: the keys and the bound over many blocks per cloud
        const int64_t nchunk = (L.N + kPickSlots - 1) / kPickSlots;
        const dim3 grid((unsigned)(nchunk < kPickBlocks ? nchunk : kPickBlocks), (unsigned)L.B);
        uint32_t* base = at<uint32_t>(ws, L.sel_base);
        uint32_t* take = at<uint32_t>(ws, L.sel_take);
        k_sel_pick<<<grid, kPickThreads, 0, s>>>(L.N, nvox, M, key_mode, seed, pick, at<uint32_t>(ws, L.sel_keys),
                                                 at<uint32_t>(ws, L.sel_bins), at<uint32_t>(ws, L.sel_ghist),
                                                 at<uint32_t>(ws, L.sel_cnt), thr, m_valid, base, take);
        k_sel_emit_chunks<<<dim3((unsigned)nchunk, (unsigned)L.B), kPickThreads, 0, s>>>(
            L.N, nvox, at<uint32_t>(ws, L.vox_lin), M, key_mode, seed, pick, thr, base, take, center_lin);
        return hipGetLastError();
    } else {
        k_sel_threshold<<<L.B, kSelThreads, 0, s>>>(L.N, L.tiles_s, nvox, M, key_mode, seed, pick, thr, m_valid,
                                                    desc_s, status);
    }
    k_sel_emit<<<(unsigned)(L.B * L.tiles_s), kScanThreads, 0, s>>>(L.N, L.tiles_s, nvox,
                                                                   at<uint32_t>(ws, L.vox_lin), M, key_mode, seed,
                                                                   pick, thr, center_lin, desc_s, status, nullptr, 0,
                                                                   nullptr);
    return hipGetLastError();
}

hipError_t launch_select_cas(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, uint32_t beta_q16,
                             int32_t* center_lin, int32_t* m_valid, hipStream_t s) {
    if (!(L.has_nbr32 && d.radius == 1 && beta_q16 == 0))
        return launch_select(L, ws, M, 1, 0, center_lin, m_valid, s);
    const CasPtrs ctl = cas_ptrs(L, ws);
    const int64_t side = 2 * (int64_t)d.radius + 1;
    uint64_t* thr = at<uint64_t>(ws, L.sel_thr);
    uint64_t* desc_s = at<uint64_t>(ws, L.desc_s);
    int* status = at<int>(ws, L.status);
    const int32_t* nvox = at<int32_t>(ws, L.nvox);
    // the neighbour-list kernel has cleared the compaction's scan state
    k_sel_emit<<<(unsigned)(L.B * L.tiles_s), kScanThreads, 0, s>>>(L.N, L.tiles_s, nvox,
                                                                   at<uint32_t>(ws, L.vox_lin), M, 1, 0,
                                                                   at<uint64_t>(ws, L.cas_pick), thr, center_lin,
                                                                   desc_s, status, ctl.uhist, 65536 * side * side * side,
                                                                   m_valid);
    return hipGetLastError();
}

hipError_t run_cas(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, uint32_t beta_q16,
                   hipStream_t s, int* status_out) {
    *status_out = CAGQ_OK;
    const int32_t B = L.B, N = L.N, BN = B * N;
    const int pb = (BN + 255) / 256;
    CasPtrs ctl = cas_ptrs(L, ws);
    CasState st;
    st.cover = at<uint32_t>(ws, L.cas_cover);
    st.key = at<uint64_t>(ws, L.cas_key);
    st.pick = at<uint64_t>(ws, L.cas_pick);
    st.round = at<uint32_t>(ws, L.cas_round);
    st.blocker = at<int32_t>(ws, L.cas_blocker);
    st.dirty = at<uint32_t>(ws, L.cas_dirty);
    GridDims g;
    for (int a = 0; a < 3; ++a) g.D[a] = d.dims[a];
    const int32_t rad = d.radius;
    if (rad != 1 && rad != 2) {
        *status_out = CAGQ_ERR_INVALID_ARG;
        return hipSuccess;
    }
    const int64_t side = 2 * rad + 1;
    const int64_t lam = side * side * side;
    const int32_t* nvox = at<int32_t>(ws, L.nvox);
    const uint32_t* vox_lin = at<uint32_t>(ws, L.vox_lin);
    const uint64_t* bitmap = at<uint64_t>(ws, L.bitmap);
    const uint32_t* word_rank = at<uint32_t>(ws, L.word_rank);
    hipError_t e = hipSuccess;
    // neighbour lists replace the row scans where the layout holds them, and
    // then a round is one kernel that keeps the keys exact by itself
    const bool lists = L.has_nbr32 && rad == 1;
    // with lists, the list kernel also sets the round-0 keys: nothing is
    // covered yet, so the score is 2^16 * lambda * (occupied voxels within r)
    // (and clears the rounds' state, which takes a launch of its own otherwise)
    const int32_t init_n = std::max(BN, B * kCasParts * kCasUBins);
    if (lists) {
        const CasClear clr{st.cover, st.pick, st.round, st.blocker, st.dirty, ctl.gpart, ctl.cpart, ctl.done,
                           ctl.ndone, ctl.uhist, kCasBufs * B * kCasParts, B * kCasParts * kCasUBins,
                           at<uint64_t>(ws, L.desc_s), (int32_t)(B * L.tiles_s), at<int>(ws, L.status) + kStTicketSel};
        if ((e = launch_cas_nbr(L, d, ws, s, st.key, 65536 * lam, &clr)) != hipSuccess) return e;
    } else {
        k_cas_init<<<(init_n + 63) / 64, 64, 0, s>>>(BN, B, st, ctl);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const uint32_t* nbr = lists ? at<uint32_t>(ws, L.cas_nbr32) : nullptr;

    int64_t R = 0;
    auto launch_batch = [&](int rounds) {
        for (int i = 0; i < rounds; ++i, ++R) {
            if (lists) {
                k_cas_round<<<(BN + kRoundThreads - 1) / kRoundThreads, kRoundThreads, 0, s>>>(
                    (int32_t)R, B, N, 65536 * lam, beta_q16, M, nvox, nbr, st, ctl);
            } else if (rad == 1) {
                k_cas_score<1><<<pb, 256, 0, s>>>((int32_t)R, B, N, L.W, g, lam, beta_q16, M, nvox,
                                                         vox_lin, bitmap, word_rank, st, ctl);
                k_cas_pick<1><<<pb, 256, 0, s>>>((int32_t)R, B, N, L.W, g, nvox, vox_lin, bitmap,
                                                        word_rank, st, ctl);
            } else {
                k_cas_score<2><<<pb, 256, 0, s>>>((int32_t)R, B, N, L.W, g, lam, beta_q16, M, nvox,
                                                         vox_lin, bitmap, word_rank, st, ctl);
                k_cas_pick<2><<<pb, 256, 0, s>>>((int32_t)R, B, N, L.W, g, nvox, vox_lin, bitmap,
                                                        word_rank, st, ctl);
            }
        }
        return hipGetLastError();
    };
    // every round picks at least the best unpicked voxel, so min(M, N) + 3
    // rounds always suffice (the last ones only count and record that the
    // cloud is done)
    const int64_t max_rounds = (int64_t)(M < N ? M : N) + 3;
    // every cloud needs several rounds: the first batch is long, later ones
    // short so that few rounds run after the last cloud is done
    const int first_batch = 6, batch = 1;
    PollBuffer* poll = poll_buffer();
    if (!poll) {
        // synchronous polling, a few rounds per copy of the done count
        const int sync_batch = 4;
        while (true) {
            if ((e = launch_batch(sync_batch)) != hipSuccess) return e;
            uint32_t nd = 0;
            if ((e = hipMemcpyAsync(&nd, ctl.ndone, sizeof nd, hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
            if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
            if (nd == (uint32_t)B) return hipSuccess;
            if (R > max_rounds + 2 * sync_batch) break;
        }
        *status_out = CAGQ_ERR_CAPACITY;
        return hipSuccess;
    }
    const int ahead = 2;
    // The round kernel publishes its round and, once every cloud is done, a
    // done flag in pinned host memory, both tagged with this call's epoch.
    // The host keeps at least `ahead` rounds queued until it sees the flag:
    // no copies and no events on the stream, so the GPU does not idle
    // between rounds. A word of another epoch is stale: it reads as no
    // progress.
    void* dev_words = nullptr;
    if ((e = hipHostGetDevicePointer(&dev_words, poll->words, 0)) != hipSuccess) return e;
    if (++poll->epoch == 0) ++poll->epoch;  // 0 is never an epoch
    const uint64_t tag = (uint64_t)poll->epoch << 32;
    volatile uint64_t* words = poll->words;
    ctl.host = static_cast<uint64_t*>(dev_words);
    ctl.epoch = tag;
    // an error return first lets the rounds already queued finish, so that
    // none of them runs after the call
    auto fail = [&](hipError_t err, int status) {
        const hipError_t q = hipStreamSynchronize(s);
        *status_out = status;
        return err != hipSuccess ? err : q;
    };
    if ((e = launch_batch(first_batch)) != hipSuccess) return fail(e, CAGQ_OK);
    auto progress = [&]() -> int64_t {  // the round being run, or -1 before this call's first
        const uint64_t w = words[1];
        return (w & 0xFFFFFFFF00000000ull) == tag ? (int64_t)(uint32_t)w : -1;
    };
    uint32_t seen = ~0u;
    auto seen_at = std::chrono::steady_clock::now();
    for (uint64_t spins = 1;; ++spins) {
        if (words[0] == (tag | 1u)) return hipSuccess;
        if (progress() + ahead >= R) {  // fewer than `ahead` rounds still queued
            if (R > max_rounds + 2 * batch) return fail(hipSuccess, CAGQ_ERR_CAPACITY);
            if ((e = launch_batch(batch)) != hipSuccess) return fail(e, CAGQ_OK);
            continue;
        }
        // A failed stream ends the wait. The stream is queried only once no
        // round has started for a millisecond: a query of a busy stream puts
        // a marker into its queue, which holds back the next round by ~5 us.
        if ((spins & 1023) == 0) {
            const uint32_t w = (uint32_t)progress();
            const auto now = std::chrono::steady_clock::now();
            if (w != seen) {
                seen = w;
                seen_at = now;
            } else if (now - seen_at > std::chrono::milliseconds(1)) {
                const hipError_t q = hipStreamQuery(s);
                if (q != hipSuccess && q != hipErrorNotReady) return q;
                seen_at = now;
            }
        }
    }
}

}  // namespace cagq
