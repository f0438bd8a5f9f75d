// Coverage-Aware Sampling (Sec. 3.2, Eqs. 1-2, greedy reading) for small
// clouds: one 1024-thread workgroup per cloud runs every round with all of
// its state in LDS, then selects and emits the centers, in one launch.
//
// The greedy, its exact round formulation and its tie-break are those of the
// many-kernel path in cagq_sample.hip; only the storage and the scheduling
// differ. With beta = 0 a score is 2^16 * lambda * U with U the number of
// uncovered voxels of the neighbourhood, so the key (score, -lin) orders
// exactly as the 32-bit key (U << 25) | (2^25 - 1 - slot): slots are ranks of
// lin, and an unpicked voxel's key is never 0.
//
// Every round walks, for some voxels, the occupied voxels within distance r
// (scoring) or 2r (picking, marking): the neighbour lists of
// cagq_cas_nbr.hip, written once before the rounds, so that the rounds need
// no geometry at all.
//
// Per round, each thread first looks at the slots it owns (slot tid + k*1024)
// and puts those that need real work into an LDS queue; the workgroup then
// drains the queue, one voxel per lane (or 16 lanes per voxel for a short
// queue with r = 1), packed into as few waves as possible. With r = 1 the
// keys stay exact by lowering (rounds_lowering): the queue holds the voxels
// that their cached blocker no longer beats, and after the picks one lane per
// voxel within r of a winner lowers the keys around it. With r = 2 a round
// first rescores the voxels near the last picks, then queues the voxels
// for picking. A voxel picked in round R keeps its key as a competitor for
// the rest of round R; after that its key drops below every unpicked key (to
// 0 with r = 2; to 2^30 with r = 1, where unpicked keys carry 2^31) and its
// pick key is kept in the two 16-bit words that an unpicked voxel uses for
// its blocker and its rescoring round.
#include "cagq_internal.h"

namespace cagq {

namespace {

constexpr int kT = 1024;                   // threads of the workgroup
constexpr int kNW = kT / kWave;            // waves of the workgroup
constexpr int kKS = kCasLdsMaxN / kT;      // owned slots per thread
constexpr int kKeyShift = 25;              // key = (U << 25) | (2^25 - 1 - slot)
constexpr uint32_t kSlotMask = (1u << kKeyShift) - 1;
constexpr uint32_t kUnpicked = 1u << 31;      // r = 1: offset of an unpicked voxel's key
constexpr uint16_t kNone = 0xFFFF;
constexpr int kPre = 4;                    // entry groups of 8 loaded with a list's header

// Lane i of a 16-lane row reads lane i - N of the row (0 beyond its start).
template <int N>
__device__ __forceinline__ uint32_t row_shr(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 + N, 0xF, 0xF, false);
}

// Value of lane `lane ^ J` within the 16-lane row (J = 1, 2, 4, 8).
template <int J>
__device__ __forceinline__ uint32_t row_xor(uint32_t v) {
    if constexpr (J == 1) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, true);  // quad_perm 1,0,3,2
    if constexpr (J == 2) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, true);  // quad_perm 2,3,0,1
    if constexpr (J == 4) {
        const uint32_t up = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x104, 0xF, 0xF, true);  // row_shl:4
        const uint32_t dn = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x114, 0xF, 0xF, true);  // row_shr:4
        return (threadIdx.x & 4) ? dn : up;
    }
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, true);  // row_ror:8
}

// Minimum over the 16 lanes of a row, in every lane of it.
__device__ __forceinline__ uint32_t row_min16(uint32_t v) {
    uint32_t o = row_xor<1>(v);
    v = o < v ? o : v;
    o = row_xor<2>(v);
    v = o < v ? o : v;
    o = row_xor<4>(v);
    v = o < v ? o : v;
    o = row_xor<8>(v);
    return o < v ? o : v;
}

// Maximum and sum over the wave, as a value uniform across it: an inclusive
// scan within each 16-lane row by row shifts, then the rows' last lanes read
// as scalars. Every lane of the wave must call them.
__device__ __forceinline__ uint32_t wmax32(uint32_t v) {
    uint32_t o = row_shr<1>(v);
    v = o > v ? o : v;
    o = row_shr<2>(v);
    v = o > v ? o : v;
    o = row_shr<4>(v);
    v = o > v ? o : v;
    o = row_shr<8>(v);
    v = o > v ? o : v;
    const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v, 15), b = (uint32_t)__builtin_amdgcn_readlane((int)v, 31);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v, 47), d = (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
    const uint32_t ab = a > b ? a : b, cd = c > d ? c : d;
    return ab > cd ? ab : cd;
}

__device__ __forceinline__ uint32_t wsum32(uint32_t v) {
    v += row_shr<1>(v);
    v += row_shr<2>(v);
    v += row_shr<4>(v);
    v += row_shr<8>(v);
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 15) + (uint32_t)__builtin_amdgcn_readlane((int)v, 31) +
           (uint32_t)__builtin_amdgcn_readlane((int)v, 47) + (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Appends the slots s = tid + k*kT with bit k of `want` set to the queue.
// One LDS atomic per wave. Every thread of the workgroup must call it.
__device__ __forceinline__ void enqueue(uint32_t want, uint16_t* q, uint32_t* s_qn) {
    const int lane = lane_id();
    const uint64_t below = (1ull << lane) - 1;
    uint64_t bal[kKS];
    uint32_t tot = 0;
#pragma unroll
    for (int k = 0; k < kKS; ++k) {
        bal[k] = __ballot((want >> k) & 1u);
        tot += (uint32_t)__popcll(bal[k]);
    }
    uint32_t base = 0;
    if (lane == 0 && tot) base = atomicAdd(s_qn, tot);
    base = (uint32_t)__builtin_amdgcn_readfirstlane((int)base);
#pragma unroll
    for (int k = 0; k < kKS; ++k) {
        if ((want >> k) & 1u) q[base + (uint32_t)__popcll(bal[k] & below)] = (uint16_t)(threadIdx.x + k * kT);
        base += (uint32_t)__popcll(bal[k]);
    }
}

// Entry j (0..7) of a 16-byte group of list entries.
__device__ __forceinline__ uint32_t entry(const uint4& v, int j) {
    const uint32_t w = j < 2 ? v.x : j < 4 ? v.y : j < 6 ? v.z : v.w;
    return (j & 1) ? w >> 16 : w & 0xFFFFu;
}

// Number of entries base..base+7 of a list (of n entries) whose voxel is
// not covered.
__device__ __forceinline__ uint32_t uncovered(const uint4& v, uint32_t base, uint32_t n, const uint8_t* cov) {
    uint32_t cv[8], u = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) cv[j] = base + j < n ? cov[entry(v, j)] : 1u;
#pragma unroll
    for (int j = 0; j < 8; ++j) u += cv[j] == 0 ? 1u : 0u;
    return u;
}

// A winner's marks on entries base..base+7 of its list: rescoring for the
// unpicked ones other than the winner itself (it and earlier picks keep
// their pick key in dty), coverage for the first n_r (those within distance
// r).
__device__ __forceinline__ void mark(const uint4& v, uint32_t base, uint32_t n_r, uint32_t n2, uint32_t self,
                                     uint16_t cur, const uint16_t* rnd, uint16_t* dty, uint8_t* cov) {
    uint32_t sl[8];
    uint16_t rr[8];
    uint8_t cc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sl[j] = base + j < n2 ? entry(v, j) : self;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        rr[j] = rnd[sl[j]];
        cc[j] = cov[sl[j]];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (base + j < n2) {
            if (rr[j] == 0 && sl[j] != self) dty[sl[j]] = cur;
            if (base + j < n_r) cov[sl[j]] = (uint8_t)(cc[j] + 1);
        }
    }
}

// The picking pass over the queued voxels, P lanes per voxel: lane `sub`
// of a voxel's P takes the groups of 8 list entries sub, sub + P, ...,
// kPre of them per load (the first kPre with the header, clamped to the
// list's storage; later ones clamped to its last group). A voxel is beaten
// when some entry within 2r holds a larger key; the lowest such position
// over the P lanes is the same blocker a single lane's in-order scan finds.
// A winner takes its pick round and key. With LOWER it joins the round's
// winner table (the lowering pass that follows updates coverage and keys);
// otherwise its lanes mark their groups: rescoring within 2r, coverage
// within r. A round's winners are more than 2r apart, so no other winner is
// on the list and their r-neighbourhoods are disjoint: plain updates are
// exact.
template <int P, int ST, bool LOWER>
__device__ __forceinline__ void drain_picks(uint32_t qb, int tid, uint16_t cur, const uint16_t* nb,
                                            const uint16_t* que, const uint32_t* key, uint16_t* rnd,
                                            uint16_t* blk, uint16_t* dty, uint8_t* cov, uint16_t* wtab,
                                            uint32_t* s_nw, uint16_t* ptab, uint32_t* s_np) {
    constexpr uint32_t kRoom = (ST - 8) / 8;  // groups a slot's storage holds after its header
    constexpr int KB = (int)((kRoom + P - 1) / P) < kPre ? (int)((kRoom + P - 1) / P) : kPre;  // groups per load
    const uint32_t sub = (uint32_t)tid & (P - 1);
    for (uint32_t i = (uint32_t)tid / P; i < qb; i += kT / P) {
        const uint32_t s = que[i];
        const uint32_t my = key[s];
        const uint4* e = reinterpret_cast<const uint4*>(nb + (size_t)s * ST);
        uint4 pre[KB];
        const uint4 h = e[0];
#pragma unroll
        for (int t = 0; t < KB; ++t) {
            const uint32_t c = sub + (uint32_t)(P * t);
            pre[t] = e[1 + (c < kRoom ? c : kRoom - 1)];
        }
        const uint32_t n_r = h.x & 0xFFFFu, n2 = h.x >> 16;
        const uint32_t nch = (n2 + 7) / 8;  // groups of 8 entries (n2 >= 1: the voxel itself)
        uint32_t hit = ~0u;                 // (position << 16) | slot of this lane's first larger key
        for (uint32_t t0 = 0; sub + P * t0 < nch && hit == ~0u; t0 += KB) {
            uint4 q[KB];
#pragma unroll
            for (int j = 0; j < KB; ++j) {
                const uint32_t c = sub + P * (t0 + j);
                q[j] = t0 == 0 ? pre[j] : e[1 + (c < nch ? c : nch - 1)];
            }
#pragma unroll
            for (int jj = 0; jj < KB; ++jj) {
                const uint32_t c = sub + P * (t0 + jj);
                if (c >= nch || hit != ~0u) break;
                uint32_t sl[8], kk[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) sl[j] = c * 8 + j < n2 ? entry(q[jj], j) : s;
#pragma unroll
                for (int j = 0; j < 8; ++j) kk[j] = key[sl[j]];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (hit == ~0u && kk[j] > my) hit = ((c * 8 + (uint32_t)j) << 16) | sl[j];
            }
        }
        static_assert(P == 1 || P == 16, "lanes per voxel");
        if constexpr (P == 16) hit = row_min16(hit);
        if (hit != ~0u) {
            if (sub == 0) blk[s] = (uint16_t)(hit & 0xFFFFu);
            continue;
        }
        if (sub == 0) {
            rnd[s] = cur;
            blk[s] = (uint16_t)(my >> 16);
            dty[s] = (uint16_t)(my & 0xFFFFu);
            if (LOWER) wtab[atomicAdd(s_nw, 1u)] = (uint16_t)s;
        }
        if constexpr (LOWER) {
            // the entries within r (the first n_r, in groups 0..kPre-1 held
            // by lanes 0..kPre-1) go to the round's pair table
            static_assert(P == 16 && KB == 1, "lane `sub` holds group `sub`");
            const uint32_t cnt = n_r > sub * 8 ? (n_r - sub * 8 < 8 ? n_r - sub * 8 : 8u) : 0u;
            if (sub < (uint32_t)kPre && cnt) {
                const uint32_t base = atomicAdd(s_np, cnt);
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if ((uint32_t)j < cnt) ptab[base + j] = (uint16_t)entry(pre[0], j);
            }
            continue;
        }
        for (uint32_t t0 = 0; sub + P * t0 < nch; t0 += KB) {
            uint4 q[KB];
#pragma unroll
            for (int j = 0; j < KB; ++j) {
                const uint32_t c = sub + P * (t0 + j);
                q[j] = t0 == 0 ? pre[j] : e[1 + (c < nch ? c : nch - 1)];
            }
#pragma unroll
            for (int jj = 0; jj < KB; ++jj) {
                const uint32_t c = sub + P * (t0 + jj);
                if (c < nch) mark(q[jj], c * 8, n_r, n2, s, cur, rnd, dty, cov);
            }
        }
    }
}

// The picking pass over a long queue (r = 1): one lane per voxel checks the
// kPre groups of entries loaded with its list's header. A voxel that none of
// them beats and whose list is longer (an open voxel) goes on to a second
// stage in which 16 lanes of its wave take it, four voxels at a time: lanes
// 0..11 load and check one group each of those after the first kPre. A
// winner joins the round's winner table. Every lane of the wave must call it.
template <int ST>
__device__ __forceinline__ void drain_mixed(uint32_t qb, int tid, uint16_t cur, const uint16_t* nb,
                                            const uint16_t* que, const uint32_t* key, uint16_t* rnd,
                                            uint16_t* blk, uint16_t* dty, uint16_t* wtab, uint32_t* s_nw,
                                            uint16_t* ptab, uint32_t* s_np) {
    constexpr int kRoom = (ST - 8) / 8;  // groups a slot's storage holds after its header
    static_assert(kRoom == 16 && kPre == 4, "16 lanes take the 16 groups of an r = 1 list");
    const int lane = lane_id();
    const int sub = lane & 15, quad = lane >> 4;
    // the group lane `sub` of a voxel's 16 checks in the second stage
    const uint32_t gq = (uint32_t)(kPre + sub);
    for (uint32_t i0 = (uint32_t)(tid - lane); i0 < qb; i0 += kT) {
        const uint32_t i = i0 + (uint32_t)lane;
        uint32_t s = 0, my = 0, n_r = 0, n2 = 0;
        bool open = false;
        uint4 pre[kPre];
        // a winner's entries within r (the first n_r) to the round's pair table
        auto pairs = [&]() {
            const uint32_t base = atomicAdd(s_np, n_r);
#pragma unroll
            for (int j = 0; j < kPre * 8; ++j)
                if ((uint32_t)j < n_r) ptab[base + j] = (uint16_t)entry(pre[j / 8], j % 8);
        };
        if (i < qb) {
            s = que[i];
            my = key[s];
            const uint4* e = reinterpret_cast<const uint4*>(nb + (size_t)s * ST);
            const uint4 h = e[0];
#pragma unroll
            for (int t = 0; t < kPre; ++t) pre[t] = e[1 + t];
            n_r = h.x & 0xFFFFu;
            n2 = h.x >> 16;
            const uint32_t nch = (n2 + 7) / 8;  // n2 >= 1: the voxel itself
            uint32_t hit = ~0u;
#pragma unroll
            for (int t = 0; t < kPre; ++t) {
                if ((uint32_t)t >= nch || hit != ~0u) break;
                uint32_t sl[8], kk[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) sl[j] = (uint32_t)(t * 8 + j) < n2 ? entry(pre[t], j) : s;
#pragma unroll
                for (int j = 0; j < 8; ++j) kk[j] = key[sl[j]];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (hit == ~0u && kk[j] > my) hit = ((uint32_t)(t * 8 + j) << 16) | sl[j];
            }
            if (hit != ~0u) {
                blk[s] = (uint16_t)(hit & 0xFFFFu);
            } else if (nch > (uint32_t)kPre) {
                open = true;
            } else {  // a short list, all checked: a winner
                rnd[s] = cur;
                blk[s] = (uint16_t)(my >> 16);
                dty[s] = (uint16_t)(my & 0xFFFFu);
                wtab[atomicAdd(s_nw, 1u)] = (uint16_t)s;
                pairs();
            }
        }
        for (uint64_t om = __ballot(open); om;) {
            // the quad-th open lane of the next four
            uint64_t m = om;
            for (int k = 0; k < quad && m; ++k) m &= m - 1;
            const bool act = m != 0;
            const int src = act ? __ffsll((unsigned long long)m) - 1 : 0;
            for (int k = 0; k < 4 && om; ++k) om &= om - 1;
            const uint32_t vs = (uint32_t)__shfl((int)s, src, kWave);
            const uint32_t vmy = (uint32_t)__shfl((int)my, src, kWave);
            const uint32_t vn2 = (uint32_t)__shfl((int)n2, src, kWave);
            const uint32_t vnch = (vn2 + 7) / 8;
            const bool mine = act && gq < vnch;  // this lane's group holds entries of the list
            uint4 q = make_uint4(0u, 0u, 0u, 0u);
            if (mine) q = reinterpret_cast<const uint4*>(nb + (size_t)vs * ST)[1 + gq];
            uint32_t hit = ~0u;
            if (mine) {
                uint32_t sl[8], kk[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) sl[j] = gq * 8 + (uint32_t)j < vn2 ? entry(q, j) : vs;
#pragma unroll
                for (int j = 0; j < 8; ++j) kk[j] = key[sl[j]];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (hit == ~0u && kk[j] > vmy) hit = ((gq * 8 + (uint32_t)j) << 16) | sl[j];
            }
            hit = row_min16(hit);
            if (act && sub == 0) {
                if (hit != ~0u) {
                    blk[vs] = (uint16_t)(hit & 0xFFFFu);
                } else {
                    rnd[vs] = cur;
                    blk[vs] = (uint16_t)(vmy >> 16);
                    dty[vs] = (uint16_t)(vmy & 0xFFFFu);
                    wtab[atomicAdd(s_nw, 1u)] = (uint16_t)vs;
                }
            }
        }
        // an open voxel that won (its pick round was written above, by this
        // wave) gives its pairs from the groups it holds
        if (open && rnd[s] == cur) pairs();
    }
}

// The rounds with r = 1, keys kept exact by lowering (the scheme of the
// many-kernel rounds on lists, in LDS). Keys start at U = n_r, the occupied
// voxels within r (nothing is covered). Per round, three phases between
// barriers:
// * owned slots: the picks above the previous round's best unpicked key G
//   are counted (when they reach m they are the sequential greedy's first m,
//   and the rounds stop: one round after the round-by-round bound would
//   allow); the best unpicked key is taken; an unpicked voxel still beaten
//   by its cached blocker stays out, the rest is queued;
// * the picking drain over the queue against the round-start keys: a voxel
//   is beaten by the first larger key on its 2r-list, else it wins and
//   joins the winner table;
// * the lowering: the winners put the voxels u within r of them into a pair
//   table (winners are more than 2r apart, so their r-neighbourhoods are
//   disjoint: at most one entry per voxel, and no coverage count is raised
//   twice in a round); one lane per u raises u's coverage count and, when u
//   was uncovered, lowers by one U the key of every unpicked voxel within r
//   of u (LDS atomics: such a voxel can lie within r of several newly
//   covered voxels). The winners' keys become 0: they compete no more.
// Keys carry 2^31 while the voxel is unpicked; a winner's key drops to 2^30.
// A picked voxel's key is then lowered by at most 27 * 2^25 < 2^30 more, so
// it stays positive and below every unpicked key: the lowering needs no
// test of who is picked. The pick keys (with the offset) order as before.
// Returns whether the rounds reached m picks.
template <int ST>
__device__ __forceinline__ bool rounds_lowering(int32_t nv, int32_t m, int tid, int lane, const uint16_t* nb,
                                                uint32_t* key, uint16_t* rnd, uint16_t* blk, uint16_t* dty,
                                                uint16_t* que, uint16_t* wtab, uint16_t* ptab, uint8_t* cov,
                                                uint32_t* s_max, uint32_t* s_cnt, uint32_t* s_qb, uint32_t* s_nw,
                                                uint32_t* s_np) {
    for (int32_t s = tid; s < nv; s += kT) {
        const uint32_t n_r = reinterpret_cast<const uint4*>(nb + (size_t)s * ST)[0].x & 0xFFFFu;
        key[s] = kUnpicked | (n_r << kKeyShift) | (kSlotMask - (uint32_t)s);
    }
    if (tid == 0) {
        *s_max = 0;
        *s_cnt = 0;
        *s_qb = 0;
    }
    uint32_t G = ~0u;  // the previous round's best unpicked key (none before the first round)
    const int32_t max_r = m + 3;
    for (int32_t R = 0; R < max_r; ++R) {
        const uint16_t cur = (uint16_t)(R + 1);
        __syncthreads();
        if (tid == 0) {
            *s_nw = 0;
            *s_np = 0;
        }
        uint32_t lmax = 0, above = 0, want = 0;
#pragma unroll
        for (int k = 0; k < kKS; ++k) {
            const int32_t s = tid + k * kT;
            if (s < nv) {
                const uint16_t r = rnd[s], bl = blk[s];
                if (r != 0) {
                    const uint32_t pk = ((uint32_t)bl << 16) | dty[s];
                    above += pk > G ? 1u : 0u;
                } else {
                    const uint32_t kv = key[s];
                    lmax = kv > lmax ? kv : lmax;
                    const bool beaten = bl != kNone && key[bl] > kv;
                    want |= beaten ? 0u : 1u << k;
                }
            }
        }
        lmax = wmax32(lmax);
        above = wsum32(above);
        if (lane == 0 && lmax) atomicMax(s_max, lmax);
        if (lane == 0 && above) atomicAdd(s_cnt, above);
        enqueue(want, que, s_qb);
        __syncthreads();
        if (*s_cnt >= (uint32_t)m) return true;
        G = *s_max;
        const uint32_t qb = *s_qb;
        if (qb <= kT / 8)
            drain_picks<16, ST, true>(qb, tid, cur, nb, que, key, rnd, blk, dty, cov, wtab, s_nw, ptab, s_np);
        else
            drain_mixed<ST>(qb, tid, cur, nb, que, key, rnd, blk, dty, wtab, s_nw, ptab, s_np);
        __syncthreads();
        if (tid == 0) {
            *s_max = 0;
            *s_cnt = 0;
            *s_qb = 0;
        }
        // the winners leave the competition; each voxel u within r of one
        // is covered once more and, if it was uncovered, lowers the keys
        // within r of it
        const uint32_t nw = *s_nw, np = *s_np;
        for (uint32_t p = (uint32_t)tid; p < nw; p += kT) key[wtab[p]] = kUnpicked >> 1;
        for (uint32_t p0 = 0; p0 < np; p0 += kT) {
            const uint32_t p = p0 + (uint32_t)tid;
            uint32_t nru = 0;
            uint4 gu[kPre];  // the first kPre groups hold every entry within r
            if (p < np) {
                const uint32_t u = ptab[p];
                const uint8_t c = cov[u];
                cov[u] = (uint8_t)(c + 1);
                if (c == 0) {
                    const uint4* eu = reinterpret_cast<const uint4*>(nb + (size_t)u * ST);
                    const uint4 hu = eu[0];
#pragma unroll
                    for (int t = 0; t < kPre; ++t) gu[t] = eu[1 + t];
                    nru = hu.x & 0xFFFFu;
                }
            }
            const uint32_t nmax = wmax32(nru);
#pragma unroll
            for (int i = 0; i < kPre * 8; ++i) {
                if ((uint32_t)i >= nmax) break;
                if ((uint32_t)i < nru) atomicSub(&key[entry(gu[i / 8], i % 8)], 1u << kKeyShift);
            }
        }
    }
    return false;
}

template <int RAD>
__global__ __launch_bounds__(kT) void k_cas_lds(int32_t N, int32_t M, int32_t cap,
                                                const int32_t* __restrict__ nvox,
                                                const uint32_t* __restrict__ vox_lin,
                                                const uint16_t* __restrict__ nbr,
                                                int32_t* __restrict__ center_lin, int32_t* __restrict__ m_valid,
                                                int* __restrict__ status) {
    constexpr int ST = nbr_stride(RAD);
    extern __shared__ __align__(16) unsigned char lds[];
    uint32_t* key = reinterpret_cast<uint32_t*>(lds);           // competitor key, 0 once out
    uint16_t* rnd = reinterpret_cast<uint16_t*>(key + cap);     // round that picked it + 1, 0 = unpicked
    uint16_t* blk = rnd + cap;   // unpicked: a neighbour that beat it; picked: pick key >> 16
    uint16_t* dty = blk + cap;   // unpicked: round that must rescore it; picked: pick key & 0xFFFF
    uint16_t* que = dty + cap;   // work queue of slots
    uint16_t* wtab = que + cap;  // r = 1: the round's winners
    uint16_t* ptab = wtab + cap; // r = 1: the voxels within r of the round's winners
    uint8_t* cov = reinterpret_cast<uint8_t*>(ptab + cap);      // centers covering the voxel
    __shared__ uint32_t s_max, s_cnt, s_qa, s_qb;  // s_qa / s_qb: scoring / picking queue lengths
    __shared__ uint32_t s_nw, s_np;                // r = 1: winners and pairs of the round
    __shared__ uint32_t s_hist[128];
    __shared__ uint32_t s_digit, s_below;
    __shared__ uint32_t s_wsum[kNW];

    const int32_t b = blockIdx.x;
    const int tid = threadIdx.x, lane = lane_id(), wv = tid / kWave;
    const int32_t nv = nvox[b];
    const int32_t m = M < nv ? M : nv;
    if (m <= 0) {  // no occupied voxel (the build has raised an error): nothing to choose
        if (tid == 0) m_valid[b] = 0;
        return;
    }
    const uint32_t* vl = vox_lin + (size_t)b * N;
    const uint16_t* nb = nbr + (size_t)b * N * ST;
    for (int32_t s = tid; s < nv; s += kT) {
        rnd[s] = 0;
        blk[s] = kNone;
        dty[s] = 0;
        cov[s] = 0;
    }
    if (tid == 0) {
        s_max = 0;
        s_qa = 0;
    }

    bool done = false;
    if constexpr (RAD == 1) {
        done = rounds_lowering<ST>(nv, m, tid, lane, nb, key, rnd, blk, dty, que, wtab, ptab, cov, &s_max, &s_cnt,
                                   &s_qb, &s_nw, &s_np);
    } else {
    const int32_t max_r = m + 2;
    for (int32_t R = 0; R < max_r; ++R) {
        const uint16_t cur = (uint16_t)(R + 1);
        // Each counter is cleared at a point where every thread is past its
        // last read and a barrier separates it from its next update:
        // s_cnt and s_qb here, s_qa once G is read, s_max after the picking
        // queue is complete.
        __syncthreads();
        if (tid == 0) {
            s_cnt = 0;
            s_qb = 0;
        }
        // -- scoring. Owned slots: last round's picks leave the competition,
        // clean unpicked keys count towards the maximum, the rest is queued.
        uint32_t lmax = 0, want = 0;
#pragma unroll
        for (int k = 0; k < kKS; ++k) {
            const int32_t s = tid + k * kT;
            if (s < nv) {
                const uint16_t r = rnd[s];
                if (R > 0 && r == (uint16_t)R) key[s] = 0;
                const bool dirty = r == 0 && (R == 0 || dty[s] == (uint16_t)R);
                if (r == 0 && !dirty) {
                    const uint32_t kv = key[s];
                    lmax = kv > lmax ? kv : lmax;
                }
                want |= dirty ? 1u << k : 0u;
            }
        }
        enqueue(want, que, &s_qa);
        __syncthreads();
        const uint32_t qa = s_qa;
        for (uint32_t i = tid; i < qa; i += kT) {
            const uint32_t s = que[i];
            const uint4* e = reinterpret_cast<const uint4*>(nb + (size_t)s * ST);
            // the header and the first kPre groups of entries are loaded
            // together (every list has room for them), so a list within r
            // of up to 8 * kPre entries costs one load latency
            uint4 pre[kPre];
            const uint4 h = e[0];
#pragma unroll
            for (int c = 0; c < kPre; ++c) pre[c] = e[1 + c];
            const uint32_t n_r = h.x & 0xFFFFu;
            uint32_t U = 0;
#pragma unroll
            for (int c = 0; c < kPre; ++c)
                if ((uint32_t)c * 8 < n_r) U += uncovered(pre[c], c * 8, n_r, cov);
            const uint32_t ncr = (n_r + 7) / 8;
            for (uint32_t c0 = kPre; c0 < ncr; c0 += kPre) {
                uint4 q[kPre];
#pragma unroll
                for (int j = 0; j < kPre; ++j) q[j] = e[1 + (c0 + j < ncr ? c0 + j : ncr - 1)];
#pragma unroll
                for (int j = 0; j < kPre; ++j)
                    if (c0 + j < ncr) U += uncovered(q[j], (c0 + j) * 8, n_r, cov);
            }
            const uint32_t kv = (U << kKeyShift) | (kSlotMask - s);
            key[s] = kv;
            lmax = kv > lmax ? kv : lmax;
        }
        lmax = wmax32(lmax);
        if (lane == 0 && lmax) atomicMax(&s_max, lmax);
        __syncthreads();
        const uint32_t G = s_max;
        if (tid == 0) s_qa = 0;
        // -- picking. Owned slots: earlier picks above the best unpicked key
        // are counted; an unpicked voxel still beaten by its cached blocker
        // stays out; the rest is queued for a pass over its list.
        uint32_t above = 0;
        want = 0;
#pragma unroll
        for (int k = 0; k < kKS; ++k) {
            const int32_t s = tid + k * kT;
            if (s < nv) {
                const uint16_t r = rnd[s], bl = blk[s];
                if (r != 0) {
                    const uint32_t pk = ((uint32_t)bl << 16) | dty[s];
                    above += pk > G ? 1u : 0u;
                } else {
                    const bool beaten = bl != kNone && key[bl] > key[s];
                    want |= beaten ? 0u : 1u << k;
                }
            }
        }
        above = wsum32(above);
        if (lane == 0 && above) atomicAdd(&s_cnt, above);
        enqueue(want, que, &s_qb);
        __syncthreads();
        if (tid == 0) s_max = 0;
        // the picks above the best unpicked key are the sequential greedy's
        // first ones; the voxels this round would pick all have keys <= G
        if (s_cnt >= (uint32_t)m) {
            done = true;
            break;
        }
        const uint32_t qb = s_qb;
        // with r = 1 a short queue gets 16 lanes per voxel, one group of
        // list entries each, in at most two passes (2, 4 or 8 lanes per
        // voxel spill registers here); a longer one gets 16 lanes only for
        // the voxels that the first groups of their lists do not decide
        drain_picks<1, ST, false>(qb, tid, cur, nb, que, key, rnd, blk, dty, cov, wtab, &s_nw, ptab, &s_np);
    }
    }
    if (!done && tid == 0) raise_error(status, CAGQ_ERR_CAPACITY);
    __syncthreads();

    // The m largest pick keys. A pick key is (U << 25) | (2^25 - 1 - slot)
    // (with r = 1 plus 2^31, which adds 64 to every U below):
    // with U* the largest U for which at least m picks have U >= U*, the
    // chosen picks are those with U > U* and, of those with U = U*, the
    // `need` lowest slots.
    // the owned slots' linear ids for the emit below, loaded now (from
    // indices clamped into the cloud's row) so that the histogram's phases
    // cover their latency
    uint32_t lv[kKS];
#pragma unroll
    for (int k = 0; k < kKS; ++k) {
        const int32_t s = k * kT + tid;
        lv[k] = vl[s < N ? s : N - 1];
    }
    uint32_t pk[kKS];
    for (int32_t i = tid; i < 128; i += kT) s_hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kKS; ++k) {
        const int32_t s = tid + k * kT;
        pk[k] = 0;
        if (s < nv && rnd[s] != 0) pk[k] = ((uint32_t)blk[s] << 16) | dty[s];
        const bool act = pk[k] != 0;
        const uint32_t u = pk[k] >> kKeyShift;
        uint64_t am = __ballot(act);
        // one LDS atomic per distinct U for the first few values of the wave
        for (int rr = 0; rr < 4 && am; ++rr) {
            const int leader = __ffsll((unsigned long long)am) - 1;
            const uint32_t u0 = (uint32_t)__shfl((int)u, leader, kWave);
            const uint64_t same = __ballot(act && u == u0) & am;
            if (lane == leader) atomicAdd(&s_hist[u0], (uint32_t)__popcll(same));
            am &= ~same;
        }
        if ((am >> lane) & 1ull) atomicAdd(&s_hist[u], 1u);
    }
    __syncthreads();
    if (tid < kWave) {
        // lane l holds U = 127 - 2l and 126 - 2l: the scan counts from the top
        const uint32_t h0 = s_hist[127 - 2 * tid], h1 = s_hist[126 - 2 * tid];
        const uint32_t incl = wave_incl_scan<uint32_t>(h0 + h1);
        const uint32_t run0 = incl - h0 - h1, run1 = run0 + h0;
        if (run0 < (uint32_t)m && run0 + h0 >= (uint32_t)m) {
            s_digit = (uint32_t)(127 - 2 * tid);
            s_below = (uint32_t)m - run0;
        }
        if (run1 < (uint32_t)m && run1 + h1 >= (uint32_t)m) {
            s_digit = (uint32_t)(126 - 2 * tid);
            s_below = (uint32_t)m - run1;
        }
    }
    __syncthreads();
    const uint32_t ustar = s_digit, need = s_below;

    // chosen slots in ascending slot (= lin) order; position p < m also
    // fills p + m, p + 2m, ... < M (cyclic padding)
    int32_t* out = center_lin + (size_t)b * M;
    const uint64_t below = (1ull << lane) - 1;
    uint32_t base_h = 0, base_t = 0;
#pragma unroll
    for (int k = 0; k < kKS; ++k) {
        const uint32_t u = pk[k] >> kKeyShift;
        const bool hi = pk[k] != 0 && u > ustar, tie = pk[k] != 0 && u == ustar;
        const uint64_t bh = __ballot(hi), bt = __ballot(tie);
        if (lane == 0) s_wsum[wv] = (uint32_t)__popcll(bh) | ((uint32_t)__popcll(bt) << 16);
        __syncthreads();
        uint32_t off = 0, tot = 0;
        for (int w = 0; w < kNW; ++w) {
            const uint32_t c = s_wsum[w];
            if (w < wv) off += c;
            tot += c;
        }
        const uint32_t hb = base_h + (off & 0xFFFFu) + (uint32_t)__popcll(bh & below);
        const uint32_t tb = base_t + (off >> 16) + (uint32_t)__popcll(bt & below);
        if (hi || (tie && tb < need)) {
            const uint32_t pos = hb + (tb < need ? tb : need);
            const int32_t lin = (int32_t)lv[k];
            for (int32_t j = (int32_t)pos; j < M; j += m) out[j] = lin;
        }
        base_h += tot & 0xFFFFu;
        base_t += tot >> 16;
        __syncthreads();
    }
    if (tid == 0) m_valid[b] = m;
}

int32_t lds_cap(int32_t N) { return (N + 3) & ~3; }
size_t lds_bytes(int32_t cap) { return (size_t)17 * cap + 16; }

}  // namespace

bool cas_lds_fits(const Layout& L, const cagq_grid_desc& d, uint32_t beta_q16) {
    return beta_q16 == 0 && (d.radius == 1 || d.radius == 2) && L.N <= kCasLdsMaxN && L.has_nbr16;
}

hipError_t launch_cas_lds(const Layout& L, const cagq_grid_desc& d, void* ws, int32_t M, int32_t* center_lin,
                          int32_t* m_valid, hipStream_t s) {
    hipError_t e = launch_cas_nbr(L, d, ws, s);
    if (e != hipSuccess) return e;
    const int32_t cap = lds_cap(L.N);
    const size_t bytes = lds_bytes(cap);
    const int32_t* nvox = at<int32_t>(ws, L.nvox);
    const uint32_t* vox_lin = at<uint32_t>(ws, L.vox_lin);
    const uint16_t* nbr = at<uint16_t>(ws, L.cas_nbr);
    auto go = [&](auto kern) {
        hipError_t r = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (r != hipSuccess) return r;
        kern<<<L.B, kT, bytes, s>>>(L.N, M, cap, nvox, vox_lin, nbr, center_lin, m_valid, at<int>(ws, L.status));
        return hipGetLastError();
    };
    return d.radius == 1 ? go(k_cas_lds<1>) : go(k_cas_lds<2>);
}

}  // namespace cagq
