/*
 * CAGQ CPU oracle -- TEST INFRASTRUCTURE ONLY (see cagq_oracle.h).
 *
 * Plain single-threaded C99, compiled with -O2 -ffp-contract=off
 * -fno-fast-math (SSE2 scalar float on x86-64: every fp32 operation is one
 * IEEE-754 round-to-nearest-even operation, no contraction, no x87).
 *
 * What the paper fixes, and the reading taken where it is silent:
 *   voxelize  Sec. 3.2: Vid = floor(x / v) per axis. Reading: an explicit
 *             grid origin o and dims D; t = (p - o) / s in fp32 (one rounded
 *             subtract, one correctly rounded divide); g = clamp(floor(t), 0,
 *             D - 1) evaluated exactly; lin = gx + Dx * (gy + Dy * gz).
 *   table     Appendix D, general procedure, step 1: O_v is the set of
 *             non-empty voxels; each voxel stores at most n_v points, the
 *             ones a sequential pass over the points visits first, i.e. the
 *             lowest point indices. Reading: slots are the ranks of lin
 *             (ascending), lists ascending, off = exclusive prefix of
 *             min(count, n_v).
 *   RVS       Sec. 3.2: every occupied voxel equally likely. Reading: the
 *             min(M, |O_v|) slots with the smallest key
 *             (hi32(h(seed, 1, b, slot)) << 32 | slot), emitted in slot
 *             order, cyclic padding up to M.
 *   CAS       Sec. 3.2, Eqs. 1-2: coverage gain H_add of a challenger,
 *             delta(C_V) minus beta * C_V / lambda summed over pi(v).
 *             Reading: greedy -- each of min(M, |O_v|) steps picks the
 *             unpicked voxel of largest integer score
 *             2^16 * lambda * U(v) - beta_q16 * sum C_V (= 2^16 * lambda *
 *             H_add exactly), ties to the lowest lin; lambda = (2r+1)^3.
 *             The chosen set is emitted in ascending lin (as for RVS); the
 *             pick order and pick-time scores are returned separately.
 *   CAS-P     Sec. 3.2, Eqs. 2-3, the paper's own procedure: M random
 *             incumbents; every other occupied voxel challenges a random
 *             incumbent and replaces it when H_add > H_rmv, with
 *             H_rmv = #{V in pi(I): C_V = 1}. Reading: the incumbents are
 *             the RVS choice with the same seed, held in slots 0..m-1 in
 *             ascending lin; the challengers are the other occupied voxels
 *             in ascending lin, each challenging once (a replaced incumbent
 *             does not challenge again); challenge t goes to slot
 *             hi32(h(seed, 3, b, t)) mod m; both heuristics are compared
 *             scaled by 2^16 * lambda, as integers. Output in ascending lin.
 *   pi(v)     Sec. 3.2 and the notation table: the occupied voxels of the
 *             (2r+1)^3 cube around v, v included, clipped to the grid.
 *   query     Sec. 3.2: Cube Query picks K context points at random, k-NN
 *             the K nearest. Reading: keep the min(K, c) context points of
 *             smallest 64-bit key, in ascending key order; cube key
 *             hi32(h(seed, 2, b, lin(v), i)) << 32 | i, k-NN key
 *             bits(d^2) << 32 | i with d measured from the center of voxel
 *             v and d^2 = (dx*dx + dy*dy) + dz*dz. Slots k >= n repeat slot 0.
 *   k-NN by   Appendix D, "CAGQ k-NN" (mode 2): levels 0, 1, ..., r of pi(v)
 *   levels    (Chebyshev distance exactly i); a level that fits in what is
 *             left of K is appended whole, in gathering order (voxels by
 *             ascending lin, stored points ascending), otherwise its nearest
 *             points by the k-NN key; stop at K. Not exact: a level-1 point
 *             can be nearer than a level-0 one.
 *   center    Appendix E, Eqs. 7-8: w_c = sum w_j, chi_c = sum w_j chi_j /
 *             w_c over the n valid nodes. Reading: the fp32 sum is pairwise
 *             in node order (stride 1, 2, 4, ...), then one fp32 divide.
 *   upsample  Sec. 3.1: centers given from outside, only nodes queried.
 *             Reading: a center point's voxel v by the voxelize rule (v need
 *             not be occupied); context and cube key as for query; the k-NN
 *             reference is the center point itself; an empty context gives
 *             n = 0 and index -1 in every slot.
 *   context   Sec. 3.3, grid context pooling: every context point of a
 *             center. Reading: voxels of pi(v) in ascending lin, stored
 *             points ascending, concatenated over the batch (CSR offsets).
 *   RPS, FPS, Ball Query (Sec. 4, the comparison methods): RPS = the M
 *             points of smallest key hi32(h(seed, 4, b, i)) << 32 | i in
 *             ascending index; FPS from point 0, farthest by d^2 to the
 *             chosen set, ties to the lowest index, pick order; Ball Query =
 *             the first K points in index order with d^2 < R^2.
 *   coverage  Sec. 4: occupied voxels holding a node point / |O_v|.
 *   h         splitmix64 chain: h(seed, tag, a1..ak) =
 *             sm64(...sm64(sm64(seed ^ tag) ^ a1)... ^ ak), tags RVS=1,
 *             CUBE=2, CAS-P=3, RPS=4 (splitmix64: Steele, Lea, Flood, OOPSLA 2014).
 *
 * Pins (tests marked "not gpu"): splitmix64 published outputs; voxelize vs
 * a numpy fp32 re-derivation and hand-placed boundary points; the table vs
 * numpy unique/argsort; RVS vs an explicit lexsort and a chi-square test of
 * equal inclusion probability; CAS vs brute-force recomputation at every
 * step, exhaustive optimum on <= 64 voxels (1 - 1/e bound, equality at
 * M = 1), disjoint-neighbourhood closed form; CAS-P: covered space strictly
 * grows with every accepted swap at beta = 0 (recomputed from the replayed
 * incumbent sets), slot draws vs an independent hash, no swap among
 * isolated voxels, hand-worked examples; k-NN vs brute force and vs
 * global k-NN when the cap never binds; cube subset / frequency checks;
 * centers vs closed forms and an fp64 error bound; upsampling k-NN vs a
 * numpy brute force over the block around each center point, and vs
 * global k-NN; context lists vs a numpy enumeration of the block's stored
 * points; level-wise k-NN vs a hand-worked example of the algorithm, the
 * K nearest of the center voxel when it holds K points, the whole context
 * in level order when it holds at most K.
 */
#include "cagq_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORC_EINVAL (-1)
#define ORC_ENONFINITE (-4)
#define ORC_ECAPACITY (-5)
#define ORC_ENOTOCC (-7)

uint64_t orc_splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static int grid_ok(const orc_grid* g) {
    int64_t v = 1;
    for (int a = 0; a < 3; ++a) {
        if (g->dims[a] < 1) return 0;
        if (!(g->voxel_size[a] > 0.0f) || !isfinite(g->voxel_size[a])) return 0;
        if (!isfinite(g->origin[a])) return 0;
        v *= g->dims[a];
        if (v > 2147483647LL) return 0;
    }
    return g->n_v >= 1 && g->radius >= 1;
}

/* One axis of the voxel index: clamp(floor((p - o) / s), 0, D - 1). */
static int32_t axis_index(float p, float o, float s, int32_t D) {
    float diff = p - o;
    float t = diff / s;
    float f = floorf(t);
    if (f < 0.0f) return 0;
    if (f >= 2147483648.0f) return D - 1;
    int64_t gi = (int64_t)f;
    return gi > (int64_t)(D - 1) ? D - 1 : (int32_t)gi;
}

int orc_voxelize(const float* pts, int64_t n, const orc_grid* g, uint32_t* lin) {
    if (!pts || !g || !lin || n < 0 || !grid_ok(g)) return ORC_EINVAL;
    int rc = 0;
    for (int64_t i = 0; i < n; ++i) {
        int32_t gg[3];
        for (int a = 0; a < 3; ++a) {
            float p = pts[3 * i + a];
            if (!isfinite(p)) {
                rc = ORC_ENONFINITE;
                gg[a] = 0;
            } else {
                gg[a] = axis_index(p, g->origin[a], g->voxel_size[a], g->dims[a]);
            }
        }
        lin[i] = (uint32_t)gg[0] + (uint32_t)g->dims[0] * ((uint32_t)gg[1] + (uint32_t)g->dims[1] * (uint32_t)gg[2]);
    }
    return rc;
}

static int cmp_u64(const void* a, const void* b) {
    uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
    return (x > y) - (x < y);
}

int orc_build_table(const float* pts, int32_t B, int32_t N, const orc_grid* g,
                    int32_t* nvox, uint32_t* vox_lin, uint32_t* vox_count,
                    uint32_t* vox_off, uint32_t* pt_list) {
    if (!pts || !g || !nvox || !vox_lin || !vox_count || !vox_off || !pt_list) return ORC_EINVAL;
    if (B < 1 || N < 1 || !grid_ok(g)) return ORC_EINVAL;
    uint32_t* lin = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)N);
    uint64_t* key = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)N);
    if (!lin || !key) { free(lin); free(key); return ORC_EINVAL; }
    int rc = 0;
    for (int32_t b = 0; b < B; ++b) {
        int r = orc_voxelize(pts + (size_t)b * N * 3, N, g, lin);
        if (r) rc = r;
        /* sort the points by (voxel, point index): the runs are the voxels of
         * O_v in ascending lin, each run's points in ascending index */
        for (int32_t i = 0; i < N; ++i) key[i] = ((uint64_t)lin[i] << 32) | (uint32_t)i;
        qsort(key, (size_t)N, sizeof(uint64_t), cmp_u64);
        uint32_t* vl = vox_lin + (size_t)b * N;
        uint32_t* vc = vox_count + (size_t)b * N;
        uint32_t* vo = vox_off + (size_t)b * (N + 1);
        uint32_t* pl = pt_list + (size_t)b * N;
        int32_t s = -1;
        for (int32_t j = 0; j < N; ++j) {
            uint32_t l = (uint32_t)(key[j] >> 32);
            if (s < 0 || vl[s] != l) {
                ++s;
                vl[s] = l;
                vc[s] = 0;
            }
            vc[s] += 1;
        }
        nvox[b] = s + 1;
        vo[0] = 0;
        for (int32_t t = 0; t < nvox[b]; ++t) {
            uint32_t stored = vc[t] < (uint32_t)g->n_v ? vc[t] : (uint32_t)g->n_v;
            vo[t + 1] = vo[t] + stored;
        }
        /* the first min(count, n_v) points of each run are its stored list */
        s = -1;
        uint32_t k = 0;
        for (int32_t j = 0; j < N; ++j) {
            uint32_t l = (uint32_t)(key[j] >> 32);
            if (s < 0 || vl[s] != l) { ++s; k = 0; }
            if (k < (uint32_t)g->n_v) pl[vo[s] + k] = (uint32_t)(key[j] & 0xFFFFFFFFu);
            ++k;
        }
    }
    free(lin);
    free(key);
    return rc;
}

/* slot of linear id l in batch b, or -1 when the voxel is not occupied */
static int32_t find_slot(const orc_table* t, int32_t b, uint32_t l) {
    const uint32_t* vl = t->vox_lin + (size_t)b * t->N;
    int32_t lo = 0, hi = t->nvox[b] - 1;
    while (lo <= hi) {
        int32_t mid = lo + (hi - lo) / 2;
        if (vl[mid] == l) return mid;
        if (vl[mid] < l) lo = mid + 1; else hi = mid - 1;
    }
    return -1;
}

/* pi(v): slots of the occupied voxels whose grid index differs from that of
 * lin by at most rad on every axis (v itself included), inside the grid. */
static int32_t neighbours(const orc_table* t, int32_t b, uint32_t l, int32_t rad, int32_t* out) {
    const int32_t* D = t->g.dims;
    int32_t gx = (int32_t)(l % (uint32_t)D[0]);
    int32_t gy = (int32_t)((l / (uint32_t)D[0]) % (uint32_t)D[1]);
    int32_t gz = (int32_t)(l / ((uint32_t)D[0] * (uint32_t)D[1]));
    int32_t n = 0;
    for (int32_t dz = -rad; dz <= rad; ++dz)
        for (int32_t dy = -rad; dy <= rad; ++dy)
            for (int32_t dx = -rad; dx <= rad; ++dx) {
                int32_t x = gx + dx, y = gy + dy, z = gz + dz;
                if (x < 0 || y < 0 || z < 0 || x >= D[0] || y >= D[1] || z >= D[2]) continue;
                uint32_t nl = (uint32_t)x + (uint32_t)D[0] * ((uint32_t)y + (uint32_t)D[1] * (uint32_t)z);
                int32_t s = find_slot(t, b, nl);
                if (s >= 0) out[n++] = s;
            }
    return n;
}

static int table_ok(const orc_table* t) {
    return t && t->B >= 1 && t->N >= 1 && grid_ok(&t->g) && t->nvox && t->vox_lin &&
           t->vox_count && t->vox_off && t->pt_list;
}

static void pad_cyclic(int32_t* c, int32_t m, int32_t M) {
    for (int32_t j = m; j < M; ++j) c[j] = c[j % m];
}

int orc_sample_rvs(const orc_table* t, int32_t M, uint64_t seed,
                   int32_t* center_lin, int32_t* m_valid) {
    if (!table_ok(t) || M < 1 || !center_lin || !m_valid) return ORC_EINVAL;
    uint64_t* key = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)t->N);
    uint64_t* sel = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)t->N);
    if (!key || !sel) { free(key); free(sel); return ORC_EINVAL; }
    for (int32_t b = 0; b < t->B; ++b) {
        int32_t nv = t->nvox[b];
        int32_t m = M < nv ? M : nv;
        uint64_t hb = orc_splitmix64(orc_splitmix64(seed ^ 1ull) ^ (uint64_t)b);
        for (int32_t s = 0; s < nv; ++s) {
            uint64_t h = orc_splitmix64(hb ^ (uint64_t)s);
            key[s] = ((h >> 32) << 32) | (uint32_t)s;
        }
        qsort(key, (size_t)nv, sizeof(uint64_t), cmp_u64);
        for (int32_t j = 0; j < m; ++j) sel[j] = key[j] & 0xFFFFFFFFu;  /* chosen slots */
        qsort(sel, (size_t)m, sizeof(uint64_t), cmp_u64);
        int32_t* c = center_lin + (size_t)b * M;
        for (int32_t j = 0; j < m; ++j) c[j] = (int32_t)t->vox_lin[(size_t)b * t->N + sel[j]];
        pad_cyclic(c, m, M);
        m_valid[b] = m;
    }
    free(key);
    free(sel);
    return 0;
}

/* Eq. 2 scaled by 2^16 * lambda: 2^16*lambda*#{V in pi(v): C_V = 0} - beta_q16 * sum C_V */
static int64_t cas_score(const int32_t* nb_off, const int32_t* nb, const uint32_t* C,
                         int32_t v, int64_t lambda, uint32_t beta_q16) {
    int64_t uncovered = 0, covsum = 0;
    for (int32_t k = nb_off[v]; k < nb_off[v + 1]; ++k) {
        uint32_t c = C[nb[k]];
        if (c == 0) uncovered += 1;
        covsum += c;
    }
    return 65536LL * lambda * uncovered - (int64_t)beta_q16 * covsum;
}

static int cmp_i32(const void* a, const void* b) {
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

int orc_sample_cas(const orc_table* t, int32_t M, uint32_t beta_q16,
                   int32_t* center_lin, int32_t* m_valid,
                   int32_t* pick_lin, int64_t* pick_score) {
    if (!table_ok(t) || M < 1 || !center_lin || !m_valid) return ORC_EINVAL;
    int32_t rad = t->g.radius;
    int32_t side = 2 * rad + 1;
    int64_t lambda = (int64_t)side * side * side;
    int rc = 0;
    for (int32_t b = 0; b < t->B && rc == 0; ++b) {
        int32_t nv = t->nvox[b];
        int32_t m = M < nv ? M : nv;
        const uint32_t* vl = t->vox_lin + (size_t)b * t->N;
        /* pi(v) of every occupied voxel, as a CSR list of slots */
        int32_t* nb_off = (int32_t*)malloc(sizeof(int32_t) * (size_t)(nv + 1));
        int32_t* nb = (int32_t*)malloc(sizeof(int32_t) * (size_t)nv * (size_t)lambda);
        uint32_t* C = (uint32_t*)calloc((size_t)nv, sizeof(uint32_t));
        unsigned char* picked = (unsigned char*)calloc((size_t)nv, 1);
        int64_t* score = (int64_t*)malloc(sizeof(int64_t) * (size_t)nv);
        if (!nb_off || !nb || !C || !picked || !score) {
            rc = ORC_EINVAL;
        } else {
            nb_off[0] = 0;
            for (int32_t v = 0; v < nv; ++v) {
                int32_t n = neighbours(t, b, vl[v], rad, nb + nb_off[v]);
                nb_off[v + 1] = nb_off[v] + n;
            }
            for (int32_t v = 0; v < nv; ++v) score[v] = cas_score(nb_off, nb, C, v, lambda, beta_q16);
            int32_t* c = center_lin + (size_t)b * M;
            for (int32_t step = 0; step < m; ++step) {
                /* argmax over unpicked voxels; scanning slots in ascending lin
                 * with a strict comparison keeps the lowest lin on ties */
                int32_t best = -1;
                for (int32_t v = 0; v < nv; ++v)
                    if (!picked[v] && (best < 0 || score[v] > score[best])) best = v;
                picked[best] = 1;
                c[step] = (int32_t)vl[best];
                if (pick_lin) pick_lin[(size_t)b * M + step] = (int32_t)vl[best];
                if (pick_score) pick_score[(size_t)b * M + step] = score[best];
                for (int32_t k = nb_off[best]; k < nb_off[best + 1]; ++k) C[nb[k]] += 1;
                /* a score sums over pi(u); C changed on pi(best), so every u
                 * with some V of pi(best) in pi(u) -- u in pi(V) -- is
                 * recomputed from its definition */
                for (int32_t k = nb_off[best]; k < nb_off[best + 1]; ++k) {
                    int32_t V = nb[k];
                    for (int32_t q = nb_off[V]; q < nb_off[V + 1]; ++q) {
                        int32_t u = nb[q];
                        score[u] = cas_score(nb_off, nb, C, u, lambda, beta_q16);
                    }
                }
            }
            for (int32_t j = m; j < M; ++j) {
                if (pick_lin) pick_lin[(size_t)b * M + j] = pick_lin[(size_t)b * M + j % m];
                if (pick_score) pick_score[(size_t)b * M + j] = pick_score[(size_t)b * M + j % m];
            }
            /* the chosen set is emitted in ascending lin, as RVS emits it */
            qsort(c, (size_t)m, sizeof(int32_t), cmp_i32);
            pad_cyclic(c, m, M);
            m_valid[b] = m;
        }
        free(nb_off);
        free(nb);
        free(C);
        free(picked);
        free(score);
    }
    return rc;
}

/* CAS-P: the paper's challenger / incumbent procedure (Sec. 3.2, Eqs. 2-3).
 * decision [B][N] (may be NULL): for challenge t, the incumbent slot it
 * challenged if the swap was accepted, -(slot + 1) if it was refused;
 * n_swaps [B] (may be NULL): accepted swaps. */
int orc_sample_cas_swap(const orc_table* t, int32_t M, uint64_t seed, uint32_t beta_q16,
                        int32_t* center_lin, int32_t* m_valid, int32_t* decision, int32_t* n_swaps) {
    if (!table_ok(t) || M < 1 || !center_lin || !m_valid) return ORC_EINVAL;
    int rc = orc_sample_rvs(t, M, seed, center_lin, m_valid);
    if (rc != 0) return rc;
    int32_t rad = t->g.radius;
    int32_t side = 2 * rad + 1;
    int64_t lambda = (int64_t)side * side * side;
    for (int32_t b = 0; b < t->B && rc == 0; ++b) {
        int32_t nv = t->nvox[b];
        int32_t m = m_valid[b];
        const uint32_t* vl = t->vox_lin + (size_t)b * t->N;
        int32_t* c = center_lin + (size_t)b * M;
        int32_t* inc = (int32_t*)malloc(sizeof(int32_t) * (size_t)m);        /* slot -> voxel (its slot in O_v) */
        unsigned char* initial = (unsigned char*)calloc((size_t)nv, 1);      /* in the RVS choice */
        uint32_t* C = (uint32_t*)calloc((size_t)nv, sizeof(uint32_t));       /* incumbents covering V */
        int32_t* pc = (int32_t*)malloc(sizeof(int32_t) * (size_t)lambda);
        int32_t* pi = (int32_t*)malloc(sizeof(int32_t) * (size_t)lambda);
        if (!inc || !initial || !C || !pc || !pi) {
            rc = ORC_EINVAL;
        } else {
            for (int32_t j = 0; j < m; ++j) {
                inc[j] = find_slot(t, b, (uint32_t)c[j]);
                initial[inc[j]] = 1;
                int32_t n = neighbours(t, b, (uint32_t)c[j], rad, pc);
                for (int32_t k = 0; k < n; ++k) C[pc[k]] += 1;
            }
            uint64_t hb = orc_splitmix64(orc_splitmix64(seed ^ 3ull) ^ (uint64_t)b);
            int32_t tch = 0, swaps = 0;
            for (int32_t v = 0; v < nv; ++v) {
                if (initial[v]) continue;
                int32_t j = (int32_t)((orc_splitmix64(hb ^ (uint64_t)tch) >> 32) % (uint64_t)m);
                int32_t I = inc[j];
                int32_t nc = neighbours(t, b, vl[v], rad, pc);
                int32_t ni = neighbours(t, b, vl[I], rad, pi);
                /* Eq. 2 and Eq. 3, both scaled by 2^16 * lambda */
                int64_t uncovered = 0, covsum = 0, single = 0;
                for (int32_t k = 0; k < nc; ++k) {
                    if (C[pc[k]] == 0) uncovered += 1;
                    covsum += C[pc[k]];
                }
                for (int32_t k = 0; k < ni; ++k)
                    if (C[pi[k]] == 1) single += 1;
                int64_t h_add = 65536LL * lambda * uncovered - (int64_t)beta_q16 * covsum;
                int64_t h_rmv = 65536LL * lambda * single;
                int accept = h_add > h_rmv;
                if (accept) {
                    for (int32_t k = 0; k < ni; ++k) C[pi[k]] -= 1;
                    for (int32_t k = 0; k < nc; ++k) C[pc[k]] += 1;
                    inc[j] = v;
                    ++swaps;
                }
                if (decision) decision[(size_t)b * t->N + tch] = accept ? j : -(j + 1);
                ++tch;
            }
            for (int32_t j = 0; j < m; ++j) c[j] = (int32_t)vl[inc[j]];
            qsort(c, (size_t)m, sizeof(int32_t), cmp_i32);
            pad_cyclic(c, m, M);
            if (n_swaps) n_swaps[b] = swaps;
        }
        free(inc);
        free(initial);
        free(C);
        free(pc);
        free(pi);
    }
    return rc;
}

static uint32_t float_bits(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return u;
}

/* k-NN key of point i from reference q: bits(d^2) << 32 | i. */
static uint64_t knn_key(const float* P, uint64_t i, const float* q) {
    float dx = P[3 * i + 0] - q[0];
    float dy = P[3 * i + 1] - q[1];
    float dz = P[3 * i + 2] - q[2];
    float xx = dx * dx, yy = dy * dy, zz = dz * dz;
    float s = xx + yy;
    float d2 = s + zz;
    return ((uint64_t)float_bits(d2) << 32) | i;
}

/* Appendix D, "CAGQ k-NN" (the level-wise procedure). Level i of pi(v) is
 * the voxels at Chebyshev distance exactly i from v. For level 0, 1, ...:
 * gather the level's stored points (voxels in ascending lin, each voxel's
 * points ascending), kl of them; topkl = min(K - counter, kl); when topkl is
 * kl the whole level is appended as gathered, otherwise the topkl nearest
 * to q (by knn_key, ascending); stop once counter reaches K. The appended
 * points go to nodes[0..counter); layer has room for one level. */
static int32_t knn_by_levels(const orc_table* t, int32_t b, uint32_t l, const float* P, const float* q,
                             int32_t K, uint64_t* layer, int32_t* nodes) {
    const int32_t* D = t->g.dims;
    const int32_t rad = t->g.radius;
    const uint32_t* vo = t->vox_off + (size_t)b * (t->N + 1);
    const uint32_t* pl = t->pt_list + (size_t)b * t->N;
    int32_t gx = (int32_t)(l % (uint32_t)D[0]);
    int32_t gy = (int32_t)((l / (uint32_t)D[0]) % (uint32_t)D[1]);
    int32_t gz = (int32_t)(l / ((uint32_t)D[0] * (uint32_t)D[1]));
    int32_t counter = 0;
    for (int32_t lev = 0; lev <= rad; ++lev) {
        int32_t kl = 0;
        for (int32_t dz = -lev; dz <= lev; ++dz)
            for (int32_t dy = -lev; dy <= lev; ++dy)
                for (int32_t dx = -lev; dx <= lev; ++dx) {
                    int32_t m = abs(dx) > abs(dy) ? abs(dx) : abs(dy);
                    m = abs(dz) > m ? abs(dz) : m;
                    if (m != lev) continue;
                    int32_t x = gx + dx, y = gy + dy, z = gz + dz;
                    if (x < 0 || y < 0 || z < 0 || x >= D[0] || y >= D[1] || z >= D[2]) continue;
                    uint32_t nl = (uint32_t)x + (uint32_t)D[0] * ((uint32_t)y + (uint32_t)D[1] * (uint32_t)z);
                    int32_t sl = find_slot(t, b, nl);
                    if (sl < 0) continue;
                    for (uint32_t u = vo[sl]; u < vo[sl + 1]; ++u) layer[kl++] = pl[u];
                }
        int32_t topkl = K - counter < kl ? K - counter : kl;
        if (topkl == kl) {
            for (int32_t e = 0; e < kl; ++e) nodes[counter + e] = (int32_t)layer[e];
        } else {
            for (int32_t e = 0; e < kl; ++e) layer[e] = knn_key(P, layer[e], q);
            qsort(layer, (size_t)kl, sizeof(uint64_t), cmp_u64);
            for (int32_t e = 0; e < topkl; ++e) nodes[counter + e] = (int32_t)(layer[e] & 0xFFFFFFFFu);
        }
        counter += topkl;
        if (counter >= K) break;
    }
    return counter;
}

int orc_query(const orc_table* t, const float* pts, const uint32_t* weights,
              const int32_t* center_lin, const int32_t* m_valid, int32_t M, int32_t K,
              int32_t mode, uint64_t seed,
              int32_t* node_idx, float* node_xyz, int32_t* n_valid,
              float* center_xyz, uint32_t* center_w, int32_t* ctx_count) {
    if (!table_ok(t) || !pts || !center_lin || !m_valid || M < 1 || K < 1) return ORC_EINVAL;
    if (mode < 0 || mode > 2) return ORC_EINVAL;
    if (!node_idx || !n_valid || !center_xyz || !center_w) return ORC_EINVAL;
    int32_t rad = t->g.radius;
    int32_t side = 2 * rad + 1;
    int32_t lambda = side * side * side;
    int32_t* nbs = (int32_t*)malloc(sizeof(int32_t) * (size_t)lambda);
    uint64_t* key = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)lambda * (size_t)t->g.n_v);
    float* term = (float*)malloc(sizeof(float) * 3 * (size_t)K);
    int32_t* nodes = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
    if (!nbs || !key || !term || !nodes) { free(nbs); free(key); free(term); free(nodes); return ORC_EINVAL; }
    const int32_t* D = t->g.dims;
    int rc = 0;
    for (int32_t b = 0; b < t->B; ++b) {
        const float* P = pts + (size_t)b * t->N * 3;
        const uint32_t* W = weights ? weights + (size_t)b * t->N : NULL;
        const uint32_t* vo = t->vox_off + (size_t)b * (t->N + 1);
        const uint32_t* pl = t->pt_list + (size_t)b * t->N;
        uint64_t hb = orc_splitmix64(orc_splitmix64(seed ^ 2ull) ^ (uint64_t)b);
        for (int32_t j = 0; j < M; ++j) {
            size_t cj = (size_t)b * M + j;
            uint32_t l = (uint32_t)center_lin[cj];
            if (center_lin[cj] < 0 || find_slot(t, b, l) < 0) { rc = ORC_ENOTOCC; continue; }
            /* context points: the stored lists of every voxel of pi(v) */
            int32_t nn = neighbours(t, b, l, rad, nbs);
            int32_t c = 0, nlev = 0;
            for (int32_t q = 0; q < nn; ++q)
                for (uint32_t e = vo[nbs[q]]; e < vo[nbs[q] + 1]; ++e) key[c++] = pl[e];
            if (mode == 0) {
                uint64_t hc = orc_splitmix64(hb ^ (uint64_t)l);
                for (int32_t e = 0; e < c; ++e) {
                    uint64_t i = key[e];
                    uint64_t h = orc_splitmix64(hc ^ i);
                    key[e] = ((h >> 32) << 32) | i;
                }
            } else {
                int32_t g[3];
                g[0] = (int32_t)(l % (uint32_t)D[0]);
                g[1] = (int32_t)((l / (uint32_t)D[0]) % (uint32_t)D[1]);
                g[2] = (int32_t)(l / ((uint32_t)D[0] * (uint32_t)D[1]));
                float q[3];
                for (int a = 0; a < 3; ++a) {
                    float gc = (float)g[a] + 0.5f;
                    float off = gc * t->g.voxel_size[a];
                    q[a] = t->g.origin[a] + off;
                }
                if (mode == 1)
                    for (int32_t e = 0; e < c; ++e) key[e] = knn_key(P, key[e], q);
                else
                    nlev = knn_by_levels(t, b, l, P, q, K, key, nodes);
            }
            if (mode != 2) qsort(key, (size_t)c, sizeof(uint64_t), cmp_u64);
            int32_t n = c < K ? c : K;
            if (mode == 2) {
                n = nlev;
                for (int32_t k = 0; k < n; ++k) key[k] = (uint64_t)(uint32_t)nodes[k];
            }
            int32_t* ni = node_idx + cj * K;
            for (int32_t k = 0; k < K; ++k) ni[k] = (int32_t)(key[k < n ? k : 0] & 0xFFFFFFFFu);
            if (node_xyz)
                for (int32_t k = 0; k < K; ++k)
                    for (int a = 0; a < 3; ++a) node_xyz[(cj * K + k) * 3 + a] = P[3 * (size_t)ni[k] + a];
            /* Eqs. 7-8 over the n valid nodes: w_c = sum w_k; the weighted sum
             * of positions is taken pairwise -- at stride h = 1, 2, 4, ...,
             * entry k (a multiple of 2h) adds entry k + h when k + h < n */
            uint32_t wc = 0;
            for (int32_t k = 0; k < n; ++k) {
                uint32_t w = W ? W[ni[k]] : 1u;
                wc += w;
                float wf = (float)w;
                for (int a = 0; a < 3; ++a) term[a * K + k] = wf * P[3 * (size_t)ni[k] + a];
            }
            for (int32_t h = 1; h < n; h *= 2)
                for (int32_t k = 0; k + h < n; k += 2 * h)
                    for (int a = 0; a < 3; ++a) term[a * K + k] = term[a * K + k] + term[a * K + k + h];
            float wcf = (float)wc;
            for (int a = 0; a < 3; ++a) center_xyz[cj * 3 + a] = term[a * K] / wcf;
            center_w[cj] = wc;
            n_valid[cj] = n;
            if (ctx_count) ctx_count[cj] = c;
        }
    }
    free(nbs);
    free(key);
    free(term);
    free(nodes);
    return rc;
}

/* Upsampling query (Sec. 3.1: in the upsampling layers the centers arrive
 * through long-range connections and CAGQ only queries their node points).
 * Each given center point falls into voxel v by the voxelize rule (v need
 * not be occupied); its context is the stored points of pi(v); the min(K, c)
 * context points of smallest key are kept. Cube key as for orc_query (it
 * depends on v only); k-NN key bits(d^2) << 32 | i with d measured from the
 * center point itself. An empty context gives n = 0 and every slot -1 (xyz
 * 0); otherwise slots k >= n repeat slot 0.
 *   centers [B][M][3]; center_lin [B][M] (may be NULL) receives lin(v). */
int orc_query_points(const orc_table* t, const float* pts, const float* centers, int32_t M, int32_t K,
                     int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz, int32_t* n_valid,
                     int32_t* ctx_count, int32_t* center_lin) {
    if (!table_ok(t) || !pts || !centers || M < 1 || K < 1) return ORC_EINVAL;
    if (mode < 0 || mode > 2) return ORC_EINVAL;
    if (!node_idx || !n_valid) return ORC_EINVAL;
    int32_t rad = t->g.radius;
    int32_t side = 2 * rad + 1;
    int32_t lambda = side * side * side;
    int32_t* nbs = (int32_t*)malloc(sizeof(int32_t) * (size_t)lambda);
    uint64_t* key = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)lambda * (size_t)t->g.n_v);
    int32_t* nodes = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
    if (!nbs || !key || !nodes) { free(nbs); free(key); free(nodes); return ORC_EINVAL; }
    int rc = 0;
    for (int32_t b = 0; b < t->B; ++b) {
        const float* P = pts + (size_t)b * t->N * 3;
        const uint32_t* vo = t->vox_off + (size_t)b * (t->N + 1);
        const uint32_t* pl = t->pt_list + (size_t)b * t->N;
        uint64_t hb = orc_splitmix64(orc_splitmix64(seed ^ 2ull) ^ (uint64_t)b);
        for (int32_t j = 0; j < M; ++j) {
            size_t cj = (size_t)b * M + j;
            const float* q = centers + cj * 3;
            uint32_t l;
            int vr = orc_voxelize(q, 1, &t->g, &l);
            if (vr != 0) rc = vr;
            if (center_lin) center_lin[cj] = (int32_t)l;
            /* context points: the stored lists of every voxel of pi(v) */
            int32_t nn = neighbours(t, b, l, rad, nbs);
            int32_t c = 0;
            for (int32_t e = 0; e < nn; ++e)
                for (uint32_t u = vo[nbs[e]]; u < vo[nbs[e] + 1]; ++u) key[c++] = pl[u];
            if (mode == 0) {
                uint64_t hc = orc_splitmix64(hb ^ (uint64_t)l);
                for (int32_t e = 0; e < c; ++e) {
                    uint64_t i = key[e];
                    uint64_t h = orc_splitmix64(hc ^ i);
                    key[e] = ((h >> 32) << 32) | i;
                }
            } else if (mode == 1) {
                for (int32_t e = 0; e < c; ++e) key[e] = knn_key(P, key[e], q);
            }
            int32_t n = c < K ? c : K;
            if (mode == 2) {
                n = knn_by_levels(t, b, l, P, q, K, key, nodes);
                for (int32_t k = 0; k < n; ++k) key[k] = (uint64_t)(uint32_t)nodes[k];
            } else {
                qsort(key, (size_t)c, sizeof(uint64_t), cmp_u64);
            }
            int32_t* ni = node_idx + cj * K;
            for (int32_t k = 0; k < K; ++k) ni[k] = n ? (int32_t)(key[k < n ? k : 0] & 0xFFFFFFFFu) : -1;
            if (node_xyz)
                for (int32_t k = 0; k < K; ++k)
                    for (int a = 0; a < 3; ++a)
                        node_xyz[(cj * K + k) * 3 + a] = n ? P[3 * (size_t)ni[k] + a] : 0.0f;
            n_valid[cj] = n;
            if (ctx_count) ctx_count[cj] = c;
        }
    }
    free(nbs);
    free(key);
    free(nodes);
    return rc;
}

/* Context lists for grid context pooling (Sec. 3.3: the context feature is
 * pooled over every context point of a group, the points CAGQ already
 * associated with the center voxel). Per center voxel v (any voxel of the
 * grid, occupied or not): the stored points of the occupied voxels of
 * pi(v), voxels in ascending lin, each voxel's stored points ascending.
 *   ctx_off [B*M + 1]: ctx_off[b*M + j] = number of context points of the
 *   centers before (b, j) in batch order; ctx_off[B*M] = the total.
 *   ctx_idx [capacity] (may be NULL): the lists, concatenated in the same
 *   order; entries past capacity are not written (returns -5 then).
 * A lin outside the grid gets an empty list and returns -7. */
int orc_context_list(const orc_table* t, const int32_t* center_lin, int32_t M, int64_t* ctx_off,
                     int32_t* ctx_idx, int64_t capacity) {
    if (!table_ok(t) || !center_lin || M < 1 || !ctx_off || capacity < 0) return ORC_EINVAL;
    int32_t rad = t->g.radius;
    int32_t side = 2 * rad + 1;
    int32_t* nbs = (int32_t*)malloc(sizeof(int32_t) * (size_t)(side * side * side));
    if (!nbs) return ORC_EINVAL;
    const int64_t V = (int64_t)t->g.dims[0] * t->g.dims[1] * t->g.dims[2];
    int rc = 0;
    int64_t total = 0;
    for (int32_t b = 0; b < t->B; ++b) {
        const uint32_t* vo = t->vox_off + (size_t)b * (t->N + 1);
        const uint32_t* pl = t->pt_list + (size_t)b * t->N;
        for (int32_t j = 0; j < M; ++j) {
            size_t cj = (size_t)b * M + j;
            ctx_off[cj] = total;
            int32_t l = center_lin[cj];
            if (l < 0 || (int64_t)l >= V) { rc = ORC_ENOTOCC; continue; }
            int32_t nn = neighbours(t, b, (uint32_t)l, rad, nbs);
            for (int32_t e = 0; e < nn; ++e)
                for (uint32_t u = vo[nbs[e]]; u < vo[nbs[e] + 1]; ++u) {
                    if (ctx_idx && total < capacity) ctx_idx[total] = (int32_t)pl[u];
                    ++total;
                }
        }
    }
    ctx_off[(size_t)t->B * M] = total;
    free(nbs);
    if (rc == 0 && ctx_idx && total > capacity) rc = ORC_ECAPACITY;
    return rc;
}

/* ------------------------------------------------------------------------
 * Comparison methods of Sec. 4 (tab:query): Random Point Sampling, Farthest
 * Point Sampling and Ball Query, and the occupied-space coverage metric.
 * They are what CAGQ is measured against, not CAGQ.
 * ------------------------------------------------------------------------ */

/* d^2 between points a and b, fp32: (dx*dx + dy*dy) + dz*dz. */
static float dist2(const float* a, const float* b) {
    float dx = a[0] - b[0], dy = a[1] - b[1], dz = a[2] - b[2];
    float xx = dx * dx, yy = dy * dy, zz = dz * dz;
    float s = xx + yy;
    return s + zz;
}

/* RPS (mode 0): M input points, every point equally likely -- the M points
 * of smallest key (hi32(h(seed, 4, b, i)) << 32) | i, in ascending index.
 * FPS (mode 1): start at point 0; each next center is the point farthest
 * (largest d^2 to its nearest chosen center; ties to the lowest index) from
 * the chosen ones, in pick order. 1 <= M <= N. center_idx [B][M]. */
int orc_sample_points(const float* pts, int32_t B, int32_t N, int32_t M, int32_t mode, uint64_t seed,
                      int32_t* center_idx) {
    if (!pts || !center_idx || B < 1 || N < 1 || M < 1 || M > N || (mode != 0 && mode != 1)) return ORC_EINVAL;
    uint64_t* key = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)N);
    float* dmin = (float*)malloc(sizeof(float) * (size_t)N);
    if (!key || !dmin) { free(key); free(dmin); return ORC_EINVAL; }
    for (int32_t b = 0; b < B; ++b) {
        const float* P = pts + (size_t)b * N * 3;
        int32_t* c = center_idx + (size_t)b * M;
        if (mode == 0) {
            uint64_t hb = orc_splitmix64(orc_splitmix64(seed ^ 4ull) ^ (uint64_t)b);
            for (int32_t i = 0; i < N; ++i) key[i] = ((orc_splitmix64(hb ^ (uint64_t)i) >> 32) << 32) | (uint32_t)i;
            qsort(key, (size_t)N, sizeof(uint64_t), cmp_u64);
            for (int32_t j = 0; j < M; ++j) key[j] &= 0xFFFFFFFFu;
            qsort(key, (size_t)M, sizeof(uint64_t), cmp_u64);
            for (int32_t j = 0; j < M; ++j) c[j] = (int32_t)key[j];
        } else {
            int32_t cur = 0;
            for (int32_t i = 0; i < N; ++i) dmin[i] = INFINITY;
            for (int32_t j = 0; j < M; ++j) {
                c[j] = cur;
                int32_t best = 0;
                float bd = -1.0f;
                for (int32_t i = 0; i < N; ++i) {
                    float d = dist2(P + 3 * (size_t)i, P + 3 * (size_t)cur);
                    if (d < dmin[i]) dmin[i] = d;
                    if (dmin[i] > bd) { bd = dmin[i]; best = i; }
                }
                cur = best;
            }
        }
    }
    free(key);
    free(dmin);
    return 0;
}

/* Ball Query: per center point, the first K points in index order with
 * d^2 < radius2 (fp32 as dist2) among all N points of its cloud; n_valid =
 * their number; slots k >= n repeat slot 0 (n >= 1 when the center is one
 * of the points). center_idx [B][M], node_idx [B][M][K], n_valid [B][M]. */
int orc_ball_query(const float* pts, int32_t B, int32_t N, const int32_t* center_idx, int32_t M, int32_t K,
                   float radius2, int32_t* node_idx, int32_t* n_valid) {
    if (!pts || !center_idx || !node_idx || !n_valid || B < 1 || N < 1 || M < 1 || K < 1) return ORC_EINVAL;
    for (int32_t b = 0; b < B; ++b) {
        const float* P = pts + (size_t)b * N * 3;
        for (int32_t j = 0; j < M; ++j) {
            size_t cj = (size_t)b * M + j;
            int32_t ci = center_idx[cj];
            if (ci < 0 || ci >= N) return ORC_EINVAL;
            int32_t* ni = node_idx + cj * K;
            int32_t n = 0;
            for (int32_t i = 0; i < N && n < K; ++i)
                if (dist2(P + 3 * (size_t)i, P + 3 * (size_t)ci) < radius2) ni[n++] = i;
            for (int32_t k = n; k < K; ++k) ni[k] = n ? ni[0] : -1;
            n_valid[cj] = n;
        }
    }
    return 0;
}

/* Occupied-space coverage (Sec. 4): per cloud, the number of occupied
 * voxels holding at least one valid node point of any group (the metric is
 * this over |O_v|). node_idx [B][M][K] point indices, n_valid [B][M];
 * covered [B]. */
int orc_coverage(const orc_table* t, const float* pts, const int32_t* node_idx, const int32_t* n_valid, int32_t M,
                 int32_t K, int32_t* covered) {
    if (!table_ok(t) || !pts || !node_idx || !n_valid || !covered || M < 1 || K < 1) return ORC_EINVAL;
    uint32_t* lin = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)t->N);
    uint8_t* hit = (uint8_t*)malloc((size_t)t->N);
    if (!lin || !hit) { free(lin); free(hit); return ORC_EINVAL; }
    int rc = 0;
    for (int32_t b = 0; b < t->B; ++b) {
        orc_voxelize(pts + (size_t)b * t->N * 3, t->N, &t->g, lin);
        memset(hit, 0, (size_t)t->N);
        for (int32_t j = 0; j < M; ++j) {
            size_t cj = (size_t)b * M + j;
            for (int32_t k = 0; k < n_valid[cj] && k < K; ++k) {
                int32_t i = node_idx[cj * K + k];
                if (i < 0 || i >= t->N) { rc = ORC_EINVAL; continue; }
                int32_t s = find_slot(t, b, lin[i]);
                if (s >= 0) hit[s] = 1;
            }
        }
        int32_t n = 0;
        for (int32_t s = 0; s < t->nvox[b]; ++s) n += hit[s];
        covered[b] = n;
    }
    free(lin);
    free(hit);
    return rc;
}
