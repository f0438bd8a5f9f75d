/*
 * CAGQ CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded C99 statement of what Coverage-Aware Grid
 * Query computes (Xu et al., "Grid-GCN for Fast and Scalable Point Cloud
 * Learning", Sec. 3.2, Appendix D "Algorithms of CAGQ" -- the general
 * procedure and the k-NN procedure -- and Appendix E, Eqs. 7-8). Only the
 * test-suite, the smoke check and the benchmark's CPU-baseline leg may load
 * it. It shares no code, header or constant with the HIP library.
 *
 * All pointers are host pointers. Shapes are row-major. Every function
 * returns 0 on success or a negative code:
 *   -1 invalid argument, -4 non-finite coordinate, -5 output capacity
 *   exceeded, -7 center voxel not occupied (or outside the grid).
 *
 * Parity pins (what each function is checked against, beyond itself) are
 * listed in the header comment of cagq_oracle.c.
 */
#ifndef CAGQ_ORACLE_H
#define CAGQ_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    float origin[3];      /* grid corner o_a */
    float voxel_size[3];  /* voxel edge s_a (the paper's v_x, v_y, v_z) */
    int32_t dims[3];      /* D_x, D_y, D_z */
    int32_t n_v;          /* max points stored per voxel */
    int32_t radius;       /* neighbourhood half-width r: (2r+1)^3 voxels */
} orc_grid;

/* The occupied-voxel table of a batch (all arrays host, caller-owned). */
typedef struct {
    int32_t B, N;
    orc_grid g;
    const int32_t* nvox;        /* [B] |O_v| */
    const uint32_t* vox_lin;    /* [B][N] linear id of slot s (ascending) */
    const uint32_t* vox_count;  /* [B][N] full point count of slot s */
    const uint32_t* vox_off;    /* [B][N+1] exclusive prefix of min(count, n_v) */
    const uint32_t* pt_list;    /* [B][N] stored point indices, per slot ascending */
} orc_table;

uint64_t orc_splitmix64(uint64_t x);

/* Linear voxel id of each of n points [n][3]. */
int orc_voxelize(const float* pts, int64_t n, const orc_grid* g, uint32_t* lin);

/* Occupied-voxel table (Algorithm "CAGQ general procedure", step 1). */
int orc_build_table(const float* pts, int32_t B, int32_t N, const orc_grid* g,
                    int32_t* nvox, uint32_t* vox_lin, uint32_t* vox_count,
                    uint32_t* vox_off, uint32_t* pt_list);

/* Random Voxel Sampling (Sec. 3.2): center_lin [B][M], m_valid [B]. */
int orc_sample_rvs(const orc_table* t, int32_t M, uint64_t seed,
                   int32_t* center_lin, int32_t* m_valid);

/* Coverage-Aware Sampling, greedy reading of Eqs. 1-2: center_lin [B][M] in
 * ascending lin, m_valid [B]; pick_lin / pick_score [B][M] (each may be
 * NULL) receive the picks in pick order and their integer score at the
 * time they were picked. */
int orc_sample_cas(const orc_table* t, int32_t M, uint32_t beta_q16,
                   int32_t* center_lin, int32_t* m_valid,
                   int32_t* pick_lin, int64_t* pick_score);

/* Coverage-Aware Sampling, the paper's challenger / incumbent procedure
 * (Sec. 3.2, Eqs. 2-3), starting from the RVS choice: center_lin [B][M] in
 * ascending lin, m_valid [B]; decision [B][N] (may be NULL) per challenge t
 * the slot challenged, >= 0 if the swap was accepted, -(slot + 1) if not;
 * n_swaps [B] (may be NULL) the accepted swaps. */
int orc_sample_cas_swap(const orc_table* t, int32_t M, uint64_t seed, uint32_t beta_q16,
                        int32_t* center_lin, int32_t* m_valid, int32_t* decision, int32_t* n_swaps);

/* Node query (Sec. 3.2: Cube Query when mode == 0, k-NN when mode == 1, the
 * level-wise k-NN of Appendix D when mode == 2) and
 * group centers (Appendix E). weights [B][N] may be NULL (all 1). */
int orc_query(const orc_table* t, const float* pts, const uint32_t* weights,
              const int32_t* center_lin, const int32_t* m_valid, int32_t M, int32_t K,
              int32_t mode, uint64_t seed,
              int32_t* node_idx, float* node_xyz, int32_t* n_valid,
              float* center_xyz, uint32_t* center_w, int32_t* ctx_count);

/* Upsampling query (Sec. 3.1): node points around given center points
 * [B][M][3]; k-NN distances from the center point; an empty context gives
 * n_valid 0 and -1 in every node slot. ctx_count, center_lin [B][M] and
 * node_xyz may be NULL. */
int orc_query_points(const orc_table* t, const float* pts, const float* centers, int32_t M, int32_t K,
                     int32_t mode, uint64_t seed, int32_t* node_idx, float* node_xyz, int32_t* n_valid,
                     int32_t* ctx_count, int32_t* center_lin);

/* Context lists (Sec. 3.3, grid context pooling): ctx_off [B*M + 1] CSR
 * offsets over the batch, ctx_idx [capacity] (may be NULL) the point
 * indices, per center the voxels of pi(v) in ascending lin. */
int orc_context_list(const orc_table* t, const int32_t* center_lin, int32_t M, int64_t* ctx_off,
                     int32_t* ctx_idx, int64_t capacity);

/* Comparison methods of Sec. 4 and the coverage metric (not CAGQ).
 * orc_sample_points: mode 0 Random Point Sampling (M smallest
 * hi32(h(seed,4,b,i)) << 32 | i, ascending index), mode 1 Farthest Point
 * Sampling from point 0 (pick order); 1 <= M <= N; center_idx [B][M]. */
int orc_sample_points(const float* pts, int32_t B, int32_t N, int32_t M, int32_t mode, uint64_t seed,
                      int32_t* center_idx);

/* Ball Query: the first K points in index order with d^2 < radius2 around
 * each center point; slots past n repeat slot 0 (-1 when n = 0). */
int orc_ball_query(const float* pts, int32_t B, int32_t N, const int32_t* center_idx, int32_t M, int32_t K,
                   float radius2, int32_t* node_idx, int32_t* n_valid);

/* Occupied-space coverage (Sec. 4): covered [B] = occupied voxels holding a
 * valid node point (the metric is covered / nvox). */
int orc_coverage(const orc_table* t, const float* pts, const int32_t* node_idx, const int32_t* n_valid, int32_t M,
                 int32_t K, int32_t* covered);

#ifdef __cplusplus
}
#endif
#endif
