/*
 * cagq.h -- C ABI of the MI355X (gfx950) Coverage-Aware Grid Query library.
 *
 * CAGQ is the data-structuring stage of Grid-GCN (Xu et al., arXiv
 * 1912.02984, Sec. 3.2; Appendix D, "CAGQ general procedure"): voxelize a
 * batch of point clouds, index the occupied voxels with at most n_v points
 * each, choose M center voxels (Random Voxel Sampling or Coverage-Aware
 * Sampling) and gather K node points per center from its (2r+1)^3 voxel
 * neighbourhood (Cube Query or k-NN), then form each group's center
 * (Appendix E, Eqs. 7-8).
 *
 * Conventions for every entry point:
 *   - Pointers named "device" are HIP device pointers owned by the caller;
 *     the library never allocates or frees device memory and keeps no
 *     pointer to caller memory past a call (a cagq_grid record borrows the
 *     caller's points and workspace; it is the caller's). Host pointers are
 *     read before the call returns. One exception holds host memory: the
 *     many-kernel CAS path (cagq_sample_centers) keeps one 64-byte pinned
 *     host block per calling thread, allocated at its first use and kept
 *     until the process ends, through which its round kernels report
 *     progress to the waiting host thread.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued asynchronously on it; results are valid once the
 *     stream has reached the enqueued work. cagq_sample_centers with the
 *     CAS mode may block the calling thread until its rounds finish (see
 *     there); such a call cannot be captured into a HIP graph.
 *   - Argument errors are detected on the host before anything is
 *     enqueued and returned synchronously. Data-dependent errors
 *     (non-finite coordinates, center voxels that are not occupied) are
 *     recorded in the workspace and reported by cagq_get_device_status.
 *   - Calls on one workspace are ordered by the stream; distinct
 *     workspaces are independent. The library's only state beyond the
 *     caller's memory is the pinned block above (each call on it is told
 *     apart by a per-call tag) and per-device kernel attributes it caches.
 *   - Array shapes are row-major; [B][N][3] means point n of cloud b has
 *     x, y, z at ((b*N)+n)*3 + {0,1,2}.
 */
#ifndef CAGQ_H
#define CAGQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Symbols of the C ABI are the only ones the shared library exports. */
#if defined(__GNUC__) || defined(__clang__)
#define CAGQ_API __attribute__((visibility("default")))
#else
#define CAGQ_API
#endif

/* Status codes. */
#define CAGQ_OK 0
#define CAGQ_ERR_INVALID_ARG (-1)       /* a pointer, size or mode out of range */
#define CAGQ_ERR_GRID_TOO_LARGE (-2)    /* D_x*D_y*D_z > 2^31-1 */
#define CAGQ_ERR_WORKSPACE_TOO_SMALL (-3)
#define CAGQ_ERR_NONFINITE_INPUT (-4)   /* device-side: a NaN/Inf coordinate */
#define CAGQ_ERR_CAPACITY (-5)          /* device-side: an internal table or an output overflowed */
#define CAGQ_ERR_HIP (-6)               /* a HIP runtime call failed */
#define CAGQ_ERR_CENTER_NOT_OCCUPIED (-7) /* device-side: a query center is not in O_v (or not in the grid) */

#define CAGQ_SAMPLE_RVS 0   /* Random Voxel Sampling (Sec. 3.2) */
#define CAGQ_SAMPLE_CAS 1   /* Coverage-Aware Sampling, greedy (Sec. 3.2, Eqs. 1-2) */
#define CAGQ_SAMPLE_CAS_SWAP 2  /* Coverage-Aware Sampling, challenger / incumbent swaps (Sec. 3.2, Eqs. 2-3) */
#define CAGQ_QUERY_CUBE 0   /* Cube Query (Sec. 3.2) */
#define CAGQ_QUERY_KNN 1    /* k-NN among the context points (Sec. 3.2) */
#define CAGQ_QUERY_KNN_RING 2  /* level-wise k-NN (Appendix D, "CAGQ k-NN"); approximate */

#define CAGQ_POINTS_RPS 0   /* Random Point Sampling (comparison method, Sec. 4) */
#define CAGQ_POINTS_FPS 1   /* Farthest Point Sampling (comparison method, Sec. 4) */

/* Library limits (checked on the host). */
#define CAGQ_MAX_K 128      /* node points per group */
#define CAGQ_MAX_NV 64      /* points stored per voxel */
#define CAGQ_MAX_RADIUS 3   /* neighbourhood half-width r */

/*
 * Voxel grid (Sec. 3.2: "voxelize the input space by setting up a voxel size
 * (v_x, v_y, v_z)"). A point p maps, per axis a, to
 *   g_a = clamp(floor((p_a - origin_a) / voxel_size_a), 0, dims_a - 1)
 * (fp32 subtract then fp32 correctly rounded divide; points outside the
 * grid are clamped onto its border voxels, never dropped), and to the
 * linear id lin = g_x + D_x * (g_y + D_y * g_z).
 * n_v: at most n_v points are stored per voxel (1..CAGQ_MAX_NV).
 * radius: pi(v) is the (2r+1)^3 block of voxels around v (1..CAGQ_MAX_RADIUS).
 */
typedef struct cagq_grid_desc {
    float origin[3];
    float voxel_size[3];   /* > 0 and finite */
    int32_t dims[3];       /* >= 1, product <= 2^31-1 */
    int32_t n_v;
    int32_t radius;
} cagq_grid_desc;

/*
 * Byte offsets of the arrays a built grid exposes inside the caller's
 * workspace (each 256-byte aligned), and the total size the workspace needs.
 *   nvox      int32  [B]           |O_v| per cloud
 *   vox_lin   uint32 [B][N]        lin of slot s; slots are ranks of lin, so
 *                                  ascending; entries s < nvox[b] are valid
 *   vox_count uint32 [B][N]        points falling in slot s
 *   vox_off   uint32 [B][N+1]      exclusive prefix of min(count, n_v); entry
 *                                  nvox[b] holds the stored total S_b
 *   pt_list   uint32 [B][N]        stored point indices (0..N-1): slot s owns
 *                                  [vox_off[s], vox_off[s+1]), the
 *                                  min(count, n_v) lowest indices ascending
 */
typedef struct cagq_layout {
    size_t total_bytes;
    size_t nvox, vox_lin, vox_count, vox_off, pt_list;
} cagq_layout;

/*
 * A built grid: a host-side record borrowing the caller's points and
 * workspace. Filled by cagq_build_grid; valid while both stay alive and the
 * workspace is not rebuilt.
 */
typedef struct cagq_grid {
    int32_t B, N;
    cagq_grid_desc desc;
    const float* points;   /* device [B][N][3], borrowed */
    void* workspace;       /* device, borrowed */
    size_t workspace_bytes;
} cagq_grid;

/*
 * Grid descriptors from a bounding box (host only, pure: no device work, no
 * state). Sec. 3.2 voxelizes the input space "by setting up a voxel size
 * (v_x, v_y, v_z)"; these helpers fix the origin and extent it leaves open.
 * lo, hi: host float[3], the box's corners (finite, lo_a <= hi_a).
 *
 * cagq_desc_from_voxel_size: origin = lo, voxel_size = vs (host float[3],
 *   > 0 and finite), and per axis dims_a = floor(t_a) + 1 with t_a =
 *   (hi_a - lo_a) / vs_a in fp32 (one rounded subtract, one correctly
 *   rounded divide: the voxelize rule of cagq_grid_desc). The voxelize rule
 *   then puts lo in voxel 0 and hi in voxel dims_a - 1 on every axis, so no
 *   point of [lo, hi] is clamped; it is the smallest such grid at origin lo.
 * cagq_desc_from_dims: origin = lo, dims = dims (host int32[3], >= 1), and
 *   voxel_size_a = (hi_a - lo_a) / dims_a in fp32 (correctly rounded), or 1
 *   when hi_a == lo_a. A point of [lo, hi] whose quotient rounds up to dims_a
 *   is clamped onto the last voxel by the voxelize rule.
 * Both copy n_v and radius into `out` (host) and validate the result as
 * cagq_build_grid does. Return CAGQ_OK; CAGQ_ERR_INVALID_ARG for a null
 * pointer, a non-finite or inverted box, a voxel size that is not positive
 * and finite (given or computed), or n_v / radius out of range;
 * CAGQ_ERR_GRID_TOO_LARGE when a dimension or the voxel count exceeds
 * 2^31-1. `out` is written only on CAGQ_OK.
 */
CAGQ_API int cagq_desc_from_voxel_size(const float lo[3], const float hi[3], const float vs[3], int32_t n_v,
                                       int32_t radius, cagq_grid_desc* out);
CAGQ_API int cagq_desc_from_dims(const float lo[3], const float hi[3], const int32_t dims[3], int32_t n_v,
                                 int32_t radius, cagq_grid_desc* out);

/* Host only, no device work. Fills `out` for a batch of B clouds of N points
 * on `desc`. Returns CAGQ_OK, CAGQ_ERR_INVALID_ARG or CAGQ_ERR_GRID_TOO_LARGE. */
CAGQ_API int cagq_workspace_layout(int32_t B, int32_t N, const cagq_grid_desc* desc, cagq_layout* out);

/*
 * Voxelize and index a batch (Appendix D, general procedure, step 1: for each
 * point, quantize it to its voxel, add the voxel to O_v on its first visit,
 * and push the point index while the voxel stores fewer than n_v points).
 * The stored points of a voxel are its n_v lowest point indices, the ones a
 * sequential pass visits first.
 *   points     device float [B][N][3]
 *   workspace  device, >= cagq_workspace_layout(...).total_bytes bytes,
 *              no alignment requirement beyond 256 bytes
 *   out        host; receives the grid record
 * 1 <= B, 1 <= N, B*N <= 2^31-1. A non-finite coordinate is clamped to voxel
 * 0 on that axis and raises CAGQ_ERR_NONFINITE_INPUT in the device status.
 */
CAGQ_API int cagq_build_grid(const float* points, int32_t B, int32_t N, const cagq_grid_desc* desc,
                    void* workspace, size_t workspace_bytes, void* stream, cagq_grid* out);

/*
 * cagq_build_grid without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc). The same build, bit for bit, into a
 * library-owned array of CAGQ_STATIC_WORKSPACE_BYTES per GPU, resident from
 * the library's load until the process ends; the call itself allocates
 * nothing. `out` borrows the array of the current device (its workspace is
 * that array's device address). Every grid built this way on one GPU shares
 * that array: a build overwrites the previous one (whose grid record is
 * then stale), and calls that overlap on one GPU race. The build clears
 * what must start at zero itself. Sampling and querying take the grid like
 * any other; with RVS, or CAS on clouds of at most 4096 points, nothing on
 * the path allocates.
 * Returns CAGQ_ERR_WORKSPACE_TOO_SMALL when cagq_workspace_layout's
 * total_bytes exceeds CAGQ_STATIC_WORKSPACE_BYTES (for example B = 1 with
 * 81920 points on a 168x168x68 grid fits, B = 2 does not), otherwise the
 * errors of cagq_build_grid.
 */
#define CAGQ_STATIC_WORKSPACE_BYTES (64u << 20)
CAGQ_API int cagq_build_grid_static(const float* points, int32_t B, int32_t N, const cagq_grid_desc* desc,
                                    void* stream, cagq_grid* out);

/*
 * Choose M center voxels per cloud (Sec. 3.2, "center voxels sampling";
 * Appendix D step 2). m_valid[b] = min(M, nvox[b]) distinct voxels are chosen
 * and written as linear ids in ascending order to center_lin[b][0..m_valid);
 * slots j >= m_valid repeat center_lin[b][j mod m_valid].
 *   mode CAGQ_SAMPLE_RVS: every occupied voxel equally likely. Slot s gets the
 *     key (hi32(h(seed,1,b,s)) << 32) | s, h the splitmix64 chain
 *     h(seed,t,a1..ak) = sm64(..sm64(sm64(seed ^ t) ^ a1).. ^ ak); the
 *     m_valid smallest keys are chosen.
 *   mode CAGQ_SAMPLE_CAS: coverage-aware greedy (Eqs. 1-2): repeatedly take
 *     the unchosen voxel v maximising
 *       2^16*lambda*#{V in pi(v): C_V = 0} - beta_q16 * sum_{V in pi(v)} C_V
 *     (C_V = chosen voxels whose neighbourhood holds V, lambda = (2r+1)^3,
 *     beta = beta_q16 / 2^16), ties to the lowest lin; the first m_valid
 *     picks are the centers. Requires (2^16 + beta_q16) * lambda^2 < 2^31.
 *     `seed` is unused. With beta_q16 = 0, r <= 2 and N <= 4096 (one
 *     workgroup per cloud holds the whole state) the call is asynchronous.
 *     Otherwise (r <= 2 only: r = 3 returns CAGQ_ERR_INVALID_ARG) its round
 *     count is data dependent: the calling thread issues rounds and spins
 *     until the kernels report every cloud done (without synchronising
 *     `stream` as a whole); up to two rounds with nothing left to do may
 *     still be queued when it returns. On an error return it first waits
 *     for the rounds it queued.
 *   mode CAGQ_SAMPLE_CAS_SWAP: the paper's own procedure (Eqs. 2-3). The
 *     m_valid incumbents start as the RVS choice for `seed`, held in slots
 *     0..m_valid-1 in ascending lin; every other occupied voxel C, in
 *     ascending lin, challenges slot hi32(h(seed,3,b,t)) mod m_valid (t =
 *     0, 1, ... counts the challenges) holding incumbent I, and replaces it
 *     when
 *       2^16*lambda*#{V in pi(C): C_V = 0} - beta_q16 * sum_{V in pi(C)} C_V
 *         > 2^16*lambda*#{V in pi(I): C_V = 1}
 *     with C_V the incumbents whose neighbourhood holds V. A replaced
 *     incumbent does not challenge again. The procedure is sequential (one
 *     workgroup per cloud walks the challengers); the call only enqueues.
 *     Both sides are compared as 64-bit integers (any beta_q16, r <= 3).
 *     Requires 4*M + 4*ceil(N/32) + (r <= 2 ? 1 : 2) * N <= 159728 bytes
 *     (the state one workgroup holds), else returns CAGQ_ERR_CAPACITY.
 *   center_lin  device int32 [B][M];  m_valid  device int32 [B]
 */
CAGQ_API int cagq_sample_centers(const cagq_grid* g, int32_t M, int32_t mode, uint64_t seed,
                        uint32_t beta_q16, int32_t* center_lin, int32_t* m_valid,
                        void* stream);

/*
 * Gather K node points per center and form the group centers (Sec. 3.2 node
 * points querying; Appendix D step 3; Appendix E). The context of center
 * voxel v is the stored points of the occupied voxels of pi(v) (v included);
 * c = their number. The n = min(K, c) context points of smallest 64-bit key
 * are kept in ascending key order:
 *   CAGQ_QUERY_CUBE: key = (hi32(h(seed,2,b,lin(v),i)) << 32) | i  (random subset)
 *   CAGQ_QUERY_KNN:  key = (bits(d2) << 32) | i, d2 = (dx*dx + dy*dy) + dz*dz
 *                    in fp32 from q_a = origin_a + ((float)g_a + 0.5f) * voxel_size_a
 *   CAGQ_QUERY_KNN_RING: the level-wise procedure of Appendix D. Level l of
 *                    pi(v) is the voxels at Chebyshev distance exactly l; for
 *                    l = 0, 1, ..., r a level whose points fit in what is
 *                    left of K is taken whole, in gathering order (voxels by
 *                    ascending lin, stored points ascending), otherwise its
 *                    nearest points by the CAGQ_QUERY_KNN key; the search
 *                    stops at K. Approximate: a level-1 point can be nearer
 *                    than a level-0 one. Nodes are kept in that order.
 * Node slots k >= n repeat slot 0. Group center (Eqs. 7-8):
 *   w_c = sum of the n node weights (uint32);
 *   chi_c = S / (float)w_c per axis, S the fp32 pairwise sum of
 *   (float)w_k * p_k over the n nodes: at stride h = 1, 2, 4, ..., entry k
 *   (k a multiple of 2h) adds entry k + h when k + h < n.
 *   weights     device uint32 [B][N] or NULL (all 1: raw points)
 *   center_lin  device int32 [B][M], every entry an occupied voxel's lin
 *   node_idx    device int32 [B][M][K]    point indices 0..N-1
 *   node_xyz    device float [B][M][K][3] or NULL; bit copies of the points
 *   n_valid     device int32 [B][M]
 *   center_xyz  device float [B][M][3]
 *   center_w    device uint32 [B][M]
 *   ctx_count   device int32 [B][M] or NULL; c
 * 1 <= K <= CAGQ_MAX_K. A center that is not occupied raises
 * CAGQ_ERR_CENTER_NOT_OCCUPIED in the device status; its outputs are zero.
 */
CAGQ_API int cagq_query_context(const cagq_grid* g, const uint32_t* weights, const int32_t* center_lin,
                       int32_t M, int32_t K, int32_t mode, uint64_t seed,
                       int32_t* node_idx, float* node_xyz, int32_t* n_valid,
                       float* center_xyz, uint32_t* center_w, int32_t* ctx_count,
                       void* stream);

/*
 * Upsampling query (Sec. 3.1: in the upsampling layers the group centers
 * arrive through long-range connections, and CAGQ only queries their node
 * points). Center point q falls into voxel v by the voxelize rule of
 * cagq_grid_desc; v need not be occupied. The context is the stored points
 * of the occupied voxels of pi(v), c points; the n = min(K, c) of smallest
 * 64-bit key are kept in ascending key order:
 *   CAGQ_QUERY_CUBE: key = (hi32(h(seed,2,b,lin(v),i)) << 32) | i, as in
 *                    cagq_query_context (it depends on v only)
 *   CAGQ_QUERY_KNN:  key = (bits(d2) << 32) | i, d2 = (dx*dx + dy*dy) + dz*dz
 *                    in fp32 with d = p_i - q, the center point itself
 *   CAGQ_QUERY_KNN_RING: the level-wise procedure (see cagq_query_context)
 *                    with distances from q
 * Node slots k >= n repeat slot 0; an empty context (c = 0) gives n = 0, -1
 * in every node slot and zero coordinates. No group center is formed.
 *   centers     device float [B][M][3]
 *   node_idx    device int32 [B][M][K]
 *   node_xyz    device float [B][M][K][3] or NULL; bit copies of the points
 *   n_valid     device int32 [B][M]
 *   ctx_count   device int32 [B][M] or NULL; c
 *   center_lin  device int32 [B][M] or NULL; lin(v), for cagq_context_*
 * 1 <= K <= CAGQ_MAX_K. A non-finite center coordinate maps to voxel 0 on
 * that axis and raises CAGQ_ERR_NONFINITE_INPUT in the device status.
 */
CAGQ_API int cagq_query_points(const cagq_grid* g, const float* centers, int32_t M, int32_t K, int32_t mode,
                               uint64_t seed, int32_t* node_idx, float* node_xyz, int32_t* n_valid,
                               int32_t* ctx_count, int32_t* center_lin, void* stream);

/*
 * Context lists for grid context pooling (Sec. 3.3: a group's context
 * feature is pooled over all of its context points, which CAGQ has already
 * associated with the center voxel). The context of center voxel v (any
 * voxel of the grid, occupied or not) is the stored points of the occupied
 * voxels of pi(v), voxels in ascending lin, each voxel's stored points in
 * ascending index. Two calls:
 *   cagq_context_offsets writes ctx_off, device int64 [B*M + 1]:
 *     ctx_off[b*M + j] = the number of context points of all centers before
 *     (b, j) in batch order, ctx_off[B*M] = the total T.
 *   cagq_context_list writes ctx_idx, device int32 [capacity]: entries
 *     [ctx_off[b*M+j], ctx_off[b*M+j+1]) hold the context of center (b, j)
 *     as point indices 0..N-1 of cloud b. ctx_off must hold the offsets of
 *     the same centers (enqueued before on the stream). Entries at or past
 *     `capacity` are not written; then CAGQ_ERR_CAPACITY is raised in the
 *     device status. Read ctx_off[B*M] to size ctx_idx.
 *   center_lin  device int32 [B][M]; a lin outside [0, D_x*D_y*D_z) gets an
 *               empty context and raises CAGQ_ERR_CENTER_NOT_OCCUPIED.
 */
CAGQ_API int cagq_context_offsets(const cagq_grid* g, const int32_t* center_lin, int32_t M, int64_t* ctx_off,
                                  void* stream);
CAGQ_API int cagq_context_list(const cagq_grid* g, const int32_t* center_lin, int32_t M, const int64_t* ctx_off,
                               int32_t* ctx_idx, int64_t capacity, void* stream);

/*
 * The comparison methods of Sec. 4 (the latency and coverage tables): what
 * CAGQ replaces, provided to measure it against. They work on raw points
 * and need no grid.
 * cagq_sample_points chooses M of the N points of each cloud:
 *   CAGQ_POINTS_RPS: Random Point Sampling, every point equally likely: the
 *     M points of smallest key (hi32(h(seed,4,b,i)) << 32) | i (h as in
 *     cagq_sample_centers), in ascending index;
 *   CAGQ_POINTS_FPS: Farthest Point Sampling from point 0: each next center
 *     is the point whose d^2 to its nearest chosen center is largest (ties
 *     to the lowest index), in pick order; one workgroup per cloud keeps
 *     the distances in registers, so N <= 81920.
 *   points [B][N][3], center_idx [B][M] (point indices), 1 <= M <= N.
 * cagq_ball_query: per center point p_c, the first K points in index order
 *   with d^2 < radius2 among all N points of its cloud (the O(MN) search);
 *   n_valid = their number; slots k >= n repeat slot 0. A center index
 *   outside [0, N) gets n = 0 and -1 in every slot.
 *   center_idx [B][M], node_idx [B][M][K], n_valid [B][M].
 * d^2 = (dx*dx + dy*dy) + dz*dz in fp32 throughout.
 */
CAGQ_API int cagq_sample_points(const float* points, int32_t B, int32_t N, int32_t M, int32_t mode, uint64_t seed,
                                int32_t* center_idx, void* stream);
CAGQ_API int cagq_ball_query(const float* points, int32_t B, int32_t N, const int32_t* center_idx, int32_t M,
                             int32_t K, float radius2, int32_t* node_idx, int32_t* n_valid, void* stream);

/*
 * Occupied-space coverage (Sec. 4: the voxels occupied by the node points of
 * all groups over the voxels occupied by the N points), on the voxels of a
 * built grid: covered[b] = the occupied voxels of cloud b holding at least
 * one valid node point (node slots k < n_valid); the metric is covered[b] /
 * nvox[b]. Node indices refer to the grid's points; any method's nodes
 * qualify (cagq_query_*, cagq_ball_query).
 *   node_idx device int32 [B][M][K], n_valid device int32 [B][M],
 *   covered  device int32 [B]. Uses the grid's workspace.
 */
CAGQ_API int cagq_coverage(const cagq_grid* g, const int32_t* node_idx, const int32_t* n_valid, int32_t M,
                           int32_t K, int32_t* covered, void* stream);

/* Synchronises `stream` and returns the first device-side error recorded in
 * g's workspace since it was last built (CAGQ_OK if none). */
CAGQ_API int cagq_get_device_status(const cagq_grid* g, void* stream);

/* Static, human-readable name of a status code. */
CAGQ_API const char* cagq_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif
