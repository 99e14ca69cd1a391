/*
 * mpm.h -- C ABI of the Mutual Pair Merging (MPM) token-reduction path,
 * implemented with hand-written HIP kernels for MI355X (gfx950, CDNA4).
 *
 * MPM (arXiv 2604.05718, Sec. 3.2, Alg. 1) reduces the N x D image tokens of a
 * ViT block input:
 *   1. normalise each token to unit L2 norm and form the cosine affinity
 *      S = Xn Xn^T with the diagonal excluded (Eq. 1);
 *   2. b(i) = argmax_{j != i} S_ij;
 *   3. keep the mutual pairs (b(b(i)) = i), lower index as representative;
 *   4. give clusters (pairs and singletons) compact ids r(i) by a
 *      left-to-right scan (Alg. 1), partners inherit the representative's id;
 *   5. replace each cluster by the mean of its members (Eq. 2).
 * Merge maps of successive insertions compose as r*(i) = r2(r1(i)) (Eq. 3),
 * and the full grid is rebuilt by a gather Z_up[i] = Z[r*(i)] (Eq. 4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All array pointers are DEVICE pointers owned by the caller. The library
 *   allocates and frees nothing.
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *   stream) and never synchronises the host. Counts and offsets stay on the
 *   device; the caller reads them when it needs them.
 * - Token rows are D contiguous elements; rows are 16-byte aligned
 *   (D % 8 == 0 for bfloat16, D % 4 == 0 for float32) and base pointers are
 *   16-byte aligned.
 * - A batch holds B images of at most N tokens each. Token rows are either
 *   DENSE (offsets pointer NULL: image b owns rows [b*N, b*N + N)) or PACKED
 *   (offsets pointer = device int32[B+1], image b owns rows
 *   [off[b], off[b+1]), n_b = off[b+1] - off[b] with 0 <= n_b <= N, offsets
 *   non-decreasing). An empty image (n_b = 0) gets no merged rows and a map of
 *   -1. Packed offsets are data on the device; violating these rules is
 *   undefined behaviour, not a reported error.
 * - Per-token integer arrays (nb, map) use a [B][N] slot layout: entry
 *   b*N + i belongs to token i of image b, for i < n_b. Ids are 0-based and
 *   image-local.
 * - Ties: the argmax keeps the lowest index j among equal scores.
 * - `schedule` (an mpm_schedule value) picks the affinity kernel's work
 *   decomposition for that call only; results never depend on it.
 * - Argument errors are reported synchronously, before anything is launched:
 *     MPM_ERR_INVALID_ARG  null or misaligned pointer, B < 1, N < 1, D < 1,
 *                          D not a multiple of 8 (bf16) / 4 (f32), bad dtype,
 *                          unknown schedule;
 *     MPM_ERR_UNSUPPORTED  N above MPM_MAX_N, B above MPM_MAX_B, D above MPM_MAX_D;
 *     MPM_ERR_WORKSPACE    workspace smaller than mpm_workspace_bytes;
 *     MPM_ERR_HIP          a launch failed; mpm_last_hip_error() holds the
 *                          hipError_t (per host thread).
 *   Device-side faults surface at the caller's next synchronisation.
 * - Results are deterministic: the same inputs give bitwise-identical outputs.
 * - Reentrant: no mutable global state besides the per-thread last HIP error
 *   and, for mpm_merge_noalloc and the checked mode below, the device address of
 *   a library array per GPU (set once). Calls that share a workspace must be
 *   ordered (one stream, or events).
 * - Fault injection: with MPM_FAULT_INJECT=launch in the environment (read once,
 *   at the first call), every entry point that would launch a kernel returns
 *   MPM_ERR_HIP with hipErrorLaunchFailure recorded, after its argument checks and
 *   before any HIP call, so that callers' error paths can be tested without a GPU.
 * - Checked mode (debugging): with MPM_CHECKED=1 in the environment (read once, at
 *   the first call), every entry point also validates on the device the data
 *   preconditions that are otherwise undefined behaviour, before launching its
 *   operation: packed offsets (0 <= n_b <= N; merged-row offsets also at most the
 *   tokens they come from, within B*N rows; the padded layout's any n_b >= 0), token
 *   values and given inverse norms (finite; norms positive), grid positions (in
 *   range, rows non-decreasing), neighbours (in [0, n_b), not the token itself, -1
 *   for a one-token image), merged-row sources (in [0, n_b)) and maps (in [-1, N),
 *   or [-1, n_z) where they index merged rows). Offsets are validated first; the
 *   rows they address must exist. On a violation the call returns
 *   MPM_ERR_INVALID_ARG and launches nothing of its operation. A checked call
 *   synchronises its stream (it reads the verdict back; so not under graph
 *   capture), and checked calls are serialised by a lock. Without the variable
 *   nothing of this runs.
 */
#ifndef MPM_H
#define MPM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MPM_OK = 0,
    MPM_ERR_INVALID_ARG = 1,
    MPM_ERR_UNSUPPORTED = 2,
    MPM_ERR_WORKSPACE = 3,
    MPM_ERR_HIP = 4
} mpm_status;

typedef enum {
    MPM_F32 = 0,   /* float32 storage, float32 arithmetic */
    MPM_BF16 = 1   /* bfloat16 storage, float32 accumulation */
} mpm_dtype;

/*
 * Work schedule of the affinity kernel. The affinity of an image is symmetric
 * (Eq. 1), so MPM_SCHEDULE_SYMMETRIC computes only the 256 x 256 blocks on and
 * above the block diagonal and takes each off-diagonal block's argmax in both
 * directions (about half the matrix-core work for large images, for a
 * cross-lane reduction per block); when an XCD group's blocks would leave a
 * last round on at most half of its workgroups (rows a whole number of
 * 128-byte chunks), that many diagonal blocks run in a second launch as two
 * halves of their queries each. MPM_SCHEDULE_FULL_64 computes every pair of
 * 64 x 64 blocks, so that a small batch (a single image of 1024 tokens has 16
 * blocks of 256 x 256 but 256 of 64 x 64) still occupies every compute unit.
 * MPM_SCHEDULE_AUTO takes the 64 x 64 blocks when the batch has at most 32
 * blocks of 256 x 256, else the symmetric schedule when it needs fewer work
 * rounds on the device's compute units, else the full one. The choice applies
 * to rows whose byte length is a multiple of 64; other rows use a kernel
 * without one. The partials (and everything reduced from them) are
 * bit-identical under every schedule.
 */
typedef enum {
    MPM_SCHEDULE_AUTO = 0,
    MPM_SCHEDULE_FULL = 1,      /* every (query block, candidate tile) pair of 256 x 256 */
    MPM_SCHEDULE_SYMMETRIC = 2, /* pairs on and above the block diagonal only */
    MPM_SCHEDULE_FULL_64 = 3    /* every pair of 64 x 64 blocks (small batches) */
} mpm_schedule;

#define MPM_MAX_N 16384   /* tokens per image */
#define MPM_MAX_B 65535   /* images per call */
#define MPM_MAX_D 16384   /* channels per token */

/* Library version string, e.g. "mpm 0.2.0 gfx950". Never NULL. */
const char* mpm_version(void);

/* Human-readable name of a status code. Never NULL. */
const char* mpm_status_string(int status);

/* hipError_t of the last MPM_ERR_HIP returned on this host thread (0 if none). */
int mpm_last_hip_error(void);

/*
 * Device workspace of mpm_affinity, mpm_affinity_compact, mpm_argmax and
 * mpm_merge: bytes needed for a batch of B images of at most N tokens. The
 * caller allocates it (256-byte aligned) and owns it; calls ordered on one
 * stream may reuse it, for any B and N it is large enough for. Layout, as byte
 * offsets returned by mpm_workspace_offsets (each 256-byte aligned):
 *   sync  int32[MPM_MAX_B + 1]  arrival counters of the fused compaction
 *                               (always at offset 0, the same for every shape);
 *   nb    int32[B*N]            nearest neighbour per token (slot layout);
 *   src   int32[2*B*N]          (representative, partner) of cluster k of image
 *                               b at 2*(b*N + k) (partner == representative for
 *                               a singleton);
 *   pv    float[B*T*N], pi int32[B*T*N]  per-candidate-tile argmax partials,
 *                               T = ceil(N / 64) slots per token: tile t of image b
 *                               for token i at (b*T + t)*N + i; a launch fills the
 *                               first ceil(n_b / w) slots, w = the block width of
 *                               its schedule (64 or 256 tokens).
 * The sync region must be zero before a workspace's first use by
 * mpm_affinity_compact or mpm_merge (mpm_workspace_init); every call leaves it
 * zero again (an interrupted call may not). Returns 0 for B < 1 or N < 1.
 */
size_t mpm_workspace_bytes(int32_t B, int32_t N);

/* Byte offsets of the workspace regions listed above; any pointer may be NULL.
 * Returns MPM_OK, or MPM_ERR_INVALID_ARG for B < 1 or N < 1. */
int mpm_workspace_offsets(int32_t B, int32_t N, size_t* sync, size_t* nb, size_t* src, size_t* pv, size_t* pi);

/*
 * Zeroes the sync region of a workspace of ws_bytes bytes (at least the
 * region's 256 KB) with a fill kernel on `stream` (no memset node, so it may
 * be captured in a HIP graph). Needed once after allocating a workspace.
 */
int mpm_workspace_init(void* ws, size_t ws_bytes, void* stream);

/*
 * Cosine affinity and its self-masked row argmax, per candidate tile (Eq. 1
 * and the argmax of Sec. 3.2), into the workspace partials: for every query i
 * and candidate tile t, the best score (x_i . x_j) / max(||x_j||, 1e-12) over
 * the tile's candidates j != i, j < n_b, and that j (lowest j among equal
 * scores). The dot products are accumulated in float32 on MFMA from the
 * stored values (bfloat16 products are exact in float32); the N x N affinity
 * is never written to memory. Dividing by ||x_i|| too would not move the
 * argmax of row i, so it is not applied.
 *   x, x_off: rows of dtype `dt`, dense or packed;
 *   x_inv (may be NULL): the inverse row norms 1 / max(||x_r||, 1e-12), one
 *     float per row of x (packed like x; rows past an image's end are not
 *     read), given instead of summed in the kernel's K loop (about a tenth of
 *     its time), as mpm_pair_average writes them for the next insertion's
 *     input (Sec. 3.3). Bfloat16 rows whose byte length is a multiple of 64
 *     only: other rows return MPM_ERR_UNSUPPORTED with a non-NULL x_inv;
 *   start_event / stop_event (may be NULL): hipEvent_t the caller created
 *     (timing enabled) and owns, bound to the kernels' own dispatches
 *     (hipExtLaunchKernel): start to the first launch, stop to the last, so
 *     hipEventElapsedTime(start, stop) is the step's duration on the device
 *     without extra stream commands. The step is one launch, or two when the
 *     symmetric schedule runs deferred diagonal blocks in a second launch.
 */
int mpm_affinity(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D,
                 int32_t dt, int32_t schedule, void* ws, size_t ws_bytes, void* start_event, void* stop_event,
                 void* stream);

/*
 * One insertion's affinity step and compaction step (Sec. 3.2, Alg. 1 steps 2-6)
 * in one call: mpm_affinity, then the compaction kernel, which reduces each
 * image's partials to nb (larger score, then smaller index; images with more
 * than a few candidate tiles are reduced by a separate parallel launch first),
 * tests the pairs for mutuality, marks representatives and assigns compact ids
 * by a left-to-right scan, one workgroup per image; the workgroup that finishes
 * the last image (found with the arrival counter in the workspace's sync
 * region, no waiting) turns the per-image cluster counts into offsets. Writes
 *   map[b*N + i] = r(i) for i < n_b, -1 for n_b <= i < N;
 *   y_off[0] = 0, y_off[b+1] = y_off[b] + n'_b (int32[B+1]);
 *   the workspace's nb and src regions (src read by mpm_pair_average).
 * The timing events are bound to the affinity kernel's dispatches only.
 * Arguments as mpm_affinity otherwise; the workspace's sync region must be zero
 * (mpm_workspace_init).
 */
int mpm_affinity_compact(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D,
                         int32_t dt, int32_t schedule, int32_t* map, int32_t* y_off, void* ws, size_t ws_bytes,
                         void* start_event, void* stop_event, void* stream);

/*
 * The schedule (MPM_SCHEDULE_FULL, MPM_SCHEDULE_SYMMETRIC or
 * MPM_SCHEDULE_FULL_64, never AUTO) that mpm_affinity runs for B images of at
 * most N tokens of D channels of dtype dt under `schedule` on the current
 * device, written to *used (a host pointer). For reporting the matrix-core
 * work a call issues: about 2 * w^2 * D flops per w x w block, nb^2 blocks per
 * image of nb = ceil(n_b / w) blocks under the full schedules (w = 256, or 64
 * for MPM_SCHEDULE_FULL_64) and nb (nb + 1) / 2 under the symmetric one
 * (w = 256). Rows whose byte length is not a multiple of 64 always report
 * MPM_SCHEDULE_FULL. Returns MPM_OK, MPM_ERR_INVALID_ARG for bad sizes, an
 * unknown schedule or a NULL pointer, or MPM_ERR_HIP when the device cannot be
 * queried.
 */
int mpm_affinity_schedule_used(int32_t B, int32_t N, int32_t D, int32_t dt, int32_t schedule, int32_t* used);

/*
 * The block size mpm_merge_local's affinity runs for this shape, window and requested
 * block_rows on the current device, written to *rows (a host pointer): 256 or 128
 * (square blocks on the symmetric schedule; with block_rows 0, whichever an estimate of
 * the launch on a full raster grid of grid_w columns, at this window, finds faster), or
 * N for rows whose byte length is not a multiple of 64 (a kernel that runs each query
 * block's whole band). For reporting. Returns MPM_OK, MPM_ERR_INVALID_ARG for bad
 * sizes, grid_w, window or block_rows (as mpm_merge_local) or a NULL pointer, or
 * MPM_ERR_HIP when the device cannot be queried.
 */
int mpm_local_block_rows(int32_t B, int32_t N, int32_t D, int32_t dt, int32_t grid_w, int32_t window,
                         int32_t block_rows, int32_t* rows);

/*
 * Nearest neighbours: mpm_affinity (norms summed in the kernel), then the
 * reduction of the partials.
 *   nb[b*N + i] = argmax_{j != i, j < n_b} cos(x_i, x_j), lowest j on equal
 *                 scores; -1 when n_b == 1. Entries i >= n_b are not written.
 *   best[b*N + i] (optional, may be NULL) = the float32 cosine of that pair.
 * nb and best are caller arrays (not the workspace).
 */
int mpm_argmax(const void* x, const int32_t* x_off, int32_t B, int32_t N, int32_t D, int32_t dt, int32_t schedule,
               int32_t* nb, float* best, void* ws, size_t ws_bytes, void* stream);

/*
 * Mutual pairs and compact ids (Sec. 3.2, Alg. 1) from given neighbours nb
 * (slot layout, values in [0, n_b) or -1 for n_b == 1).
 *   map[b*N + i] = r(i) for i < n_b, -1 for n_b <= i < N;
 *   src[2*(b*N + k)], src[2*(b*N + k) + 1] = (representative, partner) of
 *     cluster k < n'_b (partner == representative for a singleton);
 *   y_off[0] = 0, y_off[b+1] = y_off[b] + n'_b.
 * x_off: the offsets of the tokens nb was computed on (NULL = dense, n_b = N).
 * Two launches (one workgroup per image, then the offsets).
 */
int mpm_pair_compact(const int32_t* nb, const int32_t* x_off, int32_t B, int32_t N, int32_t* map, int32_t* src,
                     int32_t* y_off, void* stream);

/*
 * Cluster means (Eq. 2), packed by the offsets the compaction wrote:
 *   y[y_off[b] + k] = mean of the rows src names for cluster k of image b,
 *     computed in float32 and rounded once (nearest even) to `dt`; a
 *     singleton is copied bit for bit;
 *   y_inv (optional, may be NULL): y_inv[y_off[b] + k] = 1 / max(||y_k||, 1e-12)
 *     from the stored values of y in float32, summed in a fixed order (the same
 *     on every run): the x_inv of y for the next insertion's affinity.
 * src in the slot layout above (the workspace's src region after
 * mpm_affinity_compact, or mpm_pair_compact's output); y has room for
 * y_off[B] rows (at most B*N). x as in mpm_affinity.
 */
int mpm_pair_average(const void* x, const int32_t* x_off, const int32_t* src, const int32_t* y_off, int32_t B,
                     int32_t N, int32_t D, int32_t dt, void* y, float* y_inv, void* stream);

/*
 * One MPM insertion (Alg. 1) = mpm_affinity_compact, then mpm_pair_average
 * (src from the workspace), in order on `stream`.
 *   x, x_off, x_inv: input tokens (dense or packed) and optional given inverse
 *       norms, as in mpm_affinity;
 *   y, y_off: merged tokens, packed (capacity B*N rows), offsets int32[B+1];
 *   y_inv (may be NULL): inverse norms of the merged rows, as in mpm_pair_average;
 *   map: int32[B*N] merge map in slot layout (-1 beyond n_b);
 *   ws: workspace of at least mpm_workspace_bytes(B, N) bytes whose sync
 *       region is zero (mpm_workspace_init); nb and src are readable there
 *       after the call.
 * Feed (y, y_off, y_inv) as (x, x_off, x_inv) of the next insertion.
 */
int mpm_merge(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D, int32_t dt,
              int32_t schedule, void* y, int32_t* y_off, float* y_inv, int32_t* map, void* ws, size_t ws_bytes,
              void* stream);

/*
 * One locality-constrained insertion: mpm_merge with the candidates of each token
 * restricted to a window around it on the token grid, the mitigation of the
 * quadratic affinity that the paper proposes (Sec. 5, also Sec. 4.3). A token's
 * position is its raster index on a grid of grid_w columns (row = pos / grid_w,
 * column = pos % grid_w):
 *   x_inv (may be NULL): given inverse norms of the rows of x, as in mpm_affinity;
 *   y_inv (may be NULL): inverse norms of the merged rows, as in mpm_pair_average;
 *   pos (may be NULL): int32 per row of x, packed like x; NULL means each token's
 *       index in its image (the raster order of a full grid, as for a first
 *       insertion); positions must be non-decreasing in row along each image;
 *   window >= 0: j is a candidate of i when |row_i - row_j| <= window and
 *       |col_i - col_j| <= window;
 *   block_rows: 0, 128 or 256: the rows of the square blocks the affinity runs in
 *       (0: the library's pick, as mpm_local_block_rows reports); results never
 *       depend on it;
 *   nb[i] = argmax over the candidates of the cosine (lowest j on equal scores), or
 *       -1 when the window holds no other token (i is then a singleton);
 *   y_pos[y_off[b] + k] = the position of cluster k's representative (int32, packed
 *       like y): the pos of the merged rows for the next insertion, which keeps the
 *       raster order since ids follow the left-to-right scan.
 * Feed (y, y_off, y_inv, y_pos) as (x, x_off, x_inv, pos) of the next insertion.
 * Only the candidate tiles a query block's window reaches are computed. The
 * workspace as in mpm_merge (nb and src readable after the call). start_event /
 * stop_event (may be NULL) are bound to the affinity kernel's dispatch, as in
 * mpm_affinity. Errors as mpm_merge, plus MPM_ERR_INVALID_ARG for grid_w < 1,
 * grid_w > MPM_MAX_N, window < 0 or another block_rows. Positions outside
 * [0, grid_w * MPM_MAX_N) are undefined behaviour.
 */
int mpm_merge_local(const void* x, const int32_t* x_off, const float* x_inv, const int32_t* pos, int32_t B,
                    int32_t N, int32_t D, int32_t dt, int32_t grid_w, int32_t window, int32_t block_rows, void* y,
                    int32_t* y_off, float* y_inv, int32_t* y_pos, int32_t* map, void* ws, size_t ws_bytes,
                    void* start_event, void* stop_event, void* stream);

/*
 * Padded batch layout (the paper pads each batch to its longest image, Sec. 4.2): the
 * packed rows of B images (offsets z_off, int32[B+1], as the merges write them) to a
 * dense [B][P][row_bytes] array, image b's rows first and zero rows after them:
 *   out[b][k] = z[z_off[b] + k] for k < min(n_b, P), zeros for n_b <= k < P.
 * For the parts of a model that need equal-length images (batched attention with a
 * key mask), while the per-token parts keep the packed rows. Rows are copied as
 * bytes: row_bytes a positive multiple of 16 (any dtype, several heads' features in
 * one row, ...). P is the caller's choice, usually the batch's largest n_b (read from
 * z_off) or N. Errors: MPM_ERR_INVALID_ARG for B < 1, P < 1, a row size that is not a
 * positive multiple of 16 or bad pointers; MPM_ERR_UNSUPPORTED for B, P or rows above
 * the maxima (MPM_MAX_B, MPM_MAX_N, 4 * MPM_MAX_D bytes).
 */
int mpm_pad(const void* z, const int32_t* z_off, int32_t B, int32_t P, int32_t row_bytes, void* out, void* stream);

/* The inverse of mpm_pad: z[z_off[b] + k] = padded[b][k] for k < min(n_b, P); padded
 * rows k >= n_b are not read. Arguments and errors as mpm_pad. */
int mpm_unpad(const void* padded, const int32_t* z_off, int32_t B, int32_t P, int32_t row_bytes, void* z,
              void* stream);

/*
 * mpm_merge for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the workspace
 * is a file-scope device array of MPM_NOALLOC_SCRATCH_BYTES that each GPU the
 * library runs on holds until the process ends; its address is looked up on the
 * first call on a GPU, whose stream also gets one small fill kernel that clears
 * its arrival counters. No call allocates or frees anything (no hipMalloc,
 * hipFree or allocating library routine). Shapes whose mpm_workspace_bytes(B, N)
 * exceed the array return MPM_ERR_WORKSPACE (B = 64 at N = 1024, B = 16 at
 * N = 4096 and B = 32 at N = 2304 fit). Every call on a GPU shares that GPU's
 * array and leaves its arrival counters zero, but its other contents are the last
 * call's: calls that overlap on one GPU (several streams or threads) race and give
 * wrong results, so order them. Arguments, results and other errors as mpm_merge
 * (without the workspace, so nb and src are not readable).
 */
#define MPM_NOALLOC_SCRATCH_BYTES (48u << 20)
int mpm_merge_noalloc(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D,
                      int32_t dt, int32_t schedule, void* y, int32_t* y_off, float* y_inv, int32_t* map, void* stream);

/*
 * Composition of merge maps (Eq. 3): map_ab[b*N + i] = map_b[b*N + map_a[b*N + i]],
 * or -1 where map_a[b*N + i] < 0. Both maps in slot layout; map_a's values
 * index image b's entries of map_b. map_ab may alias map_a.
 */
int mpm_compose(const int32_t* map_a, const int32_t* map_b, int32_t B, int32_t N,
                int32_t* map_ab, void* stream);

/*
 * Gather reconstruction (Eq. 4) with E special rows in front.
 *   out is dense [B][E + N][D];
 *   out[b][e]     = z_spec[b][e]                   for e < E (z_spec [B][E][D]; may be NULL iff E == 0);
 *   out[b][E + i] = z[z_off[b] + map[b*N + i]]     for map >= 0 (bit copy),
 *                   zeros                          where map < 0.
 * z, z_off: merged rows, packed (z_off NULL = dense [B][N][D] rows).
 */
int mpm_unmerge(const void* z, const int32_t* z_off, const int32_t* map, const void* z_spec, int32_t E,
                int32_t B, int32_t N, int32_t D, int32_t dt, void* out, void* stream);

/*
 * Composition folded into the gather (Eq. 3 and Eq. 4 in one pass over the grid):
 *   r*(i) = map_b[b*N + map_a[b*N + i]], or -1 where map_a[b*N + i] < 0;
 *   out as mpm_unmerge with map = r*;
 *   map_ab (optional, may be NULL) receives r* in slot layout.
 * map_ab must not alias map_a or map_b (MPM_ERR_INVALID_ARG if it does). Other
 * arguments and errors as mpm_unmerge and mpm_compose.
 */
int mpm_compose_unmerge(const void* z, const int32_t* z_off, const int32_t* map_a, const int32_t* map_b,
                        int32_t* map_ab, const void* z_spec, int32_t E, int32_t B, int32_t N, int32_t D, int32_t dt,
                        void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MPM_H */
