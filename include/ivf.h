/*
 * ivf.h -- C ABI of the MI355X (gfx950) IVF routing and construction hot path
 * of InSituANN (arXiv 2608.08751).
 *
 * What is computed (paper references are to sections and equations):
 *   - coarse search, Eq. (1), Sec. "ANN Search and IVF": for each query the
 *     nprobe centroids of smallest squared L2 distance;
 *   - the distances are evaluated as in Eq. (6), Sec. "GPU coarse search"
 *     (||q||^2 + ||c||^2 - 2 q.c, the -2 q.c term as a dense MFMA contraction
 *     over LDS-staged centroid tiles, never written to memory), with the
 *     row-wise top-P selected on the device so that only O(B*P) ids and
 *     distances are produced ("On-device list selection", same section);
 *   - IVF construction, Sec. "System Architecture" (index layout) and
 *     Sec. "Fast Index Construction": Lloyd k-means iterations (assignment +
 *     mean update) and the assignment of every base vector to its nearest
 *     centroid, stored cluster-major with per-list offset, length and ids.
 *
 * Exactness contract. Every id, label, count, offset and permutation entry is
 * exactly what the definition gives with distances evaluated in fp64 as
 *     s = 0; for d = 0..D-1: t = (double)x_d - (double)c_d; s = fma(t, t, s)
 * and ties broken by the lower centroid id. Returned distances are that s
 * rounded to fp32. The MFMA contraction only screens candidates; a rigorous
 * error bound decides which candidates are re-evaluated in fp64 and when a
 * query or row falls back to an exact fp64 scan of all centroids. Which
 * matrix unit screens depends on the data type:
 *   - fp32 queries and rows: fp32 MFMA (v_mfma_f32_32x32x2_f32); the bound is
 *     the fp32 dot-product rounding bound for any summation order;
 *   - uint8 rows (k-means and assignment): int8 MFMA
 *     (v_mfma_i32_32x32x32_i8) on rows x - 128 against quantised centroids,
 *     whose integer scores are exact; the bound is the quantisation error
 *     alone. For D <= 128 one int8 plane rint(c - 128) screens first and
 *     settles most rows; the rows it leaves are screened on two int8 planes
 *     of the 16-bit fixed-point value rint(256 (c - 128)). A call whose
 *     centroids have a coordinate outside [0, 255.998] (which does not
 *     quantise) is screened on fp32 MFMA instead; the switch happens on the
 *     device, without a host synchronisation.
 *   - uint8-valued fp32 queries (every value an integer in [0, 255]) routed
 *     against more than 2,048 centroids: the threshold-sample keys and the
 *     candidate filter run on the two int8 planes (x - 128 against
 *     rint(256 (c - 128))), with a bound of (390 + ||x - 128||_1) / 2 in the
 *     planes' key units; any other value in the call, or a centroid that does
 *     not quantise, sends the call to the fp32 kernels (device flag, no host
 *     synchronisation). IVF_OPT_FP32_SCREEN forces the fp32 kernels.
 * Either way the results are the exact ones above; the screen chosen changes
 * speed only.
 *
 * Conventions shared by every call:
 *   - Array arguments are DEVICE pointers on the context's device, row-major,
 *     contiguous, 16-byte aligned, allocated and owned by the caller. The
 *     library never frees or retains them beyond the call.
 *   - Calls are asynchronous: IVF_OK means every kernel was enqueued on the
 *     context's stream. No call synchronises with the host. Device faults
 *     surface at ivf_sync() as IVF_EDEVICE.
 *   - Arguments are validated before anything is enqueued; on any status other
 *     than IVF_OK nothing was enqueued and the outputs are untouched, and
 *     ivf_last_error() describes the problem.
 *   - Scratch memory is a caller-provided device workspace (ivf_set_workspace)
 *     of at least ivf_workspace_bytes() for the call; too small gives
 *     IVF_ENOMEM with the required size in ivf_last_error(). Two calls that
 *     share a context must not overlap on different streams.
 *   - Q, N == 0 is a no-op returning IVF_OK.
 *   - Supported shapes: 4 <= D <= 256 with D % 4 == 0 (else IVF_EUNSUPPORTED);
 *     the row-major register tiles of the screens hold at most 256 dims.
 *   - Row counts N up to 2^32 - 1 (row ids are uint32 in the permutation);
 *     the assignment screens rows in slices of 2^28, so row ids inside a
 *     launch always fit int32.
 *   - Input values must be finite, with squared vector norms below FLT_MAX;
 *     results are unspecified otherwise (inputs are not scanned for this).
 */
#ifndef IVF_H
#define IVF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    IVF_OK = 0,
    IVF_EINVAL = 1,       /* bad argument: sizes, null pointers, aliasing */
    IVF_EUNSUPPORTED = 2, /* valid but outside the supported shapes */
    IVF_ENOMEM = 3,       /* workspace missing or too small */
    IVF_EDEVICE = 4       /* HIP runtime error (launch failure, device fault) */
} ivf_status;

typedef enum { IVF_F32 = 0, IVF_U8 = 1 } ivf_dtype;

/* Operation codes for ivf_workspace_bytes. */
typedef enum {
    IVF_OP_ROUTE = 0,
    IVF_OP_KMEANS_STEP = 1,
    IVF_OP_ASSIGN_BUILD = 2,
    IVF_OP_BUILD_LISTS = 3,
    IVF_OP_PQ_TRAIN_STEP = 4,
    IVF_OP_ADC_SCAN = 5
} ivf_op;

typedef struct ivf_ctx ivf_ctx;

/* Creates a context bound to HIP device `device` and to `hip_stream`
 * (a hipStream_t; NULL = the device's null stream). *out receives the handle.
 * Errors: IVF_EINVAL (out == NULL, bad device), IVF_EDEVICE. */
ivf_status ivf_create(int device, void *hip_stream, ivf_ctx **out);

/* Destroys a context; NULL is ignored. Does not free the workspace. */
void ivf_destroy(ivf_ctx *ctx);

/* Host string describing the last non-OK status of this context ("" if none).
 * Valid until the next call on the context. */
const char *ivf_last_error(const ivf_ctx *ctx);

/* Rebinds the context to another stream (NULL = null stream). */
ivf_status ivf_set_stream(ivf_ctx *ctx, void *hip_stream);

/* Device workspace bytes that `op` needs for the given sizes:
 *   IVF_OP_ROUTE        rows = Q, k = nprobe
 *   IVF_OP_KMEANS_STEP  rows = N (k ignored)
 *   IVF_OP_ASSIGN_BUILD rows = N (k ignored)
 *   IVF_OP_BUILD_LISTS  rows = N (D, k ignored)
 *   IVF_OP_PQ_TRAIN_STEP rows = n, C = M (D, k ignored)
 *   IVF_OP_ADC_SCAN     rows = B queries, C = P probes per query, k = handoff
 * Returns 0 for sizes that the op rejects. */
size_t ivf_workspace_bytes(int op, int64_t rows, int64_t C, int32_t D, int32_t k);

/* Hands the context a caller-owned device buffer (256-byte aligned) used as
 * scratch by later calls. The buffer must stay allocated while calls that use
 * it are in flight. NULL/0 detaches it. */
ivf_status ivf_set_workspace(ivf_ctx *ctx, void *dev_ptr, size_t bytes);

/* Waits for the context's stream. IVF_EDEVICE if the device reported an error. */
ivf_status ivf_sync(ivf_ctx *ctx);

/* Coarse search, Eq. (1) with Eq. (6) (Sec. "GPU coarse search").
 *   queries   [Q, D] fp32           centroids [C, D] fp32
 *   nprobe    1 <= nprobe <= min(C, 1024)
 *   out_ids   [Q, nprobe] int32     centroid ids, ascending (distance, id)
 *   out_dist  [Q, nprobe] fp32      squared L2 distances (fp64 rounded to
 *                                   fp32), may be NULL
 * Outputs must not overlap the inputs or each other.
 * Errors: IVF_EINVAL (Q < 0, C < 1, nprobe out of range, NULL required
 * pointer, misaligned pointer, aliasing), IVF_EUNSUPPORTED (D), IVF_ENOMEM. */
ivf_status ivf_route(ivf_ctx *ctx, const float *queries, int64_t Q, const float *centroids,
                     int64_t C, int32_t D, int32_t nprobe, int32_t *out_ids, float *out_dist);

/* ivf_route for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * same arguments, results and errors as ivf_route, but no workspace is used
 * and nothing is allocated (no hipMalloc, hipFree, event or library
 * allocation; IVF_OPT_PROFILE records nothing for it). The scratch memory is
 * a static device array of 64 MiB held on every device the library runs on
 * until the process ends; queries are processed in batches that fit it
 * (smaller batches than ivf_route's, so throughput can be lower). Sizes that
 * need more than 64 MiB for a single query (C above about 16M, or nprobe and
 * C giving a larger candidate layout) are refused with IVF_EUNSUPPORTED.
 * Every call on a device shares that device's array and leaves its contents
 * behind (the call clears what it needs itself): two calls that overlap on
 * one device, from any contexts or streams, race and give undefined results. */
ivf_status ivf_route_noalloc(ivf_ctx *ctx, const float *queries, int64_t Q, const float *centroids,
                             int64_t C, int32_t D, int32_t nprobe, int32_t *out_ids, float *out_dist);

/* One Lloyd iteration of k-means (k-means training, Sec. "Fast Index
 * Construction"): assignment against `centroids`, then the mean update.
 *   train          [N, D] fp32 or uint8 (dt), N >= 1
 *   centroids      [C, D] fp32 input centroids c^(t)
 *   seed, iter     select the training row that replaces an empty cluster j:
 *                  row = SplitMix64 output ((iter << 32) | j) + 1 of a
 *                  generator seeded with `seed`, mod N
 *   out_labels     [N] int32, nearest input centroid, ties to the lower id
 *   out_centroids  [C, D] fp32 c^(t+1): for a non-empty cluster
 *                  (float)(sum / (double)count) where the sum is exact for
 *                  uint8 data and an fp64 sum in ascending row order for fp32
 *                  data; an empty cluster takes the reseed row. Must not alias
 *                  `centroids`.
 *   out_counts     [C] int64 cluster sizes before reseeding, may be NULL
 *   out_objective  device fp64 scalar: sum over rows of the squared distance
 *                  to the assigned input centroid, may be NULL
 *   hint_labels    [N] int32 or NULL: a label per row from an earlier step
 *                  (the previous iteration's out_labels). Speed only: the
 *                  single-plane int8 screen starts each row's keep threshold
 *                  from the hinted centroid's score, so fewer centroids met
 *                  early in the scan are inserted; results never depend on it.
 *                  Entries outside [0, C) are ignored. Must not alias an output.
 * Errors: as ivf_route; N > 2^32 - 1 is IVF_EUNSUPPORTED. */
ivf_status ivf_kmeans_step(ivf_ctx *ctx, const void *train, int dt, int64_t N,
                           const float *centroids, int64_t C, int32_t D, uint64_t seed,
                           int32_t iter, int32_t *out_labels, float *out_centroids,
                           int64_t *out_counts, double *out_objective, const int32_t *hint_labels);

/* Full assignment and inverted-list build (Sec. "System Architecture", index
 * layout: cluster-major lists with offset, length and vector ids).
 *   base         [N, D] fp32 or uint8 (dt), N <= 2^32 - 1
 *   centroids    [C, D] fp32
 *   out_labels   [N] int32 nearest centroid, ties to the lower id
 *   out_counts   [C] int64 list lengths
 *   out_offsets  [C + 1] int64 exclusive prefix sum of counts, offsets[C] = N
 *   out_perm     [N] uint32 row ids grouped by list, ascending inside a list
 * Errors: as ivf_kmeans_step. */
ivf_status ivf_assign_build(ivf_ctx *ctx, const void *base, int dt, int64_t N,
                            const float *centroids, int64_t C, int32_t D, int32_t *out_labels,
                            int64_t *out_counts, int64_t *out_offsets, uint32_t *out_perm);

/* The inverted-list build alone, for given labels in [0, C) (the list-build
 * step of ivf_assign_build). Outputs as in ivf_assign_build. Labels outside
 * [0, C) give undefined lists (not detected on the host). */
ivf_status ivf_build_lists(ivf_ctx *ctx, const int32_t *labels, int64_t N, int64_t C,
                           int64_t *out_counts, int64_t *out_offsets, uint32_t *out_perm);

/* Diagnostics of the last call on this context, copied synchronously from
 * the workspace (waits on the stream):
 *   out[0] queries / rows that went to the full fp64 fallback scan
 *   out[1] rows whose top-1 was settled by fp64 re-evaluation of 2 candidates
 *   out[2] route: sum over queries of screened candidates kept
 *   out[3] route: queries whose candidate list overflowed
 *   out[4] route: centroids in the threshold sample
 *   out[5] assignment of uint8 rows: 1 when screened on int8 MFMA
 *   out[6] assignment of uint8 rows: rows the single-plane int8 screen left
 *          to the two-plane int8 screen
 *   out[7] reserved (0) */
ivf_status ivf_last_stats(ivf_ctx *ctx, int64_t out[8]);

/* Test, tuning and profiling knobs (values persist on the context):
 *   IVF_OPT_FORCE_FALLBACK  1 = every query / row takes the exact fp64
 *                           fallback scan (results must not change)
 *   IVF_OPT_SAMPLE_RANK     rank used for the routing threshold (0 = default);
 *                           changes speed only, never results or sizes
 *   IVF_OPT_PROFILE         1 = record a HIP event pair on the context stream
 *                           around every kernel launch of each call
 *   IVF_OPT_BUILD_BLOCKS    cap on the row blocks of the single-pass list build
 *                           (more than 65,536 lists; 0 = default); speed only
 *   IVF_OPT_SCREEN_WAVES    wave64s per workgroup of the fp32 distance-
 *                           screening kernel, 4 or 8 (D > 128 always uses 4);
 *                           speed only, never results
 *   IVF_OPT_FP32_SCREEN     1 = uint8 rows, and uint8-valued queries in
 *                           ivf_route, are screened on fp32 MFMA like fp32
 *                           data (default 0: int8 MFMA whenever every
 *                           centroid coordinate c has rint(256 (c - 128)) in
 *                           [-32768, 32767], i.e. c in [0, 255.998]);
 *                           speed only, never results
 *   IVF_OPT_I8_TWO_PLANE_ONLY  1 = no single-plane int8 pre-screen (default 0:
 *                           for D <= 128, uint8 rows are first screened on one
 *                           int8 plane rint(c - 128), which settles most rows
 *                           with half the MFMA work, when every coordinate has
 *                           rint(c - 128) in [-128, 127]); speed only
 *   IVF_OPT_FORCE_RESCREEN  1 = the single-plane screen settles no row: every
 *                           row goes on to the two-plane screen (results must
 *                           not change)
 *   IVF_OPT_RESCREEN_CAP    > 0: capacity of the single plane's list of rows
 *                           for the two-plane screen (default 4,096 + N / 16;
 *                           past it the two-plane screen takes every row);
 *                           speed only, never results
 *   IVF_OPT_ASSIGN_SLICE    > 0: rows per assignment slice, below the
 *                           default 2^28 (each slice is screened with its own
 *                           worklists); speed only, never results
 *   IVF_OPT_S1_ID_ORDER     1 = the single-plane screen visits centroids in id
 *                           order (default 0: in ascending distance to the
 *                           mean of the centroids, a stable counting sort per
 *                           call, so that rows meet good centroids early and
 *                           the scan inserts fewer scores); speed only, never
 *                           results */
typedef enum {
    IVF_OPT_FORCE_FALLBACK = 0,
    IVF_OPT_SAMPLE_RANK = 1,
    IVF_OPT_PROFILE = 2,
    IVF_OPT_BUILD_BLOCKS = 3,
    IVF_OPT_SCREEN_WAVES = 4,
    IVF_OPT_FP32_SCREEN = 5,
    IVF_OPT_I8_TWO_PLANE_ONLY = 6,
    IVF_OPT_FORCE_RESCREEN = 7,
    IVF_OPT_RESCREEN_CAP = 8,
    IVF_OPT_ASSIGN_SLICE = 9,
    IVF_OPT_S1_ID_ORDER = 10
} ivf_option;
ivf_status ivf_set_option(ivf_ctx *ctx, int option, int64_t value);

/* Candidate-restricted assignment (the fast construction mode of Sec. "Fast
 * Index Construction": each vector is scored against a few candidate
 * centroids only; the paper takes them from a CAGRA search over the
 * centroids). The candidates of row i are graph[prev[i]][0 .. S): e.g. each
 * centroid's S nearest centroids (ivf_route of the centroids against
 * themselves with nprobe = S) and the row's previous label. out_labels[i] is
 * the candidate of smallest distance by (distance, id), the distance exact as
 * in the contract above; candidate ids outside [0, C) are skipped, and a row
 * without any valid candidate (or with prev[i] outside [0, C)) gets -1 and an
 * infinite distance. The result is exact for the candidate sets, not for the
 * full centroid table.
 *   rows       [N, D] fp32 or uint8 (dt), N <= 2^32 - 1
 *   centroids  [C, D] fp32      graph [C, S] int32, 1 <= S <= 64
 *   prev       [N] int32        out_labels [N] int32
 *   order      [N] uint32 processing order, or NULL (row order): results do
 *              not depend on it, speed does (rows with the same previous
 *              label next to each other share their candidates' loads; the
 *              previous step's list permutation is that order; an order
 *              that does not group them is slower than NULL). Entries >= N
 *              are skipped; a row that order does not list is left untouched.
 *   out_dist   [N] fp32 squared distance (fp64 rounded), may be NULL
 * No workspace. Errors: IVF_EINVAL, IVF_EUNSUPPORTED (D, N), IVF_EDEVICE. */
ivf_status ivf_assign_graph(ivf_ctx *ctx, const void *rows, int dt, int64_t N,
                            const float *centroids, int64_t C, int32_t D, const int32_t *graph,
                            int32_t S, const int32_t *prev, const uint32_t *order,
                            int32_t *out_labels, float *out_dist);

/* Candidates for rows that have no previous label (the graph-assisted
 * assignment of the full base set, Sec. "Fast Index Building Details": the
 * paper retrieves a few candidate centroids per vector from a CAGRA search
 * over the centroid table). Here the candidates come from a coarse partition
 * of the centroids into G cells and a greedy walk over a centroid graph:
 * row i first takes the member of its cell cell[i] of smallest (distance, id)
 * (cell_members[cell_offsets[c] .. cell_offsets[c + 1]), both offsets clamped
 * into [0, M], the second to at least the first), then, up to `hops` times,
 * moves to the neighbour graph[b][0 .. S) of smallest (distance, id) if that
 * neighbour comes before the current choice b in (distance, id) order, and
 * stops otherwise. Distances are exact as in the contract above; ids outside
 * [0, C) are skipped; a row whose cell lies outside [0, G) or holds no valid
 * member gets -1 and an infinite distance. The result is exact for that
 * procedure, not for the full centroid table. Typical inputs: the cells from
 * ivf_assign_build of the centroids (as fp32 rows) against a coarse table of
 * G centroids (its offsets and permutation are cell_offsets and
 * cell_members), the rows' cells from ivf_assign_build of the rows against
 * the same table, and the graph from ivf_route of the centroids against
 * themselves.
 *   rows          [N, D] fp32 or uint8 (dt), N <= 2^32 - 1
 *   centroids     [C, D] fp32
 *   cell          [N] int32, cell of each row
 *   cell_offsets  [G + 1] int64, 1 <= G <= 2^31 - 1
 *   cell_members  [M] uint32 centroid ids grouped by cell (may be NULL when M = 0)
 *   graph         [C, S] int32 or NULL (no walk), 1 <= S <= 64
 *   hops          0 <= hops <= 1024
 *   order         [N] uint32 processing order, or NULL (row order): results
 *                 do not depend on it, speed does (rows of one cell next to
 *                 each other share their members' loads; the permutation
 *                 from ivf_assign_build of the rows against the coarse table
 *                 is that order). Entries >= N are skipped; a row that order
 *                 does not list keeps whatever out_labels/out_dist held.
 *   out_labels    [N] int32;  out_dist [N] fp32 squared distance or NULL
 * No workspace. Errors: IVF_EINVAL (sizes, NULL pointers, misalignment,
 * aliasing), IVF_EUNSUPPORTED (D, N), IVF_EDEVICE. */
ivf_status ivf_assign_cells(ivf_ctx *ctx, const void *rows, int dt, int64_t N,
                            const float *centroids, int64_t C, int32_t D, const int32_t *cell,
                            int64_t G, const int64_t *cell_offsets, const uint32_t *cell_members,
                            int64_t M, const int32_t *graph, int32_t S, int32_t hops,
                            const uint32_t *order, int32_t *out_labels, float *out_dist);

/* List-major layout of the base vectors and their residuals (Sec. "List-major
 * contiguous scans": every IVF list is one contiguous range; Sec.
 * "Residual-PQ Candidate Reduction": the residual x - c(x) to the assigned
 * centroid is what residual PQ encodes).
 *   base          [N, D] fp32 or uint8 (dt), N <= 2^32 - 1
 *   centroids     [C, D] fp32
 *   offsets       [C + 1] int64 list offsets and
 *   perm          [N] uint32 list-major row ids, as ivf_assign_build returns
 *                 them (offsets non-decreasing, offsets[0] = 0, offsets[C] = N)
 *   pos0, n       the output covers list-major positions [pos0, pos0 + n)
 *                 (batches of a large base), 0 <= pos0 <= pos0 + n <= N
 *   out_rows      [n, D] same type as base: row perm[pos0 + i], may be NULL
 *   out_residuals [n, D] fp32: that row minus the centroid of the list holding
 *                 position pos0 + i, one fp32 subtraction per element (the
 *                 exact difference rounded once), may be NULL (not both,
 *                 unless n == 0, which is a no-op)
 * A perm entry >= N yields a zero row and NaN residuals (nothing is read for
 * it); offsets that are not a valid list layout give unspecified lists but no
 * access outside the arrays. No workspace is used.
 * Errors: IVF_EINVAL (sizes, positions, NULL pointers, misalignment,
 * aliasing), IVF_EUNSUPPORTED (D, N), IVF_EDEVICE. */
ivf_status ivf_list_major(ivf_ctx *ctx, const void *base, int dt, int64_t N,
                          const float *centroids, int64_t C, int32_t D, const int64_t *offsets,
                          const uint32_t *perm, int64_t pos0, int64_t n, void *out_rows,
                          float *out_residuals);

/* Product quantisation (the PQ encoding equation, Sec. "ANN Search and IVF";
 * applied to the residuals x - c(x), Sec. "Residual-PQ Candidate
 * Reduction"). A D-dim vector is cut into M sub-vectors of D / M consecutive
 * dims (M divides D, at most 16 dims per subspace); subspace m has 256
 * codewords codebooks[m][j][0 .. D/M), fp32, [M, 256, D/M] row-major.
 *
 * ivf_pq_encode: out_codes [n, M] uint8, code m of row i = the codeword of
 * subspace m nearest to sub-vector m of x[i] by (distance, index), the
 * distance in fp64 as in the exactness contract.
 *   x [n, D] fp32 (e.g. residuals from ivf_list_major); n == 0 is a no-op.
 * No workspace. Errors: IVF_EINVAL (M does not divide D, NULL, misaligned,
 * aliasing), IVF_EUNSUPPORTED (D, more than 16 dims per subspace). */
ivf_status ivf_pq_encode(ivf_ctx *ctx, const float *x, int64_t n, int32_t D, int32_t M,
                         const float *codebooks, uint8_t *out_codes);

/* One Lloyd iteration of every subspace codebook (codebook training for
 * residual PQ): subspace m runs exactly the ivf_kmeans_step definition on
 * the sub-vectors x[.][m D/M .. (m+1) D/M) with 256 centroids and seed + m
 * (fp64 sums in ascending row order; an empty codeword takes the
 * sub-vector of the reseed row).
 *   x              [n, D] fp32, 1 <= n <= 2^32 - 1
 *   codebooks      [M, 256, D/M] input codebooks
 *   out_codebooks  [M, 256, D/M], must not alias the input
 *   out_counts     [M, 256] int64 codeword populations before reseeding,
 *                  may be NULL
 *   out_objective  [M] fp64 device array: per subspace, the sum over rows of
 *                  the squared distance to the assigned input codeword, may
 *                  be NULL
 * Workspace: ivf_workspace_bytes(IVF_OP_PQ_TRAIN_STEP, n, M, D, 0).
 * Errors: as ivf_pq_encode, plus IVF_ENOMEM. */
ivf_status ivf_pq_train_step(ivf_ctx *ctx, const float *x, int64_t n, int32_t D, int32_t M,
                             const float *codebooks, uint64_t seed, int32_t iter,
                             float *out_codebooks, int64_t *out_counts, double *out_objective);

/* Residual-PQ approximate-distance scan of the probed lists (Sec.
 * "Residual-PQ Candidate Reduction": per probed list, the query residual
 * r = q - c_l, lookup tables LUT[m][j] = ||r^(m) - codeword_{m,j}||^2 and
 * ADC sums; Sec. "Compact PQ-Code Offloading": chunked scan with local
 * top-K and a hierarchical merge into a bounded handoff of N_rerank = k
 * candidates per query for exact re-ranking).
 * Definition: r = q - c_l in fp32; LUT[m][j] = the fp64 distance of the
 * contract rounded to fp32; for every position p of list l,
 * d~ = ((0 + LUT[0][a_0]) + LUT[1][a_1]) + ... in fp32 with a = codes[p];
 * the output is each query's k smallest (d~, perm[p]) pairs, ascending, with
 * missing entries id 0xFFFFFFFF and distance +inf. Exact: the kernels
 * reproduce these operations and select by the (d~, id) order.
 *   queries    [B, D] fp32          centroids [C, D] fp32
 *   probes     [B, P] int32 list ids (e.g. ivf_route output); ids outside
 *              [0, C) are skipped; the lists of a query must be distinct
 *   offsets    [C + 1] int64, perm [N] uint32: the list layout
 *              (ivf_assign_build)
 *   codes      [N, M] uint8 PQ codes in list-major order (ivf_pq_encode of
 *              the ivf_list_major residuals); M divides D, M <= 60
 *   codebooks  [M, 256, D/M] fp32
 *   k          handoff per query, 1 <= k <= 1024; P <= 4096
 *   out_ids    [B, k] uint32 row ids     out_dist [B, k] fp32
 * Workspace: ivf_workspace_bytes(IVF_OP_ADC_SCAN, B, P, D, k) = 8 B*P*k
 * bytes (+256): large batches can be scanned in slices of queries.
 * Errors: IVF_EINVAL, IVF_EUNSUPPORTED (D, M, N), IVF_ENOMEM, IVF_EDEVICE. */
ivf_status ivf_adc_scan(ivf_ctx *ctx, const float *queries, int64_t B, int32_t D,
                        const float *centroids, int64_t C, const int32_t *probes, int32_t P,
                        const int64_t *offsets, const uint32_t *perm, int64_t N,
                        const uint8_t *codes, int32_t M, const float *codebooks, int32_t k,
                        uint32_t *out_ids, float *out_dist);

/* Measures the fp32 MFMA pipe for reporting: enqueues a probe kernel that
 * runs only v_mfma_f32_32x32x2_f32 (register operands, two waves per SIMD on
 * every CU) for `iters` rounds of 16 instructions per wave (after one
 * untimed round that loads the kernel), waits for it
 * (this call synchronises the context's stream), and stores its duration in
 * *out_ms and its rate in *out_tflops (either may be NULL, not both).
 * Errors: IVF_EINVAL (iters outside [1, 2^20], both outputs NULL),
 * IVF_EUNSUPPORTED (validation-only context), IVF_EDEVICE. */
ivf_status ivf_mfma_probe(ivf_ctx *ctx, int32_t iters, float *out_ms, double *out_tflops);

/* The same measurement for the int8 MFMA pipe that screens uint8 rows:
 * v_mfma_i32_32x32x32_i8 with register operands holding pseudo-random bytes
 * (the part runs the int8 pipe at a power-limited clock on data that
 * toggles, well below the published peak), two waves per SIMD on every CU;
 * *out_tops in 1e12 int8 operations per second. Same arguments, errors and
 * synchronisation as ivf_mfma_probe. */
ivf_status ivf_mfma_probe_i8(ivf_ctx *ctx, int32_t iters, float *out_ms, double *out_tops);

/* Kernel timeline recorded while IVF_OPT_PROFILE is on, across calls, since
 * the last complete read: waits on the stream, then fills up to `max` entries
 * of names[] (strings owned by the context, valid until the next read) and
 * ms[] (event-to-event time of each launch, in launch order). Either array
 * may be NULL. When max >= the number recorded, the timeline is cleared.
 * Returns the number of launches recorded, or -1 on error. */
int ivf_kernel_times(ivf_ctx *ctx, int max, const char **names, float *ms);

#ifdef __cplusplus
}
#endif

#endif /* IVF_H */
