/*
 * CPU oracle for the IVF routing / construction hot path of InSituANN
 * (arXiv 2608.08751).
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, obviously correct
 * definition that the GPU path is checked against. Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product library never links, calls or falls back to it. It shares no code,
 * header, table or helper with the HIP path.
 *
 * Everything is computed in fp64 in a fixed, documented operation order and
 * compiled with -ffp-contract=off, so the only fused operation is the explicit
 * fma() below.
 *
 * What each function follows:
 *   oracle_dist          squared L2 distance, the left-hand side of Eq. (6)
 *                        (Sec. "GPU coarse search"), evaluated directly.
 *   oracle_route         coarse search, Eq. (1) (Sec. "ANN Search and IVF"):
 *                        the nprobe nearest centroids, ordered by (distance, id).
 *   oracle_assign        IVF construction: every vector goes to its nearest
 *                        centroid (Sec. "ANN Search and IVF"; Sec. "System
 *                        Architecture", index layout), ties to the lower id.
 *   oracle_kmeans_update Lloyd's mean update (k-means training cited in the
 *                        introduction and in "Fast Index Construction").
 *   oracle_build_lists   cluster-major inverted lists with offset, length and
 *                        vector ids (Sec. "System Architecture", index layout).
 *   oracle_assign_graph  candidate-restricted assignment (fast construction
 *                        mode, Sec. "Fast Index Construction").
 *   oracle_assign_cells  candidates for rows without a previous label: the
 *                        members of the row's coarse cell, then a greedy walk
 *                        over a centroid graph (Sec. "Fast Index Building
 *                        Details", graph-assisted assignment of the base).
 *   oracle_adc_scan      residual-PQ approximate-distance scan of the probed
 *                        lists with a bounded handoff (Sec. "Residual-PQ
 *                        Candidate Reduction", Sec. "Compact PQ-Code
 *                        Offloading").
 *   oracle_list_major    list-major copy of the vectors and their residuals
 *                        x - c(x) (Sec. "List-major contiguous scans" and
 *                        Sec. "Residual-PQ Candidate Reduction").
 *   oracle_pq_encode,    product quantisation of vectors (residuals) and one
 *   oracle_pq_train_step Lloyd step per subspace codebook (PQ encoding
 *                        equation, Sec. "ANN Search and IVF"; Sec.
 *                        "Residual-PQ Candidate Reduction").
 *   oracle_reseed_row    deterministic choice of a training row for an empty
 *                        cluster; the paper is silent, the reading is SplitMix64
 *                        (Steele, Lea & Flood, OOPSLA 2014).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include "oracle.h"

/* ---------------------------------------------------------------- helpers */

static int resolve_threads(int nthreads)
{
    if (nthreads > 0) return nthreads;
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

/* Runs body(ctx, begin, end) over [0, n) split into contiguous ranges. */
typedef void (*range_fn)(void *ctx, int64_t begin, int64_t end);
typedef struct {
    range_fn fn;
    void *ctx;
    int64_t begin, end;
} range_job;

static void *range_thread(void *arg)
{
    range_job *j = (range_job *)arg;
    j->fn(j->ctx, j->begin, j->end);
    return NULL;
}

static void parallel_for(int64_t n, int nthreads, range_fn fn, void *ctx)
{
    int t = resolve_threads(nthreads);
    if (t > n) t = (int)(n > 0 ? n : 1);
    if (t <= 1) {
        fn(ctx, 0, n);
        return;
    }
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)t);
    range_job *jobs = (range_job *)malloc(sizeof(range_job) * (size_t)t);
    for (int i = 0; i < t; ++i) {
        jobs[i].fn = fn;
        jobs[i].ctx = ctx;
        jobs[i].begin = n * i / t;
        jobs[i].end = n * (i + 1) / t;
        pthread_create(&th[i], NULL, range_thread, &jobs[i]);
    }
    for (int i = 0; i < t; ++i) pthread_join(th[i], NULL);
    free(th);
    free(jobs);
}

/* Element d of row i as a double, for either storage type. */
static double elem(const void *x, int dtype, int64_t i, int D, int d)
{
    if (dtype == ORACLE_U8) return (double)((const uint8_t *)x)[i * (int64_t)D + d];
    return (double)((const float *)x)[i * (int64_t)D + d];
}

/* ------------------------------------------------------------- distance */

/* Squared L2 distance ||x - c||^2: s = 0; for d ascending: t = x_d - c_d;
 * s = fma(t, t, s). All in fp64, round to nearest even. */
double oracle_dist_row(const void *x, int dtype, int64_t i, const float *c, int D)
{
    double s = 0.0;
    for (int d = 0; d < D; ++d) {
        double t = elem(x, dtype, i, D, d) - (double)c[d];
        s = fma(t, t, s);
    }
    return s;
}

double oracle_dist(const float *x, const float *c, int D)
{
    return oracle_dist_row(x, ORACLE_F32, 0, c, D);
}

/* (d1, id1) < (d2, id2) in the canonical total order used everywhere. */
static int before(double d1, int64_t id1, double d2, int64_t id2)
{
    return d1 < d2 || (d1 == d2 && id1 < id2);
}

/* ---------------------------------------------------------------- route */

typedef struct {
    const float *q;
    int64_t nq;
    const float *c;
    int64_t nc;
    int D;
    int k;
    int32_t *ids;
    float *dist;
} route_ctx;

static void route_range(void *vctx, int64_t begin, int64_t end)
{
    route_ctx *r = (route_ctx *)vctx;
    double *bd = (double *)malloc(sizeof(double) * (size_t)r->k);
    int64_t *bi = (int64_t *)malloc(sizeof(int64_t) * (size_t)r->k);
    for (int64_t qi = begin; qi < end; ++qi) {
        int have = 0;
        for (int64_t j = 0; j < r->nc; ++j) {
            double d = oracle_dist_row(r->q, ORACLE_F32, qi, r->c + j * r->D, r->D);
            if (have == r->k && !before(d, j, bd[have - 1], bi[have - 1])) continue;
            /* insert (d, j) into the sorted list, dropping the last if full */
            int pos = have < r->k ? have : r->k - 1;
            while (pos > 0 && before(d, j, bd[pos - 1], bi[pos - 1])) {
                bd[pos] = bd[pos - 1];
                bi[pos] = bi[pos - 1];
                --pos;
            }
            bd[pos] = d;
            bi[pos] = j;
            if (have < r->k) ++have;
        }
        for (int t = 0; t < r->k; ++t) {
            r->ids[qi * r->k + t] = (int32_t)bi[t];
            if (r->dist) r->dist[qi * r->k + t] = (float)bd[t];
        }
    }
    free(bd);
    free(bi);
}

int oracle_route(const float *queries, int64_t nq, const float *centroids, int64_t nc, int D,
                 int nprobe, int32_t *out_ids, float *out_dist, int nthreads)
{
    if (nq < 0 || nc < 1 || D < 1 || nprobe < 1 || nprobe > nc) return ORACLE_EINVAL;
    if (nq == 0) return ORACLE_OK;
    route_ctx ctx = {queries, nq, centroids, nc, D, nprobe, out_ids, out_dist};
    parallel_for(nq, nthreads, route_range, &ctx);
    return ORACLE_OK;
}

/* --------------------------------------------------------------- assign */

typedef struct {
    const void *x;
    int dtype;
    const float *c;
    int64_t nc;
    int D;
    int32_t *labels;
    double *mind;
} assign_ctx;

static void assign_range(void *vctx, int64_t begin, int64_t end)
{
    assign_ctx *a = (assign_ctx *)vctx;
    for (int64_t i = begin; i < end; ++i) {
        double best = 0.0;
        int64_t arg = -1;
        for (int64_t j = 0; j < a->nc; ++j) {
            double d = oracle_dist_row(a->x, a->dtype, i, a->c + j * a->D, a->D);
            if (arg < 0 || before(d, j, best, arg)) {
                best = d;
                arg = j;
            }
        }
        a->labels[i] = (int32_t)arg;
        if (a->mind) a->mind[i] = best;
    }
}

int oracle_assign(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc, int D,
                  int32_t *out_labels, double *out_mindist, int nthreads)
{
    if (n < 0 || nc < 1 || D < 1 || (dtype != ORACLE_F32 && dtype != ORACLE_U8)) return ORACLE_EINVAL;
    if (n == 0) return ORACLE_OK;
    assign_ctx ctx = {x, dtype, centroids, nc, D, out_labels, out_mindist};
    parallel_for(n, nthreads, assign_range, &ctx);
    return ORACLE_OK;
}

/* Candidate-restricted assignment (the fast construction mode of Sec. "Fast
 * Index Construction", which scores every vector against a few candidate
 * centroids only): the candidates of row i are graph[prev[i]][0 .. S), and
 * label_i is the candidate of smallest distance by (distance, id). The paper
 * draws its candidates from a CAGRA search over the centroids; here the
 * graph is any [nc, S] table of centroid ids (e.g. each centroid's S nearest
 * centroids) and prev[i] is the row's previous label. Candidate ids outside
 * [0, nc) are skipped; a row with none gets label -1 and distance +inf. */
typedef struct {
    const void *x;
    int dtype;
    const float *c;
    int64_t nc;
    int D;
    const int32_t *graph;
    int S;
    const int32_t *prev;
    int32_t *labels;
    double *mind;
} graph_ctx;

static void graph_range(void *vctx, int64_t begin, int64_t end)
{
    graph_ctx *a = (graph_ctx *)vctx;
    for (int64_t i = begin; i < end; ++i) {
        double best = INFINITY;
        int64_t arg = -1;
        const int32_t p = a->prev[i];
        if (p >= 0 && p < a->nc) {
            for (int s = 0; s < a->S; ++s) {
                const int64_t j = a->graph[(int64_t)p * a->S + s];
                if (j < 0 || j >= a->nc) continue;
                const double d = oracle_dist_row(a->x, a->dtype, i, a->c + j * a->D, a->D);
                if (arg < 0 || before(d, j, best, arg)) {
                    best = d;
                    arg = j;
                }
            }
        }
        a->labels[i] = (int32_t)arg;
        if (a->mind) a->mind[i] = best;
    }
}

int oracle_assign_graph(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc,
                        int D, const int32_t *graph, int S, const int32_t *prev,
                        int32_t *out_labels, double *out_mindist, int nthreads)
{
    if (n < 0 || nc < 1 || D < 1 || S < 1 || (dtype != ORACLE_F32 && dtype != ORACLE_U8))
        return ORACLE_EINVAL;
    if (n == 0) return ORACLE_OK;
    graph_ctx ctx = {x, dtype, centroids, nc, D, graph, S, prev, out_labels, out_mindist};
    parallel_for(n, nthreads, graph_range, &ctx);
    return ORACLE_OK;
}

/* Candidate source for rows that have no previous label (the graph-assisted
 * assignment of the full base set, Sec. "Fast Index Building Details"): a
 * coarse partition of the centroid table into G cells (each centroid a member
 * of one cell) gives the first candidates, and a greedy walk over a graph of
 * centroids refines them. Row i is given its cell cell[i] (e.g. its nearest
 * coarse centroid). Its first choice b is the member of that cell of smallest
 * (distance, id); members are members[offsets[c] .. offsets[c + 1]), the two
 * offsets clamped into [0, n_members] (the second at least the first), and
 * member ids outside [0, nc) are skipped. Then up to `hops` times: among the
 * valid ids graph[b][0 .. S) take the one of smallest (distance, id); if it
 * comes before b in (distance, id) order it becomes b, otherwise the walk
 * stops. The label is the final b; a row whose cell lies outside [0, G) or
 * holds no valid member gets -1 and distance +inf. */
typedef struct {
    const void *x;
    int dtype;
    const float *c;
    int64_t nc;
    int D;
    const int32_t *cell;
    int64_t G;
    const int64_t *offsets;
    const uint32_t *members;
    int64_t n_members;
    const int32_t *graph;
    int S;
    int hops;
    int32_t *labels;
    double *mind;
} cells_ctx;

static void cells_range(void *vctx, int64_t begin, int64_t end)
{
    cells_ctx *a = (cells_ctx *)vctx;
    for (int64_t i = begin; i < end; ++i) {
        double best = INFINITY;
        int64_t arg = -1;
        const int32_t g = a->cell[i];
        if (g >= 0 && g < a->G) {
            int64_t m0 = a->offsets[g], m1 = a->offsets[g + 1];
            if (m0 < 0) m0 = 0;
            if (m0 > a->n_members) m0 = a->n_members;
            if (m1 < m0) m1 = m0;
            if (m1 > a->n_members) m1 = a->n_members;
            for (int64_t e = m0; e < m1; ++e) {
                const int64_t j = a->members[e];
                if (j >= a->nc) continue;
                const double d = oracle_dist_row(a->x, a->dtype, i, a->c + j * a->D, a->D);
                if (arg < 0 || before(d, j, best, arg)) {
                    best = d;
                    arg = j;
                }
            }
        }
        for (int h = 0; arg >= 0 && a->graph && h < a->hops; ++h) {
            double nb = INFINITY;
            int64_t narg = -1;
            for (int s = 0; s < a->S; ++s) {
                const int64_t j = a->graph[arg * a->S + s];
                if (j < 0 || j >= a->nc) continue;
                const double d = oracle_dist_row(a->x, a->dtype, i, a->c + j * a->D, a->D);
                if (narg < 0 || before(d, j, nb, narg)) {
                    nb = d;
                    narg = j;
                }
            }
            if (narg < 0 || !before(nb, narg, best, arg)) break;
            best = nb;
            arg = narg;
        }
        a->labels[i] = (int32_t)arg;
        if (a->mind) a->mind[i] = best;
    }
}

int oracle_assign_cells(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc, int D,
                        const int32_t *cell, int64_t G, const int64_t *cell_offsets,
                        const uint32_t *cell_members, int64_t n_members, const int32_t *graph, int S,
                        int hops, int32_t *out_labels, double *out_mindist, int nthreads)
{
    if (n < 0 || nc < 1 || D < 1 || G < 1 || n_members < 0 || hops < 0 || (graph && S < 1) ||
        (dtype != ORACLE_F32 && dtype != ORACLE_U8))
        return ORACLE_EINVAL;
    if (n == 0) return ORACLE_OK;
    cells_ctx ctx = {x, dtype, centroids, nc, D, cell, G, cell_offsets, cell_members, n_members,
                     graph, S, hops, out_labels, out_mindist};
    parallel_for(n, nthreads, cells_range, &ctx);
    return ORACLE_OK;
}

/* ---------------------------------------------------------- k-means update */

/* SplitMix64 (Steele, Lea & Flood 2014): the generator state advances by the
 * odd constant gamma, and each output is the state passed through the
 * variant-13 finaliser. The n-th output (n >= 1) of a generator seeded with s
 * is therefore mix(s + n * gamma). */
#define SPLITMIX_GAMMA 0x9E3779B97F4A7C15ULL

uint64_t oracle_splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t oracle_splitmix64_nth(uint64_t seed, uint64_t n)
{
    return oracle_splitmix64_mix(seed + n * SPLITMIX_GAMMA);
}

/* Row that replaces empty cluster j at Lloyd iteration `iter`: the output
 * number ((iter << 32) | j) + 1 of SplitMix64 seeded with `seed`, mod N. */
int64_t oracle_reseed_row(uint64_t seed, int32_t iter, int64_t j, int64_t n)
{
    uint64_t key = ((uint64_t)(uint32_t)iter << 32) | (uint64_t)(uint32_t)j;
    return (int64_t)(oracle_splitmix64_nth(seed, key + 1) % (uint64_t)n);
}

/* Lloyd update for fixed labels.
 *   counts_j = #{i : label_i = j}                      (before any reseed)
 *   S_j      = sum of x_i with label j, in ascending i: an exact integer sum
 *              for u8 data, a left-to-right fp64 sum for f32 data
 *   c'_j     = (float)(S_j / (double)counts_j)          when counts_j > 0
 *   c'_j     = (float)x_r, r = oracle_reseed_row(...)   when counts_j = 0 */
int oracle_kmeans_update(const void *x, int dtype, int64_t n, int D, const int32_t *labels,
                         int64_t nc, uint64_t seed, int32_t iter, float *out_centroids,
                         int64_t *out_counts)
{
    if (n < 1 || nc < 1 || D < 1 || (dtype != ORACLE_F32 && dtype != ORACLE_U8)) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i)
        if (labels[i] < 0 || labels[i] >= nc) return ORACLE_EINVAL;

    int64_t *counts = (int64_t *)calloc((size_t)nc, sizeof(int64_t));
    double *fsum = NULL;
    uint64_t *isum = NULL;
    if (dtype == ORACLE_U8)
        isum = (uint64_t *)calloc((size_t)(nc * D), sizeof(uint64_t));
    else
        fsum = (double *)calloc((size_t)(nc * D), sizeof(double));

    for (int64_t i = 0; i < n; ++i) {
        int64_t j = labels[i];
        counts[j] += 1;
        for (int d = 0; d < D; ++d) {
            if (isum)
                isum[j * D + d] += ((const uint8_t *)x)[i * D + d];
            else
                fsum[j * D + d] = fsum[j * D + d] + (double)((const float *)x)[i * D + d];
        }
    }
    for (int64_t j = 0; j < nc; ++j) {
        if (counts[j] > 0) {
            for (int d = 0; d < D; ++d) {
                double s = isum ? (double)isum[j * D + d] : fsum[j * D + d];
                out_centroids[j * D + d] = (float)(s / (double)counts[j]);
            }
        } else {
            int64_t r = oracle_reseed_row(seed, iter, j, n);
            for (int d = 0; d < D; ++d) out_centroids[j * D + d] = (float)elem(x, dtype, r, D, d);
        }
        if (out_counts) out_counts[j] = counts[j];
    }
    free(counts);
    free(isum);
    free(fsum);
    return ORACLE_OK;
}

/* J = sum_i dist(x_i, c_{label_i}), accumulated in fp64 in ascending i. */
int oracle_objective(const void *x, int dtype, int64_t n, int D, const int32_t *labels,
                     const float *centroids, int64_t nc, double *out_j)
{
    if (n < 0 || nc < 1 || D < 1) return ORACLE_EINVAL;
    double j = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        if (labels[i] < 0 || labels[i] >= nc) return ORACLE_EINVAL;
        j = j + oracle_dist_row(x, dtype, i, centroids + (int64_t)labels[i] * D, D);
    }
    *out_j = j;
    return ORACLE_OK;
}

/* One Lloyd iteration: assignment against the input centroids, then the
 * update, then the objective of the assignment (against the input centroids). */
int oracle_kmeans_step(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc,
                       int D, uint64_t seed, int32_t iter, int32_t *out_labels,
                       float *out_centroids, int64_t *out_counts, double *out_objective,
                       int nthreads)
{
    int rc = oracle_assign(x, dtype, n, centroids, nc, D, out_labels, NULL, nthreads);
    if (rc != ORACLE_OK) return rc;
    rc = oracle_kmeans_update(x, dtype, n, D, out_labels, nc, seed, iter, out_centroids, out_counts);
    if (rc != ORACLE_OK) return rc;
    if (out_objective) rc = oracle_objective(x, dtype, n, D, out_labels, centroids, nc, out_objective);
    return rc;
}

/* ----------------------------------------------------------- list build */

/* counts = histogram of labels; offsets = exclusive prefix sum of counts
 * (offsets[nc] = n); perm = ids 0..n-1 ordered by (label, id), i.e. a
 * counting sort that keeps ids ascending inside each list. */
int oracle_build_lists(const int32_t *labels, int64_t n, int64_t nc, int64_t *out_counts,
                       int64_t *out_offsets, uint32_t *out_perm)
{
    if (n < 0 || nc < 1 || n > (int64_t)UINT32_MAX) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i)
        if (labels[i] < 0 || labels[i] >= nc) return ORACLE_EINVAL;
    memset(out_counts, 0, sizeof(int64_t) * (size_t)nc);
    for (int64_t i = 0; i < n; ++i) out_counts[labels[i]] += 1;
    out_offsets[0] = 0;
    for (int64_t j = 0; j < nc; ++j) out_offsets[j + 1] = out_offsets[j] + out_counts[j];
    int64_t *cursor = (int64_t *)malloc(sizeof(int64_t) * (size_t)nc);
    memcpy(cursor, out_offsets, sizeof(int64_t) * (size_t)nc);
    for (int64_t i = 0; i < n; ++i) out_perm[cursor[labels[i]]++] = (uint32_t)i;
    free(cursor);
    return ORACLE_OK;
}

/* ------------------------------------------------ list-major layout */

/* List-major copy of the base vectors and their residuals (Sec. "List-major
 * contiguous scans": vectors stored in list order; Sec. "Residual-PQ
 * Candidate Reduction", residual encoding: r = x - c(x) with c(x) the
 * assigned centroid). For output position i, row = perm[i]:
 *   out_rows[i]    = x[row]                       (same element type)
 *   out_res[i][d]  = (float)x[row][d] - c[labels[row]][d]   (one fp32
 *                    subtraction: the exact difference rounded once)
 * Either output may be NULL. */
int oracle_list_major(const void *x, int dtype, int64_t n_rows, const float *centroids, int64_t nc,
                      int D, const int32_t *labels, const uint32_t *perm, int64_t n,
                      void *out_rows, float *out_res)
{
    if (n_rows < 0 || n < 0 || nc < 1 || D < 1 || (dtype != ORACLE_F32 && dtype != ORACLE_U8))
        return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        if ((int64_t)perm[i] >= n_rows) return ORACLE_EINVAL;
        const int32_t l = labels[perm[i]];
        if (l < 0 || l >= nc) return ORACLE_EINVAL;
    }
    for (int64_t i = 0; i < n; ++i) {
        const int64_t row = (int64_t)perm[i];
        const float *c = centroids + (int64_t)labels[row] * D;
        for (int d = 0; d < D; ++d) {
            float v;
            if (dtype == ORACLE_U8) {
                const uint8_t b = ((const uint8_t *)x)[row * D + d];
                v = (float)b;
                if (out_rows) ((uint8_t *)out_rows)[i * D + d] = b;
            } else {
                v = ((const float *)x)[row * D + d];
                if (out_rows) ((float *)out_rows)[i * D + d] = v;
            }
            if (out_res) {
                const float diff = v - c[d];
                out_res[i * D + d] = diff;
            }
        }
    }
    return ORACLE_OK;
}

/* --------------------------------------------------- product quantisation */

/* Product quantisation (Sec. "ANN Search and IVF", the PQ encoding equation;
 * applied to residuals in Sec. "Residual-PQ Candidate Reduction"): a vector
 * of D dims is cut into M sub-vectors of D/M consecutive dims, subspace m
 * has K = 256 codewords codebooks[m][j][.], and code m of a vector is the
 * nearest codeword of its sub-vector by (distance, index). Training is one
 * Lloyd step per subspace on the sub-vectors, exactly oracle_kmeans_step with
 * seed + m (reseeding an empty codeword of subspace m from the sub-vectors).
 * Both take the sub-vectors out of x into a contiguous copy first. */
#define ORACLE_PQ_K 256

static float *pq_slice(const float *x, int64_t n, int D, int m, int dsub)
{
    float *s = (float *)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1) * (size_t)dsub);
    if (!s) return NULL;
    for (int64_t i = 0; i < n; ++i)
        for (int d = 0; d < dsub; ++d) s[i * dsub + d] = x[i * D + (int64_t)m * dsub + d];
    return s;
}

int oracle_pq_encode(const float *x, int64_t n, int D, int M, const float *codebooks,
                     uint8_t *out_codes, int nthreads)
{
    if (n < 0 || D < 1 || M < 1 || D % M != 0) return ORACLE_EINVAL;
    const int dsub = D / M;
    int32_t *lab = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    if (!lab) return ORACLE_EINVAL;
    int rc = ORACLE_OK;
    for (int m = 0; m < M && rc == ORACLE_OK; ++m) {
        float *s = pq_slice(x, n, D, m, dsub);
        if (!s) { rc = ORACLE_EINVAL; break; }
        if (n > 0)
            rc = oracle_assign(s, ORACLE_F32, n, codebooks + (int64_t)m * ORACLE_PQ_K * dsub, ORACLE_PQ_K,
                               dsub, lab, NULL, nthreads);
        for (int64_t i = 0; i < n && rc == ORACLE_OK; ++i) out_codes[i * M + m] = (uint8_t)lab[i];
        free(s);
    }
    free(lab);
    return rc;
}

int oracle_pq_train_step(const float *x, int64_t n, int D, int M, const float *codebooks,
                         uint64_t seed, int32_t iter, float *out_codebooks, int64_t *out_counts,
                         double *out_objective, int nthreads)
{
    if (n < 1 || D < 1 || M < 1 || D % M != 0) return ORACLE_EINVAL;
    const int dsub = D / M;
    int32_t *lab = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
    if (!lab) return ORACLE_EINVAL;
    int rc = ORACLE_OK;
    for (int m = 0; m < M && rc == ORACLE_OK; ++m) {
        float *s = pq_slice(x, n, D, m, dsub);
        if (!s) { rc = ORACLE_EINVAL; break; }
        const int64_t cb = (int64_t)m * ORACLE_PQ_K * dsub;
        rc = oracle_kmeans_step(s, ORACLE_F32, n, codebooks + cb, ORACLE_PQ_K, dsub, seed + (uint64_t)m,
                                iter, lab, out_codebooks + cb,
                                out_counts ? out_counts + (int64_t)m * ORACLE_PQ_K : NULL,
                                out_objective ? out_objective + m : NULL, nthreads);
        free(s);
    }
    free(lab);
    return rc;
}

/* ------------------------------------------------ residual-PQ ADC scan */

/* Approximate-distance scan of the probed lists (Sec. "Residual-PQ Candidate
 * Reduction": lookup table and ADC sum; Sec. "Compact PQ-Code Offloading":
 * the bounded per-query handoff of N_rerank candidates). For query b and
 * each probed list l = probes[b][s] (ids outside [0, nc) are skipped):
 *   r[d]        = q[d] - c_l[d]                      (fp32 subtraction)
 *   LUT[m][j]   = (float) dist(r^(m), cb[m][j])       (fp64 distance of the
 *                 contract, rounded to fp32: the paper's fp32 LUTs)
 *   d~(x)       = ((0 + LUT[0][a_0]) + LUT[1][a_1]) + ... + LUT[M-1][a_M-1]
 *                 (fp32 additions in subspace order) for every position p of
 *                 list l, a = codes[p], candidate id = perm[p]
 * and out_ids/out_dist[b] are the k smallest candidates by (d~, id),
 * ascending; missing entries are id 0xFFFFFFFF and +inf. */
typedef struct {
    float d;
    uint32_t id;
} adc_cand;

static int adc_before(const void *pa, const void *pb)
{
    const adc_cand *a = (const adc_cand *)pa, *b = (const adc_cand *)pb;
    if (a->d != b->d) return a->d < b->d ? -1 : 1;
    return a->id < b->id ? -1 : (a->id > b->id ? 1 : 0);
}

int oracle_adc_scan(const float *queries, int64_t nq, int D, const float *centroids, int64_t nc,
                    const int32_t *probes, int P, const int64_t *offsets, const uint32_t *perm,
                    const uint8_t *codes, int M, const float *codebooks, int k,
                    uint32_t *out_ids, float *out_dist)
{
    if (nq < 0 || D < 1 || nc < 1 || P < 1 || M < 1 || D % M != 0 || k < 1) return ORACLE_EINVAL;
    const int dsub = D / M;
    float *r = (float *)malloc(sizeof(float) * (size_t)D);
    float *lut = (float *)malloc(sizeof(float) * (size_t)M * ORACLE_PQ_K);
    if (!r || !lut) {
        free(r);
        free(lut);
        return ORACLE_EINVAL;
    }
    int rc = ORACLE_OK;
    for (int64_t b = 0; b < nq && rc == ORACLE_OK; ++b) {
        int64_t total = 0;
        for (int s = 0; s < P; ++s) {
            const int32_t l = probes[b * P + s];
            if (l >= 0 && l < nc) total += offsets[l + 1] - offsets[l];
        }
        adc_cand *cand = (adc_cand *)malloc(sizeof(adc_cand) * (size_t)(total > 0 ? total : 1));
        if (!cand) {
            rc = ORACLE_EINVAL;
            break;
        }
        int64_t nc_b = 0;
        for (int s = 0; s < P; ++s) {
            const int32_t l = probes[b * P + s];
            if (l < 0 || l >= nc) continue;
            for (int d = 0; d < D; ++d) r[d] = queries[b * D + d] - centroids[(int64_t)l * D + d];
            for (int m = 0; m < M; ++m)
                for (int j = 0; j < ORACLE_PQ_K; ++j)
                    lut[m * ORACLE_PQ_K + j] = (float)oracle_dist(
                        r + m * dsub, codebooks + ((int64_t)m * ORACLE_PQ_K + j) * dsub, dsub);
            for (int64_t p = offsets[l]; p < offsets[l + 1]; ++p) {
                float acc = 0.0f;
                for (int m = 0; m < M; ++m) acc = acc + lut[m * ORACLE_PQ_K + codes[p * M + m]];
                cand[nc_b].d = acc;
                cand[nc_b].id = perm[p];
                ++nc_b;
            }
        }
        qsort(cand, (size_t)nc_b, sizeof(adc_cand), adc_before);
        for (int t = 0; t < k; ++t) {
            out_ids[b * k + t] = t < nc_b ? cand[t].id : 0xFFFFFFFFu;
            out_dist[b * k + t] = t < nc_b ? cand[t].d : INFINITY;
        }
        free(cand);
    }
    free(r);
    free(lut);
    return rc;
}

int oracle_num_threads(int nthreads) { return resolve_threads(nthreads); }
