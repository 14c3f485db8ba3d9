/*
 * CPU oracle for the IVF hot path (InSituANN, arXiv 2608.08751).
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * benchmark's CPU-baseline leg; never by the product library.
 *
 * All arrays are host memory, row-major and contiguous. Functions return
 * ORACLE_OK or ORACLE_EINVAL (bad sizes, out-of-range labels); nothing else.
 * nthreads <= 0 means one thread per online CPU.
 */
#ifndef IVF_ORACLE_H
#define IVF_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_OK = 0, ORACLE_EINVAL = 1 };
enum { ORACLE_F32 = 0, ORACLE_U8 = 1 };

double oracle_dist(const float *x, const float *c, int D);
double oracle_dist_row(const void *x, int dtype, int64_t i, const float *c, int D);

int oracle_route(const float *queries, int64_t nq, const float *centroids, int64_t nc, int D,
                 int nprobe, int32_t *out_ids, float *out_dist, int nthreads);

int oracle_assign(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc, int D,
                  int32_t *out_labels, double *out_mindist, int nthreads);

int oracle_assign_graph(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc,
                        int D, const int32_t *graph, int S, const int32_t *prev,
                        int32_t *out_labels, double *out_mindist, int nthreads);

int oracle_assign_cells(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc, int D,
                        const int32_t *cell, int64_t G, const int64_t *cell_offsets,
                        const uint32_t *cell_members, int64_t n_members, const int32_t *graph, int S,
                        int hops, int32_t *out_labels, double *out_mindist, int nthreads);

uint64_t oracle_splitmix64_mix(uint64_t z);
uint64_t oracle_splitmix64_nth(uint64_t seed, uint64_t n);
int64_t oracle_reseed_row(uint64_t seed, int32_t iter, int64_t j, int64_t n);

int oracle_kmeans_update(const void *x, int dtype, int64_t n, int D, const int32_t *labels,
                         int64_t nc, uint64_t seed, int32_t iter, float *out_centroids,
                         int64_t *out_counts);
int oracle_objective(const void *x, int dtype, int64_t n, int D, const int32_t *labels,
                     const float *centroids, int64_t nc, double *out_j);
int oracle_kmeans_step(const void *x, int dtype, int64_t n, const float *centroids, int64_t nc,
                       int D, uint64_t seed, int32_t iter, int32_t *out_labels,
                       float *out_centroids, int64_t *out_counts, double *out_objective,
                       int nthreads);

int oracle_build_lists(const int32_t *labels, int64_t n, int64_t nc, int64_t *out_counts,
                       int64_t *out_offsets, uint32_t *out_perm);

int oracle_list_major(const void *x, int dtype, int64_t n_rows, const float *centroids, int64_t nc,
                      int D, const int32_t *labels, const uint32_t *perm, int64_t n,
                      void *out_rows, float *out_res);
int oracle_pq_encode(const float *x, int64_t n, int D, int M, const float *codebooks,
                     uint8_t *out_codes, int nthreads);
int oracle_pq_train_step(const float *x, int64_t n, int D, int M, const float *codebooks,
                         uint64_t seed, int32_t iter, float *out_codebooks, int64_t *out_counts,
                         double *out_objective, int nthreads);
int oracle_adc_scan(const float *queries, int64_t nq, int D, const float *centroids, int64_t nc,
                    const int32_t *probes, int P, const int64_t *offsets, const uint32_t *perm,
                    const uint8_t *codes, int M, const float *codebooks, int k,
                    uint32_t *out_ids, float *out_dist);
int oracle_num_threads(int nthreads);

#ifdef __cplusplus
}
#endif

#endif
