// Internal declarations of the gfx950 IVF library: launch parameters shared
// between the C-ABI layer (api.cpp) and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ivf {

// ---- screening kernel geometry -------------------------------------------
// One workgroup = W wave64s (4 or 8). Each wave owns 32 rows (queries or data
// vectors) whose fp32 values live in registers as MFMA B fragments; all waves
// share a chunk of kChunk centroids staged in LDS (double-buffered). 8/W
// workgroups run per CU (two waves per SIMD).
constexpr int kChunk = 64;

enum ScreenMode { kModeKeys = 0, kModeFilter = 1, kModeTop1 = 2 };
enum RowType { kRowF32 = 0, kRowU8 = 1 };

// Stats slots (uint64 each) in the workspace scalar area.
enum StatSlot {
    kStatFallback = 0,
    kStatRefine2 = 1,
    kStatCandidates = 2,
    kStatOverflow = 3,
    kStatSample = 4,
    kStatScreenI8 = 5,  // 1 when the uint8 rows were screened on int8 MFMA
    kStatRescreen = 6,  // rows the single-plane int8 screen left to the two-plane screen
    kNumStats = 8
};

struct ScreenArgs {
    const void *rows;       // [nrows, D] fp32 or u8
    int64_t nrows;
    int D;
    const float *cent;      // [C, D]
    const float *cnorm;     // [C] fl32(||c||^2)
    int64_t c_begin;        // first centroid of the range (multiple of kChunk)
    int64_t c_end;          // one past the last centroid of the range
    int64_t nchunks;        // chunks of kChunk centroids the kernel visits
    // chunk k of the visit is physical chunk (c_begin / kChunk) + k, except:
    // keys mode with cstride > 1: chunk k * cstride (a spread sample); filter
    // mode with skip_n > 0: the k-th chunk that is not one of the skip_n
    // sampled chunks j * skip_s
    int64_t cstride;
    int64_t skip_n, skip_s;
    // keys mode
    float *keys;            // [nrows, nchunks * kChunk]
    float *kmin;            // [nrows, nchunks * kChunk / 16]: the minimum of every 16 keys
    // filter mode
    const float *tau;       // [nrows]
    uint32_t *cand_cnt;     // [nrows]
    uint2 *cand;            // [nrows, L] (key bits, centroid id)
    int L;
    // top-1 mode
    const uint32_t *mc2_bits;  // max_j fl32(||c_j||^2) as float bits
    double bound_coef;         // gamma_{DP+2} with u = 2^-23
    int32_t *labels;           // [nrows]
    int32_t *wl;               // fallback worklist
    uint32_t *wl_cnt;
    int64_t wl_cap;
    unsigned long long *stats;
    int force_fallback;
    // when non-null and *gate == 0, the int8 screen has taken the call and
    // this kernel returns at once
    const uint32_t *gate;
};

// waves: 4 or 8 per workgroup; the grid fills every CU with two waves per SIMD.
hipError_t launch_screen(int mode, int rowtype, int DP, const ScreenArgs &a, int waves, int num_cus,
                         hipStream_t s);

// ---- int8 screening of uint8 rows (screen_i8.hip) ---------------------------
// Quantised centroids: qc [cpad][2 * DP] int8 (plane H, then plane Ls), negb
// [cpad] int32 (-B); cpad = C rounded up to 64, the padding scores lowest.
struct ScreenI8Args {
    const uint8_t *rows;   // [nrows, D]
    int64_t nrows;
    int D;
    const float *cent;     // [C, D] (exact re-evaluation)
    const int8_t *qc;
    const int32_t *negb;
    int64_t cpad;
    int64_t nchunks;       // cpad / 64
    const uint32_t *q_bad; // nonzero: some centroid did not quantise, fp32 takes over
    int32_t *labels;
    int32_t *wl;
    uint32_t *wl_cnt;
    int64_t wl_cap;
    unsigned long long *stats;
    int force_fallback;
    // rows left by the single-plane screen (null: screen every row); when
    // *q_bad1 is set or the list overflowed, every row is screened
    const int32_t *list;
    const uint32_t *list_cnt;
    int64_t list_cap;
    const uint32_t *q_bad1;
    // single-plane screen (DP <= 128): plane [quantized_pad1(ncent)][DP]
    // int8, biases -b1 (the launcher sets its own cpad and nchunks from ncent),
    // the largest coordinate residual (float bits), real centroid count, and
    // a test knob that lists every row for the two-plane screen
    const int8_t *qc1;
    const int32_t *negb1;
    const uint32_t *e_bits;
    const uint32_t *r2_bits;  // the largest residual norm ||c' - H1||_2 (float bits; null: E only)
    int64_t ncent;
    int force_rescreen;
    // single plane: a label per row from an earlier step, or null; the row's
    // keep threshold starts from that centroid's score (speed only)
    const int32_t *hint;
    // single plane in visiting order (null: id order): plane row p holds
    // centroid ord1[p], and centroid c sits at plane row pos1[c]
    const uint32_t *ord1;
    const int32_t *pos1;
};
int64_t quantized_pad(int64_t C);
// the single plane (qc1, negb1) is padded to whole staged chunks of 256
int64_t quantized_pad1(int64_t C);
// skip (may be null): when *skip is nonzero the kernel does nothing
hipError_t launch_quantize_centroids(const float *cent, int64_t C, int D, int DP, int8_t *qc, int32_t *negb,
                                     uint32_t *q_bad, hipStream_t s, const uint32_t *skip = nullptr);
// Eight waves per workgroup (two per SIMD), one workgroup per CU.
hipError_t launch_screen_i8(int DP, const ScreenI8Args &a, int num_cus, hipStream_t s);
// Single-plane int8 screen (DP <= 128): plane rint(c - 128) [quantized_pad1(C)][DP],
// biases, *q_bad1 when some centroid does not fit, *e_bits = the largest
// coordinate residual as float bits (both zeroed by the caller).
// ord (null: id order) puts centroid ord[p] at plane row p and records
// pos[ord[p]] = p.
hipError_t launch_quantize_centroids1(const float *cent, int64_t C, int D, int DP, int8_t *q1, int32_t *negb1,
                                      uint32_t *q_bad1, uint32_t *e_bits, uint32_t *r2_bits, hipStream_t s,
                                      const uint32_t *ord = nullptr, int32_t *pos = nullptr);
// Visiting order of the single plane: keys[c] = a 15-bit bucket of
// ||c - mean||^2 (mean over the centroids; the float's exponent and top 7
// mantissa bits, so buckets are 0.8 % wide at any scale). part holds
// order1_parts(C) x D doubles, mean D floats.
constexpr int kOrder1Keys = 32768;
int64_t order1_parts(int64_t C);
hipError_t launch_order1_keys(const float *cent, int64_t C, int D, double *part, float *mean, int32_t *keys,
                              hipStream_t s);
hipError_t launch_screen_i8_single(int DP, const ScreenI8Args &a, int num_cus, hipStream_t s);

// ---- norms, selection, fallbacks (select.hip) -----------------------------
hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t s);
hipError_t launch_centroid_norms(const float *cent, int64_t C, int D, float *cnorm,
                                 uint32_t *mc2_bits, hipStream_t s);
hipError_t launch_row_norms(const float *rows, int64_t n, int D, double *out, hipStream_t s);

struct RouteArgs {
    const float *queries;  // [nq, D] (already offset to the batch)
    int64_t nq;
    const float *cent;
    int64_t C;
    int D;
    int k;
    int L;
    int64_t Cs;             // centroids in the threshold sample
    int64_t sstride;        // the sample is the chunks j * sstride of kChunk centroids (0: 1)
    int rank_j;
    const float *keys;      // [nq, Cs]
    const float *kmin;      // [nq, Cs / 16] the minimum of every 16 sample keys (fp32 keys)
    float *tau;             // [nq]
    uint32_t *cand_cnt;     // [nq]
    uint2 *cand;            // [nq, L]
    const double *qn2;      // [nq]
    const uint32_t *mc2_bits;
    double bound_coef;
    int force_fallback;
    int32_t *out_ids;       // [nq, k]
    float *out_dist;        // [nq, k] or null
    int32_t *wl;            // [nq]
    uint32_t *wl_cnt;
    unsigned long long *stats;
    // keys from the int8 route kernels while *i8_off == 0 (null: fp32 only):
    // their per-query bound qbound replaces the fp32 key bound
    const uint32_t *i8_off;
    const float *qbound;    // [nq]
};

hipError_t launch_route_threshold(const RouteArgs &a, hipStream_t s);
// Int8 routing of uint8-valued queries on the two quantised planes
// (screen_i8.hip): keys of the threshold sample and the candidate filter,
// run only while *off == 0; route_i8_check raises *off when some query value
// is not an integer in [0, 255], route_i8_bound when *q_bad is set, and
// writes the per-query bound of the int8 keys.
constexpr int kQuantChunk = 64;  // centroids per staged chunk of the two-plane kernels
constexpr int kRouteKeys = 0;
constexpr int kRouteFilter = 1;
struct RouteI8Args {
    const float *queries;   // [nq, D]
    int64_t nq;
    int D;
    const int8_t *qc;       // two planes [cpad][2 DP] and biases [cpad] (quantize_kernel)
    const int32_t *negb;
    int64_t cpad;
    int64_t c_begin, c_end; // centroid range; chunks of 64 from c_begin
    int64_t nchunks;
    int64_t cstride;        // keys mode: chunk k of the range is physical chunk k * cstride (0: 1)
    const uint32_t *off;
    float *keys;            // keys mode: group minima [nq, (c_end - c_begin) / 16] (c_begin, c_end multiples of 16)
    const float *tau;       // filter mode: [nq], lists [nq, L]
    uint32_t *cand_cnt;
    uint2 *cand;
    int L;
    unsigned long long *stats;  // [kStatScreenI8] = 1 when the int8 filter ran
};
hipError_t launch_route_i8_check(const float *queries, int64_t nq, int D, uint32_t *off, hipStream_t s);
hipError_t launch_route_i8_bound(const float *queries, int64_t nq, int D, const uint32_t *q_bad, uint32_t *off,
                                 float *qbound, hipStream_t s);
hipError_t launch_route_i8(int mode, int DP, const RouteI8Args &a, int num_cus, hipStream_t s);
hipError_t launch_route_select(const RouteArgs &a, hipStream_t s);
hipError_t launch_route_fallback(const RouteArgs &a, int grid, hipStream_t s);

// Exact fp64 scan of the rows on the assignment worklist (labels -1). The
// first kFbSplitWindows windows of 8 rows are split into kFbSeg centroid
// segments over the whole grid; split_d / split_i hold their partial
// results (kFbSplitWindows * kFbSeg * 8 entries each).
constexpr int kFbSplitWindows = 256;
constexpr int kFbSeg = 64;
constexpr int64_t kFbSplitEntries = (int64_t)kFbSplitWindows * kFbSeg * 8;
hipError_t launch_assign_fallback(const void *rows, int rowtype, int64_t N, int D,
                                  const float *cent, int64_t C, int32_t *labels,
                                  const int32_t *wl, const uint32_t *wl_cnt, int64_t wl_cap,
                                  double *split_d, int32_t *split_i, int grid, hipStream_t s);

// ---- inverted-list build (lists.hip) ---------------------------------------
constexpr int kSlice = 16384;    // buckets per workgroup (LDS counters)
constexpr int kBuildThreads = 1024;
constexpr int kSub = 4096;       // rows per scatter sub-chunk (4 per thread)

struct BuildPlan {
    int64_t N, C;
    int nslices;
    int nblocks;
    int64_t R;               // rows per block (multiple of kSub)
};
// max_blocks > 0 caps the number of row blocks (fewer open write frontiers)
BuildPlan plan_build(int64_t N, int64_t C, int num_cus, int max_blocks = 0);
size_t build_scratch_bytes(const BuildPlan &p);  // count matrix bytes
hipError_t launch_build_hist(const BuildPlan &p, const int32_t *labels, uint32_t *cntmat,
                             hipStream_t s);
hipError_t launch_build_scan(const BuildPlan &p, uint32_t *cntmat, int64_t *counts, int64_t *offsets,
                             hipStream_t s);
hipError_t launch_build_scatter(const BuildPlan &p, const int32_t *labels, const uint32_t *cntmat,
                                const int64_t *offsets, uint32_t *perm, hipStream_t s);

// ---- inverted-list build for C <= 65,536 (lists_radix.hip) -----------------
constexpr int64_t kRadixMaxLists = 65536;

struct RadixPlan {
    int64_t N, C;
    int64_t R0;      // rows per level-0 block (multiple of the 4,096-row tile)
    int nblocks0;
    int64_t R1;      // rows per level-1 sub-block
    int max_sub1;    // upper bound on the number of level-1 sub-blocks
};
struct RadixScratch {
    uint32_t *cnt0, *tot0, *astart, *sbstart, *cnt1, *tmp_ids;
    uint8_t *tmp_lo;
};
RadixPlan plan_radix(int64_t N, int64_t C, int num_cus);
size_t radix_scratch_bytes(const RadixPlan &p);
RadixScratch carve_radix(const RadixPlan &p, void *base);
hipError_t launch_radix_level0(const RadixPlan &p, const int32_t *labels, const RadixScratch &s,
                               hipStream_t st);
hipError_t launch_radix_level1_counts(const RadixPlan &p, const RadixScratch &s, int64_t *counts,
                                      hipStream_t st);
hipError_t launch_radix_level1_scatter(const RadixPlan &p, const RadixScratch &s, const int64_t *offsets,
                                       uint32_t *perm, hipStream_t st);
hipError_t launch_offsets(const int64_t *counts, int64_t C, int64_t *offsets, hipStream_t st);

// ---- k-means update (kmeans.hip) --------------------------------------------
// `groups` independent problems in one launch (product-quantisation
// subspaces): group g's rows start g * x_group elements further, its
// centroids, counts, offsets, permutation and objective parts follow the
// previous group's, its reseed uses seed + g, and objective[g] gets its sum.
hipError_t launch_kmeans_update(const void *rows, int rowtype, int64_t N, int D, int64_t ld,
                                const float *cent_in, int64_t C, const int64_t *counts,
                                const int64_t *offsets, const uint32_t *perm, uint64_t seed,
                                int32_t iter, float *cent_out, double *jpart, double *objective,
                                hipStream_t s, int groups = 1, int64_t x_group = 0);

// ---- list-major layout and residuals (layout.hip) ----------------------------
hipError_t launch_list_major(const void *base, int rowtype, int64_t N, const float *cent, int64_t C,
                             int D, const int64_t *offsets, const uint32_t *perm, int64_t pos0,
                             int64_t n, void *out_rows, float *out_res, hipStream_t s);

// ---- product quantisation (pq.hip) ------------------------------------------
constexpr int kPqK = 256;         // codewords per subspace (8-bit codes)
constexpr int kPqMaxSubDims = 16; // dims per subspace
// Nearest codeword of every row in subspaces [m0, m1): codes [n, M] uint8
// and/or labels [m1 - m0][n] int32.
hipError_t launch_pq_assign(const float *X, int64_t n, int D, int dsub, int m0, int m1,
                            const float *codebooks, uint8_t *codes, int M, int32_t *labels,
                            hipStream_t s);

// ---- candidate-restricted assignment (assign_graph.hip) ---------------------
constexpr int kMaxGraphDegree = 64;
hipError_t launch_assign_graph(const void *rows, int rowtype, int64_t N, const float *cent, int64_t C,
                               int D, const int32_t *graph, int S, const int32_t *prev, const uint32_t *order,
                               int32_t *labels, float *dist, hipStream_t s);
// Cell-and-walk assignment (rows without a previous label): nearest member of
// the row's coarse cell, then up to `hops` greedy moves over graph [C, S]
// (graph may be null). D <= kCellsMaxDim.
constexpr int kCellsMaxDim = 256;
hipError_t launch_assign_cells(const void *rows, int rowtype, int64_t N, const float *cent, int64_t C, int D,
                               const int32_t *cell, int64_t G, const int64_t *offsets, const uint32_t *members,
                               int64_t M, const int32_t *graph, int S, int hops, const uint32_t *order,
                               int32_t *labels, float *dist, int num_cus, hipStream_t s);

// ---- residual-PQ ADC scan (adc.hip) -----------------------------------------
constexpr int kAdcMaxK = 1024;   // handoff per query (N_rerank)
constexpr int kAdcMaxM = 60;     // subspaces (LUT of M x 256 floats in LDS, < 64 KiB)
constexpr int kMaxAdcProbes = 4096;
// Workspace of the scan: at most 2P groups per query, each with a handoff of
// k keys and a descriptor (list id, code range), and each query's group count.
struct AdcScratch {
    uint64_t *handoff;  // [B * 2P * k]
    int32_t *hcnt;      // [B * 2P] keys the group handed over (<= k)
    int32_t *dl;        // [B * 2P] list of the group
    longlong2 *dpos;    // [B * 2P] first and end code position of the group
    int32_t *gcnt;      // [B] groups of the query
};
// ids/dist [B, k].
hipError_t launch_adc_scan(const float *Q, int64_t B, int D, const float *cent, int64_t C,
                           const int32_t *probes, int P, const int64_t *offsets, const uint32_t *perm,
                           int64_t N, const uint8_t *codes, int M, const float *codebooks, int k,
                           const AdcScratch &w, uint32_t *ids, float *dist, hipStream_t s);

// ---- fp32 MFMA throughput probe (probe.hip) ---------------------------------
// Enqueues the probe kernel for `iters` rounds; *flops = the work it does.
hipError_t launch_mfma_probe(int iters, int num_cus, hipStream_t s, double *flops);
// The same for the int8 MFMA pipe; *ops = the int8 operations it does.
hipError_t launch_mfma_probe_i8(int iters, int num_cus, hipStream_t s, double *ops);

}  // namespace ivf
