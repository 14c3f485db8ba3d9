// C ABI of the gfx950 IVF routing / construction library (declared in
// include/ivf.h). Validates arguments, sizes and carves the caller's
// workspace, and enqueues the kernels on the context's stream. No call
// synchronises with the host except ivf_sync and ivf_last_stats.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "ivf.h"
#include "ivf_internal.h"

using namespace ivf;

struct ivf_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    int num_cus = 1;
    void *ws = nullptr;
    size_t ws_bytes = 0;
    std::string err;
    int force_fallback = 0;
    int sample_rank = 0;
    int build_blocks = 0;
    int screen_waves = 8;
    int fp32_screen = 0;  // 1: uint8 rows also take the fp32 MFMA screen
    int two_plane_only = 0;  // 1: no single-plane int8 pre-screen
    int s1_id_order = 0;     // 1: the single plane visits centroids in id order
    int force_rescreen = 0;  // 1: the single-plane screen lists every row
    int64_t rescreen_cap = 0;  // > 0: smaller capacity of that list (tests)
    int64_t assign_slice = 0;  // > 0: shorter assignment slices (tests)
    unsigned long long *last_stats = nullptr;  // device, inside the workspace
    int64_t last_sample = 0;
    // kernel timing (IVF_OPT_PROFILE): an event pair per launch of the last call
    int profile = 0;
    std::vector<hipEvent_t> events;
    std::vector<std::string> knames;
    std::vector<std::string> retired;  // names handed out by the last read
    size_t kused = 0;
    const char *cur_call = "";
    ~ivf_ctx()
    {
        for (hipEvent_t e : events) (void)hipEventDestroy(e);
    }
};

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kRouteBatch = 16384;
constexpr int kMaxNprobe = 1024;
constexpr int kMaxD = 256;
constexpr int kMaxHops = 1024;  // greedy moves of ivf_assign_cells
// Rows per assignment slice (row ids inside a slice fit int32).
constexpr int64_t kAssignSlice = (int64_t)1 << 28;

// Scratch memory of ivf_route_noalloc, for callers that cannot allocate
// device memory: one copy per device, held while the library is loaded. In
// host code `scratch` names a host-side stand-in; kernels get the device
// address that hipGetSymbolAddress returns for each device.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Looks up (once per device, with that device current) the device address of
// `scratch`; nullptr on failure.
void *static_scratch(int device)
{
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        int prev = -1;
        if (hipGetDevice(&prev) != hipSuccess) return nullptr;
        if (prev != device && hipSetDevice(device) != hipSuccess) return nullptr;
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (prev != device) (void)hipSetDevice(prev);
        if (e != hipSuccess) return nullptr;
        g_scratch_ptr[device] = ptr;
    }
    return g_scratch_ptr[device];
}

ivf_status fail(ivf_ctx *ctx, ivf_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (ctx) ctx->err = buf;
    return st;
}

// Bump allocator over the workspace (base == nullptr: sizing only).
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base((char *)b) {}
    template <typename T> T *take(size_t count)
    {
        off = (off + kAlign - 1) / kAlign * kAlign;
        T *p = base ? (T *)(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

// Workspace of ivf_adc_scan for B queries, P probes, handoff k (layout only
// when base is null); returns the bytes used.
size_t layout_adc(void *base, int64_t B, int64_t P, int64_t k, AdcScratch *w)
{
    Carver c(base);
    AdcScratch s;
    s.handoff = c.take<uint64_t>((size_t)B * 2 * P * k);
    s.hcnt = c.take<int32_t>((size_t)B * 2 * P);
    s.dl = c.take<int32_t>((size_t)B * 2 * P);
    s.dpos = c.take<longlong2>((size_t)B * 2 * P);
    s.gcnt = c.take<int32_t>((size_t)B);
    if (w) *w = s;
    return c.off + kAlign;
}

// Scalar area at the start of every workspace: [0] max centroid norm bits,
// [1] worklist counter, [2] nonzero when some centroid does not quantise for
// the int8 screen, [3] the same for its single plane, [4] the single plane's
// largest coordinate residual (float bits), [5] counter of the rows the
// single plane leaves to the two planes, [6] the int8 routing gate, [7] the
// single plane's largest residual norm (float bits), then (from word 16)
// kNumStats uint64 counters.
struct Scalars {
    uint32_t *mc2_bits;
    uint32_t *wl_cnt;
    unsigned long long *stats;
};

Scalars take_scalars(Carver &c)
{
    uint32_t *p = c.take<uint32_t>(64);
    Scalars s;
    s.mc2_bits = p;
    s.wl_cnt = p ? p + 1 : nullptr;
    s.stats = p ? (unsigned long long *)(p + 16) : nullptr;
    return s;
}

int padded_dim(int D)
{
    static const int dps[] = {32, 64, 96, 128, 192, 256};
    for (int dp : dps)
        if (D <= dp) return dp;
    return 0;
}

// Padded dimension of the quantised centroids kept for the int8 screen (the
// largest when D is not a supported size: such calls fail validation anyway).
int quant_dim(int D)
{
    const int dp = padded_dim(D);
    return dp > 0 ? dp : 256;
}

double bound_coef(int DP)
{
    const double u = 0x1p-23;  // one fp32 ulp relative: covers any rounding mode
    const double n = DP + 2;
    return n * u / (1.0 - n * u);
}

int pow2_ceil(int64_t v)
{
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

struct RoutePlan {
    int64_t QB;   // queries per internal batch
    int64_t Cs;   // threshold sample size, 0 = none
    int64_t Ss;   // the sample: chunks j * Ss of kChunk centroids, j < Cs / kChunk
    int L;        // candidate capacity per query
    int rank_j;
    int qdp;      // padded dimension of the int8 route planes; 0 = fp32 kernels only
};

RoutePlan plan_route(int64_t Q, int64_t C, int k, int rank_override, int D)
{
    RoutePlan p;
    p.QB = std::max<int64_t>(1, std::min<int64_t>(Q, kRouteBatch));
    p.qdp = quant_dim(D);
    if (C <= 2048) {
        p.Cs = 0;
        p.Ss = 1;
        p.L = pow2_ceil(std::max<int64_t>(C, k));
        p.rank_j = 0;
        return p;
    }
    // sizes depend only on (Q, C, k); a rank override (a test knob) moves the
    // threshold but never the buffers, so ivf_workspace_bytes stays valid
    const int r = 32;
    const int64_t mu = std::max<int64_t>(4 * (int64_t)k, 256);
    int64_t f = mu / r;
    f = std::min<int64_t>(std::max<int64_t>(f, 4), 64);
    int64_t Cs = (C / f) / kChunk * kChunk;
    Cs = std::max<int64_t>(Cs, (int64_t)2 * r * 16);
    Cs = std::min<int64_t>(Cs, (C / 2) / kChunk * kChunk);
    Cs = std::min<int64_t>(Cs, 65536);
    Cs = std::max<int64_t>(Cs, kChunk);
    p.Cs = Cs;
    // spread over the table (a table sorted by position or by list would
    // bias a contiguous sample); Cs <= C / 2 gives a stride of at least 2
    p.Ss = (C / kChunk) / (Cs / kChunk);
    p.rank_j = (int)std::min<int64_t>(r, Cs / 16);
    const double expected = (double)p.rank_j * (double)C / (double)Cs;
    if (rank_override > 0) p.rank_j = (int)std::min<int64_t>(rank_override, Cs / 16);
    int L = pow2_ceil((int64_t)(2.5 * expected) + 1);
    L = std::max(L, std::max(512, pow2_ceil(k)));
    p.L = std::min(L, 4096);
    return p;
}

struct RouteLayout {
    Scalars sc;
    float *cnorm;
    double *qn2;
    float *tau;
    uint32_t *cand_cnt;
    uint2 *cand;
    float *keys;
    float *kmin;
    int32_t *wl;
    // int8 route planes (plan.qdp > 0): two planes [quantized_pad(C)][2 qdp],
    // biases, per-query bounds
    int8_t *qc;
    int32_t *negb;
    float *qbound;
    size_t bytes;
};

RouteLayout layout_route(void *base, const RoutePlan &p, int64_t C)
{
    Carver c(base);
    RouteLayout l;
    l.sc = take_scalars(c);
    l.cnorm = c.take<float>(C);
    l.qn2 = c.take<double>(p.QB);
    l.tau = c.take<float>(p.QB);
    l.cand_cnt = c.take<uint32_t>(p.QB);
    l.cand = c.take<uint2>((size_t)p.QB * p.L);
    l.keys = c.take<float>((size_t)p.QB * p.Cs);
    l.kmin = c.take<float>((size_t)p.QB * (p.Cs / 16));
    l.wl = c.take<int32_t>(p.QB);
    l.qc = nullptr;
    l.negb = nullptr;
    l.qbound = nullptr;
    if (p.qdp > 0) {
        l.qc = c.take<int8_t>((size_t)quantized_pad(C) * 2 * p.qdp);
        l.negb = c.take<int32_t>(quantized_pad(C));
        l.qbound = c.take<float>(p.QB);
    }
    l.bytes = c.off + kAlign;
    return l;
}

int64_t worklist_cap(int64_t N) { return std::min<int64_t>(N, 4096 + N / 64); }
// rows the single-plane int8 screen may list for the two-plane screen
// before that screen takes every row
int64_t rescreen_cap(int64_t N) { return std::min<int64_t>(N, 4096 + N / 16); }

struct AssignLayout {
    Scalars sc;
    float *cnorm;
    // quantised centroids of the int8 screen (uint8 rows)
    int8_t *qc;
    int32_t *negb;
    // single plane (padded dimension <= 128) and the rows it leaves
    int8_t *qc1;
    int32_t *negb1;
    // its visiting order: keys, column sums and mean, counting-sort scratch,
    // bucket counts and offsets, order (plane row -> id) and positions
    int32_t *okeys;
    double *opart;
    float *omean;
    void *oradix;
    int64_t *ocounts;
    int64_t *ooffsets;
    uint32_t *ord1;
    int32_t *pos1;
    int32_t *list;
    int64_t list_cap;
    int32_t *wl;
    int64_t wl_cap;
    double *fb_d;   // split fallback partial results
    int32_t *fb_i;
    // build
    uint32_t *cntmat;
    int64_t *counts;
    int64_t *offsets;
    uint32_t *perm;
    double *jpart;
    size_t bytes;
};

// Product-quantisation training step over M subspaces: labels [M][n], the
// list build of each subspace's labels (256 lists; one radix scratch reused),
// counts [M][256], offsets [M][257], permutations [M][n] and the update's
// objective parts [M][256].
struct PqLayout {
    int32_t *labels;
    void *radix;
    int64_t *counts;
    int64_t *offsets;
    uint32_t *perm;
    double *jpart;
    size_t bytes;
};

PqLayout layout_pq(void *base, int64_t n, int M, int num_cus)
{
    Carver c(base);
    PqLayout l{};
    l.labels = c.take<int32_t>((size_t)n * M);
    l.radix = c.take<unsigned char>(radix_scratch_bytes(plan_radix(n, kPqK, num_cus)));
    l.counts = c.take<int64_t>((size_t)kPqK * M);
    l.offsets = c.take<int64_t>((size_t)(kPqK + 1) * M);
    l.perm = c.take<uint32_t>((size_t)n * M);
    l.jpart = c.take<double>((size_t)kPqK * M);
    l.bytes = c.off;
    return l;
}

// need_lists: counts/offsets/perm live in the workspace (k-means step);
// need_build: count matrix for the list build; qdp > 0: quantised centroids
// of padded dimension qdp for the int8 screen.
AssignLayout layout_assign(void *base, int64_t N, int64_t C, int qdp, bool need_build, bool need_lists,
                           int num_cus)
{
    Carver c(base);
    AssignLayout l{};
    l.sc = take_scalars(c);
    l.cnorm = c.take<float>(C);
    if (qdp > 0) {
        l.qc = c.take<int8_t>((size_t)quantized_pad(C) * 2 * qdp);
        l.negb = c.take<int32_t>(quantized_pad(C));
        if (qdp <= 128) {
            l.qc1 = c.take<int8_t>((size_t)quantized_pad1(C) * qdp);
            l.negb1 = c.take<int32_t>(quantized_pad1(C));
            l.okeys = c.take<int32_t>(C);
            l.opart = c.take<double>((size_t)order1_parts(C) * qdp);
            l.omean = c.take<float>(qdp);
            l.oradix = c.take<unsigned char>(radix_scratch_bytes(plan_radix(C, kOrder1Keys, num_cus)));
            l.ocounts = c.take<int64_t>(kOrder1Keys);
            l.ooffsets = c.take<int64_t>(kOrder1Keys + 1);
            l.ord1 = c.take<uint32_t>(C);
            l.pos1 = c.take<int32_t>(C);
            l.list_cap = rescreen_cap(std::min(N, kAssignSlice));
            l.list = c.take<int32_t>(l.list_cap);
        }
    }
    l.wl_cap = worklist_cap(std::min(N, kAssignSlice));
    l.wl = c.take<int32_t>(l.wl_cap);
    l.fb_d = c.take<double>(kFbSplitEntries);
    l.fb_i = c.take<int32_t>(kFbSplitEntries);
    if (need_build) {
        if (C <= kRadixMaxLists)
            l.cntmat = (uint32_t *)c.take<unsigned char>(radix_scratch_bytes(plan_radix(N, C, num_cus)));
        else
            l.cntmat = c.take<uint32_t>(build_scratch_bytes(plan_build(N, C, num_cus)) / 4);
    }
    if (need_lists) {
        l.counts = c.take<int64_t>(C);
        l.offsets = c.take<int64_t>(C + 1);
        l.perm = c.take<uint32_t>(N);
        l.jpart = c.take<double>(C);
    }
    l.bytes = c.off + kAlign;
    return l;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void *a, size_t na, const void *b, size_t nb)
{
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev)
    {
        if (dev < 0) {  // validation-only context
            ok = false;
            return;
        }
        if (hipGetDevice(&prev) != hipSuccess) {
            ok = false;
            return;
        }
        if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
    }
    ~DeviceGuard()
    {
        int cur;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

ivf_status check_ws(ivf_ctx *ctx, size_t need)
{
    if (!ctx->ws || ctx->ws_bytes < need)
        return fail(ctx, IVF_ENOMEM, "workspace too small: %zu bytes required, %zu provided", need,
                    ctx->ws ? ctx->ws_bytes : (size_t)0);
    return IVF_OK;
}

#define HIP_TRY(expr)                                                                      \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(ctx, IVF_EDEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));  \
    } while (0)

// Drops the recorded kernel timeline.
void prof_reset(ivf_ctx *ctx) { ctx->kused = 0; ctx->knames.clear(); }

// Records the start event of a kernel launch; returns its slot or -1.
int prof_start(ivf_ctx *ctx, const char *name)
{
    if (!ctx->profile) return -1;
    const size_t i = ctx->kused++;
    while (ctx->events.size() < 2 * ctx->kused) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) {
            --ctx->kused;
            return -1;
        }
        ctx->events.push_back(e);
    }
    ctx->knames.push_back(std::string(ctx->cur_call) + "/" + name);
    (void)hipEventRecord(ctx->events[2 * i], ctx->stream);
    return (int)i;
}

void prof_stop(ivf_ctx *ctx, int slot)
{
    if (slot >= 0) (void)hipEventRecord(ctx->events[2 * slot + 1], ctx->stream);
}

// Launch with optional event timing around it.
#define TIMED(name, expr)                        \
    do {                                         \
        const int slot_ = prof_start(ctx, name); \
        HIP_TRY(expr);                           \
        prof_stop(ctx, slot_);                   \
    } while (0)

ivf_status check_common(ivf_ctx *ctx, int64_t C, int32_t D)
{
    if (C < 1) return fail(ctx, IVF_EINVAL, "C must be >= 1 (got %lld)", (long long)C);
    if (C > INT32_MAX) return fail(ctx, IVF_EUNSUPPORTED, "C must fit int32 ids");
    if (D < 4 || D > kMaxD || D % 4 != 0)
        return fail(ctx, IVF_EUNSUPPORTED, "D must be a multiple of 4 in [4, %d] (got %d)", kMaxD, D);
    return IVF_OK;
}

// Assignment of N rows (top-1 with certification and fallback) into labels.
// The centroid preparation (norms, quantised planes) runs once; the rows are
// then screened in slices of at most `slice` rows, each with its own
// worklists, so that the row ids the screens and the fallback pass around
// (int32, relative to the slice) stay below 2^31 for any N <= 2^32 - 1.
ivf_status enqueue_assign(ivf_ctx *ctx, const void *rows, int rowtype, int64_t N,
                          const float *cent, int64_t C, int D, int32_t *labels,
                          const AssignLayout &l, const int32_t *hint = nullptr)
{
    hipStream_t s = ctx->stream;
    const int DP = padded_dim(D);
    const size_t rb = (size_t)D * (rowtype == kRowU8 ? 1 : 4);
    const int64_t slice = ctx->assign_slice > 0 ? std::min<int64_t>(ctx->assign_slice, kAssignSlice) : kAssignSlice;
    TIMED("fill", launch_fill_u32(l.sc.mc2_bits, 64, 0u, s));
    TIMED("centroid_norms", launch_centroid_norms(cent, C, D, l.cnorm, l.sc.mc2_bits, s));
    const bool int8 = rowtype == kRowU8 && !ctx->fp32_screen;
    const bool single = int8 && l.qc1 && !ctx->two_plane_only;
    uint32_t *q_bad = l.sc.mc2_bits + 2;
    uint32_t *q_bad1 = l.sc.mc2_bits + 3;
    uint32_t *e_bits = l.sc.mc2_bits + 4;
    uint32_t *list_cnt = l.sc.mc2_bits + 5;
    uint32_t *r2_bits = l.sc.mc2_bits + 7;
    const uint32_t *ord1 = nullptr;
    const int32_t *pos1 = nullptr;
    if (int8) {
        // int8 MFMA screens; the fp32 kernel runs only if some centroid does not quantise
        TIMED("quantize", launch_quantize_centroids(cent, C, D, DP, l.qc, l.negb, q_bad, s));
        if (single) {
            const bool ordered = !ctx->s1_id_order;
            if (ordered) {
                // the plane's visiting order: a stable counting sort of the
                // centroids by their distance bucket
                TIMED("order1_keys", launch_order1_keys(cent, C, D, l.opart, l.omean, l.okeys, s));
                const RadixPlan rp = plan_radix(C, kOrder1Keys, ctx->num_cus);
                const RadixScratch rs = carve_radix(rp, l.oradix);
                TIMED("order1_level0", launch_radix_level0(rp, l.okeys, rs, s));
                TIMED("order1_counts", launch_radix_level1_counts(rp, rs, l.ocounts, s));
                TIMED("order1_offsets", launch_offsets(l.ocounts, kOrder1Keys, l.ooffsets, s));
                TIMED("order1_scatter", launch_radix_level1_scatter(rp, rs, l.ooffsets, l.ord1, s));
            }
            TIMED("quantize1", launch_quantize_centroids1(cent, C, D, DP, l.qc1, l.negb1, q_bad1, e_bits, r2_bits,
                                                          s, ordered ? l.ord1 : nullptr, ordered ? l.pos1 : nullptr));
            ord1 = ordered ? l.ord1 : nullptr;
            pos1 = ordered ? l.pos1 : nullptr;
        }
    }
    for (int64_t r0 = 0; r0 < N; r0 += slice) {
        const int64_t n = std::min(slice, N - r0);
        const void *xr = (const char *)rows + (size_t)r0 * rb;
        int32_t *lab = labels + r0;
        if (r0 > 0) {
            // the worklist and the single plane's list start empty for every slice
            TIMED("fill", launch_fill_u32(l.sc.wl_cnt, 1, 0u, s));
            if (single) TIMED("fill", launch_fill_u32(list_cnt, 1, 0u, s));
        }
        ScreenArgs a{};
        a.rows = xr;
        a.nrows = n;
        a.D = D;
        a.cent = cent;
        a.cnorm = l.cnorm;
        a.c_begin = 0;
        a.c_end = C;
        a.nchunks = (C + kChunk - 1) / kChunk;
        a.mc2_bits = l.sc.mc2_bits;
        a.bound_coef = bound_coef(DP);
        a.labels = lab;
        a.wl = l.wl;
        a.wl_cnt = l.sc.wl_cnt;
        a.wl_cap = l.wl_cap;
        a.stats = l.sc.stats;
        a.force_fallback = ctx->force_fallback;
        if (int8) {
            ScreenI8Args q{};
            q.rows = (const uint8_t *)xr;
            q.nrows = n;
            q.D = D;
            q.cent = cent;
            q.qc = l.qc;
            q.negb = l.negb;
            q.cpad = quantized_pad(C);
            q.nchunks = q.cpad / 64;
            q.q_bad = q_bad;
            q.labels = lab;
            q.wl = l.wl;
            q.wl_cnt = l.sc.wl_cnt;
            q.wl_cap = l.wl_cap;
            q.stats = l.sc.stats;
            q.force_fallback = ctx->force_fallback;
            q.ncent = C;
            if (single) {
                // single plane first; the two planes then screen the rows it leaves
                q.qc1 = l.qc1;
                q.negb1 = l.negb1;
                q.e_bits = e_bits;
                q.r2_bits = r2_bits;
                q.q_bad1 = q_bad1;
                q.list = l.list;
                q.list_cnt = list_cnt;
                q.list_cap = ctx->rescreen_cap > 0 ? std::min<int64_t>(ctx->rescreen_cap, l.list_cap) : l.list_cap;
                // a forced fallback passes every row on to the two planes, which send it on
                q.force_rescreen = ctx->force_rescreen || ctx->force_fallback;
                q.hint = hint ? hint + r0 : nullptr;
                q.ord1 = ord1;
                q.pos1 = pos1;
                TIMED("screen_top1_i8s", launch_screen_i8_single(DP, q, ctx->num_cus, s));
            }
            TIMED("screen_top1_i8", launch_screen_i8(DP, q, ctx->num_cus, s));
            a.gate = q_bad;
        }
        TIMED("screen_top1", launch_screen(kModeTop1, rowtype, DP, a, ctx->screen_waves, ctx->num_cus, s));
        TIMED("assign_fallback", launch_assign_fallback(xr, rowtype, n, D, cent, C, lab, l.wl, l.sc.wl_cnt,
                                                        l.wl_cap, l.fb_d, l.fb_i, 2 * ctx->num_cus, s));
    }
    ctx->last_stats = l.sc.stats;
    ctx->last_sample = 0;
    return IVF_OK;
}

// List build: the two-level radix partition for C <= 65,536 lists, the
// single-pass per-block build otherwise. `scratch` is the build area of the
// workspace.
ivf_status enqueue_build(ivf_ctx *ctx, int64_t N, int64_t C, const int32_t *labels, void *scratch,
                         int64_t *counts, int64_t *offsets, uint32_t *perm)
{
    if (C <= kRadixMaxLists) {
        const RadixPlan rp = plan_radix(N, C, ctx->num_cus);
        const RadixScratch rs = carve_radix(rp, scratch);
        if (N == 0) {
            TIMED("fill", launch_fill_u32((uint32_t *)counts, 2 * C, 0u, ctx->stream));
            TIMED("build_offsets", launch_offsets(counts, C, offsets, ctx->stream));
            return IVF_OK;
        }
        TIMED("build_level0", launch_radix_level0(rp, labels, rs, ctx->stream));
        TIMED("build_level1_counts", launch_radix_level1_counts(rp, rs, counts, ctx->stream));
        TIMED("build_offsets", launch_offsets(counts, C, offsets, ctx->stream));
        TIMED("build_level1_scatter", launch_radix_level1_scatter(rp, rs, offsets, perm, ctx->stream));
        return IVF_OK;
    }
    const BuildPlan bp = plan_build(N, C, ctx->num_cus, ctx->build_blocks);
    uint32_t *cntmat = (uint32_t *)scratch;
    TIMED("build_hist", launch_build_hist(bp, labels, cntmat, ctx->stream));
    TIMED("build_scan", launch_build_scan(bp, cntmat, counts, offsets, ctx->stream));
    TIMED("build_scatter", launch_build_scatter(bp, labels, cntmat, offsets, perm, ctx->stream));
    return IVF_OK;
}

}  // namespace

extern "C" {

ivf_status ivf_create(int device, void *hip_stream, ivf_ctx **out)
{
    if (!out) return IVF_EINVAL;
    *out = nullptr;
    if (device == -1) {  // validation-only context: checks arguments, enqueues nothing
        ivf_ctx *c = new ivf_ctx();
        c->device = -1;
        c->num_cus = 256;
        *out = c;
        return IVF_OK;
    }
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess) return IVF_EDEVICE;
    if (device < 0 || device >= n) return IVF_EINVAL;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) return IVF_EDEVICE;
    // the static scratch of ivf_route_noalloc: its address on this device
    if (!static_scratch(device)) return IVF_EDEVICE;
    ivf_ctx *c = new ivf_ctx();
    c->device = device;
    c->stream = (hipStream_t)hip_stream;
    c->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 1;
    *out = c;
    return IVF_OK;
}

void ivf_destroy(ivf_ctx *ctx) { delete ctx; }

const char *ivf_last_error(const ivf_ctx *ctx) { return ctx ? ctx->err.c_str() : "null context"; }

ivf_status ivf_set_stream(ivf_ctx *ctx, void *hip_stream)
{
    if (!ctx) return IVF_EINVAL;
    ctx->stream = (hipStream_t)hip_stream;
    return IVF_OK;
}

size_t ivf_workspace_bytes(int op, int64_t rows, int64_t C, int32_t D, int32_t k)
{
    if (C < 1 || rows < 0) return 0;
    int num_cus = 256;
    int dev;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess &&
        prop.multiProcessorCount > 0)
        num_cus = prop.multiProcessorCount;
    switch (op) {
    case IVF_OP_ROUTE:
        if (k < 1) return 0;
        return layout_route(nullptr, plan_route(rows, C, k, 0, D), C).bytes;
    case IVF_OP_KMEANS_STEP:
        return layout_assign(nullptr, std::max<int64_t>(rows, 1), C, quant_dim(D), true, true, num_cus).bytes;
    case IVF_OP_ASSIGN_BUILD:
        return layout_assign(nullptr, std::max<int64_t>(rows, 1), C, quant_dim(D), true, false, num_cus).bytes;
    case IVF_OP_BUILD_LISTS:
        return layout_assign(nullptr, std::max<int64_t>(rows, 1), C, 0, true, false, num_cus).bytes;
    case IVF_OP_ADC_SCAN:  // rows = B, C = P (probes per query), k = handoff
        if (k < 1 || k > kAdcMaxK || C < 1 || C > kMaxAdcProbes) return 0;
        return layout_adc(nullptr, rows, C, k, nullptr);
    case IVF_OP_PQ_TRAIN_STEP:  // C = M
        if (C > kMaxD) return 0;
        return layout_pq(nullptr, std::max<int64_t>(rows, 1), (int)C, num_cus).bytes;
    default:
        return 0;
    }
}

ivf_status ivf_set_workspace(ivf_ctx *ctx, void *dev_ptr, size_t bytes)
{
    if (!ctx) return IVF_EINVAL;
    if (dev_ptr && ((uintptr_t)dev_ptr % kAlign) != 0)
        return fail(ctx, IVF_EINVAL, "workspace must be %zu-byte aligned", kAlign);
    ctx->ws = dev_ptr;
    ctx->ws_bytes = dev_ptr ? bytes : 0;
    return IVF_OK;
}

ivf_status ivf_sync(ivf_ctx *ctx)
{
    if (!ctx) return IVF_EINVAL;
    if (ctx->device < 0) return IVF_OK;
    DeviceGuard g(ctx->device);
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return fail(ctx, IVF_EDEVICE, "device error: %s", hipGetErrorString(e));
    return IVF_OK;
}

ivf_status ivf_set_option(ivf_ctx *ctx, int option, int64_t value)
{
    if (!ctx) return IVF_EINVAL;
    switch (option) {
    case IVF_OPT_FORCE_FALLBACK: ctx->force_fallback = value ? 1 : 0; return IVF_OK;
    case IVF_OPT_SAMPLE_RANK:
        if (value < 0 || value > 4096) return fail(ctx, IVF_EINVAL, "sample rank out of range");
        ctx->sample_rank = (int)value;
        return IVF_OK;
    case IVF_OPT_PROFILE: ctx->profile = value ? 1 : 0; return IVF_OK;
    case IVF_OPT_SCREEN_WAVES:
        if (value != 4 && value != 8) return fail(ctx, IVF_EINVAL, "screen waves must be 4 or 8");
        ctx->screen_waves = (int)value;
        return IVF_OK;
    case IVF_OPT_FP32_SCREEN: ctx->fp32_screen = value ? 1 : 0; return IVF_OK;
    case IVF_OPT_I8_TWO_PLANE_ONLY: ctx->two_plane_only = value ? 1 : 0; return IVF_OK;
    case IVF_OPT_FORCE_RESCREEN: ctx->force_rescreen = value ? 1 : 0; return IVF_OK;
    case IVF_OPT_RESCREEN_CAP:
        if (value < 0) return fail(ctx, IVF_EINVAL, "rescreen capacity must be >= 0");
        ctx->rescreen_cap = value;
        return IVF_OK;
    case IVF_OPT_S1_ID_ORDER: ctx->s1_id_order = value ? 1 : 0; return IVF_OK;
    case IVF_OPT_ASSIGN_SLICE:
        if (value < 0) return fail(ctx, IVF_EINVAL, "assignment slice must be >= 0");
        ctx->assign_slice = value;
        return IVF_OK;
    case IVF_OPT_BUILD_BLOCKS:
        if (value < 0 || value > 65536) return fail(ctx, IVF_EINVAL, "build blocks out of range");
        ctx->build_blocks = (int)value;
        return IVF_OK;
    default: return fail(ctx, IVF_EINVAL, "unknown option %d", option);
    }
}

ivf_status ivf_last_stats(ivf_ctx *ctx, int64_t out[8])
{
    if (!ctx || !out) return IVF_EINVAL;
    for (int i = 0; i < 8; ++i) out[i] = 0;
    if (!ctx->last_stats) return IVF_OK;
    DeviceGuard g(ctx->device);
    unsigned long long h[kNumStats];
    HIP_TRY(hipMemcpyAsync(h, ctx->last_stats, sizeof h, hipMemcpyDeviceToHost, ctx->stream));
    HIP_TRY(hipStreamSynchronize(ctx->stream));
    for (int i = 0; i < 8; ++i) out[i] = (int64_t)h[i];
    out[kStatSample] = ctx->last_sample;
    return IVF_OK;
}

int ivf_kernel_times(ivf_ctx *ctx, int max, const char **names, float *ms)
{
    if (!ctx || max < 0) return -1;
    if (ctx->device < 0) return 0;
    DeviceGuard g(ctx->device);
    if (hipStreamSynchronize(ctx->stream) != hipSuccess) return -1;
    const int n = (int)ctx->kused;
    for (int i = 0; i < n && i < max; ++i) {
        if (names) names[i] = ctx->knames[i].c_str();
        if (ms) {
            float t = 0.f;
            if (hipEventElapsedTime(&t, ctx->events[2 * i], ctx->events[2 * i + 1]) != hipSuccess) t = -1.f;
            ms[i] = t;
        }
    }
    if (max > 0 && max >= n) {
        // every entry delivered: start a new timeline (names stay valid until
        // the next recorded launch)
        ctx->kused = 0;
        ctx->retired.swap(ctx->knames);
        ctx->knames.clear();
    }
    return n;
}

}  // extern "C"

namespace {

// Times one probe launch (after an untimed one that loads the kernel) and
// reports its duration and rate in units of 1e12 operations per second.
ivf_status run_probe(ivf_ctx *ctx, int32_t iters, hipError_t (*launch)(int, int, hipStream_t, double *),
                     const char *what, float *out_ms, double *out_rate)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    if (iters < 1 || iters > (1 << 20)) return fail(ctx, IVF_EINVAL, "iters must be in [1, 2^20]");
    if (!out_ms && !out_rate) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (ctx->device < 0) return fail(ctx, IVF_EUNSUPPORTED, "validation-only context");
    DeviceGuard g(ctx->device);
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
        if (e0) (void)hipEventDestroy(e0);
        return fail(ctx, IVF_EDEVICE, "hipEventCreate failed");
    }
    double ops = 0.0;
    float ms = 0.f;
    hipError_t e = launch(1, ctx->num_cus, ctx->stream, &ops);
    if (e == hipSuccess) e = hipEventRecord(e0, ctx->stream);
    if (e == hipSuccess) e = launch(iters, ctx->num_cus, ctx->stream, &ops);
    if (e == hipSuccess) e = hipEventRecord(e1, ctx->stream);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (e != hipSuccess) return fail(ctx, IVF_EDEVICE, "%s: %s", what, hipGetErrorString(e));
    if (out_ms) *out_ms = ms;
    if (out_rate) *out_rate = ms > 0.f ? ops / (ms * 1e-3) / 1e12 : 0.0;
    return IVF_OK;
}

}  // namespace

extern "C" {

ivf_status ivf_mfma_probe(ivf_ctx *ctx, int32_t iters, float *out_ms, double *out_tflops)
{
    return run_probe(ctx, iters, launch_mfma_probe, "fp32 MFMA probe", out_ms, out_tflops);
}

ivf_status ivf_mfma_probe_i8(ivf_ctx *ctx, int32_t iters, float *out_ms, double *out_tops)
{
    return run_probe(ctx, iters, launch_mfma_probe_i8, "int8 MFMA probe", out_ms, out_tops);
}

}  // extern "C"

namespace {

// Argument checks shared by ivf_route and ivf_route_noalloc (nothing is
// enqueued). *done is set when Q == 0 (a no-op).
ivf_status check_route(ivf_ctx *ctx, const float *queries, int64_t Q, const float *centroids, int64_t C,
                       int32_t D, int32_t nprobe, int32_t *out_ids, float *out_dist, bool *done)
{
    *done = false;
    if (Q < 0) return fail(ctx, IVF_EINVAL, "Q must be >= 0");
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    if (nprobe < 1 || nprobe > C)
        return fail(ctx, IVF_EINVAL, "nprobe must be in [1, C] (got %d, C = %lld)", nprobe, (long long)C);
    if (nprobe > kMaxNprobe) return fail(ctx, IVF_EUNSUPPORTED, "nprobe > %d", kMaxNprobe);
    if (Q == 0) {
        *done = true;
        return IVF_OK;
    }
    if (!queries || !centroids || !out_ids) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(queries) || !aligned16(centroids) || !aligned16(out_ids) ||
        (out_dist && !aligned16(out_dist)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const size_t qb = (size_t)Q * D * 4, cb = (size_t)C * D * 4, ob = (size_t)Q * nprobe * 4;
    if (overlap(out_ids, ob, queries, qb) || overlap(out_ids, ob, centroids, cb) ||
        overlap(out_dist, ob, queries, qb) || overlap(out_dist, ob, centroids, cb) ||
        overlap(out_ids, ob, out_dist, ob))
        return fail(ctx, IVF_EINVAL, "outputs overlap inputs or each other");
    return IVF_OK;
}

// Enqueues the routing kernels, queries in batches of p.QB, with the scratch
// memory laid out by layout_route at `ws`.
ivf_status enqueue_route(ivf_ctx *ctx, const float *queries, int64_t Q, const float *centroids, int64_t C,
                         int32_t D, int32_t nprobe, int32_t *out_ids, float *out_dist, const RoutePlan &p,
                         void *ws)
{
    const RouteLayout l = layout_route(ws, p, C);
    hipStream_t s = ctx->stream;
    const int DP = padded_dim(D);
    TIMED("fill", launch_fill_u32(l.sc.mc2_bits, 64, 0u, s));
    TIMED("centroid_norms", launch_centroid_norms(centroids, C, D, l.cnorm, l.sc.mc2_bits, s));
    // uint8-valued queries are routed on the two int8 planes; the fp32
    // kernels run instead (device flag, no host synchronisation) when a query
    // or a centroid does not fit them. Tables small enough to be candidates
    // whole (no threshold sample) stay on the fp32 kernels: there the screen
    // only copies every centroid into the candidate list.
    const bool i8 = p.qdp > 0 && p.Cs > 0 && !ctx->fp32_screen;
    uint32_t *q_bad = l.sc.mc2_bits + 2;
    uint32_t *i8_off = l.sc.mc2_bits + 6;
    if (i8) {
        TIMED("route_i8_check", launch_route_i8_check(queries, Q, D, i8_off, s));
        TIMED("quantize", launch_quantize_centroids(centroids, C, D, p.qdp, l.qc, l.negb, q_bad, s, i8_off));
    }
    for (int64_t q0 = 0; q0 < Q; q0 += p.QB) {
        const int64_t nb = std::min(p.QB, Q - q0);
        const float *qrows = queries + q0 * D;
        TIMED("fill", launch_fill_u32(l.sc.wl_cnt, 1, 0u, s));
        TIMED("row_norms", launch_row_norms(qrows, nb, D, l.qn2, s));
        ScreenArgs a{};
        a.rows = qrows;
        a.nrows = nb;
        a.D = D;
        a.cent = centroids;
        a.cnorm = l.cnorm;
        a.gate = i8 ? i8_off : nullptr;
        RouteI8Args ra{};
        ra.queries = qrows;
        ra.nq = nb;
        ra.D = D;
        ra.qc = l.qc;
        ra.negb = l.negb;
        ra.cpad = quantized_pad(C);
        ra.off = i8_off;
        ra.stats = l.sc.stats;
        if (i8) TIMED("route_i8_bound", launch_route_i8_bound(qrows, nb, D, q_bad, i8_off, l.qbound, s));
        if (p.Cs > 0) {
            a.c_begin = 0;
            a.c_end = C;
            a.nchunks = p.Cs / kChunk;
            a.cstride = p.Ss;
            a.keys = l.keys;
            a.kmin = l.kmin;
            if (i8) {
                ra.c_begin = 0;
                ra.c_end = p.Cs;
                ra.nchunks = p.Cs / kQuantChunk;
                ra.cstride = p.Ss;
                ra.keys = l.keys;
                TIMED("route_i8_keys", launch_route_i8(kRouteKeys, p.qdp, ra, ctx->num_cus, s));
            }
            TIMED("screen_keys", launch_screen(kModeKeys, kRowF32, DP, a, ctx->screen_waves, ctx->num_cus, s));
        }
        RouteArgs r{};
        r.queries = qrows;
        r.nq = nb;
        r.cent = centroids;
        r.C = C;
        r.D = D;
        r.k = nprobe;
        r.L = p.L;
        r.Cs = p.Cs;
        r.sstride = p.Ss;
        r.rank_j = p.rank_j;
        r.keys = l.keys;
        r.kmin = l.kmin;
        r.tau = l.tau;
        r.cand_cnt = l.cand_cnt;
        r.cand = l.cand;
        r.qn2 = l.qn2;
        r.mc2_bits = l.sc.mc2_bits;
        r.bound_coef = bound_coef(DP);
        r.force_fallback = ctx->force_fallback;
        r.out_ids = out_ids + q0 * nprobe;
        r.out_dist = out_dist ? out_dist + q0 * nprobe : nullptr;
        r.wl = l.wl;
        r.wl_cnt = l.sc.wl_cnt;
        r.stats = l.sc.stats;
        r.i8_off = i8 ? i8_off : nullptr;
        r.qbound = l.qbound;
        TIMED("route_threshold", launch_route_threshold(r, s));
        if (p.Cs < C) {
            // every chunk the sample left
            a.c_begin = 0;
            a.c_end = C;
            a.nchunks = (C + kChunk - 1) / kChunk - p.Cs / kChunk;
            a.cstride = 1;
            a.skip_n = p.Cs / kChunk;
            a.skip_s = p.Ss;
            a.keys = nullptr;
            a.tau = l.tau;
            a.cand_cnt = l.cand_cnt;
            a.cand = l.cand;
            a.L = p.L;
            if (i8) {
                // the int8 threshold emits no sample candidates: the filter covers every centroid
                ra.c_begin = 0;
                ra.c_end = C;
                ra.nchunks = (C + kQuantChunk - 1) / kQuantChunk;
                ra.cstride = 1;
                ra.keys = nullptr;
                ra.tau = l.tau;
                ra.cand_cnt = l.cand_cnt;
                ra.cand = l.cand;
                ra.L = p.L;
                TIMED("route_i8_filter", launch_route_i8(kRouteFilter, p.qdp, ra, ctx->num_cus, s));
            }
            TIMED("screen_filter", launch_screen(kModeFilter, kRowF32, DP, a, ctx->screen_waves, ctx->num_cus, s));
        }
        TIMED("route_select", launch_route_select(r, s));
        TIMED("route_fallback", launch_route_fallback(r, 2 * ctx->num_cus, s));
    }
    ctx->last_stats = l.sc.stats;
    ctx->last_sample = p.Cs;
    return IVF_OK;
}

}  // namespace

extern "C" {

ivf_status ivf_route(ivf_ctx *ctx, const float *queries, int64_t Q, const float *centroids,
                     int64_t C, int32_t D, int32_t nprobe, int32_t *out_ids, float *out_dist)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "route";
    bool done = false;
    ivf_status st = check_route(ctx, queries, Q, centroids, C, D, nprobe, out_ids, out_dist, &done);
    if (st != IVF_OK || done) return st;
    const RoutePlan p = plan_route(Q, C, nprobe, ctx->sample_rank, D);
    const size_t need = layout_route(nullptr, p, C).bytes;
    if ((st = check_ws(ctx, need)) != IVF_OK) return st;
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    return enqueue_route(ctx, queries, Q, centroids, C, D, nprobe, out_ids, out_dist, p, ctx->ws);
}

ivf_status ivf_route_noalloc(ivf_ctx *ctx, const float *queries, int64_t Q, const float *centroids,
                             int64_t C, int32_t D, int32_t nprobe, int32_t *out_ids, float *out_dist)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "route_noalloc";
    bool done = false;
    ivf_status st = check_route(ctx, queries, Q, centroids, C, D, nprobe, out_ids, out_dist, &done);
    if (st != IVF_OK || done) return st;
    // the batch of queries shrinks until the layout fits the static scratch;
    // sizes that do not fit with a single query are refused
    RoutePlan p = plan_route(Q, C, nprobe, ctx->sample_rank, D);
    auto one_query = [&] {
        RoutePlan q1 = p;
        q1.QB = 1;
        return layout_route(nullptr, q1, C).bytes;
    };
    // the int8 route planes are left out (fp32 kernels only) when they do not
    // fit beside one query
    if (one_query() > kStaticScratchBytes) p.qdp = 0;
    const size_t one = one_query();
    if (one > kStaticScratchBytes)
        return fail(ctx, IVF_EUNSUPPORTED,
                    "route_noalloc: C = %lld, nprobe = %d need %zu bytes of scratch for one query; the static "
                    "scratch holds %zu", (long long)C, nprobe, one, kStaticScratchBytes);
    const size_t per_query = layout_route(nullptr, RoutePlan{2, p.Cs, p.L, p.rank_j, p.qdp}, C).bytes - one;
    const int64_t fit = 1 + (int64_t)((kStaticScratchBytes - one) / std::max<size_t>(per_query, 1));
    if (p.QB > fit) p.QB = fit >= 64 ? fit / 32 * 32 : fit;
    while (p.QB > 1 && layout_route(nullptr, p, C).bytes > kStaticScratchBytes) --p.QB;
    if (ctx->device < 0) return fail(ctx, IVF_EDEVICE, "no usable device (validation-only context)");
    void *scratch_ptr = static_scratch(ctx->device);
    if (!scratch_ptr) return fail(ctx, IVF_EDEVICE, "static scratch of device %d is not available", ctx->device);
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    // no event objects are created for this call, even when profiling is on
    const int prof = ctx->profile;
    ctx->profile = 0;
    st = enqueue_route(ctx, queries, Q, centroids, C, D, nprobe, out_ids, out_dist, p, scratch_ptr);
    ctx->profile = prof;
    return st;
}

static ivf_status check_rows(ivf_ctx *ctx, const void *rows, int dt, int64_t N, int32_t D,
                             size_t *row_bytes)
{
    if (dt != IVF_F32 && dt != IVF_U8) return fail(ctx, IVF_EINVAL, "dtype must be IVF_F32 or IVF_U8");
    if (N < 0) return fail(ctx, IVF_EINVAL, "N must be >= 0");
    if (N > (int64_t)UINT32_MAX) return fail(ctx, IVF_EUNSUPPORTED, "N must be < 2^32");
    if (N > 0 && !rows) return fail(ctx, IVF_EINVAL, "null data pointer");
    if (rows && !aligned16(rows)) return fail(ctx, IVF_EINVAL, "data must be 16-byte aligned");
    *row_bytes = (size_t)D * (dt == IVF_U8 ? 1 : 4);
    return IVF_OK;
}

ivf_status ivf_kmeans_step(ivf_ctx *ctx, const void *train, int dt, int64_t N,
                           const float *centroids, int64_t C, int32_t D, uint64_t seed,
                           int32_t iter, int32_t *out_labels, float *out_centroids,
                           int64_t *out_counts, double *out_objective, const int32_t *hint_labels)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "kmeans_step";
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    size_t rb;
    if ((st = check_rows(ctx, train, dt, N, D, &rb)) != IVF_OK) return st;
    if (N == 0) return IVF_OK;
    if (!centroids || !out_labels || !out_centroids) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(centroids) || !aligned16(out_labels) || !aligned16(out_centroids) ||
        (out_counts && !aligned16(out_counts)) || (out_objective && !aligned16(out_objective)) ||
        (hint_labels && !aligned16(hint_labels)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const size_t xb = (size_t)N * rb, cb = (size_t)C * D * 4, lb = (size_t)N * 4, nb = (size_t)C * 8;
    const void *outs[4] = {out_labels, out_centroids, out_counts, out_objective};
    const size_t osz[4] = {lb, cb, nb, 8};
    for (int i = 0; i < 4; ++i) {
        if (overlap(outs[i], osz[i], train, xb) || overlap(outs[i], osz[i], centroids, cb) ||
            overlap(outs[i], osz[i], hint_labels, hint_labels ? lb : 0))
            return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
        for (int j = i + 1; j < 4; ++j)
            if (overlap(outs[i], osz[i], outs[j], osz[j])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    }
    const size_t need = layout_assign(nullptr, N, C, quant_dim(D), true, true, ctx->num_cus).bytes;
    if ((st = check_ws(ctx, need)) != IVF_OK) return st;
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);

    const AssignLayout l = layout_assign(ctx->ws, N, C, quant_dim(D), true, true, ctx->num_cus);
    const int rowtype = dt == IVF_U8 ? kRowU8 : kRowF32;
    if ((st = enqueue_assign(ctx, train, rowtype, N, centroids, C, D, out_labels, l, hint_labels)) != IVF_OK)
        return st;
    int64_t *counts = out_counts ? out_counts : l.counts;
    if ((st = enqueue_build(ctx, N, C, out_labels, l.cntmat, counts, l.offsets, l.perm)) != IVF_OK) return st;
    TIMED("kmeans_update", launch_kmeans_update(train, rowtype, N, D, D, centroids, C, counts, l.offsets, l.perm, seed,
                                 iter, out_centroids, l.jpart, out_objective, ctx->stream));
    return IVF_OK;
}

ivf_status ivf_assign_build(ivf_ctx *ctx, const void *base, int dt, int64_t N,
                            const float *centroids, int64_t C, int32_t D, int32_t *out_labels,
                            int64_t *out_counts, int64_t *out_offsets, uint32_t *out_perm)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "assign_build";
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    size_t rb;
    if ((st = check_rows(ctx, base, dt, N, D, &rb)) != IVF_OK) return st;
    if (!centroids || !out_counts || !out_offsets || (N > 0 && (!out_labels || !out_perm)))
        return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(centroids) || !aligned16(out_counts) || !aligned16(out_offsets) ||
        (out_labels && !aligned16(out_labels)) || (out_perm && !aligned16(out_perm)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const size_t xb = (size_t)N * rb, cb = (size_t)C * D * 4;
    const void *outs[4] = {out_labels, out_counts, out_offsets, out_perm};
    const size_t osz[4] = {(size_t)N * 4, (size_t)C * 8, (size_t)(C + 1) * 8, (size_t)N * 4};
    for (int i = 0; i < 4; ++i) {
        if (overlap(outs[i], osz[i], base, xb) || overlap(outs[i], osz[i], centroids, cb))
            return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
        for (int j = i + 1; j < 4; ++j)
            if (overlap(outs[i], osz[i], outs[j], osz[j])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    }
    const size_t need = layout_assign(nullptr, std::max<int64_t>(N, 1), C, quant_dim(D), true, false, ctx->num_cus).bytes;
    if ((st = check_ws(ctx, need)) != IVF_OK) return st;
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);

    const AssignLayout l = layout_assign(ctx->ws, std::max<int64_t>(N, 1), C, quant_dim(D), true, false, ctx->num_cus);
    const int rowtype = dt == IVF_U8 ? kRowU8 : kRowF32;
    if (N > 0 && (st = enqueue_assign(ctx, base, rowtype, N, centroids, C, D, out_labels, l)) != IVF_OK)
        return st;
    if ((st = enqueue_build(ctx, N, C, out_labels, l.cntmat, out_counts, out_offsets, out_perm)) != IVF_OK)
        return st;
    return IVF_OK;
}

ivf_status ivf_build_lists(ivf_ctx *ctx, const int32_t *labels, int64_t N, int64_t C,
                           int64_t *out_counts, int64_t *out_offsets, uint32_t *out_perm)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "build_lists";
    if (C < 1) return fail(ctx, IVF_EINVAL, "C must be >= 1");
    if (C > INT32_MAX) return fail(ctx, IVF_EUNSUPPORTED, "C must fit int32 ids");
    if (N < 0) return fail(ctx, IVF_EINVAL, "N must be >= 0");
    if (N > (int64_t)UINT32_MAX) return fail(ctx, IVF_EUNSUPPORTED, "N must be < 2^32");
    if (!out_counts || !out_offsets || (N > 0 && (!labels || !out_perm)))
        return fail(ctx, IVF_EINVAL, "null pointer argument");
    if ((labels && !aligned16(labels)) || !aligned16(out_counts) || !aligned16(out_offsets) ||
        (out_perm && !aligned16(out_perm)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const void *outs[3] = {out_counts, out_offsets, out_perm};
    const size_t osz[3] = {(size_t)C * 8, (size_t)(C + 1) * 8, (size_t)N * 4};
    for (int i = 0; i < 3; ++i) {
        if (overlap(outs[i], osz[i], labels, (size_t)N * 4)) return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
        for (int j = i + 1; j < 3; ++j)
            if (overlap(outs[i], osz[i], outs[j], osz[j])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    }
    const size_t need = layout_assign(nullptr, std::max<int64_t>(N, 1), C, 0, true, false, ctx->num_cus).bytes;
    ivf_status st;
    if ((st = check_ws(ctx, need)) != IVF_OK) return st;
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    const AssignLayout l = layout_assign(ctx->ws, std::max<int64_t>(N, 1), C, 0, true, false, ctx->num_cus);
    if ((st = enqueue_build(ctx, N, C, labels, l.cntmat, out_counts, out_offsets, out_perm)) != IVF_OK) return st;
    ctx->last_stats = nullptr;
    return IVF_OK;
}

ivf_status ivf_list_major(ivf_ctx *ctx, const void *base, int dt, int64_t N, const float *centroids,
                          int64_t C, int32_t D, const int64_t *offsets, const uint32_t *perm,
                          int64_t pos0, int64_t n, void *out_rows, float *out_residuals)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "list_major";
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    size_t rb;
    if ((st = check_rows(ctx, base, dt, N, D, &rb)) != IVF_OK) return st;
    if (pos0 < 0 || n < 0 || pos0 > N || n > N - pos0)
        return fail(ctx, IVF_EINVAL, "positions [pos0, pos0 + n) must lie in [0, N)");
    if (n == 0) return IVF_OK;
    if (!out_rows && !out_residuals) return fail(ctx, IVF_EINVAL, "no output requested");
    if (!centroids || !offsets || (N > 0 && !perm)) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(centroids) || !aligned16(offsets) || (perm && !aligned16(perm)) ||
        (out_rows && !aligned16(out_rows)) || (out_residuals && !aligned16(out_residuals)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const size_t ob[2] = {(size_t)n * rb, (size_t)n * D * 4};
    const void *outs[2] = {out_rows, out_residuals};
    const void *ins[4] = {base, centroids, offsets, perm};
    const size_t ib[4] = {(size_t)N * rb, (size_t)C * D * 4, (size_t)(C + 1) * 8, (size_t)N * 4};
    for (int i = 0; i < 2; ++i)
        for (int k = 0; k < 4; ++k)
            if (overlap(outs[i], ob[i], ins[k], ib[k])) return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
    if (overlap(out_rows, ob[0], out_residuals, ob[1])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    const int rowtype = dt == IVF_U8 ? kRowU8 : kRowF32;
    TIMED("list_major", launch_list_major(base, rowtype, N, centroids, C, D, offsets, perm, pos0, n,
                                          out_rows, out_residuals, ctx->stream));
    ctx->last_stats = nullptr;
    return IVF_OK;
}

ivf_status ivf_assign_graph(ivf_ctx *ctx, const void *rows, int dt, int64_t N, const float *centroids,
                            int64_t C, int32_t D, const int32_t *graph, int32_t S, const int32_t *prev,
                            const uint32_t *order, int32_t *out_labels, float *out_dist)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "assign_graph";
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    size_t rb;
    if ((st = check_rows(ctx, rows, dt, N, D, &rb)) != IVF_OK) return st;
    if (S < 1 || S > kMaxGraphDegree)
        return fail(ctx, IVF_EINVAL, "S must be in [1, %d] (got %d)", kMaxGraphDegree, S);
    if (N == 0) return IVF_OK;
    if (!centroids || !graph || !prev || !out_labels) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(centroids) || !aligned16(graph) || !aligned16(prev) || (order && !aligned16(order)) ||
        !aligned16(out_labels) || (out_dist && !aligned16(out_dist)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const void *ins[5] = {rows, centroids, graph, prev, order};
    const size_t ib[5] = {(size_t)N * rb, (size_t)C * D * 4, (size_t)C * S * 4, (size_t)N * 4,
                          order ? (size_t)N * 4 : 0};
    const void *outs[2] = {out_labels, out_dist};
    const size_t ob[2] = {(size_t)N * 4, (size_t)N * 4};
    for (int i = 0; i < 2; ++i)
        for (int k = 0; k < 5; ++k)
            if (overlap(outs[i], ob[i], ins[k], ib[k])) return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
    if (overlap(out_labels, ob[0], out_dist, ob[1])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    const int rowtype = dt == IVF_U8 ? kRowU8 : kRowF32;
    TIMED("assign_graph", launch_assign_graph(rows, rowtype, N, centroids, C, D, graph, S, prev, order,
                                              out_labels, out_dist, ctx->stream));
    ctx->last_stats = nullptr;
    return IVF_OK;
}

ivf_status ivf_assign_cells(ivf_ctx *ctx, const void *rows, int dt, int64_t N, const float *centroids,
                            int64_t C, int32_t D, const int32_t *cell, int64_t G, const int64_t *cell_offsets,
                            const uint32_t *cell_members, int64_t M, const int32_t *graph, int32_t S,
                            int32_t hops, const uint32_t *order, int32_t *out_labels, float *out_dist)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "assign_cells";
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    size_t rb;
    if ((st = check_rows(ctx, rows, dt, N, D, &rb)) != IVF_OK) return st;
    if (G < 1 || G > INT32_MAX) return fail(ctx, IVF_EINVAL, "G must be in [1, 2^31 - 1] (got %lld)", (long long)G);
    if (M < 0) return fail(ctx, IVF_EINVAL, "M must be >= 0");
    if (hops < 0 || hops > kMaxHops) return fail(ctx, IVF_EINVAL, "hops must be in [0, %d] (got %d)", kMaxHops, hops);
    if (graph && (S < 1 || S > kMaxGraphDegree))
        return fail(ctx, IVF_EINVAL, "S must be in [1, %d] (got %d)", kMaxGraphDegree, S);
    if (N == 0) return IVF_OK;
    if (!centroids || !cell || !cell_offsets || (M > 0 && !cell_members) || !out_labels)
        return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(centroids) || !aligned16(cell) || !aligned16(cell_offsets) ||
        (cell_members && !aligned16(cell_members)) || (graph && !aligned16(graph)) || (order && !aligned16(order)) ||
        !aligned16(out_labels) || (out_dist && !aligned16(out_dist)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const void *ins[7] = {rows, centroids, cell, cell_offsets, cell_members, graph, order};
    const size_t ib[7] = {(size_t)N * rb, (size_t)C * D * 4, (size_t)N * 4, (size_t)(G + 1) * 8, (size_t)M * 4,
                          graph ? (size_t)C * S * 4 : 0, order ? (size_t)N * 4 : 0};
    const void *outs[2] = {out_labels, out_dist};
    const size_t ob[2] = {(size_t)N * 4, (size_t)N * 4};
    for (int i = 0; i < 2; ++i)
        for (int k = 0; k < 7; ++k)
            if (overlap(outs[i], ob[i], ins[k], ib[k])) return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
    if (overlap(out_labels, ob[0], out_dist, ob[1])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    const int rowtype = dt == IVF_U8 ? kRowU8 : kRowF32;
    TIMED("assign_cells", launch_assign_cells(rows, rowtype, N, centroids, C, D, cell, G, cell_offsets, cell_members,
                                              M, graph, graph ? S : 0, hops, order, out_labels, out_dist,
                                              ctx->num_cus, ctx->stream));
    ctx->last_stats = nullptr;
    return IVF_OK;
}

ivf_status ivf_adc_scan(ivf_ctx *ctx, const float *queries, int64_t B, int32_t D, const float *centroids,
                        int64_t C, const int32_t *probes, int32_t P, const int64_t *offsets,
                        const uint32_t *perm, int64_t N, const uint8_t *codes, int32_t M,
                        const float *codebooks, int32_t k, uint32_t *out_ids, float *out_dist)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "adc_scan";
    ivf_status st = check_common(ctx, C, D);
    if (st != IVF_OK) return st;
    if (B < 0 || N < 0) return fail(ctx, IVF_EINVAL, "B and N must be >= 0");
    if (N > (int64_t)UINT32_MAX) return fail(ctx, IVF_EUNSUPPORTED, "N must be < 2^32");
    if (M < 1 || D % M != 0) return fail(ctx, IVF_EINVAL, "M must divide D (D = %d, M = %d)", D, M);
    if (M > kAdcMaxM) return fail(ctx, IVF_EUNSUPPORTED, "at most %d subspaces", kAdcMaxM);
    if (P < 1 || P > kMaxAdcProbes) return fail(ctx, IVF_EINVAL, "P must be in [1, %d]", kMaxAdcProbes);
    if (k < 1 || k > kAdcMaxK) return fail(ctx, IVF_EINVAL, "k must be in [1, %d]", kAdcMaxK);
    if (B == 0) return IVF_OK;
    if (!queries || !centroids || !probes || !offsets || !codebooks || !out_ids || !out_dist ||
        (N > 0 && (!perm || !codes)))
        return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(queries) || !aligned16(centroids) || !aligned16(probes) || !aligned16(offsets) ||
        (perm && !aligned16(perm)) || (codes && !aligned16(codes)) || !aligned16(codebooks) ||
        !aligned16(out_ids) || !aligned16(out_dist))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const void *ins[7] = {queries, centroids, probes, offsets, perm, codes, codebooks};
    const size_t ib[7] = {(size_t)B * D * 4, (size_t)C * D * 4, (size_t)B * P * 4, (size_t)(C + 1) * 8,
                          (size_t)N * 4, (size_t)N * M, (size_t)kPqK * D * 4};
    const void *outs[2] = {out_ids, out_dist};
    const size_t ob = (size_t)B * k * 4;
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 7; ++j)
            if (overlap(outs[i], ob, ins[j], ib[j])) return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
    if (overlap(out_ids, ob, out_dist, ob)) return fail(ctx, IVF_EINVAL, "outputs overlap");
    const size_t need = layout_adc(nullptr, B, P, k, nullptr);
    if ((st = check_ws(ctx, need)) != IVF_OK) return st;
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    AdcScratch w;
    layout_adc(ctx->ws, B, P, k, &w);
    TIMED("adc_scan", launch_adc_scan(queries, B, D, centroids, C, probes, P, offsets, perm, N, codes, M,
                                      codebooks, k, w, out_ids, out_dist, ctx->stream));
    ctx->last_stats = nullptr;
    return IVF_OK;
}

static ivf_status check_pq(ivf_ctx *ctx, int32_t D, int32_t M, int *dsub)
{
    ivf_status st = check_common(ctx, kPqK, D);
    if (st != IVF_OK) return st;
    if (M < 1 || D % M != 0) return fail(ctx, IVF_EINVAL, "M must divide D (D = %d, M = %d)", D, M);
    *dsub = D / M;
    if (*dsub > kPqMaxSubDims)
        return fail(ctx, IVF_EUNSUPPORTED, "at most %d dims per subspace (D / M = %d)", kPqMaxSubDims, *dsub);
    return IVF_OK;
}

ivf_status ivf_pq_encode(ivf_ctx *ctx, const float *x, int64_t n, int32_t D, int32_t M,
                         const float *codebooks, uint8_t *out_codes)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "pq_encode";
    int dsub = 0;
    ivf_status st = check_pq(ctx, D, M, &dsub);
    if (st != IVF_OK) return st;
    if (n < 0) return fail(ctx, IVF_EINVAL, "n must be >= 0");
    if (n == 0) return IVF_OK;
    if (!x || !codebooks || !out_codes) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(x) || !aligned16(codebooks) || !aligned16(out_codes))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const size_t ob = (size_t)n * M;
    if (overlap(out_codes, ob, x, (size_t)n * D * 4) || overlap(out_codes, ob, codebooks, (size_t)kPqK * D * 4))
        return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    TIMED("pq_assign", launch_pq_assign(x, n, D, dsub, 0, M, codebooks, out_codes, M, nullptr, ctx->stream));
    ctx->last_stats = nullptr;
    return IVF_OK;
}

ivf_status ivf_pq_train_step(ivf_ctx *ctx, const float *x, int64_t n, int32_t D, int32_t M,
                             const float *codebooks, uint64_t seed, int32_t iter, float *out_codebooks,
                             int64_t *out_counts, double *out_objective)
{
    if (!ctx) return IVF_EINVAL;
    ctx->err.clear();
    ctx->cur_call = "pq_train_step";
    int dsub = 0;
    ivf_status st = check_pq(ctx, D, M, &dsub);
    if (st != IVF_OK) return st;
    if (n < 1) return fail(ctx, IVF_EINVAL, "n must be >= 1");
    if (n > (int64_t)UINT32_MAX) return fail(ctx, IVF_EUNSUPPORTED, "n must be < 2^32");
    if (!x || !codebooks || !out_codebooks) return fail(ctx, IVF_EINVAL, "null pointer argument");
    if (!aligned16(x) || !aligned16(codebooks) || !aligned16(out_codebooks) ||
        (out_counts && !aligned16(out_counts)) || (out_objective && !aligned16(out_objective)))
        return fail(ctx, IVF_EINVAL, "arrays must be 16-byte aligned");
    const size_t xb = (size_t)n * D * 4, cb = (size_t)kPqK * D * 4;
    const void *outs[3] = {out_codebooks, out_counts, out_objective};
    const size_t osz[3] = {cb, (size_t)M * kPqK * 8, (size_t)M * 8};
    for (int i = 0; i < 3; ++i) {
        if (overlap(outs[i], osz[i], x, xb) || overlap(outs[i], osz[i], codebooks, cb))
            return fail(ctx, IVF_EINVAL, "outputs overlap inputs");
        for (int j = i + 1; j < 3; ++j)
            if (overlap(outs[i], osz[i], outs[j], osz[j])) return fail(ctx, IVF_EINVAL, "outputs overlap");
    }
    const size_t need = layout_pq(nullptr, n, M, ctx->num_cus).bytes;
    if ((st = check_ws(ctx, need)) != IVF_OK) return st;
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, IVF_EDEVICE, "no usable device (context device %d)", ctx->device);
    const PqLayout l = layout_pq(ctx->ws, n, M, ctx->num_cus);
    int64_t *counts = out_counts ? out_counts : l.counts;
    // every subspace's labels, then each subspace's lists, then one update
    // launch over all M x 256 codewords (group m = subspace m, seed + m)
    TIMED("pq_assign", launch_pq_assign(x, n, D, dsub, 0, M, codebooks, nullptr, M, l.labels, ctx->stream));
    for (int m = 0; m < M; ++m)
        if ((st = enqueue_build(ctx, n, kPqK, l.labels + (int64_t)m * n, l.radix, counts + (int64_t)m * kPqK,
                                l.offsets + (int64_t)m * (kPqK + 1), l.perm + (int64_t)m * n)) != IVF_OK)
            return st;
    TIMED("pq_update", launch_kmeans_update(x, kRowF32, n, dsub, D, codebooks, kPqK, counts, l.offsets, l.perm,
                                            seed, iter, out_codebooks, l.jpart, out_objective, ctx->stream, M,
                                            dsub));
    ctx->last_stats = nullptr;
    return IVF_OK;
}

}  // extern "C"
