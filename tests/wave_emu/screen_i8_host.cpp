// Runs the int8 screening kernels of screen_i8.hip on the host emulation, in
// the order the library enqueues them for uint8 rows (quantisation, the
// single-plane screen when the padded dimension is at most 128 and mode is 1,
// then the two-plane screen over the rows it leaves), on one case file, with
// every array in an allocation of its own; optionally followed by the exact
// fallback scan of fallback.hip (built as its own translation unit), which
// settles the rows the screens hand on. Writes the labels, the worklist and
// the statistics for the test to check against the oracle.
//   usage: screen_i8_host in.bin out.bin num_cus force_fallback
//                         [mode force_rescreen rescreen_cap run_fallback wl_cap hints.bin order]
//   hints.bin (optional, "-" for none): int32 hint labels [N] for the single plane
//   order (optional): the single plane's visiting order, either a file of
//        uint32 [C] (plane row -> centroid id) or "auto": the library's keys
//        kernel, then a stable sort by key on the host (the counting sort
//        the library runs with the list build's kernels)
//   in:  int64 N, C, D; uint8 rows [N][D]; float centroids [C][D]
//   out: int32 labels [N]; uint32 worklist count; int32 worklist [count];
//        uint64 stats [8]; uint32 quantisation flag; uint32 single-plane
//        quantisation flag; uint32 rescreen list count
#include "hip/hip_runtime.h"
#include <vector>
namespace emu {
thread_local dim3 tid, bid;
dim3 bdim, gdim;
Block *blk;
unsigned char *dyn_lds;
}  // namespace emu
#include "screen_i8_host_src.hip"
using namespace ivf;

template <typename T>
static T *alloc(size_t n, int fill)
{
    const size_t b = std::max<size_t>(n, 1) * sizeof(T);
    T *p = (T *)malloc(b);
    memset(p, fill, b);
    return p;
}

int main(int argc, char **argv)
{
    if (argc < 5) return 2;
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int64_t hdr[3];
    if (fread(hdr, 8, 3, f) != 3) return 2;
    const int64_t N = hdr[0], C = hdr[1];
    const int D = (int)hdr[2];
    uint8_t *x = alloc<uint8_t>(N * D, 0);
    float *cent = alloc<float>(C * D, 0);
    if (fread(x, 1, N * D, f) != (size_t)(N * D) || fread(cent, 4, C * D, f) != (size_t)(C * D)) return 2;
    fclose(f);
    const int num_cus = atoi(argv[3]);
    int DP = 0;
    for (int dp : {32, 64, 96, 128, 192, 256})
        if (!DP && D <= dp) DP = dp;
    if (!DP || D % 4) return 2;
    const int64_t cpad = quantized_pad(C);
    const int64_t wl_cap_arg = argc > 9 ? atoll(argv[9]) : 0;
    const int64_t wl_cap = wl_cap_arg > 0 ? std::min<int64_t>(wl_cap_arg, N) : std::min<int64_t>(N, 4096 + N / 64);
    int8_t *qc = alloc<int8_t>(cpad * 2 * DP, 0);
    int32_t *negb = alloc<int32_t>(cpad, 0);
    uint32_t *q_bad = alloc<uint32_t>(1, 0);
    uint32_t *wl_cnt = alloc<uint32_t>(1, 0);
    int32_t *wl = alloc<int32_t>(wl_cap, 0);
    int32_t *labels = alloc<int32_t>(N, 0x7f);  // 0x7f7f7f7f marks a label never written
    unsigned long long *stats = alloc<unsigned long long>(8, 0);
    const int mode = argc > 5 ? atoi(argv[5]) : 0;
    const bool single = mode == 1 && DP <= 128;
    const int64_t list_cap = std::min<int64_t>(N, 4096 + N / 16);
    const int64_t cpad1 = quantized_pad1(C);
    int8_t *qc1 = single ? alloc<int8_t>(cpad1 * DP, 0) : nullptr;
    int32_t *negb1 = single ? alloc<int32_t>(cpad1, 0) : nullptr;
    int32_t *list = single ? alloc<int32_t>(list_cap, 0) : nullptr;
    uint32_t *q_bad1 = alloc<uint32_t>(1, 0);
    uint32_t *e_bits = alloc<uint32_t>(1, 0);
    uint32_t *r2_bits = alloc<uint32_t>(1, 0);
    uint32_t *list_cnt = alloc<uint32_t>(1, 0);

    launch_quantize_centroids(cent, C, D, DP, qc, negb, q_bad, nullptr);
    ScreenI8Args a{};
    a.rows = x;
    a.nrows = N;
    a.D = D;
    a.cent = cent;
    a.qc = qc;
    a.negb = negb;
    a.cpad = cpad;
    a.nchunks = cpad / 64;
    a.q_bad = q_bad;
    a.labels = labels;
    a.wl = wl;
    a.wl_cnt = wl_cnt;
    a.wl_cap = wl_cap;
    a.stats = stats;
    a.force_fallback = atoi(argv[4]);
    a.ncent = C;
    if (single) {
        uint32_t *ord = nullptr;
        int32_t *pos = nullptr;
        if (argc > 11) {
            ord = alloc<uint32_t>(C, 0);
            pos = alloc<int32_t>(C, 0xff);
            if (strcmp(argv[11], "auto") == 0) {
                int32_t *keys = alloc<int32_t>(C, 0xff);
                double *part = alloc<double>(order1_parts(C) * D, 0);
                float *mean = alloc<float>(D, 0);
                if (launch_order1_keys(cent, C, D, part, mean, keys, nullptr) != hipSuccess) return 3;
                std::vector<uint32_t> o(C);
                for (int64_t c = 0; c < C; ++c) {
                    if (keys[c] < 0 || keys[c] >= kOrder1Keys) return 4;
                    o[c] = (uint32_t)c;
                }
                std::stable_sort(o.begin(), o.end(), [&](uint32_t u, uint32_t v) { return keys[u] < keys[v]; });
                memcpy(ord, o.data(), 4 * C);
                free(keys);
                free(part);
                free(mean);
            } else {
                FILE *of = fopen(argv[11], "rb");
                if (!of || fread(ord, 4, C, of) != (size_t)C) return 2;
                fclose(of);
            }
        }
        launch_quantize_centroids1(cent, C, D, DP, qc1, negb1, q_bad1, e_bits, r2_bits, nullptr, ord, pos);
        a.ord1 = ord;
        a.pos1 = pos;
        a.qc1 = qc1;
        a.negb1 = negb1;
        a.e_bits = e_bits;
        a.r2_bits = r2_bits;
        a.q_bad1 = q_bad1;
        a.list = list;
        a.list_cnt = list_cnt;
        const int64_t cap = argc > 7 ? atoll(argv[7]) : 0;
        a.list_cap = cap > 0 ? std::min<int64_t>(cap, list_cap) : list_cap;
        // as the library: a forced fallback passes every row on to the two planes
        a.force_rescreen = (argc > 6 ? atoi(argv[6]) : 0) || a.force_fallback;
        int32_t *hint = nullptr;
        if (argc > 10 && strcmp(argv[10], "-") != 0) {
            hint = alloc<int32_t>(N, 0);
            FILE *hf = fopen(argv[10], "rb");
            if (!hf || fread(hint, 4, N, hf) != (size_t)N) return 2;
            fclose(hf);
        }
        a.hint = hint;
        launch_screen_i8_single(DP, a, num_cus, nullptr);
    }
    launch_screen_i8(DP, a, num_cus, nullptr);
    if (argc > 8 && atoi(argv[8])) {
        double *split_d = alloc<double>(kFbSplitEntries, 0);
        int32_t *split_i = alloc<int32_t>(kFbSplitEntries, 0);
        launch_assign_fallback(x, kRowU8, N, D, cent, C, labels, wl, wl_cnt, wl_cap, split_d, split_i,
                               2 * num_cus, nullptr);
        free(split_d);
        free(split_i);
    }

    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    const uint32_t n = std::min<uint32_t>(*wl_cnt, (uint32_t)wl_cap);
    fwrite(labels, 4, N, o);
    fwrite(&n, 4, 1, o);
    fwrite(wl, 4, n, o);
    fwrite(stats, 8, 8, o);
    fwrite(q_bad, 4, 1, o);
    fwrite(q_bad1, 4, 1, o);
    fwrite(list_cnt, 4, 1, o);
    fclose(o);
    return 0;
}
