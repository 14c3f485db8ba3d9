// Runs the int8 routing kernels of screen_i8.hip on the host emulation, in
// the order the library enqueues them (two-plane quantisation, the query
// check, the per-query bounds, the keys of the threshold sample as group
// minima, the candidate filter against given thresholds), with every array in
// an allocation of its own, and writes what they produced for the test to
// check against exact integer arithmetic.
//   usage: route_i8_host in.bin out.bin num_cus [stride]
//   stride (optional, default 1): the sample is the 64-centroid chunks
//        j * stride, j < Cs / 64 (the library spreads it over the table)
//   in:  int64 Q, C, D, Cs, L; float queries [Q][D]; float centroids [C][D];
//        float tau [Q]
//   out: uint32 off flag; uint32 quantisation flag; float qbound [Q];
//        float keys [Q][Cs / 16]; uint32 cand_cnt [Q]; uint2 cand [Q][L]
#include "hip/hip_runtime.h"
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
    if (argc < 4) return 2;
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int64_t hdr[5];
    if (fread(hdr, 8, 5, f) != 5) return 2;
    const int64_t Q = hdr[0], C = hdr[1], Cs = hdr[3];
    const int D = (int)hdr[2], L = (int)hdr[4];
    float *q = alloc<float>(Q * D, 0);
    float *cent = alloc<float>(C * D, 0);
    float *tau = alloc<float>(Q, 0);
    if (fread(q, 4, Q * D, f) != (size_t)(Q * D) || fread(cent, 4, C * D, f) != (size_t)(C * D) ||
        fread(tau, 4, Q, f) != (size_t)Q)
        return 2;
    fclose(f);
    const int num_cus = atoi(argv[3]);
    int DP = 0;
    for (int dp : {32, 64, 96, 128, 192, 256})
        if (!DP && D <= dp) DP = dp;
    if (!DP || D % 4 || Cs % 64 || Cs > C) return 2;
    const int64_t cpad = quantized_pad(C);
    int8_t *qc = alloc<int8_t>(cpad * 2 * DP, 0);
    int32_t *negb = alloc<int32_t>(cpad, 0);
    uint32_t *q_bad = alloc<uint32_t>(1, 0);
    uint32_t *off = alloc<uint32_t>(1, 0);
    float *qbound = alloc<float>(Q, 0x7f);
    const int64_t G = Cs / 16;
    float *keys = alloc<float>(Q * G, 0x7f);
    uint32_t *cand_cnt = alloc<uint32_t>(Q, 0);
    uint2 *cand = alloc<uint2>(Q * (int64_t)L, 0x7f);
    unsigned long long *stats = alloc<unsigned long long>(8, 0);

    launch_route_i8_check(q, Q, D, off, nullptr);
    launch_quantize_centroids(cent, C, D, DP, qc, negb, q_bad, nullptr, off);
    launch_route_i8_bound(q, Q, D, q_bad, off, qbound, nullptr);
    RouteI8Args a{};
    a.queries = q;
    a.nq = Q;
    a.D = D;
    a.qc = qc;
    a.negb = negb;
    a.cpad = cpad;
    a.off = off;
    a.stats = stats;
    if (Cs > 0) {
        a.c_begin = 0;
        a.c_end = Cs;
        a.nchunks = Cs / kQuantChunk;
        a.cstride = argc > 4 ? atoll(argv[4]) : 1;
        a.keys = keys;
        launch_route_i8(kRouteKeys, DP, a, num_cus, nullptr);
        a.cstride = 1;
    }
    a.c_begin = 0;
    a.c_end = C;
    a.nchunks = (C + kQuantChunk - 1) / kQuantChunk;
    a.keys = nullptr;
    a.tau = tau;
    a.cand_cnt = cand_cnt;
    a.cand = cand;
    a.L = L;
    launch_route_i8(kRouteFilter, DP, a, num_cus, nullptr);

    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    fwrite(off, 4, 1, o);
    fwrite(q_bad, 4, 1, o);
    fwrite(qbound, 4, Q, o);
    fwrite(keys, 4, Q * G, o);
    fwrite(cand_cnt, 4, Q, o);
    fwrite(cand, 8, Q * (int64_t)L, o);
    fclose(o);
    return 0;
}
