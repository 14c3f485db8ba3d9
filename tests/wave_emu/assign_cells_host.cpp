// Runs the cell-and-walk assignment kernel of assign_graph.hip on the host
// emulation (or, with a graph-only header, the candidate-restricted kernel),
// with every array in an allocation of its own, and writes the labels and
// distances for the test to check against the oracle.
//   usage: assign_cells_host in.bin out.bin num_cus
//   in:  int64 N, C, D, G, M, S, hops, rowtype (0 uint8, 1 fp32), has_graph,
//        has_order; rows [N][D] (uint8 or fp32); float centroids [C][D];
//        int32 cell [N]; int64 offsets [G + 1]; uint32 members [M];
//        int32 graph [C][S] if has_graph; uint32 order [N] if has_order.
//        G = 0 selects ivf_assign_graph's kernels instead: the cell array
//        holds the previous labels (offsets then holds one unused entry,
//        members none)
//   out: int32 labels [N]; float dist [N] (entries no processing position
//        names keep the fill 0x7F7F7F7F)
#include "hip/hip_runtime.h"

#include <initializer_list>
namespace emu {
thread_local dim3 tid, bid;
dim3 bdim, gdim;
Block *blk;
unsigned char *dyn_lds;
}  // namespace emu
#include "assign_graph_host_src.hip"
using namespace ivf;

template <typename T>
static T *alloc(size_t n, int fill)
{
    const size_t b = std::max<size_t>(n, 1) * sizeof(T);
    T *p = (T *)malloc(b);
    memset(p, fill, b);
    return p;
}

template <typename T>
static bool get(FILE *f, T *p, size_t n)
{
    return fread(p, sizeof(T), n, f) == n;
}

int main(int argc, char **argv)
{
    if (argc < 4) return 2;
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int64_t h[10];
    if (!get(f, h, 10)) return 2;
    const int64_t N = h[0], C = h[1], G = h[3], M = h[4];
    const int D = (int)h[2], S = (int)h[5], hops = (int)h[6], rowtype = (int)h[7];
    const bool has_graph = h[8] != 0, has_order = h[9] != 0;
    const size_t rb = rowtype == 0 ? 1 : 4;
    unsigned char *x = alloc<unsigned char>(N * D * rb, 0);
    float *cent = alloc<float>(C * D, 0);
    int32_t *cell = alloc<int32_t>(N, 0);
    int64_t *offsets = alloc<int64_t>(G + 1, 0);
    uint32_t *members = alloc<uint32_t>(M, 0);
    int32_t *graph = has_graph ? alloc<int32_t>(C * S, 0) : nullptr;
    uint32_t *order = has_order ? alloc<uint32_t>(N, 0) : nullptr;
    if (!get(f, x, N * D * rb) || !get(f, cent, C * D) || !get(f, cell, N) || !get(f, offsets, G + 1) ||
        !get(f, members, M) || (graph && !get(f, graph, C * S)) || (order && !get(f, order, N)))
        return 2;
    fclose(f);
    int32_t *labels = alloc<int32_t>(N, 0x7f);
    float *dist = alloc<float>(N, 0x7f);
    if (G == 0) {
        if (!graph || launch_assign_graph(x, rowtype == 0 ? kRowU8 : kRowF32, N, cent, C, D, graph, S, cell, order,
                                          labels, dist, nullptr) != hipSuccess)
            return 3;
    } else if (launch_assign_cells(x, rowtype == 0 ? kRowU8 : kRowF32, N, cent, C, D, cell, G, offsets, members, M, graph,
                            graph ? S : 0, hops, order, labels, dist, atoi(argv[3]), nullptr) != hipSuccess)
        return 3;
    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    fwrite(labels, 4, N, o);
    fwrite(dist, 4, N, o);
    fclose(o);
    for (void *p : {(void *)x, (void *)cent, (void *)cell, (void *)offsets, (void *)members, (void *)graph,
                    (void *)order, (void *)labels, (void *)dist})
        free(p);
    return 0;
}
