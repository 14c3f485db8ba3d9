"""ctypes binding of libivf.so (include/ivf.h): argument marshalling only.

Every step of the computation runs in the HIP kernels behind the C ABI; this
module only passes torch device pointers, sizes and the current HIP stream,
and sizes the caller-owned workspace. There is no CPU path: if the library is
not built, or no GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libivf.so")

IVF_OK, IVF_EINVAL, IVF_EUNSUPPORTED, IVF_ENOMEM, IVF_EDEVICE = range(5)
IVF_F32, IVF_U8 = 0, 1
IVF_OP_ROUTE, IVF_OP_KMEANS_STEP, IVF_OP_ASSIGN_BUILD, IVF_OP_BUILD_LISTS, IVF_OP_PQ_TRAIN_STEP, IVF_OP_ADC_SCAN = range(6)
(IVF_OPT_FORCE_FALLBACK, IVF_OPT_SAMPLE_RANK, IVF_OPT_PROFILE, IVF_OPT_BUILD_BLOCKS, IVF_OPT_SCREEN_WAVES,
 IVF_OPT_FP32_SCREEN, IVF_OPT_I8_TWO_PLANE_ONLY, IVF_OPT_FORCE_RESCREEN, IVF_OPT_RESCREEN_CAP,
 IVF_OPT_ASSIGN_SLICE, IVF_OPT_S1_ID_ORDER) = range(11)

STATUS_NAMES = {0: "IVF_OK", 1: "IVF_EINVAL", 2: "IVF_EUNSUPPORTED", 3: "IVF_ENOMEM", 4: "IVF_EDEVICE"}

# Exported symbols and their ctypes signatures: (name, restype, argtypes).
_P = ctypes.c_void_p
_I64, _I32, _U64, _INT, _SZ = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int, ctypes.c_size_t
SIGNATURES = [
    ("ivf_create", _INT, [_INT, _P, ctypes.POINTER(_P)]),
    ("ivf_destroy", None, [_P]),
    ("ivf_last_error", ctypes.c_char_p, [_P]),
    ("ivf_set_stream", _INT, [_P, _P]),
    ("ivf_workspace_bytes", _SZ, [_INT, _I64, _I64, _I32, _I32]),
    ("ivf_set_workspace", _INT, [_P, _P, _SZ]),
    ("ivf_sync", _INT, [_P]),
    ("ivf_route", _INT, [_P, _P, _I64, _P, _I64, _I32, _I32, _P, _P]),
    ("ivf_route_noalloc", _INT, [_P, _P, _I64, _P, _I64, _I32, _I32, _P, _P]),
    ("ivf_kmeans_step", _INT, [_P, _P, _INT, _I64, _P, _I64, _I32, _U64, _I32, _P, _P, _P, _P, _P]),
    ("ivf_assign_build", _INT, [_P, _P, _INT, _I64, _P, _I64, _I32, _P, _P, _P, _P]),
    ("ivf_build_lists", _INT, [_P, _P, _I64, _I64, _P, _P, _P]),
    ("ivf_last_stats", _INT, [_P, ctypes.POINTER(_I64)]),
    ("ivf_set_option", _INT, [_P, _INT, _I64]),
    ("ivf_kernel_times", _INT, [_P, _INT, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_float)]),
    ("ivf_mfma_probe", _INT, [_P, _I32, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)]),
    ("ivf_mfma_probe_i8", _INT, [_P, _I32, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)]),
    ("ivf_list_major", _INT, [_P, _P, _INT, _I64, _P, _I64, _I32, _P, _P, _I64, _I64, _P, _P]),
    ("ivf_pq_encode", _INT, [_P, _P, _I64, _I32, _I32, _P, _P]),
    ("ivf_assign_graph", _INT, [_P, _P, _INT, _I64, _P, _I64, _I32, _P, _I32, _P, _P, _P, _P]),
    ("ivf_assign_cells", _INT, [_P, _P, _INT, _I64, _P, _I64, _I32, _P, _I64, _P, _P, _I64, _P, _I32, _I32, _P, _P, _P]),
    ("ivf_adc_scan", _INT, [_P, _P, _I64, _I32, _P, _I64, _P, _I32, _P, _P, _I64, _P, _I32, _P, _I32, _P, _P]),
    ("ivf_pq_train_step", _INT, [_P, _P, _I64, _I32, _I32, _P, _U64, _I32, _P, _P, _P]),
]

_lib = None


class IvfError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


def load_library(path: str = LIB_PATH):
    """Loads libivf.so (after torch, so that both share one HIP runtime)."""
    global _lib
    if _lib is None:
        try:
            import torch  # noqa: F401
        except ImportError:  # pragma: no cover - torch is part of the image
            pass
        if not os.path.exists(path):
            raise RuntimeError("libivf.so is not built (%s); run __graft_entry__.build()" % path)
        lib = ctypes.CDLL(path)
        for name, res, args in SIGNATURES:
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream_handle():
    import torch

    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class Context:
    """An ivf_ctx bound to a device and to torch's current stream, plus a
    grow-only workspace tensor allocated through torch."""

    def __init__(self, device: int = 0):
        import torch

        self.lib = load_library()
        self.device = device
        self._ws = None
        h = ctypes.c_void_p()
        if device >= 0:
            with torch.cuda.device(device):
                st = self.lib.ivf_create(device, _stream_handle(), ctypes.byref(h))
        else:
            st = self.lib.ivf_create(device, None, ctypes.byref(h))
        if st != IVF_OK:
            raise IvfError(st, "ivf_create(%d) failed" % device)
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            self.lib.ivf_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def error(self) -> str:
        return (self.lib.ivf_last_error(self.handle) or b"").decode()

    def check(self, st: int, what: str):
        if st != IVF_OK:
            raise IvfError(st, "%s: %s" % (what, self.error()))

    def set_option(self, option: int, value: int):
        self.check(self.lib.ivf_set_option(self.handle, option, value), "ivf_set_option")

    def ensure_workspace(self, nbytes: int):
        import torch

        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = None
            self._ws = torch.empty(max(nbytes, 1 << 20), dtype=torch.uint8, device="cuda:%d" % self.device)
        self.check(self.lib.ivf_set_workspace(self.handle, _ptr(self._ws), self._ws.numel()),
                   "ivf_set_workspace")

    def bind_stream(self):
        self.check(self.lib.ivf_set_stream(self.handle, _stream_handle()), "ivf_set_stream")

    def sync(self):
        self.check(self.lib.ivf_sync(self.handle), "ivf_sync")

    def kernel_times(self):
        """[(kernel name, ms)] of every launch recorded with IVF_OPT_PROFILE on
        since the last read (the read clears the timeline)."""
        n = self.lib.ivf_kernel_times(self.handle, 0, None, None)
        if n < 0:
            raise IvfError(IVF_EDEVICE, "ivf_kernel_times failed")
        names = (ctypes.c_char_p * max(n, 1))()
        ms = (ctypes.c_float * max(n, 1))()
        self.lib.ivf_kernel_times(self.handle, n, names, ms)
        return [(names[i].decode(), float(ms[i])) for i in range(n)]

    def mfma_probe(self, iters: int = 20000):
        """(ms, TFLOP/s) of the fp32 MFMA throughput probe (synchronises)."""
        ms = ctypes.c_float()
        tf = ctypes.c_double()
        self.bind_stream()
        self.check(self.lib.ivf_mfma_probe(self.handle, iters, ctypes.byref(ms), ctypes.byref(tf)),
                   "ivf_mfma_probe")
        return float(ms.value), float(tf.value)

    def mfma_probe_i8(self, iters: int = 20000):
        """(ms, TOP/s) of the int8 MFMA throughput probe (synchronises)."""
        ms = ctypes.c_float()
        tops = ctypes.c_double()
        self.bind_stream()
        self.check(self.lib.ivf_mfma_probe_i8(self.handle, iters, ctypes.byref(ms), ctypes.byref(tops)),
                   "ivf_mfma_probe_i8")
        return float(ms.value), float(tops.value)

    def last_stats(self):
        out = (ctypes.c_int64 * 8)()
        self.check(self.lib.ivf_last_stats(self.handle, out), "ivf_last_stats")
        keys = ("fallback", "refine2", "candidates", "overflow", "sample", "screen_i8", "rescreen")
        return {k: int(out[i]) for i, k in enumerate(keys)}


def _dtype_code(t):
    import torch

    if t.dtype == torch.uint8:
        return IVF_U8
    if t.dtype == torch.float32:
        return IVF_F32
    raise TypeError("rows must be float32 or uint8, got %s" % t.dtype)


def _device_tensor(t, name):
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("%s must be a contiguous device tensor" % name)


def ivf_route(ctx: Context, queries, centroids, nprobe: int, out_ids=None, out_dist=None,
              want_dist: bool = True):
    """Coarse search (Eq. 1 with Eq. 6): ids [Q, nprobe] int32 and squared L2
    distances [Q, nprobe] fp32, ascending (distance, id)."""
    import torch

    _device_tensor(queries, "queries")
    _device_tensor(centroids, "centroids")
    Q, D = queries.shape
    C = centroids.shape[0]
    dev = queries.device
    if out_ids is None:
        out_ids = torch.empty((Q, nprobe), dtype=torch.int32, device=dev)
    if out_dist is None and want_dist:
        out_dist = torch.empty((Q, nprobe), dtype=torch.float32, device=dev)
    ctx.ensure_workspace(ctx.lib.ivf_workspace_bytes(IVF_OP_ROUTE, Q, C, D, nprobe))
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_route(ctx.handle, _ptr(queries), Q, _ptr(centroids), C, D, nprobe,
                                _ptr(out_ids), _ptr(out_dist)), "ivf_route")
    return out_ids, out_dist


def ivf_route_noalloc(ctx: Context, queries, centroids, nprobe: int, out_ids, out_dist=None):
    """ivf_route without a workspace: the library's static device scratch is
    used and nothing is allocated by the call (out_ids / out_dist are the
    caller's). Calls that overlap on one device race."""
    _device_tensor(queries, "queries")
    _device_tensor(centroids, "centroids")
    Q, D = queries.shape
    C = centroids.shape[0]
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_route_noalloc(ctx.handle, _ptr(queries), Q, _ptr(centroids), C, D, nprobe,
                                        _ptr(out_ids), _ptr(out_dist)), "ivf_route_noalloc")
    return out_ids, out_dist


def ivf_kmeans_step(ctx: Context, train, centroids, seed: int = 0, it: int = 0, out_labels=None,
                    out_centroids=None, out_counts=None, out_objective=None, hint_labels=None):
    """One Lloyd iteration: labels [N] int32, new centroids [C, D] fp32,
    counts [C] int64 (before reseeding), objective (device fp64 scalar).
    `hint_labels` (int32 [N], e.g. the previous iteration's labels) only
    changes the speed."""
    import torch

    _device_tensor(train, "train")
    _device_tensor(centroids, "centroids")
    N, D = train.shape
    C = centroids.shape[0]
    dev = train.device
    if out_labels is None:
        out_labels = torch.empty(N, dtype=torch.int32, device=dev)
    if out_centroids is None:
        out_centroids = torch.empty((C, D), dtype=torch.float32, device=dev)
    if out_counts is None:
        out_counts = torch.empty(C, dtype=torch.int64, device=dev)
    if out_objective is None:
        out_objective = torch.empty(2, dtype=torch.float64, device=dev)
    if hint_labels is not None:
        _device_tensor(hint_labels, "hint_labels")
    ctx.ensure_workspace(ctx.lib.ivf_workspace_bytes(IVF_OP_KMEANS_STEP, N, C, D, 0))
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_kmeans_step(ctx.handle, _ptr(train), _dtype_code(train), N, _ptr(centroids),
                                      C, D, seed & (2**64 - 1), it, _ptr(out_labels),
                                      _ptr(out_centroids), _ptr(out_counts), _ptr(out_objective),
                                      _ptr(hint_labels) if hint_labels is not None else None),
              "ivf_kmeans_step")
    return out_labels, out_centroids, out_counts, out_objective


def ivf_assign_build(ctx: Context, base, centroids, out_labels=None, out_counts=None,
                     out_offsets=None, out_perm=None):
    """Full assignment + inverted lists: labels [N], counts [C], offsets [C+1], perm [N]."""
    import torch

    _device_tensor(base, "base")
    _device_tensor(centroids, "centroids")
    N, D = base.shape
    C = centroids.shape[0]
    dev = base.device
    if out_labels is None:
        out_labels = torch.empty(N, dtype=torch.int32, device=dev)
    if out_counts is None:
        out_counts = torch.empty(C, dtype=torch.int64, device=dev)
    if out_offsets is None:
        out_offsets = torch.empty(C + 1, dtype=torch.int64, device=dev)
    if out_perm is None:
        out_perm = torch.empty(N, dtype=torch.int32, device=dev)  # uint32 bit pattern
    ctx.ensure_workspace(ctx.lib.ivf_workspace_bytes(IVF_OP_ASSIGN_BUILD, N, C, D, 0))
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_assign_build(ctx.handle, _ptr(base), _dtype_code(base), N, _ptr(centroids),
                                       C, D, _ptr(out_labels), _ptr(out_counts), _ptr(out_offsets),
                                       _ptr(out_perm)), "ivf_assign_build")
    return out_labels, out_counts, out_offsets, out_perm


def ivf_build_lists(ctx: Context, labels, C: int, out_counts=None, out_offsets=None, out_perm=None):
    """Inverted lists for given labels: counts [C], offsets [C+1], perm [N] (uint32 bits in int32)."""
    import torch

    _device_tensor(labels, "labels")
    N = labels.shape[0]
    dev = labels.device
    if out_counts is None:
        out_counts = torch.empty(C, dtype=torch.int64, device=dev)
    if out_offsets is None:
        out_offsets = torch.empty(C + 1, dtype=torch.int64, device=dev)
    if out_perm is None:
        out_perm = torch.empty(N, dtype=torch.int32, device=dev)
    ctx.ensure_workspace(ctx.lib.ivf_workspace_bytes(IVF_OP_BUILD_LISTS, N, C, 0, 0))
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_build_lists(ctx.handle, _ptr(labels), N, C, _ptr(out_counts),
                                      _ptr(out_offsets), _ptr(out_perm)), "ivf_build_lists")
    return out_counts, out_offsets, out_perm


def ivf_list_major(ctx: Context, base, centroids, offsets, perm, pos0: int = 0, n=None,
                   rows: bool = True, residuals: bool = True, out_rows=None, out_residuals=None):
    """List-major copy base[perm[pos0:pos0+n]] and residuals against each
    position's list centroid (fp32). Returns (rows or None, residuals or None)."""
    import torch

    for t, name in ((base, "base"), (centroids, "centroids"), (offsets, "offsets"), (perm, "perm")):
        _device_tensor(t, name)
    N, D = base.shape
    C = centroids.shape[0]
    if n is None:
        n = N - pos0
    dev = base.device
    if rows and out_rows is None:
        out_rows = torch.empty((n, D), dtype=base.dtype, device=dev)
    if residuals and out_residuals is None:
        out_residuals = torch.empty((n, D), dtype=torch.float32, device=dev)
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_list_major(ctx.handle, _ptr(base), _dtype_code(base), N, _ptr(centroids), C, D,
                                     _ptr(offsets), _ptr(perm), pos0, n,
                                     _ptr(out_rows if rows else None),
                                     _ptr(out_residuals if residuals else None)), "ivf_list_major")
    return (out_rows if rows else None), (out_residuals if residuals else None)


PQ_K = 256


def ivf_pq_encode(ctx: Context, x, codebooks, out_codes=None):
    """PQ codes uint8 [n, M] of fp32 rows x [n, D] with codebooks [M, 256, D/M]."""
    import torch

    _device_tensor(x, "x")
    _device_tensor(codebooks, "codebooks")
    n, D = x.shape
    M = codebooks.shape[0]
    if out_codes is None:
        out_codes = torch.empty((n, M), dtype=torch.uint8, device=x.device)
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_pq_encode(ctx.handle, _ptr(x), n, D, M, _ptr(codebooks), _ptr(out_codes)),
              "ivf_pq_encode")
    return out_codes


def ivf_pq_train_step(ctx: Context, x, codebooks, seed: int = 0, it: int = 0, out_codebooks=None,
                      out_counts=None, out_objective=None):
    """One Lloyd step per subspace: (codebooks [M, 256, D/M], counts int64 [M, 256],
    objectives fp64 [M])."""
    import torch

    _device_tensor(x, "x")
    _device_tensor(codebooks, "codebooks")
    n, D = x.shape
    M = codebooks.shape[0]
    dev = x.device
    if out_codebooks is None:
        out_codebooks = torch.empty_like(codebooks)
    if out_counts is None:
        out_counts = torch.empty((M, PQ_K), dtype=torch.int64, device=dev)
    if out_objective is None:
        out_objective = torch.empty(M, dtype=torch.float64, device=dev)
    ctx.ensure_workspace(ctx.lib.ivf_workspace_bytes(IVF_OP_PQ_TRAIN_STEP, n, M, D, 0))
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_pq_train_step(ctx.handle, _ptr(x), n, D, M, _ptr(codebooks), seed & (2**64 - 1), it,
                                        _ptr(out_codebooks), _ptr(out_counts), _ptr(out_objective)),
              "ivf_pq_train_step")
    return out_codebooks, out_counts, out_objective


def ivf_assign_graph(ctx: Context, rows, centroids, graph, prev, order=None, out_labels=None, out_dist=None,
                     want_dist: bool = True):
    """Nearest of each row's candidates graph[prev[i]] (int32 [C, S]):
    labels int32 [N] and squared distances fp32 [N]. `order` (int32 [N] or
    None) only sets the processing order."""
    import torch

    for t, name in ((rows, "rows"), (centroids, "centroids"), (graph, "graph"), (prev, "prev")):
        _device_tensor(t, name)
    N, D = rows.shape
    C = centroids.shape[0]
    S = graph.shape[1]
    if out_labels is None:
        out_labels = torch.empty(N, dtype=torch.int32, device=rows.device)
    if want_dist and out_dist is None:
        out_dist = torch.empty(N, dtype=torch.float32, device=rows.device)
    ctx.bind_stream()
    if order is not None:
        _device_tensor(order, "order")
    ctx.check(ctx.lib.ivf_assign_graph(ctx.handle, _ptr(rows), _dtype_code(rows), N, _ptr(centroids), C, D,
                                       _ptr(graph), S, _ptr(prev), _ptr(order) if order is not None else None,
                                       _ptr(out_labels), _ptr(out_dist if want_dist else None)),
              "ivf_assign_graph")
    return out_labels, (out_dist if want_dist else None)


def ivf_assign_cells(ctx: Context, rows, centroids, cell, cell_offsets, cell_members, graph=None, hops: int = 0,
                     order=None, out_labels=None, out_dist=None, want_dist: bool = True):
    """Nearest member of each row's coarse cell, then up to `hops` greedy
    moves over graph (int32 [C, S] or None): labels int32 [N] and squared
    distances fp32 [N]. `order` (int32 [N] or None) only sets the processing
    order."""
    import torch

    for t, name in ((rows, "rows"), (centroids, "centroids"), (cell, "cell"), (cell_offsets, "cell_offsets"),
                    (cell_members, "cell_members")):
        _device_tensor(t, name)
    if graph is not None:
        _device_tensor(graph, "graph")
    if order is not None:
        _device_tensor(order, "order")
    N, D = rows.shape
    C = centroids.shape[0]
    G = cell_offsets.shape[0] - 1
    M = cell_members.shape[0]
    S = graph.shape[1] if graph is not None else 0
    if out_labels is None:
        out_labels = torch.empty(N, dtype=torch.int32, device=rows.device)
    if want_dist and out_dist is None:
        out_dist = torch.empty(N, dtype=torch.float32, device=rows.device)
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_assign_cells(ctx.handle, _ptr(rows), _dtype_code(rows), N, _ptr(centroids), C, D,
                                       _ptr(cell), G, _ptr(cell_offsets), _ptr(cell_members) if M else None, M,
                                       _ptr(graph) if graph is not None else None, S, hops,
                                       _ptr(order) if order is not None else None, _ptr(out_labels),
                                       _ptr(out_dist if want_dist else None)), "ivf_assign_cells")
    return out_labels, (out_dist if want_dist else None)


def ivf_adc_scan(ctx: Context, queries, centroids, probes, offsets, perm, codes, codebooks, k: int,
                 out_ids=None, out_dist=None):
    """Residual-PQ ADC scan: each query's k best (approximate distance, row id)
    over its probed lists. Returns (ids [B, k] uint32 bits in int32, dist [B, k])."""
    import torch

    for t, name in ((queries, "queries"), (centroids, "centroids"), (probes, "probes"), (offsets, "offsets"),
                    (perm, "perm"), (codes, "codes"), (codebooks, "codebooks")):
        _device_tensor(t, name)
    B, D = queries.shape
    C = centroids.shape[0]
    P = probes.shape[1]
    N, M = codes.shape
    dev = queries.device
    if out_ids is None:
        out_ids = torch.empty((B, k), dtype=torch.int32, device=dev)
    if out_dist is None:
        out_dist = torch.empty((B, k), dtype=torch.float32, device=dev)
    ctx.ensure_workspace(ctx.lib.ivf_workspace_bytes(IVF_OP_ADC_SCAN, B, P, D, k))
    ctx.bind_stream()
    ctx.check(ctx.lib.ivf_adc_scan(ctx.handle, _ptr(queries), B, D, _ptr(centroids), C, _ptr(probes), P,
                                   _ptr(offsets), _ptr(perm), N, _ptr(codes), M, _ptr(codebooks), k,
                                   _ptr(out_ids), _ptr(out_dist)), "ivf_adc_scan")
    return out_ids, out_dist
