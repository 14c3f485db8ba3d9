"""C-ABI contract on the CPU: the library loads, exports every symbol the
header declares, and validates arguments before touching any device (a
validation-only context, device -1, reports IVF_EDEVICE only after every
check has passed)."""
import ctypes
import os
import re

import pytest

import paper_2608_08751_amd as ivf
from paper_2608_08751_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ivf.h")

BASE = 0x7F0000000000  # fake, 256-byte aligned device addresses (never dereferenced)
GB = 1 << 30


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ivf_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return ivf.load_library()


@pytest.fixture()
def vctx(lib):
    ctx = ivf.Context(-1)
    yield ctx
    ctx.close()


def P(off):
    return ctypes.c_void_p(BASE + off)


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), "libivf.so does not export %s" % n
    assert sorted(n for n, _, _ in B.SIGNATURES) == names


def test_workspace_bytes(lib):
    f = lib.ivf_workspace_bytes
    assert f(B.IVF_OP_ROUTE, 1000, 1024, 128, 16) > 0
    assert f(B.IVF_OP_ROUTE, 10000, 65536, 128, 64) > f(B.IVF_OP_ROUTE, 1000, 65536, 128, 64)
    assert f(B.IVF_OP_KMEANS_STEP, 10**6, 4096, 128, 0) > f(B.IVF_OP_KMEANS_STEP, 10**5, 4096, 128, 0)
    assert f(B.IVF_OP_ROUTE, 10, 0, 128, 1) == 0
    assert f(B.IVF_OP_ROUTE, 10, 10, 128, 0) == 0
    assert f(99, 10, 10, 128, 1) == 0


def route(ctx, q=P(0), Q=1000, c=P(GB), C=4096, D=128, k=16, ids=P(2 * GB), dist=P(3 * GB)):
    return ctx.lib.ivf_route(ctx.handle, q, Q, c, C, D, k, ids, dist)


def with_ws(ctx, nbytes=4 * GB):
    ctx.lib.ivf_set_workspace(ctx.handle, P(8 * GB), nbytes)


def test_route_validation(vctx):
    with_ws(vctx)
    assert route(vctx) == B.IVF_EDEVICE  # every check passed
    assert route(vctx, k=0) == B.IVF_EINVAL
    assert route(vctx, k=4097, C=4096) == B.IVF_EINVAL
    assert route(vctx, k=2000, C=4096) == B.IVF_EUNSUPPORTED
    assert route(vctx, C=0) == B.IVF_EINVAL
    assert route(vctx, Q=-1) == B.IVF_EINVAL
    assert route(vctx, D=3) == B.IVF_EUNSUPPORTED
    assert route(vctx, D=130) == B.IVF_EUNSUPPORTED
    assert route(vctx, D=260) == B.IVF_EUNSUPPORTED
    assert route(vctx, q=None) == B.IVF_EINVAL
    assert route(vctx, ids=None) == B.IVF_EINVAL
    assert route(vctx, q=P(4)) == B.IVF_EINVAL  # misaligned
    assert "aligned" in vctx.error()
    assert route(vctx, ids=P(0)) == B.IVF_EINVAL  # output overlaps queries
    assert "overlap" in vctx.error()
    assert route(vctx, dist=P(2 * GB)) == B.IVF_EINVAL  # outputs overlap each other
    assert route(vctx, Q=0) == B.IVF_OK  # no-op
    assert route(vctx, dist=None) == B.IVF_EDEVICE  # distances are optional


def test_route_workspace_too_small(vctx):
    need = vctx.lib.ivf_workspace_bytes(B.IVF_OP_ROUTE, 1000, 4096, 128, 16)
    assert route(vctx) == B.IVF_ENOMEM
    assert "required" in vctx.error() and str(need) in vctx.error()
    with_ws(vctx, need - 1)
    assert route(vctx) == B.IVF_ENOMEM
    with_ws(vctx, need)
    assert route(vctx) == B.IVF_EDEVICE
    assert vctx.lib.ivf_set_workspace(vctx.handle, P(8 * GB + 16), need) == B.IVF_EINVAL


def kstep(ctx, x=P(0), dt=B.IVF_U8, N=10**6, c=P(GB), C=4096, D=128, lab=P(2 * GB), cout=P(3 * GB),
          cnt=P(4 * GB), obj=P(5 * GB), hint=None):
    return ctx.lib.ivf_kmeans_step(ctx.handle, x, dt, N, c, C, D, 7, 0, lab, cout, cnt, obj, hint)


def test_kmeans_validation(vctx):
    with_ws(vctx, 64 * GB)
    assert kstep(vctx) == B.IVF_EDEVICE
    assert kstep(vctx, dt=5) == B.IVF_EINVAL
    assert kstep(vctx, N=-1) == B.IVF_EINVAL
    assert kstep(vctx, N=2**32) == B.IVF_EUNSUPPORTED
    assert kstep(vctx, N=0) == B.IVF_OK
    assert kstep(vctx, cout=P(GB)) == B.IVF_EINVAL  # new centroids alias the input ones
    assert kstep(vctx, lab=P(0)) == B.IVF_EINVAL
    assert kstep(vctx, cnt=P(2 * GB)) == B.IVF_EINVAL
    assert kstep(vctx, cnt=None, obj=None) == B.IVF_EDEVICE  # optional outputs
    assert kstep(vctx, cout=None) == B.IVF_EINVAL
    assert kstep(vctx, D=8, C=0) == B.IVF_EINVAL
    assert kstep(vctx, hint=P(6 * GB)) == B.IVF_EDEVICE  # hint labels (speed only)
    assert kstep(vctx, hint=P(6 * GB + 4)) == B.IVF_EINVAL  # misaligned
    assert kstep(vctx, hint=P(2 * GB + 64)) == B.IVF_EINVAL  # overlaps the labels
    with_ws(vctx, 1024)
    assert kstep(vctx) == B.IVF_ENOMEM


def test_assign_build_and_lists_validation(vctx):
    lib, h = vctx.lib, vctx.handle
    with_ws(vctx, 64 * GB)
    ab = lambda **kw: lib.ivf_assign_build(h, kw.get("x", P(0)), B.IVF_U8, kw.get("N", 10**6), P(GB), 4096, 128,
                                           kw.get("lab", P(2 * GB)), kw.get("cnt", P(3 * GB)),
                                           kw.get("off", P(4 * GB)), kw.get("perm", P(5 * GB)))
    assert ab() == B.IVF_EDEVICE
    assert ab(perm=P(2 * GB)) == B.IVF_EINVAL
    assert ab(off=None) == B.IVF_EINVAL
    assert ab(N=2**32) == B.IVF_EUNSUPPORTED
    bl = lambda **kw: lib.ivf_build_lists(h, kw.get("lab", P(0)), kw.get("N", 10**6), kw.get("C", 4096),
                                          kw.get("cnt", P(GB)), kw.get("off", P(2 * GB)), kw.get("perm", P(3 * GB)))
    assert bl() == B.IVF_EDEVICE
    assert bl(C=0) == B.IVF_EINVAL
    assert bl(perm=P(0)) == B.IVF_EINVAL
    assert bl(N=0) == B.IVF_EDEVICE  # lists of zero rows still write counts/offsets


def test_row_counts_above_int32(vctx):
    """N up to 2^32 - 1 rows is accepted: the assignment screens rows in
    slices of 2^28, so the int32 row ids inside a launch never wrap; the
    slice-sized worklists keep the workspace of a large call modest."""
    lib, h = vctx.lib, vctx.handle
    N = 2**31 + 5
    x0, c0, o0 = 0, 1024 * GB, 1100 * GB
    ab = lambda N, D=4: lib.ivf_assign_build(h, P(x0), B.IVF_U8, N, P(c0), 4096, D, P(o0), P(o0 + 20 * GB),
                                             P(o0 + 21 * GB), P(o0 + 22 * GB))
    ws = lambda N: lib.ivf_workspace_bytes(B.IVF_OP_ASSIGN_BUILD, N, 4096, 4, 0)
    with_ws(vctx, 64 * GB)
    for n in (N, 2**32 - 1):
        assert ws(n) > 0
        assert ab(n) == B.IVF_EDEVICE  # validation passed; no device behind this context
    assert ab(2**32) == B.IVF_EUNSUPPORTED
    # past one slice, the workspace grows only by the list build's per-row
    # scratch, not by the screens' worklists
    wb = lambda N: lib.ivf_workspace_bytes(B.IVF_OP_BUILD_LISTS, N, 4096, 4, 0)
    assert ws(2**30) - ws(2**29) == wb(2**30) - wb(2**29)
    assert ws(2**28) - ws(2**27) > wb(2**28) - wb(2**27)
    assert lib.ivf_set_option(h, B.IVF_OPT_ASSIGN_SLICE, 1000) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_ASSIGN_SLICE, -1) == B.IVF_EINVAL
    assert lib.ivf_set_option(h, B.IVF_OPT_ASSIGN_SLICE, 0) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_S1_ID_ORDER, 1) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_S1_ID_ORDER, 0) == B.IVF_OK


def test_route_noalloc_validation(vctx):
    """Routing with the static scratch: same argument checks as ivf_route, and
    sizes whose layout for one query exceeds the 64 MiB scratch are refused
    (before any device use)."""
    lib, h = vctx.lib, vctx.handle
    rn = lambda Q=1000, C=4096, D=128, k=16, ids=P(2 * GB): lib.ivf_route_noalloc(h, P(0), Q, P(GB), C, D, k, ids,
                                                                                 None)
    assert rn() == B.IVF_EDEVICE  # valid; no device behind this context
    assert rn(Q=0) == B.IVF_OK
    assert rn(k=0) == B.IVF_EINVAL
    assert rn(k=2000, C=5000) == B.IVF_EUNSUPPORTED
    assert rn(D=6) == B.IVF_EUNSUPPORTED
    assert rn(ids=P(0)) == B.IVF_EINVAL
    assert rn(C=20_000_000, D=4, ids=P(8 * GB)) == B.IVF_EUNSUPPORTED
    assert "static scratch" in vctx.error()
    assert rn(C=2_000_000, D=4, k=8, ids=P(8 * GB)) == B.IVF_EDEVICE


def test_options_and_errors(vctx):
    lib, h = vctx.lib, vctx.handle
    assert lib.ivf_set_option(h, B.IVF_OPT_FORCE_FALLBACK, 1) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_SAMPLE_RANK, 16) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_SAMPLE_RANK, -3) == B.IVF_EINVAL
    assert lib.ivf_set_option(h, B.IVF_OPT_I8_TWO_PLANE_ONLY, 1) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_FORCE_RESCREEN, 1) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_RESCREEN_CAP, 5) == B.IVF_OK
    assert lib.ivf_set_option(h, B.IVF_OPT_RESCREEN_CAP, -1) == B.IVF_EINVAL
    assert lib.ivf_set_option(h, 42, 0) == B.IVF_EINVAL
    assert "unknown option" in vctx.error()
    assert lib.ivf_sync(h) == B.IVF_OK
    out = (ctypes.c_int64 * 8)()
    assert lib.ivf_last_stats(h, out) == B.IVF_OK and list(out) == [0] * 8
    assert lib.ivf_route(None, P(0), 1, P(GB), 1, 4, 1, P(2 * GB), None) == B.IVF_EINVAL


@pytest.mark.parametrize("fn", ["ivf_mfma_probe", "ivf_mfma_probe_i8"])
def test_mfma_probe_validation(vctx, fn):
    lib, h = vctx.lib, vctx.handle
    probe = getattr(lib, fn)
    ms, tf = ctypes.c_float(), ctypes.c_double()
    assert probe(h, 0, ctypes.byref(ms), ctypes.byref(tf)) == B.IVF_EINVAL
    assert probe(h, 1 << 21, ctypes.byref(ms), None) == B.IVF_EINVAL
    assert probe(h, 10, None, None) == B.IVF_EINVAL
    assert probe(h, 10, ctypes.byref(ms), None) == B.IVF_EUNSUPPORTED
    assert probe(None, 10, ctypes.byref(ms), None) == B.IVF_EINVAL


def test_list_major_validation(vctx):
    lib, h = vctx.lib, vctx.handle
    N, C, D = 1000, 10, 16
    base, cent, off, perm, rows, res = P(0), P(GB), P(2 * GB), P(3 * GB), P(4 * GB), P(5 * GB)
    call = lambda **k: lib.ivf_list_major(h, k.get("base", base), k.get("dt", B.IVF_U8), k.get("N", N),
                                          k.get("cent", cent), k.get("C", C), k.get("D", D), k.get("off", off),
                                          k.get("perm", perm), k.get("pos0", 0), k.get("n", N),
                                          k.get("rows", rows), k.get("res", res))
    assert call() == B.IVF_EDEVICE  # every check passed; no device behind the context
    assert call(pos0=10, n=N - 10) == B.IVF_EDEVICE
    assert call(pos0=10, n=N) == B.IVF_EINVAL
    assert call(pos0=-1, n=1) == B.IVF_EINVAL
    assert call(n=-1) == B.IVF_EINVAL
    assert call(n=0) == B.IVF_OK and call(n=0, rows=None, res=None) == B.IVF_OK
    assert call(rows=None, res=None) == B.IVF_EINVAL
    assert call(rows=None) == B.IVF_EDEVICE and call(res=None) == B.IVF_EDEVICE
    assert call(D=18) == B.IVF_EUNSUPPORTED
    assert call(dt=7) == B.IVF_EINVAL
    assert call(perm=None) == B.IVF_EINVAL and call(off=None) == B.IVF_EINVAL
    assert call(rows=P(GB + 64)) == B.IVF_EINVAL  # overlaps the centroids
    assert call(res=P(4 * GB + 1000)) == B.IVF_EINVAL  # overlaps out_rows
    assert call(rows=P(4 * GB + 8)) == B.IVF_EINVAL  # misaligned
    assert call(N=1 << 33, n=1) == B.IVF_EUNSUPPORTED


def test_pq_validation(vctx, lib):
    h = vctx.handle
    x, cb, out, cnt, obj = P(0), P(GB), P(2 * GB), P(3 * GB), P(4 * GB)
    assert lib.ivf_pq_encode(h, x, 1000, 128, 16, cb, out) == B.IVF_EDEVICE
    assert lib.ivf_pq_encode(h, x, 0, 128, 16, cb, out) == B.IVF_OK
    assert lib.ivf_pq_encode(h, x, 1000, 128, 12, cb, out) == B.IVF_EINVAL  # 12 does not divide 128
    assert lib.ivf_pq_encode(h, x, 1000, 128, 4, cb, out) == B.IVF_EUNSUPPORTED  # 32 dims per subspace
    assert lib.ivf_pq_encode(h, x, 1000, 130, 10, cb, out) == B.IVF_EUNSUPPORTED  # D % 4
    assert lib.ivf_pq_encode(h, x, 1000, 128, 16, None, out) == B.IVF_EINVAL
    assert lib.ivf_pq_encode(h, x, 1000, 128, 16, cb, P(GB + 128)) == B.IVF_EINVAL  # overlaps codebooks
    need = lib.ivf_workspace_bytes(B.IVF_OP_PQ_TRAIN_STEP, 1000, 16, 128, 0)
    assert need > 1000 * 8
    assert lib.ivf_pq_train_step(h, x, 1000, 128, 16, cb, 0, 0, out, cnt, obj) == B.IVF_ENOMEM
    assert "workspace" in vctx.error()
    assert lib.ivf_set_workspace(h, P(8 * GB), need) == B.IVF_OK
    assert lib.ivf_pq_train_step(h, x, 1000, 128, 16, cb, 0, 0, out, cnt, obj) == B.IVF_EDEVICE
    assert lib.ivf_pq_train_step(h, x, 1000, 128, 16, cb, 0, 0, out, None, None) == B.IVF_EDEVICE
    assert lib.ivf_pq_train_step(h, x, 0, 128, 16, cb, 0, 0, out, cnt, obj) == B.IVF_EINVAL
    assert lib.ivf_pq_train_step(h, x, 1000, 128, 16, cb, 0, 0, cb, cnt, obj) == B.IVF_EINVAL  # aliasing


def test_assign_graph_validation(vctx, lib):
    h = vctx.handle
    rows, cent, graph, prev, lab, dist, order = P(0), P(GB), P(2 * GB), P(3 * GB), P(4 * GB), P(5 * GB), P(6 * GB)
    ok = lambda **k: lib.ivf_assign_graph(h, k.get("rows", rows), B.IVF_U8, k.get("N", 1000), cent, 100, 128,
                                          k.get("graph", graph), k.get("S", 8), k.get("prev", prev),
                                          k.get("order", order), k.get("lab", lab), k.get("dist", dist))
    assert ok() == B.IVF_EDEVICE
    assert ok(dist=None) == B.IVF_EDEVICE
    assert ok(N=0) == B.IVF_OK
    assert ok(S=0) == B.IVF_EINVAL and ok(S=65) == B.IVF_EINVAL
    assert ok(graph=None) == B.IVF_EINVAL and ok(prev=None) == B.IVF_EINVAL and ok(lab=None) == B.IVF_EINVAL
    assert ok(lab=P(3 * GB + 16)) == B.IVF_EINVAL  # overlaps prev
    assert ok(dist=P(4 * GB + 64)) == B.IVF_EINVAL  # overlaps the labels
    assert ok(dist=P(5 * GB + 4)) == B.IVF_EINVAL  # misaligned
    assert ok(order=None) == B.IVF_EDEVICE and ok(order=P(6 * GB + 4)) == B.IVF_EINVAL
    assert ok(lab=P(6 * GB + 16)) == B.IVF_EINVAL  # overlaps the order


def test_assign_cells_validation(vctx, lib):
    h = vctx.handle
    rows, cent, cell, off, mem, graph, lab, dist, order = (P(i * GB) for i in range(9))
    ok = lambda **k: lib.ivf_assign_cells(h, rows, B.IVF_U8, k.get("N", 1000), cent, 100, k.get("D", 128),
                                          k.get("cell", cell), k.get("G", 10), k.get("off", off),
                                          k.get("mem", mem), k.get("M", 100), k.get("graph", graph),
                                          k.get("S", 8), k.get("hops", 4), k.get("order", order),
                                          k.get("lab", lab), k.get("dist", dist))
    assert ok() == B.IVF_EDEVICE
    assert ok(graph=None, S=0) == B.IVF_EDEVICE and ok(dist=None) == B.IVF_EDEVICE
    assert ok(mem=None, M=0) == B.IVF_EDEVICE and ok(order=None) == B.IVF_EDEVICE
    assert ok(order=P(8 * GB + 4)) == B.IVF_EINVAL  # misaligned
    assert ok(lab=P(8 * GB + 64)) == B.IVF_EINVAL  # overlaps the order
    assert ok(N=0) == B.IVF_OK
    assert ok(G=0) == B.IVF_EINVAL and ok(M=-1) == B.IVF_EINVAL
    assert ok(hops=-1) == B.IVF_EINVAL and ok(hops=1025) == B.IVF_EINVAL
    assert ok(S=0) == B.IVF_EINVAL and ok(S=65) == B.IVF_EINVAL
    assert ok(D=260) == B.IVF_EUNSUPPORTED and ok(N=1 << 32) == B.IVF_EUNSUPPORTED
    assert ok(cell=None) == B.IVF_EINVAL and ok(off=None) == B.IVF_EINVAL and ok(mem=None) == B.IVF_EINVAL
    assert ok(lab=None) == B.IVF_EINVAL
    assert ok(lab=P(2 * GB + 16)) == B.IVF_EINVAL  # overlaps cell
    assert ok(dist=P(6 * GB + 64)) == B.IVF_EINVAL  # overlaps the labels
    assert ok(off=P(3 * GB + 8)) == B.IVF_EINVAL  # misaligned


def test_adc_scan_validation(vctx, lib):
    h = vctx.handle
    q, c, pr, off, perm, codes, cb, ids, dist = (P(i * GB) for i in range(9))
    call = lambda **a: lib.ivf_adc_scan(h, q, a.get("B", 100), 128, c, 1000, pr, a.get("P", 64), off, perm,
                                        a.get("N", 100000), codes, a.get("M", 16), cb, a.get("k", 512),
                                        a.get("ids", ids), a.get("dist", dist))
    need = lib.ivf_workspace_bytes(B.IVF_OP_ADC_SCAN, 100, 64, 128, 512)
    # handoff keys (at most 2 * 64 groups of 512 per query) plus the group
    # descriptors and handoff counts
    assert 100 * 128 * 512 * 8 < need <= 100 * 128 * (512 * 8 + 24) + 100 * 4 + 6 * 256
    assert lib.ivf_workspace_bytes(B.IVF_OP_ADC_SCAN, 100, 64, 128, 2000) == 0
    assert call() == B.IVF_ENOMEM
    assert lib.ivf_set_workspace(h, P(20 * GB), need) == B.IVF_OK
    assert call() == B.IVF_EDEVICE
    assert call(B=0) == B.IVF_OK
    assert call(k=0) == B.IVF_EINVAL and call(k=1025) == B.IVF_EINVAL
    assert call(P=0) == B.IVF_EINVAL
    assert call(M=12) == B.IVF_EINVAL and call(M=64) == B.IVF_EUNSUPPORTED
    assert call(N=1 << 33) == B.IVF_EUNSUPPORTED
    assert call(ids=None) == B.IVF_EINVAL
    assert call(dist=P(7 * GB + 64)) == B.IVF_EINVAL  # overlaps the ids


def test_no_cpu_fallback_without_gpu():
    import torch

    if torch.cuda.is_available():
        pytest.skip("GPU present")
    with pytest.raises(Exception):
        ivf.Context(0)
