"""CPU oracle for the IVF hot path of InSituANN (arXiv 2608.08751).

TEST INFRASTRUCTURE ONLY. The tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module; the product package
``paper_2608_08751_amd`` never does, and shares no code with it.

The arithmetic lives in ``oracle.c`` (plain C, fp64, explicit ``fma``,
``-ffp-contract=off``); this module only builds it with gcc and marshals numpy
arrays through ctypes. Definitions followed:

* ``dist``           squared L2, the left-hand side of Eq. (6), evaluated directly;
* ``route``          coarse search, Eq. (1): nprobe nearest centroids by (distance, id);
* ``assign``         nearest centroid per vector, ties to the lower id;
* ``assign_graph``   nearest among each vector's candidate centroids (fast construction);
* ``assign_cells``   nearest among a coarse cell's member centroids, then a greedy graph walk;
* ``kmeans_update``  Lloyd mean update with deterministic reseed of empty clusters;
* ``objective``      sum of squared distances of every vector to its assigned centroid;
* ``build_lists``    cluster-major inverted lists: counts, offsets, stable permutation;
* ``list_major``     list-major copy of the vectors and their residuals x - c(x);
* ``pq_encode``      product-quantisation codes (nearest codeword per subspace);
* ``pq_train_step``  one Lloyd step per subspace codebook;
* ``adc_scan``       PQ approximate-distance scan of probed lists, k best per query.

Parity pins for each function are in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F32, U8 = 0, 1

_lib = None


def build(force: bool = False) -> str:
    """Compile ``liboracle.so`` with gcc (no GPU, no HIP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(
        os.path.getmtime(_SRC), os.path.getmtime(os.path.join(_HERE, "oracle.h"))
    ):
        tmp = _LIB + ".tmp%d" % os.getpid()
        # -mfma: fma() is emitted as the x86-64 fused multiply-add
        # instruction instead of a libm call (the same correctly rounded
        # operation, about 1.7x faster); contraction of separate multiplies
        # and adds stays off
        cmd = [
            "gcc", "-O2", "-mfma", "-std=c11", "-fPIC", "-shared", "-pthread",
            "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
            _SRC, "-o", tmp, "-lm",
        ]
        subprocess.check_call(cmd, cwd=_HERE)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        i64, i32, u64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
        ci = ctypes.c_int
        lib.oracle_dist.argtypes = [p, p, ci]
        lib.oracle_dist.restype = ctypes.c_double
        lib.oracle_route.argtypes = [p, i64, p, i64, ci, ci, p, p, ci]
        lib.oracle_assign.argtypes = [p, ci, i64, p, i64, ci, p, p, ci]
        lib.oracle_splitmix64_nth.argtypes = [u64, u64]
        lib.oracle_splitmix64_nth.restype = u64
        lib.oracle_reseed_row.argtypes = [u64, i32, i64, i64]
        lib.oracle_reseed_row.restype = i64
        lib.oracle_kmeans_update.argtypes = [p, ci, i64, ci, p, i64, u64, i32, p, p]
        lib.oracle_objective.argtypes = [p, ci, i64, ci, p, p, i64, p]
        lib.oracle_kmeans_step.argtypes = [p, ci, i64, p, i64, ci, u64, i32, p, p, p, p, ci]
        lib.oracle_build_lists.argtypes = [p, i64, i64, p, p, p]
        lib.oracle_num_threads.argtypes = [ci]
        lib.oracle_list_major.argtypes = [p, ci, i64, p, i64, ci, p, p, i64, p, p]
        lib.oracle_pq_encode.argtypes = [p, i64, ci, ci, p, p, ci]
        lib.oracle_assign_graph.argtypes = [p, ci, i64, p, i64, ci, p, ci, p, p, p, ci]
        lib.oracle_assign_cells.argtypes = [p, ci, i64, p, i64, ci, p, i64, p, p, i64, p, ci, ci, p, p, ci]
        lib.oracle_adc_scan.argtypes = [p, i64, ci, p, i64, p, ci, p, p, p, ci, p, ci, p, p]
        lib.oracle_pq_train_step.argtypes = [p, i64, ci, ci, p, u64, i32, p, p, p, ci]
        for f in (lib.oracle_route, lib.oracle_assign, lib.oracle_kmeans_update,
                  lib.oracle_objective, lib.oracle_kmeans_step, lib.oracle_build_lists,
                  lib.oracle_num_threads):
            f.restype = ci
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _data(x):
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint8:
        return x, U8
    return np.ascontiguousarray(x, dtype=np.float32), F32


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle_%s rejected its arguments (status %d)" % (what, rc))


def num_threads(nthreads: int = 0) -> int:
    return _load().oracle_num_threads(nthreads)


def dist(x, c) -> float:
    """Squared L2 distance in fp64: s = fma(x_d - c_d, x_d - c_d, s), d ascending."""
    x, c = _f32(x), _f32(c)
    assert x.shape == c.shape and x.ndim == 1
    return _load().oracle_dist(_ptr(x), _ptr(c), x.shape[0])


def route(queries, centroids, nprobe: int, nthreads: int = 0):
    """Eq. (1): per query the nprobe nearest centroids, ascending (distance, id).

    Returns (ids int32 [Q, nprobe], distances float32 [Q, nprobe]); the
    distances are the fp64 values rounded to fp32."""
    q, c = _f32(queries), _f32(centroids)
    Q, D = q.shape
    C = c.shape[0]
    ids = np.empty((Q, nprobe), np.int32)
    dd = np.empty((Q, nprobe), np.float32)
    _check(_load().oracle_route(_ptr(q), Q, _ptr(c), C, D, nprobe, _ptr(ids), _ptr(dd), nthreads), "route")
    return ids, dd


def assign(x, centroids, nthreads: int = 0, return_dist: bool = False):
    """Nearest centroid per row by (distance, id); optionally the fp64 distance."""
    x, dt = _data(x)
    c = _f32(centroids)
    N, D = x.shape
    labels = np.empty(N, np.int32)
    md = np.empty(N, np.float64) if return_dist else None
    _check(_load().oracle_assign(_ptr(x), dt, N, _ptr(c), c.shape[0], D, _ptr(labels), _ptr(md), nthreads), "assign")
    return (labels, md) if return_dist else labels


def assign_graph(x, centroids, graph, prev, nthreads: int = 0, return_dist: bool = False):
    """Candidate-restricted assignment: row i takes the nearest of the centroids
    graph[prev[i]] by (distance, id); -1 (distance inf) when it has none."""
    x, dt = _data(x)
    c = _f32(centroids)
    g = np.ascontiguousarray(graph, dtype=np.int32)
    pv = np.ascontiguousarray(prev, dtype=np.int32)
    N, D = x.shape
    labels = np.empty(N, np.int32)
    md = np.empty(N, np.float64) if return_dist else None
    _check(_load().oracle_assign_graph(_ptr(x), dt, N, _ptr(c), c.shape[0], D, _ptr(g), g.shape[1], _ptr(pv),
                                       _ptr(labels), _ptr(md), nthreads), "assign_graph")
    return (labels, md) if return_dist else labels


def assign_cells(x, centroids, cell, cell_offsets, cell_members, graph=None, hops: int = 0,
                 nthreads: int = 0, return_dist: bool = False):
    """Row i takes the nearest member of its coarse cell cell[i] by (distance,
    id), then walks graph[b] greedily up to `hops` times while a neighbour is
    nearer; -1 (distance inf) when its cell holds no valid member."""
    x, dt = _data(x)
    c = _f32(centroids)
    cl = np.ascontiguousarray(cell, dtype=np.int32)
    off = np.ascontiguousarray(cell_offsets, dtype=np.int64)
    mem = np.ascontiguousarray(cell_members, dtype=np.uint32)
    g = None if graph is None else np.ascontiguousarray(graph, dtype=np.int32)
    N, D = x.shape
    labels = np.empty(N, np.int32)
    md = np.empty(N, np.float64) if return_dist else None
    _check(_load().oracle_assign_cells(_ptr(x), dt, N, _ptr(c), c.shape[0], D, _ptr(cl), off.shape[0] - 1,
                                       _ptr(off), _ptr(mem), mem.shape[0], _ptr(g),
                                       0 if g is None else g.shape[1], hops, _ptr(labels), _ptr(md),
                                       nthreads), "assign_cells")
    return (labels, md) if return_dist else labels


def splitmix64_nth(seed: int, n: int) -> int:
    return int(_load().oracle_splitmix64_nth(seed & (2**64 - 1), n & (2**64 - 1)))


def reseed_row(seed: int, it: int, j: int, n: int) -> int:
    return int(_load().oracle_reseed_row(seed & (2**64 - 1), it, j, n))


def kmeans_update(x, labels, C: int, seed: int = 0, it: int = 0):
    """Lloyd mean update for fixed labels; returns (centroids f32 [C, D], counts int64 [C])."""
    x, dt = _data(x)
    N, D = x.shape
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    out = np.empty((C, D), np.float32)
    cnt = np.empty(C, np.int64)
    _check(_load().oracle_kmeans_update(_ptr(x), dt, N, D, _ptr(lab), C, seed & (2**64 - 1), it, _ptr(out), _ptr(cnt)), "kmeans_update")
    return out, cnt


def objective(x, labels, centroids) -> float:
    x, dt = _data(x)
    c = _f32(centroids)
    N, D = x.shape
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    out = np.zeros(1, np.float64)
    _check(_load().oracle_objective(_ptr(x), dt, N, D, _ptr(lab), _ptr(c), c.shape[0], _ptr(out)), "objective")
    return float(out[0])


def kmeans_step(x, centroids, seed: int = 0, it: int = 0, nthreads: int = 0):
    """One Lloyd iteration. Returns (labels, new centroids, counts, objective)."""
    x, dt = _data(x)
    c = _f32(centroids)
    N, D = x.shape
    C = c.shape[0]
    labels = np.empty(N, np.int32)
    out = np.empty((C, D), np.float32)
    cnt = np.empty(C, np.int64)
    obj = np.zeros(1, np.float64)
    _check(_load().oracle_kmeans_step(_ptr(x), dt, N, _ptr(c), C, D, seed & (2**64 - 1), it,
                                      _ptr(labels), _ptr(out), _ptr(cnt), _ptr(obj), nthreads), "kmeans_step")
    return labels, out, cnt, float(obj[0])


def build_lists(labels, C: int):
    """Counting sort of ids by label: returns (counts int64 [C], offsets int64 [C+1], perm uint32 [N])."""
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    N = lab.shape[0]
    counts = np.empty(C, np.int64)
    offsets = np.empty(C + 1, np.int64)
    perm = np.empty(N, np.uint32)
    _check(_load().oracle_build_lists(_ptr(lab), N, C, _ptr(counts), _ptr(offsets), _ptr(perm)), "build_lists")
    return counts, offsets, perm


def list_major(x, centroids, labels, perm, rows: bool = True, residuals: bool = True):
    """List-major copy x[perm] (same dtype) and residuals x[perm] - c[labels[perm]]
    (fp32, one fp32 subtraction per element); perm may be a slice of the
    permutation. Returns (rows or None, residuals or None)."""
    x, dt = _data(x)
    c = _f32(centroids)
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    perm = np.ascontiguousarray(perm, dtype=np.uint32)
    N, D = x.shape
    n = perm.shape[0]
    out_rows = np.empty((n, D), x.dtype) if rows else None
    out_res = np.empty((n, D), np.float32) if residuals else None
    _check(_load().oracle_list_major(_ptr(x), dt, N, _ptr(c), c.shape[0], D, _ptr(lab), _ptr(perm), n,
                                     _ptr(out_rows), _ptr(out_res)), "list_major")
    return out_rows, out_res


PQ_K = 256


def pq_encode(x, codebooks, nthreads: int = 0):
    """PQ codes uint8 [N, M] of fp32 vectors x [N, D] with codebooks [M, 256, D/M]."""
    x = _f32(x)
    cb = _f32(codebooks)
    N, D = x.shape
    M = cb.shape[0]
    assert cb.shape == (M, PQ_K, D // M)
    codes = np.empty((N, M), np.uint8)
    _check(_load().oracle_pq_encode(_ptr(x), N, D, M, _ptr(cb), _ptr(codes), nthreads), "pq_encode")
    return codes


def pq_train_step(x, codebooks, seed: int = 0, it: int = 0, nthreads: int = 0):
    """One Lloyd step per subspace. Returns (codebooks f32 [M, 256, D/M],
    counts int64 [M, 256], objectives f64 [M])."""
    x = _f32(x)
    cb = _f32(codebooks)
    N, D = x.shape
    M = cb.shape[0]
    assert cb.shape == (M, PQ_K, D // M)
    out = np.empty_like(cb)
    cnt = np.empty((M, PQ_K), np.int64)
    obj = np.zeros(M, np.float64)
    _check(_load().oracle_pq_train_step(_ptr(x), N, D, M, _ptr(cb), seed & (2**64 - 1), it, _ptr(out),
                                        _ptr(cnt), _ptr(obj), nthreads), "pq_train_step")
    return out, cnt, obj


def adc_scan(queries, centroids, probes, offsets, perm, codes, codebooks, k: int):
    """Residual-PQ ADC scan of each query's probed lists: the k smallest
    (approximate distance, row id) pairs. Returns (ids uint32 [B, k],
    distances float32 [B, k]); missing entries are 0xFFFFFFFF and inf."""
    q = _f32(queries)
    c = _f32(centroids)
    pr = np.ascontiguousarray(probes, dtype=np.int32)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    pm = np.ascontiguousarray(perm, dtype=np.uint32)
    cd = np.ascontiguousarray(codes, dtype=np.uint8)
    cb = _f32(codebooks)
    B, D = q.shape
    M = cb.shape[0]
    assert cd.shape[1] == M and cb.shape == (M, PQ_K, D // M)
    ids = np.empty((B, k), np.uint32)
    dd = np.empty((B, k), np.float32)
    _check(_load().oracle_adc_scan(_ptr(q), B, D, _ptr(c), c.shape[0], _ptr(pr), pr.shape[1], _ptr(off), _ptr(pm),
                                   _ptr(cd), M, _ptr(cb), k, _ptr(ids), _ptr(dd)), "adc_scan")
    return ids, dd


def assign_build(x, centroids, nthreads: int = 0):
    """Full assignment followed by the inverted-list build."""
    labels = assign(x, centroids, nthreads)
    counts, offsets, perm = build_lists(labels, np.asarray(centroids).shape[0])
    return labels, counts, offsets, perm
