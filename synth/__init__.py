"""Seeded synthetic inputs for the IVF hot path.

This module only draws inputs; it holds none of the method's arithmetic (no
distances, no selection, no means). Both the GPU path and the oracle consume
its outputs. The shapes follow the paper's datasets (SIFT-like 128-d values in
0..255, DEEP-like 96-d unit-norm floats); no dataset item is reproduced.

Recipes (seed 0 unless stated; every random quantity comes from its own
sub-stream so that changing one size does not shift the others):

* ``uniform_mixture_route``  C means uniform in [0, 255]^D (fp32) are the
  centroids; each query = clip(rint(mean_a + N(0, 20^2 I)), 0, 255) with a
  uniform component a, stored as fp32; ``plants`` seeded queries are replaced
  by exact copies of seeded centroids.
* ``normalised_route``  per-dimension std s_d ~ U[0.2, 1.0] drawn once; each
  centroid = m / ||m|| with m ~ N(0, diag(s^2)); each query =
  normalise(c_a + N(0, 0.05^2 I)); plants as above.
* ``mixture_rows_u8``  rows x_i = clip(rint(mean_{a_i} + 20 z), 0, 255) as
  uint8 from a counter-based generator keyed by (seed, row, dim): a_i and the
  normal pairs z come from SplitMix64 outputs (Steele, Lea & Flood 2014) and the
  Box-Muller transform (Box & Muller 1958). The same recipe runs on the device
  (``device_mixture_rows_u8``) for the 10M- and 1e9-row workloads.
* ``kmeans_init``  a seeded sample of C distinct row indices.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))

# Sub-stream identifiers.
_S_MEANS, _S_COMP, _S_NOISE, _S_PLANT, _S_INIT, _S_STD, _S_LABELS = range(1, 8)

# Per-row counter-based streams (SplitMix64 seeds derived from the user seed).
_GAMMA = 0x9E3779B97F4A7C15
_M64 = (1 << 64) - 1


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), int(stream)])))


def uniform_means(C: int, D: int, seed: int = 0) -> np.ndarray:
    return _rng(seed, _S_MEANS).uniform(0.0, 255.0, size=(C, D)).astype(np.float32)


def _plant(queries: np.ndarray, centroids: np.ndarray, plants: int, seed: int):
    Q = queries.shape[0]
    plants = min(plants, Q)
    if plants <= 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    r = _rng(seed, _S_PLANT)
    qi = r.choice(Q, size=plants, replace=False)
    ci = r.choice(centroids.shape[0], size=plants, replace=False)
    queries[qi] = centroids[ci]
    return qi.astype(np.int64), ci.astype(np.int64)


def uniform_mixture_route(C: int, Q: int, D: int = 128, seed: int = 0, plants: int = 16):
    """Centroids = uniform means; integer-valued fp32 queries around them.

    Returns dict(centroids, queries, comp, plant_q, plant_c)."""
    cent = uniform_means(C, D, seed)
    comp = _rng(seed, _S_COMP).integers(0, C, size=Q)
    noise = _rng(seed, _S_NOISE).normal(0.0, 20.0, size=(Q, D))
    q = np.clip(np.rint(cent[comp].astype(np.float64) + noise), 0, 255).astype(np.float32)
    pq, pc = _plant(q, cent, plants, seed)
    return dict(centroids=cent, queries=q, comp=comp, plant_q=pq, plant_c=pc)


def normalised_route(C: int, Q: int, D: int = 96, seed: int = 0, plants: int = 16):
    """Unit-norm anisotropic-mixture centroids and normalised noisy queries."""
    s = _rng(seed, _S_STD).uniform(0.2, 1.0, size=D)
    m = _rng(seed, _S_MEANS).normal(0.0, 1.0, size=(C, D)) * s
    cent = (m / np.linalg.norm(m, axis=1, keepdims=True)).astype(np.float32)
    comp = _rng(seed, _S_COMP).integers(0, C, size=Q)
    q = cent[comp].astype(np.float64) + _rng(seed, _S_NOISE).normal(0.0, 0.05, size=(Q, D))
    q = (q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32)
    pq, pc = _plant(q, cent, plants, seed)
    return dict(centroids=cent, queries=q, comp=comp, plant_q=pq, plant_c=pc)


# ----------------------------------------------------------------- u8 rows

def _mix(z):
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def _stream_seed(seed: int, stream: int) -> int:
    return int(_mix(np.uint64(((int(seed) * 0x100000001B3) ^ (stream * _GAMMA)) & _M64)))


def _nth(base: int, n):
    with np.errstate(over="ignore"):
        return _mix(np.uint64(base) + np.asarray(n, dtype=np.uint64) * np.uint64(_GAMMA))


def mixture_rows_u8(means: np.ndarray, row0: int, nrows: int, seed: int = 0):
    """Host version of the counter-based u8 mixture (small row counts only).

    Row i (global index) draws its component from output i+1 of the component
    stream, and dims (2p, 2p+1) from output i*D/2 + p + 1 of the noise stream:
    u1 = (top 24 bits + 1) / 2^24, u2 = (low 24 bits) / 2^24,
    z = sqrt(-2 ln u1) * (cos, sin)(2 pi u2), all in fp32."""
    C, D = means.shape
    assert D % 2 == 0
    rows = np.arange(row0, row0 + nrows, dtype=np.uint64)
    a = (_nth(_stream_seed(seed, _S_COMP), rows + np.uint64(1)) % np.uint64(C)).astype(np.int64)
    p = np.arange(D // 2, dtype=np.uint64)
    h = _nth(_stream_seed(seed, _S_NOISE), rows[:, None] * np.uint64(D // 2) + p[None, :] + np.uint64(1))
    u1 = (((h >> np.uint64(40)) + np.uint64(1)).astype(np.float32)) * np.float32(1.0 / 16777216.0)
    u2 = ((h & np.uint64(0xFFFFFF)).astype(np.float32)) * np.float32(1.0 / 16777216.0)
    r = np.sqrt(np.float32(-2.0) * np.log(u1))
    ang = np.float32(6.283185307179586) * u2
    z = np.empty((nrows, D), np.float32)
    z[:, 0::2] = r * np.cos(ang)
    z[:, 1::2] = r * np.sin(ang)
    v = means[a] + np.float32(20.0) * z
    return np.clip(np.rint(v), 0, 255).astype(np.uint8), a


def kmeans_init(n_rows: int, C: int, seed: int = 0) -> np.ndarray:
    """Seeded sample of C distinct row indices (ascending order of draw)."""
    return _rng(seed, _S_INIT).choice(n_rows, size=C, replace=False).astype(np.int64)


def random_labels(N: int, C: int, seed: int = 0, skew: float = 0.0) -> np.ndarray:
    """Seeded labels for list-build tests: uniform, or Zipf-like when skew > 0."""
    r = _rng(seed, _S_LABELS)
    if skew <= 0:
        return r.integers(0, C, size=N).astype(np.int32)
    w = 1.0 / np.arange(1, C + 1, dtype=np.float64) ** skew
    w /= w.sum()
    return r.choice(C, size=N, p=w).astype(np.int32)


# ------------------------------------------------------- device generator

_dev = None


def build_device(force: bool = False) -> str:
    """Compile the device generator library (hipcc, gfx950)."""
    src = os.path.join(_HERE, "csrc", "synth.hip")
    lib = os.path.join(_HERE, "libivfsynth.so")
    if force or not os.path.exists(lib) or os.path.getmtime(lib) < os.path.getmtime(src):
        tmp = lib + ".tmp%d" % os.getpid()
        cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
               "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               src, "-o", tmp]
        subprocess.check_call(cmd, cwd=_HERE)
        os.replace(tmp, lib)
    return lib


def _load_device():
    global _dev
    if _dev is None:
        import torch  # noqa: F401  (share torch's HIP runtime)
        lib = os.path.join(_HERE, "libivfsynth.so")
        if not os.path.exists(lib):
            raise RuntimeError("synth device generator not built: run __graft_entry__.build()")
        d = ctypes.CDLL(lib)
        d.synth_mixture_u8.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                       ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64,
                                       ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        d.synth_mixture_u8.restype = ctypes.c_int
        d.synth_labels_i32.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                       ctypes.c_void_p]
        d.synth_labels_i32.restype = ctypes.c_int
        _dev = d
    return _dev


def device_mixture_rows_u8(means_dev, row0: int, nrows: int, out_dev, seed: int = 0, stream=None):
    """Fill out_dev (torch uint8 [nrows, D] on the GPU) with rows row0.. of the mixture."""
    import torch
    d = _load_device()
    C, D = means_dev.shape
    assert means_dev.dtype == torch.float32 and means_dev.is_contiguous()
    assert out_dev.dtype == torch.uint8 and out_dev.is_contiguous() and tuple(out_dev.shape) == (nrows, D)
    s = stream if stream is not None else torch.cuda.current_stream()
    rc = d.synth_mixture_u8(means_dev.data_ptr(), C, D,
                            _stream_seed(seed, _S_COMP), _stream_seed(seed, _S_NOISE),
                            row0, nrows, out_dev.data_ptr(), ctypes.c_void_p(s.cuda_stream))
    if rc != 0:
        raise RuntimeError("synth_mixture_u8 failed (%d)" % rc)


def device_labels(N: int, C: int, out_dev, seed: int = 0, stream=None):
    """Fill out_dev (torch int32 [N] on the GPU) with uniform labels in [0, C):
    label_i = SplitMix64 output (i + 1) of the label stream, mod C."""
    import torch

    d = _load_device()
    assert out_dev.dtype == torch.int32 and out_dev.is_contiguous() and out_dev.numel() == N
    s = stream if stream is not None else torch.cuda.current_stream()
    rc = d.synth_labels_i32(_stream_seed(seed, _S_LABELS), C, N, out_dev.data_ptr(), ctypes.c_void_p(s.cuda_stream))
    if rc != 0:
        raise RuntimeError("synth_labels_i32 failed (%d)" % rc)


def labels_host(N: int, C: int, seed: int = 0) -> np.ndarray:
    """Host twin of device_labels (bit-identical: integer arithmetic only)."""
    i = np.arange(N, dtype=np.uint64)
    return (_nth(_stream_seed(seed, _S_LABELS), i + np.uint64(1)) % np.uint64(C)).astype(np.int32)
