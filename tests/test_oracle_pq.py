"""Pins for the oracle's product quantisation (CPU only).

Encoding: brute force with exact integer distances on tiny inputs (ties to
the lower codeword index), vectors assembled from codewords, and the
permutation of subspaces. Training: the special cases that reduce to the
pinned k-means step (one subspace; each subspace alone with seed + m), exact
rational means, and Lloyd's monotone objective."""
from fractions import Fraction

import numpy as np
import pytest


def test_encode_brute_force_exact_integers(oracle_mod):
    rng = np.random.default_rng(1)
    for trial in range(20):
        M, dsub, N = int(rng.integers(1, 4)), int(rng.integers(1, 4)), int(rng.integers(1, 30))
        D = M * dsub
        x = rng.integers(-4, 5, (N, D)).astype(np.float32)
        cb = rng.integers(-4, 5, (M, 256, dsub)).astype(np.float32)  # many duplicate codewords
        codes = oracle_mod.pq_encode(x, cb)
        for i in range(N):
            for m in range(M):
                sub = [int(v) for v in x[i, m * dsub:(m + 1) * dsub]]
                d = [sum((a - int(b)) ** 2 for a, b in zip(sub, cb[m, j])) for j in range(256)]
                assert codes[i, m] == min(range(256), key=lambda j: (d[j], j))


def test_encode_vectors_built_from_codewords(oracle_mod):
    rng = np.random.default_rng(2)
    M, dsub = 8, 4
    cb = rng.standard_normal((M, 256, dsub)).astype(np.float32)
    want = rng.integers(0, 256, (50, M))
    x = np.concatenate([cb[m, want[:, m]] for m in range(M)], axis=1)
    assert (oracle_mod.pq_encode(x, cb) == want).all()


def test_encode_permuting_subspaces_permutes_codes(oracle_mod):
    rng = np.random.default_rng(3)
    M, dsub = 4, 3
    x = rng.standard_normal((200, M * dsub)).astype(np.float32)
    cb = rng.standard_normal((M, 256, dsub)).astype(np.float32)
    order = [2, 0, 3, 1]
    xp = np.concatenate([x[:, m * dsub:(m + 1) * dsub] for m in order], axis=1)
    assert (oracle_mod.pq_encode(xp, cb[order]) == oracle_mod.pq_encode(x, cb)[:, order]).all()


def test_train_one_subspace_is_the_kmeans_step(oracle_mod):
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3000, 8)).astype(np.float32)
    cb = x[rng.choice(3000, 256, replace=False)].copy()
    out, cnt, obj = oracle_mod.pq_train_step(x, cb[None], seed=5, it=2)
    _, kc, kcnt, kobj = oracle_mod.kmeans_step(x, cb, seed=5, it=2)
    assert (out[0] == kc).all() and (cnt[0] == kcnt).all() and obj[0] == kobj


def test_train_each_subspace_alone(oracle_mod):
    rng = np.random.default_rng(5)
    M, dsub = 4, 2
    x = rng.standard_normal((700, M * dsub)).astype(np.float32)
    cb = rng.standard_normal((M, 256, dsub)).astype(np.float32) * 3  # far codewords: many empty
    out, cnt, obj = oracle_mod.pq_train_step(x, cb, seed=11, it=0)
    for m in range(M):
        _, kc, kcnt, kobj = oracle_mod.kmeans_step(x[:, m * dsub:(m + 1) * dsub], cb[m], seed=11 + m, it=0)
        assert (out[m] == kc).all() and (cnt[m] == kcnt).all() and obj[m] == kobj
    assert (cnt == 0).any()  # the reseed path ran


def test_train_means_are_exact(oracle_mod):
    rng = np.random.default_rng(6)
    M, dsub, N = 2, 3, 400
    x = (rng.standard_normal((N, M * dsub)) * 7).astype(np.float32)
    cb = x[rng.choice(N, 256, replace=False)].reshape(256, M, dsub).transpose(1, 0, 2).copy()
    out, cnt, _ = oracle_mod.pq_train_step(x, cb)
    codes = oracle_mod.pq_encode(x, cb)
    for m in range(M):
        for j in np.nonzero(cnt[m])[0][:40]:
            rows = np.nonzero(codes[:, m] == j)[0]
            assert len(rows) == cnt[m, j]
            for d in range(dsub):
                exact = sum(Fraction(float(v)) for v in x[rows, m * dsub + d]) / len(rows)
                assert out[m, j, d] == np.float32(float(exact)) or abs(
                    Fraction(float(out[m, j, d])) - exact) <= abs(exact) * Fraction(1, 2 ** 24)


def test_train_objective_non_increasing(oracle_mod):
    rng = np.random.default_rng(7)
    M, dsub = 4, 4
    x = (rng.standard_normal((5000, M * dsub)) + rng.integers(0, 3, (5000, 1))).astype(np.float32)
    cb = x[rng.choice(5000, 256, replace=False)].reshape(256, M, dsub).transpose(1, 0, 2).copy()
    prev = None
    for it in range(4):
        cb, _, obj = oracle_mod.pq_train_step(x, cb, seed=1, it=it)
        if prev is not None:
            assert (obj <= prev * (1 + 1e-9)).all()
        prev = obj


def test_rejects_bad_shapes(oracle_mod):
    with pytest.raises((ValueError, AssertionError)):
        oracle_mod.pq_encode(np.zeros((3, 10), np.float32), np.zeros((3, 256, 3), np.float32))
