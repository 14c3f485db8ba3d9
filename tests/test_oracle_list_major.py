"""Pins for the oracle's list-major layout (CPU only): the copy x[perm] and
the residuals x - c(x).

Rows: the inverse permutation restores the input; every list segment holds
exactly that list's vectors in ascending id order (checked through unique row
contents, independently of perm). Residuals: exact integer differences for
integer-valued data, correct rounding against exact rational arithmetic for
arbitrary fp32 data, zero for rows equal to their centroid."""
import math
from fractions import Fraction

import numpy as np
import pytest


def half_ulp32(v):
    """Half an fp32 ulp at |v| as an exact Fraction (v != 0, normal range)."""
    m, e = math.frexp(abs(float(v)))  # |v| = m 2^e, m in [0.5, 1)
    return Fraction(2) ** (e - 24) / 2


def test_inverse_permutation_restores_rows(oracle_mod):
    rng = np.random.default_rng(1)
    x = rng.integers(0, 256, (300, 16)).astype(np.uint8)
    c = rng.uniform(0, 255, (7, 16)).astype(np.float32)
    lab = rng.integers(0, 7, 300).astype(np.int32)
    perm = rng.permutation(300).astype(np.uint32)
    rows, _ = oracle_mod.list_major(x, c, lab, perm, residuals=False)
    back = np.empty_like(rows)
    back[perm] = rows
    assert (back == x).all()


def test_segments_hold_their_list_in_id_order(oracle_mod):
    rng = np.random.default_rng(2)
    N, C, D = 500, 9, 8
    # unique rows: the row id is encoded in the first two bytes
    x = rng.integers(0, 256, (N, D)).astype(np.uint8)
    x[:, 0] = np.arange(N) % 256
    x[:, 1] = np.arange(N) // 256
    lab = rng.integers(0, C, N).astype(np.int32)
    c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    counts, offsets, perm = oracle_mod.build_lists(lab, C)
    rows, _ = oracle_mod.list_major(x, c, lab, perm, residuals=False)
    ids = rows[:, 0].astype(np.int64) + 256 * rows[:, 1].astype(np.int64)
    for j in range(C):
        seg = ids[offsets[j]:offsets[j + 1]]
        assert sorted(seg.tolist()) == seg.tolist()
        assert set(seg.tolist()) == {i for i in range(N) if lab[i] == j}


def test_residuals_exact_on_integer_data(oracle_mod):
    rng = np.random.default_rng(3)
    x = rng.integers(0, 256, (200, 12)).astype(np.uint8)
    c = rng.integers(-300, 300, (5, 12)).astype(np.float32)
    lab = rng.integers(0, 5, 200).astype(np.int32)
    perm = rng.permutation(200).astype(np.uint32)
    _, res = oracle_mod.list_major(x, c, lab, perm, rows=False)
    for i, r in enumerate(perm):
        want = [int(x[r, d]) - int(c[lab[r], d]) for d in range(12)]
        assert res[i].tolist() == want


def test_residuals_correctly_rounded(oracle_mod):
    rng = np.random.default_rng(4)
    x = (rng.standard_normal((60, 8)) * 10.0 ** rng.integers(-3, 4, (60, 1))).astype(np.float32)
    c = (rng.standard_normal((4, 8)) * 10.0 ** rng.integers(-3, 4, (4, 1))).astype(np.float32)
    lab = rng.integers(0, 4, 60).astype(np.int32)
    perm = np.arange(60, dtype=np.uint32)[::-1].copy()
    rows, res = oracle_mod.list_major(x, c, lab, perm)
    assert (rows == x[::-1]).all()
    for i, r in enumerate(perm):
        for d in range(8):
            exact = Fraction(float(x[r, d])) - Fraction(float(c[lab[r], d]))
            got = Fraction(float(res[i, d]))
            if exact == 0:
                assert got == 0
            else:
                assert abs(got - exact) <= half_ulp32(res[i, d])


def test_rows_at_their_centroid_have_zero_residual(oracle_mod):
    rng = np.random.default_rng(5)
    c = rng.uniform(-5, 5, (6, 10)).astype(np.float32)
    lab = np.array([3, 0, 5, 5, 1], np.int32)
    x = c[lab].copy()
    _, res = oracle_mod.list_major(x, c, lab, np.arange(5, dtype=np.uint32), rows=False)
    assert (res == 0).all()


def test_slices_of_the_permutation(oracle_mod):
    rng = np.random.default_rng(6)
    x = rng.integers(0, 256, (100, 4)).astype(np.uint8)
    c = rng.uniform(0, 255, (3, 4)).astype(np.float32)
    lab = rng.integers(0, 3, 100).astype(np.int32)
    perm = rng.permutation(100).astype(np.uint32)
    full_rows, full_res = oracle_mod.list_major(x, c, lab, perm)
    part_rows, part_res = oracle_mod.list_major(x, c, lab, perm[30:71])
    assert (part_rows == full_rows[30:71]).all() and (part_res == full_res[30:71]).all()
    empty_rows, empty_res = oracle_mod.list_major(x, c, lab, perm[:0])
    assert empty_rows.shape == (0, 4) and empty_res.shape == (0, 4)


def test_rejects_bad_ids_and_labels(oracle_mod):
    x = np.zeros((4, 4), np.uint8)
    c = np.zeros((2, 4), np.float32)
    with pytest.raises(ValueError):
        oracle_mod.list_major(x, c, [0, 1, 0, 1], np.array([0, 4], np.uint32))
    with pytest.raises(ValueError):
        oracle_mod.list_major(x, c, [0, 2, 0, 1], np.array([1], np.uint32))
