"""Pins for the oracle's distance and coarse search (CPU only).

Distances are checked against exact integer / rational arithmetic; routing
against exhaustive enumeration of Eq. (1) (the P-subset of centroids that
minimises the summed squared distance), against an independent exact sort,
against hand-computed golden values, and against invariants (planted
queries, translation, centroid permutation)."""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def exact_d(x, c):
    """Exact squared distance of two float32 vectors as a Fraction."""
    return sum((Fraction(float(a)) - Fraction(float(b))) ** 2 for a, b in zip(x, c))


def gamma(n, u=2.0**-53):
    return n * u / (1 - n * u)


# ---------------------------------------------------------------- distance

@pytest.mark.parametrize("D", [1, 7, 96, 128])
def test_dist_integer_data_is_exact(oracle_mod, D):
    rng = np.random.default_rng(D)
    for _ in range(50):
        x = rng.integers(0, 256, D).astype(np.float32)
        c = rng.integers(0, 256, D).astype(np.float32)
        want = sum((int(a) - int(b)) ** 2 for a, b in zip(x, c))  # Python big int
        assert oracle_mod.dist(x, c) == float(want)


@pytest.mark.parametrize("D", [2, 33, 96, 256])
def test_dist_fp32_data_within_fp64_bound(oracle_mod, D):
    rng = np.random.default_rng(100 + D)
    for scale in (1e-3, 1.0, 300.0):
        x = (rng.standard_normal(D) * scale).astype(np.float32)
        c = (rng.standard_normal(D) * scale).astype(np.float32)
        ex = exact_d(x, c)
        got = Fraction(oracle_mod.dist(x, c))
        assert abs(got - ex) <= Fraction(gamma(D + 2)) * ex


def test_dist_special_cases(oracle_mod):
    rng = np.random.default_rng(7)
    x = rng.standard_normal(64).astype(np.float32)
    assert oracle_mod.dist(x, x) == 0.0
    for _ in range(100):
        a = np.float32(rng.uniform(-1e3, 1e3))
        b = np.float32(rng.uniform(-1e3, 1e3))
        # D = 1: one exact subtraction, one rounding of the square
        assert oracle_mod.dist(np.array([a]), np.array([b])) == float((Fraction(float(a)) - Fraction(float(b))) ** 2)
    # nonnegative on arbitrary data
    for _ in range(50):
        u = rng.standard_normal(17).astype(np.float32)
        v = rng.standard_normal(17).astype(np.float32)
        assert oracle_mod.dist(u, v) >= 0.0


def test_dist_is_symmetric_and_depends_on_every_dim(oracle_mod):
    rng = np.random.default_rng(3)
    x = rng.integers(0, 256, 50).astype(np.float32)
    c = rng.integers(0, 256, 50).astype(np.float32)
    assert oracle_mod.dist(x, c) == oracle_mod.dist(c, x)
    for d in (0, 24, 49):
        y = x.copy()
        y[d] += 1
        assert oracle_mod.dist(y, c) == oracle_mod.dist(x, c) + 2 * (x[d] - c[d]) + 1


# ------------------------------------------------------------------- route

def _read_route_golden():
    cents, cases = {}, []
    with open(os.path.join(GOLDEN, "route_tiny.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("centroid"):
                _, i, x, y = line.split()
                cents[int(i)] = (float(x), float(y))
            else:
                q, k, ids, ds = line[len("query"):].split("|")
                cases.append(([float(v) for v in q.split()], int(k), [int(v) for v in ids.split()],
                              [float(v) for v in ds.split()]))
    C = np.array([cents[i] for i in range(len(cents))], np.float32)
    return C, cases


def test_route_golden(oracle_mod):
    C, cases = _read_route_golden()
    for q, k, want_ids, want_d in cases:
        ids, d = oracle_mod.route(np.array([q], np.float32), C, k)
        assert ids[0].tolist() == want_ids
        assert d[0].tolist() == want_d


def test_route_matches_exhaustive_subset_enumeration(oracle_mod):
    """Eq. (1): the returned set minimises the summed distance over all
    P-subsets, and among equal sums it is the one that the (distance, id)
    order picks (ties go to lower ids)."""
    rng = np.random.default_rng(11)
    for trial in range(40):
        C = int(rng.integers(2, 9))
        k = int(rng.integers(1, min(C, 4) + 1))
        D = 3
        # small integer range so that ties occur
        cent = rng.integers(0, 4, (C, D)).astype(np.float32)
        q = rng.integers(0, 4, (1, D)).astype(np.float32)
        dist = [exact_d(q[0], cent[j]) for j in range(C)]
        best = min(sum(dist[j] for j in s) for s in itertools.combinations(range(C), k))
        ids, dd = oracle_mod.route(q, cent, k)
        got = ids[0].tolist()
        assert sum(dist[j] for j in got) == best
        # canonical choice among optimal subsets: ascending (distance, id)
        assert got == sorted(range(C), key=lambda j: (dist[j], j))[:k]
        assert dd[0].tolist() == [float(dist[j]) for j in got]


def test_route_full_sort_when_nprobe_equals_C(oracle_mod):
    rng = np.random.default_rng(5)
    cent = rng.integers(0, 256, (40, 16)).astype(np.float32)
    qs = rng.integers(0, 256, (6, 16)).astype(np.float32)
    ids, dd = oracle_mod.route(qs, cent, 40)
    for i in range(6):
        dist = [sum((int(a) - int(b)) ** 2 for a, b in zip(qs[i], cent[j])) for j in range(40)]
        order = sorted(range(40), key=lambda j: (dist[j], j))
        assert ids[i].tolist() == order
        assert dd[i].tolist() == [float(np.float32(dist[j])) for j in order]


def test_route_planted_query_hits_its_centroid(oracle_mod):
    import synth

    d = synth.uniform_mixture_route(300, 50, 32, seed=4, plants=8)
    ids, dd = oracle_mod.route(d["queries"], d["centroids"], 5)
    for qi, ci in zip(d["plant_q"], d["plant_c"]):
        assert ids[qi, 0] == ci and dd[qi, 0] == 0.0
    assert (dd >= 0).all()
    assert (np.diff(dd, axis=1) >= 0).all()


def test_route_translation_and_permutation_invariance(oracle_mod):
    rng = np.random.default_rng(9)
    cent = rng.integers(0, 200, (64, 24)).astype(np.float32)
    qs = rng.integers(0, 200, (10, 24)).astype(np.float32)
    ids, dd = oracle_mod.route(qs, cent, 8)
    shift = rng.integers(-50, 50, 24).astype(np.float32)
    ids2, dd2 = oracle_mod.route(qs + shift, cent + shift, 8)
    assert (ids == ids2).all() and (dd == dd2).all()
    perm = rng.permutation(64)
    ids3, dd3 = oracle_mod.route(qs, cent[perm], 8)
    assert (dd3 == dd).all()
    inv = np.argsort(perm)
    # a centroid that moved keeps its distance; where distances are unique
    # the ids map through the permutation
    for i in range(10):
        for t in range(8):
            if (dd[i] == dd[i, t]).sum() == 1:
                assert perm[ids3[i, t]] == ids[i, t] and inv[ids[i, t]] == ids3[i, t]


def test_route_rejects_bad_arguments(oracle_mod):
    cent = np.zeros((4, 4), np.float32)
    q = np.zeros((2, 4), np.float32)
    with pytest.raises(ValueError):
        oracle_mod.route(q, cent, 5)
    with pytest.raises(ValueError):
        oracle_mod.route(q, cent, 0)
    ids, dd = oracle_mod.route(np.zeros((0, 4), np.float32), cent, 2)
    assert ids.shape == (0, 2)
