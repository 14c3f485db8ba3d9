"""Pins for the oracle's k-means step and inverted-list build (CPU only).

Assignment: exhaustive enumeration of labelings. Update: numpy per-cluster
means, exact rational means, closed forms (C = 1, fixed points). Reseed:
published SplitMix64 outputs and invariants. Objective: Lloyd's monotone
decrease. Build: numpy bincount / cumsum / stable argsort, golden values and
exhaustive enumeration of permutations."""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def exact_d(x, c):
    return sum((Fraction(float(a)) - Fraction(float(b))) ** 2 for a, b in zip(x, c))


# -------------------------------------------------------------- assignment

def test_assign_minimises_objective_over_all_labelings(oracle_mod):
    rng = np.random.default_rng(21)
    for trial in range(30):
        N = int(rng.integers(1, 7))
        C = int(rng.integers(1, 4))
        x = rng.integers(0, 5, (N, 3)).astype(np.uint8)
        c = rng.integers(0, 5, (C, 3)).astype(np.float32)
        dist = [[exact_d(x[i], c[j]) for j in range(C)] for i in range(N)]
        best = min(sum(dist[i][l[i]] for i in range(N)) for l in itertools.product(range(C), repeat=N))
        lab = oracle_mod.assign(x, c)
        assert sum(dist[i][lab[i]] for i in range(N)) == best
        for i in range(N):  # ties go to the lower id
            assert all(dist[i][j] > dist[i][lab[i]] for j in range(lab[i]))


def test_assign_u8_and_f32_agree_and_return_min_distance(oracle_mod):
    rng = np.random.default_rng(2)
    x = rng.integers(0, 256, (200, 16)).astype(np.uint8)
    c = rng.uniform(0, 255, (30, 16)).astype(np.float32)
    l1, d1 = oracle_mod.assign(x, c, return_dist=True)
    l2 = oracle_mod.assign(x.astype(np.float32), c)
    assert (l1 == l2).all()
    for i in range(0, 200, 37):
        assert d1[i] == oracle_mod.dist(x[i].astype(np.float32), c[l1[i]])


# ------------------------------------------------------------------ update

def test_update_equals_numpy_means_for_u8(oracle_mod):
    rng = np.random.default_rng(4)
    N, C, D = 3000, 40, 24
    x = rng.integers(0, 256, (N, D)).astype(np.uint8)
    lab = rng.integers(0, C, N).astype(np.int32)
    lab[lab == 7] = 8  # cluster 7 empty -> reseeded
    cent, cnt = oracle_mod.kmeans_update(x, lab, C, seed=5, it=3)
    assert (cnt == np.bincount(lab, minlength=C)).all()
    for j in range(C):
        if cnt[j] == 0:
            continue
        want = x[lab == j].astype(np.float64).mean(axis=0).astype(np.float32)
        assert (cent[j] == want).all()
        # and within one fp32 ulp of the exact rational mean
        for d in (0, D - 1):
            ex = Fraction(int(x[lab == j, d].astype(np.int64).sum()), int(cnt[j]))
            assert abs(Fraction(float(cent[j, d])) - ex) <= Fraction(abs(float(np.spacing(np.float32(ex)))))
    r = oracle_mod.reseed_row(5, 3, 7, N)
    assert (cent[7] == x[r].astype(np.float32)).all()


def test_update_f32_is_ordered_fp64_sum(oracle_mod):
    rng = np.random.default_rng(8)
    N, C, D = 500, 5, 6
    x = (rng.standard_normal((N, D)) * 1e3).astype(np.float32)
    lab = rng.integers(0, C, N).astype(np.int32)
    cent, cnt = oracle_mod.kmeans_update(x, lab, C)
    for j in range(C):
        rows = x[lab == j].astype(np.float64)
        s = np.zeros(D)
        for r in rows:  # left-to-right fp64 sum in ascending row order
            s = s + r
        assert (cent[j] == (s / cnt[j]).astype(np.float32)).all()
        ex = [sum(Fraction(float(v)) for v in x[lab == j, d]) / int(cnt[j]) for d in range(D)]
        for d in range(D):
            assert abs(float(cent[j, d]) - float(ex[d])) <= 4 * abs(float(np.spacing(np.float32(ex[d]))))


def test_update_single_cluster_is_global_mean(oracle_mod):
    rng = np.random.default_rng(1)
    x = rng.integers(0, 256, (777, 12)).astype(np.uint8)
    c0 = x[:1].astype(np.float32)
    lab, cent, cnt, J = oracle_mod.kmeans_step(x, c0)
    assert (lab == 0).all() and cnt[0] == 777
    assert (cent[0] == x.astype(np.float64).mean(axis=0).astype(np.float32)).all()


def test_well_separated_exact_means_are_a_fixed_point(oracle_mod):
    # Each cluster: its integer mean m plus symmetric offsets +-e, so the exact
    # mean is m; clusters are far apart so every row keeps its label.
    rng = np.random.default_rng(6)
    C, D = 6, 8
    means = (np.arange(C)[:, None] * 40 + 20 + np.zeros((C, D))).astype(np.float32)
    rows = []
    for j in range(C):
        for _ in range(5):
            e = rng.integers(-3, 4, D)
            rows += [means[j] + e, means[j] - e]
    x = np.array(rows).astype(np.uint8)
    lab, cent, cnt, J = oracle_mod.kmeans_step(x, means)
    assert (lab == np.repeat(np.arange(C), 10)).all()
    assert (cent == means).all()
    lab2, cent2, _, J2 = oracle_mod.kmeans_step(x, cent)
    assert (cent2 == cent).all() and J2 == J


# ------------------------------------------------------------------ reseed

def test_splitmix64_published_outputs(oracle_mod):
    with open(os.path.join(GOLDEN, "splitmix64.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert len(rows) == 8
    for seed, n, out in rows:
        assert oracle_mod.splitmix64_nth(int(seed), int(n)) == int(out, 0)


def test_reseed_is_deterministic_and_picks_training_rows(oracle_mod):
    N = 1000
    r = [oracle_mod.reseed_row(42, 3, j, N) for j in range(200)]
    assert r == [oracle_mod.reseed_row(42, 3, j, N) for j in range(200)]
    assert all(0 <= v < N for v in r)
    assert r != [oracle_mod.reseed_row(42, 4, j, N) for j in range(200)]
    assert r != [oracle_mod.reseed_row(43, 3, j, N) for j in range(200)]
    # definition: output ((iter << 32) | j) + 1 of SplitMix64 seeded with seed, mod N
    for j in (0, 5, 199):
        assert r[j] == oracle_mod.splitmix64_nth(42, (3 << 32 | j) + 1) % N


def test_empty_cluster_takes_reseed_row(oracle_mod):
    rng = np.random.default_rng(12)
    x = rng.integers(0, 50, (100, 4)).astype(np.uint8)
    c = np.vstack([x[:3].astype(np.float32), np.full((2, 4), 1e4, np.float32)])  # 3,4 far away
    lab, cent, cnt, J = oracle_mod.kmeans_step(x, c, seed=9, it=2)
    assert cnt[3] == 0 and cnt[4] == 0
    for j in (3, 4):
        assert (cent[j] == x[oracle_mod.reseed_row(9, 2, j, 100)]).all()


# --------------------------------------------------------------- objective

def test_objective_is_sum_of_assigned_distances(oracle_mod):
    rng = np.random.default_rng(13)
    x = rng.integers(0, 256, (300, 10)).astype(np.uint8)
    c = x[rng.choice(300, 12, replace=False)].astype(np.float32)
    lab, cent, cnt, J = oracle_mod.kmeans_step(x, c)
    want = sum(int(((x[i].astype(np.int64) - c[lab[i]].astype(np.int64)) ** 2).sum()) for i in range(300))
    assert J == float(want)


def test_objective_non_increasing_over_lloyd_iterations(oracle_mod):
    import synth

    means = synth.uniform_means(64, 16, seed=3)
    x, _ = synth.mixture_rows_u8(means, 0, 4000, seed=3)
    c = x[synth.kmeans_init(4000, 48, seed=3)].astype(np.float32)
    Js = []
    for it in range(8):
        lab, c, cnt, J = oracle_mod.kmeans_step(x, c, seed=3, it=it)
        Js.append(J)
    for a, b in zip(Js, Js[1:]):
        assert b <= a * (1 + 1e-9)
    assert Js[-1] < Js[0]


# ------------------------------------------------------------------- build

def test_build_golden(oracle_mod):
    vals = {}
    with open(os.path.join(GOLDEN, "build_tiny.txt")) as f:
        for l in f:
            if l.strip() and not l.startswith("#"):
                k, *v = l.split()
                vals[k] = [int(t) for t in v]
    counts, offsets, perm = oracle_mod.build_lists(np.array(vals["labels"]), 4)
    assert counts.tolist() == vals["counts"]
    assert offsets.tolist() == vals["offsets"]
    assert perm.tolist() == vals["perm"]


@pytest.mark.parametrize("skew", [0.0, 1.1])
def test_build_matches_numpy(oracle_mod, skew):
    import synth

    for N, C in ((1, 1), (5000, 1), (10000, 300), (20000, 5000)):
        lab = synth.random_labels(N, C, seed=N + C, skew=skew)
        counts, offsets, perm = oracle_mod.build_lists(lab, C)
        assert (counts == np.bincount(lab, minlength=C)).all()
        assert offsets[0] == 0 and (offsets[1:] == np.cumsum(counts)).all() and offsets[-1] == N
        assert (perm == np.argsort(lab, kind="stable")).all()


def test_build_unique_valid_permutation_by_enumeration(oracle_mod):
    rng = np.random.default_rng(17)
    for trial in range(20):
        N = int(rng.integers(1, 7))
        C = int(rng.integers(1, 4))
        lab = rng.integers(0, C, N).astype(np.int32)
        valid = [p for p in itertools.permutations(range(N))
                 if all((lab[p[a]], p[a]) < (lab[p[a + 1]], p[a + 1]) for a in range(N - 1))]
        assert len(valid) == 1
        counts, offsets, perm = oracle_mod.build_lists(lab, C)
        assert tuple(perm.tolist()) == valid[0]
        for j in range(C):  # list j holds exactly its ids, ascending
            seg = perm[offsets[j]:offsets[j + 1]]
            assert (lab[seg] == j).all() and (np.diff(seg.astype(np.int64)) > 0).all()


def test_build_edge_cases(oracle_mod):
    counts, offsets, perm = oracle_mod.build_lists(np.zeros(0, np.int32), 3)
    assert counts.tolist() == [0, 0, 0] and offsets.tolist() == [0, 0, 0, 0] and perm.size == 0
    with pytest.raises(ValueError):
        oracle_mod.build_lists(np.array([0, 3]), 3)
    with pytest.raises(ValueError):
        oracle_mod.build_lists(np.array([-1]), 3)


def test_update_f32_order_golden(oracle_mod):
    """fp32 rows: the cluster sums are fp64 sums in ascending row order. The
    golden rows make that order and that precision visible: a reversed or
    exact sum, fp32 or extended-precision accumulation each change a mean."""
    rows, labels, want = [], [], {}
    for line in open(os.path.join(GOLDEN, "kmeans_update_f32_order.txt")):
        f = line.split("#")[0].split()
        if not f:
            continue
        if f[0] == "row":
            v = int(f[1])
            assert float(np.float32(v)) == v  # every row value is an fp32 number
            rows.append(v)
            labels.append(int(f[2]))
        elif f[0] == "centroid":
            want[int(f[1])] = float(f[2])
    x = np.array(rows, np.float32).reshape(-1, 1)
    lab = np.array(labels, np.int32)
    cent, cnt = oracle_mod.kmeans_update(x, lab, 4)
    assert (cnt == np.bincount(lab, minlength=4)).all()
    for j in range(4):
        assert float(cent[j, 0]) == want[j], (j, float(cent[j, 0]), want[j])

    # the reading, worked out in exact arithmetic with one fp64 rounding per
    # addition (float(Fraction) is correctly rounded), gives the golden means;
    # the other readings give different ones in the clusters built for them
    def mean(vals, acc="f64", order=1):
        s = Fraction(0)
        for v in vals[::order]:
            if acc == "f64":
                s = Fraction(float(s + v))
            elif acc == "f32":
                s = Fraction(float(np.float32(float(s + v))))
            else:
                s = s + v
        return float(np.float32(float(Fraction(float(s)) / len(vals))))

    members = {j: [Fraction(v) for v, l in zip(rows, labels) if l == j] for j in range(4)}
    for j in range(4):
        assert mean(members[j]) == want[j]
    assert mean(members[0], order=-1) != want[0] and mean(members[0], acc="exact") != want[0]
    assert mean(members[1], order=-1) != want[1] and mean(members[1], acc="exact") != want[1]
    assert mean(members[2], acc="f32") != want[2]
