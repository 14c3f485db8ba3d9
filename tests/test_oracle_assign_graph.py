"""Pins for the oracle's candidate-restricted assignment (CPU only).

When every centroid is a candidate it is the full assignment (itself pinned by
enumeration); on tiny inputs it matches brute force over the candidates with
exact integer distances and the id tie-break; the label is always a
candidate; invalid candidate ids are skipped."""
import numpy as np


def test_all_candidates_is_the_full_assignment(oracle_mod):
    rng = np.random.default_rng(1)
    x = rng.integers(0, 256, (500, 16)).astype(np.uint8)
    c = rng.uniform(0, 255, (12, 16)).astype(np.float32)
    graph = np.tile(np.arange(12, dtype=np.int32)[::-1], (12, 1))  # every centroid, reversed
    prev = rng.integers(0, 12, 500).astype(np.int32)
    lab, d = oracle_mod.assign_graph(x, c, graph, prev, return_dist=True)
    full, fd = oracle_mod.assign(x, c, return_dist=True)
    assert (lab == full).all() and (d == fd).all()


def test_brute_force_exact_integers(oracle_mod):
    rng = np.random.default_rng(2)
    for trial in range(30):
        N, C, D, S = int(rng.integers(1, 20)), int(rng.integers(1, 9)), int(rng.integers(1, 5)), int(rng.integers(1, 5))
        x = rng.integers(0, 4, (N, D)).astype(np.uint8)
        c = rng.integers(0, 4, (C, D)).astype(np.float32)
        graph = rng.integers(0, C, (C, S)).astype(np.int32)
        prev = rng.integers(0, C, N).astype(np.int32)
        lab = oracle_mod.assign_graph(x, c, graph, prev)
        for i in range(N):
            cands = set(int(j) for j in graph[prev[i]])
            d = {j: sum((int(a) - int(b)) ** 2 for a, b in zip(x[i], c[j])) for j in cands}
            assert lab[i] == min(cands, key=lambda j: (d[j], j))


def test_label_is_a_candidate_and_bad_ids_are_skipped(oracle_mod):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((300, 8)).astype(np.float32)
    c = rng.standard_normal((20, 8)).astype(np.float32)
    graph = rng.integers(0, 20, (20, 4)).astype(np.int32)
    graph[:, 0] = -1
    graph[3, :] = [-5, 20, 99, 7]
    prev = rng.integers(0, 20, 300).astype(np.int32)
    prev[:5] = 3
    prev[5] = 25  # no candidates at all
    lab, d = oracle_mod.assign_graph(x, c, graph, prev, return_dist=True)
    assert (lab[:5] == 7).all()
    assert lab[5] == -1 and np.isinf(d[5])
    for i in range(6, 300):
        assert lab[i] in set(graph[prev[i]].tolist())
