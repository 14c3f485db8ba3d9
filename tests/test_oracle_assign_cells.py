"""Pins for the oracle's cell-and-walk candidate assignment (CPU only).

Rows without a previous label take their first candidates from a coarse cell
of centroids and refine them by a greedy walk over a centroid graph (the
graph-assisted assignment of the full base set, Sec. "Fast Index Building
Details"). The pins:

* one cell holding every centroid is the full assignment (pinned by
  enumeration elsewhere), and no walk can leave the global nearest;
* a graph whose every row lists every centroid reaches the global nearest in
  one hop from any start;
* centroids on a line joined to their two neighbours: the walk moves one
  centroid per hop, so the label after h hops has a closed form;
* the id tie-break of the first choice and of the walk (an equally near
  neighbour with a higher id is not a move, one with a lower id is);
* invalid cells, member ids and graph entries are skipped, and offsets are
  clamped into the member array."""
import numpy as np


def test_one_cell_of_all_centroids_is_the_full_assignment(oracle_mod):
    rng = np.random.default_rng(1)
    x = rng.integers(0, 256, (400, 16)).astype(np.uint8)
    c = rng.uniform(0, 255, (23, 16)).astype(np.float32)
    members = rng.permutation(23).astype(np.uint32)
    full, fd = oracle_mod.assign(x, c, return_dist=True)
    graph = rng.integers(0, 23, (23, 5)).astype(np.int32)
    for hops in (0, 3):
        lab, d = oracle_mod.assign_cells(x, c, np.zeros(400, np.int32), [0, 23], members, graph, hops,
                                         return_dist=True)
        assert (lab == full).all() and (d == fd).all()


def test_complete_graph_reaches_the_nearest_in_one_hop(oracle_mod):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((300, 8)).astype(np.float32)
    c = rng.standard_normal((40, 8)).astype(np.float32)
    # eight cells of five centroids each; every graph row lists all 40
    members = rng.permutation(40).astype(np.uint32)
    offsets = np.arange(0, 41, 5, dtype=np.int64)
    graph = np.tile(rng.permutation(40).astype(np.int32), (40, 1))
    cell = rng.integers(0, 8, 300).astype(np.int32)
    full = oracle_mod.assign(x, c)
    assert (oracle_mod.assign_cells(x, c, cell, offsets, members, graph, 1) == full).all()
    # without hops the label is the nearest member of the row's own cell
    lab0 = oracle_mod.assign_cells(x, c, cell, offsets, members, graph, 0)
    for i in range(300):
        own = members[offsets[cell[i]]:offsets[cell[i] + 1]]
        assert lab0[i] in own
        d = ((x[i].astype(np.float64) - c[own].astype(np.float64)) ** 2).sum(1)
        assert d[list(own).index(lab0[i])] == d.min()


def test_walk_along_a_line_moves_one_centroid_per_hop(oracle_mod):
    k = 9
    c = np.zeros((k, 4), np.float32)
    c[:, 0] = np.arange(k) * 10.0
    graph = np.stack([np.arange(k) - 1, np.arange(k) + 1], 1).astype(np.int32)
    graph[graph >= k] = -1  # the ends have one neighbour
    x = np.zeros((1, 4), np.uint8)
    x[0, 0] = 83  # nearest centroid: 8 (at 80)
    for hops in range(0, 12):
        lab, d = oracle_mod.assign_cells(x, c, [0], [0, 1], [0], graph, hops, return_dist=True)
        want = min(hops, 8)
        assert lab[0] == want
        assert d[0] == (83 - 10 * want) ** 2
    # from the far end (cell holding centroid 8) the walk stays put
    assert oracle_mod.assign_cells(x, c, [0], [0, 1], [8], graph, 5)[0] == 8


def test_ties_go_to_the_lower_id(oracle_mod):
    c = np.array([[0, 0], [2, 0], [4, 0], [2, 0]], np.float32)  # 1 and 3 coincide
    x = np.array([[2, 0]], np.uint8)
    # first choice between the equal members 3 and 1: the lower id
    assert oracle_mod.assign_cells(x, c, [0], [0, 2], [3, 1], None, 0)[0] == 1
    # start at 3; its neighbour 1 is equally near with a lower id: a move
    g = np.array([[0], [3], [1], [1]], np.int32)
    assert oracle_mod.assign_cells(x, c, [0], [0, 1], [3], g, 1)[0] == 1
    # start at 1; its neighbour 3 is equally near with a higher id: no move
    assert oracle_mod.assign_cells(x, c, [0], [0, 1], [1], g, 1)[0] == 1


def test_brute_force_exact_integers(oracle_mod):
    """Small random cases against the definition with exact integer
    distances (first choice over the cell, then the greedy walk)."""
    rng = np.random.default_rng(4)
    for trial in range(40):
        N, C, D = int(rng.integers(1, 15)), int(rng.integers(1, 10)), int(rng.integers(1, 5))
        G, S, hops = int(rng.integers(1, 4)), int(rng.integers(1, 4)), int(rng.integers(0, 4))
        x = rng.integers(0, 4, (N, D)).astype(np.uint8)
        c = rng.integers(0, 4, (C, D)).astype(np.float32)
        members = rng.integers(0, C, int(rng.integers(0, 12))).astype(np.uint32)
        cuts = np.sort(rng.integers(0, members.size + 1, G - 1))
        offsets = np.concatenate([[0], cuts, [members.size]]).astype(np.int64)
        graph = rng.integers(-1, C, (C, S)).astype(np.int32)
        cell = rng.integers(0, G, N).astype(np.int32)
        lab = oracle_mod.assign_cells(x, c, cell, offsets, members, graph, hops)

        def dist(i, j):
            return sum((int(a) - int(b)) ** 2 for a, b in zip(x[i], c[j]))

        for i in range(N):
            own = [int(j) for j in members[offsets[cell[i]]:offsets[cell[i] + 1]]]
            if not own:
                assert lab[i] == -1
                continue
            b = min(own, key=lambda j: (dist(i, j), j))
            for _ in range(hops):
                nb = [int(j) for j in graph[b] if j >= 0]
                if not nb:
                    break
                n = min(nb, key=lambda j: (dist(i, j), j))
                if (dist(i, n), n) >= (dist(i, b), b):
                    break
                b = n
            assert lab[i] == b


def test_invalid_cells_members_and_offsets(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((6, 4)).astype(np.float32)
    c = rng.standard_normal((5, 4)).astype(np.float32)
    members = np.array([7, 2, 4, 99], np.uint32)  # ids 7 and 99 do not exist
    offsets = np.array([0, 2, 4, 4], np.int64)    # cell 2 is empty
    cell = np.array([0, 1, 2, -1, 3, 1], np.int32)
    lab, d = oracle_mod.assign_cells(x, c, cell, offsets, members, None, 2, return_dist=True)
    assert lab[0] == 2 and lab[1] == 4 and lab[5] == 4
    assert (lab[2:5] == -1).all() and np.isinf(d[2:5]).all()
    # offsets past the member array are clamped to it
    lab = oracle_mod.assign_cells(x, c, np.zeros(6, np.int32), [-3, 50], members, None, 0)
    full = oracle_mod.assign(x, c[[2, 4]])
    assert (lab == np.array([2, 4])[full]).all()
