"""GPU parity of ivf_assign_cells (candidates for rows without a previous
label: the nearest member of the row's coarse cell, then a greedy walk over a
centroid graph) against the oracle: labels bit-identical and distances equal
to the oracle's fp64 distance rounded to fp32, on ragged shapes, empty cells,
invalid members and graph entries, ties, hop limits 0 ... 64, and a
full-size assignment of 10M base rows to 65,536 centroids whose cells come
from a coarse table of 1,024 centroids (trained with ivf_kmeans_step on the
centroids) and whose graph comes from ivf_route."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ivf_ctx():
    import torch

    import paper_2608_08751_amd as ivf

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ctx = ivf.Context(0)
    yield ctx
    ctx.close()


def to_dev(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run(ctx, x, c, cell, offsets, members, graph, hops, order=None):
    import torch

    import paper_2608_08751_amd as ivf

    lab, dist = ivf.ivf_assign_cells(ctx, to_dev(x), to_dev(c), to_dev(cell.astype(np.int32)),
                                     to_dev(offsets.astype(np.int64)), to_dev(members.view(np.int32)),
                                     None if graph is None else to_dev(graph.astype(np.int32)), hops,
                                     order=None if order is None else to_dev(order.astype(np.int32)))
    torch.cuda.synchronize()
    return lab.cpu().numpy(), dist.cpu().numpy()


def random_cells(rng, C, G, extra_invalid=0):
    members = rng.permutation(C).astype(np.uint32)
    if extra_invalid:
        members = np.concatenate([members, rng.integers(C, C + 50, extra_invalid).astype(np.uint32)])
        members = members[rng.permutation(members.size)]
    cuts = np.sort(rng.integers(0, members.size + 1, G - 1))
    offsets = np.concatenate([[0], cuts, [members.size]]).astype(np.int64)
    return offsets, members


@pytest.mark.parametrize("N,C,D,G,S,hops,dt", [
    (1, 1, 4, 1, 1, 0, "u8"), (1000, 50, 16, 7, 3, 2, "u8"), (5000, 300, 128, 20, 8, 4, "u8"),
    (4097, 200, 96, 16, 8, 8, "f32"), (3000, 100, 256, 3, 64, 64, "f32"), (2000, 700, 36, 5, 17, 3, "u8"),
    (777, 1000, 128, 40, 2, 1, "f32"), (1500, 90, 128, 9, 8, 0, "u8"),
])
def test_assign_cells_exact(ivf_ctx, oracle_mod, N, C, D, G, S, hops, dt):
    rng = np.random.default_rng(N + C + G + hops)
    if dt == "u8":
        x = rng.integers(0, 256, (N, D)).astype(np.uint8)
        c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    else:
        x = rng.standard_normal((N, D)).astype(np.float32)
        c = rng.standard_normal((C, D)).astype(np.float32)
    offsets, members = random_cells(rng, C, G)
    graph = rng.integers(0, C, (C, S)).astype(np.int32)
    cell = rng.integers(0, G, N).astype(np.int32)
    olab, od = oracle_mod.assign_cells(x, c, cell, offsets, members, graph, hops, return_dist=True)
    # any processing order gives the same result: row order, a random
    # permutation, and rows grouped by cell
    for order in (None, rng.permutation(N), np.argsort(cell, kind="stable")):
        lab, dist = run(ivf_ctx, x, c, cell, offsets, members, graph, hops, order)
        assert (lab == olab).all()
        assert (dist == od.astype(np.float32)).all()


def test_assign_cells_order_skips_and_leaves_rows(ivf_ctx, oracle_mod):
    """Order entries past N are skipped; rows the order does not list keep
    the output buffer's contents."""
    import torch

    import paper_2608_08751_amd as ivf

    rng = np.random.default_rng(6)
    N, C, D, G = 500, 40, 32, 5
    x = rng.integers(0, 256, (N, D)).astype(np.uint8)
    c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    offsets, members = random_cells(rng, C, G)
    cell = rng.integers(0, G, N).astype(np.int32)
    order = rng.permutation(N).astype(np.int64)
    order[:7] = N + np.arange(7)  # not rows
    left = np.setdiff1d(np.arange(N), order)
    lab = torch.full((N,), -77, dtype=torch.int32, device="cuda")
    dist = torch.full((N,), 5.0, dtype=torch.float32, device="cuda")
    ivf.ivf_assign_cells(ivf_ctx, to_dev(x), to_dev(c), to_dev(cell), to_dev(offsets), to_dev(members.view(np.int32)),
                         None, 0, order=to_dev(order.astype(np.uint32).view(np.int32)), out_labels=lab,
                         out_dist=dist)
    torch.cuda.synchronize()
    olab, od = oracle_mod.assign_cells(x, c, cell, offsets, members, None, 0, return_dist=True)
    lab, dist = lab.cpu().numpy(), dist.cpu().numpy()
    done = np.setdiff1d(np.arange(N), left)
    assert (lab[done] == olab[done]).all() and (dist[done] == od[done].astype(np.float32)).all()
    assert (lab[left] == -77).all() and (dist[left] == 5.0).all()


def test_assign_cells_ties_invalid_and_no_graph(ivf_ctx, oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.integers(0, 3, (3000, 8)).astype(np.uint8)
    c = rng.integers(0, 3, (40, 8)).astype(np.float32)  # many exact ties
    offsets, members = random_cells(rng, 40, 6, extra_invalid=15)
    offsets[3] = offsets[2]  # an empty cell
    graph = rng.integers(-3, 45, (40, 12)).astype(np.int32)  # invalid ids and duplicates
    cell = rng.integers(-2, 8, 3000).astype(np.int32)  # some cells outside [0, G)
    for g, hops in ((graph, 5), (None, 3)):
        lab, dist = run(ivf_ctx, x, c, cell, offsets, members, g, hops)
        olab, od = oracle_mod.assign_cells(x, c, cell, offsets, members, g, hops, return_dist=True)
        assert (lab == olab).all()
        assert (dist == od.astype(np.float32)).all()
        assert (lab == -1).any() and np.isinf(dist[lab == -1]).all()


def test_assign_cells_long_walk(ivf_ctx, oracle_mod):
    """Centroids on a line joined to their neighbours: a start at one end
    walks one centroid per hop, for up to 300 hops."""
    k = 400
    c = np.zeros((k, 4), np.float32)
    c[:, 0] = np.arange(k) * 0.5
    graph = np.stack([np.arange(k) - 1, np.arange(k) + 1], 1).astype(np.int32)
    graph[graph >= k] = -1
    x = np.zeros((64, 4), np.float32)
    x[:, 0] = np.linspace(0, 250, 64)
    for hops in (0, 1, 37, 300):
        lab, dist = run(ivf_ctx, x, c, np.zeros(64, np.int32), np.array([0, 1]), np.array([0], np.uint32),
                        graph, hops)
        olab, od = oracle_mod.assign_cells(x, c, np.zeros(64, np.int32), [0, 1], [0], graph, hops,
                                           return_dist=True)
        assert (lab == olab).all() and (dist == od.astype(np.float32)).all()
        assert lab.max() == min(hops, 399)


def test_assign_cells_base_full_size(ivf_ctx, oracle_mod):
    """10M base rows of the assign-build generator, 65,536 centroids (the
    mixture means), no previous labels. Coarse table: 1,024 centroids from
    three Lloyd steps over the centroid table; cells of the centroids and of
    the rows from ivf_assign_build against it; graph: each centroid's 8
    nearest (ivf_route). Sampled rows match the oracle; every label is at
    least as near as the row's first choice and no nearer than the exact
    nearest; the agreement with the exact assignment is printed."""
    import torch

    import paper_2608_08751_amd as ivf

    N, C, D, G, S, hops = 10_000_000, 65536, 128, 1024, 8, 8
    means = synth.uniform_means(C, D, seed=0)
    cent = to_dev(means)
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(cent, 0, N, x, seed=0)
    coarse = cent[to_dev(synth.kmeans_init(C, G, seed=1))].contiguous()
    for it in range(3):
        _, coarse, _, _ = ivf.ivf_kmeans_step(ivf_ctx, cent, coarse, seed=1, it=it)
    _, _, c_off, c_mem = ivf.ivf_assign_build(ivf_ctx, cent, coarse)
    cell, _, _, by_cell = ivf.ivf_assign_build(ivf_ctx, x, coarse)
    graph, _ = ivf.ivf_route(ivf_ctx, cent, cent, S)
    lab, dist = ivf.ivf_assign_cells(ivf_ctx, x, cent, cell, c_off, c_mem, graph, hops, order=by_cell)
    first, fdist = ivf.ivf_assign_cells(ivf_ctx, x, cent, cell, c_off, c_mem, None, 0, order=by_cell)
    exact, _, _, _ = ivf.ivf_assign_build(ivf_ctx, x, cent)
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    rows = np.sort(rng.choice(N, 8192, replace=False))
    xs = x[to_dev(rows)].cpu().numpy()
    olab, od = oracle_mod.assign_cells(xs, means, cell.cpu().numpy()[rows], c_off.cpu().numpy(),
                                       c_mem.cpu().numpy().view(np.uint32), graph.cpu().numpy(), hops,
                                       return_dist=True)
    assert (lab.cpu().numpy()[rows] == olab).all()
    assert (dist.cpu().numpy()[rows] == od.astype(np.float32)).all()
    assert bool((lab >= 0).all())
    assert bool((dist <= fdist).all())
    ex = exact.long()
    dex = torch.empty(N, dtype=torch.float64, device="cuda")
    for r0 in range(0, N, 1 << 20):
        r1 = min(N, r0 + (1 << 20))
        dex[r0:r1] = ((x[r0:r1].double() - cent[ex[r0:r1]].double()) ** 2).sum(1)
    assert bool((dist.double() >= dex.float().double() * (1 - 1e-6)).all())
    agree = float((lab == exact).float().mean())
    agree0 = float((first == exact).float().mean())
    print("cell-and-walk labels equal to the exact assignment: %.5f (first choice alone %.5f)" % (agree, agree0))
    assert agree > 0.5
