"""GPU parity of ivf_assign_graph (candidate-restricted assignment) against
the oracle: labels bit-identical and distances equal to the oracle's fp64
distance rounded to fp32, for every candidate degree 1 ... 64, duplicate and
invalid candidates, ties, and a full-size fast k-means iteration whose
candidates come from the centroids' nearest-centroid graph (ivf_route)."""
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


def run(ctx, x, c, graph, prev, order=None):
    import torch

    import paper_2608_08751_amd as ivf

    lab, dist = ivf.ivf_assign_graph(ctx, to_dev(x), to_dev(c), to_dev(graph), to_dev(prev),
                                     order=None if order is None else to_dev(order.astype(np.int32)))
    torch.cuda.synchronize()
    return lab.cpu().numpy(), dist.cpu().numpy()


@pytest.mark.parametrize("N,C,D,S,dt", [
    (1, 1, 4, 1, "u8"), (1000, 50, 16, 3, "u8"), (5000, 300, 128, 8, "u8"), (4097, 200, 96, 8, "f32"),
    (3000, 100, 256, 64, "f32"), (2000, 70, 36, 17, "u8"), (777, 1000, 128, 2, "f32"),
])
def test_assign_graph_exact(ivf_ctx, oracle_mod, N, C, D, S, dt):
    rng = np.random.default_rng(N + C + S)
    if dt == "u8":
        x = rng.integers(0, 256, (N, D)).astype(np.uint8)
        c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    else:
        x = rng.standard_normal((N, D)).astype(np.float32)
        c = rng.standard_normal((C, D)).astype(np.float32)
    graph = rng.integers(0, C, (C, S)).astype(np.int32)
    prev = rng.integers(0, C, N).astype(np.int32)
    olab, od = oracle_mod.assign_graph(x, c, graph, prev, return_dist=True)
    # any processing order gives the same result
    for order in (None, rng.permutation(N), np.argsort(prev, kind="stable")):
        lab, dist = run(ivf_ctx, x, c, graph, prev, order)
        assert (lab == olab).all()
        assert (dist == od.astype(np.float32)).all()


def test_assign_graph_ties_duplicates_and_invalid(ivf_ctx, oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.integers(0, 3, (3000, 8)).astype(np.uint8)
    c = rng.integers(0, 3, (40, 8)).astype(np.float32)  # many exact ties
    graph = rng.integers(-3, 45, (40, 12)).astype(np.int32)  # invalid ids and duplicates
    prev = rng.integers(-2, 42, 3000).astype(np.int32)  # some rows without candidates
    lab, dist = run(ivf_ctx, x, c, graph, prev)
    olab, od = oracle_mod.assign_graph(x, c, graph, prev, return_dist=True)
    assert (lab == olab).all()
    assert (dist == od.astype(np.float32)).all()
    assert (lab == -1).any() and np.isinf(dist[lab == -1]).all()


def test_fast_kmeans_iteration_full_size(ivf_ctx, oracle_mod):
    """10M uint8 rows: labels against the initial centroids from the exact
    k-means step, new centroids, their 8-nearest-centroid graph from
    ivf_route, then the candidate-restricted assignment. Sampled rows match
    the oracle; every row is at least as near as its previous centroid and
    no nearer than the exact assignment (the fast mode is approximate by
    design; the agreement rate is printed)."""
    import torch

    import paper_2608_08751_amd as ivf

    N, C, D, S = 10_000_000, 65536, 128, 8
    means = synth.uniform_means(C, D, seed=0)
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(to_dev(means), 0, N, x, seed=0)
    c0 = x[to_dev(synth.kmeans_init(N, C, seed=0))].float().contiguous()
    lab0, c1, _, _ = ivf.ivf_kmeans_step(ivf_ctx, x, c0, seed=0, it=0)
    graph, _ = ivf.ivf_route(ivf_ctx, c1, c1, S)
    _, _, by_prev = ivf.ivf_build_lists(ivf_ctx, lab0, C)
    lab, dist = ivf.ivf_assign_graph(ivf_ctx, x, c1, graph, lab0, order=by_prev)
    exact, _, _, _ = ivf.ivf_kmeans_step(ivf_ctx, x, c1, seed=0, it=1)
    torch.cuda.synchronize()
    rng = np.random.default_rng(9)
    rows = np.sort(rng.choice(N, 4096, replace=False))
    xs = x[to_dev(rows)].cpu().numpy()
    gh = graph.cpu().numpy()
    olab, od = oracle_mod.assign_graph(xs, c1.cpu().numpy(), gh, lab0.cpu().numpy()[rows], return_dist=True)
    assert (lab.cpu().numpy()[rows] == olab).all()
    assert (dist.cpu().numpy()[rows] == od.astype(np.float32)).all()
    # every row's previous centroid is among its candidates, and the exact
    # nearest is at least as near: d(exact) <= d(candidates) <= d(previous)
    def d_to(labels):
        out = torch.empty(N, dtype=torch.float64, device="cuda")
        for r0 in range(0, N, 1 << 20):
            xs_ = x[r0:r0 + (1 << 20)].double()
            out[r0:r0 + (1 << 20)] = ((xs_ - c1[labels[r0:r0 + (1 << 20)].long()].double()) ** 2).sum(1)
        return out
    dg = dist.double()
    assert bool((dg <= d_to(lab0) * (1 + 1e-6)).all())
    assert bool((dg >= d_to(exact) * (1 - 1e-6)).all())
    agree = float((lab == exact).float().mean())
    print("candidate-restricted labels equal to the exact assignment: %.5f" % agree)
    assert agree > 0.5
