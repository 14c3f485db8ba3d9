"""GPU parity of ivf_route against the oracle (ids and fp32 distances must be
identical), over the routing workloads, several tiles with ragged tails,
padded dimensions, ties, forced fallbacks and the full-size workloads on
sampled queries."""
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


def run_route(ctx, q, c, k):
    import torch

    import paper_2608_08751_amd as ivf

    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    cd = torch.from_numpy(np.ascontiguousarray(c)).cuda()
    ids, dist = ivf.ivf_route(ctx, qd, cd, k)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), dist.cpu().numpy(), ctx.last_stats()


def assert_route_equal(ctx, oracle_mod, q, c, k):
    ids, dist, stats = run_route(ctx, q, c, k)
    oids, odist = oracle_mod.route(q, c, k)
    bad = np.nonzero((ids != oids).any(axis=1) | (dist != odist).any(axis=1))[0]
    assert bad.size == 0, "rows %s differ (first: gpu %s / %s, oracle %s / %s)" % (
        bad[:5], ids[bad[0]][:8], dist[bad[0]][:8], oids[bad[0]][:8], odist[bad[0]][:8])
    return stats


def test_route_tiny_workload_exact(ivf_ctx, oracle_mod):
    """1,024 centroids, 1,000 integer-valued queries, nprobe 16 (every query)."""
    d = synth.uniform_mixture_route(1024, 1000, 128, seed=0)
    stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], 16)
    ids, dist, _ = run_route(ivf_ctx, d["queries"], d["centroids"], 16)
    for qi, ci in zip(d["plant_q"], d["plant_c"]):
        assert ids[qi, 0] == ci and dist[qi, 0] == 0.0
    assert (dist >= 0).all()
    assert stats["fallback"] == 0


@pytest.mark.parametrize("C,Q,D,k", [(8192, 600, 128, 64), (6000, 333, 128, 16), (4097, 257, 128, 100)])
def test_route_uint8_valued(ivf_ctx, oracle_mod, C, Q, D, k):
    d = synth.uniform_mixture_route(C, Q, D, seed=C)
    stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], k)
    assert stats["sample"] > 0
    assert stats["fallback"] <= max(2, Q // 50)


@pytest.mark.parametrize("C,Q,D,k", [(12288, 500, 96, 128), (3000, 260, 96, 8)])
def test_route_normalised(ivf_ctx, oracle_mod, C, Q, D, k):
    d = synth.normalised_route(C, Q, D, seed=C)
    stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], k)
    assert stats["fallback"] <= max(2, Q // 50)


@pytest.mark.parametrize("C,Q,D,k", [
    (1, 5, 4, 1), (7, 33, 12, 7), (65, 257, 36, 10), (3001, 300, 100, 32),
    (2049, 64, 160, 20), (2500, 40, 256, 50), (5000, 3, 64, 1), (4100, 17, 32, 1024),
    (2048, 513, 128, 2048 // 4),
])
def test_route_shapes(ivf_ctx, oracle_mod, C, Q, D, k):
    rng = np.random.default_rng(C * 7 + D)
    c = rng.integers(0, 256, (C, D)).astype(np.float32)
    q = rng.integers(0, 256, (Q, D)).astype(np.float32)
    assert_route_equal(ivf_ctx, oracle_mod, q, c, k)


def test_route_ties_go_to_lower_id(ivf_ctx, oracle_mod):
    rng = np.random.default_rng(3)
    base = rng.integers(0, 8, (1500, 16)).astype(np.float32)
    c = np.repeat(base, 2, axis=0)  # every centroid twice -> exact ties
    q = rng.integers(0, 8, (200, 16)).astype(np.float32)
    assert_route_equal(ivf_ctx, oracle_mod, q, c, 12)
    ids, dist, _ = run_route(ivf_ctx, q, c, 12)
    tie = dist[:, 1:] == dist[:, :-1]
    assert (ids[:, 1:][tie] > ids[:, :-1][tie]).all()


def test_route_forced_fallback_is_identical(ivf_ctx, oracle_mod):
    import paper_2608_08751_amd as ivf

    d = synth.uniform_mixture_route(5000, 300, 128, seed=11)
    ivf_ctx.set_option(ivf.IVF_OPT_FORCE_FALLBACK, 1)
    try:
        stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], 64)
        assert stats["fallback"] == 300
    finally:
        ivf_ctx.set_option(ivf.IVF_OPT_FORCE_FALLBACK, 0)


@pytest.mark.parametrize("rank", [1, 3, 400])
def test_route_extreme_threshold_ranks_stay_exact(ivf_ctx, oracle_mod, rank):
    """Too-tight thresholds (underflow) and too-loose ones (overflow) must
    land in the exact fallback, not change results."""
    import paper_2608_08751_amd as ivf

    d = synth.normalised_route(20000, 200, 96, seed=rank)
    ivf_ctx.set_option(ivf.IVF_OPT_SAMPLE_RANK, rank)
    try:
        assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], 64)
    finally:
        ivf_ctx.set_option(ivf.IVF_OPT_SAMPLE_RANK, 0)


def test_route_deterministic(ivf_ctx):
    d = synth.uniform_mixture_route(9000, 700, 128, seed=5)
    a = run_route(ivf_ctx, d["queries"], d["centroids"], 64)
    b = run_route(ivf_ctx, d["queries"], d["centroids"], 64)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all()


def _sampled_full_size(ctx, oracle_mod, d, k, nsample):
    ids, dist, stats = run_route(ctx, d["queries"], d["centroids"], k)
    Q = d["queries"].shape[0]
    rng = np.random.default_rng(123)
    sample = np.union1d(rng.choice(Q, nsample, replace=False), d["plant_q"])
    oids, odist = oracle_mod.route(d["queries"][sample], d["centroids"], k)
    assert (ids[sample] == oids).all()
    assert (dist[sample] == odist).all()
    for qi, ci in zip(d["plant_q"], d["plant_c"]):
        assert ids[qi, 0] == ci and dist[qi, 0] == 0.0
    assert (dist >= 0).all() and (np.diff(dist, axis=1) >= 0).all()
    # every row holds k distinct valid ids
    s = np.sort(ids, axis=1)
    assert (s[:, 1:] != s[:, :-1]).all() and ids.min() >= 0 and ids.max() < d["centroids"].shape[0]
    return stats


def test_route_uint8_full_size_sampled(ivf_ctx, oracle_mod):
    """65,536 centroids, 10,000 integer-valued queries, nprobe 64 (the int8
    planes): 200 sampled queries against the oracle."""
    d = synth.uniform_mixture_route(65536, 10000, 128, seed=0, plants=0)
    stats = _sampled_full_size(ivf_ctx, oracle_mod, d, 64, 200)
    print("route u8 full-size stats:", stats)
    assert stats["screen_i8"] == 1
    assert stats["fallback"] < 100  # < 1% of queries


def test_route_uint8_full_size_with_plants_sampled(ivf_ctx, oracle_mod):
    """The same workload with 16 queries replaced by (non-integral) centroids:
    the call takes the fp32 kernels; the plants route to their centroid at
    distance 0."""
    d = synth.uniform_mixture_route(65536, 10000, 128, seed=0)
    stats = _sampled_full_size(ivf_ctx, oracle_mod, d, 64, 100)
    assert stats["screen_i8"] == 0
    assert stats["fallback"] < 100


def test_route_normalised_full_size_sampled(ivf_ctx, oracle_mod):
    """262,144 unit-norm centroids (D = 96), 10,000 queries, nprobe 128."""
    d = synth.normalised_route(262144, 10000, 96, seed=0)
    stats = _sampled_full_size(ivf_ctx, oracle_mod, d, 128, 60)
    print("route normalised full-size stats:", stats)
    assert stats["fallback"] < 100


def _route_with_option(ctx, q, c, k, option, value):
    import paper_2608_08751_amd as ivf

    ctx.set_option(option, value)
    try:
        return run_route(ctx, q, c, k)
    finally:
        ctx.set_option(option, 0)


@pytest.mark.parametrize("C,Q,D,k", [(9000, 700, 128, 64), (2100, 130, 64, 16), (2500, 50, 96, 30),
                                     (4500, 300, 256, 40), (3001, 77, 36, 5)])
def test_route_int8_and_fp32_paths_agree(ivf_ctx, oracle_mod, C, Q, D, k):
    """Uint8-valued queries are routed on the two int8 planes (tables above
    2,048 centroids); forcing the fp32 kernels must give the same ids and
    distances (both exact)."""
    import paper_2608_08751_amd as ivf

    d = synth.uniform_mixture_route(C, Q, D, seed=C + D, plants=0)
    stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], k)
    assert stats["screen_i8"] == 1
    ids, dist, _ = run_route(ivf_ctx, d["queries"], d["centroids"], k)
    fids, fdist, fstats = _route_with_option(ivf_ctx, d["queries"], d["centroids"], k, ivf.IVF_OPT_FP32_SCREEN, 1)
    assert fstats["screen_i8"] == 0
    assert (ids == fids).all() and (dist == fdist).all()


@pytest.mark.parametrize("where", ["query", "centroid_high", "centroid_low"])
def test_route_values_outside_the_int8_path_take_fp32(ivf_ctx, oracle_mod, where):
    """A non-integral query value or a centroid outside the two planes'
    range sends the whole call to the fp32 kernels, with exact results."""
    d = synth.uniform_mixture_route(6000, 200, 128, seed=7, plants=0)
    q, c = d["queries"].copy(), d["centroids"].copy()
    if where == "query":
        q[123, 45] += 0.5
    elif where == "centroid_high":
        c[4321, 7] = 300.0
    else:
        c[17, 100] = -2.0
    stats = assert_route_equal(ivf_ctx, oracle_mod, q, c, 32)
    assert stats["screen_i8"] == 0


def test_route_int8_forced_fallback_and_extreme_ranks(ivf_ctx, oracle_mod):
    """The int8 keys and filter feed the same certified selection: too tight
    or too loose thresholds and forced fallbacks stay exact."""
    import paper_2608_08751_amd as ivf

    d = synth.uniform_mixture_route(20000, 150, 128, seed=21, plants=0)
    for opt, val in ((ivf.IVF_OPT_SAMPLE_RANK, 1), (ivf.IVF_OPT_SAMPLE_RANK, 400), (ivf.IVF_OPT_FORCE_FALLBACK, 1)):
        ivf_ctx.set_option(opt, val)
        try:
            stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], d["centroids"], 64)
            assert stats["screen_i8"] == 1
        finally:
            ivf_ctx.set_option(opt, 0)


@pytest.mark.parametrize("kind", ["uint8", "normalised"])
def test_route_sorted_table_keeps_threshold(ivf_ctx, oracle_mod, kind):
    """A centroid table in spatial order (sorted by norm, or along the axis
    of largest spread), as a table ordered by list or position would be: the
    threshold sample is spread over the table, so the threshold is not
    biased: no query overflows its candidate list or falls back, and ids and
    distances equal the oracle's."""
    if kind == "uint8":
        d = synth.uniform_mixture_route(16384, 400, 128, seed=5, plants=0)
        c, k = d["centroids"], 64
        order = np.argsort((c.astype(np.float64) ** 2).sum(axis=1), kind="stable")
    else:
        d = synth.normalised_route(32768, 300, 96, seed=5, plants=0)
        c, k = d["centroids"], 128
        order = np.argsort(c[:, int(np.argmax(c.var(axis=0)))], kind="stable")
    c = np.ascontiguousarray(c[order])
    stats = assert_route_equal(ivf_ctx, oracle_mod, d["queries"], c, k)
    assert stats["fallback"] == 0 and stats["overflow"] == 0
    assert stats["sample"] > 0
