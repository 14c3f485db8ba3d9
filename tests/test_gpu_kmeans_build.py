"""GPU parity of ivf_kmeans_step, ivf_assign_build and ivf_build_lists
against the oracle: labels, counts, offsets, permutation and centroids must
be bit-identical; the objective agrees to fp64 summation-order rounding."""
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


def gpu_step(ctx, x, c, seed, it):
    import torch

    import paper_2608_08751_amd as ivf

    lab, cen, cnt, obj = ivf.ivf_kmeans_step(ctx, to_dev(x), to_dev(c), seed=seed, it=it)
    torch.cuda.synchronize()
    return lab.cpu().numpy(), cen.cpu().numpy(), cnt.cpu().numpy(), float(obj[0].cpu()), ctx.last_stats()


def assert_step_equal(ctx, oracle_mod, x, c, seed, it):
    lab, cen, cnt, obj, stats = gpu_step(ctx, x, c, seed, it)
    olab, ocen, ocnt, oobj = oracle_mod.kmeans_step(x, c, seed=seed, it=it)
    assert (lab == olab).all(), "labels differ at rows %s" % np.nonzero(lab != olab)[0][:10]
    assert (cnt == ocnt).all()
    assert (cen == ocen).all(), "centroids differ in clusters %s" % np.unique(np.nonzero(cen != ocen)[0])[:10]
    assert abs(obj - oobj) <= 1e-12 * max(oobj, 1e-300)
    return cen, obj, stats


def test_kmeans_chain_uint8(ivf_ctx, oracle_mod):
    """Four Lloyd iterations on 20,000 u8 rows (ragged tile), 300 clusters."""
    means = synth.uniform_means(400, 128, seed=1)
    x, _ = synth.mixture_rows_u8(means, 0, 20000, seed=1)
    c = x[synth.kmeans_init(20000, 300, seed=1)].astype(np.float32)
    objs = []
    for it in range(4):
        c, obj, stats = assert_step_equal(ivf_ctx, oracle_mod, x, c, 1, it)
        objs.append(obj)
    assert all(b <= a * (1 + 1e-9) for a, b in zip(objs, objs[1:]))


def test_kmeans_float_rows(ivf_ctx, oracle_mod):
    rng = np.random.default_rng(2)
    x = (rng.standard_normal((6001, 64)) * 3 + rng.integers(0, 5, (6001, 1))).astype(np.float32)
    c = x[rng.choice(6001, 100, replace=False)].copy()
    for it in range(2):
        c, _, _ = assert_step_equal(ivf_ctx, oracle_mod, x, c, 9, it)


def test_kmeans_empty_clusters_reseed(ivf_ctx, oracle_mod):
    rng = np.random.default_rng(4)
    x = rng.integers(0, 60, (3000, 32)).astype(np.uint8)
    c = np.vstack([x[:20].astype(np.float32), np.full((30, 32), 5000.0, np.float32)])
    cen, _, _ = assert_step_equal(ivf_ctx, oracle_mod, x, c, 77, 5)
    for j in range(20, 50):
        assert (cen[j] == x[oracle_mod.reseed_row(77, 5, j, 3000)]).all()


@pytest.mark.parametrize("N,C,D", [(1, 1, 4), (500, 1, 8), (257, 256, 16), (1000, 1000, 36),
                                   (3000, 300, 200), (2000, 150, 256), (1200, 90, 32), (4000, 40, 64),
                                   (300, 400, 128)])
def test_kmeans_small_shapes(ivf_ctx, oracle_mod, N, C, D):
    rng = np.random.default_rng(N + C)
    x = rng.integers(0, 256, (N, D)).astype(np.uint8)
    c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    assert_step_equal(ivf_ctx, oracle_mod, x, c, 3, 1)


@pytest.mark.parametrize("D", [160, 256])
def test_kmeans_wide_float_rows(ivf_ctx, oracle_mod, D):
    """Wide rows run the screening kernel with one wave per SIMD."""
    rng = np.random.default_rng(D)
    x = (rng.standard_normal((2500, D)) * 2 + rng.integers(0, 4, (2500, 1))).astype(np.float32)
    c = x[rng.choice(2500, 70, replace=False)].copy()
    assert_step_equal(ivf_ctx, oracle_mod, x, c, 5, 0)


def test_kmeans_forced_fallback_is_identical(ivf_ctx, oracle_mod):
    import paper_2608_08751_amd as ivf

    means = synth.uniform_means(100, 64, seed=6)
    x, _ = synth.mixture_rows_u8(means, 0, 5000, seed=6)
    c = x[synth.kmeans_init(5000, 80, seed=6)].astype(np.float32)
    ivf_ctx.set_option(ivf.IVF_OPT_FORCE_FALLBACK, 1)
    try:
        _, _, stats = assert_step_equal(ivf_ctx, oracle_mod, x, c, 6, 0)
        assert stats["fallback"] == 5000
    finally:
        ivf_ctx.set_option(ivf.IVF_OPT_FORCE_FALLBACK, 0)


# ------------------------------------------------------------------ lists

def gpu_lists(ctx, labels, C):
    import torch

    import paper_2608_08751_amd as ivf

    cnt, off, perm = ivf.ivf_build_lists(ctx, to_dev(labels), C)
    torch.cuda.synchronize()
    return cnt.cpu().numpy(), off.cpu().numpy(), perm.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("N,C,skew", [
    (0, 5, 0.0), (1, 1, 0.0), (1000, 1, 0.0), (12345, 300, 0.0), (100003, 20000, 0.0),
    (2000001, 65536, 0.0), (1000000, 40000, 1.1), (300000, 3, 0.0), (4099, 70000, 0.0),
    (20000003, 65536, 0.0), (9000000, 65536, 1.05),
])
def test_build_lists_exact(ivf_ctx, oracle_mod, N, C, skew):
    lab = synth.random_labels(N, C, seed=N + C, skew=skew)
    cnt, off, perm = gpu_lists(ivf_ctx, lab, C)
    ocnt, ooff, operm = oracle_mod.build_lists(lab, C)
    assert (cnt == ocnt).all() and (off == ooff).all()
    assert (perm == operm).all()


def test_build_lists_deterministic(ivf_ctx):
    """Several tiles per block and per sub-block: two runs are bit-identical."""
    lab = synth.random_labels(12_000_000, 65536, seed=3)
    a = gpu_lists(ivf_ctx, lab, 65536)
    b = gpu_lists(ivf_ctx, lab, 65536)
    assert all((x == y).all() for x, y in zip(a, b))


def test_build_lists_single_list_all_rows(ivf_ctx, oracle_mod):
    lab = np.full(200000, 7, np.int32)
    cnt, off, perm = gpu_lists(ivf_ctx, lab, 20)
    assert cnt[7] == 200000 and (perm == np.arange(200000, dtype=np.uint32)).all()


@pytest.mark.parametrize("dt", ["u8", "f32"])
def test_assign_build_small(ivf_ctx, oracle_mod, dt):
    import torch

    import paper_2608_08751_amd as ivf

    means = synth.uniform_means(300, 128, seed=8)
    x, _ = synth.mixture_rows_u8(means, 0, 30001, seed=8)
    if dt == "f32":
        x = x.astype(np.float32)
    c = means[:250]
    lab, cnt, off, perm = ivf.ivf_assign_build(ivf_ctx, to_dev(x), to_dev(c))
    torch.cuda.synchronize()
    olab = oracle_mod.assign(x, c)
    ocnt, ooff, operm = oracle_mod.build_lists(olab, 250)
    assert (lab.cpu().numpy() == olab).all()
    assert (cnt.cpu().numpy() == ocnt).all() and (off.cpu().numpy() == ooff).all()
    assert (perm.cpu().numpy().view(np.uint32) == operm).all()


@pytest.mark.parametrize("N,C,D", [(30000, 700, 128), (9000, 300, 64), (12000, 520, 96)])
def test_kmeans_label_hints_change_nothing(ivf_ctx, oracle_mod, N, C, D):
    """Hint labels only seed the single plane's keep threshold: the previous
    iteration's labels, garbage (negative, >= C, random) and a mix give the
    same labels, centroids, counts and objective as no hints, and the oracle's
    step."""
    import torch

    import paper_2608_08751_amd as ivf

    means = synth.uniform_means(max(C // 2, 1), D, seed=N)
    x, _ = synth.mixture_rows_u8(means, 0, N, seed=N)
    c0 = x[synth.kmeans_init(N, C, seed=1)].astype(np.float32)
    xd = to_dev(x)
    lab0, c1, _, _ = ivf.ivf_kmeans_step(ivf_ctx, xd, to_dev(c0), seed=0, it=0)
    ref = ivf.ivf_kmeans_step(ivf_ctx, xd, c1, seed=0, it=1)
    torch.cuda.synchronize()
    ref = [t.cpu().numpy() for t in ref]
    olab, ocen, ocnt, _ = oracle_mod.kmeans_step(x, c1.cpu().numpy(), seed=0, it=1)
    assert (ref[0] == olab).all() and (ref[1] == ocen).all() and (ref[2] == ocnt).all()
    rng = np.random.default_rng(N + C)
    garbage = rng.integers(-3, C + 50, size=N).astype(np.int32)
    mix = np.where(rng.random(N) < 0.5, lab0.cpu().numpy(), garbage).astype(np.int32)
    for hint in (lab0, to_dev(garbage), to_dev(mix)):
        out = ivf.ivf_kmeans_step(ivf_ctx, xd, c1, seed=0, it=1, hint_labels=hint)
        torch.cuda.synchronize()
        out = [t.cpu().numpy() for t in out]
        assert (out[0] == ref[0]).all() and (out[1] == ref[1]).all() and (out[2] == ref[2]).all()
        assert out[3][0] == ref[3][0]


@pytest.mark.parametrize("N,C,D", [(30000, 700, 128), (12000, 2600, 64)])
def test_single_plane_visiting_order_changes_nothing(ivf_ctx, oracle_mod, N, C, D):
    """The single plane's visiting order (ascending distance to the centroid
    mean, the default) against id order: the same labels, centroids, counts,
    objective and statistics on a k-means step from mean centroids (with and
    without hint labels) and on an assign-build, and the oracle's labels."""
    import torch

    import paper_2608_08751_amd as ivf

    means = synth.uniform_means(max(C // 2, 1), D, seed=N)
    x, _ = synth.mixture_rows_u8(means, 0, N, seed=N)
    c0 = x[synth.kmeans_init(N, C, seed=1)].astype(np.float32)
    xd = to_dev(x)
    lab0, c1, _, _ = ivf.ivf_kmeans_step(ivf_ctx, xd, to_dev(c0), seed=0, it=0)
    outs = {}
    for id_order in (1, 0):
        ivf_ctx.set_option(ivf.IVF_OPT_S1_ID_ORDER, id_order)
        try:
            k = ivf.ivf_kmeans_step(ivf_ctx, xd, c1, seed=0, it=1)
            torch.cuda.synchronize()
            st = ivf_ctx.last_stats()
            kh = ivf.ivf_kmeans_step(ivf_ctx, xd, c1, seed=0, it=1, hint_labels=lab0)
            a = ivf.ivf_assign_build(ivf_ctx, xd, c1)
            torch.cuda.synchronize()
            # the objective is element 0 of its buffer
            outs[id_order] = ([t.cpu().numpy() for t in k[:3]] + [k[3][:1].cpu().numpy()], st,
                              [t.cpu().numpy() for t in kh[:3]] + [kh[3][:1].cpu().numpy()],
                              [t.cpu().numpy() for t in a])
        finally:
            ivf_ctx.set_option(ivf.IVF_OPT_S1_ID_ORDER, 0)
    (k1, s1, h1, a1), (k0, s0, h0, a0) = outs[1], outs[0]
    olab = oracle_mod.assign(x, c1.cpu().numpy())
    assert (k0[0] == olab).all() and (a0[0] == olab).all()
    for u, v in ((k0, k1), (h0, h1), (h0, k1), (a0, a1)):
        assert all((p == q).all() for p, q in zip(u, v))
    assert s0 == s1 and s0["rescreen"] > 0 and s0["refine2"] > 0
