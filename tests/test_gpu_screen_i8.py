"""GPU parity of the int8-MFMA screens used for uint8 rows (assignment and the
k-means step): labels must equal the oracle's exactly on every path: the
default (one int8 plane, then two int8 planes for the rows it leaves), two
planes alone (IVF_OPT_I8_TWO_PLANE_ONLY), and the fp32 path the library takes
when centroids do not quantise (or when IVF_OPT_FP32_SCREEN forces it),
including near-ties that the quantised scores cannot separate."""
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


# screen paths: (name, options)
PATHS = {
    "default": {},
    "two_planes": {"IVF_OPT_I8_TWO_PLANE_ONLY": 1},
    "fp32": {"IVF_OPT_FP32_SCREEN": 1},
}


def gpu_assign(ctx, x, c, path="default", **extra):
    import torch

    import paper_2608_08751_amd as ivf

    opts = dict(PATHS[path], **extra)
    for k, v in opts.items():
        ctx.set_option(getattr(ivf, k), v)
    try:
        lab, cnt, off, perm = ivf.ivf_assign_build(ctx, to_dev(x), to_dev(c))
        torch.cuda.synchronize()
        stats = ctx.last_stats()
    finally:
        for k in opts:
            ctx.set_option(getattr(ivf, k), 0)
    return lab.cpu().numpy(), cnt.cpu().numpy(), off.cpu().numpy(), perm.cpu().numpy(), stats


def check_assign(ctx, oracle_mod, x, c, expect_i8=True):
    olab = oracle_mod.assign(x, c)
    ocnt, ooff, operm = oracle_mod.build_lists(olab, c.shape[0])
    out = {}
    for path in PATHS:
        lab, cnt, off, perm, st = gpu_assign(ctx, x, c, path)
        print("%s stats %s" % (path, st), flush=True)
        bad = np.nonzero(lab != olab)[0]
        assert bad.size == 0, "%s: labels differ at rows %s" % (path, bad[:10])
        assert (cnt == ocnt).all() and (off == ooff).all() and (perm == operm).all()
        assert st["screen_i8"] == (1 if (expect_i8 and path != "fp32") else 0)
        if path != "default" or not expect_i8:
            assert st["rescreen"] == 0
        out[path] = st
    return out


def rows_and_centroids(N, C, D, seed):
    rng = np.random.default_rng(seed)
    means = rng.uniform(0.0, 255.0, size=(max(C // 2, 1), D)).astype(np.float32)
    x, _ = synth.mixture_rows_u8(means, 0, N, seed=seed)
    if C <= N:
        c = x[rng.choice(N, C, replace=False)].astype(np.float32)
    else:
        c = rng.uniform(0.0, 255.0, size=(C, D)).astype(np.float32)
    c += rng.uniform(-0.5, 0.5, size=c.shape).astype(np.float32)  # fractional coordinates
    np.clip(c, 0.0, 255.0, out=c)
    return x, c


@pytest.mark.parametrize(
    "N,C,D",
    [(5000, 1000, 128), (3001, 257, 100), (2500, 130, 36), (1500, 70, 200), (1200, 65, 256),
     (700, 1, 32), (700, 2, 64), (701, 3, 96), (4099, 640, 252), (513, 64, 128), (1, 100, 128)],
)
def test_i8_parity_shapes(ivf_ctx, oracle_mod, N, C, D):
    print("case N=%d C=%d D=%d" % (N, C, D), flush=True)
    x, c = rows_and_centroids(N, C, D, seed=N + C + D)
    check_assign(ivf_ctx, oracle_mod, x, c)


def test_i8_near_ties(ivf_ctx, oracle_mod):
    """Centroids that collide or nearly collide after quantisation (exact
    duplicates, offsets of 1e-3 and of half a quantisation step) and rows on
    or midway between them: the certificate must hand these to the exact
    re-evaluation or the fallback, and the labels must still be exact."""
    rng = np.random.default_rng(11)
    D = 128
    base = rng.integers(20, 236, size=(40, D)).astype(np.float32)
    variants = [base, base.copy(), base + 1e-3, base - 1.0 / 512, base + 1.0 / 512, base + 0.5]
    c = np.vstack(variants).astype(np.float32)
    x = [np.rint(base), np.floor(base + 0.25), np.clip(np.rint(base + 1.0), 0, 255)]
    mid = np.rint(base).copy()
    mid[:, 0] += 1  # one unit off the tie
    x.append(mid)
    x.append(rng.integers(0, 256, size=(500, D)))
    x = np.clip(np.vstack(x), 0, 255).astype(np.uint8)
    st = check_assign(ivf_ctx, oracle_mod, x, c)
    assert st["default"]["refine2"] + st["default"]["fallback"] > 0
    assert st["two_planes"]["refine2"] + st["two_planes"]["fallback"] > 0
    assert st["default"]["rescreen"] > 0


def test_i8_extreme_values(ivf_ctx, oracle_mod):
    """Rows of all 0 / all 255 against centroids at the ends of the range:
    the largest scores and bounds the int32 arithmetic has to hold."""
    D = 256
    rng = np.random.default_rng(3)
    x = np.vstack([np.zeros((3, D)), np.full((3, D), 255), rng.integers(0, 256, size=(300, D))]).astype(np.uint8)
    c = np.vstack([np.zeros((1, D)), np.full((1, D), 255.99), np.full((1, D), 127.5),
                   rng.uniform(0, 255.99, size=(97, D))]).astype(np.float32)
    check_assign(ivf_ctx, oracle_mod, x, c)


@pytest.mark.parametrize("bad", [256.0, -0.5, 255.999, 300.0, -1e6])
def test_i8_unquantisable_centroids_take_fp32(ivf_ctx, oracle_mod, bad):
    """One coordinate outside what 16-bit fixed point around 128 holds: the
    int8 kernel stands down and the fp32 screen gives the same exact labels."""
    x, c = rows_and_centroids(3000, 200, 128, seed=5)
    c[17, 5] = bad
    check_assign(ivf_ctx, oracle_mod, x, c, expect_i8=False)


def test_i8_edge_of_range_quantises(ivf_ctx, oracle_mod):
    """255.998 and 0.0 still fit (-32768 <= rint(256 (c - 128)) <= 32767)."""
    x, c = rows_and_centroids(2000, 100, 64, seed=8)
    c[3, :] = 255.998
    c[4, :] = 0.0
    check_assign(ivf_ctx, oracle_mod, x, c)


def test_i8_kmeans_step_all_paths(ivf_ctx, oracle_mod):
    """Two Lloyd iterations from sampled rows (several centroids per mixture
    component, so near-ties occur): every screen gives the oracle's step. The
    first iteration's centroids are integer rows, which the single plane
    settles alone; the second's are means."""
    import torch

    import paper_2608_08751_amd as ivf

    means = synth.uniform_means(150, 128, seed=21)
    x, _ = synth.mixture_rows_u8(means, 0, 12000, seed=21)
    c = x[synth.kmeans_init(12000, 600, seed=21)].astype(np.float32)
    for it in range(2):
        olab, ocen, ocnt, oobj = oracle_mod.kmeans_step(x, c, seed=3, it=it)
        for path, opts in PATHS.items():
            for k, v in opts.items():
                ivf_ctx.set_option(getattr(ivf, k), v)
            try:
                lab, cen, cnt, obj = ivf.ivf_kmeans_step(ivf_ctx, to_dev(x), to_dev(c), seed=3, it=it)
                torch.cuda.synchronize()
                st = ivf_ctx.last_stats()
            finally:
                for k in opts:
                    ivf_ctx.set_option(getattr(ivf, k), 0)
            print("it %d %s stats %s" % (it, path, st), flush=True)
            assert st["screen_i8"] == (0 if path == "fp32" else 1)
            if path == "default" and it == 0:
                assert st["rescreen"] <= 5
            assert (lab.cpu().numpy() == olab).all()
            assert (cnt.cpu().numpy() == ocnt).all()
            assert (cen.cpu().numpy() == ocen).all()
        c = ocen


@pytest.mark.parametrize("N", [1500, 3000, 5000])
def test_i8_forced_fallback_is_identical(ivf_ctx, oracle_mod, N):
    """Every row through the exact fallback scan: 1,500 rows fit the
    centroid-split windows, 3,000 also use the whole-row windows, and 5,000
    overflow the worklist (min(N, 4096 + N / 64) entries), so the scan finds
    the rows by their -1 labels."""
    import paper_2608_08751_amd as ivf

    x, c = rows_and_centroids(N, 90, 128, seed=13)
    olab = oracle_mod.assign(x, c)
    ivf_ctx.set_option(ivf.IVF_OPT_FORCE_FALLBACK, 1)
    try:
        lab, _, _, _, st = gpu_assign(ivf_ctx, x, c)
    finally:
        ivf_ctx.set_option(ivf.IVF_OPT_FORCE_FALLBACK, 0)
    assert st["screen_i8"] == 1 and st["fallback"] == N
    assert (lab == olab).all()


@pytest.mark.parametrize("N,C,D,cap", [(4000, 300, 128, 0), (2500, 130, 100, 7), (3000, 200, 64, 1)])
def test_i8_single_plane_rescreen_forced_and_overflow(ivf_ctx, oracle_mod, N, C, D, cap):
    """Every row handed from the single plane to the two planes
    (IVF_OPT_FORCE_RESCREEN), or a list capacity of 7 or 1 that overflows so
    that the two planes screen every row: the labels do not change."""
    import paper_2608_08751_amd as ivf

    x, c = rows_and_centroids(N, C, D, seed=N + C)
    olab = oracle_mod.assign(x, c)
    if cap == 0:
        lab, _, _, _, st = gpu_assign(ivf_ctx, x, c, IVF_OPT_FORCE_RESCREEN=1)
        assert st["rescreen"] == N
    else:
        lab, _, _, _, st = gpu_assign(ivf_ctx, x, c, IVF_OPT_RESCREEN_CAP=cap)
        assert st["rescreen"] > cap
    print("cap %d stats %s" % (cap, st), flush=True)
    assert st["screen_i8"] == 1
    assert (lab == olab).all()


@pytest.mark.parametrize("bad", [255.5, 255.7, 255.99])
def test_i8_single_plane_stands_down(ivf_ctx, oracle_mod, bad):
    """A coordinate that rounds to 128 on the single plane (outside int8) but
    fits the two planes: the two planes screen every row, exactly."""
    x, c = rows_and_centroids(3000, 150, 128, seed=7)
    c[9, 11] = bad
    st = check_assign(ivf_ctx, oracle_mod, x, c)
    assert st["default"]["rescreen"] == 0


def test_i8_single_plane_integer_centroids(ivf_ctx, oracle_mod):
    """Integer-valued centroids (sampled rows, as the k-means initialisation):
    no rounding on the single plane, which settles (almost) every row."""
    means = synth.uniform_means(200, 128, seed=31)
    x, _ = synth.mixture_rows_u8(means, 0, 20000, seed=31)
    c = x[synth.kmeans_init(20000, 700, seed=31)].astype(np.float32)
    st = check_assign(ivf_ctx, oracle_mod, x, c)
    assert st["default"]["rescreen"] <= 10


@pytest.mark.parametrize("slice_rows,extra", [(1000, {}), (997, {"IVF_OPT_FORCE_RESCREEN": 1}),
                                              (4096, {"IVF_OPT_FORCE_FALLBACK": 1}),
                                              (1500, {"IVF_OPT_RESCREEN_CAP": 3})])
@pytest.mark.parametrize("path", ["default", "fp32"])
def test_assignment_in_row_slices(ivf_ctx, oracle_mod, slice_rows, extra, path):
    """The assignment screens rows in slices (2^28 rows by default, so that
    row ids inside a launch fit int32); short slices (IVF_OPT_ASSIGN_SLICE)
    with ragged last slices, every row handed on, every row in the fallback,
    or an overflowing list: the labels, counts, offsets and permutation do not
    change, and the statistics add up over the slices."""
    x, c = rows_and_centroids(12345, 333, 128, seed=71)
    olab = oracle_mod.assign(x, c)
    ocnt, ooff, operm = oracle_mod.build_lists(olab, c.shape[0])
    lab, cnt, off, perm, st = gpu_assign(ivf_ctx, x, c, path, IVF_OPT_ASSIGN_SLICE=slice_rows, **extra)
    print("slice %d %s %s stats %s" % (slice_rows, path, extra, st), flush=True)
    assert (lab == olab).all()
    assert (cnt == ocnt).all() and (off == ooff).all() and (perm == operm).all()
    if "IVF_OPT_FORCE_FALLBACK" in extra:
        assert st["fallback"] == 12345
    if "IVF_OPT_FORCE_RESCREEN" in extra and path == "default":
        assert st["rescreen"] == 12345
