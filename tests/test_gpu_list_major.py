"""GPU parity of ivf_list_major against the oracle: the list-major copy of the
rows and the residuals x - c(x) are bit-identical, for whole layouts, slices
of positions, empty and skewed lists, and on a full-size layout produced by
ivf_assign_build (sampled positions plus invariants over every row)."""
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


def gpu_layout(ctx, x, c, offsets, perm, pos0=0, n=None):
    import torch

    import paper_2608_08751_amd as ivf

    rows, res = ivf.ivf_list_major(ctx, to_dev(x), to_dev(c), to_dev(offsets),
                                   to_dev(perm.view(np.int32)), pos0=pos0, n=n)
    torch.cuda.synchronize()
    return rows.cpu().numpy(), res.cpu().numpy()


def case(N, C, D, dt, skew, seed):
    rng = np.random.default_rng(seed)
    if dt == "u8":
        x = rng.integers(0, 256, (N, D)).astype(np.uint8)
        c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    else:
        x = (rng.standard_normal((N, D)) * 3).astype(np.float32)
        c = (rng.standard_normal((C, D)) * 3).astype(np.float32)
    lab = synth.random_labels(N, C, seed=seed, skew=skew)
    return x, c, lab


@pytest.mark.parametrize("N,C,D,dt,skew", [
    (1, 1, 4, "u8", 0.0), (1000, 7, 16, "u8", 0.0), (5003, 300, 128, "u8", 0.0),
    (5003, 300, 96, "f32", 0.0), (20000, 2000, 128, "u8", 1.2), (3001, 5000, 36, "f32", 0.0),
    (4096, 64, 256, "f32", 0.0),
])
def test_list_major_exact(ivf_ctx, oracle_mod, N, C, D, dt, skew):
    x, c, lab = case(N, C, D, dt, skew, N + C + D)
    _, offsets, perm = oracle_mod.build_lists(lab, C)
    rows, res = gpu_layout(ivf_ctx, x, c, offsets, perm)
    orows, ores = oracle_mod.list_major(x, c, lab, perm)
    assert (rows == orows).all()
    assert (res.view(np.uint32) == ores.view(np.uint32)).all()


@pytest.mark.parametrize("pos0,n", [(0, 1), (1234, 5000), (9999, 1), (4321, 0), (5000, 5000)])
def test_list_major_slices(ivf_ctx, oracle_mod, pos0, n):
    x, c, lab = case(10000, 500, 64, "u8", 0.8, 7)
    _, offsets, perm = oracle_mod.build_lists(lab, 500)
    rows, res = gpu_layout(ivf_ctx, x, c, offsets, perm, pos0=pos0, n=n)
    orows, ores = oracle_mod.list_major(x, c, lab, perm[pos0:pos0 + n])
    assert rows.shape == (n, 64) and (rows == orows).all()
    assert (res.view(np.uint32) == ores.view(np.uint32)).all()


def test_list_major_bad_row_ids_are_not_read(ivf_ctx, oracle_mod):
    x, c, lab = case(3000, 40, 32, "u8", 0.0, 9)
    _, offsets, perm = oracle_mod.build_lists(lab, 40)
    bad = perm.copy()
    bad[[5, 1700]] = [3000, 0xFFFFFFFF]
    rows, res = gpu_layout(ivf_ctx, x, c, offsets, bad)
    good = np.ones(3000, bool)
    good[[5, 1700]] = False
    orows, ores = oracle_mod.list_major(x, c, lab, perm)
    assert (rows[good] == orows[good]).all() and (res[good] == ores[good]).all()
    assert (rows[~good] == 0).all() and np.isnan(res[~good]).all()


def test_list_major_full_size_from_assign_build(ivf_ctx, oracle_mod):
    """10M uint8 rows of the 65,536-component mixture assigned by
    ivf_assign_build, then laid out list-major: sampled positions match the
    oracle bit for bit, and over every position the copy is x[perm] and the
    residual is that row minus its list's centroid (torch's fp32 subtraction
    on the device as the independent check)."""
    import torch

    import paper_2608_08751_amd as ivf

    N, C, D = 10_000_000, 65536, 128
    means = synth.uniform_means(C, D, seed=0)
    md = to_dev(means)
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(md, 0, N, x, seed=0)
    lab, cnt, off, perm = ivf.ivf_assign_build(ivf_ctx, x, md)
    rows, res = ivf.ivf_list_major(ivf_ctx, x, md, off, perm)
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    pos = np.sort(rng.choice(N, 4096, replace=False))
    permh = perm.cpu().numpy().view(np.uint32)
    labh = lab.cpu().numpy()
    xs = x[to_dev(permh[pos].astype(np.int64))].cpu().numpy()
    # the oracle on the sampled positions (labels of the sampled rows only)
    sub_lab = labh[permh[pos]]
    orows, ores = oracle_mod.list_major(xs, means, sub_lab, np.arange(len(pos), dtype=np.uint32))
    assert (rows[to_dev(pos)].cpu().numpy() == orows).all()
    assert (res[to_dev(pos)].cpu().numpy().view(np.uint32) == ores.view(np.uint32)).all()
    # every position: the copy is x[perm], and the residual is x[perm] minus the list's centroid
    permd = perm.long() & 0xFFFFFFFF
    assert bool((rows == x[permd]).all())
    listd = lab.long()[permd]
    assert bool((res == x[permd].float() - md[listd]).all())
