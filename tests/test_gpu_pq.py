"""GPU parity of product quantisation against the oracle: codes, trained
codebooks and counts are bit-identical; per-subspace objectives agree to fp64
summation-order rounding. Shapes cover the paper's subspace widths (D / M =
1 ... 16), ties (integer data with duplicate codewords), empty codewords
(reseeds), and residuals of a full-size list-major layout."""
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


SHAPES = [(1, 8, 8), (1000, 16, 4), (5001, 128, 16), (3000, 96, 16), (2000, 100, 20), (4000, 128, 32),
          (777, 48, 3), (600, 96, 32), (300, 100, 50)]


def data(n, D, M, seed, integer=False):
    rng = np.random.default_rng(seed)
    if integer:
        x = rng.integers(-3, 4, (n, D)).astype(np.float32)
        cb = rng.integers(-3, 4, (M, 256, D // M)).astype(np.float32)
    else:
        x = (rng.standard_normal((n, D)) * 4 + rng.integers(0, 3, (n, 1))).astype(np.float32)
        cb = x[rng.choice(n, 256, replace=n < 256)].reshape(256, M, D // M).transpose(1, 0, 2).copy()
        cb += rng.standard_normal(cb.shape).astype(np.float32) * 0.1
    return x, cb


@pytest.mark.parametrize("n,D,M", SHAPES)
@pytest.mark.parametrize("integer", [False, True])
def test_pq_encode_exact(ivf_ctx, oracle_mod, n, D, M, integer):
    import torch

    import paper_2608_08751_amd as ivf

    x, cb = data(n, D, M, n + D + M, integer)
    codes = ivf.ivf_pq_encode(ivf_ctx, to_dev(x), to_dev(cb))
    torch.cuda.synchronize()
    assert (codes.cpu().numpy() == oracle_mod.pq_encode(x, cb)).all()


@pytest.mark.parametrize("n,D,M", SHAPES)
def test_pq_train_chain_exact(ivf_ctx, oracle_mod, n, D, M):
    import torch

    import paper_2608_08751_amd as ivf

    x, cb = data(n, D, M, 3 * n + M)
    cb_g = to_dev(cb)
    for it in range(3):
        out, cnt, obj = ivf.ivf_pq_train_step(ivf_ctx, to_dev(x), cb_g, seed=7, it=it)
        torch.cuda.synchronize()
        oout, ocnt, oobj = oracle_mod.pq_train_step(x, cb, seed=7, it=it)
        assert (cnt.cpu().numpy() == ocnt).all()
        assert (out.cpu().numpy().view(np.uint32) == oout.view(np.uint32)).all()
        g = obj.cpu().numpy()
        assert np.all(np.abs(g - oobj) <= 1e-12 * np.maximum(oobj, 1e-300))
        cb, cb_g = oout, out
    if n < 256:
        assert (cnt.cpu().numpy() == 0).any()


def test_pq_on_list_major_residuals(ivf_ctx, oracle_mod):
    """Residuals of 2M uint8 mixture rows laid out list-major (65,536 lists):
    one training step on a 262,144-row slice and the encoding of all rows
    match the oracle (codes on a row sample)."""
    import torch

    import paper_2608_08751_amd as ivf

    N, C, D, M = 2_000_000, 65536, 128, 16
    means = synth.uniform_means(C, D, seed=0)
    md = to_dev(means)
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(md, 0, N, x, seed=0)
    lab, cnt, off, perm = ivf.ivf_assign_build(ivf_ctx, x, md)
    _, res = ivf.ivf_list_major(ivf_ctx, x, md, off, perm, rows=False)
    rng = np.random.default_rng(3)
    sample = to_dev(np.sort(rng.choice(N, 262144, replace=False)))
    train = res[sample].contiguous()
    trh = train.cpu().numpy()
    cb0 = trh[rng.choice(262144, 256, replace=False)].reshape(256, M, D // M).transpose(1, 0, 2).copy()
    cb, cntg, objg = ivf.ivf_pq_train_step(ivf_ctx, train, to_dev(cb0), seed=1, it=0)
    codes = ivf.ivf_pq_encode(ivf_ctx, res, cb)
    torch.cuda.synchronize()
    ocb, ocnt, oobj = oracle_mod.pq_train_step(trh, cb0, seed=1, it=0)
    assert (cntg.cpu().numpy() == ocnt).all()
    assert (cb.cpu().numpy().view(np.uint32) == ocb.view(np.uint32)).all()
    rows = np.sort(rng.choice(N, 20000, replace=False))
    want = oracle_mod.pq_encode(res[to_dev(rows)].cpu().numpy(), ocb)
    assert (codes[to_dev(rows)].cpu().numpy() == want).all()
