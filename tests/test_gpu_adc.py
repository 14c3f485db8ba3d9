"""GPU parity of ivf_adc_scan (residual-PQ approximate-distance scan with a
bounded handoff) against the oracle: ids and approximate distances
bit-identical, for short and long lists (the local top-k pool trims),
k = 1 ... 1024, subspace counts on both code-loading paths, invalid probes,
empty lists, and a full pipeline (assign-build -> list-major residuals ->
PQ training and encoding -> routing -> ADC scan) on sampled queries."""
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


def gpu_adc(ctx, q, c, probes, off, perm, codes, cb, k):
    import torch

    import paper_2608_08751_amd as ivf

    ids, dist = ivf.ivf_adc_scan(ctx, to_dev(q), to_dev(c), to_dev(probes), to_dev(off),
                                 to_dev(perm.view(np.int32)), to_dev(codes), to_dev(cb), k)
    torch.cuda.synchronize()
    return ids.cpu().numpy().view(np.uint32), dist.cpu().numpy()


def setup(seed, B, C, D, M, N, P, skew=0.0):
    rng = np.random.default_rng(seed)
    c = rng.standard_normal((C, D)).astype(np.float32) * 2
    q = rng.standard_normal((B, D)).astype(np.float32) * 2
    cb = rng.standard_normal((M, 256, D // M)).astype(np.float32)
    lab = synth.random_labels(N, C, seed=seed, skew=skew)
    order = np.argsort(lab, kind="stable").astype(np.uint32)
    off = np.concatenate([[0], np.cumsum(np.bincount(lab, minlength=C))]).astype(np.int64)
    codes = rng.integers(0, 256, (N, M)).astype(np.uint8)
    probes = np.stack([rng.choice(C, P, replace=False) for _ in range(B)]).astype(np.int32)
    return q, c, probes, off, order, codes, cb


@pytest.mark.parametrize("B,C,D,M,N,P,k,skew", [
    (7, 50, 32, 16, 3000, 5, 16, 0.0),        # short lists, no trim
    (5, 4, 64, 16, 40000, 3, 512, 0.0),       # lists of ~10,000: several trims per list
    (9, 30, 100, 20, 20000, 10, 100, 1.0),    # skewed lists
    (4, 20, 100, 50, 8000, 20, 1024, 0.0),    # byte-loaded codes, k = max
    (6, 12, 96, 3, 12000, 4, 1, 0.0),         # k = 1
    (3, 300, 128, 16, 600, 64, 512, 0.0),     # many empty lists, fewer candidates than k
])
def test_adc_scan_exact(ivf_ctx, oracle_mod, B, C, D, M, N, P, k, skew):
    q, c, probes, off, perm, codes, cb = setup(B + C + N, B, C, D, M, N, P, skew)
    ids, dist = gpu_adc(ivf_ctx, q, c, probes, off, perm, codes, cb, k)
    oids, odist = oracle_mod.adc_scan(q, c, probes, off, perm, codes, cb, k)
    assert (ids == oids).all()
    assert (dist.view(np.uint32) == odist.view(np.uint32)).all()


@pytest.mark.parametrize("B,C,D,M,N,P,k,skew", [
    (3, 8, 64, 16, 120000, 4, 512, 2.0),      # one list far longer than the rest: spread over groups
    (4, 6, 32, 8, 60000, 1, 256, 0.0),        # one probe: a single group of every chunk
    (5, 2000, 64, 16, 200000, 64, 512, 1.2),  # Zipf-skewed lists, 64 probes
    (2, 5, 32, 8, 50000, 5, 1000, 0.0),       # every list probed
])
def test_adc_scan_chunk_groups(ivf_ctx, oracle_mod, B, C, D, M, N, P, k, skew):
    """Lists cut into 1,024-code chunks and grouped per query (at most P
    groups): long lists spread over several groups, many short lists
    packed into one."""
    q, c, probes, off, perm, codes, cb = setup(7 * B + C + N, B, C, D, M, N, P, skew)
    ids, dist = gpu_adc(ivf_ctx, q, c, probes, off, perm, codes, cb, k)
    oids, odist = oracle_mod.adc_scan(q, c, probes, off, perm, codes, cb, k)
    assert (ids == oids).all()
    assert (dist.view(np.uint32) == odist.view(np.uint32)).all()


def test_adc_scan_queries_without_candidates(ivf_ctx, oracle_mod):
    """Queries whose probed lists are all empty or invalid have no chunk and
    no group; their handoff is all padding."""
    q, c, probes, off, perm, codes, cb = setup(11, 4, 50, 32, 8, 5000, 3)
    probes[0, :] = -1
    off[7] = off[8] = off[6]  # list 7 empty (offsets stay non-decreasing)
    off[9:] = np.maximum(off[9:], off[8])
    probes[1, :] = [7, -5, 51]
    ids, dist = gpu_adc(ivf_ctx, q, c, probes, off, perm, codes, cb, 64)
    oids, odist = oracle_mod.adc_scan(q, c, probes, off, perm, codes, cb, 64)
    assert (ids == oids).all() and (dist.view(np.uint32) == odist.view(np.uint32)).all()
    assert (ids[:2] == 0xFFFFFFFF).all() and np.isinf(dist[:2]).all()


def test_adc_scan_invalid_probes(ivf_ctx, oracle_mod):
    q, c, probes, off, perm, codes, cb = setup(5, 6, 40, 32, 8, 10000, 6)
    probes[:, 2] = -1
    probes[1, 4] = 40
    ids, dist = gpu_adc(ivf_ctx, q, c, probes, off, perm, codes, cb, 300)
    oids, odist = oracle_mod.adc_scan(q, c, probes, off, perm, codes, cb, 300)
    assert (ids == oids).all() and (dist.view(np.uint32) == odist.view(np.uint32)).all()


def test_adc_pipeline_sampled(ivf_ctx, oracle_mod):
    """2M uint8 rows of the 65,536-component mixture: assign-build, list-major
    residuals, PQ (M = 16) trained on 262,144 residuals and encoding all rows,
    1,000 queries routed with nprobe 64, ADC scan with k = 512: 32 sampled
    queries match the oracle bit for bit."""
    import torch

    import paper_2608_08751_amd as ivf

    N, C, D, M, Q, P, K = 2_000_000, 65536, 128, 16, 1000, 64, 512
    means = synth.uniform_means(C, D, seed=0)
    md = to_dev(means)
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(md, 0, N, x, seed=0)
    qrows = torch.empty((Q, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(md, N, Q, qrows, seed=0)
    qf = qrows.float().contiguous()
    lab, cnt, off, perm = ivf.ivf_assign_build(ivf_ctx, x, md)
    _, res = ivf.ivf_list_major(ivf_ctx, x, md, off, perm, rows=False)
    rng = np.random.default_rng(1)
    train = res[to_dev(np.sort(rng.choice(N, 262144, replace=False)))].contiguous()
    cb0 = train[to_dev(rng.choice(262144, 256, replace=False))].reshape(256, M, D // M).permute(1, 0, 2).contiguous()
    cb, _, _ = ivf.ivf_pq_train_step(ivf_ctx, train, cb0)
    codes = ivf.ivf_pq_encode(ivf_ctx, res, cb)
    probes, _ = ivf.ivf_route(ivf_ctx, qf, md, P, want_dist=False)
    ids, dist = ivf.ivf_adc_scan(ivf_ctx, qf, md, probes, off, perm, codes, cb, K)
    torch.cuda.synchronize()
    sample = np.sort(rng.choice(Q, 32, replace=False))
    oids, odist = oracle_mod.adc_scan(qf.cpu().numpy()[sample], means, probes.cpu().numpy()[sample],
                                      off.cpu().numpy(), perm.cpu().numpy().view(np.uint32),
                                      codes.cpu().numpy(), cb.cpu().numpy(), K)
    assert (ids.cpu().numpy().view(np.uint32)[sample] == oids).all()
    assert (dist.cpu().numpy()[sample].view(np.uint32) == odist.view(np.uint32)).all()
