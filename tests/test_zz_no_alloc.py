"""ivf_route_noalloc (routing with the library's static device scratch, for
callers that cannot allocate) against ivf_route on the same inputs: ids and
distances bit-identical, on two calls in a row, the second smaller, through
the C ABI with caller-allocated outputs."""
import ctypes

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


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def route_both(ctx, d, k):
    import torch

    import paper_2608_08751_amd as ivf

    q = torch.from_numpy(d["queries"]).cuda()
    c = torch.from_numpy(d["centroids"]).cuda()
    Q, D = q.shape
    C = c.shape[0]
    ref_ids, ref_dist = ivf.ivf_route(ctx, q, c, k)
    ids = torch.full((Q, k), -7, dtype=torch.int32, device="cuda")
    dist = torch.full((Q, k), -7.0, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    ctx.bind_stream()
    st = ctx.lib.ivf_route_noalloc(ctx.handle, _p(q), Q, _p(c), C, D, k, _p(ids), _p(dist))
    assert st == ivf.IVF_OK, ctx.error()
    assert ctx.lib.ivf_sync(ctx.handle) == ivf.IVF_OK, ctx.error()
    stats = ctx.last_stats()
    return (ids.cpu().numpy(), dist.cpu().numpy(), ref_ids.cpu().numpy(), ref_dist.cpu().numpy(), stats)


def test_route_noalloc_matches_route_twice(ivf_ctx):
    # first call: 65,536 centroids, 4,000 queries (several batches of the
    # static scratch); second call: fewer centroids and queries, so stale
    # contents of the scratch from the first call lie beyond what it writes
    # (the first call has integer-valued queries only, so it routes on the
    # int8 planes; the planted queries of the second send it to fp32)
    cases = [(synth.uniform_mixture_route(65536, 4000, 128, seed=3, plants=0), 64, 1),
             (synth.uniform_mixture_route(3000, 300, 64, seed=4), 16, 0)]
    for d, k, i8 in cases:
        ids, dist, rids, rdist, st = route_both(ivf_ctx, d, k)
        print("noalloc route Q=%d C=%d k=%d stats %s" % (d["queries"].shape[0], d["centroids"].shape[0], k, st),
              flush=True)
        assert st["screen_i8"] == i8
        assert np.array_equal(ids, rids)
        assert np.array_equal(dist.view(np.uint32), rdist.view(np.uint32))
        for qi, ci in zip(d["plant_q"], d["plant_c"]):
            assert ids[qi, 0] == ci and dist[qi, 0] == 0.0


def test_route_noalloc_refuses_oversized(ivf_ctx):
    """A centroid table whose norms alone exceed the static scratch is refused
    before anything is enqueued (the pointers are never dereferenced)."""
    import paper_2608_08751_amd as ivf

    lib, h = ivf_ctx.lib, ivf_ctx.handle
    GB = 1 << 30
    st = lib.ivf_route_noalloc(h, ctypes.c_void_p(GB), 10, ctypes.c_void_p(2 * GB), 20_000_000, 4, 8,
                               ctypes.c_void_p(4 * GB), None)
    assert st == ivf.IVF_EUNSUPPORTED
    assert "static scratch" in ivf_ctx.error()
