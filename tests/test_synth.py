"""Generator sanity (CPU): shapes, value ranges, reproducibility, plants."""
import numpy as np

import synth


def test_uniform_mixture_route_shapes_and_plants():
    a = synth.uniform_mixture_route(500, 120, 32, seed=1, plants=7)
    b = synth.uniform_mixture_route(500, 120, 32, seed=1, plants=7)
    q, c = a["queries"], a["centroids"]
    assert q.shape == (120, 32) and c.shape == (500, 32)
    assert q.dtype == np.float32 and c.dtype == np.float32
    assert (q == b["queries"]).all() and (c == b["centroids"]).all()
    assert c.min() >= 0 and c.max() <= 255
    notplanted = np.setdiff1d(np.arange(120), a["plant_q"])
    assert (q[notplanted] == np.rint(q[notplanted])).all()
    assert q.min() >= 0 and q.max() <= 255
    for qi, ci in zip(a["plant_q"], a["plant_c"]):
        assert (q[qi] == c[ci]).all()
    assert not (synth.uniform_mixture_route(500, 120, 32, seed=2)["queries"] == q).all()


def test_normalised_route_unit_norm():
    a = synth.normalised_route(1000, 50, 96, seed=0)
    n = np.linalg.norm(a["centroids"].astype(np.float64), axis=1)
    assert np.abs(n - 1).max() < 1e-6
    n = np.linalg.norm(a["queries"].astype(np.float64), axis=1)
    assert np.abs(n - 1).max() < 1e-6


def test_mixture_rows_u8_statistics_and_reproducibility():
    m = synth.uniform_means(32, 16, seed=5)
    x, a = synth.mixture_rows_u8(m, 0, 4000, seed=5)
    x2, a2 = synth.mixture_rows_u8(m, 1000, 500, seed=5)
    assert x.dtype == np.uint8 and x.shape == (4000, 16)
    assert (x[1000:1500] == x2).all() and (a[1000:1500] == a2).all()
    resid = x.astype(np.float64) - m[a]
    inner = (m[a] > 80) & (m[a] < 175)  # away from the clipping range
    assert abs(resid[inner].std() - 20.0) < 0.5
    assert abs(resid[inner].mean()) < 0.5
    assert np.bincount(a, minlength=32).min() > 60


def test_kmeans_init_distinct_and_labels():
    idx = synth.kmeans_init(10000, 512, seed=0)
    assert len(np.unique(idx)) == 512 and idx.min() >= 0 and idx.max() < 10000
    lab = synth.random_labels(10000, 64, seed=0, skew=1.2)
    assert lab.min() >= 0 and lab.max() < 64 and np.bincount(lab)[0] > np.bincount(lab, minlength=64)[-1]
