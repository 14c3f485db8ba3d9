"""Host model of the int8 screen's arithmetic (no GPU): the quantisation of
centroids to P = rint(256 (c - 128)) = 256 H + Ls + 128 with int8 H and Ls,
the integer score s = 256 (x'.H - Bh) + x'.Ls with Bh = rint(||c'||^2 / 2),
the bound |s + 128 k + 128 sum(x')| < 129 + ||x'||_1 / 2 on which the
kernel's certificate rests (k = ||c'||^2 - 2 x'.c', x' = x - 128,
c' = c - 128), and the prefilter inequality s <= 256 h + 128 ||x'||_1 with
h = x'.H - Bh. Distances are evaluated exactly with rational arithmetic on a
subset. The single-plane screen's arithmetic: one int8 plane H1 = rint(c'),
the score s1 = x'.H1 - b1 with b1 = rint(||c'||^2 / 2), and the bound
|g - s1| <= min(E ||x'||_1, R2 ||x'||_2) + 1/2 with g = x'.c' - ||c'||^2 / 2
= -k / 2, E the largest coordinate residual |c' - H1| and R2 the largest
residual norm ||c' - H1||_2 (Cauchy-Schwarz), on which its window
T = ceil(2 min(E ||x'||_1, R2 ||x'||_2)) + 2 rests."""
from fractions import Fraction

import numpy as np


def quantise(c):
    cp = c.astype(np.float64) - 128.0
    P = np.rint(256.0 * cp)
    assert np.all((P >= -32768) & (P <= 32767))
    P = P.astype(np.int64)
    H = P >> 8
    Ls = P - 256 * H - 128
    Bh = np.rint(0.5 * np.sum(cp * cp, axis=1)).astype(np.int64)
    return P, H, Ls, Bh


def hpart(x, H, Bh):
    xp = x.astype(np.int64) - 128
    return xp @ H.T - Bh[None, :]


def score(x, H, Ls, Bh):
    xp = x.astype(np.int64) - 128
    return 256 * hpart(x, H, Bh) + xp @ Ls.T


def centroids(rng, C, D):
    c = rng.uniform(0.0, 255.99, size=(C, D)).astype(np.float32)
    # values on and next to the rounding boundaries of the 1/256 grid
    k = rng.integers(0, 256 * 255, size=(C // 4, D))
    c[: C // 4] = ((k + 0.5) / 256.0).astype(np.float32)
    c[C // 4: C // 2] = np.nextafter(((k + 0.5) / 256.0).astype(np.float32), np.float32(300))
    c[0] = 0.0
    c[1] = np.float32(255.998)
    c[2] = np.float32(2.0 ** -60)  # c - 128 is not exact in fp64 (rounding slack of the bound)
    return c


def test_planes_are_int8_and_recompose():
    rng = np.random.default_rng(0)
    c = centroids(rng, 256, 64)
    P, H, Ls, _ = quantise(c)
    assert H.min() >= -128 and H.max() <= 127
    assert Ls.min() >= -128 and Ls.max() <= 127
    assert np.array_equal(256 * H + Ls + 128, P)


def test_score_error_within_bound_exact_arithmetic():
    rng = np.random.default_rng(1)
    D, C = 16, 40
    c = centroids(rng, C, D)
    x = rng.integers(0, 256, size=(30, D))
    x[0] = 0
    x[1] = 255
    _, H, Ls, B = quantise(c)
    s = score(x, H, Ls, B)
    cf = [[Fraction(float(v)) - 128 for v in row] for row in c]
    worst = Fraction(0)
    for i in range(x.shape[0]):
        xp = [int(v) - 128 for v in x[i]]
        sx = sum(xp)
        R1 = 129 + Fraction(sum(abs(v) for v in xp), 2)
        for j in range(C):
            k = sum(v * v for v in cf[j]) - 2 * sum(a * b for a, b in zip(xp, cf[j]))
            e = Fraction(int(s[i, j])) + 128 * k + 128 * sx
            assert abs(e) < R1, (i, j, float(e), float(R1))
            worst = max(worst, abs(e) / R1)
    # the bound is not vacuous: errors reach a good part of it
    assert worst > Fraction(1, 20)


def test_certificate_never_excludes_the_nearest():
    """On a wide random problem, whenever the best score beats the second by
    more than 2R the best-scored centroid is the exact nearest (fp64 direct
    distances), and whenever it beats the third by more than 2R the nearest
    is one of the two best scored."""
    rng = np.random.default_rng(2)
    D, C, N = 128, 300, 400
    c = centroids(rng, C, D)
    base = np.rint(c[rng.integers(0, C, N)]).clip(0, 255)
    x = np.clip(base + rng.integers(-3, 4, size=(N, D)), 0, 255).astype(np.int64)
    _, H, Ls, B = quantise(c)
    s = score(x, H, Ls, B)
    d = ((x[:, None, :].astype(np.float64) - c[None, :, :].astype(np.float64)) ** 2).sum(axis=2)
    l1 = np.abs(x - 128).sum(axis=1)
    twoR = 262 + l1
    order = np.argsort(-s, axis=1, kind="stable")
    top = np.take_along_axis(s, order[:, :3], axis=1)
    nearest = np.argmin(d, axis=1)
    n1 = n2 = 0
    for i in range(N):
        if top[i, 0] - top[i, 1] > twoR[i]:
            assert order[i, 0] == nearest[i]
            n1 += 1
        elif top[i, 0] - top[i, 2] > twoR[i]:
            assert nearest[i] in order[i, :2]
            n2 += 1
    assert n1 > N // 2


def test_prefilter_never_rejects_a_larger_score():
    """s <= 256 h + 128 ||x'||_1 for every row and centroid, so a group whose
    H values are all <= (k3 - 128 ||x'||_1) >> 8 holds no score above k3."""
    rng = np.random.default_rng(4)
    D = 96
    c = centroids(rng, 200, D)
    x = rng.integers(0, 256, size=(300, D))
    x[0] = 0
    x[1] = 255
    _, H, Ls, Bh = quantise(c)
    s = score(x, H, Ls, Bh)
    h = hpart(x, H, Bh)
    lmax = 128 * np.abs(x - 128).sum(axis=1)
    assert np.all(s <= 256 * h + lmax[:, None])
    k3 = np.sort(s, axis=1)[:, -3]
    t3 = (k3 - lmax) >> 8
    above = s > k3[:, None]
    assert np.all(h[above] > np.repeat(t3[:, None], s.shape[1], axis=1)[above])


def test_int32_headroom_at_the_largest_dimension():
    """D = 256 with every |x'| = 128 and P at both ends: the partial sums the
    kernel forms (x'.H - Bh shifted by 8, x'.Ls, and their sum) stay inside
    int32, above the padding score -2^31."""
    D = 256
    c = np.full((2, D), 0.0, np.float32)
    c[1] = np.float32(255.998)
    for xv in (0, 255):
        x = np.full((1, D), xv, np.int64)
        _, H, Ls, Bh = quantise(c)
        hi = 256 * hpart(x, H, Bh)
        lo = (x - 128) @ Ls.T
        for v in (hi, lo, hi + lo):
            assert np.abs(v).max() < 2 ** 31 - 2 ** 24
        assert hpart(x, H, Bh).min() > -(2 ** 23)


# ---------------------------------------------------------------- single plane

def _f32_up(v):
    f = np.float32(v)
    return float(np.nextafter(f, np.float32(np.inf))) if float(f) < v else float(f)


def quantise1(c):
    """One int8 plane, its biases, E and R2 rounded up to fp32 (as the
    kernel: R2 from the fp64 sum of squared residuals, its square root
    times 1 + 2^-40)."""
    cp = c.astype(np.float64) - 128.0
    H1 = np.rint(cp)
    assert np.all((H1 >= -128) & (H1 <= 127))
    b1 = np.rint(0.5 * np.sum(cp * cp, axis=1)).astype(np.int64)
    e = float(np.max(np.abs(cp - H1))) if c.size else 0.0
    r = float(np.max(np.sqrt(np.sum((cp - H1) ** 2, axis=1)))) if c.size else 0.0
    return H1.astype(np.int64), b1, _f32_up(e), _f32_up(r * (1.0 + 2.0 ** -40))


def window(x, E, R2):
    xp = x.astype(np.int64) - 128
    l1 = np.abs(xp).sum(axis=1)
    l2 = np.sqrt((xp * xp).sum(axis=1).astype(np.float64))
    return np.ceil(2.0 * np.minimum(E * l1, l2 * R2)).astype(np.int64) + 2


def test_single_plane_range_and_integer_centroids():
    """rint(c - 128) fits int8 for c in [-0.5, 255.5); integer centroids have
    E = 0; 255.5 rounds (half to even) to 128 and does not fit."""
    rng = np.random.default_rng(5)
    c = rng.uniform(-0.49, 255.49, size=(300, 40)).astype(np.float32)
    H1, _, E, R2 = quantise1(c)
    assert H1.min() >= -128 and H1.max() <= 127 and 0.0 < E <= 0.5 and 0.0 < R2 <= 0.5 * 40 ** 0.5 + 1e-6
    ci = rng.integers(0, 256, size=(50, 40)).astype(np.float32)
    assert quantise1(ci)[2:] == (0.0, 0.0)
    assert np.rint(np.float64(np.float32(255.5)) - 128.0) == 128.0


def test_single_plane_error_within_bound_exact_arithmetic():
    """|g - s1| <= min(E ||x'||_1, R2 ||x'||_2) + 1/2 in exact rational
    arithmetic (the second bound compared squared), including centroids on
    and next to the half-unit rounding boundaries; R2 bounds every residual
    norm; the kernel's window T exceeds twice the error."""
    rng = np.random.default_rng(6)
    D, C = 16, 40
    c = rng.uniform(0.0, 255.4, size=(C, D)).astype(np.float32)
    k = rng.integers(0, 255, size=(C // 4, D))
    c[: C // 4] = (k + 0.5).astype(np.float32)
    c[C // 4: C // 2] = np.nextafter((k + 0.5).astype(np.float32), np.float32(300))
    c[0] = 0.0
    c[1] = np.float32(2.0 ** -60)
    x = rng.integers(0, 256, size=(30, D))
    x[0] = 0
    x[1] = 255
    H1, b1, E, R2 = quantise1(c)
    s1 = (x - 128) @ H1.T - b1[None, :]
    T = window(x, E, R2)
    cf = [[Fraction(float(v)) - 128 for v in row] for row in c]
    for j in range(C):  # R2 bounds each residual norm
        assert sum((cf[j][d] - int(H1[j, d])) ** 2 for d in range(D)) <= Fraction(R2) ** 2
    worst = Fraction(0)
    for i in range(x.shape[0]):
        xp = [int(v) - 128 for v in x[i]]
        W1 = Fraction(E) * sum(abs(v) for v in xp)
        n2 = sum(v * v for v in xp)
        for j in range(C):
            g = sum(a * b for a, b in zip(xp, cf[j])) - sum(v * v for v in cf[j]) / 2
            e = abs(g - int(s1[i, j]))
            assert e <= W1 + Fraction(1, 2), (i, j, float(e), float(W1))
            if e > Fraction(1, 2):
                assert (e - Fraction(1, 2)) ** 2 <= n2 * Fraction(R2) ** 2, (i, j, float(e))
            assert 2 * e < int(T[i])
            worst = max(worst, e / (W1 + Fraction(1, 2)))
    assert worst > Fraction(1, 20)


def test_single_plane_certificate_never_excludes_the_nearest():
    """The kernel's decision on the single plane: the best-scored centroid
    when it beats the second by more than T, the nearest of the two best
    (fp64) when it beats the third by more than T, the two-plane screen
    otherwise. Settled rows carry the exact nearest centroid, for mean-like
    centroids (E near 1/2) and for integer ones (E = 0)."""
    rng = np.random.default_rng(7)
    D, C, N = 128, 300, 500
    for integer in (False, True):
        c = rng.uniform(0.0, 255.0, size=(C, D))
        c[1::3] = c[0::3][: len(c[1::3])] + rng.normal(0, 2.0, size=c[1::3].shape)  # near pairs
        c = np.clip(c, 0, 255).astype(np.float32)
        if integer:
            c = np.rint(c).astype(np.float32)
        base = np.rint(c[rng.integers(0, C, N)])
        x = np.clip(base + rng.integers(-20, 21, size=(N, D)), 0, 255).astype(np.int64)
        H1, b1, E, R2 = quantise1(c)
        s1 = (x - 128) @ H1.T - b1[None, :]
        T = window(x, E, R2)
        if not integer:  # the norm bound is the tighter one for mean-like centroids
            l1 = np.abs(x - 128).sum(axis=1)
            assert np.mean(T) < 0.85 * np.mean(np.ceil(2.0 * E * l1) + 2)
        d = ((x[:, None, :].astype(np.float64) - c[None, :, :].astype(np.float64)) ** 2).sum(axis=2)
        nearest = np.argmin(d, axis=1)
        order = np.argsort(-s1, axis=1, kind="stable")
        top = np.take_along_axis(s1, order[:, :3], axis=1)
        settled = 0
        for i in range(N):
            if top[i, 0] - top[i, 1] > T[i]:
                assert order[i, 0] == nearest[i]
                settled += 1
            elif top[i, 0] - top[i, 2] > T[i]:
                a, b = order[i, 0], order[i, 1]
                assert nearest[i] == (a if (d[i, a], a) <= (d[i, b], b) else b)
                settled += 1
        assert settled > N // 2


def test_single_plane_int32_headroom():
    """D = 128 with |x'| = 128 and H1 at both ends: |s1| < 2^23 (the padding
    bias -2^26 stays below every real score) and well inside int32."""
    D = 128
    c = np.stack([np.zeros(D), np.full(D, 255.4)]).astype(np.float32)
    H1, b1, _, _ = quantise1(c)
    for xv in (0, 255):
        x = np.full((1, D), xv, np.int64)
        s1 = (x - 128) @ H1.T - b1[None, :]
        assert np.abs(s1).max() < 2 ** 23


def _f32(v):
    return float(np.float32(v))


def test_route_key_bound_exact_arithmetic():
    """Routing of uint8-valued queries keys each centroid by -(float)s: its
    distance to 128 k + 128 sum(x') stays below B = (390 + ||x'||_1) / 2
    (the screening bound R = 131 + ||x'||_1 / 2 plus 64 for rounding s to
    fp32), including scores beyond 2^24 where the rounding is not exact."""
    rng = np.random.default_rng(7)
    for D in (16, 256):
        C = 24
        c = centroids(rng, C, D)
        c[3] = 0.0     # large ||c'||^2 and x'.c' magnitudes
        c[4] = 255.99
        x = rng.integers(0, 256, size=(12, D))
        x[0] = 0
        x[1] = 255
        _, H, Ls, Bh = quantise(c)
        s = score(x, H, Ls, Bh)
        assert np.abs(s).max() > 2 ** 24  # the fp32 rounding of s is exercised
        cf = [[Fraction(float(v)) - 128 for v in row] for row in c]
        for i in range(x.shape[0]):
            xp = [int(v) - 128 for v in x[i]]
            B = Fraction(390 + sum(abs(v) for v in xp), 2)
            for j in range(C):
                k = sum(v * v for v in cf[j]) - 2 * sum(a * b for a, b in zip(xp, cf[j]))
                key = Fraction(-_f32(int(s[i, j])))
                assert abs(key - (128 * k + 128 * sum(xp))) < B


def test_route_filter_thresholds_are_necessary():
    """The filter keeps -(float)s <= tau; its integer test s >= ceil(-tau - 64)
    and its prefilter h >= floor((-tau - 64 - 128 ||x'||_1) / 256) on the H
    plane (h = x'.H - Bh) never reject a score that passes."""
    import math

    rng = np.random.default_rng(8)
    D, C = 128, 64
    c = centroids(rng, C, D)
    x = rng.integers(0, 256, size=(8, D))
    _, H, Ls, Bh = quantise(c)
    s = score(x, H, Ls, Bh)
    h = hpart(x, H, Bh)
    l1 = np.abs(x.astype(np.int64) - 128).sum(axis=1)
    for i in range(x.shape[0]):
        for j in range(C):
            key = -_f32(int(s[i, j]))
            # thresholds at, just above and just below the key (fp32 grid)
            for tau in (key, _f32(np.nextafter(np.float32(key), np.float32(np.inf))),
                        _f32(np.nextafter(np.float32(key), np.float32(-np.inf)))):
                passes = key <= tau
                sthr = math.ceil(-tau - 64.0)
                t3 = math.floor((-tau - 64.0 - 128.0 * float(l1[i])) / 256.0)
                if passes:
                    assert int(s[i, j]) >= sthr and int(h[i, j]) >= t3
