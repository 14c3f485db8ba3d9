"""The int8 routing kernels (screen_i8.hip: the query check, the per-query
bounds, the keys of the threshold sample as group minima and the candidate
filter on the two int8 planes) built for the host against the wave64
emulation (tests/wave_emu) and run under AddressSanitizer, against the exact
integer arithmetic of the two-plane score
    s = 256 (x'.H - Bh) + x'.Ls,   x' = q - 128, P = rint(256 (c - 128)) = 256 H + Ls + 128,
with centroids on a grid of 1/4 so that Bh = rint(||c - 128||^2 / 2) is exact
whatever the summation order: the keys are -fl32(s), the group minima those of
16 consecutive sample centroids, the candidates every centroid with key <= tau
(as a set, with their keys), the bound (390 + ||x'||_1) / 2. Several
workgroups split each query tile's chunks, so ranges start mid-table. No GPU
is involved."""
import os
import subprocess

import numpy as np
import pytest

from test_emu_screen_i8 import CLANG, CSRC, HERE, strip_fences

NOT_WRITTEN = 0x7F7F7F7F


@pytest.fixture(scope="module")
def emu_route(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("clang++ of the ROCm toolchain not found")
    d = tmp_path_factory.mktemp("wave_emu_route")
    with open(os.path.join(CSRC, "screen_i8.hip")) as f:
        src = strip_fences(f.read())
    with open(d / "screen_i8_host_src.hip", "w") as f:
        f.write(src)
    exe = str(d / "route_i8_host")
    cmd = [CLANG, "-std=c++20", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
           "-I", os.path.join(HERE, "wave_emu"), "-I", str(d), "-I", CSRC,
           os.path.join(HERE, "wave_emu", "route_i8_host.cpp"), "-o", exe, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def run(exe, tmp_path, q, c, Cs, L, tau, num_cus=2, stride=1):
    Q, D = q.shape
    C = c.shape[0]
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        np.array([Q, C, D, Cs, L], np.int64).tofile(f)
        np.ascontiguousarray(q, np.float32).tofile(f)
        np.ascontiguousarray(c, np.float32).tofile(f)
        np.ascontiguousarray(tau, np.float32).tofile(f)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    r = subprocess.run([exe, str(src), str(dst), str(num_cus), str(stride)], capture_output=True, text=True,
                       timeout=900, env=env)
    assert r.returncode == 0 and "AddressSanitizer" not in r.stderr, r.stderr[-6000:]
    raw = np.fromfile(dst, np.uint8)
    o = 0

    def take(n, dt):
        nonlocal o
        v = raw[o: o + n * np.dtype(dt).itemsize].view(dt)
        o += n * np.dtype(dt).itemsize
        return v

    off, q_bad = int(take(1, np.uint32)[0]), int(take(1, np.uint32)[0])
    qbound = take(Q, np.float32)
    keys = take(Q * (Cs // 16), np.float32).reshape(Q, Cs // 16)
    cnt = take(Q, np.uint32)
    cand = take(Q * L * 2, np.uint32).reshape(Q, L, 2)
    return off, q_bad, qbound, keys, cnt, cand


def exact_scores(q, c):
    cp = c.astype(np.float64) - 128.0
    P = np.rint(256.0 * cp).astype(np.int64)
    H = P >> 8
    Ls = P - 256 * H - 128
    Bh = np.rint(0.5 * np.sum(cp * cp, axis=1)).astype(np.int64)
    xp = q.astype(np.int64) - 128
    return 256 * (xp @ H.T - Bh[None, :]) + xp @ Ls.T


def f32key(s):
    return -(s.astype(np.float32))


def case(Q, C, D, seed):
    rng = np.random.default_rng(seed)
    c = (rng.integers(0, 1021, size=(C, D)) / 4.0).astype(np.float32)  # 1/4 grid in [0, 255]
    c[0] = 0.0
    c[1] = 255.0
    q = rng.integers(0, 256, size=(Q, D)).astype(np.float32)
    q[0] = 0.0
    q[-1] = 255.0
    return q, c


def taus(s, rng):
    """Per query: the key of a random rank (5 .. 40), some +inf and -inf."""
    Q, C = s.shape
    keys = np.sort(f32key(s), axis=1)
    t = keys[np.arange(Q), rng.integers(5, min(40, C), size=Q)].copy()
    t[1] = np.inf
    t[2] = -np.inf
    return t


@pytest.mark.parametrize("Q,C,D,Cs,cus,stride", [(40, 300, 36, 128, 2, 2), (70, 200, 128, 64, 3, 3),
                                                 (33, 130, 256, 64, 2, 1), (20, 193, 96, 128, 4, 1)])
def test_emulated_route_keys_and_filter(emu_route, tmp_path, Q, C, D, Cs, cus, stride):
    """Keys of the threshold sample (contiguous, or the 64-centroid chunks
    j * stride spread over the table) and the candidate filter over every
    centroid."""
    q, c = case(Q, C, D, seed=Q + C + D)
    s = exact_scores(q, c)
    rng = np.random.default_rng(D)
    tau = taus(s, rng)
    L = C + 8
    off, q_bad, qbound, keys, cnt, cand = run(emu_route, tmp_path, q, c, Cs, L, tau, num_cus=cus, stride=stride)
    assert off == 0 and q_bad == 0
    l1 = np.abs(q.astype(np.int64) - 128).sum(axis=1)
    assert np.array_equal(qbound, (0.5 * (390 + l1)).astype(np.float32))
    sample = np.concatenate([np.arange(64 * j * stride, 64 * j * stride + 64) for j in range(Cs // 64)])
    assert sample[-1] < C
    gmin = f32key(s[:, sample].reshape(Q, Cs // 16, 16).max(axis=2))
    assert np.array_equal(keys.view(np.uint32), gmin.view(np.uint32))
    k = f32key(s)
    for i in range(Q):
        want = np.nonzero(k[i] <= tau[i])[0]
        assert int(cnt[i]) == want.size, (i, int(cnt[i]), want.size)
        got = cand[i, : want.size]
        order = np.argsort(got[:, 1])
        assert np.array_equal(got[order, 1], want)
        assert np.array_equal(got[order, 0], k[i, want].view(np.uint32))


def test_emulated_route_candidate_list_overflow(emu_route, tmp_path):
    """A list shorter than the candidates: the count is exact, the stored
    entries are valid candidates, nothing is written past the list."""
    q, c = case(30, 260, 64, seed=5)
    s = exact_scores(q, c)
    tau = np.full(30, np.inf, np.float32)
    off, _, _, _, cnt, cand = run(emu_route, tmp_path, q, c, 64, 17, tau)
    assert off == 0 and (cnt == 260).all()
    assert (cand[:, :, 1] < 260).all()


@pytest.mark.parametrize("bad", ["query", "centroid"])
def test_emulated_route_stands_down(emu_route, tmp_path, bad):
    """A non-integral query value or a centroid outside the planes' range
    raises the flag; the keys and the filter then write nothing."""
    q, c = case(25, 150, 64, seed=6)
    if bad == "query":
        q[7, 3] = 17.5
    else:
        c[9, 1] = 256.0
    tau = np.full(25, np.inf, np.float32)
    off, q_bad, _, keys, cnt, _ = run(emu_route, tmp_path, q, c, 64, 160, tau)
    assert off == 1 and q_bad == (1 if bad == "centroid" else 0)
    assert (keys.view(np.uint32) == NOT_WRITTEN).all() and (cnt == 0).all()
