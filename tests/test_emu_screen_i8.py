"""The int8 screening kernels (screen_i8.hip: the two-plane screen alone, and
the single-plane screen followed by the two-plane screen of the rows it
leaves) built for the host against a wave64 emulation (tests/wave_emu: one
host thread per lane, the int8 MFMA's operand layout, barriers for the wave
and the block, asynchronous loads into LDS) and run under AddressSanitizer:
every row the screens settle carries the oracle's label, the others are
exactly the fallback worklist, and no access leaves its allocation. No GPU is
involved; this checks the kernels' arithmetic, indexing and synchronisation,
not the compiled gfx950 code."""
import os
import subprocess

import numpy as np
import pytest

import synth

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2608_08751_amd", "csrc")
CLANG = "/opt/rocm/llvm/bin/clang++"
UNWRITTEN = 0x7F7F7F7F


def strip_fences(src: str) -> str:
    """The source without its empty asm statements (scheduling fences for the
    GPU compiler; their register constraints do not exist on the host)."""
    out, i = [], 0
    while True:
        j = src.find("asm volatile(", i)
        if j < 0:
            out.append(src[i:])
            return "".join(out)
        out.append(src[i:j])
        k, depth = j + len("asm volatile("), 1
        while depth:
            depth += {"(": 1, ")": -1}.get(src[k], 0)
            k += 1
        assert src[k] == ";"
        i = k + 1


def dynamic_lds(src: str) -> str:
    """The source with each dynamic LDS array (extern __shared__) bound to the
    emulator's per-block dynamic LDS allocation."""
    import re

    pat = re.compile(r"extern __shared__ __attribute__\(\(aligned\(16\)\)\) unsigned char (\w+)\[\];")
    out, n = pat.subn(lambda m: "unsigned char *%s = emu::dyn_lds;" % m.group(1), src)
    assert n > 0
    return out


@pytest.fixture(scope="module")
def emu_bin(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("clang++ of the ROCm toolchain not found")
    d = tmp_path_factory.mktemp("wave_emu")
    with open(os.path.join(CSRC, "screen_i8.hip")) as f:
        src = strip_fences(f.read())
    with open(d / "screen_i8_host_src.hip", "w") as f:
        f.write(src)
    with open(os.path.join(CSRC, "fallback.hip")) as f:
        src = dynamic_lds(f.read())
    with open(d / "fallback_host_src.hip", "w") as f:
        f.write(src)
    exe = str(d / "screen_i8_host")
    cmd = [CLANG, "-std=c++20", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
           "-I", os.path.join(HERE, "wave_emu"), "-I", str(d), "-I", CSRC,
           os.path.join(HERE, "wave_emu", "screen_i8_host.cpp"), os.path.join(HERE, "wave_emu", "fallback_host.cpp"),
           "-o", exe, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def run(exe, tmp_path, x, c, num_cus=3, force_fallback=0, mode=0, force_rescreen=0, rescreen_cap=0,
        run_fallback=0, wl_cap=0, hints=None, order=None):
    N, D = x.shape
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        np.array([N, c.shape[0], D], np.int64).tofile(f)
        np.ascontiguousarray(x, np.uint8).tofile(f)
        np.ascontiguousarray(c, np.float32).tofile(f)
    extra = []
    if hints is not None:
        hp = tmp_path / "hints.bin"
        np.ascontiguousarray(hints, np.int32).tofile(hp)
        extra = [str(hp)]
    if order is not None:
        extra = extra or ["-"]
        if isinstance(order, str):
            extra.append(order)
        else:
            op = tmp_path / "order.bin"
            np.ascontiguousarray(order, np.uint32).tofile(op)
            extra.append(str(op))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    r = subprocess.run([exe, str(src), str(dst), str(num_cus), str(force_fallback), str(mode),
                        str(force_rescreen), str(rescreen_cap), str(run_fallback), str(wl_cap)] + extra,
                       capture_output=True, text=True, timeout=900, env=env)
    assert r.returncode == 0 and "AddressSanitizer" not in r.stderr, r.stderr[-6000:]
    raw = np.fromfile(dst, np.uint8)
    lab = raw[: 4 * N].view(np.int32)
    n = int(raw[4 * N: 4 * N + 4].view(np.uint32)[0])
    o = 4 * N + 4
    wl = raw[o: o + 4 * n].view(np.int32)
    o += 4 * n
    stats = raw[o: o + 64].view(np.uint64)
    q_bad = int(raw[o + 64: o + 68].view(np.uint32)[0])
    run.q_bad1 = int(raw[o + 68: o + 72].view(np.uint32)[0])
    run.listed = int(raw[o + 72: o + 76].view(np.uint32)[0])
    return lab, wl, stats, q_bad


def rows_and_centroids(N, C, D, seed):
    rng = np.random.default_rng(seed)
    means = rng.uniform(0.0, 255.0, size=(max(C // 2, 1), D)).astype(np.float32)
    x, _ = synth.mixture_rows_u8(means, 0, N, seed=seed)
    if C <= N:
        c = x[rng.choice(N, C, replace=False)].astype(np.float32)
    else:
        c = rng.uniform(0.0, 255.0, size=(C, D)).astype(np.float32)
    c += rng.uniform(-0.5, 0.5, size=c.shape).astype(np.float32)
    np.clip(c, 0.0, 255.0, out=c)
    return x, c


def check(oracle_mod, lab, wl, stats, x, c):
    olab = oracle_mod.assign(x, c)
    assert not (lab == UNWRITTEN).any(), "labels never written"
    fb = np.nonzero(lab == -1)[0]
    assert np.array_equal(np.sort(wl), fb), "worklist differs from the unsettled rows"
    settled = lab != -1
    bad = np.nonzero(lab[settled] != olab[settled])[0]
    assert bad.size == 0, "labels differ at rows %s" % np.nonzero(settled)[0][bad[:10]]
    assert int(stats[0]) == fb.size and int(stats[5]) == 1


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("N,C,D,cus", [(1500, 130, 128, 3), (700, 3, 96, 2), (1100, 65, 256, 3), (600, 70, 36, 1),
                                       (900, 530, 64, 2)])
def test_emulated_screen_matches_oracle(emu_bin, tmp_path, oracle_mod, N, C, D, cus, mode):
    """Several row tiles per workgroup (persistent loop), ragged last tiles,
    C not a multiple of the 64-centroid chunk, and each padded width; mode 1
    runs the single plane first (padded widths up to 128; C = 530 spans three
    of its 256-centroid staged chunks, the last one ragged)."""
    x, c = rows_and_centroids(N, C, D, seed=N + C + D)
    lab, wl, stats, q_bad = run(emu_bin, tmp_path, x, c, num_cus=cus, mode=mode)
    assert q_bad == 0
    check(oracle_mod, lab, wl, stats, x, c)
    if mode == 1 and D <= 128:
        # non-integer centroids: some rows need the finer two planes
        assert run.q_bad1 == 0 and run.listed == int(stats[6]) and run.listed < N


def test_emulated_single_plane_integer_centroids(emu_bin, tmp_path, oracle_mod):
    """Integer-valued centroids (rows sampled as the k-means initialisation):
    E = 0, the single plane settles every row that has no tie within one unit."""
    x, _ = rows_and_centroids(1200, 90, 128, seed=3)
    rng = np.random.default_rng(4)
    c = x[rng.choice(1200, 90, replace=False)].astype(np.float32)
    lab, wl, stats, _ = run(emu_bin, tmp_path, x, c, mode=1)
    check(oracle_mod, lab, wl, stats, x, c)
    assert run.listed <= 12


@pytest.mark.parametrize("mode", [0, 1])
def test_emulated_near_ties(emu_bin, tmp_path, oracle_mod, mode):
    """Pairs of nearly equal centroids (two candidates: the exact fp64
    evaluation) and crowds of five (the fallback worklist)."""
    rng = np.random.default_rng(11)
    D = 64
    pa = rng.integers(20, 236, size=(15, D)).astype(np.float32)
    cr = rng.integers(20, 236, size=(15, D)).astype(np.float32)
    c = np.vstack([pa, pa + 1e-3, cr, cr.copy(), cr + 1e-3, cr - 1.0 / 512, cr + 0.5]).astype(np.float32)
    x = np.vstack([np.rint(pa), np.rint(pa + 0.25), np.rint(cr), rng.integers(0, 256, size=(200, D))])
    x = np.clip(x, 0, 255).astype(np.uint8)
    lab, wl, stats, _ = run(emu_bin, tmp_path, x, c, mode=mode)
    check(oracle_mod, lab, wl, stats, x, c)
    assert int(stats[0]) > 0 and int(stats[1]) > 0


@pytest.mark.parametrize("force_rescreen,cap", [(1, 0), (0, 1), (1, 5)])
def test_emulated_rescreen_forced_and_overflow(emu_bin, tmp_path, oracle_mod, force_rescreen, cap):
    """Every row listed for the two planes; a list of one or five entries
    that overflows (the two planes then screen every row)."""
    x, c = rows_and_centroids(900, 75, 100, seed=8)
    lab, wl, stats, _ = run(emu_bin, tmp_path, x, c, mode=1, force_rescreen=force_rescreen, rescreen_cap=cap)
    check(oracle_mod, lab, wl, stats, x, c)
    if force_rescreen:
        assert run.listed == 900 and int(stats[6]) == 900
    else:
        assert run.listed > cap


def test_emulated_single_plane_unquantisable(emu_bin, tmp_path, oracle_mod):
    """A coordinate of 255.7 rounds to 128 on the single plane (outside int8)
    but fits the two planes: the single plane stands down, the two planes
    screen every row."""
    x, c = rows_and_centroids(700, 50, 128, seed=9)
    c[11, 5] = 255.7
    lab, wl, stats, q_bad = run(emu_bin, tmp_path, x, c, mode=1)
    assert q_bad == 0 and run.q_bad1 == 1 and run.listed == 0
    check(oracle_mod, lab, wl, stats, x, c)


def test_emulated_forced_fallback_and_unquantisable(emu_bin, tmp_path, oracle_mod):
    x, c = rows_and_centroids(800, 40, 128, seed=5)
    lab, wl, stats, _ = run(emu_bin, tmp_path, x, c, force_fallback=1)
    assert (lab == -1).all() and np.array_equal(np.sort(wl), np.arange(800)) and int(stats[0]) == 800
    c[7, 3] = 256.0  # outside the 16-bit fixed point: the kernel stands down
    lab, wl, stats, q_bad = run(emu_bin, tmp_path, x, c)
    assert q_bad == 1 and (lab == UNWRITTEN).all() and wl.size == 0 and int(stats[5]) == 0


@pytest.mark.parametrize("mode,force_fallback,wl_cap,N", [
    (0, 0, 3, 300),   # the worklist overflows: the scan for labels of -1 finds the rows
    (0, 1, 0, 120),   # every row listed: centroid-split windows and their merge
    (1, 1, 5, 300),   # every row through both planes, overflowing worklist
])
def test_emulated_pipeline_with_fallback(emu_bin, tmp_path, oracle_mod, mode, force_fallback, wl_cap, N):
    """The screens followed by the exact fallback scan (fallback.hip), in the
    library's order: every row ends with the oracle's label. The worklist
    either holds every row the screens hand on, or overflows (capacity 1, 3,
    5 or 100), in which case the fallback finds the rows by their labels of
    -1; every row forced through the fallback covers the centroid-split
    windows, their merge and the whole-row windows. Under AddressSanitizer,
    with the dynamic LDS of every block a fresh allocation."""
    rng = np.random.default_rng(N + wl_cap)
    D = 64
    pa = rng.integers(20, 236, size=(20, D)).astype(np.float32)
    c = np.vstack([pa, pa + 1e-3, pa + 0.5, rng.uniform(0, 255, size=(97, D))]).astype(np.float32)
    x = np.vstack([np.rint(pa), np.rint(pa + 0.25), rng.integers(0, 256, size=(N - 40, D))])
    x = np.clip(x, 0, 255).astype(np.uint8)
    lab, wl, st, _ = run(emu_bin, tmp_path, x, c, num_cus=2, force_fallback=force_fallback, mode=mode,
                         run_fallback=1, wl_cap=wl_cap)
    handed = int(st[0])  # rows the screens handed to the fallback
    assert handed > 0
    if wl_cap:
        assert handed > wl_cap  # the worklist overflowed
    if force_fallback:
        assert handed == N
    olab = oracle_mod.assign(x, c)
    bad = np.nonzero(lab != olab)[0]
    assert bad.size == 0, "labels differ at rows %s" % bad[:10]


def test_emulated_single_plane_with_hints(emu_bin, tmp_path, oracle_mod):
    """Hinted labels (speed only) start each row's keep threshold from the
    hinted centroid's score: the exact labels, garbage (out of range,
    negative, random) and a mix give the same settled labels, worklist and
    rescreen list as no hints."""
    x, c = rows_and_centroids(500, 140, 128, seed=12)
    lab0, wl0, st0, _ = run(emu_bin, tmp_path, x, c, mode=1)
    listed0 = run.listed
    check(oracle_mod, lab0, wl0, st0, x, c)
    olab = oracle_mod.assign(x, c).astype(np.int32)
    rng = np.random.default_rng(13)
    garbage = rng.integers(-5, 200, size=500).astype(np.int32)
    garbage[:10] = np.iinfo(np.int32).min
    for hints in (olab, garbage, np.where(rng.random(500) < 0.5, olab, garbage).astype(np.int32)):
        lab, wl, st, _ = run(emu_bin, tmp_path, x, c, mode=1, hints=hints)
        check(oracle_mod, lab, wl, st, x, c)
        assert np.array_equal(lab, lab0) and np.array_equal(np.sort(wl), np.sort(wl0))
        assert run.listed == listed0 and int(st[1]) == int(st0[1])


@pytest.mark.parametrize("case", ["mixture", "ties"])
def test_emulated_single_plane_visiting_order(emu_bin, tmp_path, oracle_mod, case):
    """The single plane in another visiting order (plane row p holds centroid
    ord[p]): a random permutation (with and without hint labels, which then
    go through the positions) and the library's own order (its keys kernel,
    then a stable sort by key, without hints) settle the same rows with the same labels,
    hand on the same rows and count the same refinements as id order. C = 300
    spans two staged chunks, the second ragged; pairs and crowds of equal and
    nearly equal centroids put equal scores in different plane-row order."""
    if case == "mixture":
        x, c = rows_and_centroids(300, 300, 64, seed=21)
    else:
        rng = np.random.default_rng(22)
        D = 64
        pa = rng.integers(20, 236, size=(12, D)).astype(np.float32)
        cr = rng.integers(20, 236, size=(12, D)).astype(np.float32)
        c = np.vstack([pa, pa + 1e-3, cr, cr.copy(), cr + 1e-3, cr - 1.0 / 512, cr + 0.5,
                       rng.uniform(0, 255, size=(60, D))]).astype(np.float32)
        x = np.vstack([np.rint(pa), np.rint(pa + 0.25), np.rint(cr), rng.integers(0, 256, size=(100, D))])
        x = np.clip(x, 0, 255).astype(np.uint8)
    C = c.shape[0]
    lab0, wl0, st0, _ = run(emu_bin, tmp_path, x, c, mode=1)
    listed0 = run.listed
    check(oracle_mod, lab0, wl0, st0, x, c)
    rng = np.random.default_rng(23)
    perm = rng.permutation(C).astype(np.uint32)
    olab = oracle_mod.assign(x, c).astype(np.int32)
    for order, hints in ((perm, None), (perm, olab), ("auto", None)):
        lab, wl, st, _ = run(emu_bin, tmp_path, x, c, mode=1, order=order, hints=hints)
        check(oracle_mod, lab, wl, st, x, c)
        assert np.array_equal(lab, lab0) and np.array_equal(np.sort(wl), np.sort(wl0))
        assert run.listed == listed0 and int(st[1]) == int(st0[1]) and int(st[6]) == int(st0[6])
