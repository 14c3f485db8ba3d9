"""The cell-and-walk assignment kernel and the candidate-restricted kernels
(assign_graph.hip) built for the host against the wave64 emulation
(tests/wave_emu) and run under AddressSanitizer: labels equal to the oracle's and distances equal to its
fp64 distance rounded to fp32, on tiles whose rows share one cell (the
shared-member path, rows in cell order) and tiles that mix cells (random
order), with dead slots, invalid cells and members, empty cells, cells of
more than 64 members, ties, D = 4 ... 256 (three or four waves a block), and
grids smaller and larger than the number of tiles; no access leaves its
allocation. No GPU is involved."""
import os
import subprocess

import numpy as np
import pytest

from test_emu_screen_i8 import CLANG, CSRC, HERE, dynamic_lds

UNWRITTEN = 0x7F7F7F7F


@pytest.fixture(scope="module")
def emu_cells(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("clang++ of the ROCm toolchain not found")
    d = tmp_path_factory.mktemp("wave_emu_cells")
    with open(os.path.join(CSRC, "assign_graph.hip")) as f:
        src = dynamic_lds(f.read())
    with open(d / "assign_graph_host_src.hip", "w") as f:
        f.write(src)
    exe = str(d / "assign_cells_host")
    cmd = [CLANG, "-std=c++20", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
           "-I", os.path.join(HERE, "wave_emu"), "-I", str(d), "-I", CSRC,
           os.path.join(HERE, "wave_emu", "assign_cells_host.cpp"), "-o", exe, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def run(exe, tmp_path, x, c, cell, offsets, members, graph, hops, order=None, num_cus=2):
    N, D = x.shape
    C = c.shape[0]
    S = 0 if graph is None else graph.shape[1]
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    hdr = [N, C, D, len(offsets) - 1, len(members), S, hops, 0 if x.dtype == np.uint8 else 1,
           graph is not None, order is not None]
    with open(src, "wb") as f:
        f.write(np.array(hdr, np.int64).tobytes())
        f.write(np.ascontiguousarray(x).tobytes())
        f.write(np.ascontiguousarray(c, np.float32).tobytes())
        f.write(np.ascontiguousarray(cell, np.int32).tobytes())
        f.write(np.ascontiguousarray(offsets, np.int64).tobytes())
        f.write(np.ascontiguousarray(members, np.uint32).tobytes())
        if graph is not None:
            f.write(np.ascontiguousarray(graph, np.int32).tobytes())
        if order is not None:
            f.write(np.ascontiguousarray(order, np.uint32).tobytes())
    r = subprocess.run([exe, str(src), str(dst), str(num_cus)], capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stderr[-4000:]
    out = np.fromfile(dst, np.uint8)
    return out[:4 * N].view(np.int32), out[4 * N:].view(np.float32)


def cells(rng, C, G, extra_invalid=0):
    members = rng.permutation(C).astype(np.uint32)
    if extra_invalid:
        members = np.concatenate([members, rng.integers(C, C + 50, extra_invalid).astype(np.uint32)])
        members = members[rng.permutation(members.size)]
    cuts = np.sort(rng.integers(0, members.size + 1, G - 1))
    return np.concatenate([[0], cuts, [members.size]]).astype(np.int64), members


def check(exe, tmp_path, oracle_mod, x, c, cell, offsets, members, graph, hops, order, num_cus):
    lab, dist = run(exe, tmp_path, x, c, cell, offsets, members, graph, hops, order, num_cus)
    olab, od = oracle_mod.assign_cells(x, c, cell, offsets, members, graph, hops, return_dist=True)
    N = x.shape[0]
    done = np.arange(N) if order is None else np.unique(order[order < N]).astype(np.int64)
    left = np.setdiff1d(np.arange(N), done)
    assert (lab[done] == olab[done]).all()
    assert (dist[done] == od[done].astype(np.float32)).all()
    assert (lab[left] == UNWRITTEN).all() and (dist[left].view(np.int32) == UNWRITTEN).all()
    return lab


@pytest.mark.parametrize("N,C,D,G,S,hops,dt,cus", [
    (203, 90, 128, 5, 5, 3, "u8", 2), (100, 70, 256, 3, 8, 2, "f32", 1), (77, 300, 4, 2, 3, 4, "f32", 40),
    (130, 40, 36, 4, 17, 1, "u8", 3),
])
def test_emulated_assign_cells(emu_cells, tmp_path, oracle_mod, N, C, D, G, S, hops, dt, cus):
    rng = np.random.default_rng(N + D)
    if dt == "u8":
        x = rng.integers(0, 256, (N, D)).astype(np.uint8)
        c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    else:
        x = rng.standard_normal((N, D)).astype(np.float32)
        c = rng.standard_normal((C, D)).astype(np.float32)
    offsets, members = cells(rng, C, G)
    graph = rng.integers(0, C, (C, S)).astype(np.int32)
    cell = rng.integers(0, G, N).astype(np.int32)
    by_cell = np.argsort(cell, kind="stable")
    for order in (by_cell, rng.permutation(N), None):
        check(emu_cells, tmp_path, oracle_mod, x, c, cell, offsets, members, graph, hops, order, cus)


def test_emulated_assign_cells_dead_slots_and_invalid(emu_cells, tmp_path, oracle_mod):
    """Cell-ordered tiles with order entries past N among their rows (dead
    slots in a shared tile), rows of invalid cells, an empty cell, invalid
    member and graph ids, and many exact ties."""
    rng = np.random.default_rng(3)
    N, C, D = 150, 40, 8
    x = rng.integers(0, 3, (N, D)).astype(np.uint8)
    c = rng.integers(0, 3, (C, D)).astype(np.float32)
    offsets, members = cells(rng, C, 6, extra_invalid=15)
    offsets[3] = offsets[2]
    graph = rng.integers(-3, 45, (C, 12)).astype(np.int32)
    cell = rng.integers(0, 6, N).astype(np.int32)
    cell[rng.choice(N, 9, replace=False)] = rng.choice([-2, -1, 6, 7], 9)
    order = np.argsort(cell, kind="stable").astype(np.int64)
    order[rng.choice(N, 12, replace=False)] = N + np.arange(12)
    for g, hops in ((graph, 5), (None, 2)):
        lab = check(emu_cells, tmp_path, oracle_mod, x, c, cell, offsets, members, g, hops, order, 2)
        assert (lab == -1).any()


def test_emulated_assign_cells_large_cells(emu_cells, tmp_path, oracle_mod):
    """Cells of 64, 65 and 150 members: lanes take one, and several, members
    each on the shared path."""
    rng = np.random.default_rng(9)
    N, C, D = 96, 279, 16
    x = rng.standard_normal((N, D)).astype(np.float32)
    c = rng.standard_normal((C, D)).astype(np.float32)
    members = rng.permutation(C).astype(np.uint32)
    offsets = np.array([0, 64, 129, 279], np.int64)
    cell = np.repeat(np.arange(3), 32).astype(np.int32)
    graph = rng.integers(0, C, (C, 6)).astype(np.int32)
    check(emu_cells, tmp_path, oracle_mod, x, c, cell, offsets, members, graph, 3, None, 1)


def run_graph(exe, tmp_path, x, c, graph, prev, order=None):
    """ivf_assign_graph's kernels on the emulation (a header with G = 0)."""
    return run(exe, tmp_path, x, c, prev, np.zeros(1, np.int64), np.zeros(0, np.uint32), graph, 0, order)


@pytest.mark.parametrize("N,C,D,S,labels_used,dt", [
    (300, 40, 128, 8, 10, "u8"), (200, 30, 36, 12, 4, "f32"), (130, 50, 8, 3, 50, "u8"), (150, 20, 16, 17, 3, "f32"),
])
def test_emulated_assign_graph(emu_cells, tmp_path, oracle_mod, N, C, D, S, labels_used, dt):
    """Rows grouped by previous label (labels covering whole waves: the
    shared-candidate passes), random order (the one-lane-per-row rows), row
    order; invalid previous labels and graph ids; S = 17 takes the lane-group
    kernel."""
    rng = np.random.default_rng(N + S)
    if dt == "u8":
        x = rng.integers(0, 256, (N, D)).astype(np.uint8)
        c = rng.uniform(0, 255, (C, D)).astype(np.float32)
    else:
        x = rng.standard_normal((N, D)).astype(np.float32)
        c = rng.standard_normal((C, D)).astype(np.float32)
    graph = rng.integers(-2, C + 2, (C, S)).astype(np.int32)
    prev = rng.integers(0, labels_used, N).astype(np.int32)
    prev[rng.choice(N, 5, replace=False)] = rng.choice([-3, -1, C, C + 7], 5)
    olab, od = oracle_mod.assign_graph(x, c, graph, prev, return_dist=True)
    by_prev = np.argsort(prev, kind="stable")
    for order in (by_prev, rng.permutation(N), None):
        lab, dist = run_graph(emu_cells, tmp_path, x, c, graph, prev, order)
        assert (lab == olab).all()
        assert (dist == od.astype(np.float32)).all()
    assert (olab == -1).any()
