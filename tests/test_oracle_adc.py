"""Pins for the oracle's residual-PQ ADC scan (CPU only).

On integer-valued data every fp32 operation is exact, so the approximate
distance equals the exact integer sum over subspaces of
||r_q^(m) - codeword||^2 with r_q = q - c_list; the result is checked against
Python integer brute force with the (distance, id) order. The order of the
probes does not matter, ids come from the probed lists, invalid probes are
skipped, and missing entries are padded."""
import numpy as np


def make(seed, B=6, C=9, D=8, M=4, N=300, P=3):
    rng = np.random.default_rng(seed)
    dsub = D // M
    c = rng.integers(-3, 4, (C, D)).astype(np.float32)
    q = rng.integers(-3, 4, (B, D)).astype(np.float32)
    cb = rng.integers(-3, 4, (M, 256, dsub)).astype(np.float32)
    lab = rng.integers(0, C, N).astype(np.int32)
    order = np.argsort(lab, kind="stable").astype(np.uint32)
    counts = np.bincount(lab, minlength=C)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    codes = rng.integers(0, 256, (N, M)).astype(np.uint8)
    probes = np.stack([rng.choice(C, P, replace=False) for _ in range(B)]).astype(np.int32)
    return q, c, probes, offsets, order, codes, cb


def brute(q, c, probes, offsets, perm, codes, cb, k):
    M, _, dsub = cb.shape
    ids, ds = [], []
    for b in range(q.shape[0]):
        cand = []
        for l in probes[b]:
            if not 0 <= l < c.shape[0]:
                continue
            r = [int(q[b, d]) - int(c[l, d]) for d in range(q.shape[1])]
            for p in range(offsets[l], offsets[l + 1]):
                tot = 0
                for m in range(M):
                    w = cb[m, codes[p, m]]
                    tot += sum((r[m * dsub + e] - int(w[e])) ** 2 for e in range(dsub))
                cand.append((tot, int(perm[p])))
        cand.sort()
        cand = cand[:k] + [(float("inf"), 0xFFFFFFFF)] * max(0, k - len(cand))
        ds.append([t[0] for t in cand])
        ids.append([t[1] for t in cand])
    return np.array(ids, np.uint32), np.array(ds, np.float64)


def test_adc_brute_force_exact_integers(oracle_mod):
    for seed in range(6):
        q, c, probes, offsets, perm, codes, cb = make(seed)
        for k in (1, 7, 40, 500):
            ids, dd = oracle_mod.adc_scan(q, c, probes, offsets, perm, codes, cb, k)
            bi, bd = brute(q, c, probes, offsets, perm, codes, cb, k)
            assert (ids == bi).all()
            assert (dd.astype(np.float64) == bd).all()


def test_probe_order_and_membership(oracle_mod):
    q, c, probes, offsets, perm, codes, cb = make(11, P=5)
    ids, dd = oracle_mod.adc_scan(q, c, probes, offsets, perm, codes, cb, 30)
    ids2, dd2 = oracle_mod.adc_scan(q, c, probes[:, ::-1].copy(), offsets, perm, codes, cb, 30)
    assert (ids == ids2).all() and (dd == dd2).all()
    for b in range(q.shape[0]):
        members = set()
        for l in probes[b]:
            members |= set(perm[offsets[l]:offsets[l + 1]].tolist())
        got = [i for i in ids[b].tolist() if i != 0xFFFFFFFF]
        assert set(got) <= members and len(set(got)) == len(got)


def test_invalid_probes_skipped_and_padding(oracle_mod):
    q, c, probes, offsets, perm, codes, cb = make(12, P=3)
    bad = probes.copy()
    bad[:, 1] = -1
    bad[0, 2] = 99
    ids, dd = oracle_mod.adc_scan(q, c, bad, offsets, perm, codes, cb, 400)
    bi, bd = brute(q, c, bad, offsets, perm, codes, cb, 400)
    assert (ids == bi).all() and (dd.astype(np.float64) == bd).all()
    assert (ids == 0xFFFFFFFF).any() and np.isinf(dd[ids == 0xFFFFFFFF]).all()


# ----------------------------------------------- fp32 rounding of the tables

def _r32(x):
    """Exact value x (a Fraction) rounded to the nearest fp32, ties to even."""
    from fractions import Fraction

    x = Fraction(x)
    f = np.float32(float(x))
    near = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    return min(near, key=lambda v: (abs(Fraction(float(v)) - x), int(np.array(v).view(np.uint32)) & 1))


def _read_adc_golden():
    import os

    path = os.path.join(os.path.dirname(__file__), "golden", "adc_fp32_rounding.txt")
    cases = []
    for line in open(path):
        line = line.split("#")[0].strip()
        if not line:
            continue
        name, dm, q, c, w, want = [f.strip() for f in line.split("|")]
        D, M = map(int, dm.split())
        cases.append((name, D, M, [float(v) for v in q.split()], [float(v) for v in c.split()],
                      [float(v) for v in w.split()], float(want)))
    return cases


def _reading(q, c, w, M, order=1, lut_f32=True, sum_f32=True, res_f32=True, sub_f64=True):
    """The ADC distance of one point whose codes are all 0, computed step by
    step in exact rational arithmetic with the roundings a reading puts in."""
    from fractions import Fraction as Fr

    D = len(q)
    dsub = D // M
    r = [(_r32(Fr(q[d]) - Fr(c[d])) if res_f32 else Fr(q[d]) - Fr(c[d])) for d in range(D)]
    r = [Fr(float(v)) if not isinstance(v, Fr) else v for v in r]
    luts = []
    for m in range(M):
        s = Fr(0)
        for e in range(dsub):
            t = r[m * dsub + e] - Fr(w[m * dsub + e])
            s = s + t * t if sub_f64 else Fr(float(_r32(s + Fr(float(_r32(t * t))))))
        luts.append(Fr(float(_r32(s))) if lut_f32 else s)
    acc = Fr(0)
    for v in luts[::order]:
        acc = Fr(float(_r32(acc + v))) if sum_f32 else acc + v
    return float(_r32(acc))


def test_adc_fp32_rounding_golden(oracle_mod):
    """Each golden case fixes one rounding of the reading: the oracle must give
    the listed d~ bit for bit, the reading worked out exactly must give it
    too, and the named other reading must give a different value (so that a
    change of order or precision in the oracle fails here)."""
    other = {
        "sum_order": [dict(sum_f32=False), dict(order=-1)],
        "lut_rounding": [dict(lut_f32=False, sum_f32=False)],
        "lut_fp64": [dict(sub_f64=False)],
        "residual_f32": [dict(res_f32=False)],
    }
    cases = _read_adc_golden()
    assert {c[0] for c in cases} == set(other)
    for name, D, M, q, c, w, want in cases:
        dsub = D // M
        cb = np.full((M, 256, dsub), 1e6, np.float32)
        for m in range(M):
            cb[m, 0] = w[m * dsub:(m + 1) * dsub]
        qa = np.array([q], np.float32)
        ca = np.array([c], np.float32)
        ids, dd = oracle_mod.adc_scan(qa, ca, np.zeros((1, 1), np.int32), np.array([0, 1], np.int64),
                                      np.zeros(1, np.uint32), np.zeros((1, M), np.uint8), cb, 1)
        assert ids[0, 0] == 0
        assert float(dd[0, 0]) == want, (name, float(dd[0, 0]), want)
        assert _reading(q, c, w, M) == want, name
        for alt in other[name]:
            assert _reading(q, c, w, M, **alt) != want, (name, alt)
