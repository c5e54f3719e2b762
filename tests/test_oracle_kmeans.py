"""Pins of the CPU oracle's kernel-level k-means (Sec. 3.1, Eq. 1) to things
other than itself: exact rational arithmetic on tiny inputs, closed forms,
fixed points, the monotonicity of Lloyd's objective, and scikit-learn's Lloyd
k-means on inputs where both definitions coincide."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

U32 = 2.0 ** -24  # unit roundoff of fp32


def exact_d(x, c):
    return sum((Fraction(float(a)) - Fraction(float(b))) ** 2 for a, b in zip(x, c))


def exact_assign(X, C):
    """Exact squared distances (rationals), argmin with ties to the lowest index."""
    idx, best, second = [], [], []
    for x in X:
        ds = [exact_d(x, c) for c in C]
        m = min(ds)
        idx.append(ds.index(m))
        rest = sorted(ds)
        best.append(m)
        second.append(rest[1] if len(rest) > 1 else None)
    return np.array(idx), best, second


def tiny_cases():
    rng = np.random.default_rng(11)
    for t in range(12):
        n = int(rng.integers(1, 64))
        k = int(rng.integers(1, 9))
        X = rng.standard_normal((n, 9)).astype(np.float32)
        C = rng.standard_normal((k, 9)).astype(np.float32)
        yield X, C
    # small integers: every fp32 and fp64 distance is exact, and ties are planted
    for t in range(6):
        n, k = 40, 6
        X = rng.integers(-3, 4, (n, 9)).astype(np.float32)
        C = rng.integers(-3, 4, (k, 9)).astype(np.float32)
        C[3] = C[1]          # duplicate entries: the lower index must win
        yield X, C


@pytest.mark.parametrize("case", list(range(18)))
def test_assign_equals_exact_bruteforce(case):
    X, C = list(tiny_cases())[case]
    ref_idx, best, second = exact_assign(X, C)
    out = oracle.assign(X, C)
    # fp64 decision: exact except where the exact gap is below fp64 resolution
    for i in range(X.shape[0]):
        if out["idx64"][i] != ref_idx[i]:
            assert exact_d(X[i], C[out["idx64"][i]]) - best[i] <= Fraction(1, 10 ** 12) * best[i]
        assert abs(Fraction(out["d1"][i]) - best[i]) <= Fraction(2 ** -50) * best[i]
        if second[i] is not None:
            assert abs(Fraction(out["d2"][i]) - second[i]) <= Fraction(2 ** -50) * second[i]
        else:
            assert np.isinf(out["d2"][i])
    # fp32 decision: the exact winner unless the exact gap is within fp32 error
    for i in range(X.shape[0]):
        j = out["idx"][i]
        if j != ref_idx[i]:
            gap = exact_d(X[i], C[j]) - best[i]
            assert gap <= Fraction(24 * U32) * exact_d(X[i], C[j])
        d_exact = best[i] if j == ref_idx[i] else exact_d(X[i], C[j])
        assert abs(Fraction(float(out["d32"][i])) - d_exact) <= Fraction(12 * U32) * d_exact


def test_assign_planted_ties_lowest_index():
    X = np.zeros((3, 9), np.float32)
    X[1, 0] = 1.0
    X[2, :] = 0.5
    C = np.zeros((4, 9), np.float32)
    C[0, 0] = 1.0
    C[1, 1] = 1.0     # distance to X[0] equals that of entry 0
    C[2, 0] = 1.0     # duplicate of entry 0
    C[3, :] = 1.0
    out = oracle.assign(X, C)
    assert out["idx"].tolist() == [0, 0, 0]
    assert out["idx64"].tolist() == [0, 0, 0]
    assert out["d1"][1] == 0.0 and out["d2"][1] == 0.0      # entries 0 and 2 coincide
    assert out["d32"][2] == np.float32(2.25)                 # every entry is at 9 * 0.5^2: exact


def exact_mean_f32(rows):
    s = [sum(Fraction(float(r[d])) for r in rows) / len(rows) for d in range(9)]
    return s


def test_update_equals_exact_means():
    rng = np.random.default_rng(5)
    for t in range(8):
        n, k = int(rng.integers(1, 80)), int(rng.integers(1, 10))
        X = rng.standard_normal((n, 9)).astype(np.float32)
        idx = rng.integers(0, k, n).astype(np.int32)
        C_old = rng.standard_normal((k, 9)).astype(np.float32)
        C_new, counts = oracle.update(X, idx, C_old)
        assert counts.tolist() == np.bincount(idx, minlength=k).tolist()
        for j in range(k):
            rows = X[idx == j]
            if len(rows) == 0:
                assert np.array_equal(C_new[j], C_old[j])     # empty set keeps its entry
                continue
            m = exact_mean_f32(rows)
            for d in range(9):
                # one fp32 rounding of an fp64 value within a few fp64 ulps of the exact mean
                err = abs(Fraction(float(C_new[j, d])) - m[d])
                assert err <= Fraction(float(np.spacing(np.float32(abs(float(m[d])))))) * Fraction(1, 2) \
                    + Fraction(2 ** -40) * abs(m[d]) + Fraction(2 ** -140)


def test_update_rejects_bad_index():
    X = np.zeros((4, 9), np.float32)
    with pytest.raises(ValueError):
        oracle.update(X, np.array([0, 1, 5, 0], np.int32), np.zeros((3, 9), np.float32))


def exact_lloyd_step(X, C32):
    """One exact step from an fp32 codebook: exact assignment, exact means."""
    idx, best, second = exact_assign(X, C32)
    means = {}
    for j in range(C32.shape[0]):
        rows = X[idx == j]
        means[j] = exact_mean_f32(rows) if len(rows) else None
    return idx, best, second, means


def test_fit_step_locked_with_exact_lloyd():
    """Every oracle iteration equals an exact-arithmetic Lloyd step taken from the
    oracle's own fp32 codebook (well-separated data, so no near-ties)."""
    rng = np.random.default_rng(3)
    centers = rng.standard_normal((5, 9)) * 4
    X = (centers[rng.integers(0, 5, 60)] + 0.3 * rng.standard_normal((60, 9))).astype(np.float32)
    C = X[synth.distinct_init(X, 5, 3)]
    iters = 4
    ref = oracle.fit(X, C, iters)
    state = C.copy()
    for t in range(iters + 1):
        idx, best, _, means = exact_lloyd_step(X, state)
        o = oracle.assign(X, state)
        assert np.array_equal(o["idx"], idx)
        Jt = sum(best)
        assert abs(Fraction(ref["J"][t]) - Jt) <= Fraction(2 ** -40) * Jt
        if t == iters:
            assert np.array_equal(ref["idx"], idx)
            assert ref["counts"].tolist() == np.bincount(idx, minlength=5).tolist()
            break
        nxt, _ = oracle.update(X, idx, state)
        for j, m in means.items():
            if m is None:
                assert np.array_equal(nxt[j], state[j])
            else:
                assert np.allclose(nxt[j].astype(np.float64), [float(v) for v in m], rtol=2 * U32, atol=0)
        state = nxt
    assert np.array_equal(ref["C"], state)


def test_fit_monotone_distortion():
    """Lloyd never increases Eq. (1): J_{t+1} <= J_t (up to fp64 summation noise)."""
    for L in (synth.single_layer(k=64)[0], synth.resnet18_stack(k=16, layers=1)[0],
              synth.stress_layer(n=4096, k=128, n_centers=64)[0]):
        r = oracle.fit(L.X, L.C0, 8)
        J = r["J"]
        assert np.all(J[1:] <= J[:-1] * (1 + 1e-12)), J


def test_fit_fixed_point_distinct_kernels():
    """A codebook equal to all distinct kernels is a fixed point with J = 0."""
    rng = np.random.default_rng(8)
    base = rng.standard_normal((20, 9)).astype(np.float32)
    X = base[rng.integers(0, 20, 200)]
    k = synth.n_distinct(X)
    sel = synth.distinct_init(X, k, 1)
    C = X[sel]
    r = oracle.fit(X, C, 1)
    assert np.array_equal(r["C"], C)
    assert r["J"].tolist() == [0.0, 0.0]
    assert np.array_equal(C[r["idx"]], X)


def test_fit_single_entry_closed_form():
    """k = 1: the entry is the global mean and J is the total scatter."""
    X = synth.normal_layer(16, 32, 9)
    r = oracle.fit(X, X[:1], 2)
    mu = X.astype(np.float64).mean(axis=0)
    assert np.allclose(r["C"][0], mu, rtol=1e-6, atol=1e-9)
    scatter = float(((X.astype(np.float64) - r["C"][0].astype(np.float64)) ** 2).sum())
    assert r["J"][-1] == pytest.approx(scatter, rel=1e-12)
    assert np.all(r["idx"] == 0)


def test_fit_planted_clusters():
    """Two far-apart planted groups: the fitted entries are the group means."""
    rng = np.random.default_rng(4)
    a = (rng.standard_normal((50, 9)) * 0.1 + 10).astype(np.float32)
    b = (rng.standard_normal((70, 9)) * 0.1 - 10).astype(np.float32)
    X = np.concatenate([a, b])
    C0 = np.stack([a[0], b[0]])
    r = oracle.fit(X, C0, 3)
    assert np.allclose(r["C"][0], a.astype(np.float64).mean(0), rtol=1e-6)
    assert np.allclose(r["C"][1], b.astype(np.float64).mean(0), rtol=1e-6)
    assert r["counts"].tolist() == [50, 70]


def test_fit_matches_sklearn_lloyd():
    """scikit-learn's Lloyd k-means from the same initial codebook reaches the same
    labels and centres (data with separated clusters, so no empty cluster or tie)."""
    sk = pytest.importorskip("sklearn.cluster")
    rng = np.random.default_rng(21)
    centers = rng.standard_normal((8, 9)) * 3
    X = (centers[rng.integers(0, 8, 2000)] + 0.5 * rng.standard_normal((2000, 9))).astype(np.float32)
    C0 = X[synth.distinct_init(X, 8, 2)]
    r = oracle.fit(X, C0, 50)
    km = sk.KMeans(n_clusters=8, init=C0.astype(np.float64), n_init=1, max_iter=50, tol=0.0,
                   algorithm="lloyd").fit(X.astype(np.float64))
    assert np.array_equal(km.labels_, r["idx"])
    assert np.allclose(km.cluster_centers_, r["C"], rtol=1e-6, atol=1e-7)
    assert km.inertia_ == pytest.approx(r["J"][-1], rel=1e-6)


def test_threaded_assignment_is_identical():
    """The oracle's assignment loop on several host threads gives the same decisions,
    distances and fits as the sequential loop (each kernel is decided alone)."""
    L = synth.resnet18_stack(k=64, layers=1)[0]
    C = synth.random_codebook_state(L.X, 64, 3)
    try:
        oracle.set_threads(1)
        a1, f1 = oracle.assign(L.X, C), oracle.fit(L.X, L.C0, 3)
        oracle.set_threads(4)
        a4, f4 = oracle.assign(L.X, C), oracle.fit(L.X, L.C0, 3)
    finally:
        oracle.set_threads(1)
    for key in a1:
        assert np.array_equal(a1[key], a4[key]), key
    for key in f1:
        assert np.array_equal(f1[key], f4[key]), key
