"""Pins of the oracle's 6-bit kernel-codebook quantizer (Sec. 3.2): the closed
form of the uniform grid, lossless cases, the weighting (a weight w equals w
copies of the scalar), invariance to scaling all weights, and scikit-learn's
weighted Lloyd k-means where both definitions coincide."""
import numpy as np
import pytest

import oracle


def test_uniform_grid_closed_form():
    rng = np.random.default_rng(1)
    C = (rng.standard_normal((256, 9)) * 0.05).astype(np.float32)
    codes, levels, C_hat = oracle.cbq_uniform(C, 6)
    v = C.reshape(-1).astype(np.float64)
    lo, hi = v.min(), v.max()
    delta = (hi - lo) / 63
    assert levels[0] == np.float32(lo)
    assert abs(float(levels[63]) - hi) <= 2 * np.spacing(np.float32(abs(hi)))
    assert np.all(np.diff(levels.astype(np.float64)) > 0)
    # nearest grid point, q = round((v - lo) / delta), away from cell midpoints
    t = (v - lo) / delta
    q = np.floor(t + 0.5)
    far = np.abs(t - np.floor(t) - 0.5) > 1e-4
    assert np.array_equal(codes[far].astype(np.float64), q[far])
    assert codes.max() == 63 and codes.min() == 0
    assert np.array_equal(C_hat.reshape(-1), levels[codes])


def test_constant_codebook_all_codes_zero():
    C = np.full((7, 9), 0.125, np.float32)
    codes, levels, C_hat = oracle.cbq_uniform(C, 6)
    assert np.all(codes == 0) and np.all(levels == np.float32(0.125))
    codes, levels, C_hat, rounds = oracle.cbq_wkmeans(C, np.arange(7), 6)
    assert np.all(codes == 0) and np.array_equal(C_hat, C)


def test_wkmeans_lossless_on_grid_values():
    """Scalars that sit exactly on 40 of the 64 grid points are coded without loss."""
    rng = np.random.default_rng(2)
    grid = oracle.uniform_levels(-0.75, 0.5, 6)
    pick = np.concatenate([[0, 63], rng.choice(np.arange(1, 63), 38, replace=False)])
    v = grid[rng.choice(pick, 9 * 30)]
    v[:2] = grid[[0, 63]]
    C = v.reshape(30, 9).astype(np.float32)
    w = rng.integers(0, 50, 30)
    codes, levels, C_hat, rounds = oracle.cbq_wkmeans(C, w, 6)
    assert np.array_equal(C_hat, C)
    assert rounds == 1


def test_weight_equals_copies():
    """A scalar of weight w contributes exactly like w copies of weight 1."""
    rng = np.random.default_rng(3)
    C = (rng.standard_normal((12, 9)) * 0.1).astype(np.float32)
    w = rng.integers(1, 4, 12)
    codes, levels, _, _ = oracle.cbq_wkmeans(C, w, 6, iters=30)
    Crep = np.repeat(C, w, axis=0)
    codes2, levels2, _, _ = oracle.cbq_wkmeans(Crep, np.ones(len(Crep), np.int64), 6, iters=30)
    assert np.array_equal(levels, levels2)
    assert np.array_equal(np.repeat(codes.reshape(12, 9), w, axis=0).reshape(-1), codes2)


def test_weight_scaling_invariance():
    rng = np.random.default_rng(4)
    C = (rng.laplace(0, 0.04, (64, 9))).astype(np.float32)
    w = rng.integers(0, 100, 64)
    a = oracle.cbq_wkmeans(C, w, 6)
    b = oracle.cbq_wkmeans(C, w * 8, 6)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_zero_weight_levels_are_kept():
    """With every weight zero no level is ever updated: the result is the uniform grid."""
    rng = np.random.default_rng(5)
    C = (rng.standard_normal((20, 9))).astype(np.float32)
    codes, levels, C_hat, rounds = oracle.cbq_wkmeans(C, np.zeros(20, np.int64), 6)
    u_codes, u_levels, u_hat = oracle.cbq_uniform(C, 6)
    assert np.array_equal(levels, u_levels) and np.array_equal(codes, u_codes) and rounds == 1
    # only entry 0 weighted: levels no scalar of entry 0 ever used stay on the grid
    w = np.zeros(20, np.int64)
    w[0] = 3
    codes, levels, _, _ = oracle.cbq_wkmeans(C, w, 6)
    moved = np.nonzero(levels != u_levels)[0]
    assert set(moved.tolist()) <= set(u_codes[:9].tolist()) | set(codes[:9].tolist())
    assert len(moved) >= 1


@pytest.mark.parametrize("weighted", [False, True])
def test_wkmeans_matches_sklearn(weighted):
    """scikit-learn's (weighted) Lloyd k-means from the same 64-level grid: same codes
    and levels (values spread so that no level ever empties)."""
    sk = pytest.importorskip("sklearn.cluster")
    rng = np.random.default_rng(6 + weighted)
    C = rng.uniform(-1, 1, (600, 9)).astype(np.float32)
    C[0, 0], C[0, 1] = -1.0, 1.0
    w = rng.integers(1, 20, 600) if weighted else np.ones(600, np.int64)
    codes, levels, _, rounds = oracle.cbq_wkmeans(C, w, 6, iters=100)
    assert rounds < 100
    v = C.reshape(-1, 1).astype(np.float64)
    init = oracle.uniform_levels(-1.0, 1.0, 6).astype(np.float64).reshape(-1, 1)
    km = sk.KMeans(n_clusters=64, init=init, n_init=1, max_iter=300, tol=0.0, algorithm="lloyd")
    km.fit(v, sample_weight=np.repeat(w, 9).astype(np.float64))
    assert np.array_equal(km.labels_, codes)
    assert np.allclose(km.cluster_centers_[:, 0], levels, rtol=1e-6, atol=1e-7)


def test_fc_quantizer_is_the_unit_weight_codebook_quantizer():
    """The fully-connected form (end of Sec. 3.2) runs the same k-means on a flat set with
    every weight 1: arranged as rows of 9 with unit appearance counts it is identical."""
    rng = np.random.default_rng(21)
    v = (rng.laplace(0.0, 0.02, 9 * 700)).astype(np.float32)
    a = oracle.quantize_scalars(v, 6, 30)
    b = oracle.cbq_wkmeans(v.reshape(-1, 9), np.ones(700, np.int64), 6, 30)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[3] == b[3]
    assert np.array_equal(a[2], b[2].reshape(-1))


def test_fc_quantizer_matches_sklearn_lloyd_from_the_grid():
    """Unit weights reduce the method to plain 1-D Lloyd from the uniform grid: with data
    dense enough that no level empties, scikit-learn's Lloyd reaches the same partition."""
    from sklearn.cluster import KMeans
    rng = np.random.default_rng(22)
    v = (rng.standard_normal(4000) * 0.05).astype(np.float32)
    codes, levels, v_hat, rounds = oracle.quantize_scalars(v, 3, 500)
    grid = oracle.uniform_levels(float(v.min()), float(v.max()), 3).astype(np.float64)
    km = KMeans(n_clusters=8, init=grid.reshape(-1, 1), n_init=1, max_iter=1000, tol=0.0,
                algorithm="lloyd").fit(v.astype(np.float64).reshape(-1, 1))
    assert rounds < 500                                         # converged
    assert np.array_equal(km.labels_, codes.astype(np.int64))
    assert np.allclose(km.cluster_centers_.reshape(-1), levels.astype(np.float64), rtol=1e-6, atol=1e-9)
