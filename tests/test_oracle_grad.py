"""Pins of the oracle's codebook retraining step, Sec. 3.1, Eq. (2):
c_i <- c_i - gamma * mean of the gradients of the kernels mapped to entry i.

Each pin is fixed by something other than the oracle's own formula: exact rational
arithmetic, special cases with known results, and the link to Eq. (1): with the
gradient of the reconstruction loss (1/2) |W - X|^2, i.e. G = C[idx] - X, and
gamma = 1, the step lands on the mean of every kernel set, which is the k-means
update of Eq. (1)."""
from fractions import Fraction

import numpy as np

import oracle
import synth


def ulp32(v):
    return np.spacing(np.abs(np.float32(v))).astype(np.float64)


def test_exact_rational_mean_step():
    rng = np.random.default_rng(11)
    n, k = 60, 7
    G = (rng.standard_normal((n, 9)) * 1e-3).astype(np.float32)
    C = rng.standard_normal((k, 9)).astype(np.float32)
    idx = rng.integers(0, k - 1, n).astype(np.int32)          # entry k-1 stays empty
    gamma = np.float32(0.37)
    out, z = oracle.codebook_grad_step(G, idx, C, gamma)
    assert np.array_equal(z, np.bincount(idx, minlength=k))
    exact_hits = 0
    for j in range(k):
        members = np.nonzero(idx == j)[0]
        for d in range(9):
            if members.size == 0:
                assert out[j, d] == C[j, d]
                continue
            s = sum(Fraction(float(G[i, d])) for i in members)
            v = Fraction(float(C[j, d])) - Fraction(float(gamma)) * s / members.size
            assert abs(Fraction(float(out[j, d])) - v) <= Fraction(float(ulp32(float(v))))
            exact_hits += np.float32(float(v)) == out[j, d]
    assert exact_hits >= 0.95 * 9 * (k - 1)


def test_gamma_zero_keeps_the_codebook():
    L = synth.single_layer(k=64)[0]
    idx = oracle.assign(L.X, L.C0)["idx"]
    G = synth.normal_layer(64, 64, 99)
    out, _ = oracle.codebook_grad_step(G, idx, L.C0, 0.0)
    assert np.array_equal(out.view(np.uint32), L.C0.view(np.uint32))


def test_constant_gradient_per_entry_and_bad_indices():
    rng = np.random.default_rng(12)
    k, n = 5, 400
    C = rng.standard_normal((k, 9)).astype(np.float32)
    g = rng.standard_normal((k, 9)).astype(np.float32)
    idx = rng.integers(0, k, n).astype(np.int32)
    G = g[idx]
    bad = idx.copy()
    bad[:7] = k + 3
    bad[7:9] = -1
    G_bad = G.copy()
    G_bad[:9] = 1e30                                          # ignored with their indices
    for gi, ii in ((G, idx), (G_bad, bad)):
        out, z = oracle.codebook_grad_step(gi, ii, C, 0.5)
        # the mean of z equal fp32 values is that value exactly
        want = (C.astype(np.float64) - 0.5 * g.astype(np.float64)).astype(np.float32)
        assert np.array_equal(out, want)
        assert z.sum() == np.count_nonzero((ii >= 0) & (ii < k))


def test_reconstruction_gradient_gives_the_kmeans_update():
    """Eq. (2) with G = dL/dW of L = 1/2 |W - X|^2 at W = C[idx] and gamma = 1 equals the
    mean of every kernel set (Eq. 1's update), up to the fp32 rounding of G."""
    L = synth.single_layer(k=256)[0]
    C = synth.random_codebook_state(L.X, 256, 3)
    idx = oracle.assign(L.X, C)["idx"]
    G = C[idx] - L.X                                          # fp32, each within 2^-24 relative
    out, z = oracle.codebook_grad_step(G, idx, C, 1.0)
    want, wz = oracle.update(L.X, idx, C)
    assert np.array_equal(z, wz)
    dev = np.abs(C[idx].astype(np.float64) - L.X.astype(np.float64))
    slack = np.zeros((256, 9))
    np.add.at(slack, idx, dev)
    bound = 2.0 ** -24 * slack / np.maximum(z, 1)[:, None] + 2 * ulp32(want)
    assert np.all(np.abs(out.astype(np.float64) - want.astype(np.float64)) <= bound)
    # a sign or normalisation mistake would land far away
    assert np.abs(out - want).max() < 1e-6


def test_step_is_linear_in_gamma():
    L = synth.single_layer(k=128)[0]
    idx = oracle.assign(L.X, L.C0)["idx"]
    G = synth.normal_layer(64, 64, 7) * np.float32(1e-2)
    a, _ = oracle.codebook_grad_step(G, idx, L.C0, 0.25)
    b, _ = oracle.codebook_grad_step(G, idx, L.C0, 0.5)
    da = a.astype(np.float64) - L.C0
    db = b.astype(np.float64) - L.C0
    assert np.allclose(db, 2 * da, rtol=1e-3, atol=4 * ulp32(np.abs(L.C0).max()))
