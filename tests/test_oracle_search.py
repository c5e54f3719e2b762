"""Pins of the codebook-size binary search (Algorithm 1, Eq. 3) as driven here by the
k-means distortion: hand-computed traces for closed-form distortion curves, the bounds
it keeps, and its stopping rule."""
import numpy as np

import oracle


def test_trace_for_d_equal_one_over_k():
    # D(k) = 1/k, n_init = 100, r = 1: target = 2 * 0.01 = 0.02, so k >= 51 passes (1/50 = 0.02 is not below)
    k, trials, d0 = oracle.size_search(lambda k: 1.0 / k, 100, 1.0, 8)
    assert d0 == 0.01
    assert [n for n, _ in trials] == [50, 75, 62, 56, 53, 51]
    assert k == 51
    # one more iteration would test 50 + (51 - 50) // 2 = 50: a bound, so the search stopped


def test_target_follows_eq3_with_zero_error_reference():
    # a step curve: D = 1 below k = 30, D = 0.5 from k = 30 on; D(n_init) = 0.5
    step = lambda k: 1.0 if k < 30 else 0.5
    k, trials, d0 = oracle.size_search(step, 64, 0.0, 20)      # r = 0: only D < D(n_init) passes
    assert k == 64 and all(d >= 0.5 for _, d in trials)
    k, trials, d0 = oracle.size_search(step, 64, 1.5, 20)      # r = 1.5: every k passes (1.0 < 1.25)
    assert k == 1 and [n for n, _ in trials] == [32, 16, 8, 4, 2, 1]


def test_iteration_limit_and_monotone_bounds():
    rng = np.random.default_rng(4)
    for _ in range(50):
        n_init = int(rng.integers(2, 5000))
        slope = float(rng.uniform(0.5, 3.0))
        D = lambda k, s=slope: 1.0 / k ** s
        r = float(rng.uniform(0.0, 2.0))
        it = int(rng.integers(0, 12))
        k, trials, d0 = oracle.size_search(D, n_init, r, it)
        assert len(trials) <= it and 1 <= k <= n_init
        target = (1.0 + float(np.float32(r))) * d0
        assert D(k) < target or k == n_init
        lo = 0
        for n, d in trials:                                     # every tested size lies inside the bounds
            assert lo < n < n_init
            if d >= target:
                lo = max(lo, n)
        # without a limit the search ends at the smallest passing size
        k_full, _, _ = oracle.size_search(D, n_init, r, 64)
        smallest = next(q for q in range(1, n_init + 1) if D(q) < target)
        assert k_full == smallest


def test_search_on_a_layer_prefers_fewer_entries_when_allowed():
    X = np.random.default_rng(5).standard_normal((600, 9)).astype(np.float32)
    cand = X[np.random.default_rng(6).permutation(600)[:120]]
    k, trials, d0 = oracle.search_codebook_size(X, cand, 120, 0.5, 8, 5)
    assert 1 <= k < 120 and d0 > 0
    assert all(0 < n < 120 for n, _ in trials)
