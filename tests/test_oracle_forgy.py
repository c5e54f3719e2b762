"""Pins of the oracle's k-means initialisation (the reading taken for Sec. 3.1, which does
not say how the k-means starts): splitmix64 against its reference outputs, a selection
worked out by hand, and the properties the definition fixes."""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64_forgy.txt")


def golden():
    seeds, selects = {}, []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        head, vals = line.split(":")
        vals = [int(v) for v in vals.split()]
        h = head.split()
        if h[0] == "seed":
            seeds[int(h[1])] = vals
        else:  # select seed S k K
            selects.append((int(h[2]), int(h[4]), vals))
    return seeds, selects


HAND_X = np.array([[0.5] * 9, [0.0] * 9, list(range(1, 10)), [-1.0] * 9, [2.0] * 9, list(range(1, 10)),
                   [-0.0] * 9], dtype=np.float32)


def test_splitmix64_reference_outputs():
    seeds, _ = golden()
    assert set(seeds) == {0, 1234567}
    for seed, outs in seeds.items():
        g = oracle.splitmix64(seed)
        assert [next(g) for _ in outs] == outs, seed


def test_hand_worked_selection():
    _, selects = golden()
    assert np.signbit(HAND_X[6]).all() and not np.signbit(HAND_X[1]).any()
    for seed, k, expected in selects:
        assert oracle.forgy_select(HAND_X, k, seed).tolist() == expected
    # five distinct kernels (rows 5 and 6 repeat rows 2 and 1): k = 5 takes rows 0, 3, 4,
    # one of rows 1 and 6 and one of rows 2 and 5; k = 6 is refused
    sel = set(oracle.forgy_select(HAND_X, 5, 1234567).tolist())
    assert {0, 3, 4} <= sel and len(sel & {1, 6}) == 1 and len(sel & {2, 5}) == 1
    with pytest.raises(ValueError):
        oracle.forgy_select(HAND_X, 6, 1234567)


def test_selection_properties():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((400, 9)).astype(np.float32)
    X[100:150] = X[0:50]                    # fifty exact copies
    X[200, :] = 0.0
    X[201, :] = -0.0                        # the same kernel once -0 reads as +0
    X[300, 0] = np.nan                      # a NaN kernel is a value like any other
    n_distinct = 400 - 50 - 1
    for seed in (0, 1, 2 ** 64 - 1, 987654321):
        full = oracle.forgy_select(X, n_distinct, seed)
        canon = np.where(X == 0, np.float32(0), X).view(np.uint32)
        keys = {canon[i].tobytes() for i in full}
        assert len(keys) == n_distinct and len(set(full.tolist())) == n_distinct
        for k in (1, 7, 256):               # a smaller k is a prefix of a larger one
            assert np.array_equal(oracle.forgy_select(X, k, seed), full[:k])
        with pytest.raises(ValueError):
            oracle.forgy_select(X, n_distinct + 1, seed)
    assert not np.array_equal(oracle.forgy_select(X, 50, 1), oracle.forgy_select(X, 50, 2))


def test_selection_is_uniform():
    """The first pick of a full shuffle is uniform over the rows: over 3000 seeds each of
    10 rows comes first 300 +- 4.5 sigma times."""
    X = np.arange(90, dtype=np.float32).reshape(10, 9)
    first = np.bincount([int(oracle.forgy_select(X, 1, s)[0]) for s in range(3000)], minlength=10)
    sigma = np.sqrt(3000 * 0.1 * 0.9)
    assert np.all(np.abs(first - 300) <= 4.5 * sigma), first
    # and a full order is a permutation
    assert sorted(oracle.forgy_select(X, 10, 42).tolist()) == list(range(10))
