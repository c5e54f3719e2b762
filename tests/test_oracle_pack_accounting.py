"""Pins of the index stream (Eq. 4), test-time reconstruction (end of Sec. 3.2)
and the storage accounting of Eq. (4)-(7) against the figures the paper prints."""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rows(name):
    out = []
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#")[0].split()
        if line:
            out.append(line)
    return out


def test_pack_hand_examples():
    # 2-bit values 1, 2, 3 -> 01 10 11 read LSB-first -> 0b00111001
    assert oracle.pack_bits([1, 2, 3], 2).tolist() == [0b00111001]
    # 3-bit values 5, 7, 0 -> bits 101 111 000 (LSB first) -> byte0 = 0b00111101, byte1 = 0
    assert oracle.pack_bits([5, 7, 0], 3).tolist() == [0b00111101, 0b00000000]
    # 12-bit value 0xABC, then 0x123: bytes BC, 3A, 12
    assert oracle.pack_bits([0xABC, 0x123], 12).tolist() == [0xBC, 0x3A, 0x12]
    assert oracle.pack_bits([7, 7, 7], 0).size == 0


@pytest.mark.parametrize("bits", [1, 4, 6, 7, 8, 11, 12, 16])
def test_pack_roundtrip_and_length(bits):
    rng = np.random.default_rng(bits)
    n = 1000 + bits
    v = rng.integers(0, 1 << bits, n)
    s = oracle.pack_bits(v, bits)
    assert s.size == (n * bits + 7) // 8
    assert np.array_equal(oracle.unpack_bits(s, n, bits), v)


def test_index_bits():
    assert [oracle.index_bits(k) for k in (1, 2, 3, 4, 5, 192, 256, 257, 4096)] == [0, 1, 2, 2, 3, 8, 8, 9, 12]


def test_reconstruct_gather_and_mse():
    rng = np.random.default_rng(0)
    X = rng.standard_normal((500, 9)).astype(np.float32)
    C = X[:16].copy()
    a = oracle.assign(X, C)
    W = oracle.reconstruct(a["idx"], C)
    assert np.array_equal(W[:16], C)
    J = oracle.distortion(X, C, a["idx"])
    mse = float(((X.astype(np.float64) - W.astype(np.float64)) ** 2).mean())
    assert mse == pytest.approx(J / X.size, rel=1e-12)


def test_vgg_k128_ratios():
    """Sec. 4.2.1 prints CR 18 / 38.08 / 40.33 (K) and 33.15 / 40.53 / 40.98 (K+C)."""
    for layer, n, k, cr_k, cr_kc, beta_kc in rows("vgg_k128_ratios.txt"):
        n, k = int(n), int(k)
        assert abs(oracle.compression_ratio(n, k, 32) - float(cr_k)) <= 0.01
        assert abs(oracle.compression_ratio(n, k, 6) - float(cr_kc)) <= 0.01
        assert abs(oracle.bits_per_param(n, k, 6) - float(beta_kc)) <= 0.001
        # Eq. (7): beta is 32 / C_KQ
        assert oracle.bits_per_param(n, k, 6) == pytest.approx(32 / oracle.compression_ratio(n, k, 6))


@pytest.mark.parametrize("name", ["table4_vgg_layerwise.txt", "table5_resnet18_layerwise.txt"])
def test_layerwise_tables(name):
    cols = ["pctK", "pctKC", "betaK", "betaKC"]
    checked = 0
    for r in rows(name):
        n, k = int(r[1]), int(r[2])
        printed = dict(zip(cols, map(float, r[3:7])))
        flags = set(r[7].split(","))
        comp = dict(pctK=100 * oracle.bits_per_param(n, k, 32) / 32,
                    pctKC=100 * oracle.bits_per_param(n, k, 6) / 32,
                    betaK=oracle.bits_per_param(n, k, 32), betaKC=oracle.bits_per_param(n, k, 6))
        for c in cols:
            if c in flags:
                # a misprint in the paper: still within 0.2 of the formula
                assert 0.01 < abs(printed[c] - comp[c]) <= 0.2
            else:
                assert abs(printed[c] - comp[c]) <= 0.01, (r[0], c, printed[c], comp[c])
                checked += 1
    assert checked >= 18


def test_theoretical_limits():
    # Eq. (6) with k = 2 and n >> k tends to 9 * 32 / 1 = 288 for 3x3 kernels (Sec. 3.3)
    assert oracle.compression_ratio(10 ** 9, 2, 32) == pytest.approx(288, rel=1e-6)
    # Eq. (5): conventional 1-bit quantization tends to 32
    assert oracle.conventional_ratio(10 ** 9, 2, 32) == pytest.approx(32, rel=1e-6)
