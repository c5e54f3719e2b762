"""GPU parity of the large-set scalar quantizer (the fully-connected layers, end of
Sec. 3.2) through the C ABI.  Every step is exact or correctly rounded, so codes,
levels, dequantised values and the number of rounds are bit-exact against the oracle
and against the single-workgroup codebook quantizer with unit weights; at the full
VGG-16 fc6 size (too large for the oracle) the result is checked by properties that fix
it: every level is the correctly rounded mean of its scalars, every sampled code is the
nearest level, and a run that stopped early is a fixed point."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

kq = pytest.importorskip("paper_2003_05148_amd")
DEV = torch.device("cuda:0")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def data(kind, m, seed):
    rng = np.random.default_rng(seed)
    if kind == "normal":
        return (rng.standard_normal(m) * 0.01).astype(np.float32)
    if kind == "heavy":
        v = rng.laplace(0.0, 0.003, m)
        v[rng.choice(m, max(1, m // 500), replace=False)] *= 40.0
        return v.astype(np.float32)
    if kind == "constant":
        return np.full(m, -0.375, np.float32)
    if kind == "integers":                     # exact ties and midpoints between levels
        return rng.integers(-40, 41, m).astype(np.float32)
    if kind == "outliers":                      # a few far values: many thresholds share a bucket
        v = 1.0 + rng.standard_normal(m) * 0.01  # (no tiny values, so thresholds are allowed)
        v[rng.choice(m, min(m, 8), replace=False)] = rng.choice([-500.0, 500.0], min(m, 8))
        return v.astype(np.float32)
    if kind == "tiny":                          # subnormal and zero values among normal ones
        v = (rng.standard_normal(m) * 1e-3).astype(np.float32)
        v[::7] = np.float32(3e-42)
        v[::11] = 0.0
        return v
    raise ValueError(kind)


def check(v, bits, iters, tag):
    oc, ol, ov, orr = oracle.quantize_scalars(v, bits, iters)
    for search in ("auto", "thresholds"):   # the exact search below 3 * 2^20, and the threshold path
        codes, levels, v_hat, rounds = kq.kq_quantize_scalars(dev(v), bits, iters, search=search)
        assert np.array_equal(host(codes), oc), (tag, search)
        assert np.array_equal(host(levels).view(np.uint32), ol.view(np.uint32)), (tag, search)
        assert np.array_equal(host(v_hat).view(np.uint32), ov.view(np.uint32)), (tag, search)
        assert int(host(rounds)[0]) == orr, (tag, search)


@pytest.mark.parametrize("m", [1, 2, 9, 1000, 65537])
@pytest.mark.parametrize("kind", ["normal", "heavy", "integers", "tiny", "outliers"])
def test_fc_quantizer_bit_exact(m, kind):
    check(data(kind, m, m + len(kind)), 6, 30, f"{kind} m={m}")


@pytest.mark.parametrize("bits,iters", [(1, 30), (2, 5), (6, 0), (6, 1), (8, 30)])
def test_fc_quantizer_widths_and_rounds(bits, iters):
    check(data("heavy", 30001, bits * 100 + iters), bits, iters, f"bits={bits} iters={iters}")
    check(data("constant", 500, 1), bits, iters, "constant")


def test_fc_quantizer_equals_codebook_quantizer_with_unit_weights():
    v = data("normal", 9 * 900, 5)
    a = kq.kq_quantize_scalars(dev(v), 6, 30)
    C = dev(v.reshape(-1, 9))
    w = torch.ones(900, dtype=torch.int32, device=DEV)
    codes, levels, C_hat = kq.kq_quantize_codebook(C, w, 6, kq.KQ_CBQ_WKMEANS, 30)
    assert torch.equal(a[0], codes.reshape(-1)) and torch.equal(a[1], levels)
    assert torch.equal(a[2], C_hat.reshape(-1))


def test_fc_quantizer_full_size_fc6_properties():
    """VGG-16 fc6 (4096 x 25088 = 102,760,448 scalars, N(0, sqrt(2/25088)))."""
    m = 4096 * 25088
    g = torch.Generator(device=DEV)
    g.manual_seed(6)
    v = torch.randn(m, device=DEV, generator=g) * math.sqrt(2.0 / 25088)
    codes, levels, v_hat, rounds = kq.kq_quantize_scalars(v, 6, 30)
    c, L, r = host(codes), host(levels), int(host(rounds)[0])
    x = host(v)
    assert 1 <= r <= 30
    # the last codes are always computed against the final levels: nearest, lowest on ties
    rows = np.random.default_rng(3).choice(m, 20000, replace=False)
    near = np.argmin(np.abs(x[rows].astype(np.float64)[:, None] - L.astype(np.float64)[None, :]), axis=1)
    assert np.array_equal(c[rows], near)
    assert np.array_equal(host(v_hat)[rows], L[c[rows]])
    if r < 30:  # stopped early: a fixed point, every level the correctly rounded mean of its scalars
        for q in np.linspace(0, 63, 9).astype(int):
            mem = x[c == q].astype(np.float64)
            if mem.size:
                assert L[q] == np.float32(math.fsum(mem.tolist()) / mem.size), q


@pytest.mark.parametrize("kind", ["normal", "integers", "tiny", "outliers"])
def test_fc_threshold_path_equals_the_exact_search(kind):
    """From 3 * 2^20 scalars on, codes come from per-level thresholds (a bucket table over
    the data range, fp32 comparisons); with KQ_F_EXACT_SEARCH every code comes from the
    exact fp64 search.  Both agree bit for bit, also on integer data (exact midpoints
    between levels), on data whose tiny values make fp64 distances inexact (the thresholds
    are then not used) and on data with a few far values, where most thresholds fall into
    one bucket and are compared one by one."""
    m = 9 * 932068                                            # 8,388,612 >= 3 * 2^20
    vd = dev(data(kind, m, 77))
    a = kq.kq_quantize_scalars(vd, 6, 30)
    b = kq.kq_quantize_scalars(vd, 6, 30, search="exact")
    for x, y, name in zip(a, b, ["codes", "levels", "v_hat", "rounds"]):
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), (kind, name)
