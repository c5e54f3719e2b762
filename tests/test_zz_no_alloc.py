"""kq_fit_layer_noalloc (the fit with the library's static device scratch) against
kq_fit_layer with a caller workspace, through the C ABI: two calls in a row on one GPU, the
second with a smaller layer (the scratch keeps the first call's contents), then the first
shape again; every output bit for bit; sizes beyond the scratch are refused before any
launch.  Runs alone in a fresh process and after the other tests."""
import ctypes

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

kq = pytest.importorskip("paper_2003_05148_amd")
DEV = torch.device("cuda:0")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def outputs(n, k, iters):
    return (torch.full((k, 9), -1.0, device=DEV), torch.full((n,), -1, dtype=torch.int32, device=DEV),
            torch.full((k,), -1, dtype=torch.int32, device=DEV),
            torch.full((iters + 1,), -1.0, dtype=torch.float64, device=DEV))


def test_noalloc_fit_equals_workspace_fit_twice_then_smaller():
    big = synth.resnet18_stack(k=256, layers=16)[15]            # 262,144 kernels, k = 256 (fused path)
    small = synth.single_layer(k=64)[0]                          # 4,096 kernels
    mid = synth.stress_layer(n=30000, k=300, n_centers=300, seed=12)[0]   # k > 256: the separate update
    for L, iters in [(big, 6), (small, 5), (mid, 3), (big, 2)]:
        X, C0 = dev(L.X), dev(L.C0)
        ref = kq.kq_fit_layer(X, C0, iters)
        got = kq.kq_fit_layer_noalloc(X, C0, iters, *outputs(L.n, L.k, iters))
        for a, b, name in zip(ref, got, ("C", "idx", "counts", "distortion")):
            assert torch.equal(a, b), (L.name, name)
        val = kq.kq_fit_layer_noalloc(X, C0, iters, *outputs(L.n, L.k, iters), validate=True)
        for a, b in zip(ref, val):
            assert torch.equal(a, b), L.name


def test_noalloc_refuses_sizes_beyond_the_scratch():
    assert kq.lib.kq_fit_layer_noalloc_max_bytes() == 32 << 20
    n = 1666049                                                  # one kernel past the limit at k = 256
    assert kq.lib.kq_workspace_bytes(kq.KQ_OP_FIT, n, 256, 9) > kq.lib.kq_fit_layer_noalloc_max_bytes()
    assert kq.lib.kq_workspace_bytes(kq.KQ_OP_FIT, n - 1, 256, 9) <= kq.lib.kq_fit_layer_noalloc_max_bytes()
    X = torch.zeros(n, 9, device=DEV)
    C = torch.zeros(256, 9, device=DEV)
    with pytest.raises(kq.KqError) as e:
        kq.kq_fit_layer_noalloc(X, C, 1, *outputs(n, 256, 1))
    assert e.value.status == kq.KQ_ERR_WORKSPACE
