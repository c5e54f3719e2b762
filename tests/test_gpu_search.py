"""GPU parity of the codebook-size binary search (Algorithm 1 on the k-means distortion)
through the C ABI: the same tested sizes, the same answer and distortions within 1e-5 of
the oracle's search, whenever the oracle's distortions are not within that tolerance of
the target (a decision on the threshold itself could go either way and is reported)."""
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


@pytest.mark.parametrize("alpha,r,iters", [(0.3, 0.5, 8), (0.1, 0.2, 6), (0.05, 1.0, 8)])
def test_search_matches_the_oracle(alpha, r, iters):
    """ResNet-18's first 3x3 layer shape (64x64), the paper's alpha = 0.3, r = 0.5 and 8
    iterations (Sec. 4.2.2), and two other settings."""
    X = synth.laplace_layer(64, 64, 2000)
    n_init = int(alpha * X.shape[0])
    cand = X[synth.distinct_init(X, n_init, 2000)]
    T = 10
    k, C, idx, trials, d0 = kq.kq_search_codebook_size(dev(X), dev(cand), r, iters, T)
    ok, otrials, od0 = oracle.search_codebook_size(X, cand, n_init, r, iters, T)
    target = (1 + float(np.float32(r))) * od0
    assert d0 == pytest.approx(od0, rel=1e-5)
    clear = all(abs(d - target) > 1e-4 * target for _, d in otrials)
    assert clear, "an oracle distortion lies on the threshold: pick another seed"
    assert [n for n, _ in trials] == [n for n, _ in otrials]
    for (_, gd), (_, od) in zip(trials, otrials):
        assert gd == pytest.approx(od, rel=1e-5)
    assert k == ok
    # the returned codebook and assignment are the chosen fit's: its own distortion
    gi = host(idx)
    assert gi.max() < k
    o = oracle.assign(X, host(C))
    assert np.array_equal(gi, o["idx"])
