"""GPU parity of the codebook retraining step, Sec. 3.1, Eq. (2), through the C ABI.

Bar: counts exact; every stepped entry within 1e-5 of the oracle relative to the
larger of the entry and gamma times its mean gradient (the GPU sums are exact
fixed-point, the oracle's fp64 in ascending order); empty entries bit-identical;
single-layer and stack calls bit-identical; results reproducible bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

kq = pytest.importorskip("paper_2003_05148_amd")
DEV = torch.device("cuda:0")
REL = 1e-5


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def check_step(G, idx, C, gamma, tag):
    gc, gz = kq.kq_codebook_grad_step(dev(G), dev(idx), dev(C), gamma)
    gc, gz = host(gc), host(gz)
    oc, oz = oracle.codebook_grad_step(G, idx, C, gamma)
    assert np.array_equal(gz, oz), tag
    empty = oz == 0
    assert np.array_equal(gc[empty].view(np.uint32), C[empty].view(np.uint32)), tag
    # gamma times the mean gradient, for the tolerance's scale
    k = C.shape[0]
    ok = (idx >= 0) & (idx < k)
    S = np.zeros((k, 9))
    np.add.at(S, idx[ok], G[ok].astype(np.float64))
    step = abs(gamma) * np.abs(S) / np.maximum(oz, 1)[:, None]
    scale = np.maximum(np.abs(oc.astype(np.float64)), step).max(axis=1, keepdims=True)
    err = np.abs(gc.astype(np.float64) - oc.astype(np.float64))
    assert np.all(err <= REL * np.maximum(scale, 1e-38)), (tag, float((err / np.maximum(scale, 1e-38)).max()))
    return gc, gz


@pytest.mark.parametrize("n,k", [(1, 1), (100, 7), (4099, 256), (20000, 768), (20000, 769), (50000, 4096),
                                 (300001, 256)])
@pytest.mark.parametrize("gscale", [1e-9, 1.0, 1e3])
def test_grad_step_shapes_and_magnitudes(n, k, gscale):
    X = synth.normal_layer(1, n, 31 + n)[:n]
    C = synth.random_codebook_state(X, k, k + 1)
    idx = synth.random_indices(n, k, k + 2)
    if k > 4:
        idx[idx == 3] = 2                                     # entry 3 stays empty
    G = (synth.laplace_layer(1, n, 77 + n)[:n] * np.float32(gscale)).astype(np.float32)
    check_step(G, idx, C, 0.05, f"n={n} k={k} g={gscale}")


def test_grad_step_in_place_bad_indices_and_determinism():
    X = synth.normal_layer(32, 32, 5)
    n, k = X.shape[0], 64
    C = synth.random_codebook_state(X, k, 4)
    idx = synth.random_indices(n, k, 6)
    idx[:11] = 99
    idx[11:20] = -4
    G = synth.normal_layer(32, 32, 8) * np.float32(1e-4)
    want, wz = oracle.codebook_grad_step(G, idx, C, 0.3)
    Cd = dev(C)
    kq.kq_codebook_grad_step(dev(G), dev(idx), Cd, 0.3, C_new=Cd)
    assert np.allclose(host(Cd), want, rtol=REL, atol=1e-9)
    a = kq.kq_codebook_grad_step(dev(G), dev(idx), dev(C), 0.3)
    b = kq.kq_codebook_grad_step(dev(G), dev(idx), dev(C), 0.3)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_reconstruction_gradient_gives_the_update():
    """With G = C[idx] - X (gradient of 1/2 |W - X|^2 at the reconstruction) and gamma = 1
    the step lands on the kernel-set means that kq_update computes (Eq. 1)."""
    L = synth.resnet18_stack(k=256, layers=5)[4]
    C = synth.random_codebook_state(L.X, 256, 9)
    Xd, Cd = dev(L.X), dev(C)
    idx = kq.kq_assign(Xd, Cd)[0]
    G = (Cd[idx.long()] - Xd).contiguous()
    stepped, z = kq.kq_codebook_grad_step(G, idx, Cd, 1.0)
    means, z2, _ = kq.kq_update(Xd, idx, Cd, with_distortion=False)
    assert torch.equal(z, z2)
    err = (stepped.double() - means.double()).abs().max().item()
    assert err <= 1e-5 * means.abs().max().item(), err


def test_grad_step_stack_matches_single_layers():
    layers = synth.resnet18_stack(k=64, layers=5)
    Gs = [(synth.laplace_layer(1, L.n, 500 + i)[:L.n] * np.float32(1e-3)).astype(np.float32)
          for i, L in enumerate(layers)]
    idxs = [host(kq.kq_assign(dev(L.X), dev(L.C0))[0]) for L in layers]
    st = kq.Stack([dev(g) for g in Gs], [dev(L.C0) for L in layers])
    for i in range(len(layers)):
        st.idx[i].copy_(dev(idxs[i]))
    kq.kq_codebook_grad_step_stack(st, 0.7)
    for i, L in enumerate(layers):
        c, z = kq.kq_codebook_grad_step(dev(Gs[i]), dev(idxs[i]), dev(L.C0), 0.7)
        assert torch.equal(c, st.C[i]) and torch.equal(z, st.counts[i]), i
        check_step(Gs[i], idxs[i], L.C0, 0.7, f"stack layer {i}")
