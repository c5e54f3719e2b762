"""GPU parity of the Yinyang assignment (Sec. 4.1) through the C ABI.

Yinyang k-means reaches exactly the plain Lloyd result, so the bar is the plain
assignment's: for every codebook of a sequence, indices and fp32 best distances
bit-exact against the oracle's fp32 decision and against kq_assign, the distortion
equal to kq_assign's bit for bit; a Yinyang fit equal to the Lloyd fit in every output.
The scan counts check that the bounds do skip work (a run that scanned every group
would pass the parity checks too)."""
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


def same_as_plain(X, C, yy_out, tag):
    """Yinyang output == kq_assign == the oracle's fp32 decision, bit for bit."""
    gi, gd, gJ = (host(t) for t in yy_out)
    pi, pd, pJ = (host(t) for t in kq.kq_assign(dev(X), dev(C)))
    assert np.array_equal(gi, pi), (tag, np.nonzero(gi != pi)[0][:5])
    assert np.array_equal(gd.view(np.uint32), pd.view(np.uint32)), tag
    assert gJ[0] == pJ[0], tag
    o = oracle.assign(X, C)
    assert np.array_equal(gi, o["idx"]), tag
    assert np.array_equal(gd.view(np.uint32), o["d32"].view(np.uint32)), tag


def run_sequence(X, Cs, groups, tag):
    yy = kq.Yinyang(dev(X), dev(Cs[0]), groups=groups)
    same_as_plain(X, Cs[0], (yy.idx, yy.best_d, yy.distortion), f"{tag} init")
    scanned = []
    for r, C in enumerate(Cs[1:], 1):
        out = yy.assign(dev(C))
        same_as_plain(X, C, out, f"{tag} round {r}")
        scanned.append(host(yy.stats).copy())
    return scanned


def test_oracle_trajectory_step_locked():
    """The oracle's own Lloyd codebooks, round after round (64x64 layer, k = 256)."""
    L = synth.single_layer(k=256)[0]
    Cs = [L.C0]
    for _ in range(12):
        o = oracle.assign(L.X, Cs[-1])
        Cs.append(oracle.update(L.X, o["idx"], Cs[-1])[0])
    scanned = run_sequence(L.X, Cs, 0, "64x64")
    assert scanned[-1][0] < L.n, scanned         # late rounds skip kernels


@pytest.mark.parametrize("n,k,groups", [(1, 1, 0), (2, 1, 1), (63, 5, 2), (257, 7, 7), (5000, 64, 0),
                                        (5000, 64, 64), (4099, 300, 3), (3000, 1100, 1), (6000, 1500, 0)])
def test_shapes_and_groups(n, k, groups):
    X = synth.laplace_layer(1, n, 300 + n)[:n]
    C0 = synth.random_codebook_state(X, k, k)
    Cs = [C0]
    scale = float(np.std(X))
    for r, (frac, s) in enumerate([(0.0, 0.0), (0.1, 0.05), (1.0, 0.01), (0.5, 1.0), (0.02, 0.3), (0.0, 0.0)]):
        Cs.append(synth.moved_codebook(Cs[-1], frac, s * scale, 17 * r + k))
    scanned = run_sequence(X, Cs, groups, f"n={n} k={k} g={groups}")
    # the first round scans at least each kernel's own group (the initial bounds come from
    # the group centres and include the kernel's entry); after that an unmoved codebook
    # rescans only near-ties (best and second best within 2^-18)
    assert scanned[0][0] == n and scanned[-1][0] <= max(2, n // 100), scanned


def test_exact_ties_duplicates_and_far_moves():
    rng = np.random.default_rng(5)
    X = rng.integers(-2, 3, (4000, 9)).astype(np.float32)
    C0 = rng.integers(-2, 3, (256, 9)).astype(np.float32)
    C0[128:192] = C0[0:64]                      # duplicated entries: ties to the lowest index
    Cs = [C0]
    for r in range(5):
        C = Cs[-1].copy()
        sel = rng.choice(256, 40, replace=False)
        C[sel] = rng.integers(-2, 3, (40, 9)).astype(np.float32)   # jumps onto other grid points
        Cs.append(C)
    Cs.append(Cs[-1] * np.float32(8.0))         # one huge move of everything
    Cs.append(Cs[-1] * np.float32(0.125))
    for groups in (0, 1, 5, 64):
        run_sequence(X, Cs, groups, f"grid g={groups}")


def test_clustered_data_and_midpoints():
    L = synth.stress_layer(n=30000, k=1024, n_centers=1024, seed=45)[0]
    Cs = [L.C0]
    for _ in range(6):
        o = oracle.assign(L.X, Cs[-1])
        Cs.append(oracle.update(L.X, o["idx"], Cs[-1])[0])
    run_sequence(L.X, Cs, 0, "clusters")
    X = np.zeros((128, 9), np.float32)          # every kernel exactly between two entries
    C = np.zeros((2, 9), np.float32)
    C[0, 0], C[1, 0] = -1.0, 1.0
    run_sequence(X, [C, C[::-1].copy(), C], 2, "midpoint")


@pytest.mark.parametrize("which", ["single", "resnet_k64", "clusters"])
def test_fit_equals_lloyd_fit(which):
    if which == "single":
        L, T = synth.single_layer(k=256)[0], 20
    elif which == "resnet_k64":
        L, T = synth.resnet18_stack(k=64, layers=6)[5], 15
    else:
        L, T = synth.stress_layer(n=50000, k=2048, n_centers=2048, seed=46)[0], 10
    Xd, C0 = dev(L.X), dev(L.C0)
    a = kq.kq_fit_layer(Xd, C0, T)
    b = kq.kq_fit_layer_yinyang(Xd, C0, T)
    for x, y, name in zip(a, b[:4], ["C", "idx", "counts", "distortion"]):
        assert torch.equal(x, y), (which, name)
    st = host(b[4])
    assert st[-1, 0] < L.n, st                  # the last round skipped some kernels


def test_fit_groups_and_resume_state():
    L = synth.single_layer(k=256)[0]
    Xd, C0 = dev(L.X), dev(L.C0)
    ref = kq.kq_fit_layer(Xd, C0, 8)
    for groups in (1, 2, 17, 64):
        out = kq.kq_fit_layer_yinyang(Xd, C0, 8, groups=groups)
        for x, y in zip(ref, out[:4]):
            assert torch.equal(x, y), groups
    z = kq.kq_fit_layer_yinyang(Xd, C0, 0)      # no rounds: the plain assignment
    assert torch.equal(z[1], kq.kq_assign(Xd, C0)[0])


def test_stress_layer_full_size():
    """1M kernels, k = 4096, 10 rounds: the Yinyang fit equals the Lloyd fit."""
    L = synth.stress_layer()[0]
    Xd, C0 = dev(L.X), dev(L.C0)
    a = kq.kq_fit_layer(Xd, C0, 10)
    b = kq.kq_fit_layer_yinyang(Xd, C0, 10)
    for x, y, name in zip(a, b[:4], ["C", "idx", "counts", "distortion"]):
        assert torch.equal(x, y), name
    rows = np.random.default_rng(2).choice(L.n, 2000, replace=False)
    o = oracle.assign(L.X[rows], host(b[0]))
    assert np.array_equal(host(b[1])[rows], o["idx"])
    st = host(b[4])
    assert st[-1, 0] < L.n, st
