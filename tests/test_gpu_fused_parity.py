"""Step-locked oracle parity of the default fit path at full size, through the C ABI.

The fits (kq_fit_layer, kq_fit_stack, kq_compress_stack) and the benchmark run every
Lloyd round as one assignment launch that also forms the member sums (every k <= 256)
and a finish-only update.  Here each round starts both sides from the oracle's codebook:
every index must equal the oracle's fp32 decision, counts must be exact, centroids within
1e-5 of the oracle's fp64 means (per codeword, relative to its largest component) and the
distortion within 1e-5 of the oracle's fp64 value.  Also: the per-layer fixed-point scale at
small and large weight magnitudes, KQ_F_VALIDATE, and the one-call compression pass against
the oracle and the separate calls."""
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


def check_centroids(gC, oC, tag):
    err = np.abs(gC.astype(np.float64) - oC.astype(np.float64)).max(axis=1)
    scale = np.maximum(np.abs(oC.astype(np.float64)).max(axis=1), 1e-300)
    worst = float((err / scale).max())
    assert worst <= REL, (tag, worst)
    return worst


def step_locked_fused(layers, rounds, tag):
    """`rounds` Lloyd rounds of the stack through kq_assign_stack(fused_sums) +
    kq_update_stack(sums_from_assign), each started from the oracle's codebook."""
    st = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=rounds)
    C = [L.C0.copy() for L in layers]
    for t in range(rounds):
        for i in range(len(layers)):
            st.C[i].copy_(dev(C[i]))
        kq.kq_assign_stack(st, dist_slot=t, distortion=False, fused_sums=True)
        kq.kq_update_stack(st, dist_slot=t, distortion_from_assign=True, sums_from_assign=True)
        for i, L in enumerate(layers):
            a = oracle.assign(L.X, C[i])
            gi = host(st.idx[i])
            bad = np.nonzero(gi != a["idx"])[0]
            assert bad.size == 0, (tag, t, L.name, bad.size, bad[:5])
            oC, oz = oracle.update(L.X, a["idx"], C[i])
            assert np.array_equal(host(st.counts[i]), oz), (tag, t, L.name)
            check_centroids(host(st.C[i]), oC, (tag, t, L.name))
            J = float(host(st.distortion[i])[t])
            assert J == pytest.approx(oracle.distortion(L.X, C[i], a["idx"]), rel=REL, abs=1e-300), (tag, t, L.name)
            C[i] = oC
    return C


def test_fused_rounds_resnet18_k256_full_size():
    step_locked_fused(synth.resnet18_stack(k=256), 3, "resnet18 k=256")


@pytest.mark.parametrize("k", [16, 64])
def test_fused_rounds_resnet18_small_codebooks_full_size(k):
    step_locked_fused(synth.resnet18_stack(k=k), 1, f"resnet18 k={k}")


def test_fused_rounds_vgg16_k256_full_size():
    layers = synth.vgg16_stack(k=256)
    assert layers[0].k == 192                       # conv1 clamped to its distinct kernels
    step_locked_fused(layers, 1, "vgg16 k=256")


def test_fused_rounds_ragged_long_stack():
    """20 layers (two launches of at most 16), from one kernel to 50,000: layers of fewer
    64-kernel units than a workgroup has waves, unit counts that do not divide evenly over a
    layer's workgroups, and codebooks of 1 to 256 entries."""
    sizes = [1, 5, 63, 64, 65, 700, 4096, 4097, 20000, 3, 128, 129, 777, 50000, 10, 2, 9000, 837, 1000, 31]
    ks = [1, 2, 17, 64, 200, 256, 256, 255, 256, 3, 128, 64, 100, 256, 7, 2, 256, 37, 160, 31]
    layers = []
    for i, (n, k) in enumerate(zip(sizes, ks)):
        X = synth.laplace_layer(1, n, 900 + i) * np.float32(1 + 0.5 * i)
        layers.append(synth.make_layer(f"r{i}", X, k, 50 + i))
    step_locked_fused(layers, 2, "ragged")


def test_fit_stack_step_locked_resnet18():
    """kq_fit_stack itself (one Lloyd round and the final assignment per call) from the
    oracle's codebook, twice: its C, final indices, counts and both distortions."""
    layers = synth.resnet18_stack(k=256)
    C = [L.C0.copy() for L in layers]
    for t in range(2):
        st = kq.Stack([dev(L.X) for L in layers], [dev(c) for c in C], iters=1)
        kq.kq_fit_stack(st, 1)
        for i, L in enumerate(layers):
            a0 = oracle.assign(L.X, C[i])
            oC, _ = oracle.update(L.X, a0["idx"], C[i])
            gC = host(st.C[i])
            check_centroids(gC, oC, ("fit_stack", t, L.name))
            a1 = oracle.assign(L.X, gC)                 # the final assignment is exact for the GPU's C
            assert np.array_equal(host(st.idx[i]), a1["idx"]), ("fit_stack", t, L.name)
            assert np.array_equal(host(st.counts[i]), np.bincount(a1["idx"], minlength=L.k)), L.name
            J = host(st.distortion[i])
            assert J[0] == pytest.approx(oracle.distortion(L.X, C[i], a0["idx"]), rel=REL)
            assert J[1] == pytest.approx(oracle.distortion(L.X, gC, a1["idx"]), rel=REL)
            C[i] = oC


@pytest.mark.parametrize("scale", [1e-30, 1e-9, 1e-6, 1e-3, 1e3, 1e12])
def test_update_at_any_weight_magnitude(scale):
    """The fixed-point scale follows the layer's largest magnitude: means within 1e-5 of the
    oracle's fp64 means from 1e-30 to 1e12 times Kaiming-sized weights, through the
    separate update, the fused round and a fit."""
    L = synth.resnet18_stack(k=256, layers=16)[15]              # 262,144 kernels
    X = np.ascontiguousarray((L.X.astype(np.float64) * scale).astype(np.float32))
    C0 = np.ascontiguousarray((L.C0.astype(np.float64) * scale).astype(np.float32))
    a = oracle.assign(X, C0)
    oC, oz = oracle.update(X, a["idx"], C0)
    gC, gz, _ = kq.kq_update(dev(X), dev(a["idx"]), dev(C0), with_distortion=False)
    assert np.array_equal(host(gz), oz)
    w1 = check_centroids(host(gC), oC, ("update", scale))
    st = kq.Stack([dev(X)], [dev(C0)], iters=1)
    kq.kq_assign_stack(st, distortion=False, fused_sums=True)
    kq.kq_update_stack(st, distortion_from_assign=True, sums_from_assign=True)
    assert np.array_equal(host(st.idx[0]), a["idx"])
    w2 = check_centroids(host(st.C[0]), oC, ("fused", scale))
    assert np.array_equal(host(st.C[0]).view(np.uint32), host(gC).view(np.uint32))   # the same integers
    C1, _, _, _ = kq.kq_fit_layer(dev(X), dev(C0), 1)
    check_centroids(host(C1), oC, ("fit", scale))
    print(f"scale {scale:g}: worst relative error {max(w1, w2):.2e}")


def test_validate_rejects_non_finite_kernels():
    L = synth.single_layer(k=64)[0]
    for bad in (np.nan, np.inf, -np.inf):
        X = L.X.copy()
        X[1234, 5] = bad
        Xd, C0 = dev(X), dev(L.C0)
        C = torch.full((L.k, 9), 7.0, device=DEV)
        with pytest.raises(kq.KqError) as e:
            kq.kq_fit_layer(Xd, C0, 3, C=C, validate=True)
        assert e.value.status == kq.KQ_ERR_RANGE
        assert bool((C == 7.0).all())                            # nothing written
        idx = dev(oracle.assign(L.X, L.C0)["idx"])
        with pytest.raises(kq.KqError) as e:
            kq.kq_update(Xd, idx, C0, validate=True)
        assert e.value.status == kq.KQ_ERR_RANGE
        st = kq.Stack([dev(L.X), Xd], [C0, C0], iters=1)
        with pytest.raises(kq.KqError) as e:
            kq.kq_fit_stack(st, 1, validate=True)
        assert e.value.status == kq.KQ_ERR_RANGE
        assert torch.equal(st.C[0], C0)                          # the finite layer is untouched too
    # finite inputs of any size pass the check and give the unchecked results
    Xd, C0 = dev(L.X), dev(L.C0)
    a = kq.kq_fit_layer(Xd, C0, 3, validate=True)
    b = kq.kq_fit_layer(Xd, C0, 3)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


@pytest.mark.parametrize("mode", [kq.KQ_CBQ_WKMEANS, kq.KQ_CBQ_UNIFORM])
def test_compress_stack_matches_separate_calls_and_oracle(mode):
    """kq_compress_stack on a mixed stack (k from 16 to 256, one layer with C_init the
    same buffer as C's start): every output bit for bit the separate calls'; the codebook
    quantization, streams and reconstruction bit-exact against the oracle on the GPU's fit;
    the fit's final assignment exact for its codebook."""
    layers = synth.resnet18_stack(k=64, layers=4)
    layers[1] = synth.make_layer("k16", layers[1].X, 16, 5)
    layers[2] = synth.make_layer("k256", layers[2].X, 256, 6)
    T = 4
    comp = kq.Compression([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=T, bits=6, mode=mode,
                          cbq_iters=30)
    comp.run()
    comp.run()                                      # a second call on the same buffers: the same bits
    st = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=T)
    kq.kq_fit_stack(st, T)
    for i, L in enumerate(layers):
        assert torch.equal(comp.C[i], st.C[i]) and torch.equal(comp.idx[i], st.idx[i]), L.name
        assert torch.equal(comp.counts[i], st.counts[i]) and torch.equal(comp.distortion[i], st.distortion[i])
        C, z, idx = host(comp.C[i]), host(comp.counts[i]), host(comp.idx[i])
        a = oracle.assign(L.X, C)
        assert np.array_equal(idx, a["idx"]) and np.array_equal(z, np.bincount(idx, minlength=L.k))
        if mode == kq.KQ_CBQ_WKMEANS:
            oc, ol, oh, _ = oracle.cbq_wkmeans(C, z, 6, 30)
        else:
            oc, ol, oh = oracle.cbq_uniform(C, 6)
        assert np.array_equal(host(comp.codes[i]), oc), L.name
        assert np.array_equal(host(comp.levels[i]).view(np.uint32), ol.view(np.uint32)), L.name
        assert np.array_equal(host(comp.C_hat[i]).view(np.uint32), oh.reshape(-1, 9).view(np.uint32)), L.name
        b = oracle.index_bits(L.k)
        assert np.array_equal(host(comp.packed_index_stream(i)), oracle.pack_bits(idx, b)), L.name
        assert np.array_equal(host(comp.packed_code_stream(i)), oracle.pack_bits(oc, 6)), L.name
        W = oracle.reconstruct(idx, oh.reshape(-1, 9))
        assert np.array_equal(host(comp.W_hat[i]).view(np.uint32), W.view(np.uint32)), L.name
        exact = float(np.sum((L.X.astype(np.float64) - W.astype(np.float64)) ** 2))
        assert float(host(comp.sq_error)[i]) == pytest.approx(exact, rel=1e-12), L.name


def test_compress_stack_full_resnet18_matches_fit_and_validates():
    """The benchmark's call at full size: equal to kq_fit_stack + the separate quantizer,
    packers and reconstruction, and KQ_F_VALIDATE gives the same bits on finite weights."""
    layers = synth.resnet18_stack(k=256)
    T = 3
    Xs, C0s = [dev(L.X) for L in layers], [dev(L.C0) for L in layers]
    comp = kq.Compression(Xs, C0s, iters=T)
    ev = {t: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for t in (0, 2, T)}
    for a, b in ev.values():
        a.record()
        b.record()
    comp.run(validate=True, round_events=ev)     # events on the kernel launches change nothing
    torch.cuda.synchronize()
    for t, (a, b) in ev.items():
        assert 0.001 < a.elapsed_time(b) < 50.0, t   # the assignment kernel's own duration, in ms
    st = kq.Stack(Xs, C0s, iters=T)
    kq.kq_fit_stack(st, T)
    out = kq.kq_quantize_codebook_stack(st.C, st.counts, 6, kq.KQ_CBQ_WKMEANS, 30)
    for i in range(len(layers)):
        assert torch.equal(comp.C[i], st.C[i]) and torch.equal(comp.idx[i], st.idx[i])
        assert torch.equal(comp.distortion[i], st.distortion[i])
        assert torch.equal(comp.codes[i], out[i][0]) and torch.equal(comp.C_hat[i], out[i][2])
        W = kq.kq_reconstruct(st.idx[i], out[i][2])
        assert torch.equal(comp.W_hat[i], W)
