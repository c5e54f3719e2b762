"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bars: assignment indices and fp32 best distances bit-exact (the library returns the
exact fp32 argmin); distortion within 1e-5 relative of the oracle's fp64 value;
centroids within 1e-5 relative per codeword; counts, 6-bit codes and levels, packed
streams and reconstructions bit-exact."""
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


def check_assign(X, C, tag=""):
    idx, best_d, dist = kq.kq_assign(dev(X), dev(C))
    gi, gd, gJ = host(idx), host(best_d), float(host(dist)[0])
    o = oracle.assign(X, C)
    bad = np.nonzero(gi != o["idx"])[0]
    assert bad.size == 0, f"{tag}: {bad.size} indices differ, first {bad[:5]} gpu {gi[bad[:5]]} oracle {o['idx'][bad[:5]]}"
    assert np.array_equal(gd.view(np.uint32), o["d32"].view(np.uint32)), f"{tag}: best distances differ"
    J32 = float(np.sum(o["d32"].astype(np.float64)))
    assert gJ == pytest.approx(J32, rel=1e-12, abs=1e-300), tag
    J64 = float(np.sum(o["d1"]))
    assert gJ == pytest.approx(J64, rel=REL, abs=1e-30), tag
    # against the fp64 decision only near-ties may differ (best and second-best within 1e-5)
    diff = np.nonzero(o["idx"] != o["idx64"])[0]
    for i in diff:
        assert o["d2"][i] - o["d1"][i] <= REL * o["d2"][i], (tag, i)
    return diff.size


def test_assign_single_layer_64x64():
    L = synth.single_layer(k=256)[0]
    check_assign(L.X, L.C0, "64x64 k=256 init")
    check_assign(L.X, synth.random_codebook_state(L.X, 256, 5), "64x64 k=256 jittered")


@pytest.mark.parametrize("n,k", [(1, 1), (2, 1), (1, 5), (255, 3), (256, 16), (257, 31), (1000, 33),
                                 (4133, 256), (3000, 1024), (3001, 1025), (2048, 2100), (700, 4096),
                                 (300, 7000)])
def test_assign_shapes(n, k):
    X = synth.laplace_layer(1, n, 100 + n)[:n]
    C = synth.random_codebook_state(X, k, k)
    check_assign(X, C, f"n={n} k={k}")


def test_assign_exact_ties_and_near_ties():
    rng = np.random.default_rng(3)
    # small integers: many exactly equal distances, duplicated entries
    X = rng.integers(-2, 3, (3000, 9)).astype(np.float32)
    C = rng.integers(-2, 3, (200, 9)).astype(np.float32)
    C[100:150] = C[0:50]
    check_assign(X, C, "integer grid")
    # tight clusters far from the origin: strong cancellation in |c|^2 - 2 x.c
    L = synth.stress_layer(n=20000, k=1024, n_centers=1024, seed=44)[0]
    check_assign(L.X, L.C0, "clusters")
    # a point exactly between two entries
    X = np.zeros((64, 9), np.float32)
    C = np.zeros((2, 9), np.float32)
    C[0, 0], C[1, 0] = -1.0, 1.0
    check_assign(X, C, "midpoint")


def test_assign_far_entries_and_mixed_scales():
    """The guard's bound is local (|x| and the rescored distance): entries far from every
    kernel, up to norms whose fp32 |c|^2 overflows, must neither be chosen nor hide a
    nearer entry, and kernels of very different scales (zero, 1e-25, 1e-6, 1) share one
    codebook.  Bit for bit the oracle's plain fp32 argmin."""
    rng = np.random.default_rng(77)
    base = rng.laplace(0, 0.02, (256, 9)).astype(np.float32)
    far = np.zeros((12, 9), np.float32)
    for r, mag in enumerate([1e3, -1e6, 1e12, -1e15, 1e18, 3e18, -1e19, 2e19, 3e19, 1e30, -1e35, 3e38]):
        far[r] = mag * np.sign(rng.standard_normal(9)).astype(np.float32)
    far[5, 4] = 0.0  # mixed zero and huge coordinates
    C = np.concatenate([base[:100], far[:6], base[100:], far[6:]])
    X = rng.laplace(0, 0.02, (6000, 9)).astype(np.float32)
    X[:500] *= np.float32(1e-6)
    X[500:700] *= np.float32(1e-25)
    X[700:800] = 0.0
    X[800:1000] *= np.float32(50.0)
    X[1000:1064] = C[rng.integers(0, C.shape[0] - 12, 64)]  # exact hits
    check_assign(X, C, "far entries, mixed scales")
    # the same kernels against a codebook scaled down to the tiny kernels' range
    Ct = (base * np.float32(1e-6)).astype(np.float32)
    check_assign(X, Ct, "codebook at 1e-6")
    # large kernels (|x|^2 near 1e36) against far entries: Q' passes 1e37 for some
    Xl = (rng.standard_normal((3000, 9)) * 2e17).astype(np.float32)
    Cl = np.concatenate([(rng.standard_normal((200, 9)) * 2e17).astype(np.float32), far])
    check_assign(Xl, Cl, "large kernels")


def test_assign_nonfinite_inputs_match_plain_scan():
    X = synth.normal_layer(8, 8, 5)
    X[3, 2] = np.nan
    X[7, 0] = np.inf
    C = X[10:30].copy()
    idx, best_d, _ = kq.kq_assign(dev(X), dev(C))
    o = oracle.assign(X, C)
    assert np.array_equal(host(idx), o["idx"])


def check_update(X, idx, C_old, tag=""):
    C_new, counts, J = kq.kq_update(dev(X), dev(idx), dev(C_old))
    gc, gz = host(C_new), host(counts)
    oc, oz = oracle.update(X, idx, C_old)
    ok = (idx >= 0) & (idx < C_old.shape[0])
    Jo = oracle.distortion(X[ok], C_old, idx[ok])
    assert float(host(J)[0]) == pytest.approx(Jo, rel=REL, abs=1e-30), tag
    assert np.array_equal(gz, oz), tag
    empty = oz == 0
    assert np.array_equal(gc[empty], C_old[empty]), tag
    err = np.abs(gc.astype(np.float64) - oc.astype(np.float64)).max(axis=1)
    scale = np.maximum(np.abs(oc.astype(np.float64)).max(axis=1), 1e-30)
    assert np.all(err <= REL * scale), (tag, float((err / scale).max()))
    # without a distortion the rows are read in the coalesced layout (one range) or the
    # per-row layout (several ranges); the integer sums give the same bits either way
    C2, z2, _ = kq.kq_update(dev(X), dev(idx), dev(C_old), with_distortion=False)
    assert np.array_equal(host(C2).view(np.uint32), gc.view(np.uint32)), tag
    assert np.array_equal(host(z2), gz), tag
    _, z3, _ = kq.kq_update(dev(X), dev(idx), dev(C_old), with_distortion=False, counts_only=True)
    assert np.array_equal(host(z3), gz), tag
    return gc, gz


@pytest.mark.parametrize("n,k", [(1, 1), (63, 5), (65, 7), (100, 1), (4096, 16), (4099, 256), (20000, 768),
                                 (20000, 769), (50000, 4096), (9000, 20000), (300001, 256)])
def test_update_shapes(n, k):
    X = synth.normal_layer(1, n, 7 + n)[:n]
    idx = synth.random_indices(n, k, k)
    if k > 4:
        idx[idx == 3] = 2        # an empty entry keeps its value
    C_old = synth.random_codebook_state(X, k, 1)
    check_update(X, idx, C_old, f"n={n} k={k}")


def test_update_in_place_and_ignores_bad_indices():
    X = synth.normal_layer(16, 16, 3)
    n, k = X.shape[0], 32
    idx = synth.random_indices(n, k, 9)
    C = synth.random_codebook_state(X, k, 2)
    Cd = dev(C)
    kq.kq_update(dev(X), dev(idx), Cd, C_new=Cd)
    oc, _ = oracle.update(X, idx, C)
    assert np.allclose(host(Cd), oc, rtol=REL, atol=1e-12)
    bad = idx.copy()
    bad[:10] = 77
    bad[10:20] = -1
    keep = np.arange(n) >= 20
    oc, oz = oracle.update(X[keep], bad[keep], C)
    for with_d in (True, False):
        gc, gz, _ = kq.kq_update(dev(X), dev(bad), dev(C), with_distortion=with_d)
        assert np.array_equal(host(gz), oz), with_d
        assert np.allclose(host(gc), oc, rtol=REL, atol=1e-12), with_d


def test_fit_step_locked_single_layer():
    """At every round both sides start from the oracle's codebook."""
    L = synth.single_layer(k=256)[0]
    Xd = dev(L.X)
    C = L.C0.copy()
    for t in range(20):
        idx, best_d, dist = kq.kq_assign(Xd, dev(C))
        o = oracle.assign(L.X, C)
        assert np.array_equal(host(idx), o["idx"]), t
        C_g, z_g, J_g = kq.kq_update(Xd, idx, dev(C))
        assert float(host(J_g)[0]) == pytest.approx(float(np.sum(o["d1"])), rel=REL), t
        C_o, z_o = oracle.update(L.X, o["idx"], C)
        assert np.array_equal(host(z_g), z_o), t
        err = np.abs(host(C_g).astype(np.float64) - C_o).max(axis=1)
        assert np.all(err <= REL * np.maximum(np.abs(C_o).max(axis=1), 1e-30)), t
        C = C_o


def test_fit_layer_free_running():
    L = synth.single_layer(k=256)[0]
    iters = 20
    C, idx, counts, J = kq.kq_fit_layer(dev(L.X), dev(L.C0), iters)
    gC, gi, gz, gJ = host(C), host(idx), host(counts), host(J)
    ref = oracle.fit(L.X, L.C0, iters)
    assert np.all(gJ[1:] <= gJ[:-1] * (1 + 1e-9)), gJ          # Lloyd never increases Eq. (1)
    a = oracle.assign(L.X, gC)                                  # the final assignment is exact for the final C
    assert np.array_equal(gi, a["idx"]) and np.array_equal(gz, np.bincount(a["idx"], minlength=L.k))
    assert gJ[-1] == pytest.approx(float(np.sum(a["d1"])), rel=REL)
    rel = abs(gJ[-1] - ref["J"][-1]) / ref["J"][-1]
    assert rel <= 1e-3, rel                                     # trajectories may part at fp32 rounding
    if np.array_equal(gi, ref["idx"]):
        assert rel <= REL


def test_fit_determinism_and_resume():
    L = synth.resnet18_stack(k=64, layers=1)[0]
    Xd, C0 = dev(L.X), dev(L.C0)
    a = kq.kq_fit_layer(Xd, C0, 10)
    b = kq.kq_fit_layer(Xd, C0, 10)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    half = kq.kq_fit_layer(Xd, C0, 4)
    rest = kq.kq_fit_layer(Xd, half[0].clone(), 6)
    assert torch.equal(rest[0], a[0]) and torch.equal(rest[1], a[1]) and torch.equal(rest[2], a[2])
    assert torch.equal(rest[3], a[3][4:])


def test_stack_full_size_resnet18_sampled():
    """The ResNet-18-shaped stack at full size and k = 256, in the launch
    configuration the benchmark times: two Lloyd rounds through the stack calls,
    checked on sampled kernels (assignment) and in full (update, counts)."""
    layers = synth.resnet18_stack(k=256)
    st = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=2, best_d=True)
    rng = np.random.default_rng(0)
    for t in range(2):
        C_before = [host(c) for c in st.C]
        kq.kq_assign_stack(st, dist_slot=t)
        idx = [host(i) for i in st.idx]
        Ja = [float(host(d)[t]) for d in st.distortion]
        for L, Cb, gi, gd, gJ in zip(layers, C_before, idx, st.best_d, st.distortion):
            rows = rng.choice(L.n, min(L.n, 1500), replace=False)
            o = oracle.assign(L.X[rows], Cb)
            assert np.array_equal(gi[rows], o["idx"]), (L.name, t)
            assert np.array_equal(host(gd)[rows], o["d32"]), (L.name, t)
            Jo = oracle.distortion(L.X, Cb, gi)
            assert float(host(gJ)[t]) == pytest.approx(Jo, rel=REL), (L.name, t)
        kq.kq_update_stack(st, dist_slot=t)
        for Jassign, gJ in zip(Ja, st.distortion):           # update measures the same objective
            assert float(host(gJ)[t]) == pytest.approx(Jassign, rel=1e-12)
        kq.kq_update_stack(st, dist_slot=t, counts_only=True, distortion_from_assign=True)
        for Jassign, gJ in zip(Ja, st.distortion):           # the assignment's own partials: same bits
            assert float(host(gJ)[t]) == Jassign
        for L, Cb, gi, gC, gz in zip(layers, C_before, idx, st.C, st.counts):
            oc, oz = oracle.update(L.X, gi, Cb)
            assert np.array_equal(host(gz), oz), L.name
            err = np.abs(host(gC).astype(np.float64) - oc).max(axis=1)
            assert np.all(err <= REL * np.maximum(np.abs(oc).max(axis=1), 1e-30)), L.name


def test_fit_stack_matches_fit_layer():
    layers = synth.vgg16_stack(k=64, layers=4)
    st = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=5)
    kq.kq_fit_stack(st, 5)
    for i, L in enumerate(layers):
        C, idx, counts, J = kq.kq_fit_layer(dev(L.X), dev(L.C0), 5)
        assert torch.equal(C, st.C[i]) and torch.equal(idx, st.idx[i]) and torch.equal(counts, st.counts[i])
        assert torch.equal(J, st.distortion[i])


def test_stress_layer_sampled():
    """1024 x 1024 kernels from 4096 tight clusters, k = 4096 (several LDS chunks,
    many guarded kernels): sampled exact parity of one assignment and a full update."""
    L = synth.stress_layer()[0]
    Xd = dev(L.X)
    idx, best_d, dist = kq.kq_assign(Xd, dev(L.C0))
    gi, gd = host(idx), host(best_d)
    rows = np.random.default_rng(1).choice(L.n, 3000, replace=False)
    o = oracle.assign(L.X[rows], L.C0)
    assert np.array_equal(gi[rows], o["idx"])
    assert np.array_equal(gd[rows], o["d32"])
    assert float(host(dist)[0]) == pytest.approx(float(np.sum(gd.astype(np.float64))), rel=1e-12)
    check_update(L.X, gi, L.C0, "stress update")


@pytest.mark.parametrize("mode", [kq.KQ_CBQ_UNIFORM, kq.KQ_CBQ_WKMEANS])
def test_quantize_codebook_bit_exact(mode):
    cases = []
    L = synth.single_layer(k=256)[0]
    r = oracle.fit(L.X, L.C0, 5)
    cases.append((r["C"], r["counts"]))
    rng = np.random.default_rng(2)
    cases.append((rng.laplace(0, 0.03, (1000, 9)).astype(np.float32), rng.integers(0, 500, 1000)))
    cases.append((np.full((3, 9), -0.5, np.float32), np.array([1, 2, 3])))
    tiny = rng.standard_normal((40, 9)).astype(np.float32) * np.float32(1e-30)
    tiny[0, 0] = np.float32(3e-39)      # a subnormal scalar
    cases.append((tiny, rng.integers(0, 2 ** 31 - 1, 40)))
    big = (rng.standard_normal((64, 9)) * 1e30).astype(np.float32)
    cases.append((big, rng.integers(1, 1000, 64)))
    for C, w in cases:
        codes, levels, C_hat = kq.kq_quantize_codebook(dev(C), dev(w.astype(np.int32)), 6, mode, 30)
        if mode == kq.KQ_CBQ_UNIFORM:
            oc, ol, oh = oracle.cbq_uniform(C, 6)
        else:
            oc, ol, oh, _ = oracle.cbq_wkmeans(C, w, 6, 30)
        assert np.array_equal(host(codes), oc)
        assert np.array_equal(host(levels).view(np.uint32), ol.view(np.uint32))
        assert np.array_equal(host(C_hat).view(np.uint32), oh.view(np.uint32))


@pytest.mark.parametrize("bits", [1, 2, 6, 8])
@pytest.mark.parametrize("mode", [kq.KQ_CBQ_UNIFORM, kq.KQ_CBQ_WKMEANS])
def test_quantize_codebook_ties_and_widths(mode, bits):
    """Scalars exactly halfway between grid levels (ties go to the lower level), repeated
    values, and magnitudes so far apart that fp64 distances to neighbouring levels round
    to the same value; several code widths."""
    rng = np.random.default_rng(10 + bits)
    L = (1 << bits) - 1
    mid = np.concatenate([[0.0, float(L)], np.arange(L) + 0.5, rng.integers(0, L + 1, 60)])
    mid = np.resize(mid, (len(mid) + 8) // 9 * 9).astype(np.float32).reshape(-1, 9)
    pool = np.array([1.0, -1.0, 1e-20, -1e-20, 1e-19, 3e-39, 0.0, 2.0, 1e-30], np.float32)
    mixed = rng.choice(pool, (50, 9)).astype(np.float32)
    for C in (mid, mixed):
        w = rng.integers(0, 20, C.shape[0])
        codes, levels, C_hat = kq.kq_quantize_codebook(dev(C), dev(w.astype(np.int32)), bits, mode, 30)
        if mode == kq.KQ_CBQ_UNIFORM:
            oc, ol, oh = oracle.cbq_uniform(C, bits)
        else:
            oc, ol, oh, _ = oracle.cbq_wkmeans(C, w, bits, 30)
        assert np.array_equal(host(codes), oc)
        assert np.array_equal(host(levels).view(np.uint32), ol.view(np.uint32))
        assert np.array_equal(host(C_hat).view(np.uint32), oh.view(np.uint32))


def test_quantize_codebook_stack_and_unweighted():
    layers = synth.resnet18_stack(k=16, layers=3)
    Cs = [oracle.fit(L.X, L.C0, 3)["C"] for L in layers]
    out = kq.kq_quantize_codebook_stack([dev(c) for c in Cs], None, 6, kq.KQ_CBQ_WKMEANS, 30)
    for C, (codes, levels, C_hat) in zip(Cs, out):
        oc, ol, oh, _ = oracle.cbq_wkmeans(C, np.ones(C.shape[0], np.int64), 6, 30)
        assert np.array_equal(host(codes), oc) and np.array_equal(host(levels), ol)


@pytest.mark.parametrize("bits", [1, 3, 4, 6, 8, 9, 11, 12, 16])
@pytest.mark.parametrize("count", [1, 7, 31, 32, 33, 1000, 4097])
def test_pack_unpack_bit_exact(bits, count):
    rng = np.random.default_rng(bits * 1000 + count)
    v = rng.integers(0, 1 << bits, count).astype(np.int32)
    s = kq.kq_pack_bits(dev(v), bits)
    ref = oracle.pack_bits(v, bits)
    assert np.array_equal(host(s), ref)
    back = kq.kq_unpack_bits(s, count, bits)
    assert np.array_equal(host(back), v)
    if bits <= 8:
        s8 = kq.kq_pack_bits(dev(v.astype(np.uint8)), bits)
        assert np.array_equal(host(s8), ref)


def test_reconstruct_bit_exact():
    rng = np.random.default_rng(4)
    for n, k in [(1, 1), (3, 2), (4097, 256), (262144, 256), (777, 4096)]:
        C = rng.standard_normal((k, 9)).astype(np.float32)
        idx = rng.integers(0, k, n).astype(np.int32)
        W = kq.kq_reconstruct(dev(idx), dev(C))
        assert np.array_equal(host(W), oracle.reconstruct(idx, C))
        b = oracle.index_bits(k)
        packed = kq.kq_pack_bits(dev(idx), b)
        W2 = kq.kq_reconstruct_packed(packed, b, n, dev(C))
        assert np.array_equal(host(W2), oracle.reconstruct(idx, C))


def test_pack_bits_stack_matches_single_streams():
    """One launch for many streams (mixed widths and element types, empty and zero-bit
    streams) writes exactly what the oracle packs for each."""
    rng = np.random.default_rng(21)
    specs = [(4096, 8, np.int32), (2304, 6, np.uint8), (0, 6, np.uint8), (100, 0, np.int32), (1, 1, np.int32),
             (33, 5, np.int16), (262144, 8, np.int32), (777, 12, np.int32), (4097, 16, np.int32), (5, 3, np.uint8)]
    jobs, refs = [], []
    for count, bits, dt in specs:
        hi = 1 << bits if bits else 1
        v = rng.integers(0, hi, count).astype(dt)
        jobs.append((dev(v) if count else torch.zeros(0, dtype=torch.from_numpy(v).dtype, device=DEV), bits, None))
        refs.append(oracle.pack_bits(v.astype(np.int64), bits) if count and bits else np.zeros(0, np.uint8))
    outs = kq.kq_pack_bits_stack(jobs)
    for (count, bits, _), o, r in zip(specs, outs, refs):
        assert np.array_equal(host(o), r), (count, bits)


@pytest.mark.parametrize("packed", [False, True])
def test_reconstruct_stack_and_errors(packed):
    """All layers in one launch: every W_hat bit-exact against the oracle's gather; each
    layer's squared error within 1e-12 of the exact sum and the same bits on a rerun."""
    rng = np.random.default_rng(22)
    shapes = [(1, 1), (3, 2), (4097, 256), (262144, 256), (777, 4096), (913, 16), (8192, 64)]
    layers, refs = [], []
    for n, k in shapes:
        C = rng.standard_normal((k, 9)).astype(np.float32)
        idx = rng.integers(0, k, n).astype(np.int32)
        Wref = rng.standard_normal((n, 9)).astype(np.float32)
        b = oracle.index_bits(k)
        L = {"C": dev(C), "n": n, "W_ref": dev(Wref), "sq_error": torch.zeros(1, dtype=torch.float64, device=DEV)}
        if packed:
            L["packed"], L["bits"] = kq.kq_pack_bits(dev(idx), b), b
        else:
            L["idx"] = dev(idx)
        layers.append(L)
        refs.append((oracle.reconstruct(idx, C), Wref))
    outs = kq.kq_reconstruct_stack(layers)
    first = [float(host(L["sq_error"])[0]) for L in layers]
    kq.kq_reconstruct_stack(layers)
    for L, W, (ref, Wref), (n, k), e1 in zip(layers, outs, refs, shapes, first):
        assert np.array_equal(host(W).view(np.uint32), ref.view(np.uint32)), (n, k)
        e2 = float(host(L["sq_error"])[0])
        assert e1 == e2, (n, k)
        exact = float(np.sum((Wref.astype(np.float64) - ref.astype(np.float64)) ** 2))
        assert e1 == pytest.approx(exact, rel=1e-12), (n, k)
        single = float(host(kq.kq_sq_error(L["W_ref"], W))[0])
        assert e1 == pytest.approx(single, rel=1e-12), (n, k)


@pytest.mark.parametrize("bits", [2, 6, 8])
def test_quantize_codebook_wide_path(bits):
    """Codebooks of at least 16384 scalars run on the whole GPU with the entry counts as
    weights: codes, levels and C_hat bit for bit those of the oracle and of the
    one-workgroup quantizer, in a stack mixed with small codebooks; integer-valued data
    (exact ties between levels) and zero weights included."""
    rng = np.random.default_rng(30 + bits)
    big = rng.laplace(0, 0.03, (1900, 9)).astype(np.float32)          # 17,100 scalars
    ints = rng.integers(-40, 41, (4096, 9)).astype(np.float32)        # 36,864, exact ties
    small = rng.standard_normal((256, 9)).astype(np.float32)
    Cs = [big, small, ints]
    ws = [rng.integers(0, 500, len(c)) for c in Cs]
    ws[0][::13] = 0
    ws[2][::7] = 0
    wd = [dev(w.astype(np.int32)) for w in ws]
    wide = kq.kq_quantize_codebook_stack([dev(c) for c in Cs], wd, bits, kq.KQ_CBQ_WKMEANS, 30)
    one = kq.kq_quantize_codebook_stack([dev(c) for c in Cs], wd, bits, kq.KQ_CBQ_WKMEANS, 30, wide=False)
    for C, w, a, b in zip(Cs, ws, wide, one):
        oc, ol, oh, _ = oracle.cbq_wkmeans(C, w, bits, 30)
        for got in (a, b):
            assert np.array_equal(host(got[0]), oc), (len(C), bits)
            assert np.array_equal(host(got[1]).view(np.uint32), ol.view(np.uint32)), (len(C), bits)
            assert np.array_equal(host(got[2]).view(np.uint32), oh.view(np.uint32)), (len(C), bits)
    # uniform grids never take the wide path, and need no workspace
    uni = kq.kq_quantize_codebook_stack([dev(big)], None, bits, kq.KQ_CBQ_UNIFORM, 0)
    oc, ol, oh = oracle.cbq_uniform(big, bits)
    assert np.array_equal(host(uni[0][0]), oc) and np.array_equal(host(uni[0][1]).view(np.uint32), ol.view(np.uint32))


@pytest.mark.parametrize("packed", [False, True])
def test_reconstruct_unaligned_views(packed):
    """Output, reference and index arrays that start 4 bytes past a 16-byte boundary:
    W_hat bit-exact against the oracle's gather, the squared error within 1e-12."""
    rng = np.random.default_rng(23)
    shapes = [(4097, 256), (913, 16), (300, 4096)]
    layers, refs = [], []
    for n, k in shapes:
        C = rng.standard_normal((k, 9)).astype(np.float32)
        idx = rng.integers(0, k, n).astype(np.int32)
        Wref = rng.standard_normal((n, 9)).astype(np.float32)
        wbuf = torch.empty(n * 9 + 1, dtype=torch.float32, device=DEV)
        rbuf = torch.empty(n * 9 + 1, dtype=torch.float32, device=DEV)
        rbuf[1:].copy_(dev(Wref).reshape(-1))
        L = {"C": dev(C), "n": n, "W_ref": rbuf[1:].view(n, 9), "W_hat": wbuf[1:].view(n, 9),
             "sq_error": torch.zeros(1, dtype=torch.float64, device=DEV)}
        if packed:
            L["packed"], L["bits"] = kq.kq_pack_bits(dev(idx), oracle.index_bits(k)), oracle.index_bits(k)
        else:
            ibuf = torch.empty(n + 1, dtype=torch.int32, device=DEV)
            ibuf[1:].copy_(dev(idx))
            L["idx"] = ibuf[1:]
        layers.append(L)
        refs.append((oracle.reconstruct(idx, C), Wref))
    kq.kq_reconstruct_stack(layers)
    for L, (ref, Wref), (n, k) in zip(layers, refs, shapes):
        assert L["W_hat"].data_ptr() % 16 == 4
        assert np.array_equal(host(L["W_hat"]).view(np.uint32), ref.view(np.uint32)), (n, k)
        exact = float(np.sum((Wref.astype(np.float64) - ref.astype(np.float64)) ** 2))
        assert float(host(L["sq_error"])[0]) == pytest.approx(exact, rel=1e-12), (n, k)


@pytest.mark.parametrize("which", ["resnet18_k256", "vgg16_k64_mixed"])
def test_fused_sums_equal_the_separate_update(which):
    """Assignment with fused member sums + finish-only update gives the same codebooks,
    counts and distortions as the separate update pass, bit for bit (integer sums)."""
    if which == "resnet18_k256":
        layers = synth.resnet18_stack(k=256)
    else:
        layers = synth.vgg16_stack(k=64, layers=6)
        layers[2] = synth.make_layer("k200", layers[2].X, 200, 3)   # codebooks of several sizes
    T = 3
    a = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=T)
    b = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=T)
    for t in range(T + 1):
        kq.kq_assign_stack(a, dist_slot=t, distortion=False)
        kq.kq_assign_stack(b, dist_slot=t, distortion=False, fused_sums=True)
        last = t == T
        kq.kq_update_stack(a, dist_slot=t, counts_only=last, distortion_from_assign=True)
        kq.kq_update_stack(b, dist_slot=t, counts_only=last, distortion_from_assign=True, sums_from_assign=True)
        for i in range(len(layers)):
            assert torch.equal(a.C[i], b.C[i]) and torch.equal(a.counts[i], b.counts[i]), (which, t, i)
            assert torch.equal(a.idx[i], b.idx[i]), (which, t, i)
    for i in range(len(layers)):
        assert torch.equal(a.distortion[i], b.distortion[i]), i
    # the fits take the fused path by themselves: the same as the separate rounds above
    c = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=T)
    kq.kq_fit_stack(c, T)
    for i in range(len(layers)):
        assert torch.equal(a.C[i], c.C[i]) and torch.equal(a.idx[i], c.idx[i]), i
        assert torch.equal(a.counts[i], c.counts[i]) and torch.equal(a.distortion[i], c.distortion[i]), i


def test_fused_sums_need_small_codebooks():
    layers = synth.stress_layer(n=5000, k=300, n_centers=300, seed=9)
    st = kq.Stack([dev(L.X) for L in layers], [dev(L.C0) for L in layers], iters=1)
    with pytest.raises(kq.KqError):
        kq.kq_assign_stack(st, fused_sums=True)
    with pytest.raises(kq.KqError):
        kq.kq_update_stack(st, sums_from_assign=True)


@pytest.mark.parametrize("bits", [1, 3, 6])
def test_quantize_codebook_edge_weights_and_magnitudes(bits):
    """Weighted k-means codebooks bit for bit the oracle's at 1, 3 and 6 bits: codebooks on
    both sides of the size up to which the scalars are held in LDS (910 and 911 entries),
    zero weights, a level that lands a few 1e-10 from zero after the first round (weights
    near 2^30), and a value far below the largest magnitude."""
    rng = np.random.default_rng(40 + bits)
    cases = []
    for k in (1, 7, 255, 910, 911):
        C = rng.laplace(0, 0.03, (k, 9)).astype(np.float32)
        w = rng.integers(0, 300, k)
        w[::5] = 0
        cases.append((C, w))
    # the middle cell holds -1 and 1 with weights 2^30 and 2^30 + 1: its level is 1 / (2^31 + 1)
    C = np.array([[-5.0] * 9, [-1.0] * 9, [1.0] * 9, [7.0] * 9], np.float32)
    cases.append((C, np.array([1, 1 << 30, (1 << 30) + 1, 1])))
    C = rng.standard_normal((200, 9)).astype(np.float32)
    C[3, 4] = np.float32(1e-12)                                   # a value far below the largest
    cases.append((C, rng.integers(1, 50, 200)))
    for C, w in cases:
        codes, levels, C_hat = kq.kq_quantize_codebook(dev(C), dev(w.astype(np.int32)), bits, kq.KQ_CBQ_WKMEANS, 30)
        oc, ol, oh, _ = oracle.cbq_wkmeans(C, w, bits, 30)
        assert np.array_equal(host(codes), oc), (C.shape, bits)
        assert np.array_equal(host(levels).view(np.uint32), ol.view(np.uint32)), (C.shape, bits)
        assert np.array_equal(host(C_hat).view(np.uint32), oh.view(np.uint32)), (C.shape, bits)


def test_quantize_codebook_6bit_rounds_bit_exact_over_many_codebooks():
    """6-bit weighted k-means codebooks whose values meet the exactness condition run their
    rounds in integers (two 64-bit sums per level, codes from thresholds); rounds whose levels
    are unsorted or come near zero search the levels instead, and codebooks whose values do
    not meet the condition take the digit sums.  Bit for bit the oracle's over many seeds:
    sizes up to and past the 4096-scalar limit (455 and 456 entries), constant and
    few-valued codebooks (equal levels), zero and huge weights, mixed magnitudes."""
    rng = np.random.default_rng(2024)
    cases = []
    for t in range(24):
        k = int(rng.integers(1, 460))
        C = rng.laplace(0, 10.0 ** rng.uniform(-4, 1), (k, 9)).astype(np.float32)
        w = rng.integers(0, 1 << int(rng.integers(1, 31)), k)
        if t % 3 == 0:
            w[rng.random(k) < 0.3] = 0
        cases.append((C, w))
    cases.append((np.full((40, 9), 0.25, np.float32), np.ones(40, np.int64)))           # one value
    cases.append((rng.choice(np.float32([-1, 0.5, 3]), (90, 9)), rng.integers(1, 9, 90)))  # three values
    cases.append((np.zeros((7, 9), np.float32), np.ones(7, np.int64)))                   # all zero
    for k in (455, 456):
        cases.append((rng.standard_normal((k, 9)).astype(np.float32), rng.integers(1, 1000, k)))
    C = rng.standard_normal((300, 9)).astype(np.float32)
    C[17, 2] = np.float32(3e-9)                                 # below 2^(e(M) - 29): digit sums
    cases.append((C, rng.integers(1, 100, 300)))
    for i, (C, w) in enumerate(cases):
        codes, levels, C_hat = kq.kq_quantize_codebook(dev(C), dev(w.astype(np.int32)), 6, kq.KQ_CBQ_WKMEANS, 30)
        oc, ol, oh, _ = oracle.cbq_wkmeans(C, w, 6, 30)
        assert np.array_equal(host(codes), oc), i
        assert np.array_equal(host(levels).view(np.uint32), ol.view(np.uint32)), i
        assert np.array_equal(host(C_hat).view(np.uint32), oh.view(np.uint32)), i
