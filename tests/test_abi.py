"""The C-ABI library loads without a GPU, exports every function include/kq.h
declares, and rejects bad arguments on the host before touching HIP."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kq.h")

kq = pytest.importorskip("paper_2003_05148_amd")
lib = kq.lib


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kq_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 15
    raw = ctypes.CDLL(kq.LIB_PATH)
    for name in names:
        assert hasattr(raw, name), name
    assert sorted(kq.EXPORTED) == names


def test_status_strings_and_version():
    assert lib.kq_abi_version() == 10
    for s in range(6):
        assert len(lib.kq_status_string(s)) > 0
    assert lib.kq_status_string(99) == b"unknown status"


def test_workspace_sizes():
    a = lib.kq_workspace_bytes(kq.KQ_OP_ASSIGN, 4096, 256, 9)
    assert a > 0 and a % 256 == 0
    assert lib.kq_workspace_bytes(kq.KQ_OP_FIT, 4096, 256, 9) == a
    assert lib.kq_workspace_bytes(kq.KQ_OP_ASSIGN, 0, 256, 9) == 0
    assert lib.kq_workspace_bytes(kq.KQ_OP_ASSIGN, 10, 0, 9) == 0
    assert lib.kq_workspace_bytes(kq.KQ_OP_ASSIGN, 10, kq.KQ_MAX_K + 1, 9) == 0
    assert lib.kq_workspace_bytes(7, 10, 4, 9) == 0
    big = lib.kq_workspace_bytes(kq.KQ_OP_UPDATE, 1 << 20, 4096, 9)
    assert big >= 8 * 10 * 4096


FAKE = 0x10000  # a well-aligned non-null pointer value; never dereferenced on these paths


def assign(**kw):
    a = dict(X=FAKE, n=100, dim=9, C=FAKE, k=8, idx=FAKE, best_d=None, dist=None, flags=0, ws=None, wsb=0, s=None)
    a.update(kw)
    return lib.kq_assign(a["X"], a["n"], a["dim"], a["C"], a["k"], a["idx"], a["best_d"], a["dist"], a["flags"],
                         a["ws"], a["wsb"], a["s"])


def test_assign_argument_errors():
    assert assign(dim=8) == kq.KQ_ERR_UNSUPPORTED
    assert assign(k=kq.KQ_MAX_K + 1) == kq.KQ_ERR_UNSUPPORTED
    assert assign(n=0) == kq.KQ_ERR_ARG
    assert assign(n=1 << 31) == kq.KQ_ERR_ARG
    assert assign(k=0) == kq.KQ_ERR_ARG
    assert assign(X=None) == kq.KQ_ERR_ARG
    assert assign(C=None) == kq.KQ_ERR_ARG
    assert assign(idx=None) == kq.KQ_ERR_ARG
    assert assign(X=FAKE + 2) == kq.KQ_ERR_ARG
    assert assign(best_d=FAKE + 1) == kq.KQ_ERR_ARG
    assert assign(dist=FAKE + 4) == kq.KQ_ERR_ARG
    assert assign(flags=1) == kq.KQ_ERR_ARG
    # a distortion output needs a workspace of the queried size
    assert assign(dist=FAKE) == kq.KQ_ERR_WORKSPACE
    need = lib.kq_workspace_bytes(kq.KQ_OP_ASSIGN, 100, 8, 9)
    assert assign(dist=FAKE, ws=FAKE, wsb=need - 1) == kq.KQ_ERR_WORKSPACE
    assert assign(dist=FAKE, ws=FAKE + 128, wsb=need) == kq.KQ_ERR_WORKSPACE


def test_update_and_fit_argument_errors():
    up = lambda **kw: lib.kq_update(kw.get("X", FAKE), kw.get("n", 100), kw.get("dim", 9), kw.get("idx", FAKE),
                                    kw.get("k", 8), kw.get("Co", FAKE), kw.get("Cn", FAKE), kw.get("cnt", None),
                                    kw.get("dist", None), kw.get("flags", 0), kw.get("ws", None), kw.get("wsb", 0),
                                    None)
    assert up(dim=4) == kq.KQ_ERR_UNSUPPORTED
    assert up(n=-1) == kq.KQ_ERR_ARG
    assert up(Co=None) == kq.KQ_ERR_ARG
    assert up(cnt=FAKE + 2) == kq.KQ_ERR_ARG
    assert up(dist=FAKE + 4) == kq.KQ_ERR_ARG
    assert up(flags=2) == kq.KQ_ERR_ARG
    assert up() == kq.KQ_ERR_WORKSPACE
    fit = lambda **kw: lib.kq_fit_layer(FAKE, kw.get("n", 100), 9, kw.get("k", 8), kw.get("Ci", FAKE),
                                        kw.get("iters", 3), FAKE, FAKE, None, None, 0, kw.get("ws", None),
                                        kw.get("wsb", 0), None)
    assert fit(k=101) == kq.KQ_ERR_ARG          # a fit needs k <= n
    assert fit(iters=-1) == kq.KQ_ERR_ARG
    assert fit(Ci=None) == kq.KQ_ERR_ARG
    assert fit() == kq.KQ_ERR_WORKSPACE


def test_stack_argument_errors():
    arr = (kq.KqLayer * 2)()
    arr[0] = kq.KqLayer(FAKE, 4096, 256, FAKE, FAKE, None, FAKE, None)
    arr[1] = kq.KqLayer(FAKE, 100, 200, FAKE, FAKE, None, FAKE, None)
    p = ctypes.cast(arr, ctypes.c_void_p)
    need = lib.kq_stack_workspace_bytes(p, 2)
    assert need == lib.kq_workspace_bytes(0, 4096, 256, 9) + lib.kq_workspace_bytes(0, 100, 200, 9)
    assert lib.kq_fit_stack(p, 2, 3, 0, FAKE, need, None) == kq.KQ_ERR_ARG      # k > n in layer 1
    assert lib.kq_assign_stack(p, 2, 0, 0, FAKE, need - 1, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_assign_stack(p, 0, 0, 0, FAKE, need, None) == kq.KQ_ERR_ARG
    assert lib.kq_assign_stack(None, 2, 0, 0, FAKE, need, None) == kq.KQ_ERR_ARG
    assert lib.kq_assign_stack(p, 2, -1, 0, FAKE, need, None) == kq.KQ_ERR_ARG
    arr[1] = kq.KqLayer(FAKE, 100, kq.KQ_MAX_K + 1, FAKE, FAKE, None, FAKE, None)
    assert lib.kq_update_stack(p, 2, 0, 0, FAKE, need, None) == kq.KQ_ERR_UNSUPPORTED


def test_cbq_stack_workspace_rules():
    """Only weighted k-means codebooks of at least 16384 scalars need the workspace; its
    size is that of the largest; a missing or short workspace is refused before any launch."""
    arr = (kq.KqCbqLayer * 3)()
    for i, k in enumerate([16, 1821, 1820]):
        arr[i] = kq.KqCbqLayer(FAKE, k, None, FAKE, FAKE, None)
    P = ctypes.cast(arr, ctypes.c_void_p)
    need = lib.kq_quantize_codebook_stack_workspace_bytes(P, 3, 6)
    assert need == lib.kq_quantize_scalars_workspace_bytes(1821 * 9, 6) > 0
    assert lib.kq_quantize_codebook_stack_workspace_bytes(P, 1, 6) == 0      # k = 16 alone
    assert lib.kq_quantize_codebook_stack_workspace_bytes(P, 3, 9) == 0      # bits outside 1..8
    assert lib.kq_quantize_codebook_stack_ws(P, 3, 6, kq.KQ_CBQ_WKMEANS, 30, None, 0, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_quantize_codebook_stack_ws(P, 3, 6, kq.KQ_CBQ_WKMEANS, 30, FAKE, need - 1, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_quantize_codebook_stack_ws(P, 3, 9, kq.KQ_CBQ_WKMEANS, 30, FAKE, need, None) == kq.KQ_ERR_UNSUPPORTED
    assert lib.kq_quantize_codebook_stack_ws(P, 0, 6, kq.KQ_CBQ_WKMEANS, 30, FAKE, need, None) == kq.KQ_ERR_ARG


def test_cbq_pack_reconstruct_argument_errors():
    q = lambda **kw: lib.kq_quantize_codebook(kw.get("C", FAKE), kw.get("k", 8), kw.get("dim", 9), None,
                                              kw.get("bits", 6), kw.get("mode", 0), kw.get("iters", 30),
                                              kw.get("codes", FAKE), kw.get("levels", FAKE), None, None)
    assert q(dim=3) == kq.KQ_ERR_UNSUPPORTED
    assert q(bits=9) == kq.KQ_ERR_UNSUPPORTED
    assert q(bits=0) == kq.KQ_ERR_UNSUPPORTED
    assert q(mode=5) == kq.KQ_ERR_ARG
    assert q(iters=-2) == kq.KQ_ERR_ARG
    assert q(codes=None) == kq.KQ_ERR_ARG
    assert q(k=0) == kq.KQ_ERR_ARG
    assert lib.kq_pack_bits(FAKE, 4, 10, 17, FAKE, None) == kq.KQ_ERR_UNSUPPORTED
    assert lib.kq_pack_bits(FAKE, 3, 10, 4, FAKE, None) == kq.KQ_ERR_ARG
    assert lib.kq_pack_bits(FAKE, 4, 10, 4, FAKE + 2, None) == kq.KQ_ERR_ARG
    assert lib.kq_pack_bits(FAKE + 2, 4, 10, 4, FAKE, None) == kq.KQ_ERR_ARG
    assert lib.kq_pack_bits(None, 4, 0, 4, None, None) == kq.KQ_OK             # nothing to do
    assert lib.kq_pack_bits(None, 4, 10, 0, None, None) == kq.KQ_OK            # zero-bit fields
    assert lib.kq_unpack_bits(None, 10, 4, FAKE, None) == kq.KQ_ERR_ARG
    assert lib.kq_reconstruct(FAKE, 10, FAKE, 4, 9, FAKE + 2, None) == kq.KQ_ERR_ARG   # W_hat 4-B aligned
    assert lib.kq_reconstruct(FAKE, 10, FAKE, 4, 8, FAKE, None) == kq.KQ_ERR_UNSUPPORTED
    assert lib.kq_reconstruct_packed(None, 4, 10, FAKE, 4, 9, FAKE, None) == kq.KQ_ERR_ARG
    assert lib.kq_reconstruct_packed(FAKE + 2, 4, 10, FAKE, 4, 9, FAKE, None) == kq.KQ_ERR_ARG  # stream read as dwords
    assert lib.kq_workspace_init(FAKE + 8, 100, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_sq_error(FAKE, FAKE, 0, FAKE, FAKE, 1 << 20, None) == kq.KQ_ERR_ARG
    assert lib.kq_sq_error(FAKE, FAKE, 100, FAKE, FAKE, 0, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_workspace_init(FAKE, 0, None) == kq.KQ_OK


def test_python_binding_rejects_cpu_tensors():
    import torch
    X = torch.zeros(10, 9)
    with pytest.raises(TypeError):
        kq.kq_assign(X, X[:2])


def test_stack_pack_and_reconstruct_argument_errors():
    jobs = (kq.KqPackJob * 3)()
    jobs[0] = kq.KqPackJob(FAKE, 4, 8, 100, FAKE)
    jobs[1] = kq.KqPackJob(None, 1, 0, 100, None)      # zero-bit stream: nothing to write
    jobs[2] = kq.KqPackJob(FAKE, 1, 6, 0, None)        # empty stream
    p = ctypes.cast(jobs, ctypes.c_void_p)
    assert lib.kq_pack_bits_stack(None, 1, None) == kq.KQ_ERR_ARG
    assert lib.kq_pack_bits_stack(p, 0, None) == kq.KQ_ERR_ARG
    assert lib.kq_pack_bits_stack(p, kq.KQ_MAX_PACK_JOBS + 1, None) == kq.KQ_ERR_ARG
    jobs[0] = kq.KqPackJob(FAKE, 4, 17, 100, FAKE)
    assert lib.kq_pack_bits_stack(p, 3, None) == kq.KQ_ERR_UNSUPPORTED
    jobs[0] = kq.KqPackJob(FAKE, 3, 8, 100, FAKE)
    assert lib.kq_pack_bits_stack(p, 3, None) == kq.KQ_ERR_ARG
    jobs[0] = kq.KqPackJob(FAKE, 4, 8, 100, FAKE + 2)
    assert lib.kq_pack_bits_stack(p, 3, None) == kq.KQ_ERR_ARG

    lay = (kq.KqReconLayer * 2)()
    ok = kq.KqReconLayer(FAKE, None, 0, 256, 4096, FAKE, FAKE, FAKE, FAKE)
    lay[0] = ok
    lay[1] = kq.KqReconLayer(None, FAKE, 8, 256, 100, FAKE, FAKE, None, None)
    q = ctypes.cast(lay, ctypes.c_void_p)
    need = lib.kq_reconstruct_stack_workspace_bytes(q, 2)
    assert need >= 16 and need % 256 == 0        # partials of the layer that asks for its error
    assert lib.kq_reconstruct_stack(q, 2, None, 0, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_reconstruct_stack(q, 2, FAKE, need - 1, None) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_reconstruct_stack(q, 0, FAKE, need, None) == kq.KQ_ERR_ARG
    assert lib.kq_reconstruct_stack(q, kq.KQ_MAX_STACK + 1, FAKE, need, None) == kq.KQ_ERR_ARG
    lay[0] = kq.KqReconLayer(FAKE, None, 0, 256, 4096, FAKE, FAKE, None, FAKE)   # error without W_ref
    assert lib.kq_reconstruct_stack(q, 2, FAKE, need, None) == kq.KQ_ERR_ARG
    lay[0] = kq.KqReconLayer(FAKE, None, 0, kq.KQ_MAX_K + 1, 4096, FAKE, FAKE, FAKE, FAKE)
    assert lib.kq_reconstruct_stack(q, 2, FAKE, need, None) == kq.KQ_ERR_UNSUPPORTED
    lay[0] = ok
    lay[1] = kq.KqReconLayer(None, None, 8, 256, 100, FAKE, FAKE, None, None)     # no index source
    assert lib.kq_reconstruct_stack(q, 2, FAKE, need, None) == kq.KQ_ERR_ARG
    lay[1] = kq.KqReconLayer(None, FAKE, 17, 256, 100, FAKE, FAKE, None, None)
    assert lib.kq_reconstruct_stack(q, 2, FAKE, need, None) == kq.KQ_ERR_UNSUPPORTED
    assert lib.kq_reconstruct_stack_workspace_bytes(q, 2) == 0


def test_yinyang_workspace_and_argument_errors():
    a = lib.kq_yinyang_workspace_bytes(4096, 256, 0)
    assert a > lib.kq_workspace_bytes(kq.KQ_OP_FIT, 4096, 256, 9) and a % 256 == 0
    assert lib.kq_yinyang_workspace_bytes(4096, 256, 8) > lib.kq_yinyang_workspace_bytes(4096, 256, 4)
    assert lib.kq_yinyang_workspace_bytes(4096, 256, 65) == 0      # more groups than mask bits
    assert lib.kq_yinyang_workspace_bytes(100, 8, 9) == 0          # more groups than entries
    assert lib.kq_yinyang_workspace_bytes(7, 8, 0) == 0            # k > n
    assert lib.kq_yinyang_workspace_bytes(100, 1, 0) > 0           # one entry, one group
    nb = lib.kq_yinyang_workspace_bytes(100, 8, 0)

    def init(**kw):
        a = dict(X=FAKE, n=100, dim=9, C=FAKE, k=8, g=0, idx=FAKE, bd=None, dist=None, ws=FAKE, wsb=nb)
        a.update(kw)
        return lib.kq_yinyang_init(a["X"], a["n"], a["dim"], a["C"], a["k"], a["g"], a["idx"], a["bd"], a["dist"],
                                   a["ws"], a["wsb"], None)

    assert init(dim=4) == kq.KQ_ERR_UNSUPPORTED
    assert init(k=101) == kq.KQ_ERR_ARG
    assert init(g=9) == kq.KQ_ERR_ARG
    assert init(X=None) == kq.KQ_ERR_ARG
    assert init(C=FAKE + 2) == kq.KQ_ERR_ARG
    assert init(wsb=nb - 1) == kq.KQ_ERR_WORKSPACE
    assert init(ws=FAKE + 64) == kq.KQ_ERR_WORKSPACE

    def step(**kw):
        a = dict(X=FAKE, n=100, C0=FAKE, C=FAKE, k=8, idx=FAKE, st=None, ws=FAKE, wsb=nb)
        a.update(kw)
        return lib.kq_yinyang_assign(a["X"], a["n"], 9, a["C0"], a["C"], a["k"], 0, a["idx"], None, None, a["st"],
                                     a["ws"], a["wsb"], None)

    assert step(C0=None) == kq.KQ_ERR_ARG
    assert step(st=FAKE + 4) == kq.KQ_ERR_ARG
    assert step(n=0) == kq.KQ_ERR_ARG
    assert step(wsb=0) == kq.KQ_ERR_WORKSPACE

    def fit(**kw):
        a = dict(X=FAKE, n=100, k=8, C0=FAKE, it=3, C=FAKE, idx=FAKE, ws=FAKE, wsb=nb)
        a.update(kw)
        return lib.kq_fit_layer_yinyang(a["X"], a["n"], 9, a["k"], a["C0"], a["it"], 0, a["C"], a["idx"], None, None,
                                        None, a["ws"], a["wsb"], None)

    assert fit(it=-1) == kq.KQ_ERR_ARG
    assert fit(C=None) == kq.KQ_ERR_ARG
    assert fit(k=kq.KQ_MAX_K + 1) == kq.KQ_ERR_UNSUPPORTED
    assert fit(wsb=100) == kq.KQ_ERR_WORKSPACE


def test_grad_step_argument_errors():
    nb = lib.kq_workspace_bytes(kq.KQ_OP_GRAD, 100, 8, 9)
    assert nb == lib.kq_workspace_bytes(kq.KQ_OP_UPDATE, 100, 8, 9) and nb > 0

    def step(**kw):
        a = dict(G=FAKE, n=100, dim=9, idx=FAKE, k=8, C0=FAKE, gamma=0.1, C=FAKE, z=None, ws=FAKE, wsb=nb)
        a.update(kw)
        return lib.kq_codebook_grad_step(a["G"], a["n"], a["dim"], a["idx"], a["k"], a["C0"], a["gamma"], a["C"],
                                         a["z"], a["ws"], a["wsb"], None)

    assert step(dim=3) == kq.KQ_ERR_UNSUPPORTED
    assert step(k=kq.KQ_MAX_K + 1) == kq.KQ_ERR_UNSUPPORTED
    assert step(gamma=float("nan")) == kq.KQ_ERR_ARG
    assert step(gamma=float("inf")) == kq.KQ_ERR_ARG
    assert step(G=None) == kq.KQ_ERR_ARG
    assert step(C=FAKE + 1) == kq.KQ_ERR_ARG
    assert step(z=FAKE + 2) == kq.KQ_ERR_ARG
    assert step(n=0) == kq.KQ_ERR_ARG
    assert step(wsb=nb - 1) == kq.KQ_ERR_WORKSPACE
    assert lib.kq_codebook_grad_step_stack(None, 1, 0.1, FAKE, nb, None) == kq.KQ_ERR_ARG


def test_quantize_scalars_argument_errors():
    nb = lib.kq_quantize_scalars_workspace_bytes(1000, 6)
    assert nb > 0 and lib.kq_quantize_scalars_workspace_bytes(1000, 9) == 0
    assert lib.kq_quantize_scalars_workspace_bytes(0, 6) == 0
    assert lib.kq_quantize_scalars_workspace_bytes(1 << 31, 6) == 0

    def q(**kw):
        a = dict(v=FAKE, m=1000, bits=6, it=30, codes=FAKE, lev=FAKE, vh=None, r=None, fl=0, ws=FAKE, wsb=nb)
        a.update(kw)
        return lib.kq_quantize_scalars(a["v"], a["m"], a["bits"], a["it"], a["codes"], a["lev"], a["vh"], a["r"],
                                       a["fl"], a["ws"], a["wsb"], None)

    assert q(fl=kq.KQ_F_EXACT_SEARCH | kq.KQ_F_THRESHOLDS) == kq.KQ_ERR_ARG
    assert q(fl=1) == kq.KQ_ERR_ARG

    assert q(bits=0) == kq.KQ_ERR_UNSUPPORTED
    assert q(bits=9) == kq.KQ_ERR_UNSUPPORTED
    assert q(m=0) == kq.KQ_ERR_ARG
    assert q(it=-1) == kq.KQ_ERR_ARG
    assert q(v=None) == kq.KQ_ERR_ARG
    assert q(lev=FAKE + 2) == kq.KQ_ERR_ARG
    assert q(vh=FAKE + 1) == kq.KQ_ERR_ARG
    assert q(wsb=nb - 1) == kq.KQ_ERR_WORKSPACE


def test_search_argument_errors():
    nb = lib.kq_search_workspace_bytes(1000, 300, 10)
    assert nb >= lib.kq_workspace_bytes(kq.KQ_OP_FIT, 1000, 256, 9)     # covers every trial size
    assert lib.kq_search_workspace_bytes(100, 101, 10) == 0
    k = ctypes.c_int32(0)

    def srch(**kw):
        a = dict(X=FAKE, n=1000, dim=9, Cc=FAKE, ni=300, r=0.5, mi=8, li=10, C=FAKE, idx=FAKE, k=ctypes.byref(k),
                 ws=FAKE, wsb=nb)
        a.update(kw)
        return lib.kq_search_codebook_size(a["X"], a["n"], a["dim"], a["Cc"], a["ni"], a["r"], a["mi"], a["li"],
                                           a["C"], a["idx"], a["k"], None, None, None, a["ws"], a["wsb"], None)

    assert srch(dim=8) == kq.KQ_ERR_UNSUPPORTED
    assert srch(ni=1001) == kq.KQ_ERR_ARG
    assert srch(r=-0.1) == kq.KQ_ERR_ARG
    assert srch(r=float("nan")) == kq.KQ_ERR_ARG
    assert srch(mi=-1) == kq.KQ_ERR_ARG
    assert srch(k=None) == kq.KQ_ERR_ARG
    assert srch(wsb=nb - 1) == kq.KQ_ERR_WORKSPACE


# ---- host-only helpers: computed on the host, checked without a GPU -------------------------

def test_forgy_select_matches_the_oracle():
    """kq_forgy_select (host C) picks the same kernels as the oracle's reading of the
    initialisation, bit for bit, on the hand-worked case and on stacks with copies, signed
    zeros and NaN kernels; k above the number of distinct kernels is refused."""
    import numpy as np

    import oracle
    import synth
    from test_oracle_forgy import HAND_X, golden

    for seed, k, expected in golden()[1]:
        assert kq.kq_forgy_select(HAND_X, k, seed).tolist() == expected
    rng = np.random.default_rng(11)
    X = rng.standard_normal((3000, 9)).astype(np.float32)
    X[1000:1500] = X[:500]
    X[2000] = 0.0
    X[2001] = -0.0
    X[2002, 3] = np.nan
    cases = [(X, 2499, 0), (X, 64, 2 ** 64 - 1), (X, 1, 5), (synth.resnet18_stack(k=16, layers=1)[0].X, 4096, 2000),
             (synth.stress_layer(n=100000, k=4096, n_centers=4096, seed=4)[0].X, 4096, 4000)]
    for Xc, k, seed in cases:
        assert np.array_equal(kq.kq_forgy_select(Xc, k, seed), oracle.forgy_select(Xc, k, seed)), (k, seed)
    sel = np.zeros(3, np.int64)
    P = ctypes.c_void_p
    xp = np.ascontiguousarray(HAND_X).ctypes.data_as(P)
    assert lib.kq_forgy_select(xp, 7, 9, 6, 1234567, sel.ctypes.data_as(P)) == kq.KQ_ERR_ARG   # 5 distinct
    assert sel.tolist() == [0, 0, 0]                                                           # untouched
    assert lib.kq_forgy_select(xp, 7, 9, 8, 1, sel.ctypes.data_as(P)) == kq.KQ_ERR_ARG         # k > n
    assert lib.kq_forgy_select(xp, 7, 8, 3, 1, sel.ctypes.data_as(P)) == kq.KQ_ERR_UNSUPPORTED
    assert lib.kq_forgy_select(None, 7, 9, 3, 1, sel.ctypes.data_as(P)) == kq.KQ_ERR_ARG
    assert lib.kq_forgy_select(xp, 7, 9, 3, 1, None) == kq.KQ_ERR_ARG


def test_accounting_matches_the_paper_and_the_oracle():
    """Eq. (4), (6), (7) in the library: the figures of Sec. 4.2.1 (golden file) and the
    oracle's formulas, which the golden tables pin, on a grid of sizes."""
    import oracle
    from test_oracle_pack_accounting import rows

    for _layer, n, k, cr_k, cr_kc, beta_kc in rows("vgg_k128_ratios.txt"):
        B, r32, _ = kq.kq_accounting(int(n), int(k), 32)
        _, r6, b6 = kq.kq_accounting(int(n), int(k), 6)
        assert abs(r32 - float(cr_k)) <= 0.01 and abs(r6 - float(cr_kc)) <= 0.01 and abs(b6 - float(beta_kc)) <= 0.001
    for k in (1, 2, 3, 4, 5, 60, 192, 255, 256, 257, 4096, 7679, 65536):
        assert kq.index_bits(k) == oracle.index_bits(k)
        for n in (1, 192, 4096, 262144):
            for bc in (6, 32):
                B, r, beta = kq.kq_accounting(n, k, bc)
                assert B == oracle.storage_bits(n, k, bc)
                assert r == oracle.compression_ratio(n, k, bc) and beta == oracle.bits_per_param(n, k, bc)
    assert kq.kq_accounting(10 ** 9, 2, 32)[1] == pytest.approx(288, rel=1e-6)   # the limit of Sec. 3.3
    assert lib.kq_index_bits(0) == -1
    assert lib.kq_accounting(0, 4, 9, 6, None, None, None) == kq.KQ_ERR_ARG
    assert lib.kq_accounting(4, 4, 9, 0, None, None, None) == kq.KQ_ERR_ARG


def test_validate_flag_and_compress_argument_errors():
    # KQ_F_VALIDATE is accepted by the calls that form member sums, refused elsewhere
    assert lib.kq_assign(FAKE, 100, 9, FAKE, 8, FAKE, None, None, kq.KQ_F_VALIDATE, None, 0, None) == kq.KQ_ERR_ARG
    up = lambda f: lib.kq_update(FAKE, 100, 9, FAKE, 8, FAKE, FAKE, None, None, f, None, 0, None)
    assert up(kq.KQ_F_VALIDATE) == kq.KQ_ERR_WORKSPACE and up(kq.KQ_F_VALIDATE | 128) == kq.KQ_ERR_ARG
    fit = lambda f: lib.kq_fit_layer(FAKE, 100, 9, 8, FAKE, 3, FAKE, FAKE, None, None, f, None, 0, None)
    assert fit(kq.KQ_F_VALIDATE) == kq.KQ_ERR_WORKSPACE and fit(kq.KQ_F_FUSED_SUMS) == kq.KQ_ERR_ARG
    # the compression pass
    arr = (kq.KqCompressLayer * 2)()
    good = dict(X=FAKE, n=4096, k=256, C_init=FAKE, C=FAKE, idx=FAKE, counts=FAKE, distortion=None, codes=FAKE,
                levels=FAKE, C_hat=FAKE, packed_idx=FAKE, packed_codes=FAKE, W_hat=FAKE, sq_error=FAKE)
    arr[0] = kq.KqCompressLayer(**good)
    arr[1] = kq.KqCompressLayer(**dict(good, n=100, k=16))
    P = ctypes.cast(arr, ctypes.c_void_p)
    need = lib.kq_compress_workspace_bytes(P, 2, 6)
    fit_need = lib.kq_workspace_bytes(0, 4096, 256, 9) + lib.kq_workspace_bytes(0, 100, 16, 9)
    assert need >= fit_need and need % 256 == 0
    run = lambda n_layers=2, iters=30, mode=0, bits=6, cit=30, flags=0, ws=FAKE, wsb=need: lib.kq_compress_stack(
        P, n_layers, iters, mode, bits, cit, flags, None, ws, wsb, None)
    assert run(bits=9) == kq.KQ_ERR_UNSUPPORTED
    assert run(n_layers=0) == kq.KQ_ERR_ARG and run(iters=-1) == kq.KQ_ERR_ARG and run(mode=3) == kq.KQ_ERR_ARG
    assert run(cit=-1) == kq.KQ_ERR_ARG and run(flags=kq.KQ_F_FUSED_SUMS) == kq.KQ_ERR_ARG
    assert run(wsb=need - 1) == kq.KQ_ERR_WORKSPACE and run(ws=FAKE + 64) == kq.KQ_ERR_WORKSPACE
    for field, value in [("k", 4097), ("C_init", None), ("counts", None), ("C_hat", None), ("X", FAKE + 2),
                         ("packed_idx", FAKE + 2), ("W_hat", None)]:
        arr[0] = kq.KqCompressLayer(**dict(good, **{field: value}))
        assert run() == kq.KQ_ERR_ARG, field            # (W_hat None with sq_error set)
    arr[0] = kq.KqCompressLayer(**dict(good, k=kq.KQ_MAX_K + 1, n=1 << 20))
    assert run() == kq.KQ_ERR_UNSUPPORTED
    arr[0] = kq.KqCompressLayer(**dict(good, packed_idx=None, packed_codes=None, W_hat=None, sq_error=None))
    assert lib.kq_compress_workspace_bytes(P, 2, 6) >= fit_need


def test_python_stack_wrappers_check_the_distortion_slot():
    """kq_assign_stack / kq_update_stack refuse a slot outside the distortion history before
    calling the library (the C side only sees device pointers and cannot check it)."""
    import types

    import torch
    fake = types.SimpleNamespace(distortion=[torch.zeros(4, dtype=torch.float64)], layers=None, n_layers=1)
    for slot in (4, 17, -1):
        with pytest.raises(ValueError):
            kq.kq_assign_stack(fake, dist_slot=slot)
        with pytest.raises(ValueError):
            kq.kq_update_stack(fake, dist_slot=slot)
