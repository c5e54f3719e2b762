"""Plain, slow CPU oracle for Kernel Quantization (KQ): TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
(``paper_2003_05148_amd``) and never imports it.

What each function follows in the paper:

* ``forgy_select`` -- the initial codebook of the k-means (Sec. 3.1 does not say how it
  starts): k distinct kernels of the layer in a seeded random order (splitmix64 driving a
  partial Fisher-Yates shuffle).
* ``assign`` / ``update`` / ``distortion`` / ``fit`` -- kernel-level
  quantization, Sec. 3.1, Eq. (1): plain Lloyd k-means over the n = p q kernels
  of a layer, each a vector of omega^2 = 9 values (C loops in ``kq_oracle.c``).
* ``cbq_uniform`` / ``cbq_wkmeans`` -- kernel codebook quantization, Sec. 3.2:
  6-bit quantization of every scalar of a layer's codebook by k-means over those
  scalars, weighted by how often each codebook entry is used.
* ``size_search`` / ``search_codebook_size`` -- the codebook-size binary search of
  Algorithm 1 and Eq. (3), driven by the k-means distortion instead of the validation
  accuracy (a stated deviation: there is no trained network here).
* ``codebook_grad_step`` -- retraining of the kernel codebook, Sec. 3.1, Eq. (2):
  every entry moves against the mean gradient of the kernels mapped to it.
* ``quantize_scalars`` -- the same quantizer on the scalars of a fully-connected
  layer (end of Sec. 3.2), every weight 1.
* ``pack_bits`` -- the n * ceil(log2 k)-bit index stream counted by Eq. (4).
* ``reconstruct`` -- test-time recovery of the weight tensor from the codebook
  and the indices (end of Sec. 3.2).
* ``storage_bits`` / ``compression_ratio`` / ``bits_per_param`` -- Eq. (4),
  Eq. (6) and Eq. (7).

Readings of points the paper leaves open are stated at each function.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kq_oracle.c")
_LIB = os.path.join(_HERE, "libkq_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the C part of the oracle (plain loops, no FP contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared", "-fPIC",
                        _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I64, I = ctypes.c_int64, ctypes.c_int
        lib.kqo_assign.argtypes = [P, I64, I, P, I, P, P, P, P, P]
        lib.kqo_assign.restype = I
        lib.kqo_distortion.argtypes = [P, I64, I, P, P]
        lib.kqo_distortion.restype = ctypes.c_double
        lib.kqo_update.argtypes = [P, I64, I, P, I, P, P, P]
        lib.kqo_update.restype = I
        lib.kqo_fit.argtypes = [P, I64, I, I, P, I, P, P, P, P]
        lib.kqo_fit.restype = I
        lib.kqo_set_threads.argtypes = [I]
        lib.kqo_set_threads.restype = I
        _lib = lib
    return _lib


def set_threads(t: int) -> int:
    """Host threads of the assignment loop (its results do not depend on the count)."""
    return int(_load().kqo_set_threads(int(t)))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a, shape_last=None):
    a = np.ascontiguousarray(a, dtype=np.float32)
    if shape_last is not None and (a.ndim != 2 or a.shape[1] != shape_last):
        raise ValueError("expected [*, %d] array" % shape_last)
    return a


# ---- Sec. 3.1: the k-means initialisation --------------------------------------------

_MASK64 = (1 << 64) - 1


def splitmix64(seed: int):
    """The splitmix64 generator (Steele, Lea, Flood, OOPSLA 2014): the 64-bit state grows by
    0x9E3779B97F4A7C15 per draw and each draw returns the new state through the variant-13
    mixer.  Yields the draws as Python integers."""
    state = seed & _MASK64
    while True:
        state = (state + 0x9E3779B97F4A7C15) & _MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        yield z ^ (z >> 31)


def forgy_select(X, k: int, seed: int) -> np.ndarray:
    """Indices of k distinct kernels of X in a seeded random order (the reading taken for
    the k-means initialisation, which the paper leaves open).

    The order is a Fisher-Yates shuffle of 0..n-1 run only as far as needed: at step i a
    draw d of ``splitmix64(seed)`` picks j = i + (d mod (n - i)), positions i and j swap, and
    the value now at position i is the next candidate.  A candidate whose nine values equal,
    bit for bit, those of an already accepted kernel (-0 and +0 counted as equal) is
    skipped.  Raises ValueError when X holds fewer than k distinct kernels.
    """
    X = _f32(X)
    n = X.shape[0]
    bits = X.view(np.uint32).copy()
    bits[bits == 0x80000000] = 0          # -0 reads as +0
    perm = list(range(n))
    draws = splitmix64(seed)
    accepted, seen = [], set()
    for i in range(n):
        if len(accepted) == k:
            break
        j = i + next(draws) % (n - i)
        perm[i], perm[j] = perm[j], perm[i]
        cand = perm[i]
        key = bits[cand].tobytes()
        if key not in seen:
            seen.add(key)
            accepted.append(cand)
    if len(accepted) < k:
        raise ValueError(f"only {len(accepted)} distinct kernels, k={k}")
    return np.asarray(accepted, dtype=np.int64)


# ---- Sec. 3.1: kernel-level quantization (Lloyd k-means, Eq. 1) ----------------------

def assign(X, C):
    """Nearest codebook entry of every kernel.

    Returns a dict with
      idx   int32 [n]: decision on fp32 squared distances, ties to the lowest index
      d32   f32  [n]: that fp32 distance
      idx64 int32 [n]: decision on fp64 squared distances
      d1,d2 f64  [n]: best and second-best fp64 squared distances
    """
    X = _f32(X)
    C = _f32(C)
    n, dim = X.shape
    k = C.shape[0]
    out = dict(idx=np.empty(n, np.int32), d32=np.empty(n, np.float32), idx64=np.empty(n, np.int32),
               d1=np.empty(n, np.float64), d2=np.empty(n, np.float64))
    rc = _load().kqo_assign(_ptr(X), n, dim, _ptr(C), k, _ptr(out["idx"]), _ptr(out["d32"]),
                            _ptr(out["idx64"]), _ptr(out["d1"]), _ptr(out["d2"]))
    if rc:
        raise ValueError("kqo_assign failed")
    return out


def distortion(X, C, idx) -> float:
    """Eq. (1) objective of an assignment, fp64, summed in ascending kernel order."""
    X = _f32(X)
    C = _f32(C)
    idx = np.ascontiguousarray(idx, np.int32)
    return float(_load().kqo_distortion(_ptr(X), X.shape[0], X.shape[1], _ptr(C), _ptr(idx)))


def update(X, idx, C_old):
    """Each entry becomes the mean of its kernel set; an empty set keeps the old entry.

    Returns (C_new float32 [k, dim], counts int32 [k]).
    """
    X = _f32(X)
    C_old = _f32(C_old)
    idx = np.ascontiguousarray(idx, np.int32)
    k, dim = C_old.shape
    C_new = np.empty_like(C_old)
    counts = np.empty(k, np.int32)
    rc = _load().kqo_update(_ptr(X), X.shape[0], dim, _ptr(idx), k, _ptr(C_old), _ptr(C_new), _ptr(counts))
    if rc:
        raise ValueError("kqo_update failed (index out of range)")
    return C_new, counts


def fit(X, C_init, iters: int):
    """`iters` Lloyd rounds (assign, update) then a final assignment.

    Returns dict(C [k,dim] after `iters` updates, idx [n] final assignment,
    counts [k] of the final assignment, J [iters+1] distortion of each assignment).
    """
    X = _f32(X)
    C_init = _f32(C_init)
    n, dim = X.shape
    k = C_init.shape[0]
    C = np.empty_like(C_init)
    idx = np.empty(n, np.int32)
    counts = np.empty(k, np.int32)
    J = np.empty(iters + 1, np.float64)
    rc = _load().kqo_fit(_ptr(X), n, dim, k, _ptr(C_init), iters, _ptr(C), _ptr(idx), _ptr(counts), _ptr(J))
    if rc:
        raise ValueError("kqo_fit failed")
    return dict(C=C, idx=idx, counts=counts, J=J)


# ---- Alg. 1: binary search of the codebook size (on the k-means distortion) -------------

def size_search(D, n_init: int, r: float, max_iter: int):
    """The codebook-size search of Algorithm 1 with Eq. (3), on a distortion D(k) instead of
    the validation accuracy: accuracy A = -D, the unquantized layer's A_ori = 0, so
    A_target = A_base - (A_ori - A_base) r reads D_target = (1 + r) D(n_init).

    B_upper = n_init, B_lower = 0; each iteration tests N = floor((B_upper + B_lower) / 2)
    (stopping when N reaches a bound, the reading of the garbled loop condition); a size
    whose distortion is below the target becomes the new upper bound, any other the new
    lower bound.  Returns (k = B_upper, [(N, D(N)) per iteration], D(n_init)).
    """
    d0 = float(D(n_init))
    target = (1.0 + float(np.float32(r))) * d0
    upper, lower = n_init, 0
    trials = []
    for _ in range(max_iter):
        cur = (upper + lower) // 2
        if cur <= lower or cur >= upper:
            break
        d = float(D(cur))
        trials.append((cur, d))
        if d < target:
            upper = cur
        else:
            lower = cur
    return upper, trials, d0


def search_codebook_size(X, C_cand, n_init: int, r: float, max_iter: int, lloyd_iters: int):
    """``size_search`` with D(k) = the distortion of the final assignment of a Lloyd fit
    (``fit``) of k entries started from the first k rows of C_cand."""
    X = _f32(X)
    C_cand = _f32(C_cand)

    def D(k):
        return fit(X, C_cand[:k], lloyd_iters)["J"][-1]

    return size_search(D, n_init, r, max_iter)


# ---- Sec. 3.1, Eq. (2): retraining of the kernel codebook ------------------------------

def codebook_grad_step(G, idx, C, gamma):
    """One retraining step of the kernel codebook, Eq. (2):

        c_i <- c_i - gamma * (sum over the kernels m in S_i of dL/dm) / z_i.

    G [n, dim] holds dL/dm for every kernel, idx [n] the kernels' entries.  Readings:
    an entry with no kernels keeps its value (the mean over an empty set is undefined);
    indices outside [0, k) are ignored; the sum is fp64 over the members in ascending
    kernel order, the mean is that sum divided by z in fp64, and c - gamma * mean is
    evaluated in fp64 (c and the fp32 gamma widened exactly) and rounded once to fp32.

    Returns (C_new float32 [k, dim], counts int32 [k]).
    """
    G = _f32(G)
    C = _f32(C)
    idx = np.asarray(idx, np.int64)
    k, dim = C.shape
    ok = (idx >= 0) & (idx < k)
    S = np.zeros((k, dim), np.float64)
    np.add.at(S, idx[ok], G[ok].astype(np.float64))   # accumulates in ascending kernel order
    z = np.bincount(idx[ok], minlength=k)
    out = C.copy()
    has = z > 0
    mean = S[has] / z[has, None]
    out[has] = (C[has].astype(np.float64) - np.float64(np.float32(gamma)) * mean).astype(np.float32)
    return out, z.astype(np.int32)


# ---- Sec. 3.2: kernel codebook quantization -------------------------------------------

def _nearest_level(v32: np.ndarray, levels32: np.ndarray) -> np.ndarray:
    """Smallest q minimising |v - L_q|, both widened exactly to fp64."""
    diff = np.abs(v32.astype(np.float64)[:, None] - levels32.astype(np.float64)[None, :])
    return np.argmin(diff, axis=1).astype(np.uint8)


def uniform_levels(lo: float, hi: float, bits: int) -> np.ndarray:
    """2^bits levels evenly spaced on [lo, hi]: L_q = fp32(lo + q * delta),
    delta = (hi - lo) / (2^bits - 1); every operation rounded separately in fp64."""
    L = 1 << bits
    delta = (float(hi) - float(lo)) / (L - 1)
    return np.array([float(lo) + q * delta for q in range(L)], dtype=np.float64).astype(np.float32)


def cbq_uniform(C, bits: int = 6):
    """Uniform-grid quantization of all scalars of one codebook.

    Returns (codes uint8 [k*dim], levels float32 [2^bits], C_hat float32 [k, dim]).
    A constant codebook gives delta = 0 and every code 0.
    """
    C = _f32(C)
    v = C.reshape(-1)
    levels = uniform_levels(float(v.min()), float(v.max()), bits)
    codes = _nearest_level(v, levels)
    return codes, levels, levels[codes].reshape(C.shape)


def _exact_scaled(v32: np.ndarray) -> list:
    """v * 2^149 as exact Python integers (every fp32 value is a multiple of 2^-149)."""
    out = []
    for x in v32.astype(np.float64).tolist():
        num, den = x.as_integer_ratio()
        out.append(num * ((1 << 149) // den))
    return out


def cbq_wkmeans(C, weights, bits: int = 6, iters: int = 30):
    """Weighted 1-D k-means over all scalars of one codebook (Sec. 3.2).

    Scalar r = j*dim + d carries the weight of its entry j (its appearance
    count).  Initial levels: the uniform grid of ``cbq_uniform``.  Each round:
      W_q = sum of the weights of the scalars coded q (exact integer);
      N_q = sum of weight * value over those scalars, computed exactly and
            rounded once to fp64;
      L_q = fp32(N_q / W_q) (fp64 division) when W_q > 0, else L_q is kept;
      codes = nearest level (smallest q on ties).
    Stops after `iters` rounds or as soon as a round changes no code.

    Returns (codes uint8 [k*dim], levels float32 [2^bits], C_hat float32 [k, dim], rounds).
    """
    C = _f32(C)
    k, dim = C.shape
    w = np.repeat(np.asarray(weights, dtype=np.int64), dim)
    if w.shape[0] != k * dim:
        raise ValueError("weights must have one entry per codebook row")
    v = C.reshape(-1)
    codes, levels, _ = cbq_uniform(C, bits)
    vint = _exact_scaled(v)
    wl = w.tolist()
    L = 1 << bits
    rounds = 0
    for _ in range(iters):
        rounds += 1
        N = [0] * L
        W = [0] * L
        for r, q in enumerate(codes.tolist()):
            N[q] += wl[r] * vint[r]
            W[q] += wl[r]
        new_levels = levels.copy()
        for q in range(L):
            if W[q] > 0:
                Nq = N[q] / (1 << 149)          # exact integer ratio, correctly rounded to fp64
                new_levels[q] = np.float32(Nq / float(W[q]))
        new_codes = _nearest_level(v, new_levels)
        changed = bool(np.any(new_codes != codes))
        levels, codes = new_levels, new_codes
        if not changed:
            break
    return codes, levels, levels[codes].reshape(C.shape), rounds


def quantize_scalars(v, bits: int = 6, iters: int = 30):
    """Quantization of a fully-connected layer (end of Sec. 3.2), by the layer-by-layer
    k-means the codebooks are quantized with: the k-means of ``cbq_wkmeans`` on one flat
    set of scalars, every scalar carrying weight 1 (an FC weight is a parameter of its
    own, so there is no appearance count to weigh with).

    Returns (codes uint8 [m], levels float32 [2^bits], v_hat float32 [m], rounds).
    """
    v = np.ascontiguousarray(np.asarray(v, np.float32).reshape(-1, 1))
    codes, levels, v_hat, rounds = cbq_wkmeans(v, np.ones(v.shape[0], np.int64), bits, iters)
    return codes, levels, v_hat.reshape(-1), rounds


# ---- Eq. (4): the packed index stream, and test-time reconstruction ---------------------

def index_bits(k: int) -> int:
    """ceil(log2 k) bits per index (Eq. 4); 0 for k == 1."""
    return 0 if k <= 1 else int(math.ceil(math.log2(k)))


def pack_bits(values, bits: int) -> np.ndarray:
    """Concatenate `bits`-bit values LSB-first: bit t of value i is stream bit i*bits + t,
    stream bit s is bit (s % 8) of byte s // 8.  Length ceil(n * bits / 8) bytes."""
    v = np.asarray(values, dtype=np.uint64)
    if bits == 0 or v.size == 0:
        return np.zeros(0, np.uint8)
    bitmat = ((v[:, None] >> np.arange(bits, dtype=np.uint64)[None, :]) & np.uint64(1)).astype(np.uint8)
    return np.packbits(bitmat.reshape(-1), bitorder="little")


def unpack_bits(stream, count: int, bits: int) -> np.ndarray:
    s = np.unpackbits(np.asarray(stream, np.uint8), bitorder="little")[: count * bits]
    mat = s.reshape(count, bits).astype(np.int64)
    return (mat << np.arange(bits, dtype=np.int64)[None, :]).sum(axis=1).astype(np.int32)


def reconstruct(idx, C):
    """W_hat[i] = C[idx[i]] (the codebook may be the 6-bit dequantised one)."""
    return np.ascontiguousarray(np.asarray(C, np.float32)[np.asarray(idx, np.int64)])


# ---- Eq. (4), (6), (7): storage accounting ----------------------------------------------

def storage_bits(n: int, k: int, bc: int, dim: int = 9) -> int:
    """B = k * omega^2 * b_c + n * ceil(log2 k)   (Eq. 4)."""
    return k * dim * bc + n * index_bits(k)


def compression_ratio(n: int, k: int, bc: int, dim: int = 9, b_fp: int = 32) -> float:
    """C_KQ = n * omega^2 * b_FP / B   (Eq. 6)."""
    return n * dim * b_fp / storage_bits(n, k, bc, dim)


def bits_per_param(n: int, k: int, bc: int, dim: int = 9) -> float:
    """beta = B / (n * omega^2)   (Eq. 7)."""
    return storage_bits(n, k, bc, dim) / (n * dim)


def conventional_ratio(n: int, u: int, b1: int, dim: int = 9, b_fp: int = 32) -> float:
    """C_con = n omega^2 b_FP / (u b_1 + n omega^2 ceil(log2 u))   (Eq. 5)."""
    return n * dim * b_fp / (u * b1 + n * dim * index_bits(u))
