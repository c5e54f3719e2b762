"""MI355X (gfx950) hot path of Kernel Quantization (Yu et al., "Kernel Quantization for
Efficient Network Compression").

Thin Python binding of ``libkq.so`` (C ABI declared in ``include/kq.h``).  Every
function here only marshals arguments: it checks tensor devices, dtypes and shapes,
allocates outputs with torch when the caller gives none, and passes device pointers
and the current HIP stream to the library, where all the work runs.  There is no
fallback: without the built library, importing this package raises ImportError.

Entry points (same names as the C ABI):
  kq_assign, kq_update, kq_fit_layer, kq_assign_stack, kq_update_stack, kq_fit_stack,
  kq_fit_layer_yinyang (and the Yinyang class over kq_yinyang_init / kq_yinyang_assign),
  kq_codebook_grad_step, kq_codebook_grad_step_stack, kq_quantize_scalars, kq_search_codebook_size,
  kq_quantize_codebook, kq_quantize_codebook_stack, kq_pack_bits, kq_unpack_bits,
  kq_reconstruct, kq_reconstruct_packed.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkq.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(or python paper_2003_05148_amd/_build.py)")

_P = ctypes.c_void_p
_I32, _I64, _U32, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t


class KqLayer(ctypes.Structure):
    _fields_ = [("X", _P), ("n", _I64), ("k", _I32), ("C", _P), ("idx", _P), ("best_d", _P),
                ("counts", _P), ("distortion", _P)]


class KqCbqLayer(ctypes.Structure):
    _fields_ = [("C", _P), ("k", _I32), ("weights", _P), ("codes", _P), ("levels", _P), ("C_hat", _P)]


class KqPackJob(ctypes.Structure):
    _fields_ = [("values", _P), ("elem_bytes", _I32), ("bits", _I32), ("count", _I64), ("out", _P)]


class KqReconLayer(ctypes.Structure):
    _fields_ = [("idx", _P), ("packed", _P), ("bits", _I32), ("k", _I32), ("n", _I64), ("C", _P),
                ("W_hat", _P), ("W_ref", _P), ("sq_error", _P)]


class KqCompressLayer(ctypes.Structure):
    _fields_ = [("X", _P), ("n", _I64), ("k", _I32), ("C_init", _P), ("C", _P), ("idx", _P), ("counts", _P),
                ("distortion", _P), ("codes", _P), ("levels", _P), ("C_hat", _P), ("packed_idx", _P),
                ("packed_codes", _P), ("W_hat", _P), ("sq_error", _P)]


def _load():
    lib = ctypes.CDLL(LIB_PATH)
    sig = {
        "kq_status_string": ([_I32], ctypes.c_char_p),
        "kq_abi_version": ([], _I32),
        "kq_workspace_bytes": ([_I32, _I64, _I32, _I32], _SZ),
        "kq_stack_workspace_bytes": ([_P, _I32], _SZ),
        "kq_workspace_init": ([_P, _SZ, _P], _I32),
        "kq_assign": ([_P, _I64, _I32, _P, _I32, _P, _P, _P, _U32, _P, _SZ, _P], _I32),
        "kq_update": ([_P, _I64, _I32, _P, _I32, _P, _P, _P, _P, _U32, _P, _SZ, _P], _I32),
        "kq_fit_layer": ([_P, _I64, _I32, _I32, _P, _I32, _P, _P, _P, _P, _U32, _P, _SZ, _P], _I32),
        "kq_assign_stack": ([_P, _I32, _I32, _U32, _P, _SZ, _P], _I32),
        "kq_update_stack": ([_P, _I32, _I32, _U32, _P, _SZ, _P], _I32),
        "kq_fit_stack": ([_P, _I32, _I32, _U32, _P, _SZ, _P], _I32),
        "kq_quantize_codebook": ([_P, _I32, _I32, _P, _I32, _I32, _I32, _P, _P, _P, _P], _I32),
        "kq_quantize_codebook_stack": ([_P, _I32, _I32, _I32, _I32, _P], _I32),
        "kq_quantize_codebook_stack_workspace_bytes": ([_P, _I32, _I32], _SZ),
        "kq_quantize_codebook_stack_ws": ([_P, _I32, _I32, _I32, _I32, _P, _SZ, _P], _I32),
        "kq_pack_bits": ([_P, _I32, _I64, _I32, _P, _P], _I32),
        "kq_unpack_bits": ([_P, _I64, _I32, _P, _P], _I32),
        "kq_reconstruct": ([_P, _I64, _P, _I32, _I32, _P, _P], _I32),
        "kq_reconstruct_packed": ([_P, _I32, _I64, _P, _I32, _I32, _P, _P], _I32),
        "kq_sq_error": ([_P, _P, _I64, _P, _P, _SZ, _P], _I32),
        "kq_pack_bits_stack": ([_P, _I32, _P], _I32),
        "kq_reconstruct_stack_workspace_bytes": ([_P, _I32], _SZ),
        "kq_reconstruct_stack": ([_P, _I32, _P, _SZ, _P], _I32),
        "kq_codebook_grad_step": ([_P, _I64, _I32, _P, _I32, _P, ctypes.c_float, _P, _P, _P, _SZ, _P], _I32),
        "kq_codebook_grad_step_stack": ([_P, _I32, ctypes.c_float, _P, _SZ, _P], _I32),
        "kq_quantize_scalars_workspace_bytes": ([_I64, _I32], _SZ),
        "kq_quantize_scalars": ([_P, _I64, _I32, _I32, _P, _P, _P, _P, _U32, _P, _SZ, _P], _I32),
        "kq_search_workspace_bytes": ([_I64, _I32, _I32], _SZ),
        "kq_search_codebook_size": ([_P, _I64, _I32, _P, _I32, ctypes.c_float, _I32, _I32, _P, _P, _P, _P, _P, _P,
                                     _P, _SZ, _P], _I32),
        "kq_yinyang_workspace_bytes": ([_I64, _I32, _I32], _SZ),
        "kq_yinyang_init": ([_P, _I64, _I32, _P, _I32, _I32, _P, _P, _P, _P, _SZ, _P], _I32),
        "kq_yinyang_assign": ([_P, _I64, _I32, _P, _P, _I32, _I32, _P, _P, _P, _P, _P, _SZ, _P], _I32),
        "kq_fit_layer_yinyang": ([_P, _I64, _I32, _I32, _P, _I32, _I32, _P, _P, _P, _P, _P, _P, _SZ, _P], _I32),
        "kq_compress_workspace_bytes": ([_P, _I32, _I32], _SZ),
        "kq_compress_stack": ([_P, _I32, _I32, _I32, _I32, _I32, _U32, _P, _P, _SZ, _P], _I32),
        "kq_index_bits": ([_I32], _I32),
        "kq_accounting": ([_I64, _I32, _I32, _I32, _P, _P, _P], _I32),
        "kq_forgy_select": ([_P, _I64, _I32, _I32, ctypes.c_uint64, _P], _I32),
        "kq_fit_layer_noalloc_max_bytes": ([], _SZ),
        "kq_fit_layer_noalloc": ([_P, _I64, _I32, _I32, _P, _I32, _P, _P, _P, _P, _U32, _P], _I32),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


lib = _load()

# constants mirrored from include/kq.h
KQ_OK, KQ_ERR_ARG, KQ_ERR_UNSUPPORTED, KQ_ERR_WORKSPACE, KQ_ERR_RANGE, KQ_ERR_HIP = range(6)
KQ_DIM = 9
KQ_MAX_K = 65536
KQ_MAX_STACK = 16
KQ_CBQ_WKMEANS, KQ_CBQ_UNIFORM = 0, 1
KQ_OP_ASSIGN, KQ_OP_UPDATE, KQ_OP_FIT, KQ_OP_SQ_ERROR, KQ_OP_GRAD = 0, 1, 2, 3, 4
KQ_F_COUNTS_ONLY = 1
KQ_F_DISTORTION_FROM_ASSIGN = 2
KQ_F_FUSED_SUMS = 4
KQ_F_SUMS_FROM_ASSIGN = 8
KQ_F_EXACT_SEARCH = 16
KQ_F_THRESHOLDS = 32
KQ_F_VALIDATE = 64
KQ_F_REUSE_SHIFTS = 128
EXPORTED = ["kq_status_string", "kq_abi_version", "kq_workspace_bytes", "kq_stack_workspace_bytes",
            "kq_workspace_init", "kq_assign", "kq_update", "kq_fit_layer", "kq_assign_stack",
            "kq_update_stack", "kq_fit_stack", "kq_quantize_codebook", "kq_quantize_codebook_stack",
            "kq_quantize_codebook_stack_workspace_bytes", "kq_quantize_codebook_stack_ws",
            "kq_pack_bits", "kq_unpack_bits", "kq_reconstruct", "kq_reconstruct_packed", "kq_sq_error",
            "kq_pack_bits_stack", "kq_reconstruct_stack_workspace_bytes", "kq_reconstruct_stack",
            "kq_yinyang_workspace_bytes", "kq_yinyang_init", "kq_yinyang_assign", "kq_fit_layer_yinyang",
            "kq_codebook_grad_step", "kq_codebook_grad_step_stack", "kq_quantize_scalars_workspace_bytes",
            "kq_quantize_scalars", "kq_search_workspace_bytes", "kq_search_codebook_size",
            "kq_compress_workspace_bytes", "kq_compress_stack", "kq_index_bits", "kq_accounting",
            "kq_forgy_select", "kq_fit_layer_noalloc_max_bytes", "kq_fit_layer_noalloc"]
KQ_MAX_PACK_JOBS = 32


class KqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib.kq_status_string(status).decode()} (status {status})")


def _check(status: int, where: str):
    if status != KQ_OK:
        raise KqError(status, where)


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dev(t: torch.Tensor, dtype, name: str, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _ptr(t):
    return None if t is None else t.data_ptr()


def _kernels(X: torch.Tensor, name="X"):
    if X.dim() == 4:  # an OIHW 3x3 conv weight: kernel i = o * C_in + c
        if X.shape[2] * X.shape[3] != KQ_DIM:
            raise ValueError("only 3x3 kernels are supported")
        X = X.reshape(-1, KQ_DIM)
    _dev(X, torch.float32, name)
    if X.dim() != 2 or X.shape[1] != KQ_DIM:
        raise ValueError(f"{name} must be [n, 9] (or an OIHW 3x3 weight)")
    return X


class Workspace:
    """A device scratch buffer for the library (grown on demand).  Its contents need no
    initialisation; it can be reused by every call ordered on one stream."""

    def __init__(self, device=None):
        self.device = torch.device(device if device is not None else "cuda")
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=self.device)
        return self.buf


_workspaces: dict = {}


def _ws(device, nbytes):
    key = torch.device(device).index if torch.device(device).index is not None else torch.cuda.current_device()
    w = _workspaces.get(key)
    if w is None:
        w = _workspaces[key] = Workspace(torch.device("cuda", key))
    return w.get(nbytes)


# ---- Sec. 3.1, Eq. (1) ---------------------------------------------------------------

def kq_assign(X, C, idx=None, best_d=None, distortion=None, workspace=None):
    """Nearest codebook entry of every kernel (exact fp32 argmin, ties to the lowest
    index).  Returns (idx int32 [n], best_d float32 [n], distortion float64 [1])."""
    X = _kernels(X)
    C = _kernels(C, "C")
    n, k = X.shape[0], C.shape[0]
    dev = X.device
    idx = idx if idx is not None else torch.empty(n, dtype=torch.int32, device=dev)
    best_d = best_d if best_d is not None else torch.empty(n, dtype=torch.float32, device=dev)
    distortion = distortion if distortion is not None else torch.empty(1, dtype=torch.float64, device=dev)
    _dev(idx, torch.int32, "idx", (n,))
    _dev(best_d, torch.float32, "best_d", (n,))
    _dev(distortion, torch.float64, "distortion")
    nb = lib.kq_workspace_bytes(KQ_OP_ASSIGN, n, k, KQ_DIM)
    ws = workspace if workspace is not None else _ws(dev, nb)
    _check(lib.kq_assign(X.data_ptr(), n, KQ_DIM, C.data_ptr(), k, idx.data_ptr(), best_d.data_ptr(),
                         distortion.data_ptr(), 0, ws.data_ptr(), ws.numel(), _stream(dev)), "kq_assign")
    return idx, best_d, distortion


def kq_update(X, idx, C_old, C_new=None, counts=None, distortion=None, workspace=None, counts_only: bool = False,
              with_distortion: bool = True, validate: bool = False):
    """Mean of every kernel set (empty sets keep their entry) and the distortion of the
    assignment against C_old.  Returns (C_new, counts, distortion float64 [1]), the
    distortion None when `with_distortion` is False (the library is then passed NULL)."""
    X = _kernels(X)
    C_old = _kernels(C_old, "C_old")
    n, k = X.shape[0], C_old.shape[0]
    dev = X.device
    _dev(idx, torch.int32, "idx", (n,))
    C_new = C_new if C_new is not None else torch.empty_like(C_old)
    counts = counts if counts is not None else torch.empty(k, dtype=torch.int32, device=dev)
    _dev(C_new, torch.float32, "C_new", (k, KQ_DIM))
    _dev(counts, torch.int32, "counts", (k,))
    if with_distortion:
        distortion = distortion if distortion is not None else torch.empty(1, dtype=torch.float64, device=dev)
        _dev(distortion, torch.float64, "distortion")
    else:
        distortion = None
    nb = lib.kq_workspace_bytes(KQ_OP_UPDATE, n, k, KQ_DIM)
    ws = workspace if workspace is not None else _ws(dev, nb)
    _check(lib.kq_update(X.data_ptr(), n, KQ_DIM, idx.data_ptr(), k, C_old.data_ptr(), C_new.data_ptr(),
                         counts.data_ptr(), distortion.data_ptr() if distortion is not None else None,
                         (KQ_F_COUNTS_ONLY if counts_only else 0) | (KQ_F_VALIDATE if validate else 0), ws.data_ptr(),
                         ws.numel(), _stream(dev)),
           "kq_update")
    return C_new, counts, distortion


def _yy_groups_bytes(n: int, k: int, groups: int) -> int:
    nb = lib.kq_yinyang_workspace_bytes(n, k, groups)
    if nb == 0:
        raise ValueError(f"no Yinyang configuration for n={n}, k={k}, groups={groups} (needs 1 <= k <= n, "
                         f"groups <= min(64, k))")
    return nb


class Yinyang:
    """Yinyang assignment state of one layer (Sec. 4.1): the exact kq_assign result for
    every new codebook, skipping the entry groups that triangle-inequality bounds rule
    out.  The object owns its workspace (the bounds live there between calls) and a copy
    of the last codebook (the drift of the next call is measured from it)."""

    def __init__(self, X, C, groups: int = 0):
        self.X = _kernels(X)
        C = _kernels(C, "C")
        self.n, self.k, self.groups = self.X.shape[0], C.shape[0], int(groups)
        dev = self.X.device
        self.ws = torch.empty(_yy_groups_bytes(self.n, self.k, self.groups), dtype=torch.uint8, device=dev)
        self.idx = torch.empty(self.n, dtype=torch.int32, device=dev)
        self.best_d = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.distortion = torch.empty(1, dtype=torch.float64, device=dev)
        self.stats = torch.zeros(3, dtype=torch.int64, device=dev)
        self.C_prev = C.clone()
        _check(lib.kq_yinyang_init(self.X.data_ptr(), self.n, KQ_DIM, C.data_ptr(), self.k, self.groups,
                                   self.idx.data_ptr(), self.best_d.data_ptr(), self.distortion.data_ptr(),
                                   self.ws.data_ptr(), self.ws.numel(), _stream(dev)), "kq_yinyang_init")

    def assign(self, C):
        """Assignment against C (the codebook after the previous call's).  Returns
        (idx, best_d, distortion); `stats` then holds the kernels and (kernel, group) pairs
        that were scanned and the distances those scans evaluated."""
        C = _kernels(C, "C")
        if tuple(C.shape) != (self.k, KQ_DIM):
            raise ValueError(f"C must be [{self.k}, 9]")
        dev = self.X.device
        _check(lib.kq_yinyang_assign(self.X.data_ptr(), self.n, KQ_DIM, self.C_prev.data_ptr(), C.data_ptr(),
                                     self.k, self.groups, self.idx.data_ptr(), self.best_d.data_ptr(),
                                     self.distortion.data_ptr(), self.stats.data_ptr(), self.ws.data_ptr(),
                                     self.ws.numel(), _stream(dev)), "kq_yinyang_assign")
        self.C_prev.copy_(C)
        return self.idx, self.best_d, self.distortion


def kq_fit_layer_yinyang(X, C_init, iters: int, groups: int = 0, C=None, idx=None, counts=None, distortion=None,
                         stats=None, workspace=None):
    """kq_fit_layer with Yinyang assignments (Sec. 4.1); the same outputs bit for bit.
    Returns (C, idx, counts, distortion[iters+1], stats int64 [iters, 3]: kernels scanned,
    (kernel, group) pairs scanned, distances evaluated, per round)."""
    X = _kernels(X)
    C_init = _kernels(C_init, "C_init")
    n, k = X.shape[0], C_init.shape[0]
    dev = X.device
    C = C if C is not None else torch.empty_like(C_init)
    idx = idx if idx is not None else torch.empty(n, dtype=torch.int32, device=dev)
    counts = counts if counts is not None else torch.empty(k, dtype=torch.int32, device=dev)
    distortion = distortion if distortion is not None else torch.empty(iters + 1, dtype=torch.float64, device=dev)
    stats = stats if stats is not None else torch.zeros(max(iters, 1), 3, dtype=torch.int64, device=dev)
    _dev(C, torch.float32, "C", (k, KQ_DIM))
    _dev(idx, torch.int32, "idx", (n,))
    _dev(counts, torch.int32, "counts", (k,))
    _dev(distortion, torch.float64, "distortion", (iters + 1,))
    _dev(stats, torch.int64, "stats")
    nb = _yy_groups_bytes(n, k, groups)
    ws = workspace if workspace is not None else _ws(dev, nb)
    _check(lib.kq_fit_layer_yinyang(X.data_ptr(), n, KQ_DIM, k, C_init.data_ptr(), iters, groups, C.data_ptr(),
                                    idx.data_ptr(), counts.data_ptr(), distortion.data_ptr(), stats.data_ptr(),
                                    ws.data_ptr(), ws.numel(), _stream(dev)), "kq_fit_layer_yinyang")
    return C, idx, counts, distortion, stats


def kq_codebook_grad_step(G, idx, C_old, gamma: float, C_new=None, counts=None, workspace=None):
    """Eq. (2): every entry minus gamma times the mean gradient of its kernels (G [n, 9],
    or an OIHW 3x3 gradient tensor); empty entries keep their value.  C_new may be C_old
    (in place).  Returns (C_new, counts)."""
    G = _kernels(G, "G")
    C_old = _kernels(C_old, "C_old")
    n, k = G.shape[0], C_old.shape[0]
    dev = G.device
    _dev(idx, torch.int32, "idx", (n,))
    C_new = C_new if C_new is not None else torch.empty_like(C_old)
    counts = counts if counts is not None else torch.empty(k, dtype=torch.int32, device=dev)
    _dev(C_new, torch.float32, "C_new", (k, KQ_DIM))
    _dev(counts, torch.int32, "counts", (k,))
    nb = lib.kq_workspace_bytes(KQ_OP_GRAD, n, k, KQ_DIM)
    ws = workspace if workspace is not None else _ws(dev, nb)
    _check(lib.kq_codebook_grad_step(G.data_ptr(), n, KQ_DIM, idx.data_ptr(), k, C_old.data_ptr(), float(gamma),
                                     C_new.data_ptr(), counts.data_ptr(), ws.data_ptr(), ws.numel(),
                                     _stream(dev)), "kq_codebook_grad_step")
    return C_new, counts


def kq_codebook_grad_step_stack(stack, gamma: float):
    """Eq. (2) on every layer of a Stack built from the layers' gradient tensors (its X)
    and codebooks (its C, stepped in place; its counts receive the entry sizes)."""
    _check(lib.kq_codebook_grad_step_stack(ctypes.cast(stack.layers, _P), stack.n_layers, float(gamma),
                                           stack.ws.data_ptr(), stack.ws.numel(), _stream(stack.device)),
           "kq_codebook_grad_step_stack")


def kq_quantize_scalars(v, bits: int = 6, iters: int = 30, codes=None, levels=None, v_hat=None, rounds=None,
                        workspace=None, want_v_hat: bool = True, search: str = "auto"):
    """k-means quantization of every scalar of a (fully-connected) weight tensor with
    2^bits levels, the codebook quantizer's method with unit weights (end of Sec. 3.2).
    search: "auto", "exact" (KQ_F_EXACT_SEARCH) or "thresholds" (KQ_F_THRESHOLDS).
    Returns (codes uint8 [m], levels float32 [2^bits], v_hat float32 [m] or None,
    rounds int32 [1])."""
    flags = {"auto": 0, "exact": KQ_F_EXACT_SEARCH, "thresholds": KQ_F_THRESHOLDS}[search]
    if not isinstance(v, torch.Tensor) or not v.is_cuda or v.dtype != torch.float32 or not v.is_contiguous():
        raise TypeError("v must be a contiguous float32 CUDA (HIP) tensor")
    v = v.reshape(-1)
    m = v.numel()
    dev = v.device
    codes = codes if codes is not None else torch.empty(m, dtype=torch.uint8, device=dev)
    levels = levels if levels is not None else torch.empty(1 << bits, dtype=torch.float32, device=dev)
    if want_v_hat:
        v_hat = v_hat if v_hat is not None else torch.empty(m, dtype=torch.float32, device=dev)
        _dev(v_hat, torch.float32, "v_hat", (m,))
    else:
        v_hat = None
    rounds = rounds if rounds is not None else torch.zeros(1, dtype=torch.int32, device=dev)
    _dev(codes, torch.uint8, "codes", (m,))
    _dev(levels, torch.float32, "levels", (1 << bits,))
    _dev(rounds, torch.int32, "rounds", (1,))
    nb = lib.kq_quantize_scalars_workspace_bytes(m, bits)
    if nb == 0:
        raise ValueError(f"unsupported size {m} or bits {bits}")
    ws = workspace if workspace is not None else _ws(dev, nb)
    _check(lib.kq_quantize_scalars(v.data_ptr(), m, bits, iters, codes.data_ptr(), levels.data_ptr(), _ptr(v_hat),
                                   rounds.data_ptr(), flags, ws.data_ptr(), ws.numel(), _stream(dev)),
           "kq_quantize_scalars")
    return codes, levels, v_hat, rounds


def kq_search_codebook_size(X, C_cand, r: float, max_iter: int, lloyd_iters: int, workspace=None):
    """Algorithm 1's codebook-size binary search on the k-means distortion (a deviation
    from the paper's validation accuracy; see include/kq.h).  C_cand [n_init, 9] orders the
    candidate initial entries.  Returns (k, C [k, 9], idx [n], trials [(N, J(N))], J(n_init))."""
    X = _kernels(X)
    C_cand = _kernels(C_cand, "C_cand")
    n, n_init = X.shape[0], C_cand.shape[0]
    dev = X.device
    C = torch.empty_like(C_cand)
    idx = torch.empty(n, dtype=torch.int32, device=dev)
    nb = lib.kq_search_workspace_bytes(n, n_init, lloyd_iters)
    if nb == 0:
        raise ValueError("invalid search sizes")
    ws = workspace if workspace is not None else _ws(dev, nb)
    k_out = ctypes.c_int32(0)
    d0 = ctypes.c_double(0.0)
    tk = (ctypes.c_int32 * max(max_iter, 1))()
    td = (ctypes.c_double * max(max_iter, 1))()
    _check(lib.kq_search_codebook_size(X.data_ptr(), n, KQ_DIM, C_cand.data_ptr(), n_init, float(r), max_iter,
                                       lloyd_iters, C.data_ptr(), idx.data_ptr(), ctypes.byref(k_out),
                                       ctypes.cast(tk, _P), ctypes.cast(td, _P), ctypes.byref(d0), ws.data_ptr(),
                                       ws.numel(), _stream(dev)), "kq_search_codebook_size")
    trials = [(int(tk[i]), float(td[i])) for i in range(max_iter) if tk[i] > 0]
    return k_out.value, C[:k_out.value], idx, trials, d0.value


def kq_fit_layer(X, C_init, iters: int, C=None, idx=None, counts=None, distortion=None, workspace=None,
                 validate: bool = False):
    """`iters` Lloyd rounds then a final assignment.  Returns (C, idx, counts, distortion[iters+1])."""
    X = _kernels(X)
    C_init = _kernels(C_init, "C_init")
    n, k = X.shape[0], C_init.shape[0]
    dev = X.device
    C = C if C is not None else torch.empty_like(C_init)
    idx = idx if idx is not None else torch.empty(n, dtype=torch.int32, device=dev)
    counts = counts if counts is not None else torch.empty(k, dtype=torch.int32, device=dev)
    distortion = distortion if distortion is not None else torch.empty(iters + 1, dtype=torch.float64, device=dev)
    _dev(C, torch.float32, "C", (k, KQ_DIM))
    _dev(idx, torch.int32, "idx", (n,))
    _dev(counts, torch.int32, "counts", (k,))
    _dev(distortion, torch.float64, "distortion", (iters + 1,))
    nb = lib.kq_workspace_bytes(KQ_OP_FIT, n, k, KQ_DIM)
    ws = workspace if workspace is not None else _ws(dev, nb)
    _check(lib.kq_fit_layer(X.data_ptr(), n, KQ_DIM, k, C_init.data_ptr(), iters, C.data_ptr(), idx.data_ptr(),
                            counts.data_ptr(), distortion.data_ptr(), KQ_F_VALIDATE if validate else 0,
                            ws.data_ptr(), ws.numel(), _stream(dev)), "kq_fit_layer")
    return C, idx, counts, distortion


def kq_fit_layer_noalloc(X, C_init, iters: int, C, idx, counts, distortion, validate: bool = False):
    """kq_fit_layer with the library's static scratch instead of a workspace (the library
    allocates nothing; the outputs must be given).  Returns (C, idx, counts, distortion)."""
    X = _kernels(X)
    C_init = _kernels(C_init, "C_init")
    n, k = X.shape[0], C_init.shape[0]
    _dev(C, torch.float32, "C", (k, KQ_DIM))
    _dev(idx, torch.int32, "idx", (n,))
    _dev(counts, torch.int32, "counts", (k,))
    _dev(distortion, torch.float64, "distortion", (iters + 1,))
    _check(lib.kq_fit_layer_noalloc(X.data_ptr(), n, KQ_DIM, k, C_init.data_ptr(), iters, C.data_ptr(),
                                    idx.data_ptr(), counts.data_ptr(), distortion.data_ptr(),
                                    KQ_F_VALIDATE if validate else 0, _stream(X.device)), "kq_fit_layer_noalloc")
    return C, idx, counts, distortion


class Stack:
    """Device state of a conv stack for the stack calls: per layer X, C, idx, best_d,
    counts and a distortion history, plus the C descriptor array and a workspace."""

    def __init__(self, Xs, Cs, iters: int = 0, best_d: bool = False):
        self.X = [_kernels(x) for x in Xs]
        self.C = [_kernels(c, "C").clone() for c in Cs]
        dev = self.X[0].device
        self.idx = [torch.empty(x.shape[0], dtype=torch.int32, device=dev) for x in self.X]
        self.best_d = [torch.empty(x.shape[0], dtype=torch.float32, device=dev) for x in self.X] if best_d else None
        self.counts = [torch.empty(c.shape[0], dtype=torch.int32, device=dev) for c in self.C]
        self.distortion = [torch.zeros(iters + 1, dtype=torch.float64, device=dev) for _ in self.X]
        arr = (KqLayer * len(self.X))()
        for i, (x, c) in enumerate(zip(self.X, self.C)):
            arr[i] = KqLayer(x.data_ptr(), x.shape[0], c.shape[0], c.data_ptr(), self.idx[i].data_ptr(),
                             self.best_d[i].data_ptr() if best_d else None, self.counts[i].data_ptr(),
                             self.distortion[i].data_ptr())
        self.layers = arr
        self.n_layers = len(self.X)
        nb = lib.kq_stack_workspace_bytes(ctypes.cast(arr, _P), self.n_layers)
        if nb == 0:
            raise ValueError("invalid stack")
        self.ws = torch.zeros(nb, dtype=torch.uint8, device=dev)
        self.device = dev

    def set_codebooks(self, Cs):
        for c, src in zip(self.C, Cs):
            c.copy_(src)


def _check_slot(stack, dist_slot: int):
    if not 0 <= dist_slot < stack.distortion[0].numel():
        raise ValueError(f"dist_slot {dist_slot} outside the stack's distortion history "
                         f"(length {stack.distortion[0].numel()})")


def kq_assign_stack(stack: Stack, dist_slot: int = 0, distortion: bool = True, fused_sums: bool = False,
                    validate: bool = False, reuse_shifts: bool = False):
    """Assign every layer of the stack; the distortion (if asked) goes to slot dist_slot.
    fused_sums also accumulates the member sums of the new assignment (every k <= 256),
    for a following kq_update_stack(..., sums_from_assign=True); reuse_shifts takes the
    layers' fixed-point shifts from the preceding call on the stack instead of a new pass."""
    _check_slot(stack, dist_slot)
    flags = (KQ_F_FUSED_SUMS if fused_sums else 0) | (KQ_F_VALIDATE if validate else 0)
    flags |= KQ_F_REUSE_SHIFTS if reuse_shifts else 0
    if not distortion:
        saved = [(l.distortion) for l in stack.layers]
        for l in stack.layers:
            l.distortion = None
        try:
            _check(lib.kq_assign_stack(ctypes.cast(stack.layers, _P), stack.n_layers, dist_slot, flags,
                                       stack.ws.data_ptr(), stack.ws.numel(), _stream(stack.device)),
                   "kq_assign_stack")
        finally:
            for l, d in zip(stack.layers, saved):
                l.distortion = d
        return
    _check(lib.kq_assign_stack(ctypes.cast(stack.layers, _P), stack.n_layers, dist_slot, flags, stack.ws.data_ptr(),
                               stack.ws.numel(), _stream(stack.device)), "kq_assign_stack")


def kq_update_stack(stack: Stack, dist_slot: int = 0, counts_only: bool = False, distortion_from_assign=False,
                    sums_from_assign: bool = False, validate: bool = False, reuse_shifts: bool = False):
    """Update every codebook of the stack.  The distortion of the assignment goes to slot
    dist_slot; with distortion_from_assign it is the value the preceding kq_assign_stack
    left in the workspace (no second pass over the old codebook).  With sums_from_assign
    the update is finished from the member sums of the preceding fused assignment (the
    kernels are not read again; the distortion then also comes from the assignment)."""
    flags = (KQ_F_COUNTS_ONLY if counts_only else 0) | (KQ_F_DISTORTION_FROM_ASSIGN if distortion_from_assign else 0)
    flags |= (KQ_F_SUMS_FROM_ASSIGN if sums_from_assign else 0) | (KQ_F_VALIDATE if validate else 0)
    flags |= KQ_F_REUSE_SHIFTS if reuse_shifts else 0
    _check_slot(stack, dist_slot)
    _check(lib.kq_update_stack(ctypes.cast(stack.layers, _P), stack.n_layers, dist_slot, flags,
                               stack.ws.data_ptr(), stack.ws.numel(), _stream(stack.device)), "kq_update_stack")


def kq_fit_stack(stack: Stack, iters: int, validate: bool = False):
    if stack.distortion[0].numel() < iters + 1:
        raise ValueError("the stack's distortion history is shorter than iters + 1")
    _check(lib.kq_fit_stack(ctypes.cast(stack.layers, _P), stack.n_layers, iters, KQ_F_VALIDATE if validate else 0,
                            stack.ws.data_ptr(), stack.ws.numel(), _stream(stack.device)), "kq_fit_stack")


# ---- Sec. 3.2 --------------------------------------------------------------------------

def kq_quantize_codebook(C, weights=None, bits: int = 6, mode: int = KQ_CBQ_WKMEANS, iters: int = 30,
                         codes=None, levels=None, C_hat=None):
    """6-bit (by default) codebook quantization.  Returns (codes uint8 [k*9], levels [2^bits], C_hat)."""
    C = _kernels(C, "C")
    k = C.shape[0]
    dev = C.device
    if weights is not None:
        _dev(weights, torch.int32, "weights", (k,))
    codes = codes if codes is not None else torch.empty(k * KQ_DIM, dtype=torch.uint8, device=dev)
    levels = levels if levels is not None else torch.empty(1 << bits, dtype=torch.float32, device=dev)
    C_hat = C_hat if C_hat is not None else torch.empty_like(C)
    _check(lib.kq_quantize_codebook(C.data_ptr(), k, KQ_DIM, _ptr(weights), bits, mode, iters, codes.data_ptr(),
                                    levels.data_ptr(), C_hat.data_ptr(), _stream(dev)), "kq_quantize_codebook")
    return codes, levels, C_hat


def kq_quantize_codebook_stack(Cs, weights, bits: int = 6, mode: int = KQ_CBQ_WKMEANS, iters: int = 30, out=None,
                               wide: bool = True, workspace=None):
    """kq_quantize_codebook for a list of codebooks.  wide (kq_quantize_codebook_stack_ws):
    codebooks of at least 16384 scalars run on the whole GPU, the others in one launch;
    otherwise (kq_quantize_codebook_stack) one workgroup per codebook.  The results are the
    same.  Returns a list of (codes, levels, C_hat)."""
    Cs = [_kernels(c, "C") for c in Cs]
    dev = Cs[0].device
    if out is None:
        out = [(torch.empty(c.shape[0] * KQ_DIM, dtype=torch.uint8, device=dev),
                torch.empty(1 << bits, dtype=torch.float32, device=dev), torch.empty_like(c)) for c in Cs]
    arr = (KqCbqLayer * len(Cs))()
    for i, c in enumerate(Cs):
        w = weights[i] if weights is not None else None
        if w is not None:
            _dev(w, torch.int32, "weights", (c.shape[0],))
        arr[i] = KqCbqLayer(c.data_ptr(), c.shape[0], _ptr(w), out[i][0].data_ptr(), out[i][1].data_ptr(),
                            out[i][2].data_ptr())
    if not wide:
        _check(lib.kq_quantize_codebook_stack(ctypes.cast(arr, _P), len(Cs), bits, mode, iters, _stream(dev)),
               "kq_quantize_codebook_stack")
        return out
    nb = lib.kq_quantize_codebook_stack_workspace_bytes(ctypes.cast(arr, _P), len(Cs), bits)
    ws = workspace if workspace is not None else (_ws(dev, nb) if nb else None)
    _check(lib.kq_quantize_codebook_stack_ws(ctypes.cast(arr, _P), len(Cs), bits, mode, iters, _ptr(ws),
                                             0 if ws is None else ws.numel(), _stream(dev)),
           "kq_quantize_codebook_stack_ws")
    return out


# ---- Eq. (4) and test-time reconstruction -------------------------------------------------

def index_bits(k: int) -> int:
    """ceil(log2 k), the Eq. (4) index width (kq_index_bits)."""
    b = lib.kq_index_bits(int(k))
    if b < 0:
        raise ValueError("k must be >= 1")
    return b


def kq_accounting(n: int, k: int, bc: int, dim: int = KQ_DIM):
    """Eq. (4), (6), (7) for a layer of n kernels and a k-entry codebook stored at bc bits
    per value: (storage bits B, compression ratio C_KQ, bits per parameter beta)."""
    B, r, beta = ctypes.c_int64(0), ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(lib.kq_accounting(int(n), int(k), int(dim), int(bc), ctypes.byref(B), ctypes.byref(r),
                             ctypes.byref(beta)), "kq_accounting")
    return B.value, r.value, beta.value


def kq_forgy_select(X, k: int, seed: int):
    """k distinct kernels of X (host: a numpy array or CPU tensor [n, 9] float32) in the
    seeded splitmix64 partial Fisher-Yates order.  Returns their row indices (int64 numpy)."""
    import numpy as np
    if isinstance(X, torch.Tensor):
        if X.is_cuda:
            raise TypeError("kq_forgy_select takes host kernels")
        X = X.numpy()
    X = np.ascontiguousarray(X, dtype=np.float32).reshape(-1, KQ_DIM)
    sel = np.empty(max(int(k), 1), np.int64)
    _check(lib.kq_forgy_select(X.ctypes.data_as(_P), X.shape[0], KQ_DIM, int(k), int(seed) & ((1 << 64) - 1),
                               sel.ctypes.data_as(_P)), "kq_forgy_select")
    return sel[:k]


def kq_pack_bits(values, bits: int, out=None):
    """LSB-first stream of `bits`-bit fields.  values: int32, uint8 or int16 tensor."""
    eb = {torch.int32: 4, torch.uint8: 1, torch.int16: 2}.get(values.dtype)
    if eb is None:
        raise TypeError("values must be int32, int16 or uint8")
    _dev(values, values.dtype, "values")
    count = values.numel()
    nbytes = (count * bits + 7) // 8
    out = out if out is not None else torch.empty(max(nbytes, 1), dtype=torch.uint8, device=values.device)
    _check(lib.kq_pack_bits(values.data_ptr(), eb, count, bits, out.data_ptr(), _stream(values.device)),
           "kq_pack_bits")
    return out[:nbytes]


def kq_unpack_bits(stream, count: int, bits: int, out=None):
    _dev(stream, torch.uint8, "stream")
    out = out if out is not None else torch.empty(count, dtype=torch.int32, device=stream.device)
    _check(lib.kq_unpack_bits(stream.data_ptr(), count, bits, out.data_ptr(), _stream(stream.device)),
           "kq_unpack_bits")
    return out


def kq_reconstruct(idx, C, W_hat=None):
    """W_hat[i] = C[idx[i]]  ([n, 9] float32)."""
    C = _kernels(C, "C")
    _dev(idx, torch.int32, "idx")
    n = idx.numel()
    W_hat = W_hat if W_hat is not None else torch.empty(n, KQ_DIM, dtype=torch.float32, device=idx.device)
    _check(lib.kq_reconstruct(idx.data_ptr(), n, C.data_ptr(), C.shape[0], KQ_DIM, W_hat.data_ptr(),
                              _stream(idx.device)), "kq_reconstruct")
    return W_hat


def kq_reconstruct_packed(packed, bits: int, n: int, C, W_hat=None):
    C = _kernels(C, "C")
    _dev(packed, torch.uint8, "packed")
    W_hat = W_hat if W_hat is not None else torch.empty(n, KQ_DIM, dtype=torch.float32, device=packed.device)
    _check(lib.kq_reconstruct_packed(packed.data_ptr(), bits, n, C.data_ptr(), C.shape[0], KQ_DIM,
                                     W_hat.data_ptr(), _stream(packed.device)), "kq_reconstruct_packed")
    return W_hat


def kq_sq_error(A, B, out=None, workspace=None):
    """sum (A - B)^2 over all elements, fp64, fixed order.  Returns a float64 [1] tensor."""
    _dev(A, torch.float32, "A")
    _dev(B, torch.float32, "B", tuple(A.shape))
    out = out if out is not None else torch.empty(1, dtype=torch.float64, device=A.device)
    nb = lib.kq_workspace_bytes(KQ_OP_SQ_ERROR, A.numel(), 1, 1)
    ws = workspace if workspace is not None else _ws(A.device, nb)
    _check(lib.kq_sq_error(A.data_ptr(), B.data_ptr(), A.numel(), out.data_ptr(), ws.data_ptr(), ws.numel(),
                           _stream(A.device)), "kq_sq_error")
    return out


# ---- stack forms of pack and reconstruct ---------------------------------------------------

_EB = {torch.int32: 4, torch.uint8: 1, torch.int16: 2}


def kq_pack_bits_stack(jobs):
    """Pack several streams with one launch.  jobs: list of (values, bits, out) with out
    a uint8 tensor of at least ceil(count * bits / 8) bytes, or None to allocate one.
    Returns the list of streams (each trimmed to its exact length)."""
    if not 1 <= len(jobs) <= KQ_MAX_PACK_JOBS:
        raise ValueError(f"1..{KQ_MAX_PACK_JOBS} jobs per call")
    arr = (KqPackJob * len(jobs))()
    outs, dev = [], None
    for q, (values, bits, out) in enumerate(jobs):
        eb = _EB.get(values.dtype)
        if eb is None:
            raise TypeError("values must be int32, int16 or uint8")
        _dev(values, values.dtype, "values")
        dev = values.device
        nbytes = (values.numel() * bits + 7) // 8
        if out is None:
            out = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=values.device)
        else:
            _dev(out, torch.uint8, "out")
            if out.numel() < nbytes:
                raise ValueError("out is too small")
        arr[q] = KqPackJob(values.data_ptr(), eb, bits, values.numel(), out.data_ptr())
        outs.append(out[:nbytes])
    _check(lib.kq_pack_bits_stack(ctypes.cast(arr, _P), len(jobs), _stream(dev)), "kq_pack_bits_stack")
    return outs


def _recon_array(layers):
    arr = (KqReconLayer * len(layers))()
    outs, dev = [], None
    for q, L in enumerate(layers):
        C = _kernels(L["C"], "C")
        dev = C.device
        n = int(L["n"])
        idx, packed = L.get("idx"), L.get("packed")
        if idx is not None:
            _dev(idx, torch.int32, "idx", (n,))
        else:
            _dev(packed, torch.uint8, "packed")
        W_hat = L.get("W_hat")
        W_hat = W_hat if W_hat is not None else torch.empty(n, KQ_DIM, dtype=torch.float32, device=dev)
        _dev(W_hat, torch.float32, "W_hat", (n, KQ_DIM))
        W_ref, sq = L.get("W_ref"), L.get("sq_error")
        if W_ref is not None:
            W_ref = _kernels(W_ref, "W_ref")
        if sq is not None:
            _dev(sq, torch.float64, "sq_error")
        arr[q] = KqReconLayer(_ptr(idx), _ptr(packed) if idx is None else None, int(L.get("bits", 0)),
                              C.shape[0], n, C.data_ptr(), W_hat.data_ptr(), _ptr(W_ref), _ptr(sq))
        outs.append(W_hat)
    return arr, outs, dev


def recon_workspace_bytes(layers) -> int:
    """Workspace bytes kq_reconstruct_stack needs for these layers (see there)."""
    arr, _, _ = _recon_array(layers)
    return lib.kq_reconstruct_stack_workspace_bytes(ctypes.cast(arr, _P), len(layers))


def kq_reconstruct_stack(layers, workspace=None):
    """Reconstruct several layers with one launch.  layers: list of dicts with keys
    C ([k, 9] codebook), n, and either idx (int32 [n]) or packed + bits; optional W_hat
    (output [n, 9]), W_ref (original kernels [n, 9]) and sq_error (float64 [1] output,
    needs W_ref).  Returns the list of W_hat tensors."""
    if not 1 <= len(layers) <= KQ_MAX_STACK:
        raise ValueError(f"1..{KQ_MAX_STACK} layers per call")
    arr, outs, dev = _recon_array(layers)
    nb = lib.kq_reconstruct_stack_workspace_bytes(ctypes.cast(arr, _P), len(layers))
    ws = workspace if workspace is not None else (_ws(dev, nb) if nb else None)
    _check(lib.kq_reconstruct_stack(ctypes.cast(arr, _P), len(layers), _ptr(ws), 0 if ws is None else ws.numel(),
                                    _stream(dev)), "kq_reconstruct_stack")
    return outs


# ---- the whole compression pass in one call ------------------------------------------------

class Compression:
    """Device buffers of kq_compress_stack for the layers of a network: per layer X, C_init,
    the fitted C, idx, counts, the distortion history, the quantized codebook (codes, levels,
    C_hat), the packed index and code streams, W_hat and its squared error; plus the layer
    descriptor array and the workspace.  ``run()`` makes the one library call."""

    def __init__(self, Xs, C_inits, iters: int, bits: int = 6, mode: int = KQ_CBQ_WKMEANS, cbq_iters: int = 30,
                 pack: bool = True, reconstruct: bool = True, sq_error: bool = True):
        self.X = [_kernels(x) for x in Xs]
        self.C_init = [_kernels(c, "C_init") for c in C_inits]
        dev = self.X[0].device
        self.device, self.iters, self.bits, self.mode, self.cbq_iters = dev, int(iters), int(bits), int(mode), int(cbq_iters)
        ks = [c.shape[0] for c in self.C_init]
        ns = [x.shape[0] for x in self.X]
        self.C = [torch.empty(k, KQ_DIM, device=dev) for k in ks]
        self.idx = [torch.empty(n, dtype=torch.int32, device=dev) for n in ns]
        self.counts = [torch.empty(k, dtype=torch.int32, device=dev) for k in ks]
        self.distortion = [torch.zeros(self.iters + 1, dtype=torch.float64, device=dev) for _ in ns]
        self.codes = [torch.empty(k * KQ_DIM, dtype=torch.uint8, device=dev) for k in ks]
        self.levels = [torch.empty(1 << self.bits, device=dev) for _ in ks]
        self.C_hat = [torch.empty(k, KQ_DIM, device=dev) for k in ks]
        self.index_bits = [index_bits(k) for k in ks]
        # stream buffers rounded up to whole dwords (the packers store 32-bit words)
        self.packed_idx = [torch.zeros(((n * b + 7) // 8 + 3) // 4 * 4 + 4, dtype=torch.uint8, device=dev)
                           for n, b in zip(ns, self.index_bits)] if pack else None
        self.packed_codes = [torch.zeros(((k * KQ_DIM * self.bits + 7) // 8 + 3) // 4 * 4 + 4, dtype=torch.uint8,
                                         device=dev) for k in ks] if pack else None
        self.W_hat = [torch.empty(n, KQ_DIM, device=dev) for n in ns] if reconstruct else None
        self.sq_error = torch.zeros(len(ns), dtype=torch.float64, device=dev) if (reconstruct and sq_error) else None
        arr = (KqCompressLayer * len(ns))()
        for i in range(len(ns)):
            if self.C_init[i].shape != (ks[i], KQ_DIM):
                raise ValueError("C_init must be [k, 9]")
            arr[i] = KqCompressLayer(
                self.X[i].data_ptr(), ns[i], ks[i], self.C_init[i].data_ptr(), self.C[i].data_ptr(),
                self.idx[i].data_ptr(), self.counts[i].data_ptr(), self.distortion[i].data_ptr(),
                self.codes[i].data_ptr(), self.levels[i].data_ptr(), self.C_hat[i].data_ptr(),
                self.packed_idx[i].data_ptr() if pack else None, self.packed_codes[i].data_ptr() if pack else None,
                self.W_hat[i].data_ptr() if reconstruct else None,
                self.sq_error[i:i + 1].data_ptr() if self.sq_error is not None else None)
        self.layers = arr
        self.n_layers = len(ns)
        nb = lib.kq_compress_workspace_bytes(ctypes.cast(arr, _P), self.n_layers, self.bits)
        if nb == 0:
            raise ValueError("invalid compression layers")
        self.ws = torch.zeros(nb, dtype=torch.uint8, device=dev)

    def packed_index_stream(self, i: int):
        return self.packed_idx[i][:(self.X[i].shape[0] * self.index_bits[i] + 7) // 8]

    def packed_code_stream(self, i: int):
        return self.packed_codes[i][:(self.C[i].shape[0] * KQ_DIM * self.bits + 7) // 8]

    def run(self, validate: bool = False, round_events=None):
        kq_compress_stack(self, validate, round_events)


def kq_compress_stack(comp: Compression, validate: bool = False, round_events=None):
    """The compression pass of every layer of ``comp`` in one library call: Lloyd fit,
    codebook quantization, index/code packing, reconstruction and its error.
    round_events: None, or {round t: (start, end) torch.cuda.Event with timing} -- the
    library records them around the assignment launch of those Lloyd rounds."""
    ev = None
    if round_events:
        ev = (_P * (2 * (comp.iters + 1)))()
        for t, (a, b) in round_events.items():
            if not 0 <= t <= comp.iters:
                raise ValueError(f"round {t} outside 0..{comp.iters}")
            if not a.cuda_event or not b.cuda_event:
                raise ValueError("record each event once through torch first (torch creates them lazily)")
            ev[2 * t], ev[2 * t + 1] = a.cuda_event, b.cuda_event
    _check(lib.kq_compress_stack(ctypes.cast(comp.layers, _P), comp.n_layers, comp.iters, comp.mode, comp.bits,
                                 comp.cbq_iters, KQ_F_VALIDATE if validate else 0, ev, comp.ws.data_ptr(),
                                 comp.ws.numel(), _stream(comp.device)), "kq_compress_stack")
