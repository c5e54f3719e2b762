// C ABI of libkq: argument checks, workspace layout and launches.
//
// Every entry point checks its arguments before it touches HIP, so argument errors
// come back without a GPU (and without initialising the HIP runtime).  No entry point
// allocates memory; device scratch comes from the caller's workspace.
#include <string.h>

#include "kq_internal.h"

using namespace kq;

namespace {

constexpr int32_t kAbiVersion = 1;

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }
bool valid_n(int64_t n) { return n >= 1 && n < (int64_t(1) << 31); }
bool valid_k(int32_t k) { return k >= 1 && k <= KQ_MAX_K; }

kq_status hip_status(hipError_t e) { return e == hipSuccess ? KQ_OK : KQ_ERR_HIP; }

size_t stack_ws_bytes(const kq_layer* layers, int32_t n_layers) {
    size_t b = 0;
    for (int32_t l = 0; l < n_layers; ++l) b += layer_ws_bytes(layers[l].n, layers[l].k);
    return b;
}

kq_status check_ws(void* ws, size_t ws_bytes, size_t need) {
    if (ws == nullptr || !aligned(ws, 256) || ws_bytes < need) return KQ_ERR_WORKSPACE;
    return KQ_OK;
}

// fill the device descriptor of one layer; `base` is its workspace region
void fill_layer(DevLayer& d, const float* X, int64_t n, int32_t k, float* C, const float* C_old, int32_t* idx,
                float* best_d, int32_t* counts, double* dist, unsigned char* base) {
    memset(&d, 0, sizeof(d));
    d.X = X;
    d.C = C;
    d.C_old = C_old;
    d.idx = idx;
    d.best_d = best_d;
    d.counts = counts;
    d.dist = dist;
    d.n = (int)n;
    d.k = k;
    d.shift = fixed_shift(n);
    d.ctr = (unsigned*)base;
    d.part = (double*)(base + 256);
    d.acc = (unsigned long long*)(base + 256 + align256(sizeof(double) * (size_t)assign_blocks(n)));
}

// the layers [l0, l1) of a stack as launch parameters (assign or update geometry)
void stack_params(StackParams& p, const kq_layer* layers, int32_t l0, int32_t l1, unsigned char* ws, bool for_update,
                  int32_t dist_slot, bool counts_only) {
    memset(&p, 0, sizeof(p));
    size_t off = 0;
    for (int32_t l = 0; l < l0; ++l) off += layer_ws_bytes(layers[l].n, layers[l].k);
    int blk = 0;
    for (int32_t l = l0; l < l1; ++l) {
        const kq_layer& s = layers[l];
        DevLayer& d = p.L[l - l0];
        fill_layer(d, s.X, s.n, s.k, s.C, s.C, s.idx, for_update ? nullptr : s.best_d, s.counts,
                   (!for_update && s.distortion) ? s.distortion + dist_slot : nullptr, ws + off);
        d.counts_only = counts_only ? 1 : 0;
        d.blk_begin = blk;
        d.nblk = for_update ? update_blocks(s.n) : assign_blocks(s.n);
        blk += d.nblk;
        off += layer_ws_bytes(s.n, s.k);
    }
    p.nlayers = l1 - l0;
    p.total_blocks = blk;
}

kq_status check_layers(const kq_layer* layers, int32_t n_layers, bool fit) {
    if (layers == nullptr || n_layers < 1) return KQ_ERR_ARG;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_layer& s = layers[l];
        if (!valid_n(s.n)) return KQ_ERR_ARG;
        if (s.k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
        if (!valid_k(s.k) || (fit && s.k > s.n)) return KQ_ERR_ARG;
        if (!s.X || !s.C || !s.idx || !aligned(s.X, 4) || !aligned(s.C, 4) || !aligned(s.idx, 4)) return KQ_ERR_ARG;
        if ((s.best_d && !aligned(s.best_d, 4)) || (s.counts && !aligned(s.counts, 4)) ||
            (s.distortion && !aligned(s.distortion, 8)))
            return KQ_ERR_ARG;
    }
    return KQ_OK;
}

kq_status run_fit(const kq_layer* layers, int32_t n_layers, int32_t iters, unsigned char* ws, hipStream_t s) {
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        StackParams pa, pu;
        for (int32_t t = 0; t <= iters; ++t) {
            stack_params(pa, layers, l0, l1, ws, false, t, false);
            hipError_t e = launch_assign(pa, s);
            if (e != hipSuccess) return KQ_ERR_HIP;
            const bool last = (t == iters);
            stack_params(pu, layers, l0, l1, ws, true, 0, last);
            if (last) {
                bool any_counts = false;
                for (int32_t l = l0; l < l1; ++l) any_counts |= layers[l].counts != nullptr;
                if (!any_counts) break;
            }
            e = launch_update(pu, s);
            if (e != hipSuccess) return KQ_ERR_HIP;
        }
    }
    return KQ_OK;
}

}  // namespace

extern "C" {

const char* kq_status_string(kq_status st) {
    switch (st) {
        case KQ_OK: return "ok";
        case KQ_ERR_ARG: return "invalid argument";
        case KQ_ERR_UNSUPPORTED: return "unsupported size or parameter";
        case KQ_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case KQ_ERR_RANGE: return "input outside the supported range";
        case KQ_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

int32_t kq_abi_version(void) { return kAbiVersion; }

size_t kq_workspace_bytes(int32_t op, int64_t n, int32_t k) {
    if (op == KQ_OP_SQ_ERROR) {
        if (n < 1 || n >= (int64_t(1) << 40)) return 0;
        return 256 + align256(sizeof(double) * (size_t)sq_error_blocks(n));
    }
    if (!valid_n(n) || !valid_k(k)) return 0;
    if (op != KQ_OP_ASSIGN && op != KQ_OP_UPDATE && op != KQ_OP_FIT) return 0;
    return layer_ws_bytes(n, k);
}

size_t kq_stack_workspace_bytes(const kq_layer* layers, int32_t n_layers) {
    if (check_layers(layers, n_layers, false) != KQ_OK) return 0;
    return stack_ws_bytes(layers, n_layers);
}

kq_status kq_workspace_init(void* ws, size_t bytes, void* stream) {
    if (ws == nullptr || !aligned(ws, 256)) return KQ_ERR_WORKSPACE;
    if (bytes == 0) return KQ_OK;
    return hip_status(launch_fill_zero(ws, bytes, (hipStream_t)stream));
}

kq_status kq_assign(const float* X, int64_t n, int32_t dim, const float* C, int32_t k, int32_t* idx, float* best_d,
                    double* distortion, uint32_t flags, void* ws, size_t ws_bytes, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || flags != 0) return KQ_ERR_ARG;
    if (!X || !C || !idx || !aligned(X, 4) || !aligned(C, 4) || !aligned(idx, 4)) return KQ_ERR_ARG;
    if ((best_d && !aligned(best_d, 4)) || (distortion && !aligned(distortion, 8))) return KQ_ERR_ARG;
    if (distortion) {
        const kq_status w = check_ws(ws, ws_bytes, layer_ws_bytes(n, k));
        if (w != KQ_OK) return w;
    }
    kq_layer l = {X, n, k, const_cast<float*>(C), idx, best_d, nullptr, distortion};
    StackParams p;
    unsigned char scratch_base[256];  // never dereferenced: without a distortion nothing touches the workspace
    stack_params(p, &l, 0, 1, ws ? (unsigned char*)ws : scratch_base, false, 0, false);
    return hip_status(launch_assign(p, (hipStream_t)stream));
}

kq_status kq_update(const float* X, int64_t n, int32_t dim, const int32_t* idx, int32_t k, const float* C_old,
                    float* C_new, int32_t* counts, uint32_t flags, void* ws, size_t ws_bytes, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || (flags & ~KQ_F_COUNTS_ONLY) != 0) return KQ_ERR_ARG;
    if (!X || !idx || !C_old || !C_new || !aligned(X, 4) || !aligned(idx, 4) || !aligned(C_old, 4) ||
        !aligned(C_new, 4))
        return KQ_ERR_ARG;
    if (counts && !aligned(counts, 4)) return KQ_ERR_ARG;
    const kq_status w = check_ws(ws, ws_bytes, layer_ws_bytes(n, k));
    if (w != KQ_OK) return w;
    StackParams p;
    memset(&p, 0, sizeof(p));
    fill_layer(p.L[0], X, n, k, C_new, C_old, const_cast<int32_t*>(idx), nullptr, counts, nullptr, (unsigned char*)ws);
    p.L[0].nblk = update_blocks(n);
    p.L[0].counts_only = (flags & KQ_F_COUNTS_ONLY) ? 1 : 0;
    p.nlayers = 1;
    p.total_blocks = p.L[0].nblk;
    return hip_status(launch_update(p, (hipStream_t)stream));
}

kq_status kq_fit_layer(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init, int32_t iters, float* C,
                       int32_t* idx, int32_t* counts, double* distortion, uint32_t flags, void* ws, size_t ws_bytes,
                       void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || k > n || iters < 0 || flags != 0) return KQ_ERR_ARG;
    if (!C_init || !aligned(C_init, 4)) return KQ_ERR_ARG;
    kq_layer l = {X, n, k, C, idx, nullptr, counts, distortion};
    kq_status st = check_layers(&l, 1, true);
    if (st != KQ_OK) return st;
    st = check_ws(ws, ws_bytes, layer_ws_bytes(n, k));
    if (st != KQ_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    if (C_init != C) {
        if (hipMemcpyAsync(C, C_init, sizeof(float) * (size_t)k * KQ_DIM, hipMemcpyDeviceToDevice, s) != hipSuccess)
            return KQ_ERR_HIP;
    }
    return run_fit(&l, 1, iters, (unsigned char*)ws, s);
}

kq_status kq_assign_stack(const kq_layer* layers, int32_t n_layers, int32_t dist_slot, uint32_t flags, void* ws,
                          size_t ws_bytes, void* stream) {
    kq_status st = check_layers(layers, n_layers, false);
    if (st != KQ_OK) return st;
    if (dist_slot < 0 || flags != 0) return KQ_ERR_ARG;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        StackParams p;
        stack_params(p, layers, l0, l1, (unsigned char*)ws, false, dist_slot, false);
        if (launch_assign(p, (hipStream_t)stream) != hipSuccess) return KQ_ERR_HIP;
    }
    return KQ_OK;
}

kq_status kq_update_stack(const kq_layer* layers, int32_t n_layers, uint32_t flags, void* ws, size_t ws_bytes,
                          void* stream) {
    kq_status st = check_layers(layers, n_layers, false);
    if (st != KQ_OK) return st;
    if ((flags & ~KQ_F_COUNTS_ONLY) != 0) return KQ_ERR_ARG;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        StackParams p;
        stack_params(p, layers, l0, l1, (unsigned char*)ws, true, 0, (flags & KQ_F_COUNTS_ONLY) != 0);
        if (launch_update(p, (hipStream_t)stream) != hipSuccess) return KQ_ERR_HIP;
    }
    return KQ_OK;
}

kq_status kq_fit_stack(const kq_layer* layers, int32_t n_layers, int32_t iters, uint32_t flags, void* ws,
                       size_t ws_bytes, void* stream) {
    kq_status st = check_layers(layers, n_layers, true);
    if (st != KQ_OK) return st;
    if (iters < 0 || flags != 0) return KQ_ERR_ARG;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    return run_fit(layers, n_layers, iters, (unsigned char*)ws, (hipStream_t)stream);
}

static kq_status check_cbq(const kq_cbq_layer& l, int32_t bits, int32_t mode, int32_t iters) {
    if (l.k > KQ_MAX_K || bits < 1 || bits > 8) return KQ_ERR_UNSUPPORTED;
    if (!valid_k(l.k) || iters < 0 || (mode != KQ_CBQ_WKMEANS && mode != KQ_CBQ_UNIFORM)) return KQ_ERR_ARG;
    if (!l.C || !l.codes || !l.levels || !aligned(l.C, 4) || !aligned(l.levels, 4)) return KQ_ERR_ARG;
    if ((l.weights && !aligned(l.weights, 4)) || (l.C_hat && !aligned(l.C_hat, 4))) return KQ_ERR_ARG;
    return KQ_OK;
}

kq_status kq_quantize_codebook_stack(const kq_cbq_layer* layers, int32_t n_layers, int32_t bits, int32_t mode,
                                     int32_t iters, void* stream) {
    if (layers == nullptr || n_layers < 1) return KQ_ERR_ARG;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_status st = check_cbq(layers[l], bits, mode, iters);
        if (st != KQ_OK) return st;
    }
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        CbqParams p;
        memset(&p, 0, sizeof(p));
        p.nlayers = l1 - l0;
        p.bits = bits;
        p.mode = mode;
        p.iters = iters;
        for (int32_t l = l0; l < l1; ++l) {
            const kq_cbq_layer& s = layers[l];
            p.L[l - l0] = CbqLayer{s.C, s.weights, s.codes, s.levels, s.C_hat, s.k};
        }
        if (launch_cbq(p, (hipStream_t)stream) != hipSuccess) return KQ_ERR_HIP;
    }
    return KQ_OK;
}

kq_status kq_quantize_codebook(const float* C, int32_t k, int32_t dim, const int32_t* weights, int32_t bits,
                               int32_t mode, int32_t iters, uint8_t* codes, float* levels, float* C_hat, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    kq_cbq_layer l = {C, k, weights, codes, levels, C_hat};
    return kq_quantize_codebook_stack(&l, 1, bits, mode, iters, stream);
}

kq_status kq_pack_bits(const void* values, int32_t elem_bytes, int64_t count, int32_t bits, uint8_t* out,
                       void* stream) {
    if (bits < 0 || bits > 16) return KQ_ERR_UNSUPPORTED;
    if (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4) return KQ_ERR_ARG;
    if (count < 0 || count >= (int64_t(1) << 31)) return KQ_ERR_ARG;
    if (count == 0 || bits == 0) return KQ_OK;
    if (!values || !out || !aligned(values, (uintptr_t)elem_bytes) || !aligned(out, 4)) return KQ_ERR_ARG;
    return hip_status(launch_pack(values, elem_bytes, count, bits, out, (hipStream_t)stream));
}

kq_status kq_unpack_bits(const uint8_t* in, int64_t count, int32_t bits, int32_t* values, void* stream) {
    if (bits < 0 || bits > 16) return KQ_ERR_UNSUPPORTED;
    if (count < 0 || count >= (int64_t(1) << 31)) return KQ_ERR_ARG;
    if (count == 0) return KQ_OK;
    if (!values || !aligned(values, 4) || (bits > 0 && !in)) return KQ_ERR_ARG;
    return hip_status(launch_unpack(in, count, bits, values, (hipStream_t)stream));
}

kq_status kq_reconstruct(const int32_t* idx, int64_t n, const float* C, int32_t k, int32_t dim, float* W_hat,
                         void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k)) return KQ_ERR_ARG;
    if (!idx || !C || !W_hat || !aligned(idx, 4) || !aligned(C, 4) || !aligned(W_hat, 16)) return KQ_ERR_ARG;
    return hip_status(launch_reconstruct(idx, nullptr, 0, n, C, k, W_hat, (hipStream_t)stream));
}

kq_status kq_reconstruct_packed(const uint8_t* packed, int32_t bits, int64_t n, const float* C, int32_t k,
                                int32_t dim, float* W_hat, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K || bits < 0 || bits > 16) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k)) return KQ_ERR_ARG;
    if ((bits > 0 && !packed) || !C || !W_hat || !aligned(C, 4) || !aligned(W_hat, 16)) return KQ_ERR_ARG;
    return hip_status(launch_reconstruct(nullptr, packed, bits, n, C, k, W_hat, (hipStream_t)stream));
}

kq_status kq_sq_error(const float* A, const float* B, int64_t count, double* out, void* ws, size_t ws_bytes,
                      void* stream) {
    if (count < 1 || count >= (int64_t(1) << 40)) return KQ_ERR_ARG;
    if (!A || !B || !out || !aligned(A, 4) || !aligned(B, 4) || !aligned(out, 8)) return KQ_ERR_ARG;
    const kq_status w = check_ws(ws, ws_bytes, kq_workspace_bytes(KQ_OP_SQ_ERROR, count, 1));
    if (w != KQ_OK) return w;
    return hip_status(launch_sq_error(A, B, count, out, ws, (hipStream_t)stream));
}

}  // extern "C"
