// C ABI of libkq: argument checks, workspace layout and launches.
//
// Every entry point checks its arguments before it touches HIP, so argument errors
// come back without a GPU (and without initialising the HIP runtime).  No entry point
// allocates memory; device scratch comes from the caller's workspace.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "kq_internal.h"

using namespace kq;

namespace {

constexpr int32_t kAbiVersion = 10;

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

enum class Op { Assign, Update };

// Launch parameters for layers [l0, l1) of a stack.  `base` points at the workspace
// of layer 0 (the regions of the layers follow each other in order).  C_alt (nullable):
// for an assignment the codebook of each layer to assign against instead of its C; for an
// update the previous codebook (entries kept when empty, the distortion's codebook).
void stack_params(StackParams& p, const kq_layer* layers, int32_t l0, int32_t l1, unsigned char* base, Op op,
                  int32_t dist_slot, const float* const* C_alt, uint32_t kflags, bool from_assign = false) {
    memset(&p, 0, sizeof(p));
    size_t off = 0;
    for (int32_t l = 0; l < l0; ++l) off += layer_ws_bytes(layers[l].n, layers[l].k);
    int64_t weighted_n = 0;  // update: every range of a layer reads its kernels' indices
    for (int32_t l = l0; l < l1; ++l) weighted_n += layers[l].n * update_ranges(layers[l].k);
    const int kpb = update_kernels_per_block(weighted_n);
    int unit = 0;
    for (int32_t l = l0; l < l1; ++l) {
        const kq_layer& s = layers[l];
        DevLayer& d = p.L[l - l0];
        unsigned char* w = base + off;
        d.X = s.X;
        d.C = s.C;
        d.C_old = s.C;
        if (C_alt && C_alt[l]) {
            if (op == Op::Assign) d.C = const_cast<float*>(C_alt[l]);
            else d.C_old = C_alt[l];
        }
        d.idx = s.idx;
        d.n = (int)s.n;
        d.k = s.k;
        d.shift = base_shift(s.n);
        d.dist = s.distortion ? s.distortion + dist_slot : nullptr;
        d.hist = (long long*)(w + ws_assign_part(s.n) + ws_update_part(s.n, s.k));
        d.xmax = base ? (unsigned*)(w + ws_xmax_offset(s.n, s.k)) : nullptr;
        d.nxmax = absmax_blocks(s.n);
        if (op == Op::Assign) {
            d.best_d = s.best_d;
            d.part = base ? (double*)w : nullptr;  // partials whenever there is a workspace
            d.nunits = assign_units(s.n);
        } else {
            d.counts = s.counts;
            if (d.dist && from_assign) {
                d.apart = (const double*)w;
                d.napart = assign_units(s.n);
            } else if (d.dist) {
                d.part = (double*)(w + ws_assign_part(s.n));
            }
            d.ranges = update_ranges(s.k);
            d.krange = (s.k + d.ranges - 1) / d.ranges;
            d.chunk = update_chunk(s.n, s.k, kpb);
            d.nchunks = (int)((s.n + d.chunk - 1) / d.chunk);
            d.nunits = d.ranges * d.nchunks;
            d.flags = (int)kflags;
        }
        d.unit_begin = unit;
        unit += d.nunits;
        off += layer_ws_bytes(s.n, s.k);
    }
    p.nlayers = l1 - l0;
    p.total_units = unit;
    set_unit_table(p);
}

// The largest magnitudes of layers [l0, l1) (their X: kernels, or gradients) and from them
// the fixed-point shift of each layer's sums, in the workspace.  With `validate` the call
// waits for them and returns KQ_ERR_RANGE when any value is NaN or infinite.
kq_status run_xmax(const kq_layer* layers, int32_t l0, int32_t l1, unsigned char* ws, hipStream_t s, bool validate) {
    StackParams p;
    stack_params(p, layers, l0, l1, ws, Op::Update, 0, nullptr, 0);
    unsigned* flags = p.L[0].xmax + p.L[0].nxmax + 1;  // the first layer's region holds the call's flags
    p.range_flags = validate ? flags : nullptr;
    if (launch_absmax(p, s, validate) != hipSuccess) return KQ_ERR_HIP;
    if (!validate) return KQ_OK;  // the first launch that forms sums derives the shifts
    unsigned h[KQ_MAX_STACK] = {0};
    if (hipMemcpyAsync(h, flags, sizeof(unsigned) * (size_t)p.nlayers, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return KQ_ERR_HIP;
    for (int l = 0; l < p.nlayers; ++l)
        if (h[l] != 0u) return KQ_ERR_RANGE;
    return KQ_OK;
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

bool any_distortion(const kq_layer* layers, int32_t l0, int32_t l1) {
    for (int32_t l = l0; l < l1; ++l)
        if (layers[l].distortion) return true;
    return false;
}

bool fusable(const kq_layer* layers, int32_t l0, int32_t l1) {
    for (int32_t l = l0; l < l1; ++l)
        if (layers[l].k > kFuseMaxK) return false;
    return true;
}

// The assignment's workgroups over layers [l0, l1): each layer gets its own workgroups
// (assign_partition), which split its units evenly; a layer's fused partials are those of
// its workgroups.  For every layer: its first workgroup and their number; returns the grid.
int fused_slots(const kq_layer* layers, int32_t l0, int32_t l1, int* wfirst, int* nslots) {
    int units[KQ_MAX_STACK];
    for (int32_t l = l0; l < l1; ++l) units[l - l0] = assign_units(layers[l].n);
    const int grid = assign_partition(units, l1 - l0, nslots);
    int w = 0;
    for (int32_t l = 0; l < l1 - l0; ++l) {
        wfirst[l] = w;
        w += nslots[l];
    }
    return grid;
}

// assignment of layers [l0, l1) (+ the distortion finish when any layer asks for it);
// `fused` also leaves the member sums of the new assignment in the workspace (the layers'
// shifts must be in place: run_xmax)
kq_status run_assign(const kq_layer* layers, int32_t l0, int32_t l1, unsigned char* ws, int32_t slot, hipStream_t s,
                     bool fused = false, const float* const* C_alt = nullptr, void* const* events = nullptr,
                     bool derive = false) {
    StackParams p;
    stack_params(p, layers, l0, l1, ws, Op::Assign, slot, C_alt, 0);
    p.derive_shift = derive ? 1 : 0;
    {
        int wf[KQ_MAX_STACK], ns[KQ_MAX_STACK];
        p.assign_grid = fused_slots(layers, l0, l1, wf, ns);
        for (int l = 0; l < KQ_MAX_STACK; ++l) p.wg_begin[l] = l < p.nlayers ? wf[l] : 0x7fffffff;
        for (int l = 0; l < p.nlayers; ++l) p.L[l].wfirst = wf[l];
    }
    hipEvent_t e0 = events ? (hipEvent_t)events[0] : nullptr, e1 = events ? (hipEvent_t)events[1] : nullptr;
    if (launch_assign(p, s, fused, e0, e1) != hipSuccess) return KQ_ERR_HIP;
    if (any_distortion(layers, l0, l1) && launch_assign_finish(p, s) != hipSuccess) return KQ_ERR_HIP;
    return KQ_OK;
}

// `sums_from_assign`: the preceding fused assignment of the same layers left the member
// sums (and the distortion partials): only the finishing launch runs.  Otherwise the
// layers' shifts must be in place (run_xmax) unless only counts are asked for.
kq_status run_update(const kq_layer* layers, int32_t l0, int32_t l1, unsigned char* ws, int32_t slot,
                     const float* const* C_old, uint32_t kflags, hipStream_t s, bool from_assign = false,
                     bool sums_from_assign = false, bool derive = false) {
    StackParams p;
    stack_params(p, layers, l0, l1, ws, Op::Update, slot, C_old, kflags, from_assign || sums_from_assign);
    p.derive_shift = derive ? 1 : 0;
    if (sums_from_assign) {
        int wf[KQ_MAX_STACK], ns[KQ_MAX_STACK];
        fused_slots(layers, l0, l1, wf, ns);
        for (int l = 0; l < p.nlayers; ++l) p.L[l].nchunks = ns[l];
    } else if (launch_update(p, s) != hipSuccess) {
        return KQ_ERR_HIP;
    }
    if (launch_update_finish(p, s) != hipSuccess) return KQ_ERR_HIP;
    return KQ_OK;
}

// Eq. (2) on layers [l0, l1): the largest |g| and the shift of each layer, the segmented
// sums of the gradients (layers[l].X holds them), then c - gamma * mean into layers[l].C
kq_status run_grad(const kq_layer* layers, int32_t l0, int32_t l1, unsigned char* ws, const float* const* C_old,
                   float gamma, hipStream_t s) {
    kq_layer quiet[KQ_MAX_STACK];
    for (int32_t l = l0; l < l1; ++l) {
        quiet[l - l0] = layers[l];
        quiet[l - l0].distortion = nullptr;
    }
    size_t off = 0;
    for (int32_t l = 0; l < l0; ++l) off += layer_ws_bytes(layers[l].n, layers[l].k);
    kq_status st = run_xmax(quiet, 0, l1 - l0, ws + off, s, false);
    if (st != KQ_OK) return st;
    StackParams p;
    stack_params(p, quiet, 0, l1 - l0, ws + off, Op::Update, 0, C_old ? C_old + l0 : nullptr, kFlagGrad);
    p.derive_shift = 1;  // the shift pass above left the block maxima of |g|
    for (int l = 0; l < p.nlayers; ++l) p.L[l].gamma = gamma;
    if (launch_update(p, s) != hipSuccess) return KQ_ERR_HIP;
    if (launch_update_finish(p, s) != hipSuccess) return KQ_ERR_HIP;
    return KQ_OK;
}

bool finite_gamma(float g) { return g == g && g < 3.4e38f && g > -3.4e38f; }

// Lloyd rounds on a stack: the shifts of the layers' sums once (one pass over the kernels),
// then per round the assignment (leaving distortion partials, and with every k <= 256 the
// member sums, in the workspace) and the update, whose finishing kernel adds those partials;
// the final assignment is followed by a counts-only update that does the same.  C_init
// (nullable, per layer nullable): round 0 assigns against C_init[l] and keeps its entries
// when empty, so layers[l].C need not hold the start.
kq_status run_fit(const kq_layer* layers, int32_t n_layers, int32_t iters, unsigned char* ws, hipStream_t s,
                  const float* const* C_init = nullptr, bool validate = false, void* const* round_events = nullptr) {
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {  // every layer's shift (and range check) first
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        const kq_status st = run_xmax(layers, l0, l1, ws, s, validate);
        if (st != KQ_OK) return st;
    }
    kq_layer quiet[KQ_MAX_STACK];
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        for (int32_t l = l0; l < l1; ++l) {
            quiet[l - l0] = layers[l];
            quiet[l - l0].distortion = nullptr;
        }
        size_t off = 0;
        for (int32_t l = 0; l < l0; ++l) off += layer_ws_bytes(layers[l].n, layers[l].k);
        unsigned char* w = ws + off;
        const float* const* init = C_init ? C_init + l0 : nullptr;
        bool need_last = false;
        for (int32_t l = l0; l < l1; ++l) need_last |= layers[l].counts != nullptr || layers[l].distortion != nullptr;
        if (iters == 0 && init) {  // no update will write C: it takes the start as it is
            for (int32_t l = l0; l < l1; ++l) {
                if (!C_init[l] || C_init[l] == layers[l].C) continue;
                if (hipMemcpyAsync(layers[l].C, C_init[l], sizeof(float) * KQ_DIM * (size_t)layers[l].k,
                                   hipMemcpyDeviceToDevice, s) != hipSuccess)
                    return KQ_ERR_HIP;
            }
            init = nullptr;
        }
        const bool fused = fusable(layers, l0, l1);  // the member sums come with the assignment
        // with fused sums nothing reads a round's indices but the last round's: the rounds
        // before it store none (nor best distances)
        kq_layer inner[KQ_MAX_STACK];
        for (int32_t l = 0; l < l1 - l0; ++l) {
            inner[l] = quiet[l];
            inner[l].idx = nullptr;
            inner[l].best_d = nullptr;
        }
        for (int32_t t = 0; t <= iters; ++t) {
            const bool last = (t == iters);
            const float* const* from = t == 0 ? init : nullptr;
            void* const* ev = (round_events && l0 == 0) ? round_events + 2 * t : nullptr;
            // round 0 forms the shifts (from the block maxima) unless the range check did
            const bool derive = t == 0 && !validate;
            const bool fuse_t = fused && !(last && !need_last);
            kq_status st = run_assign(fuse_t && !last ? inner : quiet, 0, l1 - l0, w, 0, s, fuse_t, from, ev, derive);
            if (st != KQ_OK) return st;
            if (last && !need_last) break;
            st = run_update(layers + l0, 0, l1 - l0, w, t, from, last ? kFlagCountsOnly : 0, s, true, fused, derive);
            if (st != KQ_OK) return st;
        }
    }
    return KQ_OK;
}

// ---- Yinyang workspace: the layer's own region (assignment partials, update partials and
// histograms), then the grouping fit's region, then the Yinyang state ----------------------
struct YyLayout {
    size_t sub, Cg, labels, Cw, perm, gstart, radius, delta, cnt, Lt, B1, J1, B2, lists, mask, flist, bd, wgc, total;
};

YyLayout yy_layout(int64_t n, int32_t k, int t) {
    YyLayout L;
    size_t o = layer_ws_bytes(n, k);
    auto take = [&o](size_t b) {
        const size_t at = o;
        o += align256(b);
        return at;
    };
    const size_t tn = (size_t)t * (size_t)n;
    L.sub = take(layer_ws_bytes(k, t));
    L.Cg = take(sizeof(float) * KQ_DIM * (size_t)t);
    L.labels = take(sizeof(int32_t) * (size_t)k);
    L.Cw = take(sizeof(float) * KQ_DIM * (size_t)k);
    L.perm = take(sizeof(int32_t) * (size_t)k);
    L.gstart = take(sizeof(int32_t) * (size_t)(t + 1));
    L.radius = take(sizeof(float) * (size_t)t);
    L.delta = take(sizeof(double) * (size_t)t);
    L.cnt = take(sizeof(int32_t) * (size_t)(t + 1));
    L.Lt = take(sizeof(float) * tn);
    L.B1 = take(sizeof(float) * tn);
    L.J1 = take(sizeof(int32_t) * tn);
    L.B2 = take(sizeof(float) * tn);
    L.lists = take(sizeof(int32_t) * tn);
    L.mask = take(sizeof(unsigned long long) * (size_t)n);
    L.flist = take(sizeof(int32_t) * (size_t)n);
    L.bd = take(sizeof(float) * (size_t)n);
    L.wgc = take(sizeof(int32_t) * (size_t)(t + 1) * (size_t)((n + 255) / 256));
    L.total = o;
    return L;
}

// groups <= 0 picks the default; otherwise 1 .. min(64, k); returns 0 when invalid
int yy_groups(int32_t k, int32_t groups) {
    if (groups <= 0) return yy_default_groups(k) < k ? yy_default_groups(k) : k;
    return groups <= kYyMaxGroups && groups <= k ? groups : 0;
}

YyParams yy_params(unsigned char* ws, const YyLayout& L, const float* X, int64_t n, int32_t k, int t,
                   const float* C, const float* C_prev, int32_t* idx, float* best_d, long long* stats) {
    YyParams p;
    memset(&p, 0, sizeof(p));
    p.X = X;
    p.C = C;
    p.C_prev = C_prev;
    p.idx = idx;
    p.best_d = best_d ? best_d : (float*)(ws + L.bd);
    p.Cg = (const float*)(ws + L.Cg);
    p.labels = (const int32_t*)(ws + L.labels);
    p.perm = (int32_t*)(ws + L.perm);
    p.gstart = (int32_t*)(ws + L.gstart);
    p.radius = (float*)(ws + L.radius);
    p.delta = (double*)(ws + L.delta);
    p.cnt = (int32_t*)(ws + L.cnt);
    p.Lt = (float*)(ws + L.Lt);
    p.B1 = (float*)(ws + L.B1);
    p.J1 = (int32_t*)(ws + L.J1);
    p.B2 = (float*)(ws + L.B2);
    p.lists = (int32_t*)(ws + L.lists);
    p.mask = (unsigned long long*)(ws + L.mask);
    p.flist = (int32_t*)(ws + L.flist);
    p.wgc = (int32_t*)(ws + L.wgc);
    p.part = (double*)ws;  // the layer's assignment partials
    p.stats = stats;
    p.n = (int)n;
    p.k = k;
    p.t = t;
    p.npart = assign_units(n);
    return p;
}

// the groups of codebook C (a few Lloyd rounds on its entries, the first t entries as
// seeds), the perm / radius tables and the initial bounds of every kernel
kq_status yy_start(unsigned char* ws, const YyLayout& L, const float* X, int64_t n, const float* C, int32_t k, int t,
                   hipStream_t s) {
    float* Cg = (float*)(ws + L.Cg);
    int32_t* labels = (int32_t*)(ws + L.labels);
    if (hipMemcpyAsync(Cg, C, sizeof(float) * KQ_DIM * (size_t)t, hipMemcpyDeviceToDevice, s) != hipSuccess)
        return KQ_ERR_HIP;
    const kq_layer gl = {C, k, t, Cg, labels, nullptr, nullptr, nullptr};
    const kq_status st = run_fit(&gl, 1, kYyGroupRounds, ws + L.sub, s);
    if (st != KQ_OK) return st;
    const YyParams p = yy_params(ws, L, X, n, k, t, C, nullptr, nullptr, nullptr, nullptr);
    if (launch_yy_group(p, s) != hipSuccess) return KQ_ERR_HIP;
    return hip_status(launch_yy_bounds_init(p, s));
}

// distortion of the round's assignment from its best distances, in the order of the
// assignment kernel's partials
kq_status yy_distortion(const YyParams& p, double* distortion, hipStream_t s) {
    if (launch_yy_partials(p, s) != hipSuccess) return KQ_ERR_HIP;
    if (!distortion) return KQ_OK;
    StackParams q;
    memset(&q, 0, sizeof(q));
    q.nlayers = 1;
    q.L[0].part = p.part;
    q.L[0].dist = distortion;
    q.L[0].nunits = assign_units(p.n);
    set_unit_table(q);
    return hip_status(launch_assign_finish(q, s));
}

kq_status check_yy(const float* X, int64_t n, int32_t dim, int32_t k, int32_t groups, int32_t* idx, float* best_d,
                   double* distortion, int& t) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || k > n) return KQ_ERR_ARG;
    t = yy_groups(k, groups);
    if (t == 0) return KQ_ERR_ARG;
    if (!X || !idx || !aligned(X, 4) || !aligned(idx, 4)) return KQ_ERR_ARG;
    if ((best_d && !aligned(best_d, 4)) || (distortion && !aligned(distortion, 8))) return KQ_ERR_ARG;
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

size_t kq_workspace_bytes(int32_t op, int64_t n, int32_t k, int32_t dim) {
    if (op == KQ_OP_SQ_ERROR) {
        if (n < 1 || n >= (int64_t(1) << 40) || k != 1 || dim != 1) return 0;
        return align256(sizeof(double) * (size_t)sq_error_blocks(n));
    }
    if (!valid_n(n) || !valid_k(k) || dim != KQ_DIM) return 0;
    if (op != KQ_OP_ASSIGN && op != KQ_OP_UPDATE && op != KQ_OP_FIT && op != KQ_OP_GRAD) return 0;
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
    const kq_layer l = {X, n, k, const_cast<float*>(C), idx, best_d, nullptr, distortion};
    // without a distortion the workspace (unchecked then) is not touched
    return run_assign(&l, 0, 1, distortion ? (unsigned char*)ws : nullptr, 0, (hipStream_t)stream);
}

kq_status kq_update(const float* X, int64_t n, int32_t dim, const int32_t* idx, int32_t k, const float* C_old,
                    float* C_new, int32_t* counts, double* distortion, uint32_t flags, void* ws, size_t ws_bytes,
                    void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || (flags & ~(KQ_F_COUNTS_ONLY | KQ_F_VALIDATE)) != 0) return KQ_ERR_ARG;
    if (!X || !idx || !C_old || !C_new || !aligned(X, 4) || !aligned(idx, 4) || !aligned(C_old, 4) ||
        !aligned(C_new, 4))
        return KQ_ERR_ARG;
    if ((counts && !aligned(counts, 4)) || (distortion && !aligned(distortion, 8))) return KQ_ERR_ARG;
    const kq_status w = check_ws(ws, ws_bytes, layer_ws_bytes(n, k));
    if (w != KQ_OK) return w;
    const kq_layer l = {X, n, k, C_new, const_cast<int32_t*>(idx), nullptr, counts, distortion};
    const float* olds[1] = {C_old};
    const bool counts_only = (flags & KQ_F_COUNTS_ONLY) != 0, validate = (flags & KQ_F_VALIDATE) != 0;
    hipStream_t s = (hipStream_t)stream;
    if (!counts_only || validate) {  // the shift of the layer's sums (and the range check)
        const kq_status st = run_xmax(&l, 0, 1, (unsigned char*)ws, s, validate);
        if (st != KQ_OK) return st;
    }
    return run_update(&l, 0, 1, (unsigned char*)ws, 0, olds, counts_only ? kFlagCountsOnly : 0, s, false, false,
                      !validate);
}

kq_status kq_codebook_grad_step(const float* G, int64_t n, int32_t dim, const int32_t* idx, int32_t k,
                                const float* C_old, float gamma, float* C_new, int32_t* counts, void* ws,
                                size_t ws_bytes, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || !finite_gamma(gamma)) return KQ_ERR_ARG;
    if (!G || !idx || !C_old || !C_new || !aligned(G, 4) || !aligned(idx, 4) || !aligned(C_old, 4) ||
        !aligned(C_new, 4) || (counts && !aligned(counts, 4)))
        return KQ_ERR_ARG;
    const kq_status w = check_ws(ws, ws_bytes, layer_ws_bytes(n, k));
    if (w != KQ_OK) return w;
    const kq_layer l = {G, n, k, C_new, const_cast<int32_t*>(idx), nullptr, counts, nullptr};
    const float* olds[1] = {C_old};
    return run_grad(&l, 0, 1, (unsigned char*)ws, olds, gamma, (hipStream_t)stream);
}

kq_status kq_codebook_grad_step_stack(const kq_layer* layers, int32_t n_layers, float gamma, void* ws,
                                      size_t ws_bytes, void* stream) {
    kq_status st = check_layers(layers, n_layers, false);
    if (st != KQ_OK) return st;
    if (!finite_gamma(gamma)) return KQ_ERR_ARG;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        st = run_grad(layers, l0, l1, (unsigned char*)ws, nullptr, gamma, (hipStream_t)stream);
        if (st != KQ_OK) return st;
    }
    return KQ_OK;
}

// the FC quantizer's launch parameters over the workspace layout of fc_ws_bytes
static void fc_params(FcParams& p, const float* v, const int32_t* w, int64_t count, int32_t bits, int32_t iters,
                      uint8_t* codes, float* levels, float* v_hat, int32_t* rounds, int thr_mode, void* ws) {
    const size_t G = (size_t)fc_grid(count), nlev = (size_t)1 << bits;
    unsigned char* b = (unsigned char*)ws;
    memset(&p, 0, sizeof(p));
    p.v = v;
    p.w = w;
    p.codes = codes;
    p.levels_out = levels;
    p.v_hat = v_hat;
    p.rounds_out = rounds;
    p.m = count;
    p.bits = bits;
    p.iters = iters;
    p.thr_mode = thr_mode;
    p.minmax = (float*)b;
    p.range = p.minmax + 3 * G;
    b += align256(sizeof(float) * (3 * G + 4));
    p.part = (long long*)b;
    b += align256(sizeof(long long) * G * nlev * 12);
    p.S = (long long*)b;
    b += align256(sizeof(long long) * nlev * 12);
    p.lev = (float*)b;
    b += align256(sizeof(float) * nlev);
    p.lev_next = (float*)b;
    b += align256(sizeof(float) * nlev);
    p.thr = (float*)b;
    b += align256(sizeof(float) * nlev);
    p.state = (int*)b;
    b += align256(sizeof(int) * 4);
    p.wg_changed = (int*)b;
    b += align256(sizeof(int) * G);
    p.tbl = (unsigned*)b;
}

size_t kq_quantize_scalars_workspace_bytes(int64_t count, int32_t bits) {
    if (count < 1 || count >= (int64_t(1) << 31) || bits < 1 || bits > 8) return 0;
    return fc_ws_bytes(count, bits);
}

kq_status kq_quantize_scalars(const float* v, int64_t count, int32_t bits, int32_t iters, uint8_t* codes,
                              float* levels, float* v_hat, int32_t* rounds, uint32_t flags, void* ws, size_t ws_bytes,
                              void* stream) {
    if (bits < 1 || bits > 8) return KQ_ERR_UNSUPPORTED;
    if (count < 1 || count >= (int64_t(1) << 31) || iters < 0) return KQ_ERR_ARG;
    if ((flags & ~(KQ_F_EXACT_SEARCH | KQ_F_THRESHOLDS)) != 0 ||
        (flags & (KQ_F_EXACT_SEARCH | KQ_F_THRESHOLDS)) == (KQ_F_EXACT_SEARCH | KQ_F_THRESHOLDS))
        return KQ_ERR_ARG;
    if (!v || !codes || !levels || !aligned(v, 4) || !aligned(levels, 4)) return KQ_ERR_ARG;
    if ((v_hat && !aligned(v_hat, 4)) || (rounds && !aligned(rounds, 4))) return KQ_ERR_ARG;
    const kq_status w = check_ws(ws, ws_bytes, fc_ws_bytes(count, bits));
    if (w != KQ_OK) return w;
    FcParams p;
    fc_params(p, v, nullptr, count, bits, iters, codes, levels, v_hat, rounds,
              (flags & KQ_F_EXACT_SEARCH) ? 1 : ((flags & KQ_F_THRESHOLDS) ? 2 : 0), ws);
    return hip_status(launch_fc_quantize(p, (hipStream_t)stream));
}

// a fit workspace large enough for every codebook size up to kmax (the per-layer layout
// is not monotone in k: small codebooks keep one fused partial per assignment workgroup)
size_t fit_ws_upto(int64_t n, int32_t kmax) {
    const size_t c1024 = (size_t)((n + 1023) / 1024);
    return ws_assign_part(n) + align256(sizeof(double) * (size_t)update_ranges(kmax) * c1024) +
           align256(sizeof(int64_t) * 10 * (size_t)kmax * (size_t)std::max<int64_t>(fused_parts(n), (n + kUpdateMinKernelsPerBlock - 1) / kUpdateMinKernelsPerBlock)) +
           ws_xmax(n);
}

size_t kq_search_workspace_bytes(int64_t n, int32_t n_init, int32_t lloyd_iters) {
    if (!valid_n(n) || !valid_k(n_init) || n_init > n || lloyd_iters < 0) return 0;
    return fit_ws_upto(n, n_init) + align256(sizeof(float) * KQ_DIM * (size_t)n_init) +
           align256(sizeof(int32_t) * (size_t)n) + align256(sizeof(double) * (size_t)(lloyd_iters + 1));
}

kq_status kq_search_codebook_size(const float* X, int64_t n, int32_t dim, const float* C_cand, int32_t n_init, float r,
                                  int32_t max_iter, int32_t lloyd_iters, float* C, int32_t* idx, int32_t* k_out,
                                  int32_t* trial_k, double* trial_d, double* d_init, void* ws, size_t ws_bytes,
                                  void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (n_init > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(n_init) || n_init > n || max_iter < 0 || lloyd_iters < 0) return KQ_ERR_ARG;
    if (!(r >= 0.0f) || !finite_gamma(r)) return KQ_ERR_ARG;
    if (!X || !C_cand || !C || !idx || !k_out || !aligned(X, 4) || !aligned(C_cand, 4) || !aligned(C, 4) ||
        !aligned(idx, 4))
        return KQ_ERR_ARG;
    const size_t need = kq_search_workspace_bytes(n, n_init, lloyd_iters);
    if (check_ws(ws, ws_bytes, need) != KQ_OK) return KQ_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    unsigned char* w = (unsigned char*)ws;
    float* C_try = (float*)(w + fit_ws_upto(n, n_init));
    int32_t* idx_try = (int32_t*)((unsigned char*)C_try + align256(sizeof(float) * KQ_DIM * (size_t)n_init));
    double* J = (double*)((unsigned char*)idx_try + align256(sizeof(int32_t) * (size_t)n));
    // one fit of size k from the first k candidates; its final distortion back on the host
    auto trial = [&](int32_t k, float* Cout, int32_t* iout, double& d) -> kq_status {
        const kq_layer l = {X, n, k, Cout, iout, nullptr, nullptr, J};
        if (hipMemcpyAsync(Cout, C_cand, sizeof(float) * KQ_DIM * (size_t)k, hipMemcpyDeviceToDevice, s) !=
            hipSuccess)
            return KQ_ERR_HIP;
        const kq_status st = run_fit(&l, 1, lloyd_iters, w, s);
        if (st != KQ_OK) return st;
        if (hipMemcpyAsync(&d, J + lloyd_iters, sizeof(double), hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess)
            return KQ_ERR_HIP;
        return KQ_OK;
    };
    double d0 = 0.0;
    kq_status st = trial(n_init, C, idx, d0);  // the baseline size; its result is kept until beaten
    if (st != KQ_OK) return st;
    if (d_init) *d_init = d0;
    const double target = (1.0 + (double)r) * d0;
    int32_t upper = n_init, lower = 0;
    for (int32_t i = 0; i < max_iter; ++i) {
        const int32_t cur = (int32_t)(((int64_t)upper + lower) / 2);
        if (cur <= lower || cur >= upper) {
            for (int32_t q = i; q < max_iter; ++q) {
                if (trial_k) trial_k[q] = 0;
                if (trial_d) trial_d[q] = 0.0;
            }
            break;
        }
        double d = 0.0;
        if ((st = trial(cur, C_try, idx_try, d)) != KQ_OK) return st;
        if (trial_k) trial_k[i] = cur;
        if (trial_d) trial_d[i] = d;
        if (d < target) {  // within the allowed distortion: the new upper bound, and the result so far
            upper = cur;
            if (hipMemcpyAsync(C, C_try, sizeof(float) * KQ_DIM * (size_t)cur, hipMemcpyDeviceToDevice, s) !=
                    hipSuccess ||
                hipMemcpyAsync(idx, idx_try, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToDevice, s) != hipSuccess)
                return KQ_ERR_HIP;
        } else {
            lower = cur;
        }
    }
    *k_out = upper;
    return hip_status(hipStreamSynchronize(s));
}

// ---- kq_fit_layer_noalloc: the fit with its scratch in a static device array -------------
// Each device the library runs on holds one copy of `scratch` (until the process ends); host
// code must never pass the array's name to a kernel or a copy (on the host it names a
// stand-in, not device memory).  The device address comes from hipGetSymbolAddress, taken
// once per device with that device current, and is kept here.
static __device__ __align__(256) unsigned char scratch[KQ_NOALLOC_SCRATCH_BYTES];
constexpr int kNoAllocMaxDevices = 64;
static void* g_scratch_ptr[kNoAllocMaxDevices];
static std::mutex g_scratch_mutex;

static kq_status scratch_for_current_device(unsigned char** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return KQ_ERR_HIP;
    if (dev >= kNoAllocMaxDevices) return KQ_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return KQ_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = (unsigned char*)g_scratch_ptr[dev];
    return KQ_OK;
}

kq_status kq_fit_layer(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init, int32_t iters, float* C,
                       int32_t* idx, int32_t* counts, double* distortion, uint32_t flags, void* ws, size_t ws_bytes,
                       void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || k > n || iters < 0 || (flags & ~KQ_F_VALIDATE) != 0) return KQ_ERR_ARG;
    if (!C_init || !aligned(C_init, 4)) return KQ_ERR_ARG;
    const kq_layer l = {X, n, k, C, idx, nullptr, counts, distortion};
    kq_status st = check_layers(&l, 1, true);
    if (st != KQ_OK) return st;
    st = check_ws(ws, ws_bytes, layer_ws_bytes(n, k));
    if (st != KQ_OK) return st;
    const float* init[1] = {C_init};
    return run_fit(&l, 1, iters, (unsigned char*)ws, (hipStream_t)stream, init, (flags & KQ_F_VALIDATE) != 0);
}

size_t kq_yinyang_workspace_bytes(int64_t n, int32_t k, int32_t groups) {
    if (!valid_n(n) || !valid_k(k) || k > n) return 0;
    const int t = yy_groups(k, groups);
    if (t == 0) return 0;
    return yy_layout(n, k, t).total;
}

kq_status kq_yinyang_init(const float* X, int64_t n, int32_t dim, const float* C, int32_t k, int32_t groups,
                          int32_t* idx, float* best_d, double* distortion, void* ws, size_t ws_bytes, void* stream) {
    int t = 0;
    kq_status st = check_yy(X, n, dim, k, groups, idx, best_d, distortion, t);
    if (st != KQ_OK) return st;
    if (!C || !aligned(C, 4)) return KQ_ERR_ARG;
    const YyLayout L = yy_layout(n, k, t);
    if ((st = check_ws(ws, ws_bytes, L.total)) != KQ_OK) return st;
    unsigned char* w = (unsigned char*)ws;
    hipStream_t s = (hipStream_t)stream;
    const kq_layer l = {X, n, k, const_cast<float*>(C), idx, best_d, nullptr, distortion};
    if ((st = run_assign(&l, 0, 1, w, 0, s)) != KQ_OK) return st;
    return yy_start(w, L, X, n, C, k, t, s);
}

kq_status kq_yinyang_assign(const float* X, int64_t n, int32_t dim, const float* C_prev, const float* C, int32_t k,
                            int32_t groups, int32_t* idx, float* best_d, double* distortion, int64_t* stats, void* ws,
                            size_t ws_bytes, void* stream) {
    int t = 0;
    kq_status st = check_yy(X, n, dim, k, groups, idx, best_d, distortion, t);
    if (st != KQ_OK) return st;
    if (!C || !C_prev || !aligned(C, 4) || !aligned(C_prev, 4) || (stats && !aligned(stats, 8))) return KQ_ERR_ARG;
    const YyLayout L = yy_layout(n, k, t);
    if ((st = check_ws(ws, ws_bytes, L.total)) != KQ_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    const YyParams p = yy_params((unsigned char*)ws, L, X, n, k, t, C, C_prev, idx, best_d, (long long*)stats);
    if (launch_yy_round(p, s) != hipSuccess) return KQ_ERR_HIP;
    return distortion ? yy_distortion(p, distortion, s) : KQ_OK;
}

kq_status kq_fit_layer_yinyang(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init, int32_t iters,
                               int32_t groups, float* C, int32_t* idx, int32_t* counts, double* distortion,
                               int64_t* stats, void* ws, size_t ws_bytes, void* stream) {
    int t = 0;
    kq_status st = check_yy(X, n, dim, k, groups, idx, nullptr, distortion, t);
    if (st != KQ_OK) return st;
    if (iters < 0 || !C_init || !C || !aligned(C_init, 4) || !aligned(C, 4)) return KQ_ERR_ARG;
    if ((counts && !aligned(counts, 4)) || (stats && !aligned(stats, 8))) return KQ_ERR_ARG;
    const YyLayout L = yy_layout(n, k, t);
    if ((st = check_ws(ws, ws_bytes, L.total)) != KQ_OK) return st;
    unsigned char* w = (unsigned char*)ws;
    hipStream_t s = (hipStream_t)stream;
    const size_t cb = sizeof(float) * KQ_DIM * (size_t)k;
    if (C_init != C && hipMemcpyAsync(C, C_init, cb, hipMemcpyDeviceToDevice, s) != hipSuccess) return KQ_ERR_HIP;
    // round 0: the screened assignment (its partials stay in the workspace), groups, bounds
    const kq_layer l0 = {X, n, k, C, idx, nullptr, nullptr, nullptr};
    if ((st = run_assign(&l0, 0, 1, w, 0, s)) != KQ_OK) return st;
    if ((st = yy_start(w, L, X, n, C, k, t, s)) != KQ_OK) return st;
    if (iters > 0 && (st = run_xmax(&l0, 0, 1, w, s, false)) != KQ_OK) return st;  // the shift of the sums
    // rounds 1..iters: update from `cur` into `nxt` (the distortion of the assignment
    // before it from its partials), then the Yinyang assignment against `nxt`
    float* cur = C;
    float* nxt = (float*)(w + L.Cw);
    for (int32_t r = 0; r < iters; ++r) {
        kq_layer lu = {X, n, k, nxt, idx, nullptr, counts, distortion};
        const float* olds[1] = {cur};
        if ((st = run_update(&lu, 0, 1, w, r, olds, 0, s, true, false, r == 0)) != KQ_OK) return st;
        const YyParams p = yy_params(w, L, X, n, k, t, nxt, cur, idx, nullptr, stats ? (long long*)stats + 3 * (size_t)r : nullptr);
        if (launch_yy_round(p, s) != hipSuccess) return KQ_ERR_HIP;
        if (launch_yy_partials(p, s) != hipSuccess) return KQ_ERR_HIP;
        float* tmp = cur;
        cur = nxt;
        nxt = tmp;
    }
    if (counts || distortion) {  // counts of the final assignment, its distortion
        kq_layer lf = {X, n, k, cur, idx, nullptr, counts, distortion};
        if ((st = run_update(&lf, 0, 1, w, iters, nullptr, kFlagCountsOnly, s, true)) != KQ_OK) return st;
    }
    if (cur != C && hipMemcpyAsync(C, cur, cb, hipMemcpyDeviceToDevice, s) != hipSuccess) return KQ_ERR_HIP;
    return KQ_OK;
}

kq_status kq_assign_stack(const kq_layer* layers, int32_t n_layers, int32_t dist_slot, uint32_t flags, void* ws,
                          size_t ws_bytes, void* stream) {
    kq_status st = check_layers(layers, n_layers, false);
    if (st != KQ_OK) return st;
    if (dist_slot < 0 || (flags & ~(KQ_F_FUSED_SUMS | KQ_F_VALIDATE | KQ_F_REUSE_SHIFTS)) != 0) return KQ_ERR_ARG;
    const bool fused = (flags & KQ_F_FUSED_SUMS) != 0, validate = (flags & KQ_F_VALIDATE) != 0;
    const bool reuse = (flags & KQ_F_REUSE_SHIFTS) != 0;
    if (fused && !fusable(layers, 0, n_layers)) return KQ_ERR_UNSUPPORTED;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {  // range checks before anything is written
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        if ((validate || (fused && !reuse)) && (st = run_xmax(layers, l0, l1, (unsigned char*)ws, s, validate)) != KQ_OK)
            return st;
    }
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        st = run_assign(layers, l0, l1, (unsigned char*)ws, dist_slot, s, fused, nullptr, nullptr,
                        fused && !reuse && !validate);
        if (st != KQ_OK) return st;
    }
    return KQ_OK;
}

kq_status kq_update_stack(const kq_layer* layers, int32_t n_layers, int32_t dist_slot, uint32_t flags, void* ws,
                          size_t ws_bytes, void* stream) {
    kq_status st = check_layers(layers, n_layers, false);
    if (st != KQ_OK) return st;
    if (dist_slot < 0 ||
        (flags & ~(KQ_F_COUNTS_ONLY | KQ_F_DISTORTION_FROM_ASSIGN | KQ_F_SUMS_FROM_ASSIGN | KQ_F_VALIDATE |
                   KQ_F_REUSE_SHIFTS)) != 0)
        return KQ_ERR_ARG;
    const bool from_sums = (flags & KQ_F_SUMS_FROM_ASSIGN) != 0, validate = (flags & KQ_F_VALIDATE) != 0;
    const bool counts_only = (flags & KQ_F_COUNTS_ONLY) != 0, reuse = (flags & KQ_F_REUSE_SHIFTS) != 0;
    if (from_sums && !fusable(layers, 0, n_layers)) return KQ_ERR_UNSUPPORTED;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    // the shifts of the sums (the fused assignment left its own), and the range checks, first
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        if ((validate || (!from_sums && !counts_only && !reuse)) &&
            (st = run_xmax(layers, l0, l1, (unsigned char*)ws, s, validate)) != KQ_OK)
            return st;
    }
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        st = run_update(layers, l0, l1, (unsigned char*)ws, dist_slot, nullptr, counts_only ? kFlagCountsOnly : 0, s,
                        (flags & KQ_F_DISTORTION_FROM_ASSIGN) != 0, from_sums,
                        !validate && !from_sums && !counts_only && !reuse);
        if (st != KQ_OK) return st;
    }
    return KQ_OK;
}

kq_status kq_fit_stack(const kq_layer* layers, int32_t n_layers, int32_t iters, uint32_t flags, void* ws,
                       size_t ws_bytes, void* stream) {
    kq_status st = check_layers(layers, n_layers, true);
    if (st != KQ_OK) return st;
    if (iters < 0 || (flags & ~KQ_F_VALIDATE) != 0) return KQ_ERR_ARG;
    st = check_ws(ws, ws_bytes, stack_ws_bytes(layers, n_layers));
    if (st != KQ_OK) return st;
    return run_fit(layers, n_layers, iters, (unsigned char*)ws, (hipStream_t)stream, nullptr,
                   (flags & KQ_F_VALIDATE) != 0);
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

// codebooks of at least this many scalars (k * 9) are quantized by the FC-layer machinery
// on the whole GPU: below, its per-round launches cost more than one workgroup's pass
constexpr int64_t kCbqWideMin = 16384;

size_t kq_quantize_codebook_stack_workspace_bytes(const kq_cbq_layer* layers, int32_t n_layers, int32_t bits) {
    if (layers == nullptr || n_layers < 1 || bits < 1 || bits > 8) return 0;
    size_t b = 0;
    for (int32_t l = 0; l < n_layers; ++l) {
        const int64_t m = (int64_t)layers[l].k * KQ_DIM;
        if (layers[l].k >= 1 && layers[l].k <= KQ_MAX_K && m >= kCbqWideMin) {
            const size_t f = fc_ws_bytes(m, bits);
            b = f > b ? f : b;
        }
    }
    return b;
}

kq_status kq_quantize_codebook_stack_ws(const kq_cbq_layer* layers, int32_t n_layers, int32_t bits, int32_t mode,
                                        int32_t iters, void* ws, size_t ws_bytes, void* stream) {
    if (layers == nullptr || n_layers < 1) return KQ_ERR_ARG;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_status st = check_cbq(layers[l], bits, mode, iters);
        if (st != KQ_OK) return st;
    }
    const size_t need = kq_quantize_codebook_stack_workspace_bytes(layers, n_layers, bits);
    if (need > 0 && mode == KQ_CBQ_WKMEANS) {
        const kq_status w = check_ws(ws, ws_bytes, need);
        if (w != KQ_OK) return w;
    }
    // the small codebooks (and every codebook of a uniform grid) in one launch per 16 layers
    kq_cbq_layer small[KQ_MAX_STACK];
    int32_t ns = 0;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_cbq_layer& s = layers[l];
        if (mode == KQ_CBQ_WKMEANS && (int64_t)s.k * KQ_DIM >= kCbqWideMin) continue;
        small[ns++] = s;
        if (ns == KQ_MAX_STACK) {
            const kq_status st = kq_quantize_codebook_stack(small, ns, bits, mode, iters, stream);
            if (st != KQ_OK) return st;
            ns = 0;
        }
    }
    if (ns > 0) {
        const kq_status st = kq_quantize_codebook_stack(small, ns, bits, mode, iters, stream);
        if (st != KQ_OK) return st;
    }
    // the large ones one after another on the whole GPU, reusing the workspace (stream order)
    if (mode != KQ_CBQ_WKMEANS) return KQ_OK;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_cbq_layer& s = layers[l];
        const int64_t m = (int64_t)s.k * KQ_DIM;
        if (m < kCbqWideMin) continue;
        FcParams p;
        fc_params(p, s.C, s.weights, m, bits, iters, s.codes, s.levels, s.C_hat, nullptr, 0, ws);
        if (launch_fc_quantize(p, (hipStream_t)stream) != hipSuccess) return KQ_ERR_HIP;
    }
    return KQ_OK;
}

kq_status kq_quantize_codebook(const float* C, int32_t k, int32_t dim, const int32_t* weights, int32_t bits,
                               int32_t mode, int32_t iters, uint8_t* codes, float* levels, float* C_hat, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    const kq_cbq_layer l = {C, k, weights, codes, levels, C_hat};
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
    if (!idx || !C || !W_hat || !aligned(idx, 4) || !aligned(C, 4) || !aligned(W_hat, 4)) return KQ_ERR_ARG;
    const kq_recon_layer l = {idx, nullptr, 0, k, n, C, W_hat, nullptr, nullptr};
    return kq_reconstruct_stack(&l, 1, nullptr, 0, stream);
}

kq_status kq_reconstruct_packed(const uint8_t* packed, int32_t bits, int64_t n, const float* C, int32_t k,
                                int32_t dim, float* W_hat, void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K || bits < 0 || bits > 16) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k)) return KQ_ERR_ARG;
    if ((bits > 0 && (!packed || !aligned(packed, 4))) || !C || !W_hat || !aligned(C, 4) || !aligned(W_hat, 4))
        return KQ_ERR_ARG;
    const kq_recon_layer l = {nullptr, packed, bits, k, n, C, W_hat, nullptr, nullptr};
    return kq_reconstruct_stack(&l, 1, nullptr, 0, stream);
}

kq_status kq_sq_error(const float* A, const float* B, int64_t count, double* out, void* ws, size_t ws_bytes,
                      void* stream) {
    if (count < 1 || count >= (int64_t(1) << 40)) return KQ_ERR_ARG;
    if (!A || !B || !out || !aligned(A, 4) || !aligned(B, 4) || !aligned(out, 8)) return KQ_ERR_ARG;
    const kq_status w = check_ws(ws, ws_bytes, kq_workspace_bytes(KQ_OP_SQ_ERROR, count, 1, 1));
    if (w != KQ_OK) return w;
    return hip_status(launch_sq_error(A, B, count, out, ws, (hipStream_t)stream));
}

// ---- stack forms of pack and reconstruct --------------------------------------------------

static kq_status check_pack_job(const kq_pack_job& j) {
    if (j.bits < 0 || j.bits > 16) return KQ_ERR_UNSUPPORTED;
    if (j.elem_bytes != 1 && j.elem_bytes != 2 && j.elem_bytes != 4) return KQ_ERR_ARG;
    if (j.count < 0 || j.count >= (int64_t(1) << 31)) return KQ_ERR_ARG;
    if (j.count == 0 || j.bits == 0) return KQ_OK;
    if (!j.values || !j.out || !aligned(j.values, (uintptr_t)j.elem_bytes) || !aligned(j.out, 4)) return KQ_ERR_ARG;
    return KQ_OK;
}

kq_status kq_pack_bits_stack(const kq_pack_job* jobs, int32_t n_jobs, void* stream) {
    if (jobs == nullptr || n_jobs < 1 || n_jobs > KQ_MAX_PACK_JOBS) return KQ_ERR_ARG;
    for (int32_t q = 0; q < n_jobs; ++q) {
        const kq_status st = check_pack_job(jobs[q]);
        if (st != KQ_OK) return st;
    }
    PackParams p;
    memset(&p, 0, sizeof(p));
    p.njobs = n_jobs;
    long long words = 0;
    for (int32_t q = 0; q < n_jobs; ++q) {
        const kq_pack_job& j = jobs[q];
        const long long bytes = (j.count * (long long)j.bits + 7) / 8;
        p.J[q] = PackJob{j.values, j.out, (long long)j.count, bytes, j.elem_bytes, j.bits};
        p.word_begin[q] = words;
        words += (bytes + 3) / 4;
    }
    for (int32_t q = n_jobs; q <= KQ_MAX_PACK_JOBS; ++q) p.word_begin[q] = q == n_jobs ? words : INT64_MAX;
    return hip_status(launch_pack_stack(p, (hipStream_t)stream));
}

static kq_status check_recon_layer(const kq_recon_layer& l) {
    if (l.k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!l.idx && (l.bits < 0 || l.bits > 16)) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(l.n) || !valid_k(l.k)) return KQ_ERR_ARG;
    if (!l.C || !l.W_hat || !aligned(l.C, 4) || !aligned(l.W_hat, 4)) return KQ_ERR_ARG;
    if (l.idx ? !aligned(l.idx, 4) : (l.bits > 0 && (!l.packed || !aligned(l.packed, 4)))) return KQ_ERR_ARG;
    if (l.sq_error && (!l.W_ref || !aligned(l.sq_error, 8))) return KQ_ERR_ARG;
    if (l.W_ref && !aligned(l.W_ref, 4)) return KQ_ERR_ARG;
    return KQ_OK;
}

static size_t recon_ws_bytes(const kq_recon_layer* layers, int32_t n_layers) {
    size_t b = 0;
    for (int32_t l = 0; l < n_layers; ++l)
        if (layers[l].sq_error) b += align256(sizeof(double) * (size_t)recon_blocks(layers[l].n));
    return b;
}

size_t kq_reconstruct_stack_workspace_bytes(const kq_recon_layer* layers, int32_t n_layers) {
    if (layers == nullptr || n_layers < 1 || n_layers > KQ_MAX_STACK) return 0;
    for (int32_t l = 0; l < n_layers; ++l)
        if (check_recon_layer(layers[l]) != KQ_OK) return 0;
    return recon_ws_bytes(layers, n_layers);
}

kq_status kq_reconstruct_stack(const kq_recon_layer* layers, int32_t n_layers, void* ws, size_t ws_bytes,
                               void* stream) {
    if (layers == nullptr || n_layers < 1 || n_layers > KQ_MAX_STACK) return KQ_ERR_ARG;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_status st = check_recon_layer(layers[l]);
        if (st != KQ_OK) return st;
    }
    const size_t need = recon_ws_bytes(layers, n_layers);
    if (need > 0) {
        const kq_status w = check_ws(ws, ws_bytes, need);
        if (w != KQ_OK) return w;
    }
    ReconParams p;
    memset(&p, 0, sizeof(p));
    p.nlayers = n_layers;
    size_t off = 0;
    int blk = 0;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_recon_layer& s = layers[l];
        ReconLayer& d = p.L[l];
        d.idx = s.idx;
        d.packed = s.idx ? nullptr : s.packed;
        d.bits = s.idx ? 0 : s.bits;
        d.pbytes = (s.n * (long long)d.bits + 7) / 8;
        d.C = s.C;
        d.W = s.W_hat;
        d.W_ref = s.W_ref;
        d.n = (int)s.n;
        d.k = s.k;
        d.nblk = recon_blocks(s.n);
        if (s.sq_error) {
            d.part = (double*)((unsigned char*)ws + off);
            d.out = s.sq_error;
            off += align256(sizeof(double) * (size_t)d.nblk);
        }
        p.unit_begin[l] = blk;
        blk += d.nblk;
    }
    for (int32_t l = n_layers; l < KQ_MAX_STACK; ++l) p.unit_begin[l] = 0x7fffffff;
    p.total_blocks = blk;
    return hip_status(launch_reconstruct_stack(p, (hipStream_t)stream));
}

// ---- the whole compression pass of a stack (Sec. 3.1 fit, Sec. 3.2 codebook quantization,
// Eq. 4 index stream, test-time reconstruction) in one call ----------------------------------

static kq_status compress_layer_views(const kq_compress_layer& c, int32_t bits, kq_layer& fit, kq_cbq_layer& cbq,
                                      kq_pack_job (&jobs)[2], int& njobs, kq_recon_layer& rec) {
    fit = kq_layer{c.X, c.n, c.k, c.C, c.idx, nullptr, c.counts, c.distortion};
    cbq = kq_cbq_layer{c.C, c.k, c.counts, c.codes, c.levels, c.C_hat};
    const int32_t b = kq_index_bits(c.k);
    njobs = 0;
    if (c.packed_idx) jobs[njobs++] = kq_pack_job{c.idx, 4, b, c.n, c.packed_idx};
    if (c.packed_codes) jobs[njobs++] = kq_pack_job{c.codes, 1, bits, (int64_t)c.k * KQ_DIM, c.packed_codes};
    rec = kq_recon_layer{c.packed_idx ? nullptr : c.idx, c.packed_idx, b, c.k, c.n, c.C_hat, c.W_hat,
                         c.sq_error ? c.X : nullptr, c.sq_error};
    return KQ_OK;
}

static kq_status check_compress(const kq_compress_layer* layers, int32_t n_layers, int32_t iters, int32_t mode,
                                int32_t bits, int32_t cbq_iters, uint32_t flags) {
    if (layers == nullptr || n_layers < 1) return KQ_ERR_ARG;
    if (bits < 1 || bits > 8) return KQ_ERR_UNSUPPORTED;
    if (iters < 0 || cbq_iters < 0 || (mode != KQ_CBQ_WKMEANS && mode != KQ_CBQ_UNIFORM) ||
        (flags & ~KQ_F_VALIDATE) != 0)
        return KQ_ERR_ARG;
    for (int32_t l = 0; l < n_layers; ++l) {
        const kq_compress_layer& c = layers[l];
        if (!c.C_init || !aligned(c.C_init, 4) || !c.counts || !c.codes || !c.levels || !c.C_hat) return KQ_ERR_ARG;
        if (c.sq_error && !c.W_hat) return KQ_ERR_ARG;
        kq_layer fit;
        kq_cbq_layer cbq;
        kq_pack_job jobs[2];
        int njobs = 0;
        kq_recon_layer rec;
        compress_layer_views(c, bits, fit, cbq, jobs, njobs, rec);
        kq_status st = check_layers(&fit, 1, true);
        if (st != KQ_OK) return st;
        if ((st = check_cbq(cbq, bits, mode, cbq_iters)) != KQ_OK) return st;
        for (int q = 0; q < njobs; ++q)
            if ((st = check_pack_job(jobs[q])) != KQ_OK) return st;
        if (c.W_hat && (st = check_recon_layer(rec)) != KQ_OK) return st;
    }
    return KQ_OK;
}

// workspace regions: the fit of one chunk of up to KQ_MAX_STACK layers, the wide codebook
// quantizer, the reconstruction's error partials (chunks run one after another and share them)
struct CompressLayout {
    size_t fit, cbq, recon, total;
};

static CompressLayout compress_layout(const kq_compress_layer* layers, int32_t n_layers, int32_t bits) {
    CompressLayout L = {0, 0, 0, 0};
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        kq_layer fit[KQ_MAX_STACK];
        kq_cbq_layer cbq[KQ_MAX_STACK];
        kq_recon_layer rec[KQ_MAX_STACK];
        int nrec = 0;
        for (int32_t l = l0; l < l1; ++l) {
            kq_pack_job jobs[2];
            int njobs = 0;
            kq_recon_layer r;
            compress_layer_views(layers[l], bits, fit[l - l0], cbq[l - l0], jobs, njobs, r);
            if (layers[l].W_hat) rec[nrec++] = r;
        }
        const size_t f = stack_ws_bytes(fit, l1 - l0);
        const size_t c = kq_quantize_codebook_stack_workspace_bytes(cbq, l1 - l0, bits);
        const size_t r = nrec ? recon_ws_bytes(rec, nrec) : 0;
        L.fit = f > L.fit ? f : L.fit;
        L.cbq = align256(c) > L.cbq ? align256(c) : L.cbq;
        L.recon = align256(r) > L.recon ? align256(r) : L.recon;
    }
    L.total = L.fit + L.cbq + L.recon;
    return L;
}

size_t kq_compress_workspace_bytes(const kq_compress_layer* layers, int32_t n_layers, int32_t bits) {
    if (check_compress(layers, n_layers, 0, KQ_CBQ_WKMEANS, bits, 0, 0) != KQ_OK) return 0;
    return compress_layout(layers, n_layers, bits).total;
}

kq_status kq_compress_stack(const kq_compress_layer* layers, int32_t n_layers, int32_t iters, int32_t mode,
                            int32_t bits, int32_t cbq_iters, uint32_t flags, void* const* round_events, void* ws,
                            size_t ws_bytes, void* stream) {
    kq_status st = check_compress(layers, n_layers, iters, mode, bits, cbq_iters, flags);
    if (st != KQ_OK) return st;
    const CompressLayout L = compress_layout(layers, n_layers, bits);
    if ((st = check_ws(ws, ws_bytes, L.total)) != KQ_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    unsigned char* w = (unsigned char*)ws;
    kq_layer fit[KQ_MAX_STACK];
    const float* init[KQ_MAX_STACK];
    kq_cbq_layer cbq[KQ_MAX_STACK];
    kq_pack_job jobs[KQ_MAX_PACK_JOBS];
    kq_recon_layer rec[KQ_MAX_STACK];
    if (flags & KQ_F_VALIDATE) {  // every layer checked before any output is written
        for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
            const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
            for (int32_t l = l0; l < l1; ++l) {
                kq_pack_job j2[2];
                int nj = 0;
                kq_recon_layer r;
                compress_layer_views(layers[l], bits, fit[l - l0], cbq[l - l0], j2, nj, r);
            }
            if ((st = run_xmax(fit, 0, l1 - l0, w, s, true)) != KQ_OK) return st;
        }
    }
    for (int32_t l0 = 0; l0 < n_layers; l0 += KQ_MAX_STACK) {
        const int32_t l1 = (n_layers - l0 < KQ_MAX_STACK) ? n_layers : l0 + KQ_MAX_STACK;
        int njobs = 0, nrec = 0;
        for (int32_t l = l0; l < l1; ++l) {
            kq_pack_job j2[2];
            int nj = 0;
            kq_recon_layer r;
            compress_layer_views(layers[l], bits, fit[l - l0], cbq[l - l0], j2, nj, r);
            init[l - l0] = layers[l].C_init;
            for (int q = 0; q < nj; ++q) jobs[njobs++] = j2[q];
            if (layers[l].W_hat) rec[nrec++] = r;
        }
        if ((st = run_fit(fit, l1 - l0, iters, w, s, init, false, l0 == 0 ? round_events : nullptr)) != KQ_OK)
            return st;
        if ((st = kq_quantize_codebook_stack_ws(cbq, l1 - l0, bits, mode, cbq_iters, L.cbq ? w + L.fit : nullptr,
                                                L.cbq, stream)) != KQ_OK)
            return st;
        if (njobs > 0 && (st = kq_pack_bits_stack(jobs, njobs, stream)) != KQ_OK) return st;
        if (nrec > 0 && (st = kq_reconstruct_stack(rec, nrec, L.recon ? w + L.fit + L.cbq : nullptr, L.recon,
                                                   stream)) != KQ_OK)
            return st;
    }
    return KQ_OK;
}

// ---- host-only helpers ----------------------------------------------------------------------

int32_t kq_index_bits(int32_t k) {
    if (k < 1) return -1;
    int32_t b = 0;
    while ((int64_t(1) << b) < (int64_t)k) ++b;
    return b;
}

kq_status kq_accounting(int64_t n, int32_t k, int32_t dim, int32_t bc, int64_t* storage_bits, double* ratio,
                        double* bits_per_param) {
    if (n < 1 || k < 1 || dim < 1 || bc < 1 || bc > 64) return KQ_ERR_ARG;
    const int64_t B = (int64_t)k * dim * bc + n * kq_index_bits(k);  // Eq. (4)
    const double params = (double)n * (double)dim;
    if (storage_bits) *storage_bits = B;
    if (ratio) *ratio = params * 32.0 / (double)B;  // Eq. (6), fp32 weights
    if (bits_per_param) *bits_per_param = (double)B / params;  // Eq. (7)
    return KQ_OK;
}

// splitmix64: the state advances by the golden-ratio increment and each output is the
// state through the variant-13 mixer (Steele, Lea and Flood, OOPSLA 2014)
static uint64_t splitmix64_next(uint64_t& state) {
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

namespace {
struct KernelKey {
    uint32_t v[KQ_DIM];
    bool operator==(const KernelKey& o) const { return memcmp(v, o.v, sizeof(v)) == 0; }
};
struct KernelKeyHash {
    size_t operator()(const KernelKey& k) const {
        uint64_t h = 0x243F6A8885A308D3ull;
        for (int d = 0; d < KQ_DIM; ++d) h = (h ^ k.v[d]) * 0x100000001B3ull;
        return (size_t)(h ^ (h >> 29));
    }
};
}  // namespace

kq_status kq_forgy_select(const float* X, int64_t n, int32_t dim, int32_t k, uint64_t seed, int64_t* sel) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || k > n || !X || !sel) return KQ_ERR_ARG;
    std::unordered_map<int64_t, int64_t> moved;  // positions of the permutation that a swap changed
    std::unordered_set<KernelKey, KernelKeyHash> seen;
    std::vector<int64_t> out;
    out.reserve((size_t)k);
    uint64_t state = seed;
    for (int64_t i = 0; i < n && (int32_t)out.size() < k; ++i) {
        const int64_t j = i + (int64_t)(splitmix64_next(state) % (uint64_t)(n - i));
        const auto pi = moved.find(i), pj = moved.find(j);
        const int64_t vi = pi == moved.end() ? i : pi->second;
        const int64_t vj = pj == moved.end() ? j : pj->second;
        moved[j] = vi;  // swap positions i and j; position i is final from here on
        const int64_t cand = vj;
        KernelKey key;
        memcpy(key.v, X + cand * KQ_DIM, sizeof(key.v));
        for (int d = 0; d < KQ_DIM; ++d)
            if (key.v[d] == 0x80000000u) key.v[d] = 0u;  // -0 and +0 are the same kernel value
        if (seen.insert(key).second) out.push_back(cand);
    }
    if ((int32_t)out.size() < k) return KQ_ERR_ARG;  // fewer than k distinct kernels
    memcpy(sel, out.data(), sizeof(int64_t) * (size_t)k);
    return KQ_OK;
}

size_t kq_fit_layer_noalloc_max_bytes(void) { return (size_t)KQ_NOALLOC_SCRATCH_BYTES; }

kq_status kq_fit_layer_noalloc(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init, int32_t iters,
                               float* C, int32_t* idx, int32_t* counts, double* distortion, uint32_t flags,
                               void* stream) {
    if (dim != KQ_DIM) return KQ_ERR_UNSUPPORTED;
    if (k > KQ_MAX_K) return KQ_ERR_UNSUPPORTED;
    if (!valid_n(n) || !valid_k(k) || k > n || iters < 0 || (flags & ~KQ_F_VALIDATE) != 0) return KQ_ERR_ARG;
    if (!C_init || !aligned(C_init, 4)) return KQ_ERR_ARG;
    const kq_layer l = {X, n, k, C, idx, nullptr, counts, distortion};
    kq_status st = check_layers(&l, 1, true);
    if (st != KQ_OK) return st;
    if (layer_ws_bytes(n, k) > (size_t)KQ_NOALLOC_SCRATCH_BYTES) return KQ_ERR_WORKSPACE;  // beyond the static scratch
    unsigned char* ws = nullptr;
    if ((st = scratch_for_current_device(&ws)) != KQ_OK) return st;
    const float* init[1] = {C_init};
    return run_fit(&l, 1, iters, ws, (hipStream_t)stream, init, (flags & KQ_F_VALIDATE) != 0);
}

}  // extern "C"
