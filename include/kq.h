/*
 * kq.h -- C ABI of the MI355X (gfx950) library for the hot path of Kernel
 * Quantization (Yu, Shi, Huang, Yu: "Kernel Quantization for Efficient Network
 * Compression").
 *
 * The operations:
 *   kq_assign            Sec. 3.1, Eq. (1): nearest codebook entry of every 3x3 kernel.
 *   kq_update            Sec. 3.1, Eq. (1): every entry becomes the mean of its kernel set S_i.
 *   kq_fit_layer         Sec. 3.1: Lloyd k-means on one layer (the "k-means in Eq. (1)"
 *                        step of Algorithm 1), a fixed number of rounds then a final assignment.
 *   kq_fit_stack         the same for many layers at once (Sec. 3.1 quantizes layer by layer;
 *                        layers are independent, so one launch serves all of them).
 *   kq_search_codebook_size Alg. 1: binary search of the codebook size, on the k-means
 *                        distortion instead of validation accuracy (a flagged deviation).
 *   kq_fit_layer_yinyang Sec. 4.1: the same fit with Yinyang assignments (kq_yinyang_init,
 *                        kq_yinyang_assign), equal to kq_fit_layer bit for bit.
 *   kq_codebook_grad_step Sec. 3.1, Eq. (2): retraining step of the codebook with the mean
 *                        gradient of each entry's kernels.
 *   kq_quantize_codebook Sec. 3.2: 6-bit quantization of all scalars of a layer's codebook,
 *                        k-means weighted by how often each entry is used.
 *   kq_quantize_scalars  end of Sec. 3.2: the same k-means quantization on the scalars of a
 *                        fully-connected layer (any size).
 *   kq_pack_bits         Eq. (4): the n * ceil(log2 k)-bit index stream.
 *   kq_reconstruct       end of Sec. 3.2: recover the weight tensor from codebook + indices.
 *   kq_compress_stack    all of the above for the layers of a network in one call.
 *   kq_forgy_select      the k-means initialisation (k distinct kernels in a seeded order).
 *   kq_accounting        Eq. (4), (6), (7): storage bits, compression ratio, bits per parameter.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - dim is omega^2 and must be 9 (the paper quantizes 3x3 kernels only, Sec. 4.1);
 *    anything else returns KQ_ERR_UNSUPPORTED.
 *  - Kernels X are n rows of 9 fp32 values, row-major; for an OIHW weight tensor
 *    this is the tensor itself (kernel i = o * C_in + c).  Codebooks C are k rows of 9.
 *  - Pointers named device are device memory (hipMalloc / torch.cuda); pointers named
 *    host are host memory.  Every buffer belongs to the caller.  The library never
 *    allocates device memory and keeps no global state (kq_forgy_select, a host-only
 *    helper, uses host memory while it runs).
 *  - stream is a hipStream_t (NULL = the null stream).  Device calls only enqueue work
 *    on that stream and return; outputs are valid once the stream has been synchronised.
 *  - Arguments are checked on the host before anything is enqueued.  On an error
 *    nothing is enqueued and outputs are untouched.  No HIP call is made before the
 *    checks pass, so argument errors are reported without a GPU.
 *  - KQ_ERR_HIP: a HIP launch failed; outputs are unspecified.
 *  - workspace: device scratch of at least the size the matching *_workspace_bytes
 *    query returns, 256-byte aligned.  Its contents need no initialisation: every
 *    call writes what it later reads.  Calls that share a workspace must be ordered on one
 *    stream (concurrent calls on one workspace race).
 *  - The member sums of the update are exact 64-bit fixed-point sums at a per-layer scale
 *    taken from the layer's largest magnitude (see kq_update), so any finite kernel values
 *    are supported.  Non-finite values make the sums meaningless: calls that form sums accept
 *    KQ_F_VALIDATE, which checks every value first (one pass over the kernels, then a wait
 *    for the result) and returns KQ_ERR_RANGE, with no output written, if any is NaN or
 *    infinite.  Without the flag such inputs give unspecified codebooks (no fault).
 */
#ifndef KQ_H
#define KQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kq_status {
    KQ_OK = 0,
    KQ_ERR_ARG = 1,          /* null pointer, bad size, misaligned pointer */
    KQ_ERR_UNSUPPORTED = 2,  /* dim != 9, k above KQ_MAX_K, bits outside 1..16 */
    KQ_ERR_WORKSPACE = 3,    /* workspace missing, too small or misaligned */
    KQ_ERR_RANGE = 4,        /* KQ_F_VALIDATE: a kernel (or gradient) value is NaN or infinite */
    KQ_ERR_HIP = 5           /* a HIP runtime call failed */
} kq_status;

#define KQ_DIM 9
#define KQ_MAX_K 65536
#define KQ_MAX_STACK 16      /* layers per launch; longer stacks are split by the library */

/* codebook-quantization modes (Sec. 3.2) */
#define KQ_CBQ_WKMEANS 0     /* weighted k-means over the codebook scalars (the paper's method) */
#define KQ_CBQ_UNIFORM 1     /* the uniform grid that initialises it, without iterations */

/* workspace queries: op codes */
#define KQ_OP_ASSIGN 0
#define KQ_OP_UPDATE 1
#define KQ_OP_FIT 2
#define KQ_OP_SQ_ERROR 3     /* n = element count, k = 1 */
#define KQ_OP_GRAD 4         /* kq_codebook_grad_step */

/* flags */
#define KQ_F_COUNTS_ONLY 1u  /* kq_update / kq_update_stack: write counts only, leave C untouched */
#define KQ_F_DISTORTION_FROM_ASSIGN 2u
                             /* kq_update_stack: take the distortion from the partial sums the
                                preceding kq_assign_stack on the same layers and workspace left
                                (no second pass over the old codebook) */
#define KQ_F_FUSED_SUMS 4u   /* kq_assign_stack: also accumulate the member sums of the new
                                assignment (every k <= 256, else KQ_ERR_UNSUPPORTED) */
#define KQ_F_EXACT_SEARCH 16u /* kq_quantize_scalars: every code by the exact fp64 search (reference) */
#define KQ_F_THRESHOLDS 32u  /* kq_quantize_scalars: codes from level thresholds at any size, wherever
                                they are valid (by default only from 3 * 2^20 scalars on) */
#define KQ_F_VALIDATE 64u    /* kq_update, kq_update_stack, kq_assign_stack, kq_fit_layer,
                                kq_fit_stack, kq_compress_stack: check that every kernel value
                                is finite before anything is written; KQ_ERR_RANGE otherwise.
                                The call then waits on the stream for the check. */
#define KQ_F_REUSE_SHIFTS 128u /* kq_assign_stack (with KQ_F_FUSED_SUMS), kq_update_stack: the
                                layers' fixed-point shifts are those the preceding stack call on
                                the same layers and workspace found (a fused assignment, or an
                                update without this flag); the kernels must not have changed
                                since.  Saves the pass over the kernels that finds them. */
#define KQ_F_SUMS_FROM_ASSIGN 8u
                             /* kq_update_stack: finish the update from the sums the preceding
                                kq_assign_stack with KQ_F_FUSED_SUMS left (same layers and
                                workspace): the kernels are not read again; the distortion is
                                the assignment's, as with KQ_F_DISTORTION_FROM_ASSIGN */

/* One layer of a stack.  All pointers are device pointers. */
typedef struct kq_layer {
    const float* X;      /* [n][9] kernels */
    int64_t n;           /* number of kernels, 1 <= n < 2^31 */
    int32_t k;           /* codebook size, 1 <= k <= min(n, KQ_MAX_K) for fits */
    float* C;            /* [k][9] codebook: state in, new state out */
    int32_t* idx;        /* [n] index of the nearest entry */
    float* best_d;       /* [n] fp32 squared distance to that entry, or NULL */
    int32_t* counts;     /* [k] kernels per entry (final assignment), or NULL for assign */
    double* distortion;  /* distortion output(s), or NULL (see each call) */
} kq_layer;

/* Human-readable name of a status code (static string). */
const char* kq_status_string(kq_status s);

/* Library ABI version (incremented when a signature changes). */
int32_t kq_abi_version(void);

/*
 * Workspace bytes for one layer of n kernels of dim values and k entries for op (KQ_OP_*;
 * KQ_OP_SQ_ERROR: n values, k = 1, dim = 1).  Returns 0 for invalid or unsupported sizes.
 */
size_t kq_workspace_bytes(int32_t op, int64_t n, int32_t k, int32_t dim);

/* Workspace bytes for a stack call (kq_assign_stack / kq_update_stack / kq_fit_stack). */
size_t kq_stack_workspace_bytes(const kq_layer* layers /* host [n_layers] */, int32_t n_layers);

/* Zero-fill `bytes` of device workspace on `stream` (a fill kernel, no memset node). */
kq_status kq_workspace_init(void* ws, size_t bytes, void* stream);

/*
 * kq_assign -- Sec. 3.1, Eq. (1), the assignment half of a Lloyd round.
 *
 *   idx[i]    = the entry j minimising the fp32 squared distance
 *               d(x_i, c_j) = sum_d (x_id - c_jd)^2, evaluated term by term in
 *               dimension order as t = x - c, acc = fma(t, t, acc); ties go to the
 *               lowest j.  The result is exactly this argmin.  (Internally the
 *               distances are screened with matrix-core dot products and every
 *               kernel whose winner could be in doubt is rescored in that form.)
 *   best_d[i] = that fp32 distance (device [n], may be NULL).
 *   *distortion = sum_i best_d[i] in fp64 in a fixed order (device scalar, may be NULL).
 *
 *   X device [n][9] fp32, 4-byte aligned; C device [k][9] fp32; idx device [n] int32.
 *   1 <= n < 2^31, 1 <= k <= KQ_MAX_K (k > n is allowed).
 */
kq_status kq_assign(const float* X, int64_t n, int32_t dim, const float* C, int32_t k,
                    int32_t* idx, float* best_d, double* distortion, uint32_t flags,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * kq_update -- Sec. 3.1, Eq. (1), the update half of a Lloyd round.
 *
 *   counts[j] = |S_j| = #{i : idx[i] == j}
 *   C_new[j]  = mean of the kernels in S_j, or C_old[j] when S_j is empty.
 *   The member sums are exact integer sums of q(x) = rint(x * 2^s) with
 *   s = 62 - ceil(log2 n) - e, e the smallest integer with max_i |x_i| < 2^e (-126 if that
 *   maximum is subnormal; a first pass over X finds it), so no sum can overflow and the resolution is
 *   2^-(62 - ceil(log2 n)) of the largest magnitude at any scale of the weights; the sums
 *   do not depend on summation order, and the mean is fp32( (double(sum) * 2^-s) / |S_j| ).
 *
 *   *distortion = the Eq. (1) objective of the given assignment against C_old:
 *               sum_i d(x_i, C_old[idx[i]]) with d the fp32 distance of kq_assign,
 *               summed in fp64 in a fixed order (device scalar, may be NULL).
 *
 *   X device [n][9]; idx device [n] values in [0, k) (out-of-range indices are
 *   ignored); C_old, C_new device [k][9] (may alias); counts device [k] or NULL.
 *   flags: KQ_F_COUNTS_ONLY to compute only the counts (C_new untouched); KQ_F_VALIDATE.
 */
kq_status kq_update(const float* X, int64_t n, int32_t dim, const int32_t* idx, int32_t k,
                    const float* C_old, float* C_new, int32_t* counts, double* distortion,
                    uint32_t flags, void* ws, size_t ws_bytes, void* stream);

/*
 * kq_fit_layer -- Lloyd k-means on one layer (Sec. 3.1, Eq. 1).
 *
 *   C := C_init; repeat iters times { idx := assign(C); C := update(idx, C) };
 *   then a final idx := assign(C).
 *   C [k][9] ends as the codebook after `iters` updates, idx [n] the final
 *   assignment, counts [k] (may be NULL) its member counts, distortion
 *   device [iters+1] (may be NULL) the distortion of every assignment.
 *   Requires 1 <= k <= n.  C_init may equal C (it is only read).  flags: 0 or KQ_F_VALIDATE.
 */
kq_status kq_fit_layer(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init,
                       int32_t iters, float* C, int32_t* idx, int32_t* counts, double* distortion,
                       uint32_t flags, void* ws, size_t ws_bytes, void* stream);

/*
 * kq_codebook_grad_step -- Sec. 3.1, Eq. (2): one retraining step of the kernel codebook.
 *
 *   Every entry moves against the elementwise mean of the gradients of the kernels mapped
 *   to it:  c_i := c_i - gamma * (sum over m in S_i of dL/dm) / z_i,  z_i = |S_i|.
 *   G [n][9] holds dL/dm for every kernel (the gradient of the loss with respect to the
 *   weight tensor, OIHW, evaluated at the reconstructed weights), idx [n] the kernels'
 *   entries.  An entry with no kernels keeps its value; indices outside [0, k) are ignored.
 *   The sums are exact 64-bit fixed-point sums at a per-layer scale set from max |g| (any
 *   finite gradient magnitude, independent of the order of the work); the mean is
 *   fp64(sum) / z and c - gamma * mean is evaluated in fp64 and rounded once to fp32.
 *   counts [k] (may be NULL) receives z.  C_old and C_new may alias (in-place step).
 *   G, C_old, C_new device [.][9] fp32; idx device [n]; gamma finite (else KQ_ERR_ARG).
 *   workspace: kq_workspace_bytes(KQ_OP_GRAD, n, k, 9).
 *   kq_codebook_grad_step_stack: the same for every layer of a stack in one launch set;
 *   layers[l].X holds the layer's gradients and layers[l].C is stepped in place
 *   (workspace: kq_stack_workspace_bytes).
 */
kq_status kq_codebook_grad_step(const float* G, int64_t n, int32_t dim, const int32_t* idx, int32_t k,
                                const float* C_old, float gamma, float* C_new, int32_t* counts, void* ws,
                                size_t ws_bytes, void* stream);
kq_status kq_codebook_grad_step_stack(const kq_layer* layers, int32_t n_layers, float gamma, void* ws,
                                      size_t ws_bytes, void* stream);

/*
 * kq_quantize_scalars -- end of Sec. 3.2: the 6-bit quantization of a fully-connected
 * layer by the k-means the codebooks are quantized with, i.e. the algorithm of
 * kq_quantize_codebook (KQ_CBQ_WKMEANS) on one flat set of `count` scalars, every weight 1,
 * for sets far larger than a codebook (a VGG-16 fc6 weight has 102,760,448 scalars).
 *
 *   Grid on [min, max], codes = nearest level (smallest index on ties), then up to
 *   `iters` rounds of: level q = fp32(exact sum of its scalars rounded once to fp64 /
 *   their count) (kept when empty), recompute the codes; stop early after a round that
 *   changes no code.  iters = 0 gives the uniform grid alone.  The sums are exact, so the
 *   result is a pure function of v: bit for bit that of kq_quantize_codebook on the same
 *   scalars with unit weights.
 *   With sorted levels the code of a value never decreases as the value grows, so from
 *   3 * 2^20 scalars on each round first finds, per level boundary, the smallest value that
 *   takes the next code (a search over fp32 values with the exact search, started at the
 *   midpoint of the two levels) and then codes
 *   every scalar with fp32 comparisons only.  This is used only where every fp64 distance
 *   between a data value and a level is exact (no nonzero value or level below 2^-29 of the
 *   largest magnitude), so it gives the exact search's codes; KQ_F_EXACT_SEARCH /
 *   KQ_F_THRESHOLDS force one way (flags 0 = the size rule).
 *   v device [count] fp32 (finite); codes device [count] uint8; levels device [2^bits] fp32;
 *   v_hat device [count] (= levels[codes], may be NULL); rounds device int32 (level updates
 *   made, may be NULL).  1 <= count < 2^31; bits 1..8 (else KQ_ERR_UNSUPPORTED).
 *   workspace: kq_quantize_scalars_workspace_bytes(count, bits).
 */
size_t kq_quantize_scalars_workspace_bytes(int64_t count, int32_t bits);
kq_status kq_quantize_scalars(const float* v, int64_t count, int32_t bits, int32_t iters, uint8_t* codes,
                              float* levels, float* v_hat, int32_t* rounds, uint32_t flags, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * kq_search_codebook_size -- the codebook-size binary search of Sec. 3.1 (Algorithm 1,
 * Eq. 3), driven by the k-means distortion J (Eq. 1, the final assignment of each fit)
 * in place of the validation accuracy.  This is a deviation from the paper, which needs a
 * trained network and its validation set: here the "accuracy" of a codebook size is -J,
 * and the unquantized layer's is 0 (no error), so the target of Eq. (3),
 * A_target = A_base - (A_ori - A_base) r, becomes J_target = (1 + r) J(n_init).
 *
 *   Fit k = n_init (lloyd_iters rounds, kq_fit_layer); B_upper = n_init, B_lower = 0; then
 *   up to max_iter times: N = floor((B_upper + B_lower) / 2), stop if N is a bound; fit k = N;
 *   J(N) < J_target ? B_upper = N : B_lower = N.  The answer is B_upper.
 *   Every fit of size k starts from the first k rows of C_cand (the caller's order of
 *   candidate entries, e.g. seeded distinct kernels), so the trials are nested.
 *   X device [n][9]; C_cand device [n_init][9]; C device [n_init][9] receives the chosen
 *   fit's codebook in its first *k_out rows, idx device [n] its assignment; k_out host;
 *   trial_k, trial_d host [max_iter] or NULL: each iteration's N and J(N) (0 after an early
 *   stop); d_init host or NULL: J(n_init).  1 <= n_init <= n; r >= 0 finite; synchronous
 *   (it waits for every fit to read J); workspace: kq_search_workspace_bytes.
 */
size_t kq_search_workspace_bytes(int64_t n, int32_t n_init, int32_t lloyd_iters);
kq_status kq_search_codebook_size(const float* X, int64_t n, int32_t dim, const float* C_cand, int32_t n_init,
                                  float r, int32_t max_iter, int32_t lloyd_iters, float* C, int32_t* idx,
                                  int32_t* k_out, int32_t* trial_k, double* trial_d, double* d_init, void* ws,
                                  size_t ws_bytes, void* stream);

/*
 * Yinyang assignment -- Sec. 4.1: the paper runs its kernel-level k-means with Yinyang
 * k-means, which skips distance evaluations using triangle-inequality bounds and
 * reaches the same result as plain Lloyd.  These calls return exactly what kq_assign
 * returns for the same codebook (the fp32 argmin, ties to the lowest index; bit for bit,
 * including best_d and the distortion), doing less work once the codebook moves little.
 *
 *   The codebook's entries are split into `groups` groups (groups <= 0: about one per
 *   64 entries, at most 32; otherwise 1 .. min(64, k)) by a few Lloyd rounds on the
 *   entries.  For every kernel and group the workspace keeps a lower bound of the
 *   kernel's Euclidean distance to the group's entries, shifted by the group's
 *   cumulative movement.  A round moves every group's bounds down by the largest
 *   movement of its entries, skips the groups whose bound exceeds the distance to the
 *   kernel's current entry (with a margin that covers fp32 rounding), and scans the other
 *   groups' entries exactly.  The grouping decides only how much is skipped.
 *
 *   kq_yinyang_init:   assigns X against C exactly as kq_assign (idx, best_d, distortion:
 *                      each may be NULL except idx), groups C and sets the bounds.
 *   kq_yinyang_assign: the next assignment after the codebook moved from C_prev (the
 *                      codebook of the previous init/assign call on this workspace) to C.
 *                      idx must hold that call's assignment; it is replaced by the new one.
 *                      stats (device int64 [3] or NULL): kernels whose groups were scanned,
 *                      (kernel, group) pairs scanned, distances evaluated in those scans.
 *   kq_fit_layer_yinyang: kq_fit_layer with Yinyang assignments; C, idx, counts and
 *                      distortion [iters+1] equal kq_fit_layer's bit for bit.  stats
 *                      (device int64 [iters][3] or NULL): the scan counts of rounds 1..iters.
 *   X device [n][9]; C, C_prev, C_init device [k][9]; idx device [n]; best_d device [n];
 *   counts device [k].  Requires 1 <= k <= n.  Kernel and codebook values must be finite
 *   (the grouping and the fit run kq_update's fixed-point sums).
 *   workspace: kq_yinyang_workspace_bytes(n, k, groups) bytes (about 20 bytes per kernel
 *   and group plus kq_workspace_bytes); it carries the state from one call to the next,
 *   so the calls of one fit must use one workspace, in order, on one stream.
 */
size_t kq_yinyang_workspace_bytes(int64_t n, int32_t k, int32_t groups);
kq_status kq_yinyang_init(const float* X, int64_t n, int32_t dim, const float* C, int32_t k, int32_t groups,
                          int32_t* idx, float* best_d, double* distortion, void* ws, size_t ws_bytes,
                          void* stream);
kq_status kq_yinyang_assign(const float* X, int64_t n, int32_t dim, const float* C_prev, const float* C,
                            int32_t k, int32_t groups, int32_t* idx, float* best_d, double* distortion,
                            int64_t* stats, void* ws, size_t ws_bytes, void* stream);
kq_status kq_fit_layer_yinyang(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init,
                               int32_t iters, int32_t groups, float* C, int32_t* idx, int32_t* counts,
                               double* distortion, int64_t* stats, void* ws, size_t ws_bytes, void* stream);

/*
 * Stack versions: one launch per step for up to KQ_MAX_STACK layers (more are split).
 *   kq_assign_stack: assigns every layer against its C; writes idx, best_d (if set) and
 *                    distortion[dist_slot] (if distortion is set).
 *   kq_update_stack: updates every C in place from its idx; writes counts (if set) and
 *                    the distortion of idx against the old C into distortion[dist_slot]
 *                    (with KQ_F_DISTORTION_FROM_ASSIGN, the value the preceding
 *                    kq_assign_stack computed, which is the same objective).
 *   kq_fit_stack:    kq_fit_layer on every layer (C in place, distortion [iters+1]).
 *   layers is a host array; the pointers in it are device pointers.
 *   With every k <= 256, the fits (and kq_assign_stack with KQ_F_FUSED_SUMS followed by
 *   kq_update_stack with KQ_F_SUMS_FROM_ASSIGN) add the member sums inside the assignment
 *   and skip the update's second read of the kernels; the sums are the same integers, so
 *   every output is the same bit for bit.
 */
kq_status kq_assign_stack(const kq_layer* layers, int32_t n_layers, int32_t dist_slot, uint32_t flags,
                          void* ws, size_t ws_bytes, void* stream);
kq_status kq_update_stack(const kq_layer* layers, int32_t n_layers, int32_t dist_slot, uint32_t flags,
                          void* ws, size_t ws_bytes, void* stream);
kq_status kq_fit_stack(const kq_layer* layers, int32_t n_layers, int32_t iters, uint32_t flags,
                       void* ws, size_t ws_bytes, void* stream);

/*
 * kq_quantize_codebook -- Sec. 3.2, 6-bit quantization of one layer's codebook.
 *
 *   The k*9 scalars v_r (r = 9 j + d) are coded with 2^bits fp32 levels.
 *   Grid: lo = min v, hi = max v, delta = (hi - lo) / (2^bits - 1) in fp64,
 *         L_q = fp32(lo + q * delta) (fp64 multiply, fp64 add).
 *   code_r = the smallest q minimising |v_r - L_q| (fp64).
 *   KQ_CBQ_UNIFORM stops there.  KQ_CBQ_WKMEANS then runs up to `iters` rounds of
 *   weighted 1-D Lloyd, scalar r carrying weight weights[r / 9] (the appearance
 *   count of its entry; NULL = every weight 1):
 *     W_q = sum of weights coded q, N_q = exact sum of weight * value over them
 *     rounded once to fp64, L_q = fp32(N_q / W_q) if W_q > 0 (else kept);
 *     recompute the codes; stop early when no code changes.
 *   Every step is exact or correctly rounded, so the result does not depend on
 *   the order of the work.
 *
 *   C device [k][9]; weights device [k] int32 >= 0 or NULL; codes device [k*9] uint8;
 *   levels device [2^bits] fp32; C_hat device [k][9] (= levels[codes], may be NULL).
 *   1 <= bits <= 8 here; 1 <= k <= KQ_MAX_K.
 */
kq_status kq_quantize_codebook(const float* C, int32_t k, int32_t dim, const int32_t* weights,
                               int32_t bits, int32_t mode, int32_t iters, uint8_t* codes,
                               float* levels, float* C_hat, void* stream);

/* One layer for kq_quantize_codebook_stack (device pointers). */
typedef struct kq_cbq_layer {
    const float* C;          /* [k][9] */
    int32_t k;
    const int32_t* weights;  /* [k] or NULL */
    uint8_t* codes;          /* [k*9] */
    float* levels;           /* [2^bits] */
    float* C_hat;            /* [k][9] or NULL */
} kq_cbq_layer;

/* kq_quantize_codebook on every layer of a host array, one workgroup per layer. */
kq_status kq_quantize_codebook_stack(const kq_cbq_layer* layers, int32_t n_layers, int32_t bits,
                                     int32_t mode, int32_t iters, void* stream);

/*
 * kq_quantize_codebook_stack_ws -- the same results (Sec. 3.2, bit for bit) with large
 *   codebooks spread over the whole GPU.  In KQ_CBQ_WKMEANS mode every codebook of at least
 *   16384 scalars (k >= 1821) runs the kq_quantize_scalars machinery with the entry counts
 *   as integer weights (each of an entry's 9 scalars weighs its count; weights <= 0 add
 *   nothing), one such codebook after another; the smaller ones (and every codebook of a
 *   KQ_CBQ_UNIFORM call) take one workgroup each as in kq_quantize_codebook_stack.
 *   ws/ws_bytes: device workspace of at least
 *   kq_quantize_codebook_stack_workspace_bytes(layers, n_layers, bits) bytes (256-byte
 *   aligned; contents need no initialisation; NULL allowed when that size is 0 or the mode
 *   is KQ_CBQ_UNIFORM), else KQ_ERR_WORKSPACE.  Other errors as kq_quantize_codebook.
 */
size_t kq_quantize_codebook_stack_workspace_bytes(const kq_cbq_layer* layers, int32_t n_layers, int32_t bits);
kq_status kq_quantize_codebook_stack_ws(const kq_cbq_layer* layers, int32_t n_layers, int32_t bits,
                                        int32_t mode, int32_t iters, void* ws, size_t ws_bytes, void* stream);

/*
 * kq_pack_bits -- the index stream of Eq. (4).
 *   Value i (its low `bits` bits) occupies stream bits [i*bits, (i+1)*bits), least
 *   significant bit first; stream bit s is bit (s % 8) of byte s / 8.  Writes exactly
 *   ceil(count * bits / 8) bytes; unused high bits of the last byte are zero.
 *   values device [count], elem_bytes 1 (uint8), 2 (uint16) or 4 (int32);
 *   out device, 4-byte aligned.  0 <= bits <= 16 (bits = 0 writes nothing).
 */
kq_status kq_pack_bits(const void* values, int32_t elem_bytes, int64_t count, int32_t bits,
                       uint8_t* out, void* stream);

/* Inverse of kq_pack_bits: values device [count] int32. */
kq_status kq_unpack_bits(const uint8_t* in, int64_t count, int32_t bits, int32_t* values, void* stream);

/*
 * kq_reconstruct -- end of Sec. 3.2: W_hat[i][d] = C[idx[i]][d].
 *   Pass the 6-bit dequantised codebook (C_hat of kq_quantize_codebook) for K+C.
 *   idx device [n] values in [0, k) (others give zeros); C device [k][9];
 *   W_hat device [n][9]; every pointer 4-byte aligned.
 */
kq_status kq_reconstruct(const int32_t* idx, int64_t n, const float* C, int32_t k, int32_t dim,
                         float* W_hat, void* stream);

/*
 * kq_reconstruct_packed -- the same from the stored form: indices read from a
 * kq_pack_bits stream of `bits` = ceil(log2 k) bits each (packed device, 4-byte aligned,
 * ceil(n * bits / 8) bytes; nothing past its end is read).
 */
kq_status kq_reconstruct_packed(const uint8_t* packed, int32_t bits, int64_t n, const float* C,
                                int32_t k, int32_t dim, float* W_hat, void* stream);

/*
 * kq_sq_error -- the l2 reconstruction error the paper reports (Sec. 4.2.1):
 *   *out = sum_i (double(A[i]) - double(B[i]))^2 over `count` fp32 values, in fp64,
 *   in a fixed order (the same bits on every run).
 *   A, B device [count] fp32, 4-byte aligned; out device fp64 scalar;
 *   workspace of kq_workspace_bytes(KQ_OP_SQ_ERROR, count, 1, 1) bytes.
 */
kq_status kq_sq_error(const float* A, const float* B, int64_t count, double* out,
                      void* ws, size_t ws_bytes, void* stream);

/*
 * Stack forms of the storage and recovery steps, for the layers of a network at once
 * (Eq. 4 and the end of Sec. 3.2); each runs as one launch (plus one small finishing
 * launch for the errors) instead of one or two per layer.
 */

/* One stream of kq_pack_bits_stack (device pointers); fields as in kq_pack_bits. */
typedef struct kq_pack_job {
    const void* values;   /* [count] */
    int32_t elem_bytes;   /* 1, 2 or 4 */
    int32_t bits;         /* 0..16 */
    int64_t count;        /* >= 0 */
    uint8_t* out;         /* ceil(count * bits / 8) bytes, 4-byte aligned */
} kq_pack_job;
#define KQ_MAX_PACK_JOBS 32

/* kq_pack_bits on every job of a host array (1 <= n_jobs <= KQ_MAX_PACK_JOBS); each
 * stream is bit-identical to what kq_pack_bits writes. */
kq_status kq_pack_bits_stack(const kq_pack_job* jobs, int32_t n_jobs, void* stream);

/* One layer of kq_reconstruct_stack (device pointers). */
typedef struct kq_recon_layer {
    const int32_t* idx;      /* [n] indices, or NULL to read them from `packed` */
    const uint8_t* packed;   /* kq_pack_bits stream of `bits`-bit indices (when idx is NULL), 4-byte aligned */
    int32_t bits;            /* 0..16, used with `packed` */
    int32_t k;               /* 1..KQ_MAX_K; indices outside [0, k) give zero rows */
    int64_t n;               /* 1 <= n < 2^31 */
    const float* C;          /* [k][9] codebook (the 6-bit C_hat for K+C) */
    float* W_hat;            /* [n][9] output */
    const float* W_ref;      /* [n][9] original kernels, or NULL */
    double* sq_error;        /* device scalar, or NULL: sum over the 9n values of
                                (W_ref - W_hat)^2 in fp64, in a fixed order (the same bits on
                                every run; needs W_ref) */
} kq_recon_layer;

/* Workspace bytes of kq_reconstruct_stack (0 for invalid sizes). */
size_t kq_reconstruct_stack_workspace_bytes(const kq_recon_layer* layers /* host */, int32_t n_layers);

/* kq_reconstruct / kq_reconstruct_packed (and the squared error of each layer) for
 * every layer of a host array, 1 <= n_layers <= KQ_MAX_STACK; all pointers 4-byte aligned. */
kq_status kq_reconstruct_stack(const kq_recon_layer* layers, int32_t n_layers, void* ws, size_t ws_bytes,
                               void* stream);

/*
 * kq_compress_stack -- the whole compression pass of Sec. 3 for the layers of a network, in
 * one call (one stream-ordered sequence of launches; nothing waits on the host unless
 * KQ_F_VALIDATE is set):
 *   1. Sec. 3.1, Eq. (1): `iters` Lloyd rounds from C_init and a final assignment
 *      (kq_fit_stack): C, idx, counts, distortion [iters + 1];
 *   2. Sec. 3.2: quantization of every codebook to 2^bits levels with the entry counts as
 *      weights (kq_quantize_codebook_stack_ws, `mode`, `cbq_iters` rounds): codes, levels,
 *      C_hat;
 *   3. Eq. (4): the ceil(log2 k)-bit index stream and the `bits`-bit code stream
 *      (kq_pack_bits; each optional);
 *   4. end of Sec. 3.2: W_hat = C_hat[idx] from the packed stream when there is one
 *      (kq_reconstruct_stack; optional), and the squared error of W_hat against X.
 *   Every output is bit for bit what the separate calls give.
 *   All pointers are device pointers; C_init is only read (it may equal C).  1 <= k <= n;
 *   1 <= bits <= 8; n_layers >= 1 (processed KQ_MAX_STACK layers at a time).
 *   flags: 0 or KQ_F_VALIDATE.  workspace: kq_compress_workspace_bytes(layers, n_layers, bits).
 *   round_events: NULL, or a host array of 2 * (iters + 1) hipEvent_t handles created by the
 *   caller, any of them NULL: entries 2t and 2t + 1 take the start and the end time of the
 *   assignment kernel of Lloyd round t (t = iters: the final assignment) of the first
 *   KQ_MAX_STACK layers (hipExtLaunchKernel), so the caller can time that kernel inside the pass.
 */
typedef struct kq_compress_layer {
    const float* X;          /* [n][9] kernels */
    int64_t n;
    int32_t k;
    const float* C_init;     /* [k][9] initial codebook */
    float* C;                /* [k][9] codebook after `iters` rounds */
    int32_t* idx;            /* [n] final assignment */
    int32_t* counts;         /* [k] kernels per entry (final assignment) */
    double* distortion;      /* [iters + 1] or NULL */
    uint8_t* codes;          /* [k * 9] */
    float* levels;           /* [2^bits] */
    float* C_hat;            /* [k][9] levels[codes] */
    uint8_t* packed_idx;     /* ceil(n * ceil(log2 k) / 8) bytes, 4-byte aligned, or NULL */
    uint8_t* packed_codes;   /* ceil(9 k bits / 8) bytes, 4-byte aligned, or NULL */
    float* W_hat;            /* [n][9] or NULL */
    double* sq_error;        /* scalar or NULL (needs W_hat): sum of (X - W_hat)^2 over 9n values, fp64 */
} kq_compress_layer;

size_t kq_compress_workspace_bytes(const kq_compress_layer* layers, int32_t n_layers, int32_t bits);
kq_status kq_compress_stack(const kq_compress_layer* layers, int32_t n_layers, int32_t iters, int32_t mode,
                            int32_t bits, int32_t cbq_iters, uint32_t flags, void* const* round_events, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * Host-only helpers (no HIP call, no device memory).
 *
 * kq_index_bits: ceil(log2 k), the index width of Eq. (4) (0 for k = 1; -1 for k < 1).
 *
 * kq_accounting -- storage of a quantized layer of n kernels of dim = omega^2 values with a
 *   codebook of k entries stored at bc bits per value:
 *     Eq. (4): B = k * dim * bc + n * ceil(log2 k) bits;
 *     Eq. (6): C_KQ = 32 * n * dim / B (against fp32 weights);
 *     Eq. (7): beta = B / (n * dim) bits per parameter.
 *   bc = 32 for the fp32 codebook (K), 6 for the 6-bit one (K+C); the table of 2^bits levels
 *   is not counted.  Each output pointer may be NULL.  n, k, dim >= 1, 1 <= bc <= 64.
 *
 * kq_forgy_select -- the initial codebook of the k-means: k bitwise-distinct kernels of X
 *   (-0 and +0 count as equal) in a seeded random order.  Generator: splitmix64 (state +=
 *   0x9E3779B97F4A7C15, output mixed by the variant-13 finalizer), state = seed.  Order: a
 *   partial Fisher-Yates shuffle of 0 .. n-1: for i = 0, 1, ...: j = i + (next() mod (n - i)),
 *   swap positions i and j, candidate = the value now at position i; a candidate whose
 *   kernel equals an accepted one is skipped; stop at k accepted.  sel[q] = the q-th
 *   accepted kernel.  X host [n][9]; sel host [k].  KQ_ERR_ARG when X has fewer than k
 *   distinct kernels (sel untouched).  Host memory of O(k + draws) entries is used while it
 *   runs and released before it returns.
 */
int32_t kq_index_bits(int32_t k);
kq_status kq_accounting(int64_t n, int32_t k, int32_t dim, int32_t bc, int64_t* storage_bits, double* ratio,
                        double* bits_per_param);
kq_status kq_forgy_select(const float* X, int64_t n, int32_t dim, int32_t k, uint64_t seed, int64_t* sel);

/*
 * kq_fit_layer_noalloc -- kq_fit_layer for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid hipMalloc): the same
 * arguments without the workspace, and the same outputs bit for bit.  Its scratch is a
 * static device array of KQ_NOALLOC_SCRATCH_BYTES (32 MiB) in the library, one per GPU the
 * library runs on, held until the process ends; its address is looked up once per device
 * (hipGetSymbolAddress, on the first call with that device current).  The call allocates
 * nothing.  The stream must belong to the current device.
 *   Sizes whose kq_workspace_bytes(KQ_OP_FIT, n, k, 9) exceeds the scratch (for k = 256, n
 *   above 1,666,048 kernels) return KQ_ERR_WORKSPACE, before anything is enqueued.
 *   All calls on one GPU share that GPU's scratch: calls that overlap on one device (two
 *   streams, two host threads) race and give unspecified results; order them on one stream.
 *   Nothing in the scratch needs to start at zero (every call writes what it reads).
 *   kq_fit_layer_noalloc_max_bytes() returns the scratch size.
 */
#define KQ_NOALLOC_SCRATCH_BYTES (32u << 20)
size_t kq_fit_layer_noalloc_max_bytes(void);
kq_status kq_fit_layer_noalloc(const float* X, int64_t n, int32_t dim, int32_t k, const float* C_init, int32_t iters,
                               float* C, int32_t* idx, int32_t* counts, double* distortion, uint32_t flags,
                               void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KQ_H */
