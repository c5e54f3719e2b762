/*
 * Plain CPU oracle for kernel-level quantization (KQ): TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may load
 * this file's library.  It shares nothing with the HIP path: no headers, no
 * helpers, no tables.  Everything here is a direct, slow loop over the
 * definitions in Sec. 3.1 of the paper (kernel-level quantization):
 *
 *   - each 3x3 kernel m_i is a vector in R^{omega^2} (the weight tensor reshaped
 *     into n = p q kernels);
 *   - k-means (Eq. 1) alternates an assignment of every kernel to its nearest
 *     codebook entry and a replacement of every entry by the mean of its kernel
 *     set S_i (plain Lloyd iterations; Sec. 4.1 states that the Yinyang variant
 *     used by the authors gives exactly the results of plain k-means).
 *
 * Readings where the paper is silent:
 *   - the nearest entry is decided on squared distances evaluated in fp32 (the
 *     precision of the paper's full-precision weights), term by term in
 *     dimension order as t = x_d - c_d, acc = fma(t, t, acc); ties go to the
 *     lowest entry index;
 *   - the same decision is also reported in fp64 together with the best and
 *     second-best fp64 distances, so callers can identify near-ties;
 *   - an entry whose kernel set is empty keeps its previous value;
 *   - the mean is an fp64 sum over members in ascending kernel order, divided
 *     by the member count, rounded once to fp32;
 *   - the distortion of an assignment is the fp64 sum, in ascending kernel
 *     order, of the fp64 squared distances to the assigned entries.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC kq_oracle.c -lm
 * (contraction off, so every multiply and add below rounds separately unless
 * fmaf is written out).  The assignment's loop over kernels may run on several
 * host threads (kqo_set_threads): every kernel's decision is computed alone, so
 * the results are the same on any number of threads; the distortion and the
 * update stay sequential sums in ascending kernel order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Squared distance in fp32: t = x_d - c_d, acc = fmaf(t, t, acc), d ascending. */
static float sqdist_f32(const float* x, const float* c, int dim) {
    float acc = 0.0f;
    for (int d = 0; d < dim; ++d) {
        float t = x[d] - c[d];
        acc = fmaf(t, t, acc);
    }
    return acc;
}

/* Squared distance in fp64 (each term and each partial sum rounded to fp64). */
static double sqdist_f64(const float* x, const float* c, int dim) {
    double acc = 0.0;
    for (int d = 0; d < dim; ++d) {
        double t = (double)x[d] - (double)c[d];
        acc = acc + t * t;
    }
    return acc;
}

static int kqo_threads = 1;

/* Host threads for the assignment loop (1 = plain sequential loop).  Returns the count. */
int kqo_set_threads(int t) {
    kqo_threads = t < 1 ? 1 : t;
    return kqo_threads;
}

/*
 * Assignment step of Eq. (1): nearest codebook entry of every kernel.
 *   X [n][dim], C [k][dim] row-major fp32.
 *   idx32/d32: decision and distance in fp32 (nullable).
 *   idx64/d1/d2: decision in fp64, best and second-best fp64 distances
 *                (nullable; d2 is +inf when k == 1).
 * Returns 0, or -1 on bad sizes.
 */
int kqo_assign(const float* X, int64_t n, int dim, const float* C, int k,
               int32_t* idx32, float* d32, int32_t* idx64, double* d1, double* d2) {
    if (n < 0 || dim < 1 || k < 1) return -1;
#pragma omp parallel for schedule(static) num_threads(kqo_threads) if (kqo_threads > 1)
    for (int64_t i = 0; i < n; ++i) {
        const float* x = X + i * dim;
        if (idx32 || d32) {
            float best = INFINITY;
            int32_t bj = 0;
            for (int j = 0; j < k; ++j) {
                float d = sqdist_f32(x, C + (int64_t)j * dim, dim);
                if (d < best) { best = d; bj = j; }
            }
            if (idx32) idx32[i] = bj;
            if (d32) d32[i] = best;
        }
        if (idx64 || d1 || d2) {
            double best = INFINITY, second = INFINITY;
            int32_t bj = 0;
            for (int j = 0; j < k; ++j) {
                double d = sqdist_f64(x, C + (int64_t)j * dim, dim);
                if (d < best) { second = best; best = d; bj = j; }
                else if (d < second) { second = d; }
            }
            if (idx64) idx64[i] = bj;
            if (d1) d1[i] = best;
            if (d2) d2[i] = second;
        }
    }
    return 0;
}

/* Distortion of an assignment: sum over i (ascending) of |x_i - c_{idx_i}|^2 in fp64. */
double kqo_distortion(const float* X, int64_t n, int dim, const float* C, const int32_t* idx) {
    double J = 0.0;
    for (int64_t i = 0; i < n; ++i) J = J + sqdist_f64(X + i * dim, C + (int64_t)idx[i] * dim, dim);
    return J;
}

/*
 * Update step of Eq. (1): every entry becomes the mean of its kernel set S_j.
 *   counts[j] = |S_j|; C_new[j] = fp32(fp64 sum of members, ascending i, / |S_j|);
 *   an empty set keeps C_old[j].  C_new may alias C_old.
 * Returns 0, or -1 if an index is out of range.
 */
int kqo_update(const float* X, int64_t n, int dim, const int32_t* idx, int k,
               const float* C_old, float* C_new, int32_t* counts) {
    double* S = (double*)calloc((size_t)k * dim, sizeof(double));
    int64_t* z = (int64_t*)calloc((size_t)k, sizeof(int64_t));
    if (!S || !z) { free(S); free(z); return -2; }
    for (int64_t i = 0; i < n; ++i) {
        int32_t j = idx[i];
        if (j < 0 || j >= k) { free(S); free(z); return -1; }
        z[j] += 1;
        for (int d = 0; d < dim; ++d) S[(int64_t)j * dim + d] = S[(int64_t)j * dim + d] + (double)X[i * dim + d];
    }
    for (int j = 0; j < k; ++j) {
        if (counts) counts[j] = (int32_t)z[j];
        for (int d = 0; d < dim; ++d) {
            int64_t r = (int64_t)j * dim + d;
            C_new[r] = z[j] > 0 ? (float)(S[r] / (double)z[j]) : C_old[r];
        }
    }
    free(S);
    free(z);
    return 0;
}

/*
 * Lloyd k-means on one layer: `iters` rounds of (assign, update), then a final
 * assignment against the last codebook.
 *   C_init [k][dim] -> C_out [k][dim] (state after `iters` updates)
 *   idx_out [n]   : final assignment (fp32 decision)
 *   counts_out [k]: member counts of the final assignment
 *   J_out [iters+1]: J_out[t] is the distortion of assignment t (t = 0..iters)
 *                    against the codebook it was made with.
 * Returns 0 or a negative error.
 */
int kqo_fit(const float* X, int64_t n, int dim, int k, const float* C_init, int iters,
            float* C_out, int32_t* idx_out, int32_t* counts_out, double* J_out) {
    if (n < 1 || dim < 1 || k < 1 || iters < 0) return -1;
    memcpy(C_out, C_init, sizeof(float) * (size_t)k * dim);
    for (int t = 0; t <= iters; ++t) {
        int rc = kqo_assign(X, n, dim, C_out, k, idx_out, NULL, NULL, NULL, NULL);
        if (rc) return rc;
        if (J_out) J_out[t] = kqo_distortion(X, n, dim, C_out, idx_out);
        if (t < iters) {
            rc = kqo_update(X, n, dim, idx_out, k, C_out, C_out, NULL);
            if (rc) return rc;
        }
    }
    if (counts_out) {
        for (int j = 0; j < k; ++j) counts_out[j] = 0;
        for (int64_t i = 0; i < n; ++i) counts_out[idx_out[i]] += 1;
    }
    return 0;
}
