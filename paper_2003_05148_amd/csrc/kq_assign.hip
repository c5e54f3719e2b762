// Assignment step of kernel-level quantization (Sec. 3.1, Eq. 1) for gfx950.
//
// idx[i] = argmin_j d(x_i, c_j) with d the fp32 squared distance evaluated term by
// term in dimension order (t = x - c, acc = fma(t, t, acc)), ties to the lowest j.
//
// Screening on the matrix cores.  Up to the constant |x|^2, d(x, c_j) is the score
//     s_j = |c_j|^2 - 2 x . c_j = [x, 1] . [-2 c_j, |c_j|^2]
// a K = 10 dot product.  One v_mfma_f32_32x32x2f32 per 2 of those 10 dims gives the
// 32 x 32 scores of 32 codebook entries (rows, operand A) against 32 kernels
// (columns, operand B): 5 MFMAs per tile, 90% of the MACs useful.  In the 32x32 D
// layout lane l holds column l % 32 and 16 rows, so every lane sees 16 entries of one
// kernel and keeps, per register slot, the best score, the second-best score and the
// codebook tile of the best (4 VALU ops per score: cmp, 2 cndmask, med3).
//
// Exactness guard.  The screened winner is the fp32 argmin whenever the gap between
// the two best screened scores exceeds theta = 2^-16 (|x| + max_j |c_j|)^2 + 2^-100,
// a bound on the screening error plus the rounding of the fp32 distances (see the
// derivation in the design notes of this library).  Kernels below the gap are
// rescored over the whole codebook in the exact fp32 form, one wave per kernel, after
// the block's screening pass.  So the output equals the plain fp32 argmin bit for bit.
//
// Layout: X is [n][9] fp32 (36-byte rows), the codebook is staged in LDS in the MFMA
// A-operand order [tile][k-step][lane] (conflict-free ds_read_b32), up to 1024
// entries at a time.  Each block covers 256 consecutive kernels of one layer; a
// descriptor table in the kernel arguments maps blocks to layers, so a whole conv
// stack is one launch.  The block's distortion partial (fp64, fixed tree order) goes
// to the workspace and the last block of a layer to finish sums them in block order.
#include "kq_internal.h"

namespace kq {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float sqdist9(const float* x, const float* __restrict__ c) {
    float acc = 0.0f;
#pragma unroll
    for (int d = 0; d < kDim; ++d) {
        const float t = x[d] - c[d];
        acc = __fmaf_rn(t, t, acc);
    }
    return acc;
}

// merge two (best, index, second) summaries; ties of best go to the lower index
__device__ __forceinline__ void merge_top2(float& b, int& j, float& s, float ob, int oj, float os) {
    s = fminf(fminf(s, os), fmaxf(b, ob));
    if (ob < b || (ob == b && oj < j)) {
        b = ob;
        j = oj;
    }
}

template <int R>
__global__ __launch_bounds__(kAssignWaves * kWave, 2) void assign_kernel(const StackParams p) {
    static_assert(R == 2, "one kernel per lane in the epilogue needs R == 2");
    __shared__ float s_cb[kAssignChunk * 10];
    __shared__ float s_dist[kAssignKernelsPerBlock];
    __shared__ int s_flag[kAssignKernelsPerBlock];
    __shared__ int s_nflag;
    __shared__ float s_cmax[kAssignWaves];
    __shared__ int s_last;

    const int li = find_layer(p, blockIdx.x);
    const DevLayer& L = p.L[li];
    const int lb = blockIdx.x - L.blk_begin;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, half = lane >> 5;
    const int n = L.n, k = L.k;
    const float* __restrict__ X = L.X;
    const float* __restrict__ C = L.C;
    const int kblk = lb * kAssignKernelsPerBlock;
    const int kbase = kblk + wave * (32 * R);

    if (tid == 0) s_nflag = 0;

    // B operands: lane (col, half) holds dims 2m + half of kernel kbase + 32 r + col
    float bx[R][5];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = kbase + 32 * r + col;
#pragma unroll
        for (int m = 0; m < 5; ++m) {
            const int d = 2 * m + half;
            bx[r][m] = (i < n) ? (d < kDim ? X[(size_t)i * kDim + d] : 1.0f) : 0.0f;
        }
    }

    float best[R][16], sec[R][16];
    int tl[R][16];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            best[r][s] = __builtin_inff();
            sec[r][s] = __builtin_inff();
            tl[r][s] = 0;
        }

    float cmax2 = 0.0f;
    const int kpad = (k + 31) & ~31;
    const f32x16 zero = {0.0f};
    for (int c0 = 0; c0 < kpad; c0 += kAssignChunk) {
        const int cn = min(kAssignChunk, kpad - c0);
        __syncthreads();
        for (int e = tid; e < cn * 10; e += kAssignWaves * kWave) {
            const int t = e / 320;
            const int rem = e - t * 320;
            const int m = rem >> 6, l = rem & 63;
            const int j = c0 + t * 32 + (l & 31);
            const int d = 2 * m + (l >> 5);
            float v;
            if (j < k) {
                if (d < kDim) {
                    v = -2.0f * C[(size_t)j * kDim + d];
                } else {
                    float nn = 0.0f;
#pragma unroll
                    for (int dd = 0; dd < kDim; ++dd) {
                        const float c = C[(size_t)j * kDim + dd];
                        nn = __fmaf_rn(c, c, nn);
                    }
                    v = nn;
                    cmax2 = fmaxf(cmax2, nn);
                }
            } else {
                v = (d < kDim) ? 0.0f : __builtin_inff();
            }
            s_cb[e] = v;
        }
        __syncthreads();

        const int ntile = cn >> 5;
        const int tbase = c0 >> 5;
#pragma unroll 1
        for (int t = 0; t < ntile; ++t) {
            float a[5];
#pragma unroll
            for (int m = 0; m < 5; ++m) a[m] = s_cb[(t * 5 + m) * 64 + lane];
            f32x16 acc[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                acc[r] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], bx[r][0], zero, 0, 0, 0);
#pragma unroll
                for (int m = 1; m < 5; ++m)
                    acc[r] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[m], bx[r][m], acc[r], 0, 0, 0);
            }
            const int tg = tbase + t;
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int s = 0; s < 16; ++s) {
                    const float sc = acc[r][s];
                    const bool lt = sc < best[r][s];
                    sec[r][s] = __builtin_amdgcn_fmed3f(best[r][s], sec[r][s], sc);
                    best[r][s] = lt ? sc : best[r][s];
                    tl[r][s] = lt ? tg : tl[r][s];
                }
        }
    }

    // largest codebook norm of the layer (upper bound for the guard)
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) cmax2 = fmaxf(cmax2, __shfl_xor(cmax2, off));
    if (lane == 0) s_cmax[wave] = cmax2;

    // collapse the 16 slots, then the two half-waves; lane l then owns kernel kbase + l
    float fb = __builtin_inff(), fs = __builtin_inff();
    int fj = 0x7fffffff;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        float b = __builtin_inff(), s2 = __builtin_inff();
        int j = 0x7fffffff;
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            const int js = tl[r][s] * 32 + 8 * (s >> 2) + 4 * half + (s & 3);
            merge_top2(b, j, s2, best[r][s], js, sec[r][s]);
        }
        const float ob = __shfl_xor(b, 32);
        const int oj = __shfl_xor(j, 32);
        const float os = __shfl_xor(s2, 32);
        merge_top2(b, j, s2, ob, oj, os);
        if (r == half) {
            fb = b;
            fj = j;
            fs = s2;
        }
    }
    __syncthreads();
    float cm2 = s_cmax[0];
#pragma unroll
    for (int w = 1; w < kAssignWaves; ++w) cm2 = fmaxf(cm2, s_cmax[w]);
    const float cmax = sqrtf(cm2);

    const int i = kbase + lane;
    const int il = i - kblk;
    float dist = 0.0f;
    if (i < n) {
        float x[kDim];
        float xn2 = 0.0f;
#pragma unroll
        for (int d = 0; d < kDim; ++d) {
            x[d] = X[(size_t)i * kDim + d];
            xn2 = __fmaf_rn(x[d], x[d], xn2);
        }
        const float rr = sqrtf(xn2) + cmax;
        const float theta = 0x1p-16f * rr * rr + 0x1p-100f;
        const bool sure = (fs - fb > theta) && (fj < k);
        if (sure) {
            dist = sqdist9(x, C + (size_t)fj * kDim);
            L.idx[i] = fj;
            if (L.best_d) L.best_d[i] = dist;
        } else {
            const int slot = atomicAdd(&s_nflag, 1);
            s_flag[slot] = i;
        }
    }
    s_dist[il] = dist;
    __syncthreads();

    // exact fp32 rescoring of the kernels the guard could not settle: one wave each
    const int nf = s_nflag;
    for (int f = wave; f < nf; f += kAssignWaves) {
        const int ii = s_flag[f];
        float x[kDim];
#pragma unroll
        for (int d = 0; d < kDim; ++d) x[d] = X[(size_t)ii * kDim + d];
        float bd = __builtin_inff();
        int bj = 0x7fffffff;
        for (int j = lane; j < k; j += kWave) {
            const float d = sqdist9(x, C + (size_t)j * kDim);
            if (d < bd) {
                bd = d;
                bj = j;
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const float od = __shfl_xor(bd, off);
            const int oj = __shfl_xor(bj, off);
            if (od < bd || (od == bd && oj < bj)) {
                bd = od;
                bj = oj;
            }
        }
        if (lane == 0) {
            if (bj == 0x7fffffff) bj = 0;  // every distance NaN or +inf: entry 0, as a plain scan gives
            L.idx[ii] = bj;
            if (L.best_d) L.best_d[ii] = bd;
            s_dist[ii - kblk] = bd;
        }
    }

    if (L.dist == nullptr) return;
    __syncthreads();
    if (wave == 0) {
        double acc = 0.0;
#pragma unroll
        for (int q = 0; q < kAssignKernelsPerBlock / kWave; ++q) acc += (double)s_dist[lane + kWave * q];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
        if (lane == 0) {
            L.part[lb] = acc;
            __threadfence();
            const unsigned old = atomicInc(&L.ctr[0], (unsigned)(L.nblk - 1));
            s_last = (old == (unsigned)(L.nblk - 1));
        }
    }
    __syncthreads();
    if (s_last && wave == 0) {
        __threadfence();
        double acc = 0.0;
        for (int q = lane; q < L.nblk; q += kWave) {
            acc += __builtin_nontemporal_load(L.part + q);
            L.part[q] = 0.0;  // the workspace goes back to all-zero
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
        if (lane == 0) *L.dist = acc;
    }
}

hipError_t launch_assign(const StackParams& p, hipStream_t s) {
    hipLaunchKernelGGL(assign_kernel<kAssignTilesPerWave>, dim3(p.total_blocks), dim3(kAssignWaves * kWave), 0, s, p);
    return hipGetLastError();
}

}  // namespace kq
