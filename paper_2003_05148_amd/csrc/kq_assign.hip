// Assignment step of kernel-level quantization (Sec. 3.1, Eq. 1) for gfx950.
//
// idx[i] = argmin_j d(x_i, c_j) with d the fp32 squared distance evaluated term by
// term in dimension order (t = x - c, acc = fma(t, t, acc)), ties to the lowest j.
//
// Screening on the matrix cores.  Up to the constant |x|^2, d(x, c_j) is the score
//     s_j = |c_j|^2 - 2 x . c_j = sum_{d < 10} w_jd y_d,  w_j = (-2 c_j, |c_j|^2), y = (x, 1).
// Every fp32 value v is split into three bf16 parts v = v_h + v_m + v_l (each part the
// round-to-nearest bf16 of what the previous ones leave), and the six cross terms that
// carry fp32 precision, w_h y_h + w_h y_m + w_m y_h + w_h y_l + w_l y_h + w_m y_m, form a
// K = 60 (padded to 64) bf16 contraction: four v_mfma_f32_32x32x16_bf16 per 32 x 32
// tile of (codebook entries, kernels), products exact and sums in fp32.  In the 32x32
// D layout lane l holds column (kernel) l % 32 and 16 rows (entries); per register slot
// it keeps the best and the second-best score, the best carrying its codebook tile in
// its low mantissa bits (3 VALU ops per score: and-or and two med3).
//
// Exactness guard.  Let Q = (|x| + max_j |c_j|)^2 and u = 2^-24.  A screened score is
// within 84 u Q of its exact value (dropped cross terms and split remainders 7 u Q, at
// most 68 fp32 roundings in the MFMA sums, 9 u Q in the fp32 norm) plus 32 u Q for the
// packed tile bits, and the fp32 distance of any entry is within 12 u of its exact value.
// So when the two best screened scores are more than theta = 2^-15 Q + 2^-100 apart
// (512 u Q, against 257 u Q needed) the screened winner is the fp32 argmin.  Kernels
// below that gap are rescored over the whole codebook in the exact fp32 form by their
// wave.  The output is therefore the plain fp32 argmin, bit for bit.
//
// Grid.  Kernels are cut into tiles of 256 (one per workgroup pass); tiles of all
// layers of a stack are numbered layer after layer and a persistent grid of at most
// kAssignGridMax workgroups walks contiguous runs of them.  A codebook of up to 512
// entries is split and staged once per layer in LDS in the MFMA A-operand order
// [tile][k-step][lane][8 x bf16] (one conflict-free ds_read_b128 per MFMA); larger
// ones are streamed through LDS in 512-entry chunks.  The next tile's kernels are
// loaded while the current one is scored.  After the scoring each wave settles its own
// 64 kernels (no workgroup barrier) and, when asked, writes an fp64 distortion
// partial; a second kernel sums the partials in a fixed order.
#include "kq_internal.h"

namespace kq {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// ---- the bf16 contraction ----------------------------------------------------------------
// term k < 60 of the contraction: dimension k % 10 of cross term k / 10; the cross terms
// (entry part, kernel part) are (h,h), (h,m), (m,h), (h,l), (l,h), (m,m); k >= 60 is zero.
__host__ __device__ constexpr int term_dim(int k) { return k % 10; }
__host__ __device__ constexpr int term_wpart(int k) { return (k / 10 == 2 || k / 10 == 5) ? 1 : (k / 10 == 4 ? 2 : 0); }
__host__ __device__ constexpr int term_ypart(int k) { return (k / 10 == 1 || k / 10 == 5) ? 1 : (k / 10 == 3 ? 2 : 0); }

__device__ __forceinline__ float bf16_round(float v) { return (float)(__bf16)v; }

// v = h + m + l with h, m, l representable in bf16 (up to a remainder below 2^-25 |v|)
__device__ __forceinline__ void split3(float v, float& h, float& m, float& l) {
    h = bf16_round(v);
    const float r = v - h;  // exact
    m = bf16_round(r);
    l = bf16_round(r - m);  // r - m exact
}

// B operands (kernel side) of one kernel: lane half `half` holds terms 16 kk + 8 half + e
__device__ __forceinline__ void build_b(const float (&x)[kDim], bool valid, int half, bf16x8 (&b)[4]) {
    float p[3][10];
#pragma unroll
    for (int d = 0; d < kDim; ++d) split3(valid ? x[d] : 0.0f, p[0][d], p[1][d], p[2][d]);
    p[0][9] = valid ? 1.0f : 0.0f;
    p[1][9] = 0.0f;
    p[2][9] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int k0 = 16 * kk + e, k1 = 16 * kk + 8 + e;
            const float v0 = k0 < 60 ? p[term_ypart(k0)][term_dim(k0)] : 0.0f;
            const float v1 = k1 < 60 ? p[term_ypart(k1)][term_dim(k1)] : 0.0f;
            b[kk][e] = (__bf16)(half ? v1 : v0);
        }
}

// Scores are folded with the codebook tile (0..15 within a 512-entry chunk) packed into
// their 5 lowest mantissa bits, so one med3 keeps the best score and its tile.  The
// packing moves a score by less than 2^-19 of its magnitude; the guard allows for it.
constexpr unsigned kTileMask = 31u;
constexpr float kPadScore = 1e38f;  // score of padding entries: finite, so packing keeps a number

__device__ __forceinline__ float sqdist9(const float* x, const float* c) {
    float acc = 0.0f;
#pragma unroll
    for (int d = 0; d < kDim; ++d) {
        const float t = x[d] - c[d];
        acc = __fmaf_rn(t, t, acc);
    }
    return acc;
}

// merge two (best, index, second) summaries; exact ties of the screened best are always
// caught by the guard (the second then equals the best), so any winner is fine here
__device__ __forceinline__ void merge_top2(float& b, int& j, float& s, float ob, int oj, float os) {
    const float mx = __builtin_amdgcn_fmed3f(b, ob, __builtin_inff());
    s = __builtin_amdgcn_fmed3f(__builtin_amdgcn_fmed3f(s, os, -__builtin_inff()), mx, -__builtin_inff());
    const bool lt = ob < b;
    b = lt ? ob : b;
    j = lt ? oj : j;
}

// the 32 x 32 scores of one codebook tile (A operands a) against the wave's R kernel tiles
template <int R>
__device__ __forceinline__ void score_tile(f32x16 (&acc)[R], const bf16x8 (&a)[4], const bf16x8 (&b)[R][4]) {
    const f32x16 zero = {0.0f};
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[r][0], zero, 0, 0, 0);
#pragma unroll
    for (int kk = 1; kk < 4; ++kk)
#pragma unroll
        for (int r = 0; r < R; ++r)
            acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], b[r][kk], acc[r], 0, 0, 0);
}

// per register slot: second = med3(best, second, s), best = med3(best, s, -FLT_MAX)
// = min(best, s) -- 3 VALU ops (v_and_or_b32 with the tile held in a VGPR, 2 v_med3_f32)
template <int R>
__device__ __forceinline__ void fold_tile(const f32x16 (&acc)[R], unsigned tile, float (&best)[R][16],
                                          float (&sec)[R][16]) {
    unsigned vt;
    asm("v_mov_b32 %0, %1" : "=v"(vt) : "s"(tile));
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const float sp = __uint_as_float((__float_as_uint(acc[r][q]) & ~kTileMask) | vt);
            sec[r][q] = __builtin_amdgcn_fmed3f(best[r][q], sec[r][q], sp);
            best[r][q] = __builtin_amdgcn_fmed3f(best[r][q], sp, -3.402823466e38f);
        }
}

// this lane's kernel (kernel 256 t + 64 wave + lane of the layer); zeros past the end
__device__ __forceinline__ void load_kernel(const DevLayer& L, int tile, int wave, int lane, float (&x)[kDim]) {
    const int i = tile * kAssignKernelsPerTile + wave * kWave + lane;
    const int ic = i < L.n ? i : L.n - 1;
#pragma unroll
    for (int d = 0; d < kDim; ++d) x[d] = L.X[(size_t)ic * kDim + d];
}

__device__ __forceinline__ void global_entry(const float* __restrict__ C, int j, float (&c)[kDim]) {
#pragma unroll
    for (int d = 0; d < kDim; ++d) c[d] = C[(size_t)j * kDim + d];
}

template <int R>
__global__ __launch_bounds__(kAssignWaves * kWave, 2) void assign_kernel(const StackParams p) {
    static_assert(R == 2, "one kernel per lane in the epilogue needs R == 2");
    __shared__ bf16x8 s_a[kAssignChunk / 32 * 4 * kWave];  // [tile][k-step][lane] A operands
    __shared__ float s_wmax[kAssignWaves];                  // per-wave max |c|^2 of the staged codebook

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, half = lane >> 5;
    const long long T = p.total_units;
    int t = (int)((long long)blockIdx.x * T / gridDim.x);
    const int t_end = (int)((long long)(blockIdx.x + 1) * T / gridDim.x);
    if (t >= t_end) return;

    int li = find_layer(p, t);
    int staged = -1;  // layer whose whole codebook is resident in LDS
    float xo[kDim];   // this lane's kernel of the current tile
    load_kernel(p.L[li], t - p.L[li].unit_begin, wave, lane, xo);

#pragma unroll 1
    for (; t < t_end; ++t) {
        while (li + 1 < p.nlayers && t >= p.L[li + 1].unit_begin) ++li;
        const DevLayer& L = p.L[li];
        const int n = L.n, k = L.k;
        const float* __restrict__ C = L.C;
        const int lt = t - L.unit_begin;
        const int i = lt * kAssignKernelsPerTile + wave * kWave + lane;
        const bool valid = i < n;

        // prefetch the next tile's kernel; it arrives while this tile is scored
        float xn[kDim];
        if (t + 1 < t_end) {
            int ln = li;
            while (ln + 1 < p.nlayers && t + 1 >= p.L[ln + 1].unit_begin) ++ln;
            load_kernel(p.L[ln], t + 1 - p.L[ln].unit_begin, wave, lane, xn);
        }

        // B operands: kernel tile r of this wave is kernels 64 wave + 32 r + col, i.e. the
        // kernel of lane col + 32 r; lanes swap kernels with their partner half
        bf16x8 bop[R][4];
        {
            float xp[kDim];
#pragma unroll
            for (int d = 0; d < kDim; ++d) xp[d] = __shfl_xor(xo[d], 32);
            const bool vp = __shfl_xor((int)valid, 32) != 0;
            // tile `half` is this lane's own kernel, tile 1 - half the partner's
            bf16x8 own[4], par[4];
            build_b(xo, valid, half, own);
            build_b(xp, vp, half, par);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                bop[0][kk] = half ? par[kk] : own[kk];
                bop[1][kk] = half ? own[kk] : par[kk];
            }
        }

        float rb[R], rs[R];
        int rj[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            rb[r] = __builtin_inff();
            rs[r] = __builtin_inff();
            rj[r] = 0x7fffffff;
        }

        const int kpad = (k + 31) & ~31;
        const bool resident = kpad <= kAssignChunk;
        float tmax = 0.0f;
#pragma unroll 1
        for (int c0 = 0; c0 < kpad; c0 += kAssignChunk) {
            const int cn = min(kAssignChunk, kpad - c0);
            if (!resident || staged != li) {
                __syncthreads();  // every wave is done with the previous contents
                for (int jl = tid; jl < cn; jl += kAssignWaves * kWave) {
                    const int j = c0 + jl;
                    float w[3][10];
                    if (j < k) {
                        float c[kDim];
                        global_entry(C, j, c);
                        float nn = 0.0f;
#pragma unroll
                        for (int d = 0; d < kDim; ++d) {
                            nn = __fmaf_rn(c[d], c[d], nn);
                            split3(-2.0f * c[d], w[0][d], w[1][d], w[2][d]);
                        }
                        split3(nn, w[0][9], w[1][9], w[2][9]);
                        tmax = fmaxf(tmax, nn);
                    } else {
#pragma unroll
                        for (int d = 0; d < kDim; ++d) w[0][d] = w[1][d] = w[2][d] = 0.0f;
                        split3(kPadScore, w[0][9], w[1][9], w[2][9]);
                    }
                    const int tl = jl >> 5, row = jl & 31;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            bf16x8 v;
#pragma unroll
                            for (int e = 0; e < 8; ++e) {
                                const int kt = 16 * kk + 8 * h + e;
                                v[e] = (__bf16)(kt < 60 ? w[term_wpart(kt)][term_dim(kt)] : 0.0f);
                            }
                            s_a[(tl * 4 + kk) * kWave + row + 32 * h] = v;
                        }
                }
                if (c0 + cn >= kpad) {  // last chunk: publish this wave's max norm
                    float wm = tmax;
#pragma unroll
                    for (int off = 32; off >= 1; off >>= 1) wm = fmaxf(wm, __shfl_xor(wm, off));
                    if (lane == 0) s_wmax[wave] = wm;
                }
                __syncthreads();
                staged = resident ? li : -1;
            }

            float best[R][16], sec[R][16];
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    best[r][q] = __builtin_inff();
                    sec[r][q] = __builtin_inff();
                }
            const int ntile = cn >> 5;
#pragma unroll 1
            for (int tt = 0; tt < ntile; ++tt) {
                bf16x8 a[4];
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) a[kk] = s_a[(tt * 4 + kk) * kWave + lane];
                f32x16 acc[R];
                score_tile<R>(acc, a, bop);
                fold_tile<R>(acc, (unsigned)tt, best, sec);
            }
            // fold this chunk's 16 slots into the running summaries
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int j = c0 + (int)(__float_as_uint(best[r][q]) & kTileMask) * 32 + 8 * (q >> 2) + 4 * half +
                                  (q & 3);
                    merge_top2(rb[r], rj[r], rs[r], best[r][q], j, sec[r][q]);
                }
        }

        // the two half-waves; lane l then owns kernel 64 wave + l (tile r = half)
        float fb = __builtin_inff(), fs = __builtin_inff();
        int fj = 0x7fffffff;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float b = rb[r], s2 = rs[r];
            int j = rj[r];
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

        float xn2 = 0.0f;
#pragma unroll
        for (int d = 0; d < kDim; ++d) xn2 = __fmaf_rn(xo[d], xo[d], xn2);
        float cm2 = s_wmax[0];
#pragma unroll
        for (int w = 1; w < kAssignWaves; ++w) cm2 = fmaxf(cm2, s_wmax[w]);
        const float rr = sqrtf(xn2) + sqrtf(cm2);
        const float theta = 0x1p-15f * rr * rr + 0x1p-100f;

        const bool sure = valid && (fs - fb > theta) && (fj < k);
        float dist = 0.0f;
        if (sure) {
            float c[kDim];
            global_entry(C, fj, c);
            dist = sqdist9(xo, c);
            L.idx[i] = fj;
            if (L.best_d) L.best_d[i] = dist;
        }

        // exact fp32 rescoring of the kernels the guard could not settle, one at a time
        unsigned long long fl = __ballot(valid && !sure);
        while (fl) {
            const int f = __ffsll((long long)fl) - 1;
            fl &= fl - 1;
            float xf[kDim];
#pragma unroll
            for (int d = 0; d < kDim; ++d) xf[d] = __shfl(xo[d], f);
            float bd = __builtin_inff();
            int bj = 0x7fffffff;
            for (int j = lane; j < k; j += kWave) {
                float c[kDim];
                global_entry(C, j, c);
                const float d = sqdist9(xf, c);
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
            if (lane == f) {
                if (bj == 0x7fffffff) bj = 0;  // every distance NaN or +inf: entry 0, as a plain scan gives
                L.idx[i] = bj;
                if (L.best_d) L.best_d[i] = bd;
                dist = bd;
            }
        }

        if (L.part) {
            double v = valid ? (double)dist : 0.0;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
            if (lane == 0) L.part[lt * kAssignWaves + wave] = v;
        }

#pragma unroll
        for (int d = 0; d < kDim; ++d) xo[d] = xn[d];
    }
}

// distortion of each layer: its per-wave partials summed in a fixed order
__global__ __launch_bounds__(kSumThreads) void assign_finish_kernel(const StackParams p) {
    __shared__ double s_w[kSumThreads / kWave];
    const DevLayer& L = p.L[blockIdx.x];
    if (L.dist == nullptr) return;
    const double v = block_fixed_sum<kSumThreads>(L.part, L.nunits * kAssignWaves, s_w);
    if (threadIdx.x == 0) *L.dist = v;
}

hipError_t launch_assign(const StackParams& p, hipStream_t s) {
    const int grid = p.total_units < kAssignGridMax ? p.total_units : kAssignGridMax;
    hipLaunchKernelGGL(assign_kernel<kAssignTilesPerWave>, dim3(grid), dim3(kAssignWaves * kWave), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_assign_finish(const StackParams& p, hipStream_t s) {
    hipLaunchKernelGGL(assign_finish_kernel, dim3(p.nlayers), dim3(kSumThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace kq
