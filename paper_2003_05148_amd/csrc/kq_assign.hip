// Assignment step of kernel-level quantization (Sec. 3.1, Eq. 1) for gfx950.
//
// idx[i] = argmin_j d(x_i, c_j) with d the fp32 squared distance evaluated term by
// term in dimension order (t = x - c, acc = fma(t, t, acc)), ties to the lowest j.
//
// Screening on the matrix cores.  Up to the constant |x|^2, d(x, c_j) is the score
//     s_j = |c_j|^2 - 2 x . c_j = sum_{d < 10} w_jd y_d,  w_j = (-2 c_j, |c_j|^2), y = (x, 1).
// Every fp32 value v is split exactly into v = v_h + v_m + v_l with v_h = bf16(v) and
// v_m = bf16(v - v_h) (round to nearest), and the three cross terms w_h y_h + w_h y_m +
// w_m y_h form a K = 30 (padded to 32) bf16 contraction: two v_mfma_f32_32x32x16_bf16
// per 32 x 32 tile of (codebook entries, kernels), products exact and sums in fp32.  In
// the 32x32 D layout lane l holds column (kernel) l % 32 and 16 of its rows (entries);
// the 32 rows of a kernel are its "slots", slot r holding entries r, r + 32, r + 64, ...
// Each lane keeps the minimum score of each slot, one v_min3 per two scores.
//
// Exactness.  Write u = 2^-24 and P_j = 2 |x| |c_j| + |c_j|^2 <= (|x| + |c_j|)^2.  A
// screened score differs from s_j by at most 823 u P_j (dropped cross terms
// 3 * 2^-16 (1 + 2^-7), at most 33 fp32 roundings in the MFMA sums, 9 u in the fp32
// norm), and a slot minimum that carries its slot number in its 4 lowest mantissa bits
// moves by at most 30 u of its magnitude.  The entries of the slot with the smallest
// minimum are rescored in the plain fp32 form: d* is their smallest distance, taken at
// the lowest index; M2 is the smallest minimum of the other slots, so every entry j
// outside the slot has a screened score >= M2.  With R = 2 |x| + (1 + 2^-9) sqrt(d*) +
// 2^-61 and Q = R^2, such an entry either has |c_j| > R - |x|, and then lies farther
// than (1 + 2^-9) sqrt(d*) from x, so that its fp32 distance (every term positive,
// relative error <= 12 u) exceeds d*; or has P_j <= Q, and then its fp32 distance is at
// least (1 - 12 u) (M2 + |x|^2 - 823 u Q), which exceeds d* once
// M2 + |x|^2 - d* > 870 u Q (packing, the fp32 |x|^2, the distance's rounding and the
// guard's own two roundings included).  The guard asks for more than
// theta = 2^-14 Q' + 2^-100 with Q' = 1.03 (2 sqrt(fl |x|^2) + sqrt(d*) + 2^-60)^2 >= Q
// (1024 u Q; the hardware square roots' errors sit far inside the factor 1.03, and
// 2^-100 covers underflow).  A kernel that passes ends with the slot's fp32 argmin;
// the others are rescored over the whole codebook in the exact fp32 form by their
// wave.  The output is therefore the plain fp32 argmin, bit for bit.  Q' < 1e37 is also
// asked for: every entry with P_j <= Q then has finite partial sums, while a screened
// score of a farther entry may overflow to +inf or NaN, which the slot minima skip.
//
// Grid.  Kernels are cut into units of 64 (one kernel per lane of a wave).  The grid of
// at most kAssignGridMax workgroups is split per layer: layer l gets ceil(U_l / t)
// workgroups, t the smallest unit count per workgroup for which the total fits, and its
// U_l units are spread evenly over them, so a workgroup works within one layer; its waves
// take consecutive units round by round.  A codebook of up to kAssignChunk entries is
// split and staged once in LDS, in the MFMA A-operand
// order [tile][k-step][lane][8 x bf16] (one conflict-free ds_read_b128 per MFMA
// operand) and as fp32 rows for the slot rescoring; larger ones are streamed through LDS
// chunk by chunk.  Each lane splits its own kernel; the B operands of the two 32-kernel
// tiles of a wave are exchanged between the lane halves with v_permlane32_swap.  The next
// round's kernels are loaded while the current ones are scored.  After the scoring each wave
// settles its own 64 kernels (no workgroup barrier) and, when asked, writes an fp64
// distortion partial; a second kernel sums the partials in a fixed order.
#include <hip/hip_ext.h>

#include "kq_internal.h"

namespace kq {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowFloats = 12;      // fp32 codebook rows in LDS: 9 values, padded to 48 bytes
constexpr float kPadScore = 1e38f;  // score of padding entries: finite and above any trusted score
constexpr float kTrustQ = 1e37f;    // Q' at or above this: rescored over the whole codebook
static_assert(kAssignChunk % 64 == 0, "chunks hold whole pairs of 32-entry tiles");

// two fp32 values split exactly: v = h + m + l with h = bf16(v), m = bf16(v - h); H and M
// hold (h(a), h(b)) and (m(a), m(b)) packed, a in the low half
__device__ __forceinline__ void split2(float a, float b, unsigned& H, unsigned& M) {
    const f32x2 v = {a, b};
    H = __builtin_bit_cast(unsigned, __builtin_convertvector(v, bf16x2));
    const f32x2 r = {a - __uint_as_float(H << 16), b - __uint_as_float(H & 0xffff0000u)};  // exact
    M = __builtin_bit_cast(unsigned, __builtin_convertvector(r, bf16x2));
}

__device__ __forceinline__ float sqdist9(const float* x, const float* c) {
    float acc = 0.0f;
#pragma unroll
    for (int d = 0; d < kDim; ++d) {
        const float t = x[d] - c[d];
        acc = __fmaf_rn(t, t, acc);
    }
    return acc;
}

__device__ __forceinline__ float min2(float a, float b) { return __builtin_amdgcn_fmed3f(a, b, -3.402823466e38f); }
// the smallest of three finite values (v_min3_f32 without the compiler's NaN canonicalisation:
// the operands are never NaN)
__device__ __forceinline__ float min3f(float a, float b, float c) {
    float r;
    asm("v_min3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// scores of codebook tiles 2p and 2p + 1 (A operands a) against one kernel tile (B operands b)
__device__ __forceinline__ void score_pair(f32x16 (&acc)[2], const u32x4 (&a)[2][2], const u32x4 (&b)[2]) {
    const f32x16 zero = {0.0f};
#pragma unroll
    for (int u = 0; u < 2; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[u][0]),
                                                         __builtin_bit_cast(bf16x8, b[0]), zero, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 2; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[u][1]),
                                                         __builtin_bit_cast(bf16x8, b[1]), acc[u], 0, 0, 0);
}

// slot minima: one v_min3 per two scores
__device__ __forceinline__ void fold_pair(float (&best)[16], const f32x16 (&acc)[2]) {
#pragma unroll
    for (int q = 0; q < 16; ++q) best[q] = __builtin_fminf(__builtin_fminf(best[q], acc[0][q]), acc[1][q]);
}

// (d, j) becomes the lexicographic minimum of the pair and its partner's (o_d, o_j); a
// partner holding the same pair leaves it unchanged, so both lanes end with the same pair
__device__ __forceinline__ void argmin_take(float& d, int& j, float od, int oj) {
    const bool take = od < d || (od == d && oj < j);
    d = take ? od : d;
    j = take ? oj : j;
}
template <int CTL>
__device__ __forceinline__ void argmin_dpp(float& d, int& j) {
    const float od = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(d), CTL, 0xF, 0xF, true));
    const int oj = __builtin_amdgcn_mov_dpp(j, CTL, 0xF, 0xF, true);
    argmin_take(d, j, od, oj);
}
// the wave's lexicographic minimum of the lanes' (distance, index) pairs, in every lane:
// partners 32 and 16 lanes away by the half and row swaps, then DPP moves inside a row
// (the rotation by four meets a lane that holds the same pair as the lane 4 away)
__device__ __forceinline__ void wave_argmin(float& d, int& j) {
    {
        const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(d), __float_as_uint(d), false, false);
        const auto b = __builtin_amdgcn_permlane32_swap((unsigned)j, (unsigned)j, false, false);
        d = __uint_as_float(a[0]);
        j = (int)b[0];
        argmin_take(d, j, __uint_as_float(a[1]), (int)b[1]);
    }
    {
        const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(d), __float_as_uint(d), false, false);
        const auto b = __builtin_amdgcn_permlane16_swap((unsigned)j, (unsigned)j, false, false);
        d = __uint_as_float(a[0]);
        j = (int)b[0];
        argmin_take(d, j, __uint_as_float(a[1]), (int)b[1]);
    }
    argmin_dpp<0x128>(d, j);  // row_ror:8
    argmin_dpp<0x124>(d, j);  // row_ror:4
    argmin_dpp<0x4E>(d, j);   // quad_perm [2,3,0,1]
    argmin_dpp<0xB1>(d, j);   // quad_perm [1,0,3,2]
}

// the first pair's slot minima, capped at the largest finite float
__device__ __forceinline__ void first_pair(float (&best)[16], const f32x16 (&acc)[2]) {
#pragma unroll
    for (int q = 0; q < 16; ++q) best[q] = __builtin_fminf(__builtin_fminf(acc[0][q], acc[1][q]), 3.402823466e38f);
}

// A operands (entries) of codebook tiles 2 p and 2 p + 1
__device__ __forceinline__ void lds_a(u32x4 (&a)[2][2], const u32x4* s_a, int p, int lane) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) a[t][kk] = s_a[((2 * p + t) * 2 + kk) * kWave + lane];
}

// this lane's kernel of unit u of the layer (kernel 64 u + lane); a valid row past the end
__device__ __forceinline__ void load_kernel(const DevLayer& L, int u, int lane, float (&x)[kDim]) {
    const int i = u * kWave + lane;
    const int ic = i < L.n ? i : L.n - 1;
#pragma unroll
    for (int d = 0; d < kDim; ++d) x[d] = L.X[(size_t)ic * kDim + d];
}

// (best, second, index, distance) summaries; a tie of the screened bests makes the second
// equal to the best, which the guard rejects, so either winner may be kept
__device__ __forceinline__ void merge_top2(float& b, float& s, int& j, float& d, float ob, float os, int oj,
                                           float od) {
    const float mx = __builtin_amdgcn_fmed3f(b, ob, __builtin_inff());  // the larger (neither is NaN)
    s = fminf(fminf(s, os), mx);
    const bool lt = ob < b;
    b = lt ? ob : b;
    j = lt ? oj : j;
    d = lt ? od : d;
}

// Fused variant (every codebook of at most kFuseMaxK entries): each lane also adds its
// settled kernel to the workgroup's LDS histogram of exact fixed-point member sums, which
// is stored as the partial of (layer, workgroup) when the workgroup's units are done; the
// update then needs only its finishing launch.
__device__ __forceinline__ void fused_store(const DevLayer& H, const unsigned long long* s_sum, const unsigned* s_cnt,
                                            int tid) {
    __syncthreads();  // every wave has added its kernels
    unsigned long long* out = (unsigned long long*)H.hist + (size_t)(blockIdx.x - H.wfirst) * H.k * 10;
    for (int e = tid; e < H.k * 10; e += kAssignWaves * kWave) {
        const int j = e / 10, d = e - 10 * j;
        out[e] = d == 9 ? (unsigned long long)s_cnt[j] : s_sum[j * kDim + d];
    }
}

template <int R, bool FUSED>
__global__ __launch_bounds__(kAssignWaves * kWave, 1) void assign_kernel(const StackParams p) {
    static_assert(R == 2, "one kernel per lane and the half exchange need two kernel tiles per wave");
    constexpr int kAssignChunk = FUSED ? kFuseChunk : ::kq::kAssignChunk;
    __shared__ u32x4 s_a[kAssignChunk / 32 * 2 * kWave];  // [tile][k-step][lane] A operands
    __shared__ f32x4 s_c[kAssignChunk * kRowFloats / 4];   // fp32 rows of the staged entries
    __shared__ unsigned long long s_sum[FUSED ? kFuseMaxK * kDim : 1];  // fused: member sums
    __shared__ unsigned s_cnt[FUSED ? kFuseMaxK : 1];                   // fused: member counts
    __shared__ int s_next;                                              // fused: the next unit to hand out
    __shared__ unsigned s_mx;                                           // fused: the layer's largest magnitude

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    // this workgroup's run: a share of one layer's units (the layer's workgroups split them evenly)
    // (the table of first workgroups is read once, and the layer's fields in one batch after
    // it: every dependent load of the arguments is a memory round trip before any work)
    int lb = 0, g0 = 0, g1 = (int)gridDim.x;
#pragma unroll
    for (int l = 1; l < KQ_MAX_STACK; ++l) lb += (int)blockIdx.x >= p.wg_begin[l] ? 1 : 0;
#pragma unroll
    for (int l = 0; l < KQ_MAX_STACK; ++l) {  // past the last layer the table holds 0x7fffffff
        g0 = l == lb ? p.wg_begin[l] : g0;
        g1 = l == lb + 1 ? min(p.wg_begin[l], (int)gridDim.x) : g1;
    }
    const int gl = g1 - g0;
    const DevLayer& L = p.L[lb];
    const int n = L.n, k = L.k, U = L.nunits, j = (int)blockIdx.x - g0;
    const float* __restrict__ C = L.C;
    const float* const Xl = L.X;
    const unsigned* const xmax = L.xmax;
    const int nxmax = L.nxmax, derive = p.derive_shift;
    asm volatile("" ::"s"(n), "s"(k), "s"(U), "s"(C), "s"(Xl), "s"(xmax), "s"(nxmax), "s"(derive));
    const int q = U / gl, r = U - q * gl;  // workgroup j: q units, one more for the first r
    int ub = j * q + min(j, r);            // units of the layer, [ub, u_end)
    const int u_end = ub + q + (j < r ? 1 : 0);
    if (ub >= u_end) return;

    // The plain kernel goes in rounds of kAssignWaves consecutive units, unit ub + wave for
    // each wave (a wave past the run's end idles, but takes part in every barrier: a streamed
    // codebook is staged chunk by chunk).  The fused kernel's codebook is always resident, so
    // its loop has no barrier: each wave starts with unit ub + wave and then takes the next
    // unit from an LDS counter, so that a wave its SIMD serves less often takes fewer units.
    float xo[kDim];  // this lane's kernel of the current round
    load_kernel(L, ub + wave, lane, xo);
    // fused: the layer's shift, loaded with the first kernels (a later load would be one more
    // round trip before the first unit)
    const unsigned shift_word = FUSED && !derive ? xmax[nxmax] : 0u;
    const float* s_cf = reinterpret_cast<const float*>(s_c);
    // entries c0 .. c0 + cn - 1 of layer L into LDS: A operands [w_h | w_h | w_m] of w = (-2c, |c|^2)
    // and the fp32 rows (padding entries: screened far away, never taken by the rescoring)
    auto stage = [&](const DevLayer& L, int c0, int cn) {
        const int k = L.k;
        for (int jl = tid; jl < cn; jl += kAssignWaves * kWave) {
            const int j = c0 + jl;
            float c[kDim], w[10];
            if (j < k) {
#pragma unroll
                for (int d = 0; d < kDim; ++d) c[d] = L.C[(size_t)j * kDim + d];
                float nn = 0.0f;
#pragma unroll
                for (int d = 0; d < kDim; ++d) {
                    nn = __fmaf_rn(c[d], c[d], nn);
                    w[d] = -2.0f * c[d];
                }
                w[9] = nn;
            } else {  // padding: screened far away, and never taken by the rescoring
#pragma unroll
                for (int d = 0; d < kDim; ++d) {
                    c[d] = __builtin_inff();
                    w[d] = 0.0f;
                }
                w[9] = kPadScore;
            }
            unsigned H[5], M[5], A[16];
#pragma unroll
            for (int q = 0; q < 5; ++q) split2(w[2 * q], w[2 * q + 1], H[q], M[q]);
            // [w_h pairs 0..4 | w_h pairs 0..4 | w_m pairs 0..4 | 0]
#pragma unroll
            for (int q = 0; q < 5; ++q) {
                A[q] = H[q];
                A[5 + q] = H[q];
                A[10 + q] = M[q];
            }
            A[15] = 0u;
            const int tl = jl >> 5, row = jl & 31;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int e0 = 8 * kk + 4 * h;
                    const u32x4 v = {A[e0], A[e0 + 1], A[e0 + 2], A[e0 + 3]};
                    s_a[(tl * 2 + kk) * kWave + row + 32 * h] = v;
                }
            const f32x4 r0 = {c[0], c[1], c[2], c[3]}, r1 = {c[4], c[5], c[6], c[7]}, r2 = {c[8], 0.f, 0.f, 0.f};
            s_c[jl * 3 + 0] = r0;
            s_c[jl * 3 + 1] = r1;
            s_c[jl * 3 + 2] = r2;
        }
    };
    // the codebook, staged now so that its loads and the first kernels' are in flight together
    const int kpad = (k + 63) & ~63;
    const bool resident = kpad <= kAssignChunk;  // the whole codebook stays in LDS
    if (FUSED && !resident) return;              // (the host fuses only codebooks that fit)
    if (resident) stage(L, 0, kpad);
    if (FUSED) {
        if (tid == 0) s_next = ub + kAssignWaves;
        for (int e = tid; e < kFuseMaxK * kDim; e += kAssignWaves * kWave) s_sum[e] = 0ull;
        for (int e = tid; e < kFuseMaxK; e += kAssignWaves * kWave) s_cnt[e] = 0u;
    }
    // fused: the scale of the layer's fixed-point sums, read once (or formed from the block
    // maxima, and then stored by the layer's first workgroup for the launches after)
    double fsc = 0.0;
    if (FUSED) {
        int shift;
        if (derive) {
            shift = derive_shift<kAssignWaves * kWave>(L, &s_mx);
            if (j == 0 && tid == 0) L.xmax[L.nxmax] = (unsigned)shift;
        } else {
            shift = (int)shift_word;
        }
        fsc = fixed_scale(shift);
    }
    __syncthreads();

    // fused: this wave's unit (uniform over the wave); plain: the round's first unit
    int cur = FUSED ? __builtin_amdgcn_readfirstlane(ub + wave) : ub;
#pragma unroll 1
    while (cur < u_end) {
        const int lu = FUSED ? cur : cur + wave;  // this wave's unit of the layer
        const int i = lu * kWave + lane;
        const bool active = FUSED || lu < u_end;
        const bool valid = active && i < n;

        // the next unit's kernel, prefetched while this one is scored (every wave loads: past
        // the run's end a clamped row or another workgroup's, after its last unit this unit's
        // rows again; none is used)
        int nxt;
        if constexpr (FUSED) {
            int g = 0;
            if (lane == 0) g = atomicAdd(&s_next, 1);
            nxt = __builtin_amdgcn_readfirstlane(g);
        } else {
            nxt = cur + kAssignWaves;
        }
        float xn[kDim];
        load_kernel(L, nxt < u_end ? (FUSED ? nxt : nxt + wave) : lu, lane, xn);

        // B operands.  Kernel tile r of this wave is kernels 64 lu + 32 r + (lane % 32), the
        // kernels of lanes 32 r .. 32 r + 31.  A lane past the end holds a copy of the last
        // kernel and its results are dropped.  Lane (col, half) needs, for k-step kk, dwords
        // 8 kk + 4 half .. + 3 of the column's kernel; dword e packs terms 2e, 2e + 1:
        // [y_h pairs 0..4 | y_m pairs 0..4 | y_h pairs 0..4 | 0].
        u32x4 bop[R][2];
        {
            unsigned H[5], M[5];
#pragma unroll
            for (int q = 0; q < 4; ++q) split2(xo[2 * q], xo[2 * q + 1], H[q], M[q]);
            split2(xo[8], 1.0f, H[4], M[4]);
            unsigned D[16];
#pragma unroll
            for (int q = 0; q < 5; ++q) {
                D[q] = H[q];
                D[5 + q] = M[q];
                D[10 + q] = H[q];
            }
            D[15] = 0u;
            // lanes < 32 own tile 0 and lanes >= 32 tile 1: swapping (D[8kk+e], D[8kk+4+e])
            // across the halves leaves tile 0's operand in the first result, tile 1's in the second
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const auto sw = __builtin_amdgcn_permlane32_swap(D[8 * kk + e], D[8 * kk + 4 + e], false, false);
                    bop[0][kk][e] = sw[0];
                    bop[1][kk][e] = sw[1];
                }
        }

        float rb = __builtin_inff(), rs = __builtin_inff(), rd = __builtin_inff();  // running summary
        int rj = 0x7fffffff;
#pragma unroll 1
        for (int c0 = 0; c0 < kpad; c0 += kAssignChunk) {
            const int cn = min(kAssignChunk, kpad - c0);
            if (!FUSED && !resident) {
                __syncthreads();  // every wave is done with the previous contents
                stage(L, c0, cn);
                __syncthreads();
            }

            if (!active) continue;  // an idle wave only helps to stage

            // slot minima over the chunk (cn >= 64), two codebook tiles per step; the first
            // pair starts them, capped at the largest finite float so that packing keeps a number
            float best[R][16];
            const int npair = cn >> 6;
            u32x4 aN[2][2];
            {
                u32x4 a[2][2];
                lds_a(a, s_a, 0, lane);
                lds_a(aN, s_a, min(1, npair - 1), lane);  // the next pair's operands
                f32x16 acc[R][2];
#pragma unroll
                for (int r = 0; r < R; ++r) score_pair(acc[r], a, bop[r]);
#pragma unroll
                for (int r = 0; r < R; ++r) first_pair(best[r], acc[r]);
            }
#pragma unroll 1
            for (int tp = 1; tp < npair; ++tp) {
                u32x4 a[2][2];
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int kk = 0; kk < 2; ++kk) a[u][kk] = aN[u][kk];
                lds_a(aN, s_a, min(tp + 1, npair - 1), lane);  // the next pair's operands
                f32x16 acc[R][2];
#pragma unroll
                for (int r = 0; r < R; ++r) score_pair(acc[r], a, bop[r]);
#pragma unroll
                for (int r = 0; r < R; ++r) fold_pair(best[r], acc[r]);
            }

            // per kernel tile: smallest and second smallest slot minimum, the slot number q
            // (rows 8 (q / 4) + 4 half + q % 4) packed into the low bits.  A tournament: the
            // smallest and second smallest of each triple (min3, med3); for groups with such
            // pairs (m, s), the set's smallest is the least m and its second smallest the
            // smaller of the groups' second-least m and the least s (an s of a group that does
            // not hold the minimum is at least that group's m)
            float m1[R], m2[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float pq[16];
#pragma unroll
                for (int q = 0; q < 16; ++q) pq[q] = __uint_as_float((__float_as_uint(best[r][q]) & ~15u) | (unsigned)q);
                float tm[5], ts[5];
#pragma unroll
                for (int t = 0; t < 5; ++t) {
                    tm[t] = min3f(pq[3 * t], pq[3 * t + 1], pq[3 * t + 2]);
                    ts[t] = __builtin_amdgcn_fmed3f(pq[3 * t], pq[3 * t + 1], pq[3 * t + 2]);
                }
                const float ma = min3f(tm[0], tm[1], tm[2]);
                const float sa = min2(__builtin_amdgcn_fmed3f(tm[0], tm[1], tm[2]), min3f(ts[0], ts[1], ts[2]));
                const float mb = min3f(tm[3], tm[4], pq[15]);
                const float sb = min2(__builtin_amdgcn_fmed3f(tm[3], tm[4], pq[15]), min2(ts[3], ts[4]));
                m1[r] = min2(ma, mb);
                m2[r] = __builtin_amdgcn_fmed3f(ma, mb, min2(sa, sb));
            }
            // own kernel: lanes < 32 tile 0, lanes >= 32 tile 1; first from the lower half's rows
            const auto x1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(m1[0]), __float_as_uint(m1[1]), false, false);
            const auto x2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(m2[0]), __float_as_uint(m2[1]), false, false);
            const float lo1 = __uint_as_float(x1[0]), hi1 = __uint_as_float(x1[1]);
            const float lo2 = __uint_as_float(x2[0]), hi2 = __uint_as_float(x2[1]);
            const float M1 = min2(lo1, hi1);
            const float M2 = __builtin_amdgcn_fmed3f(lo1, hi1, min2(lo2, hi2));
            const int qs = (int)(__float_as_uint(M1) & 15u);
            const int slot = 8 * (qs >> 2) + (qs & 3) + (hi1 < lo1 ? 4 : 0);

            // exact fp32 rescoring of the winning slot's entries, in increasing index order
            // (padding rows are +inf: never taken)
            float bd = __builtin_inff();
            int bt = -1;  // tile of the best entry so far
            const int ntile = cn >> 5;  // the same trip count in every lane
            auto rescore = [&](int tq) {
                const int jl = slot + 32 * tq;
                const f32x4 r0 = s_c[jl * 3 + 0], r1 = s_c[jl * 3 + 1];
                const float c8 = s_cf[jl * kRowFloats + 8];
                const float c[kDim] = {r0[0], r0[1], r0[2], r0[3], r1[0], r1[1], r1[2], r1[3], c8};
                const float d = sqdist9(xo, c);
                const bool take = d < bd;
                bd = take ? d : bd;
                bt = take ? tq : bt;
            };
            if (ntile == 8) {  // 256 entries: constant tile numbers
#pragma unroll
                for (int tq = 0; tq < 8; ++tq) rescore(tq);
            } else {
#pragma unroll 4
                for (int tq = 0; tq < ntile; ++tq) rescore(tq);
            }
            const int bj = bt < 0 ? 0x7fffffff : c0 + slot + 32 * bt;
            if (c0 == 0) {  // the first chunk starts the summary
                rb = M1;
                rs = M2;
                rj = bj;
                rd = bd;
            } else {
                merge_top2(rb, rs, rj, rd, M1, M2, bj, bd);
            }
        }
        if (active) {  // settle this wave's unit
            float xn2 = 0.0f;
#pragma unroll
            for (int d = 0; d < kDim; ++d) xn2 = __fmaf_rn(xo[d], xo[d], xn2);
            // the local bound Q' from |x| and the rescored distance; the hardware square roots
            // will do (their errors are far below the factor 1.03)
            const float rr = 2.0f * __builtin_amdgcn_sqrtf(xn2) + __builtin_amdgcn_sqrtf(rd) + 0x1p-60f;
            const float q2 = rr * rr * 1.03f;
            const float theta = 0x1p-14f * q2 + 0x1p-100f;

            const bool sure = valid && (q2 < kTrustQ) && (rs - (rd - xn2) > theta) && (rj < k);
            float dist = 0.0f;
            int myj = rj;  // the entry this lane's kernel ends with
            if (sure) {
                dist = rd;
                if (L.idx) L.idx[i] = rj;  // (a fit's rounds before the last keep no indices)
                if (L.best_d) L.best_d[i] = rd;
            }

            // exact fp32 rescoring of the kernels the guard could not settle, one at a time
            unsigned long long fl = __ballot(valid && !sure);
            while (fl) {
                const int f = __ffsll((long long)fl) - 1;
                fl &= fl - 1;
                float xf[kDim];  // lane f's kernel, the same in every lane (f is uniform)
#pragma unroll
                for (int d = 0; d < kDim; ++d)
                    xf[d] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(xo[d]), f));
                // each lane scans entries lane, lane + 64, ... in increasing order (strict <: the
                // lowest index among equal distances), then the lanes' (distance, index) pairs
                // meet in their lexicographic minimum
                float fd = __builtin_inff();
                int fj = 0x7fffffff;
                if (resident) {  // the rows are still staged in LDS: four per lane in flight
                    constexpr int kU = 4;
                    for (int j0 = lane; j0 < k; j0 += kU * kWave) {
                        f32x4 r0[kU], r1[kU];
                        float c8[kU];
#pragma unroll
                        for (int u = 0; u < kU; ++u) {
                            const int jj = min(j0 + u * kWave, k - 1);  // a staged row past the end
                            r0[u] = s_c[jj * 3 + 0];
                            r1[u] = s_c[jj * 3 + 1];
                            c8[u] = s_cf[jj * kRowFloats + 8];
                        }
#pragma unroll
                        for (int u = 0; u < kU; ++u) {
                            const int jj = j0 + u * kWave;
                            const float c[kDim] = {r0[u][0], r0[u][1], r0[u][2], r0[u][3], r1[u][0],
                                                   r1[u][1], r1[u][2], r1[u][3], c8[u]};
                            const float d = sqdist9(xf, c);
                            const bool take = jj < k && d < fd;
                            fj = take ? jj : fj;
                            fd = take ? d : fd;
                        }
                    }
                } else {  // rows from memory: four per lane in flight, taken in index order
                    constexpr int kU = 4;
                    for (int j0 = lane; j0 < k; j0 += kU * kWave) {
                        float c[kU][kDim];
#pragma unroll
                        for (int u = 0; u < kU; ++u) {
                            const int jj = min(j0 + u * kWave, k - 1);  // a valid row past the end
#pragma unroll
                            for (int d = 0; d < kDim; ++d) c[u][d] = C[(size_t)jj * kDim + d];
                        }
#pragma unroll
                        for (int u = 0; u < kU; ++u) {
                            const int jj = j0 + u * kWave;
                            const float d = sqdist9(xf, c[u]);
                            const bool take = jj < k && d < fd;
                            fj = take ? jj : fj;
                            fd = take ? d : fd;
                        }
                    }
                }
                wave_argmin(fd, fj);
                if (lane == f) {
                    if (fj == 0x7fffffff) fj = 0;  // every distance NaN or +inf: entry 0, as a plain scan gives
                    if (L.idx) L.idx[i] = fj;
                    if (L.best_d) L.best_d[i] = fd;
                    dist = fd;
                    myj = fj;
                }
            }

            if (FUSED && valid) {  // the update's exact member sums of this kernel, at the layer's shift
                atomicAdd(&s_cnt[myj], 1u);
#pragma unroll
                for (int d = 0; d < kDim; ++d) atomicAdd(&s_sum[myj * kDim + d], fixed_bits(xo[d], fsc));
            }

            if (L.part) {
                const double v = wave_sum_f64(valid ? (double)dist : 0.0);
                if (lane == 0) L.part[lu] = v;
            }
        }

#pragma unroll
        for (int d = 0; d < kDim; ++d) xo[d] = xn[d];
        cur = nxt;
    }
    if (FUSED) fused_store(L, s_sum, s_cnt, tid);
}

// distortion of each layer: its per-wave partials summed in a fixed order
__global__ __launch_bounds__(kSumThreads) void assign_finish_kernel(const StackParams p) {
    __shared__ double s_w[kSumThreads / kWave];
    const DevLayer& L = p.L[blockIdx.x];
    if (L.dist == nullptr) return;
    const double v = block_fixed_sum<kSumThreads>(L.part, L.nunits, s_w);
    if (threadIdx.x == 0) *L.dist = v;
}


int assign_partition(const int* units, int nlayers, int* g) {
    long long T = 0;
    int umax = 1;
    for (int l = 0; l < nlayers; ++l) {
        T += units[l];
        umax = units[l] > umax ? units[l] : umax;
    }
    auto count = [&](long long t) {
        long long c = 0;
        for (int l = 0; l < nlayers; ++l) c += (units[l] + t - 1) / t;
        return c;
    };
    long long lo = (T + kAssignGridMax - 1) / kAssignGridMax, hi = umax;  // count(hi) = nlayers <= the grid
    if (lo < 1) lo = 1;
    while (lo < hi) {
        const long long mid = (lo + hi) / 2;
        if (count(mid) <= kAssignGridMax)
            hi = mid;
        else
            lo = mid + 1;
    }
    int grid = 0;
    for (int l = 0; l < nlayers; ++l) {
        g[l] = (int)((units[l] + lo - 1) / lo);
        grid += g[l];
    }
    return grid;
}

hipError_t launch_assign(const StackParams& p, hipStream_t s, bool fused, hipEvent_t start, hipEvent_t stop) {
    const int grid = p.assign_grid;
    const dim3 g(grid), b(kAssignWaves * kWave);
    if (start || stop) {  // the events take the kernel's own start and end times
        if (fused)
            hipExtLaunchKernelGGL((assign_kernel<kAssignTilesPerWave, true>), g, b, 0, s, start, stop, 0, p);
        else
            hipExtLaunchKernelGGL((assign_kernel<kAssignTilesPerWave, false>), g, b, 0, s, start, stop, 0, p);
    } else if (fused) {
        hipLaunchKernelGGL((assign_kernel<kAssignTilesPerWave, true>), g, b, 0, s, p);
    } else {
        hipLaunchKernelGGL((assign_kernel<kAssignTilesPerWave, false>), g, b, 0, s, p);
    }
    return hipGetLastError();
}

hipError_t launch_assign_finish(const StackParams& p, hipStream_t s) {
    hipLaunchKernelGGL(assign_finish_kernel, dim3(p.nlayers), dim3(kSumThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace kq
