// Yinyang assignment for gfx950.  Sec. 4.1 of the paper runs its kernel-level k-means
// with Yinyang k-means (Ding et al., ICML 2015), which skips distance evaluations with
// triangle-inequality bounds and reaches exactly the plain Lloyd result.  Here the result
// is, bit for bit, the fp32 argmin that kq_assign returns (distances evaluated term by
// term in dimension order, ties to the lowest entry index).
//
// Groups.  The codebook's entries are split into t groups once, by a few Lloyd rounds on
// the entries themselves (the grouping only decides how much work is skipped, never the
// result).  perm lists the entries group by group, ascending within a group.
//
// Bounds.  Every bound is on the true Euclidean distance e(x, c) = sqrt(sum (x - c)^2) and
// rounded towards safety.  An fp32 squared distance d32 computed term by term is within
// 12 u of the exact one (u = 2^-24; every term is non-negative) plus at most 1e-43 from
// underflow, so sqrt(d32 + 1e-43) (1 + 2^-20) bounds e from above and
// sqrt(d32 - 1e-43) (1 - 2^-20) from below.  Per kernel and group the library stores
// Lt_g = L_g + D_g rounded down to fp32, where L_g is a lower bound of e(x, c) over the
// group's entries other than the kernel's current one, and D_g the group's cumulative
// drift bound at the time (fp64, rounded up): when an entry moves by at most delta,
// distances to it change by at most delta, so Lt_g - D_g(now) stays a lower bound.
//
// One round, after the codebook moved from C_prev to C:
//   drift   per group: the largest movement of its entries (upper bound), added to D_g;
//   filter  per kernel: d_a = d32(x, c_a) for its current entry a, U = upper bound of
//           e(x, c_a) widened by (1 + 2^-18) and 1e-20.  A group with U < Lt_g - D_g
//           holds no entry whose fp32 distance can reach d_a (the widening covers the
//           12 u error on both sides and underflow), so it is skipped.  The mask of the
//           groups left is stored per kernel and counted per workgroup in LDS;
//   lists   the per-workgroup counts are scanned per group and every workgroup writes its
//           kernels into each group's list (and the list of kernels with anything to
//           scan) in ascending order: no global atomics, the same lists on every run;
//   eval    per (group, 512 listed kernels): the group's entries are staged in LDS and
//           every lane scans them for two kernels in ascending index order: smallest fp32
//           distance, its entry (strict <, so the lowest index among ties), second
//           smallest distance;
//   final   per listed kernel: the lexicographically smallest (distance, index) of the
//           current entry and the scanned groups' winners is the fp32 argmin (no finite
//           distance: entry 0, as a plain scan gives); each scanned group's bound becomes
//           its smallest distance, or its second smallest when it holds the winner; a
//           former entry that lost becomes an ordinary member of its group.
// Round 0 is the screened matrix-core assignment of kq_assign; the initial bounds come
// from the group centres: e(x, c) >= e(x, G_g) - r_g with r_g the group's radius.
#include "kq_internal.h"

namespace kq {

namespace {

constexpr double kLoRel = 1.0 - 0x1p-20;
constexpr double kHiRel = 1.0 + 0x1p-20;
constexpr double kUnderflow = 1e-43;         // absolute error of an fp32 distance from underflow
constexpr double kFilterRel = 1.0 + 0x1p-18;
constexpr double kFilterAbs = 1e-20;
constexpr double kDriftRel = 1.0 + 0x1p-50;  // cumulative drift: fp64 additions rounded up
constexpr double kStoreRel = 1.0 - 0x1p-40;  // L + D in fp64 before rounding down to fp32
constexpr float kInf = __builtin_inff();

__device__ __forceinline__ float d32(const float (&x)[kDim], const float* __restrict__ c) {
    float acc = 0.0f;
#pragma unroll
    for (int d = 0; d < kDim; ++d) {
        const float t = x[d] - c[d];
        acc = __fmaf_rn(t, t, acc);
    }
    return acc;
}

// lower / upper bound of the Euclidean distance whose fp32 square is v
__device__ __forceinline__ double dist_lo(float v) {
    if (!(v < kInf)) return v == kInf ? 1.8e19 : 0.0;  // an fp32 overflow means e >= sqrt(FLT_MAX)
    const double w = (double)v - kUnderflow;
    return w > 0.0 ? __builtin_sqrt(w) * kLoRel : 0.0;
}
__device__ __forceinline__ double dist_hi(float v) { return __builtin_sqrt((double)v + kUnderflow) * kHiRel; }

// Lt = fp32 lower bound of L + D (infinite L stays infinite)
__device__ __forceinline__ float store_lo(double L, double D) {
    const double s = L + D;
    return __double2float_rd(s > 0.0 ? s * kStoreRel : 0.0);
}

__device__ __forceinline__ void load_row(const float* __restrict__ X, long long i, float (&x)[kDim]) {
#pragma unroll
    for (int d = 0; d < kDim; ++d) x[d] = X[(size_t)i * kDim + d];
}

}  // namespace

// ---- grouping statistics: perm, group starts, radii, zero drift (one workgroup) --------
__global__ __launch_bounds__(1024) void yy_group_kernel(const YyParams p) {
    __shared__ int s_cnt[kYyMaxGroups], s_off[kYyMaxGroups];
    __shared__ int s_wc[1024 / kWave][kYyMaxGroups];
    __shared__ unsigned s_rad[kYyMaxGroups];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int k = p.k, t = p.t;
    if (tid < t) {
        s_cnt[tid] = 0;
        s_rad[tid] = 0u;
    }
    __syncthreads();
    for (int j = tid; j < k; j += 1024) {
        const int g = p.labels[j];
        float c[kDim];
        load_row(p.C, j, c);
        atomicAdd(&s_cnt[g], 1);
        const float r = __double2float_ru(dist_hi(d32(c, p.Cg + (size_t)g * kDim)));
        atomicMax(&s_rad[g], __float_as_uint(r));  // non-negative floats order as their bits
    }
    __syncthreads();
    if (tid == 0) {
        int s = 0;
        for (int g = 0; g < t; ++g) {
            p.gstart[g] = s;
            s_off[g] = s;
            s += s_cnt[g];
        }
        p.gstart[t] = s;
    }
    if (tid < t) {
        p.radius[tid] = __uint_as_float(s_rad[tid]);
        p.delta[tid] = 0.0;
    }
    __syncthreads();
    // stable scatter, 1024 entries at a time: rank among the wave's lanes of the same group,
    // then the waves before, then the chunks before
    for (int base = 0; base < k; base += 1024) {
        const int j = base + tid;
        const int g = j < k ? p.labels[j] : -1;
        int rank = 0;
        for (int gg = 0; gg < t; ++gg) {
            const unsigned long long b = __ballot(g == gg);
            if (g == gg) rank = __popcll(b & ((1ull << lane) - 1ull));
            if (lane == 0) s_wc[wave][gg] = __popcll(b);
        }
        __syncthreads();
        if (g >= 0) {
            int pos = s_off[g] + rank;
            for (int w = 0; w < wave; ++w) pos += s_wc[w][g];
            p.perm[pos] = j;
        }
        __syncthreads();
        if (tid < t)
            for (int w = 0; w < 1024 / kWave; ++w) s_off[tid] += s_wc[w][tid];
        __syncthreads();
    }
}

// ---- initial bounds from the group centres -----------------------------------------------
__global__ __launch_bounds__(256) void yy_bounds_init_kernel(const YyParams p) {
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= p.n) return;
    float x[kDim];
    load_row(p.X, i, x);
    for (int g = 0; g < p.t; ++g) {
        float Lt;
        if (p.gstart[g + 1] == p.gstart[g]) {
            Lt = kInf;  // an empty group holds nothing to find
        } else {
            const double L = dist_lo(d32(x, p.Cg + (size_t)g * kDim)) - (double)p.radius[g];
            Lt = store_lo(L > 0.0 ? L : 0.0, 0.0);
        }
        p.Lt[(size_t)g * p.n + i] = Lt;
    }
}

// ---- drift of every group between C_prev and C ----------------------------------------
__global__ __launch_bounds__(1024) void yy_drift_kernel(const YyParams p) {
    __shared__ unsigned s_mx[kYyMaxGroups];
    const int tid = threadIdx.x;
    if (tid < p.t) s_mx[tid] = 0u;
    __syncthreads();
    for (int j = tid; j < p.k; j += 1024) {
        float a[kDim];
        load_row(p.C_prev, j, a);
        const float m = __double2float_ru(dist_hi(d32(a, p.C + (size_t)j * kDim)));
        atomicMax(&s_mx[p.labels[j]], __float_as_uint(m));  // NaN bits exceed +inf: kept as NaN
    }
    __syncthreads();
    if (tid < p.t) p.delta[tid] = (p.delta[tid] + (double)__uint_as_float(s_mx[tid])) * kDriftRel;
}

// ---- filter: one kernel per thread ---------------------------------------------------------
// Writes the mask of groups to scan for every kernel (0: settled) and, per workgroup, how
// many of its kernels each group lists (row t: kernels with anything to scan).
__global__ __launch_bounds__(256) void yy_filter_kernel(const YyParams p) {
    __shared__ int s_c[kYyMaxGroups + 1];
    const int tid = threadIdx.x, lane = tid & 63;
    const long long i = (long long)blockIdx.x * 256 + tid;
    const bool valid = i < p.n;
    const int n = p.n, k = p.k, t = p.t;
    if (tid <= t) s_c[tid] = 0;
    unsigned long long mask = 0ull;
    if (valid) {
        const int a = p.idx[i];
        float x[kDim];
        load_row(p.X, i, x);
        const float da = (a >= 0 && a < k) ? d32(x, p.C + (size_t)a * kDim) : kInf;
        const double U = dist_hi(da) * kFilterRel + kFilterAbs;  // NaN fails every test below
        for (int g = 0; g < t; ++g) {
            const double L = (double)p.Lt[(size_t)g * n + i] - p.delta[g];
            if (!(U < L)) mask |= 1ull << g;
        }
        if (!(da < kInf)) mask = t >= 64 ? ~0ull : ((1ull << t) - 1ull);  // no finite distance yet: scan all
        p.best_d[i] = da;
        p.mask[i] = mask;
    }
    __syncthreads();
    for (int g = 0; g <= t; ++g) {
        const bool on = g < t ? ((mask >> g) & 1ull) != 0 : mask != 0ull;
        const unsigned long long b = __ballot(on);
        if (lane == 0 && b) atomicAdd(&s_c[g], __popcll(b));  // LDS
    }
    __syncthreads();
    if (tid <= t) p.wgc[(size_t)tid * gridDim.x + blockIdx.x] = s_c[tid];
}

// ---- per group: exclusive scan of the per-workgroup counts (one workgroup per group) ------
__global__ __launch_bounds__(1024) void yy_scan_kernel(const YyParams p, int nwg) {
    __shared__ int s_w[1024 / kWave];
    const int g = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int* row = p.wgc + (size_t)g * nwg;
    int carry = 0;
    for (int base = 0; base < nwg; base += 1024) {
        const int q = base + tid;
        const int v = q < nwg ? row[q] : 0;
        int x = v;  // inclusive scan inside the wave
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            const int y = __shfl_up(x, off);
            if (lane >= off) x += y;
        }
        if (lane == kWave - 1) s_w[wave] = x;
        __syncthreads();
        int before = carry;
        for (int w = 0; w < wave; ++w) before += s_w[w];
        int total = carry;
        for (int w = 0; w < 1024 / kWave; ++w) total += s_w[w];
        if (q < nwg) row[q] = before + x - v;
        __syncthreads();
        carry = total;
    }
    if (tid == 0) p.cnt[g] = carry;
}

// ---- scatter: every group's list in ascending kernel order --------------------------------
// Only the groups some kernel of the workgroup needs are visited (bit t of the union: the
// list of kernels with anything to scan).
__device__ __forceinline__ bool listed_in(unsigned long long mask, int g, int t) {
    return g < t ? ((mask >> g) & 1ull) != 0 : mask != 0ull;
}

__global__ __launch_bounds__(256) void yy_scatter_kernel(const YyParams p) {
    __shared__ int s_w[4][kYyMaxGroups + 1];
    __shared__ unsigned long long s_or;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const long long i = (long long)blockIdx.x * 256 + tid;
    const int n = p.n, t = p.t;
    const unsigned long long mask = i < n ? p.mask[i] : 0ull;
    const unsigned long long below = (1ull << lane) - 1ull;
    if (tid == 0) s_or = 0ull;
    __syncthreads();
    if (mask) atomicOr(&s_or, mask);
    __syncthreads();
    const unsigned long long any = s_or;
    if (any == 0ull) return;  // uniform: nothing listed in this workgroup
    // visit the groups of the union, then the list of kernels with anything to scan
    for (unsigned long long m = any;; m &= m - 1ull) {
        const int g = m ? __ffsll((long long)m) - 1 : t;
        const unsigned long long b = __ballot(listed_in(mask, g, t));
        if (lane == 0) s_w[wave][g] = __popcll(b);
        if (!m) break;
    }
    __syncthreads();
    for (unsigned long long m = any;; m &= m - 1ull) {
        const int g = m ? __ffsll((long long)m) - 1 : t;
        const bool on = listed_in(mask, g, t);
        const unsigned long long b = __ballot(on);
        if (on) {
            int pos = p.wgc[(size_t)g * gridDim.x + blockIdx.x] + __popcll(b & below);
            for (int w = 0; w < wave; ++w) pos += s_w[w][g];
            if (g < t)
                p.lists[(size_t)g * n + pos] = (int)i;
            else
                p.flist[pos] = (int)i;
        }
        if (!m) break;
    }
}

// ---- exact scan of the listed (kernel, group) pairs -------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));

// one lane's running scan of a group: smallest distance, its entry, second smallest
struct Scan {
    float b1, b2;
    int j1;
};

__device__ __forceinline__ void scan_step(Scan& s, float d, int e) {
    if (d < s.b1) {
        s.b2 = s.b1;
        s.b1 = d;
        s.j1 = e;
    } else if (d < s.b2) {
        s.b2 = d;
    }
}

// A work item is 512 listed kernels of one group, two per lane: every staged entry read
// from LDS (a broadcast) serves two distances.
__global__ __launch_bounds__(256) void yy_eval_kernel(const YyParams p) {
    __shared__ f32x4 s_c[kYyEvalChunk * 3];  // the staged entries, 48-byte rows
    __shared__ int s_j[kYyEvalChunk];
    __shared__ int s_pre[kYyMaxGroups + 1];  // first work item of each group
    constexpr int kItem = 2 * 256;
    const int tid = threadIdx.x;
    const int n = p.n, t = p.t;
    if (tid == 0) {
        int s = 0;
        for (int g = 0; g < t; ++g) {
            s_pre[g] = s;
            s += (p.cnt[g] + kItem - 1) / kItem;
        }
        s_pre[t] = s;
    }
    __syncthreads();
    const int total = s_pre[t];
    int staged_g = -1, staged_c0 = -1;
    const float* s_cf = reinterpret_cast<const float*>(s_c);
    for (int item = blockIdx.x; item < total; item += gridDim.x) {
        int g = 0;
        while (g + 1 < t && item >= s_pre[g + 1]) ++g;
        const int pos0 = (item - s_pre[g]) * kItem + tid, pos1 = pos0 + 256;
        const int cg = p.cnt[g];
        const bool has0 = pos0 < cg, has1 = pos1 < cg;
        const int pt0 = has0 ? p.lists[(size_t)g * n + pos0] : 0;
        const int pt1 = has1 ? p.lists[(size_t)g * n + pos1] : pt0;
        float x0[kDim], x1[kDim];
        load_row(p.X, pt0, x0);
        load_row(p.X, pt1, x1);
        const int g0 = p.gstart[g], m = p.gstart[g + 1] - g0;
        Scan s0 = {kInf, kInf, -1}, s1 = {kInf, kInf, -1};
        for (int c0 = 0; c0 < m; c0 += kYyEvalChunk) {
            const int cm = min(kYyEvalChunk, m - c0);
            if (staged_g != g || staged_c0 != c0) {
                __syncthreads();  // every lane is done with the previous entries
                for (int e = tid; e < cm; e += 256) {
                    const int j = p.perm[g0 + c0 + e];
                    float c[kDim];
                    load_row(p.C, j, c);
                    s_j[e] = j;
                    s_c[e * 3 + 0] = f32x4{c[0], c[1], c[2], c[3]};
                    s_c[e * 3 + 1] = f32x4{c[4], c[5], c[6], c[7]};
                    s_c[e * 3 + 2] = f32x4{c[8], 0.0f, 0.0f, 0.0f};
                }
                __syncthreads();
                staged_g = g;
                staged_c0 = c0;
            }
            // positions in the staged chunk; entries ascend with them inside a group
#pragma unroll 4
            for (int e = 0; e < cm; ++e) {
                const f32x4 r0 = s_c[e * 3 + 0], r1 = s_c[e * 3 + 1];
                const float c[kDim] = {r0[0], r0[1], r0[2], r0[3], r1[0], r1[1], r1[2], r1[3], s_cf[e * 12 + 8]};
                scan_step(s0, d32(x0, c), c0 + e);
                scan_step(s1, d32(x1, c), c0 + e);
            }
        }
        // positions to entries (the chunk that holds a position may not be staged any more)
        if (has0) {
            p.B1[(size_t)g * n + pt0] = s0.b1;
            p.J1[(size_t)g * n + pt0] = s0.j1 >= 0 ? p.perm[g0 + s0.j1] : -1;
            p.B2[(size_t)g * n + pt0] = s0.b2;
        }
        if (has1) {
            p.B1[(size_t)g * n + pt1] = s1.b1;
            p.J1[(size_t)g * n + pt1] = s1.j1 >= 0 ? p.perm[g0 + s1.j1] : -1;
            p.B2[(size_t)g * n + pt1] = s1.b2;
        }
    }
}

// ---- decision and new bounds for the listed kernels ------------------------------------
__global__ __launch_bounds__(256) void yy_final_kernel(const YyParams p) {
    const int n = p.n, t = p.t, k = p.k;
    const int nf = p.cnt[t];
    if (blockIdx.x == 0 && threadIdx.x == 0 && p.stats) {
        long long pairs = 0, evals = 0;
        for (int g = 0; g < t; ++g) {
            pairs += p.cnt[g];
            evals += (long long)p.cnt[g] * (p.gstart[g + 1] - p.gstart[g]);
        }
        p.stats[0] = nf;
        p.stats[1] = pairs;
        p.stats[2] = evals;
    }
    for (int q = blockIdx.x * 256 + threadIdx.x; q < nf; q += gridDim.x * 256) {
        const int i = p.flist[q];
        const unsigned long long mask = p.mask[i];
        const int a = p.idx[i];
        const float da = p.best_d[i];
        const bool have = da < kInf;  // a finite distance to the current entry (a is then valid)
        float bd = have ? da : kInf;
        int bj = have ? a : -1;
        for (unsigned long long m = mask; m; m &= m - 1ull) {
            const int g = __ffsll((long long)m) - 1;
            const int j1 = p.J1[(size_t)g * n + i];
            const float b1 = p.B1[(size_t)g * n + i];
            if (j1 >= 0 && (bj < 0 || b1 < bd || (b1 == bd && j1 < bj))) {
                bd = b1;
                bj = j1;
            }
        }
        if (bj < 0) {  // no finite distance: entry 0, as a plain scan gives
            bj = 0;
            bd = kInf;
        }
        const int gb = p.labels[bj];
        for (unsigned long long m = mask; m; m &= m - 1ull) {
            const int g = __ffsll((long long)m) - 1;
            const float v = (g == gb) ? p.B2[(size_t)g * n + i] : p.B1[(size_t)g * n + i];
            p.Lt[(size_t)g * n + i] = store_lo(dist_lo(v), p.delta[g]);
        }
        if (have && bj != a) {  // the former entry is now an ordinary member of its group
            const int ga = p.labels[a];
            if (!((mask >> ga) & 1ull)) {
                const double old = (double)p.Lt[(size_t)ga * n + i] - p.delta[ga];
                const double now = dist_lo(da);
                p.Lt[(size_t)ga * n + i] = store_lo(now < old ? now : old, p.delta[ga]);
            }
        }
        p.idx[i] = bj;
        p.best_d[i] = bd;
        (void)k;
    }
}

// ---- distortion partials from the best distances, in the assignment kernel's order -------
// partial w = the butterfly sum of the fp64 distances of kernels 64 w .. 64 w + 63, the same
// operations in the same order as the assignment kernel's per-wave partials
__global__ __launch_bounds__(256) void yy_partials_kernel(const YyParams p) {
    const int lane = threadIdx.x & 63;
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
    const long long i = (long long)w * kWave + lane;
    double v = i < p.n ? (double)p.best_d[i] : 0.0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0 && w < p.npart) p.part[w] = v;
}

hipError_t launch_yy_group(const YyParams& p, hipStream_t s) {
    hipLaunchKernelGGL(yy_group_kernel, dim3(1), dim3(1024), 0, s, p);
    return hipGetLastError();
}
hipError_t launch_yy_bounds_init(const YyParams& p, hipStream_t s) {
    hipLaunchKernelGGL(yy_bounds_init_kernel, dim3((unsigned)((p.n + 255) / 256)), dim3(256), 0, s, p);
    return hipGetLastError();
}
hipError_t launch_yy_round(const YyParams& p, hipStream_t s) {
    hipLaunchKernelGGL(yy_drift_kernel, dim3(1), dim3(1024), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned blocks = (unsigned)((p.n + 255) / 256);
    hipLaunchKernelGGL(yy_filter_kernel, dim3(blocks), dim3(256), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(yy_scan_kernel, dim3(p.t + 1), dim3(1024), 0, s, p, (int)blocks);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(yy_scatter_kernel, dim3(blocks), dim3(256), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const long long items = (long long)p.t * ((p.n + 511) / 512);
    const unsigned eg = (unsigned)(items < kYyEvalGrid ? items : kYyEvalGrid);
    hipLaunchKernelGGL(yy_eval_kernel, dim3(eg), dim3(256), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned fg = blocks < kYyFinalGrid ? blocks : kYyFinalGrid;
    hipLaunchKernelGGL(yy_final_kernel, dim3(fg), dim3(256), 0, s, p);
    return hipGetLastError();
}
hipError_t launch_yy_partials(const YyParams& p, hipStream_t s) {
    hipLaunchKernelGGL(yy_partials_kernel, dim3((unsigned)((p.npart + 3) / 4)), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace kq
