// Update step of kernel-level quantization (Sec. 3.1, Eq. 1): every codebook entry
// becomes the mean of its kernel set S_j; an empty set keeps its entry.
//
// The member sums are exact integers: each value is mapped to q(x) = rint(x * 2^s) with a
// per-layer shift s = min(62 - ceil(log2 n), 51) - e, max |x| < 2^e, so |q| <= 2^62 / n
// and no sum over at most n kernels can overflow int64, at any magnitude of the weights
// (each q is added as kFixedBias + q, the bit pattern of one fp64 fma, and the finish
// takes count * kFixedBias back off).
// Integer addition is associative, so the sums, and with them the new codebook, do not
// depend on the order in which blocks or lanes add.  absmax_kernel takes the maxima of |x|
// per block of 32768 values, once per call or once per fit, before any sum is formed; with a
// range check shift_kernel turns them into each layer's s (and flags non-finite values),
// otherwise the first launch that forms sums does (derive_shift: every workgroup takes the
// layer's largest block maximum, one of them stores s for the launches after).
//
// update_kernel: one launch covers every layer of a stack.  A layer's kernels are cut
// into chunks and its codebook into ranges of at most 768 entries; a workgroup of 1024
// threads takes one (chunk, range) pair: it reads the chunk's indices, one 36-byte row per
// thread and step (consecutive lanes, consecutive rows, two steps in flight), loads the
// rows whose entry lies in its range and adds them to a private LDS histogram of the range
// ([768][9] int64 sums + [768] counts at most, ds_add_u64), then stores the histogram
// into the chunk's partial ([chunks][k][10] int64).  Chunk sizes give about one workgroup
// per CU for the whole launch.  The LDS atomics, not the loads, bound it: a layout with
// fully coalesced dword loads, where each float fetched its kernel's entry with
// ds_bpermute, added LDS work and ran slower.  Asked for the distortion of a standalone
// assignment, it also sums, in a fixed order, the fp32 distances of its rows to their old
// entries.
// Codebook gradient step (Eq. 2): the same sums over a gradient tensor G instead of the
// kernels, with the same shift rule applied to max |g|; the finish then writes
// c - gamma * mean instead of the mean.
// update_finish_kernel: a workgroup of 960 threads owns 16 entries of one layer; six
// groups of 160 threads add a sixth of the partials each, nine loads in flight per thread
// (one batch for the 54 partials of the largest ResNet-18 layers; any order gives the same
// integers), then it divides and writes the codebook and the counts.  Fewer, fuller
// workgroups measured faster: the launch is short, and the workgroups dispatched last
// start up to 2 us after the first (528 workgroups of 640 threads at 8 entries each; 2
// or 4 entries each were slower still).  One more workgroup per layer adds the distortion
// partials in a fixed order with its first 640 threads (those of the assignment kernel
// when the distortion comes from there).  The kernel boundary orders every partial before
// its use, so no fence or atomic counter is needed.
#include "kq_internal.h"

namespace kq {

__device__ __forceinline__ float sqdist9u(const float* x, const float* __restrict__ c) {
    float acc = 0.0f;
#pragma unroll
    for (int d = 0; d < kDim; ++d) {
        const float t = x[d] - c[d];
        acc = __fmaf_rn(t, t, acc);
    }
    return acc;
}

struct UpdateCtx {
    unsigned long long* s_sum;  // [krange][9]
    unsigned* s_cnt;            // [krange]
    const float* C_old;
    double scale;               // 2^s of q(x) = rint(x * 2^s)
    int j0, kr;                 // the entry range [j0, j0 + kr)
    bool sums, want_dist;
};

// add one kernel (row x, entry j) to the histogram if j is in the range
__device__ __forceinline__ void add_kernel(const UpdateCtx& c, const float (&x)[kDim], int j, double& dacc) {
    const int jr = j - c.j0;
    if ((unsigned)jr >= (unsigned)c.kr) return;
    if (c.want_dist) dacc += (double)sqdist9u(x, c.C_old + (size_t)j * kDim);
    atomicAdd(&c.s_cnt[jr], 1u);
    if (c.sums) {
#pragma unroll
        for (int d = 0; d < kDim; ++d) atomicAdd(&c.s_sum[jr * kDim + d], fixed_bits(x[d], c.scale));
    }
}

// Thread t takes kernels i, i + 1024, ... (i = first + t): consecutive lanes read
// consecutive 36-byte rows with 9 dword loads each, two kernels in flight per thread; a row
// is loaded only when its entry lies in the workgroup's range (with a single range every
// row is, and the row loads need not wait for the indices).
template <bool NEED_X, bool RANGED>
__device__ __forceinline__ void add_rows(const UpdateCtx& c, const float* __restrict__ X,
                                         const int32_t* __restrict__ idx, int i, int i1, double& dacc) {
    for (; i < i1; i += 2 * kUpdateThreads) {
        const int ib = i + kUpdateThreads;
        const bool two = ib < i1;
        const int ja = idx[i], jb = two ? idx[ib] : -1;  // -1: nothing to add
        const bool ina = !RANGED || (unsigned)(ja - c.j0) < (unsigned)c.kr;
        const bool inb = !RANGED || (unsigned)(jb - c.j0) < (unsigned)c.kr;
        float xa[kDim], xb[kDim];
        if (NEED_X) {
            const float* pa = X + (size_t)i * kDim;
            const float* pb = X + (size_t)(two ? ib : i) * kDim;
#pragma unroll
            for (int d = 0; d < kDim; ++d) {
                xa[d] = ina ? pa[d] : 0.0f;
                xb[d] = inb ? pb[d] : 0.0f;
            }
        } else {
#pragma unroll
            for (int d = 0; d < kDim; ++d) xa[d] = xb[d] = 0.0f;
        }
        add_kernel(c, xa, ja, dacc);
        add_kernel(c, xb, jb, dacc);
    }
}

__global__ __launch_bounds__(kUpdateThreads) void update_kernel(const StackParams p) {
    extern __shared__ unsigned long long s_dyn[];  // [krange][9] sums, then [krange] u32 counts
    __shared__ double s_wd[kUpdateThreads / kWave];
    __shared__ unsigned s_mx;

    const int li = find_layer(p, blockIdx.x);
    const DevLayer& L = p.L[li];
    const int u = blockIdx.x - L.unit_begin;
    const int chunk = u / L.ranges, range = u - chunk * L.ranges;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = L.n, k = L.k;
    UpdateCtx c;
    c.j0 = range * L.krange;
    c.kr = min(k - c.j0, L.krange);
    c.s_sum = s_dyn;
    c.s_cnt = (unsigned*)(s_dyn + (size_t)c.kr * kDim);
    c.C_old = L.C_old;
    c.sums = (L.flags & kFlagCountsOnly) == 0;
    int shift = 0;
    if (c.sums) {  // set by shift_kernel before this launch, or formed here from the block maxima
        if (p.derive_shift) {
            shift = derive_shift<kUpdateThreads>(L, &s_mx);
            if (u == 0 && tid == 0) L.xmax[L.nxmax] = (unsigned)shift;  // for the launches after
        } else {
            shift = (int)L.xmax[L.nxmax];
        }
    }
    c.scale = fixed_scale(shift);
    c.want_dist = L.part != nullptr;
    const bool need_x = c.sums || c.want_dist;

    for (int e = tid; e < c.kr * kDim; e += kUpdateThreads) c.s_sum[e] = 0ull;
    for (int e = tid; e < c.kr; e += kUpdateThreads) c.s_cnt[e] = 0u;
    __syncthreads();

    double dacc = 0.0;
    const int i0 = chunk * L.chunk;
    const int i1 = min(n, i0 + L.chunk);
    if (!need_x)
        add_rows<false, false>(c, L.X, L.idx, i0 + tid, i1, dacc);
    else if (L.ranges == 1)
        add_rows<true, false>(c, L.X, L.idx, i0 + tid, i1, dacc);
    else
        add_rows<true, true>(c, L.X, L.idx, i0 + tid, i1, dacc);

    __syncthreads();
    unsigned long long* __restrict__ out = (unsigned long long*)L.hist + ((size_t)chunk * k + c.j0) * 10;
    for (int e = tid; e < c.kr * 10; e += kUpdateThreads) {
        const int j = e / 10, d = e - 10 * j;
        out[e] = (d == 9) ? (unsigned long long)c.s_cnt[j] : c.s_sum[j * kDim + d];
    }
    if (c.want_dist) {
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) dacc += __shfl_xor(dacc, off);
        if (lane == 0) s_wd[wave] = dacc;
        __syncthreads();
        if (tid == 0) {
            double v = s_wd[0];
            for (int w = 1; w < kUpdateThreads / kWave; ++w) v += s_wd[w];
            L.part[u] = v;
        }
    }
}

constexpr int kFinishGroups = 6;
constexpr int kFinishBatch = 9;
constexpr int kFinishDirectWgs = 16;  // workgroups per layer in the direct form
constexpr int kFinishDirectK = kFinishDirectWgs * kFinishEntries;  // 256
constexpr int kFinishThreads = kFinishEntries * 10 * kFinishGroups;  // 640
static_assert(kFinishThreads >= kSumThreads, "the distortion sum uses the first kSumThreads threads");

__global__ __launch_bounds__(kFinishThreads) void update_finish_kernel(const StackParams p) {
    __shared__ unsigned long long s_S[kFinishGroups][kFinishEntries * 10];
    __shared__ double s_w[kSumThreads / kWave];
    const int b = blockIdx.x;
    // The launch is short, and every dependent load of the arguments is a memory round trip.
    // With every codebook of at most kFinishDirectK entries (p.finish_direct) layer l owns
    // workgroups kFinishDirectWgs l .., so the fields of layer b / kFinishDirectWgs are read in
    // the first batch; otherwise the table of first workgroups gives the layer and its fields
    // come in later batches.
    const int ld = min(b / kFinishDirectWgs, KQ_MAX_STACK - 1);
    const DevLayer& Ld = p.L[ld];
    int k = Ld.k, nb = Ld.nchunks, flags = Ld.flags, nx = Ld.nxmax, ub = Ld.unit_begin;
    const unsigned long long* __restrict__ h = (const unsigned long long*)Ld.hist;
    const unsigned* xm = Ld.xmax;
    const float* C_old = Ld.C_old;
    const int total = p.total_units, direct = p.finish_direct;
    asm volatile("" ::"s"(k), "s"(nb), "s"(flags), "s"(nx), "s"(ub), "s"(h), "s"(xm), "s"(C_old), "s"(total),
                 "s"(direct));
    if (b >= total) {  // the last nlayers workgroups: the distortion of layer b - total
        const DevLayer& L = p.L[b - total];
        double* const dist = L.dist;
        const double *const ap = L.apart, *const pp = L.part;
        const int na = L.napart, nu = L.nunits;
        asm volatile("" ::"s"(dist), "s"(ap), "s"(pp), "s"(na), "s"(nu));
        const double* const src = ap ? ap : pp;
        const int m = ap ? na : nu;
        if (dist == nullptr) return;
        const double a = block_fixed_sum<kSumThreads>(src, m, s_w);
        if (threadIdx.x == 0) *dist = a;
        return;
    }
    const int lt = direct ? ld : find_layer(p, b);  // the layer
    const int li = lt;
    if (!direct) {  // layer and entry range from the table: each layer owns ceil(k / kFinishEntries) workgroups
        const DevLayer& Lt = p.L[lt];
        k = Lt.k;
        nb = Lt.nchunks;
        flags = Lt.flags;
        nx = Lt.nxmax;
        ub = Lt.unit_begin;
        h = (const unsigned long long*)Lt.hist;
        xm = Lt.xmax;
        C_old = Lt.C_old;
    }
    const DevLayer& L = p.L[li];
    const int j0 = (b - ub) * kFinishEntries;
    const int tid = threadIdx.x;
    const int g = tid / (kFinishEntries * 10), v = tid - g * (kFinishEntries * 10);
    const int j = j0 + v / 10, d = v - 10 * (v / 10);
    // the entry's old value and the layer's shift, in flight with the partials
    const bool writes_c = g == 0 && j < k && d < kDim && (flags & kFlagCountsOnly) == 0;
    float old = 0.0f;
    int shift = 0;
    if (writes_c) {
        old = C_old[(size_t)j * kDim + d];
        shift = (int)xm[nx];
    }

    unsigned long long s = 0ull;
    if (j < k) {
        const size_t stride = (size_t)k * 10;
        const unsigned long long* hp = h + (size_t)j * 10 + d;
        // partials g, g + 8, ...: kFinishBatch loads in flight at a time
#pragma unroll 1
        for (int q0 = g; q0 < nb; q0 += kFinishBatch * kFinishGroups) {
            unsigned long long v[kFinishBatch];
#pragma unroll
            for (int r = 0; r < kFinishBatch; ++r) {
                const int q = q0 + r * kFinishGroups;
                v[r] = q < nb ? hp[(size_t)q * stride] : 0ull;
            }
#pragma unroll
            for (int r = 0; r < kFinishBatch; ++r) s += v[r];
        }
    }
    s_S[g][v] = s;
    __syncthreads();
    if (g == 0 && j < k) {
        unsigned long long S = 0, z = 0;  // wrapping sums
#pragma unroll
        for (int q = 0; q < kFinishGroups; ++q) {
            S += s_S[q][v];
            z += s_S[q][(v / 10) * 10 + 9];
        }
        S -= z * kFixedBias;  // the exact sum of q(x) over the entry's kernels
        if (d == 9) {
            if (L.counts) L.counts[j] = (int32_t)z;
        } else if (writes_c) {
            float c = old;
            if (z > 0) {
                const double mean = ((double)(long long)S * ldexp(1.0, -shift)) / (double)z;
                // Eq. (2): c - gamma * mean gradient; Eq. (1): the mean of the kernels
                c = (flags & kFlagGrad) ? (float)((double)old - (double)L.gamma * mean) : (float)mean;
            }
            L.C[(size_t)j * kDim + d] = c;
        }
    }
}

// per-block maximum of |v| over 32768 values of a layer (the kernels, or the gradients of
// Eq. 2) as fp32 bits with the sign cleared: an integer maximum, so a NaN counts as the
// largest value and shift_kernel can flag it.  Blocks of 1024 threads: a grid of many small
// workgroups is slow to dispatch (the last start microseconds after the first)
__global__ __launch_bounds__(kAbsMaxThreads) void absmax_kernel(const StackParams p) {
    __shared__ unsigned s_mx;
    const int li = find_layer(p, blockIdx.x);
    const DevLayer& L = p.L[li];
    const int b = blockIdx.x - L.unit_begin;
    const long long count = (long long)L.n * kDim;
    const long long base = (long long)b * kAbsMaxPerBlock;
    if (threadIdx.x == 0) s_mx = 0u;
    __syncthreads();
    unsigned m = 0u;
    const unsigned* __restrict__ V = reinterpret_cast<const unsigned*>(L.X);
    if ((reinterpret_cast<uintptr_t>(L.X) & 15u) == 0 && base + kAbsMaxPerBlock <= count) {
        // a whole block from a 16-byte aligned tensor: eight 16-byte loads per thread in flight
        const uint4* __restrict__ V4 = reinterpret_cast<const uint4*>(V + base);
        constexpr int kPer = kAbsMaxPerBlock / (4 * kAbsMaxThreads);
        uint4 v[kPer];
#pragma unroll
        for (int u = 0; u < kPer; ++u) v[u] = V4[threadIdx.x + kAbsMaxThreads * u];
#pragma unroll
        for (int u = 0; u < kPer; ++u)
            m = max(m, max(max(v[u].x & 0x7fffffffu, v[u].y & 0x7fffffffu), max(v[u].z & 0x7fffffffu, v[u].w & 0x7fffffffu)));
    } else {
#pragma unroll 4
        for (int q = threadIdx.x; q < kAbsMaxPerBlock; q += kAbsMaxThreads) {
            const long long e = base + q;
            if (e < count) m = max(m, V[e] & 0x7fffffffu);
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, off));
    if ((threadIdx.x & 63) == 0) atomicMax(&s_mx, m);  // LDS
    __syncthreads();
    if (threadIdx.x == 0) L.xmax[b] = s_mx;
}

// one workgroup per layer: the largest of its block maxima gives the layer's shift
// (xmax[nxmax]); range_flags[layer] records whether any value was NaN or infinite
__global__ __launch_bounds__(256) void shift_kernel(const StackParams p) {
    __shared__ unsigned s_mx;
    const DevLayer& L = p.L[blockIdx.x];
    if (threadIdx.x == 0) s_mx = 0u;
    __syncthreads();
    unsigned m = 0u;
    for (int q = threadIdx.x; q < L.nxmax; q += 256) m = max(m, L.xmax[q]);
    atomicMax(&s_mx, m);  // LDS
    __syncthreads();
    if (threadIdx.x == 0) {
        L.xmax[L.nxmax] = (unsigned)layer_shift(s_mx, L.shift);
        if (p.range_flags) p.range_flags[blockIdx.x] = s_mx >= 0x7f800000u ? 1u : 0u;
    }
}

hipError_t launch_absmax(const StackParams& p, hipStream_t s, bool with_shift) {
    StackParams q = p;
    int blk = 0;
    for (int l = 0; l < q.nlayers; ++l) {
        q.L[l].unit_begin = blk;
        blk += q.L[l].nxmax;
    }
    q.total_units = blk;
    set_unit_table(q);
    hipLaunchKernelGGL(absmax_kernel, dim3(blk), dim3(kAbsMaxThreads), 0, s, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !with_shift) return e;
    hipLaunchKernelGGL(shift_kernel, dim3(q.nlayers), dim3(256), 0, s, q);
    return hipGetLastError();
}

__global__ void fill_zero_kernel(uint4* p, size_t n16, unsigned char* tail, size_t ntail) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n16; e += stride) p[e] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0)
        for (size_t e = threadIdx.x; e < ntail; e += blockDim.x) tail[e] = 0;
}

hipError_t launch_update(const StackParams& p, hipStream_t s) {
    size_t lds = 0;
    for (int l = 0; l < p.nlayers; ++l) {
        const size_t b = (size_t)p.L[l].krange * (kDim * sizeof(unsigned long long) + sizeof(unsigned));
        lds = b > lds ? b : lds;
    }
    hipLaunchKernelGGL(update_kernel, dim3(p.total_units), dim3(kUpdateThreads), lds, s, p);
    return hipGetLastError();
}

// the finishing launch numbers its workgroups per layer: ceil(k / 4) each
hipError_t launch_update_finish(const StackParams& p, hipStream_t s) {
    StackParams q = p;
    bool direct = true;  // every codebook fits kFinishDirectWgs workgroups
    for (int l = 0; l < q.nlayers; ++l) direct &= q.L[l].k <= kFinishDirectK;
    q.finish_direct = direct ? 1 : 0;
    int blk = 0;
    for (int l = 0; l < q.nlayers; ++l) {
        q.L[l].unit_begin = blk;
        blk += direct ? kFinishDirectWgs : (q.L[l].k + kFinishEntries - 1) / kFinishEntries;
    }
    q.total_units = blk;  // followed by one workgroup per layer for the distortion
    set_unit_table(q);
    // nunits keeps the number of update workgroups (partials to add)
    hipLaunchKernelGGL(update_finish_kernel, dim3(blk + q.nlayers), dim3(kFinishThreads), 0, s, q);
    return hipGetLastError();
}

hipError_t launch_fill_zero(void* ws, size_t bytes, hipStream_t s) {
    const size_t n16 = bytes / 16;
    unsigned char* tail = (unsigned char*)ws + n16 * 16;
    const size_t ntail = bytes - n16 * 16;
    size_t blocks = (n16 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint4*)ws, n16, tail, ntail);
    return hipGetLastError();
}

}  // namespace kq
