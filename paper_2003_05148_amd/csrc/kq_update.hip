// Update step of kernel-level quantization (Sec. 3.1, Eq. 1): every codebook entry
// becomes the mean of its kernel set S_j; an empty set keeps its entry.
//
// The member sums are exact integers: each value is mapped to q(x) = rint(x * 2^s)
// with s = 57 - ceil(log2 n), so |q| < 2^62 / n and no sum over at most n kernels can
// overflow int64 (|x| < 32).  Integer addition is associative, so the sums, and with
// them the new codebook, do not depend on the order in which blocks or lanes add.
//
// A block reads 4096 consecutive kernels of one layer (36-byte rows + the index),
// accumulates a private LDS histogram ([k][9] int64 sums + [k] counts, ds_add_u64),
// and flushes its non-zero bins into the layer's [k][10] int64 accumulators with
// global atomics.  Entries above kUpdateLdsMaxK skip the LDS stage and add straight
// to the global accumulators.  The last block of a layer to finish (atomicInc on a
// self-resetting counter) divides, writes the codebook and counts and zeroes the
// accumulators for the next call.
#include "kq_internal.h"

namespace kq {

__global__ __launch_bounds__(kUpdateThreads) void update_kernel(const StackParams p) {
    __shared__ unsigned long long s_sum[kUpdateLdsMaxK * kDim];
    __shared__ unsigned s_cnt[kUpdateLdsMaxK];
    __shared__ int s_last;

    const int li = find_layer(p, blockIdx.x);
    const DevLayer& L = p.L[li];
    const int lb = blockIdx.x - L.blk_begin;
    const int tid = threadIdx.x;
    const int n = L.n, k = L.k;
    const bool use_lds = k <= kUpdateLdsMaxK;
    const bool sums = !L.counts_only;
    const double scale = ldexp(1.0, L.shift);
    const float* __restrict__ X = L.X;
    const int32_t* __restrict__ idx = L.idx;
    unsigned long long* __restrict__ acc = L.acc;

    if (use_lds) {
        for (int e = tid; e < k * kDim; e += kUpdateThreads) s_sum[e] = 0ull;
        for (int e = tid; e < k; e += kUpdateThreads) s_cnt[e] = 0u;
        __syncthreads();
    }

    const int i0 = lb * kUpdateKernelsPerBlock;
    const int i1 = min(n, i0 + kUpdateKernelsPerBlock);
#pragma unroll 2
    for (int i = i0 + tid; i < i1; i += kUpdateThreads) {
        const int j = idx[i];
        if ((unsigned)j >= (unsigned)k) continue;
        float x[kDim];
        if (sums) {
#pragma unroll
            for (int d = 0; d < kDim; ++d) x[d] = X[(size_t)i * kDim + d];
        }
        if (use_lds) {
            atomicAdd(&s_cnt[j], 1u);
            if (sums) {
#pragma unroll
                for (int d = 0; d < kDim; ++d)
                    atomicAdd(&s_sum[j * kDim + d], (unsigned long long)__double2ll_rn((double)x[d] * scale));
            }
        } else {
            atomicAdd(&acc[(size_t)j * 10 + 9], 1ull);
            if (sums) {
#pragma unroll
                for (int d = 0; d < kDim; ++d)
                    atomicAdd(&acc[(size_t)j * 10 + d], (unsigned long long)__double2ll_rn((double)x[d] * scale));
            }
        }
    }

    if (use_lds) {
        __syncthreads();
        for (int e = tid; e < k * 10; e += kUpdateThreads) {
            const int j = e / 10, d = e - 10 * (e / 10);
            const unsigned long long v = (d == 9) ? (unsigned long long)s_cnt[j] : s_sum[j * kDim + d];
            if (v) atomicAdd(&acc[e], v);
        }
    }

    // the last block of the layer finalises (counter wraps back to 0 by itself)
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const unsigned old = atomicInc(&L.ctr[1], (unsigned)(L.nblk - 1));
        s_last = (old == (unsigned)(L.nblk - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const double inv_scale = ldexp(1.0, -L.shift);
    for (int j = tid; j < k; j += kUpdateThreads) {
        unsigned long long* a = acc + (size_t)j * 10;
        const long long z = (long long)__builtin_nontemporal_load(a + 9);
        if (L.counts) L.counts[j] = (int32_t)z;
        if (sums) {
#pragma unroll
            for (int d = 0; d < kDim; ++d) {
                float c;
                if (z > 0) {
                    const long long S = (long long)__builtin_nontemporal_load(a + d);
                    c = (float)(((double)S * inv_scale) / (double)z);
                } else {
                    c = L.C_old[(size_t)j * kDim + d];
                }
                L.C[(size_t)j * kDim + d] = c;
            }
        }
#pragma unroll
        for (int d = 0; d < 10; ++d) a[d] = 0ull;
    }
}

__global__ void fill_zero_kernel(uint4* p, size_t n16, unsigned char* tail, size_t ntail) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n16; e += stride) p[e] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0)
        for (size_t e = threadIdx.x; e < ntail; e += blockDim.x) tail[e] = 0;
}

hipError_t launch_update(const StackParams& p, hipStream_t s) {
    hipLaunchKernelGGL(update_kernel, dim3(p.total_blocks), dim3(kUpdateThreads), 0, s, p);
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
