// Storage form and test-time recovery (Eq. 4 and the end of Sec. 3.2).
//
//   pack:        values -> LSB-first stream of `bits`-bit fields (value i at bit i*bits),
//                one thread per output 32-bit word, so every store is a full aligned word
//                except the partial last one.
//   unpack:      the inverse, one thread per value.
//   reconstruct: W_hat[i][d] = C[idx_i][d], one thread per four consecutive outputs
//                (a 16-byte store), indices either plain int32 or read from a packed
//                stream.  HBM traffic per kernel: 4 bytes of index (or bits/8 packed)
//                + 36 bytes written; the codebook stays in cache.
#include "kq_internal.h"

namespace kq {

__device__ __forceinline__ unsigned load_value(const void* v, int eb, long long i) {
    if (eb == 1) return ((const uint8_t*)v)[i];
    if (eb == 2) return ((const uint16_t*)v)[i];
    return (unsigned)((const int32_t*)v)[i];
}

__global__ void pack_kernel(const void* __restrict__ v, int eb, long long count, int bits,
                            uint8_t* __restrict__ out, long long total_bytes) {
    const long long w = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long nw = (total_bytes + 3) / 4;
    if (w >= nw) return;
    const long long bit0 = w * 32;
    const long long i0 = bit0 / bits;
    long long i1 = (bit0 + 31) / bits;
    if (i1 > count - 1) i1 = count - 1;
    const unsigned mask = (bits >= 32) ? 0xffffffffu : ((1u << bits) - 1u);
    unsigned long long word = 0;
    for (long long i = i0; i <= i1; ++i) {
        const unsigned long long val = load_value(v, eb, i) & mask;
        const long long off = i * bits - bit0;
        word |= off >= 0 ? (val << off) : (val >> (-off));
    }
    const unsigned wd = (unsigned)word;
    if (4 * w + 4 <= total_bytes) {
        ((unsigned*)out)[w] = wd;
    } else {
        for (long long b = 0; 4 * w + b < total_bytes; ++b) out[4 * w + b] = (uint8_t)(wd >> (8 * b));
    }
}

__device__ __forceinline__ int read_packed(const uint8_t* __restrict__ in, int bits, long long i, long long total_bytes) {
    const long long bit = i * bits;
    const long long byte0 = bit >> 3;
    unsigned w = 0;
#pragma unroll
    for (int b = 0; b < 3; ++b)
        if (byte0 + b < total_bytes) w |= (unsigned)in[byte0 + b] << (8 * b);
    return (int)((w >> (bit & 7)) & ((1u << bits) - 1u));
}

__global__ void unpack_kernel(const uint8_t* __restrict__ in, long long count, int bits, int32_t* __restrict__ v,
                              long long total_bytes) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= count) return;
    v[i] = bits ? read_packed(in, bits, i, total_bytes) : 0;
}

__global__ void reconstruct_kernel(const int32_t* __restrict__ idx, const uint8_t* __restrict__ packed, int bits,
                                   long long n, const float* __restrict__ C, int k, float* __restrict__ W,
                                   long long packed_bytes) {
    const long long e = 4 * ((long long)blockIdx.x * blockDim.x + threadIdx.x);
    const long long total = n * kDim;
    if (e >= total) return;
    float o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const long long ee = e + q;
        o[q] = 0.0f;
        if (ee < total) {
            const long long i = ee / kDim;
            const int d = (int)(ee - i * kDim);
            const int j = idx ? idx[i] : (bits ? read_packed(packed, bits, i, packed_bytes) : 0);
            if ((unsigned)j < (unsigned)k) o[q] = C[(size_t)j * kDim + d];
        }
    }
    if (e + 4 <= total) {
        *(float4*)(W + e) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
        for (int q = 0; e + q < total; ++q) W[e + q] = o[q];
    }
}

// sum of squared differences, fp64, fixed order: per-thread strided sums, a
// butterfly inside each wave, waves in order; a second kernel adds the block
// partials in block order.
__global__ __launch_bounds__(kSqThreads) void sq_error_kernel(const float* __restrict__ A, const float* __restrict__ B,
                                                             long long count, double* part) {
    __shared__ double s_w[kSqThreads / kWave];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const long long base = (long long)blockIdx.x * kSqPerBlock;
    double acc = 0.0;
#pragma unroll 4
    for (int q = 0; q < kSqPerBlock / kSqThreads; ++q) {
        const long long e = base + (long long)q * kSqThreads + tid;
        if (e < count) {
            const double d = (double)A[e] - (double)B[e];
            acc += d * d;
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) s_w[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        double v = s_w[0];
        for (int w = 1; w < kSqThreads / kWave; ++w) v += s_w[w];
        part[blockIdx.x] = v;
    }
}

__global__ __launch_bounds__(kWave) void sq_finish_kernel(const double* part, int nblk, double* out) {
    const int lane = threadIdx.x;
    double v = 0.0;
    for (int q = lane; q < nblk; q += kWave) v += part[q];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) *out = v;
}

static unsigned grid_for(long long items, int block) {
    return (unsigned)((items + block - 1) / block);
}

hipError_t launch_pack(const void* v, int eb, int64_t count, int bits, uint8_t* out, hipStream_t s) {
    const long long total = (count * (long long)bits + 7) / 8;
    const long long nw = (total + 3) / 4;
    if (nw == 0) return hipSuccess;
    hipLaunchKernelGGL(pack_kernel, dim3(grid_for(nw, 256)), dim3(256), 0, s, v, eb, (long long)count, bits, out, total);
    return hipGetLastError();
}

hipError_t launch_unpack(const uint8_t* in, int64_t count, int bits, int32_t* v, hipStream_t s) {
    if (count == 0) return hipSuccess;
    const long long total = (count * (long long)bits + 7) / 8;
    hipLaunchKernelGGL(unpack_kernel, dim3(grid_for(count, 256)), dim3(256), 0, s, in, (long long)count, bits, v, total);
    return hipGetLastError();
}

hipError_t launch_reconstruct(const int32_t* idx, const uint8_t* packed, int bits, int64_t n, const float* C, int k,
                              float* W, hipStream_t s) {
    const long long total = n * (long long)kDim;
    const long long threads = (total + 3) / 4;
    const long long pbytes = (n * (long long)bits + 7) / 8;
    hipLaunchKernelGGL(reconstruct_kernel, dim3(grid_for(threads, 256)), dim3(256), 0, s, idx, packed, bits,
                       (long long)n, C, k, W, pbytes);
    return hipGetLastError();
}

hipError_t launch_sq_error(const float* A, const float* B, int64_t count, double* out, void* ws, hipStream_t s) {
    const int nblk = sq_error_blocks(count);
    double* part = (double*)ws;
    hipLaunchKernelGGL(sq_error_kernel, dim3(nblk), dim3(kSqThreads), 0, s, A, B, (long long)count, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sq_finish_kernel, dim3(1), dim3(kWave), 0, s, (const double*)part, nblk, out);
    return hipGetLastError();
}

}  // namespace kq
