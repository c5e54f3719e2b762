// Storage form and test-time recovery (Eq. 4 and the end of Sec. 3.2).
//
//   pack:        values -> LSB-first stream of `bits`-bit fields (value i at bit i*bits),
//                one thread per output 32-bit word, so every store is a full aligned word
//                except the partial last one.
//   unpack:      the inverse, one thread per value.
//   reconstruct: W_hat[i][d] = C[idx_i][d] for the layers of a stack in one launch (a
//                single layer is a stack of one), 64 rows per wave step written with
//                coalesced accesses, indices either plain int32 or read from a packed
//                stream, the codebook gathered from LDS.  HBM traffic per kernel: 4 bytes of index (or bits/8 packed)
//                + 36 bytes written (+ 36 bytes read when the squared error against
//                the original row is asked for).
//   pack stack:  one launch for the streams of a whole network.
#include "kq_internal.h"

namespace kq {

__device__ __forceinline__ unsigned load_value(const void* v, int eb, long long i) {
    if (eb == 1) return ((const uint8_t*)v)[i];
    if (eb == 2) return ((const uint16_t*)v)[i];
    return (unsigned)((const int32_t*)v)[i];
}

// output word w of a stream: the fields overlapping bits [32 w, 32 w + 32)
__device__ __forceinline__ void pack_word(const void* __restrict__ v, int eb, long long count, int bits,
                                          uint8_t* __restrict__ out, long long total_bytes, long long w) {
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

__global__ void pack_kernel(const void* __restrict__ v, int eb, long long count, int bits,
                            uint8_t* __restrict__ out, long long total_bytes) {
    const long long w = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= (total_bytes + 3) / 4) return;
    pack_word(v, eb, count, bits, out, total_bytes, w);
}

// every stream of a stack: one thread per output word of the concatenated streams
__global__ void pack_stack_kernel(const PackParams p) {
    const long long wg = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (wg >= p.word_begin[p.njobs]) return;
    // the last job starting at or before wg (jobs without words start where the next does)
    int jb = 0;
#pragma unroll
    for (int q = 1; q < KQ_MAX_PACK_JOBS; ++q) jb += wg >= p.word_begin[q] ? 1 : 0;
    const PackJob& J = p.J[jb];
    pack_word(J.v, J.eb, J.count, J.bits, J.out, J.bytes, wg - p.word_begin[jb]);
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

// Every layer of a stack: workgroup b of a layer rebuilds rows [2048 b, 2048 b + 2048) of
// W_hat.  Each wave takes 64 consecutive rows (576 floats, 2304 bytes) per step and works
// in the coalesced layout: lane l handles floats l + 64 q (q < 9) of the step, which are
// dimension (l + 64 q) % 9 of row (l + 64 q) / 9.  Lane r first obtains the index of row r
// (an int32 load, or its field of the packed stream: the step's 8 * bits bytes are loaded
// as dwords by the first 2 * bits lanes and each lane extracts its field with two
// ds_bpermute); each float then takes its row's index from that row's lane (ds_bpermute)
// and gathers its value from the codebook, copied into LDS first when it holds at most
// kReconLdsFloats values (48-byte rows).  Loads and stores are all full 256-byte wave accesses, and the
// next step's index and reference values load while the current step is rebuilt.  When the
// layer asks for it, each lane also sums (W_ref - W_hat)^2 in fp64 over its floats in a
// fixed order; the lanes of a wave are combined by a butterfly, the waves in order, and a
// second kernel adds the workgroup partials in order.

constexpr int kReconRowFloats = 12;  // staged codebook rows: 9 values, padded to 48 bytes

// the index of the step's row `lane` (rows b0 .. b0 + cnt - 1), or -1 past the end of the layer
__device__ __forceinline__ int recon_step_index(const ReconLayer& L, int b0, int cnt, int lane) {
    if (L.idx) return lane < cnt ? L.idx[b0 + lane] : -1;
    const int b = L.bits;
    if (b == 0) return lane < cnt ? 0 : -1;
    // dwords [2 b s, 2 b s + 2 b) of the stream hold the step's fields (b0 = 64 s)
    const long long w = (long long)(b0 / kWave) * 2 * b + lane;
    unsigned dw = 0;
    if (lane < 2 * b) {
        if (4 * w + 4 <= L.pbytes) {
            dw = ((const unsigned*)L.packed)[w];
        } else {  // the stream's last, partial dword
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (4 * w + t < L.pbytes) dw |= (unsigned)L.packed[4 * w + t] << (8 * t);
        }
    }
    const int bit = lane * b, wi = bit >> 5, o = bit & 31;
    const unsigned lo = (unsigned)__builtin_amdgcn_ds_bpermute(wi * 4, (int)dw);
    const unsigned hi = (unsigned)__builtin_amdgcn_ds_bpermute((wi + 1) * 4, (int)dw);
    const unsigned v = (unsigned)((((unsigned long long)hi << 32) | lo) >> o) & ((1u << b) - 1u);
    return lane < cnt ? (int)v : -1;
}

struct ReconStep {
    int j;             // index of this lane's row
    float x[kDim];     // reference floats l + 64 q of the step
};

__device__ __forceinline__ void recon_load(ReconStep& s, const ReconLayer& L, int b0, int cnt, int lane, bool err) {
    s.j = recon_step_index(L, b0, cnt, lane);
    if (!err) return;
    const float* __restrict__ ref = L.W_ref + (size_t)b0 * kDim;
    if (cnt == kWave) {
#pragma unroll
        for (int q = 0; q < kDim; ++q) s.x[q] = ref[lane + kWave * q];
    } else {
        const int nf = cnt * kDim;
#pragma unroll
        for (int q = 0; q < kDim; ++q) s.x[q] = lane + kWave * q < nf ? ref[lane + kWave * q] : 0.0f;
    }
}

// The steps of one wave.  LDS selects where the codebook is gathered from; the two
// cases are separate instantiations so that the LDS gathers are ds_read instructions
// (a generic pointer that may point into LDS compiles to FLAT loads, whose LDS
// aperture is decided from the address before the instruction offset is added).
template <bool LDS>
__device__ __forceinline__ double recon_steps(const ReconLayer& L, const float* __restrict__ s_cb, int i0, int i1,
                                              int lane, int wave, bool err) {
    constexpr int kWaves = kReconThreads / kWave;
    int src[kDim], dim[kDim];  // row lane (byte address for ds_bpermute) and dimension of float q
#pragma unroll
    for (int q = 0; q < kDim; ++q) {
        const int f = lane + kWave * q, r = f / kDim;
        src[q] = r * 4;
        dim[q] = f - kDim * r;
    }
    const int nsteps = (i1 - i0 + kWave - 1) / kWave;
    double acc = 0.0;
    int st = wave;
    if (st >= nsteps) return acc;
    ReconStep cur, nxt;
    recon_load(cur, L, i0 + st * kWave, min(kWave, i1 - i0 - st * kWave), lane, err);
    for (;;) {
        const int b0 = i0 + st * kWave;
        const int cnt = min(kWave, i1 - b0), nf = cnt * kDim;
        const int sn = st + kWaves;
        const bool more = sn < nsteps;
        if (more) recon_load(nxt, L, i0 + sn * kWave, min(kWave, i1 - i0 - sn * kWave), lane, err);
        float* __restrict__ out = L.W + (size_t)b0 * kDim;
#pragma unroll
        for (int q = 0; q < kDim; ++q) {
            const int jq = __builtin_amdgcn_ds_bpermute(src[q], cur.j);
            float v = 0.0f;
            if ((unsigned)jq < (unsigned)L.k) v = LDS ? s_cb[jq * kReconRowFloats + dim[q]] : L.C[jq * kDim + dim[q]];
            if (lane + kWave * q < nf) {
                __builtin_nontemporal_store(v, &out[lane + kWave * q]);  // streamed, not re-read here
                if (err) {
                    const double df = (double)cur.x[q] - (double)v;
                    acc += df * df;
                }
            }
        }
        if (!more) break;
        cur = nxt;
        st = sn;
    }
    return acc;
}

// The same with 16-byte accesses, for W_hat (and W_ref) aligned to 16 bytes: lane r gathers
// its row's codeword (three ds_read_b128 from 48-byte rows) into the wave's stage, a
// 576-float row-major tile of the step (rows 9 dwords apart: no bank conflicts), and the
// tile leaves as 144 float4 stores (lane l takes float4s l, l + 64, l + 128), with the
// reference read as the same float4s for the error.
typedef float rf32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void recon_ref4(rf32x4 (&x)[3], const ReconLayer& L, int b0, int nf, int lane) {
    const float* __restrict__ ref = L.W_ref + (size_t)b0 * kDim;
#pragma unroll
    for (int u = 0; u < 3; ++u) {
        const int t = lane + kWave * u;
        if (4 * t + 4 <= nf) {
            x[u] = reinterpret_cast<const rf32x4*>(ref)[t];
        } else {
            rf32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * t + e < nf) v[e] = ref[4 * t + e];
            x[u] = v;
        }
    }
}

template <bool LDS>
__device__ __forceinline__ double recon_steps_vec(const ReconLayer& L, const float* __restrict__ s_cb,
                                                  float* __restrict__ s_st, int i0, int i1, int lane, int wave,
                                                  bool err) {
    constexpr int kWaves = kReconThreads / kWave;
    const int nsteps = (i1 - i0 + kWave - 1) / kWave;
    double acc = 0.0;
    int st = wave;
    if (st >= nsteps) return acc;
    int j = recon_step_index(L, i0 + st * kWave, min(kWave, i1 - i0 - st * kWave), lane);
    rf32x4 xr[3];
    if (err) recon_ref4(xr, L, i0 + st * kWave, min(kWave, i1 - i0 - st * kWave) * kDim, lane);
    for (;;) {
        const int b0 = i0 + st * kWave;
        const int nf = min(kWave, i1 - b0) * kDim;
        const int sn = st + kWaves;
        const bool more = sn < nsteps;
        int jn = 0;
        rf32x4 xn[3];
        if (more) {
            jn = recon_step_index(L, i0 + sn * kWave, min(kWave, i1 - i0 - sn * kWave), lane);
            if (err) recon_ref4(xn, L, i0 + sn * kWave, min(kWave, i1 - i0 - sn * kWave) * kDim, lane);
        }
        float c[kDim];  // this lane's row (zeros for an index outside the codebook)
        if ((unsigned)j < (unsigned)L.k) {
            if (LDS) {
                const rf32x4* __restrict__ r = reinterpret_cast<const rf32x4*>(s_cb) + (size_t)j * 3;
                const rf32x4 r0 = r[0], r1 = r[1], r2 = r[2];
                c[0] = r0[0]; c[1] = r0[1]; c[2] = r0[2]; c[3] = r0[3];
                c[4] = r1[0]; c[5] = r1[1]; c[6] = r1[2]; c[7] = r1[3];
                c[8] = r2[0];
            } else {
#pragma unroll
                for (int d = 0; d < kDim; ++d) c[d] = L.C[(size_t)j * kDim + d];
            }
        } else {
#pragma unroll
            for (int d = 0; d < kDim; ++d) c[d] = 0.0f;
        }
#pragma unroll
        for (int d = 0; d < kDim; ++d) s_st[lane * kDim + d] = c[d];
        float* __restrict__ out = L.W + (size_t)b0 * kDim;
#pragma unroll
        for (int u = 0; u < 3; ++u) {
            const int t = lane + kWave * u;
            if (4 * t >= nf) continue;
            const rf32x4 v = reinterpret_cast<const rf32x4*>(s_st)[t];
            if (4 * t + 4 <= nf) {
                __builtin_nontemporal_store(v, reinterpret_cast<rf32x4*>(out) + t);  // streamed, not re-read here
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * t + e < nf) __builtin_nontemporal_store(v[e], out + 4 * t + e);
            }
            if (err) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * t + e < nf) {
                        const double df = (double)xr[u][e] - (double)v[e];
                        acc += df * df;
                    }
            }
        }
        if (!more) break;
        j = jn;
#pragma unroll
        for (int u = 0; u < 3; ++u) xr[u] = xn[u];
        st = sn;
    }
    return acc;
}

__global__ __launch_bounds__(kReconThreads) void reconstruct_stack_kernel(const ReconParams p) {
    extern __shared__ __attribute__((aligned(16))) float s_cb[];  // the codebook in 48-byte rows when it is staged, then the waves' stages
    __shared__ double s_w[kReconThreads / kWave];
    constexpr int kWaves = kReconThreads / kWave;
    int li = 0;
#pragma unroll
    for (int q = 1; q < KQ_MAX_STACK; ++q) li += (int)blockIdx.x >= p.unit_begin[q] ? 1 : 0;
    const ReconLayer& L = p.L[li];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lb = (int)blockIdx.x - p.unit_begin[li];
    const int i0 = lb * kReconRows;
    const int i1 = min(L.n, i0 + kReconRows);
    const bool err = L.part != nullptr;
    const bool staged = L.k * kReconRowFloats <= kReconLdsFloats;
    // 16-byte stores where W_hat (and W_ref) allow them
    const bool vec = ((reinterpret_cast<uintptr_t>(L.W) | (err ? reinterpret_cast<uintptr_t>(L.W_ref) : 0)) & 15u) == 0;
    float* s_st = s_cb + (staged ? L.k * kReconRowFloats : 0) + wave * kWave * kDim;
    double acc;
    if (staged) {
        for (int e = tid; e < L.k * kDim; e += kReconThreads) s_cb[(e / kDim) * kReconRowFloats + e % kDim] = L.C[e];
        __syncthreads();
        acc = vec ? recon_steps_vec<true>(L, s_cb, s_st, i0, i1, lane, wave, err)
                  : recon_steps<true>(L, s_cb, i0, i1, lane, wave, err);
    } else {
        acc = vec ? recon_steps_vec<false>(L, s_cb, s_st, i0, i1, lane, wave, err)
                  : recon_steps<false>(L, s_cb, i0, i1, lane, wave, err);
    }
    if (!err) return;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) s_w[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        double v = s_w[0];
        for (int q = 1; q < kWaves; ++q) v += s_w[q];
        L.part[lb] = v;
    }
}

// one wave per layer: the partials in the order of sq_finish_kernel
__global__ __launch_bounds__(kWave) void reconstruct_stack_finish_kernel(const ReconParams p) {
    const ReconLayer& L = p.L[blockIdx.x];
    if (L.part == nullptr) return;
    const int lane = threadIdx.x;
    double v = 0.0;
    for (int q = lane; q < L.nblk; q += kWave) v += L.part[q];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) *L.out = v;
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

hipError_t launch_pack_stack(const PackParams& p, hipStream_t s) {
    const long long words = p.word_begin[p.njobs];
    if (words == 0) return hipSuccess;
    hipLaunchKernelGGL(pack_stack_kernel, dim3(grid_for(words, 256)), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_reconstruct_stack(const ReconParams& p, hipStream_t s) {
    size_t lds = 0;  // the largest codebook that is staged (48-byte rows), then the waves' stages
    for (int l = 0; l < p.nlayers; ++l) {
        const size_t f = (size_t)p.L[l].k * kReconRowFloats;
        if (f <= (size_t)kReconLdsFloats && f * sizeof(float) > lds) lds = f * sizeof(float);
    }
    lds += sizeof(float) * kReconThreads * kDim;
    hipLaunchKernelGGL(reconstruct_stack_kernel, dim3(p.total_blocks), dim3(kReconThreads), lds, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    bool any = false;
    for (int l = 0; l < p.nlayers; ++l) any |= p.L[l].part != nullptr;
    if (!any) return hipSuccess;
    hipLaunchKernelGGL(reconstruct_stack_finish_kernel, dim3(p.nlayers), dim3(kWave), 0, s, p);
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
