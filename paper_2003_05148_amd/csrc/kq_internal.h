// Internal declarations shared by the HIP translation units of libkq.
// Device-side layer descriptors, workspace layout and the launchers that the
// C-ABI layer (kq_api.hip) calls after it has validated the arguments.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kq.h"

namespace kq {

constexpr int kDim = 9;
constexpr int kWave = 64;

// ---- assignment kernel geometry -----------------------------------------------------
// A workgroup is 4 waves; each wave scores kAssignTilesPerWave tiles of 32 kernels
// against 32-entry codebook tiles with v_mfma_f32_32x32x2f32 (K = 10 = 9 dims + norm).
constexpr int kAssignWaves = 4;
constexpr int kAssignTilesPerWave = 2;
constexpr int kAssignKernelsPerBlock = kAssignWaves * kAssignTilesPerWave * 32;   // 256
constexpr int kAssignChunk = 1024;   // codebook entries staged in LDS at a time

// ---- update kernel geometry ---------------------------------------------------------
constexpr int kUpdateThreads = 256;
constexpr int kUpdateKernelsPerBlock = 4096;
constexpr int kUpdateLdsMaxK = 768;  // LDS histogram [k][9] int64 + [k] u32 up to this k

// ---- squared-error reduction ------------------------------------------------------------
constexpr int kSqThreads = 256;
constexpr int kSqPerBlock = 8192;

inline int assign_blocks(int64_t n) { return (int)((n + kAssignKernelsPerBlock - 1) / kAssignKernelsPerBlock); }
inline int update_blocks(int64_t n) { return (int)((n + kUpdateKernelsPerBlock - 1) / kUpdateKernelsPerBlock); }

inline int sq_error_blocks(int64_t count) { return (int)((count + kSqPerBlock - 1) / kSqPerBlock); }

// fixed-point scale of the exact member sums: q(x) = rint(x * 2^s), s = 57 - ceil(log2 n)
inline int fixed_shift(int64_t n) {
    int c = 0;
    while ((int64_t(1) << c) < n) ++c;
    return 57 - c;
}

// ---- per-layer workspace ---------------------------------------------------------------
//   [0, 256)            : counters (u32 assign, u32 update)
//   [256, +8*assign_blk): fp64 per-block distortion partials
//   [.., +8*10*k)       : int64 accumulators, 9 member sums + 1 count per entry
inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
inline size_t layer_ws_bytes(int64_t n, int32_t k) {
    return 256 + align256(sizeof(double) * (size_t)assign_blocks(n)) + align256(sizeof(int64_t) * 10 * (size_t)k);
}

struct DevLayer {
    const float* X;
    float* C;                 // codebook read by assign / written by update
    const float* C_old;       // update: entries kept when empty
    int32_t* idx;
    float* best_d;
    int32_t* counts;
    double* dist;             // assign: where this call's distortion goes (or null)
    unsigned* ctr;            // [0] assign, [1] update
    double* part;             // assign partials
    unsigned long long* acc;  // update accumulators [k][10]
    int n;
    int k;
    int blk_begin;            // first workgroup of this layer in the launch
    int nblk;                 // workgroups of this layer
    int shift;                // fixed-point scale (update)
    int counts_only;          // update: histogram only, C untouched
};

struct StackParams {
    int nlayers;
    int total_blocks;
    DevLayer L[KQ_MAX_STACK];
};

// device-side: the layer a workgroup belongs to (layers are laid out in order)
__device__ __forceinline__ int find_layer(const StackParams& p, int b) {
    int l = 0;
#pragma unroll 1
    for (int i = 1; i < p.nlayers; ++i)
        if (b >= p.L[i].blk_begin) l = i;
    return l;
}

// launchers (return hipSuccess or the launch error)
hipError_t launch_assign(const StackParams& p, hipStream_t s);
hipError_t launch_update(const StackParams& p, hipStream_t s);
hipError_t launch_fill_zero(void* ws, size_t bytes, hipStream_t s);

struct CbqLayer {
    const float* C;
    const int32_t* w;
    uint8_t* codes;
    float* levels;
    float* C_hat;
    int k;
};
struct CbqParams {
    int nlayers;
    int bits;
    int mode;
    int iters;
    CbqLayer L[KQ_MAX_STACK];
};
hipError_t launch_cbq(const CbqParams& p, hipStream_t s);

hipError_t launch_pack(const void* v, int elem_bytes, int64_t count, int bits, uint8_t* out, hipStream_t s);
hipError_t launch_unpack(const uint8_t* in, int64_t count, int bits, int32_t* v, hipStream_t s);
hipError_t launch_sq_error(const float* A, const float* B, int64_t count, double* out, void* ws, hipStream_t s);
hipError_t launch_reconstruct(const int32_t* idx, const uint8_t* packed, int bits, int64_t n, const float* C,
                              int k, float* W, hipStream_t s);

}  // namespace kq
