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
// A wave scores kAssignTilesPerWave tiles of 32 kernels (a "unit" of 64 kernels, one per
// lane) against 32-entry codebook tiles with v_mfma_f32_32x32x16_bf16 (an exact bf16 split
// of the K = 10 fp32 contraction, 9 dims + norm, into three cross terms).  The grid is
// persistent: one workgroup of kAssignWaves waves per CU (three per SIMD), each walking a
// contiguous run of the stack's units, one unit per wave at a time.
constexpr int kAssignWaves = 12;
constexpr int kAssignTilesPerWave = 2;
// codebook entries staged in LDS at a time by the plain assignment (64 B of operands + 48 B
// of fp32 row each: 112 KB of the CU's 160 KB; codebooks up to this size stay resident, and
// a larger one takes fewer chunks, each costing a staging pass between two barriers)
constexpr int kAssignChunk = 1024;
constexpr int kAssignGridMax = 256;  // the persistent grid: one workgroup per CU

// ---- update kernel geometry ---------------------------------------------------------
// One launch updates every layer of a stack.  A layer's kernels are cut into chunks and
// its codebook into ranges of at most kUpdateLdsMaxK entries (the LDS histogram of one
// range); a workgroup adds the kernels of one chunk whose entry lies in one range.
// Chunks hold about the number of kernels that gives one workgroup per CU for the whole
// launch (a multiple of 256, at least kUpdateMinKernelsPerBlock), and a layer has at
// most update_max_chunks(n, k) of them (that bounds its partial histograms).
constexpr int kUpdateThreads = 1024;
constexpr int kUpdateMinKernelsPerBlock = 1024;
constexpr int kUpdateTargetBlocks = 256;
constexpr int kUpdateLdsMaxK = 768;     // LDS histogram [768][9] int64 + [768] u32
constexpr int kFinishEntries = 16;  // codebook entries per finishing workgroup
constexpr size_t kUpdatePartialBudget = size_t(1) << 24;  // bytes of partials per layer above 768 entries

inline int update_ranges(int32_t k) { return (k + kUpdateLdsMaxK - 1) / kUpdateLdsMaxK; }
inline int update_max_chunks(int64_t n, int32_t k) {
    const int64_t c = (n + kUpdateMinKernelsPerBlock - 1) / kUpdateMinKernelsPerBlock;
    if (k <= kUpdateLdsMaxK) return (int)c;
    int64_t cap = (int64_t)(kUpdatePartialBudget / (sizeof(int64_t) * 10 * (size_t)k));
    if (cap < 1) cap = 1;
    return (int)(c < cap ? c : cap);
}
// kernels per chunk for a launch whose layers weigh `weighted_n` = sum of ranges x n
inline int update_kernels_per_block(int64_t weighted_n) {
    int64_t kpb = (weighted_n / kUpdateTargetBlocks + 255) & ~int64_t(255);
    if (kpb < kUpdateMinKernelsPerBlock) kpb = kUpdateMinKernelsPerBlock;
    if (kpb > (int64_t(1) << 30)) kpb = int64_t(1) << 30;
    return (int)kpb;
}
inline int update_chunk(int64_t n, int32_t k, int kpb) {
    const int64_t mc = update_max_chunks(n, k);
    int64_t cs = ((n + mc - 1) / mc + 255) & ~int64_t(255);
    if (cs < kpb) cs = kpb;
    return (int)cs;
}

// ---- squared-error reduction ------------------------------------------------------------
constexpr int kSqThreads = 256;
constexpr int kSqPerBlock = 8192;

// units of 64 kernels of a layer (one wave's work at a time; one distortion partial each)
inline int assign_units(int64_t n) { return (int)((n + kWave - 1) / kWave); }
// fused partials of a layer: one per workgroup of the layer, at most one per unit
inline int fused_parts(int64_t n) { return assign_units(n) < kAssignGridMax ? assign_units(n) : kAssignGridMax; }
inline int sq_error_blocks(int64_t count) { return (int)((count + kSqPerBlock - 1) / kSqPerBlock); }

// Fixed-point scale of the exact member sums.  A layer's sums use q(x) = rint(x * 2^s) with
//     s = min(62 - ceil(log2 n), 51) - e,   e the smallest integer with max |x| < 2^e (-126
//                                  when the largest magnitude is subnormal, 0 for an
//                                  all-zero layer),
// so |q| < 2^51 and |q| <= 2^(62 - ceil(log2 n)): no sum over at most n values can leave
// int64, while the resolution stays 2^-min(62 - ceil(log2 n), 51) of the layer's largest
// magnitude whatever that magnitude is.  base_shift(n) = min(57 - ceil(log2 n), 46) is s for
// 16 <= max |x| < 32; the device derives s from it and the layer's maxima of |x| (the same
// rule serves the gradient sums of Eq. 2).
inline int base_shift(int64_t n) {
    int c = 0;
    while ((int64_t(1) << c) < n) ++c;
    return 57 - c < 46 ? 57 - c : 46;
}

// q(x) travels in the low bits of a double: fma(x, 2^s, 1.5 * 2^52) rounds x * 2^s to an
// integer (ties to even, as rint) inside the binade [2^52, 2^53), where doubles are one
// apart, so its bit pattern is kFixedBias + q(x) for |q| < 2^51.  Sums of these patterns
// in wrapping 64-bit integer arithmetic, less count * kFixedBias, are the exact sums of q.
// Two full-rate instructions per value (a conversion and an fma in fp64).
constexpr unsigned long long kFixedBias = 0x4338000000000000ull;  // the bits of 1.5 * 2^52
__device__ __forceinline__ double fixed_scale(int shift) { return __builtin_ldexp(1.0, shift); }

// the layer's shift from its largest magnitude (fp32 bits, sign cleared):
// s = base + 5 - e with max < 2^e, where base = min(57 - ceil(log2 n), 46) (e = -126 for a subnormal
// maximum, e = 0 for an all-zero layer; a non-finite maximum gives e >= 129 and a shift
// that keeps the sums finite but meaningless, which KQ_F_VALIDATE reports)
__device__ __forceinline__ int layer_shift(unsigned maxbits, int base) {
    const int be = (int)(maxbits >> 23);                          // biased exponent (255: inf or NaN)
    const int e = maxbits == 0u ? 0 : (be == 0 ? -126 : be - 126);  // max < 2^e
    return base + 5 - e;
}
__device__ __forceinline__ unsigned long long fixed_bits(float x, double scale) {
    return __builtin_bit_cast(unsigned long long, __builtin_fma((double)x, scale, 0x1.8p52));
}

// ---- fused assignment + member sums ------------------------------------------------------
// With every codebook of at most kFuseMaxK entries, the assignment kernel can also add each
// settled kernel to a per-workgroup LDS histogram of exact member sums (the update's
// fixed-point sums) and store it per (layer, workgroup) as a partial, so the update needs
// only its finishing launch.  A layer's partials are those of its workgroups (the grid is
// split per layer; fused_parts(n) at most).
constexpr int kFuseMaxK = 256;
constexpr int kFuseChunk = 256;  // codebook entries staged at a time by the fused variant

// ---- per-layer workspace ---------------------------------------------------------------
//   assign distortion partials : fp64 [assign_units(n)]                          (overwritten each call)
//   update distortion partials : fp64 [ranges * max chunks]                      (overwritten each call)
//   update histograms          : int64 [max chunks][k][10] per-chunk partial sums (overwritten each call)
//   magnitudes                 : u32 [absmax_blocks(n) + 1 + KQ_MAX_STACK] (below)
inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
inline size_t ws_assign_part(int64_t n) { return align256(sizeof(double) * (size_t)assign_units(n)); }
inline size_t ws_update_part(int64_t n, int32_t k) {
    return align256(sizeof(double) * (size_t)update_ranges(k) * (size_t)update_max_chunks(n, k));
}
inline size_t ws_hist(int64_t n, int32_t k) {
    size_t parts = (size_t)update_max_chunks(n, k);
    if (k <= kFuseMaxK && (size_t)fused_parts(n) > parts) parts = (size_t)fused_parts(n);  // fused partials
    return align256(sizeof(int64_t) * 10 * (size_t)k * parts);
}
// Largest magnitudes of the values whose fixed-point sums a call forms (the kernels, or the
// gradients of Eq. 2): one maximum of |v| per block of 32768 values (fp32 bits with the sign
// cleared, so a NaN orders above +inf and every finite value), then the layer's shift, then
// -- used in the first layer's region of a call -- one non-finite flag per layer of the call.
constexpr int kAbsMaxThreads = 1024;
constexpr int kAbsMaxPerBlock = 32 * kAbsMaxThreads;  // eight 16-byte loads per thread
inline int absmax_blocks(int64_t n) { return (int)((n * kDim + kAbsMaxPerBlock - 1) / kAbsMaxPerBlock); }
inline size_t ws_xmax(int64_t n) {
    return align256(sizeof(unsigned) * ((size_t)absmax_blocks(n) + 1 + KQ_MAX_STACK));
}
inline size_t ws_xmax_offset(int64_t n, int32_t k) { return ws_assign_part(n) + ws_update_part(n, k) + ws_hist(n, k); }
inline size_t layer_ws_bytes(int64_t n, int32_t k) { return ws_xmax_offset(n, k) + ws_xmax(n); }

enum : int { kFlagCountsOnly = 1, kFlagGrad = 2 };

struct DevLayer {
    const float* X;
    float* C;                 // assign: the codebook; update: where the new codebook goes
    const float* C_old;       // update: entries kept when empty; the codebook of the assignment
    int32_t* idx;
    float* best_d;
    int32_t* counts;
    double* dist;             // this call's distortion output, or null
    double* part;             // distortion partials (assign: per wave and tile; update: per block)
    const double* apart;      // update finish: the assignment's partials to add instead, or null
    long long* hist;          // update histograms (see the workspace layout)
    int n;
    int k;
    int unit_begin;           // first tile (assign) or workgroup (update) of this layer
    int nunits;               // units or workgroups of this layer
    int shift;                // base_shift(n); the device turns it into the layer's fixed-point shift
    int flags;                // kFlag*
    int napart;               // number of assignment partials
    int ranges;               // update: codebook ranges (workgroups per chunk)
    int krange;               // update: entries per range
    int chunk;                // update: kernels per chunk
    int nchunks;              // update: chunks (= partial histograms)
    float gamma;              // gradient step: learning rate
    unsigned* xmax;           // per-block maxima of |x| (or |g|) as fp32 bits, then the shift (xmax[nxmax])
    int nxmax;                // number of those blocks
    int wfirst;               // fused assignment: the layer's first workgroup
};

// Kernel arguments of a stack launch.  The first unit of every layer is repeated in a
// compact table at the front (INT_MAX past the last layer), so a workgroup finds its
// layer with one scalar load instead of a chain of dependent ones through the layer
// records.
struct StackParams {
    int nlayers;
    int total_units;
    unsigned* range_flags;    // per layer: a non-finite value was seen (absmax launches), or null
    int unit_begin[KQ_MAX_STACK];
    int wg_begin[KQ_MAX_STACK];  // assignment: first workgroup of each layer (0x7fffffff past the last)
    int assign_grid;             // assignment: the number of workgroups
    int finish_direct;           // update finish: layer l owns a fixed block of workgroups
    int derive_shift;            // 1: the shift pass left only the block maxima; a launch that
                                 // needs a layer's shift forms it from them, and one of the
                                 // layer's workgroups stores it at xmax[nxmax] for the launches after
    DevLayer L[KQ_MAX_STACK];
};

// host-side: fill the table from the layer records
inline void set_unit_table(StackParams& p) {
    for (int l = 0; l < KQ_MAX_STACK; ++l) p.unit_begin[l] = l < p.nlayers ? p.L[l].unit_begin : 0x7fffffff;
}

// device-side: the layer's shift from its block maxima (what shift_kernel stores at
// xmax[nxmax]), called by every thread of a workgroup of THREADS threads (two barriers)
template <int THREADS>
__device__ __forceinline__ int derive_shift(const DevLayer& L, unsigned* s_mx) {
    if (threadIdx.x == 0) *s_mx = 0u;
    __syncthreads();
    unsigned m = 0u;
    for (int q = threadIdx.x; q < L.nxmax; q += THREADS) m = max(m, L.xmax[q]);
    if (m != 0u) atomicMax(s_mx, m);  // LDS
    __syncthreads();
    return layer_shift(*s_mx, L.shift);
}

// device-side: the layer a unit (tile or workgroup) belongs to (layers are in order)
__device__ __forceinline__ int find_layer(const StackParams& p, int u) {
    int l = 0;
#pragma unroll
    for (int i = 1; i < KQ_MAX_STACK; ++i) l += u >= p.unit_begin[i] ? 1 : 0;
    return l;
}

// v plus the value that DPP control CTL brings from another lane of the row
template <int CTL>
__device__ __forceinline__ double dpp_add(double v) {
    // every source lane of these row moves exists: no "old" value is needed
    const unsigned plo = __builtin_amdgcn_mov_dpp((unsigned)__double2loint(v), CTL, 0xF, 0xF, true);
    const unsigned phi = __builtin_amdgcn_mov_dpp((unsigned)__double2hiint(v), CTL, 0xF, 0xF, true);
    return v + __hiloint2double((int)phi, (int)plo);
}
// v summed over the 64 lanes by the butterfly of partner offsets 32, 16, 8, 4, 2, 1; every
// lane gets the total and the lanes agree bit for bit.  The partners come from the half and
// row swaps and from DPP moves inside a row, not from LDS permutes.  Offset 4 uses a rotation
// by four lanes, which meets the lane 4 apart or 12 apart; the offset-8 step has already made
// those two equal, so each step adds the same two numbers as a plain exchange would.
__device__ __forceinline__ double wave_sum_f64(double v) {
    unsigned lo = (unsigned)__double2loint(v), hi = (unsigned)__double2hiint(v);
    {
        const auto a = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
        const auto b = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
        v = __hiloint2double((int)b[0], (int)a[0]) + __hiloint2double((int)b[1], (int)a[1]);
    }
    lo = (unsigned)__double2loint(v), hi = (unsigned)__double2hiint(v);
    {
        const auto a = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
        const auto b = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
        v = __hiloint2double((int)b[0], (int)a[0]) + __hiloint2double((int)b[1], (int)a[1]);
    }
    v = dpp_add<0x128>(v);  // row_ror:8
    v = dpp_add<0x124>(v);  // row_ror:4
    v = dpp_add<0x4E>(v);   // quad_perm [2,3,0,1]
    return dpp_add<0xB1>(v);  // quad_perm [1,0,3,2]
}

// Sum of m fp64 values in a fixed order by a workgroup of NT threads (a multiple of 64):
// thread t adds values t, t + NT, ... in turn, each wave combines its lanes with a
// butterfly, and thread 0 adds the wave totals in wave order.  Every thread of the
// workgroup must call it; the result is valid in thread 0.
template <int NT>
__device__ __forceinline__ double block_fixed_sum(const double* __restrict__ src, int m, double* s_w) {
    // (threads NT and up of a larger workgroup take part in the barrier only)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double a = 0.0;
    for (int q = tid; tid < NT && q < m; q += 8 * NT) {  // eight loads in flight, added in order
        double v[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) v[r] = q + r * NT < m ? src[q + r * NT] : 0.0;
#pragma unroll
        for (int r = 0; r < 8; ++r) a += v[r];
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) a += __shfl_xor(a, off);
    if (lane == 0 && tid < NT) s_w[wave] = a;
    __syncthreads();
    double r = 0.0;
    if (tid == 0)
        for (int w = 0; w < NT / 64; ++w) r += s_w[w];
    return r;
}
constexpr int kSumThreads = 640;

// launchers (return hipSuccess or the launch error)
// the assignment's workgroups per layer (every workgroup works on one layer): g[l] =
// ceil(units_l / t) for the smallest t with sum g[l] <= kAssignGridMax; returns the grid
int assign_partition(const int* units, int nlayers, int* g);
hipError_t launch_assign(const StackParams& p, hipStream_t s, bool fused = false, hipEvent_t start = nullptr,
                         hipEvent_t stop = nullptr);
hipError_t launch_assign_finish(const StackParams& p, hipStream_t s);
hipError_t launch_update(const StackParams& p, hipStream_t s);
hipError_t launch_update_finish(const StackParams& p, hipStream_t s);
hipError_t launch_fill_zero(void* ws, size_t bytes, hipStream_t s);
// the block maxima of |x| (or |g|) and, with `with_shift`, each layer's shift and non-finite
// flag; without it the next launch that forms sums derives the shift (StackParams::derive_shift)
hipError_t launch_absmax(const StackParams& p, hipStream_t s, bool with_shift);

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

// 2^bits-level k-means over one large flat set of scalars (fully-connected layers)
constexpr int kFcThreads = 256;
constexpr int kFcGrid = 1024;  // persistent workgroups
struct FcParams {
    const float* v;
    const int32_t* w;      // weight of scalar r: w[r / 9] (a codebook entry's count), or null for 1
    uint8_t* codes;
    float* levels_out;
    float* v_hat;          // levels[codes], or null
    int32_t* rounds_out;   // level updates made, or null
    long long m;
    int bits, iters;
    int thr_mode;          // codes from thresholds: 0 from 2^23 scalars on, 1 never, 2 whenever valid
    float* minmax;         // [grid][3] per-workgroup min, max, smallest nonzero magnitude
    float* range;          // [4] the data's min, max, smallest nonzero magnitude; the bucket scale
    long long* part;       // [grid][levels][12] per-workgroup digits and counts
    long long* S;          // [levels][12] running exact sums and counts
    float* lev;            // [levels] current levels
    float* lev_next;       // [levels] candidate levels
    float* thr;            // [levels] code thresholds of the current levels (last one +inf)
    int* state;            // [0] converged, [1] level updates made, [2] levels unsorted, [3] thresholds valid
    int* wg_changed;       // [grid] a code changed in the workgroup
    unsigned* tbl;         // [kFcBuckets][2] bucket table of the thresholds (range[3] > 0: valid)
};
// threshold rounds: the data range is cut into this many buckets of equal width; a scalar's
// bucket gives the count of the thresholds below the bucket and the first one inside it
constexpr int kFcBuckets = 2048;
int fc_grid(long long m);
inline size_t fc_ws_bytes(long long m, int bits) {
    const size_t G = (size_t)fc_grid(m), nlev = (size_t)1 << bits;
    return align256(sizeof(float) * (3 * G + 4)) + align256(sizeof(long long) * G * nlev * 12) +
           align256(sizeof(long long) * nlev * 12) + 3 * align256(sizeof(float) * nlev) + align256(sizeof(int) * 4) +
           align256(sizeof(int) * G) + align256(sizeof(unsigned) * 2 * kFcBuckets);
}
hipError_t launch_fc_quantize(const FcParams& p, hipStream_t s);

// stack forms of pack and reconstruct (+ squared error): a compact unit table first
struct PackJob {
    const void* v;
    uint8_t* out;
    long long count;
    long long bytes;  // ceil(count * bits / 8)
    int eb;
    int bits;
};
struct PackParams {
    int njobs;
    int pad;
    long long word_begin[KQ_MAX_PACK_JOBS + 1];  // first output word of each job; [njobs] = total
    PackJob J[KQ_MAX_PACK_JOBS];
};
struct ReconLayer {
    const int32_t* idx;
    const uint8_t* packed;
    const float* C;
    float* W;
    const float* W_ref;
    double* part;     // squared-error partials [blocks], or null
    double* out;      // squared error, or null
    long long pbytes; // packed stream bytes
    int n, k, bits, nblk;
};
struct ReconParams {
    int nlayers;
    int total_blocks;
    int unit_begin[KQ_MAX_STACK];  // first workgroup of each layer, INT_MAX past the last
    ReconLayer L[KQ_MAX_STACK];
};
constexpr int kReconThreads = 512;
constexpr int kReconRows = 2048;  // rows per workgroup of the stack reconstruction
constexpr int kReconLdsFloats = 16384;  // codebooks up to this many values are gathered from LDS
inline int recon_blocks(int64_t n) { return (int)((n + kReconRows - 1) / kReconRows); }
hipError_t launch_pack_stack(const PackParams& p, hipStream_t s);
hipError_t launch_reconstruct_stack(const ReconParams& p, hipStream_t s);


// ---- Yinyang assignment ----------------------------------------------------------------
constexpr int kYyMaxGroups = 64;     // groups per codebook (one bit each in a 64-bit mask)
constexpr int kYyEvalChunk = 1024;   // group entries staged in LDS at a time
constexpr int kYyEvalGrid = 2048;    // persistent workgroups of the exact group scan
constexpr int kYyFinalGrid = 8192;   // workgroups of the final decision (grid-stride beyond)
constexpr int kYyGroupRounds = 5;    // Lloyd rounds that group the codebook's entries

// default number of groups for k entries: about 64 entries per group, 1 to 32 groups
inline int yy_default_groups(int32_t k) {
    int t = k / 64;
    return t < 1 ? 1 : (t > 32 ? 32 : t);
}

struct YyParams {
    const float* X;
    const float* C;            // the codebook of this round
    const float* C_prev;       // the codebook of the previous round (drift)
    int32_t* idx;              // current entry in, new entry out
    float* best_d;             // fp32 distance to the entry
    const float* Cg;           // group centres [t][9]
    const int32_t* labels;     // group of every entry [k]
    int32_t* perm;             // entries group by group, ascending inside a group [k]
    int32_t* gstart;           // first position of every group in perm [t + 1]
    float* radius;             // upper bound of the distance of a group's entries to its centre [t]
    double* delta;             // cumulative drift bound of every group [t]
    int32_t* cnt;              // listed pairs per group [t], listed kernels [t]
    float* Lt;                 // stored bounds [t][n]
    float* B1;                 // smallest distance in a scanned group [t][n]
    int32_t* J1;               // its entry [t][n]
    float* B2;                 // second smallest distance in a scanned group [t][n]
    int32_t* lists;            // kernels listed per group [t][n]
    unsigned long long* mask;  // groups to scan per listed kernel [n]
    int32_t* flist;            // listed kernels [n]
    int32_t* wgc;              // per-workgroup list counts, then offsets [t + 1][ceil(n / 256)]
    double* part;              // distortion partials, one per 64 kernels
    long long* stats;          // device [3]: listed kernels, listed pairs, distances evaluated; or null
    int n, k, t, npart;
};
hipError_t launch_yy_group(const YyParams& p, hipStream_t s);
hipError_t launch_yy_bounds_init(const YyParams& p, hipStream_t s);
hipError_t launch_yy_round(const YyParams& p, hipStream_t s);
hipError_t launch_yy_partials(const YyParams& p, hipStream_t s);

hipError_t launch_pack(const void* v, int elem_bytes, int64_t count, int bits, uint8_t* out, hipStream_t s);
hipError_t launch_unpack(const uint8_t* in, int64_t count, int bits, int32_t* v, hipStream_t s);
hipError_t launch_sq_error(const float* A, const float* B, int64_t count, double* out, void* ws, hipStream_t s);

}  // namespace kq
