// Kernel codebook quantization (Sec. 3.2): every scalar of a layer's codebook is
// coded with one of 2^bits fp32 levels found by k-means over those scalars, each
// scalar weighted by the appearance count of its codebook entry.
//
// One workgroup per layer.  The weighted sums are exact: a scalar v = M 2^e (fp32)
// times its integer weight w is the integer w M shifted to a fixed position, split
// into 32-bit digits and added to per-level int64 digit accumulators in LDS
// (ds_add_u64).  Integer addition makes the sums independent of the order of the
// work; the exact sum is then rounded once to fp64 (round to nearest even), divided
// by the exact weight total in fp64 and rounded to fp32.  Grid, codes and level
// updates use only correctly rounded fp64 operations, so the codes and levels are
// a pure function of the codebook and the weights.
#include <type_traits>

#include "kq_internal.h"

namespace kq {

constexpr int kCbqThreads = 1024;
constexpr int kCbqMaxLevels = 256;
constexpr int kDigits = 11;  // 32-bit digits: |sum of w v| * 2^149 < 2^328

// smallest q minimising fl64(|v - L_q|), by scanning every level
__device__ __forceinline__ int nearest_level(float v, const float* lev, int nlev) {
    const double vd = (double)v;
    double best = fabs(vd - (double)lev[0]);
    int bq = 0;
    for (int q = 1; q < nlev; ++q) {
        const double d = fabs(vd - (double)lev[q]);
        if (d < best) {
            best = d;
            bq = q;
        }
    }
    return bq;
}

// the same, kept as a loop (for rare rounds, where a fully unrolled scan would only cost registers)
__device__ __forceinline__ int nearest_level_loop(float v, const float* lev, int nlev) {
    const double vd = (double)v;
    double best = fabs(vd - (double)lev[0]);
    int bq = 0;
#pragma unroll 1
    for (int q = 1; q < nlev; ++q) {
        const double d = fabs(vd - (double)lev[q]);
        if (d < best) {
            best = d;
            bq = q;
        }
    }
    return bq;
}

// the same when the levels are sorted (L_0 <= L_1 <= ...): the distances in fp64 do not
// grow towards v from either side, so the answer is the first level >= v or, if not
// farther, the lowest-indexed level whose distance equals that of the last level < v
__device__ __forceinline__ int nearest_sorted(float v, const float* lev, int nlev) {
    int q0 = 0;  // number of levels < v (a prefix, as the levels are sorted)
#pragma unroll
    for (int step = kCbqMaxLevels; step >= 1; step >>= 1)
        if (q0 + step <= nlev && lev[q0 + step - 1] < v) q0 += step;
    const double vd = (double)v;
    int q = q0;
    const double da = q0 < nlev ? fabs(vd - (double)lev[q0]) : __builtin_inf();
    if (q0 > 0) {
        int b = q0 - 1;
        const double db = fabs(vd - (double)lev[b]);
        while (b > 0 && fabs(vd - (double)lev[b - 1]) == db) --b;
        if (db <= da) q = b;
    }
    return q;
}

// add w * v * 2^149 (an exact integer) to the digit accumulators of one level
__device__ __forceinline__ void add_exact(unsigned long long* dig, float v, unsigned w) {
    const unsigned u = __float_as_uint(v);
    const unsigned e = (u >> 23) & 0xffu;
    const unsigned mant = u & 0x7fffffu;
    const unsigned M = e ? (mant | 0x800000u) : mant;
    const int sh = e ? (int)e - 1 : 0;  // v * 2^149 = M * 2^sh
    const unsigned long long P = (unsigned long long)w * M;  // < 2^55
    if (P == 0) return;
    const int d0 = sh >> 5, b = sh & 31;
    const unsigned long long lo = P << b;
    const unsigned long long hi = b ? (P >> (64 - b)) : 0ull;
    long long t0 = (long long)(lo & 0xffffffffull), t1 = (long long)(lo >> 32), t2 = (long long)hi;
    if (u >> 31) {
        t0 = -t0;
        t1 = -t1;
        t2 = -t2;
    }
    atomicAdd(&dig[d0], (unsigned long long)t0);
    atomicAdd(&dig[d0 + 1], (unsigned long long)t1);
    if (t2) atomicAdd(&dig[d0 + 2], (unsigned long long)t2);
}

// the exact integer sum_i dig[i] 2^(32 i), times 2^-149, rounded to nearest-even fp64
// (every loop has a fixed trip count, so the limbs stay in registers)
__device__ double digits_to_double(const unsigned long long* dig) {
    unsigned limb[kDigits + 1];
    long long carry = 0;
#pragma unroll
    for (int i = 0; i < kDigits; ++i) {
        const long long t = (long long)dig[i] + carry;
        limb[i] = (unsigned)(t & 0xffffffffll);
        carry = t >> 32;
    }
    limb[kDigits] = (unsigned)carry;
    const bool neg = carry < 0;
    if (neg) {  // two's complement negate
        unsigned c = 1;
#pragma unroll
        for (int i = 0; i <= kDigits; ++i) {
            const unsigned long long t = (unsigned long long)(~limb[i]) + c;
            limb[i] = (unsigned)t;
            c = (unsigned)(t >> 32);
        }
    }
    int h = -1;  // highest nonzero limb
#pragma unroll
    for (int i = 0; i <= kDigits; ++i) h = limb[i] ? i : h;
    if (h < 0) return 0.0;
    unsigned top = 0, l1 = 0, next = 0;
    bool sticky = false;
#pragma unroll
    for (int i = 0; i <= kDigits; ++i) {
        top = i == h ? limb[i] : top;
        l1 = i == h - 1 ? limb[i] : l1;
        next = i == h - 2 ? limb[i] : next;
        sticky |= (i <= h - 3) && limb[i] != 0u;
    }
    const int lz = __clz(top);
    const unsigned long long hi64 = ((unsigned long long)top << 32) | l1;
    unsigned long long win;
    if (lz) {
        win = (hi64 << lz) | (unsigned long long)(next >> (32 - lz));
        sticky |= (next << lz) != 0u;
    } else {
        win = hi64;
        sticky |= next != 0u;
    }
    unsigned long long mant = win >> 11;
    const unsigned rnd = (unsigned)(win & 0x7ffull);
    if (rnd > 0x400u || (rnd == 0x400u && (sticky || (mant & 1ull)))) ++mant;
    const int pos = 32 * h + 31 - lz;  // bit index of the leading one
    const double r = ldexp((double)mant, pos - 52 - 149);
    return neg ? -r : r;
}

// Nearest level of x among NLEV sorted levels (the answer of nearest_sorted): the number
// of levels below x from every eighth level (registers) and one block of eight (LDS), then
// the exact fp64 comparison of the two neighbours, walking down over equal distances.
template <int NLEV>
__device__ __forceinline__ int nearest_sorted_fast(float x, const float* s_lev, const float (&coarse)[NLEV / 8 + 1]) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    int q0;
    if (NLEV >= 8) {
        int c = 0;
        if (NLEV == 64) {  // sorted: three branch-free halving steps and a check of the last
            const bool h4 = coarse[3] < x;
            const bool h2 = (h4 ? coarse[5] : coarse[1]) < x;
            const bool h1 = (h4 ? (h2 ? coarse[6] : coarse[4]) : (h2 ? coarse[2] : coarse[0])) < x;
            c = (h4 ? 4 : 0) + (h2 ? 2 : 0) + (h1 ? 1 : 0);
            c += (c == 7 && coarse[7] < x) ? 1 : 0;
        } else {
#pragma unroll
            for (int i = 0; i < NLEV / 8; ++i) c += coarse[i] < x ? 1 : 0;
        }
        if (c == NLEV / 8) {
            q0 = NLEV;  // the last level is below x, and with it every level
        } else {
            // the block's last level is coarse[c], not below x: halving steps over the other seven
            const f32x4 a = reinterpret_cast<const f32x4*>(s_lev)[2 * c];
            const f32x4 b = reinterpret_cast<const f32x4*>(s_lev)[2 * c + 1];
            const bool f4 = a[3] < x;
            const bool f2 = (f4 ? b[1] : a[1]) < x;
            const bool f1 = (f4 ? (f2 ? b[2] : b[0]) : (f2 ? a[2] : a[0])) < x;
            q0 = 8 * c + (f4 ? 4 : 0) + (f2 ? 2 : 0) + (f1 ? 1 : 0);
        }
    } else {
        q0 = 0;
#pragma unroll
        for (int i = 0; i < NLEV; ++i) q0 += s_lev[i] < x ? 1 : 0;
    }
    const double vd = (double)x;
    int q = q0;
    const double da = q0 < NLEV ? fabs(vd - (double)s_lev[q0]) : __builtin_inf();
    if (q0 > 0) {
        int bq = q0 - 1;
        const double db = fabs(vd - (double)s_lev[bq]);
        while (bq > 0 && fabs(vd - (double)s_lev[bq - 1]) == db) --bq;
        if (db <= da) q = bq;
    }
    return q;
}

// Code thresholds.  With sorted levels the code of v (nearest level, lowest index on
// ties, fp64 distances) never decreases as v grows: the distance to a lower level only
// grows and to a higher one only shrinks.  So code(v) = the number of q < nlev - 1 with
// t_q <= v, where t_q is the smallest fp32 value whose code exceeds q (+inf if none).
// t_q is found by bisection over the fp32 values in their order, evaluating code() with
// nearest_sorted; afterwards each scalar needs only fp32 comparisons.
__device__ __forceinline__ unsigned ordered_key(float f) {
    const unsigned u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(unsigned k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}
// Searched within the data range [vmin, vmax] only, and used only where every fp64
// distance |v - L| there is exact (see exact_floor): rounding could otherwise make
// distances to distinct levels equal for far values and send them to a lower index.
// The boundary lies next to the midpoint of levels q and q + 1, so the search starts there:
// it steps away from the midpoint by 1, 2, 4, ... keys until the code crosses q, then
// bisects the last step.  Every probe keeps code(lo) <= q < code(hi), and the code does not
// decrease with the value, so the answer is the same as bisecting [vmin, vmax] from the
// start; the midpoint only saves probes (about 5 instead of 32).
__device__ float code_threshold(int q, const float* lev, int nlev, float vmin, float vmax) {
    unsigned lo = ordered_key(vmin), hi = ordered_key(vmax);
    auto above = [&](unsigned key) { return nearest_sorted(key_value(key), lev, nlev) > q; };
    if (!above(hi)) return __builtin_inff();
    if (above(lo)) return key_value(lo);
    if (q + 1 < nlev) {
        const unsigned g = ordered_key((float)(0.5 * ((double)lev[q] + (double)lev[q + 1])));
        if (g > lo && g < hi) {
            if (above(g)) {  // the boundary is at g or below: step down from g
                hi = g;
                for (unsigned st = 1u; hi - lo > st; st *= 2u) {
                    if (!above(hi - st)) {
                        lo = hi - st;
                        break;
                    }
                    hi -= st;
                }
            } else {  // above g: step up from g
                lo = g;
                for (unsigned st = 1u; hi - lo > st; st *= 2u) {
                    if (above(lo + st)) {
                        hi = lo + st;
                        break;
                    }
                    lo += st;
                }
            }
        }
    }
    while (hi - lo > 1u) {  // code(lo) <= q < code(hi)
        const unsigned mid = lo + (hi - lo) / 2u;
        if (above(mid))
            hi = mid;
        else
            lo = mid;
    }
    return key_value(hi);
}

// fp32 values v, L with |v|, |L| <= M differ exactly in fp64 when neither is a nonzero
// value below 2^(e(M) - 29) (e = floor(log2)): their exponents then differ by at most 29,
// so v - L needs at most 53 bits.  Returns that floor (0 when M is subnormal or zero).
__device__ __forceinline__ float exact_floor(float M) {
    const int be = (int)((__float_as_uint(M) >> 23) & 255u);
    return be == 0 ? 0.0f : __builtin_ldexpf(1.0f, be - 127 - 29);
}

// code of x from NLEV - 1 sorted thresholds (s_thr[NLEV - 1] = +inf): every eighth from
// registers, then one block of eight from LDS
template <int NLEV>
__device__ __forceinline__ int code_from_thresholds(float x, const float* s_thr, const float (&coarse)[NLEV / 8 + 1]) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    if (NLEV < 8) {
        int q = 0;
#pragma unroll
        for (int i = 0; i < NLEV - 1; ++i) q += s_thr[i] <= x ? 1 : 0;
        return q;
    }
    int c = 0;
    if (NLEV == 64) {
        // the thresholds do not decrease, so the count of the eight coarse ones at or below
        // x takes three halving steps (selects, no branches) and a last check of the eighth
        const bool h4 = coarse[3] <= x;
        const bool h2 = (h4 ? coarse[5] : coarse[1]) <= x;
        const bool h1 = (h4 ? (h2 ? coarse[6] : coarse[4]) : (h2 ? coarse[2] : coarse[0])) <= x;
        c = (h4 ? 4 : 0) + (h2 ? 2 : 0) + (h1 ? 1 : 0);
        c += (c == 7 && coarse[7] <= x) ? 1 : 0;
    } else {
#pragma unroll
        for (int i = 0; i < NLEV / 8; ++i) c += coarse[i] <= x ? 1 : 0;  // coarse[NLEV / 8 - 1] = +inf
    }
    const f32x4 a = reinterpret_cast<const f32x4*>(s_thr)[2 * c];
    const f32x4 b = reinterpret_cast<const f32x4*>(s_thr)[2 * c + 1];
    // the block's eighth threshold is coarse[c] > x: three halving steps over the other seven
    const bool f4 = a[3] <= x;
    const bool f2 = (f4 ? b[1] : a[1]) <= x;
    const bool f1 = (f4 ? (f2 ? b[2] : b[0]) : (f2 ? a[2] : a[0])) <= x;
    return 8 * c + (f4 ? 4 : 0) + (f2 ? 2 : 0) + (f1 ? 1 : 0);
}

// ---- codebooks of at most kCbqFastMax scalars whose values all meet the exactness condition
// (finite, no nonzero magnitude below 2^(e(M) - 29), M the largest magnitude): the rounds
// in integers.  Every value is then a multiple of 2^-S with S = 52 - e(M) (149 when M is
// subnormal), so w v 2^S is an integer below 2^84 in magnitude, held as a 2^42 + b with
// 0 <= b < 2^42; a level keeps the sums A of the a and B of the b of its members (below
// 2^54 for 4096 scalars) and W of their weights in three 64-bit LDS accumulators.  Its new
// value is the exact integer A 2^42 + B rounded once to fp64, times 2^-S, over W in fp64,
// rounded to fp32: the value the digit sums give, bit for bit.  When a round's levels are
// sorted and none is a nonzero value below 2^(e(M) - 29) either, every fp64 distance is
// exact, the nearest level of v (lowest index on ties) changes from q to q + 1 exactly
// above the midpoint of L_q and L_{q+1} (exact in fp64), and the code of v is the number of
// thresholds t_q <= v, t_q the smallest fp32 value above that midpoint (t_q = t_{q+1} when
// L_q = L_{q+1}, whose upper level never wins).  Other rounds search the levels as
// cbq_kernel does.  The scalars, their weights and codes live in LDS; one wave computes the
// levels and thresholds; in a threshold round every scalar checks that it still lies in its
// code's interval [t_{c-1}, t_c), and the few that left it are queued and searched by dense
// lanes, which move their (a, b, w) between the two levels' sums (three barriers a round).
constexpr int kCbqFastMax = 4096;                           // scalars of a codebook
constexpr int kCbqFastLevels = 64;                          // six bits

// an int128 rounded to nearest-even fp64
__device__ __forceinline__ double i128_to_double(__int128 x) {
    const bool neg = x < 0;
    const unsigned __int128 u = neg ? (unsigned __int128)(-x) : (unsigned __int128)x;
    const unsigned long long hi = (unsigned long long)(u >> 64), lo = (unsigned long long)u;
    double r;
    if (hi == 0) {
        r = (double)lo;  // correctly rounded conversion of 64 bits
    } else {
        const int lz = __clzll((long long)hi);  // 0..63
        const unsigned long long top = lz ? (hi << lz) | (lo >> (64 - lz)) : hi;
        const bool sticky = (lz ? (lo << lz) : lo) != 0ull;
        unsigned long long mant = top >> 11;
        const unsigned rnd = (unsigned)(top & 0x7ffull);
        if (rnd > 0x400u || (rnd == 0x400u && (sticky || (mant & 1ull)))) ++mant;
        r = ldexp((double)mant, 64 + 63 - lz - 52);
    }
    return neg ? -r : r;
}

// the smallest fp32 value above y (y finite, within fp32 range)
__device__ __forceinline__ float fp32_above(double y) {
    const float f = (float)y;  // nearest; a larger fp32 below y cannot exist
    if ((double)f > y) return f;
    const unsigned u = __float_as_uint(f);
    if (u == 0x80000000u || u == 0u) return __uint_as_float(1u);  // above a zero: the smallest subnormal
    return __uint_as_float((u & 0x80000000u) ? u - 1u : u + 1u);
}

__device__ void cbq_exact_rounds(const CbqParams& p, const CbqLayer& L, int m, float lo, float hi, float M, float* s_x,
                                 unsigned* s_wt, uint8_t* s_cd, unsigned short* s_q) {
    __shared__ __attribute__((aligned(16))) float s_flev[kCbqFastLevels];
    __shared__ __attribute__((aligned(16))) float s_thr[kCbqFastLevels];
    __shared__ __attribute__((aligned(16))) float s_coarse[kCbqFastLevels / 8];  // every eighth of s_flev or s_thr
    __shared__ unsigned long long s_A[kCbqFastLevels], s_B[kCbqFastLevels], s_W[kCbqFastLevels];
    __shared__ int s_mode;
    __shared__ int s_chg[2];
    __shared__ unsigned s_qn;  // scalars queued this round
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int beM = (int)((__float_as_uint(M) >> 23) & 255u);
    const int S = beM == 0 ? 149 : 179 - beM;
    const float fl = exact_floor(M);

    // the scalars, their weights (those <= 0 add nothing) and, later, their codes in LDS
    for (int r = tid; r < m; r += kCbqThreads) {
        s_x[r] = L.C[r];
        const int w = L.w ? L.w[r / kDim] : 1;
        s_wt[r] = w > 0 ? (unsigned)w : 0u;
    }
    // w v 2^S as a 2^42 + b: v 2^S from the bits (the integer mantissa shifted into place,
    // 0 <= shift <= 29 for every value that meets the condition), times w in 128 bits
    auto contrib = [&](float xv, unsigned w, long long& a, unsigned long long& b) {
        const unsigned bits = __float_as_uint(xv);
        const int be = (int)((bits >> 23) & 255u);
        const unsigned long long mant = (unsigned long long)((bits & 0x7fffffu) | (be ? 0x800000u : 0u));
        const long long vs = mant ? (long long)(mant << ((be ? be : 1) - 150 + S)) : 0ll;
        const __int128 X = (__int128)((bits >> 31) ? -vs : vs) * (__int128)w;
        a = (long long)(X >> 42);
        b = (unsigned long long)X & ((1ull << 42) - 1ull);
    };
    // scalar r moves into level q (and, unless `first`, out of level c)
    auto move = [&](int r, int c, int q, bool first) {
        const unsigned w = s_wt[r];
        if (!w) return;
        long long a;
        unsigned long long b;
        contrib(s_x[r], w, a, b);
        if (!first) {
            atomicAdd(&s_A[c], (unsigned long long)(-a));
            atomicAdd(&s_B[c], (unsigned long long)(-(long long)b));
            atomicAdd(&s_W[c], (unsigned long long)(-(long long)w));
        }
        atomicAdd(&s_A[q], (unsigned long long)a);
        atomicAdd(&s_B[q], b);
        atomicAdd(&s_W[q], (unsigned long long)w);
    };
    if (tid < kCbqFastLevels) {
        s_A[tid] = s_B[tid] = s_W[tid] = 0ull;
        const double delta = ((double)hi - (double)lo) / (double)(kCbqFastLevels - 1);
        s_flev[tid] = (float)__dadd_rn((double)lo, __dmul_rn((double)tid, delta));
    }
    if (tid < 2) s_chg[tid] = 0;

    // level q from its sums (unchanged when empty or without `update`): N = A 2^42 + B with
    // B's carries moved into A; while |A| <= 2^53 both parts are exact doubles and one fp64
    // addition rounds N correctly
    auto level_of = [&](int q, bool update) {
        float Lq = s_flev[q];
        const unsigned long long W = s_W[q];
        if (update && W > 0ull) {
            const unsigned long long B = s_B[q];
            const long long A = (long long)s_A[q] + (long long)(B >> 42);
            const unsigned long long Bl = B & ((1ull << 42) - 1ull);
            double N;
            if (A <= (1ll << 53) && A >= -(1ll << 53))
                N = __builtin_ldexp((double)A, 42) + (double)Bl;
            else
                N = i128_to_double(((__int128)A << 42) + (__int128)Bl);
            Lq = (float)(ldexp(N, -S) / (double)W);
        }
        return Lq;
    };
    // wave 0: the levels (from the sums, when `update`), whether they are sorted and exact,
    // and then the thresholds; s_mode = 2 (thresholds), 1 (sorted levels) or 0 (unsorted)
    auto levels = [&](bool update) {
        const int q = lane;
        const float Lq = level_of(q, update);
        s_flev[q] = Lq;
        const float Ln = __shfl_down(Lq, 1);  // the level above (lane 63: its own)
        const bool srt = __all(q == kCbqFastLevels - 1 || Lq <= Ln);
        const bool ex = __all(Lq == 0.0f || fabsf(Lq) >= fl);
        float t = __builtin_inff();
        int src = -1;  // a duplicate takes the threshold of the next level up
        if (q < kCbqFastLevels - 1) {
            if (Lq == Ln)
                src = q + 1;
            else
                t = fp32_above(0.5 * ((double)Lq + (double)Ln));
        }
        if (__any(src >= 0)) {
#pragma unroll
            for (int st = 0; st < 6; ++st) {  // pointer jumping over runs of equal levels
                const float ts = __shfl(t, src < 0 ? q : src);
                const int ss = __shfl(src, src < 0 ? q : src);
                if (src >= 0) {
                    t = ts;
                    src = ss;
                }
            }
        }
        const int mode = srt ? (ex ? 2 : 1) : 0;
        s_thr[q] = t;
        if ((q & 7) == 7) s_coarse[q >> 3] = mode == 2 ? t : Lq;
        if (q == 0) {
            s_mode = mode;
            s_qn = 0u;
        }
    };
    __syncthreads();  // scalars and grid in place
    if (wave == 0) levels(false);
    __syncthreads();

    auto load_coarse = [&](float (&coarse)[kCbqFastLevels / 8 + 1]) {
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        const f32x4 c0 = reinterpret_cast<const f32x4*>(s_coarse)[0], c1 = reinterpret_cast<const f32x4*>(s_coarse)[1];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            coarse[i] = c0[i];
            coarse[4 + i] = c1[i];
        }
        coarse[kCbqFastLevels / 8] = 0.0f;
    };
    // code of x against the current levels (the mode decides how)
    auto search = [&](float x, int mode, const float (&coarse)[kCbqFastLevels / 8 + 1]) {
        return mode == 2 ? code_from_thresholds<kCbqFastLevels>(x, s_thr, coarse)
                         : (mode == 1 ? nearest_sorted_fast<kCbqFastLevels>(x, s_flev, coarse)
                                      : nearest_level_loop(x, s_flev, kCbqFastLevels));
    };

    {  // the first codes, and with them the sums
        const int mode = __builtin_amdgcn_readfirstlane(s_mode);
        float coarse[kCbqFastLevels / 8 + 1];
        load_coarse(coarse);
        for (int r = tid; r < m; r += kCbqThreads) {
            const int q = search(s_x[r], mode, coarse);
            s_cd[r] = (uint8_t)q;
            move(r, 0, q, true);
        }
    }
    __syncthreads();

    for (int it = 0; it < p.iters; ++it) {
        if (wave == 0) {
            levels(true);
            if (lane == 0) s_chg[it & 1] = 0;  // last read before the previous round's first barrier
        }
        __syncthreads();
        const int mode = __builtin_amdgcn_readfirstlane(s_mode);
        int chg = 0;
        if (mode == 2) {
            // code c stays while t_{c-1} <= v < t_c; the scalars that left their interval are
            // queued and searched by dense lanes (a few per round: no wave runs the search for
            // one lane)
            // (a thread's up to four scalars: every code read first, then every bound)
            constexpr int kPer = kCbqFastMax / kCbqThreads;
            int c[kPer];
            float x[kPer], tl[kPer], th[kPer];
#pragma unroll
            for (int u = 0; u < kPer; ++u) {
                const int r = tid + u * kCbqThreads;
                c[u] = r < m ? s_cd[r] : 0;
                x[u] = r < m ? s_x[r] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kPer; ++u) {
                tl[u] = s_thr[c[u] > 0 ? c[u] - 1 : 0];
                th[u] = s_thr[c[u]];
            }
#pragma unroll
            for (int u = 0; u < kPer; ++u) {
                const int r = tid + u * kCbqThreads;
                if (r < m && !((c[u] == 0 || tl[u] <= x[u]) && x[u] < th[u]))
                    s_q[atomicAdd(&s_qn, 1u)] = (unsigned short)r;
            }
            __syncthreads();
            const int n = (int)s_qn;
            if (tid < n) {
                float coarse[kCbqFastLevels / 8 + 1];
                load_coarse(coarse);
                for (int e = tid; e < n; e += kCbqThreads) {
                    const int r = s_q[e];
                    const int c = s_cd[r];
                    const int q = code_from_thresholds<kCbqFastLevels>(s_x[r], s_thr, coarse);  // differs from c
                    move(r, c, q, false);
                    s_cd[r] = (uint8_t)q;
                }
                chg = 1;
            }
        } else {
            float coarse[kCbqFastLevels / 8 + 1];
            load_coarse(coarse);
            for (int r = tid; r < m; r += kCbqThreads) {
                const int c = s_cd[r];
                const int q = search(s_x[r], mode, coarse);
                if (q != c) {
                    move(r, c, q, false);
                    s_cd[r] = (uint8_t)q;
                    chg = 1;
                }
            }
        }
        if (chg) s_chg[it & 1] = 1;
        __syncthreads();
        if (!s_chg[it & 1]) break;
    }

    if (tid < kCbqFastLevels) L.levels[tid] = s_flev[tid];
    for (int r = tid; r < m; r += kCbqThreads) {
        const int c = s_cd[r];
        L.codes[r] = (uint8_t)c;
        if (L.C_hat) L.C_hat[r] = s_flev[c];
    }
}

// Thread tid handles scalars r = tid, tid + 1024, ...  With LDS (codebooks of at most
// kCbqLdsScalars scalars) the scalars, their weights and codes are copied into LDS once;
// otherwise every pass reads them from memory.  The level sums are kept up to date
// incrementally: after the first full accumulation only scalars whose code changes move
// their (exact) contribution between two levels, which leaves the same integers as
// summing from scratch.
constexpr int kCbqLdsScalars = 8192;

// FAST64: 64 levels (6 bits, the paper's width), searched with nearest_sorted_fast
template <bool LDS, bool FAST64>
__global__ __launch_bounds__(kCbqThreads) void cbq_kernel(const CbqParams p) {
    __shared__ __attribute__((aligned(16))) float s_lev[kCbqMaxLevels];
    __shared__ unsigned long long s_dig[kCbqMaxLevels * kDigits];
    __shared__ unsigned long long s_w[kCbqMaxLevels];
    __shared__ float s_lo[kCbqThreads / kWave], s_hi[kCbqThreads / kWave], s_sm[kCbqThreads / kWave];
    __shared__ int s_changed;
    __shared__ int s_unsorted;
    __shared__ float s_v[LDS ? kCbqLdsScalars : 1];
    __shared__ int s_wt[LDS ? kCbqLdsScalars : 1];
    __shared__ uint8_t s_code[LDS ? kCbqLdsScalars : 1];

    const CbqLayer& L = p.L[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m = L.k * kDim;
    const int nlev = 1 << p.bits;
    const bool wk = p.mode == KQ_CBQ_WKMEANS;
    const float* __restrict__ v = L.C;
    uint8_t* __restrict__ codes = L.codes;
    auto val = [&](int r) { return LDS ? s_v[r] : v[r]; };
    auto wgt = [&](int r) { return LDS ? s_wt[r] : (L.w ? L.w[r / kDim] : 1); };
    auto code = [&](int r) { return LDS ? (int)s_code[r] : (int)codes[r]; };
    auto set_code = [&](int r, int q) {
        if (LDS)
            s_code[r] = (uint8_t)q;
        else
            codes[r] = (uint8_t)q;
    };

    // grid on [min, max]; for the integer rounds also the smallest nonzero magnitude and
    // whether a value is not finite
    float lo = __builtin_inff(), hi = -__builtin_inff(), sm = __builtin_inff();
    bool nonfinite = false;
    for (int r = tid; r < m; r += kCbqThreads) {
        const float x = v[r];
        lo = fminf(lo, x);
        hi = fmaxf(hi, x);
        if (x != 0.0f) sm = fminf(sm, fabsf(x));
        nonfinite |= !(fabsf(x) <= 3.402823466e38f);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, off));
        hi = fmaxf(hi, __shfl_xor(hi, off));
        sm = fminf(sm, __shfl_xor(sm, off));
    }
    nonfinite = __any(nonfinite);
    if (lane == 0) {
        s_lo[wave] = lo;
        s_hi[wave] = hi;
        s_sm[wave] = nonfinite ? -1.0f : sm;
    }
    if (tid == 0) s_unsorted = 0;
    __syncthreads();
    lo = s_lo[0];
    hi = s_hi[0];
    sm = s_sm[0];
    for (int w = 1; w < kCbqThreads / kWave; ++w) {
        lo = fminf(lo, s_lo[w]);
        hi = fmaxf(hi, s_hi[w]);
        sm = s_sm[w] < 0.0f || sm < 0.0f ? -1.0f : fminf(sm, s_sm[w]);
    }
    if (FAST64 && wk && m <= kCbqFastMax && sm >= 0.0f) {
        const float M = fmaxf(fabsf(lo), fabsf(hi));
        if (!(sm < exact_floor(M))) {  // every value meets the exactness condition
            if constexpr (LDS) {
                cbq_exact_rounds(p, L, m, lo, hi, M, s_v, reinterpret_cast<unsigned*>(s_wt), s_code,
                                 reinterpret_cast<unsigned short*>(s_dig));
                return;
            }
        }
    }
    if (LDS) {
        for (int r = tid; r < m; r += kCbqThreads) {
            s_v[r] = v[r];
            s_wt[r] = L.w ? L.w[r / kDim] : 1;
        }
    }
    for (int e = tid; e < nlev * kDigits; e += kCbqThreads) s_dig[e] = 0ull;
    for (int e = tid; e < nlev; e += kCbqThreads) s_w[e] = 0ull;
    if (tid < nlev) {
        const double delta = ((double)hi - (double)lo) / (double)(nlev - 1);
        s_lev[tid] = (float)__dadd_rn((double)lo, __dmul_rn((double)tid, delta));
    }
    __syncthreads();
    if (tid + 1 < nlev && !(s_lev[tid] <= s_lev[tid + 1])) s_unsorted = 1;
    __syncthreads();
    bool sorted = s_unsorted == 0;
    float coarse[64 / 8 + 1];  // every eighth level, for the 64-level search
    auto load_coarse = [&]() {
#pragma unroll
        for (int i = 0; i < 64 / 8; ++i) coarse[i] = FAST64 ? s_lev[8 * i + 7] : 0.0f;
        coarse[64 / 8] = 0.0f;
    };
    auto nearest = [&](float x) {
        if (!sorted) return nearest_level(x, s_lev, nlev);
        return FAST64 ? nearest_sorted_fast<64>(x, s_lev, coarse) : nearest_sorted(x, s_lev, nlev);
    };
    load_coarse();

    // initial codes, and with them the level sums
    for (int r = tid; r < m; r += kCbqThreads) {
        const float x = val(r);
        const int q = nearest(x);
        set_code(r, q);
        const int w = wgt(r);
        if (wk && w > 0) {
            add_exact(s_dig + q * kDigits, x, (unsigned)w);
            atomicAdd(&s_w[q], (unsigned long long)w);
        }
    }
    __syncthreads();

    if (wk) {
        for (int it = 0; it < p.iters; ++it) {
            if (tid == 0) {
                s_changed = 0;
                s_unsorted = 0;
            }
            if (tid < nlev && s_w[tid] > 0ull) {
                const double N = digits_to_double(s_dig + tid * kDigits);
                s_lev[tid] = (float)(N / (double)s_w[tid]);
            }
            __syncthreads();
            if (tid + 1 < nlev && !(s_lev[tid] <= s_lev[tid + 1])) s_unsorted = 1;
            __syncthreads();
            sorted = s_unsorted == 0;
            load_coarse();
            int changed = 0;
            for (int r = tid; r < m; r += kCbqThreads) {
                const float x = val(r);
                const int q = nearest(x);
                const int c = code(r);
                if (q != c) {
                    const int w = wgt(r);
                    if (w > 0) {  // move the exact contribution from level c to level q
                        add_exact(s_dig + c * kDigits, -x, (unsigned)w);
                        add_exact(s_dig + q * kDigits, x, (unsigned)w);
                        atomicAdd(&s_w[c], (unsigned long long)(-(long long)w));
                        atomicAdd(&s_w[q], (unsigned long long)w);
                    }
                    set_code(r, q);
                    changed = 1;
                }
            }
            if (changed) s_changed = 1;
            __syncthreads();
            const int any = s_changed;
            __syncthreads();
            if (!any) break;
        }
    }

    if (tid < nlev) L.levels[tid] = s_lev[tid];
    for (int r = tid; r < m; r += kCbqThreads) {
        const int c = code(r);
        if (LDS) codes[r] = (uint8_t)c;
        if (L.C_hat) L.C_hat[r] = s_lev[c];
    }
}

// ---- large scalar sets (the fully-connected layers, end of Sec. 3.2) ---------------------
// The same method on one flat vector of m scalars, every weight 1, spread over a
// persistent grid.  Per round:
//   fc_assign_kernel  every workgroup codes its scalars against the current levels (LDS)
//                     and adds, in LDS, the exact contributions it moves: in the first
//                     pass every scalar's, later only those of scalars whose code changed
//                     (subtracted from the old level, added to the new); it stores the
//                     per-level digits and counts as its partial and whether it changed
//                     any code;
//   fc_sum_kernel     one workgroup per level adds the partials (stored per level, one per
//                     coding workgroup) to the level's running
//                     exact sum and forms the candidate level fp32(round64(sum) / count);
//   fc_state_kernel   one workgroup: a round that changed no code ends the run (every
//                     later launch returns at once); otherwise the candidates become the
//                     levels while fewer than `iters` updates were made.
// Integer sums make the levels, and with them the codes, independent of the grid and the
// order of the work: the result is the single-workgroup quantizer's, bit for bit.
constexpr int kFcCols = kDigits + 1;  // digits, then the count
// scalars from which codes come from thresholds: below, the per-round boundary search costs
// more than the exact search it saves (measured per round: about even at 2^21 scalars,
// 35 instead of 42 us at 3 * 2^20)
constexpr long long kFcThresholdMin = 3ll << 20;
// whether rounds may take their codes from thresholds: unweighted sets only (weighted
// codebooks stay far below that size), by the size rule unless a flag forces a way; the
// device's choice and the host's launch of the threshold kernel use the same rule
__host__ __device__ __forceinline__ bool fc_thr_wanted(const FcParams& p) {
    return p.w == nullptr && (p.thr_mode == 2 || (p.thr_mode == 0 && p.m >= kFcThresholdMin));
}

__device__ __forceinline__ bool fc_done(const FcParams& p) { return p.state[0] != 0; }

// per workgroup: min, max and smallest nonzero magnitude of its scalars
__global__ __launch_bounds__(kFcThreads) void fc_minmax_kernel(const FcParams p) {
    __shared__ float s_lo[kFcThreads / kWave], s_hi[kFcThreads / kWave], s_sm[kFcThreads / kWave];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float lo = __builtin_inff(), hi = -__builtin_inff(), sm = __builtin_inff();
    auto take = [&](float x) {
        lo = fminf(lo, x);
        hi = fmaxf(hi, x);
        if (x != 0.0f) sm = fminf(sm, fabsf(x));
    };
    long long r0 = 0;  // scalars from here on: one at a time
    if ((reinterpret_cast<uintptr_t>(p.v) & 15u) == 0) {  // float4 groups, four per thread in flight
        constexpr int kPer = 4;
        const long long ng = p.m >> 2;
        const float4* __restrict__ v4 = reinterpret_cast<const float4*>(p.v);
        for (long long g0 = (long long)blockIdx.x * kFcThreads * kPer + tid; g0 < ng;
             g0 += (long long)gridDim.x * kFcThreads * kPer) {
            float4 xv[kPer];
#pragma unroll
            for (int j = 0; j < kPer; ++j) {
                const long long g = g0 + (long long)j * kFcThreads;
                xv[j] = g < ng ? v4[g] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
#pragma unroll
            for (int j = 0; j < kPer; ++j)
                if (g0 + (long long)j * kFcThreads < ng) {
                    take(xv[j].x);
                    take(xv[j].y);
                    take(xv[j].z);
                    take(xv[j].w);
                }
        }
        r0 = 4 * ng;
    }
    for (long long r = r0 + (long long)blockIdx.x * kFcThreads + tid; r < p.m; r += (long long)gridDim.x * kFcThreads)
        take(p.v[r]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, off));
        hi = fmaxf(hi, __shfl_xor(hi, off));
        sm = fminf(sm, __shfl_xor(sm, off));
    }
    if (lane == 0) {
        s_lo[wave] = lo;
        s_hi[wave] = hi;
        s_sm[wave] = sm;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < kFcThreads / kWave; ++w) {
            lo = fminf(lo, s_lo[w]);
            hi = fmaxf(hi, s_hi[w]);
            sm = fminf(sm, s_sm[w]);
        }
        p.minmax[3 * blockIdx.x] = lo;
        p.minmax[3 * blockIdx.x + 1] = hi;
        p.minmax[3 * blockIdx.x + 2] = sm;
    }
}

// the bucket of x: (x - lo) * sc clamped to [0, kFcBuckets - 1] (NaN to 0), truncated.  Each
// step is monotone, so x <= y gives bucket(x) <= bucket(y); the table and the coding launch
// compute it with the same operations on the same lo and sc.
__device__ __forceinline__ int fc_bucket(float x, float lo, float sc) {
    const float t = (x - lo) * sc;
    return (int)fminf(fmaxf(t, 0.0f), (float)(kFcBuckets - 1));
}

// thresholds of the levels s_lev (sorted unless s_unsorted) when every distance from the
// data range to them is exact in fp64 (state[3]); otherwise state[3] = 0 and the codes
// are found by the exact search.  With thresholds and a finite bucket scale the bucket
// table follows: for bucket b, c = the number of thresholds whose bucket is below b (all
// of them below every value of b) and n = the number inside b; entry b = (c | n << 8,
// threshold c or +inf).  A value's code is then c plus the count of the n thresholds
// c .. c + n - 1 at or below it.  Every thread of the workgroup calls it.
__device__ void set_thresholds(const FcParams& p, const float* s_lev, int nlev, int unsorted, int* s_bad, float vmin,
                               float vmax, float vsm) {
    const int tid = threadIdx.x;
    const float fl = exact_floor(fmaxf(fabsf(vmin), fabsf(vmax)));
    // the boundary search costs a few microseconds per round: worth it only for large sets
    const bool wanted = fc_thr_wanted(p);
    if (tid == 0) *s_bad = (unsorted || vsm < fl || !wanted) ? 1 : 0;
    __syncthreads();
    if (tid < nlev && s_lev[tid] != 0.0f && fabsf(s_lev[tid]) < fl) *s_bad = 1;
    __syncthreads();
    const int ok = *s_bad == 0;
    float t = __builtin_inff();
    if (tid < nlev) {
        t = (ok && tid + 1 < nlev) ? code_threshold(tid, s_lev, nlev, vmin, vmax) : __builtin_inff();
        p.thr[tid] = t;
    }
    if (tid == 0) p.state[3] = ok;
    __shared__ float s_t[kCbqMaxLevels];
    const float sc = (float)kFcBuckets / (vmax - vmin);
    const bool table = ok && vmax > vmin && sc > 0.0f && sc < __builtin_inff();  // the same in every thread
    if (tid == 0) p.range[3] = table ? sc : 0.0f;
    if (!table) return;
    // per bucket the number of thresholds in it; then each thread takes kPerThread consecutive
    // buckets, and c of its first bucket is the exclusive prefix sum of the threads before it
    static_assert(kFcBuckets % kCbqMaxLevels == 0, "whole runs of buckets per thread");
    constexpr int kPerThread = kFcBuckets / kCbqMaxLevels;
    __shared__ int s_n[kFcBuckets];
    __shared__ int s_wsum[kCbqMaxLevels / kWave];
    for (int b = tid; b < kFcBuckets; b += kCbqMaxLevels) s_n[b] = 0;
    if (tid < nlev) s_t[tid] = t;
    __syncthreads();
    if (tid + 1 < nlev) atomicAdd(&s_n[fc_bucket(t, vmin, sc)], 1);  // thresholds 0 .. nlev - 2
    __syncthreads();
    int n[kPerThread], tot = 0;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        n[i] = s_n[kPerThread * tid + i];
        tot += n[i];
    }
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    int inc = tot;  // inclusive scan over the wave
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(inc, off);
        if (lane >= off) inc += o;
    }
    if (lane == kWave - 1) s_wsum[wave] = inc;
    __syncthreads();
    int c = inc - tot;
    for (int w = 0; w < wave; ++w) c += s_wsum[w];
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        const int b = kPerThread * tid + i;
        p.tbl[2 * b] = (unsigned)c | ((unsigned)n[i] << 8);
        p.tbl[2 * b + 1] = __float_as_uint(n[i] > 0 ? s_t[c] : __builtin_inff());
        c += n[i];
    }
}

// the uniform grid on [min, max]; clears the run state and the running sums
__global__ __launch_bounds__(kCbqMaxLevels) void fc_grid_kernel(const FcParams p, int nblk) {
    __shared__ float s_lo, s_hi, s_sm;
    __shared__ float s_lev[kCbqMaxLevels];
    __shared__ int s_unsorted, s_bad;
    __shared__ float s_w[3][kCbqMaxLevels / kWave];
    const int tid = threadIdx.x, nlev = 1 << p.bits;
    {  // the workgroups' minima and maxima: strided per thread, then across the wave and the waves
        float lo = __builtin_inff(), hi = -__builtin_inff(), sm = __builtin_inff();
        for (int b = tid; b < nblk; b += kCbqMaxLevels) {
            lo = fminf(lo, p.minmax[3 * b]);
            hi = fmaxf(hi, p.minmax[3 * b + 1]);
            sm = fminf(sm, p.minmax[3 * b + 2]);
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            lo = fminf(lo, __shfl_xor(lo, off));
            hi = fmaxf(hi, __shfl_xor(hi, off));
            sm = fminf(sm, __shfl_xor(sm, off));
        }
        if ((tid & (kWave - 1)) == 0) {
            s_w[0][tid / kWave] = lo;
            s_w[1][tid / kWave] = hi;
            s_w[2][tid / kWave] = sm;
        }
    }
    __syncthreads();
    if (tid == 0) {
        float lo = s_w[0][0], hi = s_w[1][0], sm = s_w[2][0];
        for (int w = 1; w < kCbqMaxLevels / kWave; ++w) {
            lo = fminf(lo, s_w[0][w]);
            hi = fmaxf(hi, s_w[1][w]);
            sm = fminf(sm, s_w[2][w]);
        }
        s_lo = lo;
        s_hi = hi;
        s_sm = sm;
        p.range[0] = lo;
        p.range[1] = hi;
        p.range[2] = sm;
        s_unsorted = 0;
        p.state[0] = 0;  // not converged
        p.state[1] = 0;  // level updates made
    }
    __syncthreads();
    if (tid < nlev) {
        const double delta = ((double)s_hi - (double)s_lo) / (double)(nlev - 1);
        s_lev[tid] = (float)__dadd_rn((double)s_lo, __dmul_rn((double)tid, delta));
        p.lev[tid] = s_lev[tid];
    }
    for (int e = tid; e < nlev * kFcCols; e += blockDim.x) p.S[e] = 0ll;
    __syncthreads();
    if (tid + 1 < nlev && !(s_lev[tid] <= s_lev[tid + 1])) s_unsorted = 1;
    __syncthreads();
    if (tid == 0) p.state[2] = s_unsorted;
    set_thresholds(p, s_lev, nlev, s_unsorted, &s_bad, s_lo, s_hi, s_sm);
}

// Each thread takes four scalars per step (r0 + 256 j, consecutive lanes consecutive
// scalars), their loads issued together; with sorted levels a code is the number of
// thresholds at or below the value (fp32 comparisons only).
// THR: the launch for rounds whose codes come from thresholds (true) or from the exact
// searches (false); the state decides on the device, and the other launch returns at once.
// Apart, the light threshold code keeps its register count low.
template <bool INIT, int NLEV, bool THR>
__global__ __launch_bounds__(kFcThreads) void fc_assign_kernel(const FcParams p) {
    __shared__ __attribute__((aligned(16))) float s_lev[NLEV < 8 ? 8 : NLEV];
    __shared__ __attribute__((aligned(16))) float s_thr[NLEV < 8 ? 8 : NLEV];
    __shared__ unsigned long long s_dig[NLEV * kFcCols];
    __shared__ uint2 s_tbl[THR ? kFcBuckets : 1];
    // threshold rounds: per wave a queue of the scalars whose code changed (value, old and new
    // code), whose sums are moved 64 at a time by the whole wave
    constexpr int kQCap = 4 * kWave + kWave;  // a group step adds at most 4 per lane
    __shared__ float s_qv[THR ? kFcThreads / kWave : 1][THR ? kQCap : 1];
    __shared__ unsigned short s_qc[THR ? kFcThreads / kWave : 1][THR ? kQCap : 1];
    __shared__ int s_changed;
    if (fc_done(p)) return;
    if ((p.state[3] != 0) != THR) return;  // the other launch codes this round
    const int tid = threadIdx.x;
    for (int e = tid; e < NLEV; e += kFcThreads) {
        s_lev[e] = p.lev[e];
        s_thr[e] = p.thr[e];  // thr[NLEV - 1] is +inf
    }
    const float blo = p.range[0], bsc = p.range[3];
    const bool table = THR && bsc > 0.0f;  // the bucket table of this round's thresholds
    if (table)
        for (int e = tid; e < kFcBuckets; e += kFcThreads) s_tbl[e] = make_uint2(p.tbl[2 * e], p.tbl[2 * e + 1]);
    for (int e = tid; e < NLEV * kFcCols; e += kFcThreads) s_dig[e] = 0ull;
    if (tid == 0) s_changed = 0;
    __syncthreads();
    const bool sorted = p.state[2] == 0;
    float coarse[NLEV / 8 + 1], coarse_lev[NLEV / 8 + 1];
#pragma unroll
    for (int i = 0; i < NLEV / 8; ++i) {
        coarse[i] = s_thr[8 * i + 7];
        coarse_lev[i] = s_lev[8 * i + 7];
    }
    coarse[NLEV / 8] = coarse_lev[NLEV / 8] = 0.0f;
    int changed = 0;
    constexpr int kPer = 4;
    const long long m = p.m;
    // one instantiation per search (bucket table, thresholds, sorted levels, full scan): the choice is
    // the same for every scalar of the round
    auto run = [&](auto mode, auto weighted) {
        constexpr int kMode = decltype(mode)::value;
        constexpr bool kWeighted = decltype(weighted)::value;
        // the code of scalar r (value x, old code c); moves its exact contribution (weight
        // times value, and the weight into the count) when the code changes.  A weight of
        // zero or less contributes nothing, as in the single-workgroup quantizer.
        // the code of value x: the bucket table (two or more thresholds in the bucket: the
        // rest one by one), or a search of the thresholds or levels
        auto table_fixup = [&](float x, uint2 e, int q) {
            if (e.x >= 512u) {  // two or more thresholds in the bucket
                const int c = (int)(e.x & 255u), n = (int)(e.x >> 8);
                for (int j = 1; j < n; ++j) q += s_thr[c + j] <= x ? 1 : 0;
            }
            return q;
        };
        auto search = [&](float x) {
            if constexpr (kMode == 3) {
                const uint2 e = s_tbl[fc_bucket(x, blo, bsc)];
                return table_fixup(x, e, (int)(e.x & 255u) + (__uint_as_float(e.y) <= x ? 1 : 0));
            } else {
                return kMode == 0   ? code_from_thresholds<NLEV>(x, s_thr, coarse)
                       : kMode == 1 ? nearest_sorted_fast<NLEV>(x, s_lev, coarse_lev)
                                    : nearest_level(x, s_lev, NLEV);
            }
        };
        // scalar r (value x, old code c) takes code q: its exact contribution (weight times
        // value, and the weight into the count) moves when the code changes.  A weight of
        // zero or less contributes nothing, as in the single-workgroup quantizer.
        auto recode = [&](long long r, float x, int c, int q) {
            const int wt = kWeighted ? p.w[(unsigned)r / (unsigned)kDim] : 1;  // r < 2^31
            if (INIT) {
                if (wt > 0) {
                    add_exact(s_dig + q * kFcCols, x, (unsigned)wt);
                    atomicAdd(&s_dig[q * kFcCols + kDigits], (unsigned long long)wt);
                }
            } else if (q != c) {
                if (wt > 0) {
                    add_exact(s_dig + c * kFcCols, -x, (unsigned)wt);
                    add_exact(s_dig + q * kFcCols, x, (unsigned)wt);
                    atomicAdd(&s_dig[c * kFcCols + kDigits], (unsigned long long)(-(long long)wt));
                    atomicAdd(&s_dig[q * kFcCols + kDigits], (unsigned long long)wt);
                }
                changed = 1;
            }
            return q;
        };
        // the wave's queue of changed scalars (threshold rounds, unweighted): a lane whose scalar
        // changed appends (value, old code, new code) at the wave's count plus the number of
        // lower lanes appending; drain moves the sums of 64 entries at a time from the queue's
        // end, one per lane (all of them when `all`)
        const int wv = tid / kWave, ln = tid & (kWave - 1);
        int qn = 0;  // the same in every lane of the wave
        auto enqueue = [&](bool ch, float x, int c, int q) {
            if constexpr (THR) {
                const unsigned long long mk = __ballot(ch);
                if (mk == 0ull) return;
                changed = 1;
                if (ch) {
                    const int pos = qn + (int)__builtin_amdgcn_mbcnt_hi((unsigned)(mk >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo((unsigned)mk, 0u));
                    s_qv[wv][pos] = x;
                    s_qc[wv][pos] = (unsigned short)(c | (q << 8));
                }
                qn += __popcll(mk);
            }
        };
        auto drain = [&](bool all) {
            if constexpr (THR) {
                while (qn >= kWave || (all && qn > 0)) {
                    __builtin_amdgcn_wave_barrier();  // this wave's queue writes come first
                    const int take = qn < kWave ? qn : kWave;
                    if (ln < take) {
                        const int at = qn - take + ln;
                        const float x = s_qv[wv][at];
                        const unsigned cq = s_qc[wv][at];
                        const int c = (int)(cq & 255u), q = (int)(cq >> 8);
                        add_exact(s_dig + c * kFcCols, -x, 1u);
                        add_exact(s_dig + q * kFcCols, x, 1u);
                        atomicAdd(&s_dig[c * kFcCols + kDigits], (unsigned long long)-1ll);
                        atomicAdd(&s_dig[q * kFcCols + kDigits], 1ull);
                    }
                    __builtin_amdgcn_wave_barrier();  // read before the slots are reused
                    qn -= take;
                }
            }
        };
        // the grouped loop for threshold rounds (the large sets); the exact searches (small
        // sets, weighted codebooks, data where thresholds are refused) take one scalar at a time
        if ((kMode == 0 || kMode == 3) && (reinterpret_cast<uintptr_t>(p.v) & 15u) == 0 &&
            (reinterpret_cast<uintptr_t>(p.codes) & 3u) == 0) {
            // groups of four scalars: one float4 of values and one word of four codes per
            // group, kGPer groups per thread and step, the next step's loaded while this one is
            // coded; a group whose codes change stores its word
            constexpr int kGPer = 2;
            const long long ng = m >> 2;
            const long long step = (long long)gridDim.x * kFcThreads * kGPer;
            const float4* __restrict__ v4 = reinterpret_cast<const float4*>(p.v);
            unsigned* __restrict__ c4 = reinterpret_cast<unsigned*>(p.codes);
            auto load = [&](long long g0, float4 (&xv)[kGPer], unsigned (&cw)[kGPer]) {
#pragma unroll
                for (int j = 0; j < kGPer; ++j) {
                    const long long g = g0 + (long long)j * kFcThreads;
                    xv[j] = g < ng ? v4[g] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                    cw[j] = (!INIT && g < ng) ? c4[g] : 0u;
                }
            };
            long long g0 = (long long)blockIdx.x * kFcThreads * kGPer + tid;
            // kDepth steps in flight: this one and the next (a sweep of groups per step and
            // depth kept 2 and 2)
            constexpr int kDepth = 2;
            float4 xb[kDepth][kGPer];
            unsigned cb[kDepth][kGPer];
#pragma unroll
            for (int d = 0; d < kDepth - 1; ++d)
                if (g0 + d * step < ng) load(g0 + d * step, xb[d], cb[d]);
            for (; g0 < ng; g0 += step) {
                if (g0 + (kDepth - 1) * step < ng) load(g0 + (kDepth - 1) * step, xb[kDepth - 1], cb[kDepth - 1]);
                float4 (&xv)[kGPer] = xb[0];
                unsigned (&cw)[kGPer] = cb[0];
                float xs[kGPer][4];
#pragma unroll
                for (int j = 0; j < kGPer; ++j) {
                    xs[j][0] = xv[j].x;
                    xs[j][1] = xv[j].y;
                    xs[j][2] = xv[j].z;
                    xs[j][3] = xv[j].w;
                }
                int qs[kGPer][4];
                if constexpr (kMode == 3) {  // the step's table reads issued together
                    uint2 te[kGPer][4];
#pragma unroll
                    for (int j = 0; j < kGPer; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e) te[j][e] = s_tbl[fc_bucket(xs[j][e], blo, bsc)];
                    unsigned many = 0u;
#pragma unroll
                    for (int j = 0; j < kGPer; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            qs[j][e] = (int)(te[j][e].x & 255u) + (__uint_as_float(te[j][e].y) <= xs[j][e] ? 1 : 0);
                            many |= te[j][e].x;
                        }
                    if (many >= 512u)
#pragma unroll
                        for (int j = 0; j < kGPer; ++j)
#pragma unroll
                            for (int e = 0; e < 4; ++e) qs[j][e] = table_fixup(xs[j][e], te[j][e], qs[j][e]);
                }
#pragma unroll
                for (int j = 0; j < kGPer; ++j) {
                    const long long g = g0 + (long long)j * kFcThreads;
                    const bool have = g < ng;
                    unsigned nw = 0u;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int q = kMode == 3 ? qs[j][e] : search(xs[j][e]);
                        const int c = (int)((cw[j] >> (8 * e)) & 255u);
                        if (INIT) {
                            if (have) recode(4 * g + e, xs[j][e], c, q);
                        } else {
                            enqueue(have && q != c, xs[j][e], c, q);
                        }
                        nw |= (unsigned)q << (8 * e);
                    }
                    if (have && (INIT || nw != cw[j])) c4[g] = nw;
                    if (!INIT) drain(false);
                }
#pragma unroll
                for (int d = 0; d + 1 < kDepth; ++d)
#pragma unroll
                    for (int j = 0; j < kGPer; ++j) {
                        xb[d][j] = xb[d + 1][j];
                        cb[d][j] = cb[d + 1][j];
                    }
            }
            if (!INIT) drain(true);
            if (blockIdx.x == 0)  // the last m % 4 scalars
                for (long long r = 4 * ng + tid; r < m; r += kFcThreads) {
                    const float x = p.v[r];
                    const int q = recode(r, x, INIT ? 0 : (int)p.codes[r], search(x));
                    if (INIT || q != (int)p.codes[r]) p.codes[r] = (uint8_t)q;
                }
        } else {
            const long long step = (long long)gridDim.x * kFcThreads * kPer;
            for (long long r0 = (long long)blockIdx.x * kFcThreads * kPer + tid; r0 < m; r0 += step) {
                float x[kPer];
                int c[kPer];
#pragma unroll
                for (int j = 0; j < kPer; ++j) {
                    const long long r = r0 + (long long)j * kFcThreads;
                    x[j] = r < m ? p.v[r] : 0.0f;
                    c[j] = (!INIT && r < m) ? (int)p.codes[r] : 0;
                }
#pragma unroll
                for (int j = 0; j < kPer; ++j) {
                    const long long r = r0 + (long long)j * kFcThreads;
                    if (r >= m) continue;
                    const int q = recode(r, x[j], c[j], search(x[j]));
                    if (INIT || q != c[j]) p.codes[r] = (uint8_t)q;
                }
            }
        }
    };
    // weights or none: decided once, so unweighted scalars spend nothing on them
    auto pick = [&](auto mode) {
        if (p.w)
            run(mode, std::integral_constant<bool, true>{});
        else
            run(mode, std::integral_constant<bool, false>{});
    };
    if constexpr (THR) {  // never weighted
        if (table)
            run(std::integral_constant<int, 3>{}, std::integral_constant<bool, false>{});
        else
            run(std::integral_constant<int, 0>{}, std::integral_constant<bool, false>{});
    } else {
        if (sorted)
            pick(std::integral_constant<int, 1>{});
        else
            pick(std::integral_constant<int, 2>{});
    }
    if (changed) s_changed = 1;
    __syncthreads();
    // partial of level q at [q][workgroup]: a level's partials are contiguous for fc_sum_kernel
    unsigned long long* part = (unsigned long long*)p.part;
    for (int e = tid; e < NLEV * kFcCols; e += kFcThreads) {
        const int q = e / kFcCols, c = e - q * kFcCols;
        part[((size_t)q * gridDim.x + blockIdx.x) * kFcCols + c] = s_dig[e];
    }
    if (tid == 0) p.wg_changed[blockIdx.x] = INIT ? 1 : s_changed;
}

template <bool INIT>
hipError_t launch_fc_assign(const FcParams& p, int G, hipStream_t s) {
    // the threshold launch only where the state may choose thresholds
    const bool thr = fc_thr_wanted(p);
    switch (p.bits) {
#define KQ_FC_CASE(B)                                                                                          \
    case B:                                                                                                    \
        if (thr) hipLaunchKernelGGL((fc_assign_kernel<INIT, (1 << B), true>), dim3(G), dim3(kFcThreads), 0, s, p); \
        hipLaunchKernelGGL((fc_assign_kernel<INIT, (1 << B), false>), dim3(G), dim3(kFcThreads), 0, s, p);       \
        break;
        KQ_FC_CASE(1)
        KQ_FC_CASE(2)
        KQ_FC_CASE(3)
        KQ_FC_CASE(4)
        KQ_FC_CASE(5)
        KQ_FC_CASE(6)
        KQ_FC_CASE(7)
        KQ_FC_CASE(8)
#undef KQ_FC_CASE
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// one workgroup per level: running exact sum += the partials; candidate level
// v summed over the wave's 64 lanes (wrapping integer adds, any order), in every lane: the half
// and row swaps, then DPP moves inside a row (the butterfly of the fp64 wave sum)
__device__ __forceinline__ long long wave_sum_i64(long long v) {
    auto add_pair = [](long long x, unsigned lo, unsigned hi) {
        return x + (long long)(((unsigned long long)hi << 32) | lo);
    };
    {
        const auto a = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
        const auto b = __builtin_amdgcn_permlane32_swap((unsigned)(v >> 32), (unsigned)(v >> 32), false, false);
        v = add_pair(add_pair(0, a[0], b[0]), a[1], b[1]);
    }
    {
        const auto a = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
        const auto b = __builtin_amdgcn_permlane16_swap((unsigned)(v >> 32), (unsigned)(v >> 32), false, false);
        v = add_pair(add_pair(0, a[0], b[0]), a[1], b[1]);
    }
    auto dpp = [&](auto ctl) {
        constexpr int C = decltype(ctl)::value;
        const unsigned lo = __builtin_amdgcn_mov_dpp((unsigned)v, C, 0xF, 0xF, true);
        const unsigned hi = __builtin_amdgcn_mov_dpp((unsigned)(v >> 32), C, 0xF, 0xF, true);
        v = add_pair(v, lo, hi);
    };
    dpp(std::integral_constant<int, 0x128>{});  // row_ror:8
    dpp(std::integral_constant<int, 0x124>{});  // row_ror:4
    dpp(std::integral_constant<int, 0x4E>{});   // quad_perm [2,3,0,1]
    dpp(std::integral_constant<int, 0xB1>{});   // quad_perm [1,0,3,2]
    return v;
}

// one 1024-thread workgroup per level: thread b reads partial b (the partials of a level are
// contiguous); a workgroup whose codes did not change added nothing and is skipped (every
// first-pass partial is read)
constexpr int kFcSumThreads = kFcGrid;
__global__ __launch_bounds__(kFcSumThreads) void fc_sum_kernel(const FcParams p, int nblk) {
    __shared__ long long s_acc[kFcSumThreads / kWave][kFcCols];
    if (fc_done(p)) return;
    const int q = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    long long a[kFcCols], run[kFcCols];
#pragma unroll
    for (int c = 0; c < kFcCols; ++c) a[c] = 0;
    if (tid == 0)  // the level's running sums, loaded while the partials are
#pragma unroll
        for (int c = 0; c < kFcCols; ++c) run[c] = p.S[q * kFcCols + c];
    if (tid < nblk && p.wg_changed[tid] != 0) {
        const long long* src = p.part + ((size_t)q * nblk + tid) * kFcCols;
#pragma unroll
        for (int c = 0; c < kFcCols; ++c) a[c] = src[c];
    }
#pragma unroll
    for (int c = 0; c < kFcCols; ++c) a[c] = wave_sum_i64(a[c]);
    if (lane == 0)
        for (int c = 0; c < kFcCols; ++c) s_acc[wave][c] = a[c];
    __syncthreads();
    if (tid == 0) {
        unsigned long long S[kDigits];
#pragma unroll
        for (int c = 0; c < kFcCols; ++c) {
            long long t = run[c];
            for (int w = 0; w < kFcSumThreads / kWave; ++w) t += s_acc[w][c];
            run[c] = t;
            if (c < kDigits) S[c] = (unsigned long long)t;
        }
#pragma unroll
        for (int c = 0; c < kFcCols; ++c) p.S[q * kFcCols + c] = run[c];
        const long long W = run[kDigits];
        p.lev_next[q] = W > 0 ? (float)(digits_to_double(S) / (double)W) : p.lev[q];
    }
}

// run state: stop after a round without a changed code, else take the candidates
__global__ __launch_bounds__(kCbqMaxLevels) void fc_state_kernel(const FcParams p, int nblk) {
    __shared__ int s_any, s_unsorted, s_bad;
    __shared__ float s_lev[kCbqMaxLevels];
    if (fc_done(p)) return;
    const int tid = threadIdx.x, nlev = 1 << p.bits;
    if (tid == 0) {
        s_any = 0;
        s_unsorted = 0;
    }
    __syncthreads();
    for (int b = tid; b < nblk; b += blockDim.x)
        if (p.wg_changed[b]) s_any = 1;
    __syncthreads();
    const bool update = s_any && p.state[1] < p.iters;
    if (update && tid < nlev) {
        s_lev[tid] = p.lev_next[tid];
        p.lev[tid] = s_lev[tid];
    }
    __syncthreads();
    if (update && tid + 1 < nlev && !(s_lev[tid] <= s_lev[tid + 1])) s_unsorted = 1;
    __syncthreads();
    if (update) set_thresholds(p, s_lev, nlev, s_unsorted, &s_bad, p.range[0], p.range[1], p.range[2]);  // uniform
    if (tid == 0) {
        if (update) {
            p.state[1] += 1;
            p.state[2] = s_unsorted;
        } else {
            p.state[0] = 1;
        }
    }
}

__global__ __launch_bounds__(kFcThreads) void fc_output_kernel(const FcParams p) {
    __shared__ float s_lev[kCbqMaxLevels];
    const int tid = threadIdx.x, nlev = 1 << p.bits;
    for (int e = tid; e < nlev; e += kFcThreads) s_lev[e] = p.lev[e];
    __syncthreads();
    if (blockIdx.x == 0) {
        for (int e = tid; e < nlev; e += kFcThreads) p.levels_out[e] = s_lev[e];
        if (tid == 0 && p.rounds_out) *p.rounds_out = p.state[1];
    }
    if (!p.v_hat) return;
    long long r0 = 0;  // scalars from here on: one at a time
    if ((reinterpret_cast<uintptr_t>(p.v_hat) & 15u) == 0 && (reinterpret_cast<uintptr_t>(p.codes) & 3u) == 0) {
        // a word of four codes in, a float4 out; four groups per thread in flight
        constexpr int kPer = 4;
        const long long ng = p.m >> 2;
        const unsigned* __restrict__ c4 = reinterpret_cast<const unsigned*>(p.codes);
        float4* __restrict__ o4 = reinterpret_cast<float4*>(p.v_hat);
        for (long long g0 = (long long)blockIdx.x * kFcThreads * kPer + tid; g0 < ng;
             g0 += (long long)gridDim.x * kFcThreads * kPer) {
            unsigned cw[kPer];
#pragma unroll
            for (int j = 0; j < kPer; ++j) {
                const long long g = g0 + (long long)j * kFcThreads;
                cw[j] = g < ng ? c4[g] : 0u;
            }
#pragma unroll
            for (int j = 0; j < kPer; ++j) {
                const long long g = g0 + (long long)j * kFcThreads;
                if (g < ng)
                    o4[g] = make_float4(s_lev[cw[j] & 255u], s_lev[(cw[j] >> 8) & 255u], s_lev[(cw[j] >> 16) & 255u],
                                        s_lev[cw[j] >> 24]);
            }
        }
        r0 = 4 * ng;
    }
    for (long long r = r0 + (long long)blockIdx.x * kFcThreads + tid; r < p.m; r += (long long)gridDim.x * kFcThreads)
        p.v_hat[r] = s_lev[p.codes[r]];
}

int fc_grid(long long m) {
    const long long b = (m + 4 * kFcThreads - 1) / (4 * kFcThreads);
    return (int)(b < kFcGrid ? (b < 1 ? 1 : b) : kFcGrid);
}

hipError_t launch_fc_quantize(const FcParams& p, hipStream_t s) {
    const int G = fc_grid(p.m), nlev = 1 << p.bits;
    hipLaunchKernelGGL(fc_minmax_kernel, dim3(G), dim3(kFcThreads), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fc_grid_kernel, dim3(1), dim3(kCbqMaxLevels), 0, s, p, G);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // the initial codes and sums, then `iters` rounds of (levels, codes)
    for (int r = 0; r <= p.iters; ++r) {
        e = r == 0 ? launch_fc_assign<true>(p, G, s) : launch_fc_assign<false>(p, G, s);
        if (e != hipSuccess) return e;
        if (r == p.iters) break;  // the last codes need no further levels
        hipLaunchKernelGGL(fc_sum_kernel, dim3(nlev), dim3(kFcSumThreads), 0, s, p, G);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(fc_state_kernel, dim3(1), dim3(kCbqMaxLevels), 0, s, p, G);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fc_output_kernel, dim3(G), dim3(kFcThreads), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_cbq(const CbqParams& p, hipStream_t s) {
    int mmax = 0;
    for (int l = 0; l < p.nlayers; ++l) mmax = p.L[l].k * kDim > mmax ? p.L[l].k * kDim : mmax;
    const bool fast = p.bits == 6;
    if (mmax <= kCbqLdsScalars && fast)
        hipLaunchKernelGGL((cbq_kernel<true, true>), dim3(p.nlayers), dim3(kCbqThreads), 0, s, p);
    else if (mmax <= kCbqLdsScalars)
        hipLaunchKernelGGL((cbq_kernel<true, false>), dim3(p.nlayers), dim3(kCbqThreads), 0, s, p);
    else if (fast)
        hipLaunchKernelGGL((cbq_kernel<false, true>), dim3(p.nlayers), dim3(kCbqThreads), 0, s, p);
    else
        hipLaunchKernelGGL((cbq_kernel<false, false>), dim3(p.nlayers), dim3(kCbqThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace kq
