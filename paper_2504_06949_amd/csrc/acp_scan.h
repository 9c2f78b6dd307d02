// Workgroup-wide scans and reductions for the 1024-thread per-head kernels
// (stage 1 and the decoding set-up), double-double sums for the cumulative
// gates, and the float32 last-bit position used to bound their span.
#pragma once

#include "acp_device.h"

namespace acp {

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;

// Reductions over the 16 lanes of each row of a wave (DPP: swap neighbours, swap
// pairs, mirror halves of 8, mirror the 16); every lane of the row ends with the
// row's result.
__device__ __forceinline__ double dpp_f64(double v, int ctrl_id) {
    const unsigned long long b = __double_as_longlong(v);
    int lo = (int)(unsigned)b, hi = (int)(unsigned)(b >> 32);
    switch (ctrl_id) {
        case 0: lo = __builtin_amdgcn_mov_dpp(lo, 0xB1, 0xF, 0xF, false);
                hi = __builtin_amdgcn_mov_dpp(hi, 0xB1, 0xF, 0xF, false); break;
        case 1: lo = __builtin_amdgcn_mov_dpp(lo, 0x4E, 0xF, 0xF, false);
                hi = __builtin_amdgcn_mov_dpp(hi, 0x4E, 0xF, 0xF, false); break;
        case 2: lo = __builtin_amdgcn_mov_dpp(lo, 0x141, 0xF, 0xF, false);
                hi = __builtin_amdgcn_mov_dpp(hi, 0x141, 0xF, 0xF, false); break;
        default: lo = __builtin_amdgcn_mov_dpp(lo, 0x140, 0xF, 0xF, false);
                 hi = __builtin_amdgcn_mov_dpp(hi, 0x140, 0xF, 0xF, false); break;
    }
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
__device__ __forceinline__ int dpp_i32(int v, int ctrl_id) {
    switch (ctrl_id) {
        case 0: return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);
        case 1: return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);
        case 2: return __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false);
        default: return __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false);
    }
}
template <typename Op>
__device__ __forceinline__ double row16_reduce(double v, Op op) {
#pragma unroll
    for (int c = 0; c < 4; ++c) v = op(v, dpp_f64(v, c));
    return v;
}
template <typename Op>
__device__ __forceinline__ int row16_reduce(int v, Op op) {
#pragma unroll
    for (int c = 0; c < 4; ++c) v = op(v, dpp_i32(v, c));
    return v;
}

// DPP move of a double (both halves): lanes whose source lies outside their row,
// and rows outside ROW_MASK, receive 0.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ double dpp_f64_or_zero(double v) {
    const unsigned long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)b, CTRL, ROW_MASK, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(b >> 32), CTRL, ROW_MASK, 0xF, true);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

// Inclusive prefix sum over the 64 lanes of a wave: within each row of 16 by
// zero-filled shifts of 1, 2, 4 and 8, then the last lane of row 0 into row 1 and
// of row 2 into row 3, then lane 31 into rows 2 and 3 (any association: the
// callers only add values whose float64 sums are exact).
__device__ __forceinline__ double wave_inclusive_scan_f64(double v) {
    v += dpp_f64_or_zero<0x111>(v);         // row_shr:1
    v += dpp_f64_or_zero<0x112>(v);         // row_shr:2
    v += dpp_f64_or_zero<0x114>(v);         // row_shr:4
    v += dpp_f64_or_zero<0x118>(v);         // row_shr:8
    v += dpp_f64_or_zero<0x142, 0xA>(v);    // row_bcast:15
    v += dpp_f64_or_zero<0x143, 0xC>(v);    // row_bcast:31
    return v;
}

__device__ __forceinline__ int readlane_any(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ double readlane_f64(double v, int l);
__device__ __forceinline__ double readlane_any(double v, int l) { return readlane_f64(v, l); }
__device__ __forceinline__ double readlane_f64(double v, int l) {
    const unsigned long long b = __double_as_longlong(v);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)b, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(b >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}


// The value of lane 0 (wave-uniform), as a scalar.
__device__ __forceinline__ double readfirst_f64(double v) {
    const unsigned long long b = __double_as_longlong(v);
    const unsigned lo = (unsigned)__builtin_amdgcn_readfirstlane((int)(unsigned)b);
    const unsigned hi = (unsigned)__builtin_amdgcn_readfirstlane((int)(unsigned)(b >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Inclusive prefix sum over the workgroup of one double per thread (any
// association: the callers only add values whose float64 sums are exact).
__device__ inline double block_inclusive_scan(double v, double* s_wave) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v = wave_inclusive_scan_f64(v);
    if (lane == 63) s_wave[wid] = v;
    __syncthreads();
    if (wid == 0) {
        double w = lane < kPlanWaves ? s_wave[lane] : 0.0;
        w = wave_inclusive_scan_f64(w);
        if (lane < kPlanWaves) s_wave[lane] = w;   // inclusive wave totals
    }
    __syncthreads();
    const double before = wid > 0 ? s_wave[wid - 1] : 0.0;
    const double out = v + before;
    __syncthreads();  // s_wave may be reused by the caller
    return out;
}

template <typename V, typename Op>
__device__ inline V block_reduce(V v, V* s_wave, Op op) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const V rr = row16_reduce(v, op);   // then the four rows' results
    v = op(op(readlane_any(rr, 0), readlane_any(rr, 16)), op(readlane_any(rr, 32), readlane_any(rr, 48)));
    if (lane == 0) s_wave[wid] = v;
    __syncthreads();
    V r = s_wave[0];
    for (int w = 1; w < kPlanWaves; ++w) r = op(r, s_wave[w]);
    __syncthreads();
    return r;
}

// Position of the last bit of a float32 value: it is an integer multiple of
// 2^lsb_exp(x).  Subnormals share the exponent of the smallest normal.
__device__ __forceinline__ int lsb_exp(float x) {
    const int biased = (int)((__float_as_uint(x) >> 23) & 0xff);
    return (biased > 0 ? biased : 1) - 150;
}

// ---- double-double sums of log f ---------------------------------------------------
// c is the float32 rounding of the exact prefix sum of the float32 gates.  A sum
// is carried as a pair (hi, lo): hi the float64 rounding of the value, lo the
// exact remainder.  Every gate is a multiple of 2^lsb (lsb the smallest ulp
// exponent among them) and every partial sum, in any association, lies below
// 2^E (the least power of two above sum |log f|).  Adding two such pairs by
// TwoSum (Knuth) on the leading parts, a plain sum of the remainders and the
// error, and TwoSum again keeps the pair exact while E - lsb <= 105: the
// remainders are then multiples of 2^lsb below 2^(E - 52), which float64 holds
// exactly.  Stage 1 flags wider spans (flag bit 2).
struct DD {
    double hi, lo;
};
constexpr int kExactSpanBits = 105;   // flag bit 2 from this span on

// (a non-finite sum keeps lo = 0, so that an infinite or NaN gate propagates
// through hi as it would through a plain float64 sum)
__device__ __forceinline__ DD two_sum(double a, double b) {
    const double s = a + b;
    const double bb = s - a;
    const double e = (a - (s - bb)) + (b - bb);
    return DD{s, __builtin_isfinite(s) ? e : 0.0};
}
__device__ __forceinline__ DD dd_add(DD a, DD b) {
    const DD s = two_sum(a.hi, b.hi);
    return two_sum(s.hi, (a.lo + b.lo) + s.lo);
}
__device__ __forceinline__ DD dd_add(DD a, double b) {
    const DD s = two_sum(a.hi, b);
    return two_sum(s.hi, a.lo + s.lo);
}
__device__ __forceinline__ DD dd_neg(DD a) { return DD{-a.hi, -a.lo}; }

// Running sums of float32 gates in either precision (float64 where the span
// allows it, else pairs), and their float32 value.
__device__ __forceinline__ double sum_add(double r, float x) { return r + (double)x; }
__device__ __forceinline__ DD sum_add(DD r, float x) { return dd_add(r, (double)x); }

// The float32 rounding (to nearest, ties to even) of hi + lo.  hi is the nearest
// float64 to the value and every float32 midpoint is a float64, so the rounding
// of hi is that of the value unless hi is itself a midpoint; then lo decides.
__device__ __forceinline__ float dd_to_f32(DD a) {
    float r = (float)a.hi;
    if (a.lo == 0.0) return r;
    const double rd = (double)r;
    if (__builtin_isinf(r)) {
        // hi at or beyond the overflow threshold (the largest float32 plus half an
        // ulp): the value stays below it only if hi is exactly that threshold and
        // lo points back
        const double thr = 3.4028235677973366e38;   // (2 - 2^-24) 2^127
        if (__builtin_fabs(a.hi) == thr && (a.lo < 0.0) == (a.hi > 0.0))
            r = a.hi > 0.0 ? 3.4028234663852886e38f : -3.4028234663852886e38f;
        return r;
    }
    if (a.hi == rd) return r;                       // hi is a float32: |lo| is below its half ulp
    // the float32 on the other side of hi (same sign: rounding keeps it)
    const unsigned rb = __float_as_uint(r);
    const unsigned mag = rb & 0x7fffffffu;
    const bool away = __builtin_fabs(a.hi) > __builtin_fabs(rd);
    const float other = __uint_as_float((rb & 0x80000000u) | (away ? mag + 1u : mag - 1u));
    const double od = (double)other;
    if (a.hi == 0.5 * (rd + od) && ((a.lo > 0.0) == (od > rd))) r = other;
    return r;
}

__device__ __forceinline__ float sum_f32(double r) { return (float)r; }
__device__ __forceinline__ float sum_f32(DD r) { return dd_to_f32(r); }
__device__ __forceinline__ double sum_hi(double r) { return r; }
__device__ __forceinline__ double sum_lo(double) { return 0.0; }
__device__ __forceinline__ double sum_hi(DD r) { return r.hi; }
__device__ __forceinline__ double sum_lo(DD r) { return r.lo; }

// Least E with |value| < 2^E for a positive pair (the span bound above).
__device__ __forceinline__ int dd_top_exp(DD a) {
    const unsigned long long b = (unsigned long long)__double_as_longlong(a.hi);
    const int biased = (int)((b >> 52) & 0x7ff);
    int top = (biased > 0 ? biased : 1) - 1023 + 1;       // hi in [2^(top-1), 2^top)
    if ((b & 0xFFFFFFFFFFFFFull) == 0 && biased > 0 && a.lo < 0.0) --top;   // just below a power of two
    return top;
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ DD dpp_dd_or_zero(DD v) {
    return DD{dpp_f64_or_zero<CTRL, ROW_MASK>(v.hi), dpp_f64_or_zero<CTRL, ROW_MASK>(v.lo)};
}
// wave_inclusive_scan_f64 on pairs
__device__ __forceinline__ DD wave_inclusive_scan_dd(DD v) {
    v = dd_add(v, dpp_dd_or_zero<0x111>(v));
    v = dd_add(v, dpp_dd_or_zero<0x112>(v));
    v = dd_add(v, dpp_dd_or_zero<0x114>(v));
    v = dd_add(v, dpp_dd_or_zero<0x118>(v));
    v = dd_add(v, dpp_dd_or_zero<0x142, 0xA>(v));
    v = dd_add(v, dpp_dd_or_zero<0x143, 0xC>(v));
    return v;
}
__device__ __forceinline__ DD row16_sum_dd(DD v) {
#pragma unroll
    for (int c = 0; c < 4; ++c) v = dd_add(v, DD{dpp_f64(v.hi, c), dpp_f64(v.lo, c)});
    return v;
}
__device__ __forceinline__ DD readlane_dd(DD v, int l) {
    return DD{readlane_f64(v.hi, l), readlane_f64(v.lo, l)};
}
// Sum over the 64 lanes of a wave, every lane receiving it.
__device__ __forceinline__ DD wave_sum_dd(DD v) {
    const DD r = row16_sum_dd(v);
    return dd_add(dd_add(readlane_dd(r, 0), readlane_dd(r, 16)),
                  dd_add(readlane_dd(r, 32), readlane_dd(r, 48)));
}
// Sum over the 64 lanes in float64 when that is exact: every lane's low part is
// zero and no addition rounds (each one's TwoSum error is checked off the
// critical path).  Returns false, uniformly over the wave, otherwise; the caller
// then takes wave_sum_dd.
__device__ __forceinline__ bool wave_sum_f64_if_exact(DD v, double& out) {
    bool inexact = v.lo != 0.0;
    double s = v.hi;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const DD t = two_sum(s, dpp_f64(s, c));
        inexact = inexact || t.lo != 0.0;
        s = t.hi;
    }
    const DD a = two_sum(readlane_f64(s, 0), readlane_f64(s, 16));
    const DD b = two_sum(readlane_f64(s, 32), readlane_f64(s, 48));
    const DD r = two_sum(a.hi, b.hi);
    inexact = inexact || a.lo != 0.0 || b.lo != 0.0 || r.lo != 0.0;
    out = r.hi;
    return __ballot(inexact) == 0ull;
}
// Inclusive prefix sum over the 1024-thread workgroup (s_hi, s_lo: kPlanWaves each).
__device__ inline DD block_inclusive_scan_dd(DD v, double* s_hi, double* s_lo) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v = wave_inclusive_scan_dd(v);
    if (lane == 63) {
        s_hi[wid] = v.hi;
        s_lo[wid] = v.lo;
    }
    __syncthreads();
    if (wid == 0) {
        DD w = lane < kPlanWaves ? DD{s_hi[lane], s_lo[lane]} : DD{0.0, 0.0};
        w = wave_inclusive_scan_dd(w);
        if (lane < kPlanWaves) {
            s_hi[lane] = w.hi;
            s_lo[lane] = w.lo;
        }
    }
    __syncthreads();
    const DD out = wid > 0 ? dd_add(v, DD{s_hi[wid - 1], s_lo[wid - 1]}) : v;
    __syncthreads();
    return out;
}
// Sum over the workgroup, every thread receiving it.
__device__ inline DD block_sum_dd(DD v, double* s_hi, double* s_lo) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v = wave_sum_dd(v);
    if (lane == 0) {
        s_hi[wid] = v.hi;
        s_lo[wid] = v.lo;
    }
    __syncthreads();
    DD r{s_hi[0], s_lo[0]};
    for (int w = 1; w < kPlanWaves; ++w) r = dd_add(r, DD{s_hi[w], s_lo[w]});
    __syncthreads();
    return r;
}

}  // namespace acp
