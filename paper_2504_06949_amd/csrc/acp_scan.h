// Workgroup-wide scans and reductions for the 1024-thread per-head kernels
// (stage 1 and the decoding set-up), and the float32 last-bit position used to
// check that float64 prefix sums of log f are exact.
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

}  // namespace acp
