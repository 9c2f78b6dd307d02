// Backward of Forgetting Attention over the blocks kept by ACP.
//
// The paper states only that the backward pass is built like the forward
// (Sec. 2, FlashAttention paragraph).  With x_ij = q_i.k_j/sqrt(d) + c_i - c_j,
// P = softmax_row(x) on the kept, causal entries, and the pruning mask held
// constant, the chain rule through eq. 2 and c gives
//   dV = P^T dO,  dP = dO V^T,  Delta_i = dO_i . O_i,  dS = P o (dP - Delta),
//   dQ = dS K / sqrt(d),  dK = dS^T Q / sqrt(d),
//   dc_i = sum_j dS_ij - sum_j dS_ji,  dlog f_l = sum_{i >= l} dc_i.
//
// Four launches:
//   dsum_kernel   Delta = rowdot(dO, O) (float32 path; the bf16 dQ pass forms
//                 Delta itself from the rows of O and dO it holds)
//   dq kernel     per query block, loops over kept key blocks: dQ, then
//                 Delta'_i = sum_j P_ij dP_ij (replacing Delta) and the row sums
//                 of dS (bf16: fox_bwd_mfma.hip; fp32: below)
//   dkdv kernel   per key block, loops over the query blocks that keep it: dK,
//                 dV and the column sums of dS
//   dlogf_kernel  reverse cumulative sum of (row sum - column sum)
// dQ is produced by its own pass (recomputing S and dP) rather than by atomic
// accumulation from the key-block pass, so every output is written once.
#include "acp_device.h"
#include "acp_internal.h"
#include "acp_scan.h"

namespace acp {

// ---------------------------------------------------------------------------
// Delta_i = sum_d dO_id O_id: 16 lanes per row.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void dsum_kernel(const float* __restrict__ dO,
                                                   const float* __restrict__ O,
                                                   float* __restrict__ dsum, size_t rows) {
    constexpr int E = D / 16;
    const size_t gt = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t row = gt / 16;
    const int sub = (int)(gt % 16);
    float acc = 0.f;
    if (row < rows) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const size_t off = row * D + sub * E + e;
            acc = __builtin_fmaf(dO[off], O[off], acc);
        }
    }
    acc += __shfl_xor(acc, 8);
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 1);
    if (row < rows && sub == 0) dsum[row] = acc;
}

// ---------------------------------------------------------------------------
// fp32 path (plain VALU): dQ/rowsum with one thread per query, dK/dV/colsum
// with one thread per key, tiles staged in LDS.  Off the diagonal tile the decay
// c_i - c_j is split at R, the gate at the boundary of the thread's own block
// (first query, resp. last key), into two parts of the same sign; on the
// diagonal tile it is formed per entry (see fox_fwd.hip).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void dq_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ dO, const float* __restrict__ cg,
    const int* __restrict__ row_start, const float* __restrict__ lse2,
    float* __restrict__ dsum, float* __restrict__ dQ, float* __restrict__ rowsum,
    int L, int M, float kscale, float qscale) {
    __shared__ float ks[64 * D];
    __shared__ float vs[64 * D];
    __shared__ float nc[64];   // (R - c_j) log2(e), or c_j on the diagonal tile
    const int bh = blockIdx.x / M, m = blockIdx.x % M, t = threadIdx.x;
    const size_t head = (size_t)bh * L;
    const size_t row = head + 64 * m + t;
    float q[D], go[D], acc[D];
#pragma unroll
    for (int k = 0; k < D; ++k) { q[k] = Q[row * D + k]; go[k] = dO[row * D + k]; acc[k] = 0.f; }
    const float rref = cg[head + 64 * m];
    const float ci = cg[row];
    const float l2 = (ci - rref) * kLog2e - lse2[row], l2d = -lse2[row], dl = dsum[row];
    float pdp = 0.f, psum = 0.f;
    for (int n = row_start[(size_t)bh * M + m]; n <= m; ++n) {
        __syncthreads();
        for (int i = t; i < 64 * D; i += 64) {
            ks[i] = K[(head + 64 * n) * D + i];
            vs[i] = V[(head + 64 * n) * D + i];
        }
        const float cj = cg[head + 64 * n + t];
        nc[t] = n == m ? cj : (rref - cj) * kLog2e;
        __syncthreads();
        const int jmax = (n == m) ? t : 63;
        for (int j = 0; j <= jmax; ++j) {
            float s = 0.f, dp = 0.f;
#pragma unroll
            for (int k = 0; k < D; ++k) {
                s = __builtin_fmaf(q[k], ks[j * D + k], s);
                dp = __builtin_fmaf(go[k], vs[j * D + k], dp);
            }
            const float p = n == m ? fast_exp2(__builtin_fmaf(s, kscale, (ci - nc[j]) * kLog2e) + l2d)
                                   : fast_exp2(__builtin_fmaf(s, kscale, nc[j]) + l2);
            const float dsv = p * (dp - dl);
            pdp = __builtin_fmaf(p, dp, pdp);
            psum += p;
#pragma unroll
            for (int k = 0; k < D; ++k) acc[k] = __builtin_fmaf(dsv, ks[j * D + k], acc[k]);
        }
    }
#pragma unroll
    for (int k = 0; k < D; ++k) dQ[row * D + k] = acc[k] * qscale;
    dsum[row] = pdp;               // Delta' as in the bfloat16 pass
    rowsum[row] = pdp - pdp * psum;
}

template <int D>
__global__ __launch_bounds__(64) void dkdv_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ dO, const float* __restrict__ cg,
    const int* __restrict__ col_end, const float* __restrict__ lse2,
    const float* __restrict__ dsum, float* __restrict__ dK, float* __restrict__ dV,
    float* __restrict__ colsum, int L, int M, float kscale, float qscale) {
    __shared__ float qs[64 * D];
    __shared__ float os[64 * D];
    __shared__ float ls[64];   // (c_i - R) log2(e) - L_i, or -L_i on the diagonal tile
    __shared__ float lcs[64];  // c_i (diagonal tile)
    __shared__ float dls[64];
    const int bh = blockIdx.x / M, n = blockIdx.x % M, t = threadIdx.x;
    const size_t head = (size_t)bh * L;
    const size_t row = head + 64 * n + t;
    float kk[D], vv[D], gk[D], gv[D];
#pragma unroll
    for (int k = 0; k < D; ++k) { kk[k] = K[row * D + k]; vv[k] = V[row * D + k]; gk[k] = 0.f; gv[k] = 0.f; }
    const float rref = cg[head + 64 * n + 63];
    const float cj = cg[row];
    const float nk = (rref - cj) * kLog2e;
    float cs = 0.f;
    const int mend = col_end[(size_t)bh * M + n];
    for (int m = n; m <= mend; ++m) {
        __syncthreads();
        for (int i = t; i < 64 * D; i += 64) {
            qs[i] = Q[(head + 64 * m) * D + i];
            os[i] = dO[(head + 64 * m) * D + i];
        }
        const float cr = cg[head + 64 * m + t];
        ls[t] = m == n ? -lse2[head + 64 * m + t] : (cr - rref) * kLog2e - lse2[head + 64 * m + t];
        lcs[t] = cr;
        dls[t] = dsum[head + 64 * m + t];
        __syncthreads();
        const int i0 = (m == n) ? t : 0;
        for (int i = i0; i < 64; ++i) {
            float s = 0.f, dp = 0.f;
#pragma unroll
            for (int k = 0; k < D; ++k) {
                s = __builtin_fmaf(qs[i * D + k], kk[k], s);
                dp = __builtin_fmaf(os[i * D + k], vv[k], dp);
            }
            const float p = m == n ? fast_exp2(__builtin_fmaf(s, kscale, (lcs[i] - cj) * kLog2e) + ls[i])
                                   : fast_exp2(__builtin_fmaf(s, kscale, nk) + ls[i]);
            const float dsv = p * (dp - dls[i]);
            cs += dsv;
#pragma unroll
            for (int k = 0; k < D; ++k) {
                gv[k] = __builtin_fmaf(p, os[i * D + k], gv[k]);
                gk[k] = __builtin_fmaf(dsv, qs[i * D + k], gk[k]);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < D; ++k) {
        dK[row * D + k] = gk[k] * qscale;
        dV[row * D + k] = gv[k];
    }
    colsum[row] = cs;
}

// ---------------------------------------------------------------------------
// dlog f_l = sum_{i >= l} (rowsum_i - colsum_i), accumulated in float64.  Each
// thread owns a contiguous run (held in registers up to kScanHeld values); one
// round through LDS carries the waves' totals for the suffix sums.
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 1024;
constexpr int kScanHeld = 16;

__global__ __launch_bounds__(kScanThreads) void dlogf_kernel(const float* __restrict__ rowsum,
                                                             const float* __restrict__ colsum,
                                                             float* __restrict__ dlog_f, int L) {
    constexpr int kWaves = kScanThreads / 64;
    __shared__ double s_tot[kWaves];
    const int bh = blockIdx.x, t = threadIdx.x, lane = t & 63, wid = t >> 6;
    const size_t head = (size_t)bh * L;
    const int per = (L + kScanThreads - 1) / kScanThreads;
    const int beg = min(t * per, L), n = min(beg + per, L) - beg;
    const bool held = per <= kScanHeld;
    const bool vec = held && (per & 3) == 0;   // then n is per or 0: float4 accesses
    double dv[kScanHeld];
    if (vec) {
#pragma unroll
        for (int i = 0; i < kScanHeld; i += 4) {
            float4 r = make_float4(0.f, 0.f, 0.f, 0.f), c = r;
            if (i < n) {
                r = *reinterpret_cast<const float4*>(rowsum + head + beg + i);
                c = *reinterpret_cast<const float4*>(colsum + head + beg + i);
            }
            dv[i] = (double)r.x - (double)c.x;
            dv[i + 1] = (double)r.y - (double)c.y;
            dv[i + 2] = (double)r.z - (double)c.z;
            dv[i + 3] = (double)r.w - (double)c.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < kScanHeld; ++i)
            dv[i] = held && i < n ? (double)rowsum[head + beg + i] - (double)colsum[head + beg + i] : 0.0;
    }
    double local = 0.0;
    if (held) {
#pragma unroll
        for (int i = 0; i < kScanHeld; ++i) local += dv[i];
    } else {
        for (int i = 0; i < n; ++i) local += (double)rowsum[head + beg + i] - (double)colsum[head + beg + i];
    }
    // inclusive suffix sums over the lanes of the wave: within each row of 16 by
    // zero-filled shifts toward lower lanes, then the totals of the later rows
    // (lane 16 r holds row r's)
    double suf = local;
    suf += dpp_f64_or_zero<0x101>(suf);   // row_shl:1
    suf += dpp_f64_or_zero<0x102>(suf);   // row_shl:2
    suf += dpp_f64_or_zero<0x104>(suf);   // row_shl:4
    suf += dpp_f64_or_zero<0x108>(suf);   // row_shl:8
    {
        const double t1 = readlane_f64(suf, 16), t2 = readlane_f64(suf, 32), t3 = readlane_f64(suf, 48);
        const int row = lane >> 4;
        suf += row == 0 ? (t1 + t2) + t3 : row == 1 ? t2 + t3 : row == 2 ? t3 : 0.0;
    }
    if (lane == 0) s_tot[wid] = suf;
    __syncthreads();
    // the waves after this one: lane l < 16 takes wave l's total, summed over the row
    double after;
    {
        const double v = lane < kWaves && lane > wid ? s_tot[lane] : 0.0;
        after = readlane_f64(row16_reduce(v, [](double x, double y) { return x + y; }), 0);
    }
    double run = after + (suf - local);   // sum over the threads after this one
    if (vec) {
#pragma unroll
        for (int i = kScanHeld - 4; i >= 0; i -= 4) {
            if (i < n) {
                float4 o;
                run += dv[i + 3]; o.w = (float)run;
                run += dv[i + 2]; o.z = (float)run;
                run += dv[i + 1]; o.y = (float)run;
                run += dv[i];     o.x = (float)run;
                *reinterpret_cast<float4*>(dlog_f + head + beg + i) = o;
            }
        }
    } else if (held) {
#pragma unroll
        for (int i = kScanHeld - 1; i >= 0; --i) {
            if (i < n) {
                run += dv[i];
                dlog_f[head + beg + i] = (float)run;
            }
        }
    } else {
        for (int i = n - 1; i >= 0; --i) {
            run += (double)rowsum[head + beg + i] - (double)colsum[head + beg + i];
            dlog_f[head + beg + i] = (float)run;
        }
    }
}

// ---------------------------------------------------------------------------
hipError_t launch_bwd(const BwdArgs& a, hipStream_t s) {
    const int BH = a.B * a.H, M = a.L / 64;
    const float kscale = kLog2e / sqrtf((float)a.d);
    const float qscale = 1.0f / sqrtf((float)a.d);
    const size_t rows = (size_t)BH * a.L;
    const unsigned dgrid = (unsigned)((rows * 16 + 255) / 256);
    hipError_t e;
    if (!a.bf16) {
        trace_begin(ACP_K_DSUM, s);
        if (a.d == 64)
            hipLaunchKernelGGL(dsum_kernel<64>, dim3(dgrid), dim3(256), 0, s,
                               (const float*)a.dO, (const float*)a.O, a.dsum, rows);
        else
            hipLaunchKernelGGL(dsum_kernel<128>, dim3(dgrid), dim3(256), 0, s,
                               (const float*)a.dO, (const float*)a.O, a.dsum, rows);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        trace_end(ACP_K_DSUM, s);
    }

    trace_begin(ACP_K_DQ, s);
    if (a.bf16) {
        e = launch_dq_bf16(a, s);
    } else {
#define ACP_DQ32(DD)                                                                       \
    hipLaunchKernelGGL(dq_f32_kernel<DD>, dim3(BH * M), dim3(64), 0, s,                    \
                       (const float*)a.Q, (const float*)a.K, (const float*)a.V,            \
                       (const float*)a.dO, a.c, a.row_start, a.lse2, a.dsum,               \
                       (float*)a.dQ, a.rowsum, a.L, M, kscale, qscale)
        if (a.d == 64) { ACP_DQ32(64); } else { ACP_DQ32(128); }
#undef ACP_DQ32
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    trace_end(ACP_K_DQ, s);

    trace_begin(ACP_K_DKDV, s);
    if (a.bf16) {
        e = launch_dkdv_bf16(a, s);
    } else {
#define ACP_DKV32(DD)                                                                      \
    hipLaunchKernelGGL(dkdv_f32_kernel<DD>, dim3(BH * M), dim3(64), 0, s,                  \
                       (const float*)a.Q, (const float*)a.K, (const float*)a.V,            \
                       (const float*)a.dO, a.c, a.col_end, a.lse2, a.dsum,                 \
                       (float*)a.dK, (float*)a.dV, a.colsum, a.L, M, kscale, qscale)
        if (a.d == 64) { ACP_DKV32(64); } else { ACP_DKV32(128); }
#undef ACP_DKV32
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    trace_end(ACP_K_DKDV, s);

    trace_begin(ACP_K_DLOGF, s);
    hipLaunchKernelGGL(dlogf_kernel, dim3(BH), dim3(kScanThreads), 0, s, a.rowsum, a.colsum,
                       a.dlog_f, a.L);
    e = hipGetLastError();
    trace_end(ACP_K_DLOGF, s);
    return e;
}

}  // namespace acp
