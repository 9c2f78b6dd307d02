// Stage 1 of ACP on the GPU: logit bound, threshold, cumulative gates and the
// pruning boundary (Sec. 3 of the paper: "Safe pruning via a dynamically set
// threshold", "Block-level pruning", "Two-stage implementation", Algorithm 1).
//
// Two launches:
//   rownorm_max_kernel  - HBM-bound pass over Q and K: per 128-row chunk, the
//                         largest float64 squared row norm (ascending-k sums).
//   plan_kernel         - one workgroup per (batch, head): reduce the chunk
//                         maxima to rho_q^2, rho_k^2, form U and delta, scan
//                         log f into c, then find every row's first kept block
//                         and every column's last kept block.
// With QK-norm scale bounds (App. E: U = gamma_q gamma_k sqrt(d)) the first
// launch is skipped and the plan kernel takes U from the scales.
#include "acp_device.h"
#include "acp_internal.h"
#include "acp_scan.h"

namespace acp {

constexpr int kNormRows = 128;  // rows per norm workgroup, one per thread

template <typename T, int D>
__global__ __launch_bounds__(kNormRows) void rownorm_max_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, int L, int nchunk,
    double* __restrict__ part) {
    constexpr int kRowBytes = D * (int)sizeof(T);
    constexpr int kChunks = kRowBytes / 16;   // 16-byte pieces per row
    constexpr int kStride = kRowBytes + 16;   // padded LDS row (spreads banks)
    constexpr int kPer = 16 / (int)sizeof(T); // elements per piece
    __shared__ __attribute__((aligned(16))) unsigned char tile[kNormRows * kStride];
    __shared__ double wave_max[kNormRows / 64];

    const int chunk = blockIdx.x, bh = blockIdx.y, which = blockIdx.z;
    const int row0 = chunk * kNormRows;
    const int rows = min(kNormRows, L - row0);
    const T* X = (which == 0 ? Q : K) + ((size_t)bh * L + row0) * D;
    const unsigned char* src = reinterpret_cast<const unsigned char*>(X);

    // Coalesced copy of the chunk into LDS, one padded row per query/key.
    for (int i = threadIdx.x; i < rows * kChunks; i += kNormRows) {
        const uint4 v = *reinterpret_cast<const uint4*>(src + (size_t)i * 16);
        *reinterpret_cast<uint4*>(tile + (i / kChunks) * kStride + (i % kChunks) * 16) = v;
    }
    __syncthreads();

    // Each thread: sum of squares of its row in ascending feature order, in
    // float64.  Squares of float32/bfloat16 values are exact in float64, so
    // fma(x, x, acc) rounds exactly like acc + x*x.
    double acc = 0.0;
    if ((int)threadIdx.x < rows) {
        const unsigned char* rp = tile + threadIdx.x * kStride;
        for (int ch = 0; ch < kChunks; ++ch) {
            const uint4 v = *reinterpret_cast<const uint4*>(rp + ch * 16);
            const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
            for (int t = 0; t < kPer; ++t) {
                const double x = to_f64(e[t]);
                acc = __builtin_fma(x, x, acc);
            }
        }
    }
    // max over the workgroup (order-free)
    double m = acc;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = nan_max(m, __shfl_xor(m, off));
    if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        double r = wave_max[0];
        for (int w = 1; w < kNormRows / 64; ++w) r = nan_max(r, wave_max[w]);
        part[((size_t)bh * 2 + which) * nchunk + chunk] = r;
    }
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(
    const float* __restrict__ log_f, const double* __restrict__ part, int nchunk,
    const float* __restrict__ gamma_q, const float* __restrict__ gamma_k, int H,
    int L, int d, double log_l_over_eps,
    float* __restrict__ c_out,
    double* __restrict__ u_out, double* __restrict__ delta_out,
    int* __restrict__ row_start, int* __restrict__ col_end,
    long long* __restrict__ kept_out, int* __restrict__ flags_out) {
    __shared__ double s_dbl[kPlanWaves];
    __shared__ double s_dbl2[kPlanWaves];
    __shared__ int s_int[kPlanWaves];
    __shared__ long long s_ll[kPlanWaves];
    __shared__ float s_first[kMaxBlocks];  // c at the first row of each block
    __shared__ float s_last[kMaxBlocks];   // c at the last row of each block
    __shared__ int s_rs[kMaxBlocks];
    __shared__ double s_delta;

    const int bh = blockIdx.x, t = threadIdx.x;
    const int M = L / kBlock;

    // ---- rho_q^2, rho_k^2 (maxima are order-free) -------------------------
    int flags = 0;
    if (gamma_q == nullptr) {
        double mq = 0.0, mk = 0.0;
        for (int i = t; i < nchunk; i += kPlanThreads) {
            mq = nan_max(mq, part[((size_t)bh * 2 + 0) * nchunk + i]);
            mk = nan_max(mk, part[((size_t)bh * 2 + 1) * nchunk + i]);
        }
        auto nmax = [](double a, double b) { return nan_max(a, b); };
        mq = block_reduce(mq, s_dbl, nmax);
        mk = block_reduce(mk, s_dbl, nmax);
        if (t == 0) {
            // U = rho_q rho_k / sqrt(d) evaluated as sqrt(rho_q^2 rho_k^2 / d);
            // delta = -2U - log L + log eps, every step rounded to nearest.
            const double u = __builtin_sqrt((mq * mk) / (double)d);
            const double delta = -(2.0 * u + log_l_over_eps);
            s_delta = delta;
            u_out[bh] = u;
            delta_out[bh] = delta;
            if (!(mq <= 1.7976931348623157e308) || !(mk <= 1.7976931348623157e308)) flags |= 8;
        }
    } else if (t == 0) {
        // QK-norm (App. E): an RMS-normalised row has norm sqrt(d) and a scale of
        // magnitude at most gamma stretches it by at most gamma, so
        // U = gamma_q gamma_k sqrt(d), evaluated as (gamma_q gamma_k) sqrt(d)
        // (the product of two floats is exact in float64).
        const int h = bh % H;
        const double gq = (double)gamma_q[h], gk = (double)gamma_k[h];
        const double u = (gq * gk) * __builtin_sqrt((double)d);
        const double delta = -(2.0 * u + log_l_over_eps);
        s_delta = delta;
        u_out[bh] = u;
        delta_out[bh] = delta;
        if (!(gq >= 0.0 && gq <= 3.4028234663852886e38) || !(gk >= 0.0 && gk <= 3.4028234663852886e38))
            flags |= 8;
    }

    // ---- c = cumsum(log f): each thread owns a contiguous run -------------
    const float* x = log_f + (size_t)bh * L;
    const int per = (L + kPlanThreads - 1) / kPlanThreads;
    const int beg = min(t * per, L), end = min(beg + per, L);
    double local = 0.0, local_abs = 0.0;
    int min_lsb = 1 << 30;
    for (int i = beg; i < end; ++i) {
        const float v = x[i];
        if (!__builtin_isfinite(v)) flags |= 2;
        else {
            if (v > 0.0f) flags |= 1;
            if (v != 0.0f) min_lsb = min(min_lsb, lsb_exp(v));
        }
        local += (double)v;
        local_abs += __builtin_fabs((double)v);
    }
    const double incl = block_inclusive_scan(local, s_dbl);
    double run = incl - local;  // exclusive prefix: exact when the span check passes
    auto sum = [](double a, double b) { return a + b; };
    auto imin = [](int a, int b) { return min(a, b); };
    auto ior = [](int a, int b) { return a | b; };
    const double total_abs = block_reduce(local_abs, s_dbl2, sum);
    min_lsb = block_reduce(min_lsb, s_int, imin);
    if (t == 0 && total_abs > 0.0) {
        // every partial sum is a multiple of 2^min_lsb and below 2^(ilogb+2)
        const int biased = (int)((__double_as_longlong(total_abs) >> 52) & 0x7ff);
        const int top = (biased > 0 ? biased : 1) - 1023 + 2;
        if (top - min_lsb > 53) flags |= 4;
    }
    for (int i = beg; i < end; ++i) {
        run += (double)x[i];
        const float cf = (float)run;
        c_out[(size_t)bh * L + i] = cf;
        if ((i & (kBlock - 1)) == 0) s_first[i / kBlock] = cf;
        if ((i & (kBlock - 1)) == kBlock - 1) s_last[i / kBlock] = cf;
    }
    flags = block_reduce(flags, s_int, ior);   // also orders the LDS writes above

    // ---- boundary: first kept key block of every query block ---------------
    // Block (m, n < m) is kept iff its top-right entry c_{64m} - c_{64n+63} is
    // >= delta.  With non-increasing c that entry grows with n, so the first
    // kept block is found by bisection; the diagonal block is always kept.
    const double delta = s_delta;
    long long kept = 0;
    for (int m = t; m < M; m += kPlanThreads) {
        const double f = (double)s_first[m];
        int lo = 0, hi = m;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (f - (double)s_last[mid] >= delta) hi = mid;
            else lo = mid + 1;
        }
        s_rs[m] = lo;
        row_start[(size_t)bh * M + m] = lo;
        kept += (long long)(m - lo + 1);
    }
    __syncthreads();
    // last query block that keeps key block n: largest m with row_start[m] <= n
    for (int n = t; n < M; n += kPlanThreads) {
        int lo = n, hi = M - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_rs[mid] <= n) lo = mid;
            else hi = mid - 1;
        }
        col_end[(size_t)bh * M + n] = lo;
    }
    auto lsum = [](long long a, long long b) { return a + b; };
    kept = block_reduce(kept, s_ll, lsum);
    if (t == 0) {
        kept_out[bh] = kept;
        flags_out[bh] = flags;
    }
}

// ---- launchers ---------------------------------------------------------------

template <typename T, int D>
static hipError_t launch_norm_t(const void* Q, const void* K, int BH, int L, int nchunk,
                                double* part, hipStream_t s) {
    hipLaunchKernelGGL((rownorm_max_kernel<T, D>), dim3(nchunk, BH, 2), dim3(kNormRows), 0, s,
                       (const T*)Q, (const T*)K, L, nchunk, part);
    return hipGetLastError();
}

int norm_chunks(int L) { return (L + kNormRows - 1) / kNormRows; }

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
    hipError_t e;
    const int BH = a.B * a.H;
    if (a.gamma_q == nullptr) {
        trace_begin(ACP_K_ROWNORM, s);
        if (a.bf16) {
            e = a.d == 64 ? launch_norm_t<__bf16, 64>(a.Q, a.K, BH, a.L, a.nchunk, a.part, s)
                          : launch_norm_t<__bf16, 128>(a.Q, a.K, BH, a.L, a.nchunk, a.part, s);
        } else {
            e = a.d == 64 ? launch_norm_t<float, 64>(a.Q, a.K, BH, a.L, a.nchunk, a.part, s)
                          : launch_norm_t<float, 128>(a.Q, a.K, BH, a.L, a.nchunk, a.part, s);
        }
        if (e != hipSuccess) return e;
        trace_end(ACP_K_ROWNORM, s);
    }
    trace_begin(ACP_K_PLAN, s);
    hipLaunchKernelGGL(plan_kernel, dim3(BH), dim3(kPlanThreads), 0, s,
                       a.log_f, a.part, a.nchunk, a.gamma_q, a.gamma_k, a.H, a.L, a.d,
                       a.log_l_over_eps,
                       a.c, a.u, a.delta, a.row_start, a.col_end, a.kept, a.flags);
    e = hipGetLastError();
    trace_end(ACP_K_PLAN, s);
    return e;
}

}  // namespace acp
