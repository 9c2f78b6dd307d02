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
// launch is skipped and the plan kernel takes U from the scales.  After the
// gate producer (acp_gate.hip), which leaves c and the gates' statistics in
// place, the plan kernel reads the block corners of c instead of scanning log f.
#include "acp_device.h"
#include "acp_internal.h"
#include "acp_scan.h"

namespace acp {

constexpr int kNormRows = 128;     // rows per chunk (one float64 maximum each)
constexpr int kNormThreads = 256;  // a workgroup takes two chunks per step, a thread per row

// LDS of one workgroup of rownorm_max_kernel: two chunks, rows padded by 16 bytes
template <typename T, int D>
constexpr int norm_lds_bytes() { return 2 * kNormRows * (D * (int)sizeof(T) + 16); }

// Persistent over pairs of chunks: while a pair is reduced from LDS, the next
// pair's rows are already on their way into registers.  Chunk u of the grid is
// (bh, which, chunk) with u = (2 bh + which) nchunk + chunk, which is also its
// slot in part.
template <typename T, int D>
__global__ __launch_bounds__(kNormThreads) void rownorm_max_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, int BH, int L, int nchunk,
    double* __restrict__ part) {
    constexpr int kRowBytes = D * (int)sizeof(T);
    constexpr int kPieces = kRowBytes / 16;   // 16-byte pieces per row (and per thread)
    constexpr int kStride = kRowBytes + 16;   // padded LDS row (spreads banks)
    constexpr int kPer = 16 / (int)sizeof(T); // elements per piece
    __shared__ __attribute__((aligned(16))) unsigned char tile[2][kNormRows * kStride];
    __shared__ double wave_max[kNormThreads / 64];

    const int tid = threadIdx.x, half = tid >> 7, r = tid & (kNormRows - 1);
    const int npairs = BH * nchunk;           // 2 BH nchunk chunks
    auto chunk_of = [&](int p, const unsigned char*& src, int& rows) {
        const int u = 2 * p + half;
        const int bh = u / (2 * nchunk), which = (u / nchunk) & 1, c = u % nchunk;
        const T* X = (which == 0 ? Q : K) + ((size_t)bh * L + (size_t)c * kNormRows) * D;
        src = reinterpret_cast<const unsigned char*>(X);
        rows = min(kNormRows, L - c * kNormRows);
        return u;
    };
    // Thread r of a half loads pieces r, r + 128, ... of its chunk (coalesced).
    uint4 buf[kPieces];
    auto load = [&](int p) __attribute__((always_inline)) {
        const unsigned char* src;
        int rows;
        chunk_of(p, src, rows);
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            const int i = r + kNormRows * k;
            buf[k] = i < rows * kPieces ? *reinterpret_cast<const uint4*>(src + (size_t)i * 16)
                                        : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    int p = blockIdx.x;
    if (p < npairs) load(p);
    for (; p < npairs; p += gridDim.x) {
        const unsigned char* src;
        int rows;
        const int u = chunk_of(p, src, rows);
        __syncthreads();                      // the previous pair's tile reads are done
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            const int i = r + kNormRows * k;
            *reinterpret_cast<uint4*>(tile[half] + (i / kPieces) * kStride + (i % kPieces) * 16) = buf[k];
        }
        if (p + (int)gridDim.x < npairs) load(p + gridDim.x);
        __syncthreads();

        // Each thread: sum of squares of its row in ascending feature order, in
        // float64.  Squares of float32/bfloat16 values are exact in float64, so
        // fma(x, x, acc) rounds exactly like acc + x*x.
        double acc = 0.0;
        if (r < rows) {
            const unsigned char* rp = tile[half] + r * kStride;
            for (int ch = 0; ch < kPieces; ++ch) {
                const uint4 v = *reinterpret_cast<const uint4*>(rp + ch * 16);
                const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
                for (int t = 0; t < kPer; ++t) {
                    const double x = to_f64(e[t]);
                    acc = __builtin_fma(x, x, acc);
                }
            }
        }
        // max over the chunk's rows (order-free), two waves per chunk
        double m = acc;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) m = nan_max(m, __shfl_xor(m, off));
        if ((tid & 63) == 0) wave_max[tid >> 6] = m;
        __syncthreads();
        if (r == 0) part[u] = nan_max(wave_max[2 * half], wave_max[2 * half + 1]);
    }
}

// One workgroup of 1024 threads per (batch, head); each thread owns a contiguous
// run of log f, read and written as float4s when the run length is a multiple of
// 4 (at L = 4096 one float4 per thread, so every access is coalesced), and kept
// in registers up to kPlanHeld values.  Three barriers in all, none of which
// waits for global stores: one round through LDS carries the scan's wave totals
// together with every reduction (|log f| sum, last-bit position, flags, norm
// maxima), one publishes the block corners of c, one the first kept blocks.
// U and delta are formed by every thread from the same LDS values, so they are
// identical everywhere without another round.  Cross-lane traffic is kept low:
// the gate flags go through wave ballots, and the norm maxima are reduced only
// by the waves that hold partials.
constexpr int kPlanHeld = 16;   // log f values a thread keeps in registers (L <= 16384)
constexpr int kWideBit = 1 << 16;   // (inside the kernel only) the gated mode needs pairs

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(
    const float* __restrict__ log_f, const double* __restrict__ part, int nchunk,
    const float* __restrict__ gamma_q, const float* __restrict__ gamma_k,
    const GateStats* __restrict__ gate, int H, int L, int d, double log_l_over_eps,
    float* __restrict__ c_out,
    double* __restrict__ u_out, double* __restrict__ delta_out,
    int* __restrict__ row_start, int* __restrict__ col_end,
    long long* __restrict__ kept_out, int* __restrict__ flags_out) {
    __shared__ double s_sum[kPlanWaves], s_abs[kPlanWaves], s_mq[kPlanWaves], s_mk[kPlanWaves];
    __shared__ double s_dsum[2][kPlanWaves], s_dabs[2][kPlanWaves];   // double-double round
    __shared__ int s_lsb[kPlanWaves], s_flg[kPlanWaves];
    __shared__ float s_first[kMaxBlocks];  // c at the first row of each block
    __shared__ float s_last[kMaxBlocks];   // c at the last row of each block
    __shared__ int s_rs[kMaxBlocks];

    const int bh = blockIdx.x, t = threadIdx.x, lane = t & 63, wid = t >> 6;
    const int M = L / kBlock;

    // ---- requests: this thread's run of log f and the norm partials -----------
    const float* x = log_f + (size_t)bh * L;
    float* cw = c_out + (size_t)bh * L;
    const int per = (L + kPlanThreads - 1) / kPlanThreads;
    const bool gated = gate != nullptr;   // c in place: no gates to read or scan
    const int beg = min(t * per, L), n = gated ? 0 : min(beg + per, L) - beg;
    const bool held = per <= kPlanHeld;
    const bool vec = held && (per & 3) == 0;   // then n is per or 0
    float xv[kPlanHeld];
    if (vec) {
#pragma unroll
        for (int i = 0; i < kPlanHeld; i += 4) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (i < n) v = *reinterpret_cast<const float4*>(x + beg + i);
            xv[i] = v.x; xv[i + 1] = v.y; xv[i + 2] = v.z; xv[i + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < kPlanHeld; ++i) xv[i] = held && i < n ? x[beg + i] : 0.f;
    }
    double mq = 0.0, mk = 0.0;   // squared norms are >= 0; a NaN wins nan_max
    const bool norms = gamma_q == nullptr;
    if (norms) {
        for (int i = t; i < nchunk; i += kPlanThreads) {
            mq = nan_max(mq, part[((size_t)bh * 2 + 0) * nchunk + i]);
            mk = nan_max(mk, part[((size_t)bh * 2 + 1) * nchunk + i]);
        }
    }

    // ---- this thread's sums and checks --------------------------------------------
    // First in float64, which is exact in any association while the partial sums
    // span at most 53 bits (the read below decides); a head whose sums span more
    // is summed again in double-double, exact up to 105 bits.
    double local = 0.0, local_abs = 0.0;
    int min_lsb = 1 << 30;
    bool positive = false, nonfinite = false;
    auto take = [&](float v) __attribute__((always_inline)) {
        if (!__builtin_isfinite(v)) nonfinite = true;
        else {
            if (v > 0.0f) positive = true;
            if (v != 0.0f) min_lsb = min(min_lsb, lsb_exp(v));
        }
        local += (double)v;
        local_abs += __builtin_fabs((double)v);
    };
    int gate_flags = 0;
    DD gate_abs{0.0, 0.0};
    bool gate_lo = false;   // a block's |log f| sum needed its low part
    if (gated) {
        // the producer's per-block statistics (sum of |log f| as a pair, smallest
        // ulp exponent, flags) take the place of the gates themselves
        const int M0 = L / kBlock;
        for (int m = t; m < M0; m += kPlanThreads) {
            const GateStats g = gate[(size_t)bh * M0 + m];
            local_abs += g.abs_sum;
            gate_lo = gate_lo || g.abs_lo != 0.0;
            gate_abs = dd_add(gate_abs, DD{g.abs_sum, g.abs_lo});
            min_lsb = min(min_lsb, g.min_lsb);
            gate_flags |= g.flags;
        }
    } else if (held) {
#pragma unroll
        for (int i = 0; i < kPlanHeld; ++i)
            if (i < n) take(xv[i]);
    } else {
        for (int i = 0; i < n; ++i) take(x[beg + i]);
    }

    // ---- one round through LDS --------------------------------------------------------
    // (cross-lane steps by DPP within rows of 16, then the four rows' results by
    // readlane: lane 0 writes the wave's entries)
    const double incl = wave_inclusive_scan_f64(local);
    {
        const auto add = [](double a, double b) { return a + b; };
        const double ra = row16_reduce(local_abs, add);
        local_abs = ((readlane_f64(ra, 0) + readlane_f64(ra, 16)) + readlane_f64(ra, 32)) +
                    readlane_f64(ra, 48);
        const int rl = row16_reduce(min_lsb, [](int a, int b) { return min(a, b); });
        min_lsb = min(min(__builtin_amdgcn_readlane(rl, 0), __builtin_amdgcn_readlane(rl, 16)),
                      min(__builtin_amdgcn_readlane(rl, 32), __builtin_amdgcn_readlane(rl, 48)));
    }
    const int wflags = (__ballot(positive) != 0ull ? 1 : 0) |
                       (__ballot(nonfinite || (gate_flags & 2)) != 0ull ? 2 : 0) |
                       (__ballot(gate_flags & 32) != 0ull ? 32 : 0) |
                       (__ballot(gate_lo) != 0ull ? kWideBit : 0);
    if (norms && wid * 64 < nchunk) {   // only waves that loaded partials
        const auto mx = [](double a, double b) { return nan_max(a, b); };
        const double rq = row16_reduce(mq, mx), rk = row16_reduce(mk, mx);
        mq = nan_max(nan_max(readlane_f64(rq, 0), readlane_f64(rq, 16)),
                     nan_max(readlane_f64(rq, 32), readlane_f64(rq, 48)));
        mk = nan_max(nan_max(readlane_f64(rk, 0), readlane_f64(rk, 16)),
                     nan_max(readlane_f64(rk, 32), readlane_f64(rk, 48)));
    }
    if (lane == 63) s_sum[wid] = incl;
    if (lane == 0) {
        s_abs[wid] = local_abs;
        s_lsb[wid] = min_lsb;
        s_flg[wid] = wflags;
        s_mq[wid] = mq;
        s_mk[wid] = mk;
    }
    lds_barrier();
    // Every wave combines the 16 waves' entries itself, lane l < 16 taking wave l's
    // (one LDS read per quantity, then a reduction over the row of 16 lanes; row 0
    // is read out).  The float64 sums are exact whenever the span check passes, so
    // their association does not matter.
    double before, total_abs;
    int flags;
    {
        const bool in = lane < kPlanWaves;
        const int l = in ? lane : 0;
        const auto add = [](double a, double b) { return a + b; };
        double vs = in && lane < wid ? s_sum[l] : 0.0;
        double va = in ? s_abs[l] : 0.0;
        int vl = in ? s_lsb[l] : (1 << 30);
        int vf = in ? s_flg[l] : 0;
        double vq = in ? s_mq[l] : 0.0;   // squared norms are >= 0; a NaN wins nan_max
        double vk = in ? s_mk[l] : 0.0;
        vs = row16_reduce(vs, add);
        va = row16_reduce(va, add);
        vl = row16_reduce(vl, [](int a, int b) { return min(a, b); });
        vf = row16_reduce(vf, [](int a, int b) { return a | b; });
        vq = row16_reduce(vq, [](double a, double b) { return nan_max(a, b); });
        vk = row16_reduce(vk, [](double a, double b) { return nan_max(a, b); });
        before = readfirst_f64(vs);
        total_abs = readfirst_f64(va);
        min_lsb = __builtin_amdgcn_readfirstlane(vl);
        flags = __builtin_amdgcn_readfirstlane(vf);
        mq = readfirst_f64(vq);
        mk = readfirst_f64(vk);
    }
    // ---- the span, and double-double sums where float64 is not enough -------------
    // Every partial sum is a multiple of 2^min_lsb and below 2^E, the least power
    // of two above sum |log f|.  Up to 53 bits the float64 total is exact, so E is
    // right and every float64 sum is exact; beyond, its rounding can lose one power
    // of two, and 54 bits would read as 53.  So from a read of 53 bits on (or, in
    // the gated mode, when a block's sum of |log f| has a low part) the head is
    // summed again in double-double, where the same argument holds up to 105
    // bits: flag bit 2 from a span of 105 on.  The test is uniform over the
    // workgroup.
    bool wide = (flags & kWideBit) != 0;
    flags &= ~kWideBit;
    if (total_abs > 0.0) {
        const int biased = (int)((__double_as_longlong(total_abs) >> 52) & 0x7ff);
        const int top = (biased > 0 ? biased : 1) - 1023 + 1;
        wide = wide || top - min_lsb >= 53;
    }
    DD run_dd{0.0, 0.0};
    if (wide) {
        DD l{0.0, 0.0}, la = gate_abs;
        if (held) {
#pragma unroll
            for (int i = 0; i < kPlanHeld; ++i) {
                if (i < n) {
                    l = dd_add(l, (double)xv[i]);
                    la = dd_add(la, __builtin_fabs((double)xv[i]));
                }
            }
        } else {
            for (int i = 0; i < n; ++i) {
                const double v = (double)x[beg + i];
                l = dd_add(l, v);
                la = dd_add(la, __builtin_fabs(v));
            }
        }
        const DD inc = wave_inclusive_scan_dd(l);
        la = wave_sum_dd(la);
        if (lane == 63) {
            s_dsum[0][wid] = inc.hi;
            s_dsum[1][wid] = inc.lo;
        }
        if (lane == 0) {
            s_dabs[0][wid] = la.hi;
            s_dabs[1][wid] = la.lo;
        }
        lds_barrier();
        const bool in = lane < kPlanWaves;
        const int li = in ? lane : 0;
        const bool lower = in && lane < wid;
        DD vs{lower ? s_dsum[0][li] : 0.0, lower ? s_dsum[1][li] : 0.0};
        DD va{in ? s_dabs[0][li] : 0.0, in ? s_dabs[1][li] : 0.0};
        vs = row16_sum_dd(vs);
        va = row16_sum_dd(va);
        const DD total{readfirst_f64(va.hi), readfirst_f64(va.lo)};
        if (total.hi > 0.0) {
            if (dd_top_exp(total) - min_lsb >= kExactSpanBits) flags |= 4;
            // c leaves the float32 range (|c| <= sum |log f|, reached at the end
            // when no gate is positive)
            if (__builtin_isinf(dd_to_f32(total))) flags |= 2;
        }
        run_dd = dd_add(DD{readfirst_f64(vs.hi), readfirst_f64(vs.lo)}, dd_add(inc, dd_neg(l)));
    } else if (total_abs > 0.0 && !__builtin_isfinite((float)total_abs)) {
        flags |= 2;   // (the float64 total is exact here)
    }

    // ---- U and delta ---------------------------------------------------------------------
    double u;
    if (norms) {
        // U = rho_q rho_k / sqrt(d) evaluated as sqrt(rho_q^2 rho_k^2 / d);
        // delta = -2U - log L + log eps, every step rounded to nearest.
        u = __builtin_sqrt((mq * mk) / (double)d);
        if (!(mq <= 1.7976931348623157e308) || !(mk <= 1.7976931348623157e308)) flags |= 8;
    } else {
        // QK-norm (App. E): an RMS-normalised row has norm sqrt(d) and a scale of
        // magnitude at most gamma stretches it by at most gamma, so
        // U = gamma_q gamma_k sqrt(d), evaluated as (gamma_q gamma_k) sqrt(d)
        // (the product of two floats is exact in float64).
        const int h = bh % H;
        const double gq = (double)gamma_q[h], gk = (double)gamma_k[h];
        u = (gq * gk) * __builtin_sqrt((double)d);
        if (!(gq >= 0.0 && gq <= 3.4028234663852886e38) || !(gk >= 0.0 && gk <= 3.4028234663852886e38))
            flags |= 8;
    }
    const double delta = -(2.0 * u + log_l_over_eps);
    if (t == 0) {
        u_out[bh] = u;
        delta_out[bh] = delta;
    }

    // ---- c = cumsum(log f) and the block corners ----------------------------------------
    auto corner = [&](int j, float cf) __attribute__((always_inline)) {
        if ((j & (kBlock - 1)) == 0) s_first[j / kBlock] = cf;
        if ((j & (kBlock - 1)) == kBlock - 1) s_last[j / kBlock] = cf;
    };
    // run: the exclusive prefix (float64 or a pair), exact when the span check passes
    auto emit = [&](auto run) __attribute__((always_inline)) {
        if (vec) {
#pragma unroll
            for (int i = 0; i < kPlanHeld; i += 4) {
                if (i < n) {
                    float4 cv;
                    run = sum_add(run, xv[i]);     cv.x = sum_f32(run);
                    run = sum_add(run, xv[i + 1]); cv.y = sum_f32(run);
                    run = sum_add(run, xv[i + 2]); cv.z = sum_f32(run);
                    run = sum_add(run, xv[i + 3]); cv.w = sum_f32(run);
                    *reinterpret_cast<float4*>(cw + beg + i) = cv;
                    corner(beg + i, cv.x);            // beg + i is a multiple of 4
                    corner(beg + i + 3, cv.w);
                }
            }
        } else if (held) {
#pragma unroll
            for (int i = 0; i < kPlanHeld; ++i) {
                if (i < n) {
                    run = sum_add(run, xv[i]);
                    const float cf = sum_f32(run);
                    cw[beg + i] = cf;
                    corner(beg + i, cf);
                }
            }
        } else {
            for (int i = 0; i < n; ++i) {
                run = sum_add(run, x[beg + i]);
                const float cf = sum_f32(run);
                cw[beg + i] = cf;
                corner(beg + i, cf);
            }
        }
    };
    if (gated) {
        for (int m = t; m < M; m += kPlanThreads) {
            s_first[m] = cw[kBlock * m];
            s_last[m] = cw[kBlock * m + kBlock - 1];
        }
    } else if (wide) {
        emit(run_dd);
    } else {
        emit(before + (incl - local));
    }
    lds_barrier();

    // ---- boundary: first kept key block of every query block ---------------------------
    // Block (m, n < m) is kept iff its top-right entry c_{64m} - c_{64n+63} is
    // >= delta.  With non-increasing c that entry grows with n, so the first
    // kept block is found by bisection; the diagonal block is always kept.
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
    }
    lds_barrier();
    // last query block that keeps key block n: largest m with row_start[m] <= n
    for (int nn = t; nn < M; nn += kPlanThreads) {
        int lo = nn, hi = M - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_rs[mid] <= nn) lo = mid;
            else hi = mid - 1;
        }
        col_end[(size_t)bh * M + nn] = lo;
    }
    if (wid == kPlanWaves - 1) {   // (no col_end work for this wave unless M > 960)
        long long kept = 0;
        for (int m = lane; m < M; m += 64) kept += (long long)(m - s_rs[m] + 1);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) kept += __shfl_xor(kept, off);
        if (lane == 0) {
            kept_out[bh] = kept;
            flags_out[bh] = flags;
        }
    }
}

// ---- workgroup schedule of the attention kernels ---------------------------------
// The attention kernels' workgroups each take 128 query rows (forward, dQ) or
// 128 keys (dK/dV) of one head.  Workgroup ids are dealt round-robin to the 8
// XCDs; xcd_logical_id turns that into a contiguous range of logical ids per XCD,
// and this kernel fills, per XCD range, which (head, block) each logical id
// takes, so that
//   - a head's workgroups all run on one XCD (its K and V stay in one L2);
//   - with at most 8 heads per XCD (B*H a multiple of 8, <= 64) the heads are
//     placed by kept-block count: sorted largest first, each on the least loaded
//     XCD that still has room (the same number of heads per XCD, so every range
//     holds whole heads); with more heads per XCD they stay in bh order;
//   - inside each XCD range the workgroups run largest first (a counting sort
//     on their kept-tile counts), so that the range ends on small ones.
// Grid (8, 2): x = XCD, y = 0 for the query-block table, 1 for the key-block one.
// Entry = bh * nb + block.  Equal counts keep no particular order.
constexpr int kPlaceMax = 64;
constexpr int kSchedThreads = 1024;

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(
    const long long* __restrict__ kept, const int* __restrict__ row_start,
    const int* __restrict__ col_end, int BH, int M, int nb, int* __restrict__ sched_q,
    int* __restrict__ sched_k) {
    __shared__ int s_sorted[kPlaceMax];
    __shared__ int s_place[kPlaceMax];
    __shared__ int s_hist[2 * kMaxBlocks + 2];   // a block's count is at most 2M <= 4096
    __shared__ double s_wave[kPlanWaves];
    static_assert(kSchedThreads == kPlanThreads, "block_inclusive_scan takes 1024 threads");
    const int x = blockIdx.x, table = blockIdx.y, t = threadIdx.x;
    const bool place = BH % 8 == 0 && BH >= 8 && BH <= kPlaceMax;
    if (place && t < 64) {
        // Wave 0 alone: rank the heads by kept count (largest first, ties by
        // index), then place them in that order.  Lanes 0-7 hold the load and head
        // count of XCD 0-7; each step takes the least loaded XCD with room (lowest
        // index on ties) as the minimum of load << 3 | xcd over lanes 0-7.  A head
        // keeps at most M (M + 1) / 2 < 2^22 blocks and an XCD at most 8 heads, so
        // the key fits 32 bits.  (A single wave's LDS accesses complete in order,
        // so no barrier is needed between its write and read of s_sorted.)
        const int kt_l = t < BH ? (int)min(max(kept[t], 0ll), 1ll << 22) : 0;
        int rank = 0;
        for (int j = 0; j < BH; ++j) {
            const int kj = __builtin_amdgcn_readlane(kt_l, j);
            rank += (kj > kt_l || (kj == kt_l && j < t)) ? 1 : 0;
        }
        if (t < BH) s_sorted[rank] = t;
        const int hd_l = t < BH ? s_sorted[t] : 0;
        const int k_l = __shfl(kt_l, hd_l);
        const int per = BH / 8;
        unsigned load = 0u;
        int count = 0, mypos = 0;
        for (int i = 0; i < BH; ++i) {
            unsigned key = t < 8 && count < per ? (load << 3) | (unsigned)t : 0xffffffffu;
            // minimum over each group of 8 lanes: swap neighbours, pairs, quads
            key = min(key, (unsigned)__builtin_amdgcn_mov_dpp((int)key, 0xB1, 0xF, 0xF, false));
            key = min(key, (unsigned)__builtin_amdgcn_mov_dpp((int)key, 0x4E, 0xF, 0xF, false));
            key = min(key, (unsigned)__builtin_amdgcn_mov_dpp((int)key, 0x141, 0xF, 0xF, false));
            const int best = (int)((unsigned)__builtin_amdgcn_readfirstlane((int)key) & 7u);
            const int pos = per * best + __builtin_amdgcn_readlane(count, best);
            if (t == best) {
                count += 1;
                load += (unsigned)__builtin_amdgcn_readlane(k_l, i);
            }
            if (t == i) mypos = pos;
        }
        if (t < BH) s_place[mypos] = hd_l;
    }
    const int nbins = 2 * M + 2;
    for (int i = t; i < nbins; i += kSchedThreads) s_hist[i] = 0;
    __syncthreads();

    // this XCD's range of logical ids (as xcd_logical_id deals them)
    const int nblocks = BH * nb, q = nblocks >> 3, r = nblocks & 7;
    const int lo = x * q + min(x, r), hi = lo + q + (x < r ? 1 : 0);
    int* out = table == 0 ? sched_q : sched_k;
    // the item of a logical id in the unsorted order and its kept-tile count
    auto item = [&](int lid, int& work) {
        const int slot = lid / nb, idx = lid % nb;
        const int bh = place ? s_place[slot] : slot;
        const int blk = table == 0 ? nb - 1 - idx : idx;   // longest rows / first keys first
        work = 0;
        for (int u = 0; u < 2; ++u) {
            const int m = 2 * blk + u;
            if (m < M) {
                work += table == 0 ? m - row_start[(size_t)bh * M + m] + 1
                                   : col_end[(size_t)bh * M + m] - m + 1;
            }
        }
        return bh * nb + blk;
    };
    for (int lid = lo + t; lid < hi; lid += kSchedThreads) {
        int work;
        item(lid, work);
        atomicAdd(&s_hist[work], 1);
    }
    __syncthreads();
    {
        // start of each count's run, largest count first: the bins in descending
        // order, thread t owning positions [kPer t, kPer t + kPer) of that order
        constexpr int kPer = (2 * kMaxBlocks + 2 + kSchedThreads - 1) / kSchedThreads;
        int cnt[kPer];
        int tot = 0;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int e = kPer * t + i;
            cnt[i] = e < nbins ? s_hist[nbins - 1 - e] : 0;
            tot += cnt[i];
        }
        // (the scan's barriers also order every thread's reads above before the
        // writes below)
        int run = lo + (int)block_inclusive_scan((double)tot, s_wave) - tot;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int e = kPer * t + i;
            if (e < nbins) s_hist[nbins - 1 - e] = run;
            run += cnt[i];
        }
    }
    __syncthreads();
    for (int lid = lo + t; lid < hi; lid += kSchedThreads) {
        int work;
        const int it = item(lid, work);
        out[atomicAdd(&s_hist[work], 1)] = it;
    }
}

hipError_t launch_schedule(const long long* kept, const int* row_start, const int* col_end,
                           int BH, int M, int nb, int* sched_q, int* sched_k, hipStream_t s) {
    trace_begin(ACP_K_SCHEDULE, s);
    hipLaunchKernelGGL(schedule_kernel, dim3(8, 2), dim3(kSchedThreads), 0, s, kept, row_start,
                       col_end, BH, M, nb, sched_q, sched_k);
    const hipError_t e = hipGetLastError();
    if (e == hipSuccess) trace_end(ACP_K_SCHEDULE, s);
    return e;
}

// ---- launchers ---------------------------------------------------------------

template <typename T, int D>
static hipError_t launch_norm_t(const void* Q, const void* K, int BH, int L, int nchunk,
                                double* part, hipStream_t s) {
    // as many workgroups as the CUs hold at once (LDS-bound), at most one per pair
    const int per_cu = (160 * 1024) / norm_lds_bytes<T, D>();
    const int grid = min(BH * nchunk, 256 * per_cu);
    hipLaunchKernelGGL((rownorm_max_kernel<T, D>), dim3(grid), dim3(kNormThreads), 0, s,
                       (const T*)Q, (const T*)K, BH, L, nchunk, part);
    return hipGetLastError();
}

int norm_chunks(int L) { return (L + kNormRows - 1) / kNormRows; }

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
    hipError_t e;
    const int BH = a.B * a.H;
    if (a.gamma_q == nullptr && !a.norms_ready) {
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
                       a.log_f, a.part, a.nchunk, a.gamma_q, a.gamma_k, a.gate, a.H, a.L, a.d,
                       a.log_l_over_eps,
                       a.c, a.u, a.delta, a.row_start, a.col_end, a.kept, a.flags);
    e = hipGetLastError();
    trace_end(ACP_K_PLAN, s);
    return e;
}

}  // namespace acp
