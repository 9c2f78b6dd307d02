// Decoding with ACP (paper Sec. 5, inference; the threshold of Sec. 3).
//
// With a logit bound U fixed for the whole sequence (from QK-norm scales,
// App. E) the threshold delta is fixed too, and since the cumulative gate c_t
// only falls as t grows, a key block pruned for query t stays pruned for every
// later query.  Each (batch, head) therefore keeps a pointer to the first key
// block its latest query keeps; it never moves back, and the cache entries
// behind it can be dropped.  The cache is a ring of C slots (position j in
// slot j mod C), so its memory is what the kept window needs, not the context.
//
// Kernels:
//   decode_init_kernel    prompt of L0 tokens -> delta, the float64 running
//                         cumsum, c of the prompt's last C positions, the
//                         pointer of query L0 - 1, and its K/V rows in the ring
//   decode_append_kernel  one token: cumsum, c_t, pointer advance, K/V append
//   decode_attn_kernel    query t over its kept keys, 256 keys per workgroup
//   decode_combine_kernel the workgroups' partial softmax sums merged
#include "acp_device.h"
#include "acp_internal.h"
#include "acp_scan.h"

namespace acp {

constexpr int kDecChunk = 256;   // keys per attention workgroup (one per thread)

size_t decode_partials_floats(int BH, int C, int d) {
    const int nsplit = (C + kDecChunk - 1) / kDecChunk;
    return (size_t)BH * nsplit * (d + 2);
}

// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kPlanThreads) void decode_init_kernel(
    const T* __restrict__ K, const T* __restrict__ V, const float* __restrict__ log_f,
    const float* __restrict__ gamma_q, const float* __restrict__ gamma_k, int H, int L0, int C,
    double log_lmax_over_eps, T* __restrict__ Kc, T* __restrict__ Vc, float* __restrict__ cc,
    double* __restrict__ cs_out, int* __restrict__ ptr_out, double* __restrict__ delta_out,
    int* __restrict__ flags_out) {
    __shared__ double s_dbl[kPlanWaves];
    __shared__ double s_dbl2[kPlanWaves];
    __shared__ int s_int[kPlanWaves];
    __shared__ float s_last[kMaxBlocks];   // c at the last row of each full block
    __shared__ double s_delta;
    __shared__ float s_ct;

    const int bh = blockIdx.x, t = threadIdx.x;
    int flags = 0;
    if (t == 0) {
        // U = (gamma_q gamma_k) sqrt(d), delta = -(2U + log L_max - log eps)
        const int h = bh % H;
        const double gq = (double)gamma_q[h], gk = (double)gamma_k[h];
        const double u = (gq * gk) * __builtin_sqrt((double)D);
        const double delta = -(2.0 * u + log_lmax_over_eps);
        s_delta = delta;
        delta_out[bh] = delta;
        if (!(gq >= 0.0 && gq <= 3.4028234663852886e38) || !(gk >= 0.0 && gk <= 3.4028234663852886e38))
            flags |= 8;
    }

    // c = cumsum(log f) of the prompt, each thread a contiguous run (as in stage 1)
    const float* x = log_f + (size_t)bh * L0;
    const int per = (L0 + kPlanThreads - 1) / kPlanThreads;
    const int beg = min(t * per, L0), end = min(beg + per, L0);
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
    double run = incl - local;
    auto sum = [](double a, double b) { return a + b; };
    auto imin = [](int a, int b) { return min(a, b); };
    auto ior = [](int a, int b) { return a | b; };
    const double total_abs = block_reduce(local_abs, s_dbl2, sum);
    min_lsb = block_reduce(min_lsb, s_int, imin);
    if (t == 0 && total_abs > 0.0) {
        const int biased = (int)((__double_as_longlong(total_abs) >> 52) & 0x7ff);
        const int top = (biased > 0 ? biased : 1) - 1023 + 2;
        if (top - min_lsb > 53) flags |= 4;
    }
    for (int i = beg; i < end; ++i) {
        run += (double)x[i];
        const float cf = (float)run;
        if (i >= L0 - C) cc[(size_t)bh * C + (i % C)] = cf;
        if ((i & (kBlock - 1)) == kBlock - 1) s_last[i / kBlock] = cf;
        if (i == L0 - 1) {
            cs_out[bh] = run;
            s_ct = cf;
        }
    }
    flags = block_reduce(flags, s_int, ior);   // also orders the LDS writes above

    if (t == 0) {
        // first kept block of query L0 - 1: c_t - c_{64n+63} >= delta grows with n
        const int nb = (L0 - 1) / kBlock;
        const double ct = (double)s_ct, delta = s_delta;
        int lo = 0, hi = nb;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (ct - (double)s_last[mid] >= delta) hi = mid;
            else lo = mid + 1;
        }
        // The ring holds positions L0 - C .. L0 - 1: a kept key before them is lost,
        // and the pointer does not go below the block of the oldest position held.
        const int first = L0 - C;
        if (kBlock * lo < first) flags |= 16;
        ptr_out[bh] = max(lo, first > 0 ? first / kBlock : 0);
        flags_out[bh] = flags;
    }

    // the prompt's last min(L0, C) K and V rows into their slots
    constexpr int kVec = 16 / (int)sizeof(T);
    constexpr int kPerRow = D / kVec;
    const int j0 = max(0, L0 - C);
    const int nrow = L0 - j0;
    for (int i = t; i < nrow * kPerRow; i += kPlanThreads) {
        const int j = j0 + i / kPerRow, e = (i % kPerRow) * kVec;
        const size_t src = ((size_t)bh * L0 + j) * D + e;
        const size_t dst = ((size_t)bh * C + (j % C)) * D + e;
        *reinterpret_cast<uint4*>(Kc + dst) = *reinterpret_cast<const uint4*>(K + src);
        *reinterpret_cast<uint4*>(Vc + dst) = *reinterpret_cast<const uint4*>(V + src);
    }
}

// ---------------------------------------------------------------------------
// Token t of every (batch, head): one workgroup of 64 threads.
template <typename T, int D>
__global__ __launch_bounds__(64) void decode_append_kernel(
    const T* __restrict__ k, const T* __restrict__ v, const float* __restrict__ log_f, int t,
    int C, T* __restrict__ Kc, T* __restrict__ Vc, float* __restrict__ cc,
    double* __restrict__ cs, int* __restrict__ ptr, const double* __restrict__ delta,
    int* __restrict__ flags) {
    const int bh = blockIdx.x, lane = threadIdx.x;
    const int slot = t % C;
    if (lane == 0) {
        int fl = flags[bh];
        const float lff = log_f[bh];
        if (!__builtin_isfinite(lff)) fl |= 2;
        else if (lff > 0.0f) fl |= 1;
        const double old = cs[bh], lf = (double)lff;
        const double s2 = old + lf;
        // the running sum stays the exact prefix sum only while no addition rounds
        const double bb = s2 - old;
        if ((old - (s2 - bb)) + (lf - bb) != 0.0) fl |= 4;
        const float ct = (float)s2;
        const double dl = delta[bh];
        const float* crow = cc + (size_t)bh * C;
        // Before slot t mod C is overwritten the ring holds positions t - C .. t - 1.
        // A kept key is lost iff the block of position t - C is kept (the blocks
        // before it are then kept too); its last key is one of those positions.
        const int nb = t / kBlock, gone = t - C;
        if (gone >= 0) {
            const int nx = gone / kBlock;
            if ((double)ct - (double)crow[(kBlock * nx + kBlock - 1) % C] >= dl) fl |= 16;
        }
        // advance from the old pointer, or from the block of the oldest position
        // still held after the append, to the first kept block
        int n = max(ptr[bh], gone + 1 > 0 ? (gone + 1) / kBlock : 0);
        while (n < nb && (double)ct - (double)crow[(kBlock * n + kBlock - 1) % C] < dl) ++n;
        ptr[bh] = n;
        cs[bh] = s2;
        cc[(size_t)bh * C + slot] = ct;
        flags[bh] = fl;
    }
    constexpr int kVec = 16 / (int)sizeof(T);
    for (int e = lane * kVec; e < D; e += 64 * kVec) {
        const size_t dst = ((size_t)bh * C + slot) * D + e;
        *reinterpret_cast<uint4*>(Kc + dst) = *reinterpret_cast<const uint4*>(k + (size_t)bh * D + e);
        *reinterpret_cast<uint4*>(Vc + dst) = *reinterpret_cast<const uint4*>(v + (size_t)bh * D + e);
    }
}

// ---------------------------------------------------------------------------
// Query t over keys [j_lo, t], j_lo = max(64 ptr, t - C + 1): workgroup s takes
// keys j_lo + 256 s .. + 255, wave w of it the 64 keys from 64 w.  Rows are read
// whole by groups of G lanes (16 bytes each), so every load instruction covers
// 64 / G consecutive cache rows.  Writes the workgroup's (max, sum, unnormalised
// O) with logits in log2 units.
template <typename T, int D>
__global__ __launch_bounds__(kDecChunk) void decode_attn_kernel(
    const T* __restrict__ q, const T* __restrict__ Kc, const T* __restrict__ Vc,
    const float* __restrict__ cc, const int* __restrict__ ptr, int t, int C, int nsplit,
    float kscale, float* __restrict__ part) {
    constexpr int kVec = 16 / (int)sizeof(T);   // elements per 16-byte piece
    constexpr int G = D / kVec;                 // lanes per cache row
    constexpr int kRows = 64 / G;               // rows per wave load
    constexpr int kIter = 64 / kRows;           // loads per wave for its 64 rows
    constexpr int kWaves = kDecChunk / 64;
    __shared__ float x_s[kDecChunk];
    __shared__ float red[kWaves][D];
    __shared__ float s_red[kWaves];

    const int bh = blockIdx.y, sp = blockIdx.x, tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int j_lo = max(kBlock * ptr[bh], t - C + 1);
    const int j0 = j_lo + sp * kDecChunk;
    float* out = part + ((size_t)bh * nsplit + sp) * (D + 2);
    if (j0 > t) {                                // past this query's window
        if (tid < D) out[2 + tid] = 0.f;
        if (tid == 0) { out[0] = -INFINITY; out[1] = 0.f; }
        return;
    }
    const int nk = min(kDecChunk, t - j0 + 1);
    const size_t head = (size_t)bh * C;
    const int e0 = (lane % G) * kVec;
    float qv[kVec];
    {
        const uint4 raw = *reinterpret_cast<const uint4*>(q + (size_t)bh * D + e0);
        const T* ev = reinterpret_cast<const T*>(&raw);
#pragma unroll
        for (int i = 0; i < kVec; ++i) qv[i] = to_f32(ev[i]);
    }

    // q . k_j for the wave's rows, reduced over the G lanes of each row
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int kk = 64 * wid + kRows * it + lane / G;
        float dot = 0.f;
        if (kk < nk) {
            const int j = j0 + kk;
            const uint4 raw = *reinterpret_cast<const uint4*>(Kc + (head + j % C) * D + e0);
            const T* ev = reinterpret_cast<const T*>(&raw);
#pragma unroll
            for (int i = 0; i < kVec; ++i) dot = __builtin_fmaf(qv[i], to_f32(ev[i]), dot);
        }
#pragma unroll
        for (int off = 1; off < G; off <<= 1) dot += __shfl_xor(dot, off);
        if (lane % G == 0 && kk < nk) x_s[kk] = dot;
    }
    const float ct = cc[head + t % C];
    __syncthreads();

    float x = -INFINITY;
    if (tid < nk)
        x = __builtin_fmaf(x_s[tid], kscale, (ct - cc[head + (j0 + tid) % C]) * kLog2e);
    float m = x;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if (lane == 0) s_red[wid] = m;
    __syncthreads();
    m = s_red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) m = fmaxf(m, s_red[w]);
    __syncthreads();
    const float p = tid < nk ? fast_exp2(x - m) : 0.f;
    float l = p;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) l += __shfl_xor(l, off);
    if (lane == 0) s_red[wid] = l;
    x_s[tid] = p;
    __syncthreads();
    l = s_red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) l += s_red[w];

    // P V over the same rows, then over the lanes that hold the same columns
    float acc[kVec];
#pragma unroll
    for (int i = 0; i < kVec; ++i) acc[i] = 0.f;
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int kk = 64 * wid + kRows * it + lane / G;
        if (kk < nk) {
            const int j = j0 + kk;
            const float pj = x_s[kk];
            const uint4 raw = *reinterpret_cast<const uint4*>(Vc + (head + j % C) * D + e0);
            const T* ev = reinterpret_cast<const T*>(&raw);
#pragma unroll
            for (int i = 0; i < kVec; ++i) acc[i] = __builtin_fmaf(pj, to_f32(ev[i]), acc[i]);
        }
    }
#pragma unroll
    for (int off = G; off < 64; off <<= 1)
#pragma unroll
        for (int i = 0; i < kVec; ++i) acc[i] += __shfl_xor(acc[i], off);
    if (lane < G)
#pragma unroll
        for (int i = 0; i < kVec; ++i) red[wid][e0 + i] = acc[i];
    __syncthreads();
    if (tid < D) {
        float o = red[0][tid];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) o += red[w][tid];
        out[2 + tid] = o;
    }
    if (tid == 0) { out[0] = m; out[1] = l; }
}

// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(
    const float* __restrict__ part, int nsplit, T* __restrict__ O, float* __restrict__ lse) {
    const int bh = blockIdx.x, tid = threadIdx.x;
    const float* P = part + (size_t)bh * nsplit * (D + 2);
    float M = -INFINITY;
    for (int s = 0; s < nsplit; ++s) M = fmaxf(M, P[(size_t)s * (D + 2)]);
    float l = 0.f, o = 0.f;
    for (int s = 0; s < nsplit; ++s) {
        const float* ps = P + (size_t)s * (D + 2);
        const float w = fast_exp2(ps[0] - M);          // 0 for workgroups past the window
        l = __builtin_fmaf(w, ps[1], l);
        o = __builtin_fmaf(w, ps[2 + tid], o);
    }
    O[(size_t)bh * D + tid] = from_f32<T>(o / l);
    if (tid == 0) lse[bh] = (M + fast_log2(l)) * kLn2;
}

// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t init_t(const DecodeInitArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((decode_init_kernel<T, D>), dim3(a.B * a.H), dim3(kPlanThreads), 0, s,
                       (const T*)a.K, (const T*)a.V, a.log_f, a.gamma_q, a.gamma_k, a.H, a.L0,
                       a.C, a.log_lmax_over_eps, (T*)a.Kc, (T*)a.Vc, a.cc, a.cs, a.ptr, a.delta,
                       a.flags);
    return hipGetLastError();
}

hipError_t launch_decode_init(const DecodeInitArgs& a, hipStream_t s) {
    trace_begin(ACP_K_DECODE_INIT, s);
    hipError_t e;
    if (a.bf16) e = a.d == 64 ? init_t<__bf16, 64>(a, s) : init_t<__bf16, 128>(a, s);
    else e = a.d == 64 ? init_t<float, 64>(a, s) : init_t<float, 128>(a, s);
    if (e == hipSuccess) trace_end(ACP_K_DECODE_INIT, s);
    return e;
}

template <typename T, int D>
static hipError_t step_t(const DecodeArgs& a, hipStream_t s) {
    const int BH = a.B * a.H;
    const int nsplit = (min(a.t + 1, a.C) + kDecChunk - 1) / kDecChunk;
    hipLaunchKernelGGL((decode_append_kernel<T, D>), dim3(BH), dim3(64), 0, s,
                       (const T*)a.k, (const T*)a.v, a.log_f, a.t, a.C, (T*)a.Kc, (T*)a.Vc, a.cc,
                       a.cs, a.ptr, a.delta, a.flags);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((decode_attn_kernel<T, D>), dim3(nsplit, BH), dim3(kDecChunk), 0, s,
                       (const T*)a.q, (const T*)a.Kc, (const T*)a.Vc, a.cc, a.ptr, a.t, a.C,
                       nsplit, kLog2e / sqrtf((float)D), a.part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((decode_combine_kernel<T, D>), dim3(BH), dim3(D), 0, s, a.part, nsplit,
                       (T*)a.O, a.lse);
    return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t s) {
    trace_begin(ACP_K_DECODE, s);
    hipError_t e;
    if (a.bf16) e = a.d == 64 ? step_t<__bf16, 64>(a, s) : step_t<__bf16, 128>(a, s);
    else e = a.d == 64 ? step_t<float, 64>(a, s) : step_t<float, 128>(a, s);
    if (e == hipSuccess) trace_end(ACP_K_DECODE, s);
    return e;
}

}  // namespace acp
