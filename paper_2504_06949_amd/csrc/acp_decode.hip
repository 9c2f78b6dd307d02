// Decoding with ACP (paper App. F, inference-time ACP; the threshold of Sec. 3).
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
//   decode_init_kernel  prompt of L0 tokens -> delta, the running cumsum (a
//                       double-double pair),
//                       c of the prompt's last C positions, the pointer of query
//                       L0 - 1
//   decode_copy_kernel  the prompt's last K/V rows into the ring
//   decode_step_kernel  one token: c_t, the pointer advance, query t over its
//                       kept keys (256 per workgroup, partial softmax sums), and
//                       the append of k_t, v_t
//   decode_combine_kernel  the partial sums of each head merged into O and lse
//                       (a second launch: its start orders every workgroup's
//                       partials before it without a device-wide fence, which
//                       would write back a whole L2 per workgroup)
//
// The running sum and the pointer are kept twice, the values after position p
// in copy p mod 2: every workgroup of step t reads copy (t - 1) mod 2 while the
// first one writes copy t mod 2, so no workgroup sees a half-updated state.
// The ring slot that token t takes over held position t - C, which no query from
// t on attends to; the workgroups read k_t and v_t from the inputs, not the ring.
#include "acp_device.h"
#include "acp_internal.h"
#include "acp_scan.h"

namespace acp {

constexpr int kDecChunk = 256;   // keys per attention workgroup (64 per wave)

size_t decode_partials_floats(int BH, int C, int d) {
    const int nsplit = (C + kDecChunk - 1) / kDecChunk;
    return (size_t)BH * nsplit * (d + 2);
}

// ring slot of position j (j >= 0)
__device__ __forceinline__ int ring(int j, int C) { return j % C; }

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kPlanThreads) void decode_init_kernel(
    const float* __restrict__ log_f,
    const float* __restrict__ gamma_q, const float* __restrict__ gamma_k, int H, int L0, int C,
    double log_lmax_over_eps, float* __restrict__ cc,
    double* __restrict__ cs_out, int* __restrict__ ptr_out, double* __restrict__ delta_out,
    int* __restrict__ flags_out) {
    __shared__ double s_dbl[2][kPlanWaves];
    __shared__ double s_dbl2[2][kPlanWaves];
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
    // float64 first, double-double for a head whose sums span 53 bits or more (the
    // rule of the plan kernel, which explains it)
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
    const double incl = block_inclusive_scan(local, s_dbl[0]);
    auto sum = [](double a, double b) { return a + b; };
    auto imin = [](int a, int b) { return min(a, b); };
    auto ior = [](int a, int b) { return a | b; };
    const double total_abs = block_reduce(local_abs, s_dbl2[0], sum);
    min_lsb = block_reduce(min_lsb, s_int, imin);
    bool wide = false;   // uniform: every thread holds the same totals
    if (total_abs > 0.0) {
        const int biased = (int)((__double_as_longlong(total_abs) >> 52) & 0x7ff);
        const int top = (biased > 0 ? biased : 1) - 1023 + 1;
        wide = top - min_lsb >= 53;
    }
    auto emit = [&](auto run) __attribute__((always_inline)) {
        for (int i = beg; i < end; ++i) {
            run = sum_add(run, x[i]);
            const float cf = sum_f32(run);
            if (i >= L0 - C) cc[(size_t)bh * C + (i % C)] = cf;
            if ((i & (kBlock - 1)) == kBlock - 1) s_last[i / kBlock] = cf;
            if (i == L0 - 1) {
                double* cs = cs_out + 2 * ((size_t)((L0 - 1) & 1) * gridDim.x + bh);
                cs[0] = sum_hi(run);
                cs[1] = sum_lo(run);
                s_ct = cf;
            }
        }
    };
    if (wide) {
        DD l{0.0, 0.0}, la{0.0, 0.0};
        for (int i = beg; i < end; ++i) {
            const double v = (double)x[i];
            l = dd_add(l, v);
            la = dd_add(la, __builtin_fabs(v));
        }
        const DD inc = block_inclusive_scan_dd(l, s_dbl[0], s_dbl[1]);
        const DD total = block_sum_dd(la, s_dbl2[0], s_dbl2[1]);
        if (t == 0 && total.hi > 0.0) {
            if (dd_top_exp(total) - min_lsb >= kExactSpanBits) flags |= 4;
            if (__builtin_isinf(dd_to_f32(total))) flags |= 2;
        }
        emit(dd_add(inc, dd_neg(l)));
    } else {
        if (t == 0 && total_abs > 0.0 && !__builtin_isfinite((float)total_abs)) flags |= 2;
        emit(incl - local);
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
        ptr_out[(size_t)((L0 - 1) & 1) * gridDim.x + bh] = max(lo, first > 0 ? first / kBlock : 0);
        flags_out[bh] = flags;
    }
}

// The prompt's last min(L0, C) K and V rows into their ring slots: grid
// (ceil(rows / 64), B*H), each workgroup 64 rows of both tensors, every lane's
// 16-byte pieces requested before any is stored.
constexpr int kCopyRows = 64;

template <typename T, int D>
__global__ __launch_bounds__(256) void decode_copy_kernel(
    const T* __restrict__ K, const T* __restrict__ V, int L0, int C, T* __restrict__ Kc,
    T* __restrict__ Vc) {
    constexpr int kVec = 16 / (int)sizeof(T);
    constexpr int kPerRow = D / kVec;                  // 16-byte pieces per row
    constexpr int kPer = kCopyRows * kPerRow / 256;    // pieces per thread and tensor
    const int bh = blockIdx.y, t = threadIdx.x;
    const int j0 = max(0, L0 - C);
    const int r0 = j0 + blockIdx.x * kCopyRows;
    uint4 kv[kPer], vv[kPer];
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
        // rows past the prompt read its last row again (branch-free)
        const int i = t + 256 * p, j = min(r0 + i / kPerRow, L0 - 1), e = (i % kPerRow) * kVec;
        const size_t src = ((size_t)bh * L0 + j) * D + e;
        kv[p] = *reinterpret_cast<const uint4*>(K + src);
        vv[p] = *reinterpret_cast<const uint4*>(V + src);
    }
    __builtin_amdgcn_sched_barrier(0);   // all requests out before the first store
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
        // (a row past the prompt rewrites the last row's slot with the same bytes)
        const int i = t + 256 * p, j = min(r0 + i / kPerRow, L0 - 1), e = (i % kPerRow) * kVec;
        const size_t dst = ((size_t)bh * C + (j % C)) * D + e;
        *reinterpret_cast<uint4*>(Kc + dst) = kv[p];
        *reinterpret_cast<uint4*>(Vc + dst) = vv[p];
    }
}

// ---------------------------------------------------------------------------
// Token t of every (batch, head); grid (nsplit, B*H), nsplit workgroups of 256
// threads per head, enough to cover min(t + 1, C) keys.
//   1. The previous pointer p fixes the key range [j_base, t], j_base =
//      max(64 p, t - C + 1); workgroup s takes keys j_base + 256 s .. + 255,
//      wave w of it the 64 from 64 w.  Rows are read whole by groups of G lanes
//      (16 bytes each); the K rows, the V rows (held in registers when they fit)
//      and the c of the keys are requested together.
//   2. Meanwhile every wave forms c_t = float32(cum + log f_t) and finds the new
//      pointer n, the first kept block from max(p, block of position t - C + 1)
//      on, 64 blocks per ballot; keys below max(64 n, t - C + 1) are masked.
//   3. Softmax over the workgroup's keys and P V; the workgroup writes (max, sum,
//      unnormalised O) with logits in log2 units, or max = -inf if it kept none.
//   4. Workgroup 0 writes the state of position t: cum, pointer, flags, c_t, and
//      k_t, v_t in slot t mod C.
template <typename T, int D>
__global__ __launch_bounds__(kDecChunk) void decode_step_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ log_f, int t, int C, T* __restrict__ Kc, T* __restrict__ Vc,
    float* __restrict__ cc, double* __restrict__ cum, int* __restrict__ ptr,
    const double* __restrict__ delta, int* __restrict__ flags, float* __restrict__ part,
    float kscale) {
    constexpr int kVec = 16 / (int)sizeof(T);   // elements per 16-byte piece
    constexpr int G = D / kVec;                 // lanes per cache row
    constexpr int kRows = 64 / G;               // rows per wave load
    constexpr int kIter = 64 / kRows;           // loads per wave for its 64 rows
    constexpr int kWaves = kDecChunk / 64;
    constexpr bool kHoldV = kIter <= 8;         // V rows requested with the K rows
    constexpr int kHeld = kHoldV ? kIter : 1;
    __shared__ float x_s[kDecChunk];
    __shared__ float red[kWaves][D];
    __shared__ float s_red[kWaves];

    const int bh = blockIdx.y, sp = blockIdx.x, nsplit = gridDim.x, BH = gridDim.y;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const size_t head = (size_t)bh * C;
    const float* crow = cc + head;
    float* pml = part + (size_t)bh * nsplit * 2;                            // [nsplit][2]
    float* po = part + (size_t)BH * nsplit * 2 + (size_t)bh * nsplit * D;   // [nsplit][D]

    const int rd = (t - 1) & 1;
    const int nb = t / kBlock, gone = t - C;
    const int first = gone + 1 > 0 ? gone + 1 : 0;          // oldest position held
    // (clamped to [0, nb], so that even a corrupted state indexes inside the ring)
    const int p_old = min(max(ptr[(size_t)rd * BH + bh], 0), nb);
    const DD cs_old{cum[2 * ((size_t)rd * BH + bh)], cum[2 * ((size_t)rd * BH + bh) + 1]};
    const float lff = log_f[bh];
    const double dl = delta[bh];
    const int e0 = (lane % G) * kVec;
    const uint4 qraw = *reinterpret_cast<const uint4*>(q + (size_t)bh * D + e0);

    const int j0 = max(kBlock * p_old, first) + sp * kDecChunk;
    if (j0 > t) {                             // past the window (never workgroup 0)
        if (tid == 0) {
            pml[2 * sp] = -INFINITY;          // weight 0 in the merge
            pml[2 * sp + 1] = 0.f;
        }
        return;
    }
    const int nk = min(kDecChunk, t - j0 + 1);                // keys in this chunk

    // c at the last key of blocks n_start .. n_start + 63 for the pointer search,
    // requested first so that it returns before the rows (loads complete in order)
    const int n_start = max(p_old, first / kBlock);
    // (with nb = 0 every lane is kept anyway; slot 63 is read only to stay branch-free)
    float cb = crow[ring(kBlock * min(n_start + lane, max(nb - 1, 0)) + kBlock - 1, C)];

    // ---- 1. requests for the chunk's rows ----------------------------------------
    // Slot of key j0 + kk: at most one wrap, since kk < nk <= C.  Lanes past the
    // chunk load its last row again (branch-free and in bounds) and are masked.
    const int s0 = ring(j0, C);
    auto slot = [&](int kk) {
        const int sl = s0 + kk;
        return sl >= C ? sl - C : sl;
    };
    const int kk_max = nk - 1;
    uint4 kraw[kIter];
    uint4 vraw[kHeld];
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int kk = min(64 * wid + kRows * it + lane / G, kk_max);
        const bool last = j0 + kk == t;      // k_t, v_t come from the inputs
        const size_t row = (head + slot(kk)) * D + e0;
        const T* kr = last ? k + (size_t)bh * D + e0 : Kc + row;
        kraw[it] = *reinterpret_cast<const uint4*>(kr);
        if constexpr (kHoldV) {
            const T* vr = last ? v + (size_t)bh * D + e0 : Vc + row;
            vraw[it] = *reinterpret_cast<const uint4*>(vr);
        }
    }
    float cj = crow[slot(min(tid, kk_max))];
    // all requests above are issued before anything waits for the first of them
    asm volatile("" : "+v"(cb) : : "memory");

    // ---- 2. c_t and the new pointer --------------------------------------------------
    // cum + log f_t as a pair: TwoSum of the leading parts, then the remainders
    // (the one addition that can round; step 4 checks it), then TwoSum again
    const DD s1 = two_sum(cs_old.hi, (double)lff);
    const DD lo_sum = two_sum(cs_old.lo, s1.lo);
    const DD s2 = two_sum(s1.hi, lo_sum.hi);
    const float ct = dd_to_f32(s2);
    // blocks n .. n + 63 per ballot; the block holding t (n >= nb) is always kept
    int n = n_start;
    unsigned long long bal = __ballot(n + lane >= nb || (double)ct - (double)cb >= dl);
    while (bal == 0ull) {                     // a jump of more than 64 blocks (rare)
        n += 64;
        const float c2 = crow[ring(kBlock * min(n + lane, nb - 1) + kBlock - 1, C)];
        bal = __ballot(n + lane >= nb || (double)ct - (double)c2 >= dl);
    }
    n += __builtin_ctzll(bal);
    // The rows stay opaque until here, so that the compiler neither waits for them
    // before the search nor unpacks them early into twice the registers.
#pragma unroll
    for (int it = 0; it < kIter; ++it)
        asm volatile("" : "+v"(kraw[it].x), "+v"(kraw[it].y), "+v"(kraw[it].z), "+v"(kraw[it].w));
    if constexpr (kHoldV) {
#pragma unroll
        for (int it = 0; it < kHeld; ++it)
            asm volatile("" : "+v"(vraw[it].x), "+v"(vraw[it].y), "+v"(vraw[it].z), "+v"(vraw[it].w));
    }
    const int j_lo = max(kBlock * n, first);
    // this chunk's kept keys: kk in [kk_lo, nk)
    const int kk_lo = min(max(j_lo - j0, 0), nk);

    // ---- 3. softmax and P V ------------------------------------------------------------
    if (kk_lo < nk) {
        float qv[kVec];
        {
            const T* ev = reinterpret_cast<const T*>(&qraw);
#pragma unroll
            for (int i = 0; i < kVec; ++i) qv[i] = to_f32(ev[i]);
        }
#pragma unroll
        for (int it = 0; it < kIter; ++it) {
            const int kk = 64 * wid + kRows * it + lane / G;
            const T* ev = reinterpret_cast<const T*>(&kraw[it]);
            float dot = 0.f;
#pragma unroll
            for (int i = 0; i < kVec; ++i) dot = __builtin_fmaf(qv[i], to_f32(ev[i]), dot);
#pragma unroll
            for (int off = 1; off < G; off <<= 1) dot += __shfl_xor(dot, off);
            if (lane % G == 0 && kk < nk) x_s[kk] = dot;
        }
        __syncthreads();

        float x = -INFINITY;
        if (tid >= kk_lo && tid < nk) {
            if (j0 + tid == t) cj = ct;         // the ring's slot still holds t - C
            x = __builtin_fmaf(x_s[tid], kscale, (ct - cj) * kLog2e);
        }
        float m = x;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
        if (lane == 0) s_red[wid] = m;
        __syncthreads();
        m = s_red[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) m = fmaxf(m, s_red[w]);
        __syncthreads();
        const float p = (tid >= kk_lo && tid < nk) ? fast_exp2(x - m) : 0.f;
        float l = p;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) l += __shfl_xor(l, off);
        if (lane == 0) s_red[wid] = l;
        x_s[tid] = p;
        __syncthreads();
        l = s_red[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) l += s_red[w];

        float acc[kVec];
#pragma unroll
        for (int i = 0; i < kVec; ++i) acc[i] = 0.f;
#pragma unroll
        for (int it = 0; it < kIter; ++it) {
            const int kk = 64 * wid + kRows * it + lane / G;
            if (kk >= kk_lo && kk < nk) {
                const float pj = x_s[kk];
                uint4 raw;
                if constexpr (kHoldV) {
                    raw = vraw[it];
                } else {
                    const T* vr = j0 + kk == t ? v + (size_t)bh * D + e0
                                               : Vc + (head + slot(kk)) * D + e0;
                    raw = *reinterpret_cast<const uint4*>(vr);
                }
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
            po[(size_t)sp * D + tid] = o;
        }
        if (tid == 0) {
            pml[2 * sp] = m;
            pml[2 * sp + 1] = l;
        }
    } else if (tid == 0) {
        pml[2 * sp] = -INFINITY;              // no kept key here: weight 0 in the merge
        pml[2 * sp + 1] = 0.f;
    }

    // ---- 4. the state of position t ---------------------------------------------------
    if (sp == 0) {
        if (tid == 0) {
            int fl = flags[bh];
            if (!__builtin_isfinite(lff)) fl |= 2;
            else if (lff > 0.0f) fl |= 1;
            // the running pair stays the exact prefix sum only while the sum of the
            // remainders does not round
            if (lo_sum.lo != 0.0) fl |= 4;
            // A kept key is lost iff the block of position t - C is kept (the blocks
            // before it are then kept too); its last key is still in the ring.
            if (gone >= 0) {
                const int nx = gone / kBlock;
                if ((double)ct - (double)crow[ring(kBlock * nx + kBlock - 1, C)] >= dl) fl |= 16;
            }
            flags[bh] = fl;
            cum[2 * ((size_t)(t & 1) * BH + bh)] = s2.hi;
            cum[2 * ((size_t)(t & 1) * BH + bh) + 1] = s2.lo;
            ptr[(size_t)(t & 1) * BH + bh] = n;
            cc[head + ring(t, C)] = ct;
        }
        for (int e = tid * kVec; e < D; e += kDecChunk * kVec) {
            const size_t dst = (head + ring(t, C)) * D + e;
            *reinterpret_cast<uint4*>(Kc + dst) = *reinterpret_cast<const uint4*>(k + (size_t)bh * D + e);
            *reinterpret_cast<uint4*>(Vc + dst) = *reinterpret_cast<const uint4*>(v + (size_t)bh * D + e);
        }
    }
}

// ---------------------------------------------------------------------------
// The partial sums of one head merged into O and lse: one workgroup per head,
// of 256 threads, or 1024 when a long context leaves more than 256 splits (up to
// 512).  Thread i takes the (max, sum) of split i, and dim i mod D of splits
// i / D, i / D + THREADS / D, ..., whose loads it issues kBatch at a time before
// it waits for any of them (the first batch together with the (max, sum) loads).
template <typename T, int D, int THREADS>
__global__ __launch_bounds__(THREADS) void decode_combine_kernel(
    int nsplit, const float* __restrict__ part, T* __restrict__ O, float* __restrict__ lse) {
    constexpr int kWaves = THREADS / 64;
    constexpr int kGroups = THREADS / D;
    constexpr int kBatch = 8;
    __shared__ float w_s[THREADS];   // nsplit <= THREADS
    __shared__ float o_s[THREADS];
    __shared__ float s_m[kWaves], s_l[kWaves];
    const int bh = blockIdx.x, BH = gridDim.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const float* pml = part + (size_t)bh * nsplit * 2;
    const float* po = part + (size_t)BH * nsplit * 2 + (size_t)bh * nsplit * D;
    const int dim = tid % D, grp = tid / D;

    const int sm = min(tid, nsplit - 1);
    // The first batch of partial outputs is requested with the (max, sum) pairs:
    // it does not depend on them (a split without a kept key is selected away
    // below), so small merges make one round trip to memory instead of two.
    float pv0[kBatch];
#pragma unroll
    for (int r = 0; r < kBatch; ++r) pv0[r] = po[(size_t)min(grp + kGroups * r, nsplit - 1) * D + dim];
    float ms = pml[2 * sm], ls = pml[2 * sm + 1];
    if (tid >= nsplit) {
        ms = -INFINITY;
        ls = 0.f;
    }
    float M = ms;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
    if (lane == 0) s_m[wid] = M;
    __syncthreads();
    M = s_m[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, s_m[w]);
    float L = ms != -INFINITY ? ls * fast_exp2(ms - M) : 0.f;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) L += __shfl_xor(L, off);
    if (lane == 0) s_l[wid] = L;
    if (tid < nsplit) w_s[tid] = fast_exp2(ms - M);
    __syncthreads();
    L = s_l[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) L += s_l[w];
    // splits without a kept key (weight 0) hold no O: selected away, not multiplied
    float o = 0.f;
#pragma unroll
    for (int r = 0; r < kBatch; ++r) {
        const int s2 = grp + kGroups * r;
        if (s2 < nsplit) {
            const float w = w_s[s2];
            o += w != 0.f ? w * pv0[r] : 0.f;
        }
    }
    for (int s0 = grp + kGroups * kBatch; s0 < nsplit; s0 += kGroups * kBatch) {
        float pv[kBatch];
#pragma unroll
        for (int r = 0; r < kBatch; ++r)
            pv[r] = po[(size_t)min(s0 + kGroups * r, nsplit - 1) * D + dim];
#pragma unroll
        for (int r = 0; r < kBatch; ++r) {
            const int s2 = s0 + kGroups * r;
            if (s2 < nsplit) {
                const float w = w_s[s2];
                o += w != 0.f ? w * pv[r] : 0.f;
            }
        }
    }
    o_s[tid] = o;
    __syncthreads();
    if (tid < D) {
        float r = o_s[tid];
#pragma unroll
        for (int g2 = 1; g2 < kGroups; ++g2) r += o_s[g2 * D + tid];
        O[(size_t)bh * D + tid] = from_f32<T>(r / L);
    }
    if (tid == 0) lse[bh] = (M + fast_log2(L)) * kLn2;
}

// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t init_t(const DecodeInitArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((decode_init_kernel<D>), dim3(a.B * a.H), dim3(kPlanThreads), 0, s,
                       a.log_f, a.gamma_q, a.gamma_k, a.H, a.L0,
                       a.C, a.log_lmax_over_eps, a.cc, a.cs, a.ptr, a.delta, a.flags);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int rows = min(a.L0, a.C);
    hipLaunchKernelGGL((decode_copy_kernel<T, D>),
                       dim3((rows + kCopyRows - 1) / kCopyRows, a.B * a.H), dim3(256), 0, s,
                       (const T*)a.K, (const T*)a.V, a.L0, a.C, (T*)a.Kc, (T*)a.Vc);
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
    const int nsplit = (min(a.t + 1, a.C) + kDecChunk - 1) / kDecChunk;
    hipLaunchKernelGGL((decode_step_kernel<T, D>), dim3(nsplit, a.B * a.H), dim3(kDecChunk), 0, s,
                       (const T*)a.q, (const T*)a.k, (const T*)a.v, a.log_f, a.t, a.C, (T*)a.Kc,
                       (T*)a.Vc, a.cc, a.cs, a.ptr, a.delta, a.flags, a.part,
                       kLog2e / sqrtf((float)D));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    static_assert(64 * 2048 / kDecChunk <= 1024, "one split per combine thread");
    if (nsplit <= 256)
        hipLaunchKernelGGL((decode_combine_kernel<T, D, 256>), dim3(a.B * a.H), dim3(256), 0, s,
                           nsplit, a.part, (T*)a.O, a.lse);
    else
        hipLaunchKernelGGL((decode_combine_kernel<T, D, 1024>), dim3(a.B * a.H), dim3(1024), 0, s,
                           nsplit, a.part, (T*)a.O, a.lse);
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
