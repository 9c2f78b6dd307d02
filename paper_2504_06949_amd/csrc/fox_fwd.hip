// Forgetting Attention forward over the blocks kept by ACP (paper Sec. 2,
// eq. 1-2 and its FlashAttention paragraph; Sec. 3, "Two-stage implementation":
// each query block starts at its boundary block, and the K/V of pruned blocks
// are never loaded).
//
// Logits are kept in log2 units, y_ij = (q_i . k_j) log2(e)/sqrt(d) +
// (c_i - c_j) log2(e), and the decay term is split so that no float32 value
// carries more than the decay it contributes:
//   * keys of an earlier 64-key block than the query's own: with R the
//     cumulative gate at the first query of the query's pruning block,
//     c_i - c_j = (c_i - R) + (R - c_j), and c_i <= R <= c_j, so both parts are
//     <= 0 and no larger in size than c_i - c_j itself.  (c_i - R) is a row term
//     folded into the MFMA accumulator start; (R - c_j) log2(e) a key bias held
//     in LDS per tile, one copy per query block of the workgroup.  The rounding
//     of either part is relative to |c_i - c_j|, and the weight it enters is
//     e^(c_i - c_j) times the logit factor, so the error it leaves in P is a few
//     float32 ulps however strong the forgetting.
//   * the query's own block (the peeled diagonal tiles): c_i - c_j per entry
//     from the stored float32 gates, exact when they are within a factor of two
//     of each other (and relative to the difference otherwise).
// y is therefore the logit itself, with no frame to undo; c itself grows
// without bound along the sequence and never enters a sum of its own size.
// The backward recomputes P_ij = 2^(y_ij - L_i) from the log-sum-exp
// L_i = LSE_i log2(e) in the same way.
//
// Softmax stabiliser.  ACP already bounds every logit of the head: |q.k|/sqrt(d)
// <= U and c_i - c_j <= 0, so each row's logits are <= U, while the diagonal
// logit is >= -U.  Subtracting U log2(e) from y therefore keeps every exponent
// <= 0 and the largest term >= e^(-2U).  For U <= kUFixedMax that largest term
// is a normal float32 and the online running maximum (and its rescaling of the
// accumulators) is not needed: the constant is folded into the MFMA accumulator
// start, and each logit of an off-diagonal tile costs one FMA and one exp2.
// Heads with a larger U take the online-maximum variant; one launch holds both,
// and each workgroup takes its head's.
#include <type_traits>

#include "acp_device.h"
#include "acp_internal.h"

namespace acp {

constexpr int kFwdThreads = 256;
constexpr int kFwdRows = 128;
constexpr double kUFixedMax = 32.0;

// ---------------------------------------------------------------------------
// bf16 path: v_mfma_f32_16x16x32_bf16, fp32 accumulation.
//
// Workgroup = 4 waves = 128 queries (two 64-row pruning blocks); wave w owns
// 32 queries that all sit in one pruning row, so a pruned or non-causal tile is
// skipped wave-uniformly and no pruned entry is ever computed.  Key/value tiles
// of 64 rows are double-buffered in LDS (swizzled panels, filled by DMA loads
// straight from HBM/L2 while the previous tile is computed); V^T operands come
// from LDS transpose reads.
//
// S^T = K Q^T is computed (keys x queries) so that each lane holds one query and
// eight consecutive keys of P afterwards, which is exactly the B operand of
// O^T = V^T P^T.  For that, the A-operand rows of S^T are read from K in the
// order krow(kt, r) = 32 (kt / 2) + 8 (r / 4) + 4 (kt % 2) + r % 4.
// ---------------------------------------------------------------------------

template <int D>
struct alignas(1024) FwdSmem {
    unsigned char k[2][128 * D];   // 64 x D bf16 tiles (see tile_off)
    unsigned char v[2][128 * D];
    float kb[2][2][64];            // key bias (R - c_j) log2(e), per query block of the workgroup
    float kc[2][64];               // c_j (diagonal tiles)
    float qc[128];                 // c_i of the workgroup's queries (diagonal tiles)
};

template <int D, bool kFixed>
__device__ __forceinline__ void fwd_bf16_body(
    FwdSmem<D>& sm, int qb, int bh, double u_head,
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const float* __restrict__ cg, const int* __restrict__ row_start,
    __bf16* __restrict__ O, float* __restrict__ lse,
    float* __restrict__ lse2, int L, int M, int nqb, float kscale) {
    constexpr int NDS = D / 32;                     // k-steps over the head dim
    constexpr int NDT = D / 16;                     // output tiles over the head dim
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const int q0 = qb * kFwdRows;
    const int wq0 = q0 + 32 * w;
    const bool wave_on = wq0 < L;
    const int mw = wq0 / 64;
    const int m0 = q0 / 64;
    const size_t head = (size_t)bh * L;
    const int n_lo = row_start[(size_t)bh * M + m0];
    const int n_hi = min(m0 + 1, M - 1);
    const int w_lo = wave_on ? row_start[(size_t)bh * M + mw] : (1 << 30);
    // R of the workgroup's two query blocks (the second repeats the first when
    // the sequence ends after 64 rows) and of this wave's block
    const float rb0 = cg[head + q0];
    const float rb1 = q0 + 64 < L ? cg[head + q0 + 64] : rb0;
    const float rw = (w >> 1) ? rb1 : rb0;
    const float uf = (float)u_head;
    const float sqrt_d = sqrtf((float)D);

    bf16x8 qf[2][NDS];
    // MFMA accumulator starts: off-diagonal tiles carry the row term (c_i - R)
    // and the fixed stabiliser, diagonal tiles the stabiliser alone (uniform)
    f32x4 sinit[2];
    const float sdiag = kFixed ? -uf * sqrt_d : 0.f;
    float cq[2] = {0.f, 0.f};
    if (wave_on) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                qf[qt][ds] = *reinterpret_cast<const bf16x8*>(
                    Q + (head + wq0 + 16 * qt + r16) * D + 32 * ds + 8 * g);
            cq[qt] = cg[head + wq0 + 16 * qt + r16];
        }
    }
    if (tid < 128) sm.qc[tid] = q0 + tid < L ? cg[head + q0 + tid] : 0.f;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const float row = cq[qt] - rw;
        const float init = kFixed ? (row - uf) * sqrt_d : row * sqrt_d;
        sinit[qt] = f32x4{init, init, init, init};
    }

    // Tile n: K and V by DMA into LDS, the 64 gate values through registers.
    // The gate load goes first: vmcnt retires in order, so waiting for it later
    // does not wait for the tile's DMA.
    TileDma<D, 4> dma;
    dma.init(w, lane);
    auto issue = [&](int n, int buf) __attribute__((always_inline)) {
        const float4 c = tid < 16 ? *reinterpret_cast<const float4*>(cg + head + 64 * n + 4 * tid)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
        dma.issue(sm.k[buf], K + (head + (size_t)64 * n) * D, w);
        dma.issue(sm.v[buf], V + (head + (size_t)64 * n) * D, w);
        return c;
    };
    auto put_kb = [&](float4 c, int buf) __attribute__((always_inline)) {
        if (tid < 16) {
            const float4 b0 = make_float4((rb0 - c.x) * kLog2e, (rb0 - c.y) * kLog2e,
                                          (rb0 - c.z) * kLog2e, (rb0 - c.w) * kLog2e);
            const float4 b1 = make_float4((rb1 - c.x) * kLog2e, (rb1 - c.y) * kLog2e,
                                          (rb1 - c.z) * kLog2e, (rb1 - c.w) * kLog2e);
            *reinterpret_cast<float4*>(&sm.kb[buf][0][4 * tid]) = b0;
            *reinterpret_cast<float4*>(&sm.kb[buf][1][4 * tid]) = b1;
            *reinterpret_cast<float4*>(&sm.kc[buf][4 * tid]) = c;
        }
    };

    f32x4 acc[2][NDT];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float mrun[2] = {-INFINITY, -INFINITY};
    float lrun[2] = {0.f, 0.f};   // sum of the float32 weights (for the log-sum-exp)
    // Sum of the bfloat16 weights that enter P V, formed by the matrix cores: one
    // more 16-row output tile against an all-ones operand, whose rows all come out
    // as the lane's query's weight sum (fixed stabiliser only).
    f32x4 lbf[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};

    // Per-lane LDS offsets.  The swizzle of a fragment row depends only on the
    // lane, so the tile-row steps below are compile-time offsets.
    int koff[NDS], voff[NDT];
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) koff[ds] = tile_off(8 * (r16 >> 2) + (r16 & 3), 32 * ds + 8 * g);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) voff[dt] = tile_off(8 * g + (r16 >> 2), 16 * dt + 4 * (r16 & 3));

    // Each key tile is taken in two halves of 32 keys (ks = 0, 1), each in three
    // phases: A forms S^T (MFMA; key rows and key biases from LDS), B the weights
    // P (VALU), C accumulates O^T (MFMA; V^T columns from LDS).  Each phase reads
    // its LDS operands itself, holding no operand across a phase, and scheduling
    // barriers keep the compiler from hoisting them: that keeps the kernel within
    // 128 VGPRs at d = 64 (four waves per SIMD, whose interleaving hides the LDS
    // latency) and 256 at d = 128 (two waves).
    struct OpA {
        bf16x8 a[2][NDS];   // key subtiles 2 ks, 2 ks + 1
        float4 nk[2];       // key biases (diagonal tiles: gates c_j) of the lane's keys
                            // 32 ks + 8 g + (0..3 | 4..7)
    };
    struct OpC {
        bf16x8 v[NDT];
    };
    struct SHalf {
        f32x4 s[2][2];      // [subtile][qt]
    };
    auto load_a = [&](auto mask_tag, int buf, int ks) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        const float* nkrow = kMask ? sm.kc[buf] : sm.kb[buf][w >> 1];
        OpA r;
        const unsigned char* ktile = sm.k[buf];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                // row krow = 32 ks + 4 kk + (row of koff)
                r.a[kk][ds] = *reinterpret_cast<const bf16x8*>(
                    ktile + koff[ds] + 128 * (32 * ks + 4 * kk));
#pragma unroll
        for (int i = 0; i < 2; ++i)
            r.nk[i] = *reinterpret_cast<const float4*>(&nkrow[32 * ks + 8 * g + 4 * i]);
        return r;
    };
    auto load_c = [&](int buf, int ks) __attribute__((always_inline)) {
        OpC r;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) r.v[dt] = tile_col8_at(sm.v[buf] + voff[dt] + 128 * 32 * ks);
        return r;
    };
    auto phase_a = [&](auto mask_tag, const OpA& ra) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        const f32x4 sd = f32x4{sdiag, sdiag, sdiag, sdiag};
        SHalf x;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                x.s[kk][0] = mfma16(ra.a[kk][ds], qf[0][ds], ds == 0 ? (kMask ? sd : sinit[0]) : x.s[kk][0]);
                x.s[kk][1] = mfma16(ra.a[kk][ds], qf[1][ds], ds == 0 ? (kMask ? sd : sinit[1]) : x.s[kk][1]);
            }
        return x;
    };
    // The lane's keys in half ks are 32 ks + 8 g + j, j = 0..7 (j < 4 from
    // subtile 2 ks), its query qloc = 32 (w % 2) + 16 qt + r16 within the tile.
    // kMask: the tile may be this wave's diagonal one, where keys after the query
    // are dropped.  The test is 32 ks + j > qk with the lane's qk = qloc - 8 g,
    // raised out of reach on tiles that are not diagonal, so that the comparisons
    // take immediate operands.  Such tiles form the decay c_i - c_j per entry.
    // Returns P of the half for both query subtiles.
    struct PHalf {
        bf16x8 p[2];
    };
    auto phase_b = [&](auto mask_tag, const SHalf& x, const OpA& ra, int qk0, int ks) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        const float nk[8] = {ra.nk[0].x, ra.nk[0].y, ra.nk[0].z, ra.nk[0].w,
                             ra.nk[1].x, ra.nk[1].y, ra.nk[1].z, ra.nk[1].w};
        PHalf pt;
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            int qk = qk0 + 16 * qt;
            if constexpr (kMask) asm volatile("" : "+v"(qk));
            float ci = 0.f;
            if constexpr (kMask) ci = sm.qc[32 * w + 16 * qt + r16];
            // exponent of entry j: the row term is in x.s off the diagonal
            auto expo = [&](int j) __attribute__((always_inline)) {
                const float bias = kMask ? (ci - nk[j]) * kLog2e : nk[j];
                return __builtin_fmaf(x.s[j >> 2][qt][j & 3], kscale, bias);
            };
            if constexpr (kFixed) {
                float l = lrun[qt];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    float p = fast_exp2(expo(j));
                    if (kMask && 32 * ks + j > qk) p = 0.f;
                    l += p;
                    pt.p[qt][j] = (__bf16)p;
                }
                lrun[qt] = l;
            } else {
                float y[8];
                float mx = -INFINITY;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    float v = expo(j);
                    if (kMask && 32 * ks + j > qk) v = -INFINITY;
                    y[j] = v;
                    mx = fmaxf(mx, v);
                }
                mx = fmaxf(mx, __shfl_xor(mx, 16));
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const float mnew = fmaxf(mrun[qt], mx);
                // (finite: the first half of every tile holds at least one key that
                // no row of the wave masks)
                const float alpha = fast_exp2(mrun[qt] - mnew);
                mrun[qt] = mnew;
                float l = lrun[qt] * alpha;
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) acc[qt][dt] *= alpha;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float p = fast_exp2(y[j] - mnew);
                    l += p;
                    pt.p[qt][j] = (__bf16)p;
                }
                lrun[qt] = l;
            }
        }
        return pt;
    };
    // O^T += V^T P^T over the half's 32 keys
    auto phase_c = [&](const OpC& rc, const PHalf& pt) __attribute__((always_inline)) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            acc[0][dt] = mfma16(rc.v[dt], pt.p[0], acc[0][dt]);
            acc[1][dt] = mfma16(rc.v[dt], pt.p[1], acc[1][dt]);
        }
        if constexpr (kFixed) {
            bf16x8 ones;
#pragma unroll
            for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
            lbf[0] = mfma16(ones, pt.p[0], lbf[0]);
            lbf[1] = mfma16(ones, pt.p[1], lbf[1]);
        }
    };

    // tile n_lo in LDS and published; tile n_lo + 1 on its way
    put_kb(issue(n_lo, 0), 0);
    wait_vmcnt0();
    __syncthreads();
    float4 cnext = make_float4(0.f, 0.f, 0.f, 0.f);
    if (n_lo < n_hi) cnext = issue(n_lo + 1, 1);
    int buf = 0;
    auto step = [&](auto mask_tag, int n) __attribute__((always_inline)) {
        const bool act = n >= w_lo && n <= mw;
        const int qk0 = 32 * (w & 1) + r16 - 8 * g + (n == mw ? 0 : 4096);
        if (act) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                __builtin_amdgcn_sched_barrier(0);
                const OpA ra = load_a(mask_tag, buf, ks);
                const SHalf x = phase_a(mask_tag, ra);
                __builtin_amdgcn_sched_barrier(0);
                const PHalf pt = phase_b(mask_tag, x, ra, qk0, ks);
                __builtin_amdgcn_sched_barrier(0);
                const OpC rc = load_c(buf, ks);
                phase_c(rc, pt);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (n < n_hi) put_kb(cnext, buf ^ 1);
        // tile n + 1 has landed and every wave's reads of tile n are complete
        wait_vmcnt0_lgkmcnt0();
        __syncthreads();
        const bool more = n + 1 < n_hi;
        if (more && tid < 16) cnext = *reinterpret_cast<const float4*>(cg + head + 64 * (n + 2) + 4 * tid);
        if (more) dma.issue(sm.k[buf], K + (head + (size_t)64 * (n + 2)) * D, w);
        if (more) dma.issue(sm.v[buf], V + (head + (size_t)64 * (n + 2)) * D, w);
        buf ^= 1;
    };
    // The diagonal tiles (m0 for waves 0-1, m0 + 1 for waves 2-3) are the last
    // two and go through the masking variant.
    const int n_mask = max(n_lo, n_hi - 1);
    int n = n_lo;
    for (; n < n_mask; ++n) step(std::false_type{}, n);
    for (; n <= n_hi; ++n) step(std::true_type{}, n);

    if (!wave_on) return;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        float lt = lrun[qt];
        lt += __shfl_xor(lt, 16);
        lt += __shfl_xor(lt, 32);
        // O is normalised by the sum of the weights it was built from: with the
        // fixed stabiliser the largest weight is not 1, and normalising the
        // bfloat16-weighted sum by the float32 sum would leave its rounding in O.
        const float lo = kFixed ? lbf[qt][0] : lt;
        const float inv = 1.0f / lo;
        const int query = wq0 + 16 * qt + r16;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const f32x4 o = acc[qt][dt] * inv;
            const size_t off = (head + query) * D + 16 * dt + 4 * g;
            bf16x4 ob;
            ob[0] = (__bf16)o[0]; ob[1] = (__bf16)o[1]; ob[2] = (__bf16)o[2]; ob[3] = (__bf16)o[3];
            *reinterpret_cast<bf16x4*>(O + off) = ob;
        }
        if (g == 0) {
            // L_i = LSE_i log2(e): fixed variant  U log2(e) + log2(l_i);
            // online variant  max_j y_ij + log2(l_i)
            const float l2 = kFixed ? uf * kLog2e + fast_log2(lt) : mrun[qt] + fast_log2(lt);
            lse2[head + query] = l2;
            lse[head + query] = l2 * kLn2;
        }
    }
}

// One launch for both variants: the head's bound picks the body (uniform over
// the workgroup), and the two bodies share the workgroup's LDS.
template <int D>
__global__ __launch_bounds__(kFwdThreads) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 2)))
void fwd_bf16_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const float* __restrict__ cg, const int* __restrict__ row_start,
    const double* __restrict__ bound_u, const int* __restrict__ sched, __bf16* __restrict__ O,
    float* __restrict__ lse, float* __restrict__ lse2, int L, int M, int nqb, int nblocks,
    float kscale) {
    __shared__ FwdSmem<D> sm;
    const int item = sched[xcd_logical_id(blockIdx.x, nblocks)];   // bh * nqb + query block
    const int bh = item / nqb;
    const double u_head = bound_u[bh];
    if (u_head <= kUFixedMax)
        fwd_bf16_body<D, true>(sm, item % nqb, bh, u_head, Q, K, V, cg, row_start, O, lse, lse2,
                               L, M, nqb, kscale);
    else
        fwd_bf16_body<D, false>(sm, item % nqb, bh, u_head, Q, K, V, cg, row_start, O, lse, lse2,
                                L, M, nqb, kscale);
}

// ---------------------------------------------------------------------------
// fp32 path: plain VALU arithmetic, one thread per query, 64 queries (one
// pruning row) per workgroup; K/V tiles staged in LDS; online maximum.  The
// decay is split at R = c of the block's first query off the diagonal and
// formed per entry on it, as in the bf16 path.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void fwd_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ cg, const int* __restrict__ row_start,
    float* __restrict__ O, float* __restrict__ lse,
    float* __restrict__ lse2, int L, int M, float kscale) {
    __shared__ float ks[64 * D];
    __shared__ float vs[64 * D];
    __shared__ float nc[64];   // (R - c_j) log2(e), or c_j on the diagonal tile
    const int bh = blockIdx.x / M, m = blockIdx.x % M, t = threadIdx.x;
    const size_t head = (size_t)bh * L;
    const int query = 64 * m + t;
    const float rref = cg[head + 64 * m];
    const float ci = cg[head + query];
    const float row = (ci - rref) * kLog2e;
    float q[D], acc[D];
#pragma unroll
    for (int k = 0; k < D; ++k) { q[k] = Q[(head + query) * D + k]; acc[k] = 0.f; }
    float mrun = -INFINITY, lrun = 0.f;
    const int n0 = row_start[(size_t)bh * M + m];
    for (int n = n0; n <= m; ++n) {
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
            float s = 0.f;
#pragma unroll
            for (int k = 0; k < D; ++k) s = __builtin_fmaf(q[k], ks[j * D + k], s);
            const float y = n == m ? __builtin_fmaf(s, kscale, (ci - nc[j]) * kLog2e)
                                   : __builtin_fmaf(s, kscale, nc[j]) + row;
            if (y > mrun) {
                const float alpha = fast_exp2(mrun - y);
                lrun *= alpha;
#pragma unroll
                for (int k = 0; k < D; ++k) acc[k] *= alpha;
                mrun = y;
            }
            const float p = fast_exp2(y - mrun);
            lrun += p;
#pragma unroll
            for (int k = 0; k < D; ++k) acc[k] = __builtin_fmaf(p, vs[j * D + k], acc[k]);
        }
    }
    const float inv = 1.0f / lrun;
#pragma unroll
    for (int k = 0; k < D; ++k) {
        const float o = acc[k] * inv;
        O[(head + query) * D + k] = o;
    }
    const float l2 = mrun + fast_log2(lrun);
    lse2[head + query] = l2;
    lse[head + query] = l2 * kLn2;
}

// ---------------------------------------------------------------------------
template <int D>
static void launch_fwd_bf16(const FwdArgs& a, int M, float kscale, hipStream_t s) {
    const int BH = a.B * a.H;
    const int nqb = (a.L + kFwdRows - 1) / kFwdRows;
    const int nblocks = BH * nqb;
    hipLaunchKernelGGL((fwd_bf16_kernel<D>), dim3(nblocks), dim3(kFwdThreads), 0, s,
                       (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V, a.c,
                       a.row_start, a.u, a.sched, (__bf16*)a.O, a.lse, a.lse2, a.L, M, nqb,
                       nblocks, kscale);
}

hipError_t launch_fwd(const FwdArgs& a, hipStream_t s) {
    const int BH = a.B * a.H, M = a.L / 64;
    const float kscale = kLog2e / sqrtf((float)a.d);
    trace_begin(ACP_K_FWD, s);
    if (a.bf16) {
        if (a.d == 64) launch_fwd_bf16<64>(a, M, kscale, s);
        else launch_fwd_bf16<128>(a, M, kscale, s);
    } else {
        if (a.d == 64)
            hipLaunchKernelGGL(fwd_f32_kernel<64>, dim3(BH * M), dim3(64), 0, s,
                               (const float*)a.Q, (const float*)a.K, (const float*)a.V, a.c,
                               a.row_start, (float*)a.O, a.lse, a.lse2, a.L, M, kscale);
        else
            hipLaunchKernelGGL(fwd_f32_kernel<128>, dim3(BH * M), dim3(64), 0, s,
                               (const float*)a.Q, (const float*)a.K, (const float*)a.V, a.c,
                               a.row_start, (float*)a.O, a.lse, a.lse2, a.L, M, kscale);
    }
    const hipError_t e = hipGetLastError();
    trace_end(ACP_K_FWD, s);
    return e;
}

}  // namespace acp
