// bf16 backward passes of Forgetting Attention over the blocks kept by ACP
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  The formulas are the chain
// rule through eq. 2 and the cumulative gates (see fox_bwd.hip); P is
// recomputed from the forward's log-sum-exp L_i = LSE_i log2(e):
//   P_ij = 2^(q_i.k_j log2(e)/sqrt(d) + (c_i - c_j) log2(e) - L_i).
// The decay is split as in the forward (fox_fwd.hip): off the diagonal block,
// c_i - c_j = (c_i - R) + (R - c_j) with R the cumulative gate at the boundary
// of the pruning block the wave owns (its first query in the dQ pass, its last
// key in the dK/dV pass), so that both parts share the sign of c_i - c_j and
// neither is larger; on the diagonal tiles c_i - c_j is formed per entry.  The
// part that belongs to the wave's own rows goes into the MFMA accumulator start
// together with -L_i, the other part is a bias held per column.
//
// Both passes use 4 waves of 32 rows (two 64-row pruning blocks per workgroup),
// so a pruned or non-causal tile is skipped wave-uniformly, and work through
// each 64-row tile of the other operand in two halves of 32 to keep register
// pressure low; at d = 64 both fit 168 VGPRs, i.e. three waves per SIMD.  Tiles
// are double-buffered in LDS (swizzled panels filled by DMA loads while the
// previous tile is computed); operands whose contraction runs over sequence
// positions come from LDS transpose reads.
#include <type_traits>

#include "acp_device.h"
#include "acp_internal.h"

namespace acp {

constexpr int kBwdThreads = 256;
constexpr int kBwdRows = 128;

// ---------------------------------------------------------------------------
// dQ pass: one workgroup per 128 queries, loop over kept key blocks.
// S^T = K Q^T and dP^T = V dO^T are formed keys x queries so that dS^T lands
// in the B-operand layout of dQ^T = K^T dS^T.  The A-operand rows are read in
// the order krow = 32 h + 8 (r / 4) + 4 t + r % 4 (half h, subtile t).
// ---------------------------------------------------------------------------
template <int D>
struct alignas(1024) DqSmem {
    unsigned char k[2][128 * D];   // 64 x D bf16 tiles (see tile_off)
    unsigned char v[2][128 * D];
    float kb[2][2][64];            // key bias (R - c_j) log2(e), per query block of the workgroup
    float kc[2][64];               // c_j (diagonal tiles)
};

template <int D>
__global__ __launch_bounds__(kBwdThreads) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2)))
void dq_bf16_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ O, const __bf16* __restrict__ dO, const float* __restrict__ cg,
    const int* __restrict__ row_start, const float* __restrict__ lse2,
    float* __restrict__ dsum, __bf16* __restrict__ dQ, float* __restrict__ rowsum,
    const int* __restrict__ sched, int L, int M, int nqb, int nblocks, float kscale,
    float qscale) {
    constexpr int NDS = D / 32;
    constexpr int NDT = D / 16;
    __shared__ DqSmem<D> sm;

    const int item = sched[xcd_logical_id(blockIdx.x, nblocks)];   // bh * nqb + query block
    const int bh = item / nqb;
    const int qb = item % nqb;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const int q0 = qb * kBwdRows;
    const int wq0 = q0 + 32 * w;
    const bool wave_on = wq0 < L;
    const int mw = wq0 / 64;
    const int m0 = q0 / 64;
    const size_t head = (size_t)bh * L;
    const int n_lo = row_start[(size_t)bh * M + m0];
    const int n_hi = min(m0 + 1, M - 1);
    const int w_lo = wave_on ? row_start[(size_t)bh * M + mw] : (1 << 30);
    // R of the workgroup's two query blocks and of this wave's
    const float rb0 = cg[head + q0];
    const float rb1 = q0 + 64 < L ? cg[head + q0 + 64] : rb0;
    const float rw = (w >> 1) ? rb1 : rb0;

    bf16x8 qf[2][NDS], dof[2][NDS];
    float aq[2] = {0.f, 0.f}, dl[2] = {0.f, 0.f}, cq[2] = {0.f, 0.f}, lq[2] = {0.f, 0.f};
    if (wave_on) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            const size_t row = head + wq0 + 16 * qt + r16;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                qf[qt][ds] = *reinterpret_cast<const bf16x8*>(Q + row * D + 32 * ds + 8 * g);
                dof[qt][ds] = *reinterpret_cast<const bf16x8*>(dO + row * D + 32 * ds + 8 * g);
            }
            cq[qt] = cg[row];
            lq[qt] = lse2[row];
            aq[qt] = (cq[qt] - rw) * kLog2e - lq[qt];
            // Delta_i = rowdot(dO, O) over the lane's columns, then across the four
            // lanes that hold row i
            float dd = 0.f;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                const bf16x8 o8 = *reinterpret_cast<const bf16x8*>(O + row * D + 32 * ds + 8 * g);
#pragma unroll
                for (int e = 0; e < 8; ++e) dd = __builtin_fmaf((float)dof[qt][ds][e], (float)o8[e], dd);
            }
            dd += __shfl_xor(dd, 16);
            dd += __shfl_xor(dd, 32);
            dl[qt] = dd;
        }
    }

    // The small per-tile loads go first: vmcnt retires in order, so waiting for
    // them later does not wait for the tile's DMA.
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
    // per-lane LDS offsets (the swizzle of a fragment row depends only on the lane)
    int roff[NDS], coff[NDT];
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) roff[ds] = tile_off(8 * (r16 >> 2) + (r16 & 3), 32 * ds + 8 * g);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) coff[dt] = tile_off(8 * g + (r16 >> 2), 16 * dt + 4 * (r16 & 3));

    f32x4 acc[2][NDT];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Row terms folded into the MFMA accumulator starts: S starts at a_i / k' so
    // that fma(S, k', key bias) is the exponent (a_i = (c_i - R) log2(e) - L_i off
    // the diagonal, -L_i on it), and dP starts at -Delta_i so that it comes out
    // as dP - Delta.
    f32x4 sinit[2], dinit[2];
    float sdiag[2];   // (made into accumulator starts where the diagonal tiles use them)
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const float a = aq[qt] / kscale;
        sdiag[qt] = -lq[qt] / kscale;
        float b = -dl[qt];
        asm volatile("" : "+v"(b));   // the epilogue reads -Delta_i back from dinit
        sinit[qt] = f32x4{a, a, a, a};
        dinit[qt] = f32x4{b, b, b, b};
    }
    float sds[2] = {0.f, 0.f};   // sum_j dS_ij (lane partial)

    // Each key tile is taken in two halves of 32 keys, each in three phases: A
    // forms S^T and dP^T (MFMA; key rows from LDS), B the softmax terms (VALU),
    // C accumulates dQ (MFMA; key columns from LDS).  Each phase reads its own
    // LDS operands, so that the kernel fits 168 VGPRs at d = 64 (three waves per
    // SIMD) and 256 at d = 128 (two): the other waves' interleaving hides the LDS
    // latency.
    struct OpA {
        bf16x8 a[2][NDS], b[2][NDS];
        float4 lo, hi;                 // key biases (diagonal tiles: gates c_j) of the lane's 8 keys
    };
    struct OpC {
        bf16x8 ak[NDT];
    };
    struct SdP {
        f32x4 s[2][2], dp[2][2];
    };
    struct DsH {   // dS of the half in the B-operand layout of the dQ product
        bf16x8 d[2];
    };
    // diag: the tile goes through the masking variant (gates instead of biases)
    auto load_a = [&](bool diag, int buf, int h) __attribute__((always_inline)) {
        const float* nkrow = diag ? sm.kc[buf] : sm.kb[buf][w >> 1];
        OpA r;
        const unsigned char* ktile = sm.k[buf];
        const unsigned char* vtile = sm.v[buf];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            // row 32 h + 4 t + (row of roff)
            const int rstep = 128 * (32 * h + 4 * t);
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                r.a[t][ds] = *reinterpret_cast<const bf16x8*>(ktile + roff[ds] + rstep);
                r.b[t][ds] = *reinterpret_cast<const bf16x8*>(vtile + roff[ds] + rstep);
            }
        }
        r.lo = *reinterpret_cast<const float4*>(&nkrow[32 * h + 8 * g]);
        r.hi = *reinterpret_cast<const float4*>(&nkrow[32 * h + 8 * g + 4]);
        return r;
    };
    auto load_c = [&](int buf, int h) __attribute__((always_inline)) {
        OpC r;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) r.ak[dt] = tile_col8_at(sm.k[buf] + coff[dt] + 128 * 32 * h);
        return r;
    };
    auto phase_a = [&](auto mask_tag, const OpA& ra) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        f32x4 init[2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            if constexpr (kMask) {
                // formed here, so that no copy of it stays live through the loop
                float a = sdiag[qt];
                asm volatile("" : "+v"(a));
                init[qt] = f32x4{a, a, a, a};
            } else {
                init[qt] = sinit[qt];
            }
        }
        SdP x;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
                for (int qt = 0; qt < 2; ++qt) {
                    x.s[t][qt] = mfma16(ra.a[t][ds], qf[qt][ds], ds == 0 ? init[qt] : x.s[t][qt]);
                    x.dp[t][qt] = mfma16(ra.b[t][ds], dof[qt][ds], ds == 0 ? dinit[qt] : x.dp[t][qt]);
                }
        return x;
    };
    // The lane's keys are 32 h + 8 g + j, j = 0..7 (j < 4 from subtile 0), its
    // query qloc = 32 (w % 2) + 16 qt + r16 within the tile.  kMask: the tile may
    // be this wave's diagonal one, where keys after the query are dropped.  The
    // test is 32 h + j > qk with the lane's qk = qloc - 8 g, raised out of reach
    // on tiles that are not diagonal, so that the comparisons take immediates.
    // Such tiles form the decay c_i - c_j per entry.
    auto phase_b = [&](auto mask_tag, const SdP& x, const OpA& ra, int h, int qk0) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        const float nk[8] = {ra.lo.x, ra.lo.y, ra.lo.z, ra.lo.w, ra.hi.x, ra.hi.y, ra.hi.z, ra.hi.w};
        bf16x8 dsf[2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            int qk = qk0 + 16 * qt;
            if constexpr (kMask) asm volatile("" : "+v"(qk));
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int t = j >> 2, u = j & 3;
                const float bias = kMask ? (cq[qt] - nk[j]) * kLog2e : nk[j];
                float p = fast_exp2(__builtin_fmaf(x.s[t][qt][u], kscale, bias));
                if (kMask && 32 * h + j > qk) p = 0.f;
                const float dsv = p * x.dp[t][qt][u];
                sds[qt] += dsv;
                dsf[qt][j] = (__bf16)dsv;
            }
        }
        return DsH{{dsf[0], dsf[1]}};
    };
    // dQ^T += K^T dS^T over the half's 32 keys
    auto phase_c = [&](const OpC& rc, const DsH& y) __attribute__((always_inline)) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            acc[0][dt] = mfma16(rc.ak[dt], y.d[0], acc[0][dt]);
            acc[1][dt] = mfma16(rc.ak[dt], y.d[1], acc[1][dt]);
        }
    };

    // tile n_lo in LDS and published; tile n_lo + 1 on its way
    put_kb(issue(n_lo, 0), 0);
    wait_vmcnt0();
    __syncthreads();
    float4 cnext = make_float4(0.f, 0.f, 0.f, 0.f);
    if (n_lo < n_hi) cnext = issue(n_lo + 1, 1);
    int buf = 0;
    if constexpr (D == 64) {
    auto step = [&](auto mask_tag, int n) __attribute__((always_inline)) {
        const bool act = n >= w_lo && n <= mw;
        const int qk0 = 32 * (w & 1) + r16 - 8 * g + (n == mw ? 0 : 4096);
        if (act) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const OpA ra = load_a(decltype(mask_tag)::value, buf, h);
                const SdP x = phase_a(mask_tag, ra);
                const DsH y = phase_b(mask_tag, x, ra, h, qk0);
                const OpC rc = load_c(buf, h);
                phase_c(rc, y);
            }
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
    // The diagonal tiles (m0 for waves 0-1, m0 + 1 = n_hi for waves 2-3) are the
    // last two and go through the masking variant.
    const int n_mask = max(n_lo, n_hi - 1);
    int n = n_lo;
    for (; n < n_mask; ++n) step(std::false_type{}, n);
    for (; n <= n_hi; ++n) step(std::true_type{}, n);
    } else {
    // d = 128: phase A is split in two, S^T with the key rows and dP^T with the
    // value rows, each read just before its MFMAs, so that no more than one
    // operand set is live next to the wave's Q and dO fragments and dQ.
    struct OpS {
        bf16x8 a[2][NDS];
        float4 lo, hi;
    };
    struct OpD {
        bf16x8 b[2][NDS];
    };
    auto load_s = [&](bool diag, int buf, int h) __attribute__((always_inline)) {
        const float* nkrow = diag ? sm.kc[buf] : sm.kb[buf][w >> 1];
        OpS r;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int rstep = 128 * (32 * h + 4 * t);
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                r.a[t][ds] = *reinterpret_cast<const bf16x8*>(sm.k[buf] + roff[ds] + rstep);
        }
        r.lo = *reinterpret_cast<const float4*>(&nkrow[32 * h + 8 * g]);
        r.hi = *reinterpret_cast<const float4*>(&nkrow[32 * h + 8 * g + 4]);
        return r;
    };
    auto load_d = [&](int buf, int h) __attribute__((always_inline)) {
        OpD r;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int rstep = 128 * (32 * h + 4 * t);
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                r.b[t][ds] = *reinterpret_cast<const bf16x8*>(sm.v[buf] + roff[ds] + rstep);
        }
        return r;
    };
    auto phase_s = [&](auto mask_tag, const OpS& rs, SdP& x) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        f32x4 init[2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            if constexpr (kMask) {
                float a = sdiag[qt];
                asm volatile("" : "+v"(a));
                init[qt] = f32x4{a, a, a, a};
            } else {
                init[qt] = sinit[qt];
            }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
                for (int qt = 0; qt < 2; ++qt)
                    x.s[t][qt] = mfma16(rs.a[t][ds], qf[qt][ds], ds == 0 ? init[qt] : x.s[t][qt]);
    };
    auto phase_d = [&](const OpD& rd, SdP& x) __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
                for (int qt = 0; qt < 2; ++qt)
                    x.dp[t][qt] = mfma16(rd.b[t][ds], dof[qt][ds], ds == 0 ? dinit[qt] : x.dp[t][qt]);
    };
    auto step = [&](auto mask_tag, int n) __attribute__((always_inline)) {
        const bool act = n >= w_lo && n <= mw;
        const int qk0 = 32 * (w & 1) + r16 - 8 * g + (n == mw ? 0 : 4096);
        if (act) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                __builtin_amdgcn_sched_barrier(0);
                SdP x;
                const OpS rs = load_s(decltype(mask_tag)::value, buf, h);
                phase_s(mask_tag, rs, x);
                __builtin_amdgcn_sched_barrier(0);
                {
                    const OpD rd = load_d(buf, h);
                    phase_d(rd, x);
                }
                __builtin_amdgcn_sched_barrier(0);
                OpA ra;
                ra.lo = rs.lo;
                ra.hi = rs.hi;
                const DsH y = phase_b(mask_tag, x, ra, h, qk0);
                __builtin_amdgcn_sched_barrier(0);
                const OpC rc = load_c(buf, h);
                phase_c(rc, y);
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
    const int n_mask = max(n_lo, n_hi - 1);
    int n = n_lo;
    for (; n < n_mask; ++n) step(std::false_type{}, n);
    for (; n <= n_hi; ++n) step(std::true_type{}, n);
    }

    if (!wave_on) return;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const int query = wq0 + 16 * qt + r16;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const f32x4 o = acc[qt][dt] * qscale;
            bf16x4 ob;
            ob[0] = (__bf16)o[0]; ob[1] = (__bf16)o[1]; ob[2] = (__bf16)o[2]; ob[3] = (__bf16)o[3];
            *reinterpret_cast<bf16x4*>(dQ + (head + query) * D + 16 * dt + 4 * g) = ob;
        }
        // Delta'_i = sum_j P_ij dP_ij from the float32 P and dP of this pass
        // (= sum_j dS_ij + Delta_i sum_j P_ij): it is what rowdot(dO, O) equals for
        // the exact O, free of the rounding of P to bfloat16 in the forward's PV
        // product.  The dK/dV pass uses it for dS.  sum_j P_ij is 1 here up to
        // float32 rounding, since L_i is the log of the forward's float32 weight
        // sum; the row sums of dS, Delta'_i (1 - sum_j P_ij), are therefore zero
        // to that rounding, as they are exactly for any softmax (its value does not
        // change when a whole row of logits is shifted).
        float a = sds[qt];
        a += __shfl_xor(a, 16);
        a += __shfl_xor(a, 32);
        if (g == 0) {
            dsum[head + query] = a - dinit[qt][0];
            rowsum[head + query] = 0.f;
        }
    }
}

// ---------------------------------------------------------------------------
// dK/dV pass: one workgroup per 128 keys, looping over query blocks
// m = first key block .. col_end[last key block].  Each wave owns 32 keys that
// lie in one pruning column.  At d = 64 four waves each take both 32-query
// halves of every tile.  At d = 128 eight waves run, two per key group: each
// takes one half of every tile, so that its dK and dV accumulators (32 keys x
// 128 columns, twice) fit two waves per SIMD, and the pair's partial sums are
// added through LDS at the end.
// S = Q K^T and dP = dO V^T are formed queries x keys so that P and dS land in
// the B-operand layout of dV^T = dO^T P and dK^T = Q^T dS.  The A-operand rows
// (queries) are read in the order qrow = 32 h + 8 (r / 4) + 4 t + r % 4.
// ---------------------------------------------------------------------------
template <int D>
struct DkvShape {
    static constexpr int QSPLIT = D == 64 ? 1 : 2;    // waves sharing a key group
    static constexpr int NW = 4 * QSPLIT;             // waves per workgroup
    static constexpr bool kVinLds = D == 128;         // V rows from LDS (else registers)
};

template <int D>
struct alignas(1024) DkvSmem {
    unsigned char q[2][128 * D];   // 64 x D bf16 tiles (see tile_off)
    unsigned char o[2][128 * D];   // dO
    unsigned char k[2][128 * D];   // the workgroup's 128 keys (two tiles)
    // d = 128: their values (the B operand of dP)
    unsigned char v[DkvShape<D>::kVinLds ? 2 : 1][DkvShape<D>::kVinLds ? 128 * D : 16];
    float la[2][2][64];            // a_i / k',  a_i = (c_i - R) log2(e) - L_i, per key block
    float ll[2][64];               // -L_i / k' (diagonal tiles)
    float lc[2][64];               // c_i (diagonal tiles)
    float dl[2][64];               // -Delta'_i
    float kc[128];                 // c_j of the workgroup's keys (diagonal tiles)
};

template <int D>
__global__ __launch_bounds__(64 * DkvShape<D>::NW) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2)))
void dkdv_bf16_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ cg,
    const int* __restrict__ col_end, const float* __restrict__ lse2,
    const float* __restrict__ dsum, __bf16* __restrict__ dK, __bf16* __restrict__ dV,
    float* __restrict__ colsum, const int* __restrict__ sched, int L, int M, int nkb,
    int nblocks, float kscale, float qscale) {
    constexpr int NDS = D / 32;
    constexpr int NDT = D / 16;
    constexpr int QSPLIT = DkvShape<D>::QSPLIT, NW = DkvShape<D>::NW;
    constexpr bool kVinLds = DkvShape<D>::kVinLds;
    __shared__ DkvSmem<D> sm;

    const int item = sched[xcd_logical_id(blockIdx.x, nblocks)];   // bh * nkb + key block
    const int bh = item / nkb;
    const int kb = item % nkb;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kg = w & 3;                   // the wave's key group
    const int qh = w >> 2;                  // its query half (d = 128)
    const int wb = kg >> 1;                 // the key group's block in the workgroup
    const int g = lane >> 4, r16 = lane & 15;
    const int k0 = kb * kBwdRows;
    const int wk0 = k0 + 32 * kg;
    const bool wave_on = wk0 < L;
    const int nw = wk0 / 64;
    const int n0 = k0 / 64;
    const size_t head = (size_t)bh * L;
    const int m_lo = n0;
    const int m_hi = col_end[(size_t)bh * M + min(n0 + 1, M - 1)];
    const int w_hi = wave_on ? col_end[(size_t)bh * M + nw] : -1;
    const float kinv = 1.0f / kscale;
    // R of the workgroup's two key blocks (the gate at each block's last key; the
    // second repeats the first when the sequence ends after 64 keys) and of this
    // wave's block
    const float rb0 = cg[head + k0 + 63];
    const float rb1 = k0 + 64 < L ? cg[head + k0 + 127] : rb0;
    const float rw = wb ? rb1 : rb0;

    bf16x8 vf[2][kVinLds ? 1 : NDS];   // d = 64: the wave's V rows
    float nk[2] = {0.f, 0.f};          // (R - c_j) log2(e) of the lane's keys
    if (tid < 128) sm.kc[tid] = k0 + tid < L ? cg[head + k0 + tid] : 0.f;
    if (wave_on) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            const size_t row = head + wk0 + 16 * kt + r16;
            if constexpr (!kVinLds) {
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds)
                    vf[kt][ds] = *reinterpret_cast<const bf16x8*>(V + row * D + 32 * ds + 8 * g);
            }
            nk[kt] = (rw - cg[row]) * kLog2e;
        }
    }

    // The small per-row loads go first and are combined only after the tile's
    // compute: vmcnt retires in order, so using them does not wait for the DMA.
    TileDma<D, NW> dma;
    dma.init(w, lane);
    auto issue = [&](int m, int buf) __attribute__((always_inline)) {
        float3 r = make_float3(0.f, 0.f, 0.f);
        if (tid < 64) {
            const size_t row = head + 64 * m + tid;
            r = make_float3(cg[row], lse2[row], dsum[row]);
        }
        dma.issue(sm.q[buf], Q + (head + (size_t)64 * m) * D, w);
        dma.issue(sm.o[buf], dO + (head + (size_t)64 * m) * D, w);
        return r;
    };
    auto put_rows = [&](float3 r, int buf) __attribute__((always_inline)) {
        if (tid < 64) {
            sm.la[buf][0][tid] = ((r.x - rb0) * kLog2e - r.y) * kinv;
            sm.la[buf][1][tid] = ((r.x - rb1) * kLog2e - r.y) * kinv;
            sm.ll[buf][tid] = -r.y * kinv;
            sm.lc[buf][tid] = r.x;
            sm.dl[buf][tid] = -r.z;
        }
    };
    int roff[NDS], coff[NDT];
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) roff[ds] = tile_off(8 * (r16 >> 2) + (r16 & 3), 32 * ds + 8 * g);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) coff[dt] = tile_off(8 * g + (r16 >> 2), 16 * dt + 4 * (r16 & 3));

    f32x4 dk[2][NDT], dv[2][NDT];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            dk[kt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
            dv[kt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    float csum[2] = {0.f, 0.f};

    // Each query half of 32 queries is taken in four phases: S (MFMA; query rows,
    // the accumulator starts and the key rows from LDS), dP (dO rows from LDS, V
    // from registers at d = 64 and from LDS at d = 128), the softmax terms (VALU),
    // and dV, dK (MFMA; query columns from LDS).  No operand is held across a
    // phase, and scheduling barriers keep the compiler from hoisting the next
    // phase's LDS reads: the other waves on the SIMD (three at d = 64, two at
    // d = 128) fill the wait, and the kernel stays within their register budget
    // (168, resp. 256).
    struct OpS {
        bf16x8 a[2][NDS];
        f32x4 si[2];
    };
    struct OpD {
        bf16x8 b[2][NDS];
        f32x4 di[2];
    };
    struct OpC {
        bf16x8 ao[NDT], aq[NDT];
    };
    struct SdP {
        f32x4 s[2][2], dp[2][2];
    };
    struct PdS {
        bf16x8 pb[2], db[2];
    };
    // diag: the tile goes through the masking variant (S starts at -L_i / k')
    auto load_s = [&](bool diag, int buf, int h) __attribute__((always_inline)) {
        OpS r;
        const float* sirow = diag ? sm.ll[buf] : sm.la[buf][wb];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            // rows 32 h + 4 t + (row of roff); the lane's accumulator rows are the
            // queries 32 h + 8 g + 4 t + u, whose a_i / k' and -Delta'_i start S
            // and dP, so the MFMAs leave the exponent's row term and dP - Delta'
            r.si[t] = *reinterpret_cast<const f32x4*>(&sirow[32 * h + 8 * g + 4 * t]);
            const int rstep = 128 * (32 * h + 4 * t);
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                r.a[t][ds] = *reinterpret_cast<const bf16x8*>(sm.q[buf] + roff[ds] + rstep);
        }
        return r;
    };
    auto load_d = [&](int buf, int h) __attribute__((always_inline)) {
        OpD r;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            r.di[t] = *reinterpret_cast<const f32x4*>(&sm.dl[buf][32 * h + 8 * g + 4 * t]);
            const int rstep = 128 * (32 * h + 4 * t);
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                r.b[t][ds] = *reinterpret_cast<const bf16x8*>(sm.o[buf] + roff[ds] + rstep);
        }
        return r;
    };
    auto load_c = [&](int buf, int h) __attribute__((always_inline)) {
        OpC r;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            r.ao[dt] = tile_col8_at(sm.o[buf] + coff[dt] + 128 * 32 * h);
            r.aq[dt] = tile_col8_at(sm.q[buf] + coff[dt] + 128 * 32 * h);
        }
        return r;
    };
    // the wave's keys: rows 32 (kg % 2) + 16 kt + (lane % 16) of K tile kg / 2
    const int krow = 32 * (kg & 1) + r16;
    auto phase_s = [&](const OpS& rs, SdP& x) __attribute__((always_inline)) {
        bf16x8 kr[2][NDS];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) kr[kt][ds] = tile_row8(sm.k[wb], krow + 16 * kt, 32 * ds + 8 * g);
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
                    x.s[t][kt] = mfma16(rs.a[t][ds], kr[kt][ds], ds == 0 ? rs.si[t] : x.s[t][kt]);
    };
    auto phase_d = [&](const OpD& rd, SdP& x) __attribute__((always_inline)) {
        if constexpr (kVinLds) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds) {
                    const bf16x8 vr = tile_row8(sm.v[wb], krow + 16 * kt, 32 * ds + 8 * g);
#pragma unroll
                    for (int t = 0; t < 2; ++t)
                        x.dp[t][kt] = mfma16(rd.b[t][ds], vr, ds == 0 ? rd.di[t] : x.dp[t][kt]);
                }
        } else {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt)
                        x.dp[t][kt] = mfma16(rd.b[t][ds], vf[kt][ds], ds == 0 ? rd.di[t] : x.dp[t][kt]);
        }
    };
    // The lane's queries are 32 h + 8 g + j, j = 0..7 (j < 4 from subtile 0).
    // kMask: the tile may be this wave's diagonal one, where key kloc is dropped
    // for the queries before it.  The test is kq > 32 h + j with the lane's
    // kq = kloc - 8 g, lowered out of reach on tiles that are not diagonal, so
    // that the comparisons take immediate operands.  Such tiles form the decay
    // c_i - c_j per entry (c_i from LDS).
    auto phase_b = [&](auto mask_tag, const SdP& x, int buf, int h, int kq0) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask_tag)::value;
        float ci[8], ck[2];
        if constexpr (kMask) {
            const float4 a = *reinterpret_cast<const float4*>(&sm.lc[buf][32 * h + 8 * g]);
            const float4 b = *reinterpret_cast<const float4*>(&sm.lc[buf][32 * h + 8 * g + 4]);
            ci[0] = a.x; ci[1] = a.y; ci[2] = a.z; ci[3] = a.w;
            ci[4] = b.x; ci[5] = b.y; ci[6] = b.z; ci[7] = b.w;
            ck[0] = sm.kc[32 * kg + r16];
            ck[1] = sm.kc[32 * kg + 16 + r16];
        }
        PdS y;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            int kq = kq0 + 16 * kt;
            if constexpr (kMask) asm volatile("" : "+v"(kq));
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int t = j >> 2, u = j & 3;
                const float bias = kMask ? (ci[j] - ck[kt]) * kLog2e : nk[kt];
                float p = fast_exp2(__builtin_fmaf(x.s[t][kt][u], kscale, bias));
                if (kMask && kq > 32 * h + j) p = 0.f;
                const float dsv = p * x.dp[t][kt][u];
                csum[kt] += dsv;
                y.pb[kt][j] = (__bf16)p;
                y.db[kt][j] = (__bf16)dsv;
            }
        }
        return y;
    };
    // dV^T += dO^T P,  dK^T += Q^T dS over the half's 32 queries
    auto phase_c = [&](const OpC& rc, const PdS& y) __attribute__((always_inline)) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                dv[kt][dt] = mfma16(rc.ao[dt], y.pb[kt], dv[kt][dt]);
                dk[kt][dt] = mfma16(rc.aq[dt], y.db[kt], dk[kt][dt]);
            }
    };

    // The workgroup's K (and at d = 128 V) tiles; when only 64 keys are left, the
    // second block's waves hold none
    dma.issue(sm.k[0], K + (head + k0) * D, w);
    if (k0 + 64 < L) dma.issue(sm.k[1], K + (head + k0 + 64) * D, w);
    if constexpr (kVinLds) {
        dma.issue(sm.v[0], V + (head + k0) * D, w);
        if (k0 + 64 < L) dma.issue(sm.v[1], V + (head + k0 + 64) * D, w);
    }
    // tile m_lo in LDS and published; tile m_lo + 1 on its way
    put_rows(issue(m_lo, 0), 0);
    wait_vmcnt0();
    __syncthreads();
    float3 rnext = make_float3(0.f, 0.f, 0.f);
    if (m_lo < m_hi) rnext = issue(m_lo + 1, 1);
    int buf = 0;
    auto step = [&](auto mask_tag, int m) __attribute__((always_inline)) {
        const bool act = m >= nw && m <= w_hi;
        const int kq0 = 32 * (kg & 1) + r16 - 8 * g - (m == nw ? 0 : 4096);
        if (act) {
#pragma unroll
            for (int hh = 0; hh < 2 / QSPLIT; ++hh) {
                const int h = QSPLIT == 1 ? hh : qh;
                __builtin_amdgcn_sched_barrier(0);
                SdP x;
                {
                    const OpS rs = load_s(decltype(mask_tag)::value, buf, h);
                    phase_s(rs, x);
                }
                __builtin_amdgcn_sched_barrier(0);
                {
                    const OpD rd = load_d(buf, h);
                    phase_d(rd, x);
                }
                __builtin_amdgcn_sched_barrier(0);
                const PdS y = phase_b(mask_tag, x, buf, h, kq0);
                __builtin_amdgcn_sched_barrier(0);
                const OpC rc = load_c(buf, h);
                phase_c(rc, y);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (m < m_hi) put_rows(rnext, buf ^ 1);
        // tile m + 1 has landed and every wave's reads of tile m are complete
        wait_vmcnt0_lgkmcnt0();
        __syncthreads();
        const bool more = m + 1 < m_hi;
        if (more && tid < 64) {
            const size_t row = head + 64 * (m + 2) + tid;
            rnext = make_float3(cg[row], lse2[row], dsum[row]);
        }
        if (more) dma.issue(sm.q[buf], Q + (head + (size_t)64 * (m + 2)) * D, w);
        if (more) dma.issue(sm.o[buf], dO + (head + (size_t)64 * (m + 2)) * D, w);
        buf ^= 1;
    };
    // The first block's waves meet their diagonal tile at m_lo, the second
    // block's at m_lo + 1; those two tiles go through the masking variant.
    const int m_diag = min(m_lo + 1, m_hi);
    int m = m_lo;
    for (; m <= m_diag; ++m) step(std::true_type{}, m);
    for (; m <= m_hi; ++m) step(std::false_type{}, m);

    if constexpr (QSPLIT == 2) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            csum[kt] += __shfl_xor(csum[kt], 16);
            csum[kt] += __shfl_xor(csum[kt], 32);
        }
        // The second half's waves hand their partial sums to the first half's
        // through LDS, whose tiles are no longer read (the last step ended with
        // a barrier): dK in the Q and dO tiles, dV in the K and V tiles, lane-major
        // so that the 16-byte accesses do not conflict.
        static_assert(sizeof(sm.q) + sizeof(sm.o) >= 4 * 2 * NDT * 64 * sizeof(f32x4), "dK staging");
        static_assert(sizeof(sm.k) + sizeof(sm.v) >= 4 * 2 * NDT * 64 * sizeof(f32x4), "dV staging");
        f32x4* sdk = reinterpret_cast<f32x4*>(&sm.q[0][0]);
        f32x4* sdv = reinterpret_cast<f32x4*>(&sm.k[0][0]);
        if (qh == 1) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    const int e = ((kg * 2 + kt) * NDT + dt) * 64 + lane;
                    sdk[e] = dk[kt][dt];
                    sdv[e] = dv[kt][dt];
                }
                if (g == 0) sm.kc[32 * kg + 16 * kt + r16] = csum[kt];
            }
        }
        __syncthreads();
        if (qh == 1) return;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                const int e = ((kg * 2 + kt) * NDT + dt) * 64 + lane;
                dk[kt][dt] += sdk[e];
                dv[kt][dt] += sdv[e];
            }
            csum[kt] += sm.kc[32 * kg + 16 * kt + r16];
        }
    }
    if (!wave_on) return;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        const int key = wk0 + 16 * kt + r16;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const f32x4 a = dk[kt][dt] * qscale;
            const f32x4 b = dv[kt][dt];
            bf16x4 ab, bb;
            ab[0] = (__bf16)a[0]; ab[1] = (__bf16)a[1]; ab[2] = (__bf16)a[2]; ab[3] = (__bf16)a[3];
            bb[0] = (__bf16)b[0]; bb[1] = (__bf16)b[1]; bb[2] = (__bf16)b[2]; bb[3] = (__bf16)b[3];
            const size_t off = (head + key) * D + 16 * dt + 4 * g;
            *reinterpret_cast<bf16x4*>(dK + off) = ab;
            *reinterpret_cast<bf16x4*>(dV + off) = bb;
        }
        float c = csum[kt];
        if constexpr (QSPLIT == 1) {
            c += __shfl_xor(c, 16);
            c += __shfl_xor(c, 32);
        }
        if (g == 0) colsum[head + key] = c;
    }
}

// ---------------------------------------------------------------------------
hipError_t launch_dq_bf16(const BwdArgs& a, hipStream_t s) {
    const int BH = a.B * a.H, M = a.L / 64;
    const float kscale = kLog2e / sqrtf((float)a.d);
    const float qscale = 1.0f / sqrtf((float)a.d);
    const int nqb = (a.L + kBwdRows - 1) / kBwdRows;
    const int nblocks = BH * nqb;
    if (a.d == 64)
        hipLaunchKernelGGL(dq_bf16_kernel<64>, dim3(nblocks), dim3(kBwdThreads), 0, s,
                           (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                           (const __bf16*)a.O, (const __bf16*)a.dO, a.c, a.row_start, a.lse2,
                           a.dsum, (__bf16*)a.dQ, a.rowsum, a.sched_q, a.L, M, nqb, nblocks, kscale,
                           qscale);
    else
        hipLaunchKernelGGL(dq_bf16_kernel<128>, dim3(nblocks), dim3(kBwdThreads), 0, s,
                           (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                           (const __bf16*)a.O, (const __bf16*)a.dO, a.c, a.row_start, a.lse2,
                           a.dsum, (__bf16*)a.dQ, a.rowsum, a.sched_q, a.L, M, nqb, nblocks, kscale,
                           qscale);
    return hipGetLastError();
}

hipError_t launch_dkdv_bf16(const BwdArgs& a, hipStream_t s) {
    const int BH = a.B * a.H, M = a.L / 64;
    const float kscale = kLog2e / sqrtf((float)a.d);
    const float qscale = 1.0f / sqrtf((float)a.d);
    const int nkb = (a.L + kBwdRows - 1) / kBwdRows;
    const int nblocks = BH * nkb;
    if (a.d == 64)
        hipLaunchKernelGGL(dkdv_bf16_kernel<64>, dim3(nblocks), dim3(64 * DkvShape<64>::NW), 0, s,
                           (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                           (const __bf16*)a.dO, a.c, a.col_end, a.lse2, a.dsum,
                           (__bf16*)a.dK, (__bf16*)a.dV, a.colsum, a.sched_k, a.L, M, nkb,
                           nblocks, kscale, qscale);
    else
        hipLaunchKernelGGL(dkdv_bf16_kernel<128>, dim3(nblocks), dim3(64 * DkvShape<128>::NW), 0, s,
                           (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                           (const __bf16*)a.dO, a.c, a.col_end, a.lse2, a.dsum,
                           (__bf16*)a.dK, (__bf16*)a.dV, a.colsum, a.sched_k, a.L, M, nkb,
                           nblocks, kscale, qscale);
    return hipGetLastError();
}

}  // namespace acp
