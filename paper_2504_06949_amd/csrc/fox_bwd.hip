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
//   dsum_kernel   Delta from dO and the float32 copy of O kept by the forward
//   dq kernel     one workgroup per 128 queries, loops over kept key blocks:
//                 dQ, then Delta'_i = sum_j P_ij dP_ij (replacing Delta) and the
//                 row sums of dS
//   dkdv kernel   one workgroup per 128 keys, loops over the query blocks that
//                 keep them: dK, dV and the column sums of dS
//   dlogf_kernel  reverse cumulative sum of (row sum - column sum)
// dQ is produced by its own pass (recomputing S and dP) rather than by atomic
// accumulation from the key-block pass, so every output is written once.
#include "acp_device.h"
#include "acp_internal.h"

namespace acp {

constexpr int kBwdThreads = 256;
constexpr int kBwdRows = 128;

// ---------------------------------------------------------------------------
// Delta_i = sum_d dO_id O_id: 16 lanes per row.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void dsum_kernel(const T* __restrict__ dO,
                                                   const float* __restrict__ O32,
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
            acc = __builtin_fmaf(to_f32(dO[off]), O32[off], acc);
        }
    }
    acc += __shfl_xor(acc, 8);
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 1);
    if (row < rows && sub == 0) dsum[row] = acc;
}

// ---------------------------------------------------------------------------
// bf16 dQ pass.  Same decomposition as the forward: 4 waves x 32 queries, one
// pruning row per wave; S^T = K Q^T and dP^T = V dO^T are formed keys x
// queries so that dS^T lands in the B-operand layout of dQ^T = K^T dS^T.
// ---------------------------------------------------------------------------
template <int D>
struct alignas(16) DqSmem {
    static constexpr int LD = D + 8;
    alignas(16) __bf16 k[2][64 * LD];
    __bf16 v[2][64 * LD];
    float kb[2][64];   // key bias -(c_j - r) log2(e)
};

template <int D>
__global__ __launch_bounds__(kBwdThreads) void dq_bf16_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ cg,
    const int* __restrict__ row_start, const float* __restrict__ lse2,
    float* __restrict__ dsum, __bf16* __restrict__ dQ, float* __restrict__ rowsum,
    int L, int M, int nqb, int nblocks, float kscale, float qscale) {
    constexpr int LD = D + 8;
    constexpr int NDS = D / 32;
    constexpr int NDT = D / 16;
    constexpr int CPR = D / 8;
    constexpr int CH = 64 * CPR / kBwdThreads;
    __shared__ DqSmem<D> sm;

    const int lid = xcd_logical_id(blockIdx.x, nblocks);
    const int bh = lid / nqb;
    const int qb = nqb - 1 - (lid % nqb);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
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
    const float cref = cg[head + q0];   // frame of this workgroup

    bf16x8 qf[2][NDS], dof[2][NDS];
    float lq[2] = {0.f, 0.f}, dl[2] = {0.f, 0.f};
    if (wave_on) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            const size_t row = head + wq0 + 16 * qt + r16;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                qf[qt][ds] = *reinterpret_cast<const bf16x8*>(Q + row * D + 32 * ds + 8 * g);
                dof[qt][ds] = *reinterpret_cast<const bf16x8*>(dO + row * D + 32 * ds + 8 * g);
            }
            lq[qt] = (cg[row] - cref) * kLog2e - lse2[row];   // row term minus L_i
            dl[qt] = dsum[row];
        }
    }

    uint4 kreg[CH], vreg[CH];
    float4 nreg = make_float4(0.f, 0.f, 0.f, 0.f);
    auto gload = [&](int n) {
        const __bf16* kb = K + (head + (size_t)64 * n) * D;
        const __bf16* vb = V + (head + (size_t)64 * n) * D;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int i = tid + kBwdThreads * c;
            kreg[c] = *reinterpret_cast<const uint4*>(kb + i * 8);
            vreg[c] = *reinterpret_cast<const uint4*>(vb + i * 8);
        }
        if (tid < 16) nreg = *reinterpret_cast<const float4*>(cg + head + 64 * n + 4 * tid);
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int i = tid + kBwdThreads * c;
            const int row = i / CPR, ch = i % CPR;
            *reinterpret_cast<uint4*>(&sm.k[buf][row * LD + 8 * ch]) = kreg[c];
            *reinterpret_cast<uint4*>(&sm.v[buf][row * LD + 8 * ch]) = vreg[c];
        }
        if (tid < 16) {
            const float4 b = make_float4(-((nreg.x - cref) * kLog2e), -((nreg.y - cref) * kLog2e),
                                         -((nreg.z - cref) * kLog2e), -((nreg.w - cref) * kLog2e));
            *reinterpret_cast<float4*>(&sm.kb[buf][4 * tid]) = b;
        }
    };

    f32x4 acc[2][NDT];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float pdp[2] = {0.f, 0.f};   // sum_j P_ij dP_ij (lane partial)
    float psum[2] = {0.f, 0.f};  // sum_j P_ij (lane partial)

    gload(n_lo);
    sstore(0);
    int buf = 0;
    for (int n = n_lo; n <= n_hi; ++n) {
        __syncthreads();
        const bool more = n < n_hi;
        if (more) gload(n + 1);
        if (n >= w_lo && n <= mw) {
            const __bf16* ktile = sm.k[buf];
            const __bf16* vtile = sm.v[buf];
            const float* nc = sm.kb[buf];
            f32x4 s[4][2], dp[4][2];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const int krow = 32 * (kt >> 1) + 8 * (r16 >> 2) + 4 * (kt & 1) + (r16 & 3);
#pragma unroll
                for (int qt = 0; qt < 2; ++qt) {
                    s[kt][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
                    dp[kt][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(ktile + krow * LD + 32 * ds + 8 * g);
                    const bf16x8 b = *reinterpret_cast<const bf16x8*>(vtile + krow * LD + 32 * ds + 8 * g);
#pragma unroll
                    for (int qt = 0; qt < 2; ++qt) {
                        s[kt][qt] = mfma16(a, qf[qt][ds], s[kt][qt]);
                        dp[kt][qt] = mfma16(b, dof[qt][ds], dp[kt][qt]);
                    }
                }
            }
            float nk[2][8];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const float4 lo = *reinterpret_cast<const float4*>(nc + 32 * ks + 8 * g);
                const float4 hi = *reinterpret_cast<const float4*>(nc + 32 * ks + 8 * g + 4);
                nk[ks][0] = lo.x; nk[ks][1] = lo.y; nk[ks][2] = lo.z; nk[ks][3] = lo.w;
                nk[ks][4] = hi.x; nk[ks][5] = hi.y; nk[ks][6] = hi.z; nk[ks][7] = hi.w;
            }
            const bool diag = (n == mw);
            bf16x8 dsf[2][2];
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) {
                const int query = wq0 + 16 * qt + r16;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int kt = 2 * ks + (j >> 2), u = j & 3;
                        const float y = __builtin_fmaf(s[kt][qt][u], kscale, nk[ks][j]);
                        float p = fast_exp2(y + lq[qt]);
                        if (diag && (64 * n + 32 * ks + 8 * g + j) > query) p = 0.f;
                        const float dsv = p * (dp[kt][qt][u] - dl[qt]);
                        pdp[qt] = __builtin_fmaf(p, dp[kt][qt][u], pdp[qt]);
                        psum[qt] += p;
                        dsf[qt][ks][j] = (__bf16)dsv;
                    }
            }
            // dQ^T += K^T dS^T
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x8 a = lds_col8(ktile, LD, 32 * ks + 8 * g, 16 * dt, r16);
                    acc[0][dt] = mfma16(a, dsf[0][ks], acc[0][dt]);
                    acc[1][dt] = mfma16(a, dsf[1][ks], acc[1][dt]);
                }
        }
        if (more) sstore(buf ^ 1);
        buf ^= 1;
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
        // Delta'_i = sum_j P_ij dP_ij from the float32 P and dP of this pass: it is
        // what rowdot(dO, O) equals for the exact O, free of the rounding of P to
        // bfloat16 in the forward's PV product.  The dK/dV pass and both sums of
        // dS use it; rowsum(dS) is then Delta' (1 - sum_j P_ij).
        float a = pdp[qt], z = psum[qt];
        a += __shfl_xor(a, 16);
        a += __shfl_xor(a, 32);
        z += __shfl_xor(z, 16);
        z += __shfl_xor(z, 32);
        if (g == 0) {
            dsum[head + query] = a;
            rowsum[head + query] = a - a * z;
        }
    }
}

// ---------------------------------------------------------------------------
// bf16 dK/dV pass.  4 waves x 32 keys; wave w's keys lie in one pruning column,
// and the workgroup visits query blocks m = (first column) .. col_end[last
// column].  S = Q K^T and dP = dO V^T are formed queries x keys, so that P and
// dS land in the B-operand layout of dV^T = dO^T P and dK^T = Q^T dS.  The
// A-operand rows (queries) are read in the order
// qrow(qt, r) = 32 (qt / 2) + 8 (r / 4) + 4 (qt % 2) + r % 4.
// ---------------------------------------------------------------------------
template <int D>
struct alignas(16) DkvSmem {
    static constexpr int LD = D + 8;
    alignas(16) __bf16 q[2][64 * LD];
    __bf16 o[2][64 * LD];   // dO
    float lse2[2][64];   // row term minus L_i, (c_i - r) log2(e) - L_i
    float dsum[2][64];
};

template <int D>
__global__ __launch_bounds__(kBwdThreads) void dkdv_bf16_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ cg,
    const int* __restrict__ col_end, const float* __restrict__ lse2,
    const float* __restrict__ dsum, __bf16* __restrict__ dK, __bf16* __restrict__ dV,
    float* __restrict__ colsum, int L, int M, int nkb, int nblocks, float kscale,
    float qscale) {
    constexpr int LD = D + 8;
    constexpr int NDS = D / 32;
    constexpr int NDT = D / 16;
    constexpr int CPR = D / 8;
    constexpr int CH = 64 * CPR / kBwdThreads;
    __shared__ DkvSmem<D> sm;

    const int lid = xcd_logical_id(blockIdx.x, nblocks);
    const int bh = lid / nkb;
    const int kb = lid % nkb;                       // first key blocks have the most work
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int k0 = kb * kBwdRows;
    const int wk0 = k0 + 32 * w;
    const bool wave_on = wk0 < L;
    const int nw = wk0 / 64;
    const int n0 = k0 / 64;
    const size_t head = (size_t)bh * L;
    const int m_lo = n0;
    const int m_hi = col_end[(size_t)bh * M + min(n0 + 1, M - 1)];
    const int w_hi = wave_on ? col_end[(size_t)bh * M + nw] : -1;
    const float cref = cg[head + k0];   // frame of this workgroup

    bf16x8 kf[2][NDS], vf[2][NDS];
    float nk[2] = {0.f, 0.f};
    if (wave_on) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            const size_t row = head + wk0 + 16 * kt + r16;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) {
                kf[kt][ds] = *reinterpret_cast<const bf16x8*>(K + row * D + 32 * ds + 8 * g);
                vf[kt][ds] = *reinterpret_cast<const bf16x8*>(V + row * D + 32 * ds + 8 * g);
            }
            nk[kt] = -((cg[row] - cref) * kLog2e);
        }
    }

    uint4 qreg[CH], oreg[CH];
    float lreg = 0.f, dreg = 0.f;
    auto gload = [&](int m) {
        const __bf16* qb = Q + (head + (size_t)64 * m) * D;
        const __bf16* ob = dO + (head + (size_t)64 * m) * D;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int i = tid + kBwdThreads * c;
            qreg[c] = *reinterpret_cast<const uint4*>(qb + i * 8);
            oreg[c] = *reinterpret_cast<const uint4*>(ob + i * 8);
        }
        if (tid < 64) {
            lreg = (cg[head + 64 * m + tid] - cref) * kLog2e - lse2[head + 64 * m + tid];
            dreg = dsum[head + 64 * m + tid];
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int i = tid + kBwdThreads * c;
            const int row = i / CPR, ch = i % CPR;
            *reinterpret_cast<uint4*>(&sm.q[buf][row * LD + 8 * ch]) = qreg[c];
            *reinterpret_cast<uint4*>(&sm.o[buf][row * LD + 8 * ch]) = oreg[c];
        }
        if (tid < 64) {
            sm.lse2[buf][tid] = lreg;
            sm.dsum[buf][tid] = dreg;
        }
    };

    f32x4 dk[2][NDT], dv[2][NDT];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            dk[kt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
            dv[kt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    float csum[2] = {0.f, 0.f};

    gload(m_lo);
    sstore(0);
    int buf = 0;
    for (int m = m_lo; m <= m_hi; ++m) {
        __syncthreads();
        const bool more = m < m_hi;
        if (more) gload(m + 1);
        if (m >= nw && m <= w_hi) {
            const __bf16* qtile = sm.q[buf];
            const __bf16* otile = sm.o[buf];
            // S[qt][kt] = Q[qrow(qt)] K^T, dP[qt][kt] = dO[qrow(qt)] V^T
            f32x4 s[4][2], dp[4][2];
#pragma unroll
            for (int qt = 0; qt < 4; ++qt) {
                const int qrow = 32 * (qt >> 1) + 8 * (r16 >> 2) + 4 * (qt & 1) + (r16 & 3);
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    s[qt][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
                    dp[qt][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(qtile + qrow * LD + 32 * ds + 8 * g);
                    const bf16x8 b = *reinterpret_cast<const bf16x8*>(otile + qrow * LD + 32 * ds + 8 * g);
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt) {
                        s[qt][kt] = mfma16(a, kf[kt][ds], s[qt][kt]);
                        dp[qt][kt] = mfma16(b, vf[kt][ds], dp[qt][kt]);
                    }
                }
            }
            // the lane's queries: 32 ks + 8 g + j, j = 0..7 (j < 4 from tile 2ks)
            float l8[2][8], d8[2][8];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const float4 a0 = *reinterpret_cast<const float4*>(&sm.lse2[buf][32 * ks + 8 * g]);
                const float4 a1 = *reinterpret_cast<const float4*>(&sm.lse2[buf][32 * ks + 8 * g + 4]);
                const float4 b0 = *reinterpret_cast<const float4*>(&sm.dsum[buf][32 * ks + 8 * g]);
                const float4 b1 = *reinterpret_cast<const float4*>(&sm.dsum[buf][32 * ks + 8 * g + 4]);
                l8[ks][0] = a0.x; l8[ks][1] = a0.y; l8[ks][2] = a0.z; l8[ks][3] = a0.w;
                l8[ks][4] = a1.x; l8[ks][5] = a1.y; l8[ks][6] = a1.z; l8[ks][7] = a1.w;
                d8[ks][0] = b0.x; d8[ks][1] = b0.y; d8[ks][2] = b0.z; d8[ks][3] = b0.w;
                d8[ks][4] = b1.x; d8[ks][5] = b1.y; d8[ks][6] = b1.z; d8[ks][7] = b1.w;
            }
            const bool diag = (m == nw);
            bf16x8 pb[2][2], db[2][2];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                const int key = wk0 + 16 * kt + r16;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int qt = 2 * ks + (j >> 2), u = j & 3;
                        const float y = __builtin_fmaf(s[qt][kt][u], kscale, nk[kt]);
                        float p = fast_exp2(y + l8[ks][j]);
                        if (diag && key > (64 * m + 32 * ks + 8 * g + j)) p = 0.f;
                        const float dsv = p * (dp[qt][kt][u] - d8[ks][j]);
                        csum[kt] += dsv;
                        pb[kt][ks][j] = (__bf16)p;
                        db[kt][ks][j] = (__bf16)dsv;
                    }
            }
            // dV^T += dO^T P,  dK^T += Q^T dS
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x8 ao = lds_col8(otile, LD, 32 * ks + 8 * g, 16 * dt, r16);
                    const bf16x8 aq = lds_col8(qtile, LD, 32 * ks + 8 * g, 16 * dt, r16);
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt) {
                        dv[kt][dt] = mfma16(ao, pb[kt][ks], dv[kt][dt]);
                        dk[kt][dt] = mfma16(aq, db[kt][ks], dk[kt][dt]);
                    }
                }
        }
        if (more) sstore(buf ^ 1);
        buf ^= 1;
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
        c += __shfl_xor(c, 16);
        c += __shfl_xor(c, 32);
        if (g == 0) colsum[head + key] = c;
    }
}

// ---------------------------------------------------------------------------
// fp32 path (plain VALU): dQ/rowsum with one thread per query, dK/dV/colsum
// with one thread per key, tiles staged in LDS.
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
    __shared__ float nc[64];
    const int bh = blockIdx.x / M, m = blockIdx.x % M, t = threadIdx.x;
    const size_t head = (size_t)bh * L;
    const size_t row = head + 64 * m + t;
    float q[D], go[D], acc[D];
#pragma unroll
    for (int k = 0; k < D; ++k) { q[k] = Q[row * D + k]; go[k] = dO[row * D + k]; acc[k] = 0.f; }
    const float cref = cg[head + 64 * m];
    const float l2 = (cg[row] - cref) * kLog2e - lse2[row], dl = dsum[row];
    float pdp = 0.f, psum = 0.f;
    for (int n = row_start[(size_t)bh * M + m]; n <= m; ++n) {
        __syncthreads();
        for (int i = t; i < 64 * D; i += 64) {
            ks[i] = K[(head + 64 * n) * D + i];
            vs[i] = V[(head + 64 * n) * D + i];
        }
        nc[t] = -((cg[head + 64 * n + t] - cref) * kLog2e);
        __syncthreads();
        const int jmax = (n == m) ? t : 63;
        for (int j = 0; j <= jmax; ++j) {
            float s = 0.f, dp = 0.f;
#pragma unroll
            for (int k = 0; k < D; ++k) {
                s = __builtin_fmaf(q[k], ks[j * D + k], s);
                dp = __builtin_fmaf(go[k], vs[j * D + k], dp);
            }
            const float p = fast_exp2(__builtin_fmaf(s, kscale, nc[j]) + l2);
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
    __shared__ float ls[64];
    __shared__ float dls[64];
    const int bh = blockIdx.x / M, n = blockIdx.x % M, t = threadIdx.x;
    const size_t head = (size_t)bh * L;
    const size_t row = head + 64 * n + t;
    float kk[D], vv[D], gk[D], gv[D];
#pragma unroll
    for (int k = 0; k < D; ++k) { kk[k] = K[row * D + k]; vv[k] = V[row * D + k]; gk[k] = 0.f; gv[k] = 0.f; }
    const float cref = cg[head + 64 * n];
    const float nk = -((cg[row] - cref) * kLog2e);
    float cs = 0.f;
    const int mend = col_end[(size_t)bh * M + n];
    for (int m = n; m <= mend; ++m) {
        __syncthreads();
        for (int i = t; i < 64 * D; i += 64) {
            qs[i] = Q[(head + 64 * m) * D + i];
            os[i] = dO[(head + 64 * m) * D + i];
        }
        ls[t] = (cg[head + 64 * m + t] - cref) * kLog2e - lse2[head + 64 * m + t];
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
            const float p = fast_exp2(__builtin_fmaf(s, kscale, nk) + ls[i]);
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
// dlog f_l = sum_{i >= l} (rowsum_i - colsum_i), accumulated in float64.
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void dlogf_kernel(const float* __restrict__ rowsum,
                                                             const float* __restrict__ colsum,
                                                             float* __restrict__ dlog_f, int L) {
    __shared__ double s_wave[kScanThreads / 64];
    const int bh = blockIdx.x, t = threadIdx.x, lane = t & 63, wid = t >> 6;
    const size_t head = (size_t)bh * L;
    const int per = (L + kScanThreads - 1) / kScanThreads;
    const int beg = min(t * per, L), end = min(beg + per, L);
    double local = 0.0;
    for (int i = beg; i < end; ++i) local += (double)rowsum[head + i] - (double)colsum[head + i];
    // exclusive suffix sum over threads: scan with the thread order reversed
    const int rt = kScanThreads - 1 - t;  // reversed position
    // place the value of thread t at position rt and scan positions ascending
    // (done through LDS so that each wave scans contiguous positions)
    __shared__ double s_val[kScanThreads];
    s_val[rt] = local;
    __syncthreads();
    double v = s_val[t];  // value at position t
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const double o = __shfl_up(v, off);
        if (lane >= off) v += o;
    }
    if (lane == 63) s_wave[wid] = v;
    __syncthreads();
    if (wid == 0) {
        double x = lane < kScanThreads / 64 ? s_wave[lane] : 0.0;
#pragma unroll
        for (int off = 1; off < kScanThreads / 64; off <<= 1) {
            const double o = __shfl_up(x, off);
            if (lane >= off) x += o;
        }
        if (lane < kScanThreads / 64) s_wave[lane] = x;
    }
    __syncthreads();
    const double incl = v + (wid > 0 ? s_wave[wid - 1] : 0.0);  // inclusive at position t
    __syncthreads();
    s_val[t] = incl;
    __syncthreads();
    // thread t: sum over positions < rt, i.e. over threads > t
    double run = rt > 0 ? s_val[rt - 1] : 0.0;
    for (int i = end - 1; i >= beg; --i) {
        run += (double)rowsum[head + i] - (double)colsum[head + i];
        dlog_f[head + i] = (float)run;
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
    trace_begin(ACP_K_DSUM, s);
    if (a.bf16) {
        if (a.d == 64)
            hipLaunchKernelGGL((dsum_kernel<__bf16, 64>), dim3(dgrid), dim3(256), 0, s,
                               (const __bf16*)a.dO, a.O32, a.dsum, rows);
        else
            hipLaunchKernelGGL((dsum_kernel<__bf16, 128>), dim3(dgrid), dim3(256), 0, s,
                               (const __bf16*)a.dO, a.O32, a.dsum, rows);
    } else {
        if (a.d == 64)
            hipLaunchKernelGGL((dsum_kernel<float, 64>), dim3(dgrid), dim3(256), 0, s,
                               (const float*)a.dO, a.O32, a.dsum, rows);
        else
            hipLaunchKernelGGL((dsum_kernel<float, 128>), dim3(dgrid), dim3(256), 0, s,
                               (const float*)a.dO, a.O32, a.dsum, rows);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    trace_end(ACP_K_DSUM, s);

    const int nqb = (a.L + kBwdRows - 1) / kBwdRows;
    const int nblocks = BH * nqb;
    trace_begin(ACP_K_DQ, s);
    if (a.bf16) {
#define ACP_DQ(DD)                                                                         \
    hipLaunchKernelGGL(dq_bf16_kernel<DD>, dim3(nblocks), dim3(kBwdThreads), 0, s,         \
                       (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,         \
                       (const __bf16*)a.dO, a.c, a.row_start, a.lse2, a.dsum,            \
                       (__bf16*)a.dQ, a.rowsum, a.L, M, nqb, nblocks, kscale, qscale)
        if (a.d == 64) { ACP_DQ(64); } else { ACP_DQ(128); }
#undef ACP_DQ
    } else {
#define ACP_DQ32(DD)                                                                       \
    hipLaunchKernelGGL(dq_f32_kernel<DD>, dim3(BH * M), dim3(64), 0, s,                    \
                       (const float*)a.Q, (const float*)a.K, (const float*)a.V,            \
                       (const float*)a.dO, a.c, a.row_start, a.lse2, a.dsum,             \
                       (float*)a.dQ, a.rowsum, a.L, M, kscale, qscale)
        if (a.d == 64) { ACP_DQ32(64); } else { ACP_DQ32(128); }
#undef ACP_DQ32
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    trace_end(ACP_K_DQ, s);

    trace_begin(ACP_K_DKDV, s);
    if (a.bf16) {
#define ACP_DKV(DD)                                                                        \
    hipLaunchKernelGGL(dkdv_bf16_kernel<DD>, dim3(nblocks), dim3(kBwdThreads), 0, s,       \
                       (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,         \
                       (const __bf16*)a.dO, a.c, a.col_end, a.lse2, a.dsum,              \
                       (__bf16*)a.dK, (__bf16*)a.dV, a.colsum, a.L, M, nqb, nblocks,       \
                       kscale, qscale)
        if (a.d == 64) { ACP_DKV(64); } else { ACP_DKV(128); }
#undef ACP_DKV
    } else {
#define ACP_DKV32(DD)                                                                      \
    hipLaunchKernelGGL(dkdv_f32_kernel<DD>, dim3(BH * M), dim3(64), 0, s,                  \
                       (const float*)a.Q, (const float*)a.K, (const float*)a.V,            \
                       (const float*)a.dO, a.c, a.col_end, a.lse2, a.dsum,               \
                       (float*)a.dK, (float*)a.dV, a.colsum, a.L, M, kscale, qscale)
        if (a.d == 64) { ACP_DKV32(64); } else { ACP_DKV32(128); }
#undef ACP_DKV32
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    trace_end(ACP_K_DKDV, s);

    trace_begin(ACP_K_DLOGF, s);
    hipLaunchKernelGGL(dlogf_kernel, dim3(BH), dim3(kScanThreads), 0, s, a.rowsum, a.colsum,
                       a.dlog_f, a.L);
    e = hipGetLastError();
    trace_end(ACP_K_DLOGF, s);
    return e;
}

}  // namespace acp
