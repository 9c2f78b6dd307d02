// Forget-gate producer with the cumulative gates in its epilogue (Sec. 2: each
// head's gate is f_t = sigmoid(w_f^T x_t + b_f) of the layer input, and the
// FlashAttention form of Forgetting Attention needs c = cumsum(log f); Sec. 3,
// "Two-stage implementation": stage 1 then only has to read c).
//
// gate_kernel: one workgroup per (sequence b, 64-token block), one wave per
// group of 4 heads (several groups per wave when H > 16).
//   * Gate logits a = w_f^T x + b_f: each lane owns one token and sums its
//     heads' dot products in float32 in ascending feature order (a product of
//     two bfloat16 values is exact in float32, so every step rounds once), the
//     bias added last.  Token rows and weights (a float32 copy made by the
//     set-up kernel) stream through LDS.  log f = -softplus(-a) in float64, rounded once.
//   * c: a scan of the block's 64 gates per head (float64 while they span under
//     53 bits, else double-double), then a double-double chained scan across
//     the blocks of the sequence (decoupled look-back): each wave
//     first publishes its block total, then walks back over earlier blocks,
//     adding their totals until it meets one whose inclusive prefix is
//     published, and publishes its own.  The whole wave walks: 64 earlier
//     blocks per round.  Whenever the partial sums span at most 105 bits every
//     double-double sum here is exact, so c, the float32 rounding of the pair,
//     is that of the exact prefix sum whatever the association (the span is
//     checked from the statistics below, as stage 1 does).
//   * Per-block statistics for stage 1's checks: the sum of |log f| (a pair),
//     the smallest float32 ulp exponent, and flags (a non-finite gate, a
//     time-out below), written by each block to a slot of its own (stage 1
//     reduces them; same-address atomics from every block of a sequence would
//     serialise).
// A descriptor is a pair of words holding the raw float64 bits of hi and lo; a
// signalling-NaN pattern that no arithmetic produces marks a word "not
// published yet" (gate_init_kernel sets it before every call).  Each word is
// published by an agent-scope 64-bit store and read by an agent-scope load, and
// a reader takes a descriptor only once both words are published, so no fence
// is needed (the values are the message).  Blocks of one sequence wait
// only on blocks with lower workgroup ids, which were dispatched before them;
// the wait is bounded all the same, and on a time-out the wave sets flag bit 5
// and goes on, so every wave ends.
#include "acp_device.h"
#include "acp_internal.h"
#include "acp_scan.h"

namespace acp {

constexpr unsigned long long kUnpublished = 0x7FF4ACB0DEAD0001ull;   // a signalling NaN
constexpr int kGateSpinLimit = 1 << 22;

__device__ __forceinline__ float bf16_bits_to_f32(unsigned short b) {
    return __uint_as_float((unsigned)b << 16);
}

// Set-up before every call: descriptor words unpublished, and the weights as float32 in [group of 4 heads][feature][4] order (heads past H
// zero), so that the producer reads a group's four weights of a feature as one
// uniform 16-byte load.
__global__ __launch_bounds__(256) void gate_init_kernel(unsigned long long* __restrict__ agg,
                                                        unsigned long long* __restrict__ incl,
                                                        int nwords,
                                                        const unsigned short* __restrict__ W,
                                                        float4* __restrict__ wq, int Dm, int H,
                                                        int nquad) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < nquad * Dm) {
        const int quad = i / Dm, k = i % Dm, h0 = 4 * quad;
        const unsigned short* wr = W + (size_t)k * H + h0;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        v.x = bf16_bits_to_f32(wr[0]);
        if (h0 + 1 < H) v.y = bf16_bits_to_f32(wr[1]);
        if (h0 + 2 < H) v.z = bf16_bits_to_f32(wr[2]);
        if (h0 + 3 < H) v.w = bf16_bits_to_f32(wr[3]);
        wq[i] = v;
    }
    if (i < nwords) {
        agg[i] = kUnpublished;
        incl[i] = kUnpublished;
    }

}

__device__ __forceinline__ void publish(unsigned long long* w, DD v) {
    __hip_atomic_store(w, (unsigned long long)__double_as_longlong(v.hi), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(w + 1, (unsigned long long)__double_as_longlong(v.lo), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long peek(const unsigned long long* w) {
    return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double bits_f64(unsigned long long b) {
    return __longlong_as_double((long long)b);
}

// A workgroup of 4 waves takes one (sequence b, 64-token block) for every head:
// wave w computes the groups of 4 heads w, w + 4, ...  The block's token rows
// and the groups' weights stream through LDS 64 features at a time
// (double-buffered, each tile loaded once, coalesced, by the whole workgroup);
// each lane reads its token's features from its LDS row.  The tile's next
// global loads are held in named registers (an indexed array of them was
// placed in scratch memory, whose stores waited for the loads).
constexpr int kGateThreads = 256;
constexpr int kGateTile = 64;          // features per tile (d_model % 64 == 0)
constexpr int kGateRow = 72;           // bf16 per LDS row (rows padded to 144 bytes)
constexpr int kGateMaxQuad = 16;       // H <= 64

__global__ __launch_bounds__(kGateThreads) void gate_kernel(
    const __bf16* __restrict__ X, const float4* __restrict__ wq,
    const float* __restrict__ bias, int L, int Dm, int H, int nblk, int nquad,
    float* __restrict__ log_f, float* __restrict__ c, unsigned long long* __restrict__ agg,
    unsigned long long* __restrict__ incl, GateStats* __restrict__ st) {
    extern __shared__ __attribute__((aligned(16))) unsigned char gsm[];
    __bf16* xt = reinterpret_cast<__bf16*>(gsm);                           // [2][64][kGateRow]
    float4* wt = reinterpret_cast<float4*>(gsm + 2 * 64 * kGateRow * 2);  // [2][nquad][64]
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int blk = blockIdx.x % nblk, b = blockIdx.x / nblk;
    const int tok = 64 * blk + lane;
    const int ntile = Dm / kGateTile;
    const __bf16* xsrc = X + ((size_t)b * L + 64 * blk) * Dm;   // the block's 64 rows

    // tile t: 512 pieces of 16 bytes of X (row p / 8, part p % 8) and nquad * 64
    // float4 of weights; thread tid takes pieces tid, tid + 256, ...
    const int nw4 = nquad * kGateTile;
    uint4 xr0, xr1;
    float4 wr0, wr1, wr2, wr3;
    auto fetch = [&](int t) __attribute__((always_inline)) {
        const int p0 = tid, p1 = tid + kGateThreads;
        xr0 = *reinterpret_cast<const uint4*>(xsrc + (size_t)(p0 >> 3) * Dm + kGateTile * t + 8 * (p0 & 7));
        xr1 = *reinterpret_cast<const uint4*>(xsrc + (size_t)(p1 >> 3) * Dm + kGateTile * t + 8 * (p1 & 7));
        auto wload = [&](int p) __attribute__((always_inline)) {
            return p < nw4 ? wq[(size_t)(p / kGateTile) * Dm + kGateTile * t + p % kGateTile]
                           : make_float4(0.f, 0.f, 0.f, 0.f);
        };
        wr0 = wload(tid);
        wr1 = wload(tid + kGateThreads);
        wr2 = wload(tid + 2 * kGateThreads);
        wr3 = wload(tid + 3 * kGateThreads);
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
        const int p0 = tid, p1 = tid + kGateThreads;
        *reinterpret_cast<uint4*>(xt + (buf * 64 + (p0 >> 3)) * kGateRow + 8 * (p0 & 7)) = xr0;
        *reinterpret_cast<uint4*>(xt + (buf * 64 + (p1 >> 3)) * kGateRow + 8 * (p1 & 7)) = xr1;
        if (tid < nw4) wt[buf * nw4 + tid] = wr0;
        if (tid + kGateThreads < nw4) wt[buf * nw4 + tid + kGateThreads] = wr1;
        if (tid + 2 * kGateThreads < nw4) wt[buf * nw4 + tid + 2 * kGateThreads] = wr2;
        if (tid + 3 * kGateThreads < nw4) wt[buf * nw4 + tid + 3 * kGateThreads] = wr3;
    };

    // ---- logits: float32, ascending feature order -----------------------------
    float acc[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[r][j] = 0.f;
    fetch(0);
    stash(0);
    __syncthreads();
    // Each group's 64 features of a tile are taken in steps of 8, the LDS reads
    // of step g + 1 (the lane's 8 features, the group's 8 weight vectors) issued
    // before the 32 FMAs of step g, so that their latency is covered.
    for (int t = 0; t < ntile; ++t) {
        const int buf = t & 1;
        if (t + 1 < ntile) fetch(t + 1);
        const __bf16* xrow = xt + (buf * 64 + lane) * kGateRow;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int q = w + 4 * r;
            if (q >= nquad) break;
            const float4* wq_t = wt + buf * nw4 + q * kGateTile;
            bf16x8 xa = *reinterpret_cast<const bf16x8*>(xrow);
            float4 wa[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) wa[e] = wq_t[e];
#pragma unroll
            for (int g = 0; g < kGateTile / 8; ++g) {
                bf16x8 xb;
                float4 wb[8];
                if (g + 1 < kGateTile / 8) {
                    xb = *reinterpret_cast<const bf16x8*>(xrow + 8 * (g + 1));
#pragma unroll
                    for (int e = 0; e < 8; ++e) wb[e] = wq_t[8 * (g + 1) + e];
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float xe = (float)xa[e];
                    acc[r][0] = __builtin_fmaf(xe, wa[e].x, acc[r][0]);
                    acc[r][1] = __builtin_fmaf(xe, wa[e].y, acc[r][1]);
                    acc[r][2] = __builtin_fmaf(xe, wa[e].z, acc[r][2]);
                    acc[r][3] = __builtin_fmaf(xe, wa[e].w, acc[r][3]);
                }
                __builtin_amdgcn_sched_barrier(0);
                if (g + 1 < kGateTile / 8) {
                    xa = xb;
#pragma unroll
                    for (int e = 0; e < 8; ++e) wa[e] = wb[e];
                }
            }
        }
        if (t + 1 < ntile) stash(buf ^ 1);
        __syncthreads();
    }

    // ---- per group of heads: log f, statistics, the block scan, the chained
    // prefix, c ---------------------------------------------------------------------
#pragma unroll 1
    for (int r = 0; r < 4; ++r) {
        const int q = w + 4 * r;
        if (q >= nquad) break;
        const int h0 = 4 * q, nh = min(4, H - h0);
        float a4[4];   // this group's logits (selected, not indexed, from acc)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            a4[j] = r == 0 ? acc[0][j] : r == 1 ? acc[1][j] : r == 2 ? acc[2][j] : acc[3][j];
        DD excl_mine{0.0, 0.0};   // lane j < nh: exclusive prefix of head h0 + j
        DD abs_mine{0.0, 0.0};    // lane j < nh: the block's statistics of head h0 + j
        int lsb_mine = 1 << 30, flags_mine = 0;
        DD scan[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            scan[j] = DD{0.0, 0.0};
            if (j >= nh) continue;
            const double a = (double)(a4[j] + bias[h0 + j]);
            const double sp = fmax(-a, 0.0) + log1p(exp(-fabs(a)));   // softplus(-a)
            const float lf32 = (float)(-sp);
            const size_t bh = (size_t)b * H + h0 + j;
            log_f[bh * L + tok] = lf32;
            // statistics for stage 1's checks, and the block's scan: in float64
            // while the block's own 64 gates span under 53 bits (then every float64
            // sum is exact; the read is stage 1's), else in double-double
            const bool bad = !__builtin_isfinite(lf32);
            const double gv = bad ? 0.0 : (double)lf32;
            const int lsb = bad || lf32 == 0.f ? (1 << 30) : lsb_exp(lf32);
            double sabs_f = __builtin_fabs(gv);
            int slsb = lsb;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                sabs_f += __shfl_xor(sabs_f, off);
                slsb = min(slsb, __shfl_xor(slsb, off));
            }
            const int biased = (int)((__double_as_longlong(sabs_f) >> 52) & 0x7ff);
            const bool bwide = __builtin_amdgcn_readfirstlane(
                sabs_f > 0.0 && (biased > 0 ? biased : 1) - 1023 + 1 - slsb >= 53);
            DD sabs{sabs_f, 0.0};
            if (bwide) {
                sabs = wave_sum_dd(DD{__builtin_fabs(gv), 0.0});
                scan[j] = wave_inclusive_scan_dd(DD{gv, 0.0});
            } else {
                scan[j] = DD{wave_inclusive_scan_f64(gv), 0.0};
            }
            const bool anybad = __ballot(bad) != 0ull;
            if (lane == j) {
                abs_mine = sabs;
                lsb_mine = slsb;
                flags_mine = anybad ? 2 : 0;
            }
        }
        // block totals (lane j holds head h0 + j's), published before the look-back
        DD total{0.0, 0.0};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const DD tj = readlane_dd(scan[j], 63);
            if (lane == j) total = tj;
        }
        if (lane < nh) {
            const size_t d = ((size_t)b * H + h0 + lane) * nblk + blk;
            publish((blk == 0 ? incl : agg) + 2 * d, total);
        }
        // Look-back, one head at a time with the whole wave: lane l reads block
        // i0 - l's descriptors, 64 blocks per round.  The nearest block with its
        // inclusive prefix published ends the walk if every block after it has
        // its total published; otherwise the round is read again.  A round with
        // no prefix but all 64 totals adds them and moves 64 blocks back.
        for (int j = 0; j < nh; ++j) {
            if (blk == 0) break;
            const size_t d0 = ((size_t)b * H + h0 + j) * nblk;
            DD run{0.0, 0.0};
            int i0 = blk - 1, spins = 0;
            bool timed_out = false;
            while (i0 >= 0) {
                const int i = i0 - lane;
                unsigned long long p = kUnpublished, pl = kUnpublished;
                unsigned long long qq = kUnpublished, ql = kUnpublished;
                if (i >= 0) {
                    const size_t w2 = 2 * (d0 + i);
                    p = peek(&incl[w2]);
                    pl = peek(&incl[w2 + 1]);
                    qq = peek(&agg[w2]);
                    ql = peek(&agg[w2 + 1]);
                }
                // lanes whose block lies before the sequence count as published zeros
                const bool has_p = i >= 0 && p != kUnpublished && pl != kUnpublished;
                const bool has_q = i < 0 || (qq != kUnpublished && ql != kUnpublished) || has_p;
                const unsigned long long pm = __ballot(has_p);
                const int stop = pm ? __builtin_ctzll(pm) : 64;      // nearest prefix
                const unsigned long long need = stop == 64 ? ~0ull : ((1ull << stop) - 1ull);
                const unsigned long long qm = __ballot(has_q);
                if ((qm & need) == need) {
                    if (stop == 0) {   // the previous block's prefix alone: no reduction
                        run = dd_add(run, DD{readlane_f64(bits_f64(p), 0), readlane_f64(bits_f64(pl), 0)});
                        break;
                    }
                    DD v{0.0, 0.0};
                    if (lane < stop && i >= 0) v = DD{bits_f64(qq), bits_f64(ql)};
                    if (lane == stop) v = DD{bits_f64(p), bits_f64(pl)};
                    double sum;
                    run = dd_add(run, wave_sum_f64_if_exact(v, sum) ? DD{sum, 0.0} : wave_sum_dd(v));
                    if (stop < 64) break;
                    i0 -= 64;
                    spins = 0;
                    continue;
                }
                if (++spins > kGateSpinLimit) {
                    timed_out = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            if (lane == j) {
                excl_mine = run;
                if (timed_out) flags_mine |= 32;
                publish(&incl[2 * (d0 + blk)], dd_add(run, total));
            }
        }
        if (lane < nh) {
            GateStats g;
            g.abs_sum = abs_mine.hi;
            g.abs_lo = abs_mine.lo;
            g.min_lsb = lsb_mine;
            g.flags = flags_mine;
            st[((size_t)b * H + h0 + lane) * nblk + blk] = g;
        }
        // c of the block: exclusive prefix + the in-block inclusive scan
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (j >= nh) continue;
            const DD ex = readlane_dd(excl_mine, j);
            c[((size_t)b * H + h0 + j) * L + tok] = dd_to_f32(dd_add(ex, scan[j]));
        }
    }
}

hipError_t launch_gate(const GateArgs& a, hipStream_t s) {
    const int nblk = a.L / 64, nquad = (a.H + 3) / 4;
    const int ndesc = a.B * a.H * nblk;
    trace_begin(ACP_K_GATE, s);
    const int ninit = max(2 * ndesc, nquad * a.Dm);
    hipLaunchKernelGGL(gate_init_kernel, dim3((ninit + 255) / 256), dim3(256), 0, s,
                       a.agg, a.incl, 2 * ndesc, (const unsigned short*)a.W,
                       (float4*)a.wq, a.Dm, a.H, nquad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t lds = (size_t)2 * 64 * kGateRow * 2 + (size_t)2 * nquad * kGateTile * 16;
    hipLaunchKernelGGL(gate_kernel, dim3(a.B * nblk), dim3(kGateThreads), lds, s,
                       (const __bf16*)a.X, (const float4*)a.wq, a.bias, a.L, a.Dm, a.H,
                       nblk, nquad, a.log_f, a.c, a.agg, a.incl, a.stats);
    e = hipGetLastError();
    trace_end(ACP_K_GATE, s);
    return e;
}

}  // namespace acp
