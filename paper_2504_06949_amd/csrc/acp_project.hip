// Q and K projections with the row-norm maxima of stage 1 in their epilogue
// (the fusion of the bound's norm pass into the upstream producer that the
// paper's two-stage design allows: U needs only the largest row norms of the
// stored Q and K, Sec. 3).
//
//   [Q | K] = X [Wq | Wk]     X [B*L, Dm], Wq and Wk [Dm, H*d] (row-major, bf16)
//
// One workgroup of 256 threads computes a 128 x 128 tile of the product with
// bf16 MFMA (float32 accumulation), K-blocks of 64 staged through LDS by DMA and
// double-buffered.  Its epilogue rounds the tile to bfloat16, writes every row
// straight into the head-split [B, H, L, d] layout, and forms, per head in the
// tile, the largest float64 sum of squares of the stored row (ascending feature
// order), which is the 128-row chunk maximum that rownorm_max_kernel would
// produce for the same Q and K.
#include "acp_device.h"
#include "acp_internal.h"

namespace acp {

constexpr int kPrjTile = 128;   // rows (M) and columns (N) of a workgroup tile
constexpr int kPrjK = 64;       // depth of one K-block

// DMA of a 64 x 64*P bf16 block of a row-major matrix with row stride ld
// (elements) into an LDS tile laid out as tile_off describes (P column panels).
// Instruction i of the 8 P per block fills LDS bytes [1024 i, 1024 i + 1024).
template <int P, int NWAVES>
struct StridedDma {
    static constexpr int kInst = 8 * P;
    static constexpr int kPer = kInst / NWAVES;
    unsigned off[kPer];
    __device__ __forceinline__ void init(int wave, int lane, int ld) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = wave + NWAVES * k;
            const int row = 8 * (i & 7) + (lane >> 3);
            const int chunk = (lane & 7) ^ tile_swz(row);
            off[k] = (unsigned)(2 * (row * ld + ((i >> 3) << 6) + 8 * chunk));
        }
    }
    __device__ __forceinline__ void issue(unsigned char* tile, const __bf16* src, int wave) const {
        typedef __attribute__((address_space(3))) unsigned char lds_u8;
        const unsigned long long p = reinterpret_cast<unsigned long long>(src);
        const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)p);
        const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(p >> 32));
        const unsigned long long base = ((unsigned long long)hi << 32) | lo;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = wave + NWAVES * k;
            const unsigned lds = __builtin_amdgcn_readfirstlane(
                (unsigned)(unsigned long long)(const lds_u8*)(tile + 1024 * i));
            // One wait state between the SALU write of M0 and the LDS DMA that
            // reads it (a gfx9-family hazard that the compiler's hazard check
            // cannot see inside this statement).  Nothing in these kernels keeps
            // a value in M0 across it (DS instructions do not read M0 on gfx9 and
            // later), so the clobber costs nothing.
            asm volatile(
                "s_mov_b32 m0, %0\n\t"
                "s_nop 0\n\t"
                "global_load_lds_dwordx4 %1, %2"
                :
                : "s"(lds), "v"(off[k]), "s"(base)
                : "memory", "m0");
        }
    }
};

struct PrjSmem {
    union {
        struct {
            unsigned char a[2][2][64 * 128];   // X: two 64-row halves of 64 columns
            unsigned char b[2][64 * 256];      // W: 64 rows x 128 columns (two panels)
        } in;
        __bf16 out[kPrjTile][kPrjTile + 8];   // the rounded tile, padded rows
    };
    double rmax[2][4];
};

template <int D>
__global__ __launch_bounds__(256) void qk_project_kernel(
    const __bf16* __restrict__ X, const __bf16* __restrict__ Wq, const __bf16* __restrict__ Wk,
    int L, int Dm, int H, __bf16* __restrict__ Qo, __bf16* __restrict__ Ko,
    double* __restrict__ part, int nchunk) {
    __shared__ PrjSmem sm;
    const int HD = H * D;
    // All column tiles of a 128-row block of X run on one XCD (a contiguous range
    // of logical ids per XCD), so that the block is fetched into one L2 only.
    const int ntn = 2 * H * D / kPrjTile;
    const int lid = xcd_logical_id(blockIdx.x, gridDim.x);
    const int tn = lid % ntn, tm = lid / ntn;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w >> 1, wn = w & 1;            // the wave's 64 x 64 quarter
    const int g = lane >> 4, r16 = lane & 15;
    const int m0 = tm * kPrjTile;
    const int n0 = tn * kPrjTile;                 // column of [Q | K]
    const int which = n0 / HD;                    // 0: Q, 1: K (a tile never straddles)
    const __bf16* W = which == 0 ? Wq : Wk;
    const int nw0 = n0 - which * HD;              // column inside Wq or Wk

    StridedDma<1, 4> dma_a;
    StridedDma<2, 4> dma_b;
    dma_a.init(w, lane, Dm);
    dma_b.init(w, lane, HD);
    auto issue = [&](int kb, int buf) __attribute__((always_inline)) {
        const int k0 = kb * kPrjK;
        dma_a.issue(sm.in.a[buf][0], X + (size_t)m0 * Dm + k0, w);
        dma_a.issue(sm.in.a[buf][1], X + (size_t)(m0 + 64) * Dm + k0, w);
        dma_b.issue(sm.in.b[buf], W + (size_t)k0 * HD + nw0, w);
    };

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // The product is formed transposed, C^T = W^T X^T (W columns as the A operand,
    // X rows as the B operand), so that each lane ends with four consecutive
    // columns of one row of C: lane (g, r) holds C[16 i + r][16 j + 4 g + u].
    // (Spreading the next K-block's DMA over this block's MFMAs measured slower.)
    const int nkb = Dm / kPrjK;
    issue(0, 0);
    for (int kb = 0; kb < nkb; ++kb) {
        const int buf = kb & 1;
        wait_vmcnt0();
        __syncthreads();                          // block kb landed; block kb - 1 read
        const bool more = kb + 1 < nkb;
        if (more) issue(kb + 1, buf ^ 1);
        const unsigned char* at = sm.in.a[buf][wm];
        const unsigned char* bt = sm.in.b[buf];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            bf16x8 af[4], bfr[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) af[i] = tile_row8(at, 16 * i + r16, 32 * ks + 8 * g);
#pragma unroll
            for (int j = 0; j < 4; ++j) bfr[j] = tile_col8(bt, 32 * ks + 8 * g, 64 * wn + 16 * j, r16);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(bfr[j], af[i], acc[i][j]);

        }
    }

    // ---- epilogue: the rounded tile through LDS ----------------------------------
    __syncthreads();                              // every wave is done with the inputs
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            bf16x4 v;
            v[0] = (__bf16)acc[i][j][0]; v[1] = (__bf16)acc[i][j][1];
            v[2] = (__bf16)acc[i][j][2]; v[3] = (__bf16)acc[i][j][3];
            *reinterpret_cast<bf16x4*>(&sm.out[64 * wm + 16 * i + r16][64 * wn + 16 * j + 4 * g]) = v;
        }
    __syncthreads();

    // largest sum of squares per head: thread t takes row t % 128 of the tile's
    // head t / 128 (D = 64: two heads per tile; D = 128: one)
    constexpr int kHeads = kPrjTile / D;
    const int b = m0 / L, l0 = m0 % L;
    {
        const int row = tid & (kPrjTile - 1), hh = tid >> 7;
        double ss = 0.0;
        if (hh < kHeads) {
#pragma unroll 2
            for (int e8 = 0; e8 < D; e8 += 8) {
                const bf16x8 v = *reinterpret_cast<const bf16x8*>(&sm.out[row][D * hh + e8]);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const double x = (double)(float)v[e];
                    ss = __builtin_fma(x, x, ss);
                }
            }
        }
        // max over the 128 rows of the head (two waves)
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) ss = nan_max(ss, __shfl_xor(ss, off));
        if (lane == 0) sm.rmax[hh][(tid >> 6) & 1] = ss;
    }
    __syncthreads();
    if (tid < kHeads) {
        const int h = nw0 / D + tid;
        const double mx = nan_max(sm.rmax[tid][0], sm.rmax[tid][1]);
        part[((size_t)(b * H + h) * 2 + which) * nchunk + l0 / kPrjTile] = mx;
    }
    // rows into [B, H, L, d]: 16-byte pieces, consecutive lanes along a row
    __bf16* out = which == 0 ? Qo : Ko;
    constexpr int kPieces = kPrjTile / 8;         // 16-byte pieces per tile row
    for (int i = tid; i < kPrjTile * kPieces; i += 256) {
        const int row = i / kPieces, pc = i % kPieces;
        const int col = 8 * pc;                   // tile column
        const int h = (nw0 + col) / D, e = (nw0 + col) % D;
        const uint4 v = *reinterpret_cast<const uint4*>(&sm.out[row][col]);
        *reinterpret_cast<uint4*>(out + (((size_t)b * H + h) * L + l0 + row) * D + e) = v;
    }
}

hipError_t launch_qk_project(const ProjectArgs& a, hipStream_t s) {
    const int HD = a.H * a.d;
    dim3 grid((2 * HD / kPrjTile) * (a.B * a.L / kPrjTile));
    trace_begin(ACP_K_PROJECT, s);
    if (a.d == 64)
        hipLaunchKernelGGL(qk_project_kernel<64>, grid, dim3(256), 0, s, (const __bf16*)a.X,
                           (const __bf16*)a.Wq, (const __bf16*)a.Wk, a.L, a.Dm, a.H,
                           (__bf16*)a.Q, (__bf16*)a.K, a.part, a.nchunk);
    else
        hipLaunchKernelGGL(qk_project_kernel<128>, grid, dim3(256), 0, s, (const __bf16*)a.X,
                           (const __bf16*)a.Wq, (const __bf16*)a.Wk, a.L, a.Dm, a.H,
                           (__bf16*)a.Q, (__bf16*)a.K, a.part, a.nchunk);
    const hipError_t e = hipGetLastError();
    if (e == hipSuccess) trace_end(ACP_K_PROJECT, s);
    return e;
}

}  // namespace acp
