// Device-side helpers shared by the library's kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace acp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Largest supported sequence length: the boundary kernel keeps 3 * (L / 64)
// words of block corners and indices in LDS.
constexpr int kMaxBlocks = 2048;
constexpr int kBlock = 64;  // pruning grid: 64 x 64 blocks

// ---- conversions ----------------------------------------------------------
__device__ __forceinline__ double to_f64(float x) { return (double)x; }
__device__ __forceinline__ double to_f64(__bf16 x) { return (double)(float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ __bf16 from_f32<__bf16>(float x) { return (__bf16)x; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// max that lets a NaN win, so that a NaN anywhere in Q or K reaches rho^2
__device__ __forceinline__ double nan_max(double a, double b) {
    return (b > a || b != b) ? b : a;
}

// ---- MFMA ------------------------------------------------------------------
// v_mfma_f32_16x16x32_bf16.  Lane l = 16 g + r (g = l / 16, r = l % 16):
//   A[i][k]: i = r, k = 8 g + t (t = 0..7, element t of the lane's bf16x8)
//   B[k][j]: j = r, k = 8 g + t
//   D[i][j]: j = r, i = 4 g + t (t = 0..3)
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// LDS transpose read (ds_read_b64_tr_b16).  Within every group of 16 lanes,
// lane i receives element (i % 4) of the 8-byte chunks whose addresses lanes
// 4t + i / 4 (t = 0..3) supplied.  If lane L of the group passes the address
// of X[r0 + L / 4][c0 + 4 (L % 4)] of a row-major 16-bit matrix X, lane i gets
// X[r0 + t][c0 + i] for t = 0..3: four rows of one column.
__device__ __forceinline__ s16x4 lds_read_tr16(const __bf16* p) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
}

// ---- LDS tiles of 64 rows x D bf16 columns ----------------------------------
// Stored as D/64 column panels of 64 x 64 elements (128-byte rows).  Inside a
// row, 16-byte chunk c sits at position c ^ swz(row).  With this swizzle the
// fragment reads below (ds_read_b128 of one chunk from rows {0-3, 8-11, ...},
// and the transpose reads of 4 rows x 32 bytes) are free of bank conflicts on
// gfx950 (measured); padded rows cost twice as much.  Each 1 KB stretch of a
// panel (8 rows) is written by one wave-wide 16-byte-per-lane DMA load.
__device__ __forceinline__ int tile_swz(int row) { return (row & 3) | (((row >> 3) & 1) << 2); }

// byte offset of element (row, col); col % 8 selects the position in the chunk
__device__ __forceinline__ int tile_off(int row, int col) {
    return (((col >> 6) << 6) + row) * 128 + ((((col & 63) >> 3) ^ tile_swz(row)) << 4) +
           ((col & 7) << 1);
}

// 8 bf16 of row `row`, columns col .. col + 7 (col % 8 == 0)
__device__ __forceinline__ bf16x8 tile_row8(const unsigned char* tile, int row, int col) {
    return *reinterpret_cast<const bf16x8*>(tile + tile_off(row, col));
}

// Eight consecutive rows r0 .. r0 + 7 of column c0 + (lane % 16) of a tile, as an
// MFMA operand whose k index runs over the rows (two LDS transpose reads).
__device__ __forceinline__ bf16x8 tile_col8(const unsigned char* tile, int r0, int c0, int r16) {
    const int col = c0 + 4 * (r16 & 3);
    s16x4 lo = lds_read_tr16(reinterpret_cast<const __bf16*>(tile + tile_off(r0 + (r16 >> 2), col)));
    s16x4 hi = lds_read_tr16(reinterpret_cast<const __bf16*>(tile + tile_off(r0 + 4 + (r16 >> 2), col)));
    bf16x8 out;
    bf16x4 lo_b = __builtin_bit_cast(bf16x4, lo);
    bf16x4 hi_b = __builtin_bit_cast(bf16x4, hi);
    out[0] = lo_b[0]; out[1] = lo_b[1]; out[2] = lo_b[2]; out[3] = lo_b[3];
    out[4] = hi_b[0]; out[5] = hi_b[1]; out[6] = hi_b[2]; out[7] = hi_b[3];
    return out;
}

// tile_col8 with the lane's address precomputed: p = tile + tile_off(r0 + (lane % 16) / 4,
// c0 + 4 (lane % 4)); rows r0 + 4 .. r0 + 7 sit 512 bytes further (the swizzle of
// a row does not change when 4 is added to a row whose bit 2 is clear).
__device__ __forceinline__ bf16x8 tile_col8_at(const unsigned char* p) {
    s16x4 lo = lds_read_tr16(reinterpret_cast<const __bf16*>(p));
    s16x4 hi = lds_read_tr16(reinterpret_cast<const __bf16*>(p + 512));
    bf16x8 out;
    bf16x4 lo_b = __builtin_bit_cast(bf16x4, lo);
    bf16x4 hi_b = __builtin_bit_cast(bf16x4, hi);
    out[0] = lo_b[0]; out[1] = lo_b[1]; out[2] = lo_b[2]; out[3] = lo_b[3];
    out[4] = hi_b[0]; out[5] = hi_b[1]; out[6] = hi_b[2]; out[7] = hi_b[3];
    return out;
}

// Issue this wave's share of the DMA loads that fill `tile` (LDS, 64 x D bf16)
// from rows src[0 .. 63] (row-major, D columns).  Instruction i writes LDS bytes
// [1024 i, 1024 i + 1024): panel i / 8, rows 8 (i % 8) .. + 7; lane L brings the
// 16-byte chunk that belongs at position L % 8 of row 8 (i % 8) + L / 8.
// Completion is tracked by vmcnt (wait before the barrier that publishes it).
// The per-lane source offsets do not depend on the tile, so they are computed
// once and held for the whole kernel: each load is a uniform (scalar) tile base
// plus a fixed 32-bit lane offset, and its address registers are never reused
// (which would force a wait for the loads in flight).
template <int D, int NWAVES>
struct TileDma {
    static constexpr int kInst = 64 * D * 2 / 1024;   // 1 KB wave instructions per tile
    static constexpr int kPer = kInst / NWAVES;
    unsigned off[kPer];

    __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = wave + NWAVES * k;
            const int row = 8 * (i & 7) + (lane >> 3);
            const int chunk = (lane & 7) ^ tile_swz(row);
            off[k] = (unsigned)(2 * (row * D + ((i >> 3) << 6) + 8 * chunk));
        }
    }
    // src: first element of the 64-row source tile (row-major, D columns).  The
    // loads are written out (scalar base + lane offset, LDS destination in M0) so
    // that the compiler neither recomputes their addresses nor, not knowing they
    // write LDS, places conservative waits before unrelated LDS reads; their
    // completion is awaited explicitly (wait_vmcnt0) before the barrier that
    // publishes the tile, and nothing the compiler waits on is issued after them
    // inside the tile compute.
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

// s_waitcnt vmcnt(0): this wave's outstanding vector-memory loads (including DMA
// writes into LDS) have completed.
__device__ __forceinline__ void wait_vmcnt0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// s_waitcnt vmcnt(0) lgkmcnt(0): additionally, this wave's LDS reads have
// returned (before a barrier after which other waves overwrite what they read).
__device__ __forceinline__ void wait_vmcnt0_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0x0070); }

// Workgroup barrier that orders this workgroup's LDS accesses only: unlike
// __syncthreads() it does not first wait for the wave's global stores to
// complete (for kernels whose global outputs no other wave reads back).
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory");
}

// ---- workgroup -> (head, block) mapping ------------------------------------
// Workgroups are dealt round-robin to the 8 XCDs (each with its own L2).  This
// renumbering gives every XCD a contiguous range of logical ids, so the blocks
// of one head share an L2.
__device__ __forceinline__ int xcd_logical_id(int bid, int nblocks) {
    const int q = nblocks >> 3, r = nblocks & 7;
    const int x = bid & 7, k = bid >> 3;
    return x * q + (x < r ? x : r) + k;
}

}  // namespace acp
