// Shared definitions of the gfx950 (CDNA4) kernels of the MoE expert stage.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

// Dispatch: slots handled by one workgroup of the histogram / scatter kernels.
constexpr int kDispatchThreads = 256;
constexpr int kDispatchChunk = 1024;            // 4 slots per thread
constexpr int kMaxExperts = 1024;               // LDS histogram size
constexpr int kMaxLocalExperts = 256;
constexpr int kMaxLayers = 1024;
constexpr int kMaxIngestWords = 4096;            // ready words one ingest wait may poll
constexpr uint32_t kDefaultIngestSpins = 1u << 19;   // about a second of polling

// Grouped GEMM tile: 256 x 256 output, K step 64 bf16 (or 128 e4m3) = 128 B
// per row.
constexpr int kBM = 256;
constexpr int kBN = 256;

// Cache-policy operand of the raw buffer loads: non-temporal (streaming)
// data, read once, evicted first and kept out of the last-level cache.
constexpr int kNonTemporal = 2;

// Sticky error bits.
constexpr int kErrBadId = 1;
constexpr int kErrBadLayer = 2;
constexpr int kErrIngestTimeout = 4;
constexpr int kErrBadCount = 8;       // pre-grouped counts negative or past the rows buffer

// Groups with at most this many rows ("small": a DeepSeek EP32 share at
// T=4096 has ~128 rows per expert) take one full-height tile in the bf16
// small-group GEMM, which streams each weight panel exactly once; larger
// groups use the 256x256-tile GEMM.
constexpr int kSmallRows = 192;
// The down product's partition: only groups of at most this many rows take
// the small-group kernel (at ~130 rows per expert, 256-wide tiles of the down
// product's d columns fill the GPU in one round, where 128-wide small tiles
// would take 1.75 rounds; groups of a few dozen rows, as the cold experts of
// skewed routing have, stream their weights faster in the small kernel).
constexpr int kSmallRowsDown = 64;

// Device-side tables written by the dispatch scan, read by the GEMMs.
struct GroupTable {
    int32_t *row0;      // [G] first row of the group in its A matrix
    int32_t *rows;      // [G] rows of the group
    int32_t *lt_base;   // [G+1] prefix of ceil(rows / kBM) over groups with rows > kSmallRows
    int32_t *st_base;   // [G+1] prefix of 1 per group with 1 <= rows <= kSmallRows
    // Tile order of the 256-row bf16 GEMM: the full row tiles of every group
    // first, then the partial ones (rows % kBM != 0), largest first, so the
    // cheap partial tiles fill the last round of the persistent grid.
    int32_t *fl_base;   // [G+1] prefix of rows / kBM over groups with rows > kSmallRows
    int32_t *pl_list;   // [G+1] groups with rows > kSmallRows and a partial row tile,
                        //       by descending rows % kBM (ties: lower index first); count at [G]
    // The same partition at kSmallRowsDown rows (the down product's):
    int32_t *lt_base_d; // [G+1] as lt_base, groups with rows > kSmallRowsDown
    int32_t *st_base_d; // [G+1] as st_base, groups with 1 <= rows <= kSmallRowsDown
    int32_t *fl_base_d; // [G+1] as fl_base, groups with rows > kSmallRowsDown
    int32_t *pl_list_d; // [G+1] as pl_list, groups with rows > kSmallRowsDown
};

// The tables a GEMM launch reads for the down product: the partition at
// kSmallRowsDown in place of the one at kSmallRows.
__host__ __device__ inline GroupTable down_partition(const GroupTable &g)
{
    GroupTable d = g;
    d.lt_base = g.lt_base_d;
    d.st_base = g.st_base_d;
    d.fl_base = g.fl_base_d;
    d.pl_list = g.pl_list_d;
    return d;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Round-to-nearest-even fp32 -> bf16 (finite inputs).
__device__ __forceinline__ bf16 f2bf(float v) { return static_cast<bf16>(v); }
__device__ __forceinline__ float bf2f(bf16 v) { return static_cast<float>(v); }

// Two fp32 values as a pair of bf16 in one word (round to nearest even), the
// first in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t v = {static_cast<bf16>(lo), static_cast<bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

// SiLU(g) * u = g / (1 + e^-g) * u with the hardware exp2 and reciprocal
// (about 1 ulp each in fp32, far below the bf16 rounding of the result).
// g -> -inf gives e = inf and a zero reciprocal; g -> +inf gives g * u.
__device__ __forceinline__ float silu_mul(float g, float u)
{
    const float e = __builtin_amdgcn_exp2f(-1.44269504088896341f * g);
    return g * __builtin_amdgcn_rcpf(1.0f + e) * u;
}

// Swaps lanes 32..63 of x with lanes 0..31 of y (v_permlane32_swap): after
// it, x holds [x.lo, y.lo] and y holds [x.hi, y.hi].
__device__ __forceinline__ void swap_halves(uint32_t &x, uint32_t &y)
{
    const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
    x = r[0];
    y = r[1];
}

// Output of one 32x32 block of the transposed product D[feature][token]
// (v_mfma_f32_32x32x16_bf16 with the weights as its row operand): lane l
// holds token l % 32, and register r holds feature 8 (r/4) + 4 (l/32) + r%4
// of the block.  Lanes l and l ^ 32 hold the same token, so after swapping
// halves each lane has 8 consecutive features and writes 16 bytes.
//
// store_block_bf16: the block's 32 features as bf16 at row[0..31] (row =
// the token's output row at the block's first column); lane l writes
// features 8 (l/32) .. +7 and 16 + 8 (l/32) .. +7.
__device__ __forceinline__ void store_block_bf16(const f32x16 &v, bf16 *row, bool valid)
{
    uint32_t p[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        p[2 * q] = pack_bf16x2(v[4 * q], v[4 * q + 1]);
        p[2 * q + 1] = pack_bf16x2(v[4 * q + 2], v[4 * q + 3]);
    }
    swap_halves(p[0], p[2]);
    swap_halves(p[1], p[3]);
    swap_halves(p[4], p[6]);
    swap_halves(p[5], p[7]);
    const int hi = (__lane_id() >> 5) * 8;
    if (valid) {
        *(u32x4 *)(row + hi) = (u32x4){p[0], p[1], p[2], p[3]};
        *(u32x4 *)(row + 16 + hi) = (u32x4){p[4], p[5], p[6], p[7]};
    }
}

// store_block_swiglu: the packed gate/up weights interleave by 16, so
// features 0..15 of a block are gate rows and 16..31 the matching up rows:
// register r (r < 8) and r + 8 of a lane are gate and up of one h column
// 8 (r/4) + 4 (l/32) + r%4.  The block's 16 h columns go to hrow[0..15];
// lane l writes h columns 8 (l/32) .. +7.
__device__ __forceinline__ void store_block_swiglu(const f32x16 &v, bf16 *hrow, bool valid)
{
    uint32_t p[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
        p[q] = pack_bf16x2(silu_mul(v[2 * q], v[2 * q + 8]), silu_mul(v[2 * q + 1], v[2 * q + 9]));
    swap_halves(p[0], p[2]);
    swap_halves(p[1], p[3]);
    if (valid) *(u32x4 *)(hrow + (__lane_id() >> 5) * 8) = (u32x4){p[0], p[1], p[2], p[3]};
}

// e4m3 (OCP E4M3FN) code of v, round to nearest even.  |v| is clamped to 448
// first, which makes the conversion saturating.
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d)
{
    a = fminf(fmaxf(a, -448.0f), 448.0f);
    b = fminf(fmaxf(b, -448.0f), 448.0f);
    c = fminf(fmaxf(c, -448.0f), 448.0f);
    d = fminf(fmaxf(d, -448.0f), 448.0f);
    int v = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
    v = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, v, true);
    return (uint32_t)v;
}

}  // namespace moe
