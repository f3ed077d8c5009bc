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

// Device-side tables written by the dispatch scan, read by the GEMMs.
struct GroupTable {
    int32_t *row0;      // [G] first row of the group in its A matrix
    int32_t *rows;      // [G] rows of the group
    int32_t *mt_base;   // [G+1] prefix of ceil(rows / kBM) over all groups
    int32_t *lt_base;   // [G+1] same, counting only groups with rows > kSmallRows
    int32_t *st_base;   // [G+1] prefix of 1 per group with 1 <= rows <= kSmallRows
    // Tile order of the 256-row bf16 GEMM: the full row tiles of every group
    // first, then the partial ones (rows % kBM != 0), largest first, so the
    // cheap partial tiles fill the last round of the persistent grid.
    int32_t *fm_base;   // [G+1] prefix of rows / kBM over all groups
    int32_t *fl_base;   // [G+1] same, over groups with rows > kSmallRows
    int32_t *pm_list;   // [G+1] groups with a partial row tile, by descending
                        //       rows % kBM (ties: lower index first); count at [G]
    int32_t *pl_list;   // [G+1] same, over groups with rows > kSmallRows
};

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Round-to-nearest-even fp32 -> bf16 (finite inputs).
__device__ __forceinline__ bf16 f2bf(float v) { return static_cast<bf16>(v); }
__device__ __forceinline__ float bf2f(bf16 v) { return static_cast<float>(v); }

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
