// Host-side launchers of the stage's kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace moe {

struct DispatchArgs {
    const int32_t *ids;      // [T*k]
    int32_t n_slots;         // T*k
    int32_t T, k, E, e0, E_loc;
    int32_t has_shared;
    int32_t *blk_counts;     // [nb][E]
    int32_t *counts;         // [E]
    int32_t *offsets;        // [E_loc+1]
    GroupTable groups;       // G = E_loc + has_shared groups
    int32_t *slot_of_row;    // [cap]
    int32_t *row_of_slot;    // [T*k]
    int32_t *err;            // sticky error word
};

// Histogram -> scan (+ GEMM tile table) -> stable scatter.
hipError_t launch_dispatch_index(const DispatchArgs &a, hipStream_t s);

// Tile tables (GroupTable over the E_loc routed groups, no shared group) for
// rows that arrive already grouped by local expert: counts[i] rows of expert
// i, consecutive.  Counts are read on the device; a negative count is taken
// as 0 and the running total is capped at n_rows_max (later groups lose
// their rows), both reported through kErrBadCount in *err.
hipError_t launch_group_tables_from_counts(const int32_t *counts, int32_t E_loc,
                                           int32_t n_rows_max, GroupTable g, int32_t *err,
                                           hipStream_t s);

// fp8: the token scales of the routed rows, transposed: x_perm_scales[g *
// scale_ld + r] = x_scales[(slot_of_row[r] / k) * n_scales + g] for r <
// *n_rows_dev (offsets[E_loc]) and g < n_scales; max_rows bounds the rows
// (grid size only).  The e4m3 rows themselves are read by the gate/up GEMM
// through slot_of_row.
hipError_t launch_gather_scales(const float *x_scales, const int32_t *slot_of_row,
                                const int32_t *n_rows_dev, int32_t k, int32_t n_scales,
                                float *x_perm_scales, int32_t scale_ld, int32_t max_rows,
                                int num_cus, hipStream_t s);

// [rows][cols] -> [cols][ld] copy of fp32 scales.
hipError_t launch_transpose_scales(const float *src, int32_t rows, int32_t cols, float *dst,
                                   int32_t ld, hipStream_t s);

// Packed weights of one layer (device addresses); the stage keeps a device
// array of these, one per layer.
struct LayerWeights {
    const void *w1, *w2;      // gate/up and down, in MFMA fragment order
    const float *s1, *s2;     // fp8 block scales (null in bf16)
};

struct GemmArgs {
    const void *A_routed;    // [rows][K] (rows of H, or pre-grouped rows), or x itself when A_index is set
    const void *A_shared;    // [T][K] (x or H_shared) for group E_loc, if shared
    const float *As_routed;  // fp8: [rows][K/128] scales of A
    const float *As_shared;
    const void *B;           // [G][N][K] weights (K contiguous)
    const float *Bs;         // fp8: block scales
    void *C_routed;          // [rows][ldc]
    void *C_shared;
    float *Cs_routed;        // fp8 SwiGLU epilogue: [rows][f/128] scales of H
    float *Cs_shared;
    int32_t N, K;
    int32_t shared_group;    // index of the shared group, -1 if none
    GroupTable groups;
    int32_t G;
    // When A_index is set, routed row r (r < the routed rows) is row
    // A_index[r] / A_index_div of A_routed, which has A_routed_rows rows (the
    // row gather happens in the GEMM's token-row loads; A_index = slot_of_row).
    // In fp8 the A scales stay indexed by the routed row (As_routed holds the
    // gathered scales, launch_gather_scales).
    const int32_t *A_index;
    int32_t A_index_div;
    int64_t A_routed_rows;
    // Layer-oblivious weights: with layer_id set, B and Bs are taken on the
    // device from layers[*layer_id] (w1/s1, or w2/s2 when `down`); an id
    // outside [0, n_layers) is clamped and flagged in err.
    const int32_t *layer_id;
    const LayerWeights *layers;
    int32_t n_layers;
    int32_t down;
    int32_t *err;
};

// A pointer loaded from memory, made provably wave-uniform (the value is the
// same in every lane), so that buffer descriptors built from it stay in
// scalar registers instead of being re-established lane by lane at each load.
template <typename T>
__device__ __forceinline__ T *uniform_ptr(T *p)
{
    const uint64_t v = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (T *)(((uint64_t)hi << 32) | lo);
}

// The weights a GEMM launch uses: a.B / a.Bs, or the ones of the layer named
// in device memory (read once per workgroup; every wave gets the same value).
// Workgroup 0 reports an id out of range; it calls this whenever the launch
// has any tile (a launch without tiles reads no weights and checks nothing).
__device__ __forceinline__ void resolve_weights(const GemmArgs &a, const void *&B, const float *&Bs)
{
    B = a.B;
    Bs = a.Bs;
    if (a.layer_id) {
        int l = __builtin_amdgcn_readfirstlane(*a.layer_id);
        if (l < 0 || l >= a.n_layers) {
            if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(a.err, kErrBadLayer);
            l = l < 0 ? 0 : a.n_layers - 1;
        }
        const LayerWeights &lw = a.layers[l];
        B = uniform_ptr(a.down ? lw.w2 : lw.w1);
        Bs = uniform_ptr(a.down ? lw.s2 : lw.s1);
    }
}

// bf16 grouped GEMM.  swiglu = true: B is the packed [gate|up] matrix
// (N = 2f) and C receives SiLU(gate) * up as [rows][f] bf16; otherwise C
// receives the product as [rows][N] bf16.  mt_max bounds the number of
// 256-row tiles over all groups (the grid is sized from it).
hipError_t launch_gemm_bf16(const GemmArgs &a, bool swiglu, int mt_max, int num_cus,
                            hipStream_t s);
// bf16 grouped GEMM for the groups with 1..kSmallRows rows: one 256-row x
// 128-column tile per (group, column block); g_max bounds the group count.
hipError_t launch_gemm_bf16_small(const GemmArgs &a, bool swiglu, int g_max, int num_cus,
                                  hipStream_t s);

// e4m3 grouped GEMM with 128-block scales (same conventions; the A scales
// are transposed, [K/128][ld] with ld = lds_rows_routed / lds_rows_shared).
// swiglu = true writes e4m3 h with one scale per row and 128 channels
// (C and Cs, the scales transposed like the A scales).  Every group runs
// as 128-row tiles (mt_max bounds the 256-row tiles of all groups together;
// g_max is unused).
hipError_t launch_gemm_fp8(const GemmArgs &a, bool swiglu, int mt_max, int g_max, int num_cus,
                           int32_t lds_rows_routed, int32_t lds_rows_shared, hipStream_t s);

struct CombineArgs {
    const void *y_perm;        // [rows][d] bf16
    const void *y_shared;      // [T][d] bf16 or nullptr
    const int32_t *row_of_slot;
    const float *w;            // [T][k]
    void *out;                 // [T][d] bf16
    int32_t T, k, d, accumulate;
};
hipError_t launch_combine(const CombineArgs &a, int num_cus, hipStream_t s);

// Per-row, per-128-channel e4m3 quantisation of bf16 rows.  Rows: n_rows,
// or *n_rows_dev when that is not null (then n_rows is the bound used to size
// the grid).  Scales go to xs[row * (d/128) + g] (scale_ld = 0) or, when
// scale_ld > 0, transposed to xs[g * scale_ld + row].
hipError_t launch_quantize_fp8(const void *x, int32_t n_rows, const int32_t *n_rows_dev,
                               int32_t d, void *xq, float *xs, int32_t scale_ld, int num_cus,
                               hipStream_t s);

// Asynchronous ingest: a bounded device-side wait until every ready[i]
// (i < n_words) has reached `epoch` (wrapping compare); after spin_limit
// polls it gives up and sets kErrIngestTimeout in err.  signal: a release
// store of `epoch` into *word after the stream's earlier work.
hipError_t launch_ingest_wait(const uint32_t *ready, int32_t n_words, uint32_t epoch,
                              uint32_t spin_limit, int32_t *err, hipStream_t s);
hipError_t launch_ingest_signal(uint32_t *word, uint32_t epoch, hipStream_t s);

// Weight packing at create time.  Gate and up rows are interleaved in
// blocks of `interleave` rows: packed row 2*il*b + i is gate row il*b + i for
// i < il and up row il*b + (i - il) otherwise.  Both paths use il = 16: a
// 32-column bf16 MFMA block then holds matching gate and up columns, and in
// fp8 a wave's 64 columns are gate and up rows of the same 32 h channels,
// all within one 128-row scale block of each.
constexpr int kInterleaveBf16 = 16;
constexpr int kInterleaveFp8 = 16;
// bf16 weights in MFMA fragments, panel order (the layout both bf16
// grouped-GEMM kernels read B in).  The 1 KB fragment of 32-column block b and
// 16-wide K sub-step u holds, in 16-byte chunk n % 32 + 32 ((k/8) % 2), row
// n, columns k..k+7 (k % 8 == 0).  Fragments are grouped in panels of 256
// columns (8 blocks; fewer at N's end): a panel stores, for each 32-wide K
// step s, its blocks' fragments (b, 2s) and (b, 2s + 1) contiguously, block
// by block, so one K step of a panel is a single contiguous run.  With `up`
// non-null the packed rows interleave gate and up by `interleave`.
hipError_t launch_pack_frag_bf16(const void *gate, const void *up, void *dst, int32_t n_mats,
                                 int32_t N, int32_t K, int32_t interleave, hipStream_t s);
// e4m3 weights in the fragment order of the 16x16x128 f8 MFMA: chunk
// ((m * N/16 + n/16) * K/128 + k/128) * 128 + 64 ((k/16) % 2) + n % 16 +
// 16 ((k % 128) / 32) of 16 bytes holds row n, bytes k..k+15 (k % 16 == 0).
hipError_t launch_pack_frag_fp8(const void *gate, const void *up, void *dst, int32_t n_mats,
                                int32_t N, int32_t K, int32_t interleave, hipStream_t s);
// Gate/up block scales of the fp8 path, [m][f/128][gate, up][d/128], from the
// two [m][f/128][d/128] arrays.
hipError_t launch_pack_gate_up_scales(const float *gs, const float *us, float *packed_s,
                                      int32_t n_mats, int32_t f, int32_t d, hipStream_t s);

}  // namespace moe
