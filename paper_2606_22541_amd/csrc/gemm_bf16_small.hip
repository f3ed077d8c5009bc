// bf16 grouped GEMM for small groups (1..kSmallRows rows per expert).
//
// With few rows per expert the grouped GEMM is bound by streaming the
// experts' weights from HBM (at T=4096 of a DeepSeek-V3 EP32 share each of
// the 8 local experts sees ~130 rows and ~88 MB of weights).  The design
// reads every weight byte once, from all CUs at once, and keeps LDS traffic
// low enough that it does not hold the weight stream back:
//  * one tile = all rows of a group (up to 192) x 128 weight columns, so
//    each weight panel is read exactly once and there are E_loc x N/128
//    tiles (256 at T=4096) -- enough for every CU;
//  * the four wave64s form a 2 x 2 grid: wave (kh, ch) owns weight columns
//    [64 ch, 64 ch + 64) and the K half [32 kh, 32 kh + 32) of every 64-wide
//    K step, for all row blocks; the two K halves are summed through LDS
//    once per tile;
//  * weights go straight from HBM into a 4-deep register ring (each wave
//    loads only its own columns and K half: four 1 KB fragments per step,
//    each a contiguous load thanks to the fragment layout, and the four
//    waves' loads of a step together two contiguous 8 KB runs of the
//    panel-ordered weights);
//    they are read once, so the loads are non-temporal and the stream does
//    not displace the activations other kernels read next, nor force out
//    the dirty lines of earlier ones while it runs; so
//    LDS carries only the token rows: a direct-to-LDS 4-deep ring
//    (4 x 24 KB) read as MFMA fragments, two per row block per step;
//  * the K loop is unrolled by 4 so every ring index is a compile-time
//    constant, and every step issues the same loads (steps past K re-read
//    the last one), so the wait at each step is a constant: the loads of
//    the two steps issued after it;
//  * the product is formed transposed (weights as the MFMA's row operand),
//    so each lane ends with one token's accumulators: with gate/up columns
//    interleaved by 16, a lane's registers r and r + 8 are gate and up of
//    the same h column, and h leaves as 16-byte stores (store_block_swiglu);
//  * the epilogue is shared by the four waves: wave (kh, ch) hands its
//    partial sums of column block 1 - kh to its K-half partner through LDS
//    and finishes column block kh of every row block;
//  * the group tables are read in one round trip (a ballot over st_base
//    finds a tile's group), so the first fills are not held back by a chain
//    of dependent loads.
#include "kernels.h"

namespace moe {

namespace {

constexpr int kBKs = 64;                 // bf16 per K step = 128 B per row
constexpr int kRowEs = kBKs;
constexpr int kTNs = 128;                // weight columns per tile
constexpr int kWavesS = 4;
constexpr int kThreadsS = 64 * kWavesS;
constexpr int kRing = 4;                 // ring depth = unroll factor
typedef __attribute__((address_space(3))) void lds_void_s;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_s(const void *base, int64_t bytes)
{
    int32_t n = bytes > 0x7fffffff ? 0x7fffffff : (int32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

// Offset a lane reads for tile row `r` (8 rows x 128 B per load; lane l ->
// row 8 rb + l / 8, physical chunk l % 8 <- global chunk (l % 8) ^ ((row / 2)
// % 8)).  Rows past the group get an offset past every buffer range, so they
// read as zero; routed rows of an indexed A are gathered here: tile row r is
// row index[row0 + r] / div of the whole A.
__device__ __forceinline__ int token_row_offset(const int32_t *index, int div, int row0, int r,
                                                int rows_valid, int row_bytes, int lane)
{
    if (r >= rows_valid) return (int)0x80000000u;
    const int chunk = ((lane & 7) ^ ((r >> 1) & 7)) << 4;
    const int src = index ? index[row0 + r] / div : r;
    return src * row_bytes + chunk;
}

__device__ __forceinline__ bf16x8 load_b128(__amdgpu_buffer_rsrc_t r, int voff, int soff)
{
    // every weight byte is read once in the launch: non-temporal
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kNonTemporal);
    return __builtin_bit_cast(bf16x8, v);
}

}  // namespace

struct SmallTile {
    __amdgpu_buffer_rsrc_t ra, rb;
    bf16 *C;
    int row0, rows_valid, n0, N, K, KT;
    int avoff[6];      // token-row load offsets of this lane's row blocks wave + 4 i
    int vb;            // this lane's weight load offset in the 256-column panel (K step 0)
    int sstep;         // bytes of the panel per 64-wide K step
};

struct SmallLds {
    bf16 *a[kRing];   // token-row tiles, 192 rows x 64 bf16 each
};

// Per-wave constants: which K half and column half the wave owns.
struct SmallWave {
    int wave, lane, kh, ch;
};

// Fills of step j: token rows into a[I] (direct to LDS), weights into the
// register slot I; exactly NMB + 4 vector loads per wave, with no branch, so
// that the compiler's own waits on the weight registers stay exact.  Row
// blocks past the group read past the buffer range and return zeros; steps
// past K re-read the last step.  Such rows and ring slots are never used.
template <int NMB, int I>
__device__ __forceinline__ void fill_step(const SmallTile &t, const SmallLds &l, const SmallWave &w,
                                          int j, bf16x8 (&breg)[kRing][4])
{
    const int js = min(j, t.KT - 1);
#pragma unroll
    for (int i = 0; i < NMB; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            t.ra, (lds_void_s *)(l.a[I] + (w.wave + 4 * i) * 8 * kRowEs), 16, t.avoff[i],
            js * kBKs * 2, 0, 0);
    // [column block][sub-step]: q = 2 cb + m holds sub-step 2 kh + m
    const int soff = js * t.sstep;
    breg[I][0] = load_b128(t.rb, t.vb, soff);
    breg[I][1] = load_b128(t.rb, t.vb + 1024, soff);
    breg[I][2] = load_b128(t.rb, t.vb + 2048, soff);
    breg[I][3] = load_b128(t.rb, t.vb + 3072, soff);
}

// Inside the K loop the same loads are split: the step's four weight loads
// first (the HBM stream), then one token-row load after each row block's
// first two MFMAs, so that the per-CU load path is not handed the whole
// step's loads at once while the MFMAs wait behind them.  Each step still
// issues exactly NMB + 4 loads, all after the previous step's, so the waits
// keep their counts.
template <int I>
__device__ __forceinline__ void fill_weights(const SmallTile &t, const SmallWave &w, int j,
                                             bf16x8 (&breg)[kRing][4])
{
    const int js = min(j, t.KT - 1);
    const int soff = js * t.sstep;
    breg[I][0] = load_b128(t.rb, t.vb, soff);
    breg[I][1] = load_b128(t.rb, t.vb + 1024, soff);
    breg[I][2] = load_b128(t.rb, t.vb + 2048, soff);
    breg[I][3] = load_b128(t.rb, t.vb + 3072, soff);
}

template <int I>
__device__ __forceinline__ void fill_row(const SmallTile &t, const SmallLds &l, const SmallWave &w,
                                         int j, int i)
{
    const int js = min(j, t.KT - 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        t.ra, (lds_void_s *)(l.a[I] + (w.wave + 4 * i) * 8 * kRowEs), 16, t.avoff[i],
        js * kBKs * 2, 0, 0);
}

// One K step with compile-time ring index I = k % 4.
template <int NMB, int I>
__device__ __forceinline__ void small_step(const SmallTile &t, const SmallLds &l,
                                           const SmallWave &w, f32x16 (&acc)[NMB][2], int k,
                                           bf16x8 (&breg)[kRing][4])
{
    // The fills of steps k+1 and k+2 are the loads issued after step k's.
    constexpr int kAfter = 2 * (NMB + 4);
    __builtin_amdgcn_s_waitcnt((kAfter & 15) | ((kAfter >> 4) << 14) | (7 << 4) | (15 << 8));
    __builtin_amdgcn_s_barrier();          // every wave's fills of step k landed; step k-1 read
    fill_weights<(I + 3) & 3>(t, w, k + 3, breg);
    __builtin_amdgcn_sched_barrier(0);

    // Token-row fragment (mb, m) of sub-step kk = 2 kh + m: row
    // 32 mb + lane % 32, 16-byte chunk 2 kk + lane / 32, stored swizzled.
    const int rd_row = w.lane & 31;
    const int swz = (rd_row >> 1) & 7;
    const int c0 = 4 * w.kh + (w.lane >> 5);
    const bf16 *As = l.a[I];
    bf16x8 a0[NMB], a1[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
        a0[mb] = *(const bf16x8 *)&As[(mb * 32 + rd_row) * kRowEs + ((c0 ^ swz) << 3)];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
        a1[mb] = *(const bf16x8 *)&As[(mb * 32 + rd_row) * kRowEs + (((c0 + 2) ^ swz) << 3)];
    __builtin_amdgcn_sched_barrier(0);
    // transposed product: the weights are the MFMA's row operand, so a lane's
    // accumulators belong to one token (see store_block_bf16)
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
        acc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(breg[I][0], a0[mb], acc[mb][0], 0, 0, 0);
        acc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(breg[I][2], a0[mb], acc[mb][1], 0, 0, 0);
        fill_row<(I + 3) & 3>(t, l, w, k + 3, mb);
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
        acc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(breg[I][1], a1[mb], acc[mb][0], 0, 0, 0);
        acc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(breg[I][3], a1[mb], acc[mb][1], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
}

// K-half partials of column half ch: block q = 2 mb + cb (16 x 64 floats,
// 4 KB, register group g of lane l at float4 64 g + l) lives in ring buffer
// 2 ch + q / 6 at 4 KB (q % 6).  Callers pass q from fully unrolled loops, so
// it folds to a base plus an immediate.
__device__ __forceinline__ f32x4 *partial_block(const SmallLds &l, int ch, int q)
{
    return (f32x4 *)((ch ? l.a[2 + q / 6] : l.a[q / 6]) + (q % 6) * 2048);
}

// K-half exchange, step 1: wave (kh, ch) finishes column block kh of every
// row block, so it hands its partial sums of column block 1 - kh (CB = kh)
// to wave (1 - kh, ch).
template <int NMB, int CB>
__device__ __forceinline__ void give_partials(const SmallLds &l, const SmallWave &w,
                                              const f32x16 (&acc)[NMB][2])
{
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
        f32x4 *part = partial_block(l, w.ch, 2 * mb + 1 - CB) + w.lane;
        const f32x16 &v = acc[mb][1 - CB];
#pragma unroll
        for (int g = 0; g < 4; ++g)
            part[g * 64] = (f32x4){v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]};
    }
}

// Step 2: add the partner's partial sums of column block CB and write the
// block: h = SiLU(gate) * up (16 h columns) or the product (32 columns).
template <bool SWIGLU, int NMB, int CB>
__device__ __forceinline__ void finish_blocks(const SmallTile &t, const SmallLds &l,
                                              const SmallWave &w, const f32x16 (&acc)[NMB][2])
{
    const int col = t.n0 + w.ch * 64 + CB * 32;      // first weight column of the block
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
        f32x16 v = acc[mb][CB];
        const f32x4 *part = partial_block(l, w.ch, 2 * mb + CB) + w.lane;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 p = part[g * 64];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[4 * g + e] += p[e];
        }
        const int tok = mb * 32 + (w.lane & 31);
        const bool valid = tok < t.rows_valid;
        if constexpr (SWIGLU)
            store_block_swiglu(v, t.C + (int64_t)(t.row0 + tok) * (t.N / 2) + col / 2, valid);
        else
            store_block_bf16(v, t.C + (int64_t)(t.row0 + tok) * t.N + col, valid && col < t.N);
    }
}

// One tile with NMB 32-row blocks: K loop, K-half reduction and epilogue,
// fully unrolled over the row blocks so no accumulator crosses a branch.
template <bool SWIGLU, int NMB>
__device__ __forceinline__ void run_small_tile(const SmallTile &t, const SmallLds &l,
                                               const SmallWave &w)
{
    static_assert(2 * NMB <= 12, "two 24 KB ring buffers per column half");
    f32x16 acc[NMB][2];
#pragma unroll
    for (int i = 0; i < NMB; ++i) acc[i][0] = acc[i][1] = (f32x16){};
    bf16x8 breg[kRing][4];

    // Each step's loads stay together and in step order, as in the loop: the
    // compiler's wait for a weight register at the loop's first step then
    // matches the loop's own (interleaved prologue loads made it wait for
    // the next step's loads at every fourth step).
    fill_step<NMB, 0>(t, l, w, 0, breg);
    __builtin_amdgcn_sched_barrier(0);
    fill_step<NMB, 1>(t, l, w, 1, breg);
    __builtin_amdgcn_sched_barrier(0);
    fill_step<NMB, 2>(t, l, w, 2, breg);
    __builtin_amdgcn_sched_barrier(0);
    // K is a multiple of 128, so KT is even: groups of 4 steps, then 2.
    int k = 0;
    for (; k + 4 <= t.KT; k += 4) {
        small_step<NMB, 0>(t, l, w, acc, k, breg);
        small_step<NMB, 1>(t, l, w, acc, k + 1, breg);
        small_step<NMB, 2>(t, l, w, acc, k + 2, breg);
        small_step<NMB, 3>(t, l, w, acc, k + 3, breg);
    }
    if (k < t.KT) {
        small_step<NMB, 0>(t, l, w, acc, k, breg);
        small_step<NMB, 1>(t, l, w, acc, k + 1, breg);
    }
    // The look-ahead fills of steps KT..KT+2 (clamped re-reads of the last
    // step) may still be landing in ring buffers 0-2, which the K-half
    // partials overwrite next: wait for every load of this wave, then sync.
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0)
    __syncthreads();   // all ring reads done: the ring now holds the K-half partials
    // Every wave writes half the blocks: the VALU work of the epilogue (fp32
    // sums, SiLU, bf16 packing) is shared by all four.
    if (w.kh == 0) give_partials<NMB, 0>(l, w, acc); else give_partials<NMB, 1>(l, w, acc);
    __syncthreads();
    if (w.kh == 0) finish_blocks<SWIGLU, NMB, 0>(t, l, w, acc);
    else finish_blocks<SWIGLU, NMB, 1>(t, l, w, acc);
    __syncthreads();   // partials read before the next tile's fills reuse the ring
}

template <bool SWIGLU>
__global__ __launch_bounds__(kThreadsS, 1)
void k_gemm_bf16_small(GemmArgs a)
{
    __shared__ __attribute__((aligned(1024))) bf16 lds_a0[kSmallRows * kRowEs];   // 4 x 24 KB
    __shared__ __attribute__((aligned(1024))) bf16 lds_a1[kSmallRows * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a2[kSmallRows * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a3[kSmallRows * kRowEs];
    const SmallLds l{{lds_a0, lds_a1, lds_a2, lds_a3}};
    // K-half partials after the K loop: 2 x (6 x 2 x 16 x 64) floats = 96 KB,
    // the ring's four buffers, each holding six 4 KB partial blocks.
    static_assert(6 * 16 * 64 * 4 == kSmallRows * kRowEs * 2, "six partial blocks per ring buffer");

    const int tid = threadIdx.x;
    SmallWave w;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    w.kh = w.wave >> 1;
    w.ch = w.wave & 1;
    const int N = a.N, K = a.K;
    const int NT = (N + kTNs - 1) / kTNs;
    // The group tables in one round trip: with G < 64 groups, lane i holds
    // st_base[i] (i <= G), rows[i] and row0[i] (i < G), and a tile's group is
    // found by a ballot instead of a chain of dependent loads.
    const int G = a.G;
    const bool few = G < 64;
    int st_l = 0, rows_l = 0, row0_l = 0;
    if (few) {
        const int gi = min(w.lane, G - 1);
        st_l = a.groups.st_base[min(w.lane, G)];
        rows_l = a.groups.rows[gi];
        row0_l = a.groups.row0[gi];
    }
    const int total = __builtin_amdgcn_readfirstlane(
        (few ? __builtin_amdgcn_readlane(st_l, G) : a.groups.st_base[G]) * NT);
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));
    if (first >= total) return;      // no tile: leave before resolving the weights
    const void *Bw;
    const float *Bsw;
    resolve_weights(a, Bw, Bsw);


    for (int L = first; L < total; L += P) {
        // tile L: j-th small group, column block nt (an expert's column
        // blocks are consecutive, so one XCD shares its token rows in L2)
        const int j = L / NT;
        const int nt = L - j * NT;
        SmallTile t;
        int g;                                   // largest g < G with st_base[g] <= j
        if (few) {
            // st_base is nondecreasing with st_base[0] = 0 <= j
            g = __builtin_popcountll(__ballot(w.lane < G && st_l <= j)) - 1;
            g = __builtin_amdgcn_readfirstlane(g);
            t.rows_valid = __builtin_amdgcn_readlane(rows_l, g);
            t.row0 = __builtin_amdgcn_readlane(row0_l, g);
        } else {
            int lo = 0, hi = G;
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (a.groups.st_base[mid] <= j) lo = mid; else hi = mid;
            }
            g = __builtin_amdgcn_readfirstlane(lo);
            t.rows_valid = __builtin_amdgcn_readfirstlane(a.groups.rows[g]);
            t.row0 = __builtin_amdgcn_readfirstlane(a.groups.row0[g]);
        }
        t.n0 = nt * kTNs;
        t.N = N;
        t.K = K;
        t.KT = K / kBKs;
        const bool sh = (g == a.shared_group);
        const bool indexed = a.A_index != nullptr && !sh;
        const bf16 *A = indexed ? (const bf16 *)a.A_routed
                                : (const bf16 *)(sh ? a.A_shared : a.A_routed) + (int64_t)t.row0 * K;
        // panel-order weights: the tile is one half of a 256-column panel,
        // which holds per 32-wide K step its ncb column blocks' two 1 KB
        // fragments contiguously; wave (kh, ch) reads column blocks
        // 4 half + 2 ch and + 1 of the panel's K step 2 js + kh
        const int p0 = t.n0 & ~255, half = (t.n0 >> 7) & 1;
        const int ncb = min(8, (N - p0) / 32);
        const bf16 *B = (const bf16 *)Bw + ((int64_t)g * N + p0) * K;
        t.sstep = ncb * 4096;
        t.vb = w.kh * ncb * 2048 + (4 * half + 2 * w.ch) * 2048 + w.lane * 16;
        t.ra = rsrc_s(A, (indexed ? a.A_routed_rows : (int64_t)t.rows_valid) * K * 2);
#pragma unroll
        for (int i = 0; i < 6; ++i)
            t.avoff[i] = token_row_offset(indexed ? a.A_index : nullptr, a.A_index_div, t.row0,
                                          8 * (w.wave + 4 * i) + (w.lane >> 3), t.rows_valid,
                                          K * 2, w.lane);
        t.rb = rsrc_s(B, (int64_t)ncb * 32 * K * 2);
        t.C = (bf16 *)(sh ? a.C_shared : a.C_routed);
        switch ((t.rows_valid + 31) >> 5) {   // 32-row blocks holding rows: 1..6
        case 1: run_small_tile<SWIGLU, 1>(t, l, w); break;
        case 2: run_small_tile<SWIGLU, 2>(t, l, w); break;
        case 3: run_small_tile<SWIGLU, 3>(t, l, w); break;
        case 4: run_small_tile<SWIGLU, 4>(t, l, w); break;
        case 5: run_small_tile<SWIGLU, 5>(t, l, w); break;
        default: run_small_tile<SWIGLU, 6>(t, l, w); break;
        }
    }
}

hipError_t launch_gemm_bf16_small(const GemmArgs &a, bool swiglu, int g_max, int num_cus,
                                  hipStream_t s)
{
    if (g_max <= 0) return hipSuccess;
    const int64_t tiles = (int64_t)g_max * ((a.N + kTNs - 1) / kTNs);
    int grid = num_cus < tiles ? num_cus : (int)tiles;
    if (grid >= 8) grid &= ~7;
    if (swiglu)
        hipLaunchKernelGGL(k_gemm_bf16_small<true>, dim3(grid), dim3(kThreadsS), 0, s, a);
    else
        hipLaunchKernelGGL(k_gemm_bf16_small<false>, dim3(grid), dim3(kThreadsS), 0, s, a);
    return hipGetLastError();
}

}  // namespace moe
