// bf16 grouped GEMM over the local experts (the MoE "GMM": hidden states on
// the left, one expert's weights on the right; section 3.4.2).
//
// C[g] = A[g] * B[g]^T for every group g (a local expert, or the shared
// expert), where A[g] is a run of token rows (gathered from x through
// slot_of_row) or of H, K-contiguous, and
// B[g] is the expert's [N][K] weight matrix stored in MFMA fragment order
// (see launch_pack_frag_bf16).
//
// Design for gfx950:
//  * one persistent workgroup per CU walks a device-built tile list, so the
//    host never learns the per-expert row counts (no read-back, no
//    re-launch) and empty experts simply own no tiles;
//  * a 256x256 output tile per workgroup, eight wave64s (two per SIMD, so one
//    wave's MFMAs cover the other's waits) each owning a 128x64 block as 4x2
//    blocks of v_mfma_f32_32x32x16_bf16 (fp32 accumulation); in a full tile
//    the two waves of a SIMD (the tile's two 128-row halves) run the K loop
//    in opposite phases, one reading its operands from LDS while the other
//    multiplies (in a partial tile the halves have unequal work, which the
//    alternation would serialise, so all waves read, then multiply);
//  * both operands are staged once per workgroup in LDS (staging the weights
//    per wave instead would load every weight fragment twice through the
//    vector L1 and its data return path, which then limits the MFMA rate);
//    K advances 32 bf16 per step through a 4-deep ring of 32 KB stages
//    (16 KB of token rows, 16 KB of weight fragments) filled by
//    direct-to-LDS buffer loads three steps ahead, issued one at a time
//    between the MFMAs (the per-CU load path takes a 1 KB load about every
//    19 clocks, and a burst of every wave's loads stalled the waves behind it);
//  * token rows are 64 bytes per step in LDS, their 16-byte chunks
//    XOR-swizzled by (row / 4) % 4 so that the 16-lane groups of each
//    ds_read_b128 hit 64 distinct banks; weight fragments arrive in MFMA
//    fragment order, one contiguous 1 KB per load, a tile's 16 fragments of
//    a step being one contiguous 16 KB run of the panel-ordered weights
//    (see launch_pack_frag_bf16), and are read back lane-contiguous, also
//    free of bank conflicts;
//  * every step of a wave issues the same loads (steps past K re-read the
//    last one), so the wait before each step is a constant and no wait
//    drains the look-ahead;
//  * the raw buffer range check returns zeros for rows past the group's
//    end, so ragged groups need no clamping;
//  * in the size order below, a partial row tile (the last one of a group
//    whose rows are not a multiple of 256) runs only the 32-row blocks that
//    hold rows: each wave takes the instance of its K loop for its number of
//    such blocks, and a wave whose 128-row half is empty loads no token rows
//    and runs no MFMAs (it still fills its share of the weight fragments);
//  * when the persistent grid runs a single round, or its last round would
//    be at most half full, tiles are numbered full tiles first, then partial
//    tiles in decreasing order of rows (tables built by the dispatch), so the
//    cheaper partial tiles form that last round; otherwise the band order
//    below is kept, in which a partial tile reads its weight panels from L2
//    beside the full tiles of its band, and no row blocks are skipped
//    (skipping them there only shifts power to the other CUs without
//    shortening the longest list of tiles);
//  * the tile order is XCD-aware: workgroups are placed round-robin on the 8
//    XCDs, so consecutive tile numbers are handed to the 32 workgroups of one
//    XCD, and within a group (full) tiles are rastered in bands of 4 row-tiles,
//    letting one XCD's L2 serve 4 row panels x 8 weight panels at a time;
//  * the product is formed transposed (weights as the MFMA's row operand),
//    so a lane's accumulators belong to one token and the output leaves as
//    16-byte stores of 8 consecutive features (store_block_bf16);
//  * SwiGLU mode fuses h = SiLU(gate) * up into the epilogue: the weight
//    matrix packs gate and up rows in interleaved blocks of 16, so a lane's
//    registers r and r + 8 of a 32-column block are gate and up of the same
//    h column (store_block_swiglu);
//  * groups of at most kSmallRows rows (gate/up) or kSmallRowsDown rows
//    (down) are left to the small-group kernel: the launch's group tables
//    (lt_base, fl_base, pl_list) count only the other groups.
#include "kernels.h"

namespace moe {

namespace {

constexpr int kBK = 32;                       // bf16 elements per K step (2 MFMA sub-steps)
constexpr int kRowElems = kBK;                // LDS token row = 64 bytes
constexpr int kAElems = kBM * kRowElems;      // token rows of one stage (16 KB)
constexpr int kBElems = kBN * kBK;            // weight fragments of one stage (16 KB)
constexpr int kBandM = 4;                     // row-tiles per raster band
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kFill = 4;                      // direct-to-LDS loads per wave per step

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, int64_t bytes)
{
    // Raw buffer: loads whose vector offset is at or past num_records return 0.
    int32_t n = bytes > 0x7fffffff ? 0x7fffffff : (int32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

// Tile Lg of a group with Mt row tiles and NT column tiles, in bands of up
// to kBandM row tiles (row tiles fastest within a band).
__device__ __forceinline__ void band_tile(int Lg, int Mt, int NT, int &mt, int &nt)
{
    const int band = Lg / (kBandM * NT);
    const int r = Lg - band * kBandM * NT;
    const int bm = min(kBandM, Mt - band * kBandM);
    mt = band * kBandM + r % bm;
    nt = r / bm;
}

__device__ __forceinline__ void decode_tile(int L, const int32_t *__restrict__ tbase, int G,
                                            int NT, int &g, int &mt, int &nt)
{
    int lo = 0, hi = G;   // largest g with tbase[g] * NT <= L
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (tbase[mid] * NT <= L) lo = mid; else hi = mid;
    }
    g = lo;
    band_tile(L - tbase[g] * NT, tbase[g + 1] - tbase[g], NT, mt, nt);
}

typedef __attribute__((address_space(3))) void lds_void;

struct Tile {
    __amdgpu_buffer_rsrc_t ra, rb;
    int KT;
    int ncb;           // weight column blocks present in the tile (8, or fewer at N's end)
    int stepb;         // bytes of one K step of the tile's weight panel (ncb x 2 KB)
    int va0, va1;      // token fills: offsets of rows 32 w + lane / 4 (+16), swizzled chunk
};

struct WaveConst {
    int voff_b;        // weight fill: lane * 16
    int a_rd;          // LDS element offset of this lane's token row (block 0)
    int b_rd;          // LDS element offset of this lane's weight fragment (block 0)
    int wave, rd_hi, swz;
};

struct Stage {
    bf16 *a, *b;
};

// Fills of step j (token rows, then weight fragments), 4 loads per wave:
//  * token rows 32 w .. 32 w + 31: two instructions of 16 rows x 64 bytes,
//    lane l -> LDS row 16 i + 32 w + l / 4, physical chunk l % 4 <- global
//    chunk (l % 4) ^ ((row / 4) % 4);
//  * weight fragments: the stage holds 8 column blocks x 2 sub-steps, 1 KB
//    each, in that order; wave w loads fragments 2 w and 2 w + 1.
// Steps past K re-read the last step.  The row offset is in the vector
// offset, which the buffer range check covers (rows past the group read as
// zero); the scalar offset, which it does not cover, only moves along K and
// between weight column blocks that exist (absent ones re-read the last).
// Load i of a fill: 0, 1 the token rows, 2, 3 the weight fragments.
template <bool STREAM>
__device__ __forceinline__ void fill_one(const Tile &t, const WaveConst &w, const Stage &st, int j, int i)
{
    const int js = min(j, t.KT - 1);
    if (i < 2) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            t.ra, (lds_void *)(st.a + (w.wave * 32 + i * 16) * kRowElems), 16,
            i ? t.va1 : t.va0, js * kBK * 2, 0, 0);
    } else {
        const int f = w.wave * 2 + (i - 2);       // fragment of the stage: 2 cb + kk
        const int cb = min(f >> 1, t.ncb - 1), kk = f & 1;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            t.rb, (lds_void *)(st.b + f * 512), 16, w.voff_b,
            js * t.stepb + (cb * 2 + kk) * 1024, 0, STREAM ? kNonTemporal : 0);
    }
}

template <bool AROWS, bool STREAM>
__device__ __forceinline__ void fill(const Tile &t, const WaveConst &w, const Stage &st, int j)
{
#pragma unroll
    for (int i = AROWS ? 0 : 2; i < 4; ++i) fill_one<STREAM>(t, w, st, j, i);
}

// One K step: wait for this step's stage, sync, then 2 sub-steps of 2 NMB
// MFMAs with the refill of the stage freed by the previous step (step j+3)
// spread among them.
template <int S, int NMB, bool STREAM>
__device__ __forceinline__ void kstep(const Tile &t, const WaveConst &w, const Stage (&ring)[4],
                                      f32x16 (&acc)[NMB > 0 ? NMB : 1][2], int j)
{
    // The fills of steps j+1 and j+2 are the loads issued after step j's.
    constexpr int kAfter = 2 * (NMB > 0 ? 4 : 2);
    __builtin_amdgcn_s_waitcnt((kAfter & 15) | ((kAfter >> 4) << 14) | (7 << 4) | (15 << 8));
    __builtin_amdgcn_s_barrier();   // every wave's fill of step j landed; step j-1 read
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NMB == 0) fill<false, STREAM>(t, w, ring[(S + 3) & 3], j + 3);
    if constexpr (NMB > 0) {
        const bf16 *As = ring[S].a;
        const bf16 *Bs = ring[S].b;
        auto read = [&](int kk, bf16x8 (&af)[NMB], bf16x8 (&bfr)[2]) {
            const int ch = ((kk * 2 + w.rd_hi) ^ w.swz) << 3;
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
                af[mb] = *(const bf16x8 *)&As[w.a_rd + mb * 32 * kRowElems + ch];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
                bfr[nb] = *(const bf16x8 *)&Bs[w.b_rd + (nb * 2 + kk) * 512];
        };
        auto mma = [&](const bf16x8 (&af)[NMB], const bf16x8 (&bfr)[2]) {
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[nb], af[mb],
                                                                         acc[mb][nb], 0, 0, 0);
        };
        bf16x8 a0[NMB], b0[2], a1[NMB], b1[2];
        read(0, a0, b0);
        read(1, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        // the fills of step j+3 go out between the MFMAs, one per NMB MFMAs:
        // issued as one burst after the barrier (32 loads of 1 KB per CU),
        // they held back every wave's reads and MFMAs until the per-CU load
        // path had taken them
        constexpr int kM = 4 * NMB, kEvery = kM / 4;
        int nf = 0;
#pragma unroll
        for (int q = 0; q < kM; ++q) {
            const int kk = q / (2 * NMB), r = q % (2 * NMB), mb = r >> 1, nb = r & 1;
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kk ? b1[nb] : b0[nb], kk ? a1[mb] : a0[mb],
                                                                 acc[mb][nb], 0, 0, 0);
            if (q % kEvery == kEvery / 2 && nf < 4) {
                fill_one<STREAM>(t, w, ring[(S + 3) & 3], j + 3, nf);
                ++nf;
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Full tiles (256 rows: both halves hold four row blocks) run the K loop
// with the two waves of a SIMD (w and w + 4: the tile's two 128-row halves)
// in opposite phases.  In phase E of step j waves 0..3 read
// step j's operands from LDS while waves 4..7 run step j-1's MFMAs, and in
// phase O the roles swap; a workgroup barrier separates the phases.  Every
// wave's fills of step j+3 go out between its MFMAs (waves 4..7 in phase E,
// waves 0..3 in phase O), into the stage of step j-1, which both halves have
// read by then; before the barrier that opens phase E of step j each wave
// waits for its own fills of step j.

template <int S, int NMB>
__device__ __forceinline__ void read_step(const WaveConst &w, const Stage (&ring)[4],
                                          bf16x8 (&a0)[4], bf16x8 (&a1)[4], bf16x8 (&b0)[2],
                                          bf16x8 (&b1)[2])
{
    if constexpr (NMB > 0) {
        const bf16 *As = ring[S].a;
        const bf16 *Bs = ring[S].b;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int ch = ((kk * 2 + w.rd_hi) ^ w.swz) << 3;
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
                (kk ? a1 : a0)[mb] = *(const bf16x8 *)&As[w.a_rd + mb * 32 * kRowElems + ch];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
                (kk ? b1 : b0)[nb] = *(const bf16x8 *)&Bs[w.b_rd + (nb * 2 + kk) * 512];
        }
    }
}

// The 4 NMB MFMAs of one step, with this wave's fills of step jf spread
// among them (one per NMB MFMAs) when FILL; a wave without row blocks only
// fills its weight fragments.
template <int NMB, bool STREAM, bool FILL>
__device__ __forceinline__ void mma_step(const Tile &t, const WaveConst &w, const Stage &fst, int jf,
                                         f32x16 (&acc)[NMB > 0 ? NMB : 1][2], const bf16x8 (&a0)[4],
                                         const bf16x8 (&a1)[4], const bf16x8 (&b0)[2],
                                         const bf16x8 (&b1)[2])
{
    if constexpr (NMB == 0) {
        if constexpr (FILL) fill<false, STREAM>(t, w, fst, jf);
    } else {
        constexpr int kM = 4 * NMB, kEvery = kM / 4;
        int nf = 0;
#pragma unroll
        for (int q = 0; q < kM; ++q) {
            const int kk = q / (2 * NMB), r = q % (2 * NMB), mb = r >> 1, nb = r & 1;
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kk ? b1[nb] : b0[nb], kk ? a1[mb] : a0[mb],
                                                                 acc[mb][nb], 0, 0, 0);
            if (FILL && q % kEvery == kEvery / 2 && nf < 4) {
                fill_one<STREAM>(t, w, fst, jf, nf);
                ++nf;
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

__device__ __forceinline__ void phase_barrier()
{
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Step j on stage S for a wave of either half.  LEAD: waves 0..3.  PREV: the
// trailing half has a step j-1 to multiply (j > 0).
template <int S, int NMB, bool STREAM, bool LEAD, bool PREV>
__device__ __forceinline__ void pp_step(const Tile &t, const WaveConst &w, const Stage (&ring)[4],
                                        f32x16 (&acc)[NMB > 0 ? NMB : 1][2], bf16x8 (&a0)[4],
                                        bf16x8 (&a1)[4], bf16x8 (&b0)[2], bf16x8 (&b1)[2], int j)
{
    // the fills of steps j+1 and j+2 are the loads issued after step j's
    constexpr int kAfter = 2 * (NMB > 0 ? 4 : 2);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt((kAfter & 15) | ((kAfter >> 4) << 14) | (7 << 4) | (15 << 8));
    phase_barrier();                                        // E_j
    const Stage &fst = ring[(S + 3) & 3];
    if constexpr (LEAD) {
        read_step<S, NMB>(w, ring, a0, a1, b0, b1);
        phase_barrier();                                    // O_j
        mma_step<NMB, STREAM, true>(t, w, fst, j + 3, acc, a0, a1, b0, b1);
    } else {
        if constexpr (PREV) mma_step<NMB, STREAM, true>(t, w, fst, j + 3, acc, a0, a1, b0, b1);
        else fill<(NMB > 0), STREAM>(t, w, fst, j + 3);
        phase_barrier();                                    // O_j
        read_step<S, NMB>(w, ring, a0, a1, b0, b1);
        // the reads of stage S complete before E_{j+1}, where it is refilled
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));
    }
}

// The tile's epilogue for one wave: NMB row blocks of its 128-row half.
template <bool SWIGLU, int NMB>
__device__ __forceinline__ void store_tile(const f32x16 (&acc)[NMB > 0 ? NMB : 1][2], const GemmArgs &a,
                                           int N, int n0, int row0, int rows_valid, bool sh, int wm,
                                           int wn, int lane)
{
    if constexpr (NMB > 0) {
        // transposed product: lane l holds token 32 mb + l % 32 of the wave's
        // 128-row half (see store_block_bf16)
        bf16 *C = (bf16 *)(sh ? a.C_shared : a.C_routed);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
            const int tok = wm * 128 + mb * 32 + (lane & 31);
            const bool valid = tok < rows_valid;
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                const int col = n0 + wn * 64 + nb * 32;
                if constexpr (SWIGLU)
                    store_block_swiglu(acc[mb][nb], C + (int64_t)(row0 + tok) * (N / 2) + col / 2,
                                       valid);
                else
                    store_block_bf16(acc[mb][nb], C + (int64_t)(row0 + tok) * N + col,
                                     valid && col < N);
            }
        }
    }
}

// One tile for a wave whose 128-row half holds NMB non-empty 32-row blocks:
// K loop, then the epilogue.  NMB = 0 only for the upper half of a tile of
// at most 128 rows: the wave then loads no token rows (they are all past the
// group) and runs no MFMAs, but still fills its share of weight fragments.
template <bool SWIGLU, int NMB, bool STREAM>
__device__ __forceinline__ void run_tile(const Tile &t, const WaveConst &w, const Stage (&ring)[4],
                                         const GemmArgs &a, int N, int n0, int row0, int rows_valid,
                                         bool sh, int wm, int wn, int lane)
{
    f32x16 acc[NMB > 0 ? NMB : 1][2];
#pragma unroll
    for (int i = 0; i < (NMB > 0 ? NMB : 1); ++i) acc[i][0] = acc[i][1] = (f32x16){};
    fill<(NMB > 0), STREAM>(t, w, ring[0], 0);
    fill<(NMB > 0), STREAM>(t, w, ring[1], 1);
    fill<(NMB > 0), STREAM>(t, w, ring[2], 2);
    // K is a multiple of 128, so KT is a multiple of 4.
    for (int j = 0; j < t.KT; j += 4) {
        kstep<0, NMB, STREAM>(t, w, ring, acc, j);
        kstep<1, NMB, STREAM>(t, w, ring, acc, j + 1);
        kstep<2, NMB, STREAM>(t, w, ring, acc, j + 2);
        kstep<3, NMB, STREAM>(t, w, ring, acc, j + 3);
    }
    __syncthreads();   // drain the look-ahead fills before the ring is reused
    store_tile<SWIGLU, NMB>(acc, a, N, n0, row0, rows_valid, sh, wm, wn, lane);
}

// A full tile (both halves hold four row blocks), K loop in two phases.
template <bool SWIGLU, bool STREAM, bool LEAD>
__device__ __forceinline__ void run_full_tile(const Tile &t, const WaveConst &w, const Stage (&ring)[4],
                                              const GemmArgs &a, int N, int n0, int row0, bool sh,
                                              int wm, int wn, int lane)
{
    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i][0] = acc[i][1] = (f32x16){};
    bf16x8 a0[4], a1[4], b0[2], b1[2];
    fill<true, STREAM>(t, w, ring[0], 0);
    fill<true, STREAM>(t, w, ring[1], 1);
    fill<true, STREAM>(t, w, ring[2], 2);
    // K is a multiple of 128, so KT is a multiple of 4; the first step (the
    // trailing half has nothing to multiply yet), then branch-free bodies of
    // four steps (stage = step % 4)
    pp_step<0, 4, STREAM, LEAD, false>(t, w, ring, acc, a0, a1, b0, b1, 0);
    pp_step<1, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, 1);
    pp_step<2, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, 2);
    pp_step<3, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, 3);
    for (int j = 4; j < t.KT; j += 4) {
        pp_step<0, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, j);
        pp_step<1, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, j + 1);
        pp_step<2, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, j + 2);
        pp_step<3, 4, STREAM, LEAD, true>(t, w, ring, acc, a0, a1, b0, b1, j + 3);
    }
    // E_KT: the trailing half multiplies the last step
    phase_barrier();
    if constexpr (!LEAD) mma_step<4, STREAM, false>(t, w, ring[0], 0, acc, a0, a1, b0, b1);
    __syncthreads();   // drain the look-ahead fills before the ring is reused
    store_tile<SWIGLU, 4>(acc, a, N, n0, row0, kBM, sh, wm, wn, lane);
}

}  // namespace

template <bool SWIGLU>
__global__ __launch_bounds__(kThreads, 1)
void k_gemm_bf16(GemmArgs a)
{
    __shared__ __attribute__((aligned(1024))) bf16 lds_a0[kAElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a1[kAElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a2[kAElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a3[kAElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b0[kBElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b1[kBElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b2[kBElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b3[kBElems];
    const Stage ring[4] = {{lds_a0, lds_b0}, {lds_a1, lds_b1}, {lds_a2, lds_b2}, {lds_a3, lds_b3}};

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    WaveConst w;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w.wave >> 2, wn = w.wave & 3;        // 2 x 4 waves, 128 x 64 each
    const int N = a.N, K = a.K;
    const int NT = (N + kBN - 1) / kBN;
    const int32_t *tbase = a.groups.lt_base;
    const int total = __builtin_amdgcn_readfirstlane(tbase[a.G] * NT);
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));
    // a workgroup without tiles (every one, when no group is this kernel's)
    // leaves after one load instead of first resolving the weights
    if (first >= total) return;
    const void *Bw;
    const float *Bsw;
    resolve_weights(a, Bw, Bsw);
    // A last round that fills at most half the grid is worth reordering:
    // full tiles first, then the partial tiles largest first, each running
    // only its non-empty row blocks.  So is a single round (every workgroup
    // holds at most one tile, so skipping row blocks only shortens tiles).
    // Otherwise the band order keeps every partial tile next to the full
    // tiles that share its weight panels in L2.
    const int tail = total % P;
    const bool by_size = total <= P || (tail != 0 && 2 * tail <= P);
    const int32_t *fbase = a.groups.fl_base;
    const int32_t *plist = a.groups.pl_list;
    const int n_full = by_size ? __builtin_amdgcn_readfirstlane(fbase[a.G] * NT) : total;

    // token fill: lane l covers row 32 w + l / 4 (+16 for the second
    // instruction), chunk l % 4; (row / 4) % 4 = (l / 16) % 4 for both
    const int frow = w.wave * 32 + (lane >> 2);
    const int fchunk = ((lane & 3) ^ ((lane >> 4) & 3)) << 4;
    w.voff_b = lane * 16;
    const int rd_row = lane & 31;
    w.rd_hi = lane >> 5;
    w.swz = (rd_row >> 2) & 3;
    w.a_rd = (wm * 128 + rd_row) * kRowElems;
    w.b_rd = (wn * 2) * 2 * 512 + lane * 8;

    // The group tables in one round trip for the whole launch: with G < 64
    // groups, lane i holds the tile prefix at i (i <= G), rows[i] and
    // row0[i] (i < G), and a tile's group is found by a ballot instead of a
    // binary search of dependent loads per tile.
    const int G = a.G;
    const bool few = G < 64;
    const int32_t *obase = by_size ? fbase : tbase;   // the order's full-tile prefix
    int ob_l = 0, rows_l = 0, row0_l = 0;
    if (few) {
        const int gi = min(lane, G - 1);
        ob_l = obase[min(lane, G)];
        rows_l = a.groups.rows[gi];
        row0_l = a.groups.row0[gi];
    }

    for (int L = first; L < total; L += P) {
        int g, mt, nt;
        if (L < n_full) {
            if (few) {
                // largest g < G with obase[g] * NT <= L (obase is nondecreasing, obase[0] = 0)
                g = __builtin_popcountll(__ballot(lane < G && ob_l * NT <= L)) - 1;
                g = __builtin_amdgcn_readfirstlane(g);
                const int b0 = __builtin_amdgcn_readlane(ob_l, g);
                const int b1 = __builtin_amdgcn_readlane(ob_l, g + 1);
                band_tile(L - b0 * NT, b1 - b0, NT, mt, nt);
            } else {
                decode_tile(L, obase, G, NT, g, mt, nt);
            }
        } else {
            // partial row tiles, largest first; a group's column tiles are consecutive
            const int j = (L - n_full) / NT;
            nt = L - n_full - j * NT;
            g = __builtin_amdgcn_readfirstlane(plist[j]);
            mt = (few ? __builtin_amdgcn_readlane(rows_l, g) : a.groups.rows[g]) / kBM;
        }
        g = __builtin_amdgcn_readfirstlane(g);
        mt = __builtin_amdgcn_readfirstlane(mt);
        nt = __builtin_amdgcn_readfirstlane(nt);
        const int grows = __builtin_amdgcn_readfirstlane(
            few ? __builtin_amdgcn_readlane(rows_l, g) : a.groups.rows[g]);
        const int row0 = __builtin_amdgcn_readfirstlane(
            few ? __builtin_amdgcn_readlane(row0_l, g) : a.groups.row0[g]) + mt * kBM;
        const int rows_valid = min(kBM, grows - mt * kBM);
        const int n0 = nt * kBN;
        const bool sh = (g == a.shared_group);
        // routed rows of an indexed A are gathered in the token fills: tile
        // row r is row A_index[row0 + r] / A_index_div of the whole A
        const bool indexed = a.A_index != nullptr && !sh;
        const bf16 *A = indexed ? (const bf16 *)a.A_routed
                                : (const bf16 *)(sh ? a.A_shared : a.A_routed) + (int64_t)row0 * K;
        // the tile's column blocks n0/32 .. n0/32 + 7 are contiguous
        const bf16 *B = (const bf16 *)Bw + ((int64_t)g * N + n0) * K;
        Tile t;
        t.ra = make_rsrc(A, (indexed ? a.A_routed_rows : (int64_t)rows_valid) * K * 2);
        {
            // rows past the group: an offset past every buffer range reads zero
            const int r0 = frow, r1 = frow + 16;
            t.va0 = r0 < rows_valid ? (indexed ? a.A_index[row0 + r0] / a.A_index_div : r0) * K * 2 + fchunk
                                    : (int)0x80000000u;
            t.va1 = r1 < rows_valid ? (indexed ? a.A_index[row0 + r1] / a.A_index_div : r1) * K * 2 + fchunk
                                    : (int)0x80000000u;
        }
        t.rb = make_rsrc(B, (int64_t)min(kBN, N - n0) * K * 2);
        t.KT = K / kBK;
        t.ncb = min(kBN, N - n0) / 32;
        t.stepb = t.ncb * 2048;

        // 32-row blocks of this wave's 128-row half that hold rows (uniform per
        // wave); in band order every tile runs all of them
        const int nmb = by_size ? __builtin_amdgcn_readfirstlane(
                                      min(4, max(0, (rows_valid - wm * 128 + 31) >> 5)))
                                : 4;
        // A group of one row tile reads each of its weight panels once in the
        // launch: those loads are non-temporal, so the panels do not displace
        // what the caches hold for later kernels (the combine's rows) and the
        // dirty lines of earlier ones.  Groups of several row tiles share
        // their panels through L2 and keep ordinary loads.
        if (rows_valid == kBM) {
            // every wave's half is full: the two-phase loop
            if (grows <= kBM) {
                if (wm == 0) run_full_tile<SWIGLU, true, true>(t, w, ring, a, N, n0, row0, sh, wm, wn, lane);
                else run_full_tile<SWIGLU, true, false>(t, w, ring, a, N, n0, row0, sh, wm, wn, lane);
            } else {
                if (wm == 0) run_full_tile<SWIGLU, false, true>(t, w, ring, a, N, n0, row0, sh, wm, wn, lane);
                else run_full_tile<SWIGLU, false, false>(t, w, ring, a, N, n0, row0, sh, wm, wn, lane);
            }
        } else if (grows <= kBM) {
            switch (nmb) {
            case 0: run_tile<SWIGLU, 0, true>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            case 1: run_tile<SWIGLU, 1, true>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            case 2: run_tile<SWIGLU, 2, true>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            case 3: run_tile<SWIGLU, 3, true>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            default: run_tile<SWIGLU, 4, true>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            }
        } else {
            switch (nmb) {
            case 0: run_tile<SWIGLU, 0, false>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            case 1: run_tile<SWIGLU, 1, false>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            case 2: run_tile<SWIGLU, 2, false>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            case 3: run_tile<SWIGLU, 3, false>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            default: run_tile<SWIGLU, 4, false>(t, w, ring, a, N, n0, row0, rows_valid, sh, wm, wn, lane); break;
            }
        }
    }
}

hipError_t launch_gemm_bf16(const GemmArgs &a, bool swiglu, int mt_max, int num_cus,
                            hipStream_t s)
{
    if (mt_max <= 0) return hipSuccess;
    const int64_t tiles = (int64_t)mt_max * ((a.N + kBN - 1) / kBN);
    int grid = num_cus < tiles ? num_cus : (int)tiles;
    if (grid >= 8) grid &= ~7;
    if (swiglu)
        hipLaunchKernelGGL(k_gemm_bf16<true>, dim3(grid), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(k_gemm_bf16<false>, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace moe
