// bf16 grouped GEMM over the local experts (the MoE "GMM": hidden states on
// the left, one expert's weights on the right; section 3.4.2).
//
// C[g] = A[g] * B[g]^T for every group g (a local expert, or the shared
// expert), where A[g] is a run of rows of X_perm (or H) and B[g] is the
// expert's [N][K] weight matrix; both are K-contiguous.
//
// Design for gfx950:
//  * one persistent workgroup per CU walks a device-built tile list, so the
//    host never learns the per-expert row counts (no read-back, no
//    re-launch) and empty experts simply own no tiles;
//  * a 256x256 output tile per workgroup, eight wave64s (two per SIMD, so one
//    wave's MFMAs cover the other's LDS waits) each owning a 128x64 block as
//    4x2 blocks of v_mfma_f32_32x32x16_bf16 (fp32 accumulation);
//  * K advances 64 bf16 (128 bytes per row) per step through a double-
//    buffered 128 KB LDS tile filled by direct-to-LDS buffer loads (no
//    staging registers; the next step streams in while MFMAs run on the
//    current one); 16-byte chunks are XOR-swizzled by row pair, which makes
//    the 16-lane groups of each ds_read_b128 hit 64 distinct banks;
//  * the raw buffer range check returns zeros for rows past the group's
//    end, so ragged groups need no clamping;
//  * the tile order is XCD-aware: workgroups are placed round-robin on the 8
//    XCDs, so consecutive tile numbers are handed to the 32 workgroups of one
//    XCD, and within a group tiles are rastered in bands of 4 row-tiles,
//    letting one XCD's L2 serve 4 row panels x 8 weight panels at a time.
//  * SwiGLU mode fuses h = SiLU(gate) * up into the epilogue: the weight
//    matrix packs gate and up rows in interleaved blocks of 16, so every
//    32-column MFMA block holds matching gate and up columns, paired across
//    lanes l and l ^ 16;
//  * for the gate/up product, groups of at most kSmallRows rows are left to
//    the small-group kernel (large_all = 0).
#include "kernels.h"

namespace moe {

namespace {

constexpr int kBK = 64;                       // bf16 elements per K step
constexpr int kRowElems = kBK;                // LDS row = 128 bytes
constexpr int kTileElems = kBM * kRowElems;   // one operand tile in LDS
constexpr int kBandM = 4;                     // row-tiles per raster band
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, int64_t bytes)
{
    // Raw buffer: loads at or past num_records return 0.
    int32_t n = bytes > 0x7fffffff ? 0x7fffffff : (int32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

__device__ __forceinline__ void decode_tile(int L, const int32_t *__restrict__ mt_base, int G,
                                            int NT, int &g, int &mt, int &nt)
{
    int lo = 0, hi = G;   // largest g with mt_base[g] * NT <= L
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (mt_base[mid] * NT <= L) lo = mid; else hi = mid;
    }
    g = lo;
    const int Lg = L - mt_base[g] * NT;
    const int Mt = mt_base[g + 1] - mt_base[g];
    const int band = Lg / (kBandM * NT);
    const int r = Lg - band * kBandM * NT;
    const int bm = min(kBandM, Mt - band * kBandM);
    mt = band * kBandM + r % bm;
    nt = r / bm;
}

}  // namespace

typedef __attribute__((address_space(3))) void lds_void;

// Direct-to-LDS loads of one K step of one 256-row operand tile: each of the
// 8 waves issues 4 instructions of 8 rows x 128 bytes (rows 32 w .. 32 w + 31).
// Lane l fills LDS row 8 b + l / 8, physical chunk l % 8, with global chunk
// (l % 8) ^ ((row / 2) % 8).
__device__ __forceinline__ void tile_to_lds(__amdgpu_buffer_rsrc_t r, bf16 *lds_tile, int wave,
                                            int voff_even, int voff_odd, int row_step_bytes, int soff)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rb = wave * 4 + i;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            r, (lds_void *)(lds_tile + rb * 8 * kRowElems), 16,
            ((i & 1) ? voff_odd : voff_even) + i * row_step_bytes, soff, 0, 0);
    }
}

template <bool SWIGLU>
__global__ __launch_bounds__(kThreads, 1)
void k_gemm_bf16(GemmArgs a)
{
    __shared__ __attribute__((aligned(1024))) bf16 lds_a0[kTileElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b0[kTileElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a1[kTileElems];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b1[kTileElems];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 2, wn = wave & 3;            // 2 x 4 waves, 128 x 64 each
    const int N = a.N, K = a.K;
    const int NT = (N + kBN - 1) / kBN;
    const int32_t *tbase = a.large_all ? a.groups.mt_base : a.groups.lt_base;
    const int total = __builtin_amdgcn_readfirstlane(tbase[a.G] * NT);
    const int KT = K / kBK;
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));

    const int lrow = wave * 32 + (lane >> 3);
    const int voff_even = lrow * K * 2 + (((lane & 7) ^ ((lane >> 4) & 7)) << 4);
    const int voff_odd = lrow * K * 2 + (((lane & 7) ^ ((4 + (lane >> 4)) & 7)) << 4);
    const int rstep = 8 * K * 2;
    const int rd_row = lane & 31;
    const int rd_hi = lane >> 5;
    const int a_rd = (wm * 128 + rd_row) * kRowElems;
    const int b_rd = (wn * 64 + rd_row) * kRowElems;

    for (int L = first; L < total; L += P) {
        int g, mt, nt;
        decode_tile(L, tbase, a.G, NT, g, mt, nt);
        g = __builtin_amdgcn_readfirstlane(g);
        mt = __builtin_amdgcn_readfirstlane(mt);
        nt = __builtin_amdgcn_readfirstlane(nt);
        const int grows = __builtin_amdgcn_readfirstlane(a.groups.rows[g]);
        const int row0 = __builtin_amdgcn_readfirstlane(a.groups.row0[g]) + mt * kBM;
        const int rows_valid = min(kBM, grows - mt * kBM);
        const int n0 = nt * kBN;
        const bool sh = (g == a.shared_group);
        const bf16 *A = (const bf16 *)(sh ? a.A_shared : a.A_routed) + (int64_t)row0 * K;
        const bf16 *B = (const bf16 *)a.B + ((int64_t)g * N + n0) * K;
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, (int64_t)rows_valid * K * 2);
        const __amdgpu_buffer_rsrc_t rb = make_rsrc(B, (int64_t)min(kBN, N - n0) * K * 2);

        f32x16 acc[4][2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = (f32x16){};

        // One K step from one LDS buffer: operand fragments for sub-step
        // kk+1 are read while the 16 MFMAs of sub-step kk run.
        auto read_frags = [&](const bf16 *As, const bf16 *Bs, int kk, bf16x8 (&af)[4],
                              bf16x8 (&bfr)[2]) {
            const int ch = ((kk * 2 + rd_hi) ^ ((rd_row >> 1) & 7)) << 3;
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
                af[mb] = *(const bf16x8 *)&As[a_rd + mb * 32 * kRowElems + ch];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
                bfr[nb] = *(const bf16x8 *)&Bs[b_rd + nb * 32 * kRowElems + ch];
        };
        auto mfma16 = [&](const bf16x8 (&af)[4], const bf16x8 (&bfr)[2]) {
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb],
                                                                         acc[mb][nb], 0, 0, 0);
        };
        auto kstep = [&](const bf16 *As, const bf16 *Bs) {
            bf16x8 a0[4], b0[2], a1[4], b1[2];
            read_frags(As, Bs, 0, a0, b0);
            read_frags(As, Bs, 1, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mfma16(a0, b0);
            read_frags(As, Bs, 2, a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            mfma16(a1, b1);
            read_frags(As, Bs, 3, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mfma16(a0, b0);
            mfma16(a1, b1);
        };

        tile_to_lds(ra, lds_a0, wave, voff_even, voff_odd, rstep, 0);
        tile_to_lds(rb, lds_b0, wave, voff_even, voff_odd, rstep, 0);
        __builtin_amdgcn_s_waitcnt(0);   // vmcnt(0): this wave's tile loads landed
        __syncthreads();
        // K is a multiple of 128, so KT is even: steps alternate buffers 0/1.
        // The next step's direct-to-LDS loads are issued first, so they fly
        // while this step's MFMAs run.
        for (int kt = 0; kt < KT; kt += 2) {
            tile_to_lds(ra, lds_a1, wave, voff_even, voff_odd, rstep, (kt + 1) * kBK * 2);
            tile_to_lds(rb, lds_b1, wave, voff_even, voff_odd, rstep, (kt + 1) * kBK * 2);
            __builtin_amdgcn_sched_barrier(0);
            kstep(lds_a0, lds_b0);
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (kt + 2 < KT) {
                tile_to_lds(ra, lds_a0, wave, voff_even, voff_odd, rstep, (kt + 2) * kBK * 2);
                tile_to_lds(rb, lds_b0, wave, voff_even, voff_odd, rstep, (kt + 2) * kBK * 2);
            }
            __builtin_amdgcn_sched_barrier(0);
            kstep(lds_a1, lds_b1);
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
        }

        // Epilogue.  Accumulator register r of a 32x32 block holds row
        // 8 (r / 4) + 4 (lane / 32) + r % 4 and column lane % 32.
        bf16 *C = (bf16 *)(sh ? a.C_shared : a.C_routed);
        if constexpr (SWIGLU) {
            // Packed columns interleave gate and up by 16: in each 32-column
            // block, lanes 0-15 hold gate and lanes 16-31 up of the same 16
            // h columns; lane l pairs with lane l ^ 16.
            const int f = N / 2;
            const bool gl = (lane & 16) == 0;
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                const int hc = (n0 + wn * 64 + nb * 32) / 2 + (lane & 15);
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const float v = acc[mb][nb][r];
                        const float up = __shfl_xor(v, 16);
                        const int lr = wm * 128 + mb * 32 + (r >> 2) * 8 + rd_hi * 4 + (r & 3);
                        if (gl && lr < rows_valid)
                            C[(int64_t)(row0 + lr) * f + hc] = f2bf(v / (1.0f + __expf(-v)) * up);
                    }
            }
        } else {
            const int c0 = n0 + wn * 64 + (lane & 31);
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int lr = wm * 128 + mb * 32 + (r >> 2) * 8 + rd_hi * 4 + (r & 3);
                    if (lr < rows_valid) {
                        bf16 *dst = C + (int64_t)(row0 + lr) * N;
#pragma unroll
                        for (int nb = 0; nb < 2; ++nb) {
                            const int col = c0 + nb * 32;
                            if (col < N) dst[col] = f2bf(acc[mb][nb][r]);
                        }
                    }
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
