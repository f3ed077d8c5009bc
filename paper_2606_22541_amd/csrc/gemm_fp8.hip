// e4m3 grouped GEMM with DeepSeek-style block scaling (fp8 variant of the
// expert stage): activations carry one fp32 scale per row and 128-channel
// group, weights one fp32 scale per 128x128 block.  Each K step covers
// exactly one 128-wide scale group g:
//
//   t    = sum over the group of e4m3(A) * e4m3(B)     (v_mfma 16x16x128 f8)
//   acc += t * (s_A[row, g] * s_B[block, g])            (fp32 promotion)
//
// so the block scales are applied exactly once per group in fp32.  The
// hardware's per-32-element power-of-two (E8M0) MFMA scales cannot express
// these fp32 scales and are left at 1.
//
// Design for gfx950:
//  * one persistent workgroup per CU walks the device-built tile list
//    (256-row tiles, as for the bf16 path), XCD-aware tile order;
//  * a 256x256 output tile, eight wave64s (two per SIMD, so one wave's
//    promotion arithmetic runs beside the other's MFMAs), each owning a
//    128x64 block as 8x4 blocks of v_mfma_scale_f32_16x16x128_f8f6f4;
//  * the weights are packed so that every wave's 64 columns fall into one
//    128x128 scale block: gate and up rows interleave in blocks of 64, and
//    a 256-column tile covers gate and up rows [128 t, 128 t + 128), i.e.
//    exactly one 128-channel group of h.  The promotion then needs one
//    weight scale per wave and group (a scalar load) and one product per
//    row, so it costs 1.25 VALU operations per output and group;
//  * K advances one scale group (128 bytes) per step through a 2-deep LDS
//    ring of 64 KB stages filled by direct-to-LDS buffer loads one step
//    ahead: token rows as 128-byte rows whose 16-byte chunks are
//    XOR-swizzled by (row / 2) % 8, weight fragments in MFMA fragment order
//    (two lane-contiguous 1 KB halves per 16 x 128 fragment), and the
//    step's 256 row scales (stored transposed, [K/128][ld], so they are one
//    contiguous 1 KB);
//  * rows past a group's end have an offset past every buffer range and
//    read as zero; the scalar offset, which the range check does not cover,
//    only moves along K (clamped to the last group) and between weight
//    column blocks that exist;
//  * SwiGLU mode: the up waves hand their accumulators to the gate waves
//    through LDS, the gate waves form h = SiLU(gate) * up in fp32 and
//    quantise each row's 128 channels to e4m3 with one fp32 scale (the same
//    arithmetic as the activation quantiser), and the tile's 256 rows
//    of 128 codes are written out through LDS as 16-byte stores.  The down
//    product writes bf16.
#include "kernels.h"

namespace moe {

namespace {

constexpr int kGrpB = 128;                      // K bytes per step: one scale group
constexpr int kStage8 = kBM * kGrpB;            // one operand of one stage: 32 KB
constexpr int kWaves8 = 8;
constexpr int kThreads8 = 64 * kWaves8;
constexpr int kBand8 = 4;                       // row-tiles per raster band
typedef __attribute__((address_space(3))) void lds_void;
static_assert(kBM == 256 && kBN == 256, "the fp8 kernel assumes 256x256 tiles");

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc8(const void *base, int64_t bytes)
{
    int32_t n = bytes > 0x7fffffff ? 0x7fffffff : (int32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

__device__ __forceinline__ void decode_tile8(int L, const int32_t *__restrict__ mt_base, int G,
                                             int NT, int &g, int &mt, int &nt)
{
    int lo = 0, hi = G;
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (mt_base[mid] * NT <= L) lo = mid; else hi = mid;
    }
    g = lo;
    const int Lg = L - mt_base[g] * NT;
    const int Mt = mt_base[g + 1] - mt_base[g];
    const int band = Lg / (kBand8 * NT);
    const int r = Lg - band * kBand8 * NT;
    const int bm = min(kBand8, Mt - band * kBand8);
    mt = band * kBand8 + r % bm;
    nt = r / bm;
}

struct Tile8 {
    __amdgpu_buffer_rsrc_t ra, rb, rs;
    int va[4];          // token fills: rows 32 w + 8 i + lane / 8, swizzled chunk (or past the range)
    int KT, ncb, cbstride, s_ld;
    const float *sbp;   // this wave's weight scale of each K group
};

struct Ring8 {
    uint8_t *a, *b;
    float *s;
};

// Fills of K group kg (clamped to the last), 9 loads per wave:
//  * token rows 32 w .. 32 w + 31 as four 8-row instructions; lane l writes
//    LDS row 32 w + 8 i + l / 8, physical chunk l % 8, with global chunk
//    (l % 8) ^ ((row / 2) % 8);
//  * weight fragments 2 w and 2 w + 1 of the tile's 16, both 1 KB halves;
//  * 64 of the 256 row scales (waves w and w + 4 load the same ones).
__device__ __forceinline__ void fill8(const Tile8 &t, const Ring8 &st, int wave, int lane, int kg)
{
    const int ks = min(kg, t.KT - 1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(t.ra, (lds_void *)(st.a + (wave * 32 + i * 8) * kGrpB),
                                                 16, t.va[i], ks * kGrpB, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int f = wave * 2 + (i >> 1), h = i & 1;
        const int cb = min(f, t.ncb - 1);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(t.rb, (lds_void *)(st.b + f * 2048 + h * 1024), 16,
                                                 lane * 16, cb * t.cbstride + ks * 2048 + h * 1024,
                                                 0, 0);
    }
    __builtin_amdgcn_raw_ptr_buffer_load_lds(t.rs, (lds_void *)(st.s + (wave & 3) * 64), 4,
                                             (ks * t.s_ld + (wave & 3) * 64 + lane) * 4, 0, 0, 0);
}

struct Wave8 {
    int wave, lane;
    int a_rd0, a_rd1;   // LDS byte offsets of this lane's two token chunks (row block 0)
    int b_rd;           // LDS byte offset of this lane's weight chunk (column block 0)
    int s_rd;           // LDS float index of this lane's 4 row scales (row block 0)
};

// One K group: wait for its stage, sync, refill the other stage with the
// next group, then 32 MFMAs with the promotion of each row block.
// The weight scale of the next group is loaded before the fills, so that
// waiting for it never waits for them.
// RB row blocks of 16 rows per wave.  GUARD: row blocks at or past nrb (past
// the group's last row) are skipped (wave-uniform branches).
template <int S, int RB, bool GUARD>
__device__ __forceinline__ void kgroup8(const Tile8 &t, const Wave8 &w, const Ring8 (&ring)[2],
                                        f32x4 (&acc)[RB][4], float &sb_next, int kg, int nrb)
{
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0): this group's fills landed
    __builtin_amdgcn_s_barrier();                        // ... in every wave; the other stage is idle
    const float sb = sb_next;
    sb_next = t.sbp[min(kg + 1, t.KT - 1)];
    __builtin_amdgcn_sched_barrier(0);
    fill8(t, ring[S ^ 1], w.wave, w.lane, kg + 1);
    __builtin_amdgcn_sched_barrier(0);

    const uint8_t *As = ring[S].a;
    const uint8_t *Bs = ring[S].b;
    const float *Ss = ring[S].s;
    i32x8 bfr[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
        const i32x4 lo = *(const i32x4 *)&Bs[w.b_rd + cb * 2048];
        const i32x4 hi = *(const i32x4 *)&Bs[w.b_rd + cb * 2048 + 1024];
        bfr[cb] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        if (!GUARD || rb < nrb) {
            const i32x4 lo = *(const i32x4 *)&As[w.a_rd0 + rb * 16 * kGrpB];
            const i32x4 hi = *(const i32x4 *)&As[w.a_rd1 + rb * 16 * kGrpB];
            const i32x8 af = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            const f32x4 sa = *(const f32x4 *)&Ss[w.s_rd + rb * 16];
            f32x4 tq[4];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb)
                tq[cb] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bfr[cb], (f32x4){}, 0, 0,
                                                                          0, 127, 0, 127);
            const f32x4 s = sa * sb;
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) acc[rb][cb] = tq[cb] * s + acc[rb][cb];
        }
    }
}

}  // namespace

// RB = 8: 256-row tiles over the groups of more than kSmallRows rows (every
// group with large_all).  RB = 6: one 192-row tile per group of 1..kSmallRows
// rows, with the row blocks past the group's end skipped.
template <bool SWIGLU, int RB>
__global__ __launch_bounds__(kThreads8, 1)
void k_gemm_fp8(GemmArgs a, int32_t lds_rows_routed, int32_t lds_rows_shared)
{
    constexpr bool kSmall = RB < 8;
    constexpr int kWRows = 16 * RB;                     // rows per wave
    constexpr int kTRows = 2 * kWRows;                  // rows per tile
    static_assert(!kSmall || kTRows == kSmallRows, "small tiles hold a whole small group");
    __shared__ __attribute__((aligned(1024))) uint8_t lds_a0[kStage8];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_b0[kStage8];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_a1[kStage8];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_b1[kStage8];
    __shared__ __attribute__((aligned(256))) float lds_s0[kBM];
    __shared__ __attribute__((aligned(256))) float lds_s1[kBM];
    const Ring8 ring[2] = {{lds_a0, lds_b0, lds_s0}, {lds_a1, lds_b1, lds_s1}};

    const int tid = threadIdx.x;
    Wave8 w;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = w.lane;
    const int wm = w.wave >> 2, wn = w.wave & 3;        // 2 x 4 waves, 128 x 64 each
    const int N = a.N, K = a.K;
    const int NT = (N + kBN - 1) / kBN;
    const int32_t *tbase = kSmall ? a.groups.st_base : a.large_all ? a.groups.mt_base : a.groups.lt_base;
    const int total = __builtin_amdgcn_readfirstlane(tbase[a.G] * NT);
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));
    if (first >= total) return;      // no tile: leave before resolving the weights
    const void *Bw;
    const float *Bsw;
    resolve_weights(a, Bw, Bsw);

    // MFMA operand reads: lane l takes row l % 16 of a 16-row block and the
    // 32 bytes [32 (l / 16), 32 (l / 16) + 32) of its 128-byte group (the
    // weight fragments hold the same K bytes for column l % 16).
    {
        const int r = lane & 15, swz = (r >> 1) & 7, c0 = 2 * (lane >> 4);
        w.a_rd0 = (wm * kWRows + r) * kGrpB + ((c0 ^ swz) << 4);
        w.a_rd1 = (wm * kWRows + r) * kGrpB + (((c0 + 1) ^ swz) << 4);
        w.b_rd = wn * 4 * 2048 + lane * 16;
        w.s_rd = wm * kWRows + 4 * (lane >> 4);
    }
    // token fills: lane l covers row 32 w + 8 i + l / 8, physical chunk l % 8;
    // ((row / 2) % 8) = (4 (i % 2) + l / 16) % 8
    const int frow = w.wave * 32 + (lane >> 3);
    const int fch_even = ((lane & 7) ^ ((lane >> 4) & 7)) << 4;
    const int fch_odd = ((lane & 7) ^ ((4 + (lane >> 4)) & 7)) << 4;

    for (int L = first; L < total; L += P) {
        int g, mt, nt;
        if constexpr (kSmall) {
            // tile L: j-th small group, column tile nt
            const int j = L / NT;
            nt = L - j * NT;
            mt = 0;
            int lo = 0, hi = a.G;               // largest g with st_base[g] <= j
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (tbase[mid] <= j) lo = mid; else hi = mid;
            }
            g = lo;
        } else {
            decode_tile8(L, tbase, a.G, NT, g, mt, nt);
        }
        g = __builtin_amdgcn_readfirstlane(g);
        mt = __builtin_amdgcn_readfirstlane(mt);
        nt = __builtin_amdgcn_readfirstlane(nt);
        const int grows = __builtin_amdgcn_readfirstlane(a.groups.rows[g]);
        const int row0 = __builtin_amdgcn_readfirstlane(a.groups.row0[g]) + mt * kBM;
        const int rows_valid = min(kTRows, grows - mt * kBM);
        const int n0 = nt * kBN;
        const bool sh = (g == a.shared_group);
        const uint8_t *A = (const uint8_t *)(sh ? a.A_shared : a.A_routed) + (int64_t)row0 * K;
        const float *As = (sh ? a.As_shared : a.As_routed) + row0;      // [K/128][ld]
        const uint8_t *B = (const uint8_t *)Bw + ((int64_t)g * N + n0) * K;
        Tile8 t;
        t.KT = K / kGrpB;
        t.s_ld = sh ? lds_rows_shared : lds_rows_routed;
        t.ncb = min(kBN, N - n0) / 16;
        t.cbstride = t.KT * 2048;
        t.ra = rsrc8(A, (int64_t)rows_valid * K);
        t.rb = rsrc8(B, (int64_t)t.ncb * t.cbstride);
        t.rs = rsrc8(As, ((int64_t)(t.KT - 1) * t.s_ld + rows_valid) * 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = frow + 8 * i;
            t.va[i] = r < rows_valid ? r * K + ((i & 1) ? fch_odd : fch_even) : (int)0x80000000u;
        }
        if constexpr (SWIGLU) {
            // [G][f/128][gate, up][K/128]: tile nt covers gate/up scale block nt
            const int f = N / 2;
            t.sbp = Bsw + (((int64_t)g * (f / 128) + nt) * 2 + (wn & 1)) * t.KT;
        } else {
            // [G][N/128][K/128]: wave columns n0 + 64 wn .. + 63
            const int nb = min(2 * nt + (wn >> 1), N / 128 - 1);
            t.sbp = Bsw + ((int64_t)g * (N / 128) + nb) * t.KT;
        }

        f32x4 acc[RB][4];
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = (f32x4){};

        // 16-row blocks of this wave's rows that hold rows of the group
        const int nrb = __builtin_amdgcn_readfirstlane(min(RB, max(0, rows_valid - wm * kWRows + 15) / 16));
        float sb_next = t.sbp[0];
        __builtin_amdgcn_sched_barrier(0);
        fill8(t, ring[0], w.wave, lane, 0);
        for (int kg = 0; kg < t.KT; kg += 2) {
            kgroup8<0, RB, kSmall>(t, w, ring, acc, sb_next, kg, nrb);
            if (kg + 1 < t.KT) kgroup8<1, RB, kSmall>(t, w, ring, acc, sb_next, kg + 1, nrb);
        }
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // the clamped fill issued by the last group
        __syncthreads();                                     // ring idle in every wave

        // Accumulator register i of a 16x16 block holds row 4 (lane / 16) + i
        // and column lane % 16.
        if constexpr (SWIGLU) {
            const int f = N / 2;
            const int s_ld = t.s_ld;
            uint8_t *H = (uint8_t *)(sh ? a.C_shared : a.C_routed);
            float *Hs = (sh ? a.Cs_shared : a.Cs_routed) + (int64_t)nt * s_ld + row0;
            // wave pair p (same rows, same h columns): wn = 2 q (gate) and 2 q + 1 (up)
            const int q = wn >> 1;
            const int p = wm * 2 + q;
            float *xch = (float *)(p == 0 ? lds_a0 : p == 1 ? lds_b0 : p == 2 ? lds_a1 : lds_b1);
            if (wn & 1) {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb)
                        *(f32x4 *)&xch[((rb * 4 + cb) * 64 + lane) * 4] = acc[rb][cb];
            }
            __syncthreads();
            if (!(wn & 1)) {
                // h in fp32 (kept in acc), then this wave's maximum of |h| over
                // its 64 channels of each row, stored for the partner wave
                float *mx = q ? lds_s1 : lds_s0;
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    f32x4 am = (f32x4){};
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        const f32x4 up = *(const f32x4 *)&xch[((rb * 4 + cb) * 64 + lane) * 4];
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float gt = acc[rb][cb][i];
                            const float hv = gt / (1.0f + __expf(-gt)) * up[i];
                            acc[rb][cb][i] = hv;
                            am[i] = fmaxf(am[i], fabsf(hv));
                        }
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
#pragma unroll
                        for (int m = 1; m < 16; m <<= 1) am[i] = fmaxf(am[i], __shfl_xor(am[i], m, 16));
                    }
                    if ((lane & 15) == 0) *(f32x4 *)&mx[w.s_rd + rb * 16] = am;
                }
            }
            __syncthreads();
            uint8_t *stg = lds_a0;   // [256 rows][128 codes]; the up values were read above
            if (!(wn & 1)) {
                const int col = q * 64 + (lane & 15);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    const f32x4 m0 = *(const f32x4 *)&lds_s0[w.s_rd + rb * 16];
                    const f32x4 m1 = *(const f32x4 *)&lds_s1[w.s_rd + rb * 16];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float am = fmaxf(m0[i], m1[i]);
                        const float s = am > 0.0f ? am / 448.0f : 1.0f;   // IEEE division
                        const int row = wm * kWRows + rb * 16 + 4 * (lane >> 4) + i;
                        const uint32_t c4 = e4m3_pack4(acc[rb][0][i] / s, acc[rb][1][i] / s,
                                                       acc[rb][2][i] / s, acc[rb][3][i] / s);
#pragma unroll
                        for (int cb = 0; cb < 4; ++cb)
                            stg[row * kGrpB + col + cb * 16] = (uint8_t)(c4 >> (8 * cb));
                        if (q == 0 && (lane & 15) == 0 && row < rows_valid) Hs[row] = s;
                    }
                }
            }
            __syncthreads();
            for (int c = tid; c < kBM * (kGrpB / 16); c += kThreads8) {
                const int row = c >> 3, ch = c & 7;
                if (row < rows_valid)
                    *(uint4 *)&H[(int64_t)(row0 + row) * f + nt * 128 + ch * 16] =
                        *(const uint4 *)&stg[row * kGrpB + ch * 16];
            }
            __syncthreads();   // the staging area is the next tile's first stage
        } else {
            bf16 *C = (bf16 *)(sh ? a.C_shared : a.C_routed);
            const int col0 = n0 + wn * 64 + (lane & 15);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = wm * kWRows + rb * 16 + 4 * (lane >> 4) + i;
                    if (row < rows_valid) {
                        bf16 *dst = C + (int64_t)(row0 + row) * N;
#pragma unroll
                        for (int cb = 0; cb < 4; ++cb) {
                            const int col = col0 + cb * 16;
                            if (col < N) dst[col] = f2bf(acc[rb][cb][i]);
                        }
                    }
                }
        }
    }
}

hipError_t launch_gemm_fp8(const GemmArgs &a, bool swiglu, int mt_max, int g_max, int num_cus,
                           int32_t lds_rows_routed, int32_t lds_rows_shared, hipStream_t s)
{
    if (mt_max <= 0) return hipSuccess;
    if (a.K % 128 || a.N % 128 || (swiglu && a.N % 256)) return hipErrorNotSupported;
    const int64_t NT = (a.N + kBN - 1) / kBN;
    auto grid_for = [&](int64_t tiles) {
        int grid = num_cus < tiles ? num_cus : (int)tiles;
        if (grid >= 8) grid &= ~7;
        return grid;
    };
    // groups of 1..kSmallRows rows (one 192-row tile each), then the others
    // (either launch may find no tiles)
    if (!a.large_all && g_max > 0) {
        const int grid = grid_for((int64_t)g_max * NT);
        if (swiglu)
            hipLaunchKernelGGL((k_gemm_fp8<true, 6>), dim3(grid), dim3(kThreads8), 0, s, a,
                               lds_rows_routed, lds_rows_shared);
        else
            hipLaunchKernelGGL((k_gemm_fp8<false, 6>), dim3(grid), dim3(kThreads8), 0, s, a,
                               lds_rows_routed, lds_rows_shared);
    }
    const int grid = grid_for((int64_t)mt_max * NT);
    if (swiglu)
        hipLaunchKernelGGL((k_gemm_fp8<true, 8>), dim3(grid), dim3(kThreads8), 0, s, a,
                           lds_rows_routed, lds_rows_shared);
    else
        hipLaunchKernelGGL((k_gemm_fp8<false, 8>), dim3(grid), dim3(kThreads8), 0, s, a,
                           lds_rows_routed, lds_rows_shared);
    return hipGetLastError();
}

}  // namespace moe
