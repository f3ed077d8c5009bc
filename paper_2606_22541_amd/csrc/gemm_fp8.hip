// e4m3 grouped GEMM with DeepSeek-style block scaling (fp8 variant of the
// expert stage): activations carry one fp32 scale per row and 128-channel
// group, weights one fp32 scale per 128x128 block (packed gate/up weights:
// per 32 rows).  Each K step covers exactly one 128-wide scale group:
//
//   tmp  = sum over the step of e4m3(A) * e4m3(B)     (2 x v_mfma 32x32x64 f8)
//   acc += tmp * s_A[row, step] * s_B[col block, step]  (fp32 promotion)
//
// so the block scales are applied exactly once per group in fp32.  The
// hardware's per-32-element power-of-two (E8M0) MFMA scales cannot express
// these fp32 scales and are left at 1.
//
// Tile: 256 rows x 128 columns per workgroup, four wave64s each owning a
// 64 x 128 block (2 x 4 MFMA blocks, fp32 accumulators in VGPRs so the
// promotion can use them).  A, B and the A-scale column of the step stream
// into a double-buffered LDS tile with direct-to-LDS buffer loads; the
// A-scales of X_perm / H are stored transposed ([K/128][rows]) so one step's
// 256 scales are one contiguous 1 KB load.  The SwiGLU epilogue writes
// h = SiLU(gate) * up as bf16; the stage then quantises H per 128 channels.
#include "kernels.h"

namespace moe {

namespace {

constexpr int kBK8 = 128;                       // e4m3 bytes per K step (one scale group)
constexpr int kRowB = 128;                      // LDS row bytes
constexpr int kTM = 256, kTN = 128;
constexpr int kWaves8 = 4;
constexpr int kThreads8 = 64 * kWaves8;
constexpr int kBandM8 = 4;
typedef __attribute__((address_space(3))) void lds_void;

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
    const int band = Lg / (kBandM8 * NT);
    const int r = Lg - band * kBandM8 * NT;
    const int bm = min(kBandM8, Mt - band * kBandM8);
    mt = band * kBandM8 + r % bm;
    nt = r / bm;
}

// rows [8 rb, 8 rb + 8) of a 128-byte-row tile; lane l fills physical chunk
// l % 8 of row 8 rb + l / 8 with global chunk (l % 8) ^ ((row / 2) % 8).
__device__ __forceinline__ void rows_to_lds(__amdgpu_buffer_rsrc_t r, uint8_t *tile, int rb,
                                            int voff_even, int voff_odd, int row_bytes, int soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(tile + rb * 8 * kRowB), 16,
                                             ((rb & 1) ? voff_odd : voff_even) + rb * 8 * row_bytes,
                                             soff, 0, 0);
}

}  // namespace

template <bool SWIGLU>
__global__ __launch_bounds__(kThreads8, 1)
void k_gemm_fp8(GemmArgs a, int32_t lds_rows_routed, int32_t lds_rows_shared)
{
    __shared__ __attribute__((aligned(1024))) uint8_t lds_a[2][kTM * kRowB];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_b[2][kTN * kRowB];
    __shared__ __attribute__((aligned(1024))) float lds_s[2][kTM];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int N = a.N, K = a.K;
    const int NT = (N + kTN - 1) / kTN;
    const int total = __builtin_amdgcn_readfirstlane(a.groups.mt_base[a.G] * NT);
    const int KT = K / kBK8;
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));

    // DMA lane mapping (rows relative to an 8-row block)
    const int drow = lane >> 3;
    const int voff_even = drow * K + (((lane & 7) ^ ((lane >> 4) & 7)) << 4);
    const int voff_odd = drow * K + (((lane & 7) ^ ((4 + (lane >> 4)) & 7)) << 4);
    // MFMA operand reads
    const int rd_row = lane & 31;
    const int rd_hi = lane >> 5;
    const int swz = (rd_row >> 1) & 7;
    const int a_rd = (wave * 64 + rd_row) * kRowB;
    const int b_rd = rd_row * kRowB;

    for (int L = first; L < total; L += P) {
        int g, mt, nt;
        decode_tile8(L, a.groups.mt_base, a.G, NT, g, mt, nt);
        g = __builtin_amdgcn_readfirstlane(g);
        mt = __builtin_amdgcn_readfirstlane(mt);
        nt = __builtin_amdgcn_readfirstlane(nt);
        const int grows = __builtin_amdgcn_readfirstlane(a.groups.rows[g]);
        const int row0 = __builtin_amdgcn_readfirstlane(a.groups.row0[g]) + mt * kTM;
        const int rows_valid = min(kTM, grows - mt * kTM);
        const int n0 = nt * kTN;
        const bool sh = (g == a.shared_group);
        const uint8_t *A = (const uint8_t *)(sh ? a.A_shared : a.A_routed) + (int64_t)row0 * K;
        const float *As = (sh ? a.As_shared : a.As_routed) + row0;       // [K/128][ld]
        const int s_ld = sh ? lds_rows_shared : lds_rows_routed;
        const uint8_t *B = (const uint8_t *)a.B + ((int64_t)g * N + n0) * K;
        const __amdgpu_buffer_rsrc_t ra = rsrc8(A, (int64_t)rows_valid * K);
        const __amdgpu_buffer_rsrc_t rb = rsrc8(B, (int64_t)min(kTN, N - n0) * K);
        const __amdgpu_buffer_rsrc_t rs = rsrc8(As, ((int64_t)(KT - 1) * s_ld + rows_valid) * 4);
        // weight block scales: gate/up packed per 32 rows, down per 128 rows
        const int kb = K / 128;
        const float *Bs = a.Bs + (int64_t)g * (SWIGLU ? (N / 32) : (N / 128)) * kb;

        f32x16 acc[2][4];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = (f32x16){};

        auto issue = [&](int kt, int buf) {
            const int soff = kt * kBK8;
#pragma unroll
            for (int i = 0; i < 8; ++i) rows_to_lds(ra, lds_a[buf], wave * 8 + i, voff_even, voff_odd, K, soff);
#pragma unroll
            for (int i = 0; i < 4; ++i) rows_to_lds(rb, lds_b[buf], wave * 4 + i, voff_even, voff_odd, K, soff);
            // 256 scales = 64 lanes x 16 bytes, contiguous.  The step offset is
            // in the range-checked vector offset, so on the last step the
            // scales of rows past the group read as zero instead of past the
            // end of the scale array.
            if (wave == 0)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)lds_s[buf], 16,
                                                         kt * s_ld * 4 + lane * 16, 0, 0, 0);
        };

        auto step = [&](int kt, int buf) {
            const uint8_t *Al = lds_a[buf];
            const uint8_t *Bl = lds_b[buf];
            // weight scales of this step for the 4 column blocks (wave-uniform)
            float sb[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int n = n0 + nb * 32;
                const int nblk = SWIGLU ? (n >> 5) : (n >> 7);
                sb[nb] = (n < N) ? Bs[nblk * kb + kt] : 0.0f;
            }
            i32x8 bf[4][2];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const int c = kk * 4 + rd_hi * 2;
                    const i32x4 lo = *(const i32x4 *)&Bl[b_rd + nb * 32 * kRowB + (((c) ^ swz) << 4)];
                    const i32x4 hi = *(const i32x4 *)&Bl[b_rd + nb * 32 * kRowB + (((c + 1) ^ swz) << 4)];
                    bf[nb][kk] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                }
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                i32x8 af[2];
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const int c = kk * 4 + rd_hi * 2;
                    const i32x4 lo = *(const i32x4 *)&Al[a_rd + mb * 32 * kRowB + (((c) ^ swz) << 4)];
                    const i32x4 hi = *(const i32x4 *)&Al[a_rd + mb * 32 * kRowB + (((c + 1) ^ swz) << 4)];
                    af[kk] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                }
                // row scales of the 16 accumulator rows of this lane
                float sa[16];
                const int rbase = wave * 64 + mb * 32 + rd_hi * 4;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const f32x4 v = *(const f32x4 *)&lds_s[buf][rbase + j * 8];
                    sa[4 * j + 0] = v[0];
                    sa[4 * j + 1] = v[1];
                    sa[4 * j + 2] = v[2];
                    sa[4 * j + 3] = v[3];
                }
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    f32x16 t = (f32x16){};
                    t = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[0], bf[nb][0], t, 0, 0, 0, 127, 0, 127);
                    t = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[1], bf[nb][1], t, 0, 0, 0, 127, 0, 127);
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[mb][nb][r] += t[r] * (sa[r] * sb[nb]);
                }
            }
        };

        issue(0, 0);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        for (int kt = 0; kt < KT; kt += 2) {     // K/128 is even or odd: guard the second half
            if (kt + 1 < KT) issue(kt + 1, 1);
            __builtin_amdgcn_sched_barrier(0);
            step(kt, 0);
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (kt + 1 >= KT) break;
            if (kt + 2 < KT) issue(kt + 2, 0);
            __builtin_amdgcn_sched_barrier(0);
            step(kt + 1, 1);
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
        }

        // Epilogue (bf16 out), register r of a 32x32 block = row 8 (r/4) + 4 (lane/32) + r%4.
        bf16 *C = (bf16 *)(sh ? a.C_shared : a.C_routed);
        if constexpr (SWIGLU) {
            const int f = N / 2;
            const int f0 = nt * (kTN / 2) + (lane & 31);
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int lr = wave * 64 + mb * 32 + (r >> 2) * 8 + rd_hi * 4 + (r & 3);
                    if (lr < rows_valid) {
                        bf16 *dst = C + (int64_t)(row0 + lr) * f + f0;
#pragma unroll
                        for (int p = 0; p < 2; ++p) {
                            const float gt = acc[mb][2 * p][r];
                            const float up = acc[mb][2 * p + 1][r];
                            dst[p * 32] = f2bf(gt / (1.0f + __expf(-gt)) * up);
                        }
                    }
                }
        } else {
            const int c0 = n0 + (lane & 31);
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int lr = wave * 64 + mb * 32 + (r >> 2) * 8 + rd_hi * 4 + (r & 3);
                    if (lr < rows_valid) {
                        bf16 *dst = C + (int64_t)(row0 + lr) * N;
#pragma unroll
                        for (int nb = 0; nb < 4; ++nb) {
                            const int col = c0 + nb * 32;
                            if (col < N) dst[col] = f2bf(acc[mb][nb][r]);
                        }
                    }
                }
        }
    }
}

hipError_t launch_gemm_fp8(const GemmArgs &a, bool swiglu, int mt_max, int num_cus,
                           int32_t lds_rows_routed, int32_t lds_rows_shared, hipStream_t s)
{
    if (mt_max <= 0) return hipSuccess;
    if (a.K % 128) return hipErrorNotSupported;
    const int64_t tiles = (int64_t)mt_max * ((a.N + kTN - 1) / kTN);
    int grid = num_cus < tiles ? num_cus : (int)tiles;
    if (grid >= 8) grid &= ~7;
    if (swiglu)
        hipLaunchKernelGGL(k_gemm_fp8<true>, dim3(grid), dim3(kThreads8), 0, s, a, lds_rows_routed,
                           lds_rows_shared);
    else
        hipLaunchKernelGGL(k_gemm_fp8<false>, dim3(grid), dim3(kThreads8), 0, s, a, lds_rows_routed,
                           lds_rows_shared);
    return hipGetLastError();
}

}  // namespace moe
