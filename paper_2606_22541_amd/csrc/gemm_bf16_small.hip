// bf16 grouped GEMM for small groups (1..kSmallRows rows per expert).
//
// With few rows per expert the grouped GEMM is bound by streaming the
// experts' weights from HBM (at T=4096 of a DeepSeek-V3 EP32 share each of
// the 8 local experts sees ~130 rows and ~88 MB of weights).  The design
// aims at reading every weight byte once, from all CUs at once:
//  * one tile = all rows of a group (up to 192) x 128 weight columns, so
//    each weight panel is read exactly once and there are E_loc x N/128
//    tiles (256 at T=4096) -- enough for every CU;
//  * four wave64s each own 32 weight columns and all row blocks; MFMAs and
//    row fills are skipped for 32-row blocks past the group's end;
//  * a K step (64 wide) is only ~20 MFMAs per wave, so both operands are
//    fetched three steps ahead through 4-deep direct-to-LDS rings (token
//    rows: 4 x 24 KB, weights: 4 x 16 KB); the K loop is unrolled by 4 so
//    every ring index is a compile-time constant and each buffer is its own
//    LDS object, which lets the compiler see that in-flight fills never
//    alias the buffer being read; the wait at each step is computed exactly
//    from the loads this wave issued after the step's own;
//  * SwiGLU: packed gate/up columns interleave by 16, so a wave's 32
//    columns are 16 gate and 16 up columns of the same h columns, paired
//    across lanes l and l ^ 16.
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

// 8 rows x 128 B starting at row 8 rb; lane l -> row 8 rb + l / 8, physical
// chunk l % 8 <- global chunk (l % 8) ^ ((row / 2) % 8).
__device__ __forceinline__ void rows8_to_lds(__amdgpu_buffer_rsrc_t r, bf16 *tile, int rb,
                                             int voff_even, int voff_odd, int row_bytes, int soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_s *)(tile + rb * 8 * kRowEs), 16,
                                             ((rb & 1) ? voff_odd : voff_even) + rb * 8 * row_bytes,
                                             soff, 0, 0);
}

// s_waitcnt vmcnt(n) for a wave-uniform n in [0, 31] (larger n: 31).
__device__ __forceinline__ void wait_vmcnt(int n)
{
    constexpr int E = (7 << 4) | (15 << 8);          // expcnt, lgkmcnt: no wait
#define MOE_WAIT_CASE(v) case v: __builtin_amdgcn_s_waitcnt((v) | E); break;
    switch (n) {
        MOE_WAIT_CASE(0) MOE_WAIT_CASE(1) MOE_WAIT_CASE(2) MOE_WAIT_CASE(3)
        MOE_WAIT_CASE(4) MOE_WAIT_CASE(5) MOE_WAIT_CASE(6) MOE_WAIT_CASE(7)
        MOE_WAIT_CASE(8) MOE_WAIT_CASE(9) MOE_WAIT_CASE(10) MOE_WAIT_CASE(11)
        MOE_WAIT_CASE(12) MOE_WAIT_CASE(13) MOE_WAIT_CASE(14) MOE_WAIT_CASE(15)
    default:
        if (n >= 31) __builtin_amdgcn_s_waitcnt((31 & 15) | ((31 >> 4) << 14) | E);
        else if (n >= 24) __builtin_amdgcn_s_waitcnt((24 & 15) | ((24 >> 4) << 14) | E);
        else if (n >= 20) __builtin_amdgcn_s_waitcnt((20 & 15) | ((20 >> 4) << 14) | E);
        else __builtin_amdgcn_s_waitcnt((16 & 15) | ((16 >> 4) << 14) | E);
        break;
    }
#undef MOE_WAIT_CASE
}

}  // namespace

struct SmallTile {
    __amdgpu_buffer_rsrc_t ra, rb;
    bf16 *C;
    int row0, rows_valid, n0, nrb, a_cnt, N, K, KT;
};

struct SmallLds {
    bf16 *a[kRing];   // token-row tiles, 192 rows x 64 bf16 each
    bf16 *b[kRing];   // weight tiles, 128 rows x 64 bf16 each
};

// Fills of step j: token rows into a[j % 4], then weights into b[j % 4].
template <int NMB, int I>
__device__ __forceinline__ void fill_step(const SmallTile &t, const SmallLds &l, int j, int wave,
                                          int voff_even, int voff_odd)
{
    if (j >= t.KT) return;
#pragma unroll
    for (int i = 0; i < NMB; ++i) {
        const int blk = wave + 4 * i;
        if (blk < t.nrb)
            rows8_to_lds(t.ra, l.a[I], blk, voff_even, voff_odd, t.K * 2, j * kBKs * 2);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
        rows8_to_lds(t.rb, l.b[I], wave * 4 + i, voff_even, voff_odd, t.K * 2, j * kBKs * 2);
}

// One K step with compile-time ring index I = k % 4.
template <int NMB, int I>
__device__ __forceinline__ void small_step(const SmallTile &t, const SmallLds &l,
                                           f32x16 (&acc)[NMB], int k, int wave, int lane,
                                           int voff_even, int voff_odd)
{
    // Fills are issued in step order (rows j, weights j, rows j+1, ...) and
    // steps k+1 and k+2 are the ones already issued after step k's.
    wait_vmcnt((t.a_cnt + 4) * min(2, t.KT - 1 - k));
    __builtin_amdgcn_s_barrier();          // every wave's fills of step k landed; step k-1 read
    fill_step<NMB, (I + 3) & 3>(t, l, k + 3, wave, voff_even, voff_odd);
    __builtin_amdgcn_sched_barrier(0);

    const int rd_row = lane & 31;
    const int rd_hi = lane >> 5;
    const int swz = (rd_row >> 1) & 7;
    const bf16 *As = l.a[I];
    const bf16 *Bs = l.b[I];
    // Fragments of sub-step kk+1 are read while the MFMAs of kk run.
    auto read = [&](int kk, bf16x8 (&af)[NMB], bf16x8 &bfr) {
        const int ch = ((kk * 2 + rd_hi) ^ swz) << 3;
        bfr = *(const bf16x8 *)&Bs[(wave * 32 + rd_row) * kRowEs + ch];
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
            af[mb] = *(const bf16x8 *)&As[(mb * 32 + rd_row) * kRowEs + ch];
    };
    auto mma = [&](const bf16x8 (&af)[NMB], const bf16x8 &bfr) {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr, acc[mb], 0, 0, 0);
    };
    bf16x8 a0[NMB], a1[NMB], b0, b1;
    read(0, a0, b0);
    read(1, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    mma(a0, b0);
    read(2, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    mma(a1, b1);
    read(3, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    mma(a0, b0);
    mma(a1, b1);
    __builtin_amdgcn_sched_barrier(0);
}

// One tile with NMB 32-row blocks: K loop and epilogue, fully unrolled over
// the row blocks so no accumulator crosses a branch.
template <bool SWIGLU, int NMB>
__device__ __forceinline__ void run_small_tile(const SmallTile &t, const SmallLds &l, int wave,
                                               int lane, int voff_even, int voff_odd)
{
    f32x16 acc[NMB];
#pragma unroll
    for (int i = 0; i < NMB; ++i) acc[i] = (f32x16){};

    fill_step<NMB, 0>(t, l, 0, wave, voff_even, voff_odd);
    fill_step<NMB, 1>(t, l, 1, wave, voff_even, voff_odd);
    fill_step<NMB, 2>(t, l, 2, wave, voff_even, voff_odd);
    // K is a multiple of 128, so KT is even: groups of 4 steps, then 2.
    int k = 0;
    for (; k + 4 <= t.KT; k += 4) {
        small_step<NMB, 0>(t, l, acc, k, wave, lane, voff_even, voff_odd);
        small_step<NMB, 1>(t, l, acc, k + 1, wave, lane, voff_even, voff_odd);
        small_step<NMB, 2>(t, l, acc, k + 2, wave, lane, voff_even, voff_odd);
        small_step<NMB, 3>(t, l, acc, k + 3, wave, lane, voff_even, voff_odd);
    }
    if (k < t.KT) {
        small_step<NMB, 0>(t, l, acc, k, wave, lane, voff_even, voff_odd);
        small_step<NMB, 1>(t, l, acc, k + 1, wave, lane, voff_even, voff_odd);
    }
    __syncthreads();   // all LDS reads done before the next tile's fills

    // Epilogue: register r of a 32x32 block = row 8 (r/4) + 4 (lane/32) + r%4,
    // column lane % 32 of this wave's 32 columns.
    const int rd_hi = lane >> 5;
    if constexpr (SWIGLU) {
        const int f = t.N / 2;
        const bool gl = (lane & 16) == 0;
        const int hc = (t.n0 + wave * 32) / 2 + (lane & 15);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float v = acc[mb][r];
                const float up = __shfl_xor(v, 16);
                const int lr = mb * 32 + (r >> 2) * 8 + rd_hi * 4 + (r & 3);
                if (gl && lr < t.rows_valid)
                    t.C[(int64_t)(t.row0 + lr) * f + hc] = f2bf(v / (1.0f + __expf(-v)) * up);
            }
    } else {
        const int col = t.n0 + wave * 32 + (lane & 31);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int lr = mb * 32 + (r >> 2) * 8 + rd_hi * 4 + (r & 3);
                if (lr < t.rows_valid && col < t.N)
                    t.C[(int64_t)(t.row0 + lr) * t.N + col] = f2bf(acc[mb][r]);
            }
    }
}

template <bool SWIGLU>
__global__ __launch_bounds__(kThreadsS, 1)
void k_gemm_bf16_small(GemmArgs a)
{
    __shared__ __attribute__((aligned(1024))) bf16 lds_a0[kSmallRows * kRowEs];   // 4 x 24 KB
    __shared__ __attribute__((aligned(1024))) bf16 lds_a1[kSmallRows * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a2[kSmallRows * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_a3[kSmallRows * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b0[kTNs * kRowEs];         // 4 x 16 KB
    __shared__ __attribute__((aligned(1024))) bf16 lds_b1[kTNs * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b2[kTNs * kRowEs];
    __shared__ __attribute__((aligned(1024))) bf16 lds_b3[kTNs * kRowEs];
    const SmallLds l{{lds_a0, lds_a1, lds_a2, lds_a3}, {lds_b0, lds_b1, lds_b2, lds_b3}};

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int N = a.N, K = a.K;
    const int NT = (N + kTNs - 1) / kTNs;
    const int total = __builtin_amdgcn_readfirstlane(a.groups.st_base[a.G] * NT);
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));

    const int drow = lane >> 3;
    const int voff_even = drow * K * 2 + (((lane & 7) ^ ((lane >> 4) & 7)) << 4);
    const int voff_odd = drow * K * 2 + (((lane & 7) ^ ((4 + (lane >> 4)) & 7)) << 4);

    for (int L = first; L < total; L += P) {
        // tile L: j-th small group, column block nt (an expert's column
        // blocks are consecutive, so one XCD shares its token rows in L2)
        const int j = L / NT;
        const int nt = L - j * NT;
        int lo = 0, hi = a.G;                    // largest g with st_base[g] <= j
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.groups.st_base[mid] <= j) lo = mid; else hi = mid;
        }
        SmallTile t;
        const int g = __builtin_amdgcn_readfirstlane(lo);
        t.rows_valid = __builtin_amdgcn_readfirstlane(a.groups.rows[g]);
        t.row0 = __builtin_amdgcn_readfirstlane(a.groups.row0[g]);
        t.n0 = nt * kTNs;
        t.nrb = (t.rows_valid + 7) >> 3;
        t.a_cnt = max(0, (t.nrb - wave + 3) >> 2);   // row fills this wave issues per step
        t.N = N;
        t.K = K;
        t.KT = K / kBKs;
        const bool sh = (g == a.shared_group);
        const bf16 *A = (const bf16 *)(sh ? a.A_shared : a.A_routed) + (int64_t)t.row0 * K;
        const bf16 *B = (const bf16 *)a.B + ((int64_t)g * N + t.n0) * K;
        t.ra = rsrc_s(A, (int64_t)t.rows_valid * K * 2);
        t.rb = rsrc_s(B, (int64_t)min(kTNs, N - t.n0) * K * 2);
        t.C = (bf16 *)(sh ? a.C_shared : a.C_routed);
        switch ((t.rows_valid + 31) >> 5) {   // 32-row blocks holding rows: 1..6
        case 1: run_small_tile<SWIGLU, 1>(t, l, wave, lane, voff_even, voff_odd); break;
        case 2: run_small_tile<SWIGLU, 2>(t, l, wave, lane, voff_even, voff_odd); break;
        case 3: run_small_tile<SWIGLU, 3>(t, l, wave, lane, voff_even, voff_odd); break;
        case 4: run_small_tile<SWIGLU, 4>(t, l, wave, lane, voff_even, voff_odd); break;
        case 5: run_small_tile<SWIGLU, 5>(t, l, wave, lane, voff_even, voff_odd); break;
        default: run_small_tile<SWIGLU, 6>(t, l, wave, lane, voff_even, voff_odd); break;
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
