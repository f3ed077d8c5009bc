// Weighted combine back to token order (section 3.2.2: the k expert results
// of a token are reduced with its routing weights at the receiver).
//
// out[t] = base_t + sum_{j ascending, row_of_slot[t*k+j] >= 0} w[t][j] * Y[row]
// accumulated in fp32 and rounded once to bf16.  Each thread owns whole
// 8-channel chunks of one token, so the sum order is fixed and there are no
// atomics: the result is bit-identical across runs and stream layouts.
#include "kernels.h"

namespace moe {

// One workgroup per token (grid-stride past 128 per CU).  The token's k row indices and
// weights are uniform loads; thread tid owns the 16-byte channel chunks
// c = c0 + 256 u + tid.  Loads use indices clamped into the row so that they
// are unconditional (a guarded load would be issued and waited for one at a
// time); only the stores are guarded.  A scheduling barrier after each batch
// of loads keeps the compiler from interleaving them with the conversions.
constexpr int kCombineThreads = 256;
constexpr int kUnroll = 4;

// A 16-byte load that marks its line streaming (read once).  Used for the
// shared expert's rows and, in accumulate mode, the old output rows: both are
// read exactly once and at the EP8 share (T = 16384) they are 235 MB each,
// more than the 256 MB last-level cache holds beside them.  The expert rows
// (Y_perm) keep ordinary loads: the down GEMM has just written them and they
// are often still cached (measured: streaming loads of Y_perm made the
// combine of the EP32 share at T = 32768 5% slower, those of the shared rows
// made the EP8 share's 10% faster).
__device__ __forceinline__ uint4 nt_load(const uint4 *p)
{
    const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
    return *(const uint4 *)&v;
}

__device__ __forceinline__ void acc_row(float (&acc)[8], const uint4 &v, float wj)
{
    const bf16 *vb = (const bf16 *)&v;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += wj * bf2f(vb[i]);
}

__global__ __launch_bounds__(kCombineThreads)
void k_combine(const uint4 *__restrict__ y, const uint4 *__restrict__ ysh,
               const int32_t *__restrict__ row_of_slot, const float *__restrict__ w,
               uint4 *__restrict__ out, int32_t T, int32_t k, int32_t vecs, int32_t accumulate)
{
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        int nloc = 0;
        for (int j = 0; j < k; ++j) nloc += (row_of_slot[(int64_t)t * k + j] >= 0);
        if (accumulate && nloc == 0 && ysh == nullptr) continue;   // untouched
        uint4 *orow = out + (int64_t)t * vecs;
        const uint4 *shrow = ysh ? ysh + (int64_t)t * vecs : nullptr;
        for (int c0 = 0; c0 < vecs; c0 += kCombineThreads * kUnroll) {
            int cc[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                cc[u] = min(c0 + u * kCombineThreads + (int)threadIdx.x, vecs - 1);
            float acc[kUnroll][8];
            if (accumulate) {
                uint4 o[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) o[u] = nt_load(&orow[cc[u]]);
                __builtin_amdgcn_sched_barrier(0);   // all loads issued first
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const bf16 *ob = (const bf16 *)&o[u];
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[u][i] = bf2f(ob[i]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[u][i] = 0.0f;
            }
            if (shrow) {
                uint4 v[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) v[u] = nt_load(&shrow[cc[u]]);
                __builtin_amdgcn_sched_barrier(0);   // all loads issued first
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) acc_row(acc[u], v[u], 1.0f);
            }
            for (int j = 0; j < k; ++j) {                      // j ascending
                const int r = row_of_slot[(int64_t)t * k + j];
                if (r < 0) continue;
                const float wj = w[(int64_t)t * k + j];
                const uint4 *yrow = y + (int64_t)r * vecs;
                uint4 v[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) v[u] = yrow[cc[u]];
                __builtin_amdgcn_sched_barrier(0);   // all loads issued first
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) acc_row(acc[u], v[u], wj);
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int c = c0 + u * kCombineThreads + threadIdx.x;
                if (c < vecs) {
                    uint4 o;
                    bf16 *ob = (bf16 *)&o;
#pragma unroll
                    for (int i = 0; i < 8; ++i) ob[i] = f2bf(acc[u][i]);
                    // the output is not read again by the stage: stream it to
                    // HBM now rather than leave dirty lines for the next
                    // micro-batch's weight stream to evict
                    __builtin_nontemporal_store(*(const u32x4 *)&o, (u32x4 *)&orow[c]);
                }
            }
        }
    }
}

hipError_t launch_combine(const CombineArgs &a, int num_cus, hipStream_t s)
{
    if (a.T <= 0) return hipSuccess;
    const int vecs = a.d / 8;
    // One workgroup per token: with a grid-stride loop over 16 workgroups
    // per CU the EP32 share at T = 32768 (mostly rows of zeros: 470 MB of
    // non-temporal stores, 116 MB of loads) ran at 5.2 TB/s; one workgroup
    // per token at 6.3 TB/s (the hardware hands out the next token as soon
    // as a workgroup retires, and the stores in flight stay close together).
    int64_t grid = a.T;
    const int64_t cap = (int64_t)num_cus * 128;
    if (grid > cap) grid = cap;
    hipLaunchKernelGGL(k_combine, dim3((unsigned)grid), dim3(kCombineThreads), 0, s,
                       (const uint4 *)a.y_perm, (const uint4 *)a.y_shared, a.row_of_slot, a.w,
                       (uint4 *)a.out, a.T, a.k, vecs, a.accumulate);
    return hipGetLastError();
}

}  // namespace moe
