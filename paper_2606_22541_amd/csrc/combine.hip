// Weighted combine back to token order (section 3.2.2: the k expert results
// of a token are reduced with its routing weights at the receiver).
//
// out[t] = base_t + sum_{j ascending, row_of_slot[t*k+j] >= 0} w[t][j] * Y[row]
// accumulated in fp32 and rounded once to bf16.  Each lane owns whole 8-
// channel chunks of one token, so the sum order is fixed and there are no
// atomics: the result is bit-identical across runs and stream layouts.
#include "kernels.h"

namespace moe {

// One wave per token.  Lanes 0..k-1 fetch the token's rows and weights once;
// they are broadcast with readlane so the per-slot loop is wave-uniform.
// Each lane then owns 16-byte channel chunks c = lane + 64 i, and up to
// kUnroll chunks are in flight at once.
constexpr int kCombineWaves = 4;
constexpr int kUnroll = 4;

__device__ __forceinline__ void acc_row(float (&acc)[8], const uint4 &v, float wj)
{
    const bf16 *vb = (const bf16 *)&v;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += wj * bf2f(vb[i]);
}

__global__ __launch_bounds__(64 * kCombineWaves)
void k_combine(const uint4 *__restrict__ y, const uint4 *__restrict__ ysh,
               const int32_t *__restrict__ row_of_slot, const float *__restrict__ w,
               uint4 *__restrict__ out, int32_t T, int32_t k, int32_t vecs, int32_t accumulate)
{
    const int lane = threadIdx.x & 63;
    const int gw = blockIdx.x * kCombineWaves + (threadIdx.x >> 6);
    const int nw = gridDim.x * kCombineWaves;
    for (int t = gw; t < T; t += nw) {
        int my_r = -1;
        float my_w = 0.0f;
        if (lane < k) {
            my_r = row_of_slot[(int64_t)t * k + lane];
            my_w = w[(int64_t)t * k + lane];
        }
        int nloc = 0;
        for (int j = 0; j < k; ++j) nloc += (__shfl(my_r, j) >= 0);
        if (accumulate && nloc == 0 && ysh == nullptr) continue;   // untouched
        uint4 *orow = out + (int64_t)t * vecs;
        const uint4 *shrow = ysh ? ysh + (int64_t)t * vecs : nullptr;
        for (int c0 = 0; c0 < vecs; c0 += 64 * kUnroll) {
            float acc[kUnroll][8];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int c = c0 + u * 64 + lane;
                if (accumulate && c < vecs) {
                    const uint4 o = orow[c];
                    const bf16 *ob = (const bf16 *)&o;
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[u][i] = bf2f(ob[i]);
                } else {
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[u][i] = 0.0f;
                }
                if (shrow && c < vecs) acc_row(acc[u], shrow[c], 1.0f);
            }
            for (int j = 0; j < k; ++j) {                      // j ascending
                const int r = __shfl(my_r, j);
                if (r < 0) continue;
                const float wj = __shfl(my_w, j);
                const uint4 *yrow = y + (int64_t)r * vecs;
                uint4 v[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int c = c0 + u * 64 + lane;
                    v[u] = c < vecs ? yrow[c] : make_uint4(0, 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) acc_row(acc[u], v[u], wj);
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int c = c0 + u * 64 + lane;
                if (c < vecs) {
                    uint4 o;
                    bf16 *ob = (bf16 *)&o;
#pragma unroll
                    for (int i = 0; i < 8; ++i) ob[i] = f2bf(acc[u][i]);
                    orow[c] = o;
                }
            }
        }
    }
}

hipError_t launch_combine(const CombineArgs &a, int num_cus, hipStream_t s)
{
    if (a.T <= 0) return hipSuccess;
    const int vecs = a.d / 8;
    int64_t grid = ((int64_t)a.T + kCombineWaves - 1) / kCombineWaves;
    const int64_t cap = (int64_t)num_cus * 8;
    if (grid > cap) grid = cap;
    hipLaunchKernelGGL(k_combine, dim3((unsigned)grid), dim3(64 * kCombineWaves), 0, s,
                       (const uint4 *)a.y_perm, (const uint4 *)a.y_shared, a.row_of_slot, a.w,
                       (uint4 *)a.out, a.T, a.k, vecs, a.accumulate);
    return hipGetLastError();
}

}  // namespace moe
