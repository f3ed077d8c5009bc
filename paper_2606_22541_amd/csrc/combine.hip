// Weighted combine back to token order (section 3.2.2: the k expert results
// of a token are reduced with its routing weights at the receiver).
//
// out[t] = base_t + sum_{j ascending, row_of_slot[t*k+j] >= 0} w[t][j] * Y[row]
// accumulated in fp32 and rounded once to bf16.  Each thread owns 8
// consecutive channels of one token, so the sum order is fixed and there are
// no atomics: the result is bit-identical across runs and stream layouts.
#include "kernels.h"

namespace moe {

__global__ __launch_bounds__(256)
void k_combine(const uint4 *__restrict__ y, const uint4 *__restrict__ ysh,
               const int32_t *__restrict__ row_of_slot, const float *__restrict__ w,
               uint4 *__restrict__ out, int32_t T, int32_t k, int32_t vecs, int32_t accumulate)
{
    const int64_t total = (int64_t)T * vecs;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * 256) {
        const int t = (int)(q / vecs);
        const int c = (int)(q - (int64_t)t * vecs);
        float acc[8];
        bool touched = false;
        if (accumulate) {
            uint4 o = out[q];
            const bf16 *ob = (const bf16 *)&o;
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = bf2f(ob[i]);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
        }
        if (ysh != nullptr) {
            uint4 v = ysh[q];
            const bf16 *vb = (const bf16 *)&v;
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] += bf2f(vb[i]);
            touched = true;
        }
        for (int j = 0; j < k; ++j) {
            const int r = row_of_slot[(int64_t)t * k + j];
            if (r < 0) continue;
            const float wj = w[(int64_t)t * k + j];
            uint4 v = y[(int64_t)r * vecs + c];
            const bf16 *vb = (const bf16 *)&v;
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] += wj * bf2f(vb[i]);
            touched = true;
        }
        if (!accumulate || touched) {
            uint4 o;
            bf16 *ob = (bf16 *)&o;
#pragma unroll
            for (int i = 0; i < 8; ++i) ob[i] = f2bf(acc[i]);
            out[q] = o;
        }
    }
}

hipError_t launch_combine(const CombineArgs &a, int num_cus, hipStream_t s)
{
    if (a.T <= 0) return hipSuccess;
    const int vecs = a.d / 8;
    const int64_t total = (int64_t)a.T * vecs;
    int64_t grid = (total + 255) / 256;
    const int64_t cap = (int64_t)num_cus * 16;
    if (grid > cap) grid = cap;
    hipLaunchKernelGGL(k_combine, dim3((unsigned)grid), dim3(256), 0, s, (const uint4 *)a.y_perm,
                       (const uint4 *)a.y_shared, a.row_of_slot, a.w, (uint4 *)a.out, a.T, a.k,
                       vecs, a.accumulate);
    return hipGetLastError();
}

}  // namespace moe
