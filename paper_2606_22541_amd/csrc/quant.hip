// fp8 helpers: the sender-side activation quantiser and the create-time
// weight packing kernels.
#include "kernels.h"

namespace moe {

// One group of 128 channels is handled by 16 lanes, 8 channels each.
__global__ __launch_bounds__(256)
void k_quantize_fp8(const uint4 *__restrict__ x, int32_t n_rows, const int32_t *__restrict__ n_rows_dev,
                    int32_t groups_per_row, uint2 *__restrict__ xq, float *__restrict__ xs,
                    int32_t scale_ld)
{
    const int rows = n_rows_dev ? *n_rows_dev : n_rows;
    const int64_t n_groups = (int64_t)rows * groups_per_row;
    const int sub = threadIdx.x & 15;
    for (int64_t gi = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 4; gi < n_groups;
         gi += ((int64_t)gridDim.x * 256) >> 4) {
        uint4 v = x[gi * 16 + sub];
        const bf16 *vb = (const bf16 *)&v;
        float f[8];
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            f[i] = bf2f(vb[i]);
            amax = fmaxf(amax, fabsf(f[i]));
        }
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 16));
        const float s = amax > 0.0f ? amax / 448.0f : 1.0f;   // IEEE division
        uint2 q;
        q.x = e4m3_pack4(f[0] / s, f[1] / s, f[2] / s, f[3] / s);
        q.y = e4m3_pack4(f[4] / s, f[5] / s, f[6] / s, f[7] / s);
        xq[gi * 16 + sub] = q;
        if (sub == 0) {
            const int64_t row = gi / groups_per_row;
            const int g = (int)(gi - row * groups_per_row);
            if (scale_ld > 0) xs[(int64_t)g * scale_ld + row] = s;
            else xs[gi] = s;
        }
    }
}

hipError_t launch_quantize_fp8(const void *x, int32_t n_rows, const int32_t *n_rows_dev,
                               int32_t d, void *xq, float *xs, int32_t scale_ld, int num_cus,
                               hipStream_t s)
{
    if (n_rows <= 0) return hipSuccess;
    const int gpr = d / 128;
    const int64_t threads = (int64_t)n_rows * gpr * 16;
    int64_t grid = (threads + 255) / 256;
    if (grid > (int64_t)num_cus * 16) grid = (int64_t)num_cus * 16;
    hipLaunchKernelGGL(k_quantize_fp8, dim3((unsigned)grid), dim3(256), 0, s, (const uint4 *)x,
                       n_rows, n_rows_dev, gpr, (uint2 *)xq, xs, scale_ld);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight packing (create time only).
// ---------------------------------------------------------------------------
// Gate/up weight scales of the fp8 path: [m][f/128][gate, up][d/128], so
// that a 256-column tile of the packed matrix (gate and up rows
// [128 t, 128 t + 128), interleaved by 16) finds both of its scale rows
// next to each other.
__global__ void k_pack_gate_up_scales(const float *__restrict__ gs, const float *__restrict__ us,
                                      float *__restrict__ ps, int32_t n_mats, int32_t f,
                                      int32_t kblocks)
{
    const int fb_n = f / 128;
    const int64_t total = (int64_t)n_mats * fb_n * 2 * kblocks;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int kb = (int)(q % kblocks);
        int64_t rest = q / kblocks;
        const int u = (int)(rest & 1);
        rest >>= 1;
        const int fb = (int)(rest % fb_n);
        const int m = (int)(rest / fb_n);
        const float *src = u ? us : gs;
        ps[q] = src[((int64_t)m * fb_n + fb) * kblocks + kb];
    }
}

hipError_t launch_pack_gate_up_scales(const float *gs, const float *us, float *packed_s,
                                      int32_t n_mats, int32_t f, int32_t d, hipStream_t s)
{
    hipLaunchKernelGGL(k_pack_gate_up_scales, dim3(256), dim3(256), 0, s, gs, us, packed_s,
                       n_mats, f, d / 128);
    return hipGetLastError();
}

// e4m3 weights in the fragment order of v_mfma_scale_f32_16x16x128_f8f6f4.
// Row n (of N) and byte k (of K) of matrix m go to 16-byte chunk
// ((m * N/16 + n/16) * K/128 + k/128) * 128 + 64 h + lane, byte k % 16, with
// lane = n % 16 + 16 * ((k % 128) / 32) and h = (k / 16) % 2: a 16-column x
// 128-K fragment is 2 KB of consecutive memory, two 1 KB halves of one
// 16-byte chunk per lane, and lane l's 32 bytes are the K bytes
// [32 (l / 16), 32 (l / 16) + 32) of the group for column l % 16 (the token
// rows are read with the same K assignment).  With `up` given, packed row n
// interleaves gate and up rows in blocks of `il` (N = 2 f rows per matrix).
__global__ void k_pack_frag_fp8(const uint4 *__restrict__ gate, const uint4 *__restrict__ up,
                                uint4 *__restrict__ dst, int32_t n_mats, int32_t N, int32_t K,
                                int32_t il)
{
    const int64_t total = (int64_t)n_mats * N * (K / 16);
    const int kgs = K / 128, nbs = N / 16, row_vecs = K / 16;
    const int rows_per_src = up ? N / 2 : N;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int lane = (int)(q & 63);
        const int h = (int)((q >> 6) & 1);
        int64_t rest = q >> 7;
        const int kg = (int)(rest % kgs);
        rest /= kgs;
        const int nb = (int)(rest % nbs);
        const int m = (int)(rest / nbs);
        const int n = nb * 16 + (lane & 15);
        const int kv = kg * 8 + 2 * (lane >> 4) + h;       // 16-byte chunk along K
        const uint4 *src = gate;
        int srow = n;
        if (up) {
            const int b = n / (2 * il), i = n % (2 * il);
            src = (i < il) ? gate : up;
            srow = b * il + (i % il);
        }
        dst[q] = src[((int64_t)m * rows_per_src + srow) * row_vecs + kv];
    }
}

hipError_t launch_pack_frag_fp8(const void *gate, const void *up, void *dst, int32_t n_mats,
                                int32_t N, int32_t K, int32_t interleave, hipStream_t s)
{
    hipLaunchKernelGGL(k_pack_frag_fp8, dim3(4096), dim3(256), 0, s, (const uint4 *)gate,
                       (const uint4 *)up, (uint4 *)dst, n_mats, N, K, interleave);
    return hipGetLastError();
}

// bf16 weights in MFMA fragments, panel order.  Row n (of N) and column k
// (of K) of matrix m go to chunk `lane` = n % 32 + 32 ((k / 8) % 2) of the
// fragment of column block n / 32 and K sub-step k / 16, element k % 8: the 64
// lanes' operands of one 32-column x 16-K B fragment of
// v_mfma_f32_32x32x16_bf16 are 1 KB of consecutive memory.  Blocks form
// panels of 8 (256 columns; the last panel may hold fewer), and a panel
// stores each 32-wide K step's fragments together ([K step][block][sub-step]),
// so a GEMM tile's weights for one K step are one contiguous run.  With `up`
// given, packed row n interleaves gate and up rows in blocks of `il` (N = 2 f
// rows per matrix).
__global__ void k_pack_frag_bf16(const uint4 *__restrict__ gate, const uint4 *__restrict__ up,
                                 uint4 *__restrict__ dst, int32_t n_mats, int32_t N, int32_t K,
                                 int32_t il)
{
    const int64_t total = (int64_t)n_mats * N * (K / 8);
    const int kc = K / 16, nbs = N / 32, row_vecs = K / 8;
    const int rows_per_src = up ? N / 2 : N;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int lane = (int)(q & 63);
        int64_t rest = q >> 6;
        const int kk = (int)(rest % kc);
        rest /= kc;
        const int nb = (int)(rest % nbs);
        const int m = (int)(rest / nbs);
        const int n = nb * 32 + (lane & 31);
        const int kv = kk * 2 + (lane >> 5);           // 8-element chunk along K
        const uint4 *src = gate;
        int srow = n;
        if (up) {
            const int b = n / (2 * il), i = n % (2 * il);
            src = (i < il) ? gate : up;
            srow = b * il + (i % il);
        }
        // panel order: 256-column tile t = nb / 8 holds, per 32-wide K step,
        // its column blocks' two 1 KB fragments contiguously
        const int t = nb >> 3, lb = nb & 7, ncb = min(8, nbs - 8 * t);
        const int64_t off = ((int64_t)m * nbs + 8 * t) * (int64_t)kc * 64       // tiles before
                            + (int64_t)(kk >> 1) * ncb * 128                     // K steps before
                            + (lb * 2 + (kk & 1)) * 64 + lane;
        dst[off] = src[((int64_t)m * rows_per_src + srow) * row_vecs + kv];
    }
}

hipError_t launch_pack_frag_bf16(const void *gate, const void *up, void *dst, int32_t n_mats,
                                 int32_t N, int32_t K, int32_t interleave, hipStream_t s)
{
    hipLaunchKernelGGL(k_pack_frag_bf16, dim3(4096), dim3(256), 0, s, (const uint4 *)gate,
                       (const uint4 *)up, (uint4 *)dst, n_mats, N, K, interleave);
    return hipGetLastError();
}

}  // namespace moe
