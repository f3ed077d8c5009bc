// Dispatch of one micro-batch: per-expert histogram, scan, stable counting-sort
// scatter and coalesced row gather.
//
// The per-expert token counts are the metadata the paper's MoE devices receive
// with each batch, and the payload is grouped by expert (section 3.2.1,
// Table 2).  Here the stage derives them itself from the top-k ids.
//
// The order within an expert is ascending slot index s = t*k + j.  It is
// produced without any atomic deciding an order: each workgroup owns a
// contiguous chunk of slots, each wave a contiguous part of the chunk, and
// ranks inside a 64-slot step come from wave ballots, so the result is the
// stable counting sort, bit for bit.
#include "kernels.h"

namespace moe {

// ---------------------------------------------------------------------------
// 1. Histogram over all experts, one row of counts per workgroup.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kDispatchThreads)
void k_hist(const int32_t *__restrict__ ids, int32_t n_slots, int32_t E,
            int32_t *__restrict__ blk_counts, int32_t *__restrict__ err)
{
    __shared__ int32_t h[kMaxExperts];
    for (int e = threadIdx.x; e < E; e += kDispatchThreads) h[e] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kDispatchChunk;
    int bad = 0;
    for (int i = threadIdx.x; i < kDispatchChunk; i += kDispatchThreads) {
        int64_t s = base + i;
        if (s >= n_slots) break;
        int e = ids[s];
        if (e >= 0 && e < E) atomicAdd(&h[e], 1);       // integer counts: order-free
        else if (e != -1) bad = 1;
    }
    if (bad) atomicOr(err, kErrBadId);
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += kDispatchThreads)
        blk_counts[(int64_t)blockIdx.x * E + e] = h[e];
}

// ---------------------------------------------------------------------------
// 2. Scan (single workgroup): global counts, local offsets, per-workgroup
//    bases, and the grouped-GEMM tile table.  Nothing returns to the host.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024)
void k_scan(const int32_t *__restrict__ blk_counts, int32_t nb, int32_t E, int32_t e0,
            int32_t E_loc, int32_t T, int32_t has_shared, int32_t *__restrict__ counts,
            int32_t *__restrict__ offsets, int32_t *__restrict__ blk_base, GroupTable g)
{
    __shared__ int32_t c[kMaxExperts];
    __shared__ int32_t off[kMaxLocalExperts + 1];
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        int acc = 0;
        for (int b = 0; b < nb; ++b) acc += blk_counts[(int64_t)b * E + e];
        c[e] = acc;
        counts[e] = acc;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int i = 0; i < E_loc; ++i) { off[i] = run; run += c[e0 + i]; }
        off[E_loc] = run;
        // tile tables over G = E_loc (+1 shared) groups
        int mt = 0, lt = 0, st = 0;
        const int G = E_loc + (has_shared ? 1 : 0);
        for (int i = 0; i < G; ++i) {
            const int rows = (i < E_loc) ? c[e0 + i] : T;
            g.row0[i] = (i < E_loc) ? off[i] : 0;
            g.rows[i] = rows;
            g.mt_base[i] = mt;
            g.lt_base[i] = lt;
            g.st_base[i] = st;
            const int m = (rows + kBM - 1) / kBM;
            mt += m;
            if (rows > kSmallRows) lt += m;
            else if (rows > 0) st += 1;
        }
        g.mt_base[G] = mt;
        g.lt_base[G] = lt;
        g.st_base[G] = st;
    }
    __syncthreads();
    for (int i = threadIdx.x; i <= E_loc; i += blockDim.x) offsets[i] = off[i];
    for (int i = threadIdx.x; i < E_loc; i += blockDim.x) {
        int run = off[i];
        for (int b = 0; b < nb; ++b) {
            blk_base[(int64_t)b * E_loc + i] = run;
            run += blk_counts[(int64_t)b * E + e0 + i];
        }
    }
}

// ---------------------------------------------------------------------------
// 3. Stable scatter.  Wave w of workgroup b owns slots
//    [b*chunk + w*chunk/4, b*chunk + (w+1)*chunk/4) and walks them in 64-slot
//    steps; within a step, lanes holding the same expert are ranked by lane
//    order with a ballot.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kDispatchThreads)
void k_scatter(const int32_t *__restrict__ ids, int32_t n_slots, int32_t E, int32_t e0,
               int32_t E_loc, const int32_t *__restrict__ blk_base,
               int32_t *__restrict__ slot_of_row, int32_t *__restrict__ row_of_slot)
{
    constexpr int kWaves = kDispatchThreads / 64;
    constexpr int kPerWave = kDispatchChunk / kWaves;
    __shared__ int32_t wbase[kWaves][kMaxLocalExperts];
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int64_t wstart = (int64_t)blockIdx.x * kDispatchChunk + (int64_t)wave * kPerWave;

    for (int i = lane; i < E_loc; i += 64) wbase[wave][i] = 0;
    __syncthreads();
    // per-wave local counts
    for (int st = 0; st < kPerWave; st += 64) {
        int64_t s = wstart + st + lane;
        int e = (s < n_slots) ? ids[s] : -1;
        int i = e - e0;
        if (e >= 0 && e < E && i >= 0 && i < E_loc) atomicAdd(&wbase[wave][i], 1);
    }
    __syncthreads();
    // exclusive scan over waves, seeded with this workgroup's base
    for (int i = threadIdx.x; i < E_loc; i += kDispatchThreads) {
        int run = blk_base[(int64_t)blockIdx.x * E_loc + i];
        for (int w = 0; w < kWaves; ++w) {
            int t = wbase[w][i];
            wbase[w][i] = run;
            run += t;
        }
    }
    __syncthreads();
    volatile int32_t *mybase = wbase[wave];
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int st = 0; st < kPerWave; st += 64) {
        int64_t s = wstart + st + lane;
        bool in = s < n_slots;
        int e = in ? ids[s] : -1;
        int i = e - e0;
        bool loc = in && e >= 0 && e < E && i >= 0 && i < E_loc;
        uint64_t pending = __ballot(loc);
        int pos = -1;
        while (pending) {
            int leader = __ffsll((unsigned long long)pending) - 1;
            int il = __shfl(i, leader);
            uint64_t m = __ballot(loc && i == il);
            int b = mybase[il];
            if (loc && i == il) pos = b + __popcll(m & lt_mask);
            if (lane == leader) mybase[il] = b + __popcll(m);
            pending &= ~m;
        }
        if (in) {
            row_of_slot[s] = pos;
            if (pos >= 0) slot_of_row[pos] = (int32_t)s;
        }
    }
}

// ---------------------------------------------------------------------------
// Fused single-workgroup dispatch for micro-batches of up to
// kFusedMaxSlots slots (a 4096-token DeepSeek-V3 batch has 32768): the
// histogram, scan, tile tables and stable scatter of the three kernels above
// in one launch, so the dispatch costs one launch instead of three.  Wave w
// owns the contiguous slot range [w * per, (w + 1) * per).
// ---------------------------------------------------------------------------
constexpr int kFusedThreads = 1024;
constexpr int kFusedWaves = kFusedThreads / 64;
constexpr int kFusedMaxSlots = 65536;

__global__ __launch_bounds__(kFusedThreads)
void k_dispatch_fused(const int32_t *__restrict__ ids, int32_t n_slots, int32_t E, int32_t e0,
                      int32_t E_loc, int32_t T, int32_t has_shared, int32_t *__restrict__ counts,
                      int32_t *__restrict__ offsets, GroupTable g,
                      int32_t *__restrict__ slot_of_row, int32_t *__restrict__ row_of_slot,
                      int32_t *__restrict__ err)
{
    __shared__ int32_t h[kMaxExperts];
    __shared__ int32_t wbase[kFusedWaves][kMaxLocalExperts];
    __shared__ int32_t off[kMaxLocalExperts + 1];
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int per = ((n_slots + kFusedWaves * 64 - 1) / (kFusedWaves * 64)) * 64;
    const int64_t wstart = (int64_t)wave * per;

    for (int e = threadIdx.x; e < E; e += kFusedThreads) h[e] = 0;
    for (int i = lane; i < E_loc; i += 64) wbase[wave][i] = 0;
    __syncthreads();
    int bad = 0;
    for (int st = 0; st < per; st += 64) {
        const int64_t s = wstart + st + lane;
        if (s >= n_slots) break;
        const int e = ids[s];
        if (e >= 0 && e < E) {
            atomicAdd(&h[e], 1);                       // integer counts: order-free
            const int i = e - e0;
            if (i >= 0 && i < E_loc) atomicAdd(&wbase[wave][i], 1);
        } else if (e != -1) {
            bad = 1;
        }
    }
    if (bad) atomicOr(err, kErrBadId);
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += kFusedThreads) counts[e] = h[e];
    if (threadIdx.x == 0) {
        int run = 0;
        for (int i = 0; i < E_loc; ++i) { off[i] = run; run += h[e0 + i]; }
        off[E_loc] = run;
        int mt = 0, lt = 0, stt = 0;
        const int G = E_loc + (has_shared ? 1 : 0);
        for (int i = 0; i < G; ++i) {
            const int rows = (i < E_loc) ? h[e0 + i] : T;
            g.row0[i] = (i < E_loc) ? off[i] : 0;
            g.rows[i] = rows;
            g.mt_base[i] = mt;
            g.lt_base[i] = lt;
            g.st_base[i] = stt;
            const int m = (rows + kBM - 1) / kBM;
            mt += m;
            if (rows > kSmallRows) lt += m;
            else if (rows > 0) stt += 1;
        }
        g.mt_base[G] = mt;
        g.lt_base[G] = lt;
        g.st_base[G] = stt;
    }
    __syncthreads();
    for (int i = threadIdx.x; i <= E_loc; i += kFusedThreads) offsets[i] = off[i];
    // exclusive scan of the per-wave counts, seeded with the expert offsets
    for (int i = threadIdx.x; i < E_loc; i += kFusedThreads) {
        int run = off[i];
        for (int w = 0; w < kFusedWaves; ++w) {
            const int t = wbase[w][i];
            wbase[w][i] = run;
            run += t;
        }
    }
    __syncthreads();
    volatile int32_t *mybase = wbase[wave];
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int st = 0; st < per; st += 64) {
        const int64_t s = wstart + st + lane;
        const bool in = s < n_slots;
        const int e = in ? ids[s] : -1;
        const int i = e - e0;
        const bool loc = in && e >= 0 && e < E && i >= 0 && i < E_loc;
        uint64_t pending = __ballot(loc);
        int pos = -1;
        while (pending) {
            const int leader = __ffsll((unsigned long long)pending) - 1;
            const int il = __shfl(i, leader);
            const uint64_t m = __ballot(loc && i == il);
            const int b = mybase[il];
            if (loc && i == il) pos = b + __popcll(m & lt_mask);
            if (lane == leader) mybase[il] = b + __popcll(m);
            pending &= ~m;
        }
        if (in) {
            row_of_slot[s] = pos;
            if (pos >= 0) slot_of_row[pos] = (int32_t)s;
        }
    }
}

hipError_t launch_dispatch_index(const DispatchArgs &a, hipStream_t s)
{
    if (a.n_slots <= kFusedMaxSlots) {
        hipLaunchKernelGGL(k_dispatch_fused, dim3(1), dim3(kFusedThreads), 0, s, a.ids, a.n_slots,
                           a.E, a.e0, a.E_loc, a.T, a.has_shared, a.counts, a.offsets, a.groups,
                           a.slot_of_row, a.row_of_slot, a.err);
        return hipGetLastError();
    }
    const int nb = (a.n_slots + kDispatchChunk - 1) / kDispatchChunk;
    if (nb > 0) {
        hipLaunchKernelGGL(k_hist, dim3(nb), dim3(kDispatchThreads), 0, s, a.ids, a.n_slots, a.E,
                           a.blk_counts, a.err);
    }
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, a.blk_counts, nb, a.E, a.e0, a.E_loc,
                       a.T, a.has_shared, a.counts, a.offsets, a.blk_base, a.groups);
    if (nb > 0) {
        hipLaunchKernelGGL(k_scatter, dim3(nb), dim3(kDispatchThreads), 0, s, a.ids, a.n_slots,
                           a.E, a.e0, a.E_loc, a.blk_base, a.slot_of_row, a.row_of_slot);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// 4. Row gather: one workgroup per row (grid-stride), each thread moving up
//    to 4 16-byte chunks of the row with all loads issued before the stores.
// ---------------------------------------------------------------------------
constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 4;

__global__ __launch_bounds__(kGatherThreads)
void k_gather(const uint4 *__restrict__ x, const float *__restrict__ xs,
              const int32_t *__restrict__ slot_of_row, const int32_t *__restrict__ n_rows_dev,
              int32_t k, int32_t row_vecs, int32_t n_scales, uint4 *__restrict__ xp,
              float *__restrict__ xps, int32_t scale_ld)
{
    const int n_rows = *n_rows_dev;
    for (int r = blockIdx.x; r < n_rows; r += gridDim.x) {
        const int t = slot_of_row[r] / k;
        const uint4 *src = x + (int64_t)t * row_vecs;
        uint4 *dst = xp + (int64_t)r * row_vecs;
        for (int c0 = 0; c0 < row_vecs; c0 += kGatherThreads * kGatherUnroll) {
            uint4 v[kGatherUnroll];
#pragma unroll
            for (int u = 0; u < kGatherUnroll; ++u) {
                const int c = c0 + u * kGatherThreads + threadIdx.x;
                if (c < row_vecs) v[u] = src[c];
            }
#pragma unroll
            for (int u = 0; u < kGatherUnroll; ++u) {
                const int c = c0 + u * kGatherThreads + threadIdx.x;
                if (c < row_vecs) dst[c] = v[u];
            }
        }
        if (xs != nullptr)
            for (int c = threadIdx.x; c < n_scales; c += kGatherThreads)
                xps[(int64_t)c * scale_ld + r] = xs[(int64_t)t * n_scales + c];
    }
}

hipError_t launch_gather_rows(const void *x, const float *x_scales, const int32_t *slot_of_row,
                              const int32_t *n_rows_dev, int32_t k, int32_t row_bytes,
                              int32_t n_scales, void *x_perm, float *x_perm_scales,
                              int32_t scale_ld, int32_t max_rows, int num_cus, hipStream_t s)
{
    if (max_rows <= 0) return hipSuccess;
    int grid = num_cus * 16;
    if (grid > max_rows) grid = max_rows;
    hipLaunchKernelGGL(k_gather, dim3(grid), dim3(kGatherThreads), 0, s, (const uint4 *)x,
                       x_scales, slot_of_row, n_rows_dev, k, row_bytes / 16, n_scales,
                       (uint4 *)x_perm, x_perm_scales, scale_ld);
    return hipGetLastError();
}

__global__ void k_transpose_scales(const float *__restrict__ src, int32_t rows, int32_t cols,
                                   float *__restrict__ dst, int32_t ld)
{
    const int64_t total = (int64_t)rows * cols;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(q / cols);
        const int c = (int)(q - (int64_t)r * cols);
        dst[(int64_t)c * ld + r] = src[q];
    }
}

hipError_t launch_transpose_scales(const float *src, int32_t rows, int32_t cols, float *dst,
                                   int32_t ld, hipStream_t s)
{
    const int64_t total = (int64_t)rows * cols;
    if (total <= 0) return hipSuccess;
    int64_t grid = (total + 255) / 256;
    if (grid > 1024) grid = 1024;
    hipLaunchKernelGGL(k_transpose_scales, dim3((unsigned)grid), dim3(256), 0, s, src, rows, cols,
                       dst, ld);
    return hipGetLastError();
}

}  // namespace moe
