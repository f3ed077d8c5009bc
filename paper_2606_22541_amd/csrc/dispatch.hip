// Dispatch of one micro-batch: per-expert histogram, scan, stable counting-sort
// scatter and the gather of the fp8 token scales.
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

constexpr int kWaves = kDispatchThreads / 64;
constexpr int kPerWave = kDispatchChunk / kWaves;     // slots per wave
constexpr int kSteps = kPerWave / 64;                 // 64-slot steps per wave

// Exclusive prefix sum of one value per thread over the workgroup; *total
// receives the sum of all values.  Every thread of the workgroup must call it.
__device__ int block_excl_scan(int v, int32_t *wsum, int &total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int pre = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        const int t = wsum[w];
        if (w < wave) pre += t;
        tot += t;
    }
    __syncthreads();
    total = tot;
    return pre + x - v;
}

// ---------------------------------------------------------------------------
// 1. Histogram over all experts, one row of counts per workgroup of
//    kDispatchChunk slots.  Loads use clamped indices so that each thread
//    issues all of its loads before the first use.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kDispatchThreads)
void k_hist(const int32_t *__restrict__ ids, int32_t n_slots, int32_t E,
            int32_t *__restrict__ blk_counts, int32_t *__restrict__ err)
{
    __shared__ int32_t h[kMaxExperts];
    for (int e = threadIdx.x; e < E; e += kDispatchThreads) h[e] = 0;
    const int64_t base = (int64_t)blockIdx.x * kDispatchChunk + threadIdx.x;
    constexpr int kPer = kDispatchChunk / kDispatchThreads;
    int v[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int64_t sl = base + (int64_t)j * kDispatchThreads;
        v[j] = ids[sl < n_slots ? sl : n_slots - 1];
    }
    __syncthreads();
    int bad = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        if (base + (int64_t)j * kDispatchThreads >= n_slots) continue;
        if (v[j] >= 0 && v[j] < E) atomicAdd(&h[v[j]], 1);   // integer counts: order-free
        else if (v[j] != -1) bad = 1;
    }
    if (bad) atomicOr(err, kErrBadId);
    __syncthreads();
    for (int x = threadIdx.x; x < E; x += kDispatchThreads)
        blk_counts[(int64_t)blockIdx.x * E + x] = h[x];
}

// Exclusive prefix sum over the 64 lanes of a wave; *total receives the sum.
__device__ __forceinline__ int wave_excl_scan(int v, int lane, int &total)
{
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    total = __shfl(x, 63);
    return x - v;
}

// Grouped-GEMM tile tables over G = E_loc (+1 shared) groups (GroupTable),
// built by one wave in chunks of 64 groups with shuffle scans, so no
// workgroup barrier sits in the dispatch for them.  rows[i] is the local
// expert's token count (tot), or T for the shared expert.
__device__ void build_group_tables(const GroupTable &g, const int32_t *tot, int E_loc,
                                   int has_shared, int T, int lane)
{
    const int G = E_loc + (has_shared ? 1 : 0);
    int c_row = 0;
    int c_lt[2] = {0, 0}, c_st[2] = {0, 0}, c_fl[2] = {0, 0}, c_pl[2] = {0, 0};
    int32_t *lt_base[2] = {g.lt_base, g.lt_base_d}, *st_base[2] = {g.st_base, g.st_base_d};
    int32_t *fl_base[2] = {g.fl_base, g.fl_base_d}, *pl_list[2] = {g.pl_list, g.pl_list_d};
    constexpr int kThresh[2] = {kSmallRows, kSmallRowsDown};
    for (int c0 = 0; c0 < G; c0 += 64) {
        const int i = c0 + lane;
        const int rows = i < E_loc ? tot[i] : (i < G ? T : 0);
        const int m = (rows + kBM - 1) / kBM;
        const int fm = rows / kBM, rem = rows - fm * kBM;
        int t_row;
        const int p_row = wave_excl_scan(i < E_loc ? rows : 0, lane, t_row);
        if (i < G) {
            g.row0[i] = i < E_loc ? c_row + p_row : 0;
            g.rows[i] = rows;
        }
        // the two partitions into small groups (the small-group kernel) and
        // large ones (the 256-row kernel): gate/up at kSmallRows, down at
        // kSmallRowsDown
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const bool large = rows > kThresh[q];
            int t_lt, t_st, t_fl, t_pl;
            const int p_lt = wave_excl_scan(large ? m : 0, lane, t_lt);
            const int p_st = wave_excl_scan(rows > 0 && !large ? 1 : 0, lane, t_st);
            const int p_fl = wave_excl_scan(large ? fm : 0, lane, t_fl);
            wave_excl_scan(rem > 0 && large ? 1 : 0, lane, t_pl);
            if (i < G) {
                lt_base[q][i] = c_lt[q] + p_lt;
                st_base[q][i] = c_st[q] + p_st;
                fl_base[q][i] = c_fl[q] + p_fl;
            }
            c_lt[q] += t_lt;
            c_st[q] += t_st;
            c_fl[q] += t_fl;
            c_pl[q] += t_pl;
        }
        if (i < G && rem > 0) {
            // rank among the large groups' partial row tiles: more rows first,
            // then lower index
            int rank_l[2] = {0, 0};
            for (int j = 0; j < G; ++j) {
                const int rj = j < E_loc ? tot[j] : T;
                const int qj = rj % kBM;
                const bool before = qj > 0 && (qj > rem || (qj == rem && j < i));
                rank_l[0] += (before && rj > kThresh[0]) ? 1 : 0;
                rank_l[1] += (before && rj > kThresh[1]) ? 1 : 0;
            }
            if (rows > kThresh[0]) pl_list[0][rank_l[0]] = i;
            if (rows > kThresh[1]) pl_list[1][rank_l[1]] = i;
        }
        c_row += t_row;
    }
    if (lane == 0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            lt_base[q][G] = c_lt[q];
            st_base[q][G] = c_st[q];
            fl_base[q][G] = c_fl[q];
            pl_list[q][G] = c_pl[q];
        }
    }
}

// ---------------------------------------------------------------------------
// 2. Placement.  Workgroup b owns the same kDispatchChunk slots as histogram
//    workgroup b; wave w owns slots [b*chunk + w*chunk/4, b*chunk +
//    (w+1)*chunk/4) and walks them in 64-slot steps.  Every workgroup reads
//    the local-expert columns of the histogram rows to get the expert totals
//    and the counts of the workgroups before it, so no single-workgroup scan
//    sits between the two kernels.  Workgroup b also writes the global counts
//    of experts b, b + grid, ...; workgroup 0 writes the offsets, and the
//    last workgroup, which owns no slots, the grouped-GEMM tile tables.
//    Within a step, lanes holding the same expert are ranked by lane order
//    with a ballot.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kDispatchThreads)
void k_place(const int32_t *__restrict__ ids, int32_t n_slots, int32_t nb_hist, int32_t E,
             int32_t e0, int32_t E_loc, int32_t T, int32_t has_shared,
             const int32_t *__restrict__ blk_counts, int32_t *__restrict__ counts,
             int32_t *__restrict__ offsets, GroupTable g, int32_t *__restrict__ slot_of_row,
             int32_t *__restrict__ row_of_slot)
{
    __shared__ int32_t tot[kMaxLocalExperts], pre[kMaxLocalExperts];
    __shared__ int32_t wbase[kWaves][kMaxLocalExperts];
    __shared__ int32_t cnt_my[kMaxExperts];
    __shared__ int32_t wsum[kWaves];
    const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int64_t wstart = (int64_t)b * kDispatchChunk + (int64_t)wave * kPerWave + lane;

    // The ids loads are issued first; the LDS set-up uses a barrier that
    // waits for LDS stores only, so the histogram-row loads below are
    // issued while the ids are still in flight (one latency, not two).
    int v[kSteps];
    if (n_slots > 0) {
#pragma unroll
        for (int j = 0; j < kSteps; ++j) {
            const int64_t sl = wstart + j * 64;
            v[j] = ids[sl < n_slots ? sl : n_slots - 1];
        }
    }
    const int n_my = b < E ? (E - 1 - b) / (int)gridDim.x + 1 : 0;
    for (int i = tid; i < E_loc; i += kDispatchThreads) {
        tot[i] = 0;
        pre[i] = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) wbase[w][i] = 0;
    }
    for (int q = tid; q < n_my; q += kDispatchThreads) cnt_my[q] = 0;
    // first histogram value of this thread's share of the global counts,
    // loaded now so that it arrives with the ones below instead of a round
    // trip later
    const int n_cnt = n_my * nb_hist;
    int cnt0 = 0;
    if (tid < n_cnt) {
        const int q = tid / nb_hist, bb = tid - q * nb_hist;
        cnt0 = blk_counts[(int64_t)bb * E + b + q * (int)gridDim.x];
    }
    __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));   // lgkmcnt(0) only
    __builtin_amdgcn_s_barrier();

    // expert totals and the part of them in earlier workgroups
    {
        const int tpe = E_loc < kDispatchThreads ? kDispatchThreads / E_loc : 1;
        const int i = tid / tpe, sub = tid - i * tpe;
        if (i < E_loc) {
            int t = 0, p = 0;
            for (int bb = sub; bb < nb_hist; bb += tpe) {
                const int c = blk_counts[(int64_t)bb * E + e0 + i];
                t += c;
                if (bb < b) p += c;
            }
            atomicAdd(&tot[i], t);
            atomicAdd(&pre[i], p);
        }
    }
    // local expert index of each slot this lane owns (-1: not local / none)
    int li[kSteps];
#pragma unroll
    for (int j = 0; j < kSteps; ++j) {
        const int i = v[j] - e0;
        li[j] = (n_slots > 0 && wstart + j * 64 < n_slots && v[j] >= 0 && v[j] < E && i >= 0 &&
                 i < E_loc) ? i : -1;
    }
    // per-wave counts of this workgroup's slots
#pragma unroll
    for (int j = 0; j < kSteps; ++j)
        if (li[j] >= 0) atomicAdd(&wbase[wave][li[j]], 1);
    // global counts of experts b, b + grid, ...
    if (tid < n_cnt) atomicAdd(&cnt_my[tid / nb_hist], cnt0);
    for (int it = tid + kDispatchThreads; it < n_cnt; it += kDispatchThreads) {
        const int q = it / nb_hist, bb = it - q * nb_hist;
        atomicAdd(&cnt_my[q], blk_counts[(int64_t)bb * E + b + q * (int)gridDim.x]);
    }
    __syncthreads();
    for (int q = tid; q < n_my; q += kDispatchThreads) counts[b + q * (int)gridDim.x] = cnt_my[q];

    // offsets (E_loc <= 256: one local expert per thread) and wave bases
    int total = 0;
    const int off_i = block_excl_scan(tid < E_loc ? tot[tid] : 0, wsum, total);
    if (tid < E_loc) {
        int run = off_i + pre[tid];
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int t = wbase[w][tid];
            wbase[w][tid] = run;
            run += t;
        }
    }
    if (b == 0) {
        if (tid < E_loc) offsets[tid] = off_i;
        if (tid == 0) offsets[E_loc] = total;
    }
    __syncthreads();

    volatile int32_t *mybase = wbase[wave];
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int j = 0; j < kSteps; ++j) {
        const int64_t sl = wstart + j * 64;
        const int i = li[j];
        const bool loc = i >= 0;
        uint64_t pending = __ballot(loc);
        int pos = -1;
        while (pending) {
            const int leader = __ffsll((unsigned long long)pending) - 1;
            const int il = __shfl(i, leader);
            const uint64_t m = __ballot(loc && i == il);
            const int bse = mybase[il];
            if (loc && i == il) pos = bse + __popcll(m & lt_mask);
            if (lane == leader) mybase[il] = bse + __popcll(m);
            pending &= ~m;
        }
        if (sl < n_slots) {
            row_of_slot[sl] = pos;
            if (pos >= 0) slot_of_row[pos] = (int32_t)sl;
        }
    }
    // the last workgroup owns no slots (the launch adds it for this): its
    // first wave builds the tables while the others place their slots
    if (b == (int)gridDim.x - 1 && wave == 0) build_group_tables(g, tot, E_loc, has_shared, T, lane);
}

// Tile tables for pre-grouped rows (the receive region of section 3.2.1 in
// its grouped form: the senders supply the per-expert counts).  One wave:
// validate the counts in order, then the same table build as the dispatch.
__global__ __launch_bounds__(64)
void k_group_tables_from_counts(const int32_t *__restrict__ counts, int32_t E_loc,
                                int32_t n_rows_max, GroupTable g, int32_t *__restrict__ err)
{
    __shared__ int32_t tot[kMaxLocalExperts];
    const int lane = threadIdx.x;
    int carry = 0, bad = 0;
    for (int c0 = 0; c0 < E_loc; c0 += 64) {
        const int i = c0 + lane;
        int c = i < E_loc ? counts[i] : 0;
        bad |= c < 0;
        c = c < 0 ? 0 : c;
        int t;
        const int before = carry + wave_excl_scan(c, lane, t);
        // rows past n_rows_max are dropped: the group keeps what fits
        const int keep = min(c, max(0, n_rows_max - before));
        bad |= keep != c;
        if (i < E_loc) tot[i] = keep;
        carry += t;
    }
    if (__any(bad) && lane == 0) atomicOr(err, kErrBadCount);
    __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));   // LDS stores done
    __builtin_amdgcn_wave_barrier();
    build_group_tables(g, tot, E_loc, 0, 0, lane);
}

hipError_t launch_group_tables_from_counts(const int32_t *counts, int32_t E_loc,
                                           int32_t n_rows_max, GroupTable g, int32_t *err,
                                           hipStream_t s)
{
    hipLaunchKernelGGL(k_group_tables_from_counts, dim3(1), dim3(64), 0, s, counts, E_loc,
                       n_rows_max, g, err);
    return hipGetLastError();
}

hipError_t launch_dispatch_index(const DispatchArgs &a, hipStream_t s)
{
    const int nb = (a.n_slots + kDispatchChunk - 1) / kDispatchChunk;
    if (nb > 0) {
        hipLaunchKernelGGL(k_hist, dim3(nb), dim3(kDispatchThreads), 0, s, a.ids, a.n_slots, a.E,
                           a.blk_counts, a.err);
    }
    // one workgroup per histogram row, plus one without slots for the tables
    hipLaunchKernelGGL(k_place, dim3(nb + 1), dim3(kDispatchThreads), 0, s, a.ids,
                       a.n_slots, nb, a.E, a.e0, a.E_loc, a.T, a.has_shared, a.blk_counts,
                       a.counts, a.offsets, a.groups, a.slot_of_row, a.row_of_slot);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// 4. Scale gather (fp8): the grouped GEMMs read the token rows of x through
//    slot_of_row themselves, but they take the step's token scales as one
//    contiguous run per 128-channel group, so the scales of the routed rows
//    are gathered here into the transposed [n_scales][scale_ld] layout.
//    Work item i (grid-stride) moves the scales of groups 8 (i / n_rows) ..
//    + 7 of row i % n_rows: the stores of a group are consecutive across a
//    wave, and each thread has its eight loads in flight at once.
// ---------------------------------------------------------------------------
constexpr int kGatherThreads = 256;
constexpr int kScalesPerItem = 8;

__global__ __launch_bounds__(kGatherThreads)
void k_gather_scales(const float *__restrict__ xs, const int32_t *__restrict__ slot_of_row,
                     const int32_t *__restrict__ n_rows_dev, int32_t k, int32_t n_scales,
                     float *__restrict__ xps, int32_t scale_ld)
{
    const int n_rows = *n_rows_dev;
    if (n_rows <= 0) return;
    const int64_t chunks = (n_scales + kScalesPerItem - 1) / kScalesPerItem;
    const int64_t total = (int64_t)n_rows * chunks;
    for (int64_t i = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * kGatherThreads) {
        const int c = (int)(i / n_rows);
        const int r = (int)(i - (int64_t)c * n_rows);
        const int g0 = c * kScalesPerItem;
        const float *src = xs + (int64_t)(slot_of_row[r] / k) * n_scales;
        float v[kScalesPerItem];
#pragma unroll
        for (int u = 0; u < kScalesPerItem; ++u) v[u] = src[min(g0 + u, n_scales - 1)];
#pragma unroll
        for (int u = 0; u < kScalesPerItem; ++u)
            if (g0 + u < n_scales) xps[(int64_t)(g0 + u) * scale_ld + r] = v[u];
    }
}

hipError_t launch_gather_scales(const float *x_scales, const int32_t *slot_of_row,
                                const int32_t *n_rows_dev, int32_t k, int32_t n_scales,
                                float *x_perm_scales, int32_t scale_ld, int32_t max_rows,
                                int num_cus, hipStream_t s)
{
    if (max_rows <= 0 || n_scales <= 0) return hipSuccess;
    const int64_t work = (int64_t)max_rows * ((n_scales + kScalesPerItem - 1) / kScalesPerItem);
    int64_t grid = (work + kGatherThreads - 1) / kGatherThreads;
    if (grid > (int64_t)num_cus * 4) grid = (int64_t)num_cus * 4;
    hipLaunchKernelGGL(k_gather_scales, dim3((unsigned)grid), dim3(kGatherThreads), 0, s, x_scales,
                       slot_of_row, n_rows_dev, k, n_scales, x_perm_scales, scale_ld);
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
