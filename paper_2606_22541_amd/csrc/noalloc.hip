// Dispatch index without any allocation: the histogram, scan and stable
// counting-sort scatter of moe_dispatch (the per-expert counts and the
// grouping of section 3.2.1), for callers that cannot allocate device memory
// (code under HIP graph capture, serving loops, harnesses that forbid it).
//
// The kernels are the stage's own (k_hist, k_place).  What the stage keeps in
// a slot's workspace -- one histogram row per 1024-slot workgroup and the
// grouped-GEMM tile tables the placement kernel writes -- lives here in one
// file-scope device array.  Its device address is looked up once per device
// with hipGetSymbolAddress (in host code the array's name is not a device
// address) and only that address is ever handed to a kernel.
//
// Every call on a device shares that device's array: calls that overlap on
// one device (other streams, other threads) race on it.  Nothing in it needs
// clearing between calls: k_hist writes every entry of each histogram row it
// owns, and the table build writes every table entry the placement reads.
#include <mutex>

#include "kernels.h"
#include "moe_stage.h"

using namespace moe;

namespace {

// Histogram rows: ceil(T*k / 1024) rows of n_experts counts.
constexpr int64_t kHistInts = int64_t(1) << 20;                  // 4 MiB
// Tile tables: two arrays of G and eight of G + 1 entries, G <= 256.
constexpr int64_t kTableStride = kMaxLocalExperts + 64;          // >= G + 1, 256-byte multiple
constexpr int kTables = 10;
constexpr int64_t kTableInts = kTables * kTableStride;
constexpr int64_t kErrInts = 64;                                 // the fallback error word
constexpr int64_t kScratchInts = kHistInts + kTableInts + kErrInts;
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) int32_t scratch[kScratchInts];

namespace {

std::mutex g_scratch_mu;
int32_t *g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device, looked up on the
// first call there (with that device current) and kept.
moe_status scratch_for_current_device(int32_t **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MOE_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return MOE_EHIP;
        }
        g_scratch_ptr[dev] = (int32_t *)p;
    }
    *out = g_scratch_ptr[dev];
    return MOE_OK;
}

}  // namespace

extern "C" moe_status moe_dispatch_index_noalloc(const int32_t *topk_ids, int32_t n_tokens,
                                                 int32_t top_k, int32_t n_experts,
                                                 int32_t first_local_expert,
                                                 int32_t n_local_experts, int32_t *counts,
                                                 int32_t *offsets, int32_t *slot_of_row,
                                                 int32_t *row_of_slot, int32_t *err,
                                                 void *stream)
{
    if (n_tokens < 0 || top_k < 1 || top_k > 32) return MOE_EINVAL;
    if (n_experts < 1 || n_experts > kMaxExperts) return MOE_EINVAL;
    if (first_local_expert < 0 || n_local_experts < 1 || n_local_experts > kMaxLocalExperts ||
        first_local_expert + n_local_experts > n_experts)
        return MOE_EINVAL;
    const int64_t n_slots = (int64_t)n_tokens * top_k;
    if (n_slots >= ((int64_t)1 << 31)) return MOE_EINVAL;
    if (!counts || !offsets) return MOE_EINVAL;
    if (n_slots > 0 && (!topk_ids || !slot_of_row || !row_of_slot)) return MOE_EINVAL;
    const int64_t nb = (n_slots + kDispatchChunk - 1) / kDispatchChunk;
    if (nb * n_experts > kHistInts) return MOE_EUNSUPPORTED;     // past the scratch array

    int32_t *base = nullptr;
    const moe_status st = scratch_for_current_device(&base);
    if (st != MOE_OK) return st;
    int32_t *tables = base + kHistInts;
    DispatchArgs a{};
    a.ids = topk_ids;
    a.n_slots = (int32_t)n_slots;
    a.T = n_tokens;
    a.k = top_k;
    a.E = n_experts;
    a.e0 = first_local_expert;
    a.E_loc = n_local_experts;
    a.has_shared = 0;
    a.blk_counts = base;
    a.counts = counts;
    a.offsets = offsets;
    a.groups = GroupTable{tables + 0 * kTableStride, tables + 1 * kTableStride,
                          tables + 2 * kTableStride, tables + 3 * kTableStride,
                          tables + 4 * kTableStride, tables + 5 * kTableStride,
                          tables + 6 * kTableStride, tables + 7 * kTableStride,
                          tables + 8 * kTableStride, tables + 9 * kTableStride};
    static_assert(kTables == 10, "one array per GroupTable member");
    a.slot_of_row = slot_of_row;
    a.row_of_slot = row_of_slot;
    a.err = err ? err : base + kHistInts + kTableInts;
    return launch_dispatch_index(a, (hipStream_t)stream) == hipSuccess ? MOE_OK : MOE_EHIP;
}
