// Host runtime of the MoE expert stage: the C ABI declared in moe_stage.h.
//
// Everything the hot path needs is allocated in moe_stage_create (weights
// packed for the grouped GEMM, and one workspace per in-flight micro-batch
// slot), following the paper's statically allocated, process-lifetime
// buffers (section 3.2).  The enqueue calls only validate arguments and
// launch kernels on the caller's stream; per-expert row counts stay on the
// device (section 3.4.2: host round trips are the bubble to avoid).
#include <stdio.h>
#include <string.h>

#include <new>
#include <vector>

#include "kernels.h"
#include "moe_stage.h"

using namespace moe;

namespace {

struct SlotWs {
    int32_t *blk_counts = nullptr, *counts = nullptr, *offsets = nullptr;
    int32_t *g_row0 = nullptr, *g_rows = nullptr;
    int32_t *g_lt_base = nullptr, *g_st_base = nullptr;
    int32_t *g_fl_base = nullptr, *g_pl_list = nullptr;
    int32_t *g_lt_base_d = nullptr, *g_st_base_d = nullptr, *g_fl_base_d = nullptr,
            *g_pl_list_d = nullptr;
    GroupTable tables() const
    {
        return GroupTable{g_row0,    g_rows,      g_lt_base,   g_st_base,   g_fl_base,
                          g_pl_list, g_lt_base_d, g_st_base_d, g_fl_base_d, g_pl_list_d};
    }
    int32_t *slot_of_row = nullptr, *row_of_slot = nullptr;
    float *x_perm_s = nullptr;     // fp8: the routed rows' x scales, transposed
    void *h = nullptr;
    float *h_s = nullptr;
    void *y_perm = nullptr;
    void *h_sh = nullptr;
    float *h_sh_s = nullptr;
    void *y_sh = nullptr;
    float *xsh_s = nullptr;      // fp8 mode with shared expert: x scales, transposed
    hipEvent_t ev = nullptr;
    bool ev_recorded = false;
    bool has_mb = false;
    moe_microbatch mb{};
};

struct Sizes {
    int64_t G, cap, nb_max, eb, n_slots_tok;
    int64_t w1, w2, s1, s2;                 // bytes, all layers
    int64_t w1l, w2l, s1l, s2l;             // bytes of one layer
    int64_t per_slot;                       // bytes
};

bool desc_ok(const moe_stage_desc *d);

// MOE_OK, MOE_EINVAL for a malformed descriptor, or MOE_EUNSUPPORTED for a
// well-formed shape the kernels do not take: d or f not a multiple of 128
// (one K step of every GEMM is 128 bytes of fp8 or a multiple of 64 bf16).
moe_status desc_check(const moe_stage_desc *d)
{
    if (!d) return MOE_EINVAL;
    if (d->d_model <= 0 || d->d_ff <= 0) return MOE_EINVAL;
    if (d->d_model % 128 || d->d_ff % 128) return MOE_EUNSUPPORTED;
    return desc_ok(d) ? MOE_OK : MOE_EINVAL;
}

bool desc_ok(const moe_stage_desc *d)
{
    if (!d) return false;
    if (d->d_model <= 0 || d->d_model % 128 || d->d_ff <= 0 || d->d_ff % 128) return false;
    if (d->n_experts < 1 || d->n_experts > kMaxExperts) return false;
    if (d->first_local_expert < 0 || d->n_local_experts < 1 ||
        d->n_local_experts > kMaxLocalExperts ||
        d->first_local_expert + d->n_local_experts > d->n_experts)
        return false;
    if (d->top_k < 1 || d->top_k > 32) return false;
    if (d->max_tokens < 0 || d->n_slots < 1 || d->n_slots > 64) return false;
    if (d->dtype != MOE_DTYPE_BF16 && d->dtype != MOE_DTYPE_FP8_E4M3_B128) return false;
    if (d->has_shared_expert != 0 && d->has_shared_expert != 1) return false;
    if (d->n_layers < 1 || d->n_layers > kMaxLayers) return false;
    // 32-bit slot and row indices; 32-bit byte offsets inside one GEMM tile
    if ((int64_t)d->max_tokens * d->top_k >= (int64_t)1 << 31) return false;
    if ((int64_t)256 * d->d_model * 2 >= (int64_t)1 << 31) return false;
    if ((int64_t)256 * d->d_ff * 2 >= (int64_t)1 << 31) return false;
    // the bf16 gate/up GEMM addresses token rows of x with 32-bit byte offsets
    if ((int64_t)d->max_tokens * d->d_model * 2 >= (int64_t)1 << 31) return false;
    return true;
}

int64_t align256(int64_t b) { return (b + 255) & ~(int64_t)255; }

Sizes sizes_of(const moe_stage_desc *d)
{
    Sizes s{};
    const int64_t D = d->d_model, F = d->d_ff, E = d->n_experts, El = d->n_local_experts;
    const int64_t k = d->top_k, T = d->max_tokens;
    const bool fp8 = d->dtype == MOE_DTYPE_FP8_E4M3_B128;
    s.G = El + d->has_shared_expert;
    s.eb = fp8 ? 1 : 2;
    s.cap = T * k;   // a token may repeat a local id, so every slot can be local
    s.n_slots_tok = T * k;
    s.nb_max = (s.n_slots_tok + kDispatchChunk - 1) / kDispatchChunk;
    if (s.nb_max < 1) s.nb_max = 1;
    s.w1l = align256(s.G * 2 * F * D * s.eb);
    s.w2l = align256(s.G * D * F * s.eb);
    s.s1l = fp8 ? align256(s.G * (2 * F / 128) * (D / 128) * 4) : 0;
    s.s2l = fp8 ? align256(s.G * (D / 128) * (F / 128) * 4) : 0;
    s.w1 = s.w1l * d->n_layers;
    s.w2 = s.w2l * d->n_layers;
    s.s1 = s.s1l * d->n_layers;
    s.s2 = s.s2l * d->n_layers;
    const int64_t cap1 = s.cap > 0 ? s.cap : 1;
    const int64_t T1 = T > 0 ? T : 1;
    int64_t b = 0;
    b += align256(s.nb_max * E * 4) + align256(E * 4) + align256((El + 1) * 4);
    b += 2 * align256(s.G * 4) + 8 * align256((s.G + 1) * 4);
    b += align256(cap1 * 4) + align256((s.n_slots_tok > 0 ? s.n_slots_tok : 1) * 4);
    if (fp8) b += align256(cap1 * (D / 128) * 4);   // gathered token scales (fp8 only)
    b += align256(cap1 * F * s.eb) + (fp8 ? align256(cap1 * (F / 128) * 4) : 0);
    b += align256(cap1 * D * 2);
    if (d->has_shared_expert) {
        b += align256(T1 * F * s.eb) + (fp8 ? align256(T1 * (F / 128) * 4) : 0);
        b += align256(T1 * D * 2);
        if (fp8) b += align256(T1 * (D / 128) * 4);
    }
    s.per_slot = b;
    return s;
}

}  // namespace

struct ProfRec {
    int kind;
    hipEvent_t a, b;
};

struct moe_stage {
    moe_stage_desc desc{};
    bool prof_on = false;
    std::vector<ProfRec> prof;
    Sizes sz{};
    int device = 0;
    int num_cus = 0;
    void *w1 = nullptr, *w2 = nullptr;
    float *s1 = nullptr, *s2 = nullptr;
    LayerWeights *layers = nullptr;   // device table, one entry per layer
    int32_t *err = nullptr;
    hipStream_t own = nullptr;
    std::vector<SlotWs> slots;
    std::vector<void *> allocs;
    int next_slot = 0;
};

namespace {

void release(moe_stage *st)
{
    if (!st) return;
    for (auto &p : st->prof) {
        hipEventSynchronize(p.b);
        hipEventDestroy(p.a);
        hipEventDestroy(p.b);
    }
    for (auto &sl : st->slots) {
        if (sl.ev) {
            hipEventSynchronize(sl.ev);
            hipEventDestroy(sl.ev);
        }
    }
    if (st->own) {
        hipStreamSynchronize(st->own);
        hipStreamDestroy(st->own);
    }
    for (void *p : st->allocs) hipFree(p);
    delete st;
}

template <typename T>
bool alloc(moe_stage *st, T **p, int64_t bytes)
{
    void *q = nullptr;
    if (hipMalloc(&q, (size_t)align256(bytes > 0 ? bytes : 4)) != hipSuccess) return false;
    st->allocs.push_back(q);
    *p = (T *)q;
    return true;
}

bool slot_ok(const moe_stage *st, int32_t slot)
{
    return st && slot >= 0 && slot < (int32_t)st->slots.size();
}

// Event pair around a kernel group when profiling is on.
struct ProfScope {
    moe_stage *st;
    int kind;
    hipStream_t s;
    hipEvent_t a = nullptr;
    ProfScope(moe_stage *st_, int kind_, hipStream_t s_) : st(st_), kind(kind_), s(s_)
    {
        if (st->prof_on && hipEventCreateWithFlags(&a, hipEventDisableSystemFence) == hipSuccess)
            hipEventRecord(a, s);
    }
    ~ProfScope()
    {
        if (!a) return;
        hipEvent_t b = nullptr;
        if (hipEventCreateWithFlags(&b, hipEventDisableSystemFence) == hipSuccess &&
            hipEventRecord(b, s) == hipSuccess)
            st->prof.push_back(ProfRec{kind, a, b});
        else
            hipEventDestroy(a);
    }
};

moe_status record(SlotWs &sl, hipStream_t s)
{
    if (hipEventRecord(sl.ev, s) != hipSuccess) return MOE_EHIP;
    sl.ev_recorded = true;
    return MOE_OK;
}

// Packs one layer's weights into w1/w2 (and fp8 scales into s1/s2) in MFMA
// fragment order; the shared expert is group E_loc.  [gate|up] is
// interleaved by 16 rows.
hipError_t pack_layer(const moe_stage_desc *d, const Sizes &z, const moe_weights *w, void *w1,
                      void *w2, float *s1, float *s2, hipStream_t s)
{
    const bool fp8 = d->dtype == MOE_DTYPE_FP8_E4M3_B128;
    const int64_t D = d->d_model, F = d->d_ff, El = d->n_local_experts;
    hipError_t e = hipSuccess;
    const int64_t w1_mat = 2 * F * D * z.eb, w2_mat = D * F * z.eb;
    if (fp8) {
        e = launch_pack_frag_fp8(w->w_gate, w->w_up, w1, (int32_t)El, (int32_t)(2 * F),
                                 (int32_t)D, kInterleaveFp8, s);
        if (e == hipSuccess)
            e = launch_pack_frag_fp8(w->w_down, nullptr, w2, (int32_t)El, (int32_t)D,
                                     (int32_t)F, 0, s);
        if (e == hipSuccess && d->has_shared_expert) {
            e = launch_pack_frag_fp8(w->sh_gate, w->sh_up, (char *)w1 + El * w1_mat, 1,
                                     (int32_t)(2 * F), (int32_t)D, kInterleaveFp8, s);
            if (e == hipSuccess)
                e = launch_pack_frag_fp8(w->sh_down, nullptr, (char *)w2 + El * w2_mat, 1,
                                         (int32_t)D, (int32_t)F, 0, s);
        }
    } else {
        e = launch_pack_frag_bf16(w->w_gate, w->w_up, w1, (int32_t)El, (int32_t)(2 * F),
                                  (int32_t)D, kInterleaveBf16, s);
        if (e == hipSuccess)
            e = launch_pack_frag_bf16(w->w_down, nullptr, w2, (int32_t)El, (int32_t)D,
                                      (int32_t)F, 0, s);
        if (e == hipSuccess && d->has_shared_expert) {
            e = launch_pack_frag_bf16(w->sh_gate, w->sh_up, (char *)w1 + El * w1_mat, 1,
                                      (int32_t)(2 * F), (int32_t)D, kInterleaveBf16, s);
            if (e == hipSuccess)
                e = launch_pack_frag_bf16(w->sh_down, nullptr, (char *)w2 + El * w2_mat, 1,
                                          (int32_t)D, (int32_t)F, 0, s);
        }
    }
    if (e == hipSuccess && fp8) {
        const int64_t s1_mat = (2 * F / 128) * (D / 128), s2_mat = (D / 128) * (F / 128);
        e = launch_pack_gate_up_scales(w->s_gate, w->s_up, s1, (int32_t)El, (int32_t)F,
                                       (int32_t)D, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(s2, w->s_down, (size_t)(El * s2_mat * 4),
                               hipMemcpyDeviceToDevice, s);
        if (e == hipSuccess && d->has_shared_expert) {
            e = launch_pack_gate_up_scales(w->sh_s_gate, w->sh_s_up, s1 + El * s1_mat, 1,
                                           (int32_t)F, (int32_t)D, s);
            if (e == hipSuccess)
                e = hipMemcpyAsync(s2 + El * s2_mat, w->sh_s_down, (size_t)(s2_mat * 4),
                                   hipMemcpyDeviceToDevice, s);
        }
    }
    return e;
}

}  // namespace

extern "C" {

const char *moe_status_string(moe_status s)
{
    switch (s) {
    case MOE_OK: return "ok";
    case MOE_EINVAL: return "invalid argument";
    case MOE_ENOMEM: return "out of device memory";
    case MOE_EHIP: return "HIP runtime error";
    case MOE_EBADID: return "expert id outside [-1, n_experts) seen on the device";
    case MOE_EUNSUPPORTED: return "unsupported shape or mode";
    case MOE_EBUSY: return "slot busy";
    case MOE_EBADLAYER: return "layer id outside [0, n_layers) seen on the device (clamped)";
    case MOE_ETIMEOUT: return "an ingest wait gave up before every ready word reached its epoch";
    case MOE_EBADCOUNT: return "pre-grouped counts negative or past the rows buffer (rows dropped)";
    default: return "unknown status";
    }
}

moe_status moe_stage_workspace_bytes(const moe_stage_desc *desc, int64_t *bytes)
{
    if (!bytes) return MOE_EINVAL;
    const moe_status dc = desc_check(desc);
    if (dc != MOE_OK) return dc;
    Sizes s = sizes_of(desc);
    *bytes = s.w1 + s.w2 + s.s1 + s.s2 + 256 + align256(desc->n_layers * (int64_t)sizeof(LayerWeights)) +
             s.per_slot * desc->n_slots;
    return MOE_OK;
}

moe_status moe_stage_create(const moe_stage_desc *desc, const moe_weights *w, moe_stage **out)
{
    if (!out) return MOE_EINVAL;
    *out = nullptr;
    const moe_status dc = desc_check(desc);
    if (dc != MOE_OK) return dc;
    if (!w) return MOE_EINVAL;
    const bool fp8 = desc->dtype == MOE_DTYPE_FP8_E4M3_B128;
    for (int l = 0; l < desc->n_layers; ++l) {
        const moe_weights &wl = w[l];
        if (!wl.w_gate || !wl.w_up || !wl.w_down) return MOE_EINVAL;
        if (fp8 && (!wl.s_gate || !wl.s_up || !wl.s_down)) return MOE_EINVAL;
        if (desc->has_shared_expert) {
            if (!wl.sh_gate || !wl.sh_up || !wl.sh_down) return MOE_EINVAL;
            if (fp8 && (!wl.sh_s_gate || !wl.sh_s_up || !wl.sh_s_down)) return MOE_EINVAL;
        }
    }

    moe_stage *st = new (std::nothrow) moe_stage();
    if (!st) return MOE_ENOMEM;
    st->desc = *desc;
    st->sz = sizes_of(desc);
    const Sizes &z = st->sz;
    if (hipGetDevice(&st->device) != hipSuccess ||
        hipDeviceGetAttribute(&st->num_cus, hipDeviceAttributeMultiprocessorCount, st->device) !=
            hipSuccess ||
        hipStreamCreateWithFlags(&st->own, hipStreamNonBlocking) != hipSuccess) {
        release(st);
        return MOE_EHIP;
    }
    const int64_t D = desc->d_model, F = desc->d_ff, El = desc->n_local_experts;
    bool ok = alloc(st, &st->w1, z.w1) && alloc(st, &st->w2, z.w2) && alloc(st, &st->err, 4) &&
              alloc(st, &st->layers, desc->n_layers * (int64_t)sizeof(LayerWeights));
    if (ok && fp8) ok = alloc(st, &st->s1, z.s1) && alloc(st, &st->s2, z.s2);
    if (!ok) {
        release(st);
        return MOE_ENOMEM;
    }
    // Pack every layer's weights and build the device table of their addresses.
    hipError_t e = hipSuccess;
    std::vector<LayerWeights> table(desc->n_layers);
    for (int l = 0; l < desc->n_layers && e == hipSuccess; ++l) {
        LayerWeights &lw = table[l];
        lw.w1 = (char *)st->w1 + l * z.w1l;
        lw.w2 = (char *)st->w2 + l * z.w2l;
        lw.s1 = fp8 ? (float *)((char *)st->s1 + l * z.s1l) : nullptr;
        lw.s2 = fp8 ? (float *)((char *)st->s2 + l * z.s2l) : nullptr;
        e = pack_layer(desc, z, &w[l], (void *)lw.w1, (void *)lw.w2, (float *)lw.s1,
                       (float *)lw.s2, st->own);
    }
    if (e == hipSuccess)
        e = hipMemcpyAsync(st->layers, table.data(), table.size() * sizeof(LayerWeights),
                           hipMemcpyHostToDevice, st->own);
    if (e == hipSuccess) e = hipMemsetAsync(st->err, 0, 4, st->own);
    if (e != hipSuccess) {
        release(st);
        return MOE_EHIP;
    }

    st->slots.resize(desc->n_slots);
    const int64_t E = desc->n_experts, cap1 = z.cap > 0 ? z.cap : 1;
    const int64_t T1 = desc->max_tokens > 0 ? desc->max_tokens : 1;
    for (auto &sl : st->slots) {
        ok = alloc(st, &sl.blk_counts, z.nb_max * E * 4) && alloc(st, &sl.counts, E * 4) &&
             alloc(st, &sl.offsets, (El + 1) * 4) &&
             alloc(st, &sl.g_row0, z.G * 4) && alloc(st, &sl.g_rows, z.G * 4) &&
             alloc(st, &sl.g_lt_base, (z.G + 1) * 4) && alloc(st, &sl.g_st_base, (z.G + 1) * 4) &&
             alloc(st, &sl.g_fl_base, (z.G + 1) * 4) &&
             alloc(st, &sl.g_pl_list, (z.G + 1) * 4) && alloc(st, &sl.g_lt_base_d, (z.G + 1) * 4) &&
             alloc(st, &sl.g_st_base_d, (z.G + 1) * 4) && alloc(st, &sl.g_fl_base_d, (z.G + 1) * 4) &&
             alloc(st, &sl.g_pl_list_d, (z.G + 1) * 4) && alloc(st, &sl.slot_of_row, cap1 * 4) &&
             alloc(st, &sl.row_of_slot, (z.n_slots_tok > 0 ? z.n_slots_tok : 1) * 4) &&
             alloc(st, &sl.h, cap1 * F * z.eb) &&
             alloc(st, &sl.y_perm, cap1 * D * 2);
        // no X_perm: the gate/up GEMM gathers the token rows itself; fp8 keeps
        // the gathered token scales
        if (ok && fp8) ok = alloc(st, &sl.x_perm_s, cap1 * (D / 128) * 4) &&
                            alloc(st, &sl.h_s, cap1 * (F / 128) * 4);
        if (ok && desc->has_shared_expert) {
            ok = alloc(st, &sl.h_sh, T1 * F * z.eb) && alloc(st, &sl.y_sh, T1 * D * 2);
            if (ok && fp8)
                ok = alloc(st, &sl.h_sh_s, T1 * (F / 128) * 4) &&
                     alloc(st, &sl.xsh_s, T1 * (D / 128) * 4);
        }
        if (!ok) {
            release(st);
            return MOE_ENOMEM;
        }
        if (hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming | hipEventDisableSystemFence) != hipSuccess) {
            release(st);
            return MOE_EHIP;
        }
    }
    if (hipStreamSynchronize(st->own) != hipSuccess) {
        release(st);
        return MOE_EHIP;
    }
    *out = st;
    return MOE_OK;
}

void moe_stage_destroy(moe_stage *st) { release(st); }

static bool mb_ok(const moe_stage *st, const moe_microbatch *mb)
{
    if (!st || !mb) return false;
    const moe_stage_desc &d = st->desc;
    const int32_t T = mb->n_tokens;
    if (T < 0 || T > d.max_tokens) return false;
    if (mb->combine_mode != MOE_COMBINE_OVERWRITE && mb->combine_mode != MOE_COMBINE_ACCUMULATE)
        return false;
    if (T > 0 && (!mb->x || !mb->topk_ids || !mb->topk_w || !mb->out)) return false;
    if (T > 0 && d.dtype == MOE_DTYPE_FP8_E4M3_B128 && !mb->x_scales) return false;
    return true;
}

// CUs the kernels of `stream` may run on: the stream's CU mask when it has
// one (hipExtStreamCreateWithCUMask), else every CU.  The persistent GEMMs
// size their grids by it, so a masked stream gets one workgroup per CU it
// may use instead of a second round of workgroups.
static int stream_cus(const moe_stage *st, hipStream_t s)
{
    if (!s) return st->num_cus;
    uint32_t mask[32] = {};
    if (hipExtStreamGetCUMask(s, 32, mask) != hipSuccess) {
        (void)hipGetLastError();
        return st->num_cus;
    }
    int n = 0;
    for (uint32_t m : mask) n += __builtin_popcount(m);
    return (n > 0 && n < st->num_cus) ? n : st->num_cus;
}

// The three phases.  `rec` records the slot's event at the end; a submit
// records it once, after the combine, since every record is a release that
// stalls the stream for several microseconds.
static moe_status dispatch_impl(moe_stage *st, int32_t slot, const moe_microbatch *mb,
                                void *stream, bool rec)
{
    if (!slot_ok(st, slot) || !mb_ok(st, mb)) return MOE_EINVAL;
    const moe_stage_desc &d = st->desc;
    const int32_t T = mb->n_tokens;
    const bool fp8 = d.dtype == MOE_DTYPE_FP8_E4M3_B128;
    hipStream_t s = (hipStream_t)stream;
    SlotWs &sl = st->slots[slot];
    sl.mb = *mb;
    sl.has_mb = true;

    DispatchArgs a{};
    a.ids = mb->topk_ids;
    a.n_slots = T * d.top_k;
    a.T = T;
    a.k = d.top_k;
    a.E = d.n_experts;
    a.e0 = d.first_local_expert;
    a.E_loc = d.n_local_experts;
    a.has_shared = d.has_shared_expert;
    a.blk_counts = sl.blk_counts;
    a.counts = sl.counts;
    a.offsets = sl.offsets;
    a.groups = sl.tables();
    a.slot_of_row = sl.slot_of_row;
    a.row_of_slot = sl.row_of_slot;
    a.err = st->err;
    {
        ProfScope ps(st, 0, s);
        if (launch_dispatch_index(a, s) != hipSuccess) return MOE_EHIP;
    }
    // The gate/up GEMM reads the token rows of x through slot_of_row; fp8
    // gathers the rows' scales (transposed) for it.
    const int64_t max_rows = (int64_t)T * d.top_k;
    if (fp8 && max_rows > 0) {
        ProfScope ps(st, 1, s);
        if (launch_gather_scales(mb->x_scales, sl.slot_of_row, sl.offsets + d.n_local_experts,
                                 d.top_k, d.d_model / 128, sl.x_perm_s, (int32_t)st->sz.cap,
                                 (int32_t)max_rows, stream_cus(st, s), s) != hipSuccess)
            return MOE_EHIP;
        if (fp8 && d.has_shared_expert &&
            launch_transpose_scales(mb->x_scales, T, d.d_model / 128, sl.xsh_s, d.max_tokens,
                                    s) != hipSuccess)
            return MOE_EHIP;
    }
    return rec ? record(sl, s) : MOE_OK;
}

// The two grouped GEMMs of one FFN pass on `s`: gate/up with the fused
// SiLU*up epilogue (fp8: and the quantisation of h), then down.  mt_max bounds
// the 256-row tiles of all groups together (grid sizes only).
static moe_status launch_ffn(moe_stage *st, GemmArgs &g1, GemmArgs &g2, int64_t mt_max,
                             hipStream_t s)
{
    const moe_stage_desc &d = st->desc;
    const bool fp8 = d.dtype == MOE_DTYPE_FP8_E4M3_B128;
    const int mt = mt_max > 0x7fffffff ? 0x7fffffff : (int)mt_max;
    const int32_t cap = (int32_t)st->sz.cap, tmax = d.max_tokens;
    hipError_t e;
    // bf16: groups of at most kSmallRows rows run in the small-group kernel,
    // the others in the 256x256-tile kernel (either may find no tiles).
    const int gmax = (int)st->sz.G;
    const int cus = stream_cus(st, s);
    {
        ProfScope ps(st, 2, s);
        if (fp8) {
            e = launch_gemm_fp8(g1, true, mt, gmax, cus, cap, tmax, s);
        } else {
            e = launch_gemm_bf16_small(g1, true, gmax, cus, s);
            if (e == hipSuccess) e = launch_gemm_bf16(g1, true, mt, cus, s);
        }
    }
    if (e == hipSuccess) {
        ProfScope ps(st, 3, s);
        if (fp8) {
            e = launch_gemm_fp8(g2, false, mt, gmax, cus, cap, tmax, s);
        } else {
            // the down product partitions the groups at kSmallRowsDown rows
            GemmArgs g2d = g2;
            g2d.groups = down_partition(g2.groups);
            e = launch_gemm_bf16_small(g2d, false, gmax, cus, s);
            if (e == hipSuccess) e = launch_gemm_bf16(g2d, false, mt, cus, s);
        }
    }
    if (e == hipErrorNotSupported) return MOE_EUNSUPPORTED;
    if (e != hipSuccess) return MOE_EHIP;
    return MOE_OK;
}

static moe_status ffn_impl(moe_stage *st, int32_t slot, void *stream, bool rec)
{
    if (!slot_ok(st, slot)) return MOE_EINVAL;
    SlotWs &sl = st->slots[slot];
    if (!sl.has_mb) return MOE_EINVAL;
    const moe_stage_desc &d = st->desc;
    const int32_t T = sl.mb.n_tokens;
    hipStream_t s = (hipStream_t)stream;
    if (T == 0) return rec ? record(sl, s) : MOE_OK;
    const bool fp8 = d.dtype == MOE_DTYPE_FP8_E4M3_B128;
    const int64_t max_rows = (int64_t)T * d.top_k;
    int64_t mt_max = (max_rows + kBM - 1) / kBM + d.n_local_experts;
    if (d.has_shared_expert) mt_max += (T + kBM - 1) / kBM;

    GemmArgs g1{};
    g1.A_routed = sl.mb.x;           // routed row r = token slot_of_row[r] / k of x
    g1.A_shared = sl.mb.x;
    g1.A_index = sl.slot_of_row;
    g1.A_index_div = d.top_k;
    g1.A_routed_rows = T;
    g1.As_routed = sl.x_perm_s;
    g1.As_shared = sl.xsh_s;
    g1.B = st->w1;
    g1.Bs = st->s1;
    g1.C_routed = sl.h;             // fp8: e4m3 codes, with their scales in Cs
    g1.C_shared = sl.h_sh;
    g1.Cs_routed = sl.h_s;
    g1.Cs_shared = sl.h_sh_s;
    g1.N = 2 * d.d_ff;
    g1.K = d.d_model;
    g1.shared_group = d.has_shared_expert ? d.n_local_experts : -1;
    g1.groups = sl.tables();
    g1.G = (int32_t)st->sz.G;
    g1.layer_id = sl.mb.layer_id;   // weights named on the device (NULL: layer 0)
    g1.layers = st->layers;
    g1.n_layers = d.n_layers;
    g1.down = 0;
    g1.err = st->err;

    GemmArgs g2 = g1;
    g2.A_index = nullptr;            // H rows are already grouped by expert
    g2.A_index_div = 0;
    g2.A_routed_rows = 0;
    g2.Cs_routed = nullptr;          // the down product writes bf16 Y
    g2.Cs_shared = nullptr;
    g2.A_routed = sl.h;
    g2.A_shared = sl.h_sh;
    g2.As_routed = sl.h_s;
    g2.As_shared = sl.h_sh_s;
    g2.B = st->w2;
    g2.Bs = st->s2;
    g2.down = 1;
    g2.C_routed = sl.y_perm;
    g2.C_shared = sl.y_sh;
    g2.N = d.d_model;
    g2.K = d.d_ff;

    const moe_status r = launch_ffn(st, g1, g2, mt_max, s);
    if (r != MOE_OK) return r;
    return rec ? record(sl, s) : MOE_OK;
}

// Pre-grouped rows: the tile tables come from the caller's device counts
// instead of the dispatch, the gate/up product reads the rows as they are,
// and the down product writes the caller's y.  No combine follows.
static moe_status ffn_grouped_impl(moe_stage *st, int32_t slot, const moe_grouped_batch *gb,
                                   hipStream_t s)
{
    if (!slot_ok(st, slot) || !gb) return MOE_EINVAL;
    const moe_stage_desc &d = st->desc;
    const bool fp8 = d.dtype == MOE_DTYPE_FP8_E4M3_B128;
    const int32_t n = gb->n_rows_max;
    if (n < 0 || n > st->sz.cap) return MOE_EINVAL;
    if (n > 0 && (!gb->rows || !gb->counts || !gb->y)) return MOE_EINVAL;
    if (n > 0 && fp8 && !gb->row_scales) return MOE_EINVAL;
    SlotWs &sl = st->slots[slot];
    sl.has_mb = false;               // nothing in this slot to combine
    if (n == 0) return record(sl, s);
    const GroupTable gt = sl.tables();
    {
        ProfScope ps(st, 0, s);
        if (launch_group_tables_from_counts(gb->counts, d.n_local_experts, n, gt, st->err, s) !=
            hipSuccess)
            return MOE_EHIP;
    }
    if (fp8) {                       // row scales, transposed as the fp8 GEMM reads them
        ProfScope ps(st, 1, s);
        if (launch_transpose_scales(gb->row_scales, n, d.d_model / 128, sl.x_perm_s,
                                    (int32_t)st->sz.cap, s) != hipSuccess)
            return MOE_EHIP;
    }
    GemmArgs g1{};
    g1.A_routed = gb->rows;
    g1.As_routed = fp8 ? sl.x_perm_s : nullptr;
    g1.B = st->w1;
    g1.Bs = st->s1;
    g1.C_routed = sl.h;
    g1.Cs_routed = sl.h_s;
    g1.N = 2 * d.d_ff;
    g1.K = d.d_model;
    g1.shared_group = -1;
    g1.groups = gt;
    g1.G = d.n_local_experts;
    g1.layer_id = gb->layer_id;
    g1.layers = st->layers;
    g1.n_layers = d.n_layers;
    g1.down = 0;
    g1.err = st->err;
    GemmArgs g2 = g1;
    g2.A_routed = sl.h;
    g2.As_routed = sl.h_s;
    g2.B = st->w2;
    g2.Bs = st->s2;
    g2.C_routed = gb->y;
    g2.Cs_routed = nullptr;
    g2.N = d.d_model;
    g2.K = d.d_ff;
    g2.down = 1;
    const moe_status r = launch_ffn(st, g1, g2, ((int64_t)n + kBM - 1) / kBM + d.n_local_experts, s);
    if (r != MOE_OK) return r;
    return record(sl, s);
}

static moe_status combine_impl(moe_stage *st, int32_t slot, void *stream, bool rec)
{
    if (!slot_ok(st, slot)) return MOE_EINVAL;
    SlotWs &sl = st->slots[slot];
    if (!sl.has_mb) return MOE_EINVAL;
    const moe_stage_desc &d = st->desc;
    hipStream_t s = (hipStream_t)stream;
    CombineArgs c{};
    c.y_perm = sl.y_perm;
    c.y_shared = d.has_shared_expert ? sl.y_sh : nullptr;
    c.row_of_slot = sl.row_of_slot;
    c.w = sl.mb.topk_w;
    c.out = sl.mb.out;
    c.T = sl.mb.n_tokens;
    c.k = d.top_k;
    c.d = d.d_model;
    c.accumulate = sl.mb.combine_mode == MOE_COMBINE_ACCUMULATE;
    {
        ProfScope ps(st, 4, s);
        if (launch_combine(c, stream_cus(st, s), s) != hipSuccess) return MOE_EHIP;
    }
    return rec ? record(sl, s) : MOE_OK;
}

moe_status moe_dispatch(moe_stage *st, int32_t slot, const moe_microbatch *mb, void *stream)
{
    return dispatch_impl(st, slot, mb, stream, true);
}

moe_status moe_expert_ffn(moe_stage *st, int32_t slot, void *stream)
{
    return ffn_impl(st, slot, stream, true);
}

moe_status moe_expert_ffn_grouped(moe_stage *st, int32_t slot, const moe_grouped_batch *gb,
                                  void *stream)
{
    return ffn_grouped_impl(st, slot, gb, (hipStream_t)stream);
}

moe_status moe_combine(moe_stage *st, int32_t slot, void *stream)
{
    return combine_impl(st, slot, stream, true);
}

moe_status moe_stage_submit_microbatch(moe_stage *st, const moe_microbatch *mb, void *stream,
                                       int32_t *slot_out)
{
    if (!mb_ok(st, mb)) return MOE_EINVAL;
    const int32_t slot = st->next_slot;
    SlotWs &sl = st->slots[slot];
    hipStream_t s = (hipStream_t)stream;
    // Backpressure: the slot's previous micro-batch must be done before its
    // workspace is reused.  The wait is on the device, for that one event.
    if (sl.ev_recorded && hipStreamWaitEvent(s, sl.ev, 0) != hipSuccess) return MOE_EHIP;
    moe_status r = dispatch_impl(st, slot, mb, stream, false);
    if (r != MOE_OK) return r;
    st->next_slot = (slot + 1) % (int32_t)st->slots.size();
    if ((r = ffn_impl(st, slot, stream, false)) != MOE_OK) return r;
    if ((r = combine_impl(st, slot, stream, true)) != MOE_OK) return r;
    if (slot_out) *slot_out = slot;
    return MOE_OK;
}

moe_status moe_quantize_fp8(const void *x_bf16, int32_t T, int32_t d, void *x_q, float *x_s,
                            void *stream)
{
    if (T < 0 || d <= 0 || d % 128) return MOE_EINVAL;
    if (T > 0 && (!x_bf16 || !x_q || !x_s)) return MOE_EINVAL;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return MOE_EHIP;
    if (launch_quantize_fp8(x_bf16, T, nullptr, d, x_q, x_s, 0, cus, (hipStream_t)stream) !=
        hipSuccess)
        return MOE_EHIP;
    return MOE_OK;
}

moe_status moe_stream_create_cu_masked(int32_t first_cu, int32_t n_cus, void **stream_out)
{
    if (!stream_out) return MOE_EINVAL;
    *stream_out = nullptr;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return MOE_EHIP;
    if (first_cu < 0 || n_cus < 1 || first_cu + n_cus > cus || cus > 32 * 32) return MOE_EINVAL;
    uint32_t mask[32] = {};
    for (int c = first_cu; c < first_cu + n_cus; ++c) mask[c >> 5] |= 1u << (c & 31);
    const uint32_t words = (uint32_t)((cus + 31) / 32);
    hipStream_t s = nullptr;
    const hipError_t e = hipExtStreamCreateWithCUMask(&s, words, mask);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return e == hipErrorOutOfMemory ? MOE_ENOMEM : MOE_EHIP;
    }
    *stream_out = (void *)s;
    return MOE_OK;
}

moe_status moe_stream_destroy(void *stream)
{
    if (!stream) return MOE_EINVAL;
    if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return MOE_EHIP;
    return hipStreamDestroy((hipStream_t)stream) == hipSuccess ? MOE_OK : MOE_EHIP;
}

moe_status moe_stage_poll(moe_stage *st, int32_t slot)
{
    if (!slot_ok(st, slot)) return MOE_EINVAL;
    SlotWs &sl = st->slots[slot];
    if (!sl.ev_recorded) return MOE_OK;
    const hipError_t e = hipEventQuery(sl.ev);
    if (e == hipSuccess) return MOE_OK;
    if (e == hipErrorNotReady) return MOE_EBUSY;
    return MOE_EHIP;
}

moe_status moe_stage_query(moe_stage *st, int32_t slot, moe_dispatch_view *v)
{
    if (!slot_ok(st, slot) || !v) return MOE_EINVAL;
    SlotWs &sl = st->slots[slot];
    v->counts = sl.counts;
    v->offsets = sl.offsets;
    v->slot_of_row = sl.slot_of_row;
    v->row_of_slot = sl.row_of_slot;
    v->x_perm = nullptr;              // the row gather is part of the gate/up GEMM
    v->x_perm_scales = sl.x_perm_s;
    v->h = sl.h;
    v->h_scales = sl.h_s;
    v->y_perm = sl.y_perm;
    v->h_shared = sl.h_sh;
    v->h_shared_scales = sl.h_sh_s;
    v->y_shared = sl.y_sh;
    v->capacity_rows = (int32_t)st->sz.cap;
    v->n_tokens = sl.has_mb ? sl.mb.n_tokens : 0;
    return MOE_OK;
}

moe_status moe_stage_profile(moe_stage *st, int32_t enable)
{
    if (!st) return MOE_EINVAL;
    st->prof_on = enable != 0;
    return MOE_OK;
}

moe_status moe_stage_profile_read(moe_stage *st, double *ms, int32_t *launches)
{
    if (!st || !ms || !launches) return MOE_EINVAL;
    for (int i = 0; i < MOE_PROF_KINDS; ++i) {
        ms[i] = 0.0;
        launches[i] = 0;
    }
    moe_status r = MOE_OK;
    for (auto &p : st->prof) {
        float t = 0.0f;
        if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&t, p.a, p.b) != hipSuccess)
            r = MOE_EHIP;
        else if (p.kind >= 0 && p.kind < MOE_PROF_KINDS) {
            ms[p.kind] += t;
            launches[p.kind] += 1;
        }
        hipEventDestroy(p.a);
        hipEventDestroy(p.b);
    }
    st->prof.clear();
    return r;
}

moe_status moe_ingest_wait(moe_stage *st, const uint32_t *ready, int32_t n_words, uint32_t epoch,
                           uint32_t spin_limit, void *stream)
{
    if (!st || !ready || n_words < 1 || n_words > kMaxIngestWords) return MOE_EINVAL;
    if (launch_ingest_wait(ready, n_words, epoch, spin_limit ? spin_limit : kDefaultIngestSpins,
                           st->err, (hipStream_t)stream) != hipSuccess)
        return MOE_EHIP;
    return MOE_OK;
}

moe_status moe_ingest_signal(uint32_t *word, uint32_t epoch, void *stream)
{
    if (!word) return MOE_EINVAL;
    return launch_ingest_signal(word, epoch, (hipStream_t)stream) == hipSuccess ? MOE_OK : MOE_EHIP;
}

moe_status moe_stage_sync(moe_stage *st)
{
    if (!st) return MOE_EINVAL;
    for (auto &sl : st->slots)
        if (sl.ev_recorded && hipEventSynchronize(sl.ev) != hipSuccess) return MOE_EHIP;
    int32_t err = 0;
    if (hipMemcpyAsync(&err, st->err, 4, hipMemcpyDeviceToHost, st->own) != hipSuccess ||
        hipStreamSynchronize(st->own) != hipSuccess)
        return MOE_EHIP;
    if (err) {
        if (hipMemsetAsync(st->err, 0, 4, st->own) != hipSuccess ||
            hipStreamSynchronize(st->own) != hipSuccess)
            return MOE_EHIP;
        return (err & kErrBadId)      ? MOE_EBADID
               : (err & kErrBadLayer) ? MOE_EBADLAYER
               : (err & kErrBadCount) ? MOE_EBADCOUNT
                                      : MOE_ETIMEOUT;
    }
    return MOE_OK;
}

}  // extern "C"
