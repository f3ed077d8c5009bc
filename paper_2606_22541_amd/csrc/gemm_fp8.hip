// e4m3 grouped GEMM with DeepSeek-style block scaling (fp8 variant of the
// expert stage): activations carry one fp32 scale per row and 128-channel
// group, weights one fp32 scale per 128x128 block.  Each K step covers
// exactly one 128-wide scale group g:
//
//   t    = sum over the group of e4m3(W) * e4m3(X)     (v_mfma 16x16x128 f8)
//   acc += t * (s_X[token, g] * s_W[block, g])          (fp32 promotion)
//
// so the block scales are applied exactly once per group in fp32.  The
// hardware's per-32-element power-of-two (E8M0) MFMA scales cannot express
// these fp32 scales and are left at 1.
//
// Design for gfx950:
//  * one persistent workgroup per CU walks the tiles of every group
//    (128-token x 256-feature tiles; the per-group tile counts are a prefix
//    the workgroup builds in LDS from the device row counts), XCD-aware:
//    consecutive tile numbers go to the 32 workgroups of one XCD, rastered
//    in bands of up to 8 token tiles so that each weight panel is read by
//    one XCD;
//  * the product is formed transposed, D[feature][token] = W X^T: the
//    weights are the MFMA's row operand and the tokens its column operand,
//    so each lane holds four consecutive features of ONE token and the
//    token's fp32 scale is a single value per lane and 16-token block;
//  * eight wave64s, wave w owning features 64 (w % 4) .. + 63 and tokens
//    64 (w / 4) .. + 63 of the tile as 4 x 4 blocks of
//    v_mfma_scale_f32_16x16x128_f8f6f4; the two waves of a SIMD (w and
//    w + 4) work in opposite phases, one reading its operands from LDS
//    while the other runs its MFMAs and promotion (the K loop below);
//  * K advances one scale group (128 bytes) per step through a 3-deep LDS
//    ring of 48.5 KB stages (32 KB of weight fragments, 16 KB of token rows,
//    the step's 128 token scales) filled by direct-to-LDS buffer loads two
//    groups ahead: every group issues the same seven loads per wave, so the
//    wait before a group is the constant vmcnt(7) (the next group's fills
//    stay in flight) and no wait drains the look-ahead.  The loads go out
//    one by one between the MFMAs: a stage is 49 loads of 1 KB per CU, about
//    as many clocks of the per-CU load path as the group's MFMAs take, and
//    issued as one burst they held back every wave's instructions;
//  * the weights are packed in the 16 x 128 fragment order of the MFMA (two
//    lane-contiguous 1 KB halves per fragment), gate and up rows interleaved
//    by 16, so each wave's 64 features are gate and up rows of the same 32 h
//    channels (one scalar scale each per group: the gate and the up 128 x 128
//    block) and a 256-feature gate/up tile covers exactly one 128-channel
//    group of h;
//  * token rows are 128-byte rows whose 16-byte chunks are XOR-swizzled by
//    (row / 2) % 8; rows past a group's end have an offset past every buffer
//    range and read as zero; the scalar offset, which the range check does
//    not cover, only moves along K (clamped to the last group) and between
//    weight fragments that exist;
//  * the gate/up product reads the routed token rows straight from x through
//    slot_of_row (the row gather is part of the token fills, as in bf16); the
//    rows' fp32 scales arrive already gathered and transposed, one
//    contiguous run of 128 per group, since reading them per token would cost
//    one cache line per lane and load;
//  * SwiGLU mode: every wave forms h = SiLU(gate) * up in fp32 for its 32
//    channels, the per-token |h| maximum over the tile's 128 channels meets
//    in a 2 KB LDS table, and each token's channels are quantised to e4m3
//    with one fp32 scale amax / 448 (the activation quantiser's scale;
//    the quotient is taken as a product with the scale's reciprocal), four
//    codes per lane and store.  The down product writes bf16, four
//    consecutive features per lane.
#include "kernels.h"

namespace moe {

namespace {

constexpr int kGrpB = 128;                   // K bytes per step: one scale group
constexpr int kTokT = 128;                   // tokens per tile
constexpr int kFeatT = 256;                  // features per tile
constexpr int kWBytes = kFeatT * kGrpB;      // weight fragments of one stage: 32 KB
constexpr int kXBytes = kTokT * kGrpB;       // token rows of one stage: 16 KB
constexpr int kXSBytes = kXBytes + kTokT * 4; // ... followed by the step's 128 token scales
constexpr int kWaves8 = 8;
constexpr int kThreads8 = 64 * kWaves8;
constexpr int kBand8 = 8;                    // token tiles per raster band
constexpr int kFillLoads = 7;                // loads per wave per group fill
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc8(const void *base, int64_t bytes)
{
    int32_t n = bytes > 0x7fffffff ? 0x7fffffff : (int32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

// Weight scales are read-only while a GEMM runs: reading them through the
// constant address space makes the per-group read a scalar load, which
// neither waits for nor counts against the in-flight direct-to-LDS fills (a
// flat load may alias LDS, so the compiler would drain the fills before it).
typedef const __attribute__((address_space(4))) float cfloat;

struct Tile8 {
    __amdgpu_buffer_rsrc_t rw, rx, rs;
    int vx[2];          // token fills: rows 16 w + 8 i + lane / 8, swizzled chunk (or past the range)
    int KT, ncb, cbstride, s_ld;
    const cfloat *sbp0; // weight scale of each K group: feature blocks rb = 0, 2 of this wave
    const cfloat *sbp1; //   ... and rb = 1, 3 (in SwiGLU mode the up rows; otherwise = sbp0)
};

struct Ring8 {
    uint8_t *w, *x;
    float *s;
};

// Fills of K group kg (clamped to the last) into one stage, 7 loads per wave:
//  * weight fragments 2 w and 2 w + 1 of the tile's 16, both 1 KB halves;
//  * token rows 16 w .. 16 w + 15 as two 8-row instructions; lane l writes
//    LDS row 16 w + 8 i + l / 8, physical chunk l % 8, with global chunk
//    (l % 8) ^ ((row / 2) % 8);
//  * 64 of the 128 token scales (waves w and w + 2, w + 4, w + 6 load the
//    same ones: identical data to identical addresses).
// Load i (0..6) of the fills: 0..3 the weight fragment halves, 4..5 the
// token rows, 6 the token scales.
__device__ __forceinline__ void fill8_one(const Tile8 &t, const Ring8 &st, int wave, int lane, int kg,
                                          int i)
{
    const int ks = min(kg, t.KT - 1);
    if (i < 4) {
        const int f = wave * 2 + (i >> 1), h = i & 1;
        const int cb = min(f, t.ncb - 1);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(t.rw, (lds_void *)(st.w + f * 2048 + h * 1024), 16,
                                                 lane * 16, cb * t.cbstride + ks * 2048 + h * 1024,
                                                 0, 0);
    } else if (i < 6) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(t.rx, (lds_void *)(st.x + (wave * 16 + (i - 4) * 8) * kGrpB),
                                                 16, t.vx[i - 4], ks * kGrpB, 0, 0);
    } else {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(t.rs, (lds_void *)(st.s + (wave & 1) * 64), 4,
                                                 (ks * t.s_ld + (wave & 1) * 64 + lane) * 4, 0, 0, 0);
    }
}

__device__ __forceinline__ void fill8(const Tile8 &t, const Ring8 &st, int wave, int lane, int kg)
{
#pragma unroll
    for (int i = 0; i < kFillLoads; ++i) fill8_one(t, st, wave, lane, kg, i);
}

struct Wave8 {
    int wave, lane, wf, wt;
    int w_rd;           // LDS byte offset of this lane's weight chunk (feature block 0)
    int x_rd0, x_rd1;   // LDS byte offsets of this lane's two token chunks (token block 0)
    int s_rd;           // LDS float index of this lane's token scale (token block 0)
};

// The K loop runs two waves per SIMD in opposite phases ("ping-pong"):
// waves 0..3 (tokens 0..63 of the tile) read group g's operands from LDS
// while waves 4..7 (tokens 64..127) run group g-1's MFMAs, and at the next
// barrier the roles swap, so one wave's LDS reads run under the other's
// matrix-core work instead of every wave reading, then every wave
// multiplying.  In slots E_g, O_g (one barrier before each):
//
//   slot   waves 0..3          waves 4..7
//   E_g    read g              MFMAs of g-1
//   O_g    MFMAs of g          read g
//
// Every wave issues its fills of group g+2 at the start of E_g, into the
// stage of group g-1, which waves 0..3 read in E_{g-1} (and consumed in
// O_{g-1}) and waves 4..7 in O_{g-1} (and waited for before E_g).  Before
// the barrier that starts E_g each wave waits for its own fills of g; only
// those of g+1 (seven loads) stay in flight.

// LDS reads of group g from stage S into registers: the four weight
// fragments, the NCB token fragments and their token scales.  The previous
// group's last token block is promoted here, under the reads' latency.
template <int S, int NCB>
__device__ __forceinline__ void read8(const Wave8 &w, const Ring8 (&ring)[3], i32x8 (&wfr)[4],
                                      i32x8 (&xf)[4], float (&st)[4], f32x4 (&acc)[4][4],
                                      const f32x4 (&pend)[4], const float (&ps)[2])
{
    if constexpr (NCB > 0) {
        const uint8_t *Ws = ring[S].w;
        const uint8_t *Xs = ring[S].x;
        const float *Ss = ring[S].s;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            const i32x4 lo = *(const i32x4 *)&Ws[w.w_rd + rb * 2048];
            const i32x4 hi = *(const i32x4 *)&Ws[w.w_rd + rb * 2048 + 1024];
            wfr[rb] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const i32x4 lo = *(const i32x4 *)&Xs[w.x_rd0 + cb * 16 * kGrpB];
            const i32x4 hi = *(const i32x4 *)&Xs[w.x_rd1 + cb * 16 * kGrpB];
            xf[cb] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            st[cb] = Ss[w.s_rd + cb * 16];
        }
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
            acc[rb][NCB - 1] = pend[rb] * ps[rb & 1] + acc[rb][NCB - 1];
    }
}

// The 4 x NCB MFMAs of one group, each token block's products promoted
// (acc += t * s_X * s_W) while the next block's MFMAs run; the last block's
// products are left in pend with their scales in ps.  The wave's seven fill
// loads of group kgf go out two per token block, after its second and fourth
// MFMA (the rest after the last MFMA when NCB < 4): the per-CU load path
// accepts about one 1 KB load every 19 clocks, and fills issued as one burst
// by every wave hold each wave's later instructions until the load path has
// taken them.
template <int NCB, bool FILL = true>
__device__ __forceinline__ void mfma8(const i32x8 (&wfr)[4], const i32x8 (&xf)[4],
                                      const float (&st)[4], float sb0, float sb1,
                                      f32x4 (&acc)[4][4], f32x4 (&pend)[4], float (&ps)[2],
                                      const Tile8 &t, const Ring8 &fst, int wave, int lane, int kgf)
{
    constexpr int kInter = !FILL ? 0 : (2 * NCB < kFillLoads) ? 2 * NCB : kFillLoads;
    if constexpr (NCB > 0) {
        f32x4 tq[2][4];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            // one token block: its four MFMAs with two fill loads, and the
            // previous block's promotion, in a fixed issue order (one MFMA,
            // then four promotion instructions, while the MFMA holds the
            // matrix core for 32 cycles)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const f32x4 p = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
                    wfr[rb], xf[cb], (f32x4){}, 0, 0, 0, 127, 0, 127);
                if (cb == NCB - 1) pend[rb] = p; else tq[cb & 1][rb] = p;
                const int j = 2 * cb + (rb >> 1);
                if ((rb & 1) && j < kInter) fill8_one(t, fst, wave, lane, kgf, j);
            }
            if (cb > 0) {
                const float s0 = st[cb - 1] * sb0, s1 = st[cb - 1] * sb1;
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
                    acc[rb][cb - 1] = tq[(cb - 1) & 1][rb] * ((rb & 1) ? s1 : s0) + acc[rb][cb - 1];
            }
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                        // MFMA
                if (cb > 0) __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);           // VALU
                if ((rb & 1) && 2 * cb + (rb >> 1) < kInter)
                    __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);                    // VMEM
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        ps[0] = st[NCB - 1] * sb0;
        ps[1] = st[NCB - 1] * sb1;
    }
#pragma unroll
    for (int i = kInter; i < (FILL ? kFillLoads : 0); ++i) fill8_one(t, fst, wave, lane, kgf, i);
}

// s_waitcnt operands (gfx9 encoding: vmcnt [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]).
constexpr int kWaitFills = (kFillLoads & 15) | ((kFillLoads >> 4) << 14) | (7 << 4) | (15 << 8);
constexpr int kWaitLds = 15 | (3 << 14) | (7 << 4) | (0 << 8);

// A slot boundary, with the wait before it: the scheduler moves nothing
// across it (a wait drawn into the slot before it would shorten the
// fills' look-ahead).
template <int WAIT>
__device__ __forceinline__ void slot_barrier()
{
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (WAIT >= 0) __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Group g (stage S) for a wave of either half.  LEAD: waves 0..3.  MFMA_PREV:
// the trailing half has a group g-1 to multiply (g > 0).
template <int S, int NCB, bool LEAD, bool MFMA_PREV>
__device__ __forceinline__ void group8(const Tile8 &t, const Wave8 &w, const Ring8 (&ring)[3],
                                       f32x4 (&acc)[4][4], i32x8 (&wfr)[4], i32x8 (&xf)[4],
                                       float (&st)[4], float (&sb)[2], float (&sb_next)[2],
                                       f32x4 (&pend)[4], float (&ps)[2], int kg)
{
    slot_barrier<kWaitFills>();                   // E_kg, after this wave's fills of group kg
    const Ring8 &fst = ring[(S + 2) % 3];         // group kg+2's stage, read last by group kg-1
    if constexpr (LEAD) {
        sb[0] = sb_next[0];
        sb[1] = sb_next[1];
        sb_next[0] = t.sbp0[min(kg + 1, t.KT - 1)];
        sb_next[1] = t.sbp1[min(kg + 1, t.KT - 1)];
        read8<S, NCB>(w, ring, wfr, xf, st, acc, pend, ps);
        slot_barrier<-1>();                       // O_kg
        mfma8<NCB>(wfr, xf, st, sb[0], sb[1], acc, pend, ps, t, fst, w.wave, w.lane, kg + 2);
    } else {
        if constexpr (MFMA_PREV)
            mfma8<NCB>(wfr, xf, st, sb[0], sb[1], acc, pend, ps, t, fst, w.wave, w.lane, kg + 2);
        else
            fill8(t, fst, w.wave, w.lane, kg + 2);
        slot_barrier<-1>();                       // O_kg
        sb[0] = sb_next[0];
        sb[1] = sb_next[1];
        sb_next[0] = t.sbp0[min(kg + 1, t.KT - 1)];
        sb_next[1] = t.sbp1[min(kg + 1, t.KT - 1)];
        read8<S, NCB>(w, ring, wfr, xf, st, acc, pend, ps);
        // the reads of stage S complete before E_{kg+1}, where it is refilled
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(kWaitLds);
    }
}

// The K loop of one tile for a wave of one half with NCB token blocks
// holding tokens.  Both halves pass 2 KT + 1 barriers.
template <bool LEAD, int NCB>
__device__ __forceinline__ void kloop8(const Tile8 &t, const Wave8 &w, const Ring8 (&ring)[3],
                                       f32x4 (&acc)[4][4])
{
    float sb[2] = {0.0f, 0.0f};
    float sb_next[2] = {t.sbp0[0], t.sbp1[0]};
    f32x4 pend[4] = {};
    float ps[2] = {0.0f, 0.0f};
    i32x8 wfr[4], xf[4];
    float st[4];
    __builtin_amdgcn_sched_barrier(0);
    fill8(t, ring[0], w.wave, w.lane, 0);
    fill8(t, ring[1], w.wave, w.lane, 1);
    // the first group (the trailing half has nothing to multiply yet), a
    // branch-free body of three groups (stage = group % 3), then the rest
    group8<0, NCB, LEAD, false>(t, w, ring, acc, wfr, xf, st, sb, sb_next, pend, ps, 0);
    int kg = 1;
    for (; kg + 3 <= t.KT; kg += 3) {
        group8<1, NCB, LEAD, true>(t, w, ring, acc, wfr, xf, st, sb, sb_next, pend, ps, kg);
        group8<2, NCB, LEAD, true>(t, w, ring, acc, wfr, xf, st, sb, sb_next, pend, ps, kg + 1);
        group8<0, NCB, LEAD, true>(t, w, ring, acc, wfr, xf, st, sb, sb_next, pend, ps, kg + 2);
    }
    if (kg < t.KT) group8<1, NCB, LEAD, true>(t, w, ring, acc, wfr, xf, st, sb, sb_next, pend, ps, kg);
    if (kg + 1 < t.KT) group8<2, NCB, LEAD, true>(t, w, ring, acc, wfr, xf, st, sb, sb_next, pend, ps, kg + 1);
    // E_KT: the trailing half multiplies the last group
    slot_barrier<-1>();
    if constexpr (!LEAD)
        mfma8<NCB, false>(wfr, xf, st, sb[0], sb[1], acc, pend, ps, t, ring[0], w.wave, w.lane, 0);
    if constexpr (NCB > 0) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
            acc[rb][NCB - 1] = pend[rb] * ps[rb & 1] + acc[rb][NCB - 1];
    }
}

}  // namespace

// One launch covers every group: tile L is (group, 128-token tile, 256-feature
// tile) in the band order above.
template <bool SWIGLU>
__global__ __launch_bounds__(kThreads8, 1)
void k_gemm_fp8(GemmArgs a, int32_t lds_rows_routed, int32_t lds_rows_shared)
{
    __shared__ __attribute__((aligned(1024))) uint8_t lds_w0[kWBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_w1[kWBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_w2[kWBytes];
    // token rows and token scales share one object per stage: the compiler
    // tracks a limited number of direct-to-LDS targets when it decides which
    // LDS reads must wait for which loads, and six stay within it
    __shared__ __attribute__((aligned(1024))) uint8_t lds_x0[kXSBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_x1[kXSBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_x2[kXSBytes];
    __shared__ int32_t ttab[kMaxLocalExperts + 2];    // prefix of 128-token tiles per group
    __shared__ float hmax[4][kTokT];                   // SwiGLU: |h| maximum per wave and token
    const Ring8 ring[3] = {{lds_w0, lds_x0, (float *)(lds_x0 + kXBytes)},
                           {lds_w1, lds_x1, (float *)(lds_x1 + kXBytes)},
                           {lds_w2, lds_x2, (float *)(lds_x2 + kXBytes)}};

    const int tid = threadIdx.x;
    Wave8 w;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    w.wf = w.wave & 3;
    w.wt = w.wave >> 2;
    const int lane = w.lane;
    const int N = a.N, K = a.K;
    const int NT = (N + kFeatT - 1) / kFeatT;
    const int G = a.G;

    // 128-token tiles per group, prefix over the groups (one wave)
    if (w.wave == 0) {
        int carry = 0;
        for (int c0 = 0; c0 < G; c0 += 64) {
            const int i = c0 + lane;
            const int m = i < G ? (a.groups.rows[i] + kTokT - 1) / kTokT : 0;
            int x = m;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int y = __shfl_up(x, o);
                if (lane >= o) x += y;
            }
            if (i < G) ttab[i] = carry + x - m;
            carry += __shfl(x, 63);
        }
        if (lane == 0) ttab[G] = carry;
    }
    __syncthreads();
    const int total = __builtin_amdgcn_readfirstlane(ttab[G] * NT);
    const int P = gridDim.x;
    const int first = (P & 7) ? (int)blockIdx.x : (int)((blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3));
    if (first >= total) return;      // no tile: leave before resolving the weights
    const void *Bw;
    const float *Bsw;
    resolve_weights(a, Bw, Bsw);

    // MFMA operand reads.  Weight fragment rb of this wave: feature block
    // 4 wf + rb, lane-contiguous halves.  Token block cb: lane l takes token
    // 64 wt + 16 cb + l % 16 and the 32 bytes [32 (l / 16), + 32) of its row.
    {
        const int r = w.wt * 64 + (lane & 15), swz = (r >> 1) & 7, c0 = 2 * (lane >> 4);
        w.w_rd = w.wf * 4 * 2048 + lane * 16;
        w.x_rd0 = r * kGrpB + ((c0 ^ swz) << 4);
        w.x_rd1 = r * kGrpB + (((c0 + 1) ^ swz) << 4);
        w.s_rd = r;
    }
    // token fills: lane l covers row 16 w + 8 i + l / 8, physical chunk l % 8;
    // ((row / 2) % 8) = (4 i + l / 16) % 8 since 16 w / 2 is a multiple of 8
    const int frow = w.wave * 16 + (lane >> 3);
    const int fch[2] = {((lane & 7) ^ ((lane >> 4) & 7)) << 4,
                        ((lane & 7) ^ ((4 + (lane >> 4)) & 7)) << 4};

    for (int L = first; L < total; L += P) {
        // decode: group g (largest with ttab[g] * NT <= L), then bands of up
        // to kBand8 token tiles, token tiles fastest
        int lo = 0, hi = G;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (ttab[mid] * NT <= L) lo = mid; else hi = mid;
        }
        const int g = __builtin_amdgcn_readfirstlane(lo);
        const int Lg = L - ttab[g] * NT;
        const int Mt = ttab[g + 1] - ttab[g];
        const int band = Lg / (kBand8 * NT);
        const int rr = Lg - band * kBand8 * NT;
        const int bm = min(kBand8, Mt - band * kBand8);
        const int mt = __builtin_amdgcn_readfirstlane(band * kBand8 + rr % bm);
        const int nt = __builtin_amdgcn_readfirstlane(rr / bm);
        const int grows = __builtin_amdgcn_readfirstlane(a.groups.rows[g]);
        const int row0 = __builtin_amdgcn_readfirstlane(a.groups.row0[g]) + mt * kTokT;
        const int rows_valid = min(kTokT, grows - mt * kTokT);
        const int n0 = nt * kFeatT;
        const bool sh = (g == a.shared_group);
        // routed rows of an indexed A are gathered in the token fills: tile
        // row r is row A_index[row0 + r] / A_index_div of the whole A (its
        // scales are already gathered, indexed by the routed row)
        const bool indexed = a.A_index != nullptr && !sh;
        const uint8_t *A = indexed ? (const uint8_t *)a.A_routed
                                   : (const uint8_t *)(sh ? a.A_shared : a.A_routed) + (int64_t)row0 * K;
        const float *As = (sh ? a.As_shared : a.As_routed) + row0;      // [K/128][ld]
        const uint8_t *B = (const uint8_t *)Bw + ((int64_t)g * N + n0) * K;
        Tile8 t;
        t.KT = K / kGrpB;
        t.s_ld = sh ? lds_rows_shared : lds_rows_routed;
        t.ncb = min(kFeatT, N - n0) / 16;
        t.cbstride = t.KT * 2048;
        t.rw = rsrc8(B, (int64_t)t.ncb * t.cbstride);
        t.rx = rsrc8(A, (indexed ? a.A_routed_rows : (int64_t)rows_valid) * K);
        t.rs = rsrc8(As, ((int64_t)(t.KT - 1) * t.s_ld + rows_valid) * 4);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int r = frow + 8 * i;
            t.vx[i] = r < rows_valid ? (indexed ? a.A_index[row0 + r] / a.A_index_div : r) * K + fch[i]
                                     : (int)0x80000000u;
        }
        const float *sbp0, *sbp1;
        if constexpr (SWIGLU) {
            // [G][f/128][gate, up][K/128]: tile nt covers gate/up scale block nt
            const int f = N / 2;
            sbp0 = Bsw + ((int64_t)g * (f / 128) + nt) * 2 * t.KT;
            sbp1 = sbp0 + t.KT;
        } else {
            // [G][N/128][K/128]: wave features n0 + 64 wf .. + 63
            const int nb = min(2 * nt + (w.wf >> 1), N / 128 - 1);
            sbp0 = sbp1 = Bsw + ((int64_t)g * (N / 128) + nb) * t.KT;
        }
        t.sbp0 = (const cfloat *)(uintptr_t)sbp0;
        t.sbp1 = (const cfloat *)(uintptr_t)sbp1;

        f32x4 acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = (f32x4){};

        // 16-token blocks of this wave's 64 tokens that hold tokens of the group
        const int ncbw = __builtin_amdgcn_readfirstlane(
            min(4, max(0, rows_valid - w.wt * 64 + 15) / 16));
        if (w.wt == 0) {
            switch (ncbw) {
            case 0: kloop8<true, 0>(t, w, ring, acc); break;
            case 1: kloop8<true, 1>(t, w, ring, acc); break;
            case 2: kloop8<true, 2>(t, w, ring, acc); break;
            case 3: kloop8<true, 3>(t, w, ring, acc); break;
            default: kloop8<true, 4>(t, w, ring, acc); break;
            }
        } else {
            switch (ncbw) {
            case 0: kloop8<false, 0>(t, w, ring, acc); break;
            case 1: kloop8<false, 1>(t, w, ring, acc); break;
            case 2: kloop8<false, 2>(t, w, ring, acc); break;
            case 3: kloop8<false, 3>(t, w, ring, acc); break;
            default: kloop8<false, 4>(t, w, ring, acc); break;
            }
        }
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0): the clamped look-ahead fills
        __syncthreads();                                     // ring idle in every wave

        // Accumulator register i of block (rb, cb) holds feature
        // 16 rb + 4 (lane / 16) + i of the wave and token 16 cb + lane % 16.
        const int tok = w.wt * 64 + (lane & 15);        // + 16 cb
        const int fq = 4 * (lane >> 4);                 // + 16 rb + i
        if constexpr (SWIGLU) {
            // Gate and up rows interleave by 16: blocks rb = 2 p and 2 p + 1 are
            // gate and up of h channels 32 wf + 16 p + 4 (lane / 16) + i of the
            // tile's 128, so every wave forms its own h.  A token's scale needs
            // |h| over all 128 channels: each wave reduces its 32 (lanes
            // l, l ^ 16, l ^ 32, l ^ 48 hold the same token), and the four
            // waves of the same tokens meet in LDS.
            const int f = N / 2;
            f32x4 h[2][4];
            float am[4];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                float m = 0.0f;
#pragma unroll
                for (int pq = 0; pq < 2; ++pq)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float hv = silu_mul(acc[2 * pq][cb][i], acc[2 * pq + 1][cb][i]);
                        h[pq][cb][i] = hv;
                        m = fmaxf(m, fabsf(hv));
                    }
                m = fmaxf(m, __shfl_xor(m, 16));
                am[cb] = fmaxf(m, __shfl_xor(m, 32));
                if (lane < 16) hmax[w.wf][tok + 16 * cb] = am[cb];
            }
            __syncthreads();
            uint8_t *H = (uint8_t *)(sh ? a.C_shared : a.C_routed);
            float *Hs = (sh ? a.Cs_shared : a.Cs_routed) + (int64_t)nt * t.s_ld + row0;
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const int tk = tok + 16 * cb;
                const float amax = fmaxf(fmaxf(hmax[0][tk], hmax[1][tk]), fmaxf(hmax[2][tk], hmax[3][tk]));
                const float sc = amax > 0.0f ? amax / 448.0f : 1.0f;   // the activation quantiser's scale
                const float inv = __builtin_amdgcn_rcpf(sc);
                if (tk < rows_valid) {
                    uint8_t *dst = H + (int64_t)(row0 + tk) * f + nt * 128 + w.wf * 32 + fq;
#pragma unroll
                    for (int pq = 0; pq < 2; ++pq)
                        *(uint32_t *)(dst + 16 * pq) =
                            e4m3_pack4(h[pq][cb][0] * inv, h[pq][cb][1] * inv,
                                       h[pq][cb][2] * inv, h[pq][cb][3] * inv);
                    if (w.wf == 0 && lane < 16) Hs[tk] = sc;
                }
            }
        } else {
            bf16 *C = (bf16 *)(sh ? a.C_shared : a.C_routed);
            const int fb = n0 + w.wf * 64 + fq;
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const int tk = tok + 16 * cb;
                if (tk < rows_valid) {
                    bf16 *dst = C + (int64_t)(row0 + tk) * N + fb;
#pragma unroll
                    for (int rb = 0; rb < 4; ++rb) {
                        if (fb + rb * 16 < N) {
                            typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
                            const bf16x4 v = {f2bf(acc[rb][cb][0]), f2bf(acc[rb][cb][1]),
                                              f2bf(acc[rb][cb][2]), f2bf(acc[rb][cb][3])};
                            *(bf16x4 *)(dst + rb * 16) = v;
                        }
                    }
                }
            }
        }
    }
}

hipError_t launch_gemm_fp8(const GemmArgs &a, bool swiglu, int mt_max, int g_max, int num_cus,
                           int32_t lds_rows_routed, int32_t lds_rows_shared, hipStream_t s)
{
    (void)g_max;
    if (mt_max <= 0) return hipSuccess;
    if (a.K % 128 || a.N % 128 || (swiglu && a.N % 256)) return hipErrorNotSupported;
    if (a.G < 1 || a.G > kMaxLocalExperts + 1) return hipErrorNotSupported;
    // 128-token tiles: at most two per 256-row tile of the bound
    const int64_t tiles = (int64_t)2 * mt_max * ((a.N + kFeatT - 1) / kFeatT);
    int grid = num_cus < tiles ? num_cus : (int)tiles;
    if (grid >= 8) grid &= ~7;
    if (swiglu)
        hipLaunchKernelGGL(k_gemm_fp8<true>, dim3(grid), dim3(kThreads8), 0, s, a,
                           lds_rows_routed, lds_rows_shared);
    else
        hipLaunchKernelGGL(k_gemm_fp8<false>, dim3(grid), dim3(kThreads8), 0, s, a,
                           lds_rows_routed, lds_rows_shared);
    return hipGetLastError();
}

}  // namespace moe
