// ResidualAttention decode for gfx950 (Section 5.3, Algorithm 1).
//
// One workgroup = one (work item, KV head h), four waves.  A work item is a page range
// of a segment together with the agents that read the same base pages there, in groups
// of agents whose query heads of KV head h fill the 16 rows of one matrix-core tile.  An
// item of ng groups runs on the four waves as ng groups x 4/ngp copies (ngp = ng rounded
// up to 1, 2 or 4); each copy covers its share of the pages, the copies of a group merge
// their partial rows (acc, acc_r, m, l) in LDS, and the group writes one partial per
// agent.  A second kernel merges an agent's partials (log-sum-exp combine) and applies
// Stage 3.  Without RoPE (decode_split_kernel):
//  - items of one group (private suffixes): the waves stride over the pages with a
//    register-double-buffered pipeline;
//  - items of two to four groups (shared prefixes): each base K/V block is copied once
//    from memory straight into an LDS ring (three stages ahead) and every wave applies it
//    to its own group's 16 rows, so a shared page crosses the memory hierarchy once per
//    workgroup instead of once per group.
// With RoPE (decode_rope_kernel) every wave streams its pages straight into registers and
// rebuilds its agents' keys (see there).
//
// Per page and wave (all products on the matrix cores, fp32 accumulate):
//   S^T  = K_base . Q^T                               16x16x32, all rows of the wave
//   residual key term, per agent slot s of the wave's group:
//     RoPE off: S^T += C_K,s . (B_K,s . q)^T          q folded into B_K once
//     RoPE on : U^T  = B_K,s^T . C_K,s^T              Stage 1, rebuilt in registers
//               K_lora = RoPE_p(U)                    rotate-half, fp32
//               S^T += K_lora . Q_s^T
//   online softmax (Stage 2) on S^T, rows in lanes, tokens in the 4 lane groups
//   O^T     += V_base^T . P^T                          acc of Algorithm 1
//   acc_r^T += C_V,s^T . P_s^T                         rank-space accumulator
// The reconstructed K never leaves registers; the value residual stays in rank
// space until the combine kernel applies B_V once (Eq. 4).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <type_traits>

#include "internal.hpp"
#include "lds_dma.hpp"
#include "mfma.hpp"

using namespace fkvk;

namespace {

constexpr int D = 128;
constexpr int PS = 16;
constexpr int ROWS = 16;
constexpr int WAVES = 4;
constexpr float kNegInf = -INFINITY;
constexpr int kMaxPagesPerItem = fkv::kMaxPagesPerItem;
constexpr int kBlockHalfs = PS * D;  // bf16 values in one (page, K|V, head) block
constexpr int kBlockBytes = kBlockHalfs * 2;

struct DecodeArgs {
    const uint16_t *q, *base_kv, *res_kv, *lora_b;
    const int32_t *adapter_idx, *base_bt, *res_bt, *seq_lens;
    const float *rope_cos, *rope_sin;
    const int32_t *plan;
    float *ws;
    uint16_t *out;
    int32_t hq, hkv, max_pages, ws_stride;
    int32_t off_items, off_blocks, off_ptr, off_zero, off_desc;  // plan section offsets (words)
    float scale_log2;  // softmax scale * log2(e)
    int64_t ws_bytes;  // bytes of the partial-row area of the workspace
    int32_t n_rows;    // query rows to merge: n_agents * hq
    int32_t rope_max_pos;  // rows of the RoPE tables
};

constexpr int cmax(int a, int b) { return a > b ? a : b; }

// Base-page ring of the multi-group decode path: kRing stages of two pages (K and V
// blocks of one head), written by direct memory-to-LDS copies.
constexpr int kRing = 4;
constexpr int kStageBytes = 4 * kBlockBytes;

// Ring stage hand-over: this wave's copies older than its last N vector-memory operations
// have landed in LDS (and its LDS reads of the previous stage completed inside their own
// instruction groups), then all waves meet.  A plain barrier: the copies are ordered by
// the count, not by a memory fence that would wait for every copy still in flight.
template <int N>
__device__ __forceinline__ void stage_barrier() {
    wait_vmcnt<N>();
    __builtin_amdgcn_s_barrier();
}
constexpr int cmin(int a, int b) { return a < b ? a : b; }

// Partial row record in the workspace (floats): acc[D], acc_r[R], m, l; stride
// rounded up to a multiple of 4 so every record is 16-byte aligned.
__host__ __device__ constexpr int ws_stride_of(int r) { return (D + r + 2 + 3) / 4 * 4; }

// Partial rows travel from the split kernel to the merge kernel.  They are written and read
// at device scope (cache policy sc1: coherent across the XCDs' L2 caches, no cache
// write-back or invalidation needed), 16 bytes per lane, through a buffer resource over the
// workspace (byte offsets below 4 GiB).
__device__ void raw_buffer_store_v4f32(f32x4 data, i32x4 rsrc, int voffset, int soffset, int aux) __asm("llvm.amdgcn.raw.buffer.store.v4f32");
__device__ f32x4 raw_buffer_load_v4f32(i32x4 rsrc, int voffset, int soffset, int aux) __asm("llvm.amdgcn.raw.buffer.load.v4f32");
constexpr int kDeviceCoherent = 16;  // cache-policy operand: sc1
__device__ __forceinline__ i32x4 workspace_rsrc(const float *ws, int64_t bytes) {
    return block_rsrc(reinterpret_cast<uint64_t>(ws), (int)(bytes < 0x7fffffff ? bytes : 0x7fffffff));
}

// ---------------------------------------------------------------------------
// Per-wave row state and the page update shared by both kernels.
template <int R>
struct Rows {
    static constexpr int RT = R == 0 ? 0 : (R + 15) / 16;  // 16-wide rank tiles
    static constexpr int RTX = RT > 0 ? RT : 1;
    f32x4 oacc[8];     // O^T[16mt + 4grp + i][row col]
    f32x4 racc[RTX];   // acc_r^T[16t + 4grp + i][row col]
    float m, l;
    __device__ __forceinline__ void init() {
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) oacc[mt] = f32x4{0, 0, 0, 0};
#pragma unroll
        for (int t = 0; t < RTX; ++t) racc[t] = f32x4{0, 0, 0, 0};
        m = kNegInf;
        l = 0.f;
    }
};


// Stage 2 on one page's S^T tile plus the value products.  Tokens tok0+4grp+i at or
// past `len` (this lane's row's sequence length; only tested with LEN_MASK, which a caller
// may leave off for a page inside every row's sequence) or on an invalid page get zero weight;
// vf must already be zero for tokens past every row's length, cv for tokens past its
// slot's residual length.
//
// The running maximum m is only moved (and acc, acc_r, l rescaled) when some row's new
// scores exceed it by more than 2^kLazyRescale; otherwise the weights 2^(s - m) of this
// page stay below 2^kLazyRescale.  acc, acc_r and l always refer to the same m, so the
// partial is exact whichever m it ends with.
constexpr float kLazyRescale = 8.f;

template <int R, int NS, bool LEN_MASK = true>
__device__ __forceinline__ void softmax_pv(Rows<R> &st, f32x4 sacc, bool valid, int tok0, int len, float scale_log2,
                                           const u32x2 *vf, const u32x2 (*cv)[Rows<R>::RTX], int my_slot_l,
                                           int grp) {
    float sv[4];
    float mx = kNegInf;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int tok = tok0 + 4 * grp + i;
        sv[i] = (valid && (!LEN_MASK || tok < len)) ? sacc[i] * scale_log2 : kNegInf;
        mx = fmaxf(mx, sv[i]);
    }
    mx = max_over_groups(mx);
    if (__builtin_amdgcn_ballot_w64(mx > st.m + kLazyRescale) != 0) {
        const float m_new = fmaxf(st.m, mx);
        const float alpha = fast_exp2(st.m - (m_new == kNegInf ? 0.f : m_new));
        st.l *= alpha;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) st.oacc[mt] *= alpha;
#pragma unroll
        for (int t = 0; t < Rows<R>::RT; ++t) st.racc[t] *= alpha;
        st.m = m_new;
    }
    const float m_use = st.m == kNegInf ? 0.f : st.m;
    f32x4 pv;
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        pv[i] = fast_exp2(sv[i] - m_use);
        psum += pv[i];
    }
    st.l += psum;
    const u32x2 pf = pack4(pv);
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) st.oacc[mt] = mfma16(vf[mt], pf, st.oacc[mt]);
    if constexpr (R > 0) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const u32x2 pm = my_slot_l == s ? pf : u32x2{0, 0};
#pragma unroll
            for (int t = 0; t < Rows<R>::RT; ++t) st.racc[t] = mfma16(cv[s][t], pm, st.racc[t]);
        }
    }
}

// This wave's partial rows, straight from the accumulators (l summed over lane groups).
template <int R>
__device__ __forceinline__ void write_partial(const DecodeArgs &p, Rows<R> &st, bool row_active, int64_t prow,
                                              int grp) {
    st.l += __shfl_xor(st.l, 16);
    st.l += __shfl_xor(st.l, 32);
    if (!row_active) return;
    const i32x4 rs = workspace_rsrc(p.ws, p.ws_bytes);
    const int dst = (int)(prow * p.ws_stride * 4);  // byte offset of the record
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) raw_buffer_store_v4f32(st.oacc[mt], rs, dst + (16 * mt + 4 * grp) * 4, 0, kDeviceCoherent);
#pragma unroll
    for (int t = 0; t < Rows<R>::RT; ++t)
        if (16 * t + 4 * grp < R) raw_buffer_store_v4f32(st.racc[t], rs, dst + (D + 16 * t + 4 * grp) * 4, 0, kDeviceCoherent);
    if (grp == 0) raw_buffer_store_v4f32(f32x4{st.m, st.l, 0.f, 0.f}, rs, dst + (D + R) * 4, 0, kDeviceCoherent);
}

// The wave copies of one agent group (waves my_group + ngp c, c < copies) each hold a partial
// of the same 16 rows over their share of the pages.  Copies c > 0 leave theirs in LDS (`buf`,
// at least 4 x (9 + RT) x 1 KB) and copy 0 merges them into its own (the weights 2^(m_c - M)
// of a log-sum-exp merge; acc, acc_r and l of a copy always refer to its m), so the group
// writes one partial.  Every wave of the block calls this; the LDS the block used before is
// free once all waves have arrived.
template <int R>
__device__ __forceinline__ void merge_wave_copies(Rows<R> &st, int wave, int copy, int my_group, int ngp, int copies,
                                                  f32x4 *buf) {
    constexpr int RTX = Rows<R>::RTX;
    constexpr int NF4 = 8 + RTX + 1;  // oacc, racc, (m, l) of a lane, in float4 units
    const int lane = threadIdx.x & 63;
    __syncthreads();
    if (copy > 0) {
        f32x4 *dst = buf + wave * NF4 * 64 + lane;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) dst[mt * 64] = st.oacc[mt];
#pragma unroll
        for (int t = 0; t < RTX; ++t) dst[(8 + t) * 64] = st.racc[t];
        dst[(8 + RTX) * 64] = f32x4{st.m, st.l, 0.f, 0.f};
    }
    __syncthreads();
    if (copy == 0) {
        for (int c = 1; c < copies; ++c) {
            const f32x4 *src = buf + (my_group + ngp * c) * NF4 * 64 + lane;
            const f32x4 ml = src[(8 + RTX) * 64];
            const float M = fmaxf(st.m, ml.x);
            const float Mu = M == kNegInf ? 0.f : M;
            const float w0 = fast_exp2(st.m - Mu), w1 = fast_exp2(ml.x - Mu);
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) st.oacc[mt] = st.oacc[mt] * w0 + src[mt * 64] * w1;
#pragma unroll
            for (int t = 0; t < RTX; ++t) st.racc[t] = st.racc[t] * w0 + src[(8 + t) * 64] * w1;
            st.l = st.l * w0 + ml.y * w1;
            st.m = M;
        }
    }
}
constexpr int merge_lds_bytes(int r) { return 4 * (8 + (r > 0 ? (r + 15) / 16 : 1) + 1) * 64 * 16; }

// Q^T as the B operand of the 16x16x32 products.  The head-dim index of slot j in
// k-step kk is 32kk + 16(j/4) + 4grp + j%4 for this lane group: the order in which
// a rebuilt key tile leaves the 16x16x16 accumulators and in which K blocks are
// stored, so base keys, rebuilt keys and queries all share it.
__device__ __forceinline__ void load_q(const uint16_t *qrow, bool active, int grp, u32x4 *qf) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        u32x4 v = {0, 0, 0, 0};
        if (active) {
            const u32x2 lo = ldg64(qrow + 32 * kk + 4 * grp);
            const u32x2 hi = ldg64(qrow + 32 * kk + 16 + 4 * grp);
            v = u32x4{lo.x, lo.y, hi.x, hi.y};
        }
        qf[kk] = v;
    }
}

// Lane-constant element offsets (within one agent's rCache page: C_K [16][R] then
// C_V^T [R][16]) of the fragments this lane reads, and whether they are inside R.
template <int R>
struct ResOffsets {
    static constexpr int RTX = Rows<R>::RTX;
    int ck[RTX], cv[RTX];
    bool ck_ok[RTX], cv_ok[RTX];
    __device__ __forceinline__ ResOffsets(int col, int grp) {
#pragma unroll
        for (int t = 0; t < RTX; ++t) {
            const int rho = 16 * t + col, rk = 16 * t + 4 * grp;
            cv_ok[t] = rho < R;
            ck_ok[t] = rk < R;
            cv[t] = PS * R + (rho < R ? rho : (R > 0 ? R - 1 : 0)) * PS + 4 * grp;  // C_V^T[rho][tok 4grp..]
            ck[t] = col * R + (rk < R ? rk : (R >= 4 ? R - 4 : 0));                 // C_K[tok col][rho 4grp..]
        }
    }
};

// ---------------------------------------------------------------------------
// RoPE off.  One workgroup per (work item, KV head), four waves; wave w serves agent
// group w % ngp as copy w / ngp.  Items of several groups (shared prefixes) stream their
// base pages through an LDS ring of kRing stages of two pages, written by direct
// memory-to-LDS copies kRing - 1 stages ahead (each wave copies one 4 KB block per
// stage); a wave computes its share of a stage as one step of two pages (four groups:
// the whole stage, so one 16x16x32 instruction covers 32 keys of the value products) or
// of one page (two groups: page `copy`).  Items of one group stride over their pages
// straight from memory into registers, one or two pages ahead.  Every wave's rCache
// fragments come straight from memory (one 16-byte load per slot, page and rank tile),
// two stages ahead on the ring path.
template <int R, int G>
struct SplitShape {
    static constexpr int AG = ROWS / G;                                         // agents per group
    static constexpr int RT = R == 0 ? 0 : (R + 15) / 16;                       // 16-wide rank tiles
    static constexpr int RTX = RT > 0 ? RT : 1;
    static constexpr int NG = fkv::decode_item_groups(G, R);                    // agent groups per item
    static constexpr bool MULTI = NG > 1;                                       // several groups per item
    static constexpr int NSW = fkv::decode_wave_slots(G, R);                    // agent slots per wave
    static constexpr int NSR = R > 0 ? NSW : 1;
    static constexpr int MAX_SLOTS = MULTI ? cmin(NG * AG, fkv::kMaxItemAgents) : NSW;
    static constexpr int RES_PAGE = RT * 512;                                   // rCache page (halfs)
};

template <int R, int G>
__device__ __forceinline__ void split_body(const DecodeArgs &p) {
    using S = SplitShape<R, G>;
    constexpr int AG = S::AG;
    constexpr int RT = S::RT;
    constexpr int RTX = S::RTX;
    constexpr int NSW = S::NSW;
    constexpr int NSR = S::NSR;
    struct CFrag {  // rCache fragments (C_K in .xy, C_V in .zw) of the wave's slots for its step pages
        u32x4 kv[2][NSR][RTX];
    };
    __shared__ __attribute__((aligned(16))) u32x4 lds_ring[kRing * kStageBytes / 16];

    // The block's descriptor (at an address that depends on blockIdx only) names the item:
    // page range start and capacity, KV head, the agent whose base block-table row names the
    // item's pages, every slot's agent and first partial.  Page ids, sequence lengths and
    // adapters come from the launch's own tables in the next round of loads, after which the
    // first base pages, rCache rows, queries and B_K slices are all requested together.
    const int32_t *desc = p.plan + p.off_desc + (int64_t)blockIdx.x * fkv::kDescWords;
    const int pg0 = desc[fkv::kDescPg0], pgcap = desc[fkv::kDescCap], nag = desc[fkv::kDescNag];
    const int h = desc[fkv::kDescHead], leader = desc[fkv::kDescLeader];
    const int npcap = pgcap - pg0;
    const int hkv = p.hkv;
    const int ng = (nag + AG - 1) / AG;
    if (nag <= 0 || npcap <= 0 || nag > S::MAX_SLOTS || (ng > 1 && !S::MULTI) || (ng == 1 && nag > NSW) ||
        npcap > (ng > 2 ? fkv::kMaxPagesMulti : fkv::kMaxPagesSingle))
        return;  // idle block, or rejected on the host
    const int ngp = ng == 1 ? 1 : (ng == 2 ? 2 : 4);   // groups rounded to a divisor of 4

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int my_group = wave % ngp;
    const int copy = wave / ngp;
    const int sb = my_group * AG;                       // first item slot of this wave's group
    const int my_slot = col / G;                        // this lane's row: slot within the group
    const bool row_active = my_slot < NSW && sb + my_slot < nag;
    const int qh = h * G + (col % G);
    const int64_t n = (int64_t)hkv * D;

    // lane i < nag of every wave holds item slot i: agent and first partial (plan), sequence
    // length and adapter (launch arrays); lane i (and 64 + i) holds the base page id of item
    // page i (the leader's row) and, per slot s of this wave's group, that slot's rCache page
    // id (-1: no adapter).  Entries past the capacity repeat the last one.
    const bool lane_ag = lane < nag;
    const int l_agent = lane_ag ? desc[fkv::kDescAgent + lane] : 0;
    const int l_part = lane_ag ? desc[fkv::kDescPart + lane] : 0;
    const int l_len = lane_ag ? p.seq_lens[l_agent] : 0;
    const int l_ad = (R > 0 && lane_ag) ? p.adapter_idx[l_agent] : -1;
    const int32_t *brow = p.base_bt + (int64_t)leader * p.max_pages + pg0;
    const int bid0 = brow[min(lane, npcap - 1)];
    const int bid1 = brow[min(64 + lane, npcap - 1)];
    int rid0[NSR], rid1[NSR];
#pragma unroll
    for (int s = 0; s < NSR; ++s) {
        const bool ok = R > 0 && s < NSW && sb + s < nag;
        const int ag_s = __builtin_amdgcn_readlane(l_agent, (sb + s) & 63);
        const int32_t *row = p.res_bt + (int64_t)(ok ? ag_s : 0) * p.max_pages + pg0;
        rid0[s] = ok ? row[min(lane, npcap - 1)] : -1;
        rid1[s] = (ok && npcap > 64) ? row[min(64 + lane, npcap - 1)] : -1;
    }
    // the item's longest sequence bounds the pages it reads (up to its capacity)
    int item_max_len = 0;
    for (int s = 0; s < nag; ++s) item_max_len = max(item_max_len, __builtin_amdgcn_readlane(l_len, s));
    const int npg = min(pgcap, (item_max_len + PS - 1) / PS) - pg0;
    const int pg1 = pg0 + max(npg, 0);
    // device address of the K block of (item page k, head h); V follows hkv blocks later.
    // Pages past the item repeat its last page, so loads issued ahead of the end stay valid.
    // (both table halves are read and the half is chosen on the scalar unit: no branch and
    // no vector temporary)
    auto base_addr = [&](int k) __attribute__((always_inline)) -> uint64_t {
        k = min(k, npg - 1);
        const int lo = __builtin_amdgcn_readlane(bid0, k & 63), hi = __builtin_amdgcn_readlane(bid1, k & 63);
        const int id = k < 64 ? lo : hi;
        return reinterpret_cast<uint64_t>(p.base_kv + ((int64_t)id * 2 * hkv + h) * kBlockHalfs);
    };
    // device address of the rCache page of (item page k, wave slot s); the plan's zero area
    // stands in for a slot without adapter
    const uint16_t *zero_c = reinterpret_cast<const uint16_t *>(p.plan + p.off_zero);
    auto res_addr = [&](int k, int s) __attribute__((always_inline)) -> uint64_t {
        k = min(k, npg - 1);
        const int lo = __builtin_amdgcn_readlane(rid0[s], k & 63), hi = __builtin_amdgcn_readlane(rid1[s], k & 63);
        const int id = k < 64 ? lo : hi;
        return reinterpret_cast<uint64_t>(id >= 0 ? p.res_kv + (int64_t)id * S::RES_PAGE : zero_c);
    };

    // per slot of the wave's group: adapter (or -1) and sequence length
    int slot_ad[NSR], slot_len[NSR];
    int min_len = 1 << 30, min_res = 1 << 30;  // shortest sequence / rCache among the group's slots
#pragma unroll
    for (int s = 0; s < NSR; ++s) {
        const bool ok = sb + s < nag && s < NSW;
        const int ad = __builtin_amdgcn_readlane(l_ad, (sb + s) & 63);
        const int len = __builtin_amdgcn_readlane(l_len, (sb + s) & 63);
        slot_ad[s] = (ok && R > 0) ? ad : -1;
        slot_len[s] = ok ? len : 0;
        if (ok) min_len = min(min_len, len);
        if (ok && slot_ad[s] >= 0) min_res = min(min_res, len);
        if (slot_ad[s] < 0) rid0[s] = rid1[s] = -1;   // no adapter: the zero area
    }
    const int src_lane = (sb + my_slot) & 63;
    const int sh_agent = __shfl(l_agent, src_lane), sh_len = __shfl(l_len, src_lane);
    const int my_part = __shfl(l_part, src_lane);  // this lane's row's partial
    const int my_agent = row_active ? sh_agent : 0;
    const int my_len = row_active ? sh_len : 0;
    const int64_t my_row = ((int64_t)my_part * G + col % G) * hkv + h;
    if (npg <= 0) {  // the item's agents have not reached it yet: an empty partial (weight 0)
        Rows<R> empty;
        empty.init();
        if (copy == 0) write_partial<R>(p, empty, row_active, my_row, grp);
        return;
    }

    // Query fragments and W = B_K q.  Their loads are issued after the first base pages
    // and rCache rows have been requested (each pipeline below calls this right after its
    // first loads), so the prologue's latency overlaps the start of the stream.
    u32x4 qf[4];        // Q^T fragments (B operand of the 16x16x32 products)
    u32x2 wsel[NSR][RTX];
    auto prologue_products = [&]() __attribute__((always_inline)) {
        const uint16_t *qrow = p.q + ((int64_t)my_agent * p.hq + qh) * D;
        load_q(qrow, row_active, grp, qf);

        // W = B_K q: the contraction over the head dim may take any order that both
        // operands share, so it uses the natural one (lane holds dims 32kk + 8grp .. +7),
        // in which each lane reads 16 contiguous bytes of a B_K row and of q
        u32x4 bkf[NSR][RTX][4], qn[4];
        if constexpr (R > 0) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) qn[kk] = row_active ? ldg128(qrow + 32 * kk + 8 * grp) : u32x4{0, 0, 0, 0};
#pragma unroll
            for (int s = 0; s < NSR; ++s) {
                const uint16_t *bk = p.lora_b + (int64_t)(slot_ad[s] >= 0 ? slot_ad[s] : 0) * 2 * R * n + (int64_t)h * D;
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    const int rho = 16 * t + col;
                    const int64_t ro = (int64_t)(rho < R ? rho : 0) * n;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk)
                        bkf[s][t][kk] = (slot_ad[s] >= 0 && rho < R) ? ldg128(bk + ro + 32 * kk + 8 * grp) : u32x4{0, 0, 0, 0};
                }
            }
        }
        // W^T = (B_K q)^T per slot, as the B operand of the residual key products; row
        // columns of other slots are zero, so one product serves a pair of slots (or tiles)
#pragma unroll
        for (int s = 0; s < NSR; ++s)
#pragma unroll
            for (int t = 0; t < RTX; ++t) {
                wsel[s][t] = u32x2{0, 0};
                if constexpr (R > 0) {
                    f32x4 acc = {0, 0, 0, 0};
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) acc = mfma32(bkf[s][t][kk], qn[kk], acc);
                    if (my_slot == s) wsel[s][t] = pack4(acc);
                }
            }
    };

    Rows<R> st;
    st.init();
    const float cl = p.scale_log2;
    const int64_t vbytes = (int64_t)hkv * kBlockBytes;  // K block -> V block of a (page, head)

    // rCache fragments of the wave's slots (NSA: 1 or NSR) for NP item pages from k0: one
    // 16-byte load per (page, slot, rank tile), at the address the descriptor names
    auto load_c_page = [&](auto nsa_tag, int j, int k, CFrag &c) __attribute__((always_inline)) {
        constexpr int NSA = decltype(nsa_tag)::value;
        if constexpr (R > 0) {
#pragma unroll
            for (int s = 0; s < NSA; ++s) {
                const i32x4 rs = block_rsrc(res_addr(k, s), RT * 1024);
#pragma unroll
                for (int t = 0; t < RT; ++t) c.kv[j][s][t] = buf_load16(rs, lane * 16 + t * 1024);
            }
        }
    };
    auto load_c = [&](auto nsa_tag, auto np_tag, int k0, CFrag &c) __attribute__((always_inline)) {
        constexpr int NP = decltype(np_tag)::value;
#pragma unroll
        for (int j = 0; j < NP; ++j) load_c_page(nsa_tag, j, k0 + j, c);
    };

    // ---- Stages 1-2 for NP item pages from k0, fragments in registers ----
    // kf[j][kk]: K fragments of page j (A operand of S^T = K Q^T, 32 head dims per kk);
    // vf[j][q2]: the page's value chunk q2 in its stored order, dims 32q2 + col (.xy) and
    // 32q2 + 16 + col (.zw) of tokens 4grp .. 4grp + 3.  For two pages the value product
    // takes 32 keys: the pair's two 8-byte halves form one 16x16x32 operand.
    // `hook(0)` runs after the score products, `hook(1)` before the value products: the ring
    // path issues the next stages' rCache loads there, so that the texture path works while
    // the wave computes instead of all four waves issuing together after the barrier.
    auto compute = [&](auto nsa_tag, auto np_tag, int k0, auto &&get_k, auto &&get_v, CFrag &c, auto &&hook)
        __attribute__((always_inline)) {
        constexpr int NSA = decltype(nsa_tag)::value;
        constexpr int NP = decltype(np_tag)::value;
        const int pgw = pg0 + k0;  // logical page of step page 0
        // rCache tokens past a slot's own length, or on a padding page, are unwritten: zero
        // them (one uniform branch; pages inside every rCache of the group skip it)
        if constexpr (R > 0) {
            if (pgw + NP > pg1 || (pgw + NP) * PS > min_res) {
#pragma unroll
                for (int j = 0; j < NP; ++j)
#pragma unroll
                    for (int s = 0; s < NSA; ++s) {
                        const int svis = pgw + j < pg1 ? slot_len[s] - (pgw + j) * PS : 0;
#pragma unroll
                        for (int t = 0; t < RT; ++t) {
                            const u32x4 x = c.kv[j][s][t];
                            const u32x2 k = col < svis ? u32x2{x.x, x.y} : u32x2{0, 0};
                            const u32x2 v = mask4(u32x2{x.z, x.w}, svis, grp);
                            c.kv[j][s][t] = u32x4{k.x, k.y, v.x, v.y};
                        }
                    }
            }
        }
        // rCache fragment of (page j, slot s, tile t); for rank 8 half of a tile is padding
        auto ckf = [&](int j, int s, int t) __attribute__((always_inline)) -> u32x2 {
            const u32x2 v = u32x2{c.kv[j][s][t].x, c.kv[j][s][t].y};
            if constexpr (R == 8) return grp < 2 ? v : u32x2{0, 0};
            return v;
        };
        auto cvf = [&](int j, int s, int t) __attribute__((always_inline)) -> u32x2 {
            const u32x2 v = u32x2{c.kv[j][s][t].z, c.kv[j][s][t].w};
            if constexpr (R == 8) return col < 8 ? v : u32x2{0, 0};
            return v;
        };
        // scores S^T = K_base Q^T + C_K (W)^T
        u32x4 kf[NP][4];
        get_k(kf);
        f32x4 sacc[NP];
#pragma unroll
        for (int j = 0; j < NP; ++j) {
            sacc[j] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) sacc[j] = mfma32(kf[j][kk], qf[kk], sacc[j]);
        }
        if constexpr (R > 0) {
            constexpr int NU = NSA * RT;  // (slot, tile) units, taken in pairs
#pragma unroll
            for (int j = 0; j < NP; ++j) {
#pragma unroll
                for (int u = 0; u + 1 < NU; u += 2) {
                    const int s0 = u / RT, t0 = u % RT, s1 = (u + 1) / RT, t1 = (u + 1) % RT;
                    const u32x2 c0 = ckf(j, s0, t0), c1 = ckf(j, s1, t1);
                    const u32x4 a = u32x4{c0.x, c0.y, c1.x, c1.y};
                    const u32x4 b = u32x4{wsel[s0][t0].x, wsel[s0][t0].y, wsel[s1][t1].x, wsel[s1][t1].y};
                    sacc[j] = mfma32(a, b, sacc[j]);
                }
                if constexpr (NU % 2 == 1) {
                    // the last unit alone, zero-padded: a chain that accumulates into one
                    // tile stays on the 16x16x32 form (a 16x16x16 product issued right after
                    // a 16x16x32 one onto the same accumulator read a stale value here)
                    const int s0 = (NU - 1) / RT, t0 = (NU - 1) % RT;
                    const u32x2 c0 = ckf(j, s0, t0);
                    sacc[j] = mfma32(u32x4{c0.x, c0.y, 0u, 0u}, u32x4{wsel[s0][t0].x, wsel[s0][t0].y, 0u, 0u}, sacc[j]);
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        hook(0);
        __builtin_amdgcn_sched_barrier(0);
        // Stage 2: online softmax over the step's keys (rows in lanes, keys in lane groups).
        // Keys 4grp + i of page j are visible to this lane's row when i < kv; a step inside
        // every row's sequence skips the test.
        float sv[NP][4];
        if (pgw + NP <= pg1 && (pgw + NP) * PS <= min_len) {
#pragma unroll
            for (int j = 0; j < NP; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) sv[j][i] = sacc[j][i];
        } else {
#pragma unroll
            for (int j = 0; j < NP; ++j) {
                const int kv = (pgw + j < pg1 && row_active) ? my_len - (pgw + j) * PS - 4 * grp : 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) sv[j][i] = i < kv ? sacc[j][i] : kNegInf;
            }
        }
        float mx = kNegInf;
#pragma unroll
        for (int j = 0; j < NP; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sv[j][i]);
        mx = max_over_groups(mx) * cl;
        if (__builtin_amdgcn_ballot_w64(mx > st.m + kLazyRescale) != 0) {
            const float m_new = fmaxf(st.m, mx);
            const float alpha = fast_exp2(st.m - (m_new == kNegInf ? 0.f : m_new));
            st.l *= alpha;
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) st.oacc[mt] *= alpha;
#pragma unroll
            for (int t = 0; t < RT; ++t) st.racc[t] *= alpha;
            st.m = m_new;
        }
        const float m_use = st.m == kNegInf ? 0.f : st.m;
        u32x2 pf[NP];
        float psum = 0.f;
#pragma unroll
        for (int j = 0; j < NP; ++j) {
            f32x4 pv;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                pv[i] = fast_exp2(__builtin_fmaf(sv[j][i], cl, -m_use));
                psum += pv[i];
            }
            pf[j] = pack4(pv);
        }
        st.l += psum;
        __builtin_amdgcn_sched_barrier(0);
        hook(1);
        __builtin_amdgcn_sched_barrier(0);
        u32x4 vf[NP][4];
        get_v(vf);
        // value tokens past the item's longest sequence (or on a padding page) may hold any
        // bits: zero them so that their zero weights cannot meet a NaN
        if (pgw + NP > pg1 || (pgw + NP) * PS > item_max_len) {
#pragma unroll
            for (int j = 0; j < NP; ++j) {
                const int vis = pgw + j < pg1 ? item_max_len - (pgw + j) * PS : 0;
#pragma unroll
                for (int q2 = 0; q2 < 4; ++q2) {
                    const u32x2 lo = mask4(u32x2{vf[j][q2].x, vf[j][q2].y}, vis, grp);
                    const u32x2 hi = mask4(u32x2{vf[j][q2].z, vf[j][q2].w}, vis, grp);
                    vf[j][q2] = u32x4{lo.x, lo.y, hi.x, hi.y};
                }
            }
        }
        // O^T += V^T P^T and acc_r^T += C_V^T P^T (rows of other slots masked out of P)
        if constexpr (NP == 2) {
            const u32x4 pb = u32x4{pf[0].x, pf[0].y, pf[1].x, pf[1].y};
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) {
                st.oacc[2 * q2] = mfma32(u32x4{vf[0][q2].x, vf[0][q2].y, vf[1][q2].x, vf[1][q2].y}, pb, st.oacc[2 * q2]);
                st.oacc[2 * q2 + 1] =
                    mfma32(u32x4{vf[0][q2].z, vf[0][q2].w, vf[1][q2].z, vf[1][q2].w}, pb, st.oacc[2 * q2 + 1]);
            }
            if constexpr (R > 0) {
#pragma unroll
                for (int s = 0; s < NSA; ++s) {
                    const u32x4 pm = my_slot == s ? pb : u32x4{0, 0, 0, 0};
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const u32x2 c0 = cvf(0, s, t), c1 = cvf(1, s, t);
                        st.racc[t] = mfma32(u32x4{c0.x, c0.y, c1.x, c1.y}, pm, st.racc[t]);
                    }
                }
            }
        } else {
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) {
                st.oacc[2 * q2] = mfma16(u32x2{vf[0][q2].x, vf[0][q2].y}, pf[0], st.oacc[2 * q2]);
                st.oacc[2 * q2 + 1] = mfma16(u32x2{vf[0][q2].z, vf[0][q2].w}, pf[0], st.oacc[2 * q2 + 1]);
            }
            if constexpr (R > 0) {
#pragma unroll
                for (int s = 0; s < NSA; ++s) {
                    const u32x2 pm = my_slot == s ? pf[0] : u32x2{0, 0};
#pragma unroll
                    for (int t = 0; t < RT; ++t) st.racc[t] = mfma16(cvf(0, s, t), pm, st.racc[t]);
                }
            }
        }
    };

    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using NSF = std::integral_constant<int, NSR>;

    // Base pages that no other item reads are loaded as data read once (kDescStream), so
    // that they displace less of the rCache rows the item's other KV heads re-read from L2.
    auto paths = [&](auto policy_tag) __attribute__((always_inline)) {
        constexpr int POL = decltype(policy_tag)::value;
        if (ngp > 1) {
            if constexpr (S::MULTI) {
                // Several agent groups share each base page through an LDS ring of kRing stages
                // of two pages ([K p0 | V p0 | K p1 | V p1], 4 KB each).  Memory writes a stage
                // straight into LDS (global_load_lds, no registers): wave w copies block w of
                // stage s + kRing - 1 while stage s is computed.  Four groups: every wave computes
                // both pages for its group; two groups: wave (group, copy) computes page `copy`.
                // rCache fragments go to registers two stages ahead.
                constexpr int NPW_MAX = 2;
                const int npw = ngp == 4 ? 2 : 1;
                const int n_stages = (npg + 1) / 2;
                auto dma_stage = [&](int stage, LdsU32x4 *__restrict__ buf) __attribute__((always_inline)) {
                    const i32x4 rs = block_rsrc(base_addr(2 * stage + (wave >> 1)) + ((wave & 1) ? vbytes : 0), kBlockBytes);
                    LdsU32x4 *dst = buf + wave * (kBlockBytes / 16);
#pragma unroll
                    for (int i = 0; i < 4; ++i) lds_dma16<POL>(rs, lane * 16 + i * 1024, dst + i * 64);
                };
                auto ring_buf = [&](int stage) __attribute__((always_inline)) -> LdsU32x4 * {
                    return (LdsU32x4 *)(lds_ring + (stage % kRing) * (kStageBytes / 16));
                };
                // One iteration: request the rCache rows of stage s + 2, copy stage s + kRing - 1
                // into its ring buffer, compute stage s.  The ring is read with explicit LDS
                // reads whose wait is part of the same instruction group: the compiler sees no
                // LDS load that it would have to order after the copies still in flight, which
                // are waited for (by count) before the barrier that precedes each stage.
                // The copies go first, the rCache loads of stage s + 2 one page each after the score
                // and before the value products of stage s (a stage's copies are then followed by
                // at least (kRing - 2) * (4 + NC) vector-memory operations before it is computed,
                // the count each stage waits for).
                auto iterate = [&](auto nsa_tag, auto np_tag, int s, CFrag &c_now, CFrag &c_next2) __attribute__((always_inline)) {
                    constexpr int NP = decltype(np_tag)::value;
                    dma_stage(s + kRing - 1, ring_buf(s + kRing - 1));
                    const int kc = 2 * (s + 2) + (NP == 2 ? 0 : copy);
                    auto hook = [&](int ph) __attribute__((always_inline)) {
                        if (ph < NP) load_c_page(nsa_tag, ph, kc + ph, c_next2);
                    };
                    const uint32_t cur = lds_addr(ring_buf(s)) + lane * 16;
                    // both pages' fragments under one wait (16 agents over 32K: 65.1-65.5 -> 64.2-64.5 us)
                    auto get_k = [&](u32x4 (&kf)[NP][4]) __attribute__((always_inline)) {
                        if constexpr (NP == 2) lds_read8(cur, cur + 2 * kBlockBytes, kf[0], kf[1]);
                        else lds_read4(cur + copy * 2 * kBlockBytes, kf[0]);
                    };
                    auto get_v = [&](u32x4 (&vf)[NP][4]) __attribute__((always_inline)) {
                        if constexpr (NP == 2) lds_read8(cur + kBlockBytes, cur + 3 * kBlockBytes, vf[0], vf[1]);
                        else lds_read4(cur + copy * 2 * kBlockBytes + kBlockBytes, vf[0]);
                    };
                    compute(nsa_tag, np_tag, 2 * s + (NP == 2 ? 0 : copy), get_k, get_v, c_now, hook);
                };
                auto run = [&](auto nsa_tag, auto np_tag) __attribute__((always_inline)) {
                    constexpr int NP = decltype(np_tag)::value;
                    constexpr int NC = R > 0 ? decltype(nsa_tag)::value * NP * RT : 0;  // rCache loads per iteration
                    // vm operations issued after a stage's copies until that stage is computed:
                    // kRing - 2 further iterations
                    constexpr int kWait = (kRing - 2) * (4 + NC);
                    static_assert(kWait < 64, "vmcnt range");
                    CFrag c0, c1, c2;
                    load_c(nsa_tag, np_tag, NP == 2 ? 0 : copy, c0);
                    load_c(nsa_tag, np_tag, 2 + (NP == 2 ? 0 : copy), c1);
#pragma unroll
                    for (int k = 0; k < kRing - 1; ++k) dma_stage(k, ring_buf(k));
                    prologue_products();
                    for (int s = 0;;) {
                        stage_barrier<kWait>();
                        iterate(nsa_tag, np_tag, s, c0, c2);
                        if (++s >= n_stages) break;
                        stage_barrier<kWait>();
                        iterate(nsa_tag, np_tag, s, c1, c0);
                        if (++s >= n_stages) break;
                        stage_barrier<kWait>();
                        iterate(nsa_tag, np_tag, s, c2, c1);
                        if (++s >= n_stages) break;
                    }
                    wait_vmcnt<0>();  // no copy into LDS outlives the block
                };
                (void)npw;
                if constexpr (S::NG == 4) {
                    if (ngp == 4) run(NSF{}, I2{});
                    else run(NSF{}, I1{});
                } else {
                    run(NSF{}, I1{});  // two groups at most: one page per wave and stage
                }
            }
        } else {
            // One agent group: no page is shared between waves.  Wave w computes item pages
            // w, w + 4, ... straight from registers (the stored fragment order is the operand
            // order), with the next two pages and their rCache rows in flight.
            struct PageRegs {
                u32x4 k[1][4], v[1][4];
                CFrag c;
            };
            auto load_page = [&](auto nsa_tag, int k, PageRegs &pr) __attribute__((always_inline)) {
                const uint64_t a = base_addr(k);
                const i32x4 rk = block_rsrc(a, kBlockBytes), rv = block_rsrc(a + vbytes, kBlockBytes);
#pragma unroll
                for (int i = 0; i < 4; ++i) pr.k[0][i] = buf_load16<POL>(rk, lane * 16 + i * 1024);
#pragma unroll
                for (int i = 0; i < 4; ++i) pr.v[0][i] = buf_load16<POL>(rv, lane * 16 + i * 1024);
                load_c(nsa_tag, I1{}, k, pr.c);
            };
            auto no_hook = [](int) {};
            auto regs_k = [](PageRegs &pr) {
                return [&pr](u32x4 (&kf)[1][4]) __attribute__((always_inline)) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) kf[0][i] = pr.k[0][i];
                };
            };
            auto regs_v = [](PageRegs &pr) {
                return [&pr](u32x4 (&vf)[1][4]) __attribute__((always_inline)) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) vf[0][i] = pr.v[0][i];
                };
            };
            const int n_my = wave < npg ? (npg - wave + WAVES - 1) / WAVES : 0;
            // one agent: two pages in flight; several agents (more rCache rows per page): one
            auto run2 = [&](auto nsa_tag) __attribute__((always_inline)) {
                PageRegs pa, pb;
                load_page(nsa_tag, wave, pa);
                prologue_products();
                for (int i = 0; i < n_my;) {
                    load_page(nsa_tag, wave + WAVES * (i + 1), pb);
                    compute(nsa_tag, I1{}, wave + WAVES * i, regs_k(pa), regs_v(pa), pa.c, no_hook);
                    if (++i >= n_my) break;
                    load_page(nsa_tag, wave + WAVES * (i + 1), pa);
                    compute(nsa_tag, I1{}, wave + WAVES * i, regs_k(pb), regs_v(pb), pb.c, no_hook);
                    if (++i >= n_my) break;
                }
            };
            auto run1 = [&](auto nsa_tag) __attribute__((always_inline)) {
                PageRegs pa, pb, pc;
                load_page(nsa_tag, wave, pa);
                load_page(nsa_tag, wave + WAVES, pb);
                prologue_products();
                for (int i = 0; i < n_my;) {
                    load_page(nsa_tag, wave + WAVES * (i + 2), pc);
                    compute(nsa_tag, I1{}, wave + WAVES * i, regs_k(pa), regs_v(pa), pa.c, no_hook);
                    if (++i >= n_my) break;
                    load_page(nsa_tag, wave + WAVES * (i + 2), pa);
                    compute(nsa_tag, I1{}, wave + WAVES * i, regs_k(pb), regs_v(pb), pb.c, no_hook);
                    if (++i >= n_my) break;
                    load_page(nsa_tag, wave + WAVES * (i + 2), pb);
                    compute(nsa_tag, I1{}, wave + WAVES * i, regs_k(pc), regs_v(pc), pc.c, no_hook);
                    if (++i >= n_my) break;
                }
            };
            if (R == 0 || nag == 1) run1(I1{});
            else run2(NSF{});
        }
    };
    // (not at rank 32, where the second instance would not fit the registers without scratch)
    if (R != 32 && desc[fkv::kDescStream] != 0) paths(std::integral_constant<int, R != 32 ? kCacheStream : kCacheDefault>{});
    else paths(std::integral_constant<int, kCacheDefault>{});

    static_assert(merge_lds_bytes(R) <= kRing * kStageBytes, "merge area inside the ring");
    merge_wave_copies<R>(st, wave, copy, my_group, ngp, WAVES / ngp, reinterpret_cast<f32x4 *>(lds_ring));
    if (copy == 0) write_partial<R>(p, st, row_active, my_row, grp);
}

template <int R, int G>
__global__ __launch_bounds__(256, R >= 64 ? 1 : 2) void decode_split_kernel(DecodeArgs p) {
    split_body<R, G>(p);
}


// ---------------------------------------------------------------------------
// RoPE on (deferred RoPE of the rebuilt key, Section 5.3; Algorithm 1, stage 1).  One
// workgroup per (work item, KV head h), four waves, two workgroups per compute unit.  An
// item holds up to MS agents in up to four wave groups of NSW agents; wave w serves group
// w % ngp as copy w / ngp and streams the item pages i with i % copies == copy straight
// into registers (next page in flight), independently of the other waves: the rebuild is
// vector-ALU bound, so no barrier ties the waves together.  The waves of one item read
// each base page at about the same time, so it crosses HBM once per item and reaches the
// other groups from the caches.  The B_K^T fragments of every slot of the item are built in
// LDS once per workgroup.  Per page and slot s of the wave's group (matrix-core products,
// fp32 accumulate):
//   U^T   = B_K,s^T C_K,s^T                  16x16x16
//   K_lr  = RoPE_p(U)                        rotate-half pairs (i, i + 64) in one lane, fp32
//   S^T  += K_lr Q^T                         16x16x32, kept for the slot's own rows (columns)
template <int R, int G>
struct RopeShape {
    static constexpr int RT = (R + 15) / 16;                       // 16-wide rank tiles
    static constexpr int NSW = fkv::decode_rope_wave_agents(G, R); // agent slots of a wave
    static constexpr int MS = fkv::decode_rope_item_agents(G, R);  // agent slots of an item
    static constexpr int BKT = MS * RT * 8 * 512;                  // (slot, tile, column tile) x 64 lanes x 8 B
    static constexpr int BK_UNITS = MS * RT * 128;                 // (slot, rank pair, 8-dim chunk)
    static_assert(BKT <= 64 * 1024, "two workgroups per compute unit");
    static_assert(BK_UNITS % 256 == 0 && NSW * G <= ROWS, "shape");
};

template <int R, int G>
__global__ __launch_bounds__(256, 2) void decode_rope_kernel(DecodeArgs p) {
    static_assert(R > 0, "RoPE decode needs a residual");
    using S = RopeShape<R, G>;
    using RowsT = Rows<R>;
    constexpr int RT = S::RT, NSW = S::NSW, MS = S::MS;
    constexpr int RTX = RowsT::RTX;
    // B_K^T fragments for the launch; at the end the merge area of the wave copies
    __shared__ __attribute__((aligned(16))) u32x2 bkt[cmax(S::BKT, merge_lds_bytes(R)) / 8];

    // the block's descriptor (at an address that depends on blockIdx only) names the item
    const int32_t *desc = p.plan + p.off_desc + (int64_t)blockIdx.x * fkv::kDescWords;
    const int pg0 = desc[fkv::kDescPg0], pgcap = desc[fkv::kDescCap], nag = desc[fkv::kDescNag];
    if (nag <= 0) return;  // idle block
    const int hkv = p.hkv;
    const int h = desc[fkv::kDescHead], leader = desc[fkv::kDescLeader];
    const int npcap = pgcap - pg0;
    if (nag < 1 || nag > MS || npcap < 1 || npcap > fkv::kMaxPagesSingle) return;  // rejected on the host
    const int ng = (nag + NSW - 1) / NSW;
    const int ngp = ng == 1 ? 1 : (ng == 2 ? 2 : 4);
    const int copies = WAVES / ngp;

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int my_group = wave % ngp, copy = wave / ngp;
    const int sb = my_group * NSW;                   // first item slot of this wave's group
    const int my_slot = col / G;                     // this lane's row: slot within the group
    const bool row_active = my_slot < NSW && sb + my_slot < nag;
    const int qh = h * G + (col % G);

    // lane i < nag: slot i's agent and first partial (plan), length and adapter (launch
    // arrays); lane i (and 64 + i): base page id of item page i (the leader's row) and, per
    // slot of this wave's group, its rCache page id (-1: no adapter)
    const bool lane_ag = lane < nag;
    const int l_agent = lane_ag ? desc[fkv::kDescAgent + lane] : 0;
    const int l_part = lane_ag ? desc[fkv::kDescPart + lane] : 0;
    const int l_len = lane_ag ? p.seq_lens[l_agent] : 0;
    const int l_ad = lane_ag ? p.adapter_idx[l_agent] : -1;
    const int32_t *brow = p.base_bt + (int64_t)leader * p.max_pages + pg0;
    const int bid0 = brow[min(lane, npcap - 1)];
    const int bid1 = brow[min(64 + lane, npcap - 1)];
    int rid0[NSW], rid1[NSW];
#pragma unroll
    for (int s = 0; s < NSW; ++s) {
        const bool ok = sb + s < nag;
        const int ag_s = __builtin_amdgcn_readlane(l_agent, (sb + s) & 63);
        const int32_t *row = p.res_bt + (int64_t)(ok ? ag_s : 0) * p.max_pages + pg0;
        rid0[s] = ok ? row[min(lane, npcap - 1)] : -1;
        rid1[s] = (ok && npcap > 64) ? row[min(64 + lane, npcap - 1)] : -1;
    }
    int item_max_len = 0;
    for (int s = 0; s < nag; ++s) item_max_len = max(item_max_len, __builtin_amdgcn_readlane(l_len, s));
    const int npg = min(pgcap, (item_max_len + PS - 1) / PS) - pg0;
    // the wave's slots: keys that carry a residual (0 without adapter or past the item), and
    // the shortest sequence among them: pages that end at or before it hold written keys,
    // values and rCache rows for every row of the wave, so they need no length masks
    int res_len[NSW];
    int wave_min_len = item_max_len;
#pragma unroll
    for (int s = 0; s < NSW; ++s) {
        const bool ok = sb + s < nag;
        const int ad = __builtin_amdgcn_readlane(l_ad, (sb + s) & 63);
        const int len = __builtin_amdgcn_readlane(l_len, (sb + s) & 63);
        res_len[s] = (ok && ad >= 0) ? len : 0;
        if (res_len[s] == 0) rid0[s] = rid1[s] = -1;
        if (ok) wave_min_len = min(wave_min_len, len);
    }
    const int src_lane = (sb + my_slot) & 63;
    const int sh_agent = __shfl(l_agent, src_lane), sh_len = __shfl(l_len, src_lane);
    const int my_agent = row_active ? sh_agent : 0;
    const int my_len = row_active ? sh_len : 0;
    const int my_part = __shfl(l_part, src_lane);
    const int64_t my_row = ((int64_t)my_part * G + col % G) * hkv + h;

    RowsT st;
    st.init();
    if (npg <= 0) {  // the item's agents have not reached it yet: an empty partial (weight 0)
        if (copy == 0) write_partial<R>(p, st, row_active, my_row, grp);
        return;
    }

    // B_K^T fragments of the item's slots for head h, built in LDS in rounds of four units: unit
    // (slot, rank pair, 8-dim chunk) loads ranks 2q and 2q + 1 over 8 dims (ranks past R and
    // slots without adapter: zero); lane (c, gg) of fragment (slot, tile t, column tile mt)
    // holds B_K[16t + 4gg + j][16mt + c], j < 4, as two words of rank pairs
    {
        const int64_t n = (int64_t)hkv * D;
        uint32_t *bw = reinterpret_cast<uint32_t *>(bkt);
        constexpr int UPT = S::BK_UNITS / 256, ROUND = UPT < 4 ? UPT : 4;
        for (int u0 = 0; u0 < UPT; u0 += ROUND) {
            if (256 * u0 / (RT * 128) >= nag) break;  // slots past the item's agents are never read
            u32x4 bk_lo[ROUND], bk_hi[ROUND];
#pragma unroll
            for (int u = 0; u < ROUND; ++u) {
                const int idx = threadIdx.x + 256 * (u0 + u);
                const int sl = idx / (RT * 128), rem = idx % (RT * 128);
                const int rho = 2 * (rem / 16), c8 = rem % 16;
                const int ad = __shfl(l_ad, sl & 63);
                const bool ok = sl < nag && ad >= 0 && rho < R;
                const uint16_t *src =
                    p.lora_b + ((int64_t)(ok ? ad : 0) * 2 * R + (ok ? rho : 0)) * n + (int64_t)h * D + 8 * c8;
                bk_lo[u] = ok ? ldg128(src) : u32x4{0, 0, 0, 0};
                bk_hi[u] = (ok && rho + 1 < R) ? ldg128(src + n) : u32x4{0, 0, 0, 0};
            }
#pragma unroll
            for (int u = 0; u < ROUND; ++u) {
                const int idx = threadIdx.x + 256 * (u0 + u);
                const int sl = idx / (RT * 128), rem = idx % (RT * 128);
                const int rho = 2 * (rem / 16), c8 = rem % 16;
                const int t = rho / 16, gg = (rho % 16) / 4, j2 = (rho % 4) / 2;
                if (sl >= nag) continue;
                const uint32_t lw[4] = {bk_lo[u].x, bk_lo[u].y, bk_lo[u].z, bk_lo[u].w};
                const uint32_t hw[4] = {bk_hi[u].x, bk_hi[u].y, bk_hi[u].z, bk_hi[u].w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int i = 8 * c8 + e, mt = i / 16, c = i % 16;
                    const uint32_t a = (e & 1) ? (lw[e >> 1] >> 16) : (lw[e >> 1] & 0xffffu);
                    const uint32_t b = (e & 1) ? (hw[e >> 1] >> 16) : (hw[e >> 1] & 0xffffu);
                    bw[((((sl * RT + t) * 8 + mt) * 64) + c + 16 * gg) * 2 + j2] = a | (b << 16);
                }
            }
        }
    }

    // This wave's pages: copy, copy + copies, ...  One register set holds a page's K, V and
    // rCache fragments (the stored orders are the operand orders) and the cos / sin of its
    // positions; each part is refilled with the next page's as soon as its last use is issued
    // (pages past the item repeat its last page).
    const int64_t vhalfs = (int64_t)hkv * kBlockHalfs;
    auto kblock = [&](int kk) __attribute__((always_inline)) -> const uint16_t * {
        kk = min(kk, npg - 1);
        const int lo = __builtin_amdgcn_readlane(bid0, kk & 63), hi = __builtin_amdgcn_readlane(bid1, kk & 63);
        const int id = kk < 64 ? lo : hi;
        return p.base_kv + ((int64_t)id * 2 * hkv + h) * kBlockHalfs;
    };
    u32x4 fk[4], fv[4], fc[NSW][RT];
    f32x4 cs[4], sn[4];
    auto load_k = [&](int kk) __attribute__((always_inline)) {
        const uint16_t *b = kblock(kk);
#pragma unroll
        for (int i = 0; i < 4; ++i) fk[i] = ldg128(b + i * 512 + lane * 8);
    };
    auto load_v = [&](int kk) __attribute__((always_inline)) {
        const uint16_t *b = kblock(kk) + vhalfs;
#pragma unroll
        for (int i = 0; i < 4; ++i) fv[i] = ldg128(b + i * 512 + lane * 8);
    };
    auto load_c = [&](int kk) __attribute__((always_inline)) {
        kk = min(kk, npg - 1);
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int rl = __builtin_amdgcn_readlane(rid0[s], kk & 63), rh = __builtin_amdgcn_readlane(rid1[s], kk & 63);
            const int rp = kk < 64 ? rl : rh;
            const uint16_t *rb = p.res_kv + (int64_t)(rp >= 0 ? rp : 0) * (RT * 512);
#pragma unroll
            for (int t = 0; t < RT; ++t) fc[s][t] = rp >= 0 ? ldg128(rb + t * 512 + lane * 8) : u32x4{0, 0, 0, 0};
        }
    };
    // cos / sin at position 16 * page + t (t = col) for pairs 16mt + 4grp + i: the table keeps
    // each page's 16 positions in this fragment order (tile mt, lane, 4 pairs), so lane l reads
    // 16 bytes at 256 mt + 4 l of the page's block (the page's rows, shared by every agent and
    // KV head that reads the page, come from L2 after the first reader; reading them costs fewer
    // vector instructions and registers than forming them from the page's first row by angle
    // addition: 16 agents over 32K, 156-168 -> 153-161 us)
    auto load_rope = [&](int kk) __attribute__((always_inline)) {
        kk = min(kk, npg - 1);
        const float *cr = p.rope_cos + (int64_t)(pg0 + kk) * (PS * D / 2) + 4 * lane;
        const float *sr = p.rope_sin + (int64_t)(pg0 + kk) * (PS * D / 2) + 4 * lane;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            cs[mt] = *reinterpret_cast<const f32x4 *>(cr + 256 * mt);
            sn[mt] = *reinterpret_cast<const f32x4 *>(sr + 256 * mt);
        }
    };
    const bool busy = sb < nag;  // a wave of an empty group has nothing to do
    if (busy) {
        load_k(copy);
        load_c(copy);
        load_rope(copy);
        load_v(copy);
    }
    u32x4 qf[4];
    load_q(p.q + ((int64_t)my_agent * p.hq + qh) * D, row_active, grp, qf);
    __syncthreads();  // B_K^T fragments visible to every wave

    // One page of the wave's loop.  EDGE: the page may reach past a row's sequence, so rCache
    // rows, value tokens and scores are masked by length; interior pages skip those masks.
    auto page = [&](auto edge_tag, int k) __attribute__((always_inline)) {
        constexpr bool EDGE = decltype(edge_tag)::value;
        const int next = k + copies;
        const int tok0 = (pg0 + k) * PS;
        f32x4 sbase = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) sbase = mfma32(fk[kk], qf[kk], sbase);
        load_k(next);
        // rCache fragments of slot s, tile t: tokens past the slot's own length (or all, without
        // adapter) are zero
        auto cfrag = [&](int s, int t, bool key) __attribute__((always_inline)) -> u32x2 {
            u32x2 kx = u32x2{fc[s][t].x, fc[s][t].y}, vx = u32x2{fc[s][t].z, fc[s][t].w};
            if constexpr (R == 8) {
                kx = grp < 2 ? kx : u32x2{0, 0};
                vx = col < 8 ? vx : u32x2{0, 0};
            }
            if constexpr (EDGE) {
                const int svis = res_len[s] - tok0;
                if (svis < PS) {
                    vx = mask4(vx, svis, grp);
                    kx = col < svis ? kx : u32x2{0, 0};
                }
            }
            return key ? kx : vx;
        };
        // Stage 1 per slot: U^T = B_K^T C_K^T, deferred RoPE, then K_lr Q^T, of which the
        // slot's own rows (columns) are added to the scores
        f32x4 sacc = sbase;
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int slot = sb + s;
            if (res_len[s] > tok0) {
                f32x4 sres = {0, 0, 0, 0};
                // two halves of the head dim: column tiles {2hf, 2hf + 1} and their rotate-half
                // partners {2hf + 4, 2hf + 5} are the A operands of k-steps hf and hf + 2
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    const int mts[4] = {2 * hf, 2 * hf + 1, 2 * hf + 4, 2 * hf + 5};
                    f32x4 u[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        u[j] = f32x4{0, 0, 0, 0};
#pragma unroll
                        for (int t = 0; t < RT; ++t)
                            u[j] = mfma16(bkt[((slot * RT + t) * 8 + mts[j]) * 64 + lane], cfrag(s, t, true), u[j]);
                    }
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        const int mt = mts[j];
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float x = u[j][i], y = u[j + 2][i];
                            u[j][i] = x * cs[mt][i] - y * sn[mt][i];
                            u[j + 2][i] = y * cs[mt][i] + x * sn[mt][i];
                        }
                    }
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        const u32x2 lo = pack4(u[2 * j]), hi = pack4(u[2 * j + 1]);
                        sres = mfma32(u32x4{lo.x, lo.y, hi.x, hi.y}, qf[hf + 2 * j], sres);
                    }
                }
                if (my_slot == s) sacc += sres;
            }
            __builtin_amdgcn_sched_barrier(0);  // one slot's rebuild at a time (register pressure)
        }
        u32x2 cv[NSW][RTX];
#pragma unroll
        for (int s = 0; s < NSW; ++s)
#pragma unroll
            for (int t = 0; t < RT; ++t) cv[s][t] = cfrag(s, t, false);
        load_c(next);
        load_rope(next);
        u32x2 vf[8];
#pragma unroll
        for (int q2 = 0; q2 < 4; ++q2) {
            vf[2 * q2] = u32x2{fv[q2].x, fv[q2].y};
            vf[2 * q2 + 1] = u32x2{fv[q2].z, fv[q2].w};
        }
        // value tokens past the item's longest sequence may hold any bits: zero them
        if constexpr (EDGE) {
            const int vis = item_max_len - tok0;
            if (vis < PS) {
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) vf[mt] = mask4(vf[mt], vis, grp);
            }
        }
        softmax_pv<R, NSW, EDGE>(st, sacc, row_active, tok0, my_len, p.scale_log2, vf, cv, my_slot, grp);
        load_v(next);
    };
    // interior pages first (a prefix of the wave's pages), then the rest
    int k = copy;
    for (; busy && k < npg && (pg0 + k + 1) * PS <= wave_min_len; k += copies) page(std::false_type{}, k);
    for (; busy && k < npg; k += copies) page(std::true_type{}, k);
    merge_wave_copies<R>(st, wave, copy, my_group, ngp, copies, reinterpret_cast<f32x4 *>(bkt));
    if (copy == 0) write_partial<R>(p, st, row_active, my_row, grp);
}


// Log-sum-exp merge of one agent's partials and Stage 3 of Algorithm 1 for one query
// row (agent a, query head j of KV head h = j / G), by one workgroup of CW waves:
//   O = (sum_k w_k acc_k + (sum_k w_k acc_r,k) . B_V[h]) / L,
//   w_k = 2^(m_k - M), M = max_k m_k, L = sum_k w_k l_k.
// An agent's partials are contiguous; wave w merges partials w, w + CW, ... (all of its
// share in flight at once): lane i < NV reads float4 i of every record (acc, then acc_r)
// and lane NV its (m, l); lanes past NV read float4 0 and drop it.  The waves' results
// meet in LDS and wave 0 merges them and applies Stage 3.  B_V is read at the start, as
// it does not depend on the partials.
// Waves per row: four, or sixteen when the rows are fewer than half the compute units and each
// has many partials (one KV head per GPU: a row's partials are then all the parallelism there
// is; measured on 16 agents x 4 query heads with 278 partials per row, 12.3 -> 8.8 us).
constexpr int kCombineWaves = 4, kCombineWavesFewRows = 16;
constexpr int kCus = 256;  // compute units of the GPU
constexpr int combine_batch(int cw) { return cw == kCombineWaves ? 12 : 8; }  // partials in flight per wave

__device__ __forceinline__ void lse_merge(float &M, float &L, f32x4 &acc, float mk, float lk, const f32x4 &v) {
    const float Mn = fmaxf(M, mk);
    const float Mu = Mn == kNegInf ? 0.f : Mn;
    const float e0 = fast_exp2(M - Mu), e1 = fast_exp2(mk - Mu);
    L = L * e0 + lk * e1;
    acc = acc * e0 + v * e1;
    M = Mn;
}

template <int R, int G, int CW>
__global__ __launch_bounds__(64 * CW) void decode_combine_kernel(DecodeArgs p) {
    constexpr int NV = (D + R) / 4;  // float4s of acc and acc_r; (m, l) follow
    constexpr int RB = R > 0 ? R : 1;
    constexpr int BATCH = combine_batch(CW);
    __shared__ f32x4 s_acc[CW > 1 ? CW - 1 : 1][NV + 1];
    const int row = blockIdx.x;
    const int wave = uniform(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int hq = p.hq;
    const int a = row / hq, j = row - a * hq;
    const int h = j / G, jj = j - h * G;
    const int32_t *ptr = p.plan + p.off_ptr;
    const int k0 = ptr[a], K = ptr[a + 1] - k0;
    const int ad = R > 0 ? p.adapter_idx[a] : -1;
    const int stride = p.ws_stride;
    const i32x4 rs = workspace_rsrc(p.ws, p.ws_bytes);
    // byte offsets: record of partial k0 for this row, lane's float4 (lanes past NV: float4 0)
    const int rec0 = (int)(((int64_t)k0 * G * p.hkv + jj * p.hkv + h) * stride * 4) + (lane <= NV ? 16 * lane : 0);
    const int kstride = G * p.hkv * stride * 4;

    // B_V[rho][h*D + 4 lane .. +3] for the output dims of lanes 0..31 of wave 0, requested at
    // the start: in registers of wave 0 for the four-wave merge; for the sixteen-wave one (at
    // most 128 registers per lane) in LDS, each wave copying a share of it.
    constexpr bool kBvRegs = CW == kCombineWaves;
    __shared__ u32x2 s_bv[(R > 0 && !kBvRegs) ? R * (D / 4) : 1];
    const uint16_t *bv_row = p.lora_b + ((int64_t)(ad >= 0 ? ad : 0) * 2 + 1) * R * p.hkv * D + (int64_t)h * D;
    u32x2 bv[kBvRegs ? RB : 1];
    if constexpr (R > 0 && kBvRegs) {
        if (wave == 0) {
#pragma unroll
            for (int rho = 0; rho < R; ++rho)
                bv[rho] = ad >= 0 ? ldg64(bv_row + (int64_t)rho * p.hkv * D + 4 * (lane & 31)) : u32x2{0, 0};
        }
    } else if constexpr (R > 0) {
        for (int i = threadIdx.x; i < R * (D / 4); i += 64 * CW)
            s_bv[i] = ad >= 0 ? ldg64(bv_row + (int64_t)(i / (D / 4)) * p.hkv * D + 4 * (i % (D / 4))) : u32x2{0, 0};
    }

    f32x4 acc = {0, 0, 0, 0};
    float M = kNegInf, L = 0.f;
    for (int kb = wave; kb < K; kb += BATCH * CW) {
        f32x4 v[BATCH];
#pragma unroll
        for (int u = 0; u < BATCH; ++u)
            v[u] = kb + u * CW < K ? raw_buffer_load_v4f32(rs, rec0 + (kb + u * CW) * kstride, 0, kDeviceCoherent)
                                   : f32x4{0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
            // past the last partial: weight zero (m = -inf in lane NV, zeros elsewhere)
            if (!(kb + u * CW < K && lane <= NV)) v[u] = f32x4{lane == NV ? kNegInf : 0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < BATCH; ++u) lse_merge(M, L, acc, __shfl(v[u].x, NV), __shfl(v[u].y, NV), v[u]);
    }
    if constexpr (CW > 1) {
        // lane NV's acc holds (L, 0, 0, 0) scaled alongside; carry (M, L) there instead
        if (wave > 0 && lane <= NV) s_acc[wave - 1][lane] = lane == NV ? f32x4{M, L, 0.f, 0.f} : acc;
        __syncthreads();
        if (wave > 0) return;
#pragma unroll 3
        for (int w = 0; w < CW - 1; ++w) {
            const f32x4 v = lane <= NV ? s_acc[w][lane] : f32x4{0, 0, 0, 0};
            lse_merge(M, L, acc, __shfl(v.x, NV), __shfl(v.y, NV), lane < NV ? v : f32x4{0, 0, 0, 0});
        }
    }
    // Stage 3 (Eq. 4): lanes 0..31 own output dims 4 lane .. +3; acc_r sits in lanes 32..
    f32x4 o = acc;
    auto apply_bv = [&](int rho, u32x2 b) __attribute__((always_inline)) {
        const float ar = __shfl(acc[rho % 4], D / 4 + rho / 4);
        o[0] += ar * bf16_lo(b.x);
        o[1] += ar * bf16_hi(b.x);
        o[2] += ar * bf16_lo(b.y);
        o[3] += ar * bf16_hi(b.y);
    };
    if constexpr (R > 0 && kBvRegs) {
#pragma unroll
        for (int rho = 0; rho < R; ++rho) apply_bv(rho, bv[rho]);
    } else if constexpr (R > 0) {
        // eight ranks per LDS wait keeps the sixteen-wave merge within its registers
        for (int r0 = 0; r0 < R; r0 += 8) {
#pragma unroll
            for (int i = 0; i < 8; ++i) apply_bv(r0 + i, s_bv[(r0 + i) * (D / 4) + (lane & 31)]);
        }
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    if (lane < D / 4) {
        uint16_t *dst = p.out + ((int64_t)a * hq + j) * D + 4 * lane;
        *reinterpret_cast<u32x2 *>(dst) = u32x2{pack_bf16(o[0] * inv, o[1] * inv), pack_bf16(o[2] * inv, o[3] * inv)};
    }
}

template <int R, int G, bool ROPE>
hipError_t launch_decode(const DecodeArgs &da_in, int n_blocks, int n_agents, bool wide_merge, hipStream_t st,
                         void *const *ev) {
    hipError_t e;
    DecodeArgs da = da_in;
    da.n_rows = n_agents * da.hq;
    // timing events carry the kernels' own start and end timestamps (set by the launch)
    hipEvent_t e0 = ev ? static_cast<hipEvent_t>(ev[0]) : nullptr;
    hipEvent_t e1 = ev ? static_cast<hipEvent_t>(ev[1]) : nullptr;
    hipEvent_t e2 = ev ? static_cast<hipEvent_t>(ev[2]) : nullptr;
    if constexpr (ROPE) hipExtLaunchKernelGGL((decode_rope_kernel<R, G>), dim3(n_blocks), dim3(256), 0, st, e0, e1, 0, da);
    else hipExtLaunchKernelGGL((decode_split_kernel<R, G>), dim3(n_blocks), dim3(256), 0, st, e0, e1, 0, da);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (!wide_merge)
        hipExtLaunchKernelGGL((decode_combine_kernel<R, G, kCombineWaves>), dim3(da.n_rows), dim3(64 * kCombineWaves), 0, st,
                              nullptr, e2, 0, da);
    else
        hipExtLaunchKernelGGL((decode_combine_kernel<R, G, kCombineWavesFewRows>), dim3(da.n_rows),
                              dim3(64 * kCombineWavesFewRows), 0, st, nullptr, e2, 0, da);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hipSuccess;
}

template <int R, int G>
hipError_t dispatch_rope(bool rope, const DecodeArgs &da, int nb, int na, bool wide, hipStream_t st, void *const *ev) {
    if constexpr (R == 0) {
        return launch_decode<0, G, false>(da, nb, na, wide, st, ev);
    } else {
        return rope ? launch_decode<R, G, true>(da, nb, na, wide, st, ev)
                    : launch_decode<R, G, false>(da, nb, na, wide, st, ev);
    }
}

template <int G>
hipError_t dispatch_rank(int r, bool rope, const DecodeArgs &da, int nb, int na, bool wide, hipStream_t st,
                         void *const *ev) {
    switch (r) {
    case 0: return dispatch_rope<0, G>(rope, da, nb, na, wide, st, ev);
    case 8: return dispatch_rope<8, G>(rope, da, nb, na, wide, st, ev);
    case 16: return dispatch_rope<16, G>(rope, da, nb, na, wide, st, ev);
    case 32: return dispatch_rope<32, G>(rope, da, nb, na, wide, st, ev);
    case 64: return dispatch_rope<64, G>(rope, da, nb, na, wide, st, ev);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

namespace fkv {
fkv_status validate_attn_common(const fkv_attn_args *a, const char *who);
int64_t plan_max_pages(const fkv_plan *plan);
}  // namespace fkv

namespace {

// Both decode entry points: checks, then the split and merge launches with the partial rows
// in `workspace` (`workspace_bytes` long).
fkv_status decode_impl(const fkv_attn_args *a, const fkv_plan *plan, void *stream, void *workspace,
                       size_t workspace_bytes) {
    fkv_status st = fkv::validate_attn_common(a, "fkv_residual_attention_decode");
    if (st != FKV_OK) return st;
    if (!plan || !a->plan || !workspace)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan (host and device copy) and workspace are required");
    const auto &w = plan->words;
    const int g = a->hq / a->hkv;
    if (plan->n_agents != a->n_agents || plan->hkv != a->hkv || plan->g != g)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan was built for other n_agents / heads");
    fkv_plan_info info;
    fkv_decode_plan_info(plan, a->d, a->r, &info);
    if ((int64_t)workspace_bytes < info.workspace_bytes)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: workspace too small");
    if (a->max_pages < fkv::plan_max_pages(plan))
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: block-table rows shorter than the plan's "
                                          "page capacity");
    if (a->rope_cos && (int64_t)a->rope_max_pos < fkv::plan_max_pages(plan) * a->page_size)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: RoPE table shorter than the longest sequence");
    if (g != 4 && g != 8)
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_residual_attention_decode: query heads per KV head must be 4 or 8");
    const bool rope_on = a->rope_cos != nullptr && a->r > 0;
    if (w[fkv::H_RANK] != a->r || w[fkv::H_ROPE] != (rope_on ? 1 : 0))
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: the plan was built for another rank or "
                                          "RoPE setting");
    const int hpb = w[fkv::H_HEADS_PER_BLOCK];
    if (hpb != fkv::decode_heads_per_block(a->hkv, rope_on))
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan built for another head blocking");
    if (w[fkv::H_MAX_ITEM_AGENTS] > fkv::decode_item_agent_cap(g, a->hkv, a->r, rope_on))
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: the plan puts more agents in a work item "
                                          "than this kernel takes");
    if (w[fkv::H_PAGES_PER_SPLIT] > fkv::kMaxPagesSingle)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan items longer than the kernel takes");
    if (w[fkv::H_OFF_DESC] < 0)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan has no block descriptors");
    DecodeArgs da;
    da.q = static_cast<const uint16_t *>(a->q);
    da.base_kv = static_cast<const uint16_t *>(a->base_kv);
    da.res_kv = static_cast<const uint16_t *>(a->res_kv);
    da.lora_b = static_cast<const uint16_t *>(a->lora_b);
    da.adapter_idx = a->adapter_idx;
    da.base_bt = a->base_bt;
    da.res_bt = a->res_bt;
    da.seq_lens = a->seq_lens;
    da.rope_cos = a->rope_cos;
    da.rope_sin = a->rope_sin;
    da.plan = a->plan;
    da.ws = static_cast<float *>(workspace);
    da.out = static_cast<uint16_t *>(a->out);
    da.hq = a->hq;
    da.hkv = a->hkv;
    da.max_pages = a->max_pages;
    da.ws_stride = ws_stride_of(a->r);
    da.off_items = w[fkv::H_OFF_ITEMS];
    da.off_blocks = w[fkv::H_OFF_BLOCKS];
    da.off_ptr = w[fkv::H_OFF_AGENT_PTR];
    da.off_zero = w[fkv::H_OFF_ZERO];
    da.off_desc = w[fkv::H_OFF_DESC];
    da.scale_log2 = a->scale * 1.4426950408889634f;
    da.rope_max_pos = a->rope_cos ? a->rope_max_pos : 0;
    da.ws_bytes = fkv::decode_partials_bytes(plan, a->d, a->r);
    if (da.ws_bytes >= 0x7fffffff)
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_residual_attention_decode: partial rows above 2 GiB");
    da.n_rows = a->n_agents * a->hq;
    const int nb = w[fkv::H_N_BLOCKS];
    hipStream_t hs = static_cast<hipStream_t>(stream);
    const bool rope = a->rope_cos != nullptr && a->r > 0;
    // Merge with sixteen waves per row when there are fewer rows than half the compute units
    // and each row has many partials (at least 128 on average); four otherwise.
    const int64_t total_partials = w[w[fkv::H_OFF_AGENT_PTR] + a->n_agents];
    const bool wide = (int64_t)a->n_agents * a->hq < kCus / 2 && total_partials >= 128LL * a->n_agents;
    hipError_t e = g == 4 ? dispatch_rank<4>(a->r, rope, da, nb, a->n_agents, wide, hs, a->timing_events)
                          : dispatch_rank<8>(a->r, rope, da, nb, a->n_agents, wide, hs, a->timing_events);
    if (e != hipSuccess)
        return fkv::fail(FKV_ERR_HIP, std::string("fkv_residual_attention_decode: launch failed: ") + hipGetErrorString(e));
    return FKV_OK;
}

// Partial rows of fkv_residual_attention_decode_noalloc: one array per GPU, held from the
// library's first use on that GPU until the process ends.  Host code never passes the
// array's name to a kernel (on the host it names a stand-in, not device memory): each
// device's address comes from hipGetSymbolAddress with that device current.
constexpr size_t kNoAllocBytes = FKV_NOALLOC_WORKSPACE_BYTES;
__device__ __attribute__((aligned(256))) unsigned char scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_addr[kMaxDevices] = {};

fkv_status scratch_address(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return fkv::fail(FKV_ERR_HIP, std::string("fkv_residual_attention_decode_noalloc: hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_residual_attention_decode_noalloc: device index above 63");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fkv::fail(FKV_ERR_HIP, std::string("fkv_residual_attention_decode_noalloc: hipGetSymbolAddress: ") +
                                              hipGetErrorString(e));
        g_scratch_addr[dev] = p;
    }
    *out = g_scratch_addr[dev];
    return FKV_OK;
}

}  // namespace

extern "C" fkv_status fkv_residual_attention_decode(const fkv_attn_args *a, const fkv_plan *plan, void *stream) {
    fkv::clear_error();
    if (!a) return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: null args");
    return decode_impl(a, plan, stream, a->workspace, a->workspace_bytes);
}

extern "C" fkv_status fkv_residual_attention_decode_noalloc(const fkv_attn_args *a, const fkv_plan *plan, void *stream) {
    fkv::clear_error();
    if (!a || !plan) return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode_noalloc: null argument");
    fkv_plan_info info;
    fkv_status st = fkv_decode_plan_info(plan, a->d, a->r, &info);
    if (st != FKV_OK) return st;
    if (info.workspace_bytes > (int64_t)kNoAllocBytes)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode_noalloc: the plan's partial rows (" +
                                              std::to_string(info.workspace_bytes) + " bytes) exceed the " +
                                              std::to_string(kNoAllocBytes) + "-byte static workspace");
    void *ws = nullptr;
    st = scratch_address(&ws);
    if (st != FKV_OK) return st;
    return decode_impl(a, plan, stream, ws, kNoAllocBytes);
}
