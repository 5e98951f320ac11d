// ResidualAttention decode for gfx950 (Section 5.3, Algorithm 1).
//
// One workgroup = one (work item, KV head h).  A work item is a page range of a
// segment together with up to four groups of agents that read the same base
// pages there; a group is the floor(16/g) agents whose g query heads of KV head h
// fill the 16 rows of one matrix-core tile.
//  - single-group items (typically private suffixes): the four waves stride over
//    the pages with a register-double-buffered pipeline and are merged through LDS
//    at the end;
//  - multi-group items (shared prefixes): each base page is loaded once into LDS
//    and every wave applies it to its own group's 16 rows, so a shared page crosses
//    the memory hierarchy once per workgroup instead of once per group.
// Each row leaves one partial (m, l, acc, acc_r) in the workspace; a second kernel
// merges an agent's partials (log-sum-exp combine) and applies Stage 3.
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
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "internal.hpp"
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

struct DecodeArgs {
    const uint16_t *q, *base_kv, *res_kv, *lora_b;
    const int32_t *adapter_idx, *base_bt, *res_bt, *seq_lens;
    const float *rope_cos, *rope_sin;
    const int32_t *plan;
    float *ws;
    uint16_t *out;
    int32_t hq, hkv, max_pages, ws_stride;
    float scale_log2;  // softmax scale * log2(e)
};

constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int cmin(int a, int b) { return a < b ? a : b; }

template <int R, int G, bool ROPE>
struct SplitShape {
    static constexpr int AG = ROWS / G;                                        // agents per group
    static constexpr int RT = R == 0 ? 0 : (R + 15) / 16;                      // 16-wide rank tiles
    static constexpr int MAX_SLOTS = cmin(fkv::kMaxGroups * AG, fkv::kMaxItemAgents);
    static constexpr int BKT_SLOTS = ROPE ? cmin(MAX_SLOTS, 256 / (R > 0 ? R : 1)) : 0;
    static constexpr int MERGE_BYTES = WAVES * ((8 + RT) * 256 + 2 * ROWS) * 4;
    static constexpr int STAGE_BYTES = 2 * 2 * 2 * kBlockHalfs * 2;           // [buf][page][K|V] blocks
    static constexpr int BSTAGE_BYTES = ROPE ? 4 * R * D * 2 : 0;             // B_K rows of 4 slots
    static constexpr int UNION_BYTES = cmax(MERGE_BYTES, cmax(STAGE_BYTES, BSTAGE_BYTES));
    static constexpr int BKT_BYTES = BKT_SLOTS * RT * 8 * 64 * 8;             // B_K^T fragments
    static constexpr int TABLE_WORDS = (1 + (R > 0 ? MAX_SLOTS : 0)) * kMaxPagesPerItem;
    static constexpr int LDS_BYTES = UNION_BYTES + BKT_BYTES + TABLE_WORDS * 4;
};

template <int R, int G, bool ROPE>
__global__ __launch_bounds__(256, ROPE ? 1 : 2) void decode_split_kernel(DecodeArgs p) {
    using S = SplitShape<R, G, ROPE>;
    constexpr int AG = S::AG;
    constexpr int RT = S::RT;
    constexpr int RTX = RT > 0 ? RT : 1;
    __shared__ __attribute__((aligned(16))) unsigned char lds[S::LDS_BYTES];
    float *lds_f = reinterpret_cast<float *>(lds);
    uint16_t *lds_h = reinterpret_cast<uint16_t *>(lds);
    uint32_t *lds_bkt = reinterpret_cast<uint32_t *>(lds + S::UNION_BYTES);
    int32_t *s_tab = reinterpret_cast<int32_t *>(lds + S::UNION_BYTES + S::BKT_BYTES);

    const int32_t *plan = p.plan;
    const int blk = plan[plan[fkv::H_OFF_BLOCKS] + blockIdx.x];
    if (blk < 0) return;
    const int hkv = p.hkv;
    const int item = blk / hkv;
    const int h = blk - item * hkv;
    const int32_t *rec = plan + plan[fkv::H_OFF_ITEMS] + item * fkv::kItemWords;
    const int pg0 = rec[0], pg1 = rec[1], leader = rec[2], nag = rec[3], row_base = rec[4];
    const int32_t *item_agents = rec + 5;
    const int ng = (nag + AG - 1) / AG;                 // agent groups in the item (1..4)
    const int ngp = ng == 1 ? 1 : (ng == 2 ? 2 : 4);   // groups rounded to a divisor of 4

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int my_group = wave % ngp;
    const int sb = my_group * AG;                       // first item slot of this wave's group
    const int my_slot_l = col / G;                      // this lane's row: slot within the group
    const bool row_active = my_slot_l < AG && sb + my_slot_l < nag;
    const int my_agent = row_active ? item_agents[sb + my_slot_l] : 0;
    const int my_len = row_active ? p.seq_lens[my_agent] : 0;
    const int qh = h * G + (col % G);

    int slot_ad[AG], slot_len[AG];
    int max_len = 0;  // longest sequence of the wave's group (V tokens past it are zeroed)
#pragma unroll
    for (int s = 0; s < AG; ++s) {
        const bool ok = sb + s < nag;
        const int ag_id = ok ? item_agents[sb + s] : 0;
        slot_ad[s] = (ok && R > 0) ? p.adapter_idx[ag_id] : -1;
        slot_len[s] = ok ? p.seq_lens[ag_id] : 0;
        max_len = max_len > slot_len[s] ? max_len : slot_len[s];
    }

    // Q^T as the B operand of the 16x16x32 products.  The head-dim index of slot j in
    // k-step kk is 32kk + 16(j/4) + 4grp + j%4 for this lane group: the order in which
    // a rebuilt key tile leaves the 16x16x16 accumulators and in which K blocks are
    // stored, so base keys, rebuilt keys and queries all share it.
    const uint16_t *qrow = p.q + ((int64_t)my_agent * p.hq + qh) * D;
    u32x4 qf[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        u32x4 v = {0, 0, 0, 0};
        if (row_active) {
            const u32x2 lo = ldg64(qrow + 32 * kk + 4 * grp);
            const u32x2 hi = ldg64(qrow + 32 * kk + 16 + 4 * grp);
            v = u32x4{lo.x, lo.y, hi.x, hi.y};
        }
        qf[kk] = v;
    }

    const int64_t n = (int64_t)hkv * D;
    const int64_t res_page_halfs = 2 * PS * R;
    // ---- prologue: per-agent residual key operands ----
    u32x2 wf[RTX];   // RoPE off: (B_K q) for this lane's row, bf16, B operand of 16x16x16
    if constexpr (R > 0 && !ROPE) {
        f32x4 wacc[RTX];
#pragma unroll
        for (int t = 0; t < RT; ++t) wacc[t] = f32x4{0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < AG; ++s) {
            if (slot_ad[s] < 0) continue;
            const uint16_t *bk = p.lora_b + (int64_t)slot_ad[s] * 2 * R * n + (int64_t)h * D;
#pragma unroll
            for (int t = 0; t < RT; ++t) {
                const int rho = 16 * t + col;
                f32x4 acc = {0, 0, 0, 0};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    u32x4 a = {0, 0, 0, 0};
                    if (rho < R) {
                        const u32x2 lo = ldg64(bk + (int64_t)rho * n + 32 * kk + 4 * grp);
                        const u32x2 hi = ldg64(bk + (int64_t)rho * n + 32 * kk + 16 + 4 * grp);
                        a = u32x4{lo.x, lo.y, hi.x, hi.y};
                    }
                    acc = mfma32(a, qf[kk], acc);
                }
                if (my_slot_l == s) wacc[t] = acc;
            }
        }
#pragma unroll
        for (int t = 0; t < RT; ++t) wf[t] = pack4(wacc[t]);
    }
    if constexpr (ROPE) {
        // B_K^T fragments of every item slot (lane holds B_K[16t + 4grp + i][16mt + col]),
        // built from row-major B_K slices staged four slots at a time.
        const int nstage = ngp * AG;  // unused slots of the last group get zero fragments
        for (int s0 = 0; s0 < nstage; s0 += 4) {
            const int ns = nstage - s0 < 4 ? nstage - s0 : 4;
            for (int idx = threadIdx.x; idx < ns * R * (D / 8); idx += 256) {
                const int sl = idx / (R * (D / 8));
                const int rem = idx - sl * (R * (D / 8));
                const int rho = rem / (D / 8), c8 = rem - rho * (D / 8);
                const int ad = s0 + sl < nag ? p.adapter_idx[item_agents[s0 + sl]] : -1;
                u32x4 v = {0, 0, 0, 0};
                if (ad >= 0) v = ldg128(p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)rho * n + (int64_t)h * D + 8 * c8);
                *reinterpret_cast<u32x4 *>(lds_h + (sl * R + rho) * D + 8 * c8) = v;
            }
            __syncthreads();
            for (int idx = threadIdx.x; idx < ns * RT * 8 * 64; idx += 256) {
                const int ln = idx & 63;
                const int rest = idx >> 6;  // (sl*RT + t)*8 + mt
                const int mt = rest & 7, st = rest >> 3;
                const int sl = st / RTX, t = st - sl * RTX;
                const int c = ln & 15, gg = ln >> 4;
                uint32_t w[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int r0 = 16 * t + 4 * gg + 2 * j;
                    const uint16_t lo = r0 < R ? lds_h[(sl * R + r0) * D + 16 * mt + c] : (uint16_t)0;
                    const uint16_t hi = r0 + 1 < R ? lds_h[(sl * R + r0 + 1) * D + 16 * mt + c] : (uint16_t)0;
                    w[j] = (uint32_t)lo | ((uint32_t)hi << 16);
                }
                const int o = ((((s0 + sl) * RTX + t) * 8 + mt) * 64 + ln) * 2;
                lds_bkt[o] = w[0];
                lds_bkt[o + 1] = w[1];
            }
            __syncthreads();
        }
    }
    // block-table entries of the item's pages: one round trip for the whole item
    const int npg = pg1 - pg0;
    for (int i = threadIdx.x; i < npg; i += 256) s_tab[i] = p.base_bt[(int64_t)leader * p.max_pages + pg0 + i];
    if constexpr (R > 0) {
        // slots past nag (the unused tail of the last group) read residual page 0, masked
        for (int s = 0; s < ngp * AG; ++s) {
            const int ag_id = s < nag ? item_agents[s] : 0;
            const bool has = s < nag && p.adapter_idx[ag_id] >= 0;
            for (int i = threadIdx.x; i < npg; i += 256)
                s_tab[(1 + s) * kMaxPagesPerItem + i] = has ? p.res_bt[(int64_t)ag_id * p.max_pages + pg0 + i] : 0;
        }
    }
    __syncthreads();

    // ---- state of this wave's 16 rows ----
    f32x4 oacc[8];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) oacc[mt] = f32x4{0, 0, 0, 0};
    f32x4 racc[RTX];
#pragma unroll
    for (int t = 0; t < RTX; ++t) racc[t] = f32x4{0, 0, 0, 0};
    float m_run = kNegInf, l_run = 0.f;

    // lane-constant element offsets of the rCache fragment loads
    int ck_off[RTX], cv_off[RTX];
    bool ck_ok[RTX], cv_ok[RTX];
#pragma unroll
    for (int t = 0; t < RTX; ++t) {
        const int rho = 16 * t + col, rk = 16 * t + 4 * grp;
        cv_ok[t] = rho < R;
        ck_ok[t] = rk < R;
        cv_off[t] = PS * R + (rho < R ? rho : (R > 0 ? R - 1 : 0)) * PS + 4 * grp;   // C_V^T[rho][tok 4grp..]
        ck_off[t] = col * R + (rk < R ? rk : (R >= 4 ? R - 4 : 0));                  // C_K[tok col][rho 4grp..]
    }
    auto mask4 = [&](u32x2 v, int vis) {  // zero tokens 4grp+i >= vis of a [.][tok] fragment
        if (4 * grp + 0 >= vis) v.x &= 0xffff0000u;
        if (4 * grp + 1 >= vis) v.x &= 0x0000ffffu;
        if (4 * grp + 2 >= vis) v.y &= 0xffff0000u;
        if (4 * grp + 3 >= vis) v.y &= 0x0000ffffu;
        return v;
    };
    // rCache fragments of slot sb+s for logical page pg
    auto load_res = [&](int pg, int s, u32x2 *ck, u32x2 *cv) {
        const int rpage = uniform(s_tab[(1 + sb + s) * kMaxPagesPerItem + (pg - pg0)]);
        const uint16_t *rb = p.res_kv + (int64_t)rpage * res_page_halfs;
#pragma unroll
        for (int t = 0; t < RT; ++t) {
            const u32x2 v = ldg64(rb + cv_off[t]);
            const u32x2 k = ldg64(rb + ck_off[t]);
            cv[t] = cv_ok[t] ? v : u32x2{0, 0};
            ck[t] = ck_ok[t] ? k : u32x2{0, 0};
        }
    };
    auto load_rope = [&](int pg, f32x4 *cs, f32x4 *sn) {
        const float *cr = p.rope_cos + (int64_t)pg * (PS * D / 2);
        const float *sr = p.rope_sin + (int64_t)pg * (PS * D / 2);
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            cs[mt] = *reinterpret_cast<const f32x4 *>(cr + 256 * mt + lane * 4);
            sn[mt] = *reinterpret_cast<const f32x4 *>(sr + 256 * mt + lane * 4);
        }
    };

    // One page for this wave's rows.  kf/vf hold the base K and V fragments; ck/cv the
    // rCache fragments of the NS slots; cs/sn the RoPE rows.  valid = false (a padding
    // page of a stage) masks every token.
    auto compute_page = [&](auto ns_tag, int pg, bool valid, const u32x4 *kf, u32x2 *vf, u32x2 (*ck)[RTX],
                            u32x2 (*cv)[RTX], const f32x4 *cs, const f32x4 *sn) {
        constexpr int NS = decltype(ns_tag)::value;
        const int tok0 = pg * PS;
        const int vis = max_len - tok0;   // tokens past every agent's end may hold any bits
        if (vis < PS) {
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) vf[mt] = mask4(vf[mt], vis);
        }
        f32x4 sacc = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) sacc = mfma32(kf[kk], qf[kk], sacc);
        if constexpr (R > 0) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                // slots without an adapter contribute zeros (zero W or zero B_K^T)
                // rCache tokens past the slot's own length are unwritten: zero them (a NaN
                // there would reach every row through the zero entries of the other slots)
                const int svis = slot_len[s] - tok0;
                if (svis < PS) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        cv[s][t] = mask4(cv[s][t], svis);
                        ck[s][t] = col < svis ? ck[s][t] : u32x2{0, 0};
                    }
                }
                if constexpr (!ROPE) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const u32x2 b = my_slot_l == s ? wf[t] : u32x2{0, 0};
                        sacc = mfma16(ck[s][t], b, sacc);
                    }
                } else {
                    // Stage 1: U^T = B_K^T C_K^T, deferred RoPE, then S^T += K_lora Q_s^T
                    f32x4 u[8];
#pragma unroll
                    for (int mt = 0; mt < 8; ++mt) {
                        u[mt] = f32x4{0, 0, 0, 0};
#pragma unroll
                        for (int t = 0; t < RT; ++t) {
                            const u32x2 a = *reinterpret_cast<const u32x2 *>(
                                lds_bkt + (((((sb + s) * RTX + t) * 8 + mt) * 64) + lane) * 2);
                            u[mt] = mfma16(a, ck[s][t], u[mt]);
                        }
                    }
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float x = u[mt][i], y = u[mt + 4][i];
                            u[mt][i] = x * cs[mt][i] - y * sn[mt][i];
                            u[mt + 4][i] = y * cs[mt][i] + x * sn[mt][i];
                        }
                    }
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        const u32x2 lo = pack4(u[2 * kk]), hi = pack4(u[2 * kk + 1]);
                        const u32x4 b = my_slot_l == s ? qf[kk] : u32x4{0, 0, 0, 0};
                        sacc = mfma32(u32x4{lo.x, lo.y, hi.x, hi.y}, b, sacc);
                    }
                }
            }
        }
        // Stage 2: online softmax over this page's 16 tokens (rows live in lanes)
        float sv[4];
        float mx = kNegInf;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int tok = tok0 + 4 * grp + i;
            sv[i] = (valid && row_active && tok < my_len) ? sacc[i] * p.scale_log2 : kNegInf;
            mx = fmaxf(mx, sv[i]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        const float m_use = m_new == kNegInf ? 0.f : m_new;
        const float alpha = fast_exp2(m_run - m_use);
        f32x4 pv;
        float psum = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            pv[i] = fast_exp2(sv[i] - m_use);
            psum += pv[i];
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
        const u32x2 pf = pack4(pv);
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
            oacc[mt] *= alpha;
            oacc[mt] = mfma16(vf[mt], pf, oacc[mt]);
        }
        if constexpr (R > 0) {
#pragma unroll
            for (int t = 0; t < RT; ++t) racc[t] *= alpha;
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const u32x2 pm = my_slot_l == s ? pf : u32x2{0, 0};
#pragma unroll
                for (int t = 0; t < RT; ++t) racc[t] = mfma16(cv[s][t], pm, racc[t]);
            }
        }
    };

    if (ng == 1) {
        // ---- single group: waves stride over the pages, registers double-buffered ----
        // The loop is specialised on the number NS of agent slots so that every load it
        // issues is consumed; all loads are unconditional and in a fixed order, so the
        // compiler can count them and the prefetched page stays in flight.
        auto run_pages = [&](auto ns_tag) {
            constexpr int NS = decltype(ns_tag)::value;
            constexpr int NSR = R > 0 ? NS : 1;
            struct Frag {
                f32x4 cs[ROPE ? 4 : 1], sn[ROPE ? 4 : 1];
                u32x4 kf[4];
                u32x2 vf[8];
                u32x2 ck[NSR][RTX];
                u32x2 cv[NSR][RTX];
            };
            auto load = [&](int pg, Frag &f) {
                if constexpr (ROPE) load_rope(pg, f.cs, f.sn);  // issued first: consumed first
                const int bpage = uniform(s_tab[pg - pg0]);
                const uint16_t *kblk = p.base_kv + ((int64_t)bpage * 2 * hkv + h) * kBlockHalfs;
                const uint16_t *vblk = kblk + (int64_t)hkv * kBlockHalfs;
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) f.kf[kk] = ldg128(kblk + kk * 512 + lane * 8);
#pragma unroll
                for (int q2 = 0; q2 < 4; ++q2) {
                    const u32x4 v = ldg128(vblk + q2 * 512 + lane * 8);
                    f.vf[2 * q2] = u32x2{v.x, v.y};
                    f.vf[2 * q2 + 1] = u32x2{v.z, v.w};
                }
                if constexpr (R > 0) {
#pragma unroll
                    for (int s = 0; s < NS; ++s) load_res(pg, s, f.ck[s], f.cv[s]);
                }
            };
            Frag fa, fb;
            int pg = pg0 + wave;
            if (pg < pg1) {
                const int last = pg + (pg1 - 1 - pg) / WAVES * WAVES;
                load(pg, fa);
                for (;;) {
                    load(pg + WAVES <= last ? pg + WAVES : last, fb);
                    compute_page(ns_tag, pg, true, fa.kf, fa.vf, fa.ck, fa.cv, fa.cs, fa.sn);
                    pg += WAVES;
                    if (pg > last) break;
                    load(pg + WAVES <= last ? pg + WAVES : last, fa);
                    compute_page(ns_tag, pg, true, fb.kf, fb.vf, fb.ck, fb.cv, fb.cs, fb.sn);
                    pg += WAVES;
                    if (pg > last) break;
                }
            }
        };
        using I1 = std::integral_constant<int, 1>;
        using I2 = std::integral_constant<int, cmin(2, AG)>;
        using I3 = std::integral_constant<int, cmin(3, AG)>;
        using I4 = std::integral_constant<int, cmin(4, AG)>;
        if (R == 0 || nag == 1) run_pages(I1{});
        else if (nag == 2 || AG == 2) run_pages(I2{});
        else if (nag == 3) run_pages(I3{});
        else run_pages(I4{});
    } else {
        // ---- several groups: stages of two pages, base K/V loaded once into LDS ----
        // Wave w loads block (K if w even, V if odd) of stage page w/2 for everyone and
        // computes its own group: both stage pages (4 groups) or stage page w/2 (2 groups).
        constexpr int NSR = R > 0 ? AG : 1;
        struct Stage {
            u32x4 kv[4];                                 // this wave's share of the stage's base blocks
            u32x2 ck[2][NSR][RTX], cv[2][NSR][RTX];      // rCache of the wave's pages
            f32x4 cs[2][ROPE ? 4 : 1], sn[2][ROPE ? 4 : 1];
        };
        const int last = pg1 - 1;
        const int lpage = wave >> 1, lkv = wave & 1;     // what this wave loads
        const int npages_w = ngp == 4 ? 2 : 1;           // stage pages this wave computes
        const int wpage0 = ngp == 4 ? 0 : (wave >> 1);
        auto load_stage = [&](int sp, Stage &st) {
            const int pl = sp + lpage <= last ? sp + lpage : last;
            const int bpage = uniform(s_tab[pl - pg0]);
            const uint16_t *blkp = p.base_kv + (((int64_t)bpage * 2 + lkv) * hkv + h) * kBlockHalfs;
#pragma unroll
            for (int i = 0; i < 4; ++i) st.kv[i] = ldg128(blkp + i * 512 + lane * 8);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                if (j < npages_w) {
                    const int pj = sp + wpage0 + j <= last ? sp + wpage0 + j : last;
                    if constexpr (ROPE) load_rope(pj, st.cs[j], st.sn[j]);
                    if constexpr (R > 0) {
#pragma unroll
                        for (int s = 0; s < AG; ++s) load_res(pj, s, st.ck[j][s], st.cv[j][s]);
                    }
                }
            }
        };
        auto store_stage = [&](int buf, const Stage &st) {
            uint16_t *dst = lds_h + ((buf * 2 + lpage) * 2 + lkv) * kBlockHalfs;
#pragma unroll
            for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4 *>(dst + i * 512 + lane * 8) = st.kv[i];
        };
        auto compute_stage = [&](int buf, int sp, Stage &st) {
            using IA = std::integral_constant<int, (R > 0 ? AG : 1)>;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                if (j < npages_w) {
                    const int pj = sp + wpage0 + j;
                    const uint16_t *kb = lds_h + ((buf * 2 + wpage0 + j) * 2 + 0) * kBlockHalfs;
                    const uint16_t *vb = kb + kBlockHalfs;
                    u32x4 kf[4];
                    u32x2 vf[8];
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) kf[kk] = *reinterpret_cast<const u32x4 *>(kb + kk * 512 + lane * 8);
#pragma unroll
                    for (int q2 = 0; q2 < 4; ++q2) {
                        const u32x4 v = *reinterpret_cast<const u32x4 *>(vb + q2 * 512 + lane * 8);
                        vf[2 * q2] = u32x2{v.x, v.y};
                        vf[2 * q2 + 1] = u32x2{v.z, v.w};
                    }
                    compute_page(IA{}, pj <= last ? pj : last, pj <= last, kf, vf, st.ck[j], st.cv[j], st.cs[j],
                                 st.sn[j]);
                }
            }
        };
        Stage sa, sb2;
        int sp = pg0;
        load_stage(sp, sa);
        store_stage(0, sa);
        __syncthreads();
        int buf = 0;
        for (;;) {
            load_stage(sp + 2, sb2);     // past the item end this re-reads the last page (unused)
            compute_stage(buf, sp, sa);
            store_stage(buf ^ 1, sb2);
            __syncthreads();
            sp += 2;
            buf ^= 1;
            if (sp >= pg1) break;
            load_stage(sp + 2, sa);
            compute_stage(buf, sp, sb2);
            store_stage(buf ^ 1, sa);
            __syncthreads();
            sp += 2;
            buf ^= 1;
            if (sp >= pg1) break;
        }
    }
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);

    // ---- merge the waves that hold the same group and write one partial per row ----
    __syncthreads();  // LDS stages of the main loop are dead from here on
    constexpr int TILES = 8 + RT;
    float *lds_m = lds_f + WAVES * TILES * 256;
    float *lds_l = lds_m + WAVES * ROWS;
    {
        float *mine = lds_f + wave * TILES * 256;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) *reinterpret_cast<f32x4 *>(mine + (mt * 64 + lane) * 4) = oacc[mt];
#pragma unroll
        for (int t = 0; t < RT; ++t) *reinterpret_cast<f32x4 *>(mine + ((8 + t) * 64 + lane) * 4) = racc[t];
        if (grp == 0) {
            lds_m[wave * ROWS + col] = m_run;
            lds_l[wave * ROWS + col] = l_run;
        }
    }
    __syncthreads();
    const int rows_used = nag * G;
    const int rec_len = 2 + D + R;
    const int nw = WAVES / ngp;  // waves holding each group
    for (int idx = threadIdx.x; idx < rows_used * rec_len; idx += 256) {
        const int r = idx / rec_len, k = idx - r * rec_len;
        const int gr = r / ROWS, rr = r - gr * ROWS;   // group and row within its tile
        float mw[WAVES], M = kNegInf;
#pragma unroll
        for (int i = 0; i < WAVES; ++i) {
            mw[i] = i < nw ? lds_m[(gr + i * ngp) * ROWS + rr] : kNegInf;
            M = fmaxf(M, mw[i]);
        }
        const float Mu = M == kNegInf ? 0.f : M;
        float v = 0.f;
        if (k == 0) {
            v = M;
        } else if (k == 1) {
#pragma unroll
            for (int i = 0; i < WAVES; ++i)
                if (i < nw) v += fast_exp2(mw[i] - Mu) * lds_l[(gr + i * ngp) * ROWS + rr];
        } else {
            const int e = k - 2;
            int tile, ln, ii;
            if (e < D) {
                tile = e >> 4;
                ln = rr + 16 * ((e & 15) >> 2);
                ii = e & 3;
            } else {
                const int rho = e - D;
                tile = 8 + (rho >> 4);
                ln = rr + 16 * ((rho & 15) >> 2);
                ii = rho & 3;
            }
#pragma unroll
            for (int i = 0; i < WAVES; ++i)
                if (i < nw) v += fast_exp2(mw[i] - Mu) * lds_f[(gr + i * ngp) * TILES * 256 + (tile * 64 + ln) * 4 + ii];
        }
        p.ws[((int64_t)(row_base + r) * hkv + h) * p.ws_stride + k] = v;
    }
}

// Log-sum-exp merge of one agent's partials and Stage 3 of Algorithm 1 for one query
// head j (KV head h = j / G): O = (sum_k w_k acc_k + (sum_k w_k acc_r,k) . B_V[h]) / L
// with w_k = 2^(m_k - M), M = max_k m_k, L = sum_k w_k l_k.
constexpr int kCombineThreads = 128;
constexpr int kMaxItemsPerAgent = fkv::kMaxItemsPerAgent;

template <int R, int G>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(DecodeArgs p) {
    const int hq = p.hq;
    const int a = blockIdx.x / hq;
    const int j = blockIdx.x - a * hq;
    const int h = j / G, jj = j - h * G;
    const int32_t *plan = p.plan;
    const int32_t *slots = plan + plan[fkv::H_OFF_AGENT_SLOT];
    const int k0 = plan[plan[fkv::H_OFF_AGENT_PTR] + a];
    const int K = plan[plan[fkv::H_OFF_AGENT_PTR] + a + 1] - k0;
    const int ad = R > 0 ? p.adapter_idx[a] : -1;
    const int stride = p.ws_stride;
    const int tid = threadIdx.x;
    __shared__ float sW[kMaxItemsPerAgent];
    __shared__ int sRow[kMaxItemsPerAgent];
    __shared__ float sRed[2];
    __shared__ float sAccR[R > 0 ? R : 1];

    // M = max_k m_k
    float mloc = kNegInf;
    for (int k = tid; k < K; k += kCombineThreads) {
        const int row = slots[k0 + k] + jj * p.hkv + h;
        sRow[k] = row;
        const float m = p.ws[(int64_t)row * stride];
        sW[k] = m;
        mloc = fmaxf(mloc, m);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, o));
    if ((tid & 63) == 0) sRed[tid >> 6] = mloc;
    __syncthreads();
    const float M = fmaxf(sRed[0], sRed[1]);
    const float Mu = M == kNegInf ? 0.f : M;
    __syncthreads();
    // w_k and L = sum_k w_k l_k
    float lloc = 0.f;
    for (int k = tid; k < K; k += kCombineThreads) {
        const float w = fast_exp2(sW[k] - Mu);
        sW[k] = w;
        lloc += w * p.ws[(int64_t)sRow[k] * stride + 1];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) lloc += __shfl_xor(lloc, o);
    if ((tid & 63) == 0) sRed[tid >> 6] = lloc;
    __syncthreads();
    const float L = sRed[0] + sRed[1];
    // acc_r = sum_k w_k acc_r,k
    if constexpr (R > 0) {
        if (ad >= 0 && tid < R) {
            float v = 0.f;
            for (int k = 0; k < K; ++k) v += sW[k] * p.ws[(int64_t)sRow[k] * stride + 2 + D + tid];
            sAccR[tid] = v;
        }
    }
    // acc[d] = sum_k w_k acc_k[d]
    float acc = 0.f;
    {
        const int dd = tid;
        int k = 0;
        for (; k + 4 <= K; k += 4) {
            const float a0 = p.ws[(int64_t)sRow[k] * stride + 2 + dd];
            const float a1 = p.ws[(int64_t)sRow[k + 1] * stride + 2 + dd];
            const float a2 = p.ws[(int64_t)sRow[k + 2] * stride + 2 + dd];
            const float a3 = p.ws[(int64_t)sRow[k + 3] * stride + 2 + dd];
            acc += sW[k] * a0 + sW[k + 1] * a1 + sW[k + 2] * a2 + sW[k + 3] * a3;
        }
        for (; k < K; ++k) acc += sW[k] * p.ws[(int64_t)sRow[k] * stride + 2 + dd];
    }
    if constexpr (R > 0) {
        __syncthreads();
        if (ad >= 0) {
            const uint16_t *bv = p.lora_b + ((int64_t)ad * 2 + 1) * R * p.hkv * D + (int64_t)h * D + tid;
#pragma unroll 8
            for (int rho = 0; rho < R; ++rho) acc += sAccR[rho] * bf16_to_f32(bv[(int64_t)rho * p.hkv * D]);
        }
    }
    const float o = L > 0.f ? acc / L : 0.f;
    typedef __bf16 bf1;
    p.out[((int64_t)a * hq + j) * D + tid] = __builtin_bit_cast(uint16_t, (bf1)o);
}

template <int R, int G, bool ROPE>
hipError_t launch_decode(const DecodeArgs &da, int n_blocks, int n_agents, hipStream_t st, void *const *ev) {
    hipError_t e;
    if (ev && (e = hipEventRecord(static_cast<hipEvent_t>(ev[0]), st)) != hipSuccess) return e;
    hipLaunchKernelGGL((decode_split_kernel<R, G, ROPE>), dim3(n_blocks), dim3(256), 0, st, da);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev && (e = hipEventRecord(static_cast<hipEvent_t>(ev[1]), st)) != hipSuccess) return e;
    hipLaunchKernelGGL((decode_combine_kernel<R, G>), dim3(n_agents * da.hq), dim3(kCombineThreads), 0, st, da);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev && (e = hipEventRecord(static_cast<hipEvent_t>(ev[2]), st)) != hipSuccess) return e;
    return hipSuccess;
}

template <int R, int G>
hipError_t dispatch_rope(bool rope, const DecodeArgs &da, int nb, int na, hipStream_t st, void *const *ev) {
    if constexpr (R == 0) {
        return launch_decode<0, G, false>(da, nb, na, st, ev);
    } else {
        return rope ? launch_decode<R, G, true>(da, nb, na, st, ev) : launch_decode<R, G, false>(da, nb, na, st, ev);
    }
}

template <int G>
hipError_t dispatch_rank(int r, bool rope, const DecodeArgs &da, int nb, int na, hipStream_t st, void *const *ev) {
    switch (r) {
    case 0: return dispatch_rope<0, G>(rope, da, nb, na, st, ev);
    case 8: return dispatch_rope<8, G>(rope, da, nb, na, st, ev);
    case 16: return dispatch_rope<16, G>(rope, da, nb, na, st, ev);
    case 32: return dispatch_rope<32, G>(rope, da, nb, na, st, ev);
    case 64: return dispatch_rope<64, G>(rope, da, nb, na, st, ev);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

namespace fkv {
fkv_status validate_attn_common(const fkv_attn_args *a, const char *who);
int64_t plan_max_pages(const fkv_plan *plan);
}  // namespace fkv

extern "C" fkv_status fkv_residual_attention_decode(const fkv_attn_args *a, const fkv_plan *plan, void *stream) {
    fkv::clear_error();
    fkv_status st = fkv::validate_attn_common(a, "fkv_residual_attention_decode");
    if (st != FKV_OK) return st;
    if (!plan || !a->plan || !a->workspace)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan (host and device copy) and workspace are required");
    const auto &w = plan->words;
    const int g = a->hq / a->hkv;
    if (plan->n_agents != a->n_agents || plan->hkv != a->hkv || plan->g != g)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: plan was built for other n_agents / heads");
    fkv_plan_info info;
    fkv_decode_plan_info(plan, a->d, a->r, &info);
    if ((int64_t)a->workspace_bytes < info.workspace_bytes)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: workspace too small");
    if (a->rope_cos && (int64_t)a->rope_max_pos < fkv::plan_max_pages(plan) * a->page_size)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: RoPE table shorter than the longest sequence");
    if (g != 4 && g != 8)
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_residual_attention_decode: query heads per KV head must be 4 or 8");
    if (a->rope_cos && a->r > 0 && w[fkv::H_MAX_ITEM_AGENTS] > 256 / a->r)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_decode: with RoPE the plan may hold at most 256 / r "
                                          "agents per work item (fkv_decode_plan_default_agents)");
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
    da.ws = static_cast<float *>(a->workspace);
    da.out = static_cast<uint16_t *>(a->out);
    da.hq = a->hq;
    da.hkv = a->hkv;
    da.max_pages = a->max_pages;
    da.ws_stride = (a->d + a->r + 2 + 3) / 4 * 4;
    da.scale_log2 = a->scale * 1.4426950408889634f;
    const int nb = w[fkv::H_N_BLOCKS];
    hipStream_t hs = static_cast<hipStream_t>(stream);
    const bool rope = a->rope_cos != nullptr && a->r > 0;
    hipError_t e = g == 4 ? dispatch_rank<4>(a->r, rope, da, nb, a->n_agents, hs, a->timing_events)
                          : dispatch_rank<8>(a->r, rope, da, nb, a->n_agents, hs, a->timing_events);
    if (e != hipSuccess)
        return fkv::fail(FKV_ERR_HIP, std::string("fkv_residual_attention_decode: launch failed: ") + hipGetErrorString(e));
    return FKV_OK;
}
