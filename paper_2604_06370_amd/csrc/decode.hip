// ResidualAttention decode for gfx950 (Section 5.3, Algorithm 1).
//
// One workgroup = one (work item, KV head h).  A work item is a page range of a
// segment and up to 16/g agents that share its base pages, so the 16 query rows
// of the workgroup are (agent slot, query head of h).  Four waves stride over the
// item's pages, one 16-token page per wave-step, and each keeps its own online
// softmax state; the waves are merged through LDS at the end and one partial
// (m, l, acc, acc_r) per row goes to the workspace.  A second kernel merges the
// partials of every agent (log-sum-exp combine) and applies Stage 3.
//
// Per page and wave (all products are MFMA, fp32 accumulate):
//   S^T  = K_base . Q^T                               16x16x32, shared by all rows
//   residual key term, per agent slot s with an adapter:
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

__device__ __forceinline__ int hkv_of(const DecodeArgs &p) { return p.hkv; }

template <int R>
struct RankTiles {
    static constexpr int value = R == 0 ? 0 : (R + 15) / 16;
};

template <int R, int G, bool ROPE>
struct SplitShape {
    static constexpr int AG = ROWS / G;                     // agent slots per item
    static constexpr int RT = RankTiles<R>::value;          // 16-wide rank tiles
    static constexpr int MERGE_FLOATS = WAVES * ((8 + RT) * 64 * 4 + 2 * ROWS);
    static constexpr int STAGE_HALFS = ROPE ? AG * R * D : 0;         // B_K slices, row-major
    static constexpr int BKT_WORDS = ROPE ? AG * RT * 8 * 64 * 2 : 0;  // B_K^T fragments (u32)
    static constexpr int UNION_BYTES = (MERGE_FLOATS * 4 > STAGE_HALFS * 2) ? MERGE_FLOATS * 4 : STAGE_HALFS * 2;
    static constexpr int TABLE_WORDS = (1 + (R > 0 ? AG : 0)) * kMaxPagesPerItem;  // block-table entries
    static constexpr int LDS_BYTES = UNION_BYTES + BKT_WORDS * 4 + TABLE_WORDS * 4;
};

template <int R, int G, bool ROPE>
__global__ __launch_bounds__(256, ROPE ? 1 : 2) void decode_split_kernel(DecodeArgs p) {
    using S = SplitShape<R, G, ROPE>;
    constexpr int AG = S::AG;
    constexpr int RT = S::RT;
    __shared__ __attribute__((aligned(16))) unsigned char lds[S::LDS_BYTES];
    float *lds_f = reinterpret_cast<float *>(lds);
    uint32_t *lds_bkt = reinterpret_cast<uint32_t *>(lds + S::UNION_BYTES);

    const int32_t *plan = p.plan;
    const int blk = plan[plan[fkv::H_OFF_BLOCKS] + blockIdx.x];
    if (blk < 0) return;
    const int hkv = p.hkv;
    const int item = blk / hkv;
    const int h = blk - item * hkv;
    const int32_t *rec = plan + plan[fkv::H_OFF_ITEMS] + item * fkv::kItemWords;
    const int pg0 = rec[0], pg1 = rec[1], leader = rec[2], nag = rec[3];

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int my_slot = col / G;
    const bool row_active = my_slot < nag;
    const int my_agent = row_active ? rec[4 + my_slot] : 0;
    const int my_len = row_active ? p.seq_lens[my_agent] : 0;
    const int qh = h * G + (col % G);

    int slot_agent[AG], slot_ad[AG], slot_len[AG];
    int max_len = 0;
#pragma unroll
    for (int s = 0; s < AG; ++s) {
        slot_agent[s] = s < nag ? rec[4 + s] : 0;
        slot_ad[s] = (s < nag && R > 0) ? p.adapter_idx[slot_agent[s]] : -1;
        slot_len[s] = s < nag ? p.seq_lens[slot_agent[s]] : 0;
        max_len = max_len > slot_len[s] ? max_len : slot_len[s];
    }

    // Q^T as the B operand of the 16x16x32 products.  The head-dim index of slot j in
    // k-step kk is 32kk + 16(j/4) + 4grp + j%4 for this lane group: the same order in
    // which a rebuilt key tile leaves the 16x16x16 accumulators, so base keys, rebuilt
    // keys and queries all use one permuted order.
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
    u32x2 wf[RT > 0 ? RT : 1];   // RoPE off: (B_K q) for this lane's row, bf16, B operand of 16x16x16
    if constexpr (R > 0 && !ROPE) {
        f32x4 wacc[RT];
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
                if (my_slot == s) wacc[t] = acc;
            }
        }
#pragma unroll
        for (int t = 0; t < RT; ++t) wf[t] = pack4(wacc[t]);
    }
    if constexpr (ROPE) {
        // stage B_K[ad][0..R)[h*D .. h*D+D) of every slot in LDS (row-major, coalesced) ...
        uint16_t *stage = reinterpret_cast<uint16_t *>(lds);
        for (int idx = threadIdx.x; idx < AG * R * (D / 8); idx += 256) {
            const int s = idx / (R * (D / 8));
            const int rem = idx - s * (R * (D / 8));
            const int rho = rem / (D / 8), c8 = rem - rho * (D / 8);
            u32x4 v = {0, 0, 0, 0};
            if (slot_ad[s] >= 0)
                v = ldg128(p.lora_b + (int64_t)slot_ad[s] * 2 * R * n + (int64_t)rho * n + (int64_t)h * D + 8 * c8);
            *reinterpret_cast<u32x4 *>(stage + (s * R + rho) * D + 8 * c8) = v;
        }
        __syncthreads();
        // ... and re-lay it as B_K^T fragments: lane holds B_K[16t + 4grp + i][16mt + col].
        for (int idx = threadIdx.x; idx < AG * RT * 8 * 64; idx += 256) {
            const int ln = idx & 63;
            const int rest = idx >> 6;  // (s*RT + t)*8 + mt
            const int mt = rest & 7, st = rest >> 3;
            const int s = st / RT, t = st - s * RT;
            const int c = ln & 15, gg = ln >> 4;
            uint32_t w[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int r0 = 16 * t + 4 * gg + 2 * j;
                const uint16_t lo = r0 < R ? stage[(s * R + r0) * D + 16 * mt + c] : (uint16_t)0;
                const uint16_t hi = r0 + 1 < R ? stage[(s * R + r0 + 1) * D + 16 * mt + c] : (uint16_t)0;
                w[j] = (uint32_t)lo | ((uint32_t)hi << 16);
            }
            lds_bkt[idx * 2 + 0] = w[0];
            lds_bkt[idx * 2 + 1] = w[1];
        }
    }
    // block-table entries of the item's pages: one round trip for the whole item
    int32_t *s_tab = reinterpret_cast<int32_t *>(lds + S::UNION_BYTES + S::BKT_WORDS * 4);
    const int npg = pg1 - pg0;
    for (int i = threadIdx.x; i < npg; i += 256) s_tab[i] = p.base_bt[(int64_t)leader * p.max_pages + pg0 + i];
    if constexpr (R > 0) {
#pragma unroll
        for (int s = 0; s < AG; ++s)
            for (int i = threadIdx.x; i < npg; i += 256)
                s_tab[(1 + s) * kMaxPagesPerItem + i] =
                    slot_ad[s] >= 0 ? p.res_bt[(int64_t)slot_agent[s] * p.max_pages + pg0 + i] : 0;
    }
    __syncthreads();

    // ---- main loop: this wave's pages, next page's loads in flight during compute ----
    f32x4 oacc[8];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) oacc[mt] = f32x4{0, 0, 0, 0};
    f32x4 racc[RT > 0 ? RT : 1];
#pragma unroll
    for (int t = 0; t < (RT > 0 ? RT : 1); ++t) racc[t] = f32x4{0, 0, 0, 0};
    float m_run = kNegInf, l_run = 0.f;

    const int64_t kv_block = (int64_t)PS * D;   // halfs per (page, K|V, head) block
    struct Frag {
        f32x4 cs[ROPE ? 4 : 1], sn[ROPE ? 4 : 1];
        u32x4 kf[4];
        u32x2 vf[8];
        u32x2 ck[AG][RT > 0 ? RT : 1];
        u32x2 cv[AG][RT > 0 ? RT : 1];
    };
    // Every load below is issued unconditionally and in a fixed order, so the compiler
    // can count them: a prefetch of the next page then stays in flight while the
    // current page computes.  Lanes or slots that have no data read a valid address
    // and their values are zeroed or ignored.
    auto load = [&](int pg, Frag &f) {
        const int li = pg - pg0;
        const int tok0 = pg * PS;
        if constexpr (ROPE) {  // issued first: they are consumed first
            const float *cr = p.rope_cos + (int64_t)pg * (PS * D / 2) + lane * 4;
            const float *sr = p.rope_sin + (int64_t)pg * (PS * D / 2) + lane * 4;
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                f.cs[mt] = *reinterpret_cast<const f32x4 *>(cr + 256 * mt);
                f.sn[mt] = *reinterpret_cast<const f32x4 *>(sr + 256 * mt);
            }
        }
        // K and V blocks are stored in fragment order: one 16-byte load per lane each
        const int bpage = uniform(s_tab[li]);
        const uint16_t *kblk = p.base_kv + ((int64_t)bpage * 2 * hkv + h) * kv_block;
        const uint16_t *vblk = kblk + (int64_t)hkv * kv_block;
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
            for (int s = 0; s < AG; ++s) {
                const int rpage = uniform(s_tab[(1 + s) * kMaxPagesPerItem + li]);
                const uint16_t *rb = p.res_kv + (int64_t)rpage * res_page_halfs;
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    const int rho = 16 * t + col;
                    const int rk = 16 * t + 4 * grp;
                    const u32x2 cv = ldg64(rb + PS * R + (rho < R ? rho : R - 1) * PS + 4 * grp);
                    const u32x2 ck = ldg64(rb + col * R + (rk < R ? rk : R - 4));
                    f.cv[s][t] = rho < R ? cv : u32x2{0, 0};
                    f.ck[s][t] = rk < R ? ck : u32x2{0, 0};
                }
            }
        }
    };
    auto mask4 = [&](u32x2 v, int vis) {  // zero tokens 4grp+i >= vis of a [.][tok] fragment
        if (4 * grp + 0 >= vis) v.x &= 0xffff0000u;
        if (4 * grp + 1 >= vis) v.x &= 0x0000ffffu;
        if (4 * grp + 2 >= vis) v.y &= 0xffff0000u;
        if (4 * grp + 3 >= vis) v.y &= 0x0000ffffu;
        return v;
    };
    auto compute = [&](Frag &f, int pg) {
        const int tok0 = pg * PS;
        // tokens past every agent's end are zeroed in V (they may hold any bits)
        const int vis = max_len - tok0;
        if (vis < PS) {
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) f.vf[mt] = mask4(f.vf[mt], vis);
        }
        // S^T = K_base Q^T
        f32x4 sacc = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) sacc = mfma32(f.kf[kk], qf[kk], sacc);
        if constexpr (R > 0) {
#pragma unroll
            for (int s = 0; s < AG; ++s) {
                if (slot_ad[s] < 0) continue;
                const int svis = slot_len[s] - tok0;
                if (svis < PS) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) f.cv[s][t] = mask4(f.cv[s][t], svis);
                }
                if constexpr (!ROPE) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const u32x2 b = my_slot == s ? wf[t] : u32x2{0, 0};
                        sacc = mfma16(f.ck[s][t], b, sacc);
                    }
                } else {
                    // Stage 1: U^T = B_K^T C_K^T (rows d, columns tokens), deferred RoPE, then
                    // S^T += K_lora Q_s^T with the rebuilt tile as the 16x16x32 A operand.
                    f32x4 u[8];
#pragma unroll
                    for (int mt = 0; mt < 8; ++mt) {
                        u[mt] = f32x4{0, 0, 0, 0};
#pragma unroll
                        for (int t = 0; t < RT; ++t) {
                            const u32x2 a = *reinterpret_cast<const u32x2 *>(
                                lds_bkt + ((((s * RT + t) * 8 + mt) * 64) + lane) * 2);
                            u[mt] = mfma16(a, f.ck[s][t], u[mt]);
                        }
                    }
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float x = u[mt][i], y = u[mt + 4][i];
                            u[mt][i] = x * f.cs[mt][i] - y * f.sn[mt][i];
                            u[mt + 4][i] = y * f.cs[mt][i] + x * f.sn[mt][i];
                        }
                    }
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        const u32x2 lo = pack4(u[2 * kk]), hi = pack4(u[2 * kk + 1]);
                        const u32x4 b = my_slot == s ? qf[kk] : u32x4{0, 0, 0, 0};
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
            sv[i] = (row_active && tok < my_len) ? sacc[i] * p.scale_log2 : kNegInf;
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
            oacc[mt] = mfma16(f.vf[mt], pf, oacc[mt]);
        }
        if constexpr (R > 0) {
#pragma unroll
            for (int t = 0; t < RT; ++t) racc[t] *= alpha;
#pragma unroll
            for (int s = 0; s < AG; ++s) {
                if (slot_ad[s] < 0) continue;
                const u32x2 pm = my_slot == s ? pf : u32x2{0, 0};
#pragma unroll
                for (int t = 0; t < RT; ++t) racc[t] = mfma16(f.cv[s][t], pm, racc[t]);
            }
        }
    };

    // Two register buffers: the next page (clamped to this wave's last page, so the
    // final prefetch re-reads a page that is already in cache) loads while the
    // current one computes.
    Frag fa, fb;
    int pg = pg0 + wave;
    if (pg < pg1) {
        const int last = pg + (pg1 - 1 - pg) / WAVES * WAVES;
        load(pg, fa);
        for (;;) {
            load(pg + WAVES <= last ? pg + WAVES : last, fb);
            compute(fa, pg);
            pg += WAVES;
            if (pg > last) break;
            load(pg + WAVES <= last ? pg + WAVES : last, fa);
            compute(fb, pg);
            pg += WAVES;
            if (pg > last) break;
        }
    }
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);

    // ---- merge the four waves and write one partial per row ----
    __syncthreads();  // LDS staging of the prologue is dead from here on
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
    float *wsb = p.ws + (int64_t)(item * hkv + h) * ROWS * p.ws_stride;
    for (int idx = threadIdx.x; idx < rows_used * rec_len; idx += 256) {
        const int r = idx / rec_len, k = idx - r * rec_len;
        float mw[WAVES], M = kNegInf;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            mw[w] = lds_m[w * ROWS + r];
            M = fmaxf(M, mw[w]);
        }
        const float Mu = M == kNegInf ? 0.f : M;
        float v = 0.f;
        if (k == 0) {
            v = M;
        } else if (k == 1) {
#pragma unroll
            for (int w = 0; w < WAVES; ++w) v += fast_exp2(mw[w] - Mu) * lds_l[w * ROWS + r];
        } else {
            const int e = k - 2;
            int tile, ln, i;
            if (e < D) {
                tile = e >> 4;
                ln = r + 16 * ((e & 15) >> 2);
                i = e & 3;
            } else {
                const int rho = e - D;
                tile = 8 + (rho >> 4);
                ln = r + 16 * ((rho & 15) >> 2);
                i = rho & 3;
            }
#pragma unroll
            for (int w = 0; w < WAVES; ++w)
                v += fast_exp2(mw[w] - Mu) * lds_f[w * TILES * 256 + (tile * 64 + ln) * 4 + i];
        }
        wsb[(int64_t)r * p.ws_stride + k] = v;
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
        const int row = slots[k0 + k] + h * ROWS + jj;
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
            const uint16_t *bv = p.lora_b + ((int64_t)ad * 2 + 1) * R * hkv_of(p) * D + (int64_t)h * D + tid;
#pragma unroll 8
            for (int rho = 0; rho < R; ++rho) acc += sAccR[rho] * bf16_to_f32(bv[(int64_t)rho * hkv_of(p) * D]);
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
