// ResidualAttention chunked prefill for gfx950 (Section 6 prefill kernel,
// Algorithm 1 with a block of query rows).
//
// One workgroup = (agent a, KV head h, block of query tokens); its 128 rows are
// (query token, query head of h).  Every row of the block belongs to the same
// agent, so the agent's keys are rebuilt once per 64-key tile and shared by all
// rows through LDS:
//   wave w rebuilds page w of the tile:  U^T = B_K^T C_K^T  (MFMA),
//                                        K_lora = RoPE_p(U) (rotate-half, fp32),
//                                        K = K_base + K_lora -> bf16 -> LDS
//   then every wave, for its 32 rows:    S^T = K Q^T        (16x16x32 MFMA)
//                                        causal mask + online softmax
//                                        O^T   += V^T P^T   (16x16x32 MFMA)
//                                        acc_r^T += C_V^T P^T
// and at the end O = (O + acc_r . B_V[h]) / l (Eq. 4) is written in bf16.
//
// The contraction index of the 16x16x32 products is permuted so that the
// accumulator tiles of the 16x16x16 rebuild feed them without shuffles: in
// k-step kk, slot j of lane group grp is head-dim index 32kk + 16(j/4) + 4grp +
// j%4 for the key products, and key 16(j/4) + 4grp + j%4 of a 32-key half for the
// value products.  Queries and values are loaded in the same order.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <string>

#include "internal.hpp"
#include "lds_dma.hpp"
#include "mfma.hpp"

using namespace fkvk;

namespace {

constexpr int D = 128;
constexpr int PS = 16;
constexpr int WAVES = 4;
constexpr int ROWS_PER_WAVE = 32;          // two 16-row tiles
constexpr int ROWS_PER_WG = WAVES * ROWS_PER_WAVE;
constexpr int TILE_KEYS = 64;              // four pages, one per wave
constexpr int kXcds = 8;
constexpr float kNegInf = -INFINITY;

struct PrefillArgs {
    const uint16_t *q, *base_kv, *res_kv, *lora_b;
    const int32_t *adapter_idx, *base_bt, *res_bt, *seq_lens, *q_indptr;
    const float *rope_cos, *rope_sin;
    uint16_t *out;
    int32_t n_agents, hq, hkv, max_pages, blocks_per_agent_head;
    float scale_log2;
};


// Rows of an agent's chunk that its query blocks do not reach (a max_q_per_agent below the
// agent's row count) are written as NaN by the agent's last block, so the shortfall shows in
// the output instead of leaving stale memory there.
__device__ __forceinline__ void poison_unreached_rows(const PrefillArgs &p, int q0, int nq, int h, int g, int reach) {
    const uint32_t nan2 = 0x7fc07fc0u;  // two bf16 quiet NaNs
    for (int64_t i = threadIdx.x; i < (int64_t)(nq - reach) * g * 32; i += blockDim.x) {
        const int64_t row = i / 32, c = i % 32;
        const int tok = reach + (int)(row / g), j = (int)(row % g);
        uint16_t *orow = p.out + ((int64_t)(q0 + tok) * p.hq + h * g + j) * 128;
        *reinterpret_cast<u32x2 *>(orow + 4 * c) = u32x2{nan2, nan2};
    }
}

template <int R, int G, bool ROPE>
struct PrefillShape {
    static constexpr int RT = R == 0 ? 0 : (R + 15) / 16;
    static constexpr int TOK_PER_WG = ROWS_PER_WG / G;
    static constexpr int RES_PAGE = RT * 512;                  // residual page (fragment order)
    static constexpr int SK_BYTES = 4 * 4 * 64 * 16;          // [page][kk][lane] 16 B
    static constexpr int SV_BYTES = 4 * PS * D * 2;             // [page][d][16] bf16
    static constexpr int SCV_BYTES = R > 0 ? 4 * R * PS * 2 : 16;  // [page][rho][16] bf16
    static constexpr int SBK_BYTES = (R > 0 && ROPE) ? RT * 8 * 64 * 8 : 16;  // B_K^T fragments
    static constexpr int SBV_BYTES = R > 0 ? R * D * 4 : 16;    // B_V[h] slice, fp32
    static constexpr int SACC_BYTES = R > 0 ? ROWS_PER_WG * R * 4 : 16;  // acc_r rows for the epilogue
    static constexpr int EPI_BYTES = SBV_BYTES + SACC_BYTES;
    static constexpr int MAIN_BYTES = SK_BYTES + SV_BYTES + SCV_BYTES;
    static constexpr int LDS_BYTES = (MAIN_BYTES > EPI_BYTES ? MAIN_BYTES : EPI_BYTES) + SBK_BYTES;
};

template <int R, int G, bool ROPE>
__global__ __launch_bounds__(256, 2) void prefill_kernel(PrefillArgs p) {
    using S = PrefillShape<R, G, ROPE>;
    constexpr int RT = S::RT;
    constexpr int TPW = S::TOK_PER_WG;
    __shared__ __attribute__((aligned(16))) unsigned char lds[S::LDS_BYTES];
    u32x4 *sK = reinterpret_cast<u32x4 *>(lds);
    uint16_t *sV = reinterpret_cast<uint16_t *>(lds + S::SK_BYTES);
    uint16_t *sCV = reinterpret_cast<uint16_t *>(lds + S::SK_BYTES + S::SV_BYTES);
    u32x2 *sBK = reinterpret_cast<u32x2 *>(lds + (S::MAIN_BYTES > S::EPI_BYTES ? S::MAIN_BYTES : S::EPI_BYTES));
    float *sBV = reinterpret_cast<float *>(lds);
    float *sAcc = reinterpret_cast<float *>(lds + S::SBV_BYTES);

    // Consecutive workgroup ids go round-robin to the 8 XCDs: keep all query blocks of one
    // (agent, KV head) on one XCD so the key/value tiles they all stream hit that XCD's L2.
    const int hkv = p.hkv;
    const int bpa = p.blocks_per_agent_head;
    const int xcd = blockIdx.x % kXcds, local = blockIdx.x / kXcds;
    const int pair = (local / bpa) * kXcds + xcd;
    const int qb = local - (local / bpa) * bpa;
    if (pair >= p.n_agents * hkv) return;
    const int a = pair / hkv;
    const int h = pair - a * hkv;
    const int q0 = p.q_indptr[a], nq = p.q_indptr[a + 1] - q0;
    const int tok_begin = qb * TPW;
    if (qb == bpa - 1 && nq > bpa * TPW) poison_unreached_rows(p, q0, nq, h, G, bpa * TPW);
    if (tok_begin >= nq) return;
    const int L = p.seq_lens[a];
    const int P0 = L - nq;  // position of the chunk's first query
    const int ad = R > 0 ? p.adapter_idx[a] : -1;

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int64_t n = (int64_t)hkv * D;

    // rows of this lane in the two 16-row tiles of the wave
    int row_tok[2], row_pos[2];
    bool row_ok[2];
    u32x4 qf[2][4];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const int r = wave * ROWS_PER_WAVE + nt * 16 + col;
        const int t = tok_begin + r / G;
        const int jj = r % G;
        row_ok[nt] = t < nq;
        row_tok[nt] = t;
        row_pos[nt] = P0 + t;
        const uint16_t *qr = p.q + ((int64_t)(q0 + (row_ok[nt] ? t : 0)) * p.hq + h * G + jj) * D;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            u32x4 v = {0, 0, 0, 0};
            if (row_ok[nt]) {
                const u32x2 lo = ldg64(qr + 32 * kk + 4 * grp);
                const u32x2 hi = ldg64(qr + 32 * kk + 16 + 4 * grp);
                v = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
            qf[nt][kk] = v;
        }
    }

    // B_K^T fragments for the rebuild: lane holds B_K[16t + 4grp + i][h*D + 16mt + col]
    if constexpr (R > 0 && ROPE) {
        if (ad >= 0) {
            const uint16_t *bk = p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)h * D;
            for (int idx = threadIdx.x; idx < RT * 8 * 64; idx += 256) {
                const int ln = idx & 63, rest = idx >> 6;
                const int mt = rest & 7, t = rest >> 3;
                const int c = ln & 15, gg = ln >> 4;
                uint32_t w[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int r0 = 16 * t + 4 * gg + 2 * j;
                    const uint16_t lo = r0 < R ? bk[(int64_t)r0 * n + 16 * mt + c] : (uint16_t)0;
                    const uint16_t hi = r0 + 1 < R ? bk[(int64_t)(r0 + 1) * n + 16 * mt + c] : (uint16_t)0;
                    w[j] = (uint32_t)lo | ((uint32_t)hi << 16);
                }
                sBK[idx] = u32x2{w[0], w[1]};
            }
        }
    }
    // RoPE off: the residual key term of row j is (B_K q_j) . c_p; fold it as an extra
    // contraction over the rank: S^T += C_K (B_K q)^T.
    u32x2 wq[2][RT > 0 ? RT : 1];
    if constexpr (R > 0 && !ROPE) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int t = 0; t < RT; ++t) {
                f32x4 acc = {0, 0, 0, 0};
                if (ad >= 0) {
                    const int rho = 16 * t + col;
                    const uint16_t *bk = p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)rho * n + (int64_t)h * D;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        u32x4 av = {0, 0, 0, 0};
                        if (rho < R) {
                            const u32x2 lo = ldg64(bk + 32 * kk + 4 * grp);
                            const u32x2 hi = ldg64(bk + 32 * kk + 16 + 4 * grp);
                            av = u32x4{lo.x, lo.y, hi.x, hi.y};
                        }
                        acc = mfma32(av, qf[nt][kk], acc);  // W^T[rho][row]
                    }
                }
                wq[nt][t] = pack4(acc);
            }
    }
    __syncthreads();

    f32x4 oacc[8][2];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) oacc[mt][0] = oacc[mt][1] = f32x4{0, 0, 0, 0};
    f32x4 racc[RT > 0 ? RT : 1][2];
#pragma unroll
    for (int t = 0; t < (RT > 0 ? RT : 1); ++t) racc[t][0] = racc[t][1] = f32x4{0, 0, 0, 0};
    float m_run[2] = {kNegInf, kNegInf}, l_run[2] = {0.f, 0.f};

    const int n_pages = (L + PS - 1) / PS;
    const int last_pos = P0 + (tok_begin + TPW < nq ? tok_begin + TPW : nq) - 1;
    const int n_tiles = last_pos / TILE_KEYS + 1;
    const int32_t *btb = p.base_bt + (int64_t)a * p.max_pages;
    const int32_t *btr = R > 0 ? p.res_bt + (int64_t)a * p.max_pages : nullptr;
    const int64_t kv_block = (int64_t)PS * D;

    for (int tile = 0; tile < n_tiles; ++tile) {
        // ---- stage: wave w rebuilds page w of the tile into LDS ----
        {
            const int pg = tile * 4 + wave;
            const int tok0 = pg * PS;
            const bool have = pg < n_pages;
            const int bpage = have ? btb[pg] : 0;
            const uint16_t *kblk = p.base_kv + ((int64_t)bpage * 2 * hkv + h) * kv_block;
            const uint16_t *vblk = kblk + (int64_t)hkv * kv_block;
            const int vis = L - tok0;  // valid keys in this page
            // K_base, stored in the permuted 16x16x32 A layout: one 16-byte load per k-step
            f32x4 kacc[8];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const u32x4 kb = have ? ldg128(kblk + kk * 512 + lane * 8) : u32x4{0, 0, 0, 0};
                kacc[2 * kk] = f32x4{bf16_lo(kb.x), bf16_hi(kb.x), bf16_lo(kb.y), bf16_hi(kb.y)};
                kacc[2 * kk + 1] = f32x4{bf16_lo(kb.z), bf16_hi(kb.z), bf16_lo(kb.w), bf16_hi(kb.w)};
            }
            const uint16_t *rb = nullptr;
            if constexpr (R > 0) {
                if (ad >= 0 && have) rb = p.res_kv + (int64_t)btr[pg] * S::RES_PAGE;
            }
            if constexpr (R > 0 && ROPE) {
                if (rb) {
                    f32x4 u[8];
#pragma unroll
                    for (int mt = 0; mt < 8; ++mt) u[mt] = f32x4{0, 0, 0, 0};
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const u32x2 c = ldg64(rb + t * 512 + lane * 8);
                        const u32x2 ck = (16 * t + 4 * grp < R) ? c : u32x2{0, 0};
#pragma unroll
                        for (int mt = 0; mt < 8; ++mt) u[mt] = mfma16(sBK[(t * 8 + mt) * 64 + lane], ck, u[mt]);
                    }
                    const float *cr = p.rope_cos + (int64_t)pg * (PS * D / 2) + lane * 4;
                    const float *sr = p.rope_sin + (int64_t)pg * (PS * D / 2) + lane * 4;
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt) {
                        const f32x4 cs = *reinterpret_cast<const f32x4 *>(cr + 256 * mt);
                        const f32x4 sn = *reinterpret_cast<const f32x4 *>(sr + 256 * mt);
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float x = u[mt][i], y = u[mt + 4][i];
                            kacc[mt][i] += x * cs[i] - y * sn[i];
                            kacc[mt + 4][i] += y * cs[i] + x * sn[i];
                        }
                    }
                }
            }
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const u32x2 lo = pack4(kacc[2 * kk]), hi = pack4(kacc[2 * kk + 1]);
                sK[(wave * 4 + kk) * 64 + lane] = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
            // V page as stored ([d][16 keys]); keys past the sequence end are zeroed
            for (int e = lane; e < D * PS / 4; e += 64) {
                u32x2 v = have ? ldg64(vblk + 4 * e) : u32x2{0, 0};
                const int k0 = 4 * ((((4 * e) & 511) >> 3) >> 4);  // tokens k0..k0+3 (fragment order)
                if (k0 + 0 >= vis) v.x &= 0xffff0000u;
                if (k0 + 1 >= vis) v.x &= 0x0000ffffu;
                if (k0 + 2 >= vis) v.y &= 0xffff0000u;
                if (k0 + 3 >= vis) v.y &= 0x0000ffffu;
                *reinterpret_cast<u32x2 *>(sV + wave * D * PS + 4 * e) = v;
            }
            if constexpr (R > 0) {
                // C_V^T rows of the page: lane (c, g) of tile t holds C_V[4g .. 4g+3][16t + c]
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    const int rho = 16 * t + col;
                    u32x2 v = {0, 0};
                    if (rb) v = ldg64(rb + t * 512 + lane * 8 + 4);
                    const int k0 = 4 * grp;
                    if (k0 + 0 >= vis) v.x &= 0xffff0000u;
                    if (k0 + 1 >= vis) v.x &= 0x0000ffffu;
                    if (k0 + 2 >= vis) v.y &= 0xffff0000u;
                    if (k0 + 3 >= vis) v.y &= 0x0000ffffu;
                    if (rho < R) *reinterpret_cast<u32x2 *>(sCV + wave * R * PS + rho * PS + 4 * grp) = v;
                }
            }
        }
        __syncthreads();

        // ---- scores for the 64 keys of the tile, 2 row tiles ----
        f32x4 sacc[4][2];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            sacc[kt][0] = sacc[kt][1] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const u32x4 kf = sK[(kt * 4 + kk) * 64 + lane];
                sacc[kt][0] = mfma32(kf, qf[0][kk], sacc[kt][0]);
                sacc[kt][1] = mfma32(kf, qf[1][kk], sacc[kt][1]);
            }
        }
        if constexpr (R > 0 && !ROPE) {
            if (ad >= 0) {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt) {
                    const int pg = tile * 4 + kt;
                    if (pg >= n_pages) continue;
                    const uint16_t *rb = p.res_kv + (int64_t)btr[pg] * S::RES_PAGE;
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const u32x2 c = ldg64(rb + t * 512 + lane * 8);
                        const u32x2 ck = (16 * t + 4 * grp < R) ? c : u32x2{0, 0};
                        // zero-padded 16x16x32 form: the accumulator chain stays on one
                        // instruction form (see the decode kernel)
                        const u32x4 a = u32x4{ck.x, ck.y, 0u, 0u};
                        sacc[kt][0] = mfma32(a, u32x4{wq[0][t].x, wq[0][t].y, 0u, 0u}, sacc[kt][0]);
                        sacc[kt][1] = mfma32(a, u32x4{wq[1][t].x, wq[1][t].y, 0u, 0u}, sacc[kt][1]);
                    }
                }
            }
        }

        // ---- causal mask + online softmax (rows live in lanes) ----
        u32x2 pf[4][2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            float sv[4][4];
            float mx = kNegInf;
#pragma unroll
            for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int key = tile * TILE_KEYS + kt * PS + 4 * grp + i;
                    sv[kt][i] = (row_ok[nt] && key <= row_pos[nt]) ? sacc[kt][nt][i] * p.scale_log2 : kNegInf;
                    mx = fmaxf(mx, sv[kt][i]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run[nt], mx);
            const float m_use = m_new == kNegInf ? 0.f : m_new;
            const float alpha = fast_exp2(m_run[nt] - m_use);
            float ps = 0.f;
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                f32x4 pv;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[i] = fast_exp2(sv[kt][i] - m_use);
                    ps += pv[i];
                }
                pf[kt][nt] = pack4(pv);
            }
            l_run[nt] = l_run[nt] * alpha + ps;
            m_run[nt] = m_new;
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) oacc[mt][nt] *= alpha;
#pragma unroll
            for (int t = 0; t < RT; ++t) racc[t][nt] *= alpha;
        }

        // ---- O^T += V^T P^T and acc_r^T += C_V^T P^T over two 32-key halves ----
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const u32x4 pb0 = u32x4{pf[2 * half][0].x, pf[2 * half][0].y, pf[2 * half + 1][0].x, pf[2 * half + 1][0].y};
            const u32x4 pb1 = u32x4{pf[2 * half][1].x, pf[2 * half][1].y, pf[2 * half + 1][1].x, pf[2 * half + 1][1].y};
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) {
                const int voff = (mt >> 1) * 512 + lane * 8 + 4 * (mt & 1);
                const u32x2 lo = *reinterpret_cast<const u32x2 *>(sV + (2 * half) * D * PS + voff);
                const u32x2 hi = *reinterpret_cast<const u32x2 *>(sV + (2 * half + 1) * D * PS + voff);
                const u32x4 va = u32x4{lo.x, lo.y, hi.x, hi.y};
                oacc[mt][0] = mfma32(va, pb0, oacc[mt][0]);
                oacc[mt][1] = mfma32(va, pb1, oacc[mt][1]);
            }
            if constexpr (R > 0) {
                if (ad >= 0) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const int rho = 16 * t + col;
                        u32x4 ca = {0, 0, 0, 0};
                        if (rho < R) {
                            const u32x2 lo = *reinterpret_cast<const u32x2 *>(sCV + (2 * half) * R * PS + rho * PS + 4 * grp);
                            const u32x2 hi = *reinterpret_cast<const u32x2 *>(sCV + (2 * half + 1) * R * PS + rho * PS + 4 * grp);
                            ca = u32x4{lo.x, lo.y, hi.x, hi.y};
                        }
                        racc[t][0] = mfma32(ca, pb0, racc[t][0]);
                        racc[t][1] = mfma32(ca, pb1, racc[t][1]);
                    }
                }
            }
        }
        __syncthreads();
    }

    // ---- epilogue: O = (acc + acc_r . B_V[h]) / l ----
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        l_run[nt] += __shfl_xor(l_run[nt], 16);
        l_run[nt] += __shfl_xor(l_run[nt], 32);
    }
    if constexpr (R > 0) {
        if (ad >= 0) {
            const uint16_t *bv = p.lora_b + ((int64_t)ad * 2 + 1) * R * n + (int64_t)h * D;
            for (int e = threadIdx.x; e < R * D; e += 256) sBV[e] = bf16_to_f32(bv[(int64_t)(e / D) * n + (e % D)]);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int rho = 16 * t + 4 * grp + i;
                        if (rho < R) sAcc[(wave * ROWS_PER_WAVE + nt * 16 + col) * R + rho] = racc[t][nt][i];
                    }
            __syncthreads();
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                const float *ar = sAcc + (wave * ROWS_PER_WAVE + nt * 16 + col) * R;
                for (int rho = 0; rho < R; ++rho) {
                    const float c = ar[rho];
#pragma unroll
                    for (int mt = 0; mt < 8; ++mt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) oacc[mt][nt][i] += c * sBV[rho * D + 16 * mt + 4 * grp + i];
                }
            }
        }
    }
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        if (!row_ok[nt]) continue;
        const int r = wave * ROWS_PER_WAVE + nt * 16 + col;
        const float inv = l_run[nt] > 0.f ? 1.f / l_run[nt] : 0.f;
        uint16_t *orow = p.out + ((int64_t)(q0 + row_tok[nt]) * p.hq + h * G + r % G) * D;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
            f32x4 o = oacc[mt][nt] * inv;
            *reinterpret_cast<u32x2 *>(orow + 16 * mt + 4 * grp) = pack4(o);
        }
    }
}

// ---------------------------------------------------------------------------
// Streaming kernel.  A workgroup of eight waves holds 256 query rows (twice the rows per
// key tile of the kernel above, so half the tile traffic per product), and 64-key tiles
// stream through a ring of LDS buffers by direct memory-to-LDS copies: wave w < 4 copies
// the K block (and, with an adapter, the rCache page) of page w of a tile, wave 4 + w its
// V block.  One barrier per tile hands a buffer over: every wave has waited (by count)
// for its copies of the tile, and every wave has finished reading the buffer that the
// copies issued after the barrier overwrite.
//  - RoPE off: the key residual folds into the queries (S^T += C_K (B_K q)^T), so the
//    stored blocks are used as they are; three buffers, copies two tiles ahead.
//  - RoPE on (rank up to 32): a tile also carries the table rows of its positions; two
//    buffers, copies one tile ahead.  After a tile has landed each wave rebuilds a quarter
//    of one page's keys in place (U^T = B_K^T C_K^T on the matrix cores, rotated, added to
//    K_base) and a second barrier publishes the rebuilt tile.
//
// Buffer layout (bytes): K blocks [page][4 KB], V blocks [page][4 KB], rCache pages as
// [rank tile][page][1 KB] (four pages of one rank tile are 1 KB apart).  All are stored
// verbatim: the K block's 16 bytes at k-step kk, lane l are the A fragment of the score
// product, the V block's 16 bytes at chunk q2, lane l hold dims 32q2 + col (.xy) and
// 32q2 + 16 + col (.zw) of tokens 4grp .. 4grp + 3, and the rCache fragment holds C_K
// (.xy) and C_V (.zw) of the lane.
constexpr float kLazyRescale = 8.f;

constexpr int kStreamWaves = 8;
// RoPE on, the streaming kernel serves ranks up to 32 (its LDS ring and B_K^T fragments
// fit one workgroup's LDS); rank 64 takes the kernel above
constexpr bool stream_rope(int r) { return r <= 32; }
constexpr int kStreamRows = kStreamWaves * ROWS_PER_WAVE;

template <int R, bool ROPE>
struct StreamShape {
    static constexpr int NBUF = ROPE ? 2 : 3;  // ring buffers (copies NBUF - 1 tiles ahead)
    static constexpr int RT = R == 0 ? 0 : (R + 15) / 16;
    static constexpr int SBK_BYTES = ROPE ? RT * 8 * 64 * 8 : 0;  // B_K^T fragments (RoPE on)
    static constexpr int K_OFF = 0;
    static constexpr int V_OFF = 4 * 4096;
    static constexpr int C_OFF = 8 * 4096;
    // RoPE on: table rows [page][half][cos m, cos m + 1, sin m, sin m + 1][1 KB], m = 2 half
    static constexpr int T_OFF = C_OFF + 4 * RT * 1024;
    static constexpr int BUF_BYTES = T_OFF + (ROPE ? 4 * 2 * 4096 : 0);
    static constexpr int SBV_BYTES = R > 0 ? R * D * 4 : 16;
    static constexpr int SACC_BYTES = R > 0 ? kStreamRows * R * 4 : 16;
    static constexpr int EPI_BYTES = SBV_BYTES + SACC_BYTES;
    static constexpr int RING_BYTES = NBUF * BUF_BYTES;
    static constexpr int MAIN_BYTES = RING_BYTES > EPI_BYTES ? RING_BYTES : EPI_BYTES;
    static constexpr int LDS_BYTES = MAIN_BYTES + SBK_BYTES;
    static_assert(LDS_BYTES <= 160 * 1024, "LDS of one workgroup");
};

template <int R, int G, bool ROPE>
__global__ __launch_bounds__(64 * kStreamWaves, 1) void prefill_stream_kernel(PrefillArgs p) {
    using S = StreamShape<R, ROPE>;
    constexpr int RT = S::RT;
    constexpr int RTX = RT > 0 ? RT : 1;
    constexpr int TPW = kStreamRows / G;
    __shared__ __attribute__((aligned(16))) u32x4 lds[S::LDS_BYTES / 16];
    float *sBV = reinterpret_cast<float *>(lds);
    float *sAcc = reinterpret_cast<float *>(reinterpret_cast<unsigned char *>(lds) + S::SBV_BYTES);
    const u32x2 *sBK = reinterpret_cast<const u32x2 *>(reinterpret_cast<unsigned char *>(lds) + S::MAIN_BYTES);

    const int hkv = p.hkv;
    const int bpa = p.blocks_per_agent_head;
    const int xcd = blockIdx.x % kXcds, local = blockIdx.x / kXcds;
    const int pair = (local / bpa) * kXcds + xcd;
    const int qb = local - (local / bpa) * bpa;
    if (pair >= p.n_agents * hkv) return;
    const int a = pair / hkv;
    const int h = pair - a * hkv;
    const int q0 = p.q_indptr[a], nq = p.q_indptr[a + 1] - q0;
    const int tok_begin = qb * TPW;
    if (qb == bpa - 1 && nq > bpa * TPW) poison_unreached_rows(p, q0, nq, h, G, bpa * TPW);
    if (tok_begin >= nq) return;
    const int L = p.seq_lens[a];
    const int P0 = L - nq;  // position of the chunk's first query
    const int ad = R > 0 ? p.adapter_idx[a] : -1;

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int64_t n = (int64_t)hkv * D;

    const int n_pages = (L + PS - 1) / PS;
    const int last_pos = P0 + (tok_begin + TPW < nq ? tok_begin + TPW : nq) - 1;
    const int n_tiles = last_pos / TILE_KEYS + 1;
    const int32_t *btb = p.base_bt + (int64_t)a * p.max_pages;
    const int32_t *btr = R > 0 ? p.res_bt + (int64_t)a * p.max_pages : nullptr;
    const bool use_res = R > 0 && ad >= 0;

    // This wave copies page pw of every tile: its K block and rCache page (waves 0..3) or
    // its V block (waves 4..7).
    const int pw = wave & 3;
    const int half = wave >> 2;
    const bool kwave = wave < 4;
    const bool res_copy = use_res && kwave;
    // Page ids of this wave's pages (page 4 t + pw of tile t), 64 tiles per register:
    // lane i holds the id for tile 64 c + i of chunk c (pages past the sequence repeat its
    // last page, so every copy reads a real page; their keys are masked).
    auto load_ids = [&](int c, int &idb, int &idr) __attribute__((always_inline)) {
        const int pg = min((64 * c + lane) * 4 + pw, n_pages - 1);
        idb = btb[pg];
        idr = res_copy ? btr[pg] : 0;
    };
    int idb_cur, idr_cur, idb_nxt, idr_nxt;
    load_ids(0, idb_cur, idr_cur);
    load_ids(1, idb_nxt, idr_nxt);

    auto buf = [&](int tile) __attribute__((always_inline)) -> LdsU32x4 * {
        return (LdsU32x4 *)(lds + (tile % S::NBUF) * (S::BUF_BYTES / 16));
    };
    // this wave's copies of tile `tile` (page 4 tile + pw)
    auto copy_tile = [&](int tile, int idb, int idr) __attribute__((always_inline)) {
        LdsU32x4 *b = buf(tile);
        const uint64_t kaddr = reinterpret_cast<uint64_t>(p.base_kv + ((int64_t)idb * 2 * hkv + h) * (PS * D));
        const i32x4 rs = block_rsrc(kwave ? kaddr : kaddr + (uint64_t)hkv * 4096, 4096);
        LdsU32x4 *dst = b + ((kwave ? S::K_OFF : S::V_OFF) + pw * 4096) / 16;
#pragma unroll
        for (int i = 0; i < 4; ++i) lds_dma16(rs, lane * 16 + i * 1024, dst + i * 64);
        if constexpr (R > 0) {
            if (res_copy) {
                const i32x4 rc = block_rsrc(reinterpret_cast<uint64_t>(p.res_kv + (int64_t)idr * (RT * 512)), RT * 1024);
#pragma unroll
                for (int t = 0; t < RT; ++t) lds_dma16(rc, lane * 16 + t * 1024, b + (S::C_OFF + (t * 4 + pw) * 1024) / 16);
            }
        }
        if constexpr (ROPE && R > 0) {
            if (use_res) {
                // the table rows this wave's rebuild uses: frequency tiles 2 half, 2 half + 1
                // of page pw (1 KB each, cos then sin)
                const int64_t pg = min(tile * 4 + pw, n_pages - 1);
                const uint64_t off = (uint64_t)(pg * (PS * D / 2) + 2 * half * 256) * 4;
                const i32x4 tc = block_rsrc(reinterpret_cast<uint64_t>(p.rope_cos) + off, 2048);
                const i32x4 ts = block_rsrc(reinterpret_cast<uint64_t>(p.rope_sin) + off, 2048);
                LdsU32x4 *td = b + (S::T_OFF + (pw * 2 + half) * 4096) / 16;
                lds_dma16(tc, lane * 16, td);
                lds_dma16(tc, lane * 16 + 1024, td + 64);
                lds_dma16(ts, lane * 16, td + 128);
                lds_dma16(ts, lane * 16 + 1024, td + 192);
            }
        }
    };

    // queries of this lane's rows in the two 16-row tiles of the wave, in the contraction
    // order of the stored K fragments
    int row_tok[2], row_pos[2];
    bool row_ok[2];
    u32x4 qf[2][4];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const int r = wave * ROWS_PER_WAVE + nt * 16 + col;
        const int tk = tok_begin + r / G;
        const int jj = r % G;
        row_ok[nt] = tk < nq;
        row_tok[nt] = tk;
        row_pos[nt] = P0 + tk;
        const uint16_t *qr = p.q + ((int64_t)(q0 + (row_ok[nt] ? tk : 0)) * p.hq + h * G + jj) * D;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            u32x4 v = {0, 0, 0, 0};
            if (row_ok[nt]) {
                const u32x2 lo = ldg64(qr + 32 * kk + 4 * grp);
                const u32x2 hi = ldg64(qr + 32 * kk + 16 + 4 * grp);
                v = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
            qf[nt][kk] = v;
        }
    }
    // W^T = (B_K q)^T per row tile and rank tile: the residual key term of row j is
    // (B_K q_j) . c_p, one extra contraction over the rank
    u32x2 wq[2][RTX];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int t = 0; t < RTX; ++t) wq[nt][t] = u32x2{0, 0};
    if constexpr (R > 0 && !ROPE) {
        if (use_res) {
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    f32x4 acc = {0, 0, 0, 0};
                    const int rho = 16 * t + col;
                    const uint16_t *bk = p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)(rho < R ? rho : 0) * n + (int64_t)h * D;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        u32x4 av = {0, 0, 0, 0};
                        if (rho < R) {
                            const u32x2 lo = ldg64(bk + 32 * kk + 4 * grp);
                            const u32x2 hi = ldg64(bk + 32 * kk + 16 + 4 * grp);
                            av = u32x4{lo.x, lo.y, hi.x, hi.y};
                        }
                        acc = mfma32(av, qf[nt][kk], acc);
                    }
                    wq[nt][t] = pack4(acc);
                }
        }
    }
    // RoPE on: B_K^T fragments of the agent's adapter (lane holds B_K[16t + 4grp + i][h*D +
    // 16mt + col]) in LDS for the whole launch; this wave rebuilds u tiles 2 half, 2 half + 1
    // and their rotation partners + 4 of page pw, with the table rows of frequency tiles
    // 2 half + j, loaded one tile ahead
    if constexpr (ROPE && R > 0) {
        if (use_res) {
            u32x2 *bkt = const_cast<u32x2 *>(sBK);
            const uint16_t *bk = p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)h * D;
            for (int idx = threadIdx.x; idx < RT * 8 * 64; idx += 64 * kStreamWaves) {
                const int ln = idx & 63, rest = idx >> 6;
                const int mt = rest & 7, t = rest >> 3;
                const int c = ln & 15, gg = ln >> 4;
                uint32_t w[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int r0 = 16 * t + 4 * gg + 2 * j;
                    const uint16_t lo = r0 < R ? bk[(int64_t)r0 * n + 16 * mt + c] : (uint16_t)0;
                    const uint16_t hi = r0 + 1 < R ? bk[(int64_t)(r0 + 1) * n + 16 * mt + c] : (uint16_t)0;
                    w[j] = (uint32_t)lo | ((uint32_t)hi << 16);
                }
                bkt[idx] = u32x2{w[0], w[1]};
            }
            __syncthreads();  // B_K^T fragments written (no copy into LDS is in flight yet)
        }
    }
    // the page ids must be in registers before the first copies read them
    wait_vmcnt<0>();
    copy_tile(0, __builtin_amdgcn_readlane(idb_cur, 0), __builtin_amdgcn_readlane(idr_cur, 0));
    if (S::NBUF == 3 && n_tiles > 1) copy_tile(1, __builtin_amdgcn_readlane(idb_cur, 1), __builtin_amdgcn_readlane(idr_cur, 1));

    f32x4 oacc[8][2];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) oacc[mt][0] = oacc[mt][1] = f32x4{0, 0, 0, 0};
    f32x4 racc[RTX][2];
#pragma unroll
    for (int t = 0; t < RTX; ++t) racc[t][0] = racc[t][1] = f32x4{0, 0, 0, 0};
    f32x4 lacc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};  // row sums l
    float m_run[2] = {kNegInf, kNegInf};
    const float cl = p.scale_log2;
    const u32x4 kOnes = u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};  // bf16 1.0

    for (int tile = 0; tile < n_tiles; ++tile) {
        // this wave's copies of the tile have landed (only those of the next tile, issued
        // after them, may still be in flight); after the barrier every wave's have, and
        // every wave is done with the tile before, whose buffer the next copies overwrite
        // (two buffers: nothing else is in flight)
        if (S::NBUF == 3 && tile + 1 < n_tiles) {
            if (res_copy) wait_vmcnt<4 + RT>();
            else wait_vmcnt<4>();
        } else {
            wait_vmcnt<0>();
        }
        __builtin_amdgcn_s_barrier();
        const int tn = tile + S::NBUF - 1;
        if (tn < n_tiles) {
            if ((tn & 63) == 0) {
                idb_cur = idb_nxt;
                idr_cur = idr_nxt;
                load_ids((tn >> 6) + 1, idb_nxt, idr_nxt);
            }
            copy_tile(tn, __builtin_amdgcn_readlane(idb_cur, tn & 63), __builtin_amdgcn_readlane(idr_cur, tn & 63));
        }
        const uint32_t base = lds_addr(buf(tile)) + lane * 16;
        // keys of the tile at or past the sequence end (the tile that holds it, or pages
        // past it) may hold any bits in V and C_V: zero them
        const bool ragged = (tile + 1) * TILE_KEYS > L;
        if constexpr (ROPE && R > 0) {
            if (use_res) {
                // Stage 1 for a quarter of page pw: U^T tiles, deferred RoPE, K = K_base +
                // K_lora in place (keys past the sequence end are masked out of the scores)
                u32x2 ck[RTX];
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    const u32x4 c = lds_read1(base + S::C_OFF + (t * 4 + pw) * 1024);
                    ck[t] = (16 * t + 4 * grp < R) ? u32x2{c.x, c.y} : u32x2{0, 0};
                }
                f32x4 u[4];  // u tiles 2 half, 2 half + 1, 2 half + 4, 2 half + 5
#pragma unroll
                for (int j = 0; j < 4; ++j) u[j] = f32x4{0, 0, 0, 0};
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    // (explicit reads: the copies in flight write other LDS bytes)
                    u32x2 bkf[4];
                    lds_read4_b64_tiles(lds_addr((LdsU32x4 *)lds) + S::MAIN_BYTES + ((t * 8 + 2 * half) * 64 + lane) * 8, bkf);
#pragma unroll
                    for (int j = 0; j < 4; ++j) u[j] = mfma16(bkf[j], ck[t], u[j]);
                }
                // rotate-half pairs (tile m with m + 4) at the key's position
                u32x4 rot[4];  // cos m, cos m + 1, sin m, sin m + 1 of this lane
                lds_read4(base + S::T_OFF + (pw * 2 + half) * 4096, rot);
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const f32x4 c = __builtin_bit_cast(f32x4, rot[j]), s = __builtin_bit_cast(f32x4, rot[2 + j]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float x = u[j][i], y = u[j + 2][i];
                        u[j][i] = x * c[i] - y * s[i];
                        u[j + 2][i] = y * c[i] + x * s[i];
                    }
                }
                // K fragments half (u tiles 2 half, 2 half + 1) and half + 2 (tiles + 4)
                const uint32_t ka = base + S::K_OFF + pw * 4096 + half * 1024;
                const uint32_t kb = ka + 2 * 1024;
                u32x4 kf[2];
                lds_read2_2k(ka, kf);
                u32x4 out[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const u32x4 k = kf[j];
                    const f32x4 lo = f32x4{bf16_lo(k.x), bf16_hi(k.x), bf16_lo(k.y), bf16_hi(k.y)} + u[2 * j];
                    const f32x4 hi = f32x4{bf16_lo(k.z), bf16_hi(k.z), bf16_lo(k.w), bf16_hi(k.w)} + u[2 * j + 1];
                    const u32x2 plo = pack4(lo), phi = pack4(hi);
                    out[j] = u32x4{plo.x, plo.y, phi.x, phi.y};
                }
                lds_write2(ka, out[0], kb, out[1]);
                __builtin_amdgcn_s_barrier();  // the rebuilt tile is complete
            }
        }

        // ---- scores for the 64 keys of the tile, 2 row tiles ----
        f32x4 sacc[4][2];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            u32x4 kf[4];
            lds_read4(base + S::K_OFF + kt * 4096, kf);
            sacc[kt][0] = sacc[kt][1] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                sacc[kt][0] = mfma32(kf[kk], qf[0][kk], sacc[kt][0]);
                sacc[kt][1] = mfma32(kf[kk], qf[1][kk], sacc[kt][1]);
            }
        }
        if constexpr (R > 0 && !ROPE) {
            if (use_res) {
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    // rCache fragments of the tile's four pages (C_K in .xy)
                    u32x4 cf[4];
                    lds_read4(base + S::C_OFF + t * 4096, cf);
                    // C_K of rank rows 16t + 4grp .. +3 (rank 8: half a tile is padding)
                    const bool kvalid = 16 * t + 4 * grp < R;
#pragma unroll
                    for (int kt = 0; kt < 4; ++kt) {
                        const u32x4 ak = u32x4{kvalid ? cf[kt].x : 0u, kvalid ? cf[kt].y : 0u, 0u, 0u};
                        // zero-padded 16x16x32 form: the chain stays on one instruction form
                        sacc[kt][0] = mfma32(ak, u32x4{wq[0][t].x, wq[0][t].y, 0u, 0u}, sacc[kt][0]);
                        sacc[kt][1] = mfma32(ak, u32x4{wq[1][t].x, wq[1][t].y, 0u, 0u}, sacc[kt][1]);
                    }
                }
            }
        }

        // ---- causal mask + online softmax (rows live in lanes) ----
        // A tile below every row's diagonal needs no mask.  The running maximum moves only
        // when some row's scores exceed it by more than 2^kLazyRescale (then acc, acc_r and
        // the row sums are rescaled); otherwise this tile's weights stay below 2^8.
        const bool full = (tile + 1) * TILE_KEYS - 1 <= P0 + tok_begin;
        u32x2 pf[4][2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            float sv[4][4];
            if (full) {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) sv[kt][i] = sacc[kt][nt][i];
            } else {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = tile * TILE_KEYS + kt * PS + 4 * grp + i;
                        sv[kt][i] = (row_ok[nt] && key <= row_pos[nt]) ? sacc[kt][nt][i] : kNegInf;
                    }
            }
            float mx = kNegInf;
#pragma unroll
            for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sv[kt][i]);
            mx = max_over_groups(mx) * cl;  // the scale is positive
            if (__builtin_amdgcn_ballot_w64(mx > m_run[nt] + kLazyRescale) != 0) {
                const float m_new = fmaxf(m_run[nt], mx);
                const float alpha = fast_exp2(m_run[nt] - (m_new == kNegInf ? 0.f : m_new));
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) oacc[mt][nt] *= alpha;
#pragma unroll
                for (int t = 0; t < RT; ++t) racc[t][nt] *= alpha;
                lacc[nt] *= alpha;
                m_run[nt] = m_new;
            }
            const float m_use = m_run[nt] == kNegInf ? 0.f : m_run[nt];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                f32x4 pv;
#pragma unroll
                for (int i = 0; i < 4; ++i) pv[i] = fast_exp2(__builtin_fmaf(sv[kt][i], cl, -m_use));
                pf[kt][nt] = pack4(pv);
            }
        }

        // ---- O^T += V^T P^T and acc_r^T += C_V^T P^T over two 32-key halves ----
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const u32x4 pb0 = u32x4{pf[2 * half][0].x, pf[2 * half][0].y, pf[2 * half + 1][0].x, pf[2 * half + 1][0].y};
            const u32x4 pb1 = u32x4{pf[2 * half][1].x, pf[2 * half][1].y, pf[2 * half + 1][1].x, pf[2 * half + 1][1].y};
            u32x4 v0[4], v1[4];
            lds_read8(base + S::V_OFF + (2 * half) * 4096, base + S::V_OFF + (2 * half + 1) * 4096, v0, v1);
            if (ragged) {
                const int vis0 = L - (tile * 4 + 2 * half) * PS, vis1 = vis0 - PS;
#pragma unroll
                for (int q2 = 0; q2 < 4; ++q2) {
                    const u32x2 a0 = mask4(u32x2{v0[q2].x, v0[q2].y}, vis0, grp), b0 = mask4(u32x2{v0[q2].z, v0[q2].w}, vis0, grp);
                    const u32x2 a1 = mask4(u32x2{v1[q2].x, v1[q2].y}, vis1, grp), b1 = mask4(u32x2{v1[q2].z, v1[q2].w}, vis1, grp);
                    v0[q2] = u32x4{a0.x, a0.y, b0.x, b0.y};
                    v1[q2] = u32x4{a1.x, a1.y, b1.x, b1.y};
                }
            }
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) {
                const u32x4 va = u32x4{v0[q2].x, v0[q2].y, v1[q2].x, v1[q2].y};  // dim 32q2 + col
                const u32x4 vb = u32x4{v0[q2].z, v0[q2].w, v1[q2].z, v1[q2].w};  // dim 32q2 + 16 + col
                oacc[2 * q2][0] = mfma32(va, pb0, oacc[2 * q2][0]);
                oacc[2 * q2][1] = mfma32(va, pb1, oacc[2 * q2][1]);
                oacc[2 * q2 + 1][0] = mfma32(vb, pb0, oacc[2 * q2 + 1][0]);
                oacc[2 * q2 + 1][1] = mfma32(vb, pb1, oacc[2 * q2 + 1][1]);
            }
            // row sums of the bf16 weights (every accumulator row holds the sum)
            lacc[0] = mfma32(kOnes, pb0, lacc[0]);
            lacc[1] = mfma32(kOnes, pb1, lacc[1]);
            if constexpr (R > 0) {
                if (use_res) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        // C_V of rank 16t + col, tokens 4grp .. +3 of the two pages (.zw)
                        u32x4 cf[2];
                        lds_read2(base + S::C_OFF + (t * 4 + 2 * half) * 1024, cf);
                        u32x2 c0 = u32x2{cf[0].z, cf[0].w};
                        u32x2 c1 = u32x2{cf[1].z, cf[1].w};
                        if (ragged) {
                            const int vis0 = L - (tile * 4 + 2 * half) * PS;
                            c0 = mask4(c0, vis0, grp);
                            c1 = mask4(c1, vis0 - PS, grp);
                        }
                        const bool vvalid = 16 * t + col < R;
                        const u32x4 ca = vvalid ? u32x4{c0.x, c0.y, c1.x, c1.y} : u32x4{0, 0, 0, 0};
                        racc[t][0] = mfma32(ca, pb0, racc[t][0]);
                        racc[t][1] = mfma32(ca, pb1, racc[t][1]);
                    }
                }
            }
        }
    }
    wait_vmcnt<0>();
    __syncthreads();  // the buffers are reused below

    // ---- epilogue: O = (acc + acc_r . B_V[h]) / l ----
    const float l_run[2] = {lacc[0][0], lacc[1][0]};
    if constexpr (R > 0) {
        if (use_res) {
            const uint16_t *bv = p.lora_b + ((int64_t)ad * 2 + 1) * R * n + (int64_t)h * D;
            for (int e = threadIdx.x; e < R * D; e += 64 * kStreamWaves) sBV[e] = bf16_to_f32(bv[(int64_t)(e / D) * n + (e % D)]);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int rho = 16 * t + 4 * grp + i;
                        if (rho < R) sAcc[(wave * ROWS_PER_WAVE + nt * 16 + col) * R + rho] = racc[t][nt][i];
                    }
            __syncthreads();
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                const float *ar = sAcc + (wave * ROWS_PER_WAVE + nt * 16 + col) * R;
                for (int rho = 0; rho < R; ++rho) {
                    const float c = ar[rho];
#pragma unroll
                    for (int mt = 0; mt < 8; ++mt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) oacc[mt][nt][i] += c * sBV[rho * D + 16 * mt + 4 * grp + i];
                }
            }
        }
    }
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        if (!row_ok[nt]) continue;
        const int r = wave * ROWS_PER_WAVE + nt * 16 + col;
        const float inv = l_run[nt] > 0.f ? 1.f / l_run[nt] : 0.f;
        uint16_t *orow = p.out + ((int64_t)(q0 + row_tok[nt]) * p.hq + h * G + r % G) * D;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
            f32x4 o = oacc[mt][nt] * inv;
            *reinterpret_cast<u32x2 *>(orow + 16 * mt + 4 * grp) = pack4(o);
        }
    }
}

template <int R, int G, bool ROPE>
hipError_t launch_prefill(const PrefillArgs &pa, hipStream_t st, void *const *ev) {
    using S = PrefillShape<R, G, ROPE>;
    hipError_t e;
    const int pairs = (pa.n_agents * pa.hkv + kXcds - 1) / kXcds * kXcds;
    const int grid = pairs * pa.blocks_per_agent_head;
    (void)sizeof(S);
    // timing events carry the kernel's own start and end timestamps (set by the launch)
    hipEvent_t e0 = ev ? static_cast<hipEvent_t>(ev[0]) : nullptr;
    hipEvent_t e1 = ev ? static_cast<hipEvent_t>(ev[1]) : nullptr;
    if constexpr (ROPE && !stream_rope(R))
        hipExtLaunchKernelGGL((prefill_kernel<R, G, ROPE>), dim3(grid), dim3(256), 0, st, e0, e1, 0, pa);
    else
        hipExtLaunchKernelGGL((prefill_stream_kernel<R, G, ROPE>), dim3(grid), dim3(64 * kStreamWaves), 0, st, e0, e1, 0, pa);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hipSuccess;
}

template <int G>
hipError_t dispatch_prefill(int r, bool rope, const PrefillArgs &pa, hipStream_t st, void *const *ev) {
    switch (r) {
    case 0: return launch_prefill<0, G, false>(pa, st, ev);
    case 8: return rope ? launch_prefill<8, G, true>(pa, st, ev) : launch_prefill<8, G, false>(pa, st, ev);
    case 16: return rope ? launch_prefill<16, G, true>(pa, st, ev) : launch_prefill<16, G, false>(pa, st, ev);
    case 32: return rope ? launch_prefill<32, G, true>(pa, st, ev) : launch_prefill<32, G, false>(pa, st, ev);
    case 64: return rope ? launch_prefill<64, G, true>(pa, st, ev) : launch_prefill<64, G, false>(pa, st, ev);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

namespace fkv {
fkv_status validate_attn_common(const fkv_attn_args *a, const char *who);
}

extern "C" fkv_status fkv_residual_attention_prefill(const fkv_attn_args *a, void *stream) {
    fkv::clear_error();
    fkv_status st = fkv::validate_attn_common(a, "fkv_residual_attention_prefill");
    if (st != FKV_OK) return st;
    if (!a->q_indptr || a->n_q < 1)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_prefill: q_indptr and n_q >= 1 are required");
    const int g = a->hq / a->hkv;
    if (g != 4 && g != 8)
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_residual_attention_prefill: query heads per KV head must be 4 or 8");
    if (a->rope_cos && (int64_t)a->rope_max_pos < (int64_t)a->max_pages * a->page_size)
        return fkv::fail(FKV_ERR_INVALID,
                         "fkv_residual_attention_prefill: RoPE table must cover max_pages * page_size positions");
    PrefillArgs pa;
    pa.q = static_cast<const uint16_t *>(a->q);
    pa.base_kv = static_cast<const uint16_t *>(a->base_kv);
    pa.res_kv = static_cast<const uint16_t *>(a->res_kv);
    pa.lora_b = static_cast<const uint16_t *>(a->lora_b);
    pa.adapter_idx = a->adapter_idx;
    pa.base_bt = a->base_bt;
    pa.res_bt = a->res_bt;
    pa.seq_lens = a->seq_lens;
    pa.q_indptr = a->q_indptr;
    pa.rope_cos = a->rope_cos;
    pa.rope_sin = a->rope_sin;
    pa.out = static_cast<uint16_t *>(a->out);
    pa.n_agents = a->n_agents;
    pa.hq = a->hq;
    pa.hkv = a->hkv;
    pa.max_pages = a->max_pages;
    // query blocks per (agent, KV head); blocks past an agent's own chunk exit at once
    const bool rope = a->rope_cos != nullptr && a->r > 0;
    const int tok_per_wg = ((rope && !stream_rope(a->r)) ? ROWS_PER_WG : kStreamRows) / g;
    const int maxq = a->max_q_per_agent > 0 ? a->max_q_per_agent : a->n_q;
    if (maxq > a->n_q) return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_prefill: max_q_per_agent > n_q");
    pa.blocks_per_agent_head = (maxq + tok_per_wg - 1) / tok_per_wg;
    pa.scale_log2 = a->scale * 1.4426950408889634f;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    hipError_t e = g == 4 ? dispatch_prefill<4>(a->r, rope, pa, hs, a->timing_events)
                          : dispatch_prefill<8>(a->r, rope, pa, hs, a->timing_events);
    if (e != hipSuccess)
        return fkv::fail(FKV_ERR_HIP, std::string("fkv_residual_attention_prefill: launch failed: ") + hipGetErrorString(e));
    return FKV_OK;
}
