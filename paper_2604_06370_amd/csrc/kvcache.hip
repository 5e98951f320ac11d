// Cache writes: copy-on-write page copies (Section 5.2) and scattering new tokens'
// bCache K/V and rCache C_K/C_V into their page slots.
//
// Page layouts (bf16): base page [2][Hkv][ps*d].  With ps = 16 and d = 128 the K and V
// blocks of one (page, head) are stored in the order in which the attention kernels'
// matrix-core fragments read them (one 16-byte load per lane, 1 KB per wave instruction):
//   K element (token t, dim d) at  (d/32)*512 + (t + 16*((d%16)/4))*8 + 4*((d%32)/16) + d%4
//   V element (token t, dim d) at  (d/32)*512 + (d%16 + 16*(t/4))*8 + 4*((d/16)%2) + t%4
// A residual page with ps = 16 holds ceil(r/16) tiles of 512 values; tile k holds, for
// lane L = 16*g + c of a wave, 8 values at L*8: the 4 at L*8 + i and the 4 at L*8 + 4 + i,
//   C_K[token c][16k + 4g + i]             C_V[token 4g + i][16k + c]        (i = 0..3)
// so each lane reads both of its rCache fragments of a tile with one 16-byte load (1 KB
// contiguous per wave instruction).  Rank values past r (r = 8) are padding.  Other shapes use
// plain [ps][d] (K), [d][ps] (V), [ps][r] (C_K) and [r][ps] (C_V).
#include <hip/hip_runtime.h>

#include <string>

#include "internal.hpp"
#include "mfma.hpp"

using namespace fkvk;

namespace {

// Offsets of (token t, dim dd) inside a K or V block (see the layout note above).
__device__ __forceinline__ int64_t k_off(int t, int dd, int ps, int d) {
    if (ps == 16 && d == 128) return (dd >> 5) * 512 + (t + 16 * ((dd & 15) >> 2)) * 8 + 4 * ((dd & 31) >> 4) + (dd & 3);
    return (int64_t)t * d + dd;
}
__device__ __forceinline__ int64_t v_off(int t, int dd, int ps, int d) {
    if (ps == 16 && d == 128) return (dd >> 5) * 512 + ((dd & 15) + 16 * (t >> 2)) * 8 + 4 * ((dd >> 4) & 1) + (t & 3);
    return (int64_t)dd * ps + t;
}
// Token slot of element e of a K or V block.
__device__ __forceinline__ int k_slot(int64_t e, int ps, int d) {
    if (ps == 16 && d == 128) return (int)(((e & 511) >> 3) & 15);
    return (int)(e / d);
}
__device__ __forceinline__ int v_slot(int64_t e, int ps, int d) {
    if (ps == 16 && d == 128) return (int)(4 * (((e & 511) >> 3) >> 4) + (e & 3));
    return (int)(e % ps);
}

__device__ __forceinline__ int64_t ck_off(int t, int rho, int ps, int r) {
    if (ps == 16) return (int64_t)(rho >> 4) * 512 + (((rho & 15) >> 2) * 16 + t) * 8 + (rho & 3);
    return (int64_t)t * r + rho;
}
__device__ __forceinline__ int64_t cv_off(int t, int rho, int ps, int r) {
    if (ps == 16) return (int64_t)(rho >> 4) * 512 + ((t >> 2) * 16 + (rho & 15)) * 8 + 4 + (t & 3);
    return (int64_t)ps * r + (int64_t)rho * ps + t;
}
__device__ __forceinline__ int64_t res_page_elems(int ps, int r) {
    return ps == 16 ? (int64_t)((r + 15) / 16) * 512 : 2LL * ps * r;
}
// Token slot of element e of a residual page.
__device__ __forceinline__ int c_slot(int64_t e, int ps, int r) {
    if (ps == 16) {
        const int w = (int)(e & 511);  // lane w / 8 of the tile: C_K at w % 8 < 4, else C_V
        return (w & 4) == 0 ? ((w >> 3) & 15) : 4 * (w >> 7) + (w & 3);
    }
    return e < (int64_t)ps * r ? (int)(e / r) : (int)((e - (int64_t)ps * r) % ps);
}

struct CopyArgs {
    const fkv_page_copy *copies;
    uint16_t *base_kv, *res_kv;
    int32_t hkv, d, r, ps;
};

// One workgroup per copy.  Each thread moves 16-byte chunks: in both pools' layouts every
// chunk of 8 values holds tokens of at most four consecutive slots, so a chunk whose slots are
// all below n_valid is copied whole, one with none is skipped, and one that straddles n_valid
// (a value chunk of four tokens, or an rCache chunk) is copied value by value.
template <typename SlotOf>
__device__ __forceinline__ void copy_chunks(const uint16_t *src, uint16_t *dst, int64_t elems, int n_valid,
                                            SlotOf slot_of) {
    const int64_t chunks = elems / 8;
    for (int64_t c = threadIdx.x; c < chunks; c += blockDim.x) {
        int lo = 1 << 30, hi = -1;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int sl = slot_of(8 * c + e);
            lo = min(lo, sl);
            hi = max(hi, sl);
        }
        if (hi < n_valid) {
            reinterpret_cast<u32x4 *>(dst)[c] = reinterpret_cast<const u32x4 *>(src)[c];
        } else if (lo < n_valid) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (slot_of(8 * c + e) < n_valid) dst[8 * c + e] = src[8 * c + e];
        }
    }
    for (int64_t e = chunks * 8 + threadIdx.x; e < elems; e += blockDim.x)
        if (slot_of(e) < n_valid) dst[e] = src[e];
}

__global__ __launch_bounds__(256) void page_copy_kernel(CopyArgs a) {
    const fkv_page_copy c = a.copies[blockIdx.x];
    const int n_valid = c.n_valid;
    if (c.pool == FKV_POOL_BASE) {
        const int64_t blk = (int64_t)a.ps * a.d;
        const int64_t page = 2 * a.hkv * blk;
        const uint16_t *src = a.base_kv + (int64_t)c.src * page;
        uint16_t *dst = a.base_kv + (int64_t)c.dst * page;
        const int hkv = a.hkv, ps = a.ps, d = a.d;
        if (blk % 8 == 0) {
            // chunks never straddle a block: K blocks first (hkv of them), then V blocks
            copy_chunks(src, dst, page, n_valid, [=](int64_t e) {
                const int64_t within = e % blk;
                return (e / blk) >= hkv ? v_slot(within, ps, d) : k_slot(within, ps, d);
            });
        } else {
            for (int64_t e = threadIdx.x; e < page; e += blockDim.x) {
                const int64_t within = e % blk;
                const int slot = (e / blk) >= hkv ? v_slot(within, ps, d) : k_slot(within, ps, d);
                if (slot < n_valid) dst[e] = src[e];
            }
        }
    } else {
        const int64_t page = res_page_elems(a.ps, a.r);
        const uint16_t *src = a.res_kv + (int64_t)c.src * page;
        uint16_t *dst = a.res_kv + (int64_t)c.dst * page;
        const int ps = a.ps, r = a.r;
        if (ps == 16) {
            copy_chunks(src, dst, page, n_valid, [=](int64_t e) { return c_slot(e, ps, r); });
        } else {
            for (int64_t e = threadIdx.x; e < page; e += blockDim.x)
                if (c_slot(e, ps, r) < n_valid) dst[e] = src[e];
        }
    }
}

struct ScatterArgs {
    const int32_t *bt_base, *bt_res;
    int64_t pos0, n;
    const uint16_t *k_src, *v_src, *ck_src, *cv_src;
    uint16_t *base_kv, *res_kv;
    int32_t hkv, d, r, ps;
};

// Page size 16, head dim 128: one workgroup per page the range [pos0, pos0 + n) touches.  Every
// 16-byte chunk of the fragment-ordered blocks is formed in registers from the source rows and
// stored whole: a K chunk is 8 dims of one token (two 8-byte pieces of its row); a V chunk is 2
// dims of four consecutive tokens and an rCache chunk 4 ranks of one token (C_K) and one rank of
// four tokens (C_V), so chunks whose tokens are only partly in the range are written value by
// value (slots outside the range, and the rank padding of r = 8, keep their bits).
__global__ __launch_bounds__(256) void scatter_page_kernel(ScatterArgs a) {
    constexpr int PS = 16, D = 128;
    const int64_t first_page = a.pos0 / PS;
    const int64_t lp = first_page + blockIdx.x;
    const int64_t s0 = lp * PS;  // position of slot 0 of this page
    const int t_lo = (int)max<int64_t>(0, a.pos0 - s0), t_hi = (int)min<int64_t>(PS, a.pos0 + a.n - s0);
    auto row = [&](int t) { return s0 + t - a.pos0; };  // source row of slot t
    const int hkv = a.hkv;
    if (a.k_src) {
        uint16_t *pg = a.base_kv + (int64_t)a.bt_base[lp] * 2 * hkv * PS * D;
        // K: chunk (head, quarter q, lane L = t + 16 g) = dims 32q + 4g + 0..3 and 32q + 16 + 4g + 0..3 of token t
        for (int c = threadIdx.x; c < hkv * 4 * 64; c += blockDim.x) {
            const int hh = c / 256, q = (c / 64) % 4, L = c % 64;
            const int t = L % 16, g = L / 16;
            if (t < t_lo || t >= t_hi) continue;
            const uint16_t *src = a.k_src + (row(t) * hkv + hh) * D + 32 * q + 4 * g;
            const u32x2 lo = ldg64(src), hi = ldg64(src + 16);
            *reinterpret_cast<u32x4 *>(pg + (int64_t)hh * PS * D + q * 512 + L * 8) = u32x4{lo.x, lo.y, hi.x, hi.y};
        }
        // V: chunk (head, quarter q, lane L = c + 16 tg) = dim 32q + c of tokens 4tg + 0..3, then dim 32q + 16 + c
        uint16_t *pv = pg + (int64_t)hkv * PS * D;
        for (int c = threadIdx.x; c < hkv * 4 * 64; c += blockDim.x) {
            const int hh = c / 256, q = (c / 64) % 4, L = c % 64;
            const int dc = L % 16, tg = L / 16;
            const int ta = 4 * tg, tb = ta + 4;
            if (tb <= t_lo || ta >= t_hi) continue;
            uint16_t *dst = pv + (int64_t)hh * PS * D + q * 512 + L * 8;
            if (ta >= t_lo && tb <= t_hi) {
                uint16_t v[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint16_t *src = a.v_src + (row(ta + i) * hkv + hh) * D + 32 * q + dc;
                    v[i] = src[0];
                    v[4 + i] = src[16];
                }
                u32x4 w;
                w.x = v[0] | ((uint32_t)v[1] << 16);
                w.y = v[2] | ((uint32_t)v[3] << 16);
                w.z = v[4] | ((uint32_t)v[5] << 16);
                w.w = v[6] | ((uint32_t)v[7] << 16);
                *reinterpret_cast<u32x4 *>(dst) = w;
            } else {
                for (int i = 0; i < 4; ++i) {
                    const int t = ta + i;
                    if (t < t_lo || t >= t_hi) continue;
                    const uint16_t *src = a.v_src + (row(t) * hkv + hh) * D + 32 * q + dc;
                    dst[i] = src[0];
                    dst[4 + i] = src[16];
                }
            }
        }
    }
    if (a.ck_src && a.r > 0) {
        const int r = a.r, rt = (r + 15) / 16;
        uint16_t *pg = a.res_kv + (int64_t)a.bt_res[lp] * rt * 512;
        // tile k, lane L = c + 16 g: C_K[token c][16k + 4g + 0..3] at L*8, C_V[tokens 4g + 0..3][16k + c] at L*8 + 4
        for (int c = threadIdx.x; c < rt * 64; c += blockDim.x) {
            const int k = c / 64, L = c % 64;
            const int tc = L % 16, g = L / 16;
            uint16_t *dst = pg + k * 512 + L * 8;
            if (tc >= t_lo && tc < t_hi && 16 * k + 4 * g < r) {
                const uint16_t *src = a.ck_src + row(tc) * r + 16 * k + 4 * g;
                if (r % 4 == 0) {
                    *reinterpret_cast<u32x2 *>(dst) = ldg64(src);
                } else {
                    for (int i = 0; i < 4 && 16 * k + 4 * g + i < r; ++i) dst[i] = src[i];
                }
            }
            const int rho = 16 * k + tc;
            if (rho < r) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int t = 4 * g + i;
                    if (t < t_lo || t >= t_hi) continue;
                    dst[4 + i] = a.cv_src[row(t) * r + rho];
                }
            }
        }
    }
}

// Other shapes: one workgroup per token; threads cover (head, dim) for the base pool and the
// rank for the residual pool.
__global__ __launch_bounds__(256) void scatter_kernel(ScatterArgs a) {
    const int64_t j = blockIdx.x;
    const int64_t pos = a.pos0 + j;
    const int64_t lp = pos / a.ps;
    const int slot = (int)(pos - lp * a.ps);
    if (a.k_src) {
        const int32_t page = a.bt_base[lp];
        const int64_t blk = (int64_t)a.ps * a.d;
        uint16_t *pg = a.base_kv + (int64_t)page * 2 * a.hkv * blk;
        for (int e = threadIdx.x; e < a.hkv * a.d; e += blockDim.x) {
            const int hh = e / a.d, dd = e - hh * a.d;
            pg[hh * blk + k_off(slot, dd, a.ps, a.d)] = a.k_src[j * a.hkv * a.d + e];
            pg[(a.hkv + hh) * blk + v_off(slot, dd, a.ps, a.d)] = a.v_src[j * a.hkv * a.d + e];
        }
    }
    if (a.ck_src && a.r > 0) {
        const int32_t page = a.bt_res[lp];
        uint16_t *pg = a.res_kv + (int64_t)page * res_page_elems(a.ps, a.r);
        for (int e = threadIdx.x; e < a.r; e += blockDim.x) {
            pg[ck_off(slot, e, a.ps, a.r)] = a.ck_src[j * a.r + e];
            pg[cv_off(slot, e, a.ps, a.r)] = a.cv_src[j * a.r + e];
        }
    }
}

// ---------------------------------------------------------------------------
// Producer: the cache writes of new tokens (Section 5.2 / 5.3, the step before attention).
// Per token at position pos: K = RoPE_pos(k_raw) (rotate-half pairs (i, i + d/2), angles from
// the fp32 table) and V into the base pool; C_K = x A_K^T and C_V = x A_V^T (the LoRA shrink,
// hidden -> r, fp32 accumulation on the matrix cores) into the residual pool.  Page size 16,
// head dim 128 (the fragment layouts).  Every workgroup covers one page of the call's
// position range (slots outside [pos0, pos0 + n) are left as they are).  One launch, two
// kinds of workgroups:
//  - shrink (one per four pages): wave w covers every fourth block of the hidden dimension with 16x16x32
//    products (16 bytes of one token's x row and of one row of A per lane, A L2-resident),
//    eight k-steps of loads in flight; the four partial tiles are summed through LDS.  C_K is
//    computed transposed (A as the row operand), so each lane holds 4 ranks of one token
//    and C_V 4 tokens of one rank: both are 8 contiguous bytes of the residual page;
//  - base (one per page and pair of KV heads): the page's 16 token rows of K and V of
//    each head come into LDS with 16-byte loads, all requested together; each thread then forms 16-byte chunks of the fragment-ordered blocks (K:
//    one token's dims 32a + 16h + 4b + i and their rotate-half partners 64 further on, so
//    the rotation needs nothing from other threads; V: 4 tokens x 2 dims) and stores them
//    whole (V chunks that straddle the range end are written element by element).
struct ProduceSeq {
    const int32_t *bt_base, *bt_res;
    const uint16_t *lora_a;     // null: no shrink for this sequence
    int64_t pos0, row0;         // first new position; its row in x, k_raw and v
    int32_t n, first_shrink;    // new tokens; its first shrink workgroup
    int32_t first_base, pad;    // its first base workgroup
};
constexpr int kProdMaxSeqs = 32;  // sequences per launch (kernel-argument space)
struct ProduceArgs {
    ProduceSeq seq[kProdMaxSeqs];
    int32_t nseq, n_shrink_blocks, hidden, hkv;
    const uint16_t *x, *k_raw, *v;
    const float *rope_cos, *rope_sin;
    uint16_t *base_kv, *res_kv;
};
constexpr int kProdChunk = 1024;  // hidden is a multiple of this (four waves x 8 k-steps x 32)
constexpr int kProdHeads = 2;     // KV heads per base workgroup
constexpr int kShrinkPages = 4;   // pages (16-token tiles) per shrink workgroup

template <int R>
__global__ __launch_bounds__(256, 6) void produce_kernel(ProduceArgs a) {
    constexpr int PS = 16, D = 128, HALF = D / 2;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    // the sequence served: the last one whose first workgroup of this kind is at or below ours
    const int bid = blockIdx.x;
    const bool shrink_wg = bid < a.n_shrink_blocks;
    int s = 0;
    for (int j = 1; j < a.nseq; ++j)
        if ((shrink_wg ? a.seq[j].first_shrink : a.seq[j].first_base) <= bid) s = j;
    const ProduceSeq &q = a.seq[s];
    const int lb = bid - (shrink_wg ? q.first_shrink : q.first_base);  // workgroup within the sequence
    const int64_t pos0 = q.pos0, nq = q.n;
    const int64_t page0 = pos0 / PS;
    if (shrink_wg) {
        if constexpr (R > 0) {
            constexpr int RT = (R + 15) / 16, NT = 2 * RT;
            __shared__ fkvk::f32x4 s_part[3][NT][kShrinkPages][64];
            // tile u: page page0 + kShrinkPages lb + u; token slot col of it is call index tj0[u] + col
            int64_t tj0[kShrinkPages];
            bool tok_ok[kShrinkPages];
            const uint16_t *xr[kShrinkPages];
            fkvk::f32x4 acc[NT][kShrinkPages];
#pragma unroll
            for (int u = 0; u < kShrinkPages; ++u) {
                tj0[u] = (page0 + (int64_t)kShrinkPages * lb + u) * PS - pos0;
                const int64_t tok = tj0[u] + col;
                tok_ok[u] = tok >= 0 && tok < nq;
                xr[u] = a.x + q.row0 * a.hidden + (tok_ok[u] ? tok : 0) * a.hidden + 8 * grp;
#pragma unroll
                for (int t = 0; t < NT; ++t) acc[t][u] = fkvk::f32x4{0, 0, 0, 0};
            }
            const int quarter = a.hidden / 4;
            // rows of A: shrink t / RT (K, then V), rank 16 (t % RT) + col (rows past r read row 0, zeroed)
            const uint16_t *ar[NT];
            bool rok[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int rho = 16 * (t % RT) + col;
                rok[t] = rho < R;
                ar[t] = q.lora_a + ((int64_t)((t / RT) * R + (rok[t] ? rho : 0)) * a.hidden + 8 * grp);
            }
            // KS k-steps per round, two rounds in flight (the next round's loads are issued before
            // the current round's products; the last round re-requests its own block so that
            // every load is unconditional and the wait counts stay exact).  Round k0 of wave w
            // covers hidden columns 4 k0 + w step .. + step - 1: the four waves' blocks of a round
            // are adjacent, so each token row is read in runs of 4 step columns.  Every A
            // fragment serves the kShrinkPages token tiles.
            constexpr int KS = NT <= 2 ? 2 : 1;
            constexpr int step = 32 * KS;
            auto load = [&](int k0, fkvk::u32x4 (&xa)[KS][kShrinkPages], fkvk::u32x4 (&bw)[KS][NT]) __attribute__((always_inline)) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const int off = 4 * k0 + wave * step + 32 * ks;
#pragma unroll
                    for (int u = 0; u < kShrinkPages; ++u)
                        xa[ks][u] = tok_ok[u] ? fkvk::ldg128(xr[u] + off) : fkvk::u32x4{0, 0, 0, 0};
#pragma unroll
                    for (int t = 0; t < NT; ++t) bw[ks][t] = fkvk::ldg128(ar[t] + off);
                }
            };
            auto products = [&](const fkvk::u32x4 (&xa)[KS][kShrinkPages], const fkvk::u32x4 (&bw)[KS][NT]) __attribute__((always_inline)) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const fkvk::u32x4 w = rok[t] ? bw[ks][t] : fkvk::u32x4{0, 0, 0, 0};
#pragma unroll
                        for (int u = 0; u < kShrinkPages; ++u)  // C_K^T (ranks in rows), C_V (tokens in rows)
                            acc[t][u] = t < RT ? fkvk::mfma32(w, xa[ks][u], acc[t][u]) : fkvk::mfma32(xa[ks][u], w, acc[t][u]);
                    }
            };
            fkvk::u32x4 xa0[KS][kShrinkPages], bw0[KS][NT], xa1[KS][kShrinkPages], bw1[KS][NT];
            load(0, xa0, bw0);
            for (int k0 = 0;;) {
                load(min(k0 + step, quarter - step), xa1, bw1);
                products(xa0, bw0);
                if ((k0 += step) >= quarter) break;
                load(min(k0 + step, quarter - step), xa0, bw0);
                products(xa1, bw1);
                if ((k0 += step) >= quarter) break;
            }
            if (wave > 0) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
#pragma unroll
                    for (int u = 0; u < kShrinkPages; ++u) s_part[wave - 1][t][u][lane] = acc[t][u];
            }
            __syncthreads();
            if (wave == 0) {
#pragma unroll
                for (int u = 0; u < kShrinkPages; ++u) {
                    if (tj0[u] >= nq) continue;  // page past the sequence's range: its table entry is not read
                    const int64_t pp = page0 + (int64_t)kShrinkPages * lb + u;
                    uint16_t *pg = a.res_kv + (int64_t)q.bt_res[pp] * res_page_elems(PS, R);
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        fkvk::f32x4 c = acc[t][u];
#pragma unroll
                        for (int w = 0; w < 3; ++w) c += s_part[w][t][u][lane];
                        const int kt = t % RT;
                        const fkvk::u32x2 h4 = fkvk::u32x2{fkvk::pack_bf16(c[0], c[1]), fkvk::pack_bf16(c[2], c[3])};
                        uint16_t *dst = pg + kt * 512 + (16 * grp + col) * 8;
                        if (t < RT) {
                            // C_K[token col][rank 16 kt + 4 grp + i] at dst[i]
                            if (tok_ok[u] && 16 * kt + 4 * grp < R) *reinterpret_cast<fkvk::u32x2 *>(dst) = h4;
                        } else if (16 * kt + col < R) {
                            // C_V[token 4 grp + i][rank 16 kt + col] at dst[4 + i]
                            const int64_t tf = tj0[u] + 4 * grp;
                            if (tf >= 0 && tf + 3 < nq) {
                                *reinterpret_cast<fkvk::u32x2 *>(dst + 4) = h4;
                            } else {
#pragma unroll
                                for (int i = 0; i < 4; ++i)
                                    if (tf + i >= 0 && tf + i < nq)
                                        dst[4 + i] = (uint16_t)((i & 1 ? h4[i >> 1] >> 16 : h4[i >> 1]) & 0xffffu);
                            }
                        }
                    }
                }
            }
        }
        return;
    }
    // base K (rotated) and V of one page and up to kProdHeads KV heads: every head's token
    // rows are requested before the first one is stored into LDS
    __shared__ __attribute__((aligned(16))) uint16_t s_k[kProdHeads][PS * D], s_v[kProdHeads][PS * D];  // [slot][dim]
    const int n_hg = (a.hkv + kProdHeads - 1) / kProdHeads;
    const int b = lb;
    const int h0 = (b % n_hg) * kProdHeads;
    const int nh = min(kProdHeads, a.hkv - h0);
    const int64_t pp = page0 + b / n_hg;
    const int64_t tj0 = pp * PS - pos0;  // call index of slot 0 (negative on a first partial page)
    {
        const int t = threadIdx.x >> 4, c = threadIdx.x & 15;
        const int64_t tj = tj0 + t;
        const bool ok = tj >= 0 && tj < nq;
        fkvk::u32x4 kx[kProdHeads], vx[kProdHeads];
#pragma unroll
        for (int i = 0; i < kProdHeads; ++i) {
            kx[i] = vx[i] = fkvk::u32x4{0, 0, 0, 0};
            if (ok && i < nh) {
                const int64_t src = ((q.row0 + tj) * a.hkv + h0 + i) * D + 8 * c;
                kx[i] = fkvk::ldg128(a.k_raw + src);
                vx[i] = fkvk::ldg128(a.v + src);
            }
        }
#pragma unroll
        for (int i = 0; i < kProdHeads; ++i) {
            *reinterpret_cast<fkvk::u32x4 *>(&s_k[i][t * D + 8 * c]) = kx[i];
            *reinterpret_cast<fkvk::u32x4 *>(&s_v[i][t * D + 8 * c]) = vx[i];
        }
    }
    __syncthreads();
    constexpr int64_t blk = PS * D;
    uint16_t *const pg = a.base_kv + (int64_t)q.bt_base[pp] * 2 * a.hkv * blk;
    if (threadIdx.x < 128) {
        // K chunks (a2, t, b4) and (a2 + 2, t, b4): element 4h + i is dim f = 32 a2 + 16 h + 4 b4 + i
        // (the first member of a rotate-half pair) and f + 64 (its partner)
        const int t = threadIdx.x & 15, b4 = (threadIdx.x >> 4) & 3, a2 = threadIdx.x >> 6;
        const int64_t tj = tj0 + t;
        if (tj < 0 || tj >= nq) return;
        fkvk::f32x4 cs[2], sn[2];
        if (a.rope_cos) {
            // table order [pos / 16][f / 16][pos % 16 + 16 ((f % 16) / 4)][f % 4]
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t o = pp * (PS * HALF) + (2 * a2 + h) * 256 + (t + 16 * b4) * 4;
                cs[h] = *reinterpret_cast<const fkvk::f32x4 *>(a.rope_cos + o);
                sn[h] = *reinterpret_cast<const fkvk::f32x4 *>(a.rope_sin + o);
            }
        }
        for (int hi = 0; hi < nh; ++hi) {
            float x0[8], x1[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int f = 32 * a2 + 16 * (e >> 2) + 4 * b4 + (e & 3);
                x0[e] = fkvk::bf16_to_f32(s_k[hi][t * D + f]);
                x1[e] = fkvk::bf16_to_f32(s_k[hi][t * D + f + HALF]);
            }
            if (a.rope_cos) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float c = cs[e >> 2][e & 3], s = sn[e >> 2][e & 3];
                    const float u = x0[e], w = x1[e];
                    x0[e] = u * c - w * s;
                    x1[e] = w * c + u * s;
                }
            }
            uint16_t *kb = pg + (h0 + hi) * blk + (t + 16 * b4) * 8;
            *reinterpret_cast<fkvk::u32x4 *>(kb + a2 * 512) =
                fkvk::u32x4{fkvk::pack_bf16(x0[0], x0[1]), fkvk::pack_bf16(x0[2], x0[3]), fkvk::pack_bf16(x0[4], x0[5]),
                            fkvk::pack_bf16(x0[6], x0[7])};
            *reinterpret_cast<fkvk::u32x4 *>(kb + (a2 + 2) * 512) =
                fkvk::u32x4{fkvk::pack_bf16(x1[0], x1[1]), fkvk::pack_bf16(x1[2], x1[3]), fkvk::pack_bf16(x1[4], x1[5]),
                            fkvk::pack_bf16(x1[6], x1[7])};
        }
    } else {
        // V chunks ci and ci + 128 (ci = 64 a + 16 q + c): element 4h + i is (dim 32a + 16h + c, token 4q + i)
        for (int hi = 0; hi < nh; ++hi) {
            uint16_t *vb = pg + (a.hkv + h0 + hi) * blk;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int ci = (int)threadIdx.x - 128 + 128 * half;
                const int av = ci >> 6, q = (ci >> 4) & 3, c = ci & 15;
                uint16_t e8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) e8[e] = s_v[hi][(4 * q + (e & 3)) * D + 32 * av + 16 * (e >> 2) + c];
                const int64_t tf = tj0 + 4 * q;
                if (tf >= 0 && tf + 3 < nq) {
                    fkvk::u32x4 w;
#pragma unroll
                    for (int j = 0; j < 4; ++j) w[j] = (uint32_t)e8[2 * j] | ((uint32_t)e8[2 * j + 1] << 16);
                    *reinterpret_cast<fkvk::u32x4 *>(vb + ci * 8) = w;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (tf + (e & 3) >= 0 && tf + (e & 3) < nq) vb[ci * 8 + e] = e8[e];
                }
            }
        }
    }
}

}  // namespace

extern "C" {

int64_t fkv_res_page_elems(int32_t page_size, int32_t r) {
    if (page_size < 1 || r < 0) return 0;
    return page_size == 16 ? (int64_t)((r + 15) / 16) * 512 : 2LL * page_size * r;
}

fkv_status fkv_page_copy_launch(const fkv_page_copy *copies_dev, int32_t n, void *base_kv, void *res_kv, int32_t hkv,
                                int32_t d, int32_t r, int32_t page_size, void *stream) {
    fkv::clear_error();
    if (n < 0 || (n > 0 && !copies_dev) || hkv < 1 || d < 1 || r < 0 || page_size < 1)
        return fkv::fail(FKV_ERR_INVALID, "fkv_page_copy_launch: bad argument");
    if (n == 0) return FKV_OK;
    if (!base_kv || (r > 0 && !res_kv)) return fkv::fail(FKV_ERR_INVALID, "fkv_page_copy_launch: pool pointer missing");
    CopyArgs a{copies_dev, static_cast<uint16_t *>(base_kv), static_cast<uint16_t *>(res_kv), hkv, d, r, page_size};
    hipLaunchKernelGGL(page_copy_kernel, dim3(n), dim3(256), 0, static_cast<hipStream_t>(stream), a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fkv::fail(FKV_ERR_HIP, std::string("fkv_page_copy_launch: ") + hipGetErrorString(e));
    return FKV_OK;
}

fkv_status fkv_scatter_tokens(const int32_t *bt_base, const int32_t *bt_res, int64_t pos0, int64_t n,
                              const void *k_src, const void *v_src, const void *ck_src, const void *cv_src,
                              void *base_kv, void *res_kv, int32_t hkv, int32_t d, int32_t r, int32_t page_size,
                              void *stream) {
    fkv::clear_error();
    if (pos0 < 0 || n < 0 || hkv < 1 || d < 1 || r < 0 || page_size < 1)
        return fkv::fail(FKV_ERR_INVALID, "fkv_scatter_tokens: bad argument");
    if ((k_src == nullptr) != (v_src == nullptr) || (ck_src == nullptr) != (cv_src == nullptr))
        return fkv::fail(FKV_ERR_INVALID, "fkv_scatter_tokens: K/V (and C_K/C_V) sources come in pairs");
    if (k_src && (!bt_base || !base_kv)) return fkv::fail(FKV_ERR_INVALID, "fkv_scatter_tokens: base table/pool missing");
    if (ck_src && r > 0 && (!bt_res || !res_kv))
        return fkv::fail(FKV_ERR_INVALID, "fkv_scatter_tokens: residual table/pool missing");
    if (n == 0 || (!k_src && !ck_src)) return FKV_OK;
    if (n > INT32_MAX) return fkv::fail(FKV_ERR_INVALID, "fkv_scatter_tokens: too many tokens in one call");
    ScatterArgs a{bt_base, bt_res, pos0, n,
                  static_cast<const uint16_t *>(k_src), static_cast<const uint16_t *>(v_src),
                  static_cast<const uint16_t *>(ck_src), static_cast<const uint16_t *>(cv_src),
                  static_cast<uint16_t *>(base_kv), static_cast<uint16_t *>(res_kv), hkv, d, r, page_size};
    if (page_size == 16 && d == 128) {
        const int64_t pages = (pos0 + n - 1) / 16 - pos0 / 16 + 1;
        hipLaunchKernelGGL(scatter_page_kernel, dim3((unsigned)pages), dim3(256), 0, static_cast<hipStream_t>(stream), a);
    } else {
        hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)n), dim3(256), 0, static_cast<hipStream_t>(stream), a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fkv::fail(FKV_ERR_HIP, std::string("fkv_scatter_tokens: ") + hipGetErrorString(e));
    return FKV_OK;
}

fkv_status fkv_produce_tokens_batch(const fkv_produce_seq *seqs, int32_t nseq, const void *x, int32_t hidden,
                                    const void *k_raw, const void *v, const float *rope_cos, const float *rope_sin,
                                    int64_t rope_max_pos, void *base_kv, void *res_kv, int32_t hkv, int32_t d,
                                    int32_t r, int32_t page_size, void *stream) {
    fkv::clear_error();
    if (nseq < 0 || (nseq > 0 && !seqs) || hkv < 1 || d != 128 || page_size != 16 ||
        !(r == 0 || r == 8 || r == 16 || r == 32 || r == 64))
        return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: needs d = 128, page_size = 16, r in {0, 8, 16, 32, 64}");
    if (!base_kv || !k_raw || !v) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: pool, K or V missing");
    if ((rope_cos == nullptr) != (rope_sin == nullptr))
        return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: RoPE tables come in pairs");
    // every sequence is checked before anything is launched
    for (int32_t i = 0; i < nseq; ++i) {
        const fkv_produce_seq &q = seqs[i];
        const std::string who = "fkv_produce_tokens: sequence " + std::to_string(i) + ": ";
        if (q.pos0 < 0 || q.n < 0 || q.row0 < 0) return fkv::fail(FKV_ERR_INVALID, who + "negative position, count or row");
        if (q.n > (int64_t)1 << 24) return fkv::fail(FKV_ERR_INVALID, who + "too many tokens in one call");
        if (q.n > 0 && !q.bt_base) return fkv::fail(FKV_ERR_INVALID, who + "base table missing");
        if (rope_cos && q.pos0 + q.n > rope_max_pos) return fkv::fail(FKV_ERR_INVALID, who + "RoPE table too short");
        if (q.lora_a && r > 0 && q.n > 0) {
            if (!x || hidden < kProdChunk || hidden % kProdChunk)
                return fkv::fail(FKV_ERR_INVALID, who + "x and hidden (a multiple of 1024) required with lora_a");
            if (!q.bt_res || !res_kv) return fkv::fail(FKV_ERR_INVALID, who + "residual table/pool missing");
        }
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int64_t n_hg = (hkv + kProdHeads - 1) / kProdHeads;
    for (int32_t c0 = 0; c0 < nseq; c0 += kProdMaxSeqs) {
        ProduceArgs a{};
        a.hidden = hidden;
        a.hkv = hkv;
        a.x = static_cast<const uint16_t *>(x);
        a.k_raw = static_cast<const uint16_t *>(k_raw);
        a.v = static_cast<const uint16_t *>(v);
        a.rope_cos = rope_cos;
        a.rope_sin = rope_sin;
        a.base_kv = static_cast<uint16_t *>(base_kv);
        a.res_kv = static_cast<uint16_t *>(res_kv);
        int64_t n_shrink = 0, n_base = 0;
        for (int32_t i = c0; i < nseq && i < c0 + kProdMaxSeqs; ++i) {
            const fkv_produce_seq &q = seqs[i];
            if (q.n == 0) continue;
            const int64_t pages = (q.pos0 + q.n - 1) / page_size - q.pos0 / page_size + 1;  // pages the range touches
            ProduceSeq &o = a.seq[a.nseq++];
            o.bt_base = q.bt_base;
            o.bt_res = q.bt_res;
            o.lora_a = r > 0 ? static_cast<const uint16_t *>(q.lora_a) : nullptr;
            o.pos0 = q.pos0;
            o.row0 = q.row0;
            o.n = (int32_t)q.n;
            o.first_shrink = (int32_t)n_shrink;
            o.first_base = (int32_t)n_base;  // offset by the shrink count below
            if (o.lora_a) n_shrink += (pages + kShrinkPages - 1) / kShrinkPages;
            n_base += pages * n_hg;
        }
        if (a.nseq == 0) continue;
        if (n_shrink + n_base > INT32_MAX) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: batch too large");
        for (int32_t j = 0; j < a.nseq; ++j) a.seq[j].first_base += (int32_t)n_shrink;
        a.n_shrink_blocks = (int32_t)n_shrink;
        const dim3 grid((unsigned)(n_shrink + n_base));
        switch (r) {
        case 0: hipLaunchKernelGGL(produce_kernel<0>, grid, dim3(256), 0, st, a); break;
        case 8: hipLaunchKernelGGL(produce_kernel<8>, grid, dim3(256), 0, st, a); break;
        case 16: hipLaunchKernelGGL(produce_kernel<16>, grid, dim3(256), 0, st, a); break;
        case 32: hipLaunchKernelGGL(produce_kernel<32>, grid, dim3(256), 0, st, a); break;
        default: hipLaunchKernelGGL(produce_kernel<64>, grid, dim3(256), 0, st, a); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fkv::fail(FKV_ERR_HIP, std::string("fkv_produce_tokens: ") + hipGetErrorString(e));
    }
    return FKV_OK;
}

fkv_status fkv_produce_tokens(const int32_t *bt_base, const int32_t *bt_res, int64_t pos0, int64_t n, const void *x,
                              int32_t hidden, const void *k_raw, const void *v, const void *lora_a,
                              const float *rope_cos, const float *rope_sin, int64_t rope_max_pos, void *base_kv,
                              void *res_kv, int32_t hkv, int32_t d, int32_t r, int32_t page_size, void *stream) {
    const fkv_produce_seq q{bt_base, bt_res, lora_a, pos0, n, 0};
    return fkv_produce_tokens_batch(&q, 1, x, hidden, k_raw, v, rope_cos, rope_sin, rope_max_pos, base_kv, res_kv, hkv,
                                    d, r, page_size, stream);
}

}  // extern "C"
