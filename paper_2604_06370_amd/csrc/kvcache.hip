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

// One workgroup per copy; each thread moves whole 16-bit elements whose token slot
// is below n_valid.
__global__ __launch_bounds__(256) void page_copy_kernel(CopyArgs a) {
    const fkv_page_copy c = a.copies[blockIdx.x];
    const int n_valid = c.n_valid;
    if (c.pool == FKV_POOL_BASE) {
        const int64_t blk = (int64_t)a.ps * a.d;
        const int64_t page = 2 * a.hkv * blk;
        const uint16_t *src = a.base_kv + (int64_t)c.src * page;
        uint16_t *dst = a.base_kv + (int64_t)c.dst * page;
        for (int64_t e = threadIdx.x; e < page; e += blockDim.x) {
            const int64_t within = e % blk;
            const bool is_v = (e / blk) >= a.hkv;
            const int slot = is_v ? v_slot(within, a.ps, a.d) : k_slot(within, a.ps, a.d);
            if (slot < n_valid) dst[e] = src[e];
        }
    } else {
        const int64_t page = res_page_elems(a.ps, a.r);
        const uint16_t *src = a.res_kv + (int64_t)c.src * page;
        uint16_t *dst = a.res_kv + (int64_t)c.dst * page;
        for (int64_t e = threadIdx.x; e < page; e += blockDim.x)
            if (c_slot(e, a.ps, a.r) < n_valid) dst[e] = src[e];
    }
}

struct ScatterArgs {
    const int32_t *bt_base, *bt_res;
    int64_t pos0, n;
    const uint16_t *k_src, *v_src, *ck_src, *cv_src;
    uint16_t *base_kv, *res_kv;
    int32_t hkv, d, r, ps;
};

// Grid: one workgroup per token; threads cover (head, dim) for the base pool and
// the rank for the residual pool.
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
// head dim 128 (the fragment layouts).  One launch, two kinds of workgroups:
//  - shrink: 16 tokens; wave w covers a quarter of the hidden dimension with 16x16x32
//    products (A operand: 16 bytes of one token's x row per lane; B operand: 16 bytes of one
//    row of A, read straight from memory, L2-resident), eight k-steps of loads in flight;
//    the four partial tiles are summed through LDS;
//  - base: 64 tokens of one KV head, one (token, rotate-half pair) per item.
struct ProduceArgs {
    const int32_t *bt_base, *bt_res;
    int64_t pos0;
    int32_t n, hidden, hkv, n_shrink_blocks;
    const uint16_t *x, *k_raw, *v, *lora_a;
    const float *rope_cos, *rope_sin;
    uint16_t *base_kv, *res_kv;
};
constexpr int kShrinkTok = 16;
constexpr int kBaseTok = 64;
constexpr int kProdChunk = 1024;  // hidden is a multiple of this (four waves x 8 k-steps x 32)

template <int R>
__global__ __launch_bounds__(256) void produce_kernel(ProduceArgs a) {
    constexpr int PS = 16, D = 128, HALF = D / 2;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    if ((int)blockIdx.x < a.n_shrink_blocks) {
        if constexpr (R > 0) {
            constexpr int RT = (R + 15) / 16, NT = 2 * RT;
            __shared__ fkvk::f32x4 s_part[3][NT][64];
            const int j0 = blockIdx.x * kShrinkTok;
            fkvk::f32x4 acc[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] = fkvk::f32x4{0, 0, 0, 0};
            const int tok = j0 + col;
            const bool tok_ok = tok < a.n;
            const int quarter = a.hidden / 4;
            const uint16_t *xr = a.x + (int64_t)(tok_ok ? tok : 0) * a.hidden + wave * quarter + 8 * grp;
            // B operand rows: shrink t / RT (K, then V), rank 16 (t % RT) + col (rows past r read row 0, zeroed)
            const uint16_t *ar[NT];
            bool rok[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int rho = 16 * (t % RT) + col;
                rok[t] = rho < R;
                ar[t] = a.lora_a + ((int64_t)((t / RT) * R + (rok[t] ? rho : 0)) * a.hidden + wave * quarter + 8 * grp);
            }
            for (int k0 = 0; k0 < quarter; k0 += 8 * 32) {
                fkvk::u32x4 xa[8], bw[8][NT];
#pragma unroll
                for (int ks = 0; ks < 8; ++ks) {
                    xa[ks] = tok_ok ? fkvk::ldg128(xr + k0 + 32 * ks) : fkvk::u32x4{0, 0, 0, 0};
#pragma unroll
                    for (int t = 0; t < NT; ++t) bw[ks][t] = fkvk::ldg128(ar[t] + k0 + 32 * ks);
                }
#pragma unroll
                for (int ks = 0; ks < 8; ++ks)
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        acc[t] = fkvk::mfma32(xa[ks], rok[t] ? bw[ks][t] : fkvk::u32x4{0, 0, 0, 0}, acc[t]);
            }
            if (wave > 0) {
#pragma unroll
                for (int t = 0; t < NT; ++t) s_part[wave - 1][t][lane] = acc[t];
            }
            __syncthreads();
            if (wave == 0) {
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    fkvk::f32x4 c = acc[t];
#pragma unroll
                    for (int w = 0; w < 3; ++w) c += s_part[w][t][lane];
                    // c holds C[token 4grp + i][rank 16 (t % RT) + col] of shrink t / RT
                    const int kv = t / RT, rho = 16 * (t % RT) + col;
                    if (rho >= R) continue;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int tj = j0 + 4 * grp + i;
                        if (tj >= a.n) continue;
                        const int64_t pos = a.pos0 + tj;
                        const int slot = (int)(pos % PS);
                        uint16_t *pg = a.res_kv + (int64_t)a.bt_res[pos / PS] * res_page_elems(PS, R);
                        const uint32_t h2 = fkvk::pack_bf16(c[i], 0.f);
                        pg[kv == 0 ? ck_off(slot, rho, PS, R) : cv_off(slot, rho, PS, R)] = (uint16_t)(h2 & 0xffffu);
                    }
                }
            }
        }
        return;
    }
    // base K (rotated) and V of KV head hh for 64 tokens: one (token, rotate-half pair) per item
    const int b = blockIdx.x - a.n_shrink_blocks;
    const int hh = b % a.hkv;
    const int j0 = (b / a.hkv) * kBaseTok;
    for (int e = threadIdx.x; e < kBaseTok * HALF; e += 256) {
        const int tl = e / HALF, f = e - tl * HALF;
        const int tj = j0 + tl;
        if (tj >= a.n) continue;
        const int64_t pos = a.pos0 + tj;
        const int slot = (int)(pos % PS);
        const int64_t src = ((int64_t)tj * a.hkv + hh) * D;
        float x0 = fkvk::bf16_to_f32(a.k_raw[src + f]), x1 = fkvk::bf16_to_f32(a.k_raw[src + f + HALF]);
        if (a.rope_cos) {
            // table order [pos / 16][f / 16][pos % 16 + 16 ((f % 16) / 4)][f % 4]
            const int64_t o = (pos / PS) * (PS * HALF) + (f / 16) * 256 + (slot + 16 * ((f % 16) / 4)) * 4 + f % 4;
            const float c = a.rope_cos[o], s = a.rope_sin[o];
            const float y0 = x0 * c - x1 * s, y1 = x1 * c + x0 * s;
            x0 = y0;
            x1 = y1;
        }
        constexpr int64_t blk = PS * D;
        uint16_t *pg = a.base_kv + (int64_t)a.bt_base[pos / PS] * 2 * a.hkv * blk;
        const uint32_t kk = fkvk::pack_bf16(x0, x1);
        pg[hh * blk + k_off(slot, f, PS, D)] = (uint16_t)(kk & 0xffffu);
        pg[hh * blk + k_off(slot, f + HALF, PS, D)] = (uint16_t)(kk >> 16);
        pg[(a.hkv + hh) * blk + v_off(slot, f, PS, D)] = a.v[src + f];
        pg[(a.hkv + hh) * blk + v_off(slot, f + HALF, PS, D)] = a.v[src + f + HALF];
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
    hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)n), dim3(256), 0, static_cast<hipStream_t>(stream), a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fkv::fail(FKV_ERR_HIP, std::string("fkv_scatter_tokens: ") + hipGetErrorString(e));
    return FKV_OK;
}

fkv_status fkv_produce_tokens(const int32_t *bt_base, const int32_t *bt_res, int64_t pos0, int64_t n, const void *x,
                              int32_t hidden, const void *k_raw, const void *v, const void *lora_a,
                              const float *rope_cos, const float *rope_sin, int64_t rope_max_pos, void *base_kv,
                              void *res_kv, int32_t hkv, int32_t d, int32_t r, int32_t page_size, void *stream) {
    fkv::clear_error();
    if (pos0 < 0 || n < 0 || hkv < 1 || d != 128 || page_size != 16 || !(r == 0 || r == 8 || r == 16 || r == 32 || r == 64))
        return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: needs d = 128, page_size = 16, r in {0, 8, 16, 32, 64}");
    if (!bt_base || !base_kv || !k_raw || !v) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: base table, pool, K or V missing");
    if ((rope_cos == nullptr) != (rope_sin == nullptr))
        return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: RoPE tables come in pairs");
    if (rope_cos && pos0 + n > rope_max_pos) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: RoPE table too short");
    if (lora_a && r > 0) {
        if (!x || hidden < kProdChunk || hidden % kProdChunk) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: x and hidden (a multiple of 1024) required with lora_a");
        if (!bt_res || !res_kv) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: residual table/pool missing");
    }
    if (n == 0) return FKV_OK;
    if (n > (int64_t)1 << 24) return fkv::fail(FKV_ERR_INVALID, "fkv_produce_tokens: too many tokens in one call");
    const bool shrink = lora_a && r > 0;
    const int32_t n_shrink = shrink ? (int32_t)((n + kShrinkTok - 1) / kShrinkTok) : 0;
    const int64_t n_base = (n + kBaseTok - 1) / kBaseTok * hkv;
    ProduceArgs a{bt_base, bt_res, pos0, (int32_t)n, hidden, hkv, n_shrink,
                  static_cast<const uint16_t *>(x), static_cast<const uint16_t *>(k_raw), static_cast<const uint16_t *>(v),
                  r > 0 ? static_cast<const uint16_t *>(lora_a) : nullptr, rope_cos, rope_sin,
                  static_cast<uint16_t *>(base_kv), static_cast<uint16_t *>(res_kv)};
    const dim3 grid((unsigned)(n_shrink + n_base));
    hipStream_t st = static_cast<hipStream_t>(stream);
    switch (r) {
    case 0: hipLaunchKernelGGL(produce_kernel<0>, grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL(produce_kernel<8>, grid, dim3(256), 0, st, a); break;
    case 16: hipLaunchKernelGGL(produce_kernel<16>, grid, dim3(256), 0, st, a); break;
    case 32: hipLaunchKernelGGL(produce_kernel<32>, grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL(produce_kernel<64>, grid, dim3(256), 0, st, a); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fkv::fail(FKV_ERR_HIP, std::string("fkv_produce_tokens: ") + hipGetErrorString(e));
    return FKV_OK;
}

}  // extern "C"
