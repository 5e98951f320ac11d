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

}  // extern "C"
