// Cache writes: copy-on-write page copies (Section 5.2) and scattering new tokens'
// bCache K/V and rCache C_K/C_V into their page slots.
//
// Page layouts (bf16): base page [2][Hkv][ps*d]; residual page [2][ps*r] with C_K as
// [ps][r] and C_V as [r][ps].  With ps = 16 and d = 128 the K and V blocks of one
// (page, head) are stored in the order in which the attention kernels' matrix-core
// fragments read them (one 16-byte load per lane, 1 KB per wave instruction):
//   K element (token t, dim d) at  (d/32)*512 + (t + 16*((d%16)/4))*8 + 4*((d%32)/16) + d%4
//   V element (token t, dim d) at  (d/32)*512 + (d%16 + 16*(t/4))*8 + 4*((d/16)%2) + t%4
// Other shapes use plain [ps][d] (K) and [d][ps] (V).
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
        const int64_t blk = (int64_t)a.ps * a.r;
        const int64_t page = 2 * blk;
        const uint16_t *src = a.res_kv + (int64_t)c.src * page;
        uint16_t *dst = a.res_kv + (int64_t)c.dst * page;
        for (int64_t e = threadIdx.x; e < page; e += blockDim.x) {
            const int64_t within = e % blk;
            const bool is_v = e >= blk;
            const int slot = is_v ? (int)(within % a.ps) : (int)(within / a.r);
            if (slot < n_valid) dst[e] = src[e];
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
        const int64_t blk = (int64_t)a.ps * a.r;
        uint16_t *pg = a.res_kv + (int64_t)page * 2 * blk;
        for (int e = threadIdx.x; e < a.r; e += blockDim.x) {
            pg[(int64_t)slot * a.r + e] = a.ck_src[j * a.r + e];
            pg[blk + (int64_t)e * a.ps + slot] = a.cv_src[j * a.r + e];
        }
    }
}

}  // namespace

extern "C" {

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
