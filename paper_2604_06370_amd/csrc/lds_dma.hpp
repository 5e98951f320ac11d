// Direct global-to-LDS copies and explicit LDS reads for gfx950, shared by the
// attention kernels.
//
// A copy (buffer_load ... lds) moves 16 bytes per lane from a buffer resource straight
// into LDS: lane i's bytes land at dst + 16 i, no registers involved, and the copy counts
// as an outstanding vector-memory operation of the issuing wave until it has landed.  The
// compiler does not see which LDS bytes such a copy writes, so LDS that copies write is
// read with the explicit reads below (each group of reads waits for itself), and the
// hand-over is a counted vmcnt wait followed by a barrier.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"

namespace fkvk {

typedef __attribute__((address_space(3))) u32x4 LdsU32x4;
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

__device__ void raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) uint32_t *lds, int size, int voffset,
                                    int soffset, int offset, int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

// Buffer resource over `bytes` bytes from `base` (wave-uniform); offsets past the end
// read as zero.
__device__ __forceinline__ i32x4 block_rsrc(uint64_t base, int bytes) {
    i32x4 r;
    r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)base);
    r.y = __builtin_amdgcn_readfirstlane((int)(uint32_t)(base >> 32));
    r.z = bytes;       // bytes addressable through the resource
    r.w = 0x00020000;  // raw 32-bit data format
    return r;
}
// Cache policy of a load (the instruction's cache-policy bits): kCacheStream marks data read
// once (non-temporal), so that it displaces less of what other workgroups re-read.
constexpr int kCacheDefault = 0, kCacheStream = 2;
// 16-byte buffer load into registers.
__device__ i32x4 raw_buffer_load_b128(i32x4 rsrc, int voffset, int soffset, int aux) __asm("llvm.amdgcn.raw.buffer.load.v4i32");
template <int POLICY = kCacheDefault>
__device__ __forceinline__ u32x4 buf_load16(i32x4 rsrc, int voff) {
    return __builtin_bit_cast(u32x4, raw_buffer_load_b128(rsrc, voff, 0, POLICY));
}
// Copy: lane i's 16 bytes at byte offset voff of the resource land at dst + 16 i.  The
// instruction's immediate offset stays 0 (it would shift the LDS destination as well).
template <int POLICY = kCacheDefault>
__device__ __forceinline__ void lds_dma16(i32x4 rsrc, int voff, LdsU32x4 *dst) {
    raw_buffer_load_lds(rsrc, reinterpret_cast<__attribute__((address_space(3))) uint32_t *>(dst), 16, voff, 0, 0, POLICY);
}

// LDS byte address of an LDS location.
__device__ __forceinline__ uint32_t lds_addr(const LdsU32x4 *p) {
    return (uint32_t)reinterpret_cast<uintptr_t>(p);
}
// Four 16-byte LDS reads at addr, addr + 1 KB, + 2 KB, + 3 KB (addr: this lane's byte
// address), completed before the group ends.
__device__ __forceinline__ void lds_read4(uint32_t addr, u32x4 (&out)[4]) {
    asm volatile(
        "ds_read_b128 %0, %4\n\t"
        "ds_read_b128 %1, %4 offset:1024\n\t"
        "ds_read_b128 %2, %4 offset:2048\n\t"
        "ds_read_b128 %3, %4 offset:3072\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(out[0]), "=&v"(out[1]), "=&v"(out[2]), "=&v"(out[3])  // early clobber: the address stays intact
        : "v"(addr)
        : "memory");
}
// Two 16-byte LDS reads at addr and addr + 1 KB.
__device__ __forceinline__ void lds_read2(uint32_t addr, u32x4 (&out)[2]) {
    asm volatile(
        "ds_read_b128 %0, %2\n\t"
        "ds_read_b128 %1, %2 offset:1024\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(out[0]), "=&v"(out[1])
        : "v"(addr)
        : "memory");
}
// Eight 16-byte LDS reads: four at addr0 + 0/1/2/3 KB, four at addr1 + 0/1/2/3 KB.
__device__ __forceinline__ void lds_read8(uint32_t addr0, uint32_t addr1, u32x4 (&o0)[4], u32x4 (&o1)[4]) {
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:1024\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\t"
        "ds_read_b128 %3, %8 offset:3072\n\t"
        "ds_read_b128 %4, %9\n\t"
        "ds_read_b128 %5, %9 offset:1024\n\t"
        "ds_read_b128 %6, %9 offset:2048\n\t"
        "ds_read_b128 %7, %9 offset:3072\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o0[0]), "=&v"(o0[1]), "=&v"(o0[2]), "=&v"(o0[3]), "=&v"(o1[0]), "=&v"(o1[1]), "=&v"(o1[2]), "=&v"(o1[3])
        : "v"(addr0), "v"(addr1)
        : "memory");
}

// Two 16-byte LDS writes (addr0 <- v0, addr1 <- v1), completed before the group ends.
__device__ __forceinline__ void lds_write2(uint32_t addr0, const u32x4 &v0, uint32_t addr1, const u32x4 &v1) {
    asm volatile(
        "ds_write_b128 %0, %1\n\t"
        "ds_write_b128 %2, %3\n\t"
        "s_waitcnt lgkmcnt(0)"
        :
        : "v"(addr0), "v"(v0), "v"(addr1), "v"(v1)
        : "memory");
}

// Compiler-visible forms of the reads above (same addresses and results): the compiler
// schedules these loads and their waits among the surrounding products.  Only for LDS that
// no copy in flight writes, read between barriers that LDS accesses cannot cross
// (lds_fence_barrier).  CV selects them, else the explicit reads.
__device__ __forceinline__ u32x4 lds_load(uint32_t addr) {
    return *reinterpret_cast<const __attribute__((address_space(3))) u32x4 *>((uintptr_t)addr);
}
template <bool CV>
__device__ __forceinline__ void lds_get2(uint32_t addr, u32x4 (&out)[2]) {
    if constexpr (CV) {
        out[0] = lds_load(addr);
        out[1] = lds_load(addr + 1024);
    } else {
        lds_read2(addr, out);
    }
}
template <bool CV>
__device__ __forceinline__ void lds_get4(uint32_t addr, u32x4 (&out)[4]) {
    if constexpr (CV) {
#pragma unroll
        for (int i = 0; i < 4; ++i) out[i] = lds_load(addr + 1024 * i);
    } else {
        lds_read4(addr, out);
    }
}
template <bool CV>
__device__ __forceinline__ void lds_get8(uint32_t addr0, uint32_t addr1, u32x4 (&o0)[4], u32x4 (&o1)[4]) {
    if constexpr (CV) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o0[i] = lds_load(addr0 + 1024 * i);
            o1[i] = lds_load(addr1 + 1024 * i);
        }
    } else {
        lds_read8(addr0, addr1, o0, o1);
    }
}
// Workgroup barrier after this wave's LDS accesses have completed; the compiler moves no
// memory access across it.
__device__ __forceinline__ void lds_fence_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

}  // namespace fkvk
