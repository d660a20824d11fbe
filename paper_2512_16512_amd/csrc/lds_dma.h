// Direct global -> LDS copies shared by the kernel families.
//
// gfx950 buffer loads with the `lds` modifier write their data straight into
// LDS (no register staging): lane i's bytes land at LDS address
// M0 + size*i.  Reads at a buffer offset past the buffer's record count
// return zero, which the kernels use for edge and zero-padding handling.
#pragma once

#include <hip/hip_runtime.h>

namespace xtc {

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer resource of a raw (unstructured) buffer: base address, no stride,
// `bytes` records; word 3 holds the gfx9 default data format.  Reads at an
// offset with offset + size > bytes return zero.
__device__ __forceinline__ i32x4 make_rsrc(const void *base, int bytes) {
    const unsigned long long a = reinterpret_cast<unsigned long long>(base);
    i32x4 r;
    r[0] = (int)(unsigned)(a & 0xffffffffull);
    r[1] = (int)(unsigned)((a >> 32) & 0xffffull);
    r[2] = bytes;
    r[3] = 0x00020000;
    return r;
}

// One 16-byte-per-lane copy global -> LDS: lane i's 16 bytes at buffer offset
// `voffset` land at LDS byte `lds_addr + 16*i`.  Written as inline assembly
// so that the compiler does not treat every later LDS read as dependent on
// every copy in flight (the completion of these copies is tracked with
// explicit vmcnt waits instead).  M0 carries the LDS base; one wait state
// separates its write from the copy.
__device__ __forceinline__ void dma16(const i32x4 &rsrc, unsigned lds_addr, int voffset) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voffset), "s"(rsrc)
        : "memory", "m0");
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ unsigned lds_address(const void *p) {
    return (unsigned)reinterpret_cast<unsigned long long>(
        (const __attribute__((address_space(3))) unsigned char *)(p));
}

// s_waitcnt on the vector-memory counter only (gfx9 encoding: vmcnt in bits
// 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// wait_vmcnt<N> that also waits for every LDS read of this wave (lgkmcnt 0).
// Used in front of a barrier that frees a ring slot: the reads of the slot
// have then completed, not only been issued, before any wave's copies into
// the slot start.
template <int N>
__device__ __forceinline__ void wait_vmcnt_and_lds() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

constexpr int kOOB = 0x7FFFFFF0;  // buffer offset beyond any operand (spans are < 2^31 - 1)

// 4-byte-per-lane variant of dma16 (lane i's dword lands at lds_addr + 4*i).
__device__ __forceinline__ void dma4(const i32x4 &rsrc, unsigned lds_addr, int voffset) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dword %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voffset), "s"(rsrc)
        : "memory", "m0");
}

// dma4 with a wave-uniform byte offset `soffset` added to every lane's
// address.  A lane whose `voffset` is past the end of the buffer still reads
// zero (the sum stays below 2^32 for soffset < 2^31 - 16).
__device__ __forceinline__ void dma4_so(const i32x4 &rsrc, unsigned lds_addr, int voffset,
                                        int soffset) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dword %1, %2, %3 offen lds"
        :
        : "s"(lds_addr), "v"(voffset), "s"(rsrc), "s"(soffset)
        : "memory", "m0");
}

}  // namespace xtc
