// Global -> LDS DMA helpers shared by the convolution kernels (gfx950).
// Device-only; included inside no namespace.
#pragma once

#include <hip/hip_runtime.h>

namespace quan {
namespace {

// Raw buffer resource over [base, base + bytes): loads past the end return
// zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// LDS address of a __shared__ pointer, as the 32-bit value M0 takes.
__device__ __forceinline__ unsigned lds_addr(const void *p)
{
    return __builtin_amdgcn_readfirstlane(
        (unsigned)(size_t)(const __attribute__((address_space(3))) void *)p);
}

// One 16-byte chunk per lane from byte offset voff + soff of the buffer
// [base, base + bytes) straight into LDS at m0 + 16 * lane; offsets past the
// end land as zeros.  The compiler does not see this load: the issuing wave
// waits for it with s_waitcnt vmcnt, and no wave that issues these reads LDS
// (an outstanding LDS DMA holds back the issuing wave's own LDS reads).  The
// scalar operands go through readfirstlane so they sit in SGPRs even where
// the compiler kept a copy in a VGPR.
__device__ __forceinline__ void dma16(const void *base, unsigned bytes, unsigned voff, unsigned soff,
                                      unsigned m0)
{
    const unsigned long long b = (unsigned long long)base;
    const unsigned lo = __builtin_amdgcn_readfirstlane(unsigned(b));
    const unsigned hi = __builtin_amdgcn_readfirstlane(unsigned(b >> 32));
    const __amdgpu_buffer_rsrc_t rsrc =
        make_rsrc((const void *)(((unsigned long long)hi << 32) | lo), __builtin_amdgcn_readfirstlane(bytes));
    asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff),
                 "s"(rsrc), "s"(__builtin_amdgcn_readfirstlane(soff)), "s"(__builtin_amdgcn_readfirstlane(m0))
                 : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    // vmcnt[3:0] | expcnt (7) | lgkmcnt (15) | vmcnt[5:4]
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

}  // namespace
}  // namespace quan
