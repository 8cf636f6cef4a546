// tbn_dma.h -- LDS-DMA helpers shared by the gfx950 GEMM kernels: raw buffer resources,
// buffer loads that write straight into LDS (issued from inline assembly so that the
// kernels keep control of their vmcnt waits), and explicit vmcnt waits.
//
// The compiler does not see these loads; a kernel that uses them issues no other vector
// memory loads inside its pipelined loop and waits for them with wait_vmcnt().  M0 is
// written by the DMA helpers; nothing else in these kernels uses M0.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tbn {

typedef int v4i __attribute__((ext_vector_type(4)));

// Buffer resource for raw (unstructured) buffer loads of `bytes` bytes at `base`.
__device__ __forceinline__ v4i make_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    v4i r;
    r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r.y = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xFFFFu));
    r.z = __builtin_amdgcn_readfirstlane((int)bytes);
    r.w = 0x00020000;
    return r;
}

// One LDS-DMA: lane i's 16 (or 4) bytes at byte `voff` of the buffer land at LDS
// address lds + 16*i (4*i).  An offset beyond the buffer yields zeros.  `lds` must be the
// same in every active lane (it is read from the first one into M0).
__device__ __forceinline__ void dma_b128(v4i rsrc, uint32_t lds, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(rsrc)
                 : "memory");
}
__device__ __forceinline__ void dma_b32(v4i rsrc, uint32_t lds, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(lds), "v"(voff), "s"(rsrc)
                 : "memory");
}

// s_waitcnt vmcnt(n), 0 <= n < 32 (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt and
// lgkmcnt left at their maxima); larger n waits for everything.
__device__ __forceinline__ void wait_vmcnt(int n) {
    switch (n) {
        case 0: __builtin_amdgcn_s_waitcnt(0x0F70); break;
        case 1: __builtin_amdgcn_s_waitcnt(0x0F71); break;
        case 2: __builtin_amdgcn_s_waitcnt(0x0F72); break;
        case 3: __builtin_amdgcn_s_waitcnt(0x0F73); break;
        case 4: __builtin_amdgcn_s_waitcnt(0x0F74); break;
        case 5: __builtin_amdgcn_s_waitcnt(0x0F75); break;
        case 6: __builtin_amdgcn_s_waitcnt(0x0F76); break;
        case 7: __builtin_amdgcn_s_waitcnt(0x0F77); break;
        case 8: __builtin_amdgcn_s_waitcnt(0x0F78); break;
        case 9: __builtin_amdgcn_s_waitcnt(0x0F79); break;
        case 10: __builtin_amdgcn_s_waitcnt(0x0F7A); break;
        case 11: __builtin_amdgcn_s_waitcnt(0x0F7B); break;
        case 12: __builtin_amdgcn_s_waitcnt(0x0F7C); break;
        case 13: __builtin_amdgcn_s_waitcnt(0x0F7D); break;
        case 14: __builtin_amdgcn_s_waitcnt(0x0F7E); break;
        case 15: __builtin_amdgcn_s_waitcnt(0x0F7F); break;
        case 16: __builtin_amdgcn_s_waitcnt(0x4F70); break;
        case 17: __builtin_amdgcn_s_waitcnt(0x4F71); break;
        case 18: __builtin_amdgcn_s_waitcnt(0x4F72); break;
        case 19: __builtin_amdgcn_s_waitcnt(0x4F73); break;
        case 20: __builtin_amdgcn_s_waitcnt(0x4F74); break;
        case 21: __builtin_amdgcn_s_waitcnt(0x4F75); break;
        case 22: __builtin_amdgcn_s_waitcnt(0x4F76); break;
        case 23: __builtin_amdgcn_s_waitcnt(0x4F77); break;
        case 24: __builtin_amdgcn_s_waitcnt(0x4F78); break;
        case 25: __builtin_amdgcn_s_waitcnt(0x4F79); break;
        case 26: __builtin_amdgcn_s_waitcnt(0x4F7A); break;
        case 27: __builtin_amdgcn_s_waitcnt(0x4F7B); break;
        case 28: __builtin_amdgcn_s_waitcnt(0x4F7C); break;
        case 29: __builtin_amdgcn_s_waitcnt(0x4F7D); break;
        case 30: __builtin_amdgcn_s_waitcnt(0x4F7E); break;
        case 31: __builtin_amdgcn_s_waitcnt(0x4F7F); break;
        default: __builtin_amdgcn_s_waitcnt(0x0F70); break;
    }
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

}  // namespace tbn
