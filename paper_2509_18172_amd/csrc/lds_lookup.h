// Table lookups in LDS (subset-sum tables of the prefill paths): the LDS
// address of a pointer, and base + one byte of a register as a single
// byte-select (SDWA) add -- the compiler forms a shift, a mask and an add
// for the same expression.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace sbvr {

// LDS address of a pointer into the workgroup's LDS
__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// base + byte B of v
template <int B>
__device__ __forceinline__ uint32_t add_byte(uint32_t base, uint32_t v)
{
    uint32_t r;
    if constexpr (B == 0)
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
            : "=v"(r) : "v"(base), "v"(v));
    else if constexpr (B == 1)
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
            : "=v"(r) : "v"(base), "v"(v));
    else if constexpr (B == 2)
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
            : "=v"(r) : "v"(base), "v"(v));
    else
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
            : "=v"(r) : "v"(base), "v"(v));
    return r;
}

}  // namespace sbvr
