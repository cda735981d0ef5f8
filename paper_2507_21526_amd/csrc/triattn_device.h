// Device helpers shared by the tile kernels of libtriattn.so (forward passes
// and the region-contribution probe): vector types, the global -> LDS copy,
// barriers and waits.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace triattn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Lambdas of the tile kernels are always inlined: the step loops call
// several of them more than once and must not turn them into calls.
#define TA_INLINE __attribute__((always_inline))

// Register fences: an empty volatile asm that reads and rewrites a value, so
// the computation producing it cannot be moved past this point (side-effect
// free arithmetic could otherwise be sunk across a phase boundary).
__device__ __forceinline__ void fence_regs(bf16x8 &x)
{
    asm volatile("" : "+v"(x));
}
__device__ __forceinline__ void fence_regs(float &x)
{
    asm volatile("" : "+v"(x));
}
__device__ __forceinline__ void fence_regs(double &x)
{
    asm volatile("" : "+v"(x));
}

// One wave-wide 16-byte-per-lane copy from global memory straight into LDS
// (lane l lands at lds_addr + 16 l).  Issued from inline assembly so that the
// compiler does not serialise it against unrelated LDS reads (the copy
// targets another LDS stage; barriers order it against the readers of its
// own stage): completion is tracked explicitly with vmcnt waits.  The LDS
// address is bound to M0 through the operand constraint, so the compiler
// writes M0 itself (one scalar add per copy) and knows its value; the nop
// is the wait state between that write and the copy reading it.  Compiler
// waits on its own loads stay correct beside these copies: a wait for
// vmcnt <= n then also counts the copies, which only makes it stricter.
__device__ __forceinline__ void copy_to_lds16(const void *gbase, uint32_t lane_byte_off,
                                              uint32_t lds_addr)
{
    asm volatile("s_nop 0\n\t"
                 "global_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(lane_byte_off), "s"(gbase), "{m0}"(lds_addr));
}

// A burst of N (2 or 4) such copies into consecutive 1 KB blocks of LDS
// from lds_addr on, with one M0 write and one wait state for all of them:
// copy i uses the instruction offset i KB, which the hardware adds to both
// the global and the LDS address, so its lane offset is its byte offset in
// global memory minus i KB (never negative for the tiles copied here).
template <int N>
__device__ __forceinline__ void copy_burst_to_lds16(const void *gbase, const uint32_t (&off)[N],
                                                    uint32_t lds_addr)
{
    static_assert(N == 2 || N == 4, "bursts of two or four copies");
    if constexpr (N == 4)
        asm volatile("s_nop 0\n\t"
                     "global_load_lds_dwordx4 %0, %4\n\t"
                     "global_load_lds_dwordx4 %1, %4 offset:1024\n\t"
                     "global_load_lds_dwordx4 %2, %4 offset:2048\n\t"
                     "global_load_lds_dwordx4 %3, %4 offset:3072"
                     :
                     : "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "s"(gbase),
                       "{m0}"(lds_addr));
    else
        asm volatile("s_nop 0\n\t"
                     "global_load_lds_dwordx4 %0, %2\n\t"
                     "global_load_lds_dwordx4 %1, %2 offset:1024"
                     :
                     : "v"(off[0]), "v"(off[1]), "s"(gbase), "{m0}"(lds_addr));
}

// Workgroup barrier without a memory fence: this wave's LDS reads are
// complete (lgkmcnt 0); copies into LDS are synchronised by vmcnt waits.
__device__ __forceinline__ void barrier_no_fence()
{
    asm volatile("" ::: "memory");       // no compiler motion of memory ops
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n) for a run-time n (small): the count is an immediate.
__device__ __forceinline__ void wait_vmcnt(int n)
{
    // expcnt and lgkmcnt fields left at their maximum (no wait on them)
    switch (n) {
    case 0: __builtin_amdgcn_s_waitcnt(0x0f70); break;
    case 1: __builtin_amdgcn_s_waitcnt(0x0f71); break;
    case 2: __builtin_amdgcn_s_waitcnt(0x0f72); break;
    case 3: __builtin_amdgcn_s_waitcnt(0x0f73); break;
    case 4: __builtin_amdgcn_s_waitcnt(0x0f74); break;
    case 5: __builtin_amdgcn_s_waitcnt(0x0f75); break;
    case 6: __builtin_amdgcn_s_waitcnt(0x0f76); break;
    case 7: __builtin_amdgcn_s_waitcnt(0x0f77); break;
    default: __builtin_amdgcn_s_waitcnt(0x0f78); break;
    }
}

// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

}  // namespace triattn
