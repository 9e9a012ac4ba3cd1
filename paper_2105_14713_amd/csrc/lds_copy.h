// Buffer loads straight into LDS, and the waits and flag accesses that order
// them, shared by the kernels that stage operands with such copies.
#pragma once

#include "conv_common.h"

namespace onexn {

typedef int v4i32 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

constexpr int32_t kRawBufferFlags = 0x00020000;   // buffer resource word 3: 32-bit raw data
constexpr uint32_t kBufferOutOfRange = 0x7fffffffu;   // a byte offset past any buffer here

// Raw buffer resource over [p, p + bytes).  The hardware range-checks the
// vector offset (plus the instruction's immediate) against `bytes` and
// returns zeros beyond it; the scalar offset is added after that check.
// Callers therefore put every data-dependent offset in the vector offset, so
// that padding and ragged tails read zeros and no read leaves the buffer.
__device__ __forceinline__ v4i32 buffer_rsrc(const void* p, int32_t bytes) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    v4i32 r;
    r.x = __builtin_amdgcn_readfirstlane(int32_t(uint32_t(v)));
    r.y = __builtin_amdgcn_readfirstlane(int32_t(uint32_t(v >> 32) & 0xffff));
    r.z = __builtin_amdgcn_readfirstlane(bytes);
    r.w = kRawBufferFlags;
    return r;
}

// (m0 is named as clobbered for the reader; the compiler keeps nothing in it here.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// Copies from a buffer straight into LDS: lane i's 16 (or 4) bytes at byte
// offset voff + soff land at LDS address dst + 16 i (4 i).  Written as inline
// assembly so that the compiler, which cannot tell which LDS bytes such a copy
// writes, does not make every later LDS read wait for all outstanding copies;
// callers order the copies themselves with vm_wait.
__device__ __forceinline__ void copy16_to_lds(v4i32 rs, const lds_char* dst, int32_t voff, int32_t soff) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(uint32_t(uintptr_t(dst)));
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(m0), "v"(voff), "s"(rs), "s"(soff) : "memory", "m0");
}
__device__ __forceinline__ void copy4_to_lds(v4i32 rs, const lds_char* dst, int32_t voff, int32_t soff) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(uint32_t(uintptr_t(dst)));
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                 :: "s"(m0), "v"(voff), "s"(rs), "s"(soff) : "memory", "m0");
}
#pragma clang diagnostic pop

// Waits until at most K vector-memory instructions of this wave are
// outstanding; also a compiler barrier for memory accesses.
template <int K>
__device__ __forceinline__ void vm_wait() {
    static_assert(K >= 0 && K < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(K) : "memory");
}

// Relaxed LDS flag accesses (workgroup scope).
__device__ __forceinline__ int32_t lds_flag_load(const int32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_flag_store(int32_t* p, int32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Compiler-only barrier: no memory access moves across it.
__device__ __forceinline__ void fence_compiler() { asm volatile("" ::: "memory"); }

}  // namespace onexn
