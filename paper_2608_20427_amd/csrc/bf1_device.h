// Device-side helpers shared by the forward and backward kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bf1 {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int KT = 64;  // keys (or query rows) per LDS tile
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int VMCNT0 = 0x0F70;  // s_waitcnt vmcnt(0) (expcnt, lgkmcnt unconstrained)

// LDS address (byte offset in the workgroup's LDS) of a shared-memory pointer.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const lds_void*)(p);
}

// Combine a value with the one held by the lane 32 apart (both lane halves
// hold the same query row).  v_permlane32_swap exchanges the halves in the
// vector ALU, with no LDS round trip; both halves get identical results.
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Buffer resource over `bytes` bytes from `base`: reads at byte offsets at or
// past the end return zero (the staging relies on it for rows past n).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t head_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             0x00020000);
}

// Direct buffer -> LDS load of 16 bytes per lane into the wave's 1 KB LDS
// segment (lane order); voff is the lane's byte offset inside the tile, soff
// the tile's byte offset inside the head.  (Compiler-visible form.)
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, void* lds_segment,
                                           uint32_t voff, uint32_t soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds_segment, 16, voff, soff, 0, 0);
}

// The same direct load (16 or 4 bytes per lane, SIZE) issued through inline
// assembly, so that the compiler does not treat every later LDS read as
// possibly aliasing an in-flight load and wait for all of them (vmcnt(0))
// before it; kernels using this form order these loads against their readers
// themselves, with explicit vmcnt waits and workgroup barriers.  The
// instruction has no register results (the data goes to LDS) and reads its
// operands at issue.  M0 holds the LDS destination; the compiler sets M0
// itself before each of its own uses, so overwriting it here is safe (hence
// the silenced warning).  One wait state separates the M0 write from the load.
template <int SIZE>
__device__ __forceinline__ void load_lds_async(__amdgpu_buffer_rsrc_t r, void* lds_segment,
                                               uint32_t voff, uint32_t soff) {
    static_assert(SIZE == 16 || SIZE == 4, "dwordx4 or dword");
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_addr(lds_segment));
    soff = __builtin_amdgcn_readfirstlane(soff);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    if constexpr (SIZE == 16)
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                     :
                     : "s"(m0), "v"(voff), "s"(r), "s"(soff)
                     : "memory", "m0");
    else
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                     :
                     : "s"(m0), "v"(voff), "s"(r), "s"(soff)
                     : "memory", "m0");
#pragma clang diagnostic pop
}

// One 64-bit LDS transpose read (ds_read_b64_tr_b16) at byte address a; the
// compiler schedules it and its wait.
__device__ __forceinline__ u32x2 lds_read_tr16(uint32_t a) {
    return __builtin_bit_cast(
        u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                   reinterpret_cast<lds_s16x4*>(static_cast<uintptr_t>(a))));
}

}  // namespace bf1
