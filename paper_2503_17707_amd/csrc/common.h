// Device-side helpers shared by the CDNA4 (gfx950) kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pb {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Storage-type traits: T is _Float16 or __bf16.
template <typename T> struct Mfma;

template <> struct Mfma<_Float16> {
    typedef f16x8 vec8;
    // D[16x16] += A[16x32] B[32x16]; lane l holds A row l%16, k = 8(l/16)..+7,
    // B column l%16, k = 8(l/16)..+7, and D rows 4(l/16)+i, column l%16.
    __device__ static inline f32x4 mma(vec8 a, vec8 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

template <> struct Mfma<__bf16> {
    typedef bf16x8 vec8;
    __device__ static inline f32x4 mma(vec8 a, vec8 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

template <typename T> __device__ inline float to_f32(T x) { return (float)x; }
template <typename T> __device__ inline T from_f32(float x) { return (T)x; }

// Reinterpret 16 bytes as the MFMA operand vector of T.
template <typename T> __device__ inline typename Mfma<T>::vec8 as_vec8(u32x4 v) {
    return __builtin_bit_cast(typename Mfma<T>::vec8, v);
}

// One 16-byte global -> LDS copy per lane (LDS-DMA, global_load_lds_dwordx4)
// from a wave-uniform 64-bit base (SGPRs) plus a 32-bit per-lane byte offset
// (voffset, saddr form: each lane's address costs one 32-bit offset): lane i
// writes bytes [16 i, 16 i + 16) after the wave-uniform LDS address lds_base.
// Issued from inline assembly so that the compiler, which would otherwise
// drain every outstanding load before the next LDS read, leaves the waiting
// to explicit s_waitcnt (wait_vmcnt); later compiler-placed waits only ever
// wait for more, never less.  M0 is saved and restored around the copy, so
// the compiler's own use of M0 is never disturbed, and one wait state
// separates the M0 write from the copy that reads it.
__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, uint32_t lds_base) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_base), "v"(voff), "s"(sbase)
        : "memory");
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Pack 4 floats into 4 storage-type values (8 bytes), round to nearest even.
template <typename T> __device__ inline u32x2 pack4(float a, float b, float c, float d) {
    T t[4] = {(T)a, (T)b, (T)c, (T)d};
    u32x2 r;
    __builtin_memcpy(&r, t, 8);
    return r;
}

// Barrier for exchanges through LDS only: the fences order LDS accesses
// (waiting for LDS, not for outstanding global stores as __syncthreads does).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ inline float wave_sum(float v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ inline float wave_max(float v) {
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// Timing of a span of launches by events taken from the kernels' own dispatch
// packets (no marker packets between kernels): while `stop` is set, the next
// launch records `start` as it begins and every launch records `stop` as it
// ends, so the span runs from the first kernel's start to the last one's end.
struct LaunchTiming {
    hipEvent_t start, stop;
};
extern thread_local LaunchTiming g_launch_timing;

}  // namespace pb

// Every kernel launch of the library (a plain launch unless a span is timed).
#define PB_LAUNCH(kernel, grid, block, shmem, stream, ...)                                  \
    do {                                                                                    \
        if (::pb::g_launch_timing.stop) {                                                   \
            const hipEvent_t pb_start_ = ::pb::g_launch_timing.start;                       \
            ::pb::g_launch_timing.start = nullptr;                                          \
            hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, pb_start_,            \
                                  ::pb::g_launch_timing.stop, 0, __VA_ARGS__);              \
        } else {                                                                            \
            hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);            \
        }                                                                                   \
    } while (0)
