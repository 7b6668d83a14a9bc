// Device-side helpers shared by the gfx950 kernels of the verification step.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define DSPARK_WAVE 64

namespace dspark {

// bfloat16 <-> fp32.  Widening is exact; narrowing rounds to nearest even
// (NaN stays NaN).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)0x7fc0;
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    __device__ __forceinline__ static float load(const float* p, int64_t i) { return p[i]; }
    __device__ __forceinline__ static void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    __device__ __forceinline__ static float load(const uint16_t* p, int64_t i) {
        return bf16_to_f32(p[i]);
    }
    __device__ __forceinline__ static void store(uint16_t* p, int64_t i, float v) {
        p[i] = f32_to_bf16(v);
    }
};

// Wave-wide reductions over 64 lanes (every lane gets the result).
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, DSPARK_WAVE));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, DSPARK_WAVE);
    return v;
}
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, DSPARK_WAVE);
    return v;
}

// Intra-wave LDS exchange: orders this wave's LDS writes before its later
// LDS reads (DS instructions of one wave execute in order; this stops the
// compiler from moving accesses across the point).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Workgroup barrier that orders LDS only: waits for this wave's LDS accesses
// (lgkmcnt) but leaves global loads in flight, so prefetched data keeps
// streaming across the barrier (a plain __syncthreads() waits for every
// outstanding global load as well).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Pointer into LDS (address space 3) from a 32-bit LDS byte address.
template <typename T>
__device__ __forceinline__ T* lds_ptr(uint32_t addr) {
    return (T*)(uintptr_t)addr;
}

}  // namespace dspark
