// Device-side helpers shared by the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace oc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

constexpr int WAVE = 64;

// address-space views for global_load_lds (global source, LDS destination)
typedef __attribute__((address_space(3))) void *lds_vp;
typedef __attribute__((address_space(1))) void *glb_vp;

// s_waitcnt vmcnt(n) leaving the other counters alone (gfx9 encoding; n < 64)
#define OC_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))

// Workgroup barrier for loops that stage operands with global_load_lds.
// __syncthreads() is a release fence plus s_barrier, and the fence waits for
// every outstanding LDS-DMA load (vmcnt(0)), which would drain the prefetch
// ring at each step.  Here each wave has already waited (vmcnt) for its own
// loads of the stage being published; the barrier only needs this wave's
// LDS reads to have completed (lgkmcnt(0)) before other waves may overwrite
// what they read.  The memory clobber keeps the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ float bf2f(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ float ld(const float *p) { return *p; }
    static __device__ __forceinline__ void st(float *p, float v) { *p = v; }
};
template <> struct Elem<uint16_t> {
    static __device__ __forceinline__ float ld(const uint16_t *p) { return bf2f(*p); }
    static __device__ __forceinline__ void st(uint16_t *p, float v) { *p = f2bf(v); }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
    return v;
}

// (value, index) arg-max merge: larger value wins, smaller index on ties.
__device__ __forceinline__ void argmax_merge(float &v, int &i, float v2, int i2) {
    if (v2 > v || (v2 == v && (unsigned)i2 < (unsigned)i)) { v = v2; i = i2; }
}

// Raw buffer resources (stride 0): offsets at or past num_records bytes read
// as zero.  The LDS-destination buffer load is the LLVM intrinsic, bound by
// name; the fourth word selects 32-bit data on gfx950.
typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int BUF_RSRC_WORD3 = 0x00020000;
__device__ __forceinline__ i32x4 buffer_rsrc(const void *base, int num_bytes) {
    const unsigned long a = (unsigned long)base;
    i32x4 r;
    r.x = (int)(unsigned)(a & 0xFFFFFFFFul);
    r.y = (int)(unsigned)((a >> 32) & 0xFFFFul);
    r.z = num_bytes;
    r.w = BUF_RSRC_WORD3;
    return r;
}
__device__ void buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) void *lds, int size, int voffset,
                                int soffset, int offset, int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

// Order-preserving map of a float to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t float_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;   // -0 and +0 are the same value
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inverse of float_key (-0 comes back as +0).
__device__ __forceinline__ float key_float(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k ^ 0x80000000u) : ~k);
}

// (value, index) packed into 64 bits so that the unsigned maximum is the
// arg-max with the smallest index on ties: order-preserving value key high,
// inverted index low.  0 is below every packed pair and means "none".
__device__ __forceinline__ unsigned long long pack_argmax(float v, int i) {
    return ((unsigned long long)float_key(v) << 32) | (unsigned long long)(~(uint32_t)i);
}
__device__ __forceinline__ void unpack_argmax(unsigned long long p, float &v, int &i) {
    if (p == 0ull) {
        v = -INFINITY;
        i = -1;
        return;
    }
    v = key_float((uint32_t)(p >> 32));
    i = (int)~(uint32_t)p;
}

__host__ __device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace oc
