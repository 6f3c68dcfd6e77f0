// Shared device helpers for the SDM kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SDM_WAVE 64

typedef __bf16 sdm_bf16x8 __attribute__((ext_vector_type(8)));
typedef float sdm_f32x4 __attribute__((ext_vector_type(4)));

// Input element types.  bf16 is carried as its raw 16-bit pattern.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float((uint32_t)x.bits << 16); }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Load 4 consecutive elements (8-byte aligned for bf16, 16-byte for fp32) as fp32.
__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4(const bf16_t* p) {
    uint2 w = *reinterpret_cast<const uint2*>(p);
    return make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
}

// Monotone map of fp32 to uint32 (larger float -> larger key); -0 maps like +0.
__device__ __forceinline__ uint32_t ord_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_to_float(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (SDM_WAVE - 1); }

__device__ __forceinline__ int popc64(unsigned long long m) { return __popcll(m); }

// Number of set bits of m in lanes strictly below this lane.
__device__ __forceinline__ int mbcnt64(unsigned long long m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, SDM_WAVE); }

__device__ __forceinline__ float4 shfl_xor_f4(float4 v, int m) {
    return make_float4(__shfl_xor(v.x, m, SDM_WAVE), __shfl_xor(v.y, m, SDM_WAVE),
                       __shfl_xor(v.z, m, SDM_WAVE), __shfl_xor(v.w, m, SDM_WAVE));
}

__device__ __forceinline__ float4 f4add(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
__device__ __forceinline__ float4 f4sub(float4 a, float4 b) {
    return make_float4(a.x - b.x, a.y - b.y, a.z - b.z, a.w - b.w);
}
__device__ __forceinline__ float4 f4scale(float s, float4 a) {
    return make_float4(s * a.x, s * a.y, s * a.z, s * a.w);
}
// a + s*b with a fused multiply-add per element
__device__ __forceinline__ float4 f4fma(float s, float4 b, float4 a) {
    return make_float4(fmaf(s, b.x, a.x), fmaf(s, b.y, a.y), fmaf(s, b.z, a.z), fmaf(s, b.w, a.w));
}
__device__ __forceinline__ float f4dot(float4 a, float4 b) {
    return fmaf(a.x, b.x, fmaf(a.y, b.y, fmaf(a.z, b.z, a.w * b.w)));
}
__device__ __forceinline__ float4 f4zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, SDM_WAVE);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, SDM_WAVE));
    return v;
}
__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v = min(v, __shfl_xor(v, m, SDM_WAVE));
    return v;
}

// Clang vector of 4 floats: elementwise arithmetic, kept in registers.
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));
typedef unsigned int u2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ v4f ld4(const float* p) { return *reinterpret_cast<const v4f*>(p); }
__device__ __forceinline__ void st4(float* p, v4f v) { *reinterpret_cast<v4f*>(p) = v; }
__device__ __forceinline__ v4f ld4v(const float* p) { return *reinterpret_cast<const v4f*>(p); }
__device__ __forceinline__ v4f ld4v(const bf16_t* p) {
    const uint2 w = *reinterpret_cast<const uint2*>(p);
    v4f r;
    r.x = bf16_lo(w.x);
    r.y = bf16_hi(w.x);
    r.z = bf16_lo(w.y);
    r.w = bf16_hi(w.y);
    return r;
}
__device__ __forceinline__ v4f v4zero() { return v4f{0.f, 0.f, 0.f, 0.f}; }
__device__ __forceinline__ v4f v4fma(float s, v4f b, v4f a) {
    v4f r;
    r.x = fmaf(s, b.x, a.x);
    r.y = fmaf(s, b.y, a.y);
    r.z = fmaf(s, b.z, a.z);
    r.w = fmaf(s, b.w, a.w);
    return r;
}
__device__ __forceinline__ float v4dot(v4f a, v4f b) {
    return fmaf(a.x, b.x, fmaf(a.y, b.y, fmaf(a.z, b.z, a.w * b.w)));
}
__device__ __forceinline__ v4f v4shfl_xor(v4f v, int m) {
    v4f r;
    r.x = __shfl_xor(v.x, m, SDM_WAVE);
    r.y = __shfl_xor(v.y, m, SDM_WAVE);
    r.z = __shfl_xor(v.z, m, SDM_WAVE);
    r.w = __shfl_xor(v.w, m, SDM_WAVE);
    return r;
}
__device__ __forceinline__ v4f v4sel(bool c, v4f a, v4f b) {
    v4f r;
    r.x = c ? a.x : b.x;
    r.y = c ? a.y : b.y;
    r.z = c ? a.z : b.z;
    r.w = c ? a.w : b.w;
    return r;
}

// Wait for outstanding LDS operations only (vmcnt and expcnt left at their maxima).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xc07f); }
