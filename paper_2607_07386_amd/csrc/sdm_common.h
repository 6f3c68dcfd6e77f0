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

// Gate producers of Sec. 3.1 step 2 from their pre-activations: the forget gate
// alpha = exp(-A softplus(a + b_dt)) and the input gate beta = sigma(b), with A
// and b_dt per head.  softplus is written so that neither branch overflows.
__device__ __forceinline__ float sdm_softplus(float z) {
    return z > 0.f ? z + log1pf(expf(-z)) : log1pf(expf(z));
}
__device__ __forceinline__ float sdm_sigmoid(float z) { return 1.f / (1.f + expf(-z)); }
// (al, be) hold the stored gates, or the pre-activations when A != NULL; on
// return they are the gates the recurrence uses.
__device__ __forceinline__ void sdm_gates_of(const float* A, const float* bdt, int head, float& al, float& be) {
    if (A) {
        al = expf(-A[head] * sdm_softplus(al + bdt[head]));
        be = sdm_sigmoid(be);
    }
}
// log alpha of the gates above, without forming alpha (the chunked form's decays)
__device__ __forceinline__ float sdm_log_alpha(const float* A, const float* bdt, int head, float a_pre) {
    return -A[head] * sdm_softplus(a_pre + bdt[head]);
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

// Wave mask of the lanes whose index has bit M set (M a power of two; 0 for
// M >= 64), and the same as a per-lane condition: the mask is a constant, so
// the condition costs no vector instruction.
template <int M>
__host__ __device__ constexpr unsigned long long lanes_with_bit() {
    unsigned long long m = 0ull;
    for (int l = 0; l < 64; ++l)
        if (l & M) m |= 1ull << l;
    return m;
}
template <unsigned long long MASK>
__device__ __forceinline__ bool lane_in() {
    return __builtin_amdgcn_inverse_ballot_w64(MASK);
}

// Value of lane (this lane ^ M) without going through LDS: DPP row/quad
// permutes for M <= 8, the gfx950 permlane swaps for 16 and 32.
template <int M>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v) {
    if constexpr (M == 1) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
    } else if constexpr (M == 2) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
    } else if constexpr (M == 4) {
        const int h = __builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, false);     // row_half_mirror: i ^ 7
        return (uint32_t)__builtin_amdgcn_mov_dpp(h, 0x1B, 0xF, 0xF, false);        // quad_perm [3,2,1,0]: ^ 3
    } else if constexpr (M == 8) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false);  // row_ror:8
    } else if constexpr (M == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return lane_in<lanes_with_bit<16>()>() ? r[0] : r[1];
    } else {
        static_assert(M == 32, "xor distance must be a power of two below 64");
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return lane_in<lanes_with_bit<32>()>() ? r[0] : r[1];
    }
}
// Same for a distance known only after unrolling (folds to one case).
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t v, int m) {
    switch (m) {
        case 1: return xor_lane<1>(v);
        case 2: return xor_lane<2>(v);
        case 4: return xor_lane<4>(v);
        case 8: return xor_lane<8>(v);
        case 16: return xor_lane<16>(v);
        case 32: return xor_lane<32>(v);
        default: return (uint32_t)__shfl_xor((int)v, m, SDM_WAVE);
    }
}
__device__ __forceinline__ float xor_lane_f(float v, int m) {
    return __uint_as_float(xor_lane_u32(__float_as_uint(v), m));
}
__device__ __forceinline__ float shfl_xor_f(float v, int m) { return xor_lane_f(v, m); }

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

template <int M>
__device__ __forceinline__ float xor_lane_ff(float v) {
    return __uint_as_float(xor_lane<M>(__float_as_uint(v)));
}
// Butterfly reductions over the wave (every lane receives the result).
template <int M = 32>
__device__ __forceinline__ float wave_sum(float v) {
    v += xor_lane_ff<M>(v);
    if constexpr (M > 1) return wave_sum<M / 2>(v);
    else return v;
}
template <int M = 32>
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, xor_lane_ff<M>(v));
    if constexpr (M > 1) return wave_max<M / 2>(v);
    else return v;
}
template <int M = 32>
__device__ __forceinline__ int wave_min_i(int v) {
    v = min(v, (int)xor_lane<M>((uint32_t)v));
    if constexpr (M > 1) return wave_min_i<M / 2>(v);
    else return v;
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
    r.x = xor_lane_f(v.x, m);
    r.y = xor_lane_f(v.y, m);
    r.z = xor_lane_f(v.z, m);
    r.w = xor_lane_f(v.w, m);
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

// Workgroup -> (column group, stream) for the scans, launched as a 1-D grid of
// groups x S workgroups.  Workgroups go to the 8 XCDs round-robin by linear
// id.  XCD_LOCAL (and S a multiple of 8): the groups of one stream get ids
// congruent mod 8, so they run on one XCD and read the stream's per-token
// records through one L2 (measured: the backward, 4 groups per stream, gains
// about 4%; the forward, 2 groups, loses about 1.5%).  Otherwise the groups of
// a stream are consecutive.
template <bool XCD_LOCAL>
__device__ __forceinline__ void scan_wg_coords(int groups, int& group, int& stream) {
    const int L = blockIdx.x;
    const int S = gridDim.x / groups;
    if (XCD_LOCAL && S % 8 == 0) {
        const int idx = L >> 3;
        stream = (idx / groups) * 8 + (L & 7);
        group = idx % groups;
    } else {
        stream = L / groups;
        group = L % groups;
    }
}

// Wait for outstanding LDS operations only (vmcnt and expcnt left at their maxima).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xc07f); }
