// ls_device.h - device helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/ls_ffn.h"

namespace ls {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---- weight storage types: V elements per 16-byte vector, widened to fp32 -------------
template <ls_dtype T>
struct Wt;

template <>
struct Wt<LS_F32> {
    static constexpr int V = 4;
    static constexpr int kBytes = 4;
    __device__ static inline void widen(const u32x4& r, float* o) {
        o[0] = __uint_as_float(r.x);
        o[1] = __uint_as_float(r.y);
        o[2] = __uint_as_float(r.z);
        o[3] = __uint_as_float(r.w);
    }
    __device__ static inline float scalar(const void* p, size_t i) {
        return static_cast<const float*>(p)[i];
    }
    // element i of the array from the aligned 32-bit word holding it
    __device__ static inline float from_word(uint32_t w, size_t) { return __uint_as_float(w); }
};

__device__ inline float half_bits_to_float(unsigned int bits16) {
    unsigned short s = static_cast<unsigned short>(bits16);
    return static_cast<float>(__builtin_bit_cast(_Float16, s));
}

template <>
struct Wt<LS_F16> {
    static constexpr int V = 8;
    static constexpr int kBytes = 2;
    __device__ static inline void widen(const u32x4& r, float* o) {
        o[0] = half_bits_to_float(r.x & 0xffffu);
        o[1] = half_bits_to_float(r.x >> 16);
        o[2] = half_bits_to_float(r.y & 0xffffu);
        o[3] = half_bits_to_float(r.y >> 16);
        o[4] = half_bits_to_float(r.z & 0xffffu);
        o[5] = half_bits_to_float(r.z >> 16);
        o[6] = half_bits_to_float(r.w & 0xffffu);
        o[7] = half_bits_to_float(r.w >> 16);
    }
    __device__ static inline float scalar(const void* p, size_t i) {
        return half_bits_to_float(static_cast<const unsigned short*>(p)[i]);
    }
    __device__ static inline float from_word(uint32_t w, size_t i) {
        return half_bits_to_float((i & 1) ? w >> 16 : w & 0xffffu);
    }
};

template <>
struct Wt<LS_BF16> {
    static constexpr int V = 8;
    static constexpr int kBytes = 2;
    // bfloat16 is the upper half of a binary32: widening is a shift.
    __device__ static inline void widen(const u32x4& r, float* o) {
        o[0] = __uint_as_float(r.x << 16);
        o[1] = __uint_as_float(r.x & 0xffff0000u);
        o[2] = __uint_as_float(r.y << 16);
        o[3] = __uint_as_float(r.y & 0xffff0000u);
        o[4] = __uint_as_float(r.z << 16);
        o[5] = __uint_as_float(r.z & 0xffff0000u);
        o[6] = __uint_as_float(r.w << 16);
        o[7] = __uint_as_float(r.w & 0xffff0000u);
    }
    __device__ static inline float scalar(const void* p, size_t i) {
        return __uint_as_float(static_cast<unsigned int>(static_cast<const unsigned short*>(p)[i]) << 16);
    }
    __device__ static inline float from_word(uint32_t w, size_t i) {
        return __uint_as_float((i & 1) ? w & 0xffff0000u : w << 16);
    }
};

// Sum over the 64 lanes with DPP row operations (ALU-speed, no LDS crossbar); fixed order:
// pairs, quads, half-rows, rows, then rows 0+1 and 2+3, then all four; the total is
// taken from lane 63 and returned in every lane.
template <int CTRL, int ROW_MASK>
__device__ inline float dpp_add(float v) {
    const int t = __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xf, false);
    return v + __int_as_float(t);
}
__device__ inline float wave_sum_dpp(float v) {
    v = dpp_add<0xb1, 0xf>(v);   // quad_perm [1,0,3,2]
    v = dpp_add<0x4e, 0xf>(v);   // quad_perm [2,3,0,1]
    v = dpp_add<0x141, 0xf>(v);  // row_half_mirror
    v = dpp_add<0x140, 0xf>(v);  // row_mirror
    v = dpp_add<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_add<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// RMS prenorm scale of a vector of d elements whose squares sum to ss
__device__ inline float rms_scale(float ss, int d) { return 1.f / sqrtf(ss / (float)d + 1e-6f); }

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ inline u32x4 ld_stream(const u32x4* p) { return __builtin_nontemporal_load(p); }

// 16-byte streaming load through an explicitly global pointer (a global_load, never a
// flat load: flat loads also count against the LDS counter that LDS barriers wait on).
typedef const __attribute__((address_space(1))) u32x4* gvec_ptr;
__device__ inline u32x4 gload(const void* base, size_t byte_off) {
    return __builtin_nontemporal_load((gvec_ptr)((const char*)base + byte_off));
}

// Same, for a wave-uniform base and a 32-bit per-lane offset (scalar base + vector offset
// addressing: one offset register per lane instead of a 64-bit address per load).
__device__ inline u32x4 gload_u(const void* uniform_base, uint32_t byte_off) {
    const uint64_t b = (uint64_t)uniform_base;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const char* base = (const char*)(((uint64_t)hi << 32) | lo);
    return __builtin_nontemporal_load((gvec_ptr)(base + byte_off));
}

// One aligned 32-bit word at a wave-uniform base plus a per-lane byte offset.
typedef const __attribute__((address_space(1))) uint32_t* gword_ptr;
__device__ inline uint32_t gload_word(const void* uniform_base, uint32_t byte_off) {
    const uint64_t b = (uint64_t)uniform_base;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const char* base = (const char*)(((uint64_t)hi << 32) | lo);
    return *(gword_ptr)(base + byte_off);
}

// Order-preserving map of a binary32 score to uint32: NaN -> 0 (below every number),
// -0 -> +0, otherwise a monotone bit transform.  Ties are broken by the smaller index.
__device__ inline uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace ls
