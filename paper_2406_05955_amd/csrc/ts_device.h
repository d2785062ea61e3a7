// Device-side helpers for the gfx950 kernels: 16-byte weight chunks, the
// fp32 / bf16 unpacking and wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ts {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Weight element types: float (4 per 16-byte chunk) or bfloat16 bit
// patterns stored as uint16_t (8 per chunk).
template <typename WT>
struct WTraits;
template <>
struct WTraits<float> {
    static constexpr int CE = 4;
};
template <>
struct WTraits<uint16_t> {
    static constexpr int CE = 8;
};

// Streaming 16-byte load of weights that are read once per call: the
// non-temporal hint keeps them from displacing x, the partial sums and the
// index lists in L2.
__device__ __forceinline__ u32x4 ld_stream(const void *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ u32x4 ld_cached(const void *p) { return *reinterpret_cast<const u32x4 *>(p); }

// Unpack one 16-byte chunk to fp32.  bf16 element 2m sits in the low half
// of 32-bit word m; its fp32 value is that half shifted into the top.
template <typename WT>
__device__ __forceinline__ void unpack(const u32x4 v, float *f);

template <>
__device__ __forceinline__ void unpack<float>(const u32x4 v, float *f) {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
}

template <>
__device__ __forceinline__ void unpack<uint16_t>(const u32x4 v, float *f) {
    f[0] = __uint_as_float(v.x << 16);
    f[1] = __uint_as_float(v.x & 0xffff0000u);
    f[2] = __uint_as_float(v.y << 16);
    f[3] = __uint_as_float(v.y & 0xffff0000u);
    f[4] = __uint_as_float(v.z << 16);
    f[5] = __uint_as_float(v.z & 0xffff0000u);
    f[6] = __uint_as_float(v.w << 16);
    f[7] = __uint_as_float(v.w & 0xffff0000u);
}

// Butterfly sum over the 64 lanes of a wave.  Every lane ends with the same
// bits: at each step both partners add the same two values.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

__device__ __forceinline__ int lane_prefix(uint64_t mask, int lane) {
    return __popcll(mask & ((1ull << lane) - 1ull));
}

}  // namespace ts
