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

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float readlane_f32(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Sum over the 64 lanes of a wave with DPP moves inside each 16-lane row
// (quad swaps, then rotations by 4 and 8) and the four row sums read into
// scalars and added in a fixed order.  The result is wave-uniform and the
// same bits on every run.
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f32<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f32<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_f32<0x124>(v);  // row_ror:4
    v += dpp_f32<0x128>(v);  // row_ror:8
    return (readlane_f32(v, 0) + readlane_f32(v, 16)) + (readlane_f32(v, 32) + readlane_f32(v, 48));
}

// 16-byte chunk c of a row, or zeros when c is out of range, without a
// branch: the address is clamped to a valid chunk and the value masked, so a
// run of such loads issues back to back.
__device__ __forceinline__ u32x4 ld_stream_masked(const void *row, int c, int nch, int bytes_per_chunk, bool ok) {
    const int cc = c < nch ? c : nch - 1;
    u32x4 v = ld_stream(static_cast<const char *>(row) + (size_t)cc * bytes_per_chunk);
    const bool keep = ok && c < nch;
    return keep ? v : u32x4{0u, 0u, 0u, 0u};
}

// ld_stream_masked with the default cache policy (rows many workgroups read).
__device__ __forceinline__ u32x4 ld_cached_masked(const void *row, int c, int nch, int bytes_per_chunk, bool ok) {
    const int cc = c < nch ? c : nch - 1;
    u32x4 v = ld_cached(static_cast<const char *>(row) + (size_t)cc * bytes_per_chunk);
    const bool keep = ok && c < nch;
    return keep ? v : u32x4{0u, 0u, 0u, 0u};
}

// Same without the mask: chunks past the row end re-read its last chunk.
// Callers pair such chunks with zero x values, so they add nothing.
__device__ __forceinline__ u32x4 ld_stream_clamped(const void *row, int c, int nch) {
    const int cc = c < nch ? c : nch - 1;
    return ld_stream(static_cast<const char *>(row) + (size_t)cc * 16);
}

// Raw buffer resource over `bytes` bytes at `base` (gfx9 layout, 32-bit
// dword format).  Loads through it at offsets past `bytes` return zeros and
// touch no memory, so a masked load is an ordinary load at an out-of-range
// offset: no branch, no traffic.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

constexpr uint32_t kOutOfRange = 0x80000000u;  // offset past every resource used here

// Streaming (non-temporal) 16-byte load at byte offset `off` of resource `r`.
__device__ __forceinline__ u32x4 ld_buf_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
}

// The same with the default cache policy: for data that many workgroups
// read (it stays in L2 for the ones after the first).
__device__ __forceinline__ u32x4 ld_buf_cached(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

__device__ __forceinline__ f32x4 ld_f32x4_masked(const float *p, int i4, int n4) {
    const int ii = i4 < n4 ? i4 : n4 - 1;
    f32x4 v = *reinterpret_cast<const f32x4 *>(p + (size_t)ii * 4);
    return i4 < n4 ? v : f32x4{0.f, 0.f, 0.f, 0.f};
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// x = hi + lo as two bf16 parts (16 significant bits together), the matrix
// cores' operands for fp32-level products with bf16 weights.
__device__ __forceinline__ void split_hi_lo(float x, uint32_t &hi, uint32_t &lo) {
    hi = bf16_bits(x);
    lo = bf16_bits(x - __uint_as_float(hi << 16));
}

__device__ __forceinline__ int lane_prefix(uint64_t mask, int lane) {
    return __popcll(mask & ((1ull << lane) - 1ull));
}

}  // namespace ts
