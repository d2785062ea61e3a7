// HBM probes: a streaming read that measures achievable bandwidth and a
// plain copy whose counter readings calibrate the traffic counters.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ts_device.h"
#include "ts_plan.h"
#include "ts_runtime.h"
#include "turbosparse.h"

namespace ts {

constexpr int kProbeBlocks = 4096;

// Block b reads the b-th contiguous slice with 16-byte streaming loads, four
// in flight per thread, and folds them into one float so nothing is elided.
__global__ __launch_bounds__(256) void probe_read(const u32x4 *__restrict__ src, size_t n16, float *__restrict__ sink) {
    const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const size_t b0 = blockIdx.x * per;
    const size_t b1 = b0 + per < n16 ? b0 + per : n16;
    unsigned acc = 0;
    for (size_t i = b0 + threadIdx.x; i < b1; i += 4 * 256) {
        u32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t k = i + (size_t)u * 256;
            v[u] = k < b1 ? __builtin_nontemporal_load(src + k) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    acc = (unsigned)wave_sum((float)(acc & 0xffu));
    if (threadIdx.x == 0) sink[blockIdx.x] = (float)acc;
}

__global__ __launch_bounds__(256) void probe_copy(const u32x4 *__restrict__ src, u32x4 *__restrict__ dst, size_t n16) {
    for (size_t i = blockIdx.x * (size_t)256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256)
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace ts

extern "C" {

ts_status ts_probe_read(const void *src, size_t bytes, float *sink, void *stream) {
    if (!src || !sink) return TS_ERR_NULL;
    if (bytes == 0 || bytes % 16 != 0) return TS_ERR_SHAPE;
    if (!ts::aligned16(src) || !ts::aligned4(sink)) return TS_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    ts::launch("probe_read", ts::probe_read, dim3(ts::kProbeBlocks), dim3(256), st,
               static_cast<const ts::u32x4 *>(src), bytes / 16, sink);
    return ts::check_launch("probe_read");
}

ts_status ts_probe_copy(const void *src, void *dst, size_t bytes, void *stream) {
    if (!src || !dst) return TS_ERR_NULL;
    if (bytes == 0 || bytes % 16 != 0) return TS_ERR_SHAPE;
    if (!ts::aligned16(src) || !ts::aligned16(dst)) return TS_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    ts::launch("probe_copy", ts::probe_copy, dim3(ts::kProbeBlocks), dim3(256), st,
               static_cast<const ts::u32x4 *>(src), static_cast<ts::u32x4 *>(dst), bytes / 16);
    return ts::check_launch("probe_copy");
}

}  // extern "C"
