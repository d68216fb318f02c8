// Plain HBM streaming kernels used as measurement references: a copy of known size
// (calibrates the HBM byte counters against a kernel whose traffic is known exactly;
// dwordx4 accesses, grid-stride) and a read-only stream (the achievable read bandwidth on
// this device, reported next to the nominal peak: each workgroup reads one contiguous
// chunk with sixteen dwordx4 loads in flight per thread, the fastest of the simple read
// patterns measured on MI355X).
#include <hip/hip_runtime.h>

#include "../../include/monomoe.h"

#include <stdint.h>

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
constexpr int kDepth = 8;
constexpr int kBlock = 256;
constexpr int kGrid = 1024;

__global__ __launch_bounds__(kBlock) void stream_copy(const v4i* __restrict__ src, v4i* __restrict__ dst, size_t n16) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    for (; i + (kDepth - 1) * stride < n16; i += kDepth * stride) {
        v4i v[kDepth];
#pragma unroll
        for (int d = 0; d < kDepth; ++d) v[d] = src[i + d * stride];
#pragma unroll
        for (int d = 0; d < kDepth; ++d) dst[i + d * stride] = v[d];
    }
    for (; i < n16; i += stride) dst[i] = src[i];
}

constexpr int kReadDepth = 16;
__global__ __launch_bounds__(kBlock) void stream_read(const v4i* __restrict__ src, size_t n16, v4i* sink) {
    const size_t per = (n16 + gridDim.x - 1) / gridDim.x;   // this workgroup's chunk
    const size_t lo = per * blockIdx.x, hi = lo + per < n16 ? lo + per : n16;
    size_t i = lo + threadIdx.x;
    v4i acc = {0, 0, 0, 0};
    for (; i + (kReadDepth - 1) * (size_t)kBlock < hi; i += kReadDepth * (size_t)kBlock) {
        v4i v[kReadDepth];
#pragma unroll
        for (int d = 0; d < kReadDepth; ++d) v[d] = src[i + d * (size_t)kBlock];
#pragma unroll
        for (int d = 0; d < kReadDepth; ++d) acc ^= v[d];
    }
    for (; i < hi; i += kBlock) acc ^= src[i];
    // the reduction keeps the loads alive; it is written only if it hits a marker value
    if (acc[0] == 0x7A3F19C5 && acc[1] == 0x1B2C3D4E) sink[0] = acc;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" {

int monomoe_stream_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
    if (!dst || !src || !aligned16(dst) || !aligned16(src) || (bytes & 15u)) return MONOMOE_ERR_INVALID;
    if (bytes == 0) return MONOMOE_OK;
    hipLaunchKernelGGL(stream_copy, dim3(kGrid), dim3(kBlock), 0, stream, static_cast<const v4i*>(src),
                       static_cast<v4i*>(dst), bytes / 16);
    return hipGetLastError() == hipSuccess ? MONOMOE_OK : MONOMOE_ERR_HIP;
}

int monomoe_stream_read(const void* src, size_t bytes, void* sink16, hipStream_t stream) {
    if (!src || !sink16 || !aligned16(src) || !aligned16(sink16) || (bytes & 15u)) return MONOMOE_ERR_INVALID;
    if (bytes == 0) return MONOMOE_OK;
    hipLaunchKernelGGL(stream_read, dim3(kGrid), dim3(kBlock), 0, stream, static_cast<const v4i*>(src), bytes / 16,
                       static_cast<v4i*>(sink16));
    return hipGetLastError() == hipSuccess ? MONOMOE_OK : MONOMOE_ERR_HIP;
}

}  // extern "C"
