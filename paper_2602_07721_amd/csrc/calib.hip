// Reference streaming kernels for measurement: a plain device copy and a plain
// device read, against which the benchmark states the achievable HBM bandwidth
// of this GPU and scales the rocprofv3 FETCH_SIZE / WRITE_SIZE counters.
//
// Each thread moves 4 x 16 bytes per round in a grid-stride loop, all loads of a
// round issued before its stores, with non-temporal hints (the data is touched
// once).  The read kernel folds what it reads into one word per thread and stores
// it only when it equals a caller-chosen key, which the loads cannot be optimised
// away around.

#include "internal.hpp"

namespace pariskv {

namespace {

constexpr int kCalThreads = 256;
constexpr int kCalUnroll = 4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kCalThreads) void stream_copy_kernel(u32x4* __restrict__ dst,
                                                                  const u32x4* __restrict__ src,
                                                                  int64_t n16) {
    const int64_t stride = (int64_t)gridDim.x * kCalThreads;
    int64_t i = (int64_t)blockIdx.x * kCalThreads + threadIdx.x;
    for (; i + (kCalUnroll - 1) * stride < n16; i += kCalUnroll * stride) {
        u32x4 v[kCalUnroll];
#pragma unroll
        for (int u = 0; u < kCalUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < kCalUnroll; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
    }
    for (; i < n16; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

__global__ __launch_bounds__(kCalThreads) void stream_read_kernel(const u32x4* __restrict__ src, int64_t n16,
                                                                  uint32_t key, uint32_t* __restrict__ sink) {
    const int64_t stride = (int64_t)gridDim.x * kCalThreads;
    int64_t i = (int64_t)blockIdx.x * kCalThreads + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (kCalUnroll - 1) * stride < n16; i += kCalUnroll * stride) {
        u32x4 v[kCalUnroll];
#pragma unroll
        for (int u = 0; u < kCalUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < kCalUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const u32x4 v = __builtin_nontemporal_load(src + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == key) *sink = acc;
}

// 64 blocks of 256 threads per CU on 256 CUs: of the shapes tried (2048 to 16384
// blocks, 1 to 8 rows in flight per thread, strided or contiguous per thread, with and
// without non-temporal hints) this copied fastest, 5.3 TB/s for 1 GiB, above the HIP
// runtime's own device copy (5.2 TB/s).
constexpr unsigned kCalBlocks = 256 * 64;

}  // namespace

hipError_t launch_stream_copy(void* dst, const void* src, size_t bytes, hipStream_t s) {
    const ProfEvents pe = prof_begin("stream_copy");
    hipExtLaunchKernelGGL(stream_copy_kernel, dim3(kCalBlocks), dim3(kCalThreads), 0, s, pe.start, pe.stop, 0,
                          static_cast<u32x4*>(dst), static_cast<const u32x4*>(src), (int64_t)(bytes / 16));
    return hipGetLastError();
}

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t key, uint32_t* sink, hipStream_t s) {
    const ProfEvents pe = prof_begin("stream_read");
    hipExtLaunchKernelGGL(stream_read_kernel, dim3(kCalBlocks), dim3(kCalThreads), 0, s, pe.start, pe.stop, 0,
                          static_cast<const u32x4*>(src), (int64_t)(bytes / 16), key, sink);
    return hipGetLastError();
}

}  // namespace pariskv
