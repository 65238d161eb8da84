// Streaming-read probe for the benchmark: the rate at which this part delivers a
// plain read of a buffer from HBM, the context beside the decode kernel's
// achieved bandwidth (which the roofline fraction measures against the
// published 8 TB/s). Not part of the attention path.
//
// The kernel reads `bytes` bytes as 16-byte vectors, grid-stride, with four
// loads in flight per lane, with or without the non-temporal cache hint, and
// folds them into one XOR per thread stored to `sink`, so that no load is
// optimised away. It is a separate library: nothing in libtkattn calls it.
#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
constexpr int kProbeThreads = 512;

template <bool NT>
__device__ __forceinline__ u32x4 load(const u32x4* p) {
    if constexpr (NT)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}

template <bool NT>
__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const u32x4* __restrict__ a, size_t n16,
                                                                    unsigned* __restrict__ sink) {
    const size_t T = (size_t)gridDim.x * kProbeThreads;
    const size_t t = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
    u32x4 acc = {0u, 0u, 0u, 0u};
    size_t i = t;
    for (; i + 3 * T < n16; i += 4 * T)  // every index below n16
        acc ^= load<NT>(a + i) ^ load<NT>(a + i + T) ^ load<NT>(a + i + 2 * T) ^ load<NT>(a + i + 3 * T);
    for (; i < n16; i += T) acc ^= load<NT>(a + i);
    sink[t] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

}  // namespace

extern "C" {

// Threads per workgroup of the probe: `sink` must hold grid * this many unsigned.
int tkprobe_threads(void) { return kProbeThreads; }

// Reads `bytes` bytes at `buf` (device memory, 16-byte aligned, bytes a multiple
// of 16) with `grid` workgroups of tkprobe_threads() threads on `stream`, using
// non-temporal loads when `non_temporal` is nonzero; writes one word per thread
// to `sink` (device memory). Returns 0 on success, 1 for an invalid argument
// (checked before any HIP call), 2 for a launch error.
int tkprobe_stream_read(const void* buf, size_t bytes, unsigned* sink, int grid, int non_temporal,
                        hipStream_t stream) {
    if (!buf || !sink || bytes == 0 || bytes % 16 != 0 || ((uintptr_t)buf & 15) != 0 || grid < 1 || grid > 65535)
        return 1;
    const u32x4* a = (const u32x4*)buf;
    const size_t n16 = bytes / 16;
    if (non_temporal)
        hipLaunchKernelGGL(stream_read_kernel<true>, dim3((unsigned)grid), dim3(kProbeThreads), 0, stream, a, n16,
                           sink);
    else
        hipLaunchKernelGGL(stream_read_kernel<false>, dim3((unsigned)grid), dim3(kProbeThreads), 0, stream, a, n16,
                           sink);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
