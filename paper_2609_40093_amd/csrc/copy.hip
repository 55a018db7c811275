// copy.hip -- plain streaming copy (16-byte non-temporal vectors, one 16 KiB chunk per
// workgroup, the fastest of the copy shapes measured on MI355X): the attainable HBM
// bandwidth probe and the known-size reference for hardware byte counters.
#include "ep_internal.h"

namespace ep {
namespace {

constexpr int kCopyU = 4;  // 16-byte vectors per lane: one 16 KiB chunk per workgroup

__global__ __launch_bounds__(256) void copy_kernel(u32x4 *__restrict__ dst, const u32x4 *__restrict__ src,
                                                   int64_t n) {
    const int64_t base = (int64_t)blockIdx.x * 256 * kCopyU + threadIdx.x;
    u32x4 v[kCopyU];
#pragma unroll
    for (int u = 0; u < kCopyU; ++u) {
        const int64_t i = base + u * 256;
        v[u] = i < n ? __builtin_nontemporal_load(src + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kCopyU; ++u) {
        const int64_t i = base + u * 256;
        if (i < n)
            __builtin_nontemporal_store(v[u], dst + i);
    }
}

}  // namespace

hipError_t launch_copy(void *dst, const void *src, size_t bytes, hipStream_t stream) {
    const int64_t n = (int64_t)(bytes / 16);
    if (n == 0)
        return hipSuccess;
    const int64_t blocks = (n + 256 * kCopyU - 1) / (256 * kCopyU);
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, ts.start, ts.stop, 0,
                          (u32x4 *)dst, (const u32x4 *)src, n);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("copy_probe", ts);
    return err;
}

}  // namespace ep
