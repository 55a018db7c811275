// copy.hip -- plain streaming kernels: what streaming code attains on this chip, beside
// which the path's kernels are judged.
//   copy_kernel    16-byte non-temporal vectors, one 16 KiB chunk per workgroup (the
//                  fastest copy shape measured on MI355X): the attainable-bandwidth probe
//                  and the known-size reference for hardware byte counters.
//   stream_kernel  one wave per unit: reads `reads` consecutive rows and writes `writes`
//                  consecutive rows (each written row the XOR of the rows read), so the
//                  traffic has the read:write mix of a kernel of the path with none of its
//                  routing -- 1:k like the dispatch's pack, k:1 like the combine, 1:0
//                  read-only, 0:1 write-only -- over sequential addresses, with any of the
//                  path's three store policies (RowStore).
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

constexpr int kStreamMaxGroups = 16;  // 64-vector groups per row the probe holds in registers

// Unit u reads rows [u*reads, (u+1)*reads) of src and writes rows [u*writes, (u+1)*writes)
// of dst; a row is `groups` x 64 16-byte vectors, lane l moving vector l of each group.
// With no row to write, the XOR of everything read is stored (one 16-byte vector per
// wave, into dst[unit % 64]) only if it equals a value that normal data does not give, so
// the loads cannot be dropped.
template <int G, int SP>
__global__ __launch_bounds__(256) void stream_kernel(u32x4 *__restrict__ dst, const u32x4 *__restrict__ src,
                                                     int64_t units, int32_t reads, int32_t writes) {
    const int lane = threadIdx.x & 63;
    const int64_t unit = ((int64_t)blockIdx.x * 256 + threadIdx.x) / 64;
    if (unit >= units)
        return;
    constexpr int64_t kRow = (int64_t)G * 64;
    u32x4 acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
        acc[g] = u32x4{0x9e3779b9u, 0x7f4a7c15u, 0x85ebca6bu, (uint32_t)unit};
    const u32x4 *in = src + unit * reads * kRow + lane;
    for (int r = 0; r < reads; ++r) {
        u32x4 v[G];
#pragma unroll
        for (int g = 0; g < G; ++g)
            v[g] = __builtin_nontemporal_load(in + r * kRow + g * 64);
#pragma unroll
        for (int g = 0; g < G; ++g)
            acc[g] ^= v[g];
    }
    if (writes == 0) {
        u32x4 f = acc[0];
#pragma unroll
        for (int g = 1; g < G; ++g)
            f ^= acc[g];
        if (f.x == 0x01234567u && f.y == 0x89abcdefu && f.z == 0x02468aceu && f.w == 0x13579bdfu)
            dst[unit % 64] = f;
        return;
    }
    u32x4 *out = dst + unit * writes * kRow;
    for (int w = 0; w < writes; ++w) {
        const RowStore<SP> row(out + w * kRow, (uint32_t)(kRow * 16));
#pragma unroll
        for (int g = 0; g < G; ++g)
            row.put(acc[g], g * 64 + lane);
    }
}

}  // namespace

hipError_t launch_stream_probe(void *dst, const void *src, int64_t units, int32_t row_bytes, int32_t reads,
                               int32_t writes, int store_policy, hipStream_t stream) {
    const int groups = row_bytes / 1024;
    if (units <= 0)
        return hipSuccess;
    const unsigned blocks = (unsigned)((units * 64 + 255) / 256);
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    auto go = [&](auto nt_kern, auto wt_kern, auto wts_kern) {
        auto kern = store_policy == kStoreWTStream ? wts_kern : store_policy == kStoreWT ? wt_kern : nt_kern;
        hipExtLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, stream, ts.start, ts.stop, 0, (u32x4 *)dst,
                              (const u32x4 *)src, units, reads, writes);
    };
    switch (groups) {
    case 1: go(stream_kernel<1, kStoreNT>, stream_kernel<1, kStoreWT>, stream_kernel<1, kStoreWTStream>); break;
    case 2: go(stream_kernel<2, kStoreNT>, stream_kernel<2, kStoreWT>, stream_kernel<2, kStoreWTStream>); break;
    case 4: go(stream_kernel<4, kStoreNT>, stream_kernel<4, kStoreWT>, stream_kernel<4, kStoreWTStream>); break;
    case 8: go(stream_kernel<8, kStoreNT>, stream_kernel<8, kStoreWT>, stream_kernel<8, kStoreWTStream>); break;
    case 14: go(stream_kernel<14, kStoreNT>, stream_kernel<14, kStoreWT>, stream_kernel<14, kStoreWTStream>); break;
    case 16: go(stream_kernel<16, kStoreNT>, stream_kernel<16, kStoreWT>, stream_kernel<16, kStoreWTStream>); break;
    default: return hipErrorInvalidValue;
    }
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("stream_probe", ts);
    return err;
}

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
