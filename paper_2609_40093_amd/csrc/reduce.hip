// reduce.hip -- block reduction of the dense Reduce-Scatter (Sec. 4.2 of the paper: the
// destination GPU sums the blocks the other GPUs computed for its shard with its own):
//   out[i] = sum over blocks b (in the order given) of block_b[i], fp32 accumulation,
//   stored as bf16 (round to nearest, ties to even) or fp32.
// HBM-bound: reads n_blocks * n elements, writes n.  One thread per 8 consecutive
// elements: a 16-byte vector of bf16 (two of fp32) per block, every block's load issued
// before the adds; non-temporal loads and stores (each element is touched once).
#include "ep_internal.h"

namespace ep {
namespace {

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    const b2 r = __builtin_convertvector(f2{lo, hi}, b2);  // v_cvt_pk_bf16_f32: nearest-even
    return __builtin_bit_cast(uint32_t, r);
}

template <bool F32_IN, bool F32_OUT>
__global__ __launch_bounds__(256) void block_reduce_kernel(BlockList bl, int64_t groups, void *__restrict__ out) {
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;  // group of 8 elements
    if (g >= groups)
        return;
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q)
        acc[q] = 0.f;
    // blocks in chunks of 4 with their loads in flight together
    for (int b0 = 0; b0 < bl.n; b0 += 4) {
        u32x4 v[4][F32_IN ? 2 : 1];
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
            if (b0 + bb >= bl.n)
                break;
            const u32x4 *src = static_cast<const u32x4 *>(bl.ptr[b0 + bb]) + g * (F32_IN ? 2 : 1);
#pragma unroll
            for (int h = 0; h < (F32_IN ? 2 : 1); ++h)
                v[bb][h] = __builtin_nontemporal_load(src + h);
        }
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
            if (b0 + bb >= bl.n)
                break;
            if (F32_IN) {
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    acc[q] += __uint_as_float(v[bb][q / 4][q % 4]);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[2 * q] += __uint_as_float(v[bb][0][q] << 16);
                    acc[2 * q + 1] += __uint_as_float(v[bb][0][q] & 0xffff0000u);
                }
            }
        }
    }
    if (F32_OUT) {
        u32x4 *dst = static_cast<u32x4 *>(out) + g * 2;
        __builtin_nontemporal_store(u32x4{__float_as_uint(acc[0]), __float_as_uint(acc[1]), __float_as_uint(acc[2]),
                                          __float_as_uint(acc[3])},
                                    dst);
        __builtin_nontemporal_store(u32x4{__float_as_uint(acc[4]), __float_as_uint(acc[5]), __float_as_uint(acc[6]),
                                          __float_as_uint(acc[7])},
                                    dst + 1);
    } else {
        u32x4 r;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            r[q] = pack_bf16x2(acc[2 * q], acc[2 * q + 1]);
        __builtin_nontemporal_store(r, static_cast<u32x4 *>(out) + g);
    }
}

}  // namespace

hipError_t launch_block_reduce(const BlockList &bl, bool f32_in, int64_t n, void *out, bool f32_out,
                               hipStream_t stream) {
    if (n == 0 || bl.n == 0)
        return hipSuccess;
    if (n % 8 != 0 || bl.n > kMaxBlocks)
        return hipErrorInvalidValue;
    const int64_t groups = n / 8;
    const dim3 grid((unsigned)((groups + 255) / 256)), block(256);
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    if (f32_in && f32_out)
        hipExtLaunchKernelGGL(block_reduce_kernel<true, true>, grid, block, 0, stream, ts.start, ts.stop, 0, bl, groups,
                              out);
    else if (f32_in)
        hipExtLaunchKernelGGL(block_reduce_kernel<true, false>, grid, block, 0, stream, ts.start, ts.stop, 0, bl,
                              groups, out);
    else if (f32_out)
        hipExtLaunchKernelGGL(block_reduce_kernel<false, true>, grid, block, 0, stream, ts.start, ts.stop, 0, bl,
                              groups, out);
    else
        hipExtLaunchKernelGGL(block_reduce_kernel<false, false>, grid, block, 0, stream, ts.start, ts.stop, 0, bl,
                              groups, out);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("block_reduce", ts);
    return err;
}

}  // namespace ep
