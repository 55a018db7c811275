// combine.hip -- gate-weighted top-k combine for gfx950:
//   out[t][:] = sum_{j<k} w[t*k+j] * recv[slot_pos[t*k+j]][:]
// The returned contributions of a token are added on the GPU that owns the token
// (Sec. 4.3 of the paper: a DMA engine cannot add, so the reduction stays on the GPU),
// which also returns the rows to token order.
//
// Arithmetic: fp32 accumulator, fused multiply-add per slot in order j = 0..k-1 starting
// from +0, then one round-to-nearest-even conversion to bf16 (v_cvt_pk_bf16_f32), or the
// fp32 accumulator itself.  HBM-bound: k row reads and one row write per token.
//
// Mapping: one wave per (token, column chunk of 64*U 16-byte vectors); the k slot
// positions and gates are wave-uniform scalar loads.  Slots are taken KC at a time and
// all KC*U row loads of a batch are issued before their FMAs, keeping KC*U KiB in flight
// per wave.  Rows are read once: loads and stores are non-temporal.
#include "ep_internal.h"

namespace ep {
namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2 b = __builtin_convertvector(f32x2{lo, hi}, bf16x2);
    return __builtin_bit_cast(uint32_t, b);
}

template <int U, int KC, bool F32_OUT>
__global__ __launch_bounds__(256) void combine_kernel(const u32x4 *__restrict__ recv,
                                                      const int32_t *__restrict__ slot_pos,
                                                      const float *__restrict__ topk_w, int64_t T,
                                                      int32_t V, int32_t chunks, int32_t k,
                                                      void *__restrict__ out, int64_t max_rows,
                                                      RoundSel sel) {
    const int lane = threadIdx.x & (kWave - 1);
    if (sel.round && (__hip_atomic_load(sel.round, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 1u))
        recv = static_cast<const u32x4 *>(sel.alt);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + wave;
    const int64_t t = item / chunks;
    if (t >= T)
        return;
    const int32_t v0 = (int32_t)(item - t * chunks) * (U * kWave);
    const int32_t *sp = slot_pos + t * k;
    const float *wt = topk_w + t * k;

    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q)
            acc[u][q] = 0.0f;

    for (int32_t j0 = 0; j0 < k; j0 += KC) {
        u32x4 d[KC][U];
        float g[KC];
        bool ok[KC];
#pragma unroll
        for (int jj = 0; jj < KC; ++jj) {
            const int32_t j = j0 + jj;
            const int64_t p = j < k ? (int64_t)sp[j] : -1;
            ok[jj] = p >= 0 && p < max_rows;
            g[jj] = ok[jj] ? wt[j] : 0.0f;
            const u32x4 *src = recv + (ok[jj] ? p : 0) * V;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t v = v0 + u * kWave + lane;
                d[jj][u] = ok[jj] && v < V ? __builtin_nontemporal_load(src + v) : u32x4{0u, 0u, 0u, 0u};
            }
        }
#pragma unroll
        for (int jj = 0; jj < KC; ++jj) {
            if (!ok[jj])
                continue;
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[u][2 * q] = __builtin_fmaf(g[jj], bf16_lo(d[jj][u][q]), acc[u][2 * q]);
                    acc[u][2 * q + 1] = __builtin_fmaf(g[jj], bf16_hi(d[jj][u][q]), acc[u][2 * q + 1]);
                }
        }
    }

#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int32_t v = v0 + u * kWave + lane;
        if (v >= V)
            continue;
        const int64_t o = t * V + v;
        if constexpr (F32_OUT) {
            u32x4 *dst = (u32x4 *)out + 2 * o;
            const u32x4 a = {__float_as_uint(acc[u][0]), __float_as_uint(acc[u][1]),
                             __float_as_uint(acc[u][2]), __float_as_uint(acc[u][3])};
            const u32x4 b = {__float_as_uint(acc[u][4]), __float_as_uint(acc[u][5]),
                             __float_as_uint(acc[u][6]), __float_as_uint(acc[u][7])};
            __builtin_nontemporal_store(a, dst);
            __builtin_nontemporal_store(b, dst + 1);
        } else {
            const u32x4 r = {pack_bf16x2(acc[u][0], acc[u][1]), pack_bf16x2(acc[u][2], acc[u][3]),
                             pack_bf16x2(acc[u][4], acc[u][5]), pack_bf16x2(acc[u][6], acc[u][7])};
            __builtin_nontemporal_store(r, (u32x4 *)out + o);
        }
    }
}

template <int U, int KC>
hipError_t launch_uk(const void *recv, const int32_t *slot_pos, const float *topk_w, int64_t T,
                     int32_t V, int32_t k, void *out, bool out_f32, int64_t max_rows,
                     hipStream_t stream, RoundSel sel) {
    const int32_t chunks = (V + U * kWave - 1) / (U * kWave);
    const int64_t items = T * chunks;
    const int waves_per_block = 4;
    const int64_t blocks = (items + waves_per_block - 1) / waves_per_block;
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    if (out_f32)
        hipExtLaunchKernelGGL(combine_kernel<U, KC, true>, dim3((unsigned)blocks),
                              dim3(waves_per_block * kWave), 0, stream, ts.start, ts.stop, 0,
                              (const u32x4 *)recv, slot_pos, topk_w, T, V, chunks, k, out, max_rows, sel);
    else
        hipExtLaunchKernelGGL(combine_kernel<U, KC, false>, dim3((unsigned)blocks),
                              dim3(waves_per_block * kWave), 0, stream, ts.start, ts.stop, 0,
                              (const u32x4 *)recv, slot_pos, topk_w, T, V, chunks, k, out, max_rows, sel);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("combine", ts);
    return err;
}

}  // namespace

hipError_t launch_combine(const void *recv, const int32_t *slot_pos, const float *topk_w,
                          int64_t T, int32_t H, int32_t k, void *out, bool out_f32,
                          int64_t max_rows, hipStream_t stream, RoundSel sel) {
    if (T == 0)
        return hipSuccess;
    const int32_t V = H / 8;
    // KC*U 16-byte loads per lane in flight: 16 for k >= 4, 4 for k = 2 and 3 (two-group
    // chunks: more waves, which measured faster on MI355X than four-group chunks there)
    if (k >= 8)
        return launch_uk<2, 8>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    if (k >= 4)
        return launch_uk<4, 4>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    if (k >= 2)
        return launch_uk<2, 2>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    return launch_uk<4, 1>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
}

}  // namespace ep
