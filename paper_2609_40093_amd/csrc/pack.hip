// pack.hip -- dispatch pack for gfx950: packed[slot_pos[t*k+j]][:] = x[t][:].
//
// A DMA engine moves only contiguous regions, so the rows a destination needs are first
// gathered into one contiguous segment per destination (Sec. 2.2 of the paper).  The
// kernel is HBM-bound: it reads each token row once and writes it k times.
//
// Mapping: one wave per (token, column chunk of 64*U 16-byte vectors).  The token index
// is wave-uniform, so the k slot positions are scalar loads; each lane loads U 16-byte
// vectors of the row (all in flight together) and stores them to the k destination rows.
// Consecutive lanes touch consecutive 16-byte pieces of one row: every load and store is
// a fully coalesced 1 KiB wave access.  Loads and stores are non-temporal (the rows are
// touched once; streaming stores leave no dirty lines for the end-of-kernel writeback).
// Which mapping is used follows bandwidth measured on MI355X: for rows of at most 4 KiB
// with k >= 4, one wave per (token, chunk, slot).  Rows carry no reuse across
// workgroups, so the workgroup-to-XCD placement needs no remapping.
#include "ep_internal.h"

namespace ep {
namespace {

constexpr int kPackU = 4;  // 16-byte vectors per lane per chunk

// One wave per (token, chunk): the chunk is loaded once and stored to the k rows.
template <int U>
__global__ __launch_bounds__(256) void pack_kernel(const u32x4 *__restrict__ x, int64_t T, int32_t V,
                                                   int32_t chunks, int32_t k,
                                                   const int32_t *__restrict__ slot_pos,
                                                   u32x4 *__restrict__ packed, int64_t max_rows,
                                                   uint32_t *epoch_word, uint32_t epoch, RoundSel sel,
                                                   bool fence_system) {
    const int lane = threadIdx.x & (kWave - 1);
    if (epoch_word && blockIdx.x == 0 && threadIdx.x == 0)
        *epoch_word = epoch;
    if (sel.round && (__hip_atomic_load(sel.round, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 1u))
        packed = static_cast<u32x4 *>(const_cast<void *>(sel.alt));
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + wave;
    const int64_t t = item / chunks;
    if (t >= T)
        return;
    const int32_t v0 = (int32_t)(item - t * chunks) * (U * kWave);
    const u32x4 *src = x + t * V;
    u32x4 d[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int32_t v = v0 + u * kWave + lane;
        d[u] = v < V ? __builtin_nontemporal_load(src + v) : u32x4{0u, 0u, 0u, 0u};
    }
    const int32_t *sp = slot_pos + t * k;
    for (int32_t j = 0; j < k; ++j) {
        const int64_t p = sp[j];
        if (p < 0 || p >= max_rows)
            continue;
        u32x4 *dst = packed + p * V;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t v = v0 + u * kWave + lane;
            if (v < V)
                __builtin_nontemporal_store(d[u], dst + v);
        }
    }
    if (fence_system)
        __threadfence_system();
}

// One wave per (token, chunk, slot), the k waves of a chunk adjacent: each wave writes a
// single destination row; the chunk's k reads after the first come from L2.  Faster for
// narrow rows with many slots, where each wave otherwise feeds k write streams.
template <int U>
__global__ __launch_bounds__(256) void pack_slot_kernel(const u32x4 *__restrict__ x, int64_t T, int32_t V,
                                                        int32_t chunks, int32_t k,
                                                        const int32_t *__restrict__ slot_pos,
                                                        u32x4 *__restrict__ packed, int64_t max_rows,
                                                        uint32_t *epoch_word, uint32_t epoch, RoundSel sel,
                                                        bool fence_system) {
    const int lane = threadIdx.x & (kWave - 1);
    if (epoch_word && blockIdx.x == 0 && threadIdx.x == 0)
        *epoch_word = epoch;
    if (sel.round && (__hip_atomic_load(sel.round, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 1u))
        packed = static_cast<u32x4 *>(const_cast<void *>(sel.alt));
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + wave;
    const int64_t tc = item / k;
    const int32_t j = (int32_t)(item - tc * k);
    const int64_t t = tc / chunks;
    if (t >= T)
        return;
    const int32_t v0 = (int32_t)(tc - t * chunks) * (U * kWave);
    const int64_t p = slot_pos[t * k + j];
    if (p < 0 || p >= max_rows)
        return;
    const u32x4 *src = x + t * V;
    u32x4 *dst = packed + p * V;
    u32x4 d[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int32_t v = v0 + u * kWave + lane;
        d[u] = v < V ? src[v] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int32_t v = v0 + u * kWave + lane;
        if (v < V)
            __builtin_nontemporal_store(d[u], dst + v);
    }
    if (fence_system)
        __threadfence_system();
}

}  // namespace

hipError_t launch_pack(const void *x, int64_t T, int32_t H, int32_t k, const int32_t *slot_pos,
                       void *packed, int64_t max_rows, uint32_t *epoch_word, uint32_t epoch,
                       hipStream_t stream, RoundSel sel, bool fence_system) {
    if (T == 0)
        return hipSuccess;
    const int32_t V = H / 8;
    const int32_t chunks = (V + kPackU * kWave - 1) / (kPackU * kWave);
    const bool per_slot = V <= 256 && k >= 4;   // rows of at most 4 KiB, many slots
    const int64_t items = T * chunks * (per_slot ? k : 1);
    const int waves_per_block = 4;
    const int64_t blocks = (items + waves_per_block - 1) / waves_per_block;
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    if (per_slot)
        hipExtLaunchKernelGGL(pack_slot_kernel<kPackU>, dim3((unsigned)blocks), dim3(waves_per_block * kWave), 0,
                              stream, ts.start, ts.stop, 0, (const u32x4 *)x, T, V, chunks, k, slot_pos,
                              (u32x4 *)packed, max_rows, epoch_word, epoch, sel, fence_system);
    else
        hipExtLaunchKernelGGL(pack_kernel<kPackU>, dim3((unsigned)blocks), dim3(waves_per_block * kWave), 0,
                              stream, ts.start, ts.stop, 0, (const u32x4 *)x, T, V, chunks, k, slot_pos,
                              (u32x4 *)packed, max_rows, epoch_word, epoch, sel, fence_system);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("pack", ts);
    return err;
}

}  // namespace ep
