// pack.hip -- dispatch pack for gfx950: packed[slot_pos[t*k+j]][:] = x[t][:].
//
// A DMA engine moves only contiguous regions, so the rows a destination needs are first
// gathered into one contiguous segment per destination (Sec. 2.2 of the paper).  The
// kernel is HBM-bound: it reads each token row once and writes it k times.
//
// Mapping: a row of V 16-byte vectors is G = ceil(V/64) groups of 64 (one vector per
// lane); a wave moves one chunk of `gpc` groups (all its loads in flight together) of one
// row.  Consecutive lanes touch consecutive 16-byte pieces of the row: every load and
// store is a fully coalesced 1 KiB wave access.
//   EXACT instances: V is a multiple of 64 and the chunk length U divides G, so every
//     load and store is unconditional, at a compile-time offset;
//   generic instances (rows whose length is not a multiple of 64 vectors, or G with no
//     usable divisor): chunks of up to U groups; loads stay unconditional (a group past
//     the chunk's end reloads the chunk's last group, a lane past the row's end reloads
//     the row's last vector: L2 hits, no HBM traffic); stores are guarded.
//
// Which mapping is used follows bandwidth measured on MI355X with inputs outside the
// memory-side cache:
//   k < 4:  one wave per (token, chunk): the chunk is loaded once (non-temporal) and
//           stored to the k rows;
//   k >= 4: one wave per (token, chunk, slot), the k waves of a chunk adjacent: each wave
//           writes a single destination row; the chunk's loads after the first come from
//           L2 (cached loads), and each wave feeds one write stream instead of k;
//   chunk:  the largest divisor of G of at most 16 groups (16 KiB): a whole row for rows
//           up to 16 KiB; long exact chunks measured faster than 4-group chunks and than
//           16-group chunks with guarded tails.  Rows with no divisor of at least 4 groups
//           (G a prime above 16) use the generic 16-group instance.
// Stores: non-temporal below 2 GiB written per launch, device-scope write-through buffer
// stores with the non-temporal hint from 2 GiB up (RowStore: each policy is the faster one
// at its sizes).  Rows carry
// no reuse across workgroups, so the workgroup-to-XCD placement needs no remapping.
#include "ep_internal.h"

namespace ep {
namespace {

struct PackGeom {
    int32_t V;       // 16-byte vectors per row
    int32_t G;       // groups of 64 vectors per row
    int32_t gpc;     // groups per chunk (<= the kernel's U)
    int32_t chunks;  // chunks per row
};

// Vector of the row that lane `lane` loads for group u of a generic chunk starting at
// group g0 with ng groups: always inside the row.
__device__ __forceinline__ int32_t load_index(int32_t g0, int u, int32_t ng, int lane, int32_t V) {
    return min((g0 + min(u, ng - 1)) * kWave + lane, V - 1);
}

// Whether the store of group u of a generic chunk is inside the chunk and the row.
__device__ __forceinline__ bool store_ok(int32_t g0, int u, int32_t ng, int lane, int32_t V) {
    return u < ng && (g0 + u) * kWave + lane < V;
}

// One wave per (token, chunk): the chunk is loaded once and stored to the k rows.
template <int U, bool EXACT, int SP>
__global__ __launch_bounds__(256) void pack_kernel(const u32x4 *__restrict__ x, int64_t T, PackGeom pg, int32_t k,
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
    const int64_t t = item / pg.chunks;
    if (t >= T)
        return;
    const int32_t g0 = (int32_t)(item - t * pg.chunks) * pg.gpc;
    const int32_t ng = EXACT ? U : min(pg.gpc, pg.G - g0);  // wave-uniform, >= 1
    const u32x4 *src = x + t * pg.V;
    u32x4 d[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
        d[u] = __builtin_nontemporal_load(src + (EXACT ? (g0 + u) * kWave + lane : load_index(g0, u, ng, lane, pg.V)));
    const int32_t *sp = slot_pos + t * k;
    for (int32_t j = 0; j < k; ++j) {
        const int64_t p = sp[j];
        if (p < 0 || p >= max_rows)
            continue;
        const RowStore<SP> dst(packed + p * pg.V + g0 * kWave, (uint32_t)(pg.V - g0 * kWave) * 16u);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (EXACT || store_ok(g0, u, ng, lane, pg.V))
                dst.put(d[u], u * kWave + lane);
    }
    if (fence_system)
        __threadfence_system();
}

// One wave per (token, chunk, slot), the k waves of a chunk adjacent: each wave writes a
// single destination row.
template <int U, bool EXACT, int SP>
__global__ __launch_bounds__(1024) void pack_slot_kernel(const u32x4 *__restrict__ x, int64_t T, PackGeom pg, int32_t k,
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
    const int64_t t = tc / pg.chunks;
    if (t >= T)
        return;
    const int32_t g0 = (int32_t)(tc - t * pg.chunks) * pg.gpc;
    const int32_t ng = EXACT ? U : min(pg.gpc, pg.G - g0);  // wave-uniform, >= 1
    const int64_t p = slot_pos[t * k + j];
    if (p < 0 || p >= max_rows)
        return;
    const u32x4 *src = x + t * pg.V;
    const RowStore<SP> dst(packed + p * pg.V + g0 * kWave, (uint32_t)(pg.V - g0 * kWave) * 16u);
    u32x4 d[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
        d[u] = src[EXACT ? (g0 + u) * kWave + lane : load_index(g0, u, ng, lane, pg.V)];
#pragma unroll
    for (int u = 0; u < U; ++u)
        if (EXACT || store_ok(g0, u, ng, lane, pg.V))
            dst.put(d[u], u * kWave + lane);
    if (fence_system)
        __threadfence_system();
}

template <int U, bool EXACT, int SP>
void launch_pack_u(bool per_slot, dim3 grid, dim3 block, hipStream_t stream, TraceSlot ts, const u32x4 *x, int64_t T,
                   const PackGeom &pg, int32_t k, const int32_t *slot_pos, u32x4 *packed, int64_t max_rows,
                   uint32_t *epoch_word, uint32_t epoch, RoundSel sel, bool fence_system) {
    if (per_slot)
        hipExtLaunchKernelGGL(pack_slot_kernel<U, EXACT, SP>, grid, block, 0, stream, ts.start, ts.stop, 0, x, T, pg,
                              k, slot_pos, packed, max_rows, epoch_word, epoch, sel, fence_system);
    else
        hipExtLaunchKernelGGL(pack_kernel<U, EXACT, SP>, grid, dim3(256), 0, stream, ts.start, ts.stop, 0, x, T, pg, k,
                              slot_pos, packed, max_rows, epoch_word, epoch, sel, fence_system);
}

// Chunk lengths with an EXACT instance (groups of 64 vectors), longest first.
constexpr int kExactU[] = {16, 15, 14, 13, 12, 11, 10, 9, 8, 7, 6, 5, 4, 3, 2, 1};

// Launches the instance for chunk length `exact` (0: generic) under store policy SP.
template <int SP>
void launch_chunk(int exact, bool per_slot, dim3 grid, dim3 block, hipStream_t stream, TraceSlot ts, const u32x4 *x,
                  int64_t T, const PackGeom &pg, int32_t k, const int32_t *slot_pos, u32x4 *packed, int64_t max_rows,
                  uint32_t *epoch_word, uint32_t epoch, RoundSel sel, bool fence_system) {
#define EP_PACK_ARGS per_slot, grid, block, stream, ts, x, T, pg, k, slot_pos, packed, max_rows, epoch_word, epoch, sel, fence_system
    switch (exact) {
    case 16: launch_pack_u<16, true, SP>(EP_PACK_ARGS); break;
    case 15: launch_pack_u<15, true, SP>(EP_PACK_ARGS); break;
    case 14: launch_pack_u<14, true, SP>(EP_PACK_ARGS); break;
    case 13: launch_pack_u<13, true, SP>(EP_PACK_ARGS); break;
    case 12: launch_pack_u<12, true, SP>(EP_PACK_ARGS); break;
    case 11: launch_pack_u<11, true, SP>(EP_PACK_ARGS); break;
    case 10: launch_pack_u<10, true, SP>(EP_PACK_ARGS); break;
    case 9: launch_pack_u<9, true, SP>(EP_PACK_ARGS); break;
    case 8: launch_pack_u<8, true, SP>(EP_PACK_ARGS); break;
    case 7: launch_pack_u<7, true, SP>(EP_PACK_ARGS); break;
    case 6: launch_pack_u<6, true, SP>(EP_PACK_ARGS); break;
    case 5: launch_pack_u<5, true, SP>(EP_PACK_ARGS); break;
    case 4: launch_pack_u<4, true, SP>(EP_PACK_ARGS); break;
    case 3: launch_pack_u<3, true, SP>(EP_PACK_ARGS); break;
    case 2: launch_pack_u<2, true, SP>(EP_PACK_ARGS); break;
    case 1: launch_pack_u<1, true, SP>(EP_PACK_ARGS); break;
    default:
        if (pg.gpc > 4)
            launch_pack_u<16, false, SP>(EP_PACK_ARGS);
        else
            launch_pack_u<4, false, SP>(EP_PACK_ARGS);
    }
#undef EP_PACK_ARGS
}

}  // namespace

hipError_t launch_pack(const void *x, int64_t T, int32_t H, int32_t k, const int32_t *slot_pos,
                       void *packed, int64_t max_rows, uint32_t *epoch_word, uint32_t epoch,
                       hipStream_t stream, RoundSel sel, bool fence_system) {
    if (T == 0)
        return hipSuccess;
    PackGeom pg;
    pg.V = H / 8;
    pg.G = (pg.V + kWave - 1) / kWave;
    const bool per_slot = k >= 4;
    int exact = 0;  // chunk length of the EXACT instance, 0: generic
    if (pg.V % kWave == 0)
        for (int u : kExactU)
            if (pg.G % u == 0) {
                exact = u >= (pg.G < 4 ? pg.G : 4) ? u : 0;  // no short chunks for long rows
                break;
            }
    // few tokens: shorter chunks, so that the launch keeps about 1024 waves (measured on
    // MI355X, top-2 of 14 KiB rows: 128 tokens 2.8 against 3.8 us, 512 tokens 5.5 against 6.0)
    if (exact > 1) {
        const int64_t per_chunk = per_slot ? T * k : T;
        if (per_chunk * (pg.G / exact) < 1024)
            for (int u : kExactU)
                if (u < exact && pg.G % u == 0) {
                    exact = u;
                    if (per_chunk * (pg.G / u) >= 1024)
                        break;
                }
    }
    pg.gpc = exact ? exact : (pg.G < 16 ? pg.G : 16);
    pg.chunks = (pg.G + pg.gpc - 1) / pg.gpc;
    const int64_t items = (per_slot ? T * k : T) * pg.chunks;
    // per-slot waves of one token chunk share its row through L2 only inside one workgroup
    // (consecutive workgroups run on different XCDs, each with its own L2): for k = 8 or 16
    // a workgroup of k waves holds them all, so the row is fetched from HBM once (4-wave
    // workgroups fetched it twice at k = 8; measured on MI355X)
    const int waves = per_slot && (k == 8 || k == 16) ? k : 4;
    const int64_t blocks = (items + waves - 1) / waves;
    if (blocks > INT32_MAX)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks);
    const u32x4 *xv = static_cast<const u32x4 *>(x);
    u32x4 *pv = static_cast<u32x4 *>(packed);
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    const bool wt = T * k * (int64_t)pg.V * 16 >= kWriteThroughBytes;
    if (wt)
        launch_chunk<kStoreWTStream>(exact, per_slot, grid, dim3(per_slot ? waves * kWave : 256), stream, ts, xv, T, pg, k,
                           slot_pos, pv, max_rows, epoch_word, epoch, sel, fence_system);
    else
        launch_chunk<kStoreNT>(exact, per_slot, grid, dim3(per_slot ? waves * kWave : 256), stream, ts, xv, T, pg, k,
                            slot_pos, pv, max_rows, epoch_word, epoch, sel, fence_system);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("pack", ts);
    return err;
}

}  // namespace ep
