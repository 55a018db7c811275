// ep_internal.h -- declarations shared by the library's host code and kernel files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "status_block.h"

#include <algorithm>
#include <cstddef>
#include <cstdint>

namespace ep {

// 16-byte vector: the unit every bandwidth kernel moves per lane.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Stores of one row (a packed row of the dispatch, an output row of the combine) from a
// wave-uniform base, under one of three policies that each kernel picks by the bytes a
// launch writes (measured on MI355X, inputs rotated past the memory-side cache):
//   kStoreNT:        non-temporal stores;
//   kStoreWT:        16-byte buffer stores at device scope (sc1: written through the XCD's
//                    L2 rather than held there dirty);
//   kStoreWTStream:  the same with the non-temporal hint as well (sc1 nt).
// The pack (rows of 4 and 14 KiB) stores with kStoreWTStream from 2 GiB per launch up,
// where the non-temporal rate falls with the size of the stream: at the prefill pack
// (3.76 GB written) 764 us against 772 us with kStoreWT and 778 us non-temporal;
// non-temporal is up to 20% faster at 0.1-1 GiB.  The combine writes through with kStoreWT
// below 128 MiB of output (there kStoreWTStream measured 5-8% slower); its thresholds are
// beside it.  The buffer range of a buffer-store row is the `bytes` from `base` on: a store
// past it is dropped by the hardware.
constexpr int kStoreNT = 0, kStoreWT = 1, kStoreWTStream = 2;
constexpr int64_t kWriteThroughBytes = 2ll << 30;  // the pack's
template <int POL>
struct RowStore {
    static_assert(POL == kStoreWT || POL == kStoreWTStream, "buffer-store policies");
    __amdgpu_buffer_rsrc_t rsrc;
    __device__ __forceinline__ RowStore(u32x4 *b, uint32_t bytes) {
        const uint64_t a = reinterpret_cast<uint64_t>(b);
        const uint64_t u = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                           (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
        rsrc = __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void *>(u), 0,
                                                 (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
    }
    __device__ __forceinline__ void put(u32x4 v, uint32_t vec) const {
        // cache-policy operand: 16 = sc1 (device scope), 2 = nt
        __builtin_amdgcn_raw_buffer_store_b128(v, rsrc, vec * 16u, 0, POL == kStoreWT ? 16 : 16 | 2);
    }
};
template <>
struct RowStore<kStoreNT> {
    u32x4 *base;
    __device__ __forceinline__ RowStore(u32x4 *b, uint32_t) : base(b) {}
    __device__ __forceinline__ void put(u32x4 v, uint32_t vec) const { __builtin_nontemporal_store(v, base + vec); }
};

// ---- layout geometry -----------------------------------------------------------
// The routing array is cut into tiles, one workgroup each; a workgroup has W waves and
// each wave walks `rounds` rounds of 64 entries.  W = 16 while 16 rows of per-wave
// counters fit in LDS (E <= 512), else 4.  One tile when it covers every entry in at most
// 4 rounds (W = 16) or 8 rounds (W = 4): one kernel then does the whole layout.  Otherwise
// as many tiles as keep the tile counts at most 16K words (every workgroup of the rank
// kernel reads them all) and at most 1024 tiles, with as few rounds as that allows.  No tile waits for another, so the tile count is not tied to the device.
constexpr int kMaxExperts = 2048;
constexpr int kLayoutRankCache = 8;  // rounds whose ids and in-wave ranks stay in registers
struct LayoutGeom {
    int waves;
    int rounds;
    int64_t tiles;
};
inline LayoutGeom layout_geometry(int64_t slots, int32_t experts) {
    const int waves = experts <= 512 ? 16 : 4;
    const int64_t per_round = (int64_t)kWave * waves;
    const int64_t one_tile_rounds = waves == 16 ? 4 : 8;
    if (slots <= per_round * one_tile_rounds) {
        const int64_t rounds = slots > 0 ? (slots + per_round - 1) / per_round : 1;
        return {waves, (int)rounds, 1};
    }
    int64_t max_tiles = 16384 / (experts > 0 ? experts : 1);
    max_tiles = max_tiles < 2 ? 2 : (max_tiles > 1024 ? 1024 : max_tiles);
    const int64_t rounds = (slots + per_round * max_tiles - 1) / (per_round * max_tiles);
    const int64_t tiles = (slots + per_round * rounds - 1) / (per_round * rounds);
    return {waves, (int)rounds, tiles};
}

// Routing status bits left in the layout workspace's status word.
constexpr uint32_t kRoutingIdOutOfRange = 1u;
constexpr uint32_t kRoutingDuplicate = 2u;

// Layout workspace (zero-filled before its first use):
//   byte   0  uint32 routing status of the last call
//   byte 192  int32 [3] rank count/offsets of a window layout (one segment)
//   byte 256  int32 [tiles][E] each tile's counts per expert (written by the count
//             kernel, read by the rank kernel); then uint32 [tiles] the tiles' routing
//             error bits
constexpr size_t kWorkspaceHeader = 256;
constexpr size_t kWorkspaceScratch = 192;  // 3 words the one-segment local layout writes
inline size_t layout_workspace_bytes(int64_t slots, int32_t experts) {
    const LayoutGeom g = layout_geometry(slots, experts);
    return kWorkspaceHeader + (g.tiles > 1 ? (size_t)g.tiles * ((size_t)experts + 1) * sizeof(int32_t) : 0);
}

// ---- timing events (tracing) -----------------------------------------------------
struct TraceSlot {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
// Returns a pair of timing events when tracing is enabled, else null events.
TraceSlot trace_acquire();
// Registers a launched pair under `name` (no-op for null events).
void trace_submit(const char *name, TraceSlot slot);
// Adds a host-timed span (milliseconds) under `name` while tracing is enabled.
void trace_host(const char *name, double ms);

// ---- kernel launchers (return the launch's hipError_t) ----------------------------
struct LayoutArgs {
    const int32_t *topk_idx;
    int64_t slots;  // T*k
    // E: experts grouped (the window [e_lo, e_lo + E) of all_E experts); nbits covers E,
    // all_nbits covers all_E (duplicate check over the raw ids when the window is narrower)
    int32_t k, E, R, nbits;
    int32_t e_lo = 0, all_E = 0, all_nbits = 0;
    int32_t *expert_counts, *expert_offsets, *rank_counts, *rank_offsets;
    int32_t *slot_pos, *row_src;
    uint32_t *status;        // workspace byte 0
    int32_t *tile_counts;    // workspace byte 256: [tiles][E]
    uint32_t *tile_errs;     // [tiles], after tile_counts
};
// Sets the workspace pointers of `a` (a.E and a.slots set) from the workspace base.
inline void layout_workspace(LayoutArgs &a, void *workspace) {
    char *ws = static_cast<char *>(workspace);
    const LayoutGeom g = layout_geometry(a.slots, a.E);
    a.status = reinterpret_cast<uint32_t *>(ws);
    a.tile_counts = reinterpret_cast<int32_t *>(ws + kWorkspaceHeader);
    a.tile_errs = reinterpret_cast<uint32_t *>(a.tile_counts + g.tiles * (int64_t)a.E);
}
hipError_t launch_layout(LayoutArgs a, hipStream_t stream);

// Layout and pack in one kernel for small expert counts (see fused.hip).  Same outputs
// as launch_layout followed by launch_pack; no workspace besides the status word.
struct FusedArgs {
    const int32_t *topk_idx;  // 16-byte aligned
    int64_t T;
    int32_t k, E, R, nbits;
    int32_t *expert_counts, *expert_offsets, *rank_counts, *rank_offsets;
    int32_t *slot_pos, *row_src;
    uint32_t *status;         // layout workspace byte 0
    const void *x;            // [T][H] 16-bit rows, 16-byte aligned
    int32_t H;
    void *packed;             // [max_rows][H]
    int64_t max_rows;
    uint32_t *epoch_word;     // stores `epoch` when non-null (host leg flag copies)
    uint32_t epoch;
};
// Whether the fused kernel covers these sizes (otherwise: layout, then pack).
bool fused_layout_pack_fits(int64_t T, int32_t k, int32_t E, int32_t H, const void *topk_idx);
hipError_t launch_layout_pack(const FusedArgs &a, hipStream_t stream);

// Buffer chosen at run time by the parity of a round counter in device memory (graph-
// replayed rounds): `alt` replaces the kernel's buffer argument on odd rounds.  No choice
// when `round` is null.
struct RoundSel {
    const void *alt = nullptr;
    const uint32_t *round = nullptr;
};

// Also stores `epoch` into *epoch_word (when non-null) for the host leg's flag copies.
// fence_system: every wave ends with a system-scope release (rows stored to host memory
// are visible to the host before any later kernel runs).
hipError_t launch_pack(const void *x, int64_t T, int32_t H, int32_t k, const int32_t *slot_pos,
                       void *packed, int64_t max_rows, uint32_t *epoch_word, uint32_t epoch,
                       hipStream_t stream, RoundSel sel = {}, bool fence_system = false);

hipError_t launch_combine(const void *recv, const int32_t *slot_pos, const float *topk_w,
                          int64_t T, int32_t H, int32_t k, void *out, bool out_f32,
                          int64_t max_rows, hipStream_t stream, RoundSel sel = {});

// Per-sender accumulation (combine.hip, signal.hip).  masks: device words, masks[0] the
// senders whose rows need no wait, masks[i + 1] the senders landed before pass i.
// launch_landed_set waits (bounded) until the landed set (landed[r] holds the epoch)
// grows past masks[i] (base for i = 0) and records it; launch_accumulate runs pass i
// into the fp32 partial acc [T][H], writing each token to out once its k slots are in.
hipError_t launch_landed_set(const uint32_t *landed, int32_t R, uint32_t epoch, uint32_t base, uint32_t *masks,
                             int32_t i, int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream);
hipError_t launch_accumulate(const void *recv, const int32_t *slot_pos, const float *topk_w, int64_t T, int32_t H,
                             int32_t k, const int32_t *rank_offsets, int32_t R, const uint32_t *masks, int32_t i,
                             float *acc, void *out, bool out_f32, int64_t max_rows, hipStream_t stream);

// One lane per flag polls flags[i] until (int32)(flags[i] - epoch) >= 0, at most
// timeout_ticks of the constant-rate wall clock; on expiry records the timeout in the
// status block (kStatusWords words at `status`).
hipError_t launch_wait_flags(const char *name, const uint32_t *flags, int32_t n, uint32_t epoch,
                             int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream);

// Stores 0 into *value (a DMA dependency signal) with a system-scope release.
hipError_t launch_release_signal(int64_t *value, hipStream_t stream);

// Gate over up to kMaxGate flags (see signal.hip): waits for flag[i] to hold the epoch and
// stores 0 into release[i] (per flag) or release[0] (all = 1, after every flag).
constexpr int kMaxGate = 64;
struct GateArgs {
    const uint32_t *flag[kMaxGate];
    int64_t *release[kMaxGate];
    int32_t n = 0;
    int32_t all = 0;
    uint32_t epoch = 0;
    int32_t sleep_units = 2;
    int64_t timeout_ticks = 0;
    uint32_t *status = nullptr;  // status block (kStatusWords words)
    uint32_t site = 0;           // set by launch_gate from its name
};
hipError_t launch_gate(const char *name, const GateArgs &g, hipStream_t stream);
// Words of a buffer set's device epoch row: the sources of the DMA flag copies, one word
// per flag of a merged flag copy.
constexpr int kEpochRowWords = 64;
// Stores `epoch` into the kEpochRowWords words of epoch_word[], then 0 into *value (a DMA
// start signal).
hipError_t launch_stamp_release(uint32_t *epoch_word, uint32_t epoch, int64_t *value, hipStream_t stream);
// Copies n int32 from device memory to host words host[0..n), then stores `epoch` in host[n].
hipError_t launch_mirror(const int32_t *src, int32_t n, uint32_t *host, uint32_t epoch, hipStream_t stream);

// Up to kMaxBlocks equally shaped blocks summed element-wise by launch_block_reduce.
constexpr int kMaxBlocks = 32;
struct BlockList {
    const void *ptr[kMaxBlocks];
    int32_t n = 0;
};
// out[i] = sum_b block_b[i] over n elements (n % 8 == 0, 16-byte aligned blocks), fp32
// accumulation in list order; blocks bf16 or fp32 (f32_in), out bf16 (nearest-even) or fp32.
hipError_t launch_block_reduce(const BlockList &bl, bool f32_in, int64_t n, void *out, bool f32_out,
                               hipStream_t stream);

// Round-counter kernels of graph-replayed rounds (signal.hip):
//   launch_round_advance: *round += 1;
//   launch_round_gate: waits until flags[(round % 2) * stride + i] - (round + delta) >= 0
//     (signed) for i < n, bounded like the other flag waits;
//   launch_round_stamp: after a system-scope release, words[(round % 2) * stride + i] =
//     round for i < n.
hipError_t launch_round_advance(uint32_t *round, hipStream_t stream);
hipError_t launch_round_gate(const char *name, const uint32_t *round, const uint32_t *flags, int32_t stride,
                             int32_t n, int32_t delta, int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream);
hipError_t launch_round_stamp(const uint32_t *round, uint32_t *words, int32_t stride, int32_t n, hipStream_t stream);

hipError_t launch_copy(void *dst, const void *src, size_t bytes, hipStream_t stream);
// Streaming probe of a given read:write mix (copy.hip); row_bytes = 1024 * g with g in
// {1, 2, 4, 8, 14, 16}.
hipError_t launch_stream_probe(void *dst, const void *src, int64_t units, int32_t row_bytes, int32_t reads,
                               int32_t writes, int store_policy, hipStream_t stream);

}  // namespace ep
