// ep_internal.h -- declarations shared by the library's host code and kernel files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace ep {

// 16-byte vector: the unit every bandwidth kernel moves per lane.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---- layout geometry -----------------------------------------------------------
// A workgroup of W waves ranks one tile; each wave walks kLayoutRounds rounds of 64
// routing entries.  W = 16 while W per-wave counter rows of E experts (plus the scan
// arrays) fit in 64 KiB of LDS, else 4.
constexpr int kLayoutRounds = 8;
constexpr int kMaxExperts = 2048;
constexpr int layout_waves(int32_t experts) { return experts <= 512 ? 16 : 4; }
constexpr int64_t layout_tile_slots(int waves) { return (int64_t)waves * kWave * kLayoutRounds; }

// Routing status bits left in the layout workspace's status word.
constexpr uint32_t kRoutingIdOutOfRange = 1u;
constexpr uint32_t kRoutingDuplicate = 2u;

// Layout workspace: [0,256) status word (+ padding); when more than one tile is needed,
// then int32 tile totals [num_tiles][E] and per-wave counts [num_tiles][W][E].
constexpr size_t kWorkspaceHeader = 256;
inline int64_t layout_tiles(int64_t slots, int32_t experts) {
    const int64_t tile = layout_tile_slots(layout_waves(experts));
    return (slots + tile - 1) / tile;
}
inline size_t layout_workspace_bytes(int64_t slots, int32_t experts) {
    const int64_t tiles = layout_tiles(slots, experts);
    return kWorkspaceHeader + (tiles > 1 ? (size_t)tiles * (1 + layout_waves(experts)) * (size_t)experts *
                                               sizeof(int32_t)
                                         : 0);
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

// ---- kernel launchers (return the launch's hipError_t) ----------------------------
struct LayoutArgs {
    const int32_t *topk_idx;
    int64_t slots;  // T*k
    int32_t k, E, R, nbits;
    int32_t *expert_counts, *expert_offsets, *rank_counts, *rank_offsets;
    int32_t *slot_pos, *row_src;
    uint32_t *status;
    int32_t *tile_hist;  // [tiles][E] tile totals, then [tiles][waves][E] wave counts; null for one tile
};
hipError_t launch_layout(const LayoutArgs &a, hipStream_t stream);

// Also stores `epoch` into *epoch_word (when non-null) for the host leg's flag copies.
hipError_t launch_pack(const void *x, int64_t T, int32_t H, int32_t k, const int32_t *slot_pos,
                       void *packed, int64_t max_rows, uint32_t *epoch_word, uint32_t epoch,
                       hipStream_t stream);

hipError_t launch_combine(const void *recv, const int32_t *slot_pos, const float *topk_w,
                          int64_t T, int32_t H, int32_t k, void *out, bool out_f32,
                          int64_t max_rows, hipStream_t stream);

// One lane per flag polls flags[i] until (int32)(flags[i] - epoch) >= 0, at most
// timeout_ticks of the constant-rate wall clock; on expiry stores EP_ERR_TIMEOUT to *status.
hipError_t launch_wait_flags(const char *name, const uint32_t *flags, int32_t n, uint32_t epoch,
                             int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream);

// Stores 0 into *value (a DMA dependency signal) with a system-scope release.
hipError_t launch_release_signal(int64_t *value, hipStream_t stream);

hipError_t launch_copy(void *dst, const void *src, size_t bytes, hipStream_t stream);

}  // namespace ep
