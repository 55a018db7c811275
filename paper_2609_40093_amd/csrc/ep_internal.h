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
constexpr int kLayoutThreads = 256;                       // 4 waves per workgroup
constexpr int kLayoutWaves = kLayoutThreads / kWave;
constexpr int kTileSlots = 4096;                          // routing entries per tile
constexpr int kSlotsPerWave = kTileSlots / kLayoutWaves;  // contiguous run per wave
constexpr int kRoundsPerWave = kSlotsPerWave / kWave;     // 64 entries per round
constexpr int kMaxExperts = 2048;

// Routing status bits left in the layout workspace's status word.
constexpr uint32_t kRoutingIdOutOfRange = 1u;
constexpr uint32_t kRoutingDuplicate = 2u;

// Layout workspace: [0,256) status word (+ padding), then int32 tile histogram
// [num_tiles][E] when more than one tile is needed.
constexpr size_t kWorkspaceHeader = 256;
inline int64_t layout_tiles(int64_t slots) { return (slots + kTileSlots - 1) / kTileSlots; }
inline size_t layout_workspace_bytes(int64_t slots, int32_t experts) {
    int64_t tiles = layout_tiles(slots);
    return kWorkspaceHeader + (tiles > 1 ? (size_t)tiles * (size_t)experts * sizeof(int32_t) : 0);
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
    int32_t *tile_hist;  // [tiles][E] or null for one tile
};
hipError_t launch_layout(const LayoutArgs &a, hipStream_t stream);

hipError_t launch_pack(const void *x, int64_t T, int32_t H, int32_t k, const int32_t *slot_pos,
                       void *packed, int64_t max_rows, hipStream_t stream);

hipError_t launch_combine(const void *recv, const int32_t *slot_pos, const float *topk_w,
                          int64_t T, int32_t H, int32_t k, void *out, bool out_f32,
                          int64_t max_rows, hipStream_t stream);

hipError_t launch_wait_flags(const uint32_t *flags, int32_t n, uint32_t epoch,
                             int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream);

hipError_t launch_write_flag(uint32_t *flag, uint32_t epoch, hipStream_t stream);

hipError_t launch_copy(void *dst, const void *src, size_t bytes, hipStream_t stream);

}  // namespace ep
