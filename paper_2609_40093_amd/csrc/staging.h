// staging.h -- the staging object behind the C ABI's opaque ep_staging, shared by the
// files that implement its calls (ep_api.cpp: allocation, the default host legs;
// exchange.cpp: the per-sender, duplex and remote-only legs).
#pragma once

#include "ep.h"
#include "ep_internal.h"
#include "sdma.h"
#include "status_block.h"

#include <cstdint>
#include <string>
#include <vector>

namespace ep {

// Record the message for ep_last_error and return `st`.
ep_status fail(ep_status st, const char *fmt, ...);
// Map a HIP error to EP_ERR_OOM / EP_ERR_HIP (and clear it from the runtime).
ep_status hip_fail(hipError_t e, const char *what);

// Takes and clears a status block (kStatusWords words): EP_OK, or the error it holds, with
// the expired wait described in ep_last_error; `name_flag` names the flag word at an
// address ("recv_landed[buf 1][rank 3]"), or returns "" for one it does not know.
struct FlagNamer {
    virtual std::string operator()(const uint32_t *flag) const = 0;
    virtual ~FlagNamer() = default;
};
ep_status take_status(uint32_t *block, int64_t timeout_us, const FlagNamer &name_flag);

// Host-visible argument checks of a dispatch layout call (sizes, NULL pointers, the
// workspace's size), and the kernel arguments of one with its workspace at `workspace`.
ep_status check_layout_args(const char *who, int64_t T, int32_t k, int32_t E, int32_t R, const int32_t *topk_idx,
                            const int32_t *expert_counts, const int32_t *expert_offsets, const int32_t *rank_counts,
                            const int32_t *rank_offsets, const int32_t *slot_pos, const void *workspace,
                            size_t workspace_bytes);
LayoutArgs layout_args(const int32_t *topk_idx, int64_t T, int32_t k, int32_t E, int32_t R, int32_t *expert_counts,
                       int32_t *expert_offsets, int32_t *rank_counts, int32_t *rank_offsets, int32_t *slot_pos,
                       int32_t *row_src, void *workspace);

#define EP_HIP(call)                                                                                \
    do {                                                                                            \
        hipError_t e_ = (call);                                                                     \
        if (e_ != hipSuccess)                                                                       \
            return ::ep::hip_fail(e_, #call);                                                       \
    } while (0)

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kMaxBuffers = 8;
constexpr int64_t kDefaultChunk = 64ll << 20;
constexpr size_t kEpochStride = kEpochRowWords * sizeof(uint32_t);  // one device epoch row per buffer set
constexpr int kSdmaSlots = 4;        // host-leg rounds in flight per staging

// true: the default device->host leg goes through hipMemcpyAsync instead of the SDMA lane
// (environment EP_HOSTLEG_COPY=hip; kept as a measured comparison).
bool d2h_through_hip();

// ---- host legs of graph-replayed rounds on SDMA engines (graph_legs.h)
class GraphLegs;

// ---- exchange modes (exchange.cpp)
class Exchange;
constexpr int kMaxExchangeRanks = 32;  // 2R flags fit one polling wave; a sender set fits 32 bits
constexpr int kMaskWords = 64;         // landed-set words per buffer set (EP_MODE_ACCUMULATE)
Exchange *exchange_create(int device, int nslots, std::string &err);
void exchange_destroy(Exchange *x);
const char *exchange_engines(const Exchange *x);

}  // namespace ep

struct ep_staging;

namespace ep {
// Queues the copy of rank_offsets to the host mirror of buffer set b (before the pack).
ep_status exchange_enqueue_mirror(ep_staging *s, int b, uint32_t epoch, const int32_t *rank_offsets,
                                  hipStream_t stream, const char *who);
// The reduction of a combine in EP_MODE_ACCUMULATE: run by exchange_combine itself, one
// pass per arrival of senders.
struct AccumulateCall {
    const int32_t *slot_pos;
    const float *topk_w;
    int64_t T;
    int32_t k;
    void *out;
    bool out_f32;
};
// Host legs of a dispatch (after the pack was queued) and of a combine (before the
// reduction is queued, or with the reduction when `acc` is given), in the staging's
// exchange mode.
ep_status exchange_dispatch(ep_staging *s, int b, uint32_t epoch, int64_t rows, hipStream_t stream);
ep_status exchange_combine(ep_staging *s, int b, uint32_t epoch, int64_t rows, const int32_t *rank_offsets,
                           hipStream_t stream, const AccumulateCall *acc = nullptr);
}  // namespace ep

struct ep_staging {
    int device = -1;
    ep_staging_kind kind = EP_STAGING_HBM;
    int64_t max_rows = 0;
    int32_t hidden = 0, num_ranks = 0, num_buffers = 0, max_chunks = 0;
    int64_t row_bytes = 0, buffer_bytes = 0, chunk_bytes = 0;
    void *dev_send[ep::kMaxBuffers] = {}, *dev_recv[ep::kMaxBuffers] = {};
    void *host_send[ep::kMaxBuffers] = {}, *host_recv[ep::kMaxBuffers] = {};
    // coherent pinned words: send [nbuf][max_chunks], recv [nbuf][R], the status block
    // (ep::kStatusWords words, status_block.h), then
    // inbound [nbuf][R], returned-out [nbuf][R], inbound-landed [nbuf][R],
    // recv-landed [nbuf][R], offsets mirror [nbuf][R+2], send credits [nbuf][R],
    // recv credits [nbuf], graph-round ready [nbuf], graph-round landed [nbuf]
    uint32_t *flags = nullptr;
    size_t flag_words = 0;
    char *dev_epoch = nullptr;       // device: the epoch of each buffer set's current round
    uint32_t *dev_round = nullptr;   // device: round counter of graph-replayed rounds
    ep::SdmaLane *lane = nullptr;    // default device->host leg on one SDMA engine
    ep::GraphLegs *graph_legs = nullptr;  // graph rounds' host legs on SDMA (ep_graph_legs_sdma)
    hipEvent_t ev_sysrel = nullptr;  // records a system-scope release before a DMA engine reads
    hipStream_t up = nullptr, down = nullptr;
    hipEvent_t ev_up_in[ep::kMaxBuffers] = {}, ev_up_done[ep::kMaxBuffers] = {};
    hipEvent_t ev_down_in[ep::kMaxBuffers] = {}, ev_down_done[ep::kMaxBuffers] = {};
    int64_t timeout_us = 10ll * 1000 * 1000;
    int32_t sleep_units = 2;
    int64_t wall_clock_khz = 100000;

    // exchange modes (EP_MODE_* bits) and the buffers they add
    uint32_t mode = 0;
    int32_t self_rank = 0;
    void *dev_in[ep::kMaxBuffers] = {}, *host_in[ep::kMaxBuffers] = {}, *host_ret[ep::kMaxBuffers] = {};
    std::vector<int64_t> rows_in;     // [nbuf][R] rows each sender sends this rank (host-set)
    std::vector<int64_t> off_in;      // [nbuf][R+1] where they land in dev_in (set by dispatch)
    std::vector<int32_t> offs_cache;  // [nbuf][R+1] rank offsets read through the mirror
    std::vector<uint32_t> offs_epoch; // [nbuf] epoch of offs_cache (valid when offs_valid)
    std::vector<uint8_t> offs_valid;  // [nbuf]
    std::vector<uint32_t> offs_sent;  // [nbuf] epoch of the last mirror queued (may still be in flight)
    std::vector<uint32_t> in_epoch;   // [nbuf] epoch of the last duplex dispatch (off_in valid)
    ep::Exchange *xchg = nullptr;
    // EP_MODE_ACCUMULATE: per buffer set the fp32 partial sums [T][H] (grown on demand),
    // and the landed-set words of its passes [nbuf][kMaskWords]
    float *dev_acc[ep::kMaxBuffers] = {};
    size_t acc_bytes[ep::kMaxBuffers] = {};
    uint32_t *dev_masks = nullptr;

    size_t R() const { return (size_t)num_ranks; }
    size_t nb() const { return (size_t)num_buffers; }
    uint32_t *send_flags(int b) const { return flags + (size_t)b * max_chunks; }
    uint32_t *recv_flags(int b) const { return flags + nb() * max_chunks + (size_t)b * R(); }
    uint32_t *status() const { return flags + nb() * (max_chunks + R()); }
    uint32_t *ext_base() const { return status() + ep::kStatusWords; }
    uint32_t *in_flags(int b) const { return ext_base() + (size_t)b * R(); }
    uint32_t *ret_flags(int b) const { return ext_base() + nb() * R() + (size_t)b * R(); }
    uint32_t *in_landed(int b) const { return ext_base() + 2 * nb() * R() + (size_t)b * R(); }
    uint32_t *recv_landed(int b) const { return ext_base() + 3 * nb() * R() + (size_t)b * R(); }
    uint32_t *mirror(int b) const { return ext_base() + 4 * nb() * R() + (size_t)b * (R() + 2); }
    uint32_t *send_credit(int b) const { return mirror(0) + nb() * (R() + 2) + (size_t)b * R(); }
    uint32_t *recv_credit(int b) const { return send_credit(0) + nb() * R() + (size_t)b; }
    // graph rounds with SDMA legs: the dispatch's rows are in dev_send (set by the device),
    // the returned rows are in dev_recv (set by the legs' thread)
    uint32_t *graph_ready(int b) const { return recv_credit(0) + nb() + (size_t)b; }
    uint32_t *graph_landed(int b) const { return graph_ready(0) + nb() + (size_t)b; }
    static size_t flag_words_for(int nbuf, int max_chunks, int R) {
        return (size_t)nbuf * (max_chunks + R) + ep::kStatusWords + 4 * (size_t)nbuf * R + (size_t)nbuf * (R + 2) +
               (size_t)nbuf * R + 3 * (size_t)nbuf;
    }
    uint32_t *epoch_word(int b) const { return reinterpret_cast<uint32_t *>(dev_epoch + b * ep::kEpochStride); }
};
