// layout_static.hip -- ep_dispatch_layout_static: the dispatch layout without a workspace
// argument, for callers that cannot allocate device memory (code under HIP graph capture,
// serving loops that must not allocate, harnesses that forbid it).
//
// The layout kernels' scratch (the status word and the tiles' counts and error bits of a
// multi-tile layout) is a file-scope device array of this library, one copy per GPU,
// held until the process ends.  Its size is fixed: the layout geometry keeps the tile
// counts at 16K words and the tiles at 1024 at most, whatever the number of routing
// entries, so one array serves every size ep_dispatch_layout accepts.
//
// Host code never passes the array's name to a kernel (in host code it is a stand-in, not
// a device address): the device address is read once per device with hipGetSymbolAddress,
// with that device current, and kept; kernels get that address.
//
// Every call on one GPU shares that GPU's array, which keeps the last call's contents;
// no call reads what an earlier one left there (the count kernel writes every tile count
// the rank kernel reads).  Calls that overlap on one GPU (other streams, or other host
// threads, without ordering between them) race on the array.
#include "ep.h"
#include "ep_internal.h"
#include "staging.h"

#include <mutex>

namespace {

constexpr size_t kScratchBytes = 128u << 10;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices] = {};  // device address of `scratch` on each device, once read

// The device address of this GPU's scratch (read on the first call on that device).
ep_status scratch_address(int device, void **out) {
    if (device < 0 || device >= kMaxDevices)
        return ep::fail(EP_ERR_INVALID_ARG, "ep_dispatch_layout_static: device %d out of range", device);
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return ep::hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                                "ep_dispatch_layout_static: hipGetSymbolAddress of the scratch array");
        g_scratch[device] = p;
    }
    *out = g_scratch[device];
    return EP_OK;
}

}  // namespace

extern "C" ep_status ep_dispatch_layout_static(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                                               int32_t num_experts, int32_t num_ranks, int32_t *expert_counts,
                                               int32_t *expert_offsets, int32_t *rank_counts,
                                               int32_t *rank_offsets, int32_t *slot_pos, int32_t *row_src,
                                               uint32_t *status_dev, hipStream_t stream) {
    const char *who = "ep_dispatch_layout_static";
    const int64_t T = num_tokens;
    const int32_t k = topk, E = num_experts, R = num_ranks;
    if (!status_dev)
        return ep::fail(EP_ERR_INVALID_ARG, "%s: status_dev is NULL", who);
    if (T >= 0 && k >= 1 && E >= 1 && E <= EP_MAX_EXPERTS && T * (int64_t)k <= INT32_MAX) {
        const size_t need = ep::layout_workspace_bytes(T * k, E);
        if (need > kScratchBytes)
            return ep::fail(EP_ERR_INVALID_ARG, "%s: T*k = %lld entries over %d experts need %zu bytes of scratch; "
                                                "the library holds %zu",
                            who, (long long)(T * k), E, need, kScratchBytes);
    }
    // every argument is checked before the device is touched (the workspace argument of the
    // shared checks only needs to be non-NULL here: the scratch's address is read below)
    ep_status st = ep::check_layout_args(who, T, k, E, R, topk_idx, expert_counts, expert_offsets, rank_counts,
                                         rank_offsets, slot_pos, &kScratchBytes, kScratchBytes);
    if (st != EP_OK)
        return st;
    int device = -1;
    EP_HIP(hipGetDevice(&device));
    void *ws = nullptr;
    st = scratch_address(device, &ws);
    if (st != EP_OK)
        return st;
    ep::LayoutArgs a = ep::layout_args(topk_idx, T, k, E, R, expert_counts, expert_offsets, rank_counts, rank_offsets,
                                       slot_pos, row_src, ws);
    a.status = status_dev;  // the routing status goes to the caller's word, not the scratch
    EP_HIP(ep::launch_layout(a, stream));
    return EP_OK;
}
