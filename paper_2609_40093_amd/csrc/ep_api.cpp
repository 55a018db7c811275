// ep_api.cpp -- host side of libep: the C ABI declared in include/ep.h.
//
// Argument checks, staging buffers and their DMA streams, the chunked host legs, flag
// writes and waits, and the timing-event tracer.  Every call enqueues on the caller's
// stream; the library's side streams (up = D2H, down = H2D) join the caller's stream
// through events, so the caller sees one ordered stream.
//
// Device->host legs run on an SDMA engine driven through ROCr (sdma.h), because the HIP
// runtime may turn a device->host hipMemcpyAsync into a copy kernel on the compute
// units.  Host->device legs are hipMemcpyAsync copies, which the runtime places on SDMA.
// EP_HOSTLEG_COPY=hip sends the device->host leg through hipMemcpyAsync too (the
// runtime's own choice of engine, kept as a measured comparison).
#include "ep.h"
#include "ep_internal.h"
#include "graph_legs.h"
#include "staging.h"

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace ep {

ep_status fail(ep_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

ep_status hip_fail(hipError_t e, const char *what) {
    (void)hipGetLastError();  // reported here; do not let a later launch check see it again
    return fail(e == hipErrorOutOfMemory ? EP_ERR_OOM : EP_ERR_HIP, "%s: %s (%d)", what,
                hipGetErrorString(e), (int)e);
}

bool d2h_through_hip() {
    static const bool v = [] {
        const char *e = std::getenv("EP_HOSTLEG_COPY");
        return e && std::strcmp(e, "hip") == 0;
    }();
    return v;
}

}  // namespace ep

using ep::aligned16;
using ep::d2h_through_hip;
using ep::fail;
using ep::hip_fail;
using ep::kDefaultChunk;
using ep::kEpochStride;
using ep::kMaxBuffers;
using ep::kSdmaSlots;

// ------------------------------------------------------------------------- tracing

namespace ep {
namespace {
std::atomic<bool> g_trace_on{false};
std::mutex g_trace_mu;
struct Pending {
    std::string name;
    hipEvent_t start, stop;
};
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_event_pool;
constexpr size_t kTraceSamples = 65536;  // durations kept per name for the percentiles
struct Stat {
    int64_t count = 0;
    double total = 0, mn = 1e300, mx = 0;
    std::vector<float> samples;
    void add(double ms) {
        count += 1;
        total += ms;
        mn = std::min(mn, ms);
        mx = std::max(mx, ms);
        if (samples.size() < kTraceSamples)
            samples.push_back((float)ms);
    }
};
double percentile(std::vector<float> v, double q) {  // by copy: sorted here
    if (v.empty())
        return 0.0;
    std::sort(v.begin(), v.end());
    return v[(size_t)(q * (double)(v.size() - 1) + 0.5)];
}
std::map<std::string, Stat> g_stats;

hipEvent_t pool_get() {
    if (!g_event_pool.empty()) {
        hipEvent_t e = g_event_pool.back();
        g_event_pool.pop_back();
        return e;
    }
    // timing-only events: no system-scope cache writeback folded into the measured span
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess)
        return nullptr;
    return e;
}
}  // namespace

TraceSlot trace_acquire() {
    TraceSlot s;
    if (!g_trace_on.load(std::memory_order_relaxed))
        return s;
    std::lock_guard<std::mutex> lk(g_trace_mu);
    s.start = pool_get();
    s.stop = pool_get();
    if (!s.start || !s.stop) {
        if (s.start)
            g_event_pool.push_back(s.start);
        if (s.stop)
            g_event_pool.push_back(s.stop);
        s = TraceSlot{};
    }
    return s;
}

void trace_submit(const char *name, TraceSlot slot) {
    if (!slot.start)
        return;
    std::lock_guard<std::mutex> lk(g_trace_mu);
    g_pending.push_back({name, slot.start, slot.stop});
}

void trace_host(const char *name, double ms) {
    if (!g_trace_on.load(std::memory_order_relaxed))
        return;
    std::lock_guard<std::mutex> lk(g_trace_mu);
    g_stats[name].add(ms);
}

}  // namespace ep

// ---------------------------------------------------------------------------- misc

extern "C" int32_t ep_abi_version(void) { return EP_ABI_VERSION; }

extern "C" const char *ep_status_name(int32_t status) {
    switch (status) {
    case EP_OK: return "EP_OK";
    case EP_ERR_INVALID_ARG: return "EP_ERR_INVALID_ARG";
    case EP_ERR_BAD_ROUTING: return "EP_ERR_BAD_ROUTING";
    case EP_ERR_HIP: return "EP_ERR_HIP";
    case EP_ERR_OOM: return "EP_ERR_OOM";
    case EP_ERR_TIMEOUT: return "EP_ERR_TIMEOUT";
    default: return "EP_ERR_UNKNOWN";
    }
}

extern "C" const char *ep_last_error(void) { return g_last_error.c_str(); }

// -------------------------------------------------------------------------- layout

extern "C" ep_status ep_layout_workspace_bytes(int64_t num_tokens, int32_t topk, int32_t num_experts,
                                               size_t *bytes) {
    if (!bytes)
        return fail(EP_ERR_INVALID_ARG, "ep_layout_workspace_bytes: bytes is NULL");
    if (num_tokens < 0 || topk < 1 || num_experts < 1 || num_experts > EP_MAX_EXPERTS)
        return fail(EP_ERR_INVALID_ARG, "ep_layout_workspace_bytes: bad sizes T=%lld k=%d E=%d",
                    (long long)num_tokens, topk, num_experts);
    *bytes = ep::layout_workspace_bytes(num_tokens * topk, num_experts);
    return EP_OK;
}

namespace ep {

// Host-visible argument checks of a dispatch layout call.
ep_status check_layout_args(const char *who, int64_t T, int32_t k, int32_t E, int32_t R, const int32_t *topk_idx,
                            const int32_t *expert_counts, const int32_t *expert_offsets, const int32_t *rank_counts,
                            const int32_t *rank_offsets, const int32_t *slot_pos, const void *workspace,
                            size_t workspace_bytes) {
    if (T < 0 || E < 1 || E > EP_MAX_EXPERTS || k < 1 || k > E || R < 1 || E % R != 0)
        return fail(EP_ERR_INVALID_ARG, "%s: need T >= 0, 1 <= k <= E <= %d, R >= 1, E %% R == 0 (T=%lld k=%d E=%d R=%d)",
                    who, EP_MAX_EXPERTS, (long long)T, k, E, R);
    if (T * (int64_t)k > INT32_MAX)
        return fail(EP_ERR_INVALID_ARG, "%s: T*k = %lld does not fit int32", who, (long long)(T * k));
    if (!expert_counts || !expert_offsets || !rank_counts || !rank_offsets || !workspace)
        return fail(EP_ERR_INVALID_ARG, "%s: NULL output or workspace", who);
    if (T > 0 && (!topk_idx || !slot_pos))
        return fail(EP_ERR_INVALID_ARG, "%s: NULL topk_idx or slot_pos", who);
    const size_t need = ep::layout_workspace_bytes(T * k, E);
    if (workspace_bytes < need)
        return fail(EP_ERR_INVALID_ARG, "%s: workspace of %zu bytes, need %zu", who, workspace_bytes, need);
    return EP_OK;
}

LayoutArgs layout_args(const int32_t *topk_idx, int64_t T, int32_t k, int32_t E, int32_t R, int32_t *expert_counts,
                       int32_t *expert_offsets, int32_t *rank_counts, int32_t *rank_offsets, int32_t *slot_pos,
                       int32_t *row_src, void *workspace) {
    LayoutArgs a{};
    a.topk_idx = topk_idx;
    a.slots = T * k;
    a.k = k;
    a.E = E;
    a.R = R;
    a.nbits = E > 1 ? 32 - __builtin_clz((unsigned)(E - 1)) : 0;
    a.e_lo = 0;
    a.all_E = E;
    a.all_nbits = a.nbits;
    a.expert_counts = expert_counts;
    a.expert_offsets = expert_offsets;
    a.rank_counts = rank_counts;
    a.rank_offsets = rank_offsets;
    a.slot_pos = slot_pos;
    a.row_src = row_src;
    layout_workspace(a, workspace);
    return a;
}

}  // namespace ep

using ep::check_layout_args;

extern "C" ep_status ep_dispatch_layout(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                                        int32_t num_experts, int32_t num_ranks, int32_t *expert_counts,
                                        int32_t *expert_offsets, int32_t *rank_counts,
                                        int32_t *rank_offsets, int32_t *slot_pos, int32_t *row_src,
                                        void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const int64_t T = num_tokens;
    const int32_t k = topk, E = num_experts, R = num_ranks;
    const ep_status st = check_layout_args("ep_dispatch_layout", T, k, E, R, topk_idx, expert_counts, expert_offsets,
                                           rank_counts, rank_offsets, slot_pos, workspace, workspace_bytes);
    if (st != EP_OK)
        return st;
    EP_HIP(ep::launch_layout(ep::layout_args(topk_idx, T, k, E, R, expert_counts, expert_offsets, rank_counts,
                                             rank_offsets, slot_pos, row_src, workspace),
                             stream));
    return EP_OK;
}

extern "C" ep_status ep_dispatch_layout_local(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                                              int32_t num_experts, int32_t e_lo, int32_t e_hi,
                                              int32_t *local_counts, int32_t *local_offsets, int32_t *slot_pos,
                                              int32_t *row_src, void *workspace, size_t workspace_bytes,
                                              hipStream_t stream) {
    const int64_t N = num_tokens;
    const int32_t k = topk, E = num_experts;
    if (N < 0 || E < 1 || E > EP_MAX_EXPERTS || k < 1 || k > E || e_lo < 0 || e_lo >= e_hi || e_hi > E)
        return fail(EP_ERR_INVALID_ARG,
                    "ep_dispatch_layout_local: need N >= 0, 1 <= k <= E <= %d, 0 <= e_lo < e_hi <= E "
                    "(N=%lld k=%d E=%d window [%d,%d))",
                    EP_MAX_EXPERTS, (long long)N, k, E, e_lo, e_hi);
    if (N * (int64_t)k > INT32_MAX)
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch_layout_local: N*k = %lld does not fit int32", (long long)(N * k));
    if (!local_counts || !local_offsets || !workspace)
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch_layout_local: NULL output or workspace");
    if (N > 0 && (!topk_idx || !slot_pos))
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch_layout_local: NULL topk_idx or slot_pos");
    const int32_t L = e_hi - e_lo;
    const size_t need = ep::layout_workspace_bytes(N * k, L);
    if (workspace_bytes < need)
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch_layout_local: workspace of %zu bytes, need %zu",
                    workspace_bytes, need);
    char *ws = static_cast<char *>(workspace);
    ep::LayoutArgs a{};
    a.topk_idx = topk_idx;
    a.slots = N * k;
    a.k = k;
    a.E = L;
    a.R = 1;  // one segment: the rows of the whole window
    a.nbits = L > 1 ? 32 - __builtin_clz((unsigned)(L - 1)) : 0;
    a.e_lo = e_lo;
    a.all_E = E;
    a.all_nbits = E > 1 ? 32 - __builtin_clz((unsigned)(E - 1)) : 0;
    a.expert_counts = local_counts;
    a.expert_offsets = local_offsets;
    a.rank_counts = reinterpret_cast<int32_t *>(ws + ep::kWorkspaceScratch);      // [1], unused by callers
    a.rank_offsets = reinterpret_cast<int32_t *>(ws + ep::kWorkspaceScratch + 4); // [2]
    a.slot_pos = slot_pos;
    a.row_src = row_src;
    ep::layout_workspace(a, workspace);
    EP_HIP(ep::launch_layout(a, stream));
    return EP_OK;
}

extern "C" ep_status ep_pack(const void *x_dev, int64_t num_tokens, int32_t hidden, int32_t topk,
                             const int32_t *slot_pos, void *out_dev, int64_t max_rows, hipStream_t stream) {
    if (num_tokens < 0 || topk < 1 || hidden < 8 || hidden % 8 != 0 || max_rows < 0)
        return fail(EP_ERR_INVALID_ARG, "ep_pack: need N >= 0, k >= 1, H a positive multiple of 8, max_rows >= 0");
    if (num_tokens > 0 && (!x_dev || !slot_pos || !out_dev || !aligned16(x_dev) || !aligned16(out_dev)))
        return fail(EP_ERR_INVALID_ARG, "ep_pack: x, slot_pos and a 16-byte aligned out are required");
    EP_HIP(ep::launch_pack(x_dev, num_tokens, hidden, topk, slot_pos, out_dev, max_rows, nullptr, 0, stream));
    return EP_OK;
}

extern "C" ep_status ep_combine_rows(const void *y_dev, int64_t max_rows, const int32_t *slot_pos,
                                     const float *topk_w, int64_t num_tokens, int32_t hidden, int32_t topk,
                                     void *out_dev, ep_out_dtype out_dtype, hipStream_t stream) {
    if (num_tokens < 0 || topk < 1 || hidden < 8 || hidden % 8 != 0 || max_rows < 0)
        return fail(EP_ERR_INVALID_ARG,
                    "ep_combine_rows: need N >= 0, k >= 1, H a positive multiple of 8, max_rows >= 0");
    if (out_dtype != EP_OUT_BF16 && out_dtype != EP_OUT_F32)
        return fail(EP_ERR_INVALID_ARG, "ep_combine_rows: unknown out_dtype %d", (int)out_dtype);
    if (num_tokens > 0 && (!slot_pos || !topk_w || !out_dev || !aligned16(out_dev) ||
                           (max_rows > 0 && (!y_dev || !aligned16(y_dev)))))
        return fail(EP_ERR_INVALID_ARG, "ep_combine_rows: slot_pos, topk_w and 16-byte aligned y/out are required");
    EP_HIP(ep::launch_combine(y_dev, slot_pos, topk_w, num_tokens, hidden, topk, out_dev, out_dtype == EP_OUT_F32,
                              max_rows, stream));
    return EP_OK;
}

extern "C" ep_status ep_layout_validate(const void *workspace, hipStream_t stream) {
    if (!workspace)
        return fail(EP_ERR_INVALID_ARG, "ep_layout_validate: workspace is NULL");
    EP_HIP(hipStreamSynchronize(stream));
    uint32_t word = 0;
    EP_HIP(hipMemcpy(&word, workspace, sizeof word, hipMemcpyDeviceToHost));
    if (word == 0)
        return EP_OK;
    return fail(EP_ERR_BAD_ROUTING, "routing rejected:%s%s",
                (word & ep::kRoutingIdOutOfRange) ? " expert id outside [0,E)" : "",
                (word & ep::kRoutingDuplicate) ? " expert repeated within a token row" : "");
}

// ------------------------------------------------------------------------- staging

namespace {

void staging_release(ep_staging *s) {
    // first the SDMA copies (each waits until its copies have landed), then their buffers
    if (s->graph_legs) {
        s->graph_legs->stop();
        delete s->graph_legs;
        s->graph_legs = nullptr;
    }
    if (s->lane) {
        s->lane->release();
        delete s->lane;
        s->lane = nullptr;
    }
    ep::exchange_destroy(s->xchg);
    s->xchg = nullptr;
    for (int b = 0; b < kMaxBuffers; ++b) {
        if (s->dev_send[b]) (void)hipFree(s->dev_send[b]);
        if (s->dev_recv[b]) (void)hipFree(s->dev_recv[b]);
        if (s->host_send[b]) (void)hipHostFree(s->host_send[b]);
        if (s->host_recv[b]) (void)hipHostFree(s->host_recv[b]);
        if (s->dev_in[b]) (void)hipFree(s->dev_in[b]);
        if (s->host_in[b]) (void)hipHostFree(s->host_in[b]);
        if (s->host_ret[b]) (void)hipHostFree(s->host_ret[b]);
        if (s->dev_acc[b]) (void)hipFree(s->dev_acc[b]);
        for (hipEvent_t e : {s->ev_up_in[b], s->ev_up_done[b], s->ev_down_in[b], s->ev_down_done[b]})
            if (e) (void)hipEventDestroy(e);
    }
    if (s->ev_sysrel) (void)hipEventDestroy(s->ev_sysrel);
    if (s->flags) (void)hipHostFree(s->flags);
    if (s->dev_epoch) (void)hipFree(s->dev_epoch);
    if (s->dev_round) (void)hipFree(s->dev_round);
    if (s->dev_masks) (void)hipFree(s->dev_masks);
    for (hipStream_t st : {s->up, s->down})
        if (st) (void)hipStreamDestroy(st);
    delete s;
}

ep_status check_device(const ep_staging *s, const char *who) {
    int dev = -1;
    EP_HIP(hipGetDevice(&dev));
    if (dev != s->device)
        return fail(EP_ERR_INVALID_ARG, "%s: staging lives on device %d, current device is %d", who,
                    s->device, dev);
    return EP_OK;
}

}  // namespace

extern "C" ep_status ep_staging_alloc(ep_staging_kind kind, int64_t max_rows, int32_t hidden,
                                      int32_t num_ranks, int32_t num_buffers, int64_t chunk_bytes,
                                      ep_staging **out) {
    if (!out)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_alloc: out is NULL");
    *out = nullptr;
    if (kind != EP_STAGING_HBM && kind != EP_STAGING_PINNED_HOST)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_alloc: unknown kind %d", (int)kind);
    if (max_rows < 1 || hidden < 8 || hidden % 8 != 0 || num_ranks < 1 || num_buffers < 1 ||
        num_buffers > kMaxBuffers || chunk_bytes < 0)
        return fail(EP_ERR_INVALID_ARG,
                    "ep_staging_alloc: need max_rows >= 1, hidden a positive multiple of 8, "
                    "num_ranks >= 1, 1 <= num_buffers <= %d, chunk_bytes >= 0",
                    kMaxBuffers);
    ep_staging *s = new ep_staging();
    s->kind = kind;
    s->max_rows = max_rows;
    s->hidden = hidden;
    s->num_ranks = num_ranks;
    s->num_buffers = num_buffers;
    s->row_bytes = (int64_t)hidden * 2;
    s->buffer_bytes = max_rows * s->row_bytes;
    int64_t chunk = chunk_bytes == 0 ? kDefaultChunk : chunk_bytes;
    chunk = (chunk + 4095) / 4096 * 4096;
    s->chunk_bytes = chunk;
    s->max_chunks = (int32_t)std::max<int64_t>(1, (s->buffer_bytes + chunk - 1) / chunk);
    s->rows_in.assign((size_t)num_buffers * num_ranks, 0);
    s->off_in.assign((size_t)num_buffers * (num_ranks + 1), 0);
    s->offs_cache.assign((size_t)num_buffers * (num_ranks + 1), 0);
    s->offs_epoch.assign((size_t)num_buffers, 0);
    s->offs_valid.assign((size_t)num_buffers, 0);
    s->offs_sent.assign((size_t)num_buffers, 0);
    s->in_epoch.assign((size_t)num_buffers, 0);

#define EP_ALLOC_HIP(call)                                                                          \
    do {                                                                                            \
        hipError_t e_ = (call);                                                                     \
        if (e_ != hipSuccess) {                                                                     \
            ep_status st_ = hip_fail(e_, #call);                                                    \
            staging_release(s);                                                                     \
            return st_;                                                                             \
        }                                                                                           \
    } while (0)

    EP_ALLOC_HIP(hipGetDevice(&s->device));
    int khz = 0;
    EP_ALLOC_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, s->device));
    if (khz > 0)
        s->wall_clock_khz = khz;
    for (int b = 0; b < num_buffers; ++b) {
        EP_ALLOC_HIP(hipMalloc(&s->dev_send[b], (size_t)s->buffer_bytes));
        EP_ALLOC_HIP(hipMalloc(&s->dev_recv[b], (size_t)s->buffer_bytes));
    }
    if (kind == EP_STAGING_PINNED_HOST) {
        for (int b = 0; b < num_buffers; ++b) {
            EP_ALLOC_HIP(hipHostMalloc(&s->host_send[b], (size_t)s->buffer_bytes, hipHostMallocDefault));
            EP_ALLOC_HIP(hipHostMalloc(&s->host_recv[b], (size_t)s->buffer_bytes, hipHostMallocDefault));
        }
        s->flag_words = ep_staging::flag_words_for(num_buffers, s->max_chunks, num_ranks);
        EP_ALLOC_HIP(hipHostMalloc((void **)&s->flags, s->flag_words * sizeof(uint32_t),
                                   hipHostMallocCoherent));
        std::memset(s->flags, 0, s->flag_words * sizeof(uint32_t));
        EP_ALLOC_HIP(hipStreamCreateWithFlags(&s->up, hipStreamNonBlocking));
        EP_ALLOC_HIP(hipStreamCreateWithFlags(&s->down, hipStreamNonBlocking));
        EP_ALLOC_HIP(hipMalloc((void **)&s->dev_epoch, kMaxBuffers * kEpochStride));
        EP_ALLOC_HIP(hipMalloc((void **)&s->dev_round, 256));
        EP_ALLOC_HIP(hipMemset(s->dev_round, 0, 256));
        EP_ALLOC_HIP(hipEventCreateWithFlags(&s->ev_sysrel, hipEventDisableTiming | hipEventReleaseToSystem));
        if (!d2h_through_hip()) {
            std::string err;
            s->lane = new ep::SdmaLane();
            if (!s->lane->init(s->device, kSdmaSlots, err)) {
                staging_release(s);
                return fail(EP_ERR_HIP, "ep_staging_alloc: SDMA lane: %s", err.c_str());
            }
        }
        for (int b = 0; b < num_buffers; ++b) {
            EP_ALLOC_HIP(hipEventCreateWithFlags(&s->ev_up_in[b], hipEventDisableTiming));
            EP_ALLOC_HIP(hipEventCreateWithFlags(&s->ev_up_done[b], hipEventDisableTiming));
            EP_ALLOC_HIP(hipEventCreateWithFlags(&s->ev_down_in[b], hipEventDisableTiming));
            EP_ALLOC_HIP(hipEventCreateWithFlags(&s->ev_down_done[b], hipEventDisableTiming));
        }
    }
#undef EP_ALLOC_HIP
    *out = s;
    return EP_OK;
}

extern "C" ep_status ep_staging_free(ep_staging *s) {
    if (!s)
        return EP_OK;
    int prev = -1;
    if (hipGetDevice(&prev) == hipSuccess && prev != s->device)
        (void)hipSetDevice(s->device);
    // every stream that used the staging has run (so each SDMA copy has been started)
    (void)hipDeviceSynchronize();
    staging_release(s);
    if (prev >= 0)
        (void)hipSetDevice(prev);
    return EP_OK;
}

extern "C" ep_status ep_staging_ptrs(ep_staging *s, int32_t buf, ep_staging_view *v) {
    if (!s || !v)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_ptrs: NULL argument");
    if (buf < 0 || buf >= s->num_buffers)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_ptrs: buffer %d of %d", buf, s->num_buffers);
    const bool pinned = s->kind == EP_STAGING_PINNED_HOST;
    v->kind = s->kind;
    v->num_ranks = s->num_ranks;
    v->num_buffers = s->num_buffers;
    v->hidden = s->hidden;
    v->max_rows = s->max_rows;
    v->row_bytes = s->row_bytes;
    v->buffer_bytes = s->buffer_bytes;
    v->chunk_bytes = s->chunk_bytes;
    v->max_chunks = s->max_chunks;
    v->dev_send = s->dev_send[buf];
    v->dev_recv = s->dev_recv[buf];
    v->host_send = pinned ? s->host_send[buf] : nullptr;
    v->host_recv = pinned ? s->host_recv[buf] : nullptr;
    v->send_flags = pinned ? s->send_flags(buf) : nullptr;
    v->recv_flags = pinned ? s->recv_flags(buf) : nullptr;
    v->mode = s->mode;
    v->self_rank = s->self_rank;
    v->dev_in = s->dev_in[buf];
    v->host_in = s->host_in[buf];
    v->host_ret = s->host_ret[buf];
    v->in_flags = pinned ? s->in_flags(buf) : nullptr;
    v->ret_flags = pinned ? s->ret_flags(buf) : nullptr;
    v->in_landed = pinned ? s->in_landed(buf) : nullptr;
    v->recv_landed = pinned ? s->recv_landed(buf) : nullptr;
    v->in_offsets = &s->off_in[(size_t)buf * (s->num_ranks + 1)];
    v->send_credits = pinned ? s->send_credit(buf) : nullptr;
    v->recv_credit = pinned ? s->recv_credit(buf) : nullptr;
    return EP_OK;
}

extern "C" ep_status ep_staging_set_mode(ep_staging *s, uint32_t mode, int32_t self_rank) {
    if (!s)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: staging is NULL");
    const uint32_t known = EP_MODE_PER_SENDER | EP_MODE_DUPLEX | EP_MODE_REMOTE_ONLY | EP_MODE_ACCUMULATE;
    if (mode & ~known)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: unknown mode bits 0x%x", mode & ~known);
    if (mode && s->kind != EP_STAGING_PINNED_HOST)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: exchange modes need a PINNED_HOST staging");
    if ((mode & EP_MODE_REMOTE_ONLY) && !(mode & EP_MODE_DUPLEX))
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: EP_MODE_REMOTE_ONLY needs EP_MODE_DUPLEX");
    if ((mode & EP_MODE_ACCUMULATE) && !(mode & EP_MODE_PER_SENDER))
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: EP_MODE_ACCUMULATE needs EP_MODE_PER_SENDER");
    if (mode && s->num_ranks > ep::kMaxExchangeRanks)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: at most %d ranks in the exchange modes, have %d",
                    ep::kMaxExchangeRanks, s->num_ranks);
    if (self_rank < 0 || self_rank >= s->num_ranks)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_mode: self_rank %d outside [0, %d)", self_rank,
                    s->num_ranks);
    ep_status st = check_device(s, "ep_staging_set_mode");
    if (st != EP_OK)
        return st;
    for (hipStream_t side : {s->up, s->down})  // no leg of the previous mode may still run
        if (side) EP_HIP(hipStreamSynchronize(side));
    if (mode & EP_MODE_DUPLEX) {
        // each missing buffer on its own, so a call that failed half-way leaves none NULL
        // behind a later success
        for (int b = 0; b < s->num_buffers; ++b) {
            hipError_t e = hipSuccess;
            void *p = nullptr;
            if (!s->dev_in[b] && (e = hipMalloc(&p, (size_t)s->buffer_bytes)) == hipSuccess)
                s->dev_in[b] = p;
            if (e == hipSuccess && !s->host_in[b] &&
                (e = hipHostMalloc(&p, (size_t)s->buffer_bytes, hipHostMallocDefault)) == hipSuccess)
                s->host_in[b] = p;
            if (e == hipSuccess && !s->host_ret[b] &&
                (e = hipHostMalloc(&p, (size_t)s->buffer_bytes, hipHostMallocDefault)) == hipSuccess)
                s->host_ret[b] = p;
            if (e != hipSuccess)
                return hip_fail(e, "ep_staging_set_mode: duplex buffers");
        }
    }
    if ((mode & EP_MODE_ACCUMULATE) && !s->dev_masks) {
        void *p = nullptr;
        hipError_t e = hipMalloc(&p, (size_t)ep::kMaxBuffers * ep::kMaskWords * sizeof(uint32_t));
        if (e != hipSuccess)
            return hip_fail(e, "ep_staging_set_mode: landed-set words");
        s->dev_masks = static_cast<uint32_t *>(p);
    }
    if (mode && !s->xchg) {
        std::string err;
        s->xchg = ep::exchange_create(s->device, kSdmaSlots, err);
        if (!s->xchg)
            return fail(EP_ERR_HIP, "ep_staging_set_mode: SDMA engines: %s", err.c_str());
    }
    s->mode = mode;
    s->self_rank = self_rank;
    std::fill(s->offs_valid.begin(), s->offs_valid.end(), 0);
    std::fill(s->in_epoch.begin(), s->in_epoch.end(), 0);
    return EP_OK;
}

extern "C" ep_status ep_staging_set_inbound(ep_staging *s, int32_t buf, const int64_t *rows_per_sender) {
    if (!s || !rows_per_sender)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_inbound: NULL argument");
    if (buf < 0 || buf >= s->num_buffers)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_inbound: buffer %d of %d", buf, s->num_buffers);
    int64_t total = 0;
    for (int r = 0; r < s->num_ranks; ++r) {
        if (rows_per_sender[r] < 0)
            return fail(EP_ERR_INVALID_ARG, "ep_staging_set_inbound: negative row count for sender %d", r);
        if (r != s->self_rank)
            total += rows_per_sender[r];
    }
    if (total > s->max_rows)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_inbound: %lld rows from other senders exceed %lld",
                    (long long)total, (long long)s->max_rows);
    for (int r = 0; r < s->num_ranks; ++r)
        s->rows_in[(size_t)buf * s->num_ranks + r] = r == s->self_rank ? 0 : rows_per_sender[r];
    return EP_OK;
}

extern "C" ep_status ep_staging_set_wait(ep_staging *s, int64_t timeout_us, int32_t sleep_units) {
    if (!s || timeout_us < 0 || sleep_units < 0 || sleep_units > 1000)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_set_wait: need timeout_us >= 0, 0 <= sleep_units <= 1000");
    s->timeout_us = timeout_us;
    s->sleep_units = sleep_units;
    return EP_OK;
}

namespace {

// Names a flag word of a staging by its array, buffer set and index.
struct StagingFlagNamer : ep::FlagNamer {
    const ep_staging *s;
    explicit StagingFlagNamer(const ep_staging *st) : s(st) {}
    std::string operator()(const uint32_t *f) const override {
        struct Arr {
            const char *name, *index;
            uint32_t *(ep_staging::*at)(int) const;
            size_t len;
        };
        const size_t R = s->R();
        const Arr arrs[] = {{"send_flags", "chunk", &ep_staging::send_flags, (size_t)s->max_chunks},
                            {"recv_flags", "rank", &ep_staging::recv_flags, R},
                            {"in_flags", "rank", &ep_staging::in_flags, R},
                            {"ret_flags", "rank", &ep_staging::ret_flags, R},
                            {"in_landed", "rank", &ep_staging::in_landed, R},
                            {"recv_landed", "rank", &ep_staging::recv_landed, R},
                            {"send_credits", "rank", &ep_staging::send_credit, R},
                            {"recv_credit", "word", &ep_staging::recv_credit, 1},
                            {"graph_ready", "word", &ep_staging::graph_ready, 1},
                            {"graph_landed", "word", &ep_staging::graph_landed, 1}};
        for (const Arr &a : arrs)
            for (int b = 0; b < s->num_buffers; ++b) {
                const uint32_t *base = (s->*a.at)(b);
                if (f >= base && f < base + a.len) {
                    char buf[96];
                    std::snprintf(buf, sizeof buf, "%s[buf %d][%s %d]", a.name, b, a.index, (int)(f - base));
                    return buf;
                }
            }
        return "";
    }
};

}  // namespace

namespace ep {

ep_status take_status(uint32_t *block, int64_t timeout_us, const FlagNamer &name_flag) {
    const uint32_t word = __atomic_exchange_n(block, 0u, __ATOMIC_ACQ_REL);
    if (word == 0)
        return EP_OK;
    uint32_t d[kStatusWords];
    for (int i = 1; i < kStatusWords; ++i)
        d[i] = __atomic_exchange_n(block + i, 0u, __ATOMIC_RELAXED);
    if (word != EP_ERR_TIMEOUT)
        return fail(EP_ERR_HIP, "unexpected staging status word %u", word);
    const uint32_t *flag = reinterpret_cast<const uint32_t *>((uint64_t)d[2] | ((uint64_t)d[3] << 32));
    std::string name = flag ? name_flag(flag) : std::string();
    if (name.empty()) {
        char buf[40];
        std::snprintf(buf, sizeof buf, "the flag at %p", (const void *)flag);
        name = buf;
    }
    return fail(EP_ERR_TIMEOUT,
                "a completion-flag wait expired after %lld us: %s gave up on %s, which last read %u "
                "(waited for %u)",
                (long long)timeout_us, wait_site_name(d[1]), name.c_str(), d[4], d[5]);
}

}  // namespace ep

extern "C" ep_status ep_staging_status(ep_staging *s, hipStream_t stream) {
    if (!s)
        return fail(EP_ERR_INVALID_ARG, "ep_staging_status: staging is NULL");
    ep_status st = check_device(s, "ep_staging_status");
    if (st != EP_OK)
        return st;
    EP_HIP(hipStreamSynchronize(stream));
    for (hipStream_t side : {s->up, s->down})
        if (side) EP_HIP(hipStreamSynchronize(side));
    if (!s->flags)
        return EP_OK;
    return ep::take_status(s->status(), s->timeout_us, StagingFlagNamer(s));
}

// --------------------------------------------------------------- dispatch / combine

namespace {

ep_status check_round(const ep_staging *s, const char *who, int64_t T, int32_t H, int32_t k,
                      int32_t buf, const int32_t *slot_pos) {
    if (!s)
        return fail(EP_ERR_INVALID_ARG, "%s: staging is NULL", who);
    if (T < 0 || k < 1 || H != s->hidden)
        return fail(EP_ERR_INVALID_ARG, "%s: need T >= 0, k >= 1 and H == staging hidden (%d), got T=%lld k=%d H=%d",
                    who, s->hidden, (long long)T, k, H);
    if (T * (int64_t)k > s->max_rows)
        return fail(EP_ERR_INVALID_ARG, "%s: T*k = %lld rows exceed the staging's %lld", who,
                    (long long)(T * k), (long long)s->max_rows);
    if (buf < 0 || buf >= s->num_buffers)
        return fail(EP_ERR_INVALID_ARG, "%s: buffer %d of %d", who, buf, s->num_buffers);
    if (T > 0 && !slot_pos)
        return fail(EP_ERR_INVALID_ARG, "%s: slot_pos is NULL", who);
    return check_device(s, who);
}

// Host leg of a dispatch in the default pinned mode: the packed rows of s->dev_send[buf]
// go to the host bounce buffer in chunks, one flag per chunk.
ep_status dispatch_default_legs(ep_staging *s, int32_t buf, uint32_t epoch, int64_t rows, hipStream_t stream) {
    const int64_t bytes = rows * s->row_bytes;
    const int64_t chunks = (bytes + s->chunk_bytes - 1) / s->chunk_bytes;
    char *dsrc = static_cast<char *>(s->dev_send[buf]);
    char *hdst = static_cast<char *>(s->host_send[buf]);
    if (s->lane) {
        // SDMA lane: make the packed rows visible at system scope (every XCD's L2), release
        // the lane's start signal from the stream, submit chunk + flag copies to the engine,
        // and let the stream wait (bounded) for the last flag.
        std::string err;
        ep::SdmaLane::Round round;
        if (!s->lane->begin(round, s->timeout_us, err))
            return fail(EP_ERR_TIMEOUT, "ep_dispatch: %s", err.c_str());
        EP_HIP(hipEventRecord(s->ev_sysrel, stream));
        EP_HIP(ep::launch_release_signal(round.start_value, stream));
        if (!s->lane->submit(round, hdst, dsrc, bytes, s->chunk_bytes, s->send_flags(buf), s->epoch_word(buf), err))
            return fail(EP_ERR_HIP, "ep_dispatch: %s", err.c_str());
        const int64_t ticks = s->timeout_us * s->wall_clock_khz / 1000;
        EP_HIP(ep::launch_wait_flags("wait_d2h", s->send_flags(buf) + (chunks - 1), 1, epoch, ticks,
                                     s->sleep_units, s->status(), stream));
        return EP_OK;
    }

    // hipMemcpyAsync path on the up stream: each chunk followed by a 4-byte copy of this
    // round's epoch (written by the pack kernel) into the chunk's flag.
    EP_HIP(hipEventRecord(s->ev_up_in[buf], stream));
    EP_HIP(hipStreamWaitEvent(s->up, s->ev_up_in[buf], 0));
    for (int64_t c = 0; c < chunks; ++c) {
        const int64_t off = c * s->chunk_bytes;
        const int64_t len = std::min<int64_t>(s->chunk_bytes, bytes - off);
        EP_HIP(hipMemcpyAsync(hdst + off, dsrc + off, (size_t)len, hipMemcpyDeviceToHost, s->up));
        EP_HIP(hipMemcpyAsync(s->send_flags(buf) + c, s->epoch_word(buf), sizeof(uint32_t),
                              hipMemcpyDeviceToHost, s->up));
    }
    EP_HIP(hipEventRecord(s->ev_up_done[buf], s->up));
    EP_HIP(hipStreamWaitEvent(stream, s->ev_up_done[buf], 0));
    return EP_OK;
}

}  // namespace

extern "C" ep_status ep_dispatch(const void *x_dev, int64_t num_tokens, int32_t hidden, int32_t topk,
                                 const int32_t *slot_pos, const int32_t *rank_offsets, ep_staging *s,
                                 int32_t buf, uint32_t epoch, hipStream_t stream) {
    ep_status st = check_round(s, "ep_dispatch", num_tokens, hidden, topk, buf, slot_pos);
    if (st != EP_OK)
        return st;
    if (num_tokens > 0 && (!x_dev || !aligned16(x_dev)))
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch: x must be a non-NULL 16-byte aligned pointer");
    const int64_t rows = num_tokens * topk;
    const bool pinned = s->kind == EP_STAGING_PINNED_HOST;
    const bool exchange = pinned && s->mode != 0 && rows > 0;
    if (exchange) {  // the offsets travel to the host while the pack runs
        st = ep::exchange_enqueue_mirror(s, buf, epoch, rank_offsets, stream, "ep_dispatch");
        if (st != EP_OK)
            return st;
    }
    EP_HIP(ep::launch_pack(x_dev, num_tokens, hidden, topk, slot_pos, s->dev_send[buf], s->max_rows,
                           pinned ? s->epoch_word(buf) : nullptr, epoch, stream));
    if (!pinned || rows == 0)
        return EP_OK;
    if (exchange)
        return ep::exchange_dispatch(s, buf, epoch, rows, stream);

    return dispatch_default_legs(s, buf, epoch, rows, stream);
}

extern "C" ep_status ep_dispatch_fused(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                                       int32_t num_experts, int32_t num_ranks, int32_t *expert_counts,
                                       int32_t *expert_offsets, int32_t *rank_counts, int32_t *rank_offsets,
                                       int32_t *slot_pos, int32_t *row_src, void *workspace, size_t workspace_bytes,
                                       const void *x_dev, int32_t hidden, ep_staging *s, int32_t buf, uint32_t epoch,
                                       hipStream_t stream) {
    const int64_t T = num_tokens;
    const int32_t k = topk, E = num_experts, R = num_ranks;
    // every argument of both steps is checked before anything is enqueued
    ep_status st = check_layout_args("ep_dispatch_fused", T, k, E, R, topk_idx, expert_counts, expert_offsets,
                                     rank_counts, rank_offsets, slot_pos, workspace, workspace_bytes);
    if (st != EP_OK)
        return st;
    st = check_round(s, "ep_dispatch_fused", T, hidden, k, buf, slot_pos);
    if (st != EP_OK)
        return st;
    if (T > 0 && (!x_dev || !aligned16(x_dev)))
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch_fused: x must be a non-NULL 16-byte aligned pointer");
    const bool pinned = s->kind == EP_STAGING_PINNED_HOST;
    if ((pinned && s->mode != 0) || !ep::fused_layout_pack_fits(T, k, E, hidden, topk_idx)) {
        // the two steps as separate kernels (the exchange modes also send the offsets to
        // the host between them)
        st = ep_dispatch_layout(topk_idx, T, k, E, R, expert_counts, expert_offsets, rank_counts, rank_offsets,
                                slot_pos, row_src, workspace, workspace_bytes, stream);
        if (st != EP_OK)
            return st;
        return ep_dispatch(x_dev, T, hidden, k, slot_pos, rank_offsets, s, buf, epoch, stream);
    }
    ep::FusedArgs a{};
    a.topk_idx = topk_idx;
    a.T = T;
    a.k = k;
    a.E = E;
    a.R = R;
    a.nbits = E > 1 ? 32 - __builtin_clz((unsigned)(E - 1)) : 0;
    a.expert_counts = expert_counts;
    a.expert_offsets = expert_offsets;
    a.rank_counts = rank_counts;
    a.rank_offsets = rank_offsets;
    a.slot_pos = slot_pos;
    a.row_src = row_src;
    a.status = static_cast<uint32_t *>(workspace);
    a.x = x_dev;
    a.H = hidden;
    a.packed = s->dev_send[buf];
    a.max_rows = s->max_rows;
    a.epoch_word = pinned ? s->epoch_word(buf) : nullptr;
    a.epoch = epoch;
    EP_HIP(ep::launch_layout_pack(a, stream));
    if (!pinned)
        return EP_OK;
    return dispatch_default_legs(s, buf, epoch, T * k, stream);
}

extern "C" ep_status ep_combine(ep_staging *s, int32_t buf, uint32_t epoch, const int32_t *slot_pos,
                                const int32_t *rank_offsets, const float *topk_w, int64_t num_tokens,
                                int32_t hidden, int32_t topk, void *out_dev, ep_out_dtype out_dtype,
                                hipStream_t stream) {
    ep_status st = check_round(s, "ep_combine", num_tokens, hidden, topk, buf, slot_pos);
    if (st != EP_OK)
        return st;
    if (out_dtype != EP_OUT_BF16 && out_dtype != EP_OUT_F32)
        return fail(EP_ERR_INVALID_ARG, "ep_combine: unknown out_dtype %d", (int)out_dtype);
    if (num_tokens > 0 && (!topk_w || !out_dev || !aligned16(out_dev)))
        return fail(EP_ERR_INVALID_ARG, "ep_combine: topk_w and a 16-byte aligned out are required");
    const int64_t rows = num_tokens * topk;
    if (rows == 0)
        return EP_OK;
    if (s->kind == EP_STAGING_PINNED_HOST && (s->mode & EP_MODE_ACCUMULATE)) {
        if (!rank_offsets)  // the passes find each row's sender from the device offsets
            return fail(EP_ERR_INVALID_ARG, "ep_combine: EP_MODE_ACCUMULATE needs rank_offsets");
        // fp32 partial sums of this buffer set, grown on demand (after the device has
        // finished the rounds that used the smaller buffer)
        const size_t need = (size_t)num_tokens * (size_t)hidden * sizeof(float);
        if (s->acc_bytes[buf] < need) {
            if (s->dev_acc[buf]) {
                EP_HIP(hipDeviceSynchronize());
                EP_HIP(hipFree(s->dev_acc[buf]));
                s->dev_acc[buf] = nullptr;
                s->acc_bytes[buf] = 0;
            }
            void *p = nullptr;
            EP_HIP(hipMalloc(&p, need));
            s->dev_acc[buf] = static_cast<float *>(p);
            s->acc_bytes[buf] = need;
        }
        const ep::AccumulateCall call{slot_pos, topk_w, num_tokens, topk, out_dev, out_dtype == EP_OUT_F32};
        return ep::exchange_combine(s, buf, epoch, rows, rank_offsets, stream, &call);
    }
    if (s->kind == EP_STAGING_PINNED_HOST && s->mode != 0) {
        st = ep::exchange_combine(s, buf, epoch, rows, rank_offsets, stream);
        if (st != EP_OK)
            return st;
    } else if (s->kind == EP_STAGING_PINNED_HOST) {
        // Wait (bounded) for every sender's flag, then the host leg as one copy on the
        // caller's stream: the reduction needs every row, and a copy the runtime orders
        // inside one stream reaches the next kernel sooner than one joined from another.
        const int64_t bytes = rows * s->row_bytes;
        const int64_t ticks = s->timeout_us * s->wall_clock_khz / 1000;
        EP_HIP(ep::launch_wait_flags("wait_recv", s->recv_flags(buf), s->num_ranks, epoch, ticks, s->sleep_units,
                                     s->status(), stream));
        // no timing events around this copy: on this runtime their span can exceed the
        // call that holds them, and they delay the copy
        EP_HIP(hipMemcpyAsync(s->dev_recv[buf], s->host_recv[buf], (size_t)bytes, hipMemcpyHostToDevice, stream));
    }
    EP_HIP(ep::launch_combine(s->dev_recv[buf], slot_pos, topk_w, num_tokens, hidden, topk, out_dev,
                              out_dtype == EP_OUT_F32, s->max_rows, stream));
    return EP_OK;
}

// ----------------------------------------------------------- graph-replayed rounds

namespace {

ep_status check_graph(const ep_staging *s, const char *who) {
    if (!s)
        return fail(EP_ERR_INVALID_ARG, "%s: staging is NULL", who);
    if (s->kind != EP_STAGING_PINNED_HOST || s->num_buffers != 2)
        return fail(EP_ERR_INVALID_ARG, "%s: graph rounds need a PINNED_HOST staging with 2 buffer sets", who);
    if (s->num_ranks > 64)
        return fail(EP_ERR_INVALID_ARG, "%s: at most 64 ranks, have %d", who, s->num_ranks);
    return check_device(s, who);
}

}  // namespace

extern "C" ep_status ep_round_advance(ep_staging *s, hipStream_t stream) {
    ep_status st = check_graph(s, "ep_round_advance");
    if (st != EP_OK)
        return st;
    EP_HIP(ep::launch_round_advance(s->dev_round, stream));
    return EP_OK;
}

extern "C" ep_status ep_round_read(ep_staging *s, uint32_t *round) {
    ep_status st = check_graph(s, "ep_round_read");
    if (st != EP_OK)
        return st;
    if (!round)
        return fail(EP_ERR_INVALID_ARG, "ep_round_read: round is NULL");
    EP_HIP(hipDeviceSynchronize());
    EP_HIP(hipMemcpy(round, s->dev_round, sizeof(uint32_t), hipMemcpyDeviceToHost));
    return EP_OK;
}

extern "C" ep_status ep_graph_legs_sdma(ep_staging *s, int32_t on) {
    ep_status st = check_graph(s, "ep_graph_legs_sdma");
    if (st != EP_OK)
        return st;
    if (!on) {
        if (s->graph_legs) {
            EP_HIP(hipDeviceSynchronize());  // no captured round may still wait for the thread
            s->graph_legs->stop();
            delete s->graph_legs;
            s->graph_legs = nullptr;
        }
        return EP_OK;
    }
    if (s->graph_legs)
        return EP_OK;
    // the thread starts at the round the device counter reaches next
    EP_HIP(hipDeviceSynchronize());
    uint32_t round = 0;
    EP_HIP(hipMemcpy(&round, s->dev_round, sizeof round, hipMemcpyDeviceToHost));
    ep::GraphLegsIO io{};
    for (int b = 0; b < 2; ++b) {
        io.ready[b] = s->graph_ready(b);
        io.landed[b] = s->graph_landed(b);
        io.send_flags[b] = s->send_flags(b);
        io.recv_flags[b] = s->recv_flags(b);
        io.recv_credit[b] = s->recv_credit(b);
        io.dev_send[b] = s->dev_send[b];
        io.dev_recv[b] = s->dev_recv[b];
        io.host_send[b] = s->host_send[b];
        io.host_recv[b] = s->host_recv[b];
    }
    io.send_flag_words = s->max_chunks;
    io.senders = s->num_ranks;
    io.status = s->status();
    io.row_bytes = s->row_bytes;
    io.timeout_us = s->timeout_us;
    ep::GraphLegs *g = new ep::GraphLegs();
    std::string err;
    if (!g->dma.init(s->device, err)) {
        g->dma.release();  // drops the ROCr reference init may have taken
        delete g;
        return fail(EP_ERR_HIP, "ep_graph_legs_sdma: %s", err.c_str());
    }
    g->start(io, round + 1u);
    s->graph_legs = g;
    return EP_OK;
}

extern "C" ep_status ep_dispatch_graph(const void *x_dev, int64_t num_tokens, int32_t hidden, int32_t topk,
                                       const int32_t *slot_pos, ep_staging *s, hipStream_t stream) {
    ep_status st = check_graph(s, "ep_dispatch_graph");
    if (st == EP_OK)
        st = check_round(s, "ep_dispatch_graph", num_tokens, hidden, topk, 0, slot_pos);
    if (st != EP_OK)
        return st;
    if (num_tokens > 0 && (!x_dev || !aligned16(x_dev)))
        return fail(EP_ERR_INVALID_ARG, "ep_dispatch_graph: x must be a non-NULL 16-byte aligned pointer");
    const int64_t ticks = s->timeout_us * s->wall_clock_khz / 1000;
    // buffer set round % 2 is free once every receiver credited its contents of two rounds ago
    EP_HIP(ep::launch_round_gate("wait_credits", s->dev_round, s->send_credit(0), s->num_ranks, s->num_ranks, -2,
                                 ticks, s->sleep_units, s->status(), stream));
    // the rows go to pinned memory from the compute units, or with SDMA legs to the device
    // send buffer, from which the legs' thread copies them once the ready word holds the round
    const bool sdma = s->graph_legs != nullptr;
    if (sdma)
        s->graph_legs->set_rows(num_tokens * topk);
    void *const *dst = sdma ? s->dev_send : s->host_send;
    ep::RoundSel sel;
    sel.alt = dst[1];
    sel.round = s->dev_round;
    EP_HIP(ep::launch_pack(x_dev, num_tokens, hidden, topk, slot_pos, dst[0], s->max_rows, nullptr, 0, stream, sel,
                           true));
    if (sdma)
        EP_HIP(ep::launch_round_stamp(s->dev_round, s->graph_ready(0), 1, 1, stream));
    else
        EP_HIP(ep::launch_round_stamp(s->dev_round, s->send_flags(0), s->max_chunks, 1, stream));
    return EP_OK;
}

extern "C" ep_status ep_combine_graph(ep_staging *s, const int32_t *slot_pos, const float *topk_w,
                                      int64_t num_tokens, int32_t hidden, int32_t topk, void *out_dev,
                                      ep_out_dtype out_dtype, hipStream_t stream) {
    ep_status st = check_graph(s, "ep_combine_graph");
    if (st == EP_OK)
        st = check_round(s, "ep_combine_graph", num_tokens, hidden, topk, 0, slot_pos);
    if (st != EP_OK)
        return st;
    if (out_dtype != EP_OUT_BF16 && out_dtype != EP_OUT_F32)
        return fail(EP_ERR_INVALID_ARG, "ep_combine_graph: unknown out_dtype %d", (int)out_dtype);
    if (num_tokens > 0 && (!topk_w || !out_dev || !aligned16(out_dev)))
        return fail(EP_ERR_INVALID_ARG, "ep_combine_graph: topk_w and a 16-byte aligned out are required");
    const int64_t ticks = s->timeout_us * s->wall_clock_khz / 1000;
    // the rows are read from pinned memory by the compute units, or with SDMA legs from the
    // device receive buffer once the legs' thread has copied every sender's rows there
    const bool sdma = s->graph_legs != nullptr;
    if (sdma)
        EP_HIP(ep::launch_round_gate("wait_graph_landed", s->dev_round, s->graph_landed(0), 1, 1, 0, ticks,
                                     s->sleep_units, s->status(), stream));
    else
        EP_HIP(ep::launch_round_gate("wait_returned", s->dev_round, s->recv_flags(0), s->num_ranks, s->num_ranks, 0,
                                     ticks, s->sleep_units, s->status(), stream));
    void *const *src = sdma ? s->dev_recv : s->host_recv;
    ep::RoundSel sel;
    sel.alt = src[1];
    sel.round = s->dev_round;
    EP_HIP(ep::launch_combine(src[0], slot_pos, topk_w, num_tokens, hidden, topk, out_dev, out_dtype == EP_OUT_F32,
                              s->max_rows, stream, sel));
    // the returned rows of this round are consumed: credit the buffer set to the senders
    EP_HIP(ep::launch_round_stamp(s->dev_round, s->recv_credit(0), 1, 1, stream));
    return EP_OK;
}

// ---------------------------------------------------------------------- measurement

extern "C" ep_status ep_trace_enable(int32_t on) {
    ep::g_trace_on.store(on != 0);
    return EP_OK;
}

extern "C" ep_status ep_trace_read(ep_trace_stat *stats, int32_t capacity, int32_t *count) {
    if (!count || capacity < 0 || (capacity > 0 && !stats))
        return fail(EP_ERR_INVALID_ARG, "ep_trace_read: bad arguments");
    std::lock_guard<std::mutex> lk(ep::g_trace_mu);
    // every pending pair goes back to the pool exactly once, also after a failed query
    hipError_t first = hipSuccess;
    for (auto &p : ep::g_pending) {
        float ms = 0.f;
        hipError_t e = hipEventSynchronize(p.stop);
        if (e == hipSuccess)
            e = hipEventElapsedTime(&ms, p.start, p.stop);
        if (e == hipSuccess)
            ep::g_stats[p.name].add(ms);
        else if (first == hipSuccess)
            first = e;
        ep::g_event_pool.push_back(p.start);
        ep::g_event_pool.push_back(p.stop);
    }
    ep::g_pending.clear();
    if (first != hipSuccess)
        return hip_fail(first, "ep_trace_read: timing events");
    int32_t n = 0;
    for (auto &kv : ep::g_stats) {
        if (n < capacity) {
            ep_trace_stat &o = stats[n];
            std::memset(&o, 0, sizeof o);
            std::snprintf(o.name, sizeof o.name, "%s", kv.first.c_str());
            o.count = kv.second.count;
            o.total_ms = kv.second.total;
            o.min_ms = kv.second.count ? kv.second.mn : 0.0;
            o.max_ms = kv.second.mx;
            o.p10_ms = ep::percentile(kv.second.samples, 0.1);
            o.p50_ms = ep::percentile(kv.second.samples, 0.5);
            o.p90_ms = ep::percentile(kv.second.samples, 0.9);
        }
        ++n;
    }
    *count = std::min(n, capacity);
    return EP_OK;
}

extern "C" ep_status ep_trace_reset(void) {
    std::lock_guard<std::mutex> lk(ep::g_trace_mu);
    for (auto &p : ep::g_pending) {
        (void)hipEventSynchronize(p.stop);
        ep::g_event_pool.push_back(p.start);
        ep::g_event_pool.push_back(p.stop);
    }
    ep::g_pending.clear();
    ep::g_stats.clear();
    return EP_OK;
}

extern "C" ep_status ep_copy_probe(void *dst_dev, const void *src_dev, size_t bytes, hipStream_t stream) {
    if (bytes % 16 != 0 || (bytes && (!dst_dev || !src_dev || !aligned16(dst_dev) || !aligned16(src_dev))))
        return fail(EP_ERR_INVALID_ARG, "ep_copy_probe: 16-byte aligned pointers and a multiple of 16 bytes");
    EP_HIP(ep::launch_copy(dst_dev, src_dev, bytes, stream));
    return EP_OK;
}

extern "C" ep_status ep_stream_probe(void *dst_dev, const void *src_dev, int64_t units, int32_t row_bytes,
                                     int32_t reads, int32_t writes, int32_t store_policy, hipStream_t stream) {
    const int g = row_bytes / 1024;
    const bool shape = row_bytes > 0 && row_bytes % 1024 == 0 &&
                       (g == 1 || g == 2 || g == 4 || g == 8 || g == 14 || g == 16);
    if (units < 0 || !shape || reads < 0 || writes < 0 || reads + writes == 0 || reads > 64 || writes > 64 ||
        store_policy < 0 || store_policy > 2)
        return fail(EP_ERR_INVALID_ARG, "ep_stream_probe: need units >= 0, row_bytes = 1024 * {1,2,4,8,14,16}, "
                                        "0 <= reads, writes <= 64, reads + writes > 0, store_policy 0, 1 or 2");
    if (units > 0 && (!dst_dev || !aligned16(dst_dev) || (reads > 0 && (!src_dev || !aligned16(src_dev)))))
        return fail(EP_ERR_INVALID_ARG, "ep_stream_probe: 16-byte aligned src (when reading) and dst are required");
    EP_HIP(ep::launch_stream_probe(dst_dev, src_dev, units, row_bytes, reads, writes, store_policy, stream));
    return EP_OK;
}

extern "C" ep_status ep_memcpy(void *dst, const void *src, size_t bytes, hipStream_t stream) {
    if (bytes && (!dst || !src))
        return fail(EP_ERR_INVALID_ARG, "ep_memcpy: NULL pointer");
    if (bytes)
        EP_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, stream));
    return EP_OK;
}
