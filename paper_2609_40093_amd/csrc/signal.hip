// signal.hip -- completion flags in pinned host memory (Sec. 4.4 of the paper).
//
// The payload stays contiguous and the flags live apart from it, one 32-bit word per
// sender (receive side) or per DMA chunk (send side, written by a 4-byte DMA copy queued
// behind the chunk), each with a single writer, so no atomic read-modify-write is needed.  A flag holds the epoch of the round that filled
// its data; a reader accepts it when (int32)(flag - epoch) >= 0, so a flag left over from
// an earlier round is never taken for the current one.
//
// wait_flags_kernel: one lane per remote sender polls its flag with system-scope loads
// (they bypass the GPU caches and cross PCIe) and sleeps between polls, instead of a
// large thread block spinning.  The wait is bounded by the constant-rate wall clock; on
// expiry the kernel records the timeout in the host status block (where it waited, the
// flag, the value it last read and the value it wanted) and exits, so the stream never
// hangs on a flag that does not come.
#include "ep_internal.h"

namespace ep {
namespace {

constexpr uint32_t kStatusTimeout = 5u;  // EP_ERR_TIMEOUT

// Records an expired wait in the status block: the details first, then the status word
// with release order (one lane per wave calls it).
__device__ void record_timeout(uint32_t *status, uint32_t site, const uint32_t *flag, uint32_t seen, uint32_t want) {
    const uint64_t a = reinterpret_cast<uint64_t>(flag);
    __hip_atomic_store(status + 1, site, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(status + 2, (uint32_t)a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(status + 3, (uint32_t)(a >> 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(status + 4, seen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(status + 5, want, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(status, kStatusTimeout, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// The lowest lane of the wave for which `pending` holds (-1 if none).
__device__ inline int first_lane(bool pending) {
    const uint64_t m = __ballot(pending);
    return m ? __builtin_ctzll(m) : -1;
}

__global__ __launch_bounds__(64) void wait_flags_kernel(const uint32_t *flags, int32_t n,
                                                        uint32_t epoch, int64_t timeout_ticks,
                                                        int32_t sleep_units, uint32_t *status, uint32_t site) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    bool done = i >= n;
    uint32_t seen = 0;
    const int64_t t0 = wall_clock64();
    bool late = false;
    while (!__all(done)) {
        if (!done) {
            seen = __hip_atomic_load(flags + i, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
            done = (int32_t)(seen - epoch) >= 0;
        }
        if (wall_clock64() - t0 > timeout_ticks) {
            late = true;
            break;
        }
        for (int32_t s = 0; s < sleep_units; ++s)
            __builtin_amdgcn_s_sleep(1);
    }
    if (late && (int)threadIdx.x == first_lane(!done))
        record_timeout(status, site, flags + i, seen, epoch);
}

// Releases a DMA-engine dependency: stores 0 into a signal value the engine polls.
__global__ __launch_bounds__(64) void release_signal_kernel(int64_t *value) {
    if (threadIdx.x == 0)
        __hip_atomic_store(value, (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Waits for a list of flags (any memory) and releases DMA copies as they arrive: lane i
// polls flag[i] until it holds the epoch; per-flag mode then stores 0 into release[i] at
// once (that sender's copy starts while other senders are still working), all-flags mode
// stores 0 into release[0] when the last flag is in.  A null release only waits.  On
// timeout every remaining release is still stored, so no queued copy waits forever; the
// status word records the timeout.
__global__ __launch_bounds__(64) void gate_kernel(GateArgs g) {
    const int i = threadIdx.x;
    bool done = i >= g.n;
    bool released = done || g.all || !g.release[i];
    uint32_t seen = 0;
    const int64_t t0 = wall_clock64();
    bool late = false;
    while (!__all(done)) {
        if (!done) {
            seen = __hip_atomic_load(g.flag[i], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
            if ((int32_t)(seen - g.epoch) >= 0) {
                done = true;
                if (!released) {
                    __hip_atomic_store(g.release[i], (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
                    released = true;
                }
            }
        }
        if (wall_clock64() - t0 > g.timeout_ticks) {
            late = true;
            break;
        }
        for (int32_t s = 0; s < g.sleep_units; ++s)
            __builtin_amdgcn_s_sleep(1);
    }
    if (late) {
        if (i == first_lane(!done))
            record_timeout(g.status, g.site, g.flag[i], seen, g.epoch);
        if (!released)
            __hip_atomic_store(g.release[i], (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    if (g.all && i == 0 && g.release[0])
        __hip_atomic_store(g.release[0], (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Stores the round's epoch into the row of words the DMA flag copies read (a merged flag
// copy reads one word per flag), then releases the copies.
__global__ __launch_bounds__(64) void stamp_release_kernel(uint32_t *epoch_word, uint32_t epoch, int64_t *value) {
    static_assert(kEpochRowWords <= 64, "one lane per word of the epoch row");
    if (threadIdx.x < kEpochRowWords)
        __hip_atomic_store(epoch_word + threadIdx.x, epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_store(value, (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Copies n int32 values (rank offsets) to host memory, then the epoch as a tag after them.
__global__ __launch_bounds__(64) void mirror_kernel(const int32_t *src, int32_t n, uint32_t *host, uint32_t epoch) {
    if (threadIdx.x != 0)
        return;
    for (int i = 0; i < n; ++i)  // one thread: its release below orders every store before it
        __hip_atomic_store(host + i, (uint32_t)src[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(host + n, epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Graph-replayed rounds read their round number from device memory, so the captured
// launches stay valid from one replay to the next.
__global__ __launch_bounds__(64) void round_advance_kernel(uint32_t *round) {
    if (threadIdx.x == 0)  // agent scope: every XCD's later kernels read the new value
        __hip_atomic_fetch_add(round, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until flags[(round % 2) * stride + i] has reached round + delta, i < n (one lane
// per flag, pausing between polls, bounded by the wall clock).
__global__ __launch_bounds__(64) void round_gate_kernel(const uint32_t *round_ptr, const uint32_t *flags,
                                                        int32_t stride, int32_t n, int32_t delta, int64_t timeout_ticks,
                                                        int32_t sleep_units, uint32_t *status, uint32_t site) {
    const int32_t i = threadIdx.x;
    const uint32_t round = __hip_atomic_load(round_ptr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t want = round + (uint32_t)delta;
    const uint32_t *f = flags + (round & 1u) * (uint32_t)stride + i;
    bool done = i >= n;
    uint32_t seen = 0;
    const int64_t t0 = wall_clock64();
    bool late = false;
    while (!__all(done)) {
        if (!done) {
            seen = __hip_atomic_load(f, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
            done = (int32_t)(seen - want) >= 0;
        }
        if (wall_clock64() - t0 > timeout_ticks) {
            late = true;
            break;
        }
        for (int32_t s = 0; s < sleep_units; ++s)
            __builtin_amdgcn_s_sleep(1);
    }
    if (late && i == first_lane(!done))
        record_timeout(status, site, f, seen, want);
}

// Publishes the round: after a system-scope release, words[(round % 2) * stride + i] =
// round for i < n (a send flag, or a credit for a consumed buffer).
__global__ __launch_bounds__(64) void round_stamp_kernel(const uint32_t *round_ptr, uint32_t *words, int32_t stride,
                                                         int32_t n) {
    const int32_t i = threadIdx.x;
    if (i >= n)
        return;
    const uint32_t round = __hip_atomic_load(round_ptr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(words + (round & 1u) * (uint32_t)stride + i, round, __ATOMIC_RELEASE,
                       __HIP_MEMORY_SCOPE_SYSTEM);
}

// The set of senders whose rows pass i of the per-sender accumulation may add: the set of
// pass i - 1 (masks[i]; empty before pass 0) with the senders of `base` (rows that need no
// wait) and those whose landed[r] holds the epoch.  Waits (one lane per sender, pausing
// between polls, bounded by the wall clock) until it holds a sender outside pass i - 1's
// set and `base`, or every sender, so that every pass adds a sender that was waited for
// and one pass per such sender suffices.  Records the set in masks[i + 1] (and the empty
// set in masks[0]).  On expiry it records every sender (the rows still missing are
// reduced as they are) and leaves a timeout in the status word.
__global__ __launch_bounds__(64) void landed_set_kernel(const uint32_t *landed, int32_t R, uint32_t epoch,
                                                        uint32_t base, uint32_t *masks, int32_t i,
                                                        int64_t timeout_ticks, int32_t sleep_units,
                                                        uint32_t *status) {
    const int lane = threadIdx.x;
    const uint32_t full = R >= 32 ? ~0u : ((1u << R) - 1u);
    const uint32_t prev = i == 0 ? 0u : __hip_atomic_load(masks + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t start = prev | base;
    uint32_t m = start;
    const int64_t t0 = wall_clock64();
    for (;;) {
        bool in = false;
        if (lane < R && !((start >> lane) & 1u))
            in = (int32_t)(__hip_atomic_load(landed + lane, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM) - epoch) >= 0;
        m = start | (uint32_t)__ballot(in);
        if (m != start || m == full)
            break;
        if (wall_clock64() - t0 > timeout_ticks) {
            const bool missing = lane < R && !((m >> lane) & 1u);
            if (lane == first_lane(missing))
                record_timeout(status, kSiteLandedSet, landed + lane,
                               __hip_atomic_load(landed + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM), epoch);
            m = full;
            break;
        }
        for (int32_t s = 0; s < sleep_units; ++s)
            __builtin_amdgcn_s_sleep(1);
    }
    if (lane == 0) {
        if (i == 0)
            __hip_atomic_store(masks, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(masks + i + 1, m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

}  // namespace

hipError_t launch_landed_set(const uint32_t *landed, int32_t R, uint32_t epoch, uint32_t base, uint32_t *masks,
                             int32_t i, int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream) {
    if (!landed || !masks || R < 1 || R > 32 || i < 0)
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(landed_set_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, landed, R, epoch,
                          base, masks, i, timeout_ticks, sleep_units, status);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("landed_set", ts);
    return err;
}

hipError_t launch_round_advance(uint32_t *round, hipStream_t stream) {
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(round_advance_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, round);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("round_advance", ts);
    return err;
}

hipError_t launch_round_gate(const char *name, const uint32_t *round, const uint32_t *flags, int32_t stride,
                             int32_t n, int32_t delta, int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    if (n > 64)
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(round_gate_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, round, flags, stride,
                          n, delta, timeout_ticks, sleep_units, status, wait_site(name));
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit(name, ts);
    return err;
}

hipError_t launch_round_stamp(const uint32_t *round, uint32_t *words, int32_t stride, int32_t n, hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    if (n > 64)
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(round_stamp_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, round, words,
                          stride, n);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("round_stamp", ts);
    return err;
}

hipError_t launch_gate(const char *name, const GateArgs &g, hipStream_t stream) {
    if (g.n <= 0 || g.n > kMaxGate)
        return g.n == 0 ? hipSuccess : hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    GateArgs named = g;
    named.site = wait_site(name);
    hipExtLaunchKernelGGL(gate_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, named);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit(name, ts);
    return err;
}

hipError_t launch_stamp_release(uint32_t *epoch_word, uint32_t epoch, int64_t *value, hipStream_t stream) {
    if (!epoch_word || !value)  // e.g. a signal whose value pointer could not be read
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(stamp_release_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, epoch_word,
                          epoch, value);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("release_signal", ts);
    return err;
}

hipError_t launch_mirror(const int32_t *src, int32_t n, uint32_t *host, uint32_t epoch, hipStream_t stream) {
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(mirror_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, src, n, host, epoch);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("mirror_offsets", ts);
    return err;
}

hipError_t launch_release_signal(int64_t *value, hipStream_t stream) {
    if (!value)
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(release_signal_kernel, dim3(1), dim3(64), 0, stream, ts.start, ts.stop, 0, value);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("release_signal", ts);
    return err;
}

hipError_t launch_wait_flags(const char *name, const uint32_t *flags, int32_t n, uint32_t epoch,
                             int64_t timeout_ticks, int32_t sleep_units, uint32_t *status,
                             hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(wait_flags_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, stream,
                          ts.start, ts.stop, 0, flags, n, epoch, timeout_ticks, sleep_units, status, wait_site(name));
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit(name, ts);
    return err;
}

namespace {
constexpr const char *kSiteNames[kSiteCount] = {
    "unknown wait",  "wait_d2h",      "wait_recv",    "wait_dispatch",  "wait_combine",       "wait_returned_out",
    "landed_set",    "wait_credits",  "wait_returned", "wait_allgather", "wait_reducescatter", "the inbound-copy courier",
    "wait_graph_landed", "the graph rounds' host-leg thread",
};
}  // namespace

uint32_t wait_site(const char *launch_name) {
    for (uint32_t i = 1; i < kSiteCount; ++i) {
        const char *a = kSiteNames[i], *b = launch_name;
        while (*a && *a == *b)
            ++a, ++b;
        if (!*a && !*b)
            return i;
    }
    return kSiteUnknown;
}

const char *wait_site_name(uint32_t site) { return site < kSiteCount ? kSiteNames[site] : kSiteNames[0]; }

}  // namespace ep
