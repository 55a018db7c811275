// graph_legs.cpp -- the host-leg thread of graph-replayed rounds with SDMA legs
// (graph_legs.h has the protocol).
#include "graph_legs.h"

#include "ep.h"
#include "status_block.h"

#include <immintrin.h>

#include <chrono>

namespace ep {

namespace {
using Clock = std::chrono::steady_clock;
}

void GraphLegs::start(const GraphLegsIO &io, uint32_t first) {
    io_ = io;
    slots_.init(2);
    first_ = first;
    th_ = std::thread([this] { run(); });
}

void GraphLegs::stop() {
    stop_.store(true, std::memory_order_release);
    if (th_.joinable())
        th_.join();
    std::string err;
    slots_.destroy(slots_.drain(kReleaseDrainUs, err));
    dma.release();
}

// Waits until (int32)(*w - want) >= 0.  A bounded wait gives up after the timeout and
// records the flag in the status block.
GraphLegs::Wait GraphLegs::wait_word(const uint32_t *w, uint32_t want, bool bounded) {
    const auto t0 = Clock::now();
    for (uint32_t spins = 1;; ++spins) {
        if ((int32_t)(__atomic_load_n(w, __ATOMIC_ACQUIRE) - want) >= 0)
            return kDone;
        if ((spins & 255u) != 0) {
            _mm_pause();
            continue;
        }
        if (stop_.load(std::memory_order_acquire))
            return kStopped;
        const auto waited = Clock::now() - t0;
        if (bounded && waited > std::chrono::microseconds(io_.timeout_us)) {
            record_host_timeout(io_.status, kSiteGraphLegs, w, want);
            return kLate;
        }
        if (waited > std::chrono::milliseconds(10))  // an idle caller: poll less often
            std::this_thread::sleep_for(std::chrono::microseconds(50));
        else
            std::this_thread::yield();
    }
}

// One copy on `engine`, then a bounded wait on the host until it has landed.  A copy that
// cannot be queued, or that the runtime reports as failed, leaves EP_ERR_HIP in the status
// block; one that does not land in time is recorded under the flag it precedes.
bool GraphLegs::copy(int slot, uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
                     const uint32_t *names_flag, uint32_t want) {
    std::string err;
    hsa_signal_t g{};
    if (!slots_.take(slot, g, err) || !dma.copy(engine, dst, dst_host, src, src_host, len, nullptr, 0, g, err)) {
        __atomic_store_n(io_.status, (uint32_t)EP_ERR_HIP, __ATOMIC_RELEASE);
        return false;
    }
    slots_.arm(slot, g);
    const auto t0 = Clock::now();
    for (uint32_t spins = 1;; ++spins) {
        const hsa_signal_value_t v = hsa_signal_load_scacquire(g);
        if (v <= 0) {
            if (v < 0)
                __atomic_store_n(io_.status, (uint32_t)EP_ERR_HIP, __ATOMIC_RELEASE);
            return v == 0;
        }
        if ((spins & 255u) != 0) {
            _mm_pause();
            continue;
        }
        if (Clock::now() - t0 > std::chrono::microseconds(io_.timeout_us)) {
            record_host_timeout(io_.status, kSiteGraphLegs, names_flag, want);
            return false;
        }
        std::this_thread::yield();
    }
}

void GraphLegs::run() {
    for (uint32_t r = first_;; ++r) {
        const int b = (int)(r & 1u);
        if (wait_word(io_.ready[b], r, false) == kStopped)
            return;
        const size_t bytes = (size_t)(rows_.load(std::memory_order_acquire) * io_.row_bytes);
        std::string err;
        const int slot = slots_.begin(io_.timeout_us, err);  // the copies of the slot's last use landed
        const bool have_slot = slot >= 0;
        if (!have_slot)
            record_host_timeout(io_.status, kSiteGraphLegs, io_.send_flags[b], r);
        // outbound: device send buffer -> pinned send buffer, then the send flags
        if (have_slot && bytes > 0)
            copy(slot, dma.out_engine(), io_.host_send[b], true, io_.dev_send[b], false, bytes, io_.send_flags[b], r);
        for (int c = 0; c < io_.send_flag_words; ++c)
            __atomic_store_n(io_.send_flags[b] + c, r, __ATOMIC_RELEASE);
        // inbound: every sender's rows are back and the device receive buffer is free (after
        // one wait has expired the others are not waited for: the round is already late)
        bool late = false;
        for (int i = 0; i <= io_.senders && !late; ++i) {
            const Wait w = i < io_.senders ? wait_word(io_.recv_flags[b] + i, r, true)
                                           : wait_word(io_.recv_credit[b], r - 2u, true);
            if (w == kStopped)
                return;
            late = w == kLate;
        }
        if (have_slot && bytes > 0)
            copy(slot, dma.in_engine(0), io_.dev_recv[b], false, io_.host_recv[b], true, bytes, io_.landed[b], r);
        __atomic_store_n(io_.landed[b], r, __ATOMIC_RELEASE);
    }
}

}  // namespace ep
