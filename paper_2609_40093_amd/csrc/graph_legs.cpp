// graph_legs.cpp -- host legs of graph-replayed rounds on SDMA engines (ep_graph_legs_sdma).
//
// A captured graph replays the same launches every round, so it cannot hold DMA copies
// whose source and destination change with the round's buffer set.  With these legs the
// captured kernels stay on the device side of the staging: ep_dispatch_graph packs into
// the device send buffer of set round % 2 and stamps that set's ready word in host memory;
// ep_combine_graph waits (bounded) for the set's landed word in host memory and reduces
// from the device receive buffer.  A library thread moves the rows in between on SDMA
// engines (Sec. 4.3 of the paper: bulk data on the DMA engines, no compute unit spent on
// it), round r = 1, 2, ... on set r % 2:
//   1. waits until ready[set] holds r (the packed rows are in device memory, written back
//      past every L2 by the pack's system-scope release);
//   2. copies them to the pinned send buffer on the device->host engine and, once they
//      have landed, sets the set's send flags to r (Sec. 4.4: flags after the data);
//   3. waits for every sender's recv flag of the set to reach r and for this rank's
//      receive credit of round r - 2 (the device receive buffer has been reduced);
//   4. copies the returned rows to the device receive buffer on the host->device engine
//      and, once they have landed, sets landed[set] = r.
// Each copy is queued only once the host has seen that its source is complete, so no
// engine waits on a signal that the device releases.  The waits of steps 2 to 4 are
// bounded by the staging's timeout: one that expires is recorded in the status block and
// the round goes on (its flags are still raised), so that no device wait is left to run
// out its own bound.  Step 1 has no bound: the device reaches a round whenever the
// caller replays it.
#include "exchange.h"
#include "staging.h"

#include <immintrin.h>

#include <atomic>
#include <chrono>
#include <string>
#include <thread>

namespace ep {

class GraphLegs {
public:
    explicit GraphLegs(ep_staging *s) : s_(s) {}

    // Takes SDMA engines and starts the thread at round `first` (the round the device
    // counter reaches next).
    bool start(uint32_t first, std::string &err) {
        if (!dma_.init(s_->device, err)) {
            dma_.release();  // drops the ROCr reference init may have taken
            return false;
        }
        slots_.init(2);
        first_ = first;
        th_ = std::thread([this] { run(); });
        return true;
    }
    // Rows of every round from the next one on (T * top-k of the captured dispatch).
    void set_rows(int64_t rows) { rows_.store(rows, std::memory_order_release); }
    // Ends the thread (between rounds, or in a wait), waits for its copies in flight, then
    // frees their signals and the engines' ROCr reference.
    void stop() {
        stop_.store(true, std::memory_order_release);
        if (th_.joinable())
            th_.join();
        std::string err;
        slots_.destroy(slots_.drain(kReleaseDrainUs, err));
        dma_.release();
    }
    const std::string &engines() const { return dma_.describe(); }

private:
    using Clock = std::chrono::steady_clock;
    enum Wait { kDone, kLate, kStopped };

    // Waits until (int32)(*w - want) >= 0.  A bounded wait gives up after the staging's
    // timeout and records the flag in the status block.
    Wait wait_word(const uint32_t *w, uint32_t want, bool bounded) {
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
            if (bounded && waited > std::chrono::microseconds(s_->timeout_us)) {
                record_host_timeout(s_->status(), kSiteGraphLegs, w, want);
                return kLate;
            }
            if (waited > std::chrono::milliseconds(10))  // an idle caller: poll less often
                std::this_thread::sleep_for(std::chrono::microseconds(50));
            else
                std::this_thread::yield();
        }
    }

    // One copy on `engine`, then a bounded wait on the host until it has landed.  A copy
    // that cannot be queued leaves EP_ERR_HIP in the status block.
    bool copy(int slot, uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
              const uint32_t *names_flag, uint32_t want) {
        std::string err;
        hsa_signal_t g{};
        if (!slots_.take(slot, g, err) || !dma_.copy(engine, dst, dst_host, src, src_host, len, nullptr, 0, g, err)) {
            __atomic_store_n(s_->status(), (uint32_t)EP_ERR_HIP, __ATOMIC_RELEASE);
            return false;
        }
        slots_.arm(slot, g);
        const auto t0 = Clock::now();
        for (uint32_t spins = 1;; ++spins) {
            const hsa_signal_value_t v = hsa_signal_load_scacquire(g);
            if (v <= 0) {
                if (v < 0)  // the runtime reports a failed copy
                    __atomic_store_n(s_->status(), (uint32_t)EP_ERR_HIP, __ATOMIC_RELEASE);
                return v == 0;
            }
            if ((spins & 255u) != 0) {
                _mm_pause();
                continue;
            }
            if (Clock::now() - t0 > std::chrono::microseconds(s_->timeout_us)) {
                // named by the flag the copy precedes: it is raised late, or with rows missing
                record_host_timeout(s_->status(), kSiteGraphLegs, names_flag, want);
                return false;
            }
            std::this_thread::yield();
        }
    }

    void run() {
        for (uint32_t r = first_;; ++r) {
            const int b = (int)(r & 1u);
            if (wait_word(s_->graph_ready(b), r, false) == kStopped)
                return;
            const size_t bytes = (size_t)(rows_.load(std::memory_order_acquire) * s_->row_bytes);
            std::string err;
            const int slot = slots_.begin(s_->timeout_us, err);  // both copies of the previous use landed
            const bool have_slot = slot >= 0;
            if (!have_slot)
                record_host_timeout(s_->status(), kSiteGraphLegs, s_->send_flags(b), r);
            // outbound: device send buffer -> pinned send buffer, then the send flags
            if (have_slot && bytes > 0)
                copy(slot, dma_.out_engine(), s_->host_send[b], true, s_->dev_send[b], false, bytes, s_->send_flags(b),
                     r);
            for (int c = 0; c < s_->max_chunks; ++c)
                __atomic_store_n(s_->send_flags(b) + c, r, __ATOMIC_RELEASE);
            // inbound: every sender's rows are back and the device receive buffer is free (after
            // one wait has expired the others are not waited for: the round is already late)
            bool late = false;
            for (int i = 0; i <= s_->num_ranks && !late; ++i) {
                const Wait w = i < s_->num_ranks ? wait_word(s_->recv_flags(b) + i, r, true)
                                                 : wait_word(s_->recv_credit(b), r - 2u, true);
                if (w == kStopped)
                    return;
                late = w == kLate;
            }
            if (have_slot && bytes > 0)
                copy(slot, dma_.in_engine(0), s_->dev_recv[b], false, s_->host_recv[b], true, bytes,
                     s_->graph_landed(b), r);
            __atomic_store_n(s_->graph_landed(b), r, __ATOMIC_RELEASE);
        }
    }

    ep_staging *s_;
    DmaEngines dma_;
    SignalSlots slots_;
    std::thread th_;
    std::atomic<int64_t> rows_{0};
    std::atomic<bool> stop_{false};
    uint32_t first_ = 1;
};

GraphLegs *graph_legs_create(ep_staging *s, uint32_t first_round, std::string &err) {
    GraphLegs *g = new GraphLegs(s);
    if (!g->start(first_round, err)) {
        delete g;
        return nullptr;
    }
    return g;
}

void graph_legs_destroy(GraphLegs *g) {
    if (!g)
        return;
    g->stop();
    delete g;
}

void graph_legs_set_rows(GraphLegs *g, int64_t rows) {
    if (g)
        g->set_rows(rows);
}

}  // namespace ep
