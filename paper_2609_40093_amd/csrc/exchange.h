// exchange.h -- SDMA queueing shared by the host legs of the exchange modes (exchange.cpp)
// and of the dense collectives (dense.cpp): per-call signal slots, and the courier thread
// that queues host->device copies as their senders' flags arrive.
#pragma once

#include "ep.h"
#include "sdma.h"

#include <immintrin.h>

#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <deque>
#include <functional>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

namespace ep {

// Signals and completion flags of one call (a dispatch or a combine).  A slot is reused
// only once every flag its previous call raised holds that call's epoch, i.e. once every
// copy of that call has landed and no engine still polls one of its signals.
struct XSlot {
    std::vector<hsa_signal_t> sigs;
    size_t used = 0;
    std::vector<std::pair<const uint32_t *, uint32_t>> finish;
};

// One host->device copy of a sender's rows: queued once *ready holds the epoch, then a
// 4-byte copy of the epoch into *landed.
struct InCopy {
    const uint32_t *ready;
    char *dst;
    const char *src;
    int64_t len;
    hsa_signal_t done;
    uint32_t *landed;
};

// The host->device copies of one call.  They all go to the one inbound engine and all
// depend on `start`, which the caller's stream releases once the target buffer is free.
struct InJob {
    std::vector<InCopy> copies;
    std::vector<const uint32_t *> ready_all;  // all-senders jobs: further flags to wait for
    std::function<void()> before_copies;      // all-senders jobs: host work once every flag is in
    uint32_t epoch = 0;
    bool per_sender = false;
    hsa_signal_t start{};
    const uint32_t *epoch_word = nullptr;
    hsa_signal_t landed_done{};
    uint32_t *status = nullptr;
    std::chrono::steady_clock::time_point deadline;
};

// Host thread that queues inbound copies in the order their senders' flags arrive.
// Measured on MI355X: one device->host engine next to one host->device engine fills both
// PCIe directions (about 96 GB/s together), but host->device copies on two or more engines
// at once pull the total down to about 61 GB/s.  So every inbound copy shares one engine,
// and to keep a late sender from holding up ready ones queued behind it on that in-order
// engine, a copy is queued only once its sender's flag (host memory, read without a PCIe
// round trip) holds the epoch.  With the all-senders policy a call's copies are queued
// together when the last flag is in.
class Courier {
public:
    void start(DmaEngines *dma) {
        dma_ = dma;
        th_ = std::thread([this] { run(); });
    }
    // Ends the thread, then queues every copy it still held (ready or not, without the
    // host work of all-senders jobs), so that each of them lands and raises its flag: a
    // release can then wait for all flags before freeing what the copies touch.
    void stop() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        if (th_.joinable())
            th_.join();
        while (!incoming_.empty()) {
            active_.push_back(std::move(incoming_.front()));
            incoming_.pop_front();
        }
        for (InJob &j : active_)
            for (const InCopy &c : j.copies)
                if (dma_)
                    submit(j, c);
        active_.clear();
    }
    void post(InJob &&j) {
        {
            std::lock_guard<std::mutex> lk(mu_);
            incoming_.push_back(std::move(j));
        }
        cv_.notify_one();
    }

private:
    static bool flag_ready(const InJob &j, const uint32_t *f) {
        return !f || (int32_t)(__atomic_load_n(f, __ATOMIC_ACQUIRE) - j.epoch) >= 0;
    }
    static bool ready(const InJob &j, const InCopy &c) { return flag_ready(j, c.ready); }
    bool submit(InJob &j, const InCopy &c) {
        std::string err;
        const uint32_t eng = dma_->in_engine(0);
        if (dma_->copy(eng, c.dst, false, c.src, true, (size_t)c.len, &j.start, 1, c.done, err) &&
            dma_->copy(eng, c.landed, true, j.epoch_word, false, sizeof(uint32_t), &c.done, 1, j.landed_done, err))
            return true;
        __atomic_store_n(j.status, (uint32_t)EP_ERR_HIP, __ATOMIC_RELEASE);
        return false;
    }
    // Queues what is ready; returns true once every copy of the job is queued.
    bool progress(InJob &j) {
        const bool late = std::chrono::steady_clock::now() > j.deadline;
        bool all = true;
        if (!j.per_sender && !late) {
            for (const InCopy &c : j.copies)
                all = all && ready(j, c);
            for (const uint32_t *f : j.ready_all)
                all = all && flag_ready(j, f);
        }
        if (!j.per_sender && (all || late)) {
            if (late)
                for (const uint32_t *f : j.ready_all)
                    if (!flag_ready(j, f))
                        __atomic_store_n(j.status, (uint32_t)EP_ERR_TIMEOUT, __ATOMIC_RELEASE);
            if (j.before_copies)
                j.before_copies();
            j.before_copies = nullptr;
        }
        for (size_t i = 0; i < j.copies.size();) {
            if (late || (j.per_sender ? ready(j, j.copies[i]) : all)) {
                if (late && !ready(j, j.copies[i]))
                    __atomic_store_n(j.status, (uint32_t)EP_ERR_TIMEOUT, __ATOMIC_RELEASE);
                submit(j, j.copies[i]);  // queued even when late, so no wait on the device hangs
                j.copies.erase(j.copies.begin() + (std::ptrdiff_t)i);
            } else {
                ++i;
            }
        }
        return j.copies.empty();
    }
    void run() {
        std::unique_lock<std::mutex> lk(mu_);
        for (;;) {
            if (stop_)
                return;
            while (!incoming_.empty()) {
                active_.push_back(std::move(incoming_.front()));
                incoming_.pop_front();
            }
            if (active_.empty()) {
                cv_.wait(lk, [&] { return stop_ || !incoming_.empty(); });
                continue;
            }
            lk.unlock();
            for (size_t i = 0; i < active_.size();) {
                if (progress(active_[i]))
                    active_.erase(active_.begin() + (std::ptrdiff_t)i);
                else
                    ++i;
            }
            for (int p = 0; p < 64; ++p)
                _mm_pause();
            lk.lock();
        }
    }

    DmaEngines *dma_ = nullptr;
    std::thread th_;
    std::mutex mu_;
    std::condition_variable cv_;
    std::deque<InJob> incoming_;
    std::vector<InJob> active_;
    bool stop_ = false;
};

class Exchange {
public:
    DmaEngines dma;
    Courier courier;

    bool init(int device, int nslots, std::string &err) {
        if (!dma.init(device, err))
            return false;
        slots_.resize((size_t)nslots);
        courier.start(&dma);
        return true;
    }

    // Waits (bounded) for every copy of every slot to land, then frees the signals.  Call
    // it after the streams that start the copies have run and before freeing the buffers
    // the copies touch.
    void release() {
        courier.stop();
        const auto t0 = std::chrono::steady_clock::now();
        bool drained = true;
        uint32_t spins = 0;
        for (XSlot &s : slots_)
            for (const auto &f : s.finish)
                while (drained && (int32_t)(__atomic_load_n(f.first, __ATOMIC_ACQUIRE) - f.second) < 0)
                    if (++spins % 1024 == 0) {
                        std::this_thread::yield();
                        drained = std::chrono::steady_clock::now() - t0 < std::chrono::microseconds(kReleaseDrainUs);
                    }
        if (drained)  // otherwise a copy may still wait on these signals: keep them alive
            for (XSlot &s : slots_)
                for (hsa_signal_t g : s.sigs)
                    hsa_signal_destroy(g);
        slots_.clear();
        dma.release();
    }

    XSlot *begin(int64_t timeout_us, std::string &err) {
        XSlot &s = slots_[(size_t)next_];
        const auto t0 = std::chrono::steady_clock::now();
        uint32_t spins = 0;
        for (const auto &f : s.finish) {
            while ((int32_t)(__atomic_load_n(f.first, __ATOMIC_ACQUIRE) - f.second) < 0) {
                _mm_pause();
                if (++spins % 1024 == 0) {
                    std::this_thread::yield();
                    if (std::chrono::steady_clock::now() - t0 > std::chrono::microseconds(timeout_us)) {
                        err = "the host legs of an earlier round did not finish";
                        return nullptr;
                    }
                }
            }
        }
        s.finish.clear();
        s.used = 0;
        next_ = (next_ + 1) % (int)slots_.size();
        return &s;
    }

    // A signal of this call with the given initial value (reset if reused).
    bool signal(XSlot &s, int64_t initial, hsa_signal_t &out, std::string &err) {
        if (s.used == s.sigs.size()) {
            hsa_signal_t g{};
            if (!dma.make_signal(g, err))
                return false;
            s.sigs.push_back(g);
        }
        out = s.sigs[s.used++];
        hsa_signal_store_relaxed(out, initial);
        return true;
    }

private:
    std::vector<XSlot> slots_;
    int next_ = 0;
};

}  // namespace ep
