// exchange.h -- SDMA queueing shared by the host legs of the exchange modes (exchange.cpp)
// and of the dense collectives (dense.cpp): per-call signal slots, and the courier thread
// that queues host->device copies as their senders' flags arrive.
#pragma once

#include "ep.h"
#include "sdma.h"
#include "signal_slots.h"
#include "status_block.h"

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

// One host->device copy of a sender's rows: queued once *ready holds the epoch, then a
// 4-byte copy of the epoch into *landed (none when landed is null: a piece of a larger
// transfer whose last piece carries the flag).  Each of the two copies has its own
// completion signal (done, landed_done), armed in the call's signal slot when the job is
// posted.  An eager copy goes as soon as its own flag is in, also in an all-senders job
// (a rank's own rows coming back from host memory, or a piece of a host-side result:
// they wait for no other sender).
struct InCopy {
    const uint32_t *ready;
    char *dst;
    const char *src;
    int64_t len;
    hsa_signal_t done;
    uint32_t *landed;
    hsa_signal_t landed_done;
    bool eager = false;
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
    const uint32_t *epoch_word = nullptr;  // source of the landed flags: epoch_words words of the epoch
    int epoch_words = 1;
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
// Jobs are served strictly in the order they were posted: no copy of a call is queued
// before every copy of the calls posted earlier.  A call's copies wait for its start
// signal, which the caller's stream releases only after the earlier calls' copies have
// landed; a copy queued ahead of them on the in-order engine would wait for a release that
// cannot come until the copies behind it have run.
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
            if (dma_)
                submit_all(j);
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
    // Copies a and b are next to each other in both the source and the destination.
    static bool contiguous(const InCopy &a, const InCopy &b) {
        return a.dst + a.len == b.dst && a.src + a.len == b.src;
    }
    // Queues copies [a, b) of the job, contiguous in memory, as one data copy on the
    // inbound engine (completion signal of copy a), then their landed flags on the inbound
    // flag engine after it: flags of neighbouring copies that are neighbouring words go as
    // one copy of up to epoch_words words (completion signal of its first copy).  The
    // signals that go unused are stored 0 by the host; so is every signal of a copy that
    // cannot be submitted (the staging's status records it).
    bool submit_run(InJob &j, size_t a, size_t b) {
        std::string err;
        const uint32_t eng = dma_->in_engine(0);
        int64_t len = 0;
        for (size_t m = a; m < b; ++m)
            len += j.copies[m].len;
        const InCopy &first = j.copies[a];
        const bool data = dma_->copy(eng, first.dst, false, first.src, true, (size_t)len, &j.start, 1, first.done, err);
        for (size_t m = data ? a + 1 : a; m < b; ++m)
            hsa_signal_store_screlease(j.copies[m].done, 0);
        bool ok = data;
        const uint32_t feng = dma_->in_flag_engine();
        for (size_t m = a; m < b;) {
            const InCopy &c = j.copies[m];
            if (!c.landed) {  // no flag for this piece
                hsa_signal_store_screlease(c.landed_done, 0);
                ++m;
                continue;
            }
            size_t e = m + 1;
            while (e < b && (int)(e - m) < j.epoch_words && j.copies[e].landed == c.landed + (e - m))
                ++e;
            if (!(ok && dma_->copy(feng, c.landed, true, j.epoch_word, false, (e - m) * sizeof(uint32_t), &first.done,
                                   1, c.landed_done, err))) {
                ok = false;
                hsa_signal_store_screlease(c.landed_done, 0);
            }
            for (size_t q = m + 1; q < e; ++q)
                hsa_signal_store_screlease(j.copies[q].landed_done, 0);
            m = e;
        }
        if (!ok)
            __atomic_store_n(j.status, (uint32_t)EP_ERR_HIP, __ATOMIC_RELEASE);
        return ok;
    }
    // Queues the copies marked in `go`, merging neighbours that are contiguous in memory,
    // and removes them from the job.
    void submit_marked(InJob &j, std::vector<char> &go) {
        std::vector<InCopy> rest;
        for (size_t i = 0; i < j.copies.size();) {
            if (!go[i]) {
                rest.push_back(j.copies[i++]);
                continue;
            }
            size_t e = i + 1;
            while (e < j.copies.size() && go[e] && contiguous(j.copies[e - 1], j.copies[e]))
                ++e;
            submit_run(j, i, e);
            i = e;
        }
        j.copies.swap(rest);
    }
    void submit_all(InJob &j) {
        std::vector<char> go(j.copies.size(), 1);
        submit_marked(j, go);
    }
    // Queues what is ready; returns true once every copy of the job is queued.
    bool progress(InJob &j) {
        const bool late = std::chrono::steady_clock::now() > j.deadline;
        // all-senders jobs: every sender's flag is in (eager copies go on their own flags and
        // do not count: the host work of the job may be what raises them)
        bool all = true;
        if (!j.per_sender && !late) {
            for (const InCopy &c : j.copies)
                all = all && (c.eager || ready(j, c));
            for (const uint32_t *f : j.ready_all)
                all = all && flag_ready(j, f);
        }
        if (!j.per_sender && (all || late)) {
            if (late)
                for (const uint32_t *f : j.ready_all)
                    if (!flag_ready(j, f))
                        record_host_timeout(j.status, kSiteCourier, f, j.epoch);
            if (j.before_copies)
                j.before_copies();
            j.before_copies = nullptr;
        }
        std::vector<char> go(j.copies.size(), 0);
        bool any = false;
        for (size_t i = 0; i < j.copies.size(); ++i) {
            const InCopy &c = j.copies[i];
            const bool own_flag = ready(j, c);
            go[i] = late || (own_flag && (j.per_sender || c.eager || all));
            if (late && !own_flag)
                record_host_timeout(j.status, kSiteCourier, c.ready, j.epoch);  // queued all the same,
            any = any || go[i];                                                 // so no wait on the device hangs
        }
        if (any)
            submit_marked(j, go);
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
            // the oldest job first; a later one only once the earlier ones are all queued
            while (!active_.empty() && progress(active_.front()))
                active_.erase(active_.begin());
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
    SignalSlots slots;

    bool init(int device, int nslots, std::string &err) {
        if (!dma.init(device, err))
            return false;
        slots.init(nslots);
        courier.start(&dma);
        return true;
    }
    // The same on engines chosen by the caller (flag engines 0: the flags go on the engine
    // of their data).
    void init_with(hsa_agent_t gpu, hsa_agent_t cpu, uint32_t out, const std::vector<uint32_t> &in, int nslots,
                   uint32_t out_flag = 0, uint32_t in_flag = 0) {
        dma.init_with(gpu, cpu, out, in, out_flag, in_flag);
        slots.init(nslots);
        courier.start(&dma);
    }

    // Queues every copy the courier still holds, waits (bounded) for every copy of every
    // call to land, then frees the signals (or leaves them allocated if one did not land:
    // an engine may still decrement it).  Call it after the streams that release the
    // calls' start signals have run and before freeing the buffers the copies touch.
    void release() {
        courier.stop();
        std::string err;
        slots.destroy(slots.drain(kReleaseDrainUs, err));
        dma.release();
    }

    // Reserves the signal slot of a call (see SignalSlots::begin); -1 with err on timeout.
    int begin(int64_t timeout_us, std::string &err) { return slots.begin(timeout_us, err); }

    // A start signal of call `slot` (value 1; the caller's stream stores 0 into it).  Arm it
    // once the kernel that releases it has been enqueued.
    bool start_signal(int slot, hsa_signal_t &out, std::string &err) { return slots.take(slot, out, err); }
    void arm(int slot, hsa_signal_t g) { slots.arm(slot, g); }

    // One copy of call `slot` with a completion signal of its own (returned in *done when
    // non-null), armed once submitted.
    bool copy(int slot, uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
              const hsa_signal_t *deps, int ndeps, hsa_signal_t *done, std::string &err) {
        hsa_signal_t g{};
        if (!slots.take(slot, g, err) || !dma.copy(engine, dst, dst_host, src, src_host, len, deps, ndeps, g, err))
            return false;
        slots.arm(slot, g);
        if (done)
            *done = g;
        return true;
    }

    // An inbound copy of call `slot` for the courier: its two completion signals.
    bool in_copy(int slot, const uint32_t *ready, char *dst, const char *src, int64_t len, uint32_t *landed,
                 InCopy &out, std::string &err) {
        out = InCopy{ready, dst, src, len, {}, landed, {}};
        return slots.take(slot, out.done, err) && slots.take(slot, out.landed_done, err);
    }
    // Hands a call's inbound copies to the courier and arms their signals (the courier
    // submits every copy it is given, or stores 0 into the signals of one it cannot).
    void post(int slot, InJob &&j) {
        if (j.copies.empty())
            return;
        for (const InCopy &c : j.copies) {
            slots.arm(slot, c.done);
            slots.arm(slot, c.landed_done);
        }
        courier.post(std::move(j));
    }
};

}  // namespace ep
