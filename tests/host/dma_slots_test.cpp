// dma_slots_test.cpp -- host-only test of the SDMA lane's, the exchange's and the graph
// rounds' host legs (sdma.h, exchange.h, graph_legs.h, signal_slots.h) against a stand-in
// for the ROCr runtime.
//
// The stand-in keeps the documented contract of an async copy: it starts once every
// dependency signal reads exactly 0, it writes its bytes, and afterwards it decrements
// its completion signal.  Each engine runs its copies in order on a thread of its own, and
// it applies a copy's decrement after a random delay, with the copied bytes (a flag word
// included) already visible to the host: the window in which a host that has seen a flag
// may still get that copy's decrement later.  The stand-in records as violations:
//   - a decrement landing on a signal whose value was stored again (reset for a new call),
//     or on a destroyed signal (its handle is handed out again by the next create);
//   - a dependency reading below 0 (an engine waiting for 0 would never start the copy);
//   - an engine waiting longer than the test allows.
// Destroyed handles are recycled last-in first-out, as a signal pool would.
//
// Usage: dma_slots_test lane|exchange|order|merge|bounded|graph|graph_timeout|old_rule
// [seed]; prints "violations N" and exits 0 when N == 0 and every check of the scenario
// held.
#include "exchange.h"
#include "graph_legs.h"
#include "sdma.h"
#include "signal_slots.h"

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <map>
#include <memory>
#include <mutex>
#include <random>
#include <string>
#include <thread>
#include <vector>

namespace {

using Clock = std::chrono::steady_clock;

std::atomic<int> g_violations{0};
std::mutex g_log_mu;
void violation(const char *what, uint64_t h) {
    ++g_violations;
    std::lock_guard<std::mutex> lk(g_log_mu);
    if (g_violations <= 10)
        std::printf("violation: %s (signal %llu)\n", what, (unsigned long long)h);
}

// ---------------------------------------------------------------- stand-in signals

constexpr size_t kMaxSignals = 1 << 16;
struct FakeSignal {
    volatile int64_t value;
    std::atomic<uint64_t> gen;  // bumped by every host store and by destroy
    std::atomic<bool> alive;
};
FakeSignal g_sig[kMaxSignals];
std::mutex g_sig_mu;
std::vector<uint64_t> g_free;  // recycled handles, last in first out
uint64_t g_next = 1;
std::atomic<int64_t> g_created{0}, g_destroyed{0};

FakeSignal &sig(hsa_signal_t s) { return g_sig[s.handle]; }

std::atomic<int> g_delay_max_us{200};
thread_local std::mt19937 t_rng{12345};
int rand_delay_us() {
    const int m = g_delay_max_us.load();
    if (m <= 0)
        return 0;
    std::uniform_int_distribution<int> d(0, 9);
    const int pick = d(t_rng);
    std::uniform_int_distribution<int> u(0, m);
    return pick < 6 ? 0 : u(t_rng);  // most decrements at once, some late
}

// ---------------------------------------------------------------- stand-in engines

struct Copy {
    void *dst;
    const void *src;
    size_t len;
    std::vector<hsa_signal_t> deps;
    hsa_signal_t done;
    uint64_t done_gen;
};

class Engine {
public:
    explicit Engine(uint32_t id) : id_(id), th_([this] { run(); }) {}
    ~Engine() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        th_.join();
    }
    void push(Copy c) {
        {
            std::lock_guard<std::mutex> lk(mu_);
            q_.push_back(std::move(c));
        }
        cv_.notify_all();
    }
    bool idle() {
        std::lock_guard<std::mutex> lk(mu_);
        return q_.empty() && !busy_;
    }

private:
    void run() {
        t_rng.seed(1000 + id_);
        for (;;) {
            Copy c;
            {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return stop_ || !q_.empty(); });
                if (stop_ && q_.empty())
                    return;
                c = q_.front();
                q_.pop_front();
                busy_ = true;
            }
            const auto t0 = Clock::now();
            bool stuck = false;
            for (hsa_signal_t d : c.deps) {
                for (;;) {
                    const int64_t v = __atomic_load_n(&sig(d).value, __ATOMIC_ACQUIRE);
                    if (v == 0)
                        break;
                    if (v < 0) {
                        violation("a dependency reads below 0: the copy would never start", d.handle);
                        stuck = true;
                        break;
                    }
                    if (Clock::now() - t0 > std::chrono::seconds(5)) {
                        violation("a copy waited 5 s for a dependency", d.handle);
                        stuck = true;
                        break;
                    }
                    std::this_thread::yield();
                }
                if (stuck)
                    break;
            }
            if (!stuck) {
                if (c.len % sizeof(uint32_t) == 0 && c.len <= 64 * sizeof(uint32_t)) {
                    // flag words (one, or a merged run of them): one visible store each
                    for (size_t w = 0; w < c.len / sizeof(uint32_t); ++w)
                        __atomic_store_n(static_cast<uint32_t *>(c.dst) + w,
                                         static_cast<const volatile uint32_t *>(c.src)[w], __ATOMIC_RELEASE);
                } else {
                    std::memcpy(c.dst, c.src, c.len);
                    __atomic_thread_fence(__ATOMIC_RELEASE);
                }
                const int us = rand_delay_us();
                if (us > 0)
                    std::this_thread::sleep_for(std::chrono::microseconds(us));
                FakeSignal &f = sig(c.done);
                if (!f.alive.load())
                    violation("a completion decrement landed on a destroyed signal", c.done.handle);
                else if (f.gen.load() != c.done_gen)
                    violation("a completion decrement landed after the signal was reset for a new call",
                              c.done.handle);
                __atomic_fetch_sub(&f.value, 1, __ATOMIC_ACQ_REL);
            }
            std::lock_guard<std::mutex> lk(mu_);
            busy_ = false;
        }
    }

    uint32_t id_;
    std::mutex mu_;
    std::condition_variable cv_;
    std::deque<Copy> q_;
    bool stop_ = false, busy_ = false;
    std::thread th_;
};

std::mutex g_eng_mu;
std::map<uint32_t, std::unique_ptr<Engine>> g_engines;
std::atomic<int64_t> g_copies{0}, g_copy_bytes_max{0};  // copies submitted, largest one

Engine &engine(uint32_t id) {
    std::lock_guard<std::mutex> lk(g_eng_mu);
    auto &e = g_engines[id];
    if (!e)
        e.reset(new Engine(id));
    return *e;
}
void stop_engines() {
    std::lock_guard<std::mutex> lk(g_eng_mu);
    g_engines.clear();
}

hsa_status_t submit(void *dst, const void *src, size_t len, uint32_t ndeps, const hsa_signal_t *deps,
                    hsa_signal_t done, uint32_t eng) {
    if (!dst || !src || !done.handle)
        return HSA_STATUS_ERROR_INVALID_ARGUMENT;
    Copy c{dst, src, len, std::vector<hsa_signal_t>(deps, deps + ndeps), done, sig(done).gen.load()};
    ++g_copies;
    for (int64_t m = g_copy_bytes_max.load(); (int64_t)len > m && !g_copy_bytes_max.compare_exchange_weak(m, len);)
        ;
    engine(eng).push(std::move(c));
    return HSA_STATUS_SUCCESS;
}

}  // namespace

// ---------------------------------------------------------------- the ROCr entry points used

extern "C" {

hsa_status_t hsa_amd_signal_create(hsa_signal_value_t initial_value, uint32_t, const hsa_agent_t *, uint64_t,
                                   hsa_signal_t *signal) {
    std::lock_guard<std::mutex> lk(g_sig_mu);
    uint64_t h;
    if (!g_free.empty()) {
        h = g_free.back();
        g_free.pop_back();
    } else {
        if (g_next >= kMaxSignals)
            return HSA_STATUS_ERROR_OUT_OF_RESOURCES;
        h = g_next++;
    }
    g_sig[h].value = initial_value;
    g_sig[h].gen.fetch_add(1);
    g_sig[h].alive.store(true);
    signal->handle = h;
    ++g_created;
    return HSA_STATUS_SUCCESS;
}

hsa_status_t hsa_signal_destroy(hsa_signal_t s) {
    std::lock_guard<std::mutex> lk(g_sig_mu);
    sig(s).alive.store(false);
    sig(s).gen.fetch_add(1);
    g_free.push_back(s.handle);
    ++g_destroyed;
    return HSA_STATUS_SUCCESS;
}

void hsa_signal_store_relaxed(hsa_signal_t s, hsa_signal_value_t v) {
    sig(s).gen.fetch_add(1);
    __atomic_store_n(&sig(s).value, v, __ATOMIC_RELAXED);
}

void hsa_signal_store_screlease(hsa_signal_t s, hsa_signal_value_t v) {
    sig(s).gen.fetch_add(1);
    __atomic_store_n(&sig(s).value, v, __ATOMIC_RELEASE);
}

hsa_signal_value_t hsa_signal_load_scacquire(hsa_signal_t s) { return __atomic_load_n(&sig(s).value, __ATOMIC_ACQUIRE); }

hsa_status_t hsa_amd_signal_value_pointer(hsa_signal_t s, volatile hsa_signal_value_t **p) {
    *p = &sig(s).value;
    return HSA_STATUS_SUCCESS;
}

hsa_status_t hsa_amd_memory_async_copy_on_engine(void *dst, hsa_agent_t, const void *src, hsa_agent_t, size_t size,
                                                 uint32_t ndeps, const hsa_signal_t *deps, hsa_signal_t done,
                                                 hsa_amd_sdma_engine_id_t engine_id, bool) {
    return submit(dst, src, size, ndeps, deps, done, (uint32_t)engine_id);
}

hsa_status_t hsa_amd_memory_async_copy(void *dst, hsa_agent_t, const void *src, hsa_agent_t, size_t size,
                                       uint32_t ndeps, const hsa_signal_t *deps, hsa_signal_t done) {
    return submit(dst, src, size, ndeps, deps, done, 0);
}

hsa_status_t hsa_shut_down() { return HSA_STATUS_SUCCESS; }

}  // extern "C"

// ---------------------------------------------------------------- the caller's stream

namespace {

// Work the caller's stream does in order: store 0 into a start signal (the release
// kernel), or wait for a flag word to reach an epoch (the wait kernel).
class Stream {
public:
    Stream() : th_([this] { run(); }) {}
    ~Stream() {
        finish();
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        th_.join();
    }
    void release(int64_t *value) { push({value, nullptr, 0}); }
    void wait(const uint32_t *flag, uint32_t epoch) { push({nullptr, flag, epoch}); }
    void finish() {
        std::unique_lock<std::mutex> lk(mu_);
        done_cv_.wait(lk, [&] { return q_.empty() && !busy_; });
    }

private:
    struct Item {
        int64_t *value;
        const uint32_t *flag;
        uint32_t epoch;
    };
    void push(Item it) {
        {
            std::lock_guard<std::mutex> lk(mu_);
            q_.push_back(it);
        }
        cv_.notify_all();
    }
    void run() {
        std::mt19937 rng(77);
        for (;;) {
            Item it;
            {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return stop_ || !q_.empty(); });
                if (q_.empty())
                    return;
                it = q_.front();
                q_.pop_front();
                busy_ = true;
            }
            if (it.value) {
                std::this_thread::sleep_for(std::chrono::microseconds(rng() % 50));
                __atomic_store_n(it.value, (int64_t)0, __ATOMIC_RELEASE);
            } else {
                const auto t0 = Clock::now();
                while ((int32_t)(__atomic_load_n(it.flag, __ATOMIC_ACQUIRE) - it.epoch) < 0) {
                    if (Clock::now() - t0 > std::chrono::seconds(5)) {
                        violation("the stream waited 5 s for a flag", 0);
                        break;
                    }
                    std::this_thread::yield();
                }
            }
            {
                std::lock_guard<std::mutex> lk(mu_);
                busy_ = false;
            }
            done_cv_.notify_all();
        }
    }
    std::mutex mu_;
    std::condition_variable cv_, done_cv_;
    std::deque<Item> q_;
    bool stop_ = false, busy_ = false;
    std::thread th_;
};

int g_checks_failed = 0;
void check(bool ok, const char *what) {
    if (!ok) {
        ++g_checks_failed;
        std::printf("check failed: %s\n", what);
    }
}

const hsa_agent_t kGpu{1}, kCpu{2};

// ---------------------------------------------------------------- scenarios

// Rounds of the default device->host leg with a chunk count that changes from round to
// round (so a signal's role in one round differs from its role in the last round on the
// same slot), the host running ahead of the copies, and lanes created and released
// between batches (destroyed handles recycled); the chunk flags on the data engine in
// even batches and on an engine of their own in odd ones.
void scenario_lane(uint32_t seed) {
    std::mt19937 rng(seed);
    for (int batch = 0; batch < 6; ++batch) {
        ep::SdmaLane lane;
        lane.init_with(kGpu, kCpu, 1u, 4, batch % 2 ? 3u : 0u);
        Stream stream;
        struct R {
            std::vector<uint8_t> src, dst;
            std::vector<uint32_t> flags;
            uint32_t epoch_word;
            uint32_t epoch;
        };
        std::vector<std::unique_ptr<R>> rounds;
        for (int i = 0; i < 60; ++i) {
            const int64_t chunk = 256, chunks = 1 + rng() % 6;
            const int64_t bytes = (chunks - 1) * chunk + 1 + rng() % chunk;
            std::unique_ptr<R> r(new R);
            r->src.resize((size_t)bytes);
            for (auto &b : r->src)
                b = (uint8_t)rng();
            r->dst.assign((size_t)bytes, 0);
            r->flags.assign((size_t)chunks, 0);
            r->epoch = (uint32_t)(batch * 1000 + i + 1);
            r->epoch_word = r->epoch;
            ep::SdmaLane::Round round;
            std::string err;
            if (!lane.begin(round, 5 * 1000 * 1000, err)) {
                check(false, err.c_str());
                break;
            }
            stream.release(round.start_value);
            if (!lane.submit(round, r->dst.data(), r->src.data(), bytes, chunk, r->flags.data(), &r->epoch_word, err)) {
                check(false, err.c_str());
                break;
            }
            stream.wait(&r->flags[(size_t)chunks - 1], r->epoch);
            rounds.push_back(std::move(r));
        }
        stream.finish();
        std::string err;
        check(lane.drain(5 * 1000 * 1000, err), "the lane drains");
        for (auto &r : rounds) {
            check(r->dst == r->src, "every round's bytes landed");
            for (uint32_t f : r->flags)
                check(f == r->epoch, "every chunk flag holds its round's epoch");
        }
        lane.release();
    }
}

// Calls of the exchange modes: outbound copies with their flag copies, inbound copies
// queued by the courier as simulated senders raise their flags at random times, with the
// number of copies per call changing from call to call; exchanges created and released
// between batches.  Even batches put the flags on the engines of their data, odd ones on
// two flag engines; every other call gives the courier an epoch row, so that the landed
// flags of merged inbound copies go as one flag copy.
void scenario_exchange(uint32_t seed) {
    std::mt19937 rng(seed);
    for (int batch = 0; batch < 6; ++batch) {
        ep::Exchange x;
        x.init_with(kGpu, kCpu, 1u, {2u}, 4, batch % 2 ? 3u : 0u, batch % 2 ? 4u : 0u);
        Stream stream;
        uint32_t status[ep::kStatusWords] = {};
        struct Call {
            std::vector<std::vector<uint8_t>> out_src, out_dst, in_src, in_dst;
            std::vector<uint32_t> out_flags, ready, landed;
            uint32_t epoch, epoch_word;
            uint32_t epoch_row[64];
        };
        std::vector<std::unique_ptr<Call>> calls;
        std::vector<std::thread> senders;
        for (int i = 0; i < 50; ++i) {
            std::unique_ptr<Call> c(new Call);
            c->epoch = c->epoch_word = (uint32_t)(batch * 1000 + i + 1);
            for (uint32_t &w : c->epoch_row)
                w = c->epoch;
            const int nout = (int)(rng() % 4), nin = 1 + (int)(rng() % 6);
            for (int k = 0; k < nout; ++k) {
                c->out_src.emplace_back(64 + rng() % 512);
                for (auto &b : c->out_src.back())
                    b = (uint8_t)rng();
                c->out_dst.emplace_back(c->out_src.back().size(), 0);
            }
            for (int k = 0; k < nin; ++k) {
                c->in_src.emplace_back(64 + rng() % 512);
                for (auto &b : c->in_src.back())
                    b = (uint8_t)rng();
                c->in_dst.emplace_back(c->in_src.back().size(), 0);
            }
            c->out_flags.assign((size_t)nout, 0);
            c->ready.assign((size_t)nin, 0);
            c->landed.assign((size_t)nin, 0);
            std::string err;
            const int slot = x.begin(5 * 1000 * 1000, err);
            if (slot < 0) {
                check(false, err.c_str());
                break;
            }
            hsa_signal_t start{};
            check(x.start_signal(slot, start, err), "start signal");
            stream.release(ep::DmaEngines::value_pointer(start));
            x.arm(slot, start);
            for (int k = 0; k < nout; ++k) {
                hsa_signal_t d{};
                check(x.copy(slot, 1u, c->out_dst[(size_t)k].data(), true, c->out_src[(size_t)k].data(), false,
                             c->out_src[(size_t)k].size(), &start, 1, &d, err) &&
                          x.copy(slot, x.dma.out_flag_engine(), &c->out_flags[(size_t)k], true, &c->epoch_word, false,
                                 sizeof(uint32_t), &d, 1, nullptr, err),
                      "outbound copies submitted");
                stream.wait(&c->out_flags[(size_t)k], c->epoch);
            }
            ep::InJob j;
            j.epoch = c->epoch;
            j.per_sender = rng() % 2;
            j.start = start;
            j.epoch_word = i % 2 ? c->epoch_row : &c->epoch_word;
            j.epoch_words = i % 2 ? 64 : 1;
            j.status = status;
            j.deadline = Clock::now() + std::chrono::seconds(5);
            for (int k = 0; k < nin; ++k) {
                ep::InCopy ic;
                check(x.in_copy(slot, &c->ready[(size_t)k], reinterpret_cast<char *>(c->in_dst[(size_t)k].data()),
                                reinterpret_cast<const char *>(c->in_src[(size_t)k].data()),
                                (int64_t)c->in_src[(size_t)k].size(), &c->landed[(size_t)k], ic, err),
                      "inbound copy signals");
                j.copies.push_back(ic);
                stream.wait(&c->landed[(size_t)k], c->epoch);
            }
            x.post(slot, std::move(j));
            // the senders raise their flags in a random order, a little later
            Call *cp = c.get();
            const uint32_t sseed = (uint32_t)rng();
            senders.emplace_back([cp, nin, sseed] {
                std::mt19937 r(sseed);
                std::vector<int> order((size_t)nin);
                for (int k = 0; k < nin; ++k)
                    order[(size_t)k] = k;
                std::shuffle(order.begin(), order.end(), r);
                for (int k : order) {
                    std::this_thread::sleep_for(std::chrono::microseconds(r() % 300));
                    __atomic_store_n(&cp->ready[(size_t)k], cp->epoch, __ATOMIC_RELEASE);
                }
            });
            calls.push_back(std::move(c));
        }
        for (auto &t : senders)
            t.join();
        stream.finish();
        x.release();
        check(status[0] == 0, "no courier timeout");
        for (auto &c : calls) {
            check(c->out_dst == c->out_src, "outbound bytes landed");
            check(c->in_dst == c->in_src, "inbound bytes landed");
            for (uint32_t f : c->out_flags)
                check(f == c->epoch, "outbound flags hold the epoch");
            for (uint32_t f : c->landed)
                check(f == c->epoch, "landed flags hold the epoch");
        }
    }
}

// Two calls whose senders answer out of order: the first call's sender is 50 ms late, the
// second call's sender has answered before the second call is even posted.  The second
// call's copy must not be queued on the in-order inbound engine ahead of the first call's
// (it waits for a start signal that the stream releases only after the first call's rows
// have landed).  Both calls must finish in about the late sender's delay, well inside the
// stream's 5 s bound.
void scenario_order() {
    ep::Exchange x;
    x.init_with(kGpu, kCpu, 1u, {2u}, 4);
    Stream stream;
    uint32_t status[ep::kStatusWords] = {};
    std::vector<uint8_t> src[2], dst[2];
    uint32_t ready[2] = {0, 0}, landed[2] = {0, 0}, epoch_word[2] = {1, 2};
    const auto t0 = Clock::now();
    for (int c = 0; c < 2; ++c) {
        src[c].assign(4096, (uint8_t)(c + 1));
        dst[c].assign(4096, 0);
        if (c == 1)
            __atomic_store_n(&ready[1], 2u, __ATOMIC_RELEASE);  // the second call's sender is early
        std::string err;
        const int slot = x.begin(1000 * 1000, err);
        hsa_signal_t start{};
        check(slot >= 0 && x.start_signal(slot, start, err), "slot and start signal");
        stream.release(ep::DmaEngines::value_pointer(start));
        x.arm(slot, start);
        ep::InJob j;
        j.epoch = (uint32_t)(c + 1);
        j.per_sender = true;
        j.start = start;
        j.epoch_word = &epoch_word[c];
        j.status = status;
        j.deadline = Clock::now() + std::chrono::seconds(5);
        ep::InCopy ic;
        check(x.in_copy(slot, &ready[c], reinterpret_cast<char *>(dst[c].data()),
                        reinterpret_cast<const char *>(src[c].data()), 4096, &landed[c], ic, err),
              "inbound copy");
        j.copies.push_back(ic);
        x.post(slot, std::move(j));
        stream.wait(&landed[c], (uint32_t)(c + 1));
    }
    std::thread late([&] {
        std::this_thread::sleep_for(std::chrono::milliseconds(50));
        __atomic_store_n(&ready[0], 1u, __ATOMIC_RELEASE);
    });
    late.join();
    stream.finish();
    const double ms = std::chrono::duration<double, std::milli>(Clock::now() - t0).count();
    check(ms < 1000.0, "both calls finished within a second (no wait for the bound)");
    check(landed[0] == 1 && landed[1] == 2 && dst[0] == src[0] && dst[1] == src[1], "both calls' rows landed");
    check(status[0] == 0, "no timeout recorded");
    x.release();
    std::printf("out-of-order senders: %.1f ms\n", ms);
}

// Inbound copies of one call that are next to each other in memory and whose senders
// have all answered go down as one data copy, each sender's flag after it: four senders
// ready at once give one copy of their four ranges and four flag copies.  An eager copy
// of an all-senders job (a rank's own rows) goes before the other senders answer.
void scenario_merge() {
    ep::Exchange x;
    x.init_with(kGpu, kCpu, 1u, {2u}, 4);
    Stream stream;
    uint32_t status[ep::kStatusWords] = {};
    const int n = 4;
    const int64_t part = 4096;
    std::vector<uint8_t> src((size_t)(n * part)), dst((size_t)(n * part), 0);
    for (size_t i = 0; i < src.size(); ++i)
        src[i] = (uint8_t)(i * 7 + 3);
    uint32_t ready[n] = {1, 1, 1, 1}, landed[n] = {0, 0, 0, 0}, epoch_word = 1;
    std::string err;
    int slot = x.begin(1000 * 1000, err);
    hsa_signal_t start{};
    check(slot >= 0 && x.start_signal(slot, start, err), "slot");
    stream.release(ep::DmaEngines::value_pointer(start));
    x.arm(slot, start);
    const int64_t before = g_copies.load();
    ep::InJob j;
    j.epoch = 1;
    j.per_sender = true;
    j.start = start;
    j.epoch_word = &epoch_word;
    j.status = status;
    j.deadline = Clock::now() + std::chrono::seconds(5);
    for (int r = 0; r < n; ++r) {
        ep::InCopy c;
        check(x.in_copy(slot, &ready[r], reinterpret_cast<char *>(dst.data()) + r * part,
                        reinterpret_cast<const char *>(src.data()) + r * part, part, &landed[r], c, err), "copy");
        j.copies.push_back(c);
        stream.wait(&landed[r], 1);
    }
    x.post(slot, std::move(j));
    stream.finish();
    check(g_copies.load() - before == 1 + n, "one data copy and one flag copy per sender");
    check(g_copy_bytes_max.load() == n * part, "the data copy spans the four ranges");
    check(dst == src, "every range landed");
    for (int r = 0; r < n; ++r)
        check(landed[r] == 1, "every sender's landed flag");

    // with an epoch row the landed flags of the merged copies are neighbouring words and go
    // as one flag copy (on the inbound flag engine); a landed flag that is not the next word
    // starts another flag copy
    {
        ep::Exchange y;
        y.init_with(kGpu, kCpu, 1u, {2u}, 4, 3u, 4u);
        std::vector<uint8_t> d2((size_t)(n * part), 0);
        uint32_t row[64], lnd[n + 1] = {0, 0, 0, 0, 0};
        for (uint32_t &w : row)
            w = 5;
        uint32_t rdy[n] = {5, 5, 5, 5};
        int s2 = y.begin(1000 * 1000, err);
        hsa_signal_t st2{};
        check(s2 >= 0 && y.start_signal(s2, st2, err), "slot (epoch row)");
        stream.release(ep::DmaEngines::value_pointer(st2));
        y.arm(s2, st2);
        const int64_t b2 = g_copies.load();
        ep::InJob m;
        m.epoch = 5;
        m.per_sender = true;
        m.start = st2;
        m.epoch_word = row;
        m.epoch_words = 64;
        m.status = status;
        m.deadline = Clock::now() + std::chrono::seconds(5);
        // flags of senders 0, 1, 2 are words 0, 1, 2; sender 3's is word 4 (not the next word)
        uint32_t *where[n] = {&lnd[0], &lnd[1], &lnd[2], &lnd[4]};
        for (int r = 0; r < n; ++r) {
            ep::InCopy c;
            check(y.in_copy(s2, &rdy[r], reinterpret_cast<char *>(d2.data()) + r * part,
                            reinterpret_cast<const char *>(src.data()) + r * part, part, where[r], c, err), "copy");
            m.copies.push_back(c);
            stream.wait(where[r], 5);
        }
        y.post(s2, std::move(m));
        stream.finish();
        check(g_copies.load() - b2 == 3, "one data copy, one flag copy for words 0-2, one for word 4");
        check(d2 == src, "every range landed (epoch row)");
        check(lnd[0] == 5 && lnd[1] == 5 && lnd[2] == 5 && lnd[3] == 0 && lnd[4] == 5,
              "the landed flags and nothing between them");
        y.release();
    }

    // all-senders job: the eager copy goes while another sender is still out
    std::vector<uint8_t> own(4096, 9), own_dst(4096, 0), other(4096, 5), other_dst(4096, 0);
    uint32_t own_ready = 2, other_ready = 0, own_landed = 0, other_landed = 0;
    epoch_word = 2;
    slot = x.begin(1000 * 1000, err);
    check(slot >= 0 && x.start_signal(slot, start, err), "slot 2");
    stream.release(ep::DmaEngines::value_pointer(start));
    x.arm(slot, start);
    ep::InJob k;
    k.epoch = 2;
    k.per_sender = false;
    k.start = start;
    k.epoch_word = &epoch_word;
    k.status = status;
    k.deadline = Clock::now() + std::chrono::seconds(5);
    ep::InCopy c1, c2;
    check(x.in_copy(slot, &own_ready, reinterpret_cast<char *>(own_dst.data()),
                    reinterpret_cast<const char *>(own.data()), 4096, &own_landed, c1, err) &&
              x.in_copy(slot, &other_ready, reinterpret_cast<char *>(other_dst.data()),
                        reinterpret_cast<const char *>(other.data()), 4096, &other_landed, c2, err),
          "copies");
    c1.eager = true;
    k.copies = {c1, c2};
    x.post(slot, std::move(k));
    const auto t0 = Clock::now();
    while (__atomic_load_n(&own_landed, __ATOMIC_ACQUIRE) != 2 && Clock::now() - t0 < std::chrono::seconds(2))
        std::this_thread::yield();
    check(own_landed == 2 && own_dst == own, "the eager copy landed before the other sender answered");
    check(__atomic_load_n(&other_landed, __ATOMIC_ACQUIRE) == 0, "the other copy waited");
    __atomic_store_n(&other_ready, 2u, __ATOMIC_RELEASE);
    stream.wait(&other_landed, 2);
    stream.finish();
    check(other_dst == other && status[0] == 0, "then the other copy landed");

    // all-senders job whose copies are pieces of a host-side result: its host work runs
    // once the senders' flags are in and raises each piece's flag as that piece is ready;
    // the pieces' own flags do not hold back the host work that raises them
    std::vector<uint8_t> sum(4 * 4096, 0), sum_dst(4 * 4096, 0);
    uint32_t sender = 0, piece_flag[4] = {0, 0, 0, 0}, block_landed = 0;
    epoch_word = 3;
    slot = x.begin(1000 * 1000, err);
    check(slot >= 0 && x.start_signal(slot, start, err), "slot 3");
    stream.release(ep::DmaEngines::value_pointer(start));
    x.arm(slot, start);
    ep::InJob h;
    h.epoch = 3;
    h.per_sender = false;
    h.start = start;
    h.epoch_word = &epoch_word;
    h.status = status;
    h.deadline = Clock::now() + std::chrono::seconds(5);
    h.ready_all.push_back(&sender);
    for (int c = 0; c < 4; ++c) {
        ep::InCopy piece;
        check(x.in_copy(slot, &piece_flag[c], reinterpret_cast<char *>(sum_dst.data()) + c * 4096,
                        reinterpret_cast<const char *>(sum.data()) + c * 4096, 4096, c == 3 ? &block_landed : nullptr,
                        piece, err),
              "piece");
        piece.eager = true;
        h.copies.push_back(piece);
    }
    std::thread worker;
    h.before_copies = [&]() {
        worker = std::thread([&]() {
            for (int c = 0; c < 4; ++c) {
                std::fill(sum.begin() + c * 4096, sum.begin() + (c + 1) * 4096, (uint8_t)(c + 11));
                __atomic_store_n(&piece_flag[c], 3u, __ATOMIC_RELEASE);
                std::this_thread::sleep_for(std::chrono::microseconds(200));
            }
        });
    };
    x.post(slot, std::move(h));
    stream.wait(&block_landed, 3);
    std::this_thread::sleep_for(std::chrono::milliseconds(2));
    __atomic_store_n(&sender, 3u, __ATOMIC_RELEASE);
    stream.finish();
    if (worker.joinable())
        worker.join();
    check(block_landed == 3 && sum_dst == sum, "host-side pieces went down once their flags came");
    check(status[0] == 0, "no timeout for the pieces");
    x.release();
}

// A slot whose previous call left a signal that never reaches 0 is not handed out: begin()
// gives up after its bound with a message, and succeeds once the signal retires.
void scenario_bounded() {
    ep::SignalSlots slots;
    slots.init(2);
    std::string err;
    const int a = slots.begin(1000, err);
    hsa_signal_t g{};
    check(a == 0 && slots.take(a, g, err), "first call");
    slots.arm(a, g);
    check(slots.begin(1000, err) == 1, "the other slot is free");
    const auto t0 = Clock::now();
    check(slots.begin(20000, err) == -1, "the pending slot is refused");
    check(Clock::now() - t0 >= std::chrono::milliseconds(20), "after waiting for its bound");
    check(err.find("still reads 1") != std::string::npos, "the message names the pending value");
    hsa_signal_store_screlease(g, 0);
    check(slots.begin(1000, err) == 0, "reused once the signal reads 0");
    // a negative value (a failed copy) is reported once, then the slot is usable
    check(slots.take(0, g, err), "take");
    slots.arm(0, g);
    hsa_signal_store_screlease(g, -1);
    check(slots.begin(1000, err) == 1, "slot 1");
    check(slots.begin(1000, err) == -1 && err.find("failed copy") != std::string::npos, "failed copy reported");
    check(slots.begin(1000, err) == 0, "then usable");
    // destroy leaves signals alone when the drain did not succeed
    check(slots.take(0, g, err), "take");
    slots.arm(0, g);
    const int64_t before = g_destroyed.load();
    check(!slots.drain(1000, err), "drain gives up on a pending signal");
    slots.destroy(false);
    check(g_destroyed.load() == before, "no signal destroyed while one may still be decremented");
}

// Waits (at most 5 s) until (int32)(*w - want) >= 0.
bool wait_for(const uint32_t *w, uint32_t want) {
    const auto t0 = Clock::now();
    while ((int32_t)(__atomic_load_n(w, __ATOMIC_ACQUIRE) - want) < 0) {
        if (Clock::now() - t0 > std::chrono::seconds(5))
            return false;
        std::this_thread::yield();
    }
    return true;
}

// The two buffer sets of graph-replayed rounds with SDMA legs, in host memory (the
// stand-in engines copy between any two buffers).
constexpr int kGraphSenders = 4, kGraphFlagWords = 3;
constexpr int64_t kGraphRowBytes = 64, kGraphMaxRows = 64;
struct GraphSet {
    std::vector<uint8_t> dev_send, dev_recv, host_send, host_recv;
    uint32_t ready = 0, landed = 0, recv_credit = 0;
    uint32_t send_flags[kGraphFlagWords] = {}, recv_flags[kGraphSenders] = {}, send_credits[kGraphSenders] = {};
    GraphSet() {
        for (auto *v : {&dev_send, &dev_recv, &host_send, &host_recv})
            v->assign((size_t)(kGraphMaxRows * kGraphRowBytes), 0);
    }
};
ep::GraphLegsIO graph_io(GraphSet *sets, uint32_t *status, int64_t timeout_us) {
    ep::GraphLegsIO io{};
    for (int b = 0; b < 2; ++b) {
        GraphSet &g = sets[b];
        io.ready[b] = &g.ready;
        io.landed[b] = &g.landed;
        io.send_flags[b] = g.send_flags;
        io.recv_flags[b] = g.recv_flags;
        io.recv_credit[b] = &g.recv_credit;
        io.dev_send[b] = g.dev_send.data();
        io.dev_recv[b] = g.dev_recv.data();
        io.host_send[b] = g.host_send.data();
        io.host_recv[b] = g.host_recv.data();
    }
    io.send_flag_words = kGraphFlagWords;
    io.senders = kGraphSenders;
    io.status = status;
    io.row_bytes = kGraphRowBytes;
    io.timeout_us = timeout_us;
    return io;
}
uint8_t sent_byte(uint32_t r, size_t i) { return (uint8_t)(r * 7u + i); }

// Graph-replayed rounds with SDMA legs (graph_legs.h), 200 rounds: a device stand-in (this
// thread) waits for the receivers' credits of round r - 2, packs a number of rows that
// changes from round to round into the device send buffer of set r % 2 and stamps the
// set's ready word; simulated peers wait for the last send flag, check the rows in the
// host send buffer, wait for this rank's receive credit of round r - 2, write their
// returned rows (each sent byte plus r), credit the send buffer and raise their flags in
// a random order after random delays; the device stand-in waits for the landed word,
// checks the rows in the device receive buffer and credits the set.  The stand-in engines
// apply completion decrements late.
void scenario_graph(uint32_t seed) {
    static GraphSet sets[2];
    uint32_t status[ep::kStatusWords] = {};
    ep::GraphLegs legs;
    legs.dma.init_with(kGpu, kCpu, 1u, {2u});
    legs.start(graph_io(sets, status, 5ll * 1000 * 1000), 1);
    constexpr uint32_t kRounds = 200;
    std::vector<int64_t> rows(kRounds + 1);
    std::mt19937 rng(seed);
    for (auto &n : rows)
        n = 1 + (int64_t)(rng() % kGraphMaxRows);
    std::atomic<int> peer_failures{0};
    std::thread peers([&] {
        std::mt19937 prng(seed + 1);
        for (uint32_t r = 1; r <= kRounds; ++r) {
            GraphSet &g = sets[r & 1u];
            if (!wait_for(&g.send_flags[kGraphFlagWords - 1], r)) {
                ++peer_failures;
                return;
            }
            const size_t n = (size_t)(rows[r] * kGraphRowBytes);
            for (size_t i = 0; i < n; ++i)
                if (g.host_send[i] != sent_byte(r, i)) {
                    ++peer_failures;  // a send flag came before its rows
                    break;
                }
            for (int c = 0; c < kGraphFlagWords; ++c)
                if (__atomic_load_n(&g.send_flags[c], __ATOMIC_ACQUIRE) != r)
                    ++peer_failures;
            if (!wait_for(&g.recv_credit, r - 2u)) {
                ++peer_failures;
                return;
            }
            for (size_t i = 0; i < n; ++i)
                g.host_recv[i] = (uint8_t)(g.host_send[i] + r);
            for (int i = 0; i < kGraphSenders; ++i)
                __atomic_store_n(&g.send_credits[i], r, __ATOMIC_RELEASE);
            int order[kGraphSenders] = {0, 1, 2, 3};
            std::shuffle(order, order + kGraphSenders, prng);
            for (int i : order) {
                std::this_thread::sleep_for(std::chrono::microseconds(prng() % 100));
                __atomic_store_n(&g.recv_flags[i], r, __ATOMIC_RELEASE);
            }
        }
    });
    bool rows_ok = true, landed_ok = true, credits_ok = true;
    for (uint32_t r = 1; r <= kRounds; ++r) {
        GraphSet &g = sets[r & 1u];
        for (int i = 0; i < kGraphSenders; ++i)
            credits_ok = credits_ok && wait_for(&g.send_credits[i], r - 2u);
        const size_t n = (size_t)(rows[r] * kGraphRowBytes);
        for (size_t i = 0; i < n; ++i)
            g.dev_send[i] = sent_byte(r, i);
        legs.set_rows(rows[r]);
        __atomic_store_n(&g.ready, r, __ATOMIC_RELEASE);
        if (!wait_for(&g.landed, r)) {
            landed_ok = false;
            break;
        }
        for (size_t i = 0; i < n; ++i)
            rows_ok = rows_ok && g.dev_recv[i] == (uint8_t)(sent_byte(r, i) + r);
        __atomic_store_n(&g.recv_credit, r, __ATOMIC_RELEASE);
    }
    peers.join();
    legs.stop();
    check(credits_ok, "the peers credited every send buffer");
    check(landed_ok, "every round landed");
    check(rows_ok, "every round's returned rows were in the device receive buffer when it landed");
    check(peer_failures == 0, "every send flag came after its rows, with every flag word of the set");
    check(status[0] == 0, "no wait of the legs' thread expired");
}

// Graph rounds with SDMA legs and peers that never answer: the thread copies the rows out
// and raises the send flags, gives up on the senders after its bound (20 ms), records the
// wait in the status block and still lands the round; a thread waiting for a round the
// device never reaches stops at once.
void scenario_graph_timeout() {
    static GraphSet sets[2];
    uint32_t status[ep::kStatusWords] = {};
    ep::GraphLegs legs;
    legs.dma.init_with(kGpu, kCpu, 1u, {2u});
    legs.start(graph_io(sets, status, 20 * 1000), 1);
    GraphSet &g = sets[1];
    for (size_t i = 0; i < (size_t)(8 * kGraphRowBytes); ++i)
        g.dev_send[i] = sent_byte(1, i);
    legs.set_rows(8);
    const auto t0 = Clock::now();
    __atomic_store_n(&g.ready, 1u, __ATOMIC_RELEASE);
    check(wait_for(&g.landed, 1u), "the late round still lands");
    check(Clock::now() - t0 >= std::chrono::milliseconds(20), "after the wait's bound");
    check(__atomic_load_n(&g.send_flags[0], __ATOMIC_ACQUIRE) == 1u, "the send flags are up");
    bool sent = true;
    for (size_t i = 0; i < (size_t)(8 * kGraphRowBytes); ++i)
        sent = sent && g.host_send[i] == sent_byte(1, i);
    check(sent, "the rows reached the host send buffer");
    check(__atomic_load_n(&status[0], __ATOMIC_ACQUIRE) == 5u, "the status block holds a timeout");
    check(status[1] == ep::kSiteGraphLegs, "recorded as the legs' thread's wait");
    const uint64_t flag = (uint64_t)status[2] | ((uint64_t)status[3] << 32);
    check(flag == reinterpret_cast<uint64_t>(&g.recv_flags[0]), "naming the first sender's flag");
    check(status[5] == 1u, "and the round it waited for");
    const auto t1 = Clock::now();
    legs.stop();  // the thread now waits for round 2, which never comes
    check(Clock::now() - t1 < std::chrono::milliseconds(500), "a stop ends the wait for the next round");
}

// The reuse rule this library had before, replayed directly against the stand-in: one
// completion signal shared by two flag copies, reset for the next call as soon as the
// host sees the flags.  With late decrements the stand-in must report a violation; this
// scenario checks the harness, and is expected to fail.
void scenario_old_rule(uint32_t seed) {
    std::mt19937 rng(seed);
    g_delay_max_us = 2000;
    hsa_signal_t start{}, d0{}, d1{}, shared{};
    for (hsa_signal_t *s : {&start, &d0, &d1, &shared})
        hsa_amd_signal_create(1, 0, nullptr, 0, s);
    uint32_t epoch_word = 0, flags[2] = {0, 0};
    std::vector<uint8_t> src(256, 7), dst(256);
    for (int call = 1; call <= 200 && g_violations == 0; ++call) {
        // the next call re-initialises every signal of the slot, whatever role it had
        for (hsa_signal_t s : {start, d0, d1})
            hsa_signal_store_relaxed(s, 1);
        hsa_signal_store_relaxed(shared, 2);
        epoch_word = (uint32_t)call;
        submit(dst.data(), src.data(), 128, 1, &start, d0, 1);
        submit(&flags[0], &epoch_word, 4, 1, &d0, shared, 1);
        submit(dst.data() + 128, src.data() + 128, 128, 1, &start, d1, 1);
        submit(&flags[1], &epoch_word, 4, 1, &d1, shared, 1);
        hsa_signal_store_screlease(start, 0);
        const auto t0 = Clock::now();
        while (__atomic_load_n(&flags[1], __ATOMIC_ACQUIRE) != (uint32_t)call &&
               Clock::now() - t0 < std::chrono::seconds(2))
            std::this_thread::yield();
        // roles shift: the shared completion signal becomes the first chunk's signal
        if (rng() % 2)
            std::swap(d0, shared);
    }
    g_delay_max_us = 200;
}

}  // namespace

int main(int argc, char **argv) {
    const std::string what = argc > 1 ? argv[1] : "";
    const uint32_t seed = argc > 2 ? (uint32_t)std::strtoul(argv[2], nullptr, 10) : 1u;
    if (what == "lane")
        scenario_lane(seed);
    else if (what == "exchange")
        scenario_exchange(seed);
    else if (what == "order")
        scenario_order();
    else if (what == "merge")
        scenario_merge();
    else if (what == "bounded")
        scenario_bounded();
    else if (what == "graph")
        scenario_graph(seed);
    else if (what == "graph_timeout")
        scenario_graph_timeout();
    else if (what == "old_rule")
        scenario_old_rule(seed);
    else {
        std::printf("usage: %s lane|exchange|order|merge|bounded|graph|graph_timeout|old_rule [seed]\n", argv[0]);
        return 2;
    }
    // let every queued copy finish before the engines stop
    for (;;) {
        bool idle = true;
        {
            std::lock_guard<std::mutex> lk(g_eng_mu);
            for (auto &e : g_engines)
                idle = idle && e.second->idle();
        }
        if (idle)
            break;
        std::this_thread::sleep_for(std::chrono::milliseconds(1));
    }
    stop_engines();
    std::printf("violations %d checks_failed %d signals created %lld destroyed %lld\n", g_violations.load(),
                g_checks_failed, (long long)g_created.load(), (long long)g_destroyed.load());
    return g_violations == 0 && g_checks_failed == 0 ? 0 : 1;
}
