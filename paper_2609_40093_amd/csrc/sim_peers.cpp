// sim_peers.cpp -- host thread standing in for the peer ranks of a one-GPU run
// (harness for host-staged dispatch/combine; see include/ep_sim.h).
#include "ep_sim.h"

#include <immintrin.h>

#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <mutex>
#include <thread>
#include <utility>
#include <vector>

namespace {

using Clock = std::chrono::steady_clock;

struct Round {
    int32_t buf;
    uint32_t epoch;
    int64_t rows;   // exchange staging: packed rows; dense staging: the phase (0 AG, 1 RS)
    int64_t delay_us;
    Clock::time_point posted;
    std::vector<int64_t> inbound_us, return_us;  // per sender
};

// Sleeps until `t` (or returns false once `stop` is set).
bool sleep_until(Clock::time_point t, const std::atomic<bool> &stop) {
    while (Clock::now() < t) {
        if (stop)
            return false;
        std::this_thread::sleep_for(std::min<Clock::duration>(t - Clock::now(), std::chrono::milliseconds(5)));
    }
    return true;
}

// Sender indices ordered by their delay.
std::vector<int> by_delay(const std::vector<int64_t> &d) {
    std::vector<int> o(d.size());
    for (size_t i = 0; i < o.size(); ++i)
        o[i] = (int)i;
    std::stable_sort(o.begin(), o.end(), [&](int a, int b) { return d[(size_t)a] < d[(size_t)b]; });
    return o;
}

constexpr int64_t kGiveUpMs = 60 * 1000;

}  // namespace

struct ep_sim_peers {
    ep_staging *s = nullptr;
    ep_dense *dense = nullptr;
    ep_sim_mode mode = EP_SIM_FLAGS_ONLY;
    std::thread th;
    std::mutex mu;
    std::condition_variable cv, done_cv;
    std::deque<Round> q;
    std::atomic<bool> stop{false};
    int64_t posted = 0, answered = 0;
    std::atomic<int> timed_out{0};
    std::vector<int64_t> inbound_us, return_us;  // delays for rounds posted from now on
    // graph-replayed rounds: the thread follows the rounds by itself (no posts)
    bool graph = false;
    int64_t graph_rows = 0, graph_delay_us = 0;
    bool graph_echo = true;
    std::atomic<uint32_t> graph_done{0};

    // Waits until (int32)(*w - want) >= 0; false on stop or after the give-up time.
    bool wait_word(const uint32_t *w, uint32_t want) {
        const auto t0 = Clock::now();
        uint32_t spins = 0;
        while ((int32_t)(__atomic_load_n(w, __ATOMIC_ACQUIRE) - want) < 0) {
            _mm_pause();
            if (++spins % 4096 == 0) {
                if (stop)
                    return false;
                if (Clock::now() - t0 > std::chrono::milliseconds(kGiveUpMs)) {
                    timed_out.store(1);
                    return false;
                }
            }
        }
        return true;
    }

    // Round r uses buffer set r % 2: wait for this rank's send flag, wait until this rank
    // credited the receive buffer of round r - 2, echo the rows (identity experts), credit
    // the send buffer, then raise every sender's recv flag.
    void run_graph() {
        for (uint32_t r = 1;; ++r) {
            ep_staging_view v;
            if (ep_staging_ptrs(s, (int32_t)(r & 1u), &v) != EP_OK)
                return;
            if (!wait_word(v.send_flags, r) || !wait_word(v.recv_credit, r - 2u))
                return;
            if (graph_echo)
                std::memcpy(v.host_recv, v.host_send, (size_t)(graph_rows * v.row_bytes));
            for (int i = 0; i < v.num_ranks; ++i)
                __atomic_store_n(v.send_credits + i, r, __ATOMIC_RELEASE);
            if (graph_delay_us > 0 && !sleep_until(Clock::now() + std::chrono::microseconds(graph_delay_us), stop))
                return;
            for (int i = 0; i < v.num_ranks; ++i)
                __atomic_store_n(v.recv_flags + i, r, __ATOMIC_RELEASE);
            graph_done.store(r, std::memory_order_release);
            done_cv.notify_all();
        }
    }

    void run() {
        for (;;) {
            Round r;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv.wait(lk, [&] { return stop || !q.empty(); });
                if (stop)
                    return;
                r = q.front();
                q.pop_front();
            }
            serve(r);
            {
                std::lock_guard<std::mutex> lk(mu);
                ++answered;
            }
            done_cv.notify_all();
        }
    }

    // dense staging: the other ranks' flags of one phase, in order of their delays
    void serve_dense(const Round &r) {
        ep_dense_view v;
        if (ep_dense_get(dense, r.buf, &v) != EP_OK)
            return;
        const bool ag = r.rows == 0;
        const std::vector<int64_t> &delay = ag ? r.inbound_us : r.return_us;
        uint32_t *flags = ag ? v.ag_flags : v.rs_in_flags;
        for (int i : by_delay(delay)) {
            if (i == v.self_rank)
                continue;
            if (!sleep_until(r.posted + std::chrono::microseconds(delay[(size_t)i]), stop))
                return;
            __atomic_store_n(flags + i, r.epoch, __ATOMIC_RELEASE);
        }
    }

    void serve(const Round &r) {
        if (dense) {
            serve_dense(r);
            return;
        }
        ep_staging_view v;
        if (ep_staging_ptrs(s, r.buf, &v) != EP_OK)
            return;
        if ((v.mode & EP_MODE_DUPLEX) && v.in_flags) {
            for (int i : by_delay(r.inbound_us)) {
                if (i == v.self_rank)
                    continue;
                if (!sleep_until(r.posted + std::chrono::microseconds(r.inbound_us[(size_t)i]), stop))
                    return;
                __atomic_store_n(v.in_flags + i, r.epoch, __ATOMIC_RELEASE);
            }
        }
        const int64_t bytes = r.rows * v.row_bytes;
        if (bytes > 0) {
            const int64_t last = (bytes + v.chunk_bytes - 1) / v.chunk_bytes - 1;
            const uint32_t *flag = v.send_flags + last;
            const auto t0 = Clock::now();
            uint32_t spins = 0;
            while ((int32_t)(__atomic_load_n(flag, __ATOMIC_ACQUIRE) - r.epoch) < 0) {
                _mm_pause();
                if (++spins % 4096 == 0) {
                    if (stop)
                        return;
                    if (Clock::now() - t0 > std::chrono::milliseconds(kGiveUpMs)) {
                        timed_out.store(1);
                        return;
                    }
                }
            }
            if (mode == EP_SIM_ECHO)
                std::memcpy(v.host_recv, v.host_send, (size_t)bytes);
        }
        const auto landed = Clock::now() + std::chrono::microseconds(r.delay_us);
        for (int i : by_delay(r.return_us)) {
            if (!sleep_until(landed + std::chrono::microseconds(r.return_us[(size_t)i]), stop))
                return;
            __atomic_store_n(v.recv_flags + i, r.epoch, __ATOMIC_RELEASE);
        }
    }
};

extern "C" ep_status ep_sim_peers_start(ep_staging *s, ep_sim_mode mode, ep_sim_peers **out) {
    if (!s || !out || (mode != EP_SIM_FLAGS_ONLY && mode != EP_SIM_ECHO))
        return EP_ERR_INVALID_ARG;
    ep_staging_view v;
    if (ep_staging_ptrs(s, 0, &v) != EP_OK || v.kind != EP_STAGING_PINNED_HOST)
        return EP_ERR_INVALID_ARG;
    ep_sim_peers *p = new ep_sim_peers();
    p->s = s;
    p->mode = mode;
    p->th = std::thread([p] { p->run(); });
    *out = p;
    return EP_OK;
}

extern "C" ep_status ep_sim_peers_post(ep_sim_peers *p, int32_t buf, uint32_t epoch, int64_t rows,
                                       int64_t delay_us) {
    if (!p || p->dense || rows < 0 || delay_us < 0)
        return EP_ERR_INVALID_ARG;
    ep_staging_view v;
    if (ep_staging_ptrs(p->s, buf, &v) != EP_OK || rows > v.max_rows)
        return EP_ERR_INVALID_ARG;
    {
        std::lock_guard<std::mutex> lk(p->mu);
        Round r{buf, epoch, rows, delay_us, Clock::now(), p->inbound_us, p->return_us};
        r.inbound_us.resize((size_t)v.num_ranks, 0);
        r.return_us.resize((size_t)v.num_ranks, 0);
        p->q.push_back(std::move(r));
        ++p->posted;
    }
    p->cv.notify_one();
    return EP_OK;
}

namespace {
int sim_ranks(ep_sim_peers *p) {
    if (p->dense) {
        ep_dense_view v;
        return ep_dense_get(p->dense, 0, &v) == EP_OK ? v.num_ranks : -1;
    }
    ep_staging_view v;
    return ep_staging_ptrs(p->s, 0, &v) == EP_OK ? v.num_ranks : -1;
}
}  // namespace

extern "C" ep_status ep_sim_dense_start(ep_dense *d, ep_sim_peers **out) {
    if (!d || !out)
        return EP_ERR_INVALID_ARG;
    ep_dense_view v;
    if (ep_dense_get(d, 0, &v) != EP_OK)
        return EP_ERR_INVALID_ARG;
    ep_sim_peers *p = new ep_sim_peers();
    p->dense = d;
    p->th = std::thread([p] { p->run(); });
    *out = p;
    return EP_OK;
}

extern "C" ep_status ep_sim_dense_post(ep_sim_peers *p, int32_t buf, uint32_t epoch, int32_t phase) {
    if (!p || !p->dense || (phase != 0 && phase != 1))
        return EP_ERR_INVALID_ARG;
    ep_dense_view v;
    if (ep_dense_get(p->dense, buf, &v) != EP_OK)
        return EP_ERR_INVALID_ARG;
    {
        std::lock_guard<std::mutex> lk(p->mu);
        Round r{buf, epoch, phase, 0, Clock::now(), p->inbound_us, p->return_us};
        r.inbound_us.resize((size_t)v.num_ranks, 0);
        r.return_us.resize((size_t)v.num_ranks, 0);
        p->q.push_back(std::move(r));
        ++p->posted;
    }
    p->cv.notify_one();
    return EP_OK;
}

extern "C" ep_status ep_sim_peers_set_delays(ep_sim_peers *p, const int64_t *inbound_us, const int64_t *return_us) {
    if (!p)
        return EP_ERR_INVALID_ARG;
    const int R = sim_ranks(p);
    if (R < 1)
        return EP_ERR_INVALID_ARG;
    std::vector<int64_t> in((size_t)R, 0), ret((size_t)R, 0);
    for (int i = 0; i < R; ++i) {
        in[(size_t)i] = inbound_us ? inbound_us[i] : 0;
        ret[(size_t)i] = return_us ? return_us[i] : 0;
        if (in[(size_t)i] < 0 || ret[(size_t)i] < 0)
            return EP_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> lk(p->mu);
    p->inbound_us = std::move(in);
    p->return_us = std::move(ret);
    return EP_OK;
}

extern "C" ep_status ep_sim_graph_start(ep_staging *s, int64_t rows, int64_t delay_us, int32_t echo,
                                        ep_sim_peers **out) {
    if (!s || !out || rows < 0 || delay_us < 0)
        return EP_ERR_INVALID_ARG;
    ep_staging_view v;
    if (ep_staging_ptrs(s, 0, &v) != EP_OK || v.kind != EP_STAGING_PINNED_HOST || v.num_buffers != 2 ||
        rows > v.max_rows)
        return EP_ERR_INVALID_ARG;
    ep_sim_peers *p = new ep_sim_peers();
    p->s = s;
    p->graph = true;
    p->graph_rows = rows;
    p->graph_delay_us = delay_us;
    p->graph_echo = echo != 0;
    p->th = std::thread([p] { p->run_graph(); });
    *out = p;
    return EP_OK;
}

extern "C" ep_status ep_sim_graph_wait(ep_sim_peers *p, uint32_t round, int64_t timeout_ms) {
    if (!p || !p->graph)
        return EP_ERR_INVALID_ARG;
    std::unique_lock<std::mutex> lk(p->mu);
    const bool ok = p->done_cv.wait_for(lk, std::chrono::milliseconds(timeout_ms), [&] {
        return (int32_t)(p->graph_done.load(std::memory_order_acquire) - round) >= 0 || p->timed_out.load();
    });
    return ok && !p->timed_out.load() ? EP_OK : EP_ERR_TIMEOUT;
}

extern "C" ep_status ep_sim_peers_drain(ep_sim_peers *p, int64_t timeout_ms) {
    if (!p)
        return EP_ERR_INVALID_ARG;
    std::unique_lock<std::mutex> lk(p->mu);
    const bool ok = p->done_cv.wait_for(lk, std::chrono::milliseconds(timeout_ms),
                                        [&] { return p->answered == p->posted; });
    if (!ok || p->timed_out.load())
        return EP_ERR_TIMEOUT;
    return EP_OK;
}

extern "C" ep_status ep_sim_peers_stop(ep_sim_peers *p) {
    if (!p)
        return EP_OK;
    {
        std::lock_guard<std::mutex> lk(p->mu);
        p->stop = true;
    }
    p->cv.notify_all();
    if (p->th.joinable())
        p->th.join();
    delete p;
    return EP_OK;
}
