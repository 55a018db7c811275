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

namespace {

struct Round {
    int32_t buf;
    uint32_t epoch;
    int64_t rows;
    int64_t delay_us;
};

constexpr int64_t kGiveUpMs = 60 * 1000;

}  // namespace

struct ep_sim_peers {
    ep_staging *s = nullptr;
    ep_sim_mode mode = EP_SIM_FLAGS_ONLY;
    std::thread th;
    std::mutex mu;
    std::condition_variable cv, done_cv;
    std::deque<Round> q;
    bool stop = false;
    int64_t posted = 0, answered = 0;
    std::atomic<int> timed_out{0};

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

    void serve(const Round &r) {
        ep_staging_view v;
        if (ep_staging_get(s, r.buf, &v) != EP_OK)
            return;
        const int64_t bytes = r.rows * v.row_bytes;
        if (bytes > 0) {
            const int64_t last = (bytes + v.chunk_bytes - 1) / v.chunk_bytes - 1;
            const uint32_t *flag = v.send_flags + last;
            const auto t0 = std::chrono::steady_clock::now();
            uint32_t spins = 0;
            while ((int32_t)(__atomic_load_n(flag, __ATOMIC_ACQUIRE) - r.epoch) < 0) {
                _mm_pause();
                if (++spins % 4096 == 0) {
                    if (stop)
                        return;
                    if (std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(kGiveUpMs)) {
                        timed_out.store(1);
                        return;
                    }
                }
            }
            if (mode == EP_SIM_ECHO)
                std::memcpy(v.host_recv, v.host_send, (size_t)bytes);
        }
        if (r.delay_us > 0)
            std::this_thread::sleep_for(std::chrono::microseconds(r.delay_us));
        for (int32_t i = 0; i < v.num_ranks; ++i)
            __atomic_store_n(v.recv_flags + i, r.epoch, __ATOMIC_RELEASE);
    }
};

extern "C" ep_status ep_sim_peers_start(ep_staging *s, ep_sim_mode mode, ep_sim_peers **out) {
    if (!s || !out || (mode != EP_SIM_FLAGS_ONLY && mode != EP_SIM_ECHO))
        return EP_ERR_INVALID_ARG;
    ep_staging_view v;
    if (ep_staging_get(s, 0, &v) != EP_OK || v.kind != EP_STAGING_PINNED_HOST)
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
    if (!p || rows < 0 || delay_us < 0)
        return EP_ERR_INVALID_ARG;
    ep_staging_view v;
    if (ep_staging_get(p->s, buf, &v) != EP_OK || rows > v.max_rows)
        return EP_ERR_INVALID_ARG;
    {
        std::lock_guard<std::mutex> lk(p->mu);
        p->q.push_back({buf, epoch, rows, delay_us});
        ++p->posted;
    }
    p->cv.notify_one();
    return EP_OK;
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
