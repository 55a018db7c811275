// dense.cpp -- the paper's adopted collectives (Sec. 4.2): single-step All-Gather for
// dispatch and Reduce-Scatter for combine, with pinned host memory as the shared medium.
//
// All-Gather: this rank writes its shard (T token rows) once into its slot of the host
// buffer (device->host SDMA, then an epoch flag), and reads the other ranks' slots as
// their flags arrive (host->device SDMA on the inbound engine, queued by the courier in
// arrival order).  Per GPU: S up, (N-1)S down, two phases whatever N is.
// Reduce-Scatter: this rank uploads its blocks for the other ranks (its experts'
// contributions to their shards), then either
//   - downloads the N-1 blocks for its own shard and sums them with its own block on the
//     GPU (block_reduce kernel): (N-1)S up, (N-1)S down; or
//   - (partial host reduction, Sec. 4.5) lets the host sum the N-1 remote blocks in
//     pinned memory with a thread pool, downloads that one block and adds its own on the
//     GPU: (N-1)S up, S down.
// The SDMA engines, signal slots and the courier are those of the exchange modes.
#include "exchange.h"
#include "staging.h"

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstring>

namespace {

constexpr int kDenseMaxBuffers = 8;
// The partial host reduction sums and downloads its block in up to this many pieces of at
// least 2 MiB: piece c goes down while the host sums piece c + 1.
constexpr int kReduceChunks = 16;
constexpr int64_t kReduceChunkMinBytes = 2ll << 20;

// Fixed set of host threads for the partial host reduction; run() splits [0, n) into
// `workers + 1` parts (the calling thread takes one).  run() is called by the courier
// thread; start() and stop() wait for a run() in progress before touching the workers.
class HostPool {
public:
    void start(int threads) {
        std::lock_guard<std::mutex> busy(run_mu_);
        join_all();
        stop_ = false;
        // a new worker takes only work posted after it was made (no run() can post while
        // run_mu_ is held)
        const uint64_t gen = gen_;
        for (int i = 0; i < threads; ++i)
            th_.emplace_back([this, i, gen] { loop(i, gen); });
        nworkers_.store(threads, std::memory_order_relaxed);
    }
    void stop() {
        std::lock_guard<std::mutex> busy(run_mu_);
        join_all();
    }
    int workers() const { return nworkers_.load(std::memory_order_relaxed); }
    void run(int64_t n, const std::function<void(int64_t, int64_t)> &fn) {
        std::lock_guard<std::mutex> busy(run_mu_);
        const int parts = (int)th_.size() + 1;
        {
            std::lock_guard<std::mutex> lk(mu_);
            fn_ = &fn;
            n_ = n;
            parts_ = parts;
            pending_ = parts - 1;
            ++gen_;
        }
        cv_.notify_all();
        fn(0, n / parts);
        std::unique_lock<std::mutex> lk(mu_);
        done_cv_.wait(lk, [&] { return pending_ == 0; });
        fn_ = nullptr;
    }

private:
    void join_all() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        for (std::thread &t : th_)
            if (t.joinable())
                t.join();
        th_.clear();
        nworkers_.store(0, std::memory_order_relaxed);
    }
    void loop(int i, uint64_t seen) {
        std::unique_lock<std::mutex> lk(mu_);
        for (;;) {
            cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
            if (stop_)
                return;
            seen = gen_;
            const std::function<void(int64_t, int64_t)> *fn = fn_;
            const int64_t n = n_, parts = parts_;
            lk.unlock();
            (*fn)(n * (i + 1) / parts, n * (i + 2) / parts);
            lk.lock();
            if (--pending_ == 0)
                done_cv_.notify_all();
        }
    }

    std::vector<std::thread> th_;
    std::atomic<int> nworkers_{0};
    std::mutex run_mu_;  // held by run(), start() and stop()
    std::mutex mu_;
    std::condition_variable cv_, done_cv_;
    const std::function<void(int64_t, int64_t)> *fn_ = nullptr;
    int64_t n_ = 0, parts_ = 1;
    int pending_ = 0;
    uint64_t gen_ = 0;
    bool stop_ = false;
};

// One host thread that runs queued tasks in order (the partial host reductions, so that
// the courier thread that posts them goes on queueing copies meanwhile).  stop() runs the
// tasks still queued, then ends the thread.
class Reducer {
public:
    void start() {
        stop_ = false;
        th_ = std::thread([this] { loop(); });
    }
    void stop() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        if (th_.joinable())
            th_.join();
    }
    void post(std::function<void()> task) {
        {
            std::lock_guard<std::mutex> lk(mu_);
            q_.push_back(std::move(task));
        }
        cv_.notify_one();
    }

private:
    void loop() {
        std::unique_lock<std::mutex> lk(mu_);
        for (;;) {
            cv_.wait(lk, [&] { return stop_ || !q_.empty(); });
            if (q_.empty())
                return;  // stopped, nothing left
            std::function<void()> task = std::move(q_.front());
            q_.pop_front();
            lk.unlock();
            task();
            lk.lock();
        }
    }
    std::thread th_;
    std::mutex mu_;
    std::condition_variable cv_;
    std::deque<std::function<void()>> q_;
    bool stop_ = false;
};

// IEEE binary32 -> bf16, round to nearest, ties to even (NaN kept quiet).
inline uint16_t f32_to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
inline float bf16_to_f32(uint16_t b) {
    const uint32_t u = (uint32_t)b << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

}  // namespace

struct ep_dense {
    int device = -1;
    int64_t max_tokens = 0;
    int32_t hidden = 0, R = 0, me = 0, nbuf = 0;
    bool f32_blocks = false;
    int64_t row_bytes = 0, block_row_bytes = 0;
    void *host_ag[kDenseMaxBuffers] = {}, *dev_gathered[kDenseMaxBuffers] = {};
    void *host_rs_out[kDenseMaxBuffers] = {}, *host_rs_in[kDenseMaxBuffers] = {}, *dev_rs_in[kDenseMaxBuffers] = {};
    // coherent pinned: ag, ag_landed, rs_out, rs_in, rs_landed [nbuf][R] each, then the
    // status block (ep::kStatusWords words), then the host reduction's piece flags
    // [nbuf][kReduceChunks] (epoch once the host has summed that piece)
    uint32_t *flags = nullptr;
    char *dev_epoch = nullptr;
    hipEvent_t ev_sysrel = nullptr;
    ep::Exchange *xchg = nullptr;
    HostPool pool;
    Reducer reducer;
    uint32_t reduced_epoch[kDenseMaxBuffers] = {};  // epoch of the last host reduction posted per buffer set
    uint32_t mode = 0;
    int64_t timeout_us = 10ll * 1000 * 1000;
    int32_t sleep_units = 2;
    int64_t wall_khz = 100000;
    std::atomic<int64_t> bytes_up{0}, bytes_down{0};

    uint32_t *fl(int which, int b) const { return flags + ((size_t)which * nbuf + b) * R; }
    uint32_t *ag(int b) const { return fl(0, b); }
    uint32_t *ag_landed(int b) const { return fl(1, b); }
    uint32_t *rs_out(int b) const { return fl(2, b); }
    uint32_t *rs_in(int b) const { return fl(3, b); }
    uint32_t *rs_landed(int b) const { return fl(4, b); }
    uint32_t *status() const { return flags + (size_t)5 * nbuf * R; }
    uint32_t *piece_flags(int b) const { return status() + ep::kStatusWords + (size_t)b * kReduceChunks; }
    uint32_t *epoch_word(int b) const { return reinterpret_cast<uint32_t *>(dev_epoch + b * ep::kEpochStride); }
};

namespace {

using ep::fail;
using ep::hip_fail;

void dense_release(ep_dense *d) {
    ep::exchange_destroy(d->xchg);
    d->reducer.stop();  // after the courier: no reduction is posted any more
    d->pool.stop();
    for (int b = 0; b < kDenseMaxBuffers; ++b) {
        for (void *p : {d->host_ag[b], d->host_rs_out[b], d->host_rs_in[b]})
            if (p) (void)hipHostFree(p);
        for (void *p : {d->dev_gathered[b], d->dev_rs_in[b]})
            if (p) (void)hipFree(p);
    }
    if (d->flags) (void)hipHostFree(d->flags);
    if (d->dev_epoch) (void)hipFree(d->dev_epoch);
    if (d->ev_sysrel) (void)hipEventDestroy(d->ev_sysrel);
    delete d;
}

ep_status dense_check(ep_dense *d, const char *who, int32_t buf, int64_t T) {
    if (!d)
        return fail(EP_ERR_INVALID_ARG, "%s: dense staging is NULL", who);
    if (buf < 0 || buf >= d->nbuf)
        return fail(EP_ERR_INVALID_ARG, "%s: buffer %d of %d", who, buf, d->nbuf);
    if (T < 0 || T > d->max_tokens)
        return fail(EP_ERR_INVALID_ARG, "%s: %lld tokens, the staging holds %lld per rank", who, (long long)T,
                    (long long)d->max_tokens);
    int dev = -1;
    EP_HIP(hipGetDevice(&dev));
    if (dev != d->device)
        return fail(EP_ERR_INVALID_ARG, "%s: staging lives on device %d, current device is %d", who, d->device, dev);
    return EP_OK;
}

void init_waits(ep::GateArgs &g, const ep_dense *d, uint32_t epoch) {
    g.n = 0;
    g.all = 0;
    g.epoch = epoch;
    g.sleep_units = d->sleep_units;
    g.timeout_ticks = d->timeout_us * d->wall_khz / 1000;
    g.status = d->status();
}

void add_wait(ep::GateArgs &g, const uint32_t *flag) {
    g.flag[g.n] = flag;
    g.release[g.n] = nullptr;
    ++g.n;
}

}  // namespace

extern "C" ep_status ep_dense_alloc(int64_t max_tokens, int32_t hidden, int32_t num_ranks, int32_t self_rank,
                                    int32_t num_buffers, ep_out_dtype block_dtype, ep_dense **out) {
    if (!out)
        return fail(EP_ERR_INVALID_ARG, "ep_dense_alloc: out is NULL");
    *out = nullptr;
    if (max_tokens < 1 || hidden < 8 || hidden % 8 != 0 || num_ranks < 1 || num_ranks > ep::kMaxExchangeRanks ||
        self_rank < 0 || self_rank >= num_ranks || num_buffers < 1 || num_buffers > kDenseMaxBuffers ||
        (block_dtype != EP_OUT_BF16 && block_dtype != EP_OUT_F32))
        return fail(EP_ERR_INVALID_ARG,
                    "ep_dense_alloc: need max_tokens >= 1, hidden a positive multiple of 8, 1 <= R <= %d, "
                    "0 <= self_rank < R, 1 <= num_buffers <= %d, block dtype bf16 or f32",
                    ep::kMaxExchangeRanks, kDenseMaxBuffers);
    ep_dense *d = new ep_dense();
    d->max_tokens = max_tokens;
    d->hidden = hidden;
    d->R = num_ranks;
    d->me = self_rank;
    d->nbuf = num_buffers;
    d->f32_blocks = block_dtype == EP_OUT_F32;
    d->row_bytes = (int64_t)hidden * 2;
    d->block_row_bytes = (int64_t)hidden * (d->f32_blocks ? 4 : 2);
    const size_t ag_bytes = (size_t)num_ranks * max_tokens * d->row_bytes;
    const size_t rs_bytes = (size_t)num_ranks * max_tokens * d->block_row_bytes;
#define EP_DENSE_HIP(call)                                                                          \
    do {                                                                                            \
        hipError_t e_ = (call);                                                                     \
        if (e_ != hipSuccess) {                                                                     \
            ep_status st_ = hip_fail(e_, #call);                                                    \
            dense_release(d);                                                                       \
            return st_;                                                                             \
        }                                                                                           \
    } while (0)
    EP_DENSE_HIP(hipGetDevice(&d->device));
    int khz = 0;
    EP_DENSE_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, d->device));
    if (khz > 0)
        d->wall_khz = khz;
    for (int b = 0; b < num_buffers; ++b) {
        EP_DENSE_HIP(hipHostMalloc(&d->host_ag[b], ag_bytes, hipHostMallocDefault));
        EP_DENSE_HIP(hipMalloc(&d->dev_gathered[b], ag_bytes));
        EP_DENSE_HIP(hipHostMalloc(&d->host_rs_out[b], rs_bytes, hipHostMallocDefault));
        EP_DENSE_HIP(hipHostMalloc(&d->host_rs_in[b], rs_bytes, hipHostMallocDefault));
        EP_DENSE_HIP(hipMalloc(&d->dev_rs_in[b], rs_bytes));
    }
    const size_t words = (size_t)5 * num_buffers * num_ranks + ep::kStatusWords + (size_t)num_buffers * kReduceChunks;
    EP_DENSE_HIP(hipHostMalloc((void **)&d->flags, words * sizeof(uint32_t), hipHostMallocCoherent));
    std::memset(d->flags, 0, words * sizeof(uint32_t));
    EP_DENSE_HIP(hipMalloc((void **)&d->dev_epoch, kDenseMaxBuffers * ep::kEpochStride));
    EP_DENSE_HIP(hipEventCreateWithFlags(&d->ev_sysrel, hipEventDisableTiming | hipEventReleaseToSystem));
#undef EP_DENSE_HIP
    std::string err;
    d->xchg = ep::exchange_create(d->device, ep::kSdmaSlots, err);
    if (!d->xchg) {
        dense_release(d);
        return fail(EP_ERR_HIP, "ep_dense_alloc: SDMA engines: %s", err.c_str());
    }
    const unsigned hc = std::thread::hardware_concurrency();
    d->pool.start((int)std::min<unsigned>(15u, hc > 1 ? hc - 1 : 0u));
    d->reducer.start();
    *out = d;
    return EP_OK;
}

extern "C" ep_status ep_dense_free(ep_dense *d) {
    if (!d)
        return EP_OK;
    int prev = -1;
    if (hipGetDevice(&prev) == hipSuccess && prev != d->device)
        (void)hipSetDevice(d->device);
    (void)hipDeviceSynchronize();
    dense_release(d);
    if (prev >= 0)
        (void)hipSetDevice(prev);
    return EP_OK;
}

extern "C" ep_status ep_dense_get(ep_dense *d, int32_t buf, ep_dense_view *v) {
    if (!d || !v)
        return fail(EP_ERR_INVALID_ARG, "ep_dense_get: NULL argument");
    if (buf < 0 || buf >= d->nbuf)
        return fail(EP_ERR_INVALID_ARG, "ep_dense_get: buffer %d of %d", buf, d->nbuf);
    v->num_ranks = d->R;
    v->self_rank = d->me;
    v->num_buffers = d->nbuf;
    v->hidden = d->hidden;
    v->block_dtype = d->f32_blocks ? EP_OUT_F32 : EP_OUT_BF16;
    v->max_tokens = d->max_tokens;
    v->row_bytes = d->row_bytes;
    v->block_row_bytes = d->block_row_bytes;
    v->host_ag = d->host_ag[buf];
    v->dev_gathered = d->dev_gathered[buf];
    v->host_rs_out = d->host_rs_out[buf];
    v->host_rs_in = d->host_rs_in[buf];
    v->dev_rs_in = d->dev_rs_in[buf];
    v->ag_flags = d->ag(buf);
    v->ag_landed = d->ag_landed(buf);
    v->rs_out_flags = d->rs_out(buf);
    v->rs_in_flags = d->rs_in(buf);
    v->rs_landed = d->rs_landed(buf);
    return EP_OK;
}

extern "C" ep_status ep_dense_set_policy(ep_dense *d, uint32_t mode, int64_t timeout_us, int32_t host_threads) {
    if (!d || (mode & ~EP_MODE_PER_SENDER) || timeout_us < 0 || host_threads < 0 || host_threads > 256)
        return fail(EP_ERR_INVALID_ARG,
                    "ep_dense_set_policy: mode 0 or EP_MODE_PER_SENDER, timeout_us >= 0, 0 <= host_threads <= 256");
    d->mode = mode;
    d->timeout_us = timeout_us;
    d->pool.start(host_threads > 0 ? host_threads - 1 : d->pool.workers());
    return EP_OK;
}

extern "C" ep_status ep_dense_status(ep_dense *d, hipStream_t stream) {
    if (!d)
        return fail(EP_ERR_INVALID_ARG, "ep_dense_status: NULL staging");
    EP_HIP(hipStreamSynchronize(stream));
    struct Namer : ep::FlagNamer {
        const ep_dense *d;
        explicit Namer(const ep_dense *dd) : d(dd) {}
        std::string operator()(const uint32_t *f) const override {
            static const char *names[5] = {"ag_flags", "ag_landed", "rs_out_flags", "rs_in_flags", "rs_landed"};
            for (int w = 0; w < 5; ++w)
                for (int b = 0; b < d->nbuf; ++b) {
                    const uint32_t *base = d->fl(w, b);
                    if (f >= base && f < base + d->R) {
                        char buf[80];
                        std::snprintf(buf, sizeof buf, "%s[buf %d][rank %d]", names[w], b, (int)(f - base));
                        return buf;
                    }
                }
            return "";
        }
    };
    return ep::take_status(d->status(), d->timeout_us, Namer(d));
}

extern "C" ep_status ep_dense_bytes(ep_dense *d, int64_t *up, int64_t *down) {
    if (!d || !up || !down)
        return fail(EP_ERR_INVALID_ARG, "ep_dense_bytes: NULL argument");
    *up = d->bytes_up.load();
    *down = d->bytes_down.load();
    return EP_OK;
}

extern "C" ep_status ep_allgather(ep_dense *d, int32_t buf, uint32_t epoch, const void *x_dev, int64_t num_tokens,
                                  hipStream_t stream) {
    const char *who = "ep_allgather";
    ep_status st = dense_check(d, who, buf, num_tokens);
    if (st != EP_OK)
        return st;
    const int64_t T = num_tokens, rb = d->row_bytes, shard = T * rb;
    if (T == 0)
        return EP_OK;
    if (!x_dev || !ep::aligned16(x_dev))
        return fail(EP_ERR_INVALID_ARG, "%s: x must be a non-NULL 16-byte aligned pointer", who);
    ep::Exchange &x = *d->xchg;
    std::string err;
    const int slot = x.begin(d->timeout_us, err);
    if (slot < 0)
        return fail(EP_ERR_TIMEOUT, "%s: %s", who, err.c_str());
    char *hag = static_cast<char *>(d->host_ag[buf]);
    char *dg = static_cast<char *>(d->dev_gathered[buf]);
    const int me = d->me, R = d->R;
    uint32_t *ew = d->epoch_word(buf);

    // own shard: into the gathered buffer (HBM copy) and once into host memory (SDMA)
    EP_HIP(hipMemcpyAsync(dg + me * shard, x_dev, (size_t)shard, hipMemcpyDeviceToDevice, stream));
    hsa_signal_t start{}, sent{};
    if (!x.start_signal(slot, start, err))
        return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
    EP_HIP(hipEventRecord(d->ev_sysrel, stream));
    EP_HIP(ep::launch_stamp_release(ew, epoch, ep::DmaEngines::value_pointer(start), stream));
    x.arm(slot, start);
    if (!x.copy(slot, x.dma.out_engine(), hag + me * shard, true, x_dev, false, (size_t)shard, &start, 1, &sent, err) ||
        !x.copy(slot, x.dma.out_flag_engine(), d->ag(buf) + me, true, ew, false, sizeof(uint32_t), &sent, 1, nullptr,
                err))
        return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
    d->bytes_up += shard;
    ep::GateArgs waits;
    init_waits(waits, d, epoch);
    add_wait(waits, d->ag(buf) + me);

    // the other shards, each as soon as its rank's flag is in
    std::vector<ep::InCopy> plan;
    for (int r = 0; r < R; ++r) {
        if (r == me)
            continue;
        ep::InCopy c;
        if (!x.in_copy(slot, d->ag(buf) + r, dg + r * shard, hag + r * shard, shard, d->ag_landed(buf) + r, c, err))
            return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
        plan.push_back(c);
        add_wait(waits, d->ag_landed(buf) + r);
        d->bytes_down += shard;
    }
    if (!plan.empty()) {
        ep::InJob j;
        j.copies = std::move(plan);
        j.epoch = epoch;
        j.per_sender = d->mode & EP_MODE_PER_SENDER;
        j.start = start;
        j.epoch_word = ew;
        j.epoch_words = ep::kEpochRowWords;
        j.status = d->status();
        j.deadline = std::chrono::steady_clock::now() + std::chrono::microseconds(d->timeout_us);
        x.post(slot, std::move(j));
    }
    EP_HIP(ep::launch_gate("wait_allgather", waits, stream));
    return EP_OK;
}

extern "C" ep_status ep_reducescatter(ep_dense *d, int32_t buf, uint32_t epoch, const void *blocks_dev,
                                      int64_t num_tokens, int32_t reduce_on_host, void *out_dev,
                                      ep_out_dtype out_dtype, hipStream_t stream) {
    const char *who = "ep_reducescatter";
    ep_status st = dense_check(d, who, buf, num_tokens);
    if (st != EP_OK)
        return st;
    if (out_dtype != EP_OUT_BF16 && out_dtype != EP_OUT_F32)
        return fail(EP_ERR_INVALID_ARG, "%s: unknown out_dtype %d", who, (int)out_dtype);
    const int64_t T = num_tokens, brb = d->block_row_bytes, block = T * brb;
    if (T == 0)
        return EP_OK;
    if (!blocks_dev || !out_dev || !ep::aligned16(blocks_dev) || !ep::aligned16(out_dev))
        return fail(EP_ERR_INVALID_ARG, "%s: blocks and out must be non-NULL 16-byte aligned pointers", who);
    ep::Exchange &x = *d->xchg;
    std::string err;
    const int slot = x.begin(d->timeout_us, err);
    if (slot < 0)
        return fail(EP_ERR_TIMEOUT, "%s: %s", who, err.c_str());
    const int me = d->me, R = d->R;
    const char *blocks = static_cast<const char *>(blocks_dev);
    char *hout = static_cast<char *>(d->host_rs_out[buf]);
    char *hin = static_cast<char *>(d->host_rs_in[buf]);
    char *din = static_cast<char *>(d->dev_rs_in[buf]);
    uint32_t *ew = d->epoch_word(buf);
    ep::GateArgs waits;
    init_waits(waits, d, epoch);

    // ---- up: this rank's blocks for the other ranks, each flagged as soon as written
    hsa_signal_t start{};
    if (!x.start_signal(slot, start, err))
        return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
    EP_HIP(hipEventRecord(d->ev_sysrel, stream));
    EP_HIP(ep::launch_stamp_release(ew, epoch, ep::DmaEngines::value_pointer(start), stream));
    x.arm(slot, start);
    for (int r = 0; r < R; ++r) {
        if (r == me)
            continue;
        hsa_signal_t dn{};
        if (!x.copy(slot, x.dma.out_engine(), hout + r * block, true, blocks + r * block, false, (size_t)block, &start,
                    1, &dn, err) ||
            !x.copy(slot, x.dma.out_flag_engine(), d->rs_out(buf) + r, true, ew, false, sizeof(uint32_t), &dn, 1, nullptr,
                    err))
            return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
        d->bytes_up += block;
        add_wait(waits, d->rs_out(buf) + r);
    }

    // ---- down: the blocks for this rank's shard (or their host-side sum)
    ep::BlockList bl;
    ep::InJob j;
    j.epoch = epoch;
    j.start = start;
    j.epoch_word = ew;
    j.epoch_words = ep::kEpochRowWords;
    j.status = d->status();
    j.deadline = std::chrono::steady_clock::now() + std::chrono::microseconds(d->timeout_us);
    if (R > 1 && !reduce_on_host) {
        j.per_sender = d->mode & EP_MODE_PER_SENDER;
        for (int r = 0; r < R; ++r) {
            bl.ptr[bl.n++] = r == me ? blocks + me * block : din + r * block;  // summed in rank order
            if (r == me)
                continue;
            ep::InCopy c;
            if (!x.in_copy(slot, d->rs_in(buf) + r, din + r * block, hin + r * block, block, d->rs_landed(buf) + r, c,
                           err))
                return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
            j.copies.push_back(c);
            add_wait(waits, d->rs_landed(buf) + r);
            d->bytes_down += block;
        }
    } else if (R > 1) {
        // partial host reduction: once every remote block is in, the host sums them (fp32,
        // rank order) into this rank's own slot of the host buffer, piece by piece on the
        // reducer thread; each piece goes down as soon as it is summed (its piece flag),
        // the last one followed by the block's landed flag
        const int64_t n = T * d->hidden, eb = brb / d->hidden;
        const int64_t want_pieces = std::max<int64_t>(1, std::min<int64_t>(kReduceChunks, block / kReduceChunkMinBytes));
        const int64_t per = ((n + want_pieces - 1) / want_pieces + 4095) / 4096 * 4096;  // elements, 4096-aligned
        const int pieces = (int)((n + per - 1) / per);
        uint32_t *pf = d->piece_flags(buf);
        for (int c = 0; c < pieces; ++c) {
            const int64_t e0 = c * per, e1 = std::min(n, e0 + per);
            ep::InCopy piece;
            if (!x.in_copy(slot, pf + c, din + me * block + e0 * eb, hin + me * block + e0 * eb, (e1 - e0) * eb,
                           c == pieces - 1 ? d->rs_landed(buf) + me : nullptr, piece, err))
                return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
            piece.eager = true;  // the host's sum, not a sender's rows: goes when summed
            j.copies.push_back(piece);
        }
        j.per_sender = false;
        for (int r = 0; r < R; ++r)
            if (r != me)
                j.ready_all.push_back(d->rs_in(buf) + r);
        const bool f32 = d->f32_blocks;
        HostPool *pool = &d->pool;
        Reducer *reducer = &d->reducer;
        // the previous reduction into this buffer set must have gone down before this one
        // overwrites its sum
        const uint32_t prev = d->reduced_epoch[buf];
        d->reduced_epoch[buf] = epoch;
        const uint32_t *prev_landed = d->rs_landed(buf) + me;
        uint32_t *status = d->status();
        const int64_t timeout_us = d->timeout_us;
        j.before_copies = [=]() {
            reducer->post([=]() {
                if (prev != 0) {
                    const auto w0 = std::chrono::steady_clock::now();
                    while ((int32_t)(__atomic_load_n(prev_landed, __ATOMIC_ACQUIRE) - prev) < 0) {
                        if (std::chrono::steady_clock::now() - w0 > std::chrono::microseconds(timeout_us)) {
                            ep::record_host_timeout(status, ep::kSiteCourier, prev_landed, prev);
                            break;
                        }
                        std::this_thread::yield();
                    }
                }
                const std::function<void(int64_t, int64_t)> sum = [=](int64_t lo, int64_t hi) {
                    for (int64_t i0 = lo; i0 < hi; i0 += 4096) {
                        const int64_t i1 = std::min(hi, i0 + 4096);
                        float acc[4096];
                        for (int64_t i = i0; i < i1; ++i)
                            acc[i - i0] = 0.f;
                        for (int r = 0; r < R; ++r) {
                            if (r == me)
                                continue;
                            if (f32) {
                                const float *src = reinterpret_cast<const float *>(hin + r * block);
                                for (int64_t i = i0; i < i1; ++i)
                                    acc[i - i0] += src[i];
                            } else {
                                const uint16_t *src = reinterpret_cast<const uint16_t *>(hin + r * block);
                                for (int64_t i = i0; i < i1; ++i)
                                    acc[i - i0] += bf16_to_f32(src[i]);
                            }
                        }
                        if (f32) {
                            float *dst = reinterpret_cast<float *>(hin + me * block);
                            for (int64_t i = i0; i < i1; ++i)
                                dst[i] = acc[i - i0];
                        } else {
                            uint16_t *dst = reinterpret_cast<uint16_t *>(hin + me * block);
                            for (int64_t i = i0; i < i1; ++i)
                                dst[i] = f32_to_bf16(acc[i - i0]);
                        }
                    }
                };
                // one pass of the pool: each of its `parts` threads sums its share of piece 0,
                // then of piece 1, ...; the thread that finishes a piece last raises its flag,
                // so piece c goes down while the threads sum piece c + 1
                const auto t0 = std::chrono::steady_clock::now();
                const int parts = pool->workers() + 1;
                std::atomic<int> finished[kReduceChunks];
                for (int c = 0; c < pieces; ++c)
                    finished[c].store(0, std::memory_order_relaxed);
                pool->run(parts, [&](int64_t lo, int64_t hi) {
                    for (int c = 0; c < pieces; ++c) {
                        const int64_t e0 = c * per, e1 = std::min(n, e0 + per), len = e1 - e0;
                        for (int64_t q = lo; q < hi; ++q)
                            sum(e0 + len * q / parts, e0 + len * (q + 1) / parts);
                        if (finished[c].fetch_add((int)(hi - lo), std::memory_order_acq_rel) + (int)(hi - lo) == parts)
                            __atomic_store_n(pf + c, epoch, __ATOMIC_RELEASE);
                    }
                });
                ep::trace_host("host_reduce",
                               std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count());
            });
        };
        add_wait(waits, d->rs_landed(buf) + me);
        d->bytes_down += block;
        bl.ptr[bl.n++] = blocks + me * block;
        bl.ptr[bl.n++] = din + me * block;
    } else {
        bl.ptr[bl.n++] = blocks;
    }
    x.post(slot, std::move(j));
    EP_HIP(ep::launch_gate("wait_reducescatter", waits, stream));
    EP_HIP(ep::launch_block_reduce(bl, d->f32_blocks, T * d->hidden, out_dev, out_dtype == EP_OUT_F32, stream));
    return EP_OK;
}
