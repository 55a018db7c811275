// exchange.cpp -- host legs of a PINNED_HOST staging in the exchange modes
// (EP_MODE_PER_SENDER, EP_MODE_DUPLEX, EP_MODE_REMOTE_ONLY; include/ep.h).
//
// Every byte crosses PCIe on an SDMA engine (Sec. 4.3: DMA offload), queued through ROCr
// with its dependencies expressed as signals:
//   - device->host copies (this rank's packed rows; in duplex mode also its results for
//     the other ranks) run on one engine, started by a one-lane kernel on the caller's
//     stream that stores 0 into the copies' start signal after a system-scope release;
//   - host->device copies (rows from each sender) run on one other engine, so that the
//     two PCIe directions overlap (Sec. 4.3: full-duplex transfers on two DMA contexts).
//     A host thread (the courier) queues each sender's copy the moment that sender's
//     completion flag in host memory holds the epoch (Sec. 4.4: flags apart from the
//     payload, per-sender waiting policy), or all of a call's copies once the last flag
//     is in (all-senders policy); the copies also wait for the caller's stream to release
//     the target buffer;
//   - each copy is followed on its engine by a 4-byte copy of the round's epoch into a
//     flag (send chunk, landed, or returned-out), and the caller's stream waits for
//     those flags (one polling lane per flag, pausing between polls) before the
//     reduction or the next round.
// Segment boundaries are routing-dependent and computed on the device; the host reads
// them once per round through a small mirror of rank_offsets (Sec. 4.5), which makes a
// duplex or remote-only dispatch wait on the host until the layout of that round has run.
#include "exchange.h"
#include "staging.h"

#include <algorithm>
#include <chrono>
#include <utility>

namespace ep {

Exchange *exchange_create(int device, int nslots, std::string &err) {
    Exchange *x = new Exchange();
    if (!x->init(device, nslots, err)) {
        x->release();
        delete x;
        return nullptr;
    }
    return x;
}

void exchange_destroy(Exchange *x) {
    if (!x)
        return;
    x->release();
    delete x;
}

const char *exchange_engines(const Exchange *x) { return x ? x->dma.describe().c_str() : ""; }

namespace {

constexpr uint32_t kSpinsPerClockCheck = 1024;

// Waits on the host for the mirror of buffer set b to carry `epoch`, then checks and
// caches the offsets.
ep_status wait_offsets(ep_staging *s, int b, uint32_t epoch, int64_t rows, const char *who) {
    const size_t R = s->R();
    const uint32_t *m = s->mirror(b);
    const auto t0 = std::chrono::steady_clock::now();
    uint32_t spins = 0;
    while (__atomic_load_n(m + R + 1, __ATOMIC_ACQUIRE) != epoch) {
        _mm_pause();
        if (++spins % kSpinsPerClockCheck == 0 &&
            std::chrono::steady_clock::now() - t0 > std::chrono::microseconds(s->timeout_us))
            return fail(EP_ERR_TIMEOUT, "%s: rank offsets of epoch %u never reached the host", who, epoch);
    }
    int32_t *o = &s->offs_cache[(size_t)b * (R + 1)];
    for (size_t r = 0; r <= R; ++r)
        o[r] = (int32_t)__atomic_load_n(m + r, __ATOMIC_RELAXED);
    bool ok = o[0] == 0 && o[R] == rows;
    for (size_t r = 0; ok && r < R; ++r)
        ok = o[r] <= o[r + 1];
    if (!ok)
        return fail(EP_ERR_INVALID_ARG, "%s: rank_offsets do not split the %lld rows of this round", who,
                    (long long)rows);
    s->offs_epoch[(size_t)b] = epoch;
    s->offs_valid[(size_t)b] = 1;
    return EP_OK;
}

// Hands a call's inbound copies to the courier (which arms their signals in `slot`).
void post_inbound(Exchange &x, int slot, const ep_staging *s, std::vector<InCopy> &&plan, uint32_t epoch,
                  bool per_sender, hsa_signal_t start, const uint32_t *epoch_word) {
    if (plan.empty())
        return;
    InJob j;
    j.copies = std::move(plan);
    j.epoch = epoch;
    j.per_sender = per_sender;
    j.start = start;
    j.epoch_word = epoch_word;
    j.epoch_words = kEpochRowWords;  // every call that posts inbound copies stamps the whole row
    j.status = s->status();
    j.deadline = std::chrono::steady_clock::now() + std::chrono::microseconds(s->timeout_us);
    x.post(slot, std::move(j));
}

struct Batch {
    GateArgs waits;    // flags the stream waits for after the copies
    void add_wait(const uint32_t *flag) {
        waits.flag[waits.n] = flag;
        waits.release[waits.n] = nullptr;
        ++waits.n;
    }
};

void init_gate(GateArgs &g, const ep_staging *s, uint32_t epoch) {
    g.n = 0;
    g.all = 0;
    g.epoch = epoch;
    g.sleep_units = s->sleep_units;
    g.timeout_ticks = s->timeout_us * s->wall_clock_khz / 1000;
    g.status = s->status();
}

// Flag copy: *flag = epoch (read from the device epoch word) on `engine` after `deps`.
bool flag_copy(Exchange &x, int slot, uint32_t engine, uint32_t *flag, const uint32_t *epoch_word,
               const hsa_signal_t *deps, int ndeps, std::string &err) {
    return x.copy(slot, engine, flag, true, epoch_word, false, sizeof(uint32_t), deps, ndeps, nullptr, err);
}

}  // namespace

ep_status exchange_enqueue_mirror(ep_staging *s, int b, uint32_t epoch, const int32_t *rank_offsets,
                                  hipStream_t stream, const char *who) {
    if (!rank_offsets)
        return fail(EP_ERR_INVALID_ARG, "%s: the exchange modes need rank_offsets", who);
    // a stale tag equal to this epoch would be taken for this round's offsets
    __atomic_store_n(s->mirror(b) + s->R() + 1, epoch - 1, __ATOMIC_RELEASE);
    EP_HIP(launch_mirror(rank_offsets, s->num_ranks + 1, s->mirror(b), epoch, stream));
    s->offs_valid[(size_t)b] = 0;
    s->offs_sent[(size_t)b] = epoch;
    return EP_OK;
}

ep_status exchange_dispatch(ep_staging *s, int b, uint32_t epoch, int64_t rows, hipStream_t stream) {
    const char *who = "ep_dispatch";
    const int R = s->num_ranks, me = s->self_rank;
    const int64_t rb = s->row_bytes;
    const bool duplex = s->mode & EP_MODE_DUPLEX, remote_only = s->mode & EP_MODE_REMOTE_ONLY,
               per_sender = s->mode & EP_MODE_PER_SENDER;
    // only the own segment's place depends on the offsets here: with neither duplex nor
    // remote-only legs the dispatch does not wait for them (the combine will)
    if (duplex || remote_only) {
        ep_status st = wait_offsets(s, b, epoch, rows, who);
        if (st != EP_OK)
            return st;
    }
    const int32_t *ro = &s->offs_cache[(size_t)b * (R + 1)];
    Exchange &x = *s->xchg;
    std::string err;

    // inbound layout: sender r's rows at [off_in[r], off_in[r+1]), own segment in place of r = me
    int64_t *rin = &s->rows_in[(size_t)b * R];
    int64_t *off = &s->off_in[(size_t)b * (R + 1)];
    if (duplex) {
        rin[me] = ro[me + 1] - ro[me];
        off[0] = 0;
        for (int r = 0; r < R; ++r)
            off[r + 1] = off[r] + rin[r];
        if (off[R] > s->max_rows)
            return fail(EP_ERR_INVALID_ARG, "%s: %lld inbound rows exceed the staging's %lld", who,
                        (long long)off[R], (long long)s->max_rows);
    }

    const int slot = x.begin(s->timeout_us, err);
    if (slot < 0)
        return fail(EP_ERR_TIMEOUT, "%s: %s", who, err.c_str());
    uint32_t *ew = s->epoch_word(b);
    char *dsend = static_cast<char *>(s->dev_send[b]);
    char *hsend = static_cast<char *>(s->host_send[b]);

    // ---- outbound: packed rows -> host send buffer, chunk flags (own segment skipped in
    //      remote-only mode; its chunks' flags are raised all the same)
    hsa_signal_t start{};
    if (!x.start_signal(slot, start, err))
        return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
    EP_HIP(hipEventRecord(s->ev_sysrel, stream));
    EP_HIP(launch_stamp_release(ew, epoch, DmaEngines::value_pointer(start), stream));  // the flags' epoch row
    x.arm(slot, start);
    const int64_t bytes = rows * rb, chunk = s->chunk_bytes;
    const int64_t chunks = (bytes + chunk - 1) / chunk;
    std::vector<std::pair<int64_t, int64_t>> ranges;
    if (remote_only) {
        ranges.push_back({0, ro[me] * rb});
        ranges.push_back({ro[me + 1] * rb, bytes});
    } else {
        ranges.push_back({0, bytes});
    }
    Batch bt;
    init_gate(bt.waits, s, epoch);
    if (chunks > 0) {
        const uint32_t out = x.dma.out_engine();
        for (int64_t c = 0; c < chunks; ++c) {
            const int64_t lo = c * chunk, hi = std::min(bytes, lo + chunk);
            hsa_signal_t deps[2] = {start, start};
            int nd = 0;
            for (const auto &rg : ranges) {
                const int64_t a = std::max(rg.first, lo), e = std::min(rg.second, hi);
                if (a >= e)
                    continue;
                if (!x.copy(slot, out, hsend + a, true, dsend + a, false, (size_t)(e - a), &start, 1, &deps[nd], err))
                    return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
                ++nd;
            }
            if (!flag_copy(x, slot, x.dma.out_flag_engine(), s->send_flags(b) + c, ew, deps, nd ? nd : 1, err))
                return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
        }
        bt.add_wait(s->send_flags(b) + (chunks - 1));
    }

    // ---- inbound (duplex): every sender's rows -> dev_in on the inbound engine, each
    //      sender's copy queued when its flag arrives (the courier)
    if (duplex) {
        char *din = static_cast<char *>(s->dev_in[b]);
        char *hin = static_cast<char *>(s->host_in[b]);
        std::vector<InCopy> plan;
        for (int r = 0; r < R; ++r) {
            if (rin[r] == 0)
                continue;
            char *dst = din + off[r] * rb;
            const int64_t len = rin[r] * rb;
            if (r == me && remote_only) {
                EP_HIP(hipMemcpyAsync(dst, dsend + ro[me] * rb, (size_t)len, hipMemcpyDeviceToDevice, stream));
                continue;
            }
            // own segment: back from the host send buffer once its last chunk's flag is up
            const uint32_t *ready = r == me ? s->send_flags(b) + ((ro[me + 1] * rb - 1) / chunk) : s->in_flags(b) + r;
            const char *src = r == me ? hsend + ro[me] * rb : hin + off[r] * rb;
            InCopy c;
            if (!x.in_copy(slot, ready, dst, src, len, s->in_landed(b) + r, c, err))
                return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
            c.eager = r == me;  // this rank's own rows wait for no sender
            plan.push_back(c);
            bt.add_wait(s->in_landed(b) + r);
        }
        post_inbound(x, slot, s, std::move(plan), epoch, per_sender, start, ew);
        s->in_epoch[(size_t)b] = epoch;
    }
    EP_HIP(launch_gate("wait_dispatch", bt.waits, stream));
    return EP_OK;
}

ep_status exchange_combine(ep_staging *s, int b, uint32_t epoch, int64_t rows, const int32_t *rank_offsets,
                           hipStream_t stream, const AccumulateCall *acc) {
    const char *who = "ep_combine";
    const int R = s->num_ranks, me = s->self_rank;
    if (!(s->offs_valid[(size_t)b] && s->offs_epoch[(size_t)b] == epoch)) {
        // the dispatch of this round queued the mirror already (it ran right after the
        // layout); otherwise queue one now
        ep_status st = s->offs_sent[(size_t)b] == epoch ? EP_OK
                                                         : exchange_enqueue_mirror(s, b, epoch, rank_offsets, stream, who);
        if (st == EP_OK)
            st = wait_offsets(s, b, epoch, rows, who);
        if (st != EP_OK)
            return st;
    }
    const int32_t *ro = &s->offs_cache[(size_t)b * (R + 1)];
    if (ro[R] != rows)
        return fail(EP_ERR_INVALID_ARG, "%s: %lld rows, but the dispatch of this buffer set had %d", who,
                    (long long)rows, ro[R]);
    const int64_t rb = s->row_bytes;
    const bool duplex = s->mode & EP_MODE_DUPLEX, remote_only = s->mode & EP_MODE_REMOTE_ONLY,
               per_sender = s->mode & EP_MODE_PER_SENDER;
    const int64_t *rin = &s->rows_in[(size_t)b * R];
    const int64_t *off = &s->off_in[(size_t)b * (R + 1)];
    if (duplex && s->in_epoch[(size_t)b] != epoch)
        return fail(EP_ERR_INVALID_ARG, "%s: duplex combine of epoch %u needs the duplex dispatch of that epoch "
                    "on the same buffer set", who, epoch);
    Exchange &x = *s->xchg;
    std::string err;
    const int slot = x.begin(s->timeout_us, err);
    if (slot < 0)
        return fail(EP_ERR_TIMEOUT, "%s: %s", who, err.c_str());
    uint32_t *ew = s->epoch_word(b);
    char *din = static_cast<char *>(s->dev_in[b]);
    char *drecv = static_cast<char *>(s->dev_recv[b]);
    const char *hrecv = static_cast<const char *>(s->host_recv[b]);
    char *hret = static_cast<char *>(s->host_ret[b]);

    // the flag copies of this call read the epoch word: stamp it, then start the
    // outbound copies (after a system-scope release of the expert results in dev_in)
    hsa_signal_t start{};
    if (!x.start_signal(slot, start, err))
        return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
    EP_HIP(hipEventRecord(s->ev_sysrel, stream));
    EP_HIP(launch_stamp_release(ew, epoch, DmaEngines::value_pointer(start), stream));
    x.arm(slot, start);
    Batch bt;
    init_gate(bt.waits, s, epoch);

    // ---- outbound (duplex): this rank's results for sender r's rows -> host_ret
    if (duplex) {
        const uint32_t out = x.dma.out_engine();
        for (int r = 0; r < R; ++r) {
            if (rin[r] == 0 || (r == me && remote_only))
                continue;
            hsa_signal_t d{};
            if (!x.copy(slot, out, hret + off[r] * rb, true, din + off[r] * rb, false, (size_t)(rin[r] * rb), &start,
                        1, &d, err) ||
                !flag_copy(x, slot, x.dma.out_flag_engine(), s->ret_flags(b) + r, ew, &d, 1, err))
                return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
            bt.add_wait(s->ret_flags(b) + r);
        }
    }

    // ---- inbound: sender r's returned rows for this rank's segment r -> dev_recv, on the
    //      inbound engine as each sender's flag arrives (the courier)
    uint32_t base = 0;  // senders whose rows need no wait: none, or copied inside HBM
    std::vector<InCopy> plan;
    for (int r = 0; r < R; ++r) {
        const int64_t n = ro[r + 1] - ro[r];
        if (n == 0) {
            base |= 1u << r;
            continue;
        }
        char *dst = drecv + ro[r] * rb;
        if (r == me && remote_only) {
            EP_HIP(hipMemcpyAsync(dst, din + off[me] * rb, (size_t)(n * rb), hipMemcpyDeviceToDevice, stream));
            base |= 1u << r;
            continue;
        }
        const bool own_dup = r == me && duplex;  // own results come back from host_ret
        const uint32_t *ready = own_dup ? s->ret_flags(b) + me : s->recv_flags(b) + r;
        const char *src = own_dup ? hret + off[me] * rb : hrecv + ro[r] * rb;
        InCopy c;
        if (!x.in_copy(slot, ready, dst, src, n * rb, s->recv_landed(b) + r, c, err))
            return fail(EP_ERR_HIP, "%s: %s", who, err.c_str());
        c.eager = own_dup;  // this rank's own results wait for no sender
        plan.push_back(c);
        if (!acc)
            bt.add_wait(s->recv_landed(b) + r);
    }
    post_inbound(x, slot, s, std::move(plan), epoch, per_sender, start, ew);
    if (!acc) {
        EP_HIP(launch_gate("wait_combine", bt.waits, stream));
        return EP_OK;
    }

    // ---- the reduction, one pass per growth of the set of landed senders (at most one
    //      pass per sender that needs a wait; later passes find nothing left to add)
    const int passes = std::max(1, R - __builtin_popcount(base));
    uint32_t *masks = s->dev_masks + (size_t)b * kMaskWords;
    const int64_t ticks = s->timeout_us * s->wall_clock_khz / 1000;
    for (int i = 0; i < passes; ++i) {
        EP_HIP(launch_landed_set(s->recv_landed(b), R, epoch, base, masks, i, ticks, s->sleep_units, s->status(),
                                 stream));
        EP_HIP(launch_accumulate(drecv, acc->slot_pos, acc->topk_w, acc->T, s->hidden, acc->k, rank_offsets, R,
                                 masks, i, s->dev_acc[b], acc->out, acc->out_f32, s->max_rows, stream));
    }
    if (bt.waits.n > 0)  // duplex: the results this rank returned are out of dev_in
        EP_HIP(launch_gate("wait_returned_out", bt.waits, stream));
    return EP_OK;
}

}  // namespace ep

// ---------------------------------------------------------------------- PCIe probe

using ep::DmaEngines;
using ep::fail;

namespace {

// Waits (host, at most 30 s) for a host-visible completion signal to drop below 1.
bool host_wait(hsa_signal_t sig) {
    const auto t0 = std::chrono::steady_clock::now();
    while (hsa_signal_wait_scacquire(sig, HSA_SIGNAL_CONDITION_LT, 1, 1000000, HSA_WAIT_STATE_BLOCKED) >= 1)
        if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(30))
            return false;
    return true;
}

}  // namespace

extern "C" ep_status ep_pcie_probe(void *host, void *dev, size_t bytes, int32_t dirs, double *gbps) {
    if (!host || !dev || !gbps || bytes == 0 || dirs < 1 || dirs > 3)
        return fail(EP_ERR_INVALID_ARG, "ep_pcie_probe: need host, dev, gbps, bytes > 0 and dirs in 1..3");
    int device = 0;
    EP_HIP(hipGetDevice(&device));
    EP_HIP(hipDeviceSynchronize());
    DmaEngines dma;
    std::string err;
    if (!dma.init(device, err)) {
        dma.release();
        return fail(EP_ERR_HIP, "ep_pcie_probe: %s", err.c_str());
    }
    hsa_signal_t sig[2] = {};
    for (hsa_signal_t &g : sig)
        if (hsa_signal_create(1, 0, nullptr, &g) != HSA_STATUS_SUCCESS) {
            for (hsa_signal_t made : sig)
                if (made.handle)
                    hsa_signal_destroy(made);
            dma.release();
            return fail(EP_ERR_HIP, "ep_pcie_probe: hsa_signal_create failed");
        }
    char *h = static_cast<char *>(host), *d = static_cast<char *>(dev);
    double best = 0.0;
    ep_status st = EP_OK;
    for (int rep = 0; rep < 5 && st == EP_OK; ++rep) {  // first run warms the engines
        for (hsa_signal_t g : sig)
            hsa_signal_store_relaxed(g, 1);
        const auto t0 = std::chrono::steady_clock::now();
        bool ok = true;
        if (dirs & 1)
            ok = ok && dma.copy(dma.out_engine(), h, true, d, false, bytes, nullptr, 0, sig[0], err);
        if (dirs & 2)
            ok = ok && dma.copy(dma.in_engine(0), d + bytes, false, h + bytes, true, bytes, nullptr, 0, sig[1], err);
        if (!ok) {
            st = fail(EP_ERR_HIP, "ep_pcie_probe: %s", err.c_str());
            break;
        }
        if (((dirs & 1) && !host_wait(sig[0])) || ((dirs & 2) && !host_wait(sig[1]))) {
            // a copy may still be in flight: keep its signals alive, report the timeout
            dma.release();
            return fail(EP_ERR_TIMEOUT, "ep_pcie_probe: a copy did not finish within 30 s");
        }
        const double sec = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        const double moved = (double)bytes * ((dirs & 1) + ((dirs >> 1) & 1));
        if (rep > 0)
            best = std::max(best, moved / sec / 1e9);
    }
    for (hsa_signal_t g : sig)
        hsa_signal_destroy(g);
    dma.release();
    if (st == EP_OK)
        *gbps = best;
    return st;
}
