// sdma.h -- device->host leg on one SDMA engine, driven through the ROCr runtime.
//
// The HIP runtime may run a device->host hipMemcpyAsync as a copy kernel on the compute
// units; this lane submits the leg to a chosen SDMA engine instead (Sec. 4.3 of the
// paper: bulk data moves on DMA engines so that no compute unit is spent on it).
//
// Ordering, per round:
//   stream:  pack kernel -> event with system-scope release (every XCD's L2 written
//            back) -> 1-wave kernel storing 0 into the round's start signal
//   SDMA:    [poll start signal == 0] copy chunk 0 -> [poll chunk 0 done] copy epoch word
//            -> send flag 0 -> copy chunk 1 -> ... (one engine, in order)
//   stream:  bounded wait until the last chunk's flag holds the epoch
// Signals of a round are reused only once that round's last flag is seen on the host.
#pragma once

#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <cstdint>
#include <string>
#include <vector>

namespace ep {

// Longest a release waits for copies still in flight before it frees their signals.
constexpr int64_t kReleaseDrainUs = 5ll * 1000 * 1000;

class SdmaLane {
public:
    // Finds the GPU agent of HIP device `device`, its nearest CPU agent and a free SDMA
    // engine for device->host copies.  Returns false with `err` set on failure.
    bool init(int device, int slots, std::string &err);
    void release();

    struct Round {
        int64_t *start_value = nullptr;  // device-writable value of the start signal
        int slot = -1;
    };
    // Reserves a slot whose previous round has finished (its last flag reached its epoch),
    // waiting on the host for at most timeout_us.  Resets the slot's start signal.
    bool begin(Round &r, int64_t timeout_us, std::string &err);
    // Submits the chunk copies and the flag copies of a round (after the stream work that
    // releases the start signal has been enqueued).
    bool submit(const Round &r, void *host_dst, const void *dev_src, int64_t bytes, int64_t chunk_bytes,
                uint32_t *flags, const uint32_t *epoch_word, uint32_t epoch, std::string &err);
    // Waits on the host (at most timeout_us in all) until every submitted round's last flag
    // holds its epoch, i.e. until no copy of this lane is still in flight.  Call it after
    // the streams that release the rounds' start signals have run, before freeing the
    // buffers the copies touch.  Returns false if a round did not finish in time.
    bool drain(int64_t timeout_us);

    const char *engine_name() const { return engine_name_.c_str(); }

private:
    struct Slot {
        hsa_signal_t start{};
        std::vector<hsa_signal_t> done;  // one per chunk, grown on demand
        volatile uint32_t *last_flag = nullptr;
        uint32_t epoch = 0;
        bool busy = false;
    };
    bool ensure_done_signals(Slot &s, int64_t n, std::string &err);

    hsa_agent_t gpu_{}, cpu_{};
    uint32_t engine_ = 0;  // hsa_amd_sdma_engine_id_t bit, 0 = let the runtime choose
    std::string engine_name_;
    std::vector<Slot> slots_;
    int next_ = 0;
    bool ready_ = false;
};

// SDMA engines of one GPU for the exchange legs (device->host and host->device), driven
// through ROCr.  Copies run on an engine named by its id bit, after dependency signals
// reach 0, and decrement a completion signal when they land.  One engine carries the
// device->host direction and the first other engine the host->device direction (the
// callers queue every inbound copy on that one engine).
class DmaEngines {
public:
    bool init(int device, std::string &err);
    void release();

    uint32_t out_engine() const { return out_; }
    // Engine for the i-th host->device stream of copies.
    uint32_t in_engine(int i) const { return in_.empty() ? out_ : in_[(size_t)i % in_.size()]; }
    int in_engines() const { return (int)in_.size(); }
    const std::string &describe() const { return desc_; }

    // A GPU-only signal with value 1 (the device stores 0 into it to start a copy, or a
    // copy decrements it when it lands).
    bool make_signal(hsa_signal_t &sig, std::string &err);
    static int64_t *value_pointer(hsa_signal_t sig);
    // One copy of len bytes; dst_host / src_host say which side is pinned host memory.
    bool copy(uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
              const hsa_signal_t *deps, int ndeps, hsa_signal_t done, std::string &err);

private:
    hsa_agent_t gpu_{}, cpu_{};
    uint32_t out_ = 0;
    std::vector<uint32_t> in_;
    std::string desc_;
    bool ready_ = false;
};

}  // namespace ep
