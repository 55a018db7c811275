// sdma.h -- device<->host legs on SDMA engines, driven through the ROCr runtime.
//
// The HIP runtime may run a device->host hipMemcpyAsync as a copy kernel on the compute
// units; these classes submit the legs to chosen SDMA engines instead (Sec. 4.3 of the
// paper: bulk data moves on DMA engines so that no compute unit is spent on it).
//
// SdmaLane (the default device->host leg), per round:
//   stream:  pack kernel -> event with system-scope release (every XCD's L2 written
//            back) -> 1-wave kernel storing 0 into the round's start signal
//   SDMA:    [poll start == 0] copy chunk 0 -> [poll chunk 0 done] copy epoch word
//            -> send flag 0 -> copy chunk 1 -> ... (one engine, in order)
//   stream:  bounded wait until the last chunk's flag holds the epoch
// Every copy has a completion signal of its own, and a round's signals are reused only
// once each of them reads 0 (signal_slots.h).
//
// Agent discovery needs the HIP runtime (sdma.cpp); everything else uses only ROCr
// (sdma_lane.cpp), and init_with() takes agents and engines found elsewhere.
#pragma once

#include "signal_slots.h"

#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <cstdint>
#include <string>
#include <vector>

namespace ep {

// Longest a release waits for copies still in flight before it frees their signals.
constexpr int64_t kReleaseDrainUs = 5ll * 1000 * 1000;

// The ROCr GPU agent of HIP device `device` (matched by PCI location) and its nearest CPU
// agent.  Takes a ROCr reference (hsa_init) that the caller drops with hsa_shut_down.
bool find_agents(int device, hsa_agent_t &gpu, hsa_agent_t &cpu, std::string &err);

class SdmaLane {
public:
    // Finds the GPU agent of HIP device `device`, its nearest CPU agent and a free SDMA
    // engine for device->host copies.  Returns false with `err` set on failure.
    bool init(int device, int slots, std::string &err);
    // The same with agents and engines chosen by the caller (engine 0: the runtime picks;
    // flag_engine 0: the flags go on the data engine); takes no ROCr reference.
    void init_with(hsa_agent_t gpu, hsa_agent_t cpu, uint32_t engine, int slots, uint32_t flag_engine = 0);
    // Waits (bounded) for every copy in flight, then frees the signals (or leaves them
    // allocated if a copy did not land in time).
    void release();

    struct Round {
        hsa_signal_t start{};             // released by the stream (value pointer below)
        int64_t *start_value = nullptr;  // device-writable value of the start signal
        int slot = -1;
    };
    // Reserves a slot whose previous round has fully retired (every completion signal at
    // 0), waiting on the host for at most timeout_us, and takes its start signal.
    bool begin(Round &r, int64_t timeout_us, std::string &err);
    // Submits the chunk copies of a round on the data engine and each chunk's flag copy on
    // the flag engine (after that chunk's copy has landed).  Call it after the stream work
    // that stores 0 into r.start has been enqueued.
    bool submit(const Round &r, void *host_dst, const void *dev_src, int64_t bytes, int64_t chunk_bytes,
                uint32_t *flags, const uint32_t *epoch_word, std::string &err);
    // Waits on the host (at most timeout_us in all) until every submitted copy has
    // landed.  Call it after the streams that release the rounds' start signals have run.
    bool drain(int64_t timeout_us, std::string &err);

    const char *engine_name() const { return engine_name_.c_str(); }

private:
    bool copy(int slot, uint32_t engine, void *dst, const void *src, size_t len, const hsa_signal_t *dep,
              hsa_signal_t *done, std::string &err);

    hsa_agent_t gpu_{}, cpu_{};
    uint32_t engine_ = 0;       // hsa_amd_sdma_engine_id_t bit, 0 = let the runtime choose
    uint32_t flag_engine_ = 0;  // engine of the chunk flags (0: the data engine)
    std::string engine_name_;
    SignalSlots slots_;
    bool ready_ = false, owns_rocr_ = false;
};

// SDMA engines of one GPU for the exchange legs (device->host and host->device).  Copies
// run on an engine named by its id bit, after dependency signals reach 0, and decrement
// their completion signal when they land.  One engine carries the device->host direction
// and the first other engine the host->device direction (the callers queue every inbound
// copy on that one engine).  The flag copies go on two further engines, one for the flags
// that follow outbound data and one for those that follow inbound data: a flag copy waits
// for its data copy's completion, and on the data engine that wait stalls every copy
// queued behind it (measured on MI355X: about 11 us per flag between 3.7 MB copies).
class DmaEngines {
public:
    bool init(int device, std::string &err);
    // Agents and engines chosen by the caller (no ROCr reference taken); flag engines 0:
    // the flags go on the engine of their data.
    void init_with(hsa_agent_t gpu, hsa_agent_t cpu, uint32_t out_engine, const std::vector<uint32_t> &in_engines,
                   uint32_t out_flag_engine = 0, uint32_t in_flag_engine = 0);
    void release();

    uint32_t out_engine() const { return out_; }
    // Engines of the flag copies after outbound and after inbound data.
    uint32_t out_flag_engine() const { return out_flag_ ? out_flag_ : out_; }
    uint32_t in_flag_engine() const { return in_flag_ ? in_flag_ : in_engine(0); }
    // Engine for the i-th host->device stream of copies.
    uint32_t in_engine(int i) const { return in_.empty() ? out_ : in_[(size_t)i % in_.size()]; }
    int in_engines() const { return (int)in_.size(); }
    const std::string &describe() const { return desc_; }

    static int64_t *value_pointer(hsa_signal_t sig);
    // One copy of len bytes; dst_host / src_host say which side is pinned host memory.
    bool copy(uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
              const hsa_signal_t *deps, int ndeps, hsa_signal_t done, std::string &err) const;

private:
    hsa_agent_t gpu_{}, cpu_{};
    uint32_t out_ = 0, out_flag_ = 0, in_flag_ = 0;
    std::vector<uint32_t> in_;
    std::string desc_;
    bool ready_ = false, owns_rocr_ = false;
};

}  // namespace ep
