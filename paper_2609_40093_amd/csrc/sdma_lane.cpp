// sdma_lane.cpp -- rounds of the default device->host leg and the copy submission of the
// exchange engines (sdma.h).  Uses only the ROCr API: agents and engines come from
// sdma.cpp (or from init_with).
#include "sdma.h"

#include <algorithm>

namespace ep {

// ---------------------------------------------------------------------- SdmaLane

void SdmaLane::init_with(hsa_agent_t gpu, hsa_agent_t cpu, uint32_t engine, int slots, uint32_t flag_engine) {
    gpu_ = gpu;
    cpu_ = cpu;
    engine_ = engine;
    flag_engine_ = flag_engine ? flag_engine : engine;
    engine_name_ = engine ? "sdma (caller-chosen)" : "runtime-chosen";
    slots_.init(slots);
    owns_rocr_ = false;
    ready_ = true;
}

void SdmaLane::release() {
    if (!ready_)
        return;
    std::string err;
    slots_.destroy(slots_.drain(kReleaseDrainUs, err));
    if (owns_rocr_)
        hsa_shut_down();
    ready_ = owns_rocr_ = false;
}

bool SdmaLane::begin(Round &r, int64_t timeout_us, std::string &err) {
    if (!ready_) {
        err = "SDMA lane not initialised";
        return false;
    }
    const int slot = slots_.begin(timeout_us, err);
    if (slot < 0)
        return false;
    if (!slots_.take(slot, r.start, err))
        return false;
    r.start_value = DmaEngines::value_pointer(r.start);
    if (!r.start_value) {
        err = "hsa_amd_signal_value_pointer failed";
        return false;
    }
    r.slot = slot;
    return true;
}

bool SdmaLane::copy(int slot, uint32_t engine, void *dst, const void *src, size_t len, const hsa_signal_t *dep,
                    hsa_signal_t *done, std::string &err) {
    if (!slots_.take(slot, *done, err))
        return false;
    hsa_status_t st;
    if (engine)
        st = hsa_amd_memory_async_copy_on_engine(dst, cpu_, src, gpu_, len, 1, dep, *done,
                                                 (hsa_amd_sdma_engine_id_t)engine, false);
    else
        st = hsa_amd_memory_async_copy(dst, cpu_, src, gpu_, len, 1, dep, *done);
    if (st != HSA_STATUS_SUCCESS) {
        err = "SDMA copy submission failed";
        return false;
    }
    slots_.arm(slot, *done);
    return true;
}

bool SdmaLane::submit(const Round &r, void *host_dst, const void *dev_src, int64_t bytes, int64_t chunk_bytes,
                      uint32_t *flags, const uint32_t *epoch_word, std::string &err) {
    slots_.arm(r.slot, r.start);  // the stream stores 0 into it before the first copy runs
    const int64_t chunks = (bytes + chunk_bytes - 1) / chunk_bytes;
    char *dst = static_cast<char *>(host_dst);
    const char *src = static_cast<const char *>(dev_src);
    for (int64_t c = 0; c < chunks; ++c) {
        const int64_t off = c * chunk_bytes;
        const size_t len = (size_t)std::min<int64_t>(chunk_bytes, bytes - off);
        hsa_signal_t data{}, flag{};
        if (!copy(r.slot, engine_, dst + off, src + off, len, &r.start, &data, err) ||
            !copy(r.slot, flag_engine_, flags + c, epoch_word, sizeof(uint32_t), &data, &flag, err))
            return false;
    }
    return true;
}

bool SdmaLane::drain(int64_t timeout_us, std::string &err) { return slots_.drain(timeout_us, err); }

// ---------------------------------------------------------------------- DmaEngines

void DmaEngines::init_with(hsa_agent_t gpu, hsa_agent_t cpu, uint32_t out_engine,
                           const std::vector<uint32_t> &in_engines, uint32_t out_flag_engine, uint32_t in_flag_engine) {
    gpu_ = gpu;
    cpu_ = cpu;
    out_ = out_engine;
    in_ = in_engines;
    out_flag_ = out_flag_engine;
    in_flag_ = in_flag_engine;
    desc_ = "caller-chosen engines";
    owns_rocr_ = false;
    ready_ = true;
}

void DmaEngines::release() {
    if (ready_ && owns_rocr_)
        hsa_shut_down();
    ready_ = owns_rocr_ = false;
}

int64_t *DmaEngines::value_pointer(hsa_signal_t sig) {
    volatile hsa_signal_value_t *value = nullptr;
    if (hsa_amd_signal_value_pointer(sig, &value) != HSA_STATUS_SUCCESS)
        return nullptr;
    return const_cast<int64_t *>(reinterpret_cast<volatile int64_t *>(value));
}

bool DmaEngines::copy(uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
                      const hsa_signal_t *deps, int ndeps, hsa_signal_t done, std::string &err) const {
    hsa_status_t st = hsa_amd_memory_async_copy_on_engine(
        dst, dst_host ? cpu_ : gpu_, src, src_host ? cpu_ : gpu_, len, (uint32_t)ndeps, deps, done,
        (hsa_amd_sdma_engine_id_t)engine, false);
    if (st != HSA_STATUS_SUCCESS) {
        err = "SDMA copy submission failed";
        return false;
    }
    return true;
}

}  // namespace ep
