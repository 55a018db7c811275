// sdma.cpp -- device->host leg on one SDMA engine (see sdma.h).
#include "sdma.h"

#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdio>
#include <thread>

namespace ep {
namespace {

std::string hsa_text(const char *what, hsa_status_t st) {
    const char *s = nullptr;
    if (hsa_status_string(st, &s) != HSA_STATUS_SUCCESS || !s)
        s = "unknown status";
    return std::string(what) + ": " + s;
}

struct AgentSearch {
    uint32_t bdf = 0, domain = 0;
    hsa_agent_t gpu{}, first_cpu{};
    bool found = false, have_cpu = false;
};

hsa_status_t visit_agent(hsa_agent_t a, void *data) {
    auto *s = static_cast<AgentSearch *>(data);
    hsa_device_type_t type;
    if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &type) != HSA_STATUS_SUCCESS)
        return HSA_STATUS_SUCCESS;
    if (type == HSA_DEVICE_TYPE_CPU) {
        if (!s->have_cpu) {
            s->first_cpu = a;
            s->have_cpu = true;
        }
        return HSA_STATUS_SUCCESS;
    }
    if (type != HSA_DEVICE_TYPE_GPU || s->found)
        return HSA_STATUS_SUCCESS;
    uint32_t bdf = 0, domain = 0;
    hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_BDFID), &bdf);
    hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_DOMAIN), &domain);
    if ((bdf >> 3) == (s->bdf >> 3) && domain == s->domain) {  // same bus and device
        s->gpu = a;
        s->found = true;
    }
    return HSA_STATUS_SUCCESS;
}

// The ROCr GPU agent of HIP device `device` (matched by PCI location) and its nearest CPU
// agent.  Takes a ROCr reference (hsa_init) that the caller drops with hsa_shut_down.
bool find_agents(int device, hsa_agent_t &gpu, hsa_agent_t &cpu, std::string &err) {
    hsa_status_t st = hsa_init();  // the HIP runtime initialised ROCr already; adds a reference
    if (st != HSA_STATUS_SUCCESS) {
        err = hsa_text("hsa_init", st);
        return false;
    }
    int bus = 0, dev = 0, domain = 0;
    if (hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, device) != hipSuccess ||
        hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, device) != hipSuccess ||
        hipDeviceGetAttribute(&domain, hipDeviceAttributePciDomainId, device) != hipSuccess) {
        err = "cannot read the PCI location of the HIP device";
        hsa_shut_down();
        return false;
    }
    AgentSearch search;
    search.bdf = ((uint32_t)bus << 8) | ((uint32_t)dev << 3);
    search.domain = (uint32_t)domain;
    hsa_iterate_agents(visit_agent, &search);
    if (!search.found) {
        err = "no ROCr GPU agent at the HIP device's PCI location";
        hsa_shut_down();
        return false;
    }
    gpu = search.gpu;
    hsa_agent_t near{};
    if (hsa_agent_get_info(gpu, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_NEAREST_CPU), &near) ==
            HSA_STATUS_SUCCESS && near.handle)
        cpu = near;
    else if (search.have_cpu)
        cpu = search.first_cpu;
    else {
        err = "no ROCr CPU agent";
        hsa_shut_down();
        return false;
    }
    return true;
}

int engine_index(uint32_t bit) {
    int id = 0;
    while (bit && !((bit >> id) & 1u))
        ++id;
    return id;
}

}  // namespace

bool SdmaLane::init(int device, int slots, std::string &err) {
    if (!find_agents(device, gpu_, cpu_, err))
        return false;
    hsa_status_t st;
    uint32_t avail = 0, pref = 0;
    if (hsa_amd_memory_copy_engine_status(cpu_, gpu_, &avail) != HSA_STATUS_SUCCESS)
        avail = 0;
    if (hsa_amd_memory_get_preferred_copy_engine(cpu_, gpu_, &pref) != HSA_STATUS_SUCCESS)
        pref = 0;
    const uint32_t pick = (pref & avail) ? (pref & avail) : avail;
    engine_ = pick ? (pick & (~pick + 1u)) : 0u;  // lowest usable engine
    char name[64];
    if (engine_) {
        int id = 0;
        while (!((engine_ >> id) & 1u))
            ++id;
        std::snprintf(name, sizeof name, "sdma%d (available mask 0x%x)", id, avail);
    } else {
        std::snprintf(name, sizeof name, "runtime-chosen");
    }
    engine_name_ = name;
    slots_.resize((size_t)slots);
    for (Slot &s : slots_) {
        st = hsa_amd_signal_create(1, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, &s.start);
        if (st != HSA_STATUS_SUCCESS) {
            err = hsa_text("hsa_amd_signal_create", st);
            return false;
        }
    }
    ready_ = true;
    return true;
}

void SdmaLane::release() {
    if (!drain(kReleaseDrainUs))
        slots_.clear();  // a copy may still wait on these signals: keep them alive
    for (Slot &s : slots_) {
        if (s.start.handle)
            hsa_signal_destroy(s.start);
        for (hsa_signal_t d : s.done)
            hsa_signal_destroy(d);
    }
    slots_.clear();
    if (ready_)
        hsa_shut_down();
    ready_ = false;
}

bool SdmaLane::ensure_done_signals(Slot &s, int64_t n, std::string &err) {
    while ((int64_t)s.done.size() < n + 1) {  // one per chunk, plus the flags' completion
        hsa_signal_t sig{};
        hsa_status_t st = hsa_amd_signal_create(1, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, &sig);
        if (st != HSA_STATUS_SUCCESS) {
            err = hsa_text("hsa_amd_signal_create", st);
            return false;
        }
        s.done.push_back(sig);
    }
    return true;
}

bool SdmaLane::begin(Round &r, int64_t timeout_us, std::string &err) {
    if (!ready_) {
        err = "SDMA lane not initialised";
        return false;
    }
    Slot &s = slots_[(size_t)next_];
    if (s.busy) {
        // the slot's previous round is over once its last flag holds its epoch
        const auto t0 = std::chrono::steady_clock::now();
        uint32_t spins = 0;
        while ((int32_t)(__atomic_load_n(s.last_flag, __ATOMIC_ACQUIRE) - s.epoch) < 0) {
            if (++spins % 64 == 0) {
                std::this_thread::yield();
                if (std::chrono::steady_clock::now() - t0 > std::chrono::microseconds(timeout_us)) {
                    err = "an earlier device->host leg did not finish";
                    return false;
                }
            }
        }
        s.busy = false;
    }
    hsa_signal_store_relaxed(s.start, 1);
    volatile hsa_signal_value_t *value = nullptr;
    hsa_status_t st = hsa_amd_signal_value_pointer(s.start, &value);
    if (st != HSA_STATUS_SUCCESS) {
        err = hsa_text("hsa_amd_signal_value_pointer", st);
        return false;
    }
    r.start_value = const_cast<int64_t *>(reinterpret_cast<volatile int64_t *>(value));
    r.slot = next_;
    next_ = (next_ + 1) % (int)slots_.size();
    return true;
}

bool SdmaLane::submit(const Round &r, void *host_dst, const void *dev_src, int64_t bytes, int64_t chunk_bytes,
                      uint32_t *flags, const uint32_t *epoch_word, uint32_t epoch, std::string &err) {
    Slot &s = slots_[(size_t)r.slot];
    const int64_t chunks = (bytes + chunk_bytes - 1) / chunk_bytes;
    if (!ensure_done_signals(s, chunks, err))
        return false;
    hsa_signal_t flags_done = s.done[(size_t)chunks];
    for (int64_t c = 0; c < chunks; ++c)
        hsa_signal_store_relaxed(s.done[(size_t)c], 1);
    hsa_signal_store_relaxed(flags_done, chunks);
    char *dst = static_cast<char *>(host_dst);
    const char *src = static_cast<const char *>(dev_src);
    for (int64_t c = 0; c < chunks; ++c) {
        const int64_t off = c * chunk_bytes;
        const size_t len = (size_t)std::min<int64_t>(chunk_bytes, bytes - off);
        hsa_status_t st;
        if (engine_) {
            st = hsa_amd_memory_async_copy_on_engine(dst + off, cpu_, src + off, gpu_, len, 1, &s.start,
                                                     s.done[(size_t)c], (hsa_amd_sdma_engine_id_t)engine_, false);
            if (st == HSA_STATUS_SUCCESS)
                st = hsa_amd_memory_async_copy_on_engine(flags + c, cpu_, epoch_word, gpu_, sizeof(uint32_t), 1,
                                                         &s.done[(size_t)c], flags_done,
                                                         (hsa_amd_sdma_engine_id_t)engine_, false);
        } else {
            st = hsa_amd_memory_async_copy(dst + off, cpu_, src + off, gpu_, len, 1, &s.start, s.done[(size_t)c]);
            if (st == HSA_STATUS_SUCCESS)
                st = hsa_amd_memory_async_copy(flags + c, cpu_, epoch_word, gpu_, sizeof(uint32_t), 1,
                                               &s.done[(size_t)c], flags_done);
        }
        if (st != HSA_STATUS_SUCCESS) {
            err = hsa_text("SDMA copy submission", st);
            return false;
        }
    }
    s.busy = true;
    s.last_flag = flags + (chunks - 1);
    s.epoch = epoch;
    return true;
}

bool SdmaLane::drain(int64_t timeout_us) {
    const auto t0 = std::chrono::steady_clock::now();
    uint32_t spins = 0;
    for (Slot &s : slots_) {
        if (!s.busy)
            continue;
        while ((int32_t)(__atomic_load_n(s.last_flag, __ATOMIC_ACQUIRE) - s.epoch) < 0) {
            if (++spins % 64 == 0) {
                std::this_thread::yield();
                if (std::chrono::steady_clock::now() - t0 > std::chrono::microseconds(timeout_us))
                    return false;
            }
        }
        s.busy = false;
    }
    return true;
}

// ---------------------------------------------------------------------- DmaEngines

bool DmaEngines::init(int device, std::string &err) {
    if (!find_agents(device, gpu_, cpu_, err))
        return false;
    ready_ = true;
    uint32_t out_avail = 0, out_pref = 0, in_avail = 0;
    if (hsa_amd_memory_copy_engine_status(cpu_, gpu_, &out_avail) != HSA_STATUS_SUCCESS)
        out_avail = 0;
    if (hsa_amd_memory_get_preferred_copy_engine(cpu_, gpu_, &out_pref) != HSA_STATUS_SUCCESS)
        out_pref = 0;
    if (hsa_amd_memory_copy_engine_status(gpu_, cpu_, &in_avail) != HSA_STATUS_SUCCESS)
        in_avail = 0;
    const uint32_t pick = (out_pref & out_avail) ? (out_pref & out_avail) : out_avail;
    out_ = pick & (~pick + 1u);
    if (!out_) {
        err = "no SDMA engine available for device->host copies";
        return false;
    }
    for (uint32_t m = in_avail & ~out_; m; m &= m - 1)
        in_.push_back(m & (~m + 1u));
    char buf[96];
    std::snprintf(buf, sizeof buf, "out sdma%d, in %d engines (masks out 0x%x in 0x%x)", engine_index(out_),
                  (int)in_.size(), out_avail, in_avail);
    desc_ = buf;
    return true;
}

void DmaEngines::release() {
    if (ready_)
        hsa_shut_down();
    ready_ = false;
}

bool DmaEngines::make_signal(hsa_signal_t &sig, std::string &err) {
    hsa_status_t st = hsa_amd_signal_create(1, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, &sig);
    if (st != HSA_STATUS_SUCCESS) {
        err = hsa_text("hsa_amd_signal_create", st);
        return false;
    }
    return true;
}

int64_t *DmaEngines::value_pointer(hsa_signal_t sig) {
    volatile hsa_signal_value_t *value = nullptr;
    if (hsa_amd_signal_value_pointer(sig, &value) != HSA_STATUS_SUCCESS)
        return nullptr;
    return const_cast<int64_t *>(reinterpret_cast<volatile int64_t *>(value));
}

bool DmaEngines::copy(uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
                      const hsa_signal_t *deps, int ndeps, hsa_signal_t done, std::string &err) {
    hsa_status_t st = hsa_amd_memory_async_copy_on_engine(
        dst, dst_host ? cpu_ : gpu_, src, src_host ? cpu_ : gpu_, len, (uint32_t)ndeps, deps, done,
        (hsa_amd_sdma_engine_id_t)engine, false);
    if (st != HSA_STATUS_SUCCESS) {
        err = hsa_text("SDMA copy submission", st);
        return false;
    }
    return true;
}

}  // namespace ep
