// sdma.cpp -- the parts of the SDMA legs that need the HIP runtime: finding the ROCr
// agents of a HIP device and picking engines (sdma.h).  The rounds, copies and signals
// are in sdma_lane.cpp.
#include "sdma.h"

#include <hip/hip_runtime.h>

#include <cstdio>

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

}  // namespace

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

namespace {

int engine_index(uint32_t bit) {
    int id = 0;
    while (bit && !((bit >> id) & 1u))
        ++id;
    return id;
}

// Highest engine of a mask (0 for none).  Flag engines are taken from the top of the
// mask: the runtime's own copies (hipMemcpyAsync on a stream) run on the low engines, and
// a flag copy queued behind one of them would wait for it (measured on MI355X: the decode
// layer's default legs lost 100 us per layer with their chunk flags on engine 0).
uint32_t highest_engine(uint32_t mask) {
    if (!mask)
        return 0;
    uint32_t b = 1u << 31;
    while (!(mask & b))
        b >>= 1;
    return b;
}

}  // namespace

bool SdmaLane::init(int device, int slots, std::string &err) {
    hsa_agent_t gpu{}, cpu{};
    if (!find_agents(device, gpu, cpu, err))
        return false;
    uint32_t avail = 0, pref = 0;
    if (hsa_amd_memory_copy_engine_status(cpu, gpu, &avail) != HSA_STATUS_SUCCESS)
        avail = 0;
    if (hsa_amd_memory_get_preferred_copy_engine(cpu, gpu, &pref) != HSA_STATUS_SUCCESS)
        pref = 0;
    const uint32_t pick = (pref & avail) ? (pref & avail) : avail;
    const uint32_t engine = pick ? (pick & (~pick + 1u)) : 0u;  // lowest usable engine
    const uint32_t flag_engine = engine ? highest_engine(avail & ~engine) : 0u;
    init_with(gpu, cpu, engine, slots, flag_engine);
    owns_rocr_ = true;
    char name[64];
    if (engine)
        std::snprintf(name, sizeof name, "sdma%d, flags sdma%d (available mask 0x%x)", engine_index(engine),
                      engine_index(flag_engine_), avail);
    else
        std::snprintf(name, sizeof name, "runtime-chosen");
    engine_name_ = name;
    return true;
}

bool DmaEngines::init(int device, std::string &err) {
    hsa_agent_t gpu{}, cpu{};
    if (!find_agents(device, gpu, cpu, err))
        return false;
    owns_rocr_ = true;
    ready_ = true;  // release() drops the ROCr reference even if no engine is found
    uint32_t out_avail = 0, out_pref = 0, in_avail = 0;
    if (hsa_amd_memory_copy_engine_status(cpu, gpu, &out_avail) != HSA_STATUS_SUCCESS)
        out_avail = 0;
    if (hsa_amd_memory_get_preferred_copy_engine(cpu, gpu, &out_pref) != HSA_STATUS_SUCCESS)
        out_pref = 0;
    if (hsa_amd_memory_copy_engine_status(gpu, cpu, &in_avail) != HSA_STATUS_SUCCESS)
        in_avail = 0;
    const uint32_t pick = (out_pref & out_avail) ? (out_pref & out_avail) : out_avail;
    const uint32_t out = pick & (~pick + 1u);
    if (!out) {
        err = "no SDMA engine available for device->host copies";
        return false;
    }
    std::vector<uint32_t> in;
    for (uint32_t m = in_avail & ~out; m; m &= m - 1)
        in.push_back(m & (~m + 1u));
    // the flag engines: the two highest further engines that can write host memory (none
    // left: the flags share their data's engine)
    const uint32_t spare = out_avail & ~out & ~(in.empty() ? 0u : in[0]);
    const uint32_t out_flag = highest_engine(spare), in_flag = highest_engine(spare & ~out_flag);
    init_with(gpu, cpu, out, in, out_flag, in_flag);
    owns_rocr_ = true;
    char buf[128];
    std::snprintf(buf, sizeof buf, "out sdma%d, in %d engines, flags sdma%d / sdma%d (masks out 0x%x in 0x%x)",
                  engine_index(out_), (int)in_.size(), engine_index(out_flag_engine()),
                  engine_index(in_flag_engine()), out_avail, in_avail);
    desc_ = buf;
    return true;
}

}  // namespace ep
