// status_block.h -- layout of the status block of a staging, shared by the wait kernels,
// the host threads that give up on a flag, and the calls that read and clear it.
#pragma once

#include <cstdint>

namespace ep {

// Coherent host words: [0] the status (0, or EP_ERR_TIMEOUT once a bounded wait expired)
// and, for the last wait that expired: [1] where it waited (a WaitSite), [2] and [3] the
// low and high halves of the address of the flag it gave up on, [4] the value it last read
// there, [5] the value it waited for.  The details are stored before word 0 (with release
// order), so a reader that takes word 0 with acquire order sees them.
constexpr int kStatusWords = 8;
enum WaitSite : uint32_t {
    kSiteUnknown = 0,
    kSiteD2H,             // wait_d2h: the last device->host chunk's flag of a dispatch
    kSiteRecv,            // wait_recv: the senders' flags of a default-mode combine
    kSiteDispatch,        // wait_dispatch: chunk and inbound-landed flags (exchange modes)
    kSiteCombine,         // wait_combine: returned-rows-landed flags (exchange modes)
    kSiteReturnedOut,     // wait_returned_out: this rank's results in host memory (duplex)
    kSiteLandedSet,       // landed_set: the senders of a pass of EP_MODE_ACCUMULATE
    kSiteCredits,         // wait_credits: graph rounds, the receivers' credits
    kSiteReturned,        // wait_returned: graph rounds, the senders' flags
    kSiteAllgather,       // wait_allgather
    kSiteReducescatter,   // wait_reducescatter
    kSiteCourier,         // the host thread gave up waiting for a sender's flag
    kSiteGraphLanded,     // wait_graph_landed: graph rounds with SDMA legs, the returned rows landed
    kSiteGraphLegs,       // the graph rounds' host-leg thread gave up on a flag or a copy
    kSiteCount
};
// The site of a wait kernel's launch name, and the name of a site.
uint32_t wait_site(const char *launch_name);
const char *wait_site_name(uint32_t site);

// Records, from the host, that a wait for `flag` to reach `want` gave up.
inline void record_host_timeout(uint32_t *status, uint32_t site, const uint32_t *flag, uint32_t want) {
    const uint64_t a = reinterpret_cast<uint64_t>(flag);
    __atomic_store_n(status + 1, site, __ATOMIC_RELAXED);
    __atomic_store_n(status + 2, (uint32_t)a, __ATOMIC_RELAXED);
    __atomic_store_n(status + 3, (uint32_t)(a >> 32), __ATOMIC_RELAXED);
    __atomic_store_n(status + 4, flag ? __atomic_load_n(flag, __ATOMIC_RELAXED) : 0u, __ATOMIC_RELAXED);
    __atomic_store_n(status + 5, want, __ATOMIC_RELAXED);
    __atomic_store_n(status, 5u /* EP_ERR_TIMEOUT */, __ATOMIC_RELEASE);
}

}  // namespace ep
