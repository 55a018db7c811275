// signal_slots.h -- the ROCr signals of the DMA copies of the calls in flight.
//
// A DMA copy decrements its completion signal once, after its bytes are in memory.  When
// the copy writes a flag word, a host that sees the flag cannot tell whether the engine
// has applied that decrement yet.  So this pool never gives a signal a new value, or a new
// owner, while a decrement may still be on its way:
//   - every copy has a completion signal of its own (value 1, exactly one decrement), and
//     no signal is shared by several copies, so no count can be off by a late decrement;
//   - a slot is handed to a new call only once every signal its previous call armed reads
//     0 (the copy landed, or the stream kernel that releases a start signal ran);
//   - signals are destroyed only after the same check (ROCr recycles the memory of a
//     destroyed signal, so a late decrement could land in a signal of another staging).
// A decrement landing on a signal already reset to 1 for a new call would leave it at 0
// before its own copy finished, and that copy's decrement would then take it to -1; an
// engine waits for a dependency to read exactly 0, so a copy depending on it would never
// start.  The checks above rule that out.
//
// Everything here uses only the ROCr signal API, so the pool can be exercised on the host
// against a stand-in runtime.
#pragma once

#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <chrono>
#include <cstdio>
#include <string>
#include <thread>
#include <vector>

namespace ep {

class SignalSlots {
public:
    void init(int nslots) {
        slots_.assign((size_t)(nslots > 0 ? nslots : 1), Slot{});
        next_ = 0;
    }

    // Reserves the next slot for a call: waits (at most timeout_us) until every signal the
    // slot's previous call armed reads 0 or less.  Returns the slot, or -1 with `err` set
    // (the slot is then not handed out; a later begin() tries the same slot again).
    int begin(int64_t timeout_us, std::string &err) {
        const int id = next_;
        Slot &s = slots_[(size_t)id];
        if (!retire(s, timeout_us, err, id))
            return -1;
        s.used = 0;
        next_ = (next_ + 1) % (int)slots_.size();
        return id;
    }

    // A signal of slot `id`'s current call, with value 1.  Not yet armed.
    bool take(int id, hsa_signal_t &out, std::string &err) {
        Slot &s = slots_[(size_t)id];
        if (s.used == s.sigs.size()) {
            hsa_signal_t g{};
            const hsa_status_t st = hsa_amd_signal_create(1, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, &g);
            if (st != HSA_STATUS_SUCCESS) {
                err = "hsa_amd_signal_create failed";
                return false;
            }
            s.sigs.push_back(g);
        }
        out = s.sigs[s.used++];
        hsa_signal_store_relaxed(out, 1);
        return true;
    }

    // `g` (taken from slot `id`) will be brought to 0: a copy whose completion it is was
    // submitted, or the stream kernel that releases it was enqueued.  Armed signals are
    // waited for before the slot is reused or the signals destroyed.
    void arm(int id, hsa_signal_t g) { slots_[(size_t)id].armed.push_back(g); }

    // Waits (at most timeout_us in all) until every armed signal of every slot reads 0.
    bool drain(int64_t timeout_us, std::string &err) {
        const auto t0 = std::chrono::steady_clock::now();
        for (size_t i = 0; i < slots_.size(); ++i) {
            const int64_t left =
                timeout_us - std::chrono::duration_cast<std::chrono::microseconds>(std::chrono::steady_clock::now() - t0)
                                 .count();
            if (!retire(slots_[i], left > 0 ? left : 0, err, (int)i))
                return false;
        }
        return true;
    }

    // Destroys every signal when `drained` (a drain succeeded); otherwise leaves them
    // allocated, since an engine may still decrement or wait on them.
    void destroy(bool drained) {
        if (drained)
            for (Slot &s : slots_)
                for (hsa_signal_t g : s.sigs)
                    hsa_signal_destroy(g);
        slots_.clear();
    }

private:
    struct Slot {
        std::vector<hsa_signal_t> sigs;   // owned; reused by the slot's later calls
        size_t used = 0;                  // handed to the current call
        std::vector<hsa_signal_t> armed;  // to reach 0 before reuse
    };

    // Waits for the armed signals of `s` to read <= 0 and forgets them.  A negative value
    // is the runtime reporting a failed copy: reported once, then the slot is usable.
    static bool retire(Slot &s, int64_t timeout_us, std::string &err, int id) {
        const auto t0 = std::chrono::steady_clock::now();
        uint32_t spins = 0;
        for (size_t i = 0; i < s.armed.size(); ++i) {
            hsa_signal_value_t v;
            while ((v = hsa_signal_load_scacquire(s.armed[i])) > 0) {
                if (++spins % 256 == 0) {
                    std::this_thread::yield();
                    const auto waited = std::chrono::steady_clock::now() - t0;
                    if (waited > std::chrono::microseconds(timeout_us)) {
                        char buf[200];
                        std::snprintf(buf, sizeof buf,
                                      "DMA slot %d: completion signal %zu of %zu of the previous call still reads "
                                      "%lld after %lld us (a copy of that call has not landed)",
                                      id, i, s.armed.size(), (long long)v, (long long)timeout_us);
                        err = buf;
                        return false;
                    }
                }
            }
            if (v < 0) {
                char buf[160];
                std::snprintf(buf, sizeof buf, "DMA slot %d: the runtime reported a failed copy (completion signal %zu "
                              "reads %lld)", id, i, (long long)v);
                err = buf;
                s.armed.clear();
                return false;
            }
        }
        s.armed.clear();
        return true;
    }

    std::vector<Slot> slots_;
    int next_ = 0;
};

}  // namespace ep
