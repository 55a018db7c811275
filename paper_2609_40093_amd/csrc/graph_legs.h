// graph_legs.h -- the host-leg thread of graph-replayed rounds with SDMA legs
// (ep_graph_legs_sdma; graph_legs.cpp).
//
// A captured graph replays the same launches every round, so it cannot hold DMA copies
// whose source and destination change with the round's buffer set.  With these legs the
// captured kernels stay on the device side of the staging: the dispatch packs into the
// device send buffer of set round % 2 and stamps that set's ready word in host memory; the
// combine waits (bounded) for the set's landed word in host memory and reduces from the
// device receive buffer.  This thread moves the rows in between on SDMA engines (Sec. 4.3
// of the paper: bulk data on the DMA engines, no compute unit spent on it), round r = 1,
// 2, ... on set r % 2:
//   1. waits until ready[set] holds r (the packed rows are in device memory, written back
//      past every L2 by the pack's system-scope release);
//   2. copies them to the pinned send buffer on the device->host engine and, once they
//      have landed, sets the set's send flags to r (Sec. 4.4: flags after the data);
//   3. waits for every sender's recv flag of the set to reach r and for this rank's
//      receive credit of round r - 2 (the device receive buffer has been reduced);
//   4. copies the returned rows to the device receive buffer on the host->device engine
//      and, once they have landed, sets landed[set] = r.
// Each copy is queued only once the host has seen that its source is complete, so no
// engine waits on a signal that the device releases.  The waits of steps 2 to 4 are
// bounded: one that expires is recorded in the status block and the round goes on (its
// flags are still raised), so that no device wait is left to run out its own bound.  Step
// 1 has no bound: the device reaches a round whenever the caller replays it.
//
// Only the ROCr API is used here, so the thread can be exercised on the host against a
// stand-in runtime.
#pragma once

#include "sdma.h"
#include "signal_slots.h"

#include <atomic>
#include <cstdint>
#include <string>
#include <thread>

namespace ep {

// Where the thread finds each buffer set's words and buffers (host pointers; the device
// buffers are device memory the engines read and write).
struct GraphLegsIO {
    uint32_t *ready[2];              // the device stamps the round: its rows are in dev_send
    uint32_t *landed[2];             // the thread stamps the round: the rows are in dev_recv
    uint32_t *send_flags[2];         // [send_flag_words], raised once the rows are in host_send
    int32_t send_flag_words;
    const uint32_t *recv_flags[2];   // [senders]: each sender's rows are in host_recv
    int32_t senders;
    const uint32_t *recv_credit[2];  // this rank consumed the set's receive buffer (round)
    uint32_t *status;                // status block (status_block.h)
    void *dev_send[2], *dev_recv[2], *host_send[2], *host_recv[2];
    int64_t row_bytes;
    int64_t timeout_us;  // bound of the waits for the senders and for each copy
};

class GraphLegs {
public:
    // Engines of the copies: set up by the caller before start() (init or init_with); the
    // device->host copies go on out_engine(), the host->device ones on in_engine(0).
    DmaEngines dma;

    // Starts the thread at round `first` (the round the device counter reaches next).
    void start(const GraphLegsIO &io, uint32_t first);
    // Rows of every round from the next one on (T * top-k of the captured dispatch).
    void set_rows(int64_t rows) { rows_.store(rows, std::memory_order_release); }
    // Ends the thread (between rounds, or in a wait), waits for its copies in flight, then
    // frees their signals and releases the engines.
    void stop();

private:
    enum Wait { kDone, kLate, kStopped };
    Wait wait_word(const uint32_t *w, uint32_t want, bool bounded);
    bool copy(int slot, uint32_t engine, void *dst, bool dst_host, const void *src, bool src_host, size_t len,
              const uint32_t *names_flag, uint32_t want);
    void run();

    GraphLegsIO io_{};
    SignalSlots slots_;
    std::thread th_;
    std::atomic<int64_t> rows_{0};
    std::atomic<bool> stop_{false};
    uint32_t first_ = 1;
};

}  // namespace ep
