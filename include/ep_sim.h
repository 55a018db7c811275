/*
 * ep_sim.h -- simulated peer ranks for one-GPU runs of host-staged dispatch/combine.
 *
 * HARNESS, not part of dispatch or combine.  With one GPU there are no peer ranks; a
 * host thread stands in for them on the host side of the staging, where the paper's
 * peers meet (Sec. 4.2: pinned host memory as the shared medium; Sec. 4.4: completion
 * flags in host memory).  For every posted round it
 *   0. with EP_MODE_DUPLEX, announces every other sender's inbound rows (which the
 *      harness wrote into host_in beforehand): in_flags[r] = epoch, inbound_us[r] after
 *      the post, in order of those delays,
 *   1. waits until the send flag of the round's last DMA chunk holds the round's epoch
 *      (chunks land in order, so every packed row is then in the host send buffer),
 *   2. in ECHO mode copies the host send buffer to the host recv buffer (every expert
 *      is the identity), otherwise leaves the recv buffer as the harness filled it,
 *   3. waits delay_us (emulating the peers' expert computation), then
 *   4. sets each sender's recv flag to the epoch, sender r return_us[r] later than that
 *      (skewed senders), releasing this rank's combine.
 * The thread polls with a pause instruction and gives up on a round after 60 s, which
 * ep_sim_peers_drain then reports as EP_ERR_TIMEOUT.
 */
#ifndef EP_SIM_H
#define EP_SIM_H

#include "ep.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { EP_SIM_FLAGS_ONLY = 0, EP_SIM_ECHO = 1 } ep_sim_mode;

typedef struct ep_sim_peers ep_sim_peers;

/* Starts the peer thread for a PINNED_HOST staging (EP_ERR_INVALID_ARG otherwise). */
ep_status ep_sim_peers_start(ep_staging *s, ep_sim_mode mode, ep_sim_peers **out);
/* Queues one round: `rows` packed rows were dispatched into buffer `buf` with `epoch`. */
ep_status ep_sim_peers_post(ep_sim_peers *p, int32_t buf, uint32_t epoch, int64_t rows,
                            int64_t delay_us);
/* Per-sender delays in microseconds, arrays of num_ranks (NULL = all zero), used by the
 * rounds posted after this call (steps 0 and 4 above). */
ep_status ep_sim_peers_set_delays(ep_sim_peers *p, const int64_t *inbound_us, const int64_t *return_us);
/* Simulated peers of a dense staging (ep_dense).  For each posted round the thread sets
 * the other ranks' flags, in order of their delays: phase 0 (All-Gather) ag_flags[r] =
 * epoch inbound_us[r] after the post; phase 1 (Reduce-Scatter) rs_in_flags[r] = epoch
 * return_us[r] after the post.  The harness writes the peers' shards and blocks first. */
ep_status ep_sim_dense_start(ep_dense *d, ep_sim_peers **out);
ep_status ep_sim_dense_post(ep_sim_peers *p, int32_t buf, uint32_t epoch, int32_t phase);
/* Simulated peers of graph-replayed rounds (ep_round_advance, ep_dispatch_graph,
 * ep_combine_graph) on a PINNED_HOST staging with 2 buffer sets.  The thread follows the
 * rounds r = 1, 2, ... by itself: it waits for send_flags[0] of set r % 2 to reach r and
 * for this rank's recv_credit of that set to reach r - 2, with `echo` copies the first
 * `rows` rows of the send buffer into the recv buffer (identity experts; otherwise the
 * recv buffer keeps what the harness wrote), credits the send buffer (send_credits = r),
 * waits delay_us, and sets every sender's recv flag to r. */
ep_status ep_sim_graph_start(ep_staging *s, int64_t rows, int64_t delay_us, int32_t echo, ep_sim_peers **out);
/* Blocks until the thread finished round `round` (or timeout_ms passed). */
ep_status ep_sim_graph_wait(ep_sim_peers *p, uint32_t round, int64_t timeout_ms);
/* Blocks until every posted round was answered (or timeout_ms passed). */
ep_status ep_sim_peers_drain(ep_sim_peers *p, int64_t timeout_ms);
/* Stops and joins the thread (pending rounds are dropped). */
ep_status ep_sim_peers_stop(ep_sim_peers *p);

#ifdef __cplusplus
}
#endif

#endif /* EP_SIM_H */
