/*
 * ep.h -- C ABI of the MI355X expert-parallel dispatch/combine library (libep.so).
 *
 * One GPU is one rank of an expert-parallel (EP) group of R ranks.  A MoE layer's
 * router has picked k of E experts per token; experts are placed contiguously, rank r
 * holding experts [r*L, (r+1)*L) with L = E/R.  The library computes this rank's share
 * of the layer's communication (Lee et al., "Efficient Expert-Parallel Communication on
 * PCIe-Connected Consumer GPUs"):
 *
 *   ep_dispatch_layout  counts, prefix offsets and the packed row of every (token, slot),
 *                       grouping rows by destination rank, then expert, then token
 *                       (Sec. 4.3: tokens are grouped by the experts that consume them;
 *                       Sec. 4.5: routing-aware transfer of only the rows each
 *                       destination needs).
 *   ep_dispatch         packs the token rows into that contiguous layout (Sec. 2.2:
 *                       a DMA engine moves only contiguous regions, so a kernel packs
 *                       routing-dependent rows first) and, with host staging, moves the
 *                       packed buffer to a pinned host bounce buffer on a DMA (SDMA)
 *                       stream in fixed chunks, raising one completion flag per chunk in
 *                       host memory (Sec. 4.3 DMA offload; Sec. 4.4 flags kept apart
 *                       from the payload).
 *   ep_combine          waits for the peers' completion flags (one polling lane per
 *                       sender, with pauses between polls: Sec. 4.4), moves the returned
 *                       rows host->device on a second DMA stream, and reduces each
 *                       token's k returned rows, weighted by its gates, in fp32 back into
 *                       token order on the GPU (Sec. 4.3: the reduction stays on the GPU
 *                       because a DMA engine cannot add).
 *   ep_staging_alloc    the send/receive buffers (HBM, or HBM plus pinned host bounce
 *                       buffers) with their flags and DMA streams.
 *
 * Conventions for every call:
 *   - Pointers named *_dev (and every array argument not marked "host") are device
 *     pointers on the current HIP device; the caller owns them.  bf16 data is passed as
 *     raw 16-bit patterns.  Byte offsets are 64-bit; rows are never assumed < 2^31 bytes.
 *   - Every call only enqueues work on `stream` (0 = the null stream) and returns; the
 *     outputs are valid once `stream` has reached that point.  Only ep_layout_validate,
 *     ep_staging_status, ep_staging_alloc/free and ep_trace_read block.
 *   - Argument errors a host can see are reported synchronously and nothing is enqueued.
 *     Errors that depend on device data (an expert id out of range, a token row naming
 *     an expert twice, a flag wait that expired) are recorded in a status word and read
 *     by ep_layout_validate / ep_staging_status.  No call throws.
 *   - ep_last_error() returns this thread's text for the last non-OK status.
 *   - Calls on one ep_staging must not overlap from several host threads.
 */
#ifndef EP_H
#define EP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EP_ABI_VERSION 6
#define EP_MAX_EXPERTS 2048 /* largest E the layout kernels accept */

typedef enum {
    EP_OK = 0,
    EP_ERR_INVALID_ARG = 1, /* a size, pointer or mode the call cannot accept */
    EP_ERR_BAD_ROUTING = 2, /* an expert id outside [0,E) or repeated within a token row */
    EP_ERR_HIP = 3,         /* the HIP runtime reported an error (text in ep_last_error) */
    EP_ERR_OOM = 4,         /* device or pinned host allocation failed */
    EP_ERR_TIMEOUT = 5,     /* a bounded completion-flag wait expired */
} ep_status;

typedef enum {
    EP_STAGING_HBM = 0,         /* send/recv buffers in HBM only; no host leg */
    EP_STAGING_PINNED_HOST = 1, /* plus pinned host bounce buffers, SDMA legs, host flags */
} ep_staging_kind;

typedef enum {
    EP_OUT_BF16 = 0, /* combine output rounded to nearest-even bf16 */
    EP_OUT_F32 = 1,  /* combine output as the fp32 accumulator itself (exactness tests) */
} ep_out_dtype;

typedef struct ep_staging ep_staging; /* opaque, owned by the library */

int32_t ep_abi_version(void);
const char *ep_status_name(int32_t status);
const char *ep_last_error(void);

/* ------------------------------------------------------------------------- layout */

/* Bytes of device workspace ep_dispatch_layout needs for T tokens, top-k, E experts
 * (the grouping of Sec. 4.3 counts every routing entry; the workspace holds its partial
 * counts and its status).  bytes: host out; EP_ERR_INVALID_ARG for sizes the layout does
 * not accept. */
ep_status ep_layout_workspace_bytes(int64_t num_tokens, int32_t topk, int32_t num_experts,
                                    size_t *bytes /* host out */);

/* Dispatch layout (Sec. 4.3 grouping; Sec. 4.5 routing-aware rows): a stable counting
 * sort of the T*k routing entries by expert id.
 *   topk_idx        int32 [T][k] row-major: slot j of token t selects expert topk_idx[t*k+j].
 *   expert_counts   int32 [E]: rows for expert e (one per (token, slot) selecting it).
 *   expert_offsets  int32 [E+1]: exclusive prefix sum of expert_counts; [E] = T*k.
 *   rank_counts     int32 [R]: rows for rank r = sum of its experts' counts.
 *   rank_offsets    int32 [R+1]: rank_offsets[r] = expert_offsets[r*E/R]; [R] = T*k.
 *   slot_pos        int32 [T*k]: packed row of slot t*k+j = expert_offsets[e] + number of
 *                   earlier slots (smaller flat index) with the same expert.
 *   row_src         int32 [T*k] or NULL: inverse of slot_pos (row p came from slot row_src[p]).
 *   workspace       device scratch of ep_layout_workspace_bytes() bytes, zero-filled
 *                   before its first use (e.g. hipMemset) and otherwise left alone between
 *                   calls: it holds the partial counts of the tiles of the routing array
 *                   and the status read by ep_layout_validate.  Calls that share a workspace must be ordered
 *                   (same stream or events).  No workgroup of a layout waits for another,
 *                   so a layout completes whatever else the device runs.
 * Requires T >= 0, T*k < 2^31, 1 <= k <= E <= EP_MAX_EXPERTS, R >= 1, E % R == 0.
 * T == 0 is valid: counts and offsets are written as zeros.  With an invalid expert id
 * the outputs are unspecified but every write stays inside the arrays above, and the
 * slot of that id gets slot_pos = -1. */
ep_status ep_dispatch_layout(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                             int32_t num_experts, int32_t num_ranks,
                             int32_t *expert_counts, int32_t *expert_offsets,
                             int32_t *rank_counts, int32_t *rank_offsets,
                             int32_t *slot_pos, int32_t *row_src,
                             void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Validation of the routing a layout consumed (Sec. 4.3: every routing entry names one
 * of the E experts, each at most once per token).  Synchronizes `stream`, then reads the
 * status word the last layout on `workspace` left: EP_OK, or EP_ERR_BAD_ROUTING (an id
 * outside [0,E) or an expert repeated in a row). */
ep_status ep_layout_validate(const void *workspace, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving
 * loops that must not allocate, harnesses that forbid hipMalloc): ep_dispatch_layout with
 * no workspace argument.  The layout's scratch is the library's own, a fixed 128 KiB
 * array per GPU (held until the process ends), which fits every size ep_dispatch_layout
 * accepts; sizes beyond it are refused with EP_ERR_INVALID_ARG.  Arguments, outputs and
 * results as ep_dispatch_layout, bit for bit, except:
 *   status_dev  device uint32 the routing status is written to (0, or bit 0 an id outside
 *               [0,E), bit 1 an expert repeated within a token row), as ep_layout_validate
 *               would report it; caller-owned, valid once `stream` has reached the call.
 * The call allocates nothing.  Every call on one GPU shares that GPU's scratch: calls that
 * overlap on one GPU (other streams or host threads without ordering) race. */
ep_status ep_dispatch_layout_static(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                                    int32_t num_experts, int32_t num_ranks,
                                    int32_t *expert_counts, int32_t *expert_offsets,
                                    int32_t *rank_counts, int32_t *rank_offsets,
                                    int32_t *slot_pos, int32_t *row_src, uint32_t *status_dev,
                                    hipStream_t stream);

/* ------------------------------------------------------------------------ staging */

/* Allocates the staging of one rank: the buffers every dispatch and combine moves rows
 * through.  With host staging the bounce buffers are pinned host memory, the one medium
 * that ranks without peer-to-peer access all reach over PCIe (Sec. 4.2), and the
 * completion flags are separate words in coherent host memory, each written by one
 * party only (Sec. 4.4).
 *   kind         EP_STAGING_HBM or EP_STAGING_PINNED_HOST.
 *   max_rows     rows per buffer (>= T*k of every later call), hidden = H (multiple of 8).
 *   num_ranks    R: number of senders whose completion flags ep_combine waits for.
 *   num_buffers  1..8 independent buffer sets (alternate them between rounds).
 *   chunk_bytes  size of one device->host DMA chunk (0 = 64 MiB); rounded up to 4 KiB.
 * Per buffer: HBM send (packed) and recv (returned rows) buffers of max_rows*H*2 bytes;
 * with PINNED_HOST also pinned host send/recv bounce buffers of the same size, one
 * uint32 send flag per chunk and one uint32 recv flag per sender in coherent pinned host
 * memory, all zero-initialised.  Creates two non-blocking streams at default priority,
 * up (device->host) and down (host->device), and takes SDMA engines through ROCr: one for
 * the device->host chunks and another for their flag copies (a flag copy waits for its
 * chunk to land, and on the chunk's own engine that wait would hold up the chunks behind
 * it).  With the environment variable EP_HOSTLEG_COPY=hip the device->host chunks and
 * flags go through hipMemcpyAsync on the up stream instead. */
ep_status ep_staging_alloc(ep_staging_kind kind, int64_t max_rows, int32_t hidden,
                           int32_t num_ranks, int32_t num_buffers, int64_t chunk_bytes,
                           ep_staging **out);
/* Frees a staging (NULL is a no-op): the pinned buffers and flag words of Sec. 4.2 and
 * Sec. 4.4.  Blocks: synchronises the staging's device, waits for every SDMA copy still in
 * flight (queued copies whose flags never came are started first, so that none writes
 * freed memory; at most 5 s in all, after which the copies' completion signals are left
 * allocated rather than freed under an engine), then frees the buffers.  Stop simulated
 * peers of the staging (ep_sim_peers_stop) before. */
ep_status ep_staging_free(ep_staging *s);

typedef struct {
    int32_t kind, num_ranks, num_buffers, hidden;
    int64_t max_rows, row_bytes, buffer_bytes, chunk_bytes;
    int32_t max_chunks;           /* send flags per buffer */
    void *dev_send, *dev_recv;    /* device, buffer_bytes each */
    void *host_send, *host_recv;  /* pinned host, or NULL in HBM mode */
    uint32_t *send_flags;         /* host [max_chunks], or NULL: flag c = epoch when chunk c landed */
    uint32_t *recv_flags;         /* host [num_ranks], or NULL: set to epoch by sender r */
    /* exchange modes (ep_staging_set_mode); NULL until EP_MODE_DUPLEX allocated them */
    uint32_t mode;
    int32_t self_rank;
    void *dev_in;                 /* device, buffer_bytes: rows every sender dispatched to this rank */
    void *host_in, *host_ret;     /* pinned host, buffer_bytes: inbound rows; this rank's outbound results */
    uint32_t *in_flags;           /* host [num_ranks]: sender r sets epoch when its inbound rows are in host_in */
    uint32_t *ret_flags;          /* host [num_ranks]: set to epoch once the results for rank r are in host_ret */
    uint32_t *in_landed;          /* host [num_ranks]: set to epoch once sender r's inbound rows are in dev_in */
    uint32_t *recv_landed;        /* host [num_ranks]: set to epoch once sender r's returned rows are in dev_recv */
    const int64_t *in_offsets;    /* host [num_ranks+1]: first dev_in/host_in row of each sender (last dispatch) */
    uint32_t *send_credits;       /* host [num_ranks]: receiver r sets the round once it consumed this send buffer */
    uint32_t *recv_credit;        /* host word: this rank sets the round once it consumed this recv buffer */
} ep_staging_view;

/* Pointers and sizes of buffer set `buf` (host pointers are usable from the host): the
 * device send/recv buffers, the pinned bounce buffers that stand for the shared host
 * medium of Sec. 4.2 (NULL with HBM staging), and the flag words of Sec. 4.4 that the
 * other ranks (here: simulated peers on the host) write.  The view is owned by the
 * caller; the pointers stay valid until ep_staging_free. */
ep_status ep_staging_ptrs(ep_staging *s, int32_t buf, ep_staging_view *view);

/* Bounded flag wait used by ep_combine with host staging: give up after timeout_us
 * microseconds (default 10 s), pausing sleep_units*64 cycles between polls (default 2). */
ep_status ep_staging_set_wait(ep_staging *s, int64_t timeout_us, int32_t sleep_units);

/* Synchronizes the staging's streams and `stream`, then returns and clears its status
 * block: EP_OK, or EP_ERR_TIMEOUT if a bounded flag wait (Sec. 4.4) expired since the last
 * call; ep_last_error then names the wait, the flag array, buffer set and index it gave
 * up on, the value it last read and the value it waited for. */
ep_status ep_staging_status(ep_staging *s, hipStream_t stream);

/* Exchange modes of a PINNED_HOST staging (bit flags; 0 = the default legs above).
 * Every mode reads the layout's rank_offsets on the host (a small device->host copy of
 * R+1 words, the mirror) before it queues the DMA copies, since segment boundaries come
 * from routing computed on the device (Sec. 4.5: routing-aware transfers need the
 * routing metadata on the host); the calls then wait on the host for that mirror.
 *   EP_MODE_PER_SENDER   each sender's rows are downloaded as soon as that sender's
 *                        flag arrives instead of after the last sender's (Sec. 4.4,
 *                        per-sender waiting policy): a library thread watches the flags
 *                        in host memory and queues the copies on the one host->device
 *                        SDMA engine in arrival order.
 *   EP_MODE_DUPLEX       each phase moves both PCIe directions at once (Sec. 4.3,
 *                        full-duplex transfers on two DMA contexts): dispatch also
 *                        downloads the rows every sender dispatched to this rank
 *                        (host_in -> dev_in, rows per sender from ep_staging_set_inbound),
 *                        and combine also uploads this rank's expert results for every
 *                        sender (dev_in -> host_ret, one ret flag per destination raised
 *                        as soon as its part is written).  The rank's own segment makes
 *                        the round trip through host memory like any other.
 *   EP_MODE_REMOTE_ONLY  (with DUPLEX) the rank's own segment never crosses PCIe: it is
 *                        copied inside HBM (packed -> dev_in, dev_in -> recv).
 *   EP_MODE_ACCUMULATE   (with PER_SENDER) ep_combine reduces each sender's returned rows
 *                        as they land (Sec. 4.4 per-sender policy; Sec. 4.5: computation
 *                        begins upon each sender's completion): one pass per growth of
 *                        the set of landed senders adds, for every token, the slots of the
 *                        longest prefix whose senders have all landed, to an fp32 partial
 *                        sum in device memory.  Every token's k rows still go in slot
 *                        order from +0, so `out` equals that of the single reduction bit
 *                        for bit, whatever order the senders arrive in.  Adds T*H*4 bytes
 *                        of device memory per buffer set (allocated by the first combine,
 *                        regrown when T*H grows).
 * self_rank: the rank this GPU plays (0..R-1).  The exchange modes require R <= 32.
 * Allocates host_in, dev_in and host_ret on first use of DUPLEX. */
#define EP_MODE_PER_SENDER 1u
#define EP_MODE_DUPLEX 2u
#define EP_MODE_REMOTE_ONLY 4u
#define EP_MODE_ACCUMULATE 8u
ep_status ep_staging_set_mode(ep_staging *s, uint32_t mode, int32_t self_rank);

/* Rows each sender r != self_rank dispatches to this rank in buffer set `buf` (host
 * array of num_ranks; the self entry is ignored: it is this rank's own segment).  Used by
 * EP_MODE_DUPLEX dispatches; the inbound rows of sender r occupy host_in/dev_in rows
 * [in_offsets[r], in_offsets[r+1]) in rank order. */
ep_status ep_staging_set_inbound(ep_staging *s, int32_t buf, const int64_t *rows_per_sender);

/* --------------------------------------------------------------- dispatch / combine */

/* Dispatch of one round (epoch) into buffer set `buf` (Sec. 2.2: a DMA engine moves only
 * contiguous regions, so the routed rows are packed first; Sec. 4.3: the host leg runs on
 * a DMA engine in chunks; Sec. 4.4: one completion flag per chunk, apart from the data):
 *   packed[slot_pos[t*k+j]][:] = x[t][:] for every token t and slot j   (bf16 byte copy)
 * into the staging's HBM send buffer.  x_dev: bf16 [T][H]; slot_pos: int32 [T*k] from
 * ep_dispatch_layout; rows with slot_pos outside [0, max_rows) are skipped.
 * With PINNED_HOST, the first T*k rows then go device->host on an SDMA engine in
 * chunk_bytes pieces, and after chunk c has landed send_flags[c] is set to `epoch`
 * (a 4-byte DMA copy queued behind the chunk).  `stream` waits (bounded) for the last
 * flag before later work.  Epochs should increase per
 * round (flags compare as signed 32-bit differences).
 * rank_offsets: int32 [R+1] from ep_dispatch_layout; required by the exchange modes
 * (ep_staging_set_mode), else may be NULL.  With EP_MODE_REMOTE_ONLY the chunks' flags
 * are still all raised, but no byte of the own segment is copied. */
ep_status ep_dispatch(const void *x_dev, int64_t num_tokens, int32_t hidden, int32_t topk,
                      const int32_t *slot_pos, const int32_t *rank_offsets, ep_staging *s,
                      int32_t buf, uint32_t epoch, hipStream_t stream);

/* Layout and dispatch in one call: the same results as ep_dispatch_layout(topk_idx, ...)
 * followed by ep_dispatch(x_dev, T, hidden, topk, slot_pos, rank_offsets, s, buf, epoch),
 * bit for bit, and the same arguments, ownership and errors (the layout arguments as in
 * ep_dispatch_layout, the rest as in ep_dispatch; every argument is checked before
 * anything is enqueued).  Sec. 4.3 (tokens grouped by the experts that consume them)
 * and Sec. 2.2 (rows packed into contiguous segments for the DMA engine).
 * For few routing entries one kernel does both steps, each workgroup counting every
 * routing entry itself (no exchange between workgroups, no second kernel): with HBM
 * staging or the default pinned mode, E <= 256, topk in {1, 2, 4, 8}, T*topk <= 65536
 * when E <= 64 and topk <= 4, otherwise T*topk <= 16384 (8192 when hidden > 4096),
 * hidden = 512 * g with g in {1, 2, 4, 8, 14, 16}, and topk_idx 16-byte aligned.  Otherwise the two steps run
 * as their own kernels.  The fused kernel writes only the status word of the workspace. */
ep_status ep_dispatch_fused(const int32_t *topk_idx, int64_t num_tokens, int32_t topk,
                            int32_t num_experts, int32_t num_ranks, int32_t *expert_counts,
                            int32_t *expert_offsets, int32_t *rank_counts, int32_t *rank_offsets,
                            int32_t *slot_pos, int32_t *row_src, void *workspace, size_t workspace_bytes,
                            const void *x_dev, int32_t hidden, ep_staging *s, int32_t buf, uint32_t epoch,
                            hipStream_t stream);

/* Combine of one round from buffer set `buf` (Sec. 4.4: wait for every sender's flag,
 * polling sparingly; Sec. 4.3: the gate-weighted reduction runs on the GPU, a DMA engine
 * cannot add):
 *   out[t][:] = sum_{j<k} topk_w[t*k+j] * recv[slot_pos[t*k+j]][:]
 * accumulated in fp32 with fused multiply-adds in slot order j = 0..k-1, then rounded
 * to nearest-even bf16 (EP_OUT_BF16) or stored as fp32 (EP_OUT_F32).  recv holds the
 * returned rows in the packed layout.  With PINNED_HOST, first waits (bounded, see
 * ep_staging_set_wait) until recv_flags[r] has reached `epoch` for every sender r, then
 * moves the first T*k rows host->device (one DMA copy, ordered on `stream`).
 * topk_w: float [T][k]; out: [T][H] of out_dtype.  Slots whose slot_pos is outside
 * [0, max_rows) contribute nothing.  rank_offsets as for ep_dispatch (the exchange modes
 * reuse the offsets read by the dispatch of the same buffer set and epoch). */
ep_status ep_combine(ep_staging *s, int32_t buf, uint32_t epoch, const int32_t *slot_pos,
                     const int32_t *rank_offsets, const float *topk_w, int64_t num_tokens,
                     int32_t hidden, int32_t topk, void *out_dev, ep_out_dtype out_dtype,
                     hipStream_t stream);

/* -------------------------------------------------- graph-replayed rounds (Sec. 4.5)
 *
 * For decode, where a captured HIP graph replays every layer.  The round number lives in
 * device memory and every kernel of these calls reads it there, so the captured launches
 * stay valid from one replay to the next; nothing is passed per round from the host.
 * Buffer set b = round % 2 alternates (a PINNED_HOST staging with num_buffers == 2): a
 * sender writes buffer set b only after every receiver has credited its contents of two
 * rounds ago, and credits its own receive buffer once the reduction has read it (Sec. 4.4:
 * receivers send credits by writes; the double buffer lets the next round start without
 * a global synchronization).  The rows move on the compute units (stores to and loads from
 * pinned host memory) because a captured DMA copy keeps the addresses recorded at capture
 * (Sec. 4.5); at decode sizes the compute units are not the contended resource.
 *   ep_round_advance   round += 1; the first call of each round (capture it too).
 *   ep_dispatch_graph  waits for send_credits of buffer set b to reach round - 2, packs the
 *                      rows straight into host_send of set b, then sets that set's
 *                      send_flags[0] = round.
 *   ep_combine_graph   waits for recv_flags of set b to reach round (every sender), reduces
 *                      the rows straight from host_recv of set b, then sets recv_credit of
 *                      set b = round.
 * Arguments and results as for ep_dispatch / ep_combine (slot_pos from a layout whose
 * workspace was zero-filled once: the layout is replay-safe too).  Graph rounds and the
 * other legs must not be mixed on one staging. */
ep_status ep_round_advance(ep_staging *s, hipStream_t stream);
/* Synchronizes the device and reads the round counter. */
ep_status ep_round_read(ep_staging *s, uint32_t *round);
ep_status ep_dispatch_graph(const void *x_dev, int64_t num_tokens, int32_t hidden, int32_t topk,
                            const int32_t *slot_pos, ep_staging *s, hipStream_t stream);
ep_status ep_combine_graph(ep_staging *s, const int32_t *slot_pos, const float *topk_w, int64_t num_tokens,
                           int32_t hidden, int32_t topk, void *out_dev, ep_out_dtype out_dtype, hipStream_t stream);
/* Host legs of graph-replayed rounds on SDMA engines instead of the compute units (Sec. 4.3:
 * the DMA engines move the bulk data, so no compute unit is spent on it; Sec. 4.4: flags
 * raised only after their data).  on = 1 starts a library thread (call it outside graph
 * capture, before capturing the rounds: it reads the round counter); on = 0 stops it,
 * after synchronizing the device.  With the thread running, ep_dispatch_graph packs into
 * the device send buffer of set round % 2 and stamps that set's ready word in host memory;
 * the thread sees it, copies the T*topk rows to host_send on the device->host engine, and
 * sets the set's send_flags to the round once they have landed; it then waits for every
 * sender's recv flag of the set and for this rank's recv_credit of round - 2, copies the
 * returned rows from host_recv to the device recv buffer on the host->device engine and
 * sets the set's landed word; ep_combine_graph waits (bounded) for that word and reduces
 * from the device recv buffer.  The other ranks (simulated peers) see the same flags,
 * credits and pinned buffers as with the compute-unit legs.  No copy depends on a signal
 * released by the device: each is queued once its source is complete.  The thread's
 * waits for the peers and for its copies are bounded by the staging's timeout as set when
 * the thread starts (ep_staging_set_wait); an expired one is recorded in the status block
 * (ep_staging_status) and the round goes on.
 * Which legs a round uses is fixed when its ep_dispatch_graph / ep_combine_graph calls are
 * made (or captured): replay rounds captured with the thread running only while it runs
 * (otherwise their combine waits out its bound and reports EP_ERR_TIMEOUT), and rounds
 * captured without it keep the compute-unit legs.  ep_staging_free stops the thread.
 * EP_ERR_INVALID_ARG for a staging that graph rounds cannot use; EP_ERR_HIP if no SDMA
 * engine can be taken. */
ep_status ep_graph_legs_sdma(ep_staging *s, int32_t on);

/* ------------------------------------------------------- dense collectives (Sec. 4.2)
 *
 * The paper's adopted design: dispatch is a single-step All-Gather of every rank's token
 * rows, combine a Reduce-Scatter of partial blocks, both through pinned host memory as
 * the one medium all ranks share.  For this rank (self_rank of R, T tokens per rank):
 *   ep_allgather          uploads its shard once and downloads the R-1 others as their
 *                         ranks' flags arrive: S up, (R-1)S down (S = T*H*2 bytes);
 *   ep_dispatch_layout_local, ep_pack
 *                         group the R*T gathered tokens by the experts this rank owns
 *                         (Sec. 4.3) and pack them for the expert computation;
 *   ep_combine_rows       turns the experts' outputs into R partial blocks, block d =
 *                         this rank's contribution to rank d's shard (gate-weighted sum over
 *                         its local experts, fp32 accumulation);
 *   ep_reducescatter      uploads the R-1 blocks for the other ranks and sums the blocks for
 *                         its own shard: on the GPU after downloading R-1 blocks ((R-1)S up,
 *                         (R-1)S down), or with the partial host reduction (Sec. 4.5: host
 *                         threads sum the R-1 remote blocks in pinned memory, one block goes
 *                         down, (R-1)S up, S down).
 * Every transfer runs on SDMA engines as in the exchange modes (one device->host engine,
 * one host->device engine whose copies are queued in flag-arrival order). */
typedef struct ep_dense ep_dense; /* opaque, owned by the library */

/* Buffers of `num_buffers` independent rounds for up to max_tokens tokens per rank:
 * pinned host [R][max_tokens][H] shard slots, device [R][max_tokens][H] gathered rows,
 * pinned host and device [R][max_tokens][H] blocks in block_dtype (bf16 rounded to
 * nearest-even, or fp32), coherent host flags.  R <= 32. */
ep_status ep_dense_alloc(int64_t max_tokens, int32_t hidden, int32_t num_ranks, int32_t self_rank,
                         int32_t num_buffers, ep_out_dtype block_dtype, ep_dense **out);
/* Frees a dense staging, after the device and every SDMA copy in flight as ep_staging_free. */
ep_status ep_dense_free(ep_dense *d);

typedef struct {
    int32_t num_ranks, self_rank, num_buffers, hidden, block_dtype;
    int64_t max_tokens, row_bytes, block_row_bytes;
    void *host_ag;          /* pinned: rank r's shard at rows [r*T, (r+1)*T) of a T-token call */
    void *dev_gathered;     /* device, same layout: the All-Gather's result */
    void *host_rs_out;      /* pinned: this rank's block for rank r at rows [r*T, (r+1)*T) */
    void *host_rs_in;       /* pinned: rank r's block for this rank (own slot: the host-side sum) */
    void *dev_rs_in;        /* device, same layout as host_rs_in */
    uint32_t *ag_flags;     /* host [R]: rank r sets epoch once its shard is in host_ag */
    uint32_t *ag_landed;    /* host [R]: epoch once rank r's shard is in dev_gathered */
    uint32_t *rs_out_flags; /* host [R]: epoch once this rank's block for r is in host_rs_out */
    uint32_t *rs_in_flags;  /* host [R]: rank r sets epoch once its block for this rank is in host_rs_in */
    uint32_t *rs_landed;    /* host [R]: epoch once that block (or the host sum, own slot) is on the GPU */
} ep_dense_view;
ep_status ep_dense_get(ep_dense *d, int32_t buf, ep_dense_view *view);

/* mode: 0 (download after the last rank's flag) or EP_MODE_PER_SENDER; timeout_us bounds
 * every flag wait (default 10 s); host_threads: threads of the partial host reduction
 * (0 keeps the current count).  Waits for a partial host reduction in progress. */
ep_status ep_dense_set_policy(ep_dense *d, uint32_t mode, int64_t timeout_us, int32_t host_threads);
/* Synchronizes `stream`; returns and clears the status word (EP_ERR_TIMEOUT after an expired
 * wait). */
ep_status ep_dense_status(ep_dense *d, hipStream_t stream);
/* PCIe payload bytes queued so far by this staging's collectives, each direction (flag
 * words not counted): the measured side of the volume model of Sec. 4.2. */
ep_status ep_dense_bytes(ep_dense *d, int64_t *up, int64_t *down);

/* All-Gather of round `epoch` into buffer set `buf`: x_dev bf16 [T][H] is this rank's
 * shard; afterwards the gathered rows are dev_gathered [R*T][H] (rank order). */
ep_status ep_allgather(ep_dense *d, int32_t buf, uint32_t epoch, const void *x_dev, int64_t num_tokens,
                       hipStream_t stream);

/* Reduce-Scatter of round `epoch`: blocks_dev [R][T][H] in the block dtype (block r: this
 * rank's contribution to rank r's shard); out_dev [T][H] = sum over r of the blocks for
 * this rank's shard, fp32 accumulation in rank order, stored as out_dtype.  With
 * reduce_on_host the R-1 remote blocks are first summed by host threads (fp32, rank order,
 * stored in the block dtype) and the GPU adds its own block to that sum. */
ep_status ep_reducescatter(ep_dense *d, int32_t buf, uint32_t epoch, const void *blocks_dev, int64_t num_tokens,
                           int32_t reduce_on_host, void *out_dev, ep_out_dtype out_dtype, hipStream_t stream);

/* Grouping of N (gathered) tokens by the experts [e_lo, e_hi) of E: ep_dispatch_layout
 * restricted to a window (Sec. 4.3: each rank groups the tokens it received by the
 * experts it owns).  Outputs local_counts[L], local_offsets[L+1] (L = e_hi - e_lo),
 * slot_pos[N*k] (-1 for slots naming other experts), row_src[local rows] or NULL.
 * Routing errors (ids outside [0,E), an expert twice in a row) are checked over every
 * id, as in ep_dispatch_layout.  workspace: ep_layout_workspace_bytes(N, k, L) bytes,
 * zero-filled before first use. */
ep_status ep_dispatch_layout_local(const int32_t *topk_idx, int64_t num_tokens, int32_t topk, int32_t num_experts,
                                   int32_t e_lo, int32_t e_hi, int32_t *local_counts, int32_t *local_offsets,
                                   int32_t *slot_pos, int32_t *row_src, void *workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/* out[slot_pos[t*k+j]][:] = x[t][:] for slots with slot_pos in [0, max_rows) (the pack of
 * ep_dispatch on caller-owned buffers). */
ep_status ep_pack(const void *x_dev, int64_t num_tokens, int32_t hidden, int32_t topk, const int32_t *slot_pos,
                  void *out_dev, int64_t max_rows, hipStream_t stream);

/* out[t][:] = sum_j topk_w[t*k+j] * y[slot_pos[t*k+j]][:] over slots with slot_pos in
 * [0, max_rows) (the reduction of ep_combine on caller-owned buffers; over the gathered
 * tokens with a window layout it yields the partial blocks of ep_reducescatter). */
ep_status ep_combine_rows(const void *y_dev, int64_t max_rows, const int32_t *slot_pos, const float *topk_w,
                          int64_t num_tokens, int32_t hidden, int32_t topk, void *out_dev, ep_out_dtype out_dtype,
                          hipStream_t stream);

/* ------------------------------------------------------------------ measurement */

typedef struct {
    char name[48];
    int64_t count;
    double total_ms, min_ms, max_ms;
    /* percentiles of the traced durations (the sample of rank round(q*(count-1)) in
     * sorted order; computed over the first 65536 durations of each name) */
    double p10_ms, p50_ms, p90_ms;
} ep_trace_stat;

/* While enabled, every kernel launch of the library is bracketed by HIP timing events on
 * the stream it runs on (the launch's own start and stop events), and the host's partial
 * reductions are timed on the host.  DMA copies are not bracketed: timing events around
 * an SDMA copy misreport its span (it can exceed the span of the call that holds it); the
 * flag-wait kernels after a leg (wait_d2h, ...) span the copies they wait for. */
ep_status ep_trace_enable(int32_t on);
/* Synchronizes the pending events and returns per-name totals (up to `capacity`). */
ep_status ep_trace_read(ep_trace_stat *stats, int32_t capacity, int32_t *count);
ep_status ep_trace_reset(void);

/* A plain streaming copy kernel (16-byte vectors): the attainable-bandwidth probe and
 * the calibration for hardware byte counters.  bytes must be a multiple of 16. */
ep_status ep_copy_probe(void *dst_dev, const void *src_dev, size_t bytes, hipStream_t stream);

/* Streaming probe of one read:write mix, over sequential addresses: `units` units, each
 * reading `reads` rows of row_bytes (unit u: src rows [u*reads, (u+1)*reads)) and writing
 * `writes` rows (dst rows [u*writes, (u+1)*writes)), every written row the XOR of the rows
 * read.  1:k has the traffic of the dispatch's pack, k:1 that of the combine, 1:0 is
 * read-only, 0:1 write-only: what plain streaming code attains, beside which the path's
 * kernels are judged.  row_bytes = 1024 * g, g in {1, 2, 4, 8, 14, 16}; reads, writes in
 * 0..64, not both 0.  src: units*reads*row_bytes bytes (may be NULL when reads == 0);
 * dst: units*writes*row_bytes bytes, or 1 KiB when writes == 0.  store_policy (the path's
 * three): 0 non-temporal 16-byte stores, 1 device-scope write-through buffer stores (the
 * combine below 128 MiB of output), 2 the same with the non-temporal hint (the pack from
 * 2 GiB per launch); any other value is EP_ERR_INVALID_ARG.  Traced as "stream_probe". */
ep_status ep_stream_probe(void *dst_dev, const void *src_dev, int64_t units, int32_t row_bytes, int32_t reads,
                          int32_t writes, int32_t store_policy, hipStream_t stream);

/* PCIe probe on the SDMA engines the exchange uses: `dirs` bit 0 moves `bytes`
 * device->host (dev -> host), bit 1 host->device (host + bytes -> dev + bytes), both
 * bits at once on two engines.  host: pinned, dev: device, 2*bytes each.  Blocks; runs the
 * copies five times (the first warms the engines) and writes the best host-timed aggregate
 * rate of the other four in GB/s (1e9 B/s) to *gbps. */
ep_status ep_pcie_probe(void *host, void *dev, size_t bytes, int32_t dirs, double *gbps);

/* hipMemcpyAsync(kind = default) passthrough for bindings that hold raw pointers. */
ep_status ep_memcpy(void *dst, const void *src, size_t bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* EP_H */
