// layout.hip -- dispatch layout for gfx950: a stable counting sort of the T*k routing
// entries by expert id (rows grouped by expert, token order kept inside a group, groups
// in expert order, hence contiguous per destination rank).  Sec. 4.3 of the paper groups
// tokens by the experts that consume them; Sec. 4.5 sends each destination only its rows.
// The same kernel groups only a window of experts (the receive side of the dense design,
// Sec. 4.2-4.3: a rank groups the tokens it gathered by the experts it owns); entries
// naming other experts get no row and are not errors.
//
// One kernel, one workgroup per tile of the routing array, all workgroups resident at
// once.  A workgroup has W waves; each wave owns a contiguous run of `rounds` x 64 entries.
//  1. Count.  Inside a wave, the lanes holding the same expert are found with ceil(log2 E)
//     64-lane ballots ("match any"); a lane's rank among them is a masked popcount
//     (mbcnt).  One leader lane per distinct expert adds the group's size to the wave's
//     counter row in LDS; every lane of the group reads the counter's old value first, so
//     it learns its rank among the wave's earlier entries of that expert at the same
//     time.  Routing errors (ids outside [0,E), an expert twice in one token row) are
//     found here too.  No atomic decides any position: the result is deterministic.
//  2. Exchange (several tiles).  Each workgroup publishes its per-expert totals and error
//     bits as 64-bit words tagged with the call's epoch, then reads every tile's words,
//     waiting (bounded by the wall clock) until all carry this call's tag: the sum over
//     all tiles gives the expert totals, the sum over earlier tiles the rows of each
//     expert that precede this tile.  A tag travels with each value, so neither a reset
//     of the words nor an atomic counter is needed; the first workgroup advances the
//     epoch once it has seen every tile's words, i.e. once every workgroup has read it.
//  3. Expert offsets: a workgroup-wide exclusive scan built on a DPP wave scan.
//  4. Positions: expert offset + rows in earlier tiles + rows in earlier waves + the rank
//     kept from step 1 (read-only LDS lookups, no dependency between rounds).  Runs of
//     more than kLayoutRankCache rounds (very large inputs) rank a second time instead.
#include "ep_internal.h"
#include "wave.h"

#include <mutex>

namespace ep {
namespace {

__device__ __forceinline__ uint64_t load_word(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_word(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Does entry i (expert e, slot jslot of its token row) repeat an expert named by an
// earlier slot of the same row?  m: lanes of this round with the same valid expert;
// earlier: the ids of the 64 entries before this round (rows that straddle rounds).
// Every lane must call it (the shuffles read other lanes).
__device__ __forceinline__ bool repeats_in_row(const LayoutArgs &a, int e, bool valid, uint64_t m,
                                               int earlier, int64_t i, int lane, int jslot) {
    const int k = a.k;
    if (kWave % k == 0) {
        // rounds start at multiples of 64, so a row's k entries are k neighbouring lanes
        const uint64_t row = (k == kWave ? ~0ull : ((1ull << k) - 1)) << (lane - jslot);
        return valid && __popcll(m & row) > 1;
    }
    bool dup = false;
    if (k <= kWave) {
        for (int d = 1; d < k; ++d) {
            const int src = (lane - d) & (kWave - 1);
            const int same = __shfl(e, src);
            const int prev = __shfl(earlier, src);
            dup |= valid && d <= jslot && (lane >= d ? same : prev) == e;
        }
    } else if (valid) {
        const int32_t *row = a.topk_idx + (i - jslot);
        for (int jj = 0; jj < jslot; ++jj)
            dup |= row[jj] == e;
    }
    return dup;
}

// An id names one of the grouped experts when it falls in the window [e_lo, e_lo + E).
__device__ __forceinline__ bool in_window(const LayoutArgs &a, int id) {
    return (unsigned)(id - a.e_lo) < (unsigned)a.E;
}

// Step 1 for one round: returns the entry's rank among this wave's entries of its expert
// so far (-1 when it does not name a grouped expert) and bumps the wave's counter row.

__device__ __forceinline__ int count_entry(const LayoutArgs &a, int id, int earlier, int64_t i, int lane,
                                           int jslot, int *cnt, uint32_t &err) {
    const bool in_range = i < a.slots;
    const bool id_ok = in_range && (unsigned)id < (unsigned)a.all_E;
    const bool valid = id_ok && in_window(a, id);
    const int e = id - a.e_lo;
    const uint64_t m = match_expert(e, valid, a.nbits);
    if (in_range && !id_ok)
        err |= kRoutingIdOutOfRange;
    // duplicates are judged on the raw ids, also outside the window
    const uint64_t m_all = a.E == a.all_E ? m : match_expert(id, id_ok, a.all_nbits);
    if (repeats_in_row(a, id, id_ok, m_all, earlier, i, lane, jslot))
        err |= kRoutingDuplicate;
    int rank = -1;
    if (valid) {
        const int below = lanes_below(m);
        const int old = cnt[e];
        rank = old + below;
        if (below == 0)
            cnt[e] = old + (int)__popcll(m);
    }
    return rank;
}

__device__ __forceinline__ void write_position(const LayoutArgs &a, int64_t i, int pos) {
    // positions are < T*k by construction; the check keeps every store inside the arrays
    // even if a timed-out exchange left inconsistent totals
    if ((uint64_t)(uint32_t)pos >= (uint64_t)a.slots)
        pos = -1;
    a.slot_pos[i] = pos;
    if (pos >= 0 && a.row_src)
        a.row_src[pos] = (int32_t)i;
}

// Step 2: sums the words every tile published -- over all tiles into tot[e], over the
// tiles before `tile` into pre[e] -- and ORs their error bits into *err.  Each thread
// takes one column (expert, or the error column) and a strided share of the tiles, with
// 8 loads in flight.  Returns false if some word still lacked this call's tag after
// timeout_ticks of the wall clock.
template <int kThreads>
__device__ bool gather_tiles(const LayoutArgs &a, int tiles, int tile, uint32_t want, int *tot, int *pre,
                             int *err, int tid) {
    const int cols = a.E + 1;
    const int groups = kThreads / cols > 0 ? kThreads / cols : 1;
    const int64_t t_start = wall_clock64();
    bool ok = true;
    for (int q = tid; q < cols * groups; q += kThreads) {
        const int g = q / cols, c = q - g * cols;
        int all = 0, before = 0;
        for (int t0 = g; t0 < tiles; t0 += 8 * groups) {
            uint64_t v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int t = t0 + u * groups;
                v[u] = t < tiles ? load_word(a.tile_words + (int64_t)t * cols + c) : (uint64_t)want << 32;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int t = t0 + u * groups;
                while (ok && (uint32_t)(v[u] >> 32) != want) {
                    if (wall_clock64() - t_start > a.timeout_ticks) {
                        ok = false;
                    } else {
                        __builtin_amdgcn_s_sleep(2);
                        v[u] = load_word(a.tile_words + (int64_t)t * cols + c);
                    }
                }
                const int n = (int)(uint32_t)v[u];
                if (t < tiles) {
                    if (c < cols - 1) {
                        all += n;
                        before += t < tile ? n : 0;
                    } else {
                        all |= n;
                    }
                }
            }
        }
        if (c < cols - 1) {
            atomicAdd(&tot[c], all);
            atomicAdd(&pre[c], before);
        } else {
            atomicOr(err, all);
        }
    }
    return ok;
}

template <int W>
__global__ __launch_bounds__(W * 64) void layout_kernel(LayoutArgs a, int32_t rounds, int32_t tiles) {
    constexpr int kThreads = W * kWave;
    extern __shared__ int lds[];
    const int E = a.E;
    int *wave_cnt = lds;            // [W][E]: per-wave counts, then per-wave first rows
    int *offs = wave_cnt + W * E;   // [E+1] exclusive expert offsets
    int *tot = offs + E + 1;        // [E] rows per expert over all tiles
    int *pre = tot + E;             // [E] rows per expert in earlier tiles
    int *wave_sum = pre + E;        // [W] scan carries
    int *flags = wave_sum + W;      // [0] this tile's error bits [1] all tiles' [2] timed out
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int tile = blockIdx.x;
    const int64_t run_begin = ((int64_t)tile * W + w) * rounds * kWave;
    const bool cached = rounds <= kLayoutRankCache;

    // every global read is issued up front: this wave's ids (cached runs), the 64 ids
    // before its run (rows that straddle rounds), the epoch of the workspace
    int ids[kLayoutRankCache];
    if (cached) {
#pragma unroll
        for (int r = 0; r < kLayoutRankCache; ++r) {
            const int64_t i = run_begin + r * kWave + lane;
            ids[r] = r < rounds && i < a.slots ? a.topk_idx[i] : -1;
        }
    }
    const bool aligned = kWave % a.k == 0;
    int halo = -1;
    if (!aligned) {
        const int64_t h = run_begin - kWave + lane;
        halo = h >= 0 && h < a.slots ? a.topk_idx[h] : -1;
    }
    const uint32_t want = tiles > 1 ? __hip_atomic_load(a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u : 0u;

    for (int i = tid; i < W * E; i += kThreads)
        wave_cnt[i] = 0;
    for (int i = tid; i < 2 * E; i += kThreads)
        tot[i] = 0;  // tot and pre
    if (tid < 3)
        flags[tid] = 0;
    __syncthreads();

    // 1. count, rank within the wave, routing errors
    int *cnt = wave_cnt + w * E;
    uint32_t err = 0;
    const int32_t step = kWave % a.k;
    int32_t jslot = aligned ? lane % a.k : (int32_t)((run_begin + lane) % a.k);
    int rank[kLayoutRankCache];
    if (cached) {
#pragma unroll
        for (int r = 0; r < kLayoutRankCache; ++r) {
            const int64_t round_begin = run_begin + r * kWave;
            if (r >= rounds || round_begin >= a.slots)
                break;
            if (r > 0 && step) {
                jslot += step;
                jslot -= jslot >= a.k ? a.k : 0;
            }
            rank[r] = count_entry(a, ids[r], r == 0 ? halo : ids[r == 0 ? 0 : r - 1], round_begin + lane, lane,
                                  jslot, cnt, err);
        }
    } else {
        int earlier = halo;
        int next = run_begin + lane < a.slots ? a.topk_idx[run_begin + lane] : -1;
        for (int r = 0; r < rounds; ++r) {
            const int64_t round_begin = run_begin + (int64_t)r * kWave;
            if (round_begin >= a.slots)
                break;
            const int e = next;
            const int64_t ni = round_begin + kWave + lane;
            next = r + 1 < rounds && ni < a.slots ? a.topk_idx[ni] : -1;
            if (r > 0 && step) {
                jslot += step;
                jslot -= jslot >= a.k ? a.k : 0;
            }
            (void)count_entry(a, e, earlier, round_begin + lane, lane, jslot, cnt, err);
            earlier = e;
        }
    }
    const uint32_t wave_err = (__ballot(err & kRoutingIdOutOfRange) ? kRoutingIdOutOfRange : 0u) |
                              (__ballot(err & kRoutingDuplicate) ? kRoutingDuplicate : 0u);
    if (wave_err && lane == 0)
        atomicOr(&flags[0], (int)wave_err);
    __syncthreads();

    // 2. tile totals; with several tiles, publish them and read everyone's
    for (int e = tid; e < E; e += kThreads) {
        int s = 0;
#pragma unroll
        for (int v = 0; v < W; ++v)
            s += wave_cnt[v * E + e];
        if (tiles > 1)
            store_word(a.tile_words + (int64_t)tile * (E + 1) + e, (uint64_t)want << 32 | (uint32_t)s);
        else
            tot[e] = s;
    }
    bool timed_out = false;
    if (tiles > 1) {
        if (tid == 0)
            store_word(a.tile_words + (int64_t)tile * (E + 1) + E, (uint64_t)want << 32 | (uint32_t)flags[0]);
        if (!gather_tiles<kThreads>(a, tiles, tile, want, tot, pre, &flags[1], tid))
            flags[2] = 1;
        __syncthreads();
        timed_out = flags[2] != 0;
    } else if (tid == 0) {
        flags[1] = flags[0];
    }
    if (timed_out) {
        // the totals are incomplete: report it, and give this tile's entries no row
        if (tid == 0)
            __hip_atomic_fetch_or(a.timed_out, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int64_t i = run_begin + lane, end = run_begin + (int64_t)rounds * kWave; i < end && i < a.slots;
             i += kWave)
            a.slot_pos[i] = -1;
        return;
    }
    __syncthreads();

    // 3. exclusive scan of tot over experts: each thread scans a contiguous run of
    //    experts, the runs' sums are scanned across the workgroup
    const int per = (E + kThreads - 1) / kThreads;
    const int first = tid * per;
    int s = 0;
    for (int c = 0; c < per; ++c)
        if (first + c < E)
            s += tot[first + c];
    const int incl = wave_inclusive_scan(s);
    if (lane == kWave - 1)
        wave_sum[w] = incl;
    __syncthreads();
    int carry = 0, total = 0;
#pragma unroll
    for (int v = 0; v < W; ++v) {
        carry += v < w ? wave_sum[v] : 0;
        total += wave_sum[v];
    }
    int run = carry + incl - s;
    for (int c = 0; c < per; ++c)
        if (first + c < E) {
            offs[first + c] = run;
            run += tot[first + c];
        }
    if (tid == 0)
        offs[E] = total;
    __syncthreads();

    // counts, offsets and status (first workgroup), and each wave's first row per expert
    if (tile == 0) {
        for (int e = tid; e < E; e += kThreads) {
            a.expert_counts[e] = tot[e];
            a.expert_offsets[e] = offs[e];
        }
        const int L = E / a.R;
        for (int r = tid; r < a.R; r += kThreads) {
            a.rank_offsets[r] = offs[r * L];
            a.rank_counts[r] = offs[(r + 1) * L] - offs[r * L];
        }
        if (tid == 0) {
            a.expert_offsets[E] = offs[E];
            a.rank_offsets[a.R] = offs[E];
            *a.status = (uint32_t)flags[1];
            if (tiles > 1)  // every workgroup has read the epoch: it published this call's tag
                __hip_atomic_store(a.epoch, want, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    for (int e = tid; e < E; e += kThreads) {
        int base = offs[e] + pre[e];
#pragma unroll
        for (int v = 0; v < W; ++v) {
            const int c = wave_cnt[v * E + e];
            wave_cnt[v * E + e] = base;
            base += c;
        }
    }
    __syncthreads();

    // 4. positions
    int *base = wave_cnt + w * E;
    if (cached) {
#pragma unroll
        for (int r = 0; r < kLayoutRankCache; ++r) {
            const int64_t round_begin = run_begin + r * kWave;
            if (r >= rounds || round_begin >= a.slots)
                break;
            const int64_t i = round_begin + lane;
            if (i < a.slots)
                write_position(a, i, rank[r] >= 0 ? base[ids[r] - a.e_lo] + rank[r] : -1);
        }
    } else {
        for (int r = 0; r < rounds; ++r) {
            const int64_t round_begin = run_begin + (int64_t)r * kWave;
            if (round_begin >= a.slots)
                break;
            const int64_t i = round_begin + lane;
            const bool in_range = i < a.slots;
            const int id = in_range ? a.topk_idx[i] : -1;
            const bool valid = in_range && (unsigned)id < (unsigned)a.all_E && in_window(a, id);
            const int e = id - a.e_lo;
            const uint64_t m = match_expert(e, valid, a.nbits);
            int pos = -1;
            if (valid) {
                const int below = lanes_below(m);
                const int b = base[e];
                pos = b + below;
                if (below == 0)
                    base[e] = b + (int)__popcll(m);
            }
            if (in_range)
                write_position(a, i, pos);
        }
    }
}

// Compute units and wall-clock rate of a device, read once.
struct DeviceInfo {
    int cus = 0;
    int64_t wall_khz = 0;
};
DeviceInfo device_info(int dev) {
    static std::mutex mu;
    static DeviceInfo cache[64];
    std::lock_guard<std::mutex> lock(mu);
    if (dev < 0 || dev >= 64)
        return {};
    DeviceInfo &d = cache[dev];
    if (d.cus == 0) {
        int cus = 0, khz = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
            return {};
        d.cus = cus;
        d.wall_khz = khz > 0 ? khz : 100000;
    }
    return d;
}

template <int W>
hipError_t launch_layout_w(LayoutArgs a, const LayoutGeom &g, hipStream_t stream) {
    const size_t lds = sizeof(int) * ((size_t)W * a.E + (a.E + 1) + 2 * (size_t)a.E + W + 3);
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(layout_kernel<W>, dim3((unsigned)g.tiles), dim3(W * kWave), (uint32_t)lds, stream,
                          ts.start, ts.stop, 0, a, (int32_t)g.rounds, (int32_t)g.tiles);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("layout", ts);
    return err;
}

}  // namespace

hipError_t launch_layout(LayoutArgs a, hipStream_t stream) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess)
        return err;
    const DeviceInfo info = device_info(dev);
    if (info.cus <= 0)
        return hipErrorInvalidDevice;
    // one workgroup per compute unit at most: all of them fit on the device at once
    const LayoutGeom g = layout_geometry(a.slots, a.E, std::min<int64_t>(kLayoutMaxTiles, info.cus));
    a.timeout_ticks = info.wall_khz * 1000;  // one second
    return g.waves == 16 ? launch_layout_w<16>(a, g, stream) : launch_layout_w<4>(a, g, stream);
}

}  // namespace ep
