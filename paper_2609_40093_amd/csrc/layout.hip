// layout.hip -- dispatch layout for gfx950: a stable counting sort of the T*k routing
// entries by expert id (rows grouped by expert, token order kept inside a group, groups
// in expert order, hence contiguous per destination rank).  Sec. 4.3 of the paper groups
// tokens by the experts that consume them; Sec. 4.5 sends each destination only its rows.
// The same kernels group only a window of experts (the receive side of the dense design,
// Sec. 4.2-4.3: a rank groups the tokens it gathered by the experts it owns); entries
// naming other experts get no row and are not errors.
//
// The routing array is cut into tiles of W waves x `rounds` rounds x 64 entries, one
// workgroup per tile.  Inside a wave, the lanes holding the same expert are found with
// ceil(log2 E) 64-lane ballots ("match any"); a lane's rank among them is a masked
// popcount (mbcnt).  One leader lane per distinct expert adds the group's size to the
// wave's counter row in LDS; every lane of the group reads the counter's old value first,
// so it learns its rank among the wave's earlier entries of that expert at the same time.
// No atomic decides any position: the result is deterministic.
//
// One tile (few entries): one kernel counts, scans the expert totals (a DPP wave scan with
// LDS carries) and writes every position.
// Several tiles: two kernels, and no workgroup ever waits for another (so nothing depends
// on which workgroups the device runs at once):
//   count  each tile counts its entries per expert, checks the routing (ids outside [0,E),
//          an expert twice in one token row) and stores its counts and error bits in the
//          workspace.
//   rank   each tile reads every tile's counts (a thread per run of tiles of an expert's
//          column, 16 loads in flight), which gives the expert totals and the rows of each
//          expert in earlier tiles; scans the totals; counts its own entries again (the
//          same ballots) and writes every position: expert offset + rows of the expert in
//          earlier tiles + in earlier waves + the entry's rank inside its wave.  Tile 0
//          also writes the counts, offsets and status.
// The kernel boundary orders the count kernel's stores before the rank kernel's loads: no
// fence, atomic or counter is involved, so a layout captured in a graph replays as it runs.
// Cross-tile traffic: tiles x E words written once, read by every rank workgroup (from L2
// after its XCD's first miss), and tiles error words read by tile 0.
#include "ep_internal.h"
#include "wave.h"

#include <mutex>

namespace ep {
namespace {

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

// Counting one round: returns the entry's rank among this wave's entries of its expert so
// far (-1 when it does not name a grouped expert) and bumps the wave's counter row.  With
// kCheck, also records routing errors in `err` (the rank pass of a multi-tile layout
// recounts without checking again).
template <bool kCheck>
__device__ __forceinline__ int count_entry(const LayoutArgs &a, int id, int earlier, int64_t i, int lane,
                                           int jslot, int *cnt, uint32_t &err) {
    const bool in_range = i < a.slots;
    const bool id_ok = in_range && (unsigned)id < (unsigned)a.all_E;
    const bool valid = id_ok && in_window(a, id);
    const int e = id - a.e_lo;
    const uint64_t m = match_expert(e, valid, a.nbits);
    if (kCheck) {
        if (in_range && !id_ok)
            err |= kRoutingIdOutOfRange;
        // duplicates are judged on the raw ids, also outside the window
        const uint64_t m_all = a.E == a.all_E ? m : match_expert(id, id_ok, a.all_nbits);
        if (repeats_in_row(a, id, id_ok, m_all, earlier, i, lane, jslot))
            err |= kRoutingDuplicate;
    }
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
    // whatever the workspace held
    if ((uint64_t)(uint32_t)pos >= (uint64_t)a.slots)
        pos = -1;
    a.slot_pos[i] = pos;
    if (pos >= 0 && a.row_src)
        a.row_src[pos] = (int32_t)i;
}

// Counts the tile's entries into the per-wave counter rows wave_cnt [W][E] (zeroed by the
// caller); with kCheck also ORs routing errors into flags[0].  Cached runs keep each
// entry's in-wave rank in rank[] for the positions.
template <int W, bool kCheck>
__device__ void count_tile(const LayoutArgs &a, int64_t run_begin, int rounds, int lane, int *wave_cnt, int w,
                           int *flags, const int (&ids)[kLayoutRankCache], int halo, int (&rank)[kLayoutRankCache]) {
    int *cnt = wave_cnt + w * a.E;
    uint32_t err = 0;
    const bool aligned = kWave % a.k == 0;
    const int32_t step = kWave % a.k;
    int32_t jslot = aligned ? lane % a.k : (int32_t)((run_begin + lane) % a.k);
    if (rounds <= kLayoutRankCache) {
#pragma unroll
        for (int r = 0; r < kLayoutRankCache; ++r) {
            const int64_t round_begin = run_begin + r * kWave;
            if (r >= rounds || round_begin >= a.slots)
                break;
            if (r > 0 && step) {
                jslot += step;
                jslot -= jslot >= a.k ? a.k : 0;
            }
            rank[r] = count_entry<kCheck>(a, ids[r], r == 0 ? halo : ids[r == 0 ? 0 : r - 1], round_begin + lane,
                                          lane, jslot, cnt, err);
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
            (void)count_entry<kCheck>(a, e, earlier, round_begin + lane, lane, jslot, cnt, err);
            earlier = e;
        }
    }
    if (kCheck) {
        const uint32_t wave_err = (__ballot(err & kRoutingIdOutOfRange) ? kRoutingIdOutOfRange : 0u) |
                                  (__ballot(err & kRoutingDuplicate) ? kRoutingDuplicate : 0u);
        if (wave_err && lane == 0)
            atomicOr(&flags[0], (int)wave_err);
    }
}

// Writes the tile's positions from base[W][E] (each wave's first row per expert) and the
// ranks kept by count_tile (cached runs) or found again (longer runs).
template <int W>
__device__ void write_tile(const LayoutArgs &a, int64_t run_begin, int rounds, int lane, int *base_rows,
                           const int (&ids)[kLayoutRankCache], const int (&rank)[kLayoutRankCache]) {
    int *base = base_rows;
    if (rounds <= kLayoutRankCache) {
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

// Exclusive scan of tot[0..E) into offs[0..E] (offs[E] = total) by the whole workgroup:
// each thread scans a contiguous run of experts, the runs' sums are scanned across it.
template <int W>
__device__ void scan_experts(int E, const int *tot, int *offs, int *wave_sum, int tid) {
    constexpr int kThreads = W * kWave;
    const int lane = tid & (kWave - 1), w = tid / kWave;
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
}

// Writes the expert counts and offsets, the rank counts and offsets, and the status.
template <int W>
__device__ void write_totals(const LayoutArgs &a, const int *tot, const int *offs, uint32_t status, int tid) {
    constexpr int kThreads = W * kWave;
    const int E = a.E;
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
        *a.status = status;
    }
}

enum LayoutPass { kWhole = 0, kCountPass = 1, kRankPass = 2 };
constexpr int kLastBatch = 16;  // tile counts a thread loads at once

// LDS of every pass: wave_cnt [W][E], offs [E+1], tot [E], pre [E], wave_sum [W], flags [4],
// part and part_pre [W*64] (partial column sums of the rank pass).
template <int W>
constexpr size_t layout_lds_ints(int E) {
    return (size_t)W * E + (E + 1) + 2 * E + W + 4 + 2 * W * kWave;
}

// Rank pass: every tile's counts, summed per expert into tot[e] (all tiles) and pre[e]
// (tiles before `tile`).  Column e's tiles are split into `groups` runs, one thread per
// (run, column); the runs' sums meet in LDS.  Tile 0 also ORs every tile's error bits into
// flags[0].  Ends with the workgroup synchronised.
template <int W>
__device__ void sum_tile_counts(const LayoutArgs &a, int tiles, int tile, int tid, int *tot, int *pre, int *part,
                                int *part_pre, int *flags) {
    constexpr int kThreads = W * kWave;
    const int E = a.E;
    const int groups = E < kThreads ? kThreads / E : 1;
    const int per = (tiles + groups - 1) / groups;
    for (int q = tid; q < groups * E; q += kThreads) {
        const int g = q / E, e = q - g * E;
        const int t_end = min(tiles, (g + 1) * per);
        int s = 0, b = 0;
        for (int t0 = g * per; t0 < t_end; t0 += kLastBatch) {
            int held[kLastBatch];
#pragma unroll
            for (int u = 0; u < kLastBatch; ++u)  // kLastBatch loads in flight
                held[u] = t0 + u < t_end ? a.tile_counts[(int64_t)(t0 + u) * E + e] : 0;
#pragma unroll
            for (int u = 0; u < kLastBatch; ++u) {
                s += held[u];
                b += t0 + u < tile ? held[u] : 0;
            }
        }
        if (groups > 1) {
            part[q] = s;
            part_pre[q] = b;
        } else {
            tot[e] = s;
            pre[e] = b;
        }
    }
    if (tile == 0) {
        uint32_t err_bits = 0;
        for (int t = tid; t < tiles; t += kThreads)
            err_bits |= a.tile_errs[t];
        if (err_bits)
            atomicOr(&flags[0], (int)err_bits);
    }
    __syncthreads();
    if (groups > 1) {
        for (int e = tid; e < E; e += kThreads) {
            int s = 0, b = 0;
            for (int g = 0; g < groups; ++g) {
                s += part[g * E + e];
                b += part_pre[g * E + e];
            }
            tot[e] = s;
            pre[e] = b;
        }
        __syncthreads();
    }
}

template <int W, int kPass>
__global__ __launch_bounds__(W * 64) void layout_kernel(LayoutArgs a, int32_t rounds, int32_t tiles) {
    constexpr int kThreads = W * kWave;
    extern __shared__ int lds[];
    const int E = a.E;
    int *wave_cnt = lds;            // [W][E]: per-wave counts, then per-wave first rows
    int *offs = wave_cnt + W * E;   // [E+1] exclusive expert offsets
    int *tot = offs + E + 1;        // [E] rows per expert
    int *pre = tot + E;             // [E] rows per expert in earlier tiles (rank pass)
    int *wave_sum = pre + E;        // [W] scan carries
    int *flags = wave_sum + W;      // [0] error bits
    int *part = flags + 4;          // [kThreads]
    int *part_pre = part + kThreads;  // [kThreads]
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int tile = blockIdx.x;
    const int64_t run_begin = ((int64_t)tile * W + w) * rounds * kWave;

    // every global read is issued up front: this wave's ids (cached runs) and the 64 ids
    // before its run (rows that straddle rounds)
    int ids[kLayoutRankCache], rank[kLayoutRankCache];
    if (rounds <= kLayoutRankCache) {
#pragma unroll
        for (int r = 0; r < kLayoutRankCache; ++r) {
            const int64_t i = run_begin + r * kWave + lane;
            ids[r] = r < rounds && i < a.slots ? a.topk_idx[i] : -1;
        }
    }
    int halo = -1;
    if (kPass != kRankPass && kWave % a.k != 0) {
        const int64_t h = run_begin - kWave + lane;
        halo = h >= 0 && h < a.slots ? a.topk_idx[h] : -1;
    }
    for (int i = tid; i < W * E; i += kThreads)
        wave_cnt[i] = 0;
    if (tid < 4)
        flags[tid] = 0;
    __syncthreads();

    if (kPass == kRankPass) {
        sum_tile_counts<W>(a, tiles, tile, tid, tot, pre, part, part_pre, flags);
        scan_experts<W>(E, tot, offs, wave_sum, tid);
        if (tile == 0)
            write_totals<W>(a, tot, offs, (uint32_t)flags[0], tid);
    }

    count_tile<W, kPass != kRankPass>(a, run_begin, rounds, lane, wave_cnt, w, flags, ids, halo, rank);
    __syncthreads();

    if (kPass == kCountPass) {
        // this tile's counts and error bits, for the rank kernel
        if (w == 0) {
            int32_t *counts = a.tile_counts + (int64_t)tile * E;
            for (int e = lane; e < E; e += kWave) {
                int s = 0;
#pragma unroll
                for (int v = 0; v < W; ++v)
                    s += wave_cnt[v * E + e];
                counts[e] = s;
            }
            if (lane == 0)
                a.tile_errs[tile] = (uint32_t)flags[0];
        }
        return;
    }

    // each wave's first row per expert
    if (kPass == kWhole) {
        for (int e = tid; e < E; e += kThreads) {
            int s = 0;
#pragma unroll
            for (int v = 0; v < W; ++v)
                s += wave_cnt[v * E + e];
            tot[e] = s;
        }
        __syncthreads();
        scan_experts<W>(E, tot, offs, wave_sum, tid);
        write_totals<W>(a, tot, offs, (uint32_t)flags[0], tid);
    }
    for (int e = tid; e < E; e += kThreads) {
        int base = kPass == kRankPass ? offs[e] + pre[e] : offs[e];
#pragma unroll
        for (int v = 0; v < W; ++v) {
            const int c = wave_cnt[v * E + e];
            wave_cnt[v * E + e] = base;
            base += c;
        }
    }
    __syncthreads();
    write_tile<W>(a, run_begin, rounds, lane, wave_cnt + w * E, ids, rank);
}

template <int W>
hipError_t launch_layout_w(const LayoutArgs &a, const LayoutGeom &g, hipStream_t stream) {
    const size_t lds = sizeof(int) * layout_lds_ints<W>(a.E);
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    const dim3 grid((unsigned)g.tiles), block(W * kWave);
    TraceSlot ts = trace_acquire();
    if (g.tiles == 1) {
        hipExtLaunchKernelGGL((layout_kernel<W, kWhole>), grid, block, (uint32_t)lds, stream, ts.start, ts.stop, 0, a,
                              (int32_t)g.rounds, (int32_t)g.tiles);
    } else {
        // both kernels inside one pair of timing events: the layout's time
        hipExtLaunchKernelGGL((layout_kernel<W, kCountPass>), grid, block, (uint32_t)lds, stream, ts.start, nullptr,
                              0, a, (int32_t)g.rounds, (int32_t)g.tiles);
        hipExtLaunchKernelGGL((layout_kernel<W, kRankPass>), grid, block, (uint32_t)lds, stream, nullptr, ts.stop, 0,
                              a, (int32_t)g.rounds, (int32_t)g.tiles);
    }
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("layout", ts);
    return err;
}

}  // namespace

hipError_t launch_layout(LayoutArgs a, hipStream_t stream) {
    const LayoutGeom g = layout_geometry(a.slots, a.E);
    return g.waves == 16 ? launch_layout_w<16>(a, g, stream) : launch_layout_w<4>(a, g, stream);
}

}  // namespace ep
