// layout.hip -- dispatch layout for gfx950: a stable counting sort of the T*k routing
// entries by expert id (rows grouped by expert, token order kept inside a group, groups
// in expert order, hence contiguous per destination rank).  Sec. 4.3 of the paper groups
// tokens by the experts that consume them; Sec. 4.5 sends each destination only its rows.
//
// Work split: the routing array is cut into tiles, one workgroup per tile, W waves per
// workgroup, each wave owning a contiguous run of kLayoutRounds x 64 entries.  W is 16
// (1024 lanes) when the per-wave counters of E experts fit in LDS next to each other,
// else 4, so that a tile's entries are ranked by many waves at once while each wave
// walks only a few rounds.
//  * Inside a wave, the lanes holding the same expert are found with ceil(log2 E) 64-lane
//    ballots ("match any"); a lane's rank among them is a masked popcount (mbcnt), and
//    one leader lane per distinct expert updates the wave's counter in LDS.  No atomics
//    decide any position, so the result is deterministic.
//  * Across waves and tiles, positions come from exclusive prefix sums: per-wave counts
//    in LDS (within the tile) and a per-tile histogram in the workspace (across tiles).
//  * Expert offsets are a workgroup-wide exclusive scan built on a DPP wave scan.
// One tile: a single kernel does everything.  Several tiles: a histogram kernel (tile
// totals and per-wave counts), then the ranking kernel (each workgroup re-reads the small
// [tiles][E] totals and its own per-wave counts instead of counting again).
#include "ep_internal.h"

namespace ep {
namespace {

// Mask of lanes whose `valid` is set and whose expert id equals this lane's.
__device__ __forceinline__ uint64_t match_expert(int e, bool valid, int nbits) {
    uint64_t m = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = (e >> b) & 1;
        const uint64_t bal = __ballot(bit);
        m &= bit ? bal : ~bal;
    }
    return m;
}

// Number of lanes of `m` below this lane.
__device__ __forceinline__ int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP row shifts and broadcasts.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15 -> rows 1,3
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31 -> rows 2,3
    return v;
}

// The routing ids of this wave's run, one register per round of 64 entries.
__device__ __forceinline__ void load_ids(const int32_t *__restrict__ idx, int64_t slots,
                                         int64_t run_begin, int lane, int (&ids)[kLayoutRounds]) {
#pragma unroll
    for (int r = 0; r < kLayoutRounds; ++r) {
        const int64_t i = run_begin + r * kWave + lane;
        ids[r] = i < slots ? idx[i] : -1;
    }
}

// Adds this wave's per-expert counts of its run to cnt[0..E) (LDS row owned by the wave).
__device__ __forceinline__ void wave_count(const int (&ids)[kLayoutRounds], int64_t slots,
                                           int64_t run_begin, int lane, int E, int nbits,
                                           int *cnt) {
#pragma unroll
    for (int r = 0; r < kLayoutRounds; ++r) {
        const int64_t round_begin = run_begin + r * kWave;
        if (round_begin >= slots)
            break;
        const int e = ids[r];
        const bool valid = round_begin + lane < slots && (unsigned)e < (unsigned)E;
        const uint64_t m = match_expert(e, valid, nbits);
        if (valid && lanes_below(m) == 0)
            cnt[e] += __popcll(m);
    }
}

template <int W>
__global__ __launch_bounds__(W * 64) void layout_histogram_kernel(LayoutArgs a) {
    constexpr int kThreads = W * kWave;
    extern __shared__ int lds[];  // [W][E]
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int E = a.E;
    const int64_t run_begin = (int64_t)blockIdx.x * layout_tile_slots(W) + (int64_t)w * kLayoutRounds * kWave;
    int ids[kLayoutRounds];
    load_ids(a.topk_idx, a.slots, run_begin, lane, ids);
    for (int i = tid; i < W * E; i += kThreads)
        lds[i] = 0;
    if (blockIdx.x == 0 && tid == 0)
        *a.status = 0u;  // the ranking kernel (next on the stream) records routing errors
    __syncthreads();
    wave_count(ids, a.slots, run_begin, lane, E, a.nbits, lds + w * E);
    __syncthreads();
    const int64_t tiles = gridDim.x;
    int32_t *tot = a.tile_hist + (int64_t)blockIdx.x * E;
    int32_t *per_wave = a.tile_hist + tiles * E + (int64_t)blockIdx.x * W * E;
    for (int e = tid; e < E; e += kThreads) {
        int s = 0;
#pragma unroll
        for (int v = 0; v < W; ++v) {
            const int c = lds[v * E + e];
            per_wave[v * E + e] = c;
            s += c;
        }
        tot[e] = s;
    }
}

template <int W>
__global__ __launch_bounds__(W * 64) void layout_rank_kernel(LayoutArgs a, int32_t tiles) {
    constexpr int kThreads = W * kWave;
    extern __shared__ int lds[];
    const int E = a.E;
    int *wave_cnt = lds;            // [W][E]: counts, then running bases
    int *offs = wave_cnt + W * E;   // [E+1] exclusive expert offsets
    int *tot = offs + E + 1;        // [E] rows per expert over all tiles
    int *pre = tot + E;             // [E] rows per expert in earlier tiles
    int *wave_sum = pre + E;        // [W] scan carries
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int64_t tile = blockIdx.x;

    // every global read is issued up front: this wave's ids, the 64 ids before its run
    // (for the duplicate check), and with several tiles the histogram of the first pass
    const int64_t run_begin = tile * layout_tile_slots(W) + (int64_t)w * kLayoutRounds * kWave;
    int ids[kLayoutRounds];
    load_ids(a.topk_idx, a.slots, run_begin, lane, ids);
    const int64_t halo_i = run_begin - kWave + lane;
    const int halo = halo_i >= 0 && halo_i < a.slots ? a.topk_idx[halo_i] : -1;

    // 1-2. this wave's counts, per-expert totals and rows in earlier tiles
    if (tiles == 1) {
        for (int i = tid; i < W * E; i += kThreads)
            wave_cnt[i] = 0;
        if (tid == 0)
            *a.status = 0u;
        __syncthreads();
        wave_count(ids, a.slots, run_begin, lane, E, a.nbits, wave_cnt + w * E);
        __syncthreads();
        for (int e = tid; e < E; e += kThreads) {
            int t = 0;
#pragma unroll
            for (int v = 0; v < W; ++v)
                t += wave_cnt[v * E + e];
            tot[e] = t;
            pre[e] = 0;
        }
    } else {
        const int32_t *own = a.tile_hist + (int64_t)tiles * E + tile * W * E;
        for (int i = tid; i < W * E; i += kThreads)
            wave_cnt[i] = own[i];
        for (int e = tid; e < E; e += kThreads) {
            int t = 0, p = 0;
            // batches of 16 independent loads keep the histogram reads in flight together
            for (int64_t b0 = 0; b0 < tiles; b0 += 16) {
                int c[16];
#pragma unroll
                for (int q = 0; q < 16; ++q)
                    c[q] = b0 + q < tiles ? a.tile_hist[(b0 + q) * E + e] : 0;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    t += c[q];
                    p += b0 + q < tile ? c[q] : 0;
                }
            }
            tot[e] = t;
            pre[e] = p;
        }
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

    // 4. counts and offsets (first workgroup), and each wave's first row per expert
    if (blockIdx.x == 0) {
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

    // 5. positions: running base of the expert in this wave + rank among equal lanes.
    //    A token must name k different experts: each slot compares its id with the j
    //    earlier slots of its row, read from neighbouring lanes (this round, or the
    //    previous round / the 64 entries before the run for lanes near the front).
    int *wave_base = wave_cnt + w * E;
    bool bad_id = false, dup = false;
    // slot index within the token row, advanced by 64 mod k per round (no division per round)
    const int32_t step = kWave % a.k;
    int32_t jslot = (int32_t)((run_begin + lane) % a.k);
#pragma unroll
    for (int r = 0; r < kLayoutRounds; ++r) {
        const int64_t round_begin = run_begin + r * kWave;
        if (round_begin >= a.slots)
            break;
        const int64_t i = round_begin + lane;
        const bool in_range = i < a.slots;
        const int e = ids[r];
        const bool valid = in_range && (unsigned)e < (unsigned)E;
        const uint64_t m = match_expert(e, valid, a.nbits);
        const int32_t ii = (int32_t)i;
        if (r > 0) {
            jslot += step;
            jslot -= jslot >= a.k ? a.k : 0;
        }
        if (a.k <= kWave) {
            const int earlier_round = r == 0 ? halo : ids[r == 0 ? 0 : r - 1];
            for (int d = 1; d < a.k; ++d) {
                const int src = (lane - d) & (kWave - 1);
                const int same = __shfl(e, src);
                const int prev = __shfl(earlier_round, src);
                dup |= valid && d <= jslot && (lane >= d ? same : prev) == e;
            }
        } else if (valid) {
            const int32_t *row = a.topk_idx + (ii - jslot);
            for (int32_t jj = 0; jj < jslot; ++jj)
                dup |= row[jj] == e;
        }
        int pos = -1;
        if (valid) {
            const int below = lanes_below(m);
            const int b = wave_base[e];
            pos = b + below;
            if (below == 0)
                wave_base[e] = b + __popcll(m);
        }
        bad_id |= in_range && !valid;
        if (in_range) {
            a.slot_pos[i] = pos;
            if (valid && a.row_src)
                a.row_src[pos] = (int32_t)i;
        }
    }
    const uint32_t err = (__ballot(bad_id) ? kRoutingIdOutOfRange : 0u) |
                         (__ballot(dup) ? kRoutingDuplicate : 0u);
    if (err && lane == 0)
        atomicOr(a.status, err);
}

template <int W>
hipError_t launch_layout_w(const LayoutArgs &a, hipStream_t stream) {
    const int64_t tiles = std::max<int64_t>(1, layout_tiles(a.slots, a.E));
    const size_t rank_lds = sizeof(int) * ((size_t)W * a.E + (a.E + 1) + 2 * (size_t)a.E + W);
    if (tiles > 1) {
        (void)hipGetLastError();  // drop an error left by an earlier, already reported call
        TraceSlot ts = trace_acquire();
        hipExtLaunchKernelGGL(layout_histogram_kernel<W>, dim3((unsigned)tiles), dim3(W * kWave),
                              (uint32_t)(sizeof(int) * W * a.E), stream, ts.start, ts.stop, 0, a);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess)
            return err;
        trace_submit("layout_histogram", ts);
    }
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(layout_rank_kernel<W>, dim3((unsigned)tiles), dim3(W * kWave), (uint32_t)rank_lds,
                          stream, ts.start, ts.stop, 0, a, (int32_t)tiles);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("layout_rank", ts);
    return err;
}

}  // namespace

hipError_t launch_layout(const LayoutArgs &a, hipStream_t stream) {
    return layout_waves(a.E) == 16 ? launch_layout_w<16>(a, stream) : launch_layout_w<4>(a, stream);
}

}  // namespace ep
