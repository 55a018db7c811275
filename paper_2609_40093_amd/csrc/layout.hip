// layout.hip -- dispatch layout for gfx950: a stable counting sort of the T*k routing
// entries by expert id (rows grouped by expert, token order kept inside a group, groups
// in expert order, hence contiguous per destination rank).  Sec. 4.3 of the paper groups
// tokens by the experts that consume them; Sec. 4.5 sends each destination only its rows.
//
// Work split: the routing array is cut into tiles of kTileSlots entries, one workgroup
// per tile, 4 waves per workgroup, each wave owning a contiguous run of the tile.
//  * Inside a wave, the lanes holding the same expert are found with ceil(log2 E) 64-lane
//    ballots ("match any"); a lane's rank among them is a masked popcount (mbcnt), and
//    one leader lane per distinct expert updates the wave's counter in LDS.  No atomics
//    decide any position, so the result is deterministic.
//  * Across waves and tiles, positions come from exclusive prefix sums: per-wave counts
//    in LDS (within the tile) and a per-tile histogram in the workspace (across tiles).
//  * Expert offsets are a workgroup-wide exclusive scan built on a DPP wave scan.
// One tile: a single kernel does everything.  Several tiles: a histogram kernel, then
// the ranking kernel (each workgroup re-reads the small [tiles][E] histogram).
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
                                         int64_t run_begin, int lane, int (&ids)[kRoundsPerWave]) {
#pragma unroll
    for (int r = 0; r < kRoundsPerWave; ++r) {
        const int64_t i = run_begin + r * kWave + lane;
        ids[r] = i < slots ? idx[i] : -1;
    }
}

// Adds this wave's per-expert counts of its run to cnt[0..E) (LDS row owned by the wave).
__device__ __forceinline__ void wave_count(const int (&ids)[kRoundsPerWave], int64_t slots,
                                           int64_t run_begin, int lane, int E, int nbits,
                                           int *cnt) {
#pragma unroll
    for (int r = 0; r < kRoundsPerWave; ++r) {
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

__global__ __launch_bounds__(kLayoutThreads) void layout_histogram_kernel(LayoutArgs a) {
    extern __shared__ int lds[];  // [waves][E]
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int E = a.E;
    for (int i = tid; i < kLayoutWaves * E; i += kLayoutThreads)
        lds[i] = 0;
    if (blockIdx.x == 0 && tid == 0)
        *a.status = 0u;  // the ranking kernel (next on the stream) records routing errors
    __syncthreads();
    const int64_t run_begin = (int64_t)blockIdx.x * kTileSlots + (int64_t)w * kSlotsPerWave;
    int ids[kRoundsPerWave];
    load_ids(a.topk_idx, a.slots, run_begin, lane, ids);
    wave_count(ids, a.slots, run_begin, lane, E, a.nbits, lds + w * E);
    __syncthreads();
    int32_t *hist = a.tile_hist + (int64_t)blockIdx.x * E;
    for (int e = tid; e < E; e += kLayoutThreads) {
        int s = 0;
#pragma unroll
        for (int v = 0; v < kLayoutWaves; ++v)
            s += lds[v * E + e];
        hist[e] = s;
    }
}

__global__ __launch_bounds__(kLayoutThreads) void layout_rank_kernel(LayoutArgs a, int32_t tiles) {
    extern __shared__ int lds[];
    const int E = a.E;
    int *wave_cnt = lds;                        // [waves][E]: counts, then running bases
    int *offs = wave_cnt + kLayoutWaves * E;    // [E+1] exclusive expert offsets
    int *tot = offs + E + 1;                    // [E] rows per expert over all tiles
    int *pre = tot + E;                         // [E] rows per expert in earlier tiles
    int *wave_sum = pre + E;                    // [waves] scan carries
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int64_t tile = blockIdx.x;

    for (int i = tid; i < kLayoutWaves * E; i += kLayoutThreads)
        wave_cnt[i] = 0;
    if (tiles == 1 && tid == 0)
        *a.status = 0u;
    __syncthreads();

    // 1. this wave's counts
    const int64_t run_begin = tile * kTileSlots + (int64_t)w * kSlotsPerWave;
    int ids[kRoundsPerWave];
    load_ids(a.topk_idx, a.slots, run_begin, lane, ids);
    wave_count(ids, a.slots, run_begin, lane, E, a.nbits, wave_cnt + w * E);
    __syncthreads();

    // 2. per-expert totals and rows in earlier tiles
    for (int e = tid; e < E; e += kLayoutThreads) {
        int t = 0, p = 0;
        if (tiles == 1) {
#pragma unroll
            for (int v = 0; v < kLayoutWaves; ++v)
                t += wave_cnt[v * E + e];
        } else {
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
        }
        tot[e] = t;
        pre[e] = p;
    }
    __syncthreads();

    // 3. exclusive scan of tot over experts: each thread scans a contiguous run of
    //    experts, the runs' sums are scanned across the workgroup
    const int per = (E + kLayoutThreads - 1) / kLayoutThreads;
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
    for (int v = 0; v < kLayoutWaves; ++v) {
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
        for (int e = tid; e < E; e += kLayoutThreads) {
            a.expert_counts[e] = tot[e];
            a.expert_offsets[e] = offs[e];
        }
        const int L = E / a.R;
        for (int r = tid; r < a.R; r += kLayoutThreads) {
            a.rank_offsets[r] = offs[r * L];
            a.rank_counts[r] = offs[(r + 1) * L] - offs[r * L];
        }
        if (tid == 0) {
            a.expert_offsets[E] = offs[E];
            a.rank_offsets[a.R] = offs[E];
        }
    }
    for (int e = tid; e < E; e += kLayoutThreads) {
        int base = offs[e] + pre[e];
#pragma unroll
        for (int v = 0; v < kLayoutWaves; ++v) {
            const int c = wave_cnt[v * E + e];
            wave_cnt[v * E + e] = base;
            base += c;
        }
    }
    __syncthreads();

    // 5. positions: running base of the expert in this wave + rank among equal lanes
    int *wave_base = wave_cnt + w * E;
    bool bad_id = false, dup = false;
#pragma unroll
    for (int r = 0; r < kRoundsPerWave; ++r) {
        const int64_t round_begin = run_begin + r * kWave;
        if (round_begin >= a.slots)
            break;
        const int64_t i = round_begin + lane;
        const bool in_range = i < a.slots;
        const int e = ids[r];
        const bool valid = in_range && (unsigned)e < (unsigned)E;
        const uint64_t m = match_expert(e, valid, a.nbits);
        int pos = -1;
        if (valid) {
            const int below = lanes_below(m);
            const int b = wave_base[e];
            pos = b + below;
            if (below == 0)
                wave_base[e] = b + __popcll(m);
            // a token must name k different experts
            const int32_t ii = (int32_t)i;
            const int32_t t = ii / a.k;
            const int32_t *row = a.topk_idx + (int64_t)t * a.k;
            for (int32_t jj = 0; jj < ii - t * a.k; ++jj)
                dup |= row[jj] == e;
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

}  // namespace

hipError_t launch_layout(const LayoutArgs &a, hipStream_t stream) {
    const int64_t tiles = layout_tiles(a.slots) > 0 ? layout_tiles(a.slots) : 1;
    const size_t rank_lds = sizeof(int) * ((size_t)kLayoutWaves * a.E + (a.E + 1) + 2 * (size_t)a.E + kLayoutWaves);
    if (tiles > 1) {
        (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
        hipExtLaunchKernelGGL(layout_histogram_kernel, dim3((unsigned)tiles), dim3(kLayoutThreads),
                              (uint32_t)(sizeof(int) * kLayoutWaves * a.E), stream, ts.start, ts.stop, 0, a);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess)
            return err;
        trace_submit("layout_histogram", ts);
    }
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    hipExtLaunchKernelGGL(layout_rank_kernel, dim3((unsigned)tiles), dim3(kLayoutThreads),
                          (uint32_t)rank_lds, stream, ts.start, ts.stop, 0, a, (int32_t)tiles);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("layout_rank", ts);
    return err;
}

}  // namespace ep
