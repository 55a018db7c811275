// fused.hip -- dispatch layout and pack in one kernel, for small expert counts.
//
// The layout (a stable counting sort of the T*k routing entries by expert, Sec. 4.3 of
// the paper) and the pack (each destination's rows gathered into one contiguous segment,
// Sec. 2.2) otherwise run as two kernels, and the layout's workgroups exchange their
// per-expert totals through memory.  With few experts every workgroup can afford to count
// all entries itself; that removes the exchange and the kernel boundary between layout
// and pack.  A workgroup of W waves owns W*tpw consecutive tokens (a run of tpw per
// wave); W is 4, 8 or 16 by the number of routing entries (each workgroup counts all of
// them, so fewer, larger workgroups for more entries; more, smaller ones for few -- less
// of the kernel waits on its last workgroups).  Below 1024 tokens a row is split over S
// waves instead (each moves 1/S of it; W = m*S for m tokens, one per S waves), so that
// the stores of few tokens still reach every compute unit:
//   A. each wave issues the loads of its first ids, then those of its first token row
//      (they do not depend on the layout; vector loads complete in order, so the ids
//      come first);
//   B. the workgroup counts all T*k entries (16-byte loads of 4 ids) with LDS atomic
//      adds into 16 copies of the per-expert counters, chosen by lane, so that lanes of
//      one instruction naming the same expert rarely hit the same word (vector and LDS
//      work only: a ballot per id would queue every wave of the compute unit on its one
//      scalar unit), both over all entries and over the entries before its own range;
//      routing errors (an id outside [0,E), an expert twice in one token row) are found
//      in the same pass (a top-8 row spans the 4-id groups of two neighbouring lanes);
//   C. the totals' exclusive scan (DPP; a lane per expert, or four consecutive experts
//      per lane above 64 experts) gives the expert offsets; workgroup 0 stores the
//      counts, offsets, rank counts/offsets and the status word;
//   D. wave 0 ranks the workgroup's own entries in flat order (ballot match-any and a
//      masked popcount, as the layout kernel does: stable), stores slot_pos / row_src and
//      keeps the rows in LDS;
//   E. each wave stores its tokens' rows (or its part of one) to their k packed rows
//      (non-temporal; U groups of 64 16-byte vectors, one per lane, all loads in flight
//      together).
// The outputs equal those of the layout kernel followed by the pack kernel, bit for bit.
// Workgroups never wait on each other, so nothing needs them resident together.
//
// Limits (the host falls back to the two kernels outside them): E <= 256 (four experts
// per lane in step C), k in {1, 2, 4, 8} (a token row inside one 4-id load, or two for
// top-8), T*k <= 65536 for E <= 64 and k <= 4, else T*k <= 16384 for rows up to 8 KiB and
// 8192 for longer ones (every workgroup reads and counts every id before its stores:
// beyond that the layout kernel's exchange of totals costs less), rows of 1, 2, 4, 8, 14
// or 16 groups (H = 512 * groups), a 16-byte aligned routing array.  The split runs of
// fewer than 1024 tokens keep the same limits.
#include "ep_internal.h"
#include "wave.h"

namespace ep {
namespace {

constexpr int kFMaxThreads = 16 * kWave;    // largest workgroup (16 waves)
constexpr int kFNarrowE = 64;                // experts with one lane each in step C
constexpr int kFMaxE = 4 * kWave;            // experts with four per lane (wide instances)
constexpr int64_t kFMaxSlots = 65536;        // T*k: every workgroup reads every id
// T*k for E > 64 or k = 8 (measured on MI355X: at 16384 ids the one kernel still wins
// with 4 KiB rows, 20-24 against 23-29 us, and loses with 14 KiB rows, 56 against 55 us)
constexpr int64_t kFMaxSlotsWide = 16384;    // rows of at most 8 KiB
constexpr int64_t kFMaxSlotsWideLong = 8192; // longer rows
constexpr int kFMaxOwn = 256;                // entries one workgroup owns (LDS rows)
constexpr int kFOwnRounds = kFMaxOwn / kWave;
constexpr int kFBatch = 4;                   // 16-byte id loads in flight per lane
constexpr int kFMaxWaves = 4096;             // waves in flight over the device (16 per CU)
constexpr int64_t kFSplitBelow = 1024;       // tokens below which rows are split over waves

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Does a token row inside a 4-id group name an expert twice?  Ids outside [0,E) are not
// compared (they are errors of their own).
template <int K>
__device__ __forceinline__ bool row_repeats(i32x4 v, int E) {
    auto ok = [E](int id) { return (unsigned)id < (unsigned)E; };
    if constexpr (K == 2)
        return (ok(v[0]) && v[0] == v[1]) || (ok(v[2]) && v[2] == v[3]);
    else if constexpr (K == 4)
        return (ok(v[0]) && (v[0] == v[1] || v[0] == v[2] || v[0] == v[3])) ||
               (ok(v[1]) && (v[1] == v[2] || v[1] == v[3])) || (ok(v[2]) && v[2] == v[3]);
    else
        return false;
}

// Loads the 4-id groups qw + b*threads + lane of a batch: every load is issued (an index
// past the last whole group rereads that group; the caller masks it by index), so the
// compiler can count the loads in flight and wait for the ids alone.
__device__ __forceinline__ void load_ids(const i32x4 *q, int64_t full, int64_t qw, int lane, int threads,
                                         i32x4 *v) {
#pragma unroll
    for (int b = 0; b < kFBatch; ++b)
        v[b] = q[min(qw + (int64_t)b * threads + lane, full - 1)];
}

constexpr int kFCopies = 16;  // copies of the LDS counters (lane % 16 picks one)

// Counts one id into the LDS counters (all entries, and those before this workgroup's);
// ME counters per copy.
template <int ME>
__device__ __forceinline__ void count_id(int id, bool in, bool before, int E, int *s_all, int *s_pre, int copy,
                                         bool &bad_id) {
    const bool valid = in && (unsigned)id < (unsigned)E;
    bad_id |= in && !valid;
    if (valid) {
        atomicAdd(&s_all[copy * ME + id], 1);
        if (before)
            atomicAdd(&s_pre[copy * ME + id], 1);
    }
}

// Does any id of `a` (in [0,E)) equal one of `b`?  (The two halves of a top-8 row.)
__device__ __forceinline__ bool halves_repeat(i32x4 a, i32x4 b, int E) {
    bool r = false;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        r |= (unsigned)a[i] < (unsigned)E && (a[i] == b[0] || a[i] == b[1] || a[i] == b[2] || a[i] == b[3]);
    return r;
}

// MULTI: more ids than one batch of the workgroup's loads (the count loops).  Instances
// without the loop have only straight-line loads, so the compiler's waits stay exact and
// no wave waits for its token row before the count's barrier.  WIDE: more than 64
// experts (four per lane in step C).  U: groups per wave (the row's, or 1/split of them).
template <int U, int K, bool MULTI, bool WIDE>
__global__ __launch_bounds__(kFMaxThreads) void layout_pack_kernel(FusedArgs a, int32_t tpw, int32_t split) {
    constexpr int ME = WIDE ? kFMaxE : kFNarrowE;  // counters per copy
    __shared__ int s_all[kFCopies * ME];
    __shared__ int s_pre[kFCopies * ME];
    __shared__ int s_base[ME];
    __shared__ int s_off[WIDE ? ME + 1 : 1];
    __shared__ int s_pos[kFMaxOwn];
    __shared__ int s_err;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int threads = blockDim.x, waves = threads / kWave;
    const int64_t slots = a.T * K;
    const int runs = waves / split;  // token runs of tpw tokens (split == 1: one per wave)
    const int64_t tok0 = (int64_t)blockIdx.x * runs * tpw;  // runs*tpw*K: a multiple of 4
    const int64_t tok1 = min(a.T, tok0 + (int64_t)runs * tpw);
    const int32_t col = (w % split) * U * kWave;  // this wave's first vector of a row
    const int64_t ent0 = tok0 * K, ent1 = tok1 * K;
    const int32_t V = a.H / 8;
    const u32x4 *x = static_cast<const u32x4 *>(a.x);
    const i32x4 *q = reinterpret_cast<const i32x4 *>(a.topk_idx);
    const int64_t full = slots / 4;  // whole 4-id groups; the 0..3 ids after them are the tail
    const int64_t stride = (int64_t)threads * kFBatch;

    // A. first ids, the own entries' ids (step D), then this wave's first token row (a
    //    wave past the workgroup's last token loads that token instead, storing nothing)
    i32x4 v[kFBatch];
    int64_t qw = (int64_t)w * kWave;
    if (full > 0)
        load_ids(q, full, qw, lane, threads, v);
    int own_id[kFOwnRounds];
#pragma unroll
    for (int r = 0; r < kFOwnRounds; ++r)
        own_id[r] = a.topk_idx[min(ent0 + r * kWave + lane, ent1 - 1)];  // masked by index in step D
    // the 0..3 ids after the whole 4-id groups (wave 0 counts them): loaded here, with the
    // rest, so that no load is left after the count (a load there would make every wave
    // wait for its token row before the count's barrier)
    const int64_t ti = full * 4 + lane;
    const int tail_id = a.topk_idx[min(ti, slots - 1)];
    const int tail_next = a.topk_idx[min(ti + 1, slots - 1)];
    const int64_t wtok = tok0 + (int64_t)(w / split) * tpw;
    u32x4 d[U];
    {
        const u32x4 *src = x + min(wtok, tok1 - 1) * V + col + lane;
#pragma unroll
        for (int u = 0; u < U; ++u)
            d[u] = __builtin_nontemporal_load(src + u * kWave);
    }
    for (int i = tid; i < kFCopies * ME; i += threads) {
        s_all[i] = 0;
        s_pre[i] = 0;
    }
    if (tid == 0)
        s_err = 0;
    __syncthreads();

    // B. count all entries into the LDS counters
    bool bad_id = false, dup = false;
    auto count_batch = [&](int64_t qb) {
#pragma unroll
        for (int b = 0; b < kFBatch; ++b) {
            const int64_t g = qb + (int64_t)b * threads;  // this round's first group
            if (g >= full)
                break;
            const int64_t qi = g + lane;
            const bool in = qi < full;
            // entries before this workgroup's: whole 4-id groups (ent0 is a multiple of 4)
            const bool before = qi * 4 < ent0;
            if constexpr (K == 8) {
                // a row is the groups of lanes 2m and 2m+1 (qi and lane have the same
                // parity; full = 2T is even, so both halves are in or out together)
                i32x4 o;
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    o[c] = __shfl_xor(v[b][c], 1);
                dup |= in && (row_repeats<4>(v[b], a.E) || ((lane & 1) == 0 && halves_repeat(v[b], o, a.E)));
            } else {
                dup |= in && row_repeats<K>(v[b], a.E);
            }
#pragma unroll
            for (int c = 0; c < 4; ++c)
                count_id<ME>(v[b][c], in, before, a.E, s_all, s_pre, lane % kFCopies, bad_id);
        }
    };
    // the first batch outside the loop: its wait leaves the token row's loads in flight
    if (qw < full)
        count_batch(qw);
    if (MULTI) {
        for (qw += stride; qw < full; qw += stride) {  // wave-uniform
            load_ids(q, full, qw, lane, threads, v);
            count_batch(qw);
        }
    }
    if (w == 0 && full * 4 < slots) {  // the tail: 1..3 ids (a whole token row for k <= 2)
        const bool in = ti < slots;
        const int id = in ? tail_id : -1;
        if (K == 2 && lane == 0)
            dup |= (unsigned)id < (unsigned)a.E && id == tail_next;  // the tail is one row
        count_id<ME>(id, in, ti < ent0, a.E, s_all, s_pre, lane % kFCopies, bad_id);
    }
    const uint32_t wave_err = (__ballot(bad_id) ? kRoutingIdOutOfRange : 0u) | (__ballot(dup) ? kRoutingDuplicate : 0u);
    if (lane == 0 && wave_err)
        atomicOr(&s_err, (int)wave_err);
    __syncthreads();

    if (w == 0 && WIDE) {
        // C (wide). Lane l holds experts 4l..4l+3: their totals, one scan of the lanes'
        // sums, the offsets of each expert kept in LDS (read back by other lanes of this
        // wave only, in program order)
        int tot[4], pre[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = 4 * lane + q;
            tot[q] = pre[q] = 0;
            if (e < a.E) {
#pragma unroll
                for (int c = 0; c < kFCopies; ++c) {
                    tot[q] += s_all[c * ME + e];
                    pre[q] += s_pre[c * ME + e];
                }
            }
            sum += tot[q];
        }
        const int incl = wave_inclusive_scan(sum);
        const int total = __shfl(incl, kWave - 1);
        int run = incl - sum;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = 4 * lane + q;
            if (e < a.E) {
                s_off[e] = run;
                s_base[e] = run + pre[q];
            }
            run += tot[q];
        }
        if (lane == 0)
            s_off[a.E] = total;
        __builtin_amdgcn_wave_barrier();  // the reads below follow every lane's writes
        if (blockIdx.x == 0) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (4 * lane + q < a.E)
                    a.expert_counts[4 * lane + q] = tot[q];
            const int L = a.E / a.R;
            for (int e = lane; e <= a.E; e += kWave)
                a.expert_offsets[e] = s_off[e];
            for (int r = lane; r <= a.R; r += kWave) {
                a.rank_offsets[r] = s_off[r * L];
                if (r < a.R)
                    a.rank_counts[r] = s_off[(r + 1) * L] - s_off[r * L];
            }
            if (lane == 0) {
                *a.status = (uint32_t)s_err;
                if (a.epoch_word)
                    *a.epoch_word = a.epoch;
            }
        }
    } else if (w == 0) {
        // C. totals, offsets; workgroup 0 stores the layout's counts and the status
        int tot = 0, pre = 0;
        if (lane < a.E) {
#pragma unroll
            for (int c = 0; c < kFCopies; ++c) {
                tot += s_all[c * ME + lane];
                pre += s_pre[c * ME + lane];
            }
        }
        const int incl = wave_inclusive_scan(tot);
        const int excl = incl - tot;
        const int total = __shfl(incl, kWave - 1);
        if (lane < a.E)
            s_base[lane] = excl + pre;
        if (blockIdx.x == 0) {
            if (lane < a.E)
                a.expert_counts[lane] = tot;
            if (lane <= a.E)  // lane E (< 64) holds the total too; E == 64 is stored below
                a.expert_offsets[lane] = excl;
            // rank r's first row: the exclusive offset of expert r*L (the total for r = R)
            const int L = a.E / a.R;
            auto offset_of = [&](int e) {
                const int v = __shfl(excl, min(e, kWave - 1));
                return e >= a.E ? total : v;
            };
            const int lo = offset_of(min(lane, a.R) * L);
            const int hi = offset_of(min(lane + 1, a.R) * L);
            if (lane < a.R)
                a.rank_counts[lane] = hi - lo;
            if (lane <= a.R)
                a.rank_offsets[lane] = lo;
            if (lane == 0) {
                if (a.E == kWave)
                    a.expert_offsets[kWave] = total;
                if (a.R == kWave)
                    a.rank_offsets[kWave] = total;
                *a.status = (uint32_t)s_err;
                if (a.epoch_word)
                    *a.epoch_word = a.epoch;
            }
        }
    }
    if (w == 0) {
        // D. rank the own entries in flat order (s_base as step C left it, written by this
        //    wave)
#pragma unroll
        for (int r = 0; r < kFOwnRounds; ++r) {
            const int64_t i = ent0 + r * kWave + lane;
            if (ent0 + r * kWave >= ent1)
                break;
            const int id = i < ent1 ? own_id[r] : -1;
            const bool valid = i < ent1 && (unsigned)id < (unsigned)a.E;
            const uint64_t m = match_expert(id, valid, a.nbits);
            int pos = -1;
            if (valid) {
                const int below = lanes_below(m);
                const int b = s_base[id];
                pos = b + below;
                if (below == 0)
                    s_base[id] = b + (int)__popcll(m);
            }
            if (i < ent1) {
                if ((uint64_t)(uint32_t)pos >= (uint64_t)slots)
                    pos = -1;  // cannot happen with consistent counts; keeps every store in bounds
                a.slot_pos[i] = pos;
                if (pos >= 0 && a.row_src)
                    a.row_src[pos] = (int32_t)i;
                s_pos[i - ent0] = pos;
            }
        }
    }
    __syncthreads();

    // E. store each token row (this wave's part of it) to its k packed rows
    u32x4 *packed = static_cast<u32x4 *>(a.packed);
    for (int j0 = 0; j0 < tpw; ++j0) {
        const int64_t t = wtok + j0;
        if (t >= tok1)
            break;
        if (j0 > 0) {
            const u32x4 *src = x + t * V + col + lane;
#pragma unroll
            for (int u = 0; u < U; ++u)
                d[u] = __builtin_nontemporal_load(src + u * kWave);
        }
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const int64_t p = s_pos[(t - tok0) * K + j];
            if (p < 0 || p >= a.max_rows)
                continue;
            const RowStore<kStoreNT> dst(packed + p * V + col, (uint32_t)(V - col) * 16u);
#pragma unroll
            for (int u = 0; u < U; ++u)
                dst.put(d[u], u * kWave + lane);
        }
    }
}

template <int U, int K, bool MULTI, bool WIDE>
void launch_one(const FusedArgs &a, int32_t tpw, int32_t split, unsigned blocks, int threads, hipStream_t stream,
                TraceSlot ts) {
    hipExtLaunchKernelGGL((layout_pack_kernel<U, K, MULTI, WIDE>), dim3(blocks), dim3(threads), 0, stream, ts.start,
                          ts.stop, 0, a, tpw, split);
}

// Picks the instance: the count loop only where one batch of loads does not cover every
// id (never within the wide limits: at most 16384 ids, 1024 threads x 16), four experts
// per lane above 64 experts.
template <int U>
hipError_t launch_k(const FusedArgs &a, int32_t tpw, int32_t split, unsigned blocks, int threads, hipStream_t stream,
                    TraceSlot ts) {
    const bool multi = a.T * a.k > (int64_t)threads * kFBatch * 4;  // one batch: kFBatch 4-id groups per thread
    const bool wide = a.E > kFNarrowE;
    if ((wide || a.k == 8) && multi)
        return hipErrorInvalidValue;  // excluded by the limits
    switch (a.k) {
    case 1:
        wide ? launch_one<U, 1, false, true>(a, tpw, split, blocks, threads, stream, ts)
             : (multi ? launch_one<U, 1, true, false>(a, tpw, split, blocks, threads, stream, ts)
                      : launch_one<U, 1, false, false>(a, tpw, split, blocks, threads, stream, ts));
        break;
    case 2:
        wide ? launch_one<U, 2, false, true>(a, tpw, split, blocks, threads, stream, ts)
             : (multi ? launch_one<U, 2, true, false>(a, tpw, split, blocks, threads, stream, ts)
                      : launch_one<U, 2, false, false>(a, tpw, split, blocks, threads, stream, ts));
        break;
    case 4:
        wide ? launch_one<U, 4, false, true>(a, tpw, split, blocks, threads, stream, ts)
             : (multi ? launch_one<U, 4, true, false>(a, tpw, split, blocks, threads, stream, ts)
                      : launch_one<U, 4, false, false>(a, tpw, split, blocks, threads, stream, ts));
        break;
    default:
        wide ? launch_one<U, 8, false, true>(a, tpw, split, blocks, threads, stream, ts)
             : launch_one<U, 8, false, false>(a, tpw, split, blocks, threads, stream, ts);
        break;
    }
    return hipSuccess;
}

// Workgroups of one call.  Below kFSplitBelow tokens a row is split over the fewest waves
// S (dividing its G groups, with an instance for G/S groups) that make the call at least
// kFSplitBelow waves, else over the most; a workgroup holds m tokens (m*S waves: at least
// 4, and enough threads that one batch of id loads covers every id; at most 16; m*k a
// multiple of 4, since step B splits the ids before the workgroup's own at whole 4-id
// groups).  Split
// rows measured on MI355X, 256 experts top-8, 14 KiB rows: 256 tokens 9.8 against 11.4 us,
// 512 tokens 16.1 against 16.9 us.  Otherwise 4, 8 or 16 waves by the entries (4 or 8
// win up to 8192 entries, 16 above), with tpw tokens per wave so that the workgroups hold
// at most kFMaxWaves waves.
struct FusedGeom {
    int32_t split = 1, waves = 4, tpw = 1;
    int64_t blocks = 0;
};

FusedGeom fused_geometry(int64_t T, int32_t k, int G) {
    FusedGeom g;
    const int64_t slots = T * k;
    const int64_t ids_per_wave = (int64_t)kWave * kFBatch * 4;  // one batch of 16-byte id loads
    if (T < kFSplitBelow) {
        int split = 1;
        for (int d : {2, 4, 7, 8, 14, 16}) {
            const int u = G % d == 0 ? G / d : 0;
            if (u == 1 || u == 2 || u == 4 || u == 8) {
                split = d;
                if (T * d >= kFSplitBelow)
                    break;
            }
        }
        if (split > 1) {
            int64_t m = split >= 4 ? 1 : 4 / split;
            m = std::max<int64_t>(m, (slots + split * ids_per_wave - 1) / (split * ids_per_wave));
            const int64_t q = k < 4 ? 4 / k : 1;  // m*k a multiple of 4
            m = (m + q - 1) / q * q;
            if (m * split <= 16) {
                g.split = split;
                g.waves = (int32_t)(m * split);
                g.tpw = 1;
                g.blocks = (T + m - 1) / m;
                return g;
            }
        }
    }
    g.waves = slots <= 4096 ? 4 : (slots <= 8192 ? 8 : 16);
    const int64_t max_blocks = kFMaxWaves / g.waves;
    const int64_t per_block_min = (T + max_blocks - 1) / max_blocks;
    g.tpw = (int32_t)((per_block_min + g.waves - 1) / g.waves);
    g.blocks = (T + (int64_t)g.waves * g.tpw - 1) / ((int64_t)g.waves * g.tpw);
    return g;
}

}  // namespace

bool fused_layout_pack_fits(int64_t T, int32_t k, int32_t E, int32_t H, const void *topk_idx) {
    if (T < 1 || E < 1 || E > kFMaxE || k > E || !(k == 1 || k == 2 || k == 4 || k == 8))
        return false;
    const int64_t wide_limit = H <= 4096 ? kFMaxSlotsWide : kFMaxSlotsWideLong;
    if (T * k > (E > kFNarrowE || k == 8 ? wide_limit : kFMaxSlots))
        return false;
    if (H % 512 != 0)
        return false;
    const int G = H / 512;
    return (G == 1 || G == 2 || G == 4 || G == 8 || G == 14 || G == 16) &&
           reinterpret_cast<uintptr_t>(topk_idx) % 16 == 0;
}

hipError_t launch_layout_pack(const FusedArgs &a, hipStream_t stream) {
    if (!fused_layout_pack_fits(a.T, a.k, a.E, a.H, a.topk_idx) || a.R < 1 || a.E % a.R != 0)
        return hipErrorInvalidValue;
    const int G = a.H / 512;
    const FusedGeom g = fused_geometry(a.T, a.k, G);
    if ((int64_t)(g.waves / g.split) * g.tpw * a.k > kFMaxOwn || g.blocks > INT32_MAX)
        return hipErrorInvalidValue;  // excluded by the limits above
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    const unsigned nb = (unsigned)g.blocks;
    const int threads = g.waves * kWave;
    hipError_t err;
    switch (G / g.split) {  // groups per wave
    case 1: err = launch_k<1>(a, g.tpw, g.split, nb, threads, stream, ts); break;
    case 2: err = launch_k<2>(a, g.tpw, g.split, nb, threads, stream, ts); break;
    case 4: err = launch_k<4>(a, g.tpw, g.split, nb, threads, stream, ts); break;
    case 8: err = launch_k<8>(a, g.tpw, g.split, nb, threads, stream, ts); break;
    case 14: err = launch_k<14>(a, g.tpw, g.split, nb, threads, stream, ts); break;
    default: err = launch_k<16>(a, g.tpw, g.split, nb, threads, stream, ts); break;
    }
    if (err != hipSuccess)
        return err;  // nothing was launched (unreachable within the limits)
    err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("layout_pack", ts);
    return err;
}

}  // namespace ep
