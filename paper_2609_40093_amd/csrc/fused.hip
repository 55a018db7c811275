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
// of the kernel waits on its last workgroups):
//   A. each wave issues the loads of its first ids, then those of its first token row
//      (they do not depend on the layout; vector loads complete in order, so the ids
//      come first);
//   B. the workgroup counts all T*k entries (16-byte loads of 4 ids) with LDS atomic
//      adds into 16 copies of the per-expert counters, chosen by lane, so that lanes of
//      one instruction naming the same expert rarely hit the same word (vector and LDS
//      work only: a ballot per id would queue every wave of the compute unit on its one
//      scalar unit), both over all entries and over the entries before its own range;
//      routing errors (an id outside [0,E), an expert twice in one token row) are found
//      in the same pass;
//   C. the totals' exclusive scan (DPP) gives the expert offsets; workgroup 0 stores the
//      counts, offsets, rank counts/offsets and the status word;
//   D. wave 0 ranks the workgroup's own entries in flat order (ballot match-any and a
//      masked popcount, as the layout kernel does: stable), stores slot_pos / row_src and
//      keeps the rows in LDS;
//   E. each wave stores its tokens' rows to their k packed rows (non-temporal; a row is
//      U groups of 64 16-byte vectors, one per lane, all loads in flight together).
// The outputs equal those of the layout kernel followed by the pack kernel, bit for bit.
// Workgroups never wait on each other, so nothing needs them resident together.
//
// Limits (the host falls back to the two kernels outside them): E <= 64 (a lane per
// expert in step C), k in {1, 2, 4} (a token row lies inside one 4-id load), T*k <= 65536
// (every workgroup reads every id), rows of 1, 2, 4, 8 or 16 groups (H a multiple of 512
// up to 8192), a 16-byte aligned routing array.
#include "ep_internal.h"
#include "wave.h"

namespace ep {
namespace {

constexpr int kFMaxThreads = 16 * kWave;    // largest workgroup (16 waves)
constexpr int kFMaxE = 64;                   // experts: one lane each in step C
constexpr int64_t kFMaxSlots = 65536;        // T*k: every workgroup reads every id
constexpr int kFMaxOwn = 256;                // entries one workgroup owns (LDS rows)
constexpr int kFOwnRounds = kFMaxOwn / kWave;
constexpr int kFBatch = 4;                   // 16-byte id loads in flight per lane
constexpr int kFMaxWaves = 4096;             // waves in flight over the device (16 per CU)

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

// Counts one id into the LDS counters (all entries, and those before this workgroup's).
__device__ __forceinline__ void count_id(int id, bool in, bool before, int E, int *s_all, int *s_pre, int copy,
                                         bool &bad_id) {
    const bool valid = in && (unsigned)id < (unsigned)E;
    bad_id |= in && !valid;
    if (valid) {
        atomicAdd(&s_all[copy * kFMaxE + id], 1);
        if (before)
            atomicAdd(&s_pre[copy * kFMaxE + id], 1);
    }
}

// MULTI: more ids than one batch of the workgroup's loads (the count loops).  Instances
// without the loop have only straight-line loads, so the compiler's waits stay exact and
// no wave waits for its token row before the count's barrier.
template <int U, int K, bool MULTI>
__global__ __launch_bounds__(kFMaxThreads) void layout_pack_kernel(FusedArgs a, int32_t tpw) {
    __shared__ int s_all[kFCopies * kFMaxE];
    __shared__ int s_pre[kFCopies * kFMaxE];
    __shared__ int s_base[kFMaxE];
    __shared__ int s_pos[kFMaxOwn];
    __shared__ int s_err;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int threads = blockDim.x, waves = threads / kWave;
    const int64_t slots = a.T * K;
    const int64_t tok0 = (int64_t)blockIdx.x * waves * tpw;
    const int64_t tok1 = min(a.T, tok0 + (int64_t)waves * tpw);
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
    const int64_t wtok = tok0 + (int64_t)w * tpw;
    u32x4 d[U];
    {
        const u32x4 *src = x + min(wtok, tok1 - 1) * V + lane;
#pragma unroll
        for (int u = 0; u < U; ++u)
            d[u] = __builtin_nontemporal_load(src + u * kWave);
    }
    for (int i = tid; i < kFCopies * kFMaxE; i += threads) {
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
            dup |= in && row_repeats<K>(v[b], a.E);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                count_id(v[b][c], in, before, a.E, s_all, s_pre, lane % kFCopies, bad_id);
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
        count_id(id, in, ti < ent0, a.E, s_all, s_pre, lane % kFCopies, bad_id);
    }
    const uint32_t wave_err = (__ballot(bad_id) ? kRoutingIdOutOfRange : 0u) | (__ballot(dup) ? kRoutingDuplicate : 0u);
    if (lane == 0 && wave_err)
        atomicOr(&s_err, (int)wave_err);
    __syncthreads();

    if (w == 0) {
        // C. totals, offsets; workgroup 0 stores the layout's counts and the status
        int tot = 0, pre = 0;
        if (lane < a.E) {
#pragma unroll
            for (int c = 0; c < kFCopies; ++c) {
                tot += s_all[c * kFMaxE + lane];
                pre += s_pre[c * kFMaxE + lane];
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
        // D. rank the own entries in flat order
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

    // E. store each token row to its k packed rows
    u32x4 *packed = static_cast<u32x4 *>(a.packed);
    for (int j0 = 0; j0 < tpw; ++j0) {
        const int64_t t = wtok + j0;
        if (t >= tok1)
            break;
        if (j0 > 0) {
            const u32x4 *src = x + t * V + lane;
#pragma unroll
            for (int u = 0; u < U; ++u)
                d[u] = __builtin_nontemporal_load(src + u * kWave);
        }
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const int64_t p = s_pos[(t - tok0) * K + j];
            if (p < 0 || p >= a.max_rows)
                continue;
            u32x4 *dst = packed + p * V + lane;
#pragma unroll
            for (int u = 0; u < U; ++u)
                __builtin_nontemporal_store(d[u], dst + u * kWave);
        }
    }
}

template <int U, bool MULTI>
void launch_km(const FusedArgs &a, int32_t tpw, unsigned blocks, int threads, hipStream_t stream, TraceSlot ts) {
    if (a.k == 1)
        hipExtLaunchKernelGGL((layout_pack_kernel<U, 1, MULTI>), dim3(blocks), dim3(threads), 0, stream, ts.start,
                              ts.stop, 0, a, tpw);
    else if (a.k == 2)
        hipExtLaunchKernelGGL((layout_pack_kernel<U, 2, MULTI>), dim3(blocks), dim3(threads), 0, stream, ts.start,
                              ts.stop, 0, a, tpw);
    else
        hipExtLaunchKernelGGL((layout_pack_kernel<U, 4, MULTI>), dim3(blocks), dim3(threads), 0, stream, ts.start,
                              ts.stop, 0, a, tpw);
}

template <int U>
void launch_k(const FusedArgs &a, int32_t tpw, unsigned blocks, int threads, hipStream_t stream, TraceSlot ts) {
    // one batch is kFBatch 4-id groups per thread
    if (a.T * a.k > (int64_t)threads * kFBatch * 4)
        launch_km<U, true>(a, tpw, blocks, threads, stream, ts);
    else
        launch_km<U, false>(a, tpw, blocks, threads, stream, ts);
}

}  // namespace

bool fused_layout_pack_fits(int64_t T, int32_t k, int32_t E, int32_t H, const void *topk_idx) {
    if (T < 1 || E < 1 || E > kFMaxE || !(k == 1 || k == 2 || k == 4) || T * k > kFMaxSlots)
        return false;
    if (H % 512 != 0)
        return false;
    const int G = H / 512;
    return (G == 1 || G == 2 || G == 4 || G == 8 || G == 16) && reinterpret_cast<uintptr_t>(topk_idx) % 16 == 0;
}

hipError_t launch_layout_pack(const FusedArgs &a, hipStream_t stream) {
    if (!fused_layout_pack_fits(a.T, a.k, a.E, a.H, a.topk_idx) || a.R < 1 || a.E % a.R != 0)
        return hipErrorInvalidValue;
    // workgroup size by the entries every workgroup counts (measured on MI355X: 4 or 8
    // waves win up to 8192 entries, 16 above); tokens per wave: enough that the workgroups
    // hold at most kFMaxWaves waves
    const int64_t slots = a.T * a.k;
    const int waves = slots <= 4096 ? 4 : (slots <= 8192 ? 8 : 16);
    const int64_t max_blocks = kFMaxWaves / waves;
    const int64_t per_block_min = (a.T + max_blocks - 1) / max_blocks;
    const int32_t tpw = (int32_t)((per_block_min + waves - 1) / waves);
    const int64_t blocks = (a.T + (int64_t)waves * tpw - 1) / ((int64_t)waves * tpw);
    if ((int64_t)waves * tpw * a.k > kFMaxOwn)
        return hipErrorInvalidValue;  // excluded by the limits above
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    TraceSlot ts = trace_acquire();
    switch (a.H / 512) {
    case 1: launch_k<1>(a, tpw, (unsigned)blocks, waves * kWave, stream, ts); break;
    case 2: launch_k<2>(a, tpw, (unsigned)blocks, waves * kWave, stream, ts); break;
    case 4: launch_k<4>(a, tpw, (unsigned)blocks, waves * kWave, stream, ts); break;
    case 8: launch_k<8>(a, tpw, (unsigned)blocks, waves * kWave, stream, ts); break;
    default: launch_k<16>(a, tpw, (unsigned)blocks, waves * kWave, stream, ts); break;
    }
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("layout_pack", ts);
    return err;
}

}  // namespace ep
