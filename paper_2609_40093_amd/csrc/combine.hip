// combine.hip -- gate-weighted top-k combine for gfx950:
//   out[t][:] = sum_{j<k} w[t*k+j] * recv[slot_pos[t*k+j]][:]
// The returned contributions of a token are added on the GPU that owns the token
// (Sec. 4.3 of the paper: a DMA engine cannot add, so the reduction stays on the GPU),
// which also returns the rows to token order.
//
// Arithmetic: fp32 accumulator, fused multiply-add per slot in order j = 0..k-1 starting
// from +0, then one round-to-nearest-even conversion to bf16 (v_cvt_pk_bf16_f32), or the
// fp32 accumulator itself.  HBM-bound: k row reads and one row write per token.
//
// Mapping: one wave per (token, column chunk of 64*U 16-byte vectors); the k slot
// positions and gates are wave-uniform scalar loads.  Slots are taken KC at a time and
// all KC*U row loads of a batch are issued before their FMAs, keeping KC*U KiB in flight
// per wave.  Nothing is conditional: a slot without a row reads row 0 with its bits
// masked to +0 and its gate set to -0, so it adds exactly -0, which leaves every sum
// unchanged (signs of zero included) -- a branch around it would let the compiler sink
// the slot's loads into the branch and serialize them behind the previous slot's.  In
// EXACT instances (rows a whole number of chunks) no lane carries a bounds mask either.
// Rows are read once: loads are non-temporal.  Stores are device-scope write-through
// buffer stores when the output is under 128 MiB and non-temporal from there up (RowStore),
// where the call runs as launches of about 64 MiB of output each (see the launcher):
// measured on MI355X with inputs outside the memory-side cache, write-through stores made
// the combine 2-7% faster up to 112 MiB of output (top-8 of 14 KiB rows, 2K-8K tokens;
// 4 KiB rows, 8K tokens; top-2 of 8 KiB rows, 4K tokens) and 0.5-2% slower from 128 MiB
// up (top-2, 16K tokens of 8 KiB rows; 16K and 32K tokens of 14 KiB rows).
#include "ep_internal.h"

namespace ep {
namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2 b = __builtin_convertvector(f32x2{lo, hi}, bf16x2);
    return __builtin_bit_cast(uint32_t, b);
}

// FIXED_K: k == KC (one batch of slots, its bounds known at compile time).  SEL: the
// receive buffer is chosen by a round counter in device memory (graph-replayed rounds);
// without it the kernel loads nothing before the slot positions.
template <int U, int KC, bool F32_OUT, bool EXACT, bool FIXED_K, bool SEL, bool WT>
__global__ __launch_bounds__(256) void combine_kernel(const u32x4 *__restrict__ recv,
                                                      const int32_t *__restrict__ slot_pos,
                                                      const float *__restrict__ topk_w, int64_t T,
                                                      int32_t V, int32_t chunks, int32_t k,
                                                      void *__restrict__ out, int64_t max_rows,
                                                      RoundSel sel) {
    const int lane = threadIdx.x & (kWave - 1);
    if (SEL && (__hip_atomic_load(sel.round, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 1u))
        recv = static_cast<const u32x4 *>(sel.alt);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + wave;
    const int64_t t = item / chunks;
    if (t >= T)
        return;
    const int32_t v0 = (int32_t)(item - t * chunks) * (U * kWave);
    const int32_t kk = FIXED_K ? KC : k;
    const int32_t *sp = slot_pos + t * kk;
    const float *wt = topk_w + t * kk;

    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q)
            acc[u][q] = 0.0f;

    for (int32_t j0 = 0; j0 < kk; j0 += KC) {
        u32x4 d[KC][U];
        float g[KC];
        uint32_t keep[KC];  // all ones for a slot with a row, else 0
        bool ok[KC];
        // positions first, then every row load, then the gates (needed only by the FMAs);
        // every load is issued for every jj (a slot past k has no row)
#pragma unroll
        for (int jj = 0; jj < KC; ++jj) {
            const int32_t j = j0 + jj;
            const int64_t p = j < kk ? (int64_t)sp[min(j, kk - 1)] : -1;  // wave-uniform
            ok[jj] = p >= 0 && p < max_rows;
            keep[jj] = ok[jj] ? ~0u : 0u;
            const u32x4 *src = recv + (ok[jj] ? p : 0) * V;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t v = v0 + u * kWave + lane;
                d[jj][u] = EXACT ? __builtin_nontemporal_load(src + v)
                                 : __builtin_nontemporal_load(src + min(v, V - 1));
            }
        }
#pragma unroll
        for (int jj = 0; jj < KC; ++jj) {
            const float gj = wt[min(j0 + jj, kk - 1)];
            g[jj] = ok[jj] ? gj : -0.0f;
        }
#pragma unroll
        for (int jj = 0; jj < KC; ++jj)
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t bits = d[jj][u][q] & keep[jj];
                    acc[u][2 * q] = __builtin_fmaf(g[jj], bf16_lo(bits), acc[u][2 * q]);
                    acc[u][2 * q + 1] = __builtin_fmaf(g[jj], bf16_hi(bits), acc[u][2 * q + 1]);
                }
    }

    // the token's output row: V 16-byte vectors (bf16) or 2V (fp32)
    constexpr int kVecs = F32_OUT ? 2 : 1;
    const RowStore<WT ? kStoreWT : kStoreNT> dst((u32x4 *)out + t * V * kVecs, (uint32_t)V * kVecs * 16u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int32_t v = v0 + u * kWave + lane;
        if (!EXACT && v >= V)
            continue;
        if constexpr (F32_OUT) {
            const u32x4 a = {__float_as_uint(acc[u][0]), __float_as_uint(acc[u][1]),
                             __float_as_uint(acc[u][2]), __float_as_uint(acc[u][3])};
            const u32x4 b = {__float_as_uint(acc[u][4]), __float_as_uint(acc[u][5]),
                             __float_as_uint(acc[u][6]), __float_as_uint(acc[u][7])};
            dst.put(a, 2u * (uint32_t)v);
            dst.put(b, 2u * (uint32_t)v + 1u);
        } else {
            const u32x4 r = {pack_bf16x2(acc[u][0], acc[u][1]), pack_bf16x2(acc[u][2], acc[u][3]),
                             pack_bf16x2(acc[u][4], acc[u][5]), pack_bf16x2(acc[u][6], acc[u][7])};
            dst.put(r, (uint32_t)v);
        }
    }
}

// With no rows to read every output is zero (each sum is empty).
__global__ __launch_bounds__(256) void zero_fill_kernel(u32x4 *__restrict__ out, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        out[i] = u32x4{0u, 0u, 0u, 0u};
}

constexpr int64_t kCombineWriteThroughBelow = 128ll << 20;  // output bytes
// From 128 MiB of output up the combine runs as several launches over consecutive token
// ranges of about 64 MiB of output each (measured on MI355X, top-8 of 14 KiB rows, 32K
// tokens, non-temporal stores: one launch 747 us, 2 / 4 / 8 / 16 / 32 / 64 launches 733 /
// 727 / 718 / 719 / 748 / 801 us, and the layer's pack after it unchanged; the
// write-through stores of the smaller outputs made the following pack slower when applied
// to such launches).
constexpr int64_t kCombineSplitAbove = 128ll << 20;
constexpr int64_t kCombineLaunchBytes = 64ll << 20;

template <int U, int KC, bool WT>
void launch_ukw(dim3 grid, dim3 block, hipStream_t stream, TraceSlot ts, const u32x4 *rv, const int32_t *slot_pos,
                const float *topk_w, int64_t T, int32_t V, int32_t chunks, int32_t k, void *out, bool out_f32,
                bool exact, int64_t max_rows, RoundSel sel) {
#define EP_COMBINE_ARGS grid, block, 0, stream, ts.start, ts.stop, 0, rv, slot_pos, topk_w, T, V, chunks, k, out, max_rows, sel
#define EP_COMBINE_LAUNCH(F32, EX)                                                                      \
    (k == KC ? hipExtLaunchKernelGGL((combine_kernel<U, KC, F32, EX, true, false, WT>), EP_COMBINE_ARGS) \
             : hipExtLaunchKernelGGL((combine_kernel<U, KC, F32, EX, false, false, WT>), EP_COMBINE_ARGS))
    if (sel.round && out_f32)  // graph-replayed rounds: the general instance reading the round
        hipExtLaunchKernelGGL((combine_kernel<U, KC, true, false, false, true, WT>), EP_COMBINE_ARGS);
    else if (sel.round)
        hipExtLaunchKernelGGL((combine_kernel<U, KC, false, false, false, true, WT>), EP_COMBINE_ARGS);
    else if (out_f32 && exact)
        EP_COMBINE_LAUNCH(true, true);
    else if (out_f32)
        EP_COMBINE_LAUNCH(true, false);
    else if (exact)
        EP_COMBINE_LAUNCH(false, true);
    else
        EP_COMBINE_LAUNCH(false, false);
#undef EP_COMBINE_LAUNCH
#undef EP_COMBINE_ARGS
}

template <int U, int KC>
hipError_t launch_uk(const void *recv, const int32_t *slot_pos, const float *topk_w, int64_t T,
                     int32_t V, int32_t k, void *out, bool out_f32, int64_t max_rows,
                     hipStream_t stream, RoundSel sel) {
    const int32_t chunks = (V + U * kWave - 1) / (U * kWave);
    const int waves_per_block = 4;
    const int64_t row_bytes = (int64_t)V * 16 * (out_f32 ? 2 : 1);  // one output row
    const int64_t out_bytes = T * row_bytes;
    // token ranges of the launches: one below kCombineSplitAbove bytes of output, else
    // about kCombineLaunchBytes each
    const int64_t launches = out_bytes < kCombineSplitAbove
                                 ? 1
                                 : std::min<int64_t>(T, (out_bytes + kCombineLaunchBytes - 1) / kCombineLaunchBytes);
    const int64_t per = (T + launches - 1) / launches;
    if ((per * chunks + waves_per_block - 1) / waves_per_block > INT32_MAX)
        return hipErrorInvalidValue;
    const bool exact = V % (U * kWave) == 0;
    const dim3 block(waves_per_block * kWave);
    const u32x4 *rv = static_cast<const u32x4 *>(recv);
    (void)hipGetLastError();  // drop an error left by an earlier, already reported call
    const TraceSlot ts = trace_acquire();  // one pair of events around every launch of the call
    const bool wt = out_bytes < kCombineWriteThroughBelow;
    for (int64_t t0 = 0; t0 < T; t0 += per) {
        const int64_t n = std::min(per, T - t0);
        const dim3 grid((unsigned)((n * chunks + waves_per_block - 1) / waves_per_block));
        TraceSlot part;
        part.start = t0 == 0 ? ts.start : nullptr;
        part.stop = t0 + n == T ? ts.stop : nullptr;
        const int32_t *sp = slot_pos + t0 * k;
        const float *gw = topk_w + t0 * k;
        void *o = static_cast<char *>(out) + t0 * row_bytes;
        if (wt)
            launch_ukw<U, KC, true>(grid, block, stream, part, rv, sp, gw, n, V, chunks, k, o, out_f32, exact,
                                    max_rows, sel);
        else
            launch_ukw<U, KC, false>(grid, block, stream, part, rv, sp, gw, n, V, chunks, k, o, out_f32, exact,
                                     max_rows, sel);
    }
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("combine", ts);
    return err;
}

// One pass of the per-sender accumulation (a combine that reduces each sender's returned
// rows as they land).  For a token and a set M of senders, p_M is the length of the
// longest prefix of its k slots whose rows all come from senders in M (a slot without a
// row belongs to every prefix; a row's sender is the rank segment holding it, rows past
// the last segment count as the last sender's).  Pass i adds the slots [p_prev, p_cur)
// for M = masks[i], masks[i + 1] -- in slot order, to the fp32 partial kept in `acc` (from
// +0 unless an earlier pass added a row of this token), by the very FMAs of
// combine_kernel -- and writes a token whose prefix is complete to `out`.  Sets only
// grow, so every slot is added once and in slot order: the result equals combine_kernel's
// bit for bit whatever order the senders arrive in.  A slot without a row is skipped:
// combine_kernel adds exactly -0 for it, which changes nothing.  One wave per (token,
// 64-vector chunk).
template <bool F32_OUT>
__global__ __launch_bounds__(256) void accumulate_kernel(const u32x4 *__restrict__ recv,
                                                         const int32_t *__restrict__ slot_pos,
                                                         const float *__restrict__ topk_w, int64_t T, int32_t V,
                                                         int32_t chunks, int32_t k,
                                                         const int32_t *__restrict__ rank_offsets, int32_t R,
                                                         const uint32_t *__restrict__ masks, int32_t i,
                                                         float *__restrict__ acc, void *__restrict__ out,
                                                         int64_t max_rows) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + wave;
    const int64_t t = item / chunks;
    if (t >= T)
        return;
    const int32_t v = (int32_t)(item - t * chunks) * kWave + lane;
    const bool vin = v < V;
    const int32_t ro = lane <= R ? rank_offsets[lane] : INT32_MAX;  // lane r: first row of rank r
    const uint32_t prev = masks[i], cur = masks[i + 1];
    const int32_t *sp = slot_pos + t * k;
    auto sender = [&](int64_t p) {  // the segment holding row p (wave-uniform p)
        return min((int)__popcll(__ballot(ro <= p)) - 1, R - 1);
    };
    int32_t pp = -1, pc = k;
    bool added_before = false;  // a row of this token went into acc in an earlier pass
    for (int32_t j = 0; j < k; ++j) {  // wave-uniform
        const int64_t p = sp[j];
        if (p < 0 || p >= max_rows)
            continue;
        const int r = sender(p);
        if (pp < 0) {
            if ((prev >> r) & 1u)
                added_before = true;
            else
                pp = j;
        }
        if (!((cur >> r) & 1u)) {
            pc = j;
            break;
        }
    }
    if (pp < 0) {  // every row of the token was in before this pass
        if (i != 0)
            return;    // written by an earlier pass
        pp = k;        // a token without rows: written by pass 0, as +0 (combine_kernel's sum)
    } else if (pc == pp) {
        return;
    }
    const int64_t o = t * V + (vin ? v : 0);
    float a[8];
    if (added_before && vin) {
        const u32x4 lo = reinterpret_cast<const u32x4 *>(acc)[2 * o];
        const u32x4 hi = reinterpret_cast<const u32x4 *>(acc)[2 * o + 1];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            a[q] = __uint_as_float(lo[q]);
            a[4 + q] = __uint_as_float(hi[q]);
        }
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q)
            a[q] = 0.0f;
    }
    for (int32_t j = pp; j < pc; ++j) {
        const int64_t p = sp[j];
        if (p < 0 || p >= max_rows)
            continue;
        const float g = topk_w[t * k + j];
        const u32x4 d = __builtin_nontemporal_load(recv + p * V + (vin ? v : 0));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            a[2 * q] = __builtin_fmaf(g, bf16_lo(d[q]), a[2 * q]);
            a[2 * q + 1] = __builtin_fmaf(g, bf16_hi(d[q]), a[2 * q + 1]);
        }
    }
    if (!vin)
        return;
    if (pc == k) {
        if constexpr (F32_OUT) {
            u32x4 *dst = (u32x4 *)out + 2 * o;
            __builtin_nontemporal_store(u32x4{__float_as_uint(a[0]), __float_as_uint(a[1]), __float_as_uint(a[2]),
                                              __float_as_uint(a[3])}, dst);
            __builtin_nontemporal_store(u32x4{__float_as_uint(a[4]), __float_as_uint(a[5]), __float_as_uint(a[6]),
                                              __float_as_uint(a[7])}, dst + 1);
        } else {
            const u32x4 r = {pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(a[4], a[5]),
                             pack_bf16x2(a[6], a[7])};
            __builtin_nontemporal_store(r, (u32x4 *)out + o);
        }
    } else {
        u32x4 *dst = reinterpret_cast<u32x4 *>(acc) + 2 * o;
        dst[0] = u32x4{__float_as_uint(a[0]), __float_as_uint(a[1]), __float_as_uint(a[2]), __float_as_uint(a[3])};
        dst[1] = u32x4{__float_as_uint(a[4]), __float_as_uint(a[5]), __float_as_uint(a[6]), __float_as_uint(a[7])};
    }
}

}  // namespace

hipError_t launch_combine(const void *recv, const int32_t *slot_pos, const float *topk_w,
                          int64_t T, int32_t H, int32_t k, void *out, bool out_f32,
                          int64_t max_rows, hipStream_t stream, RoundSel sel) {
    if (T == 0)
        return hipSuccess;
    const int32_t V = H / 8;
    if (max_rows <= 0) {  // the kernels below read row 0 for slots without a row
        const int64_t n = T * V * (out_f32 ? 2 : 1);
        const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
        (void)hipGetLastError();
        hipLaunchKernelGGL(zero_fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, static_cast<u32x4 *>(out), n);
        return hipGetLastError();
    }
    // KC*U 16-byte loads per lane in flight: 16 for k >= 4 (8 for k >= 8 with rows of at
    // least 12 KiB), 4 for k = 2 and 3.  Measured on MI355X: at k = 8 and 14 KiB rows,
    // one-group chunks (twice the waves) beat two-group chunks by 2% at 32768 tokens and
    // 1% at 16384, and tie at a few thousand; with 4 KiB rows two-group chunks are ahead
    // by 1%.  At k = 2, two-group chunks beat four-group ones.
    if (k >= 8 && V >= 768)
        return launch_uk<1, 8>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    if (k >= 8)
        return launch_uk<2, 8>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    if (k >= 4)
        return launch_uk<4, 4>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    if (k >= 2)
        return launch_uk<2, 2>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
    return launch_uk<4, 1>(recv, slot_pos, topk_w, T, V, k, out, out_f32, max_rows, stream, sel);
}

hipError_t launch_accumulate(const void *recv, const int32_t *slot_pos, const float *topk_w, int64_t T, int32_t H,
                             int32_t k, const int32_t *rank_offsets, int32_t R, const uint32_t *masks, int32_t i,
                             float *acc, void *out, bool out_f32, int64_t max_rows, hipStream_t stream) {
    if (T <= 0)
        return hipSuccess;
    if (!recv || !slot_pos || !topk_w || !rank_offsets || !masks || !acc || !out || H % 8 != 0 || R < 1 ||
        R > 32 || i < 0)
        return hipErrorInvalidValue;
    const int32_t V = H / 8;
    const int32_t chunks = (V + kWave - 1) / kWave;
    const int64_t blocks = (T * chunks + 3) / 4;
    if (blocks > INT32_MAX)
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    TraceSlot ts = trace_acquire();
    if (out_f32)
        hipExtLaunchKernelGGL(accumulate_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, ts.start,
                              ts.stop, 0, (const u32x4 *)recv, slot_pos, topk_w, T, V, chunks, k, rank_offsets, R,
                              masks, i, acc, out, max_rows);
    else
        hipExtLaunchKernelGGL(accumulate_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, ts.start,
                              ts.stop, 0, (const u32x4 *)recv, slot_pos, topk_w, T, V, chunks, k, rank_offsets, R,
                              masks, i, acc, out, max_rows);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess)
        trace_submit("accumulate", ts);
    return err;
}

}  // namespace ep
