/*
 * ep_oracle.c -- CPU oracle for MoE expert-parallel dispatch and combine.
 *
 * TEST INFRASTRUCTURE ONLY (see ep_oracle.h).  Plain loops, no blocking, no fusion,
 * no reordering beyond what the definitions state.  Built with -ffp-contract=off so
 * every sum and product below is rounded exactly as written.
 */
#include "ep_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Threads over which pack and combine split their tokens (ep_oracle_set_threads). */
static int g_threads = 1;

int ep_oracle_set_threads(int threads) {
#ifdef _OPENMP
    g_threads = threads > 0 ? threads : 1;
#else
    (void)threads;
    g_threads = 1;
#endif
    return g_threads;
}

/* ---- bf16 <-> double ------------------------------------------------------------ */

double ep_oracle_bf16_to_double(uint16_t b) {
    /* bf16 is the upper half of a binary32: widen by appending 16 zero bits. */
    uint32_t bits = (uint32_t)b << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

uint16_t ep_oracle_double_to_bf16(double v) {
    /* Round to the nearest bf16 value, ties to the one with an even last bit
     * (IEEE-754 roundTiesToEven), written from the format's definition:
     * 8 significant bits, exponent range of binary32, subnormal spacing 2^-133. */
    if (isnan(v))
        return signbit(v) ? 0xFFC0u : 0x7FC0u;
    uint16_t sign = signbit(v) ? 0x8000u : 0u;
    double a = fabs(v);
    if (isinf(a))
        return sign | 0x7F80u;
    if (a == 0.0)
        return sign;
    int ex;
    (void)frexp(a, &ex);                 /* a in [2^(ex-1), 2^ex) */
    int qexp = ex - 8;                   /* spacing of bf16 values in that binade */
    if (qexp < -133)
        qexp = -133;                     /* subnormal range: fixed spacing */
    double n = nearbyint(ldexp(a, -qexp)); /* default mode: nearest, ties to even */
    double r = ldexp(n, qexp);           /* exact */
    if (r >= ldexp(1.0, 128))
        return sign | 0x7F80u;           /* rounds past the largest finite value */
    float f = (float)r;                  /* exact: r is a bf16 value */
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    return sign | (uint16_t)((bits >> 16) & 0x7FFFu);
}

void ep_oracle_double_to_bf16_n(const double *v, int64_t n, uint16_t *out) {
    for (int64_t i = 0; i < n; ++i)
        out[i] = ep_oracle_double_to_bf16(v[i]);
}

/* ---- layout --------------------------------------------------------------------- */

int ep_oracle_layout(const int32_t *topk_idx, int64_t T, int32_t k, int32_t E, int32_t R,
                     int32_t *expert_counts, int32_t *expert_offsets,
                     int32_t *rank_counts, int32_t *rank_offsets,
                     int32_t *slot_pos, int32_t *row_src) {
    if (T < 0 || E < 1 || R < 1 || E % R != 0 || k < 1 || k > E)
        return EP_ORACLE_INVALID_ARG;
    if (T * (int64_t)k > INT32_MAX)
        return EP_ORACLE_INVALID_ARG;
    const int64_t n = T * (int64_t)k;
    const int32_t L = E / R;             /* experts per rank, placed contiguously */

    /* 1. every id is an expert, and a token selects k different experts (Sec. 2.1) */
    int status = EP_ORACLE_OK;
    for (int64_t t = 0; t < T; ++t) {
        for (int32_t j = 0; j < k; ++j) {
            int32_t e = topk_idx[t * k + j];
            if (e < 0 || e >= E)
                status = EP_ORACLE_BAD_ROUTING;
            for (int32_t jj = 0; jj < j; ++jj)
                if (topk_idx[t * k + jj] == e)
                    status = EP_ORACLE_BAD_ROUTING;
        }
    }
    if (status != EP_ORACLE_OK)
        return status;

    /* 2. rows per expert: one row per (token, selected expert) */
    for (int32_t e = 0; e < E; ++e)
        expert_counts[e] = 0;
    for (int64_t i = 0; i < n; ++i)
        expert_counts[topk_idx[i]] += 1;

    /* 3. each expert's group starts where the previous one ends; a rank's segment is
     *    the concatenation of its experts' groups */
    expert_offsets[0] = 0;
    for (int32_t e = 0; e < E; ++e)
        expert_offsets[e + 1] = expert_offsets[e] + expert_counts[e];
    for (int32_t r = 0; r < R; ++r) {
        rank_counts[r] = 0;
        for (int32_t e = r * L; e < (r + 1) * L; ++e)
            rank_counts[r] += expert_counts[e];
        rank_offsets[r] = expert_offsets[r * L];
    }
    rank_offsets[R] = (int32_t)n;

    /* 4. place the slots in increasing flat index, each at the next free row of its
     *    expert's group: rows of one expert keep token order */
    int32_t *cursor = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
    if (!cursor)
        abort();
    for (int32_t e = 0; e < E; ++e)
        cursor[e] = expert_offsets[e];
    for (int64_t i = 0; i < n; ++i) {
        int32_t e = topk_idx[i];
        slot_pos[i] = cursor[e];
        cursor[e] += 1;
        if (row_src)
            row_src[slot_pos[i]] = (int32_t)i;
    }
    free(cursor);
    return EP_ORACLE_OK;
}

/* ---- pack ----------------------------------------------------------------------- */

void ep_oracle_pack(const uint16_t *x, int64_t T, int32_t H, int32_t k,
                    const int32_t *slot_pos, uint16_t *packed) {
    const size_t row_bytes = (size_t)H * sizeof(uint16_t);
    /* tokens are independent: each row is written by the thread of its token */
#pragma omp parallel for schedule(static) num_threads(g_threads)
    for (int64_t t = 0; t < T; ++t)
        for (int32_t j = 0; j < k; ++j) {
            int64_t p = slot_pos[t * k + j];
            memcpy(packed + p * (int64_t)H, x + t * (int64_t)H, row_bytes);
        }
}

/* ---- combine -------------------------------------------------------------------- */

void ep_oracle_combine(const uint16_t *y, const int32_t *slot_pos, const float *topk_w,
                       int64_t T, int32_t H, int32_t k,
                       double *out_exact, uint16_t *out_bf16, float *out_f32) {
    /* tokens are independent: each token's sums are formed by one thread, in the order
     * below, whatever the thread count */
#pragma omp parallel num_threads(g_threads)
    {
    double *acc = (double *)malloc(sizeof(double) * (size_t)(H > 0 ? H : 1));
    if (!acc)
        abort();
#pragma omp for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int32_t h = 0; h < H; ++h)
            acc[h] = 0.0;
        /* contributions in slot order j = 0..k-1; each product of a binary32 gate and a
         * bf16 value is exact in double */
        for (int32_t j = 0; j < k; ++j) {
            if (slot_pos[t * k + j] < 0)
                continue;   /* routed to another rank: no contribution here */
            double w = (double)topk_w[t * k + j];
            const uint16_t *row = y + (int64_t)slot_pos[t * k + j] * H;
            for (int32_t h = 0; h < H; ++h)
                acc[h] = acc[h] + w * ep_oracle_bf16_to_double(row[h]);
        }
        for (int32_t h = 0; h < H; ++h) {
            int64_t o = t * (int64_t)H + h;
            if (out_exact)
                out_exact[o] = acc[h];
            if (out_bf16)
                out_bf16[o] = ep_oracle_double_to_bf16(acc[h]);
            if (out_f32)
                out_f32[o] = (float)acc[h];   /* C conversion: current mode, nearest-even */
        }
    }
    free(acc);
    }
}

int ep_oracle_local_layout(const int32_t *topk_idx, int64_t N, int32_t k, int32_t E, int32_t e_lo,
                           int32_t e_hi, int32_t *local_counts, int32_t *local_offsets,
                           int32_t *slot_pos, int32_t *row_src) {
    if (N < 0 || k < 1 || E < 1 || k > E || e_lo < 0 || e_lo >= e_hi || e_hi > E)
        return EP_ORACLE_INVALID_ARG;
    /* 1. validate every row: ids in [0,E), no expert twice */
    for (int64_t t = 0; t < N; ++t)
        for (int32_t j = 0; j < k; ++j) {
            int32_t e = topk_idx[t * k + j];
            if (e < 0 || e >= E)
                return EP_ORACLE_BAD_ROUTING;
            for (int32_t jj = 0; jj < j; ++jj)
                if (topk_idx[t * k + jj] == e)
                    return EP_ORACLE_BAD_ROUTING;
        }
    const int32_t L = e_hi - e_lo;
    /* 2. count the slots that name a local expert */
    for (int32_t l = 0; l < L; ++l)
        local_counts[l] = 0;
    for (int64_t i = 0; i < N * k; ++i) {
        int32_t e = topk_idx[i];
        if (e >= e_lo && e < e_hi)
            local_counts[e - e_lo] += 1;
    }
    /* 3. exclusive prefix sum */
    local_offsets[0] = 0;
    for (int32_t l = 0; l < L; ++l)
        local_offsets[l + 1] = local_offsets[l] + local_counts[l];
    /* 4. place local slots in increasing flat index; others get -1 */
    int32_t *cursor = (int32_t *)malloc(sizeof(int32_t) * (size_t)L);
    if (!cursor)
        abort();
    for (int32_t l = 0; l < L; ++l)
        cursor[l] = local_offsets[l];
    for (int64_t i = 0; i < N * k; ++i) {
        int32_t e = topk_idx[i];
        if (e < e_lo || e >= e_hi) {
            slot_pos[i] = -1;
            continue;
        }
        int32_t p = cursor[e - e_lo]++;
        slot_pos[i] = p;
        if (row_src)
            row_src[p] = (int32_t)i;
    }
    free(cursor);
    return EP_ORACLE_OK;
}

void ep_oracle_block_reduce(const double *blocks, int32_t R, int64_t n, double *out_exact,
                            uint16_t *out_bf16, float *out_f32) {
    for (int64_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int32_t d = 0; d < R; ++d)   /* blocks summed in rank order */
            acc = acc + blocks[(int64_t)d * n + i];
        if (out_exact)
            out_exact[i] = acc;
        if (out_bf16)
            out_bf16[i] = ep_oracle_double_to_bf16(acc);
        if (out_f32)
            out_f32[i] = (float)acc;
    }
}
