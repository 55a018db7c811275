/*
 * ep_oracle.h -- plain, slow, obviously correct CPU oracle for MoE expert-parallel
 * token dispatch and combine (one rank's share).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link, load or
 * call this code: only the tests, the smoke check and the benchmark's CPU-baseline leg
 * use it.  It shares no source, header, table or helper with the GPU library.
 *
 * What it computes (Lee et al., "Efficient Expert-Parallel Communication on
 * PCIe-Connected Consumer GPUs"):
 *   - Sec. 2.1 (Distributed MoE; communication patterns of dispatch and combine):
 *     each token is sent to the devices that hold its k selected experts, and the
 *     expert outputs are returned to the token's owner and combined.
 *   - Sec. 2.2 (Data transfer mechanisms): a DMA engine moves only contiguous
 *     regions, so tokens at routing-dependent places are first packed contiguously.
 *   - Sec. 4.3 (DMA engine-based communication): tokens are grouped by expert before
 *     the expert computation, and the returned contributions of a token are added up
 *     on the GPU that owns it, in token order.
 *   - Sec. 4.5 (Routing-aware communication): only the rows each destination needs
 *     are sent (one row per (token, selected expert)).
 *
 * Conventions (readings of points the paper leaves open):
 *   - Experts are placed contiguously: rank r holds experts [r*L, (r+1)*L), L = E/R.
 *   - Rows inside an expert group are ordered by ascending flat slot index t*k+j
 *     (a stable counting sort of the routing array by expert id).
 *   - Counts count slots (token, expert) pairs: they sum to T*k.
 *   - combine: out[t] = sum_j w[t][j] * y[slot_pos[t*k+j]], accumulated in double,
 *     rounded once (to nearest, ties to even) to bf16 or float.
 *
 * bf16 values are passed as uint16_t bit patterns.  All byte offsets are 64-bit.
 */
#ifndef EP_ORACLE_H
#define EP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { EP_ORACLE_OK = 0, EP_ORACLE_INVALID_ARG = 1, EP_ORACLE_BAD_ROUTING = 2 };

/* Layout of the dispatch (Sec. 4.3 grouping; Sec. 4.5 routing-aware rows).
 * topk_idx: int32 [T][k] row-major.  Outputs (caller-owned host arrays):
 *   expert_counts[E], expert_offsets[E+1], rank_counts[R], rank_offsets[R+1],
 *   slot_pos[T*k] (packed row of slot t*k+j), row_src[T*k] (inverse; may be NULL).
 * Returns EP_ORACLE_INVALID_ARG for bad sizes, EP_ORACLE_BAD_ROUTING when an expert id
 * is outside [0,E) or repeated within a token row (outputs then unspecified). */
int ep_oracle_layout(const int32_t *topk_idx, int64_t T, int32_t k, int32_t E, int32_t R,
                     int32_t *expert_counts, int32_t *expert_offsets,
                     int32_t *rank_counts, int32_t *rank_offsets,
                     int32_t *slot_pos, int32_t *row_src);

/* Pack (Sec. 2.2): packed[slot_pos[t*k+j]][:] = x[t][:], a byte copy.
 * x: bf16 [T][H]; packed: bf16 [T*k][H]. */
void ep_oracle_pack(const uint16_t *x, int64_t T, int32_t H, int32_t k,
                    const int32_t *slot_pos, uint16_t *packed);

/* Combine (Sec. 4.3 GPU-side reduction of the returned contributions):
 *   exact[t][h] = sum_{j<k} w[t][j] * y[slot_pos[t*k+j]][h]   (double)
 * y: bf16 [*][H] in packed order; w: float [T][k].  A slot with slot_pos < 0 (not routed
 * to this rank, see ep_oracle_local_layout) contributes nothing, so over the gathered
 * tokens of the dense design this gives each shard's partial block (Sec. 4.2: a GPU's
 * contribution to an output shard).  Any output pointer may be NULL:
 *   out_exact: double [T][H]; out_bf16: bf16 [T][H] (exact rounded to nearest-even);
 *   out_f32: float [T][H] (exact rounded to nearest-even). */
void ep_oracle_combine(const uint16_t *y, const int32_t *slot_pos, const float *topk_w,
                       int64_t T, int32_t H, int32_t k,
                       double *out_exact, uint16_t *out_bf16, float *out_f32);

/* Receive-side grouping of the dense design (Sec. 4.3: each GPU groups the tokens it
 * gathered by the experts it owns): the stable counting sort of ep_oracle_layout over N
 * gathered tokens, restricted to the local experts [e_lo, e_hi).  Slots naming another
 * expert get slot_pos = -1 and are not counted.  Outputs: local_counts[L],
 * local_offsets[L+1] (L = e_hi - e_lo), slot_pos[N*k], row_src[local rows] (may be NULL).
 * Returns EP_ORACLE_INVALID_ARG unless 0 <= e_lo < e_hi <= E, EP_ORACLE_BAD_ROUTING for
 * an id outside [0,E) or repeated within a token row. */
int ep_oracle_local_layout(const int32_t *topk_idx, int64_t N, int32_t k, int32_t E, int32_t e_lo,
                           int32_t e_hi, int32_t *local_counts, int32_t *local_offsets,
                           int32_t *slot_pos, int32_t *row_src);

/* Block reduction of the Reduce-Scatter (Sec. 4.2: the destination sums the blocks of the
 * other GPUs with its own):  exact[i] = sum_{d<R} blocks[d*n + i]  (double), i < n.
 * Any output pointer may be NULL; rounding as in ep_oracle_combine. */
void ep_oracle_block_reduce(const double *blocks, int32_t R, int64_t n, double *out_exact,
                            uint16_t *out_bf16, float *out_f32);

/* bf16 <-> double.  bf16 = sign, 8 exponent bits, 7 fraction bits (the upper half of an
 * IEEE-754 binary32).  The narrowing rounds to nearest, ties to even; NaN stays NaN. */
double ep_oracle_bf16_to_double(uint16_t b);
uint16_t ep_oracle_double_to_bf16(double v);

/* Element-wise ep_oracle_double_to_bf16 over n values. */
void ep_oracle_double_to_bf16_n(const double *v, int64_t n, uint16_t *out);

/* Host threads over which ep_oracle_pack and ep_oracle_combine split their tokens (1 by
 * default: the plain single-threaded oracle).  Each token's rows and sums are computed by
 * one thread exactly as in the single-threaded loops, so the outputs do not depend on the
 * count.  Returns the count in effect (1 when the library was built without OpenMP). */
int ep_oracle_set_threads(int threads);

#ifdef __cplusplus
}
#endif

#endif /* EP_ORACLE_H */
