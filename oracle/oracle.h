/*
 * oracle.h -- plain CPU oracle for budgeted weight-space merging
 * ("Access Sets Matter: Budgeting Expert Reads for Scalable Weight-Space
 * Model Merging").
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no source
 * with the GPU library and is written to be read against the paper, not to
 * be fast.
 *
 * Conventions (the readings of the paper this oracle takes):
 *  - dtype 0 = IEEE fp32, dtype 1 = bfloat16 (raw 16-bit patterns).
 *  - A "block list" describes the blocks to process: for block b, its data
 *    starts at element doff[b] of every checkpoint buffer passed and holds
 *    len[b] elements; tensor[b] / elem0[b] give its tensor id and the index,
 *    inside that tensor, of its first element (only the DARE drop mask needs
 *    them).  Full-checkpoint calls pass doff = the block's checkpoint offset.
 *  - Masks are one uint32 word per block, bit i = expert i selected.
 *  - Return value 0 = ok, negative = invalid argument.
 */
#ifndef MERGEPIPE_ORACLE_H
#define MERGEPIPE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Block partition (Section 2: deterministic blocks of each tensor). */
int64_t orc_num_blocks(int32_t n_tensors, const int64_t* numel, int64_t block_elems);
int orc_blocks(int32_t n_tensors, const int64_t* numel, int64_t block_elems,
               int64_t* off, int64_t* len, int32_t* tensor, int64_t* elem0);

/* Per-(block, expert) sum of squared deltas, canonical fp32 order.
 * sumsq[b*K + i]. */
int orc_index(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
              const void* base, const void* const* experts, int32_t K, float* sumsq);

/* Algorithm 1 (PlanGen), literal: score, sort, skip-and-continue greedy
 * over the (expert, block) units of a block catalog (sumsq, not NULL).
 * flags: 1 = score per byte of cost, 2 = units with a zero sum of squares
 * are not candidates.  stats[0]=selected cost, [1]=selected units, [2]=full
 * cost, [3]=digest, [4]=number of units. */
int orc_plan(int64_t G, const int64_t* len, int32_t dtype, int32_t K,
             const float* sumsq, const float* w, uint64_t budget, uint32_t flags,
             uint32_t* mask, uint64_t* stats);

/* Section 3's deterministic tensor-level fallback when block metadata are
 * missing: Algorithm 1 over (expert, tensor) units with statistic 1 (score
 * w_i^2, ties by tensor then expert), cost = the tensor's bytes; a selected
 * unit sets the expert's bit in every block of the tensor.  mask: [G]
 * block words; stats as orc_plan's, for the block mask. */
int orc_plan_tensors(int32_t n_tensors, const int64_t* numel, int64_t block_elems, int32_t dtype,
                     int32_t K, const float* w, uint64_t budget, uint32_t flags, uint32_t* mask,
                     uint64_t* stats);

/* Mask-aware merge operators (Eq. 4 with Appendix A.1's operators). */
int orc_merge_avg(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                  const void* base, const void* const* experts, int32_t K,
                  const uint32_t* mask, const float* alpha, void* out);
/* Selected-only AVG: the coefficients renormalised over each block's
 * selected experts (Appendix A.1's coefficient-drift variant). */
int orc_merge_avg_renorm(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                         const void* base, const void* const* experts, int32_t K,
                         const uint32_t* mask, const float* alpha, void* out);
int orc_merge_ties(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                   const void* base, const void* const* experts, int32_t K,
                   const uint32_t* mask, double density, float lambda, void* out);
int orc_merge_dare(int64_t nb, const int64_t* doff, const int64_t* len,
                   const int32_t* tensor, const int64_t* elem0, int32_t dtype,
                   const void* base, const void* const* experts, int32_t K,
                   const uint32_t* mask, double p, uint32_t seed, int32_t combine,
                   const float* alpha, float lambda, void* out);

/* TIES trim thresholds per unit (mask-independent): tau[b*K + i] = fp32
 * pattern of the k-th largest |d| of unit (block b, expert i), k =
 * orc_ties_k(len, density); all ones (a NaN pattern: nothing kept) when
 * k = 0. */
int orc_ties_thresholds(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                        const void* base, const void* const* experts, int32_t K, double density,
                        uint32_t* tau);
/* Per-tensor trim thresholds over the zero-completed masked deltas:
 * tau_t[t*K + i] = the k-th largest |d| pattern of tensor t for expert i,
 * k = orc_ties_k(n_t, density); 0 when fewer than k elements are selected;
 * all ones when k = 0.  tensor[b]: tensor id of block b (consecutive). */
int orc_ties_tensor_thresholds(int64_t nb, const int64_t* doff, const int64_t* len, const int32_t* tensor,
                               int32_t n_tensors, int32_t dtype, const void* base, const void* const* experts,
                               int32_t K, const uint32_t* mask, double density, uint32_t* tau_t);
/* TIES with given thresholds (keep iff |d| >= float(tau) and |d| > 0). */
int orc_merge_ties_tau(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                       const void* base, const void* const* experts, int32_t K,
                       const uint32_t* mask, const uint32_t* tau, float lambda, void* out);

/* One tensor's delta from a LoRA adapter (Section 3's low-rank delta
 * source): out[r*cols + c] = fl32(scale * y) in the checkpoint dtype, y the
 * fp32 rounding of sum_k B[r*rank + k] * A[k*cols + c] (exact products,
 * summed in fp64).  A: rank x cols, B: rows x rank, row-major, checkpoint
 * dtype (no ORC_DELTA bit). */
int orc_lora_delta(int32_t dtype, int64_t rows, int64_t cols, int32_t rank, const void* A, const void* B,
                   float scale, void* out);

/* Building blocks exposed so the tests can pin them. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
uint64_t orc_mix64(uint64_t x);
void orc_round_bf16(const float* x, uint16_t* y, int64_t n);
int64_t orc_ties_k(int64_t n, double density);
int orc_num_threads(void);
/* Threads of the following parallel loops (results do not depend on it). */
void orc_set_num_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
