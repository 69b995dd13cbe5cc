/*
 * mergepipe.h -- C ABI of the MI355X budgeted-merge library (libmergepipe.so).
 *
 * Budgeted weight-space merging after "Access Sets Matter: Budgeting Expert
 * Reads for Scalable Weight-Space Model Merging": index the per-block expert
 * deltas, build a deterministic access plan A with C_expert(A) <= B, and run
 * the mask-aware merge operator Psi_op over only the selected delta blocks.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Checkpoints.  A checkpoint is ONE flat, contiguous buffer holding the
 *   tensors of an mp_layout back to back, each flattened row-major, in
 *   layout order.  Elements are IEEE fp32 (MP_F32) or bfloat16 (MP_BF16).
 *   The base, the output and every expert share the layout.
 * Blocks (Section 2, the deterministic blocks of each tensor).  Each tensor
 *   is cut into consecutive blocks of layout.block_elems elements; the last
 *   block of a tensor may be shorter; blocks never cross tensors.  Blocks
 *   are numbered g = 0..G-1 in layout order.  They partition the parameter
 *   vector, as Prop. 2 assumes.
 * Units.  An access unit is (expert i, block g), uid = g*K + i (Eq. 2).  Its
 *   read cost c is the stored byte length of the block (Appendix A.1).
 * Masks.  One uint32 word per block, bit i set iff expert i is read for the
 *   block (the access mask A of Eq. 2).  K <= 32.
 * Memory.  Unless stated otherwise pointers are device pointers (memory of
 *   the current HIP device).  `experts` is a HOST array of K pointers; with
 *   residency MP_HOST_PINNED those K pointers are pinned host memory
 *   (hipHostMalloc / pinned torch tensors) and the kernels read expert
 *   blocks straight from it over PCIe -- only the blocks a call touches
 *   cross the link, with no staging copy (the host-to-device feed of
 *   Algorithm 2).  With residency MP_HOST_PAGEABLE they are host memory of
 *   any kind (ordinary pageable allocations included; each must hold the
 *   whole checkpoint, which the library cannot check): the call packs the
 *   blocks it needs into pinned staging buffers on host threads, copies
 *   them to the device on a side stream and runs the kernels over each
 *   staged chunk (Algorithm 2's stage-and-merge pipeline); it returns once
 *   every chunk is enqueued, and the experts are no longer read.  Otherwise
 *   they are device memory.  The caller owns every buffer; the library only
 *   reads inputs and writes the named outputs.  The library keeps a
 *   per-device workspace (block tables, plan scratch, byte counters,
 *   staging buffers) that mp_release() frees.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Work is
 *   enqueued on it; calls return once enqueued unless stated otherwise.
 *   Calls that fill a host-side stats struct synchronise the stream first.
 * Errors.  Every call returns MP_OK (0) or a negative MP_E_* code;
 *   mp_last_error() gives a message (thread-local).  On an argument error,
 *   and on MP_E_NOMEM, nothing is enqueued and no output is written.  On
 *   MP_E_IO (staged residencies) the chunks before the failing one may have
 *   been merged.  Asynchronous device errors surface at the next
 *   synchronising call.  No C++ exception crosses the ABI.
 * Validation (all calls): 1 <= K <= 32; block_elems > 0 and a multiple of
 *   16 / (bytes per element); every tensor numel >= 0 and a multiple of
 *   16 / (bytes per element) (each tensor starts 16-byte aligned);
 *   K * G < 2^32; non-NULL pointers; device buffers must be device memory
 *   large enough for the layout; pinned buffers must be pinned host memory.
 *   `out` must not overlap the base or any expert.
 */
#ifndef MERGEPIPE_H
#define MERGEPIPE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MP_OK 0
#define MP_E_ARG (-1)         /* invalid argument; nothing was done */
#define MP_E_UNSUPPORTED (-2) /* valid request this build does not handle */
#define MP_E_NOMEM (-3)       /* workspace allocation failed */
#define MP_E_HIP (-4)         /* a HIP runtime call failed */
#define MP_E_IO (-5)          /* reading an expert file failed */

typedef enum { MP_F32 = 0, MP_BF16 = 1 } mp_dtype;
typedef enum { MP_DEVICE = 0, MP_HOST_PINNED = 1, MP_HOST_PAGEABLE = 2, MP_HOST_FILE = 3 } mp_residency;
/* OR-ed into `residency`: the expert buffers hold the deltas
 * Delta_i = W_i - W_0 themselves (Section 3's "explicit deltas" source)
 * instead of fine-tuned weights, in the checkpoint dtype.  Then
 * d = fl32(Delta_i): the index reads no base, the merges read the base only
 * to add the merged delta to it.  Everything else is unchanged. */
enum { MP_EXPERTS_DELTA = 16 };
typedef enum { MP_COMBINE_LINEAR = 0, MP_COMBINE_SIGN_ELECT = 1 } mp_combine;
/* mp_plan options (bit flags; 0 is the literal Algorithm 1). */
typedef enum { MP_PLAN_PER_BYTE = 1, MP_PLAN_SKIP_ZERO = 2 } mp_plan_flags;

typedef struct mp_layout {
    int32_t n_tensors;     /* number of tensors (>= 0) */
    int32_t dtype;         /* mp_dtype of every checkpoint */
    const int64_t* numel;  /* HOST array [n_tensors]: elements per tensor */
    int64_t block_elems;   /* block size in elements */
} mp_layout;

typedef struct mp_plan_stats {
    uint64_t budget_bytes; /* B as passed */
    uint64_t cost_bytes;   /* C_expert(A) of the returned mask (<= B) */
    uint64_t full_bytes;   /* C_expert(1) = K * P * bytes per element */
    uint64_t n_selected;   /* units with A = 1 */
    uint64_t n_units;      /* K * G */
    uint64_t digest;       /* selected-block digest of (mask, cost) */
} mp_plan_stats;

typedef struct mp_io_stats {
    uint64_t expert_bytes; /* expert bytes the merge kernels loaded */
    uint64_t base_bytes;   /* base bytes read */
    uint64_t out_bytes;    /* output bytes written */
    uint64_t h2d_bytes;    /* expert bytes moved over PCIe (MP_HOST_PINNED: read by
                              the kernels; MP_HOST_PAGEABLE: staged copies), else 0 */
    uint64_t expert_bytes_by_expert[32]; /* expert_bytes split by expert i (0 past K) */
} mp_io_stats;

/* Number of blocks G of a layout (Section 2's block partition).
 * Host only; enqueues nothing.  Returns MP_E_ARG for an invalid layout. */
int mp_layout_blocks(const mp_layout* layout, int64_t* n_blocks);

/* Catalog statistic (Section 2 "Offline Analyze", Section 3 "Catalog"):
 * for every unit, S = sum over the block of d*d with d = float(x_i) -
 * float(x_0) the fp32 delta, summed in this fixed order: with V = 16 /
 * (bytes per element), 64 partial sums p_l, p_l takes 16-byte chunks
 * l, l+64, l+128, ... of the block in turn and their elements in order,
 * p_l = fma(d, d, p_l) from +0; then for s = 32,16,8,4,2,1 each p_l
 * becomes p_l + p_(l xor s); S = p_0.  (The paper fixes no order; a fixed
 * one makes plans reproducible bit for bit.)
 *   sumsq: device float[G*K], written at uid = g*K + i.
 * Asynchronous on `stream`.  With MP_HOST_PINNED or MP_HOST_PAGEABLE every
 * expert byte crosses PCIe once (the amortised catalog construction). */
int mp_index_blocks(const mp_layout* layout, const void* base,
                    const void* const* experts, int32_t K, int32_t residency,
                    float* sumsq, void* stream);

/* Catalog statistics for TIES (Section 3 "Catalog"; Appendix A.1's trim):
 * for every unit, the per-unit trim threshold
 *   tau[g*K + i] = fp32 bit pattern of the k-th largest |d| of the block
 *                  (multiplicity counted), k = min(n, ceil(density * n)) in
 *                  fp64, n = the block length; all ones (a NaN pattern,
 *                  which no magnitude meets: nothing is kept) if k = 0,
 * and, when sumsq is not NULL, the sum of squares of mp_index_blocks (the
 * same bits) in the same pass.  The threshold depends on the unit and the
 * density only, never on an access mask, so one catalog pass serves TIES
 * merges at every budget (mp_merge_ties_tau).
 *   tau: device uint32[G*K].  sumsq: device float[G*K] or NULL.
 * block_elems must be <= 4096 (MP_E_UNSUPPORTED otherwise).
 * Asynchronous on `stream`; with MP_HOST_PINNED every expert byte crosses
 * PCIe once. */
int mp_index_ties(const mp_layout* layout, const void* base,
                  const void* const* experts, int32_t K, int32_t residency,
                  double density, float* sumsq, uint32_t* tau, void* stream);

/* Algorithm 1 (PlanGen) over all units, budget-feasible by construction
 * (Prop. 1: C_expert(A) <= B):
 *   score  s_u = float(float(w_i * w_i) * S_u), which ranks units as
 *          |w_i| * ||Delta||_2, the retained utility of Section 2;
 *   cost   c_u = block length * bytes per element;
 *   order  decreasing score, ties by increasing uid;
 *   greedy take u iff Chat + c_u <= B, and continue past candidates that
 *          do not fit (skip-and-continue).
 *   sumsq: device float[G*K] from mp_index_blocks.  w: HOST float[K]
 *   (alpha for AVG and DARE-linear, 1 for TIES and sign-elect).
 *   flags: 0, or a combination of
 *     MP_PLAN_PER_BYTE   score per byte read, as Eq. 6 trades utility
 *                        against a byte budget: s_u = float(double(s_u) /
 *                        double(c_u)), one rounding from the fp64 quotient;
 *     MP_PLAN_SKIP_ZERO  units with S_u = 0 are not candidates (their
 *                        block is the base's, up to squares that
 *                        underflow); they are never selected.
 *   Other bits: MP_E_UNSUPPORTED.
 *   mask: device uint32[G], written for every block.
 *   stats: HOST, filled; digest = mix64(D xor Chat) with D = sum over g of
 *   mix64((g << 32) | mask[g]) mod 2^64 and mix64 the SplitMix64 output
 *   function.  B >= full_bytes yields the all-ones mask.
 * Synchronises `stream` before returning (the one blocking point). */
/* sumsq may be NULL when no block catalog exists: the planner then falls
 * back to Section 3's deterministic tensor-level plan.  A unit is (expert
 * i, tensor t), with uid t*K + i and cost the tensor's bytes; every unit's
 * statistic is 1, so the score is float(w_i * w_i) (per byte: divided by
 * the cost as above); tensors without elements are not candidates; the
 * order and the skip-and-continue greedy are those above.  A selected unit
 * sets bit i in the mask word of every block of tensor t: no tensor is
 * split.  The stats describe the block mask (n_selected counts (expert,
 * block) units).  MP_E_UNSUPPORTED if a tensor has 2^32 or more elements. */
int mp_plan(const mp_layout* layout, int32_t K, const float* sumsq,
            const float* w, uint64_t budget_bytes, uint32_t flags,
            uint32_t* mask, mp_plan_stats* stats, void* stream);

/* mp_plan without allocation, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Arguments, results, errors and the final
 * synchronisation are those of mp_plan, and it runs the same kernels: mask
 * and stats are equal bit for bit.  It calls no hipMalloc, hipFree or
 * other allocation routine and keeps no per-layout cache.  Instead, the
 * control block, the layout's tensor sizes (twice), the first block of
 * each tensor, the tensors' selection words, the block lengths and the two
 * candidate lists live in one fixed device array of 16 MiB (16,777,216
 * bytes), which each device the library runs on holds until the process
 * ends.  A layout needs the sum of these sizes, each rounded up to 256
 * bytes: about 19 KB for the control block, 8 * n_tensors, 4 * (n_tensors +
 * 1), twice 4 * n_tensors, 4 * G, and twice 4 * K * max(1, n_tensors) --
 * 1.6 MB for a 1.5B-parameter layout cut into 4096-element blocks, so up
 * to about four million blocks fit.  A larger layout
 * gets MP_E_UNSUPPORTED (with the sizes in mp_last_error) before anything
 * is enqueued.  The array keeps the last call's contents; each call
 * rebuilds everything it reads from it.  Calls hold the library's lock
 * until their stream has finished, so calls from several threads are
 * serialised and never use the array at the same time. */
int mp_plan_noalloc(const mp_layout* layout, int32_t K, const float* sumsq,
                    const float* w, uint64_t budget_bytes, uint32_t flags,
                    uint32_t* mask, mp_plan_stats* stats, void* stream);

/* Coverage of an access mask for the run's manifest (Section 3: the
 * executor records touched blocks and contributing experts).
 * cov: HOST uint64[n_tensors * K]; cov[t*K + i] = number of elements of
 * tensor t in blocks that select expert i (0: expert i contributes nothing
 * to tensor t).  mask: device uint32[G] as written by mp_plan (bits of
 * experts >= K are ignored).  Synchronises `stream` before returning. */
int mp_coverage(const mp_layout* layout, int32_t K, const uint32_t* mask,
                uint64_t* cov, void* stream);

/* Budgeted AVG (Eq. 4 with Appendix A.1's Psi_AVG): per element
 * acc = +0; for selected i in increasing order acc = fma(alpha_i, d_i, acc);
 * out = round(x_0 + acc) (round-to-nearest-even into the checkpoint dtype).
 * alpha: HOST float[K], fixed (no renormalisation over the selected
 * experts).  Unselected experts are never read.  mask: device uint32[G].
 * io: optional (NULL = none); when given the call synchronises `stream`
 * and reports the bytes the kernels loaded and stored (Prop. 1: the expert
 * bytes equal the cost of the mask, since only selected blocks are read). */
int mp_merge_avg(const mp_layout* layout, const void* base,
                 const void* const* experts, int32_t K, int32_t residency,
                 const uint32_t* mask, const float* alpha, void* out,
                 mp_io_stats* io, void* stream);

/* Selected-only budgeted AVG (Appendix A.1, the variant that renormalises
 * an additive merge over the selected experts; the coefficient-drift bound
 * there, not Prop. 2's omission bound, describes its error).  Per block g:
 * s_g = sum of alpha_i over the experts selected in g (fp32 adds from +0,
 * increasing i); beta_i = alpha_i / s_g (IEEE fp32 division) for a
 * selected i; s_g = 0 gives no coefficients (the block keeps the base).
 * Then per element as mp_merge_avg with beta in place of alpha.  Arguments,
 * residencies, reads and io as mp_merge_avg. */
int mp_merge_avg_renorm(const mp_layout* layout, const void* base,
                        const void* const* experts, int32_t K, int32_t residency,
                        const uint32_t* mask, const float* alpha, void* out,
                        mp_io_stats* io, void* stream);

/* Budgeted TIES (Appendix A.1: trim, sign election and disjoint mean over
 * the masked deltas).  Trim is per selected (expert, block): k = min(n,
 * ceil(density * n)) in fp64, tau = the k-th largest |d| of the block; d is
 * kept iff |d| >= tau and |d| > 0.  Per element, over the selected experts
 * in increasing order: P = sum of the positive kept d, N = sum of the
 * negative kept d (fp32 adds from +0), with their counts; the elected sign
 * compares the two rounded sums: + if fl32(P) > -fl32(N), - if
 * fl32(P) < -fl32(N), none if equal (the paper fixes no summation order;
 * this can differ from the sign of the exact sum: kept deltas
 * (1, -1, 2^-25) elect none); mean = P / count(+), N / count(-) or 0;
 * out = round(fma(lambda, mean, x_0)).  0 <= density <= 1.
 * block_elems must be <= 4096 (MP_E_UNSUPPORTED otherwise). */
int mp_merge_ties(const mp_layout* layout, const void* base,
                  const void* const* experts, int32_t K, int32_t residency,
                  const uint32_t* mask, double density, float lambda, void* out,
                  mp_io_stats* io, void* stream);

/* TIES trim thresholds at tensor scope (the per-tensor variant of
 * Appendix A.1's trim after masking): for each unit (g, i),
 * tau[g*K + i] = the k-th largest |d| pattern over the zero-completed
 * masked deltas of expert i in block g's tensor t (unselected blocks count
 * as zeros and are not read), k = min(n_t, ceil(density * n_t)) in fp64
 * over the tensor's n_t elements; 0 when fewer than k elements of t are
 * selected; all ones (nothing kept) when k = 0.  mp_merge_ties_tau with
 * these thresholds is the tensor-scope TIES merge.  mask: device uint32[G]
 * (the mask the merge will use); tau: device uint32[G*K].  Residency
 * MP_DEVICE or MP_HOST_PINNED (MP_E_UNSUPPORTED for MP_HOST_PAGEABLE),
 * optionally with MP_EXPERTS_DELTA.  Runs on `stream` and returns once the
 * thresholds are complete: the kernels share one scratch area per device,
 * so calls on different streams run one after the other, and a selection
 * that finds no cut (an internal error, never expected) returns MP_E_HIP
 * with tau unspecified. */
int mp_ties_tensor_thresholds(const mp_layout* layout, const void* base,
                              const void* const* experts, int32_t K, int32_t residency,
                              const uint32_t* mask, double density, uint32_t* tau,
                              void* stream);

/* Budgeted TIES with catalog thresholds: as mp_merge_ties, with d kept
 * iff |d| >= float(tau[g*K + i]) and |d| > 0 for the selected unit (g, i).
 * With the thresholds of mp_index_ties for a density the result equals
 * mp_merge_ties at that density bit for bit.  tau: device uint32[G*K].
 * Any block size. */
int mp_merge_ties_tau(const mp_layout* layout, const void* base,
                      const void* const* experts, int32_t K, int32_t residency,
                      const uint32_t* mask, const uint32_t* tau, float lambda,
                      void* out, mp_io_stats* io, void* stream);

/* Budgeted DARE (Appendix A.1: random drop and rescale with a fixed seed).
 * Element e of tensor t of expert i is dropped iff u < floor(p * 2^16),
 * u = the 16-bit draw h = e mod 8 of Philox4x32-10 (Salmon et al., SC 2011)
 * with key (seed, i) and counter (low32(e/8), high32(e/8), t, 0): bits
 * 16 (h mod 2) .. 16 (h mod 2) + 15 of output word h / 2.  The decision
 * never depends on the mask.  Kept deltas become float(d * s), s = float(1/(1-p)).
 * combine MP_COMBINE_LINEAR: acc = fma(alpha_i, t_i, acc) over selected i
 * increasing, out = round(fma(lambda, acc, x_0)).  MP_COMBINE_SIGN_ELECT:
 * TIES's sign election and disjoint mean (no trim); alpha is ignored and
 * may be NULL.  0 <= p < 1. */
int mp_merge_dare(const mp_layout* layout, const void* base,
                  const void* const* experts, int32_t K, int32_t residency,
                  const uint32_t* mask, double p, uint32_t seed, int32_t combine,
                  const float* alpha, float lambda, void* out, mp_io_stats* io,
                  void* stream);

/* One low-rank adapter record (Section 3: the delta iterator's LoRA-style
 * adapters, Hu et al. 2022).  Tensor `tensor` of the layout, viewed as a
 * rows x cols row-major matrix (rows * cols = its numel), has the delta
 * scale * B A, with A (rank x cols) and B (rows x rank) row-major in the
 * layout's dtype at element offsets a_off and b_off of each expert's
 * adapter buffer.  1 <= rank <= 64; cols a multiple of 4; numel < 2^32;
 * 0 <= a_off, b_off <= 2^48; scale finite; each tensor at most once.
 * Zero-initialise the struct (its tail padding is ignored either way). */
typedef struct mp_lora_tensor {
    int32_t tensor;
    int32_t rank;
    int64_t rows;
    int64_t cols;
    int64_t a_off;
    int64_t b_off;
    float scale;
} mp_lora_tensor;

/* Deltas drawn from adapters (Section 3, the executor's delta iterator):
 * writes expert i's delta of every selected unit (g, i) -- every unit when
 * mask is NULL -- into deltas[i], an explicit-delta checkpoint (layout
 * order, layout dtype) for the MP_EXPERTS_DELTA residency bit.  For an
 * adapted tensor, element (r, c) is float(scale * y) rounded to the dtype
 * (to nearest even), y the fp32 sum over k of B[r][k] * A[k][c] computed on
 * the matrix cores (exact products, fp32 accumulation; equal to the
 * correctly rounded sum whenever every partial sum is exact in fp32).
 * Tensors without a record get zeros.  Elements of unselected units are not
 * written.  adapters: HOST array of K device pointers (each at least the
 * largest a_off + rank*cols, b_off + rows*rank elements; the array may be
 * NULL when n_lora = 0); deltas: HOST array of K device checkpoints,
 * disjoint from each other and from the adapters; mask: device uint32[G]
 * or NULL.  The caller owns every buffer; the library reads the adapters
 * and the mask and writes only the named elements of deltas.  Errors:
 * MP_E_ARG for an invalid layout, K, record, NULL array, undersized or
 * non-device buffer, or overlap (checked before anything is enqueued);
 * MP_E_UNSUPPORTED for tensors of 2^32 or more elements; MP_E_NOMEM or
 * MP_E_HIP from the table upload, the table's scratch or the launch.
 * Records are validated and their device table is cached per (device,
 * layout, records) until mp_release.  The table also holds scratch: with a
 * mask, the row lists (the rows meeting a selected block); without one, when
 * every adapted tensor's rows are whole 16-byte chunks, an operand-order copy
 * of the adapters (K x about 2 x the adapter elements) that the pull runs
 * on.  So a call's stream first waits for the previous call that used the
 * same table's scratch (this entry point or mp_lora_merge_ties_tau), on
 * whatever stream it ran.  Asynchronous on `stream`. */
int mp_lora_materialize(const mp_layout* layout, const mp_lora_tensor* loras, int32_t n_lora,
                        const void* const* adapters, int32_t K, const uint32_t* mask,
                        void* const* deltas, void* stream);

/* Budgeted TIES from catalog thresholds with the experts given as adapters
 * (Section 3's delta iterator feeding the executor, Algorithm 2 with the
 * merge operator of Appendix A.1): the result of mp_lora_materialize(mask)
 * followed by mp_merge_ties_tau(MP_DEVICE | MP_EXPERTS_DELTA, mask, tau,
 * lambda) on those deltas, bit for bit wherever the base is finite (the
 * explicit-delta merge forms x - 0 * x0, which is NaN where x0 is not), but
 * with no delta checkpoint: each selected unit's deltas are computed by the
 * same matrix-core tiles, rounded to the dtype as the pull stores them, and
 * trimmed, elected and averaged in registers.  Writes every element of out.
 * base, out: device checkpoints (layout order and dtype); out must not
 * overlap base, an adapter, mask or tau.  adapters, loras, n_lora and K as
 * for mp_lora_materialize; mask: device uint32[G]; tau: device uint32[G*K]
 * (from mp_index_ties on the deltas, or mp_ties_tensor_thresholds).
 * MP_E_UNSUPPORTED when an adapted bf16 tensor's columns are not a multiple
 * of 8 (then use the two calls); MP_E_ARG as for the two calls, or for a
 * non-finite lambda; MP_E_NOMEM if the operand-order copy of the adapters
 * (kept with the record table, as for mp_lora_materialize's full pull, whose
 * ordering across streams applies here too) does not fit the workspace cap.
 * Asynchronous on `stream`. */
int mp_lora_merge_ties_tau(const mp_layout* layout, const void* base, const mp_lora_tensor* loras,
                           int32_t n_lora, const void* const* adapters, int32_t K,
                           const uint32_t* mask, const uint32_t* tau, float lambda, void* out,
                           void* stream);

/* Measurement aid, not part of the method: a plain stream copy of `bytes`
 * bytes (a multiple of 16, at most 2^40) from device memory src to device
 * memory dst, which must not overlap, with the merge kernels' access pattern
 * (16-byte non-temporal loads and stores, one chunk per lane) and none of
 * their arithmetic.  Timing it gives the HBM rate the device reaches on a
 * read-once, write-once stream, the practical ceiling beside the published
 * peak.  MP_E_ARG for a null, non-device or too small buffer, a size that is
 * not a multiple of 16, or overlapping buffers; MP_E_HIP if the launch fails.
 * Asynchronous on `stream`. */
int mp_stream_copy(const void* src, void* dst, uint64_t bytes, void* stream);

/* Staging for MP_HOST_PAGEABLE: the bytes of each of the two pinned host
 * buffers (and of their two device counterparts) that chunks of packed
 * expert blocks pass through; default 256 MiB, rounded down to 256 bytes.
 * Takes effect at the next host-pageable call (buffers are reallocated).
 * MP_E_ARG outside [1 MiB, 4 GiB]. */
int mp_set_stage_bytes(uint64_t bytes);

/* Cap on the library's cached workspace (block tables, plan scratch, byte
 * counters, staging buffers: the device and pinned host memory it keeps
 * between calls), in bytes; 0 (the default) means no cap.  A call whose
 * workspace allocation would pass the cap returns MP_E_NOMEM before it
 * enqueues anything, writing no output; memory already held is kept (free
 * it with mp_release).  Takes effect at the next allocation. */
int mp_set_workspace_limit(uint64_t bytes);

/* Bytes of workspace the library holds now (all devices). */
uint64_t mp_workspace_bytes(void);

/* Fault injection for tests of the staged residencies (MP_HOST_PAGEABLE,
 * MP_HOST_FILE): with the environment variable MP_FAULT_PACK_CHUNK=n set
 * when a staged call runs, the pack of its chunk n (0-based; a chunk that
 * packs at least one block) reports a failed read, as an unreadable expert
 * file does: the call returns MP_E_IO after the kernels of chunks 0..n-1
 * were enqueued, so outputs may be partly written.
 * With MP_FAULT_TENSOR_NO_CUT=1 set, mp_ties_tensor_thresholds sends its
 * first (expert, tensor) pair down the no-cut error path: the kernels finish
 * normally and the call returns MP_E_HIP. */

/* Message for the last failing call on this thread ("" if none). */
const char* mp_last_error(void);

/* Free the library's cached per-device workspaces.  No call may be in
 * flight on any stream. */
void mp_release(void);

#ifdef __cplusplus
}
#endif
#endif /* MERGEPIPE_H */
