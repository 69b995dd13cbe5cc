// Internal declarations shared by the host runtime and the kernel files of
// libmergepipe.so.  Not part of the public ABI (include/mergepipe.h).
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/mergepipe.h"

namespace mp {

constexpr int kMaxK = 32;
constexpr int kTiesMaxBlock = 4096;  // elements per block the TIES kernel holds in registers

// K expert base pointers, passed to kernels by value.
struct ExpertPtrs {
    const void* p[kMaxK];
};

// Per-expert fp32 coefficients, passed to kernels by value.
struct Coeffs {
    float v[kMaxK];
};

// Device-resident description of a layout's block partition (one per
// (device, layout) pair, cached by the runtime).
struct BlockTable {
    int device = -1;
    int32_t dtype = 0;
    int32_t esize = 0;       // bytes per element
    int64_t block_elems = 0;
    int64_t n_tensors = 0;
    int64_t G = 0;           // number of blocks
    int64_t P = 0;           // elements per checkpoint
    uint32_t max_len = 0;    // longest block
    int n_distinct_len = 0;  // distinct block lengths (bounds the plan rounds)
    int64_t n_short = 0;     // blocks shorter than block_elems
    std::vector<int64_t> numel;
    // host copies
    std::vector<uint64_t> h_off;
    std::vector<uint32_t> h_len;
    // device arrays [G]
    uint64_t* d_off = nullptr;     // element offset of the block in a checkpoint
    uint32_t* d_len = nullptr;     // elements in the block
    uint32_t* d_tensor = nullptr;  // tensor id
    uint64_t* d_elem0 = nullptr;   // index of the block's first element inside its tensor
    // runs of at most kChunkBlocks consecutive blocks of one tensor: {g0, g1 (end), tensor, 0}
    int64_t n_chunks = 0;
    uint4* d_chunk = nullptr;
    uint64_t* d_tnumel = nullptr;  // elements per tensor [n_tensors]
    // the tensor-level plan (no block catalog): elements per tensor as u32
    // (valid when every tensor has fewer than 2^32), their distinct values,
    // and the first block of every tensor [n_tensors + 1]
    uint32_t* d_tlen = nullptr;
    uint32_t* d_g0 = nullptr;
    int n_distinct_tlen = 0;
    bool tlen_fits = true;
};

constexpr int kChunkBlocks = 16;

// Device control block of the plan (see k_plan.hip).
struct PlanCtl;

// Per-device plan scratch.
struct PlanScratch {
    PlanCtl* ctl = nullptr;
    uint32_t* list[2] = {nullptr, nullptr};  // candidate uid lists for the later rounds
    int64_t list_cap = 0;
    uint32_t* tmask = nullptr;  // tensor-level plan: selection word per tensor
    int64_t tmask_cap = 0;
    uint64_t* h_stats = nullptr;  // pinned host mirror of the stats
};

// ---------------------------------------------------------------- workspace memory
// Every cached device or pinned-host allocation of the library goes through
// these, which count the bytes held and refuse (hipErrorOutOfMemory) an
// allocation that would pass the limit set by mp_set_workspace_limit
// (0: none).  Callers hold the library's lock.
hipError_t ws_malloc(void** p, size_t bytes);
hipError_t ws_host_malloc(void** p, size_t bytes);
void ws_free(void* p);
void ws_host_free(void* p);

// ---------------------------------------------------------------- launchers
// All launchers enqueue on `s` and return the launch status.

// Expert pointers are device addresses: device memory or the device view of
// pinned host memory (the kernels then read over PCIe).
hipError_t launch_index(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K,
                        float* sumsq, hipStream_t s, bool delta = false);

// Index plus the per-unit TIES thresholds for `density` (sumsq may be null).
// Blocks must hold at most kTiesMaxBlock elements.
hipError_t launch_index_ties(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K,
                             double density, float* sumsq, uint32_t* tau, hipStream_t s, bool delta = false);

// Algorithm 1 without allocation (k_plan.hip): everything the kernels need
// beyond the caller's buffers lives in a fixed device array of
// static_plan_limit() bytes.  static_plan_bytes() is what a layout needs;
// static_plan_scratch() returns the array's address on the current device
// (looked up once per device); launch_plan_static() enqueues the plan on it,
// reads the seven stats words back into `stats` and synchronises `s`.
int64_t static_plan_bytes(int64_t n_tensors, int64_t G, int64_t n_short, int K);
int64_t static_plan_limit();
hipError_t static_plan_scratch(void** ptr);
hipError_t launch_plan_static(void* ws, const int64_t* numel, int32_t n_tensors, int64_t block_elems, uint32_t es,
                              int64_t G, int64_t n_short, int K, const float* sumsq, const Coeffs& w, uint32_t flags,
                              uint64_t budget, uint64_t full_bytes, uint32_t* mask, uint64_t* stats,
                              hipStream_t s);

// Touched elements per (tensor, expert) of a mask: cov[t * K + i] (device;
// k_plan.hip).
hipError_t launch_coverage(const BlockTable& bt, int K, const uint32_t* mask, unsigned long long* cov,
                           hipStream_t s);

// Algorithm 1 on the device (k_plan.hip).  sumsq null: the tensor-level
// plan of Section 3's fallback (units (expert, tensor), statistic 1), which
// needs ps.tmask for n_tensors words and lists of K * n_tensors uids.
hipError_t launch_plan(const BlockTable& bt, PlanScratch& ps, int K, const float* sumsq,
                       const Coeffs& w, uint32_t flags, uint64_t budget, uint64_t full_bytes, uint32_t* mask,
                       hipStream_t s);

// TIES thresholds at tensor scope (k_tensor_ties.hip): per unit (g, i) the
// k-th largest |d| of tensor(g)'s zero-completed masked deltas of expert i.
// hist: device uint32[K * n_tensors * 2048], state: device uint4[K * n_tensors
// + 1]; the word after the pairs' states is set to nonzero if a selection
// found no cut (an internal error).  force_no_cut: a test hook that sends
// the first pair down that error path (the kernels still finish normally).
hipError_t launch_ties_tensor(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K,
                              const uint32_t* mask, double density, uint32_t* tau, uint32_t* hist, uint4* state,
                              hipStream_t s, bool delta, bool force_no_cut);

// ---------------------------------------------------------------- LoRA source (k_lora.hip)
constexpr int kMaxLoraRank = 64;

// Expert output pointers (the explicit-delta checkpoints written), by value.
struct OutPtrs {
    void* p[kMaxK];
};

// One adapted tensor on the device; its 64-row bands are workgroups
// tile0 .. tile0 + ceil(rows / 64) - 1 of the launch.
struct LoraDesc {
    uint64_t toff;  // element offset of the tensor in a checkpoint
    uint64_t a_off, b_off;  // element offsets of A and B in an adapter buffer
    uint32_t rows, cols, rank;
    float scale;
    uint32_t g0;  // the tensor's first block
    uint32_t tiles_n;  // 128-column tiles per band
    uint32_t tile0;
    uint32_t vec;  // every row of A starts 16-byte aligned (relative to the adapter buffer)
    uint32_t r0;   // the tensor's first entry in a row list (rows of the earlier tensors)
    uint64_t at_off, bp_off;  // element offsets of A^T and B in one expert's operand-order copy
};

// A validated set of adapter records for a layout, cached per device.
struct LoraTable {
    LoraDesc* d_desc = nullptr;  // sorted by tile0
    int n_desc = 0;
    uint32_t n_tiles = 0;  // row bands (workgroups per expert)
    uint32_t* d_zero = nullptr;  // blocks of tensors without an adapter
    uint32_t n_zero = 0;
    uint32_t rows_total = 0;     // rows of all adapted tensors
    uint32_t* d_rl = nullptr;    // masked pulls: the listed rows, K x rows_total (grown on demand)
    uint32_t* d_rc = nullptr;    //   and their counts, K x n_desc
    int rl_k = 0;                // experts the two arrays hold
    hipEvent_t ev = nullptr;     // recorded after each masked pull: the next one (any stream) waits for it
    uint32_t max_rank = 0;       // the largest adapter rank
    bool rows_chunked = true;    // every adapted tensor's rows are a whole number of 16-byte chunks
    uint32_t max_cols = 0;       // the widest adapted tensor
    uint32_t prep_rank = 16;     // depth of the operand-order copy (16 or kMaxLoraRank)
    uint64_t prep_elems = 0;     // elements of one expert's operand-order copy
    uint32_t prep_z = 1;         // 128-column (and 128-row) slices of the widest (tallest) adapted tensor
    void* d_prep = nullptr;      // the fused merge's operand-order copies, prep_k x prep_elems (grown on demand)
    int prep_k = 0;
};

// Row bands of a rows x cols tensor; *tiles_n receives the column tiles per band.
uint32_t lora_bands(uint32_t rows, uint32_t cols, uint32_t* tiles_n);

// Writes the selected units' deltas (all units when mask is null).  A masked
// pull needs lt.d_rl and lt.d_rc for at least K experts; a full pull with
// prep (K buffers of lt.prep_elems elements, rewritten) runs on the
// operand-order copy.
hipError_t launch_lora(const BlockTable& bt, const LoraTable& lt, const ExpertPtrs& ad, const OutPtrs& dl, int K,
                       const uint32_t* mask, hipStream_t s, const OutPtrs* prep = nullptr);
// The budgeted TIES merge from stored thresholds with every delta drawn from
// the adapters inside the merge (no delta checkpoint).
// prep: K device buffers of lt.prep_elems elements each, rewritten by the call.
hipError_t launch_lora_ties(const BlockTable& bt, const LoraTable& lt, const ExpertPtrs& ad, const OutPtrs& prep,
                            int K, const void* base, const uint32_t* mask, const uint32_t* tau, float lambda,
                            void* out, hipStream_t s);

// Merge operators.  `counters` is null or a device array of 256 uint64
// accumulating the expert bytes the kernels load: slot (block mod 8) * 32 + i
// holds expert i's.
enum class Op { AVG = 0, TIES = 1, DARE_LINEAR = 2, DARE_SIGN = 3, TIES_TAU = 4, AVG_RENORM = 5 };

struct MergeArgs {
    Op op = Op::AVG;
    Coeffs alpha{};
    double density = 0.0;
    float lambda = 1.0f;
    double p = 0.0;
    uint32_t seed = 0;
    const uint32_t* tau = nullptr;  // TIES_TAU: per-unit thresholds [G*K]
    float bsub = 1.0f;  // d = x_i - bsub * x_0: 1 for fine-tuned weights, 0 for explicit deltas
};

hipError_t launch_merge(const BlockTable& bt, const MergeArgs& a, const void* base,
                        const ExpertPtrs& ex, int K, const uint32_t* mask, void* out,
                        unsigned long long* counters, hipStream_t s);

// The merge over blocks [b0, b0 + nb) with the selected expert blocks staged
// in device memory: block b0 + j's selected experts lie back to back, in
// increasing expert order, from stage + soff[j].
hipError_t launch_merge_staged(const BlockTable& bt, const MergeArgs& a, const void* base, int K,
                               const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s,
                               const void* stage, const uint64_t* soff, int64_t b0, int64_t nb);

// Stream copy of nbytes (a multiple of 16, at most 2^40) of device
// memory (k_copy.hip).
hipError_t launch_stream_copy(const void* src, void* dst, uint64_t nbytes, hipStream_t s);

// z with P(|Z| > z) = rho for a standard normal Z (0 unless 0 < rho < 1);
// scales the TIES kernels' first guess at a trim threshold (k_index.hip).
double normal_two_sided_quantile(double rho);

// The TIES merge that selects its trim thresholds itself (k_merge_ties.hip);
// launch_merge and launch_merge_staged forward Op::TIES here.
hipError_t launch_merge_ties(const BlockTable& bt, const MergeArgs& a, const void* base, const ExpertPtrs& ex, int K,
                             const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s);
hipError_t launch_merge_ties_staged(const BlockTable& bt, const MergeArgs& a, const void* base, int K,
                                    const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s,
                                    const void* stage, const uint64_t* soff, int64_t b0, int64_t nb);

// ---------------------------------------------------------------- host experts (stage.hip)
// Expert checkpoints on the host: memory (ptr[i]) or files (fd[i], read
// with pread).  read() copies bytes [pos, pos + n) of expert i; a failed
// file read sets `failed` and returns false.
struct HostExperts {
    const void* const* ptr = nullptr;
    const int* fd = nullptr;
    mutable std::atomic<int> failed{0};
    bool read(int i, void* dst, size_t pos, size_t n) const;
};

// Experts in host memory of any kind, streamed through pinned staging
// buffers; h2d receives the bytes copied to the device.  The functions
// return once every chunk is enqueued on `s` (the experts are no longer
// read); staging buffers are reused by the next call after its kernels.
void set_stage_bytes(size_t bytes);
void release_stagers();
hipError_t stage_index(const BlockTable& bt, const void* base, const HostExperts& experts, int K, bool ties,
                       double density, float* sumsq, uint32_t* tau, hipStream_t s, uint64_t* h2d,
                       bool delta = false);
hipError_t stage_merge(const BlockTable& bt, const MergeArgs& a, const void* base, const HostExperts& experts,
                       int K, const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s,
                       uint64_t* h2d);

}  // namespace mp
