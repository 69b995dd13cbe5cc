// Where a merge kernel finds a selected expert block, and the realized-read
// counters, shared by the elementwise merge kernels (k_merge.hip) and the
// TIES kernel that trims inside the merge (k_merge_ties.hip).
//
// Expert i's block sits at its layout offset in expert i's buffer, which is
// device memory or pinned host memory read over PCIe (DevSrc), or in a
// device staging buffer filled from host memory (StagedSrc).
#pragma once

#include "device_common.h"
#include "mp_internal.h"

namespace mp {

namespace {

// ------------------------------------------------------------ addressing
struct DevSrc {
    ExpertPtrs ex;
    __device__ uint32_t block(int64_t b) const { return (uint32_t)b; }
    // r = rank of expert i among the block's selected experts (unused here)
    __device__ const uint4* expert(int i, int r, int64_t b, uint64_t off, uint32_t n, int es) const
    {
        return chunk_ptr(ex.p[i], off, es);
    }
    // With at most four experts the pointer is picked from the first four
    // by constant indices: the kernel loads them with its arguments, and an
    // expert read does not wait for a pointer fetched once the mask is known.
    template <bool SMALLK>
    __device__ const void* expert_block(int i, int r, int64_t b, uint64_t off, uint32_t n, int es) const
    {
        const void* p = SMALLK ? ((i == 0) ? ex.p[0] : (i == 1) ? ex.p[1] : (i == 2) ? ex.p[2] : ex.p[3]) : ex.p[i];
        return static_cast<const char*>(p) + off * (uint64_t)es;
    }
};

// Selected expert blocks staged in device memory (host experts): the
// launch covers blocks b0 .. b0 + grid - 1; block b0 + j's selected experts
// lie back to back, in increasing expert order (rank r), from stage + soff[j].
struct StagedSrc {
    const char* stage;
    const uint64_t* soff;
    int64_t b0;
    __device__ uint32_t block(int64_t b) const { return (uint32_t)(b0 + b); }
    __device__ const uint4* expert(int i, int r, int64_t b, uint64_t off, uint32_t n, int es) const
    {
        return reinterpret_cast<const uint4*>(stage + soff[b] + (uint64_t)r * n * (uint64_t)es);
    }
    template <bool SMALLK>
    __device__ const void* expert_block(int i, int r, int64_t b, uint64_t off, uint32_t n, int es) const
    {
        return stage + soff[b] + (uint64_t)r * n * (uint64_t)es;
    }
};

// Realized expert reads (Prop. 1's N^run), counted where the loads are
// issued: after loading expert i's chunks q * NT + t (q < CPT) of a block of
// nch chunks, each wave adds the bytes its lanes loaded into slot
// ((workgroup * 4 + wave) mod 8) * 32 + i, so the 256 counters sum per
// expert and the atomics spread over 8 words each.  No-op when ctr is null.
template <int NT, int CPT>
__device__ inline void count_loaded(unsigned long long* ctr, int i, uint32_t nch)
{
    if (ctr == nullptr)
        return;
    const uint32_t t = threadIdx.x;
    uint32_t nl = 0;
#pragma unroll
    for (int q = 0; q < CPT; ++q)
        nl += (uint32_t)__popcll(__ballot(q * NT + t < nch));
    if ((t & 63u) == 0u)
        atomicAdd(&ctr[(((blockIdx.x * 4u) + (t >> 6)) & 7u) << 5 | (uint32_t)i], (unsigned long long)nl * 16ull);
}

}  // namespace

}  // namespace mp
