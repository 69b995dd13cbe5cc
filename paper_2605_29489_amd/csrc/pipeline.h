// Host-to-device feed for host-resident experts (Algorithm 2's streaming
// loop with DeltaIterator.PullMasked): only selected expert blocks cross
// PCIe.  See pipeline.hip.
#pragma once

#include <string>

#include "mp_internal.h"

namespace mp {

class Pipeline {
public:
    Pipeline();
    ~Pipeline();
    Pipeline(const Pipeline&) = delete;
    Pipeline& operator=(const Pipeline&) = delete;

    // Index with pinned host experts: every expert block is staged once.
    int index(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K, float* sumsq,
              hipStream_t s, std::string* err);

    // Merge with pinned host experts: only the blocks the mask selects are
    // packed, copied and merged; io (never NULL here) gets the transfer totals.
    int merge(const BlockTable& bt, const MergeArgs& a, const void* base, const ExpertPtrs& ex, int K,
              const uint32_t* mask, void* out, unsigned long long* ctr, hipStream_t s, mp_io_stats* io,
              std::string* err);

private:
    struct Impl;
    Impl* impl_;
};

}  // namespace mp
