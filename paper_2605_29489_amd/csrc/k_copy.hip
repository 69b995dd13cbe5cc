// A plain stream copy of device memory: the access pattern of the merge
// kernels (16-byte non-temporal buffer loads and stores, one chunk per lane,
// one wave per workgroup) without their arithmetic.  It measures the HBM rate
// this device reaches on a read-once, write-once stream, the practical
// ceiling the merges are compared with beside the published peak.  Among
// 64 to 512 threads per workgroup and one to eight chunks per lane, one
// chunk per lane of a one-wave workgroup copied fastest on MI355X.
#include "device_common.h"
#include "mp_internal.h"

namespace mp {

namespace {

constexpr int kCopyT = 64;

// Workgroup w copies bytes [w * 1024, min((w + 1) * 1024, nbytes)); the
// buffer resource ends there, so lanes past the end read zeros and their
// stores are dropped.
__global__ __launch_bounds__(kCopyT) void k_stream_copy(const char* __restrict__ src, char* __restrict__ dst,
                                                        uint64_t nbytes)
{
    const uint64_t w0 = (uint64_t)blockIdx.x * (kCopyT * 16);
    const uint64_t rem = nbytes - w0;
    const uint32_t lim = (uint32_t)(rem < (uint64_t)(kCopyT * 16) ? rem : (uint64_t)(kCopyT * 16));
    const uint32_t off = threadIdx.x * 16u;
    bst16s(block_rsrc(dst + w0, lim), off, bld16s(block_rsrc(src + w0, lim), off));
}

}  // namespace

hipError_t launch_stream_copy(const void* src, void* dst, uint64_t nbytes, hipStream_t s)
{
    if (nbytes == 0)
        return hipSuccess;
    const uint64_t grid = (nbytes + kCopyT * 16 - 1) / (kCopyT * 16);
    hipLaunchKernelGGL(k_stream_copy, dim3((unsigned)grid), dim3(kCopyT), 0, s, static_cast<const char*>(src),
                       static_cast<char*>(dst), nbytes);
    return hipGetLastError();
}

}  // namespace mp
