// Block-norm index (the catalog statistic of Section 2 / Section 3
// "Catalog"): S[g*K + i] = sum over block g of d*d, d = x_i - x_0 in fp32.
//
// One 256-thread workgroup per block; wave w handles experts w, w+4, ...
// Each lane streams 16-byte chunks l, l+64, l+128, ... of the block (one
// coalesced 1 KiB row per wave load), accumulates its chunk elements in
// order with fma into one fp32 partial, and the wave folds the 64 partials
// with an xor butterfly.  This fixed order is the one the ABI documents, so
// the scores -- and therefore the plan -- are reproducible bit for bit.
// The base block is re-read per expert from L2 (it stays resident: 8-16 KiB
// per workgroup), so HBM sees it once.
#include <cmath>

// The catalog kernel keeps two copies of each window bin (the merge kernel
// that trims in place keeps four): a wave's histogram row is then 4 KiB, the
// workgroup's LDS 24 KiB and its registers fit five waves per SIMD.  More
// waves in flight pay for the extra same-address atomics: on the headline
// family the pass took 2.45-2.50 ms against 2.69 ms with four copies at four
// waves (one copy at five waves: 2.59 ms; six waves spill).
#define MP_TIES_NC 2
#include "device_common.h"
#include "mp_internal.h"
#include "ties_select.h"

namespace mp {

namespace {

constexpr int kRows = 8;  // chunk rows a lane keeps in flight per expert

// DELTA: the expert buffers hold the deltas themselves (no base read).
template <int DT, bool DELTA>
__device__ inline float block_sumsq(const uint4* __restrict__ b, const uint4* __restrict__ e,
                                    uint32_t nch, int lane)
{
    constexpr int V = Fmt<DT>::V;
    float p = 0.0f;
    for (uint32_t c0 = 0; c0 < nch; c0 += 64 * kRows) {
        uint4 xb[kRows], xe[kRows];
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const uint32_t c = c0 + r * 64 + lane;
            if (c < nch) {
                if (!DELTA)
                    xb[r] = b[c];  // re-read per expert: cached
                xe[r] = ld16s(&e[c]);
            }
        }
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const uint32_t c = c0 + r * 64 + lane;
            if (c < nch) {
                float fb[V], fe[V];
                if (!DELTA)
                    Fmt<DT>::unpack(xb[r], fb);
                Fmt<DT>::unpack(xe[r], fe);
#pragma unroll
                for (int q = 0; q < V; ++q) {
                    const float d = DELTA ? fe[q] : fe[q] - fb[q];
                    p = fmaf(d, d, p);
                }
            }
        }
    }
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1)
        p = p + __shfl_xor(p, s);
    return p;
}

template <int DT, bool DELTA>
__global__ __launch_bounds__(256) void k_index(const void* __restrict__ base, ExpertPtrs ex, int K,
                                               const uint64_t* __restrict__ boff,
                                               const uint32_t* __restrict__ blen,
                                               float* __restrict__ sumsq)
{
    const int64_t g = blockIdx.x;
    const int lane = threadIdx.x & 63;
    // wave-uniform, so that ex.p[i] is a scalar load
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t off = boff[g];
    const uint32_t nch = blen[g] / Fmt<DT>::V;
    const uint4* b = chunk_ptr(base, off, Fmt<DT>::esize);
    for (int i = wave; i < K; i += 4) {
        const uint4* e = chunk_ptr(ex.p[i], off, Fmt<DT>::esize);
        const float s = block_sumsq<DT, DELTA>(b, e, nch, lane);
        if (lane == 0)
            sumsq[g * K + i] = s;
    }
}

// Catalog statistics for TIES: per unit, the sum of squares of k_index
// (same order, same bits; optional) and the trim threshold, the fp32
// pattern of the k-th largest |d| of the (expert, block) unit for a keep
// density (all ones when k = 0: a NaN pattern, which keeps nothing).  The
// threshold depends on the unit and the density only, never on an access
// mask, so merges at any budget can reuse it.  The base block is staged in
// LDS once; wave w takes experts w, w+4, ... of the block: it holds the
// whole unit's deltas in registers (64 per lane; lane l owns chunks l, l+64,
// ...) and selects with its own LDS row, so after the staging the workgroup
// never synchronises.
#ifndef MP_CAT_WAVES
#define MP_CAT_WAVES 5
#endif
template <int DT, bool DELTA>
__global__ __launch_bounds__(256, DT == 1 ? MP_CAT_WAVES : 3) void k_index_ties(
    const void* __restrict__ base, ExpertPtrs ex, int K, const uint64_t* __restrict__ boff,
    const uint32_t* __restrict__ blen, uint32_t n_full, uint32_t k_full, double density, float gcoef,
    float* __restrict__ sumsq, uint32_t* __restrict__ tau)
{
    constexpr int V = Fmt<DT>::V;
    constexpr int R = kTiesMaxBlock / 64 / V;  // chunk rows per lane
    constexpr int E = R * V;                   // deltas per lane
    __shared__ uint32_t rows[4][ties::NB];
    __shared__ uint4 xb[R * 64];  // the base block's chunks (zeros past its end)
    const int64_t g = blockIdx.x;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // wave-uniform: ex.p[i] is a scalar load
    const uint64_t off = boff[g];
    const uint32_t n = blen[g];
    const uint32_t nch = n / V;
    uint32_t k = k_full;
    if (n != n_full) {
        const double kk = ceil(density * (double)n);
        k = (kk >= (double)n) ? n : (uint32_t)kk;
    }
    // one unit: expert i's chunks (xe) against the staged base
    auto unit = [&](int i, const uint4 (&xe)[R]) {
        float d[E];
        float p = 0.0f;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float fb[V], fe[V];
            if (!DELTA)
                Fmt<DT>::unpack(xb[r * 64 + lane], fb);
            Fmt<DT>::unpack(xe[r], fe);
#pragma unroll
            for (int q = 0; q < V; ++q) {
                d[r * V + q] = DELTA ? fe[q] : fe[q] - fb[q];  // padding: 0 - 0
                p = fmaf(d[r * V + q], d[r * V + q], p);  // + 0 on padding, exact
            }
        }
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1)
            p = p + __shfl_xor(p, s);
        // a guess at tau: gcoef times the deltas' root mean square
        const uint32_t guess = __float_as_uint(gcoef * sqrtf(p / (float)n));
        const uint32_t th = (k == 0u) ? 0xffffffffu
                                      : wave_kth_largest<E>(reinterpret_cast<char*>(&rows[0][0]), wave * ties::NB * 4,
                                                            d, k, lane, guess);
        if (lane == 0) {
            if (sumsq != nullptr)
                sumsq[g * K + i] = p;
            tau[g * K + i] = th;
        }
    };
    // Loads are buffer loads over the block's byte range: lanes past a short
    // block's end read zeros without a branch, so every load of a lane is
    // issued back to back and the waits count them exactly.
    const uint32_t nbytes = nch * 16u;
    auto load_expert = [&](int i, uint32_t bytes, uint4 (&xe)[R]) {
        const __amdgpu_buffer_rsrc_t re = block_rsrc(chunk_ptr(ex.p[i], off, Fmt<DT>::esize), bytes);
#pragma unroll
        for (int r = 0; r < R; ++r)
            xe[r] = bld16s(re, (uint32_t)(r * 64 + lane) * 16u);
    };
    // The base's chunks are requested first, then the wave's first expert
    // (a wave without one reads an empty range), so the base arrives first
    // and is staged while the expert is still in flight; further experts
    // (K > 4) are read one at a time.
    uint4 xbr[R / 4];
    if (!DELTA) {  // explicit deltas need no base
        const __amdgpu_buffer_rsrc_t rb = block_rsrc(chunk_ptr(base, off, Fmt<DT>::esize), nbytes);
#pragma unroll
        for (int q = 0; q < R / 4; ++q)
            xbr[q] = bld16s(rb, (uint32_t)(q * 256 + t) * 16u);
    }
    uint4 xf[R];
    load_expert(wave < K ? wave : 0, wave < K ? nbytes : 0u, xf);
    if (!DELTA) {
#pragma unroll
        for (int q = 0; q < R / 4; ++q)
            xb[q * 256 + t] = xbr[q];  // zeros past the block's end
        __syncthreads();
    }
    if (wave < K)
        unit(wave, xf);
    for (int i = wave + 4; i < K; i += 4) {
        uint4 xe[R];
        load_expert(i, nbytes, xe);
        unit(i, xe);
    }
}

}  // namespace

// z with P(|Z| > z) = rho for a standard normal Z (bisection on erfc).
double normal_two_sided_quantile(double rho)
{
    if (!(rho > 0.0) || rho >= 1.0)
        return 0.0;
    double lo = 0.0, hi = 40.0;
    for (int it = 0; it < 200; ++it) {
        const double mid = 0.5 * (lo + hi);
        if (erfc(mid / sqrt(2.0)) > rho)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

hipError_t launch_index_ties(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K,
                             double density, float* sumsq, uint32_t* tau, hipStream_t s, bool delta)
{
    if (bt.G == 0)
        return hipSuccess;
    const uint32_t n_full = (uint32_t)bt.block_elems;
    const double kk = ceil(density * (double)n_full);
    const uint32_t k_full = (kk >= (double)n_full) ? n_full : (uint32_t)kk;
    // The selector's first guess at a unit's threshold: 0.8 of the rho-tail
    // quantile of a normal with the deltas' RMS (for normal deltas about
    // 0.8 tau; measured on the headline family, 0.6 was slower, 0.9 the same
    // and 1.0 misses often enough to cost a second pass).  It only decides
    // which values the first histogram pass counts; the thresholds are exact
    // for any data.
    const float gcoef = (float)(0.8 * normal_two_sided_quantile(density));
    const dim3 grid((unsigned)bt.G), block(256);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, block, 0, s, base, ex, K, bt.d_off, bt.d_len, n_full, k_full, density, gcoef,
                           sumsq, tau);
    };
    if (bt.dtype == 0)
        delta ? go(k_index_ties<0, true>) : go(k_index_ties<0, false>);
    else
        delta ? go(k_index_ties<1, true>) : go(k_index_ties<1, false>);
    return hipGetLastError();
}

hipError_t launch_index(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K,
                        float* sumsq, hipStream_t s, bool delta)
{
    if (bt.G == 0)
        return hipSuccess;
    const dim3 grid((unsigned)bt.G), block(256);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, block, 0, s, base, ex, K, bt.d_off, bt.d_len, sumsq);
    };
    if (bt.dtype == 0)
        delta ? go(k_index<0, true>) : go(k_index<0, false>);
    else
        delta ? go(k_index<1, true>) : go(k_index<1, false>);
    return hipGetLastError();
}

}  // namespace mp
