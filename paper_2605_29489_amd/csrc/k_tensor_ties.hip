// TIES trim thresholds at tensor scope: for expert i and tensor t, the k-th
// largest |d| over the tensor's zero-completed masked deltas (unselected
// blocks count as zeros and are never read), k = min(n_t, ceil(rho n_t)).
// This is the per-tensor variant of Appendix A.1's trim; merges then use
// the per-unit threshold kernel with each unit taking its tensor's value.
//
// An exact MSD radix select on the 31-bit magnitude patterns, three digit
// passes (bits 30..20, 19..9, 8..0) over the selected blocks:
//   k_tt_hist     one workgroup per (run of <= 16 consecutive blocks of one
//                 tensor, expert): LDS histogram of the digit of the
//                 elements that match the prefix fixed so far, nonzero bins
//                 added to the pair's global histogram.  Each XCD takes a
//                 contiguous range of (run, expert) pairs with the expert
//                 fastest, so the K workgroups of a run read its base
//                 blocks through one L2;
//   k_tt_resolve  one wave per (expert, tensor) pair: the bin holding the
//                 k-th largest fixes the digit and the remaining rank.  In
//                 the first pass, k = 0 gives all ones (nothing kept) and
//                 fewer than k selected elements give 0 (the k-th largest
//                 is a completed zero);
//   k_tt_expand   tau[g*K + i] = the pair's threshold for every unit.
// State per pair (uint4): {prefix, remaining rank, done, tau}.
#include <cmath>

#include "device_common.h"
#include "mp_internal.h"

namespace mp {

namespace {

constexpr int kTT = 256;
constexpr int kDigBins = 2048;  // 11-bit digits (the last pass uses 9 bits)
// Digit-pass workgroups: the first pass counts every element, and equal
// top digits are common, so its histogram has four copies of each bin
// (lane l adds to copy l mod 4) in 512-thread workgroups (32 KiB of LDS, 32
// waves per CU); later passes count only the prefix's elements, with two
// copies in 256-thread workgroups.  On the Qwen2.5-1.5B-shaped family at
// B = 25/50/100%, thresholds and merge: 4.29-4.34 / 6.51-6.55 / 11.07-11.22
// ms; 4.14 / 6.42 / 12.32 ms with the later passes' form throughout, 4.39 /
// 6.52 / 10.92 ms with the first's.
constexpr int kTH0 = 512, kCop0 = 4;
constexpr int kTH = 256, kCop = 2;

__host__ __device__ inline int tt_shift(int pass) { return pass == 0 ? 20 : (pass == 1 ? 9 : 0); }
__host__ __device__ inline int tt_width(int pass) { return pass == 2 ? 9 : 11; }

__global__ __launch_bounds__(kTT) void k_tt_zero(uint32_t* __restrict__ p, int64_t n)
{
    for (int64_t q = (int64_t)blockIdx.x * kTT + threadIdx.x; q < n; q += (int64_t)gridDim.x * kTT)
        p[q] = 0u;
}

template <int DT, bool DELTA, int kTH, int kCopies>
__global__ __launch_bounds__(kTH) void k_tt_hist(const void* __restrict__ base, ExpertPtrs ex, int K,
                                                  const uint4* __restrict__ chunks,
                                                  const uint64_t* __restrict__ boff,
                                                  const uint32_t* __restrict__ blen,
                                                  const uint32_t* __restrict__ mask,
                                                  const uint4* __restrict__ state, int T, int pass,
                                                  uint32_t* __restrict__ hist, uint32_t n_pairs, uint32_t per_xcd)
{
    constexpr int V = Fmt<DT>::V;
    __shared__ __align__(16) uint32_t h[kDigBins * kCopies];  // h[bin * kCopies + copy]
    static_assert(kCopies == 1 || kCopies == 2 || kCopies == 4, "a bin's copies are one LDS read");
    // workgroup id -> (run, expert): XCD x = id mod 8 takes pairs
    // x*per_xcd .. in order
    const uint32_t pr = (blockIdx.x & 7u) * per_xcd + (blockIdx.x >> 3);
    if (pr >= n_pairs)
        return;
    const uint4 ch = chunks[pr / (uint32_t)K];
    const int i = (int)(pr % (uint32_t)K);
    const uint32_t t = ch.z;
    const uint4 st = state[(size_t)i * T + t];
    if (st.z != 0u)  // this pair's threshold is already known
        return;
    const int tid = threadIdx.x;
    // nothing to count when the expert has no selected block in the run
    static_assert(kChunkBlocks <= kTH, "a thread per block of a run");
    if (!__syncthreads_or(tid < (int)(ch.y - ch.x) && ((mask[ch.x + (uint32_t)tid] >> i) & 1u)))
        return;
    for (int q = tid; q < kDigBins * kCopies / 4; q += kTH)
        reinterpret_cast<uint4*>(h)[q] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    const uint32_t cp = (uint32_t)(tid % kCopies);
    const int sh = tt_shift(pass), wd = tt_width(pass);
    const uint32_t dmask = (1u << wd) - 1u;
    const int hsh = sh + wd;  // the bits above the digit must match the prefix
    const uint32_t prefix = st.x;
    for (uint32_t g = ch.x; g < ch.y; ++g) {
        if (!((mask[g] >> i) & 1u))
            continue;
        const uint64_t off = boff[g];
        const uint32_t nch = blen[g] / V;
        const uint4* pe = chunk_ptr(ex.p[i], off, Fmt<DT>::esize);
        const uint4* pb = chunk_ptr(base, off, Fmt<DT>::esize);
        // two chunks per thread in flight (a 4096-element bf16 block is
        // exactly two)
        for (uint32_t c0 = tid; c0 < nch; c0 += 2 * kTH) {
            uint4 re[2], rb[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const uint32_t c = c0 + (uint32_t)(u * kTH);
                re[u] = c < nch ? ld16s(pe + c) : make_uint4(0u, 0u, 0u, 0u);
                rb[u] = (!DELTA && c < nch) ? pb[c] : make_uint4(0u, 0u, 0u, 0u);  // cached: the run's other experts read it too
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                if (c0 + (uint32_t)(u * kTH) >= nch)
                    continue;
                float fe[V], fb[V];
                Fmt<DT>::unpack(re[u], fe);
                if (!DELTA)
                    Fmt<DT>::unpack(rb[u], fb);
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    const float d = DELTA ? fe[v] : fe[v] - fb[v];
                    const uint32_t mg = __float_as_uint(d) & 0x7fffffffu;
                    if (pass == 0 || (mg >> hsh) == prefix)
                        atomicAdd(&h[((mg >> sh) & dmask) * kCopies + cp], 1u);
                }
            }
        }
    }
    __syncthreads();
    uint32_t* out = hist + ((size_t)i * T + t) * kDigBins;
    for (int q = tid; q < kDigBins; q += kTH) {
        uint32_t v;
        if constexpr (kCopies == 4) {
            const uint4 w = reinterpret_cast<const uint4*>(h)[q];
            v = w.x + w.y + w.z + w.w;
        } else if constexpr (kCopies == 2) {
            const uint2 w = reinterpret_cast<const uint2*>(h)[q];
            v = w.x + w.y;
        } else {
            v = h[q];
        }
        if (v != 0u)
            atomicAdd(&out[q], v);
    }
}

__global__ __launch_bounds__(kTT) void k_tt_resolve(uint4* __restrict__ state, const uint32_t* __restrict__ hist,
                                                     const uint64_t* __restrict__ tnumel, int K, int T,
                                                     double density, int pass, uint32_t* __restrict__ err,
                                                     int force_no_cut)
{
    const int lane = threadIdx.x & 63;
    const int64_t q = (int64_t)blockIdx.x * (kTT / 64) + (threadIdx.x >> 6);
    if (q >= (int64_t)K * T)
        return;
    const int t = (int)(q % T);
    uint4 st = state[q];
    if (st.z != 0u)
        return;
    const uint32_t* h = hist + (size_t)q * kDigBins;
    const int wd = tt_width(pass);
    constexpr int per = kDigBins / 64;  // lane l holds bins [l*per, (l+1)*per) (the 9-bit pass leaves the top ones 0)
    uint32_t c[per];
    uint32_t mine = 0u;
#pragma unroll
    for (int j = 0; j < per; ++j) {
        c[j] = h[lane * per + j];
        mine += c[j];
    }
    // count in the bins above this lane's range (suffix over higher lanes)
    uint32_t incl = mine;  // inclusive sum over lanes >= lane
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_down(incl, (unsigned)off);
        if (lane + off < 64)
            incl += y;
    }
    const uint32_t total = __shfl(incl, 0);
    uint32_t rank = st.y;
    if (pass == 0) {
        const uint64_t n = tnumel[t];
        const double kk = ceil(density * (double)n);
        const uint64_t k = (kk >= (double)n) ? n : (uint64_t)kk;
        if (k == 0u || (uint64_t)total < k) {
            if (lane == 0)
                state[q] = make_uint4(0u, 0u, 1u, k == 0u ? 0xffffffffu : 0u);
            return;
        }
        rank = (uint32_t)k;
    }
    const uint32_t above = incl - mine;  // elements in bins of higher lanes
    int bin = -1;
    uint32_t before = 0u;
    if (above < rank && incl >= rank) {  // the k-th largest is in this lane's range
        uint32_t acc = above;
#pragma unroll
        for (int j = per - 1; j >= 0; --j) {
            if (bin < 0 && acc + c[j] >= rank) {
                bin = lane * per + j;
                before = acc;
            }
            acc += c[j];
        }
    }
    unsigned long long bal = __ballot(bin >= 0);
    if (force_no_cut && q == 0)
        bal = 0ull;  // test hook: pair 0 takes the error path
    if (bal == 0ull) {  // cannot happen: the prefix's elements hold the rank-th largest
        if (lane == 0) {
            state[q] = make_uint4(st.x, 0u, 1u, 0u);
            err[0] = 1u;  // the host reports an internal error
        }
        return;
    }
    const int src = __ffsll((long long)bal) - 1;
    bin = __shfl(bin, src);
    before = __shfl(before, src);
    if (lane == 0) {
        st.x = (st.x << wd) | (uint32_t)bin;
        st.y = rank - before;
        if (pass == 2) {
            st.z = 1u;
            st.w = st.x;
        }
        state[q] = st;
    }
}

__global__ __launch_bounds__(kTT) void k_tt_expand(const uint4* __restrict__ state,
                                                    const uint32_t* __restrict__ tensor, int64_t G, int K, int T,
                                                    uint32_t* __restrict__ tau)
{
    const int64_t u = (int64_t)blockIdx.x * kTT + threadIdx.x;
    if (u >= G * K)
        return;
    const int64_t g = u / K;
    const int i = (int)(u - g * K);
    tau[u] = state[(size_t)i * T + tensor[g]].w;
}

}  // namespace

hipError_t launch_ties_tensor(const BlockTable& bt, const void* base, const ExpertPtrs& ex, int K,
                              const uint32_t* mask, double density, uint32_t* tau, uint32_t* hist, uint4* state,
                              hipStream_t s, bool delta, bool force_no_cut)
{
    if (bt.G == 0)
        return hipSuccess;
    const int T = (int)bt.n_tensors;
    const int64_t pairs = (int64_t)K * T;
    const int64_t nh = pairs * kDigBins;
    // the state words and, after them, the error word start at zero
    uint32_t* err = reinterpret_cast<uint32_t*>(state + pairs);
    hipLaunchKernelGGL(k_tt_zero, dim3((unsigned)std::min<int64_t>((pairs * 4 + 4 + kTT - 1) / kTT, 1024)), dim3(kTT),
                       0, s, reinterpret_cast<uint32_t*>(state), pairs * 4 + 4);
    const uint32_t n_pairs = (uint32_t)(bt.n_chunks * K), per_xcd = (n_pairs + 7u) / 8u;
    const dim3 hgrid(8u * per_xcd);
    for (int pass = 0; pass < 3; ++pass) {
        hipLaunchKernelGGL(k_tt_zero, dim3((unsigned)std::min<int64_t>((nh + kTT - 1) / kTT, 2048)), dim3(kTT), 0, s,
                           hist, nh);
        auto go = [&](auto kern, int nth) {
            hipLaunchKernelGGL(kern, hgrid, dim3(nth), 0, s, base, ex, K, bt.d_chunk, bt.d_off, bt.d_len, mask, state,
                               T, pass, hist, n_pairs, per_xcd);
        };
        if (pass == 0) {
            if (bt.dtype == 0)
                delta ? go(k_tt_hist<0, true, kTH0, kCop0>, kTH0) : go(k_tt_hist<0, false, kTH0, kCop0>, kTH0);
            else
                delta ? go(k_tt_hist<1, true, kTH0, kCop0>, kTH0) : go(k_tt_hist<1, false, kTH0, kCop0>, kTH0);
        } else {
            if (bt.dtype == 0)
                delta ? go(k_tt_hist<0, true, kTH, kCop>, kTH) : go(k_tt_hist<0, false, kTH, kCop>, kTH);
            else
                delta ? go(k_tt_hist<1, true, kTH, kCop>, kTH) : go(k_tt_hist<1, false, kTH, kCop>, kTH);
        }
        hipLaunchKernelGGL(k_tt_resolve, dim3((unsigned)((pairs + 3) / 4)), dim3(kTT), 0, s, state, hist,
                           bt.d_tnumel, K, T, density, pass, err, force_no_cut ? 1 : 0);
    }
    hipLaunchKernelGGL(k_tt_expand, dim3((unsigned)((bt.G * K + kTT - 1) / kTT)), dim3(kTT), 0, s, state,
                       bt.d_tensor, bt.G, K, T, tau);
    return hipGetLastError();
}

}  // namespace mp
