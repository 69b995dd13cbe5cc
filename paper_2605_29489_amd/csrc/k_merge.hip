// Mask-aware merge operators Psi_op (Eq. 4; operators of Appendix A.1).
//
// One 256-thread workgroup per block.  The block's mask word is uniform, so
// the loop over the selected experts is a scalar loop: unselected experts
// are never touched (the zero-completed tuple of Appendix A.1 costs no
// reads).  Blocks are streamed as 16-byte chunks with coalesced loads.
//
//  * AVG / DARE (linear or sign-elect): elementwise.  A thread owns CPT
//    chunks of a tile and loads the chunks of up to 4 selected experts
//    before consuming them in increasing expert order.
//  * TIES: the whole block (<= 4096 elements, 16 per thread) stays in
//    registers.  Per selected expert the trim threshold tau (k-th largest
//    |d|) comes from an exact MSD radix select over the fp32 magnitude bit
//    patterns in LDS: bits 30..21 (all elements), 20..11 (only the ones in
//    the chosen bucket, with bucket min/max to stop early on ties), 10..0.
//    Any tau' with  max{|d| < tau} < tau' <= tau  gives the same keep
//    decisions, so the select stops as soon as the bucket that holds tau is
//    known to be kept entirely.  The sign election and disjoint mean run in
//    one pass over the experts with running sums per element.
//
// Addressing: device-resident experts (expert i's block at its layout
// offset) or staged experts (the selected blocks packed back to back in a
// device buffer, in increasing expert order, as the host pipeline copies
// them).
#include "device_common.h"
#include "mp_internal.h"

namespace mp {

namespace {

constexpr int kT = 256;

// ------------------------------------------------------------ addressing
struct DevSrc {
    ExpertPtrs ex;
    __device__ uint32_t block(int64_t b) const { return (uint32_t)b; }
    // r = rank of expert i among the block's selected experts (unused here)
    __device__ const uint4* expert(int i, int r, int64_t b, uint64_t off, uint32_t n, int es) const
    {
        return chunk_ptr(ex.p[i], off, es);
    }
};

struct StagedSrc {
    const char* stage;
    const uint32_t* gid;
    const uint64_t* soff;  // byte offset of the block's first selected expert
    __device__ uint32_t block(int64_t b) const { return gid[b]; }
    __device__ const uint4* expert(int i, int r, int64_t b, uint64_t off, uint32_t n, int es) const
    {
        return reinterpret_cast<const uint4*>(stage + soff[b] + (uint64_t)r * n * (uint64_t)es);
    }
};

__device__ inline void count_expert_bytes(unsigned long long* ctr, uint32_t m, uint32_t n, int es)
{
    if (ctr != nullptr && threadIdx.x == 0 && m != 0u)
        atomicAdd(&ctr[blockIdx.x & 255u], (unsigned long long)__popc(m) * n * (unsigned long long)es);
}

// ------------------------------------------------------------ elementwise family
enum { M_AVG = 0, M_DARE_LIN = 1, M_DARE_SIGN = 2 };

template <int DT, int MODE, class Src>
__global__ __launch_bounds__(kT) void k_merge_elem(Src src, const void* __restrict__ base,
                                                   const uint32_t* __restrict__ mask,
                                                   const uint64_t* __restrict__ boff,
                                                   const uint32_t* __restrict__ blen,
                                                   const uint32_t* __restrict__ btensor,
                                                   const uint64_t* __restrict__ belem0, Coeffs alpha,
                                                   float lambda, uint32_t drop_T, float scale,
                                                   uint32_t seed, uint32_t kmask, void* __restrict__ out,
                                                   unsigned long long* __restrict__ ctr)
{
    constexpr int V = Fmt<DT>::V;
    constexpr int ES = Fmt<DT>::esize;
    constexpr int CPT = (DT == 1) ? 2 : 4;  // chunks per thread per tile (4096-element blocks: 1 tile)
    constexpr int E = CPT * V;
    const int64_t b = blockIdx.x;
    const int t = threadIdx.x;
    const uint32_t g = src.block(b);
    const uint64_t off = boff[g];
    const uint32_t n = blen[g];
    const uint32_t m = mask[g] & kmask;  // bits of experts >= K are ignored
    const uint32_t nch = n / V;
    const uint4* pb = chunk_ptr(base, off, ES);
    uint4* po = reinterpret_cast<uint4*>(static_cast<char*>(out) + off * ES);
    count_expert_bytes(ctr, m, n, ES);
    uint32_t tens = 0;
    uint64_t e0 = 0;
    if (MODE != M_AVG) {
        tens = btensor[g];
        e0 = belem0[g];
    }

    for (uint32_t tile = 0; tile < nch; tile += CPT * kT) {
        float x0[E];
        bool ok[CPT];
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            const uint32_t c = tile + q * kT + t;
            ok[q] = c < nch;
            uint4 raw = make_uint4(0, 0, 0, 0);
            if (ok[q])
                raw = pb[c];
            Fmt<DT>::unpack(raw, &x0[q * V]);
        }
        float acc[E], ps[E], ns[E];
        uint32_t pc[E], nc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            acc[e] = 0.0f;
            ps[e] = 0.0f;
            ns[e] = 0.0f;
            pc[e] = 0u;
            nc[e] = 0u;
        }
        uint32_t mm = m;
        int rank = 0;
        while (mm) {
            int idx[4];
            int cnt = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                idx[j] = -1;
                if (mm) {
                    idx[j] = __builtin_ctz(mm);
                    mm &= mm - 1u;
                    ++cnt;
                }
            }
            uint4 raw[4][CPT];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (j < cnt) {
                    const uint4* pe = src.expert(idx[j], rank + j, b, off, n, ES);
#pragma unroll
                    for (int q = 0; q < CPT; ++q)
                        if (ok[q])
                            raw[j][q] = pe[tile + q * kT + t];
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (j >= cnt)
                    break;
                const int i = idx[j];
#pragma unroll
                for (int q = 0; q < CPT; ++q) {
                    if (!ok[q])
                        continue;
                    float x[V];
                    Fmt<DT>::unpack(raw[j][q], x);
                    uint32_t word[V];
                    if (MODE != M_AVG) {
                        // Philox words for elements e .. e+V-1 of tensor `tens` (V is 4 or 8)
                        const uint64_t e = e0 + (uint64_t)(tile + q * kT + t) * V;
#pragma unroll
                        for (int h = 0; h < V / 4; ++h) {
                            const uint64_t qq = (e >> 2) + h;
                            const uint4 r4 = philox4x32_10(
                                make_uint4((uint32_t)qq, (uint32_t)(qq >> 32), tens, 0u), seed, (uint32_t)i);
                            word[h * 4 + 0] = r4.x;
                            word[h * 4 + 1] = r4.y;
                            word[h * 4 + 2] = r4.z;
                            word[h * 4 + 3] = r4.w;
                        }
                    }
#pragma unroll
                    for (int v = 0; v < V; ++v) {
                        const int e = q * V + v;
                        const float d = x[v] - x0[e];
                        if (MODE == M_AVG) {
                            acc[e] = fmaf(alpha.v[i], d, acc[e]);
                        } else {
                            const float tv = (word[v] < drop_T) ? 0.0f : d * scale;
                            if (MODE == M_DARE_LIN) {
                                acc[e] = fmaf(alpha.v[i], tv, acc[e]);
                            } else {
                                acc[e] = acc[e] + tv;  // sigma
                                ps[e] = ps[e] + fmaxf(tv, 0.0f);
                                ns[e] = ns[e] + fminf(tv, 0.0f);
                                pc[e] += (tv > 0.0f) ? 1u : 0u;
                                nc[e] += (tv < 0.0f) ? 1u : 0u;
                            }
                        }
                    }
                }
            }
            rank += cnt;
        }
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            if (!ok[q])
                continue;
            float y[V];
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int e = q * V + v;
                if (MODE == M_AVG) {
                    y[v] = x0[e] + acc[e];
                } else if (MODE == M_DARE_LIN) {
                    y[v] = fmaf(lambda, acc[e], x0[e]);
                } else {
                    float mean = 0.0f;
                    if (acc[e] > 0.0f)
                        mean = ps[e] / (float)pc[e];
                    else if (acc[e] < 0.0f)
                        mean = ns[e] / (float)nc[e];
                    y[v] = fmaf(lambda, mean, x0[e]);
                }
            }
            po[tile + q * kT + t] = Fmt<DT>::pack(y);
        }
    }
}

// ------------------------------------------------------------ TIES
struct TiesSmem {
    uint32_t hA[2][1024];
    uint32_t hB[1024];
    uint32_t hBmin[1024];
    uint32_t hBmax[1024];
    uint32_t hC[2048];
    uint32_t sel[8];
};

// Wave 0 only: walk the NB-bin histogram h from the top bin down and find
// the bin holding the k-th largest element.  Writes sel[0..3] = {found,
// bin, k - count above the bin, count in the bin}; found = 0 when fewer
// than k elements were counted.
template <int NB>
__device__ inline void scan_from_top(const uint32_t* h, uint32_t k, int lane, uint32_t* sel)
{
    constexpr int PER = NB / 64;
    const int top = NB - PER * lane - 1;  // lane 0 owns the highest bins
    uint32_t loc = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        loc += h[top - j];
    uint32_t incl = loc;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, (unsigned)off);
        if (lane >= off)
            incl += y;
    }
    const uint32_t excl = incl - loc;
    const uint32_t total = __shfl(incl, 63);
    if (lane == 0 && total < k)
        sel[0] = 0u;
    if (excl < k && k <= incl) {
        uint32_t run = excl;
        for (int j = 0; j < PER; ++j) {
            const uint32_t cb = h[top - j];
            if (run + cb >= k) {
                sel[0] = 1u;
                sel[1] = (uint32_t)(top - j);
                sel[2] = k - run;
                sel[3] = cb;
                break;
            }
            run += cb;
        }
    }
}

// Block-wide: threshold tau' for the E magnitudes each thread holds (bit
// patterns of |d|, 0 for padding).  Elements are kept iff mg >= tau' and
// mg != 0.  Must be called by every thread of the workgroup.
// On entry sm.hA[it & 1], sm.hB*, sm.hC are clear; on exit sm.hA[(it+1) & 1],
// sm.hB* and sm.hC are clear again (each thread resets the pass-B/C bins it
// touched), ready for the next expert.
template <int E>
__device__ inline uint32_t ties_threshold(const uint32_t (&mg)[E], uint32_t k, int it, TiesSmem& sm)
{
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (k == 0u)
        return 0xffffffffu;  // keep nothing
    uint32_t* HA = sm.hA[it & 1];
    uint32_t* HAn = sm.hA[(it + 1) & 1];  // last used by the previous expert, whose scans are done
    for (int q = t; q < 1024; q += kT)
        HAn[q] = 0u;
    uint32_t orv = 0u;
#pragma unroll
    for (int e = 0; e < E; ++e)
        orv |= mg[e];
    if (__any(orv != 0u)) {  // a wave whose elements are all zero adds nothing above bin 0
#pragma unroll
        for (int e = 0; e < E; ++e)
            atomicAdd(&HA[mg[e] >> 21], 1u);
    }
    __syncthreads();
    if (wave == 0)
        scan_from_top<1024>(HA, k, lane, sm.sel);
    __syncthreads();
    if (sm.sel[0] == 0u)
        return 1u;  // fewer than k counted: the k-th largest is 0, keep every nonzero
    const uint32_t bA = sm.sel[1], kA = sm.sel[2], cA = sm.sel[3];
    if (cA == kA)
        return bA << 21;  // the whole bucket is kept
    // pass B: bits 20..11 of the elements in bucket bA, with bucket min / max
#pragma unroll
    for (int e = 0; e < E; ++e) {
        if ((mg[e] >> 21) == bA) {
            const uint32_t dg = (mg[e] >> 11) & 1023u;
            atomicAdd(&sm.hB[dg], 1u);
            atomicMin(&sm.hBmin[dg], mg[e]);
            atomicMax(&sm.hBmax[dg], mg[e]);
        }
    }
    __syncthreads();
    if (wave == 0) {
        scan_from_top<1024>(sm.hB, kA, lane, sm.sel);
        if (lane == 0) {
            sm.sel[4] = sm.hBmin[sm.sel[1]];
            sm.sel[5] = sm.hBmax[sm.sel[1]];
        }
    }
    __syncthreads();
    const uint32_t bB = sm.sel[1], kB = sm.sel[2], cB = sm.sel[3];
    const bool whole = (cB == kB) || (sm.sel[4] == sm.sel[5]);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        if ((mg[e] >> 21) == bA) {
            const uint32_t dg = (mg[e] >> 11) & 1023u;
            sm.hB[dg] = 0u;
            sm.hBmin[dg] = 0xffffffffu;
            sm.hBmax[dg] = 0u;
        }
    }
    const uint32_t lo = (bA << 21) | (bB << 11);
    if (whole)
        return lo;  // count matches, or every value in the bucket is equal (ties are all kept)
    // pass C: bits 10..0 of the elements in bucket (bA, bB)
    const uint32_t hiC = lo >> 11;
#pragma unroll
    for (int e = 0; e < E; ++e)
        if ((mg[e] >> 11) == hiC)
            atomicAdd(&sm.hC[mg[e] & 2047u], 1u);
    __syncthreads();
    if (wave == 0)
        scan_from_top<2048>(sm.hC, kB, lane, sm.sel);
    __syncthreads();
    const uint32_t tau = lo | sm.sel[1];
#pragma unroll
    for (int e = 0; e < E; ++e)
        if ((mg[e] >> 11) == hiC)
            sm.hC[mg[e] & 2047u] = 0u;
    return tau;
}

template <int DT, class Src>
__global__ __launch_bounds__(kT) void k_merge_ties(Src src, const void* __restrict__ base,
                                                   const uint32_t* __restrict__ mask,
                                                   const uint64_t* __restrict__ boff,
                                                   const uint32_t* __restrict__ blen, double density,
                                                   float lambda, uint32_t kmask, void* __restrict__ out,
                                                   unsigned long long* __restrict__ ctr)
{
    constexpr int V = Fmt<DT>::V;
    constexpr int ES = Fmt<DT>::esize;
    constexpr int CPT = kTiesMaxBlock / kT / V;  // 2 (bf16) or 4 (fp32)
    constexpr int E = CPT * V;                   // 16 elements per thread
    __shared__ TiesSmem sm;
    const int64_t b = blockIdx.x;
    const int t = threadIdx.x;
    const uint32_t g = src.block(b);
    const uint64_t off = boff[g];
    const uint32_t n = blen[g];
    const uint32_t m = mask[g] & kmask;  // bits of experts >= K are ignored
    const uint32_t nch = n / V;
    const uint4* pb = chunk_ptr(base, off, ES);
    uint4* po = reinterpret_cast<uint4*>(static_cast<char*>(out) + off * ES);
    count_expert_bytes(ctr, m, n, ES);

    const double kk = ceil(density * (double)n);
    const uint32_t k = (kk >= (double)n) ? n : (uint32_t)kk;

    bool ok[CPT];
    float x0[E];
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        const uint32_t c = q * kT + t;
        ok[q] = c < nch;
        uint4 raw = make_uint4(0, 0, 0, 0);
        if (ok[q])
            raw = pb[c];
        Fmt<DT>::unpack(raw, &x0[q * V]);
    }
    float sg[E], ps[E], ns[E];
    uint32_t cnt[E];  // positives in the low 16 bits, negatives in the high 16 bits
#pragma unroll
    for (int e = 0; e < E; ++e) {
        sg[e] = 0.0f;
        ps[e] = 0.0f;
        ns[e] = 0.0f;
        cnt[e] = 0u;
    }
    for (int q = t; q < 1024; q += kT) {
        sm.hA[0][q] = 0u;
        sm.hB[q] = 0u;
        sm.hBmin[q] = 0xffffffffu;
        sm.hBmax[q] = 0u;
    }
    for (int q = t; q < 2048; q += kT)
        sm.hC[q] = 0u;
    __syncthreads();

    uint32_t mm = m;
    uint4 nxt[CPT];
    int rank = 0;
    if (mm) {
        const uint4* pe = src.expert(__builtin_ctz(mm), 0, b, off, n, ES);
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            if (ok[q])
                nxt[q] = pe[q * kT + t];
    }
    int it = 0;
    while (mm) {
        mm &= mm - 1u;
        uint4 cur[CPT];
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            cur[q] = nxt[q];
        if (mm) {  // prefetch the next selected expert while this one is trimmed
            const uint4* pe = src.expert(__builtin_ctz(mm), rank + 1, b, off, n, ES);
#pragma unroll
            for (int q = 0; q < CPT; ++q)
                if (ok[q])
                    nxt[q] = pe[q * kT + t];
        }
        float d[E];
        uint32_t mg[E];
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            float x[V];
            Fmt<DT>::unpack(ok[q] ? cur[q] : make_uint4(0, 0, 0, 0), x);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int e = q * V + v;
                d[e] = ok[q] ? (x[v] - x0[e]) : 0.0f;
                mg[e] = __float_as_uint(d[e]) & 0x7fffffffu;
            }
        }
        const uint32_t tau = ties_threshold<E>(mg, k, it, sm);
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const bool keep = (mg[e] >= tau) && (mg[e] != 0u);
            const float tv = keep ? d[e] : 0.0f;
            sg[e] = sg[e] + tv;
            ps[e] = ps[e] + fmaxf(tv, 0.0f);
            ns[e] = ns[e] + fminf(tv, 0.0f);
            cnt[e] += keep ? ((d[e] > 0.0f) ? 1u : 0x10000u) : 0u;
        }
        ++it;
        ++rank;
    }
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        if (!ok[q])
            continue;
        float y[V];
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int e = q * V + v;
            float mean = 0.0f;
            if (sg[e] > 0.0f)
                mean = ps[e] / (float)(cnt[e] & 0xffffu);
            else if (sg[e] < 0.0f)
                mean = ns[e] / (float)(cnt[e] >> 16);
            y[v] = fmaf(lambda, mean, x0[e]);
        }
        po[q * kT + t] = Fmt<DT>::pack(y);
    }
}

template <int DT, class Src>
hipError_t launch_typed(const BlockTable& bt, const MergeArgs& a, const Src& src, const void* base,
                        int K, const uint32_t* mask, int64_t nb, void* out, unsigned long long* ctr,
                        hipStream_t s)
{
    const uint32_t kmask = (K >= 32) ? 0xffffffffu : ((1u << K) - 1u);
    if (nb == 0)
        return hipSuccess;
    const dim3 grid((unsigned)nb), block(kT);
    const uint32_t T = (uint32_t)floor(a.p * 4294967296.0);
    const float scale = (float)(1.0 / (1.0 - a.p));
    switch (a.op) {
    case Op::AVG:
        hipLaunchKernelGGL((k_merge_elem<DT, M_AVG, Src>), grid, block, 0, s, src, base, mask, bt.d_off,
                           bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, 0u, 1.0f, 0u, kmask, out, ctr);
        break;
    case Op::DARE_LINEAR:
        hipLaunchKernelGGL((k_merge_elem<DT, M_DARE_LIN, Src>), grid, block, 0, s, src, base, mask,
                           bt.d_off, bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, T, scale,
                           a.seed, kmask, out, ctr);
        break;
    case Op::DARE_SIGN:
        hipLaunchKernelGGL((k_merge_elem<DT, M_DARE_SIGN, Src>), grid, block, 0, s, src, base, mask,
                           bt.d_off, bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, T, scale,
                           a.seed, kmask, out, ctr);
        break;
    case Op::TIES:
        hipLaunchKernelGGL((k_merge_ties<DT, Src>), grid, block, 0, s, src, base, mask, bt.d_off,
                           bt.d_len, a.density, a.lambda, kmask, out, ctr);
        break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const BlockTable& bt, const MergeArgs& a, const void* base,
                        const ExpertPtrs& ex, int K, const uint32_t* mask, void* out,
                        unsigned long long* counters, hipStream_t s)
{
    DevSrc src{ex};
    if (bt.dtype == 0)
        return launch_typed<0>(bt, a, src, base, K, mask, bt.G, out, counters, s);
    return launch_typed<1>(bt, a, src, base, K, mask, bt.G, out, counters, s);
}

hipError_t launch_merge_staged(const BlockTable& bt, const MergeArgs& a, const void* base,
                               const void* stage, int K, const uint32_t* mask,
                               const uint32_t* gid, const uint64_t* soff, int64_t nb, void* out,
                               unsigned long long* counters, hipStream_t s)
{
    StagedSrc src{static_cast<const char*>(stage), gid, soff};
    if (bt.dtype == 0)
        return launch_typed<0>(bt, a, src, base, K, mask, nb, out, counters, s);
    return launch_typed<1>(bt, a, src, base, K, mask, nb, out, counters, s);
}

}  // namespace mp
