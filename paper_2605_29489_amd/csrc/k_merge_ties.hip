// The TIES merge operator with the trim inside the merge (Appendix A.1:
// trim, elect signs, average the sign-consistent entries, over the masked
// deltas), one workgroup per block.
//
// Two copies of each window bin: registers (about 120 per lane: the K
// experts' 16 deltas each) hold the kernel at four waves per SIMD either
// way, and halving the histogram rows (33 to 17 KiB per workgroup) took the
// merges on the Qwen2.5-1.5B-shaped family at B = 25/50/100% from 1.90 /
// 2.71 / 4.03 ms to 1.82 / 2.61 / 3.97 ms.  A fifth wave spills the deltas.
#define MP_TIES_NC 2
#include "device_common.h"
#include "merge_src.h"
#include "mp_internal.h"
#include "ties_select.h"

namespace mp {

namespace {

// Divisors for the mean of at most four agreeing entries: {den, fl32(1/den)}
// at index den (1..4; the others are unused and hold {1, 1}).
__device__ inline float2 ties_divisor(int i)
{
    const float r = (i == 2) ? 0.5f : (i == 3) ? 0x1.555556p-2f : (i == 4) ? 0.25f : 1.0f;
    return make_float2((i >= 2 && i <= 4) ? (float)i : 1.0f, r);
}

// ------------------------------------------------------------ TIES
// One 256-thread workgroup per block.  The block's deltas (<= 4096
// elements: 16 per thread and expert) stay in registers, and up to four
// selected experts are trimmed together so that they share the barriers.
// Per expert, tau = the k-th largest |d| is found on the fp32 magnitude bit
// patterns (window, bins and fallbacks as in ties_select.h):
//  A  the block maximum M (wave maxima, one value per wave in LDS);
//  B  the elements of the binade of M and of the three binades below it
//     are counted into the window histogram (nothing lies above it), first
//     only those at or above a guess at tau (a fixed fraction of the normal
//     quantile for rho at the deltas' root mean square): the bins from the
//     guess's up are then exact, and the guess keeps most elements out of
//     the LDS atomics;
//  C  one wave per expert walks the histogram from the top to the bin where
//     the count reaches k, needing r more elements from that bin (if the
//     count above the guess falls short of k, the rest of the window is
//     added and the walk repeated; rare).  If fewer
//     than r of the bin's elements lie above its floor, the floor is the
//     k-th largest value; if the whole bin is needed its floor keeps the
//     same elements as the k-th largest.  Either way the keep set is known;
//  D  otherwise (rare) the bin's elements are listed in LDS and one wave
//     resolves the low bits one at a time; if tau lies below the window
//     or the list overflows, an exact 3-level radix select over all
//     elements runs instead.
// Then one pass over the elements keeps |d| >= tau (tau is at least the
// smallest positive pattern, so a kept delta is not zero), elects a sign by
// comparing the fp32 sums P of the positive and N of the negative kept
// deltas (+ if P > -N, - if P < -N, none if equal) and takes the mean of
// the agreeing entries.
namespace ties {
using namespace ::mp::ties;  // window constants of ties_select.h
#ifndef MP_TIES_NT
#define MP_TIES_NT 256
#endif
constexpr int NT = MP_TIES_NT;           // threads per workgroup
constexpr int EPT = kTiesMaxBlock / NT;  // elements per thread and expert
constexpr int NW = NT / 64;              // waves per workgroup
constexpr int GS = 4;                    // experts trimmed together (one scanning wave each)
constexpr uint32_t RETRY = 4u;           // state: the cut lies below the first pass's floor
}  // namespace ties

// Sum over the 64 lanes of a wave, returned wave-uniform: the butterfly of
// wave_max_u32 (quad permutes, row mirrors, row broadcasts) with adds.  The
// order of the adds differs from a sequential sum; the result only guides
// the threshold guess.
template <int CTRL, int ROW_MASK, int BANK_MASK, bool BOUND_CTRL>
__device__ inline float dpp_f32(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, BANK_MASK, BOUND_CTRL));
}
__device__ inline float wave_sum_f32(float v)
{
    v = v + dpp_f32<0xb1, 0xf, 0xf, true>(v);    // quad_perm [1,0,3,2]
    v = v + dpp_f32<0x4e, 0xf, 0xf, true>(v);    // quad_perm [2,3,0,1]
    v = v + dpp_f32<0x141, 0xf, 0xf, true>(v);   // row_half_mirror
    v = v + dpp_f32<0x140, 0xf, 0xf, true>(v);   // row_mirror
    v = v + dpp_f32<0x142, 0xa, 0xf, false>(v);  // row_bcast:15
    v = v + dpp_f32<0x143, 0xc, 0xf, false>(v);  // row_bcast:31
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// The window histogram's update for the values with lo <= |d| < hi
// (magnitude patterns): the part of the window below a first pass's floor.
__device__ inline void window_add_range(char* base, uint32_t bits, uint32_t lo, uint32_t hi, uint32_t koff)
{
    using namespace ties;
    const uint32_t mg = bits & 0x7fffffffu;
    const uint32_t boff = (__builtin_amdgcn_ubfe(bits, KS, 31 - KS) << LG) + koff;
    const uint32_t inc = (min(bits & ((1u << KS) - 1u), 1u) << 16) + 1u;
    if (mg >= lo && mg < hi)
        atomicAdd(reinterpret_cast<uint32_t*>(base + boff), inc);
}

struct TiesSmem {
    uint32_t h[ties::GS][ties::NB];     // window histogram, then candidate list / radix levels
    uint32_t wmax[ties::GS][ties::NW];  // per-wave maximum |d| pattern
    float wss[ties::GS][ties::NW];      // per-wave sum of d^2 (for the guess at tau)
    uint32_t flo[ties::GS];             // floor of the first histogram pass (a bin floor)
    uint32_t st[ties::GS][4];           // state, tau (or bucket key), rank in the bucket, list length
    float2 rd[8];                       // divisors {den, 1/den} of the small-K mean
};

template <int DT, int NT, int CPT>
__device__ inline void load_chunks(const uint4* __restrict__ p, uint32_t nch, uint4 (&dst)[CPT])
{
    const int t = threadIdx.x;
#pragma unroll
    for (int q = 0; q < CPT; ++q)
        dst[q] = (q * NT + t < nch) ? ld16s(&p[q * NT + t]) : make_uint4(0u, 0u, 0u, 0u);
}

// Whole workgroup: exact k-th largest magnitude pattern of slot j over all
// of its elements (padding elements are zeros, which cannot change the k
// largest), by levels from bit 30 down in digits that fit the histogram row
// (30..20, 19..9, 8..0 for 2048 counters).  Returns the pattern (at least 1:
// a zero threshold keeps every nonzero delta).
template <int E>
__device__ inline uint32_t block_radix_select(TiesSmem& sm, int j, const float (&dj)[E], uint32_t k, int t,
                                              int lane, int wave)
{
    constexpr int WD = (ties::NB >= 2048) ? 11 : (ties::NB >= 1024) ? 10 : 9;
    constexpr int NL = (31 + WD - 1) / WD;
    uint32_t* h = sm.h[j];
    uint32_t pref = 0u, r = k;
#pragma unroll 1
    for (int lv = 0; lv < NL; ++lv) {
        const int top_bit = 31 - lv * WD;  // one past the digit's highest bit
        const int sh = (top_bit - WD > 0) ? top_bit - WD : 0;
        const int wd = top_bit - sh;
        __syncthreads();  // earlier readers of h and st are done
        for (int q = t; q < ties::NB; q += ties::NT)
            h[q] = 0u;
        __syncthreads();
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const uint32_t mg = __float_as_uint(dj[e]) & 0x7fffffffu;
            const uint32_t hi = (lv == 0) ? 0u : (mg >> (sh + wd));
            if (hi == pref)
                atomicAdd(&h[(mg >> sh) & ((1u << wd) - 1u)], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            const Cut c = wave_find_from_top<1>(h, (1 << wd) - 1, r, lane);
            if (lane == 0) {
                sm.st[j][1] = c.bin;
                sm.st[j][2] = c.rank;
            }
        }
        __syncthreads();
        pref = (pref << wd) | uniform_u32(sm.st[j][1]);
        r = uniform_u32(sm.st[j][2]);
    }
    return max(pref, 1u);
}

// Issues the loads of up to GS selected experts of one block (the set bits
// of gm, in increasing expert order; rank0 = rank of the first among all the
// block's selected experts) into raw.
template <int DT, int CPT, class Src>
__device__ inline void ties_load_group(const Src& src, int64_t b, uint64_t off, uint32_t n, uint32_t gm, int rank0,
                                       uint4 (&raw)[ties::GS][CPT], unsigned long long* ctr)
{
    constexpr int ES = Fmt<DT>::esize;
    const int ns = __popc(gm);
    const uint32_t nch = n / Fmt<DT>::V;
    uint32_t mm = gm;
#pragma unroll
    for (int j = 0; j < ties::GS; ++j) {
        if (j < ns) {
            const int i = __builtin_ctz(mm);
            mm &= mm - 1u;
            load_chunks<DT, ties::NT, CPT>(src.expert(i, rank0 + j, b, off, n, ES), nch, raw[j]);
            count_loaded<ties::NT, CPT>(ctr, i, nch);
        }
    }
}

// Phase A of a trim group: clears the histogram rows of the ns slots in use
// (their previous readers passed a barrier since), forms the deltas and
// publishes the wave maxima of |d|.
template <int DT, int CPT>
__device__ inline void ties_deltas(TiesSmem& sm, const uint4 (&raw)[ties::GS][CPT], int ns,
                                   const float (&x0)[CPT * Fmt<DT>::V], float (&d)[ties::GS][CPT * Fmt<DT>::V],
                                   float bsub)
{
    using namespace ties;
    constexpr int V = Fmt<DT>::V;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
#pragma unroll
    for (int j = 0; j < GS; ++j) {
        if (j < ns) {
#pragma unroll
            for (int q = 0; q < (NB + 4 * NT - 1) / (4 * NT); ++q) {
                const int w = 4 * (q * NT + t);
                if (NB % (4 * NT) == 0 || w < NB)
                    *reinterpret_cast<uint4*>(&sm.h[j][w]) = make_uint4(0u, 0u, 0u, 0u);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < GS; ++j) {
        if (j < ns) {
            float mx = 0.0f, ss = 0.0f;
#pragma unroll
            for (int q = 0; q < CPT; ++q) {
                float x[V];
                Fmt<DT>::unpack(raw[j][q], x);
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    d[j][q * V + v] = fmaf(-bsub, x0[q * V + v], x[v]);  // x - x0 or the delta; padding 0
                    ss = fmaf(d[j][q * V + v], d[j][q * V + v], ss);
                }
#pragma unroll
                for (int v = 0; v < V; v += 2)  // pairs: one three-way maximum each
                    mx = fmaxf(mx, fmaxf(fabsf(d[j][q * V + v]), fabsf(d[j][q * V + v + 1])));
            }
            const uint32_t w = wave_max_u32(__float_as_uint(mx));
            ss = wave_sum_f32(ss);
            if (lane == 0) {
                sm.wmax[j][wave] = w;
                sm.wss[j][wave] = ss;
            }
        }
    }
}

// Phases B-D of a trim group whose deltas are in d and whose wave maxima
// were published by ties_deltas: leaves the thresholds in tau (wave-uniform
// patterns) and returns the largest |d| pattern of the group's slots.  Every
// thread of the workgroup calls it.
template <int E>
__device__ inline uint32_t ties_select_group(TiesSmem& sm, uint32_t n, uint32_t k, int ns, float gcoef,
                                             const float (&d)[ties::GS][E], uint32_t (&tau)[ties::GS])
{
    using namespace ties;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    __syncthreads();
    // ---- B: window histograms of the values at or above each slot's guess
    uint32_t bmax[GS], flo[GS];
#pragma unroll
    for (int j = 0; j < GS; ++j) {
        bmax[j] = 0u;
        flo[j] = 0u;
        if (j < ns) {
            float ss = 0.0f;
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                bmax[j] = max(bmax[j], uniform_u32(sm.wmax[j][w]));
                ss = ss + __uint_as_float(uniform_u32(__float_as_uint(sm.wss[j][w])));
            }
            if (bmax[j] != 0u) {
                int wb;
                const uint32_t koff = window_koff(bmax[j], lane, &wb);
                const uint32_t wfloor = window_floor(wb);
                // the guess only decides which values the first pass counts
                // (any value, NaN included, leaves tau exact)
                const float gf = gcoef * __builtin_amdgcn_sqrtf(ss * __builtin_amdgcn_rcpf((float)n));
                const uint32_t guess = (gcoef > 0.0f) ? __float_as_uint(gf) : 0u;
                flo[j] = (guess > wfloor) ? (guess >> KS) << KS : wfloor;
                if (t == 0)
                    sm.flo[j] = flo[j];
                char* row = reinterpret_cast<char*>(sm.h[j]);
                uint32_t inc = 1u;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    window_add<false>(row, __float_as_uint(d[j][e]), flo[j], koff, inc);
            }
        }
    }
    __syncthreads();
    // ---- C: one wave per expert finds the bin of the k-th largest
    // wave j (all lanes): the state of slot j from a walk of its histogram
    auto walk = [&](int j, uint32_t bm, bool partial) {
        const Cut c = wave_find_from_top<NC>(sm.h[j], NBIN - 1, k, lane);
        const int wb = window_base(bm);
        uint32_t state = DONE, v1 = 1u, v2 = 0u;  // v1: tau, or the bucket key to refine
        if (!c.found) {
            state = partial ? RETRY : RADIX;  // below the first pass's floor, or below the window
        } else if (c.aux < c.rank || c.count == c.rank) {
            v1 = max((uint32_t)(wb + (int)c.bin) << KS, 1u);
        } else {
            state = LIST;
            v1 = (uint32_t)(wb + (int)c.bin);
            v2 = c.rank;
        }
        if (lane == 0) {
            sm.st[j][0] = state;
            sm.st[j][1] = v1;
            sm.st[j][2] = v2;
            sm.st[j][3] = 0u;
        }
    };
    if (wave < ns) {
        const int j = wave;
        uint32_t bm = 0u;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            bm = max(bm, uniform_u32(sm.wmax[j][w]));
        if (bm != 0u && k < n) {  // all zero, or k = n: keep every nonzero
            walk(j, bm, uniform_u32(sm.flo[j]) > window_floor(window_base(bm)));
        } else if (lane == 0) {
            sm.st[j][0] = DONE;
            sm.st[j][1] = 1u;
            sm.st[j][2] = 0u;
            sm.st[j][3] = 0u;
        }
    }
    __syncthreads();
    // ---- C' (rare): the cut lies below the guess; add the rest of the
    // window and walk again
    uint32_t anyst = 0u;
#pragma unroll
    for (int j = 0; j < GS; ++j)
        if (j < ns)
            anyst |= uniform_u32(sm.st[j][0]);
    if (anyst & RETRY) {
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            if (j < ns && uniform_u32(sm.st[j][0]) == RETRY) {
                int wb;
                const uint32_t koff = window_koff(bmax[j], lane, &wb);
                char* row = reinterpret_cast<char*>(sm.h[j]);
#pragma unroll
                for (int e = 0; e < E; ++e)
                    window_add_range(row, __float_as_uint(d[j][e]), window_floor(wb), flo[j], koff);
            }
        }
        __syncthreads();
        if (wave < ns && uniform_u32(sm.st[wave][0]) == RETRY) {
            const int j = wave;
            uint32_t bm = 0u;
#pragma unroll
            for (int w = 0; w < NW; ++w)
                bm = max(bm, uniform_u32(sm.wmax[j][w]));
            walk(j, bm, false);
        }
        __syncthreads();
        anyst = 0u;
#pragma unroll
        for (int j = 0; j < GS; ++j)
            if (j < ns)
                anyst |= uniform_u32(sm.st[j][0]);
    }
    // ---- D (rare): resolve inside the bucket, or select exactly
    if (anyst != 0u) {
        if (anyst & LIST) {
#pragma unroll
            for (int j = 0; j < GS; ++j) {
                if (j < ns && uniform_u32(sm.st[j][0]) == LIST) {
                    const uint32_t key = uniform_u32(sm.st[j][1]);
#pragma unroll
                    for (int e = 0; e < E; ++e) {
                        const uint32_t mg = __float_as_uint(d[j][e]) & 0x7fffffffu;
                        const bool in = (mg >> KS) == key;
                        const unsigned long long bal = __ballot(in);
                        if (bal) {  // wave-uniform
                            uint32_t pos0 = 0u;
                            if (lane == 0)
                                pos0 = atomicAdd(&sm.st[j][3], (uint32_t)__popcll(bal));
                            pos0 = uniform_u32(pos0);
                            const uint32_t pos =
                                pos0 + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
                            if (in && pos < (uint32_t)NB)
                                sm.h[j][pos] = mg;
                        }
                    }
                }
            }
            __syncthreads();
            if (wave < ns && uniform_u32(sm.st[wave][0]) == LIST) {
                const int j = wave;
                const uint32_t cnt = uniform_u32(sm.st[j][3]);
                if (cnt <= (uint32_t)NB) {
                    const uint32_t tv = wave_select_list(sm.h[j], cnt, uniform_u32(sm.st[j][1]),
                                                         uniform_u32(sm.st[j][2]), lane);
                    if (lane == 0) {
                        sm.st[j][0] = DONE;
                        sm.st[j][1] = max(tv, 1u);
                    }
                } else if (lane == 0) {
                    sm.st[j][0] = RADIX;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            if (j < ns && uniform_u32(sm.st[j][0]) == RADIX) {
                const uint32_t tv = block_radix_select<E>(sm, j, d[j], k, t, lane, wave);
                __syncthreads();  // every thread has read the last level's result
                if (t == 0) {
                    sm.st[j][0] = DONE;
                    sm.st[j][1] = tv;
                }
                __syncthreads();
            }
        }
    }
#pragma unroll
    for (int j = 0; j < GS; ++j)
        tau[j] = (j < ns) ? uniform_u32(sm.st[j][1]) : 0xffffffffu;
    uint32_t top = 0u;
#pragma unroll
    for (int j = 0; j < GS; ++j)
        top = max(top, bmax[j]);
    return top;
}

// Loads and trims up to GS selected experts of one block (see
// ties_load_group): leaves the deltas in d and the thresholds in tau, and
// returns the largest |d| pattern of the group.
template <int DT, int CPT, class Src>
__device__ inline uint32_t ties_trim_group(TiesSmem& sm, const Src& src, int64_t b, uint64_t off, uint32_t n,
                                       uint32_t k, uint32_t gm, int rank0, const float (&x0)[CPT * Fmt<DT>::V],
                                       float (&d)[ties::GS][CPT * Fmt<DT>::V], uint32_t (&tau)[ties::GS],
                                       float bsub, float gcoef, unsigned long long* ctr)
{
    uint4 raw[ties::GS][CPT];
    ties_load_group<DT, CPT>(src, b, off, n, gm, rank0, raw, ctr);
    const int ns = __popc(gm);
    ties_deltas<DT, CPT>(sm, raw, ns, x0, d, bsub);
    return ties_select_group<CPT * Fmt<DT>::V>(sm, n, k, ns, gcoef, d, tau);
}

// Keep test and the running signed masses of element e over NS slots, with
// the kept counts np (positive) and nn (negative).  tau is at least the
// smallest positive pattern, so d >= tau keeps a positive delta and
// -d >= tau a negative one; a zero or NaN delta is never kept.  FRESH: the
// masses and counts start here (+0 + x is x for every term, which is +0 or
// a nonzero delta, so the first term is assigned).
template <int NS, bool FRESH>
__device__ inline void ties_accumulate(const float (&d)[ties::GS][ties::EPT], const uint32_t (&tau)[ties::GS], int e,
                                       float& P, float& N, uint32_t& np, uint32_t& nn)
{
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const float dj = d[j][e];
        const float t = __uint_as_float(tau[j]);
        const bool kp = dj >= t;
        const bool kn = -dj >= t;
        if (FRESH && j == 0) {
            P = kp ? dj : 0.0f;
            N = kn ? dj : 0.0f;
            np = kp ? 1u : 0u;
            nn = kn ? 1u : 0u;
        } else {
            P = P + (kp ? dj : 0.0f);
            N = N + (kn ? dj : 0.0f);
            np += kp ? 1u : 0u;
            nn += kn ? 1u : 0u;
        }
    }
}

// Sign election (+ if the fp32 positive kept mass P exceeds -N, the negated
// negative mass, - if it is below, none if equal) and the mean of the agreeing entries, for the V elements of one
// chunk of a block with NS (2..4) selected experts; then y = lambda * mean
// + x0, rounded once, is stored.  With at most two agreeing entries the mean
// is the entry or an exact halving.  Otherwise q = mean * fl32(1/den) and one
// residual step q + fl32(mean - den*q) * fl32(1/den) give the correctly
// rounded quotient of a finite mass: for den = 1, 2, 4 the product is
// already correctly rounded and the residual term adds exactly nothing; for
// den = 3 this is Markstein's correction, checked against IEEE division on
// all 2^32 fp32 patterns (only -0 comes out as +0, and an elected mass is
// never zero).  IEEE: the block holds a |d| of at least 2^125, so a mass of
// up to four terms may be infinite (the residual step would make it NaN);
// such blocks divide.
template <int DT, int NS, bool IEEE>
__device__ inline void ties_store_small(const float (&P)[Fmt<DT>::V], const float (&N)[Fmt<DT>::V],
                                        const uint32_t (&np)[Fmt<DT>::V], const uint32_t (&nn)[Fmt<DT>::V],
                                        const float* x0, float lambda, const float2* rd,
                                        uint4* __restrict__ dst, bool ok)
{
    constexpr int V = Fmt<DT>::V;
    float y[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
        const bool up = P[v] > -N[v];
        const bool dn = P[v] < -N[v];
        const float num = up ? P[v] : (dn ? N[v] : 0.0f);
        const uint32_t den = up ? np[v] : (dn ? nn[v] : 1u);
        float q;
        if (NS <= 2) {
            q = (den == 2u) ? num * 0.5f : num;
        } else if (IEEE) {
            q = num / (float)den;
        } else {
            const float2 c = rd[den];
            const float q0 = num * c.y;
            q = fmaf(fmaf(-c.x, q0, num), c.y, q0);
        }
        y[v] = fmaf(lambda, q, x0[v]);
    }
    if (ok)
        st16s(dst, Fmt<DT>::pack(y));
}

// Election and mean for any number of agreeing entries (counts packed:
// positive in the low, negative in the high half), then the store.
template <int DT>
__device__ inline void ties_store_chunk(const float (&P)[Fmt<DT>::V], const float (&N)[Fmt<DT>::V],
                                        const uint32_t (&cnt)[Fmt<DT>::V], const float* x0, float lambda,
                                        uint4* __restrict__ dst, bool ok)
{
    constexpr int V = Fmt<DT>::V;
    float num[V];
    uint32_t den[V];
    bool odd = false;  // some agreeing count is not a power of two
#pragma unroll
    for (int v = 0; v < V; ++v) {
        const bool up = P[v] > -N[v];
        const bool dn = P[v] < -N[v];
        num[v] = up ? P[v] : (dn ? N[v] : 0.0f);
        den[v] = up ? (cnt[v] & 0xffffu) : (dn ? (cnt[v] >> 16) : 1u);
        odd |= (den[v] & (den[v] - 1u)) != 0u;
    }
    if (__any(odd)) {
#pragma unroll
        for (int v = 0; v < V; ++v)
            num[v] = num[v] / (float)den[v];
    } else {
        // division by 2^s is exact scaling (correctly rounded, as the quotient)
#pragma unroll
        for (int v = 0; v < V; ++v)
            num[v] = num[v] * __uint_as_float((127u - (uint32_t)__builtin_ctz(den[v])) << 23);
    }
    if (ok) {
        float y[V];
#pragma unroll
        for (int v = 0; v < V; ++v)
            y[v] = fmaf(lambda, num[v], x0[v]);
        st16s(dst, Fmt<DT>::pack(y));
    }
}

// All selected experts trimmed in one group: accumulate and store chunk by
// chunk (IEEE as for ties_store_small).
template <int DT, int NS, bool IEEE = false>
__device__ inline void ties_finish_single(const float (&d)[ties::GS][ties::EPT], const uint32_t (&tau)[ties::GS],
                                          const float (&x0)[ties::EPT], float lambda, const float2* rd,
                                          uint4* __restrict__ po, uint32_t nch)
{
    constexpr int V = Fmt<DT>::V, CPT = ties::EPT / V;
    const int t = threadIdx.x;
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        if (NS <= 1) {
            // one expert (or none): the elected sign is the kept delta's own, and
            // the mean of one entry is the entry
            if (q * ties::NT + t < (int)nch) {
                float y[V];
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    float mean = 0.0f;
                    if (NS == 1) {
                        const float dj = d[0][q * V + v];
                        mean = (fabsf(dj) >= __uint_as_float(tau[0])) ? dj : 0.0f;
                    }
                    y[v] = fmaf(lambda, mean, x0[q * V + v]);
                }
                st16s(&po[q * ties::NT + t], Fmt<DT>::pack(y));
            }
            continue;
        }
        float P[V], N[V];
        uint32_t np[V], nn[V];
#pragma unroll
        for (int v = 0; v < V; ++v)
            ties_accumulate<NS, true>(d, tau, q * V + v, P[v], N[v], np[v], nn[v]);
        ties_store_small<DT, NS, IEEE>(P, N, np, nn, &x0[q * V], lambda, rd, po + q * ties::NT + t,
                                       q * ties::NT + t < (int)nch);
    }
}

// Several groups: the signed masses and the packed counts are carried across
// groups.
template <int NS>
__device__ inline void ties_accumulate_all(const float (&d)[ties::GS][ties::EPT], const uint32_t (&tau)[ties::GS],
                                           float (&P)[ties::EPT], float (&N)[ties::EPT], uint32_t (&cnt)[ties::EPT])
{
#pragma unroll
    for (int e = 0; e < ties::EPT; ++e) {
        uint32_t np = 0u, nn = 0u;
        ties_accumulate<NS, false>(d, tau, e, P[e], N[e], np, nn);
        cnt[e] += np + (nn << 16);
    }
}

// MULTI = false: K <= GS, every selected expert is trimmed in one group.
// MULTI = true: groups of GS experts in increasing order, with the signed
// masses and counts carried across groups.
template <int DT, bool MULTI, class Src>
#ifndef MP_TIES_WAVES
#define MP_TIES_WAVES (ties::NT / 64)
#endif
__global__ __launch_bounds__(ties::NT, MULTI ? ties::NT / 128 : MP_TIES_WAVES) void k_merge_ties(Src src, const void* __restrict__ base,
                                                         const uint32_t* __restrict__ mask,
                                                         const uint64_t* __restrict__ boff,
                                                         const uint32_t* __restrict__ blen, double density,
                                                         uint32_t n_full, uint32_t k_full, float lambda,
                                                         uint32_t kmask, void* __restrict__ out,
                                                         unsigned long long* __restrict__ ctr, float bsub,
                                                         float gcoef)
{
    using namespace ties;
    constexpr int V = Fmt<DT>::V, ES = Fmt<DT>::esize;
    constexpr int CPT = kTiesMaxBlock / NT / V;  // chunks per thread and expert
    constexpr int E = CPT * V;
    static_assert(E == EPT, "elements per thread and expert");
    __shared__ TiesSmem sm;
    if (threadIdx.x < 8)  // read after the trim's barriers
        sm.rd[threadIdx.x] = ties_divisor((int)threadIdx.x);
    const int64_t b = blockIdx.x;
    const uint32_t g = uniform_u32(src.block(b));
    const uint64_t off = boff[g];
    const uint32_t n = blen[g];
    uint32_t k = k_full;
    if (n != n_full) {
        const double kk = ceil(density * (double)n);
        k = (kk >= (double)n) ? n : (uint32_t)kk;
    }
    const uint32_t m = (k != 0u) ? (mask[g] & kmask) : 0u;  // density 0 keeps nothing: no expert is read
    const uint32_t nch = n / V;
    uint4 x0raw[CPT];
    load_chunks<DT, NT, CPT>(chunk_ptr(base, off, ES), nch, x0raw);
    float x0[E];
    uint4* po = reinterpret_cast<uint4*>(static_cast<char*>(out) + off * ES);

    float d[GS][E];
    uint32_t tau[GS];
    if (!MULTI) {
        const int ns = __popc(m);
        // every load of the block is issued before the base is unpacked
        uint4 raw[GS][CPT];
        ties_load_group<DT, CPT>(src, b, off, n, m, 0, raw, ctr);
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            Fmt<DT>::unpack(x0raw[q], &x0[q * V]);
        uint32_t top = 0u;
        if (ns != 0) {
            ties_deltas<DT, CPT>(sm, raw, ns, x0, d, bsub);
            top = ties_select_group<E>(sm, n, k, ns, gcoef, d, tau);
        }
        const bool big = top >= 0x7e000000u;  // some |d| >= 2^125: masses may overflow
        switch (ns) {
        case 0: ties_finish_single<DT, 0>(d, tau, x0, lambda, sm.rd, po, nch); break;
        case 1: ties_finish_single<DT, 1>(d, tau, x0, lambda, sm.rd, po, nch); break;
        case 2: ties_finish_single<DT, 2>(d, tau, x0, lambda, sm.rd, po, nch); break;
        case 3:
            if (big)
                ties_finish_single<DT, 3, true>(d, tau, x0, lambda, sm.rd, po, nch);
            else
                ties_finish_single<DT, 3>(d, tau, x0, lambda, sm.rd, po, nch);
            break;
        default:
            if (big)
                ties_finish_single<DT, 4, true>(d, tau, x0, lambda, sm.rd, po, nch);
            else
                ties_finish_single<DT, 4>(d, tau, x0, lambda, sm.rd, po, nch);
            break;
        }
    } else {
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            Fmt<DT>::unpack(x0raw[q], &x0[q * V]);
        float P[E], N[E];
        uint32_t cnt[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            P[e] = 0.0f;
            N[e] = 0.0f;
            cnt[e] = 0u;
        }
        uint32_t mm = m;
        int rank0 = 0;
        while (mm) {  // wave-uniform
            uint32_t gm = 0u;
            for (int j = 0; j < GS && mm; ++j) {
                gm |= mm & (0u - mm);
                mm &= mm - 1u;
            }
            ties_trim_group<DT, CPT>(sm, src, b, off, n, k, gm, rank0, x0, d, tau, bsub, gcoef, ctr);
            const int ns = __popc(gm);
            switch (ns) {
            case 1: ties_accumulate_all<1>(d, tau, P, N, cnt); break;
            case 2: ties_accumulate_all<2>(d, tau, P, N, cnt); break;
            case 3: ties_accumulate_all<3>(d, tau, P, N, cnt); break;
            default: ties_accumulate_all<4>(d, tau, P, N, cnt); break;
            }
            rank0 += ns;
        }
        const int t = threadIdx.x;
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            float Pq[V], Nq[V];
            uint32_t cq[V];
#pragma unroll
            for (int v = 0; v < V; ++v) {
                Pq[v] = P[q * V + v];
                Nq[v] = N[q * V + v];
                cq[v] = cnt[q * V + v];
            }
            ties_store_chunk<DT>(Pq, Nq, cq, &x0[q * V], lambda, po + q * NT + t, q * NT + t < (int)nch);
        }
    }
}

template <int DT, class Src>
hipError_t launch_ties_typed(const BlockTable& bt, const MergeArgs& a, const Src& src, const void* base, int K,
                             const uint32_t* mask, int64_t nb, void* out, unsigned long long* ctr, hipStream_t s)
{
    const uint32_t kmask = (K >= 32) ? 0xffffffffu : ((1u << K) - 1u);
    if (nb == 0)
        return hipSuccess;
    const dim3 grid((unsigned)nb);
    // k for full-length blocks, as the kernel computes it for short ones
    const uint32_t n_full = (uint32_t)bt.block_elems;
    const double kk = ceil(a.density * (double)n_full);
    const uint32_t k_full = (kk >= (double)n_full) ? n_full : (uint32_t)kk;
    // the first histogram pass's guess at tau: 0.8 of the rho-tail quantile
    // of a normal with the deltas' RMS, as in the catalog pass
    const float gcoef = (float)(0.8 * normal_two_sided_quantile(a.density));
    if (K <= ties::GS)
        hipLaunchKernelGGL((k_merge_ties<DT, false, Src>), grid, dim3(ties::NT), 0, s, src, base, mask, bt.d_off,
                           bt.d_len, a.density, n_full, k_full, a.lambda, kmask, out, ctr, a.bsub, gcoef);
    else
        hipLaunchKernelGGL((k_merge_ties<DT, true, Src>), grid, dim3(ties::NT), 0, s, src, base, mask, bt.d_off,
                           bt.d_len, a.density, n_full, k_full, a.lambda, kmask, out, ctr, a.bsub, gcoef);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_merge_ties(const BlockTable& bt, const MergeArgs& a, const void* base, const ExpertPtrs& ex, int K,
                             const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s)
{
    DevSrc src{ex};
    if (bt.dtype == 0)
        return launch_ties_typed<0>(bt, a, src, base, K, mask, bt.G, out, counters, s);
    return launch_ties_typed<1>(bt, a, src, base, K, mask, bt.G, out, counters, s);
}

hipError_t launch_merge_ties_staged(const BlockTable& bt, const MergeArgs& a, const void* base, int K,
                                    const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s,
                                    const void* stage, const uint64_t* soff, int64_t b0, int64_t nb)
{
    StagedSrc src{static_cast<const char*>(stage), soff, b0};
    if (bt.dtype == 0)
        return launch_ties_typed<0>(bt, a, src, base, K, mask, nb, out, counters, s);
    return launch_ties_typed<1>(bt, a, src, base, K, mask, nb, out, counters, s);
}

}  // namespace mp
