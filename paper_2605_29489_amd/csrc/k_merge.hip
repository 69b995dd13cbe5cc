// Mask-aware merge operators Psi_op (Eq. 4; operators of Appendix A.1).
//
// One workgroup per block.  The block's mask word is uniform, so the loop
// over the selected experts is a scalar loop: unselected experts are never
// touched (the zero-completed tuple of Appendix A.1 costs no reads).  Blocks
// are streamed as 16-byte chunks with coalesced loads.
//
//  * AVG / DARE (linear or sign-elect): elementwise.  A thread owns CPT
//    chunks of a tile and loads the chunks of up to 4 selected experts
//    before consuming them in increasing expert order.
//  * TIES: the block's deltas stay in registers while the per-expert trim
//    thresholds are selected in LDS (see the TIES section).
//
// Addressing: expert i's block sits at its layout offset in expert i's
// buffer, which is device memory or pinned host memory read over PCIe.
#include <type_traits>

#include "device_common.h"
#include "mp_internal.h"
#include "ties_select.h"

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

// Divisors for the mean of at most four agreeing entries: {den, fl32(1/den)}
// at index den (1..4; the others are unused and hold {1, 1}).
__device__ inline float2 ties_divisor(int i)
{
    const float r = (i == 2) ? 0.5f : (i == 3) ? 0x1.555556p-2f : (i == 4) ? 0.25f : 1.0f;
    return make_float2((i >= 2 && i <= 4) ? (float)i : 1.0f, r);
}

// ------------------------------------------------------------ elementwise family
enum { M_AVG = 0, M_DARE_LIN = 1, M_DARE_SIGN = 2, M_TIES_TAU = 3, M_AVG_RENORM = 4 };

template <int MODE>
constexpr bool is_avg() { return MODE == M_AVG || MODE == M_AVG_RENORM; }

// Shape of the elementwise kernels (AVG, selected-only AVG, DARE, TIES from
// thresholds), chosen by measurement on MI355X.  A workgroup is one wave;
// each lane owns one 16-byte chunk (bf16) or two (fp32), eight elements, so
// a workgroup covers 512 elements and a 4096-element block takes eight
// (2^sub_log2 workgroups per block; those past the end of a shorter block
// return at once).  No kernel loops over a block: a loop made the compiler
// hoist per-expert addresses out of it and spill them.
//   * Loads are buffer loads with the block as the resource: one 32-bit
//     offset register serves the base, every expert and the output, a load
//     past the block's end returns zeros and a store past it is dropped, so
//     no lane branches.  (Loads under a per-lane condition made the compiler
//     wait for each load before issuing the next.)
//   * The selected experts are read one at a time, in increasing order, each
//     consumed before the next is loaded.  Issuing every stream's load at
//     once measured slower: on this HBM a merge of five streams into one
//     moves 0.67 of peak when each wave keeps all five reads in flight and
//     0.73-0.75 when it reads them in turn, and so did the merges.
//   * AVG (either coefficient rule) does little arithmetic per byte: it
//     reads the block's length, offset and mask together, overlaps the base
//     read with the first expert's, and runs at most 6 waves per SIMD (LDS
//     reserved per workgroup caps the workgroups per CU); fewer requests in
//     flight measured faster for it (2.86 against 3.12 ms at B = 100% on the
//     Qwen2.5-1.5B-shaped family).  The sign-elect and DARE modes, with more
//     arithmetic per element, run 8 waves per SIMD, read the length first
//     (the exit test needs it) and the base before the first expert.
//   * One-wave workgroups measured best among 64 to 512 threads, one or two
//     chunks per lane and one or two passes per workgroup.
constexpr int kTE = 64;
// LDS reserved by each AVG workgroup: 25 of them exceed the CU's 160 KiB,
// so at most 24 (6 waves per SIMD) are resident
constexpr unsigned kAvgLds = 6656;

template <int DT, int MODE, bool COUNT, bool SMALLK, class Src>
__global__ __launch_bounds__(kTE, 8) void k_merge_elem(Src src, const void* __restrict__ base,
                                                      const uint32_t* __restrict__ mask,
                                                      const uint64_t* __restrict__ boff,
                                                      const uint32_t* __restrict__ blen,
                                                      const uint32_t* __restrict__ btensor,
                                                      const uint64_t* __restrict__ belem0, Coeffs alpha,
                                                      float lambda, uint32_t drop_T, float scale, uint32_t seed,
                                                      uint32_t kmask, void* __restrict__ out,
                                                      unsigned long long* __restrict__ ctr,
                                                      const uint32_t* __restrict__ tau, int K, float bsub,
                                                      uint32_t sub_log2)
{
    constexpr int V = Fmt<DT>::V;
    constexpr int ES = Fmt<DT>::esize;
    constexpr int CPT = (DT == 1) ? 1 : 2;  // chunks per lane
    constexpr int E = CPT * V;              // elements per lane (8)
    constexpr bool DARE = MODE == M_DARE_LIN || MODE == M_DARE_SIGN;
    constexpr bool SIGN = MODE == M_DARE_SIGN || MODE == M_TIES_TAU;
    const int64_t b = blockIdx.x >> sub_log2;
    // this workgroup's first chunk of the block
    const uint32_t tile = (blockIdx.x & ((1u << sub_log2) - 1u)) * (uint32_t)(CPT * kTE);
    const int t = threadIdx.x;
    const uint32_t g = src.block(b);
    uint64_t off;
    uint32_t n, mraw;
    if (is_avg<MODE>()) {
        // the block's metadata fetched together (one memory latency)
        off = boff[g];
        n = blen[g];
        mraw = mask[g];
        __asm__ volatile("" : : "s"(off), "s"(n), "s"(mraw), "s"(base), "s"(out));
    }
    else {
        n = blen[g];
    }
    const uint32_t nch = n / V;
    if (tile >= nch)
        return;  // past the end of a shorter block
    if (!is_avg<MODE>()) {
        off = boff[g];
        mraw = mask[g];
    }
    const uint32_t m = mraw & kmask;  // bits of experts >= K are ignored
    const uint32_t nbytes = n * (uint32_t)ES;  // < 2^30 (checked by the host)
    const __amdgpu_buffer_rsrc_t rb = block_rsrc(chunk_ptr(base, off, ES), nbytes);
    const __amdgpu_buffer_rsrc_t ro = block_rsrc(static_cast<char*>(out) + off * ES, nbytes);
    uint32_t tens = 0;
    uint64_t e0 = 0;
    if (DARE) {
        tens = btensor[g];
        e0 = belem0[g];
    }
    uint32_t bo[CPT];  // byte offset of the lane's chunks in the block
    uint32_t nl = 0;   // realized reads: chunks of the block this wave loads per expert
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        const uint32_t c = tile + q * kTE + t;
        bo[q] = c * 16u;
        if (COUNT)
            nl += (uint32_t)__popcll(__ballot(c < nch));
    }
    uint4 xb[CPT];
#pragma unroll
    for (int q = 0; q < CPT; ++q)
        xb[q] = bld16s(rb, bo[q]);
    float x0[E];
    auto unpack_base = [&]() {
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            Fmt<DT>::unpack(xb[q], &x0[q * V]);
    };
    float acc[E], ps[E], ns[E];
    uint32_t cpn[E];  // sign-elect counts: positive in the low, negative in the high half
#pragma unroll
    for (int e = 0; e < E; ++e) {
        acc[e] = 0.0f;
        ps[e] = 0.0f;
        ns[e] = 0.0f;
        cpn[e] = 0u;
    }
    // selected-only AVG: the coefficients are alpha_i / s, s = the sum of the
    // selected alpha_i in increasing i (no coefficient when s = 0)
    float s_sel = 0.0f;
    if (MODE == M_AVG_RENORM) {
        uint32_t ms = m;
        __asm__ volatile("" : "+s"(ms) : : "memory");  // constant indices: a few wide scalar loads
#pragma unroll
        for (int q = 0; q < 32; ++q)
            if ((ms >> q) & 1u)
                s_sel = s_sel + alpha.v[q];
    }
    // expert i (the r-th selected) read and folded into the state
    auto expert = [&](int i, int r, bool first) {
        const __amdgpu_buffer_rsrc_t re =
            block_rsrc(src.template expert_block<SMALLK>(i, r, b, off, n, ES), nbytes);
        if (first && !is_avg<MODE>())  // the base arrives before the first expert is read
            __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        uint4 raw[CPT];
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            raw[q] = bld16s(re, bo[q]);
        if (COUNT && t == 0)
            atomicAdd(&ctr[((blockIdx.x & 7u) << 5) | (uint32_t)i], (unsigned long long)nl * 16ull);
        if (first)
            unpack_base();
        // TIES from catalog thresholds: keep |d| >= tau (at least the
        // smallest positive pattern, so a kept delta is not zero)
        float tauf = 0.0f;
        if (MODE == M_TIES_TAU)
            tauf = __uint_as_float(max(tau[(uint64_t)g * (uint32_t)K + (uint32_t)i], 1u));
        float coef = alpha.v[i];
        if (MODE == M_AVG_RENORM)
            coef = (s_sel != 0.0f) ? coef / s_sel : 0.0f;
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            float x[V];
            Fmt<DT>::unpack(raw[q], x);
            bool keep[V];  // DARE: the element survives the drop
            if (DARE) {
                // One Philox4x32-10 draw per eight elements of tensor
                // `tens`: element e takes the 16-bit half (e mod 8) of draw
                // e/8, the low half of a word first, and is dropped iff that
                // half is below drop_T >> 16.  A high half is compared in
                // place (w < drop_T), a low half as the word's low 16 bits.
                const uint64_t e = e0 + (uint64_t)(tile + q * kTE + t) * V;
                const uint64_t qq = e >> 3;
                const uint4 r4 = philox4x32_10(make_uint4((uint32_t)qq, (uint32_t)(qq >> 32), tens, 0u), seed,
                                               (uint32_t)i);
                uint32_t w[V / 2];  // the draw's words for this chunk's elements
                if (V == 8) {
                    w[0] = r4.x; w[1 % (V / 2)] = r4.y; w[2 % (V / 2)] = r4.z; w[3 % (V / 2)] = r4.w;
                } else {  // fp32: a chunk is the first or the second half of a draw
                    const bool second = (e & 4u) != 0u;
                    w[0] = second ? r4.z : r4.x;
                    w[1] = second ? r4.w : r4.y;
                }
                const uint32_t t16 = drop_T >> 16;
#pragma unroll
                for (int v = 0; v < V; ++v)
                    keep[v] = (v & 1) ? !(w[v >> 1] < drop_T) : !((w[v >> 1] & 0xffffu) < t16);
            }
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int e = q * V + v;
                // x - x0 (bsub = 1: exactly the difference), or the stored
                // delta itself (bsub = 0: explicit deltas)
                const float d = fmaf(-bsub, x0[e], x[v]);
                if (is_avg<MODE>()) {
                    acc[e] = fmaf(coef, d, acc[e]);
                } else if (MODE == M_TIES_TAU) {
                    // d >= tau keeps a positive delta, -d >= tau a negative one
                    const bool kp = d >= tauf, kn = -d >= tauf;
                    ps[e] = ps[e] + (kp ? d : 0.0f);
                    ns[e] = ns[e] + (kn ? d : 0.0f);
                    cpn[e] += kp ? 1u : (kn ? 0x10000u : 0u);
                } else {
                    if (MODE == M_DARE_LIN) {
                        acc[e] = fmaf(alpha.v[i], keep[v] ? d * scale : 0.0f, acc[e]);
                    } else {
                        // scale >= 1 is finite, so a kept d * scale has the
                        // sign of d and is zero only when d is
                        const float tv = d * scale;
                        const bool pos = keep[v] && d > 0.0f, neg = keep[v] && d < 0.0f;
                        ps[e] = ps[e] + (pos ? tv : 0.0f);
                        ns[e] = ns[e] + (neg ? tv : 0.0f);
                        cpn[e] += pos ? 1u : (neg ? 0x10000u : 0u);
                    }
                }
            }
        }
    };
    uint32_t mm = m;
    if (mm == 0u) {
        unpack_base();  // no expert selected
    } else {
        expert(__builtin_ctz(mm), 0, true);
        mm &= mm - 1u;
        for (int r = 1; mm != 0u; ++r) {
            expert(__builtin_ctz(mm), r, false);
            mm &= mm - 1u;
        }
    }
    if (SIGN) {
        // elect by comparing the rounded masses P and -N; mean of the
        // agreeing entries
        uint32_t den[E];
        bool odd = false;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const bool up = ps[e] > -ns[e];
            const bool dn = ps[e] < -ns[e];
            acc[e] = up ? ps[e] : (dn ? ns[e] : 0.0f);  // never NaN: a NaN mass elects nothing
            // with no elected sign acc is 0 and any count >= 1 gives 0
            den[e] = up ? (cpn[e] & 0xffffu) : (dn ? (cpn[e] >> 16) : 1u);
            odd |= (den[e] & (den[e] - 1u)) != 0u;
        }
        bool tiny = false;
        if (__any(odd)) {
#pragma unroll
            for (int e = 0; e < E; ++e)
                tiny |= (fabsf(acc[e]) < 0x1p-100f) & (acc[e] != 0.0f);
        }
        if (!__any(odd)) {
            // counts that are powers of two divide by exact scaling, one
            // rounding of the quotient
#pragma unroll
            for (int e = 0; e < E; ++e)
                acc[e] = acc[e] * __uint_as_float((127u - (uint32_t)__builtin_ctz(den[e])) << 23);
        } else if (!__any(tiny)) {
            // The correctly rounded quotient acc / den (1 <= den <= 32)
            // without a division.  Lane j holds h + l, two terms of 1/j:
            // h <= 1/j within an ulp, l = max(fl32((1 - j h) h), 2^-126) > 0
            // (the residual 1 - j h is exact), |h + l - 1/j| < 2^-44 / j.  Then
            // fma(a, h, a l) lies within 2^-43 of a / den (relative).  When
            // a / den is a normal number, every rounding boundary (a midpoint
            // between neighbouring floats, which a / den never equals) lies
            // at least 2^-25 / den >= 2^-30 (relative) away from it, so both
            // round to the same value.  |a| >= 2^-100 keeps a / den and a l
            // clear of the subnormal range (smaller masses divide); l > 0,
            // so an infinite mass gives a l of its own sign and stays
            // infinite.
            const float fj = (float)(t > 0 ? t : 1);
            float h = __builtin_amdgcn_rcpf(fj);
            float r = fmaf(-fj, h, 1.0f);
            if (r < 0.0f) {  // the hardware reciprocal rounded up: one ulp down
                h = __uint_as_float(__float_as_uint(h) - 1u);
                r = fmaf(-fj, h, 1.0f);
            }
            const float l = fmaxf(r * h, 0x1p-126f);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int src = (int)(den[e] << 2);
                const float he = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(h)));
                const float le = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(l)));
                acc[e] = fmaf(acc[e], he, acc[e] * le);
            }
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e)
                acc[e] = acc[e] / (float)den[e];
        }
    }
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        float y[V];
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int e = q * V + v;
            if (is_avg<MODE>())
                y[v] = x0[e] + acc[e];
            else
                y[v] = fmaf(lambda, acc[e], x0[e]);
        }
        bst16s(ro, bo[q], Fmt<DT>::pack(y));  // dropped past the block's end
    }
}

// ------------------------------------------------------------ TIES
// One 256-thread workgroup per block.  The block's deltas (<= 4096
// elements: 16 per thread and expert) stay in registers, and up to four
// selected experts are trimmed together so that they share the barriers.
// Per expert, tau = the k-th largest |d| is found on the fp32 magnitude bit
// patterns (window, bins and fallbacks as in ties_select.h):
//  A  the block maximum M (wave maxima, one value per wave in LDS);
//  B  the elements of the binade of M and of the three binades below it
//     are counted into the window histogram (nothing lies above it);
//  C  one wave per expert walks the histogram from the top to the bin where
//     the count reaches k, needing r more elements from that bin.  If fewer
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
}  // namespace ties

struct TiesSmem {
    uint32_t h[ties::GS][ties::NB];     // window histogram, then candidate list / radix levels
    uint32_t wmax[ties::GS][ties::NW];  // per-wave maximum |d| pattern
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
// largest), by levels on bits 30..20, 19..9 and 8..0.  Returns the pattern
// (at least 1: a zero threshold keeps every nonzero delta).
template <int E>
__device__ inline uint32_t block_radix_select(TiesSmem& sm, int j, const float (&dj)[E], uint32_t k, int t,
                                              int lane, int wave)
{
    uint32_t* h = sm.h[j];
    uint32_t pref = 0u, r = k;
#pragma unroll 1
    for (int lv = 0; lv < 3; ++lv) {
        const int sh = (lv == 0) ? 20 : ((lv == 1) ? 9 : 0);
        const int wd = (lv == 2) ? 9 : 11;
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
            for (int q = 0; q < NB / (4 * NT); ++q)
                *reinterpret_cast<uint4*>(&sm.h[j][4 * (q * NT + t)]) = make_uint4(0u, 0u, 0u, 0u);
        }
    }
#pragma unroll
    for (int j = 0; j < GS; ++j) {
        if (j < ns) {
            float mx = 0.0f;
#pragma unroll
            for (int q = 0; q < CPT; ++q) {
                float x[V];
                Fmt<DT>::unpack(raw[j][q], x);
#pragma unroll
                for (int v = 0; v < V; ++v)
                    d[j][q * V + v] = fmaf(-bsub, x0[q * V + v], x[v]);  // x - x0 or the delta; padding 0
#pragma unroll
                for (int v = 0; v < V; v += 2)  // pairs: one three-way maximum each
                    mx = fmaxf(mx, fmaxf(fabsf(d[j][q * V + v]), fabsf(d[j][q * V + v + 1])));
            }
            const uint32_t w = wave_max_u32(__float_as_uint(mx));
            if (lane == 0)
                sm.wmax[j][wave] = w;
        }
    }
}

// Phases B-D of a trim group whose deltas are in d and whose wave maxima
// were published by ties_deltas: leaves the thresholds in tau (wave-uniform
// patterns) and returns the largest |d| pattern of the group's slots.  Every
// thread of the workgroup calls it.
template <int E>
__device__ inline uint32_t ties_select_group(TiesSmem& sm, uint32_t n, uint32_t k, int ns,
                                             const float (&d)[ties::GS][E], uint32_t (&tau)[ties::GS])
{
    using namespace ties;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    __syncthreads();
    // ---- B: window histograms
    uint32_t bmax[GS];
#pragma unroll
    for (int j = 0; j < GS; ++j) {
        bmax[j] = 0u;
        if (j < ns) {
#pragma unroll
            for (int w = 0; w < NW; ++w)
                bmax[j] = max(bmax[j], uniform_u32(sm.wmax[j][w]));
            if (bmax[j] != 0u) {
                int wb;
                const uint32_t koff = window_koff(bmax[j], lane, &wb);
                const uint32_t flo = window_floor(wb);
                char* row = reinterpret_cast<char*>(sm.h[j]);
                uint32_t inc = 1u;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    window_add<false>(row, __float_as_uint(d[j][e]), flo, koff, inc);
            }
        }
    }
    __syncthreads();
    // ---- C: one wave per expert finds the bin of the k-th largest
    if (wave < ns) {
        const int j = wave;
        uint32_t bm = 0u;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            bm = max(bm, uniform_u32(sm.wmax[j][w]));
        uint32_t state = DONE, v1 = 1u, v2 = 0u;  // v1: tau, or the bucket key to refine
        if (bm != 0u && k < n) {                  // all zero, or k = n: keep every nonzero
            const Cut c = wave_find_from_top<NC>(sm.h[j], NBIN - 1, k, lane);
            const int wb = window_base(bm);
            if (!c.found) {
                state = RADIX;  // tau lies below the window
            } else if (c.aux < c.rank || c.count == c.rank) {
                v1 = max((uint32_t)(wb + (int)c.bin) << KS, 1u);
            } else {
                state = LIST;
                v1 = (uint32_t)(wb + (int)c.bin);
                v2 = c.rank;
            }
        }
        if (lane == 0) {
            sm.st[j][0] = state;
            sm.st[j][1] = v1;
            sm.st[j][2] = v2;
            sm.st[j][3] = 0u;
        }
    }
    __syncthreads();
    // ---- D (rare): resolve inside the bucket, or select exactly
    uint32_t anyst = 0u;
#pragma unroll
    for (int j = 0; j < GS; ++j)
        if (j < ns)
            anyst |= uniform_u32(sm.st[j][0]);
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
                                       float bsub, unsigned long long* ctr)
{
    uint4 raw[ties::GS][CPT];
    ties_load_group<DT, CPT>(src, b, off, n, gm, rank0, raw, ctr);
    const int ns = __popc(gm);
    ties_deltas<DT, CPT>(sm, raw, ns, x0, d, bsub);
    return ties_select_group<CPT * Fmt<DT>::V>(sm, n, k, ns, d, tau);
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
                                                         unsigned long long* __restrict__ ctr, float bsub)
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
            top = ties_select_group<E>(sm, n, k, ns, d, tau);
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
            ties_trim_group<DT, CPT>(sm, src, b, off, n, k, gm, rank0, x0, d, tau, bsub, ctr);
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

// The elementwise kernel with or without the read counters; AVG with the
// expert pointers picked by constant indices when K <= 4.
template <int DT, int MODE, bool COUNT, class Src, class... A>
void launch_elem_k(int K, dim3 grid, hipStream_t s, const Src& src, A... a)
{
    if constexpr (is_avg<MODE>()) {
        if (K <= 4)
            hipLaunchKernelGGL((k_merge_elem<DT, MODE, COUNT, true, Src>), grid, dim3(kTE), kAvgLds, s, src, a...);
        else
            hipLaunchKernelGGL((k_merge_elem<DT, MODE, COUNT, false, Src>), grid, dim3(kTE), kAvgLds, s, src, a...);
    } else {
        hipLaunchKernelGGL((k_merge_elem<DT, MODE, COUNT, false, Src>), grid, dim3(kTE), 0, s, src, a...);
    }
}
template <int DT, int MODE, class Src, class... A>
void launch_elem(bool count, int K, dim3 grid, hipStream_t s, const Src& src, A... a)
{
    if (count)
        launch_elem_k<DT, MODE, true>(K, grid, s, src, a...);
    else
        launch_elem_k<DT, MODE, false>(K, grid, s, src, a...);
}

template <int DT, class Src>
hipError_t launch_typed(const BlockTable& bt, const MergeArgs& a, const Src& src, const void* base,
                        int K, const uint32_t* mask, int64_t nb, void* out, unsigned long long* ctr,
                        hipStream_t s)
{
    const uint32_t kmask = (K >= 32) ? 0xffffffffu : ((1u << K) - 1u);
    if (nb == 0)
        return hipSuccess;
    // workgroups per block for the elementwise kernels: a power of two
    // covering the longest block
    const int64_t per_wg = 8 * (int64_t)kTE;  // elements of one elementwise workgroup (8 per lane)
    uint32_t sub_log2 = 0;
    while ((per_wg << sub_log2) < (int64_t)bt.max_len)
        ++sub_log2;
    const dim3 grid((unsigned)nb), egrid((unsigned)(nb << sub_log2));
    const uint32_t T = (uint32_t)floor(a.p * 65536.0) << 16;  // the 16-bit drop threshold, in the top half
    const float scale = (float)(1.0 / (1.0 - a.p));
    switch (a.op) {
    case Op::AVG:
        launch_elem<DT, M_AVG>(ctr != nullptr, K, egrid, s, src, base, mask, bt.d_off,
                           bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, 0u, 1.0f, 0u, kmask, out, ctr,
                           nullptr, K, a.bsub, sub_log2);
        break;
    case Op::AVG_RENORM:
        launch_elem<DT, M_AVG_RENORM>(ctr != nullptr, K, egrid, s, src, base, mask, bt.d_off,
                           bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, 0u, 1.0f, 0u, kmask, out, ctr,
                           nullptr, K, a.bsub, sub_log2);
        break;
    case Op::DARE_LINEAR:
        launch_elem<DT, M_DARE_LIN>(ctr != nullptr, K, egrid, s, src, base, mask,
                           bt.d_off, bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, T, scale,
                           a.seed, kmask, out, ctr, nullptr, K, a.bsub, sub_log2);
        break;
    case Op::DARE_SIGN:
        launch_elem<DT, M_DARE_SIGN>(ctr != nullptr, K, egrid, s, src, base, mask,
                           bt.d_off, bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, T, scale,
                           a.seed, kmask, out, ctr, nullptr, K, a.bsub, sub_log2);
        break;
    case Op::TIES_TAU:
        launch_elem<DT, M_TIES_TAU>(ctr != nullptr, K, egrid, s, src, base, mask,
                           bt.d_off, bt.d_len, bt.d_tensor, bt.d_elem0, a.alpha, a.lambda, 0u, 1.0f, 0u, kmask,
                           out, ctr, a.tau, K, a.bsub, sub_log2);
        break;
    case Op::TIES: {
        // k for full-length blocks, as the kernel computes it for short ones
        const uint32_t n_full = (uint32_t)bt.block_elems;
        const double kk = ceil(a.density * (double)n_full);
        const uint32_t k_full = (kk >= (double)n_full) ? n_full : (uint32_t)kk;
        if (K <= ties::GS)
            hipLaunchKernelGGL((k_merge_ties<DT, false, Src>), grid, dim3(ties::NT), 0, s, src, base, mask,
                               bt.d_off, bt.d_len, a.density, n_full, k_full, a.lambda, kmask, out, ctr, a.bsub);
        else
            hipLaunchKernelGGL((k_merge_ties<DT, true, Src>), grid, dim3(ties::NT), 0, s, src, base, mask,
                               bt.d_off, bt.d_len, a.density, n_full, k_full, a.lambda, kmask, out, ctr, a.bsub);
        break;
    }
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

hipError_t launch_merge_staged(const BlockTable& bt, const MergeArgs& a, const void* base, int K,
                               const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s,
                               const void* stage, const uint64_t* soff, int64_t b0, int64_t nb)
{
    StagedSrc src{static_cast<const char*>(stage), soff, b0};
    if (bt.dtype == 0)
        return launch_typed<0>(bt, a, src, base, K, mask, nb, out, counters, s);
    return launch_typed<1>(bt, a, src, base, K, mask, nb, out, counters, s);
}

}  // namespace mp
