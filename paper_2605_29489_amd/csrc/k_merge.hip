// Mask-aware elementwise merge operators Psi_op (Eq. 4; operators of
// Appendix A.1): AVG, selected-only AVG, DARE (linear or sign-elect) and
// TIES from stored trim thresholds.  The TIES kernel that selects its
// thresholds inside the merge lives in k_merge_ties.hip.
//
// The block's mask word is uniform, so the loop over the selected experts is
// a scalar loop: unselected experts are never touched (the zero-completed
// tuple of Appendix A.1 costs no reads).  Blocks are streamed as 16-byte
// chunks with coalesced loads.
#include <type_traits>

#include "device_common.h"
#include "merge_src.h"
#include "mp_internal.h"

namespace mp {

namespace {

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
    if (SIGN)
        ties_elect_mean<E>(ps, ns, cpn, acc, t);
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
    case Op::TIES:
        return hipErrorInvalidValue;  // launched by launch_merge_ties
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const BlockTable& bt, const MergeArgs& a, const void* base,
                        const ExpertPtrs& ex, int K, const uint32_t* mask, void* out,
                        unsigned long long* counters, hipStream_t s)
{
    if (a.op == Op::TIES)
        return launch_merge_ties(bt, a, base, ex, K, mask, out, counters, s);
    DevSrc src{ex};
    if (bt.dtype == 0)
        return launch_typed<0>(bt, a, src, base, K, mask, bt.G, out, counters, s);
    return launch_typed<1>(bt, a, src, base, K, mask, bt.G, out, counters, s);
}

hipError_t launch_merge_staged(const BlockTable& bt, const MergeArgs& a, const void* base, int K,
                               const uint32_t* mask, void* out, unsigned long long* counters, hipStream_t s,
                               const void* stage, const uint64_t* soff, int64_t b0, int64_t nb)
{
    if (a.op == Op::TIES)
        return launch_merge_ties_staged(bt, a, base, K, mask, out, counters, s, stage, soff, b0, nb);
    StagedSrc src{static_cast<const char*>(stage), soff, b0};
    if (bt.dtype == 0)
        return launch_typed<0>(bt, a, src, base, K, mask, nb, out, counters, s);
    return launch_typed<1>(bt, a, src, base, K, mask, nb, out, counters, s);
}

}  // namespace mp
