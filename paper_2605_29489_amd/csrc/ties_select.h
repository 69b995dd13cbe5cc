// Exact selection of the k-th largest delta magnitude of a block, shared by
// the TIES merge kernel (per selected unit) and the catalog kernel that
// stores every unit's threshold (k_index.hip).
//
// Magnitudes are compared as fp32 bit patterns with the sign cleared (the
// same order as the values, since they are not negative).  The window is the
// binade of the block maximum and the three binades below it, keyed by
// |d| >> KS (exponent and MB mantissa bits): NBIN bins, each with NC copies
// so that lanes holding equal values (frequent in bf16 deltas) update
// different words.  No magnitude lies above the window.  The low half of a
// counter counts the bin's elements, the high half the ones above the bin's
// floor (low bits not zero).
#pragma once

#include "device_common.h"

#ifndef MP_TIES_MB
#define MP_TIES_MB 7
#endif
#ifndef MP_TIES_NC
#define MP_TIES_NC 4
#endif
#ifndef MP_TIES_ASM
#define MP_TIES_ASM 1
#endif

namespace mp {

namespace ties {
constexpr int MB = MP_TIES_MB;  // mantissa bits in a window key
constexpr int NC = MP_TIES_NC;  // copies of each window bin (lanes spread over them)
constexpr int KS = 23 - MB;     // pattern bits below a key
constexpr int NBIN = 4 << MB;   // window bins: four binades
constexpr int NB = NBIN * NC;    // words per histogram row
static_assert(NBIN * NC == NB, "a histogram row holds every copy of every bin");
static_assert(NC == 1 || NC == 2 || NC == 4 || NC == 8 || NC == 16, "bins are 16-byte aligned or fill one");
constexpr int LG = (NC == 1) ? 2 : (NC == 2) ? 3 : (NC == 4) ? 4 : (NC == 8) ? 5 : 6;  // log2(4 NC)
enum : uint32_t { DONE = 0u, LIST = 1u, RADIX = 2u };
}  // namespace ties


struct Cut {
    uint32_t found, bin, rank, count, aux;  // wave-uniform
};

// Wave-level, all lanes: walk histogram bins downward from bin `top` and
// find the bin where the count from the top first reaches k.  A bin is NC
// consecutive words; counts are the low 16 bits of the word sums and aux
// returns the bin's high-half sum.  rank = k minus the count above the bin.
// Each round reads 1 KB: 16 consecutive bytes per lane (conflict-free), and
// prefix-sums the lane totals across the wave with DPP.
template <int NC>
__device__ inline Cut wave_find_from_top(const uint32_t* __restrict__ h, int top, uint32_t k, int lane)
{
    if (NC >= 4) {  // one bin per lane per round
        Cut r{0u, 0u, 0u, 0u, 0u};
        uint32_t above = 0;
        for (int hb = top; hb >= 0; hb -= 64) {
            const int bin = hb - lane;
            uint32_t w = 0u;
            if (bin >= 0) {
                const uint4* p = reinterpret_cast<const uint4*>(h + bin * NC);
#pragma unroll
                for (int u = 0; u < NC / 4; ++u) {
                    const uint4 raw = p[u];
                    w += raw.x + raw.y + raw.z + raw.w;
                }
            }
            const uint32_t s = w & 0xffffu;
            const uint32_t incl = wave_incl_sum(s);
            const uint32_t before = above + incl - s;
            const bool hit = before < k && k <= above + incl;
            const unsigned long long bal = __ballot(hit);
            if (bal) {
                const int src = __ffsll((long long)bal) - 1;
                r.found = 1u;
                r.bin = (uint32_t)__builtin_amdgcn_readlane(bin, src);
                r.rank = (uint32_t)__builtin_amdgcn_readlane((int)(k - before), src);
                r.count = (uint32_t)__builtin_amdgcn_readlane((int)s, src);
                r.aux = (uint32_t)__builtin_amdgcn_readlane((int)(w >> 16), src);
                return r;
            }
            above += (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
        }
        return r;
    }
    constexpr int BPL = NC >= 4 ? 1 : 4 / NC;  // bins per lane per round
    Cut r{0u, 0u, 0u, 0u, 0u};
    const int topw = top * NC + NC - 1;  // highest word
    uint32_t above = 0;
    for (int hi = topw | 3; hi >= 0; hi -= 256) {
        const int g4 = hi - 4 * lane - 3;  // multiple of 4: the lane's words are g4 .. g4+3
        uint4 raw = make_uint4(0u, 0u, 0u, 0u);
        if (g4 >= 0)
            raw = *reinterpret_cast<const uint4*>(h + g4);
        uint32_t bw[BPL];  // bin sums, highest bin first
        if (NC == 1) {
            bw[0] = raw.w; bw[BPL > 1 ? 1 : 0] = raw.z; bw[BPL > 2 ? 2 : 0] = raw.y; bw[BPL > 3 ? 3 : 0] = raw.x;
        } else if (NC == 2) {
            bw[0] = raw.z + raw.w; bw[BPL > 1 ? 1 : 0] = raw.x + raw.y;
        } else {
            bw[0] = raw.x + raw.y + raw.z + raw.w;
        }
        uint32_t s = 0u;
#pragma unroll
        for (int q = 0; q < BPL; ++q)
            s += bw[q] & 0xffffu;
        const uint32_t incl = wave_incl_sum(s);
        const uint32_t before = above + incl - s;  // count in the bins above this lane's
        const bool hit = before < k && k <= above + incl;
        const unsigned long long bal = __ballot(hit);
        if (bal) {
            uint32_t c = before, bin = 0u, cnt = 0u, aux = 0u;
            bool got = false;
#pragma unroll
            for (int q = 0; q < BPL; ++q) {
                const uint32_t cq = bw[q] & 0xffffu;
                if (!got && (c + cq >= k || q == BPL - 1)) {
                    got = true;
                    bin = (uint32_t)(g4 / NC + BPL - 1 - q);
                    cnt = cq;
                    aux = bw[q] >> 16;
                } else if (!got) {
                    c += cq;
                }
            }
            const int src = __ffsll((long long)bal) - 1;
            r.found = 1u;
            r.bin = (uint32_t)__builtin_amdgcn_readlane((int)bin, src);
            r.rank = (uint32_t)__builtin_amdgcn_readlane((int)(k - c), src);
            r.count = (uint32_t)__builtin_amdgcn_readlane((int)cnt, src);
            r.aux = (uint32_t)__builtin_amdgcn_readlane((int)aux, src);
            return r;
        }
        above += (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    }
    return r;
}

// Sum over the lanes of a wave (wave-uniform result).
__device__ inline uint32_t wave_sum_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_sum(v), 63);
}


// Wave-level: the r-th largest of the n patterns in `list`, all of which
// share the key (pattern >> KS); the low bits are fixed from the top down.
// Up to 64 patterns sit one per lane in a register, and each bit then
// costs one compare: the count is the popcount of its lane mask.
__device__ inline uint32_t wave_select_list(const uint32_t* __restrict__ list, uint32_t n, uint32_t key,
                                            uint32_t r, int lane)
{
    uint32_t pref = key << ties::KS;
    if (n <= 64u) {
        const uint32_t v = ((uint32_t)lane < n) ? list[lane] : 0u;  // 0 lies below every candidate
        // wave-uniform values, kept in scalar registers
        uint32_t sp = (uint32_t)__builtin_amdgcn_readfirstlane((int)pref);
        const uint32_t sr = (uint32_t)__builtin_amdgcn_readfirstlane((int)r);
#pragma unroll
        for (int bit = ties::KS - 1; bit >= 0; --bit) {
            const uint32_t cand = sp | (1u << bit);
            if ((uint32_t)__popcll(__ballot(v >= cand)) >= sr)
                sp = cand;
        }
        return sp;
    }
#pragma unroll 1
    for (int bit = ties::KS - 1; bit >= 0; --bit) {
        const uint32_t cand = pref | (1u << bit);
        uint32_t c = 0u;
        for (uint32_t i = (uint32_t)lane; i < n; i += 64u)
            c += (list[i] >= cand) ? 1u : 0u;
        if (wave_sum_u32(c) >= r)
            pref = cand;
    }
    return pref;
}


// The LDS operations of one wave take effect in program order; this keeps
// the compiler from reordering them across a hand-off between lanes.
__device__ inline void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Adds one element to the window histogram.  base + koff + (key << LG) is
// the byte address of the lane's copy of the element's bin (koff holds the
// row's offset from base, the lane's copy and -wb bins; see window_koff).
// Nothing lies above the window, so one test against the window's floor
// pattern selects the elements to count.  MAG: bits is a magnitude pattern
// (sign cleared; compared as an integer); otherwise a signed fp32 pattern
// whose magnitude is compared (NaN is never counted).  inc is the counter
// increment: its low half-word must hold 1; its high half-word is set to 1
// when the element lies above its bin's floor (low bits not zero).
template <bool MAG>
__device__ inline void window_add(char* base, uint32_t bits, uint32_t floor_bits, uint32_t koff, uint32_t& inc)
{
    using namespace ties;
    const bool in = MAG ? bits >= floor_bits : fabsf(__uint_as_float(bits)) >= __uint_as_float(floor_bits);
    // the address and increment are formed in every lane (one instruction
    // each either way), so inc flows from element to element unmerged
#if MP_TIES_ASM
    static_assert(KS == 16, "the low bits are the low half-word");
    uint32_t key, boff;
    asm("v_bfe_u32 %0, %1, %2, %3" : "=v"(key) : "v"(bits), "i"(KS), "i"(31 - KS));
    asm("v_lshl_add_u32 %0, %1, %2, %3" : "=v"(boff) : "v"(key), "i"(LG), "v"(koff));
    // high half-word of inc = min(low half-word of bits, 1); low half-word kept
    asm("v_min_u32_sdwa %0, %1, 1 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_0 src1_sel:DWORD"
        : "+v"(inc) : "v"(bits));
#else
    const uint32_t boff = (__builtin_amdgcn_ubfe(bits, KS, 31 - KS) << LG) + koff;
    inc = (min(bits & ((1u << KS) - 1u), 1u) << 16) + 1u;
#endif
    if (in)
        atomicAdd(reinterpret_cast<uint32_t*>(base + boff), inc);
}

// Floor pattern of the window whose bin 0 has key wb (everything at or
// above it lies in the window).
__device__ inline uint32_t window_floor(int wb)
{
    return (uint32_t)(wb > 0 ? wb : 0) << ties::KS;
}

// Key of bin 0 of the window anchored at the block maximum's pattern: the
// top bin holds the last key of the maximum's binade.
__device__ inline int window_base(uint32_t bmax)
{
    using namespace ties;
    return (int)((bmax >> 23) << MB) + (1 << MB) - NBIN;
}

// Byte offset term of window_add for the lane's copy, given the block
// maximum's pattern: key kk goes to ((kk - wb) * NC + (lane % NC)) * 4.
__device__ inline uint32_t window_koff(uint32_t bmax, int lane, int* wb_out)
{
    using namespace ties;
    const int wb = window_base(bmax);
    *wb_out = wb;
    return (uint32_t)(lane & (NC - 1)) * 4u - (uint32_t)wb * (uint32_t)(4 * NC);
}

// |x|'s pattern, formed where it is used: the rare fallbacks below do not
// keep a second copy of the values (the compiler would otherwise share one
// between them).
__device__ inline uint32_t mag_bits(float x)
{
    uint32_t r;
    asm volatile("v_and_b32 %0, 0x7fffffff, %1" : "=v"(r) : "v"(x));
    return r;
}

// max(m, |a|, |b|) in one instruction.  Written out because the compiler,
// unable to tell that these values are canonical, otherwise quiets each one
// with a v_max_f32 of its own before comparing (1.75 instructions per value
// instead of 0.5).
__device__ inline float max3_abs(float m, float a, float b)
{
    float r;
    asm("v_max3_f32 %0, %1, |%2|, |%3|" : "=v"(r) : "v"(m), "v"(a), "v"(b));
    return r;
}

// Wave-level, all lanes: exact k-th largest magnitude pattern (multiplicity
// counted) of the E values each lane holds in d (NaN is not ordered: keep
// it out), 1 <= k <= the number of values that are not padding; padding
// values are zeros, which cannot change the k largest.  The wave-private
// LDS row of NB words starts row_off bytes after base.
//
// guess (wave-uniform) is a magnitude pattern expected at or below the
// answer, 0 for none.  The histogram then first counts only the values at or
// above the floor of guess's bin: the bins from there up are exact, so a cut
// found among them is the answer, and one not found means the answer lies
// lower, when the whole window is counted again.  A good guess leaves most
// values out of the LDS atomics (and their bank conflicts).
template <int E>
__device__ inline uint32_t wave_kth_largest(char* base, int row_off, const float (&d)[E], uint32_t k, int lane,
                                            uint32_t guess = 0u)
{
    using namespace ties;
    uint32_t* __restrict__ h = reinterpret_cast<uint32_t*>(base + row_off);
    float mxf = 0.0f;
#pragma unroll
    for (int e = 0; e < E; e += 2)  // pairs: one three-way maximum each
        mxf = max3_abs(mxf, d[e], d[e + 1]);
    const uint32_t bmax = wave_max_u32(__float_as_uint(mxf));
    if (bmax == 0u)
        return 0u;  // all zero
    int wb;
    const uint32_t koff = window_koff(bmax, lane, &wb) + (uint32_t)row_off;
    const uint32_t wfloor = window_floor(wb);
    uint32_t flo = (guess > wfloor) ? (guess >> KS) << KS : wfloor;
    Cut c;
#pragma unroll 1
    for (;;) {
#pragma unroll
        for (int q = 0; q < NB / 256; ++q)
            *reinterpret_cast<uint4*>(&h[4 * (q * 64 + lane)]) = make_uint4(0u, 0u, 0u, 0u);
        wave_lds_sync();
        uint32_t inc = 1u;
#pragma unroll
        for (int e = 0; e < E; ++e)
            window_add<false>(base, __float_as_uint(d[e]), flo, koff, inc);
        wave_lds_sync();
        c = wave_find_from_top<NC>(h, NBIN - 1, k, lane);
        if (c.found || flo == wfloor)
            break;
        flo = wfloor;  // below the guess: count the whole window
        wave_lds_sync();
    }
    if (c.found) {  // else the k-th largest lies below the window
        if (c.aux < c.rank)
            return (uint32_t)(wb + (int)c.bin) << KS;  // the rank-th largest of the bin is its floor
        // list the bin's values, then fix their low bits one at a time
        const uint32_t key = (uint32_t)(wb + (int)c.bin);
        wave_lds_sync();
        uint32_t n = 0u;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const uint32_t mg = mag_bits(d[e]);
            const bool in = (mg >> KS) == key;
            const unsigned long long bal = __ballot(in);
            // position: n plus the lanes below this one that list a value
            const uint32_t pos =
                __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, n));
            const uint32_t nn = n + (uint32_t)__popcll(bal);  // wave-uniform: one bound test for all lanes
            if (in && nn <= (uint32_t)NB)
                h[pos] = mg;
            n = nn;
        }
        wave_lds_sync();
        if (n <= (uint32_t)NB)
            return wave_select_list(h, n, key, c.rank, lane);
    }
    // exact radix select over all values, from bit 30 down in digits of WD
    // bits (the row holds 2^WD counters): 30..20, 19..9, 8..0 for a row of
    // 2048 words
    constexpr int WD = (NB >= 2048) ? 11 : (NB >= 1024) ? 10 : 9;
    constexpr int NL = (31 + WD - 1) / WD;
    uint32_t pref = 0u, r = k;
#pragma unroll 1
    for (int lv = 0; lv < NL; ++lv) {
        const int top_bit = 31 - lv * WD;  // one past the digit's highest bit
        const int sh = (top_bit - WD > 0) ? top_bit - WD : 0;
        const int wd = top_bit - sh;
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < NB / 256; ++q)
            *reinterpret_cast<uint4*>(&h[4 * (q * 64 + lane)]) = make_uint4(0u, 0u, 0u, 0u);
        wave_lds_sync();
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const uint32_t mg = mag_bits(d[e]);
            const uint32_t hi = (lv == 0) ? 0u : (mg >> (sh + wd));
            if (hi == pref)
                atomicAdd(&h[(mg >> sh) & ((1u << wd) - 1u)], 1u);
        }
        wave_lds_sync();
        const Cut c = wave_find_from_top<1>(h, (1 << wd) - 1, r, lane);
        pref = (pref << wd) | c.bin;
        r = c.rank;
    }
    return pref;
}

}  // namespace mp
