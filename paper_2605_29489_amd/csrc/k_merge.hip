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
#ifndef MP_TIES_THREADS
#define MP_TIES_THREADS 512
#endif
constexpr int kTiesThreads = MP_TIES_THREADS;  // threads per block of the TIES kernel
#ifndef MP_TIES_GRID
#define MP_TIES_GRID 1024
#endif
constexpr int64_t kTiesGrid = MP_TIES_GRID;  // persistent workgroups of the TIES kernel

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
                                const bool pos = tv > 0.0f, neg = tv < 0.0f;
                                ps[e] = ps[e] + (pos ? tv : 0.0f);
                                ns[e] = ns[e] + (neg ? tv : 0.0f);
                                pc[e] += pos ? 1u : 0u;
                                nc[e] += neg ? 1u : 0u;
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
                    float mean = 0.0f;  // elect the sign of the larger signed mass
                    if (ps[e] > -ns[e])
                        mean = ps[e] / (float)pc[e];
                    else if (ps[e] < -ns[e])
                        mean = ns[e] / (float)nc[e];
                    y[v] = fmaf(lambda, mean, x0[e]);
                }
            }
            po[tile + q * kT + t] = Fmt<DT>::pack(y);
        }
    }
}

// ------------------------------------------------------------ TIES
// Threshold search for one expert block: tau = the k-th largest |d|.
// Magnitudes are compared as fp32 bit patterns (sign cleared).  Levels:
//  window  one atomic per element into a 2048-bin histogram of the key
//          |d| >> 14 (exponent + 9 mantissa bits) over the binade of the
//          block maximum and the three below it; smaller elements (zeros
//          included -- they are frequent in bf16 deltas and would all hit one
//          counter) are not counted.  The high half of each counter counts
//          elements whose 14 low bits are not zero.  If the k-th largest
//          falls in a bucket that is either kept whole or holds only values
//          with zero low bits (so all its values are equal), that bucket
//          gives tau.
//  refine  otherwise the bucket's elements are histogrammed on the next
//          bits (13..3, then 2..0), with the same exactness test; if fewer
//          than k elements lie in the window the search restarts on bits
//          30..20 of all elements.
// The window level is scanned by all waves at once: wave w owns a 256-bin
// slice and publishes its total; after one barrier every wave finds the
// slice holding the k-th largest and resolves the bin by re-reading that
// slice.  Refinement levels (rare) are one atomic pass, a barrier, a scan
// by one wave and a barrier.  Any tau' with max{|d| < tau} < tau' <= tau
// gives the same keep decisions, so a bucket that is kept whole ends the
// search.
struct TiesSmem {
    uint32_t hw[2][2048];  // per round parity: window histogram, then refinement levels
    uint32_t smax[2];      // block maximum |d| pattern per round parity
    uint32_t res[2][4];    // scan result of the current level
    uint32_t slice[2][8];  // per-wave slice totals of the window histogram
};

struct Cut {
    uint32_t found, bin, rank, count, aux;  // wave-uniform (scalar registers)
};

// Wave-level, all lanes: walk histogram bins downward from `top` and find
// the bin where the count from the top first reaches k.  Counts are the low
// 16 bits of each counter; aux returns the bin's high 16 bits.  rank = k
// minus the count above the bin.  Each round reads 256 bins, four
// consecutive bins per lane (conflict-free 16-byte LDS reads), and
// prefix-sums the lane totals across the wave with DPP.
__device__ inline Cut wave_find_from_top(const uint32_t* __restrict__ h, int top, uint32_t k, int lane)
{
    Cut r{0u, 0u, 0u, 0u, 0u};
    top |= 3;
    uint32_t above = 0;
    for (int hi = top; hi >= 0; hi -= 256) {
        const int g4 = hi - 4 * lane - 3;  // multiple of 4: the lane's bins are g4 .. g4+3
        uint4 raw = make_uint4(0u, 0u, 0u, 0u);
        if (g4 >= 0)
            raw = *reinterpret_cast<const uint4*>(h + g4);
        const uint4 v = make_uint4(raw.x & 0xffffu, raw.y & 0xffffu, raw.z & 0xffffu, raw.w & 0xffffu);
        const uint32_t s = v.x + v.y + v.z + v.w;
        const uint32_t incl = wave_incl_sum(s);
        const uint32_t before = above + incl - s;  // count in the bins above this lane's four
        const bool hit = before < k && k <= above + incl;
        const unsigned long long bal = __ballot(hit);
        if (bal) {
            uint32_t c = before, bin, cnt, aux;
            if (c + v.w >= k) {
                bin = g4 + 3; cnt = v.w; aux = raw.w;
            } else {
                c += v.w;
                if (c + v.z >= k) {
                    bin = g4 + 2; cnt = v.z; aux = raw.z;
                } else {
                    c += v.z;
                    if (c + v.y >= k) {
                        bin = g4 + 1; cnt = v.y; aux = raw.y;
                    } else {
                        c += v.y;
                        bin = g4; cnt = v.x; aux = raw.x;
                    }
                }
            }
            const int src = __ffsll((long long)bal) - 1;
            r.found = 1u;
            r.bin = (uint32_t)__builtin_amdgcn_readlane((int)bin, src);
            r.rank = (uint32_t)__builtin_amdgcn_readlane((int)(k - c), src);
            r.count = (uint32_t)__builtin_amdgcn_readlane((int)cnt, src);
            r.aux = (uint32_t)__builtin_amdgcn_readlane((int)(aux >> 16), src);
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

struct BlockInfo {
    uint32_t g, n, m, k;
    uint64_t off;
};

template <class Src>
__device__ inline BlockInfo block_info(const Src& src, int64_t b, const uint32_t* __restrict__ mask,
                                       const uint64_t* __restrict__ boff, const uint32_t* __restrict__ blen,
                                       double density, uint32_t kmask)
{
    BlockInfo bi;
    bi.g = uniform_u32(src.block(b));
    bi.off = boff[bi.g];
    bi.n = blen[bi.g];
    const double kk = ceil(density * (double)bi.n);
    bi.k = uniform_u32((kk >= (double)bi.n) ? bi.n : (uint32_t)kk);
    bi.m = (bi.k != 0u) ? (mask[bi.g] & kmask) : 0u;  // density 0 keeps nothing: no expert is read
    return bi;
}

template <int DT, int NT, int CPT>
__device__ inline void load_chunks(const uint4* __restrict__ p, uint32_t nch, uint4 (&dst)[CPT])
{
    const int t = threadIdx.x;
#pragma unroll
    for (int q = 0; q < CPT; ++q)
        dst[q] = (q * NT + t < nch) ? p[q * NT + t] : make_uint4(0u, 0u, 0u, 0u);
}

// One workgroup merges blocks b, b + gridDim.x, ... (persistent).  While an
// expert block is trimmed the next one -- or the next block's base and
// first selected expert -- is already being loaded.
template <int DT, int NT, class Src>
__global__ __launch_bounds__(NT, NT / 128) void k_merge_ties(Src src, const void* __restrict__ base,
                                                   const uint32_t* __restrict__ mask,
                                                   const uint64_t* __restrict__ boff,
                                                   const uint32_t* __restrict__ blen, double density,
                                                   float lambda, uint32_t kmask, void* __restrict__ out,
                                                   unsigned long long* __restrict__ ctr, int64_t nblocks)
{
    constexpr int V = Fmt<DT>::V;
    constexpr int ES = Fmt<DT>::esize;
    constexpr int CPT = kTiesMaxBlock / NT / V;  // chunks per thread
    constexpr int E = CPT * V;                   // elements per thread
    static_assert(CPT >= 1, "block too small for the thread count");
    __shared__ TiesSmem sm;
    const int t = threadIdx.x;
    const int lane = t & 63;
    int64_t b = blockIdx.x;
    if (b >= nblocks)
        return;

    static_assert(NT == 512, "the window scan gives each of the 8 waves a 256-bin slice");
    for (int q = t; q < 2 * 2048; q += NT)
        (&sm.hw[0][0])[q] = 0u;
    if (t < 2)
        sm.smax[t] = 0u;
    __syncthreads();
    const int wave = t >> 6;
    uint32_t par = 0u;  // parity of the expert round (LDS buffer set)

    BlockInfo cur = block_info(src, b, mask, boff, blen, density, kmask);
    uint4 x0raw[CPT], nx0raw[CPT], nxt[CPT];
    load_chunks<DT, NT, CPT>(chunk_ptr(base, cur.off, ES), cur.n / V, x0raw);
    uint32_t mm = cur.m;
    int rank = 0;
    if (mm)
        load_chunks<DT, NT, CPT>(src.expert(__builtin_ctz(mm), 0, b, cur.off, cur.n, ES), cur.n / V, nxt);

    for (;;) {
        const int64_t b2 = b + gridDim.x;
        const bool has_next = b2 < nblocks;
        BlockInfo nx{};
        if (has_next)
            nx = block_info(src, b2, mask, boff, blen, density, kmask);
        const uint32_t nch = cur.n / V;
        count_expert_bytes(ctr, cur.m, cur.n, ES);
        float x0[E];
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            Fmt<DT>::unpack(x0raw[q], &x0[q * V]);

        float ps[E], ns[E];
        uint32_t pc[E], nc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            ps[e] = 0.0f;
            ns[e] = 0.0f;
            pc[e] = 0u;
            nc[e] = 0u;
        }
        if (mm == 0u && has_next) {  // nothing to trim here: start loading the next block now
            load_chunks<DT, NT, CPT>(chunk_ptr(base, nx.off, ES), nx.n / V, nx0raw);
            if (nx.m)
                load_chunks<DT, NT, CPT>(src.expert(__builtin_ctz(nx.m), 0, b2, nx.off, nx.n, ES), nx.n / V, nxt);
        }
        while (mm) {
            mm &= mm - 1u;
            uint4 ce[CPT];
#pragma unroll
            for (int q = 0; q < CPT; ++q)
                ce[q] = nxt[q];
            if (mm) {
                load_chunks<DT, NT, CPT>(src.expert(__builtin_ctz(mm), rank + 1, b, cur.off, cur.n, ES), nch, nxt);
            } else if (has_next) {
                load_chunks<DT, NT, CPT>(chunk_ptr(base, nx.off, ES), nx.n / V, nx0raw);
                if (nx.m)
                    load_chunks<DT, NT, CPT>(src.expert(__builtin_ctz(nx.m), 0, b2, nx.off, nx.n, ES), nx.n / V,
                                             nxt);
            }
            float d[E];  // padding chunks were loaded as zeros: d = 0 there
            uint32_t mg[E];
#pragma unroll
            for (int q = 0; q < CPT; ++q) {
                float x[V];
                Fmt<DT>::unpack(ce[q], x);
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    const int e = q * V + v;
                    d[e] = x[v] - x0[e];
                    mg[e] = __float_as_uint(d[e]) & 0x7fffffffu;
                }
            }
            uint32_t* h = sm.hw[par];  // clean: cleared during the previous round
            // ---- R1: block maximum
            if (t == 0)
                sm.smax[par ^ 1u] = 0u;  // for the next round
            {
                uint32_t mx = 0u;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    mx = max(mx, mg[e]);
                const uint32_t wmx = wave_max_u32(mx);
                if (lane == 0 && wmx != 0u)
                    atomicMax(&sm.smax[par], wmx);
            }
            __syncthreads();
            // every wave is past the previous round: clear its buffer for the next round
            *reinterpret_cast<uint4*>(&sm.hw[par ^ 1u][4 * t]) = make_uint4(0u, 0u, 0u, 0u);
            const uint32_t bmax = uniform_u32(sm.smax[par]);
            uint32_t tau = 1u;  // all-zero block: nothing is kept
            if (bmax != 0u) {
                // ---- R2: window histogram over [2^(E_max - 3), max] (E_max: binade of the max)
                const uint32_t ebin = bmax >> 23;
                const uint32_t wlo = (ebin > 3u ? ebin - 3u : 0u) << 9;  // first key of the window
                const uint32_t top = (bmax >> 14) - wlo;                  // bin of the max, < 2048
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const uint32_t key = mg[e] >> 14;
                    if (key >= wlo && mg[e] != 0u) {
                        const uint32_t inc = (mg[e] & 0x3fffu) ? 0x10001u : 1u;
                        atomicAdd(&h[key - wlo], inc);
                    }
                }
                __syncthreads();
                // ---- R3 (one wave): scan; then refine while the bucket is not resolved
                // level state: elements with (mg >> pshift) == pref are histogrammed on
                // (mg >> dshift) & dmask; tau so far = pref << pshift
                // ---- all waves: slice totals
                const int g4 = 2047 - 256 * wave - 4 * lane - 3;  // this lane's four bins (slice of this wave)
                const uint4 raw = *reinterpret_cast<const uint4*>(h + g4);
                const uint32_t cnt4 = (raw.x & 0xffffu) + (raw.y & 0xffffu) + (raw.z & 0xffffu) + (raw.w & 0xffffu);
                const uint32_t stot = wave_sum_u32(cnt4);
                if (lane == 0)
                    sm.slice[par][wave] = stot;
                __syncthreads();
                // ---- every wave: the slice holding the k-th largest, then its bin
                uint32_t st = 0u, v1 = 0u, v2 = 0u;  // st 0: done (v1 = tau), 1: refine bucket, 2: restart
                {
                    uint32_t above = 0u;
                    int sl = -1;
#pragma unroll
                    for (int w = 0; w < 8; ++w) {
                        const uint32_t tw = uniform_u32(sm.slice[par][w]);
                        if (sl < 0) {
                            if (above + tw >= cur.k)
                                sl = w;
                            else
                                above += tw;
                        }
                    }
                    if (sl < 0) {
                        st = 2u;  // fewer than k nonzero elements in the window: search everything
                        v2 = cur.k;
                    } else {
                        const Cut c = wave_find_from_top(h, 2047 - 256 * sl, cur.k - above, lane);
                        const uint32_t bin = c.bin;
                        if (c.count == c.rank || c.aux == 0u) {
                            v1 = max((wlo + bin) << 14, 1u);  // the bucket is kept whole / holds one value
                        } else {
                            st = 1u;
                            v1 = wlo + bin;  // bucket key
                            v2 = c.rank;
                        }
                    }
                }
                tau = v1;
                if (st != 0u) {
                    // rare: refinement levels, all in one buffer (the other set is clean for
                    // the next round, this one is cleared at the start of the round after it)
                    uint32_t rk = v2;
                    uint32_t pref = (st == 1u) ? tau : 0u;
                    int pshift = (st == 1u) ? 14 : 31;
                    int dshift = (st == 1u) ? 3 : 20;
#pragma unroll 1
                    for (;;) {
                        __syncthreads();  // everyone has read the previous level's result
                        for (int q = t; q < 2048; q += NT)
                            h[q] = 0u;
                        __syncthreads();
                        const uint32_t lowm = (dshift > 0) ? ((1u << dshift) - 1u) : 0u;
#pragma unroll
                        for (int e = 0; e < E; ++e) {
                            const uint32_t hi = (pshift >= 31) ? 0u : (mg[e] >> pshift);
                            if (hi == pref) {
                                const uint32_t bin = (mg[e] >> dshift) & 2047u;
                                atomicAdd(&h[bin], (mg[e] & lowm) ? 0x10001u : 1u);
                            }
                        }
                        __syncthreads();
                        if (t < 64) {
                            const Cut c = wave_find_from_top(h, 2047, rk, lane);
                            if (lane == 0) {
                                sm.res[par][0] = c.found;
                                sm.res[par][1] = c.bin;
                                sm.res[par][2] = c.rank;
                                sm.res[par][3] = (c.count == c.rank || c.aux == 0u) ? 1u : 0u;
                            }
                        }
                        __syncthreads();
                        const uint32_t found = uniform_u32(sm.res[par][0]);
                        const uint32_t bin = uniform_u32(sm.res[par][1]);
                        rk = uniform_u32(sm.res[par][2]);
                        const uint32_t whole = uniform_u32(sm.res[par][3]);
                        pref = (pshift >= 31 ? 0u : (pref << (pshift - dshift))) | bin;
                        if (!found) {
                            tau = 1u;  // fewer than k nonzero: keep every nonzero
                            break;
                        }
                        if (whole || dshift == 0) {
                            tau = max(pref << dshift, 1u);
                            break;
                        }
                        pshift = dshift;
                        dshift = dshift > 11 ? dshift - 11 : 0;
                    }
                    __syncthreads();  // every wave is done with the buffer
                    for (int q = t; q < 2048; q += NT)
                        h[q] = 0u;
                }
            }
            // ---- keep, and accumulate the signed masses and their counts
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const bool keep = mg[e] >= tau;  // tau >= 1: a kept delta is not zero
                const bool posr = (int32_t)__float_as_uint(d[e]) > 0;
                const bool pos = keep && posr;
                const bool neg = keep && !posr;
                ps[e] = ps[e] + (pos ? d[e] : 0.0f);
                ns[e] = ns[e] + (neg ? d[e] : 0.0f);
                pc[e] += pos ? 1u : 0u;
                nc[e] += neg ? 1u : 0u;
            }
            par ^= 1u;
            ++rank;
        }
        // ---- output of this block
        uint4* po = reinterpret_cast<uint4*>(static_cast<char*>(out) + cur.off * ES);
        // elect the sign of the larger signed mass; mean of the agreeing entries
        float num[E];
        uint32_t den[E];
        bool any_div = false;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const bool up = ps[e] > -ns[e];
            const bool dn = ps[e] < -ns[e];
            num[e] = up ? ps[e] : (dn ? ns[e] : 0.0f);
            den[e] = up ? pc[e] : (dn ? nc[e] : 1u);
            any_div |= den[e] > 1u;
        }
        if (__any(any_div)) {  // one agreeing entry (or none) needs no division
#pragma unroll
            for (int e = 0; e < E; ++e)
                num[e] = num[e] / (float)den[e];
        }
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            if (q * NT + t >= nch)
                continue;
            float y[V];
#pragma unroll
            for (int v = 0; v < V; ++v)
                y[v] = fmaf(lambda, num[q * V + v], x0[q * V + v]);
            po[q * NT + t] = Fmt<DT>::pack(y);
        }
        if (!has_next)
            break;
        b = b2;
        cur = nx;
        mm = cur.m;
        rank = 0;
#pragma unroll
        for (int q = 0; q < CPT; ++q)
            x0raw[q] = nx0raw[q];
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
    case Op::TIES: {
        const int64_t gridT = nb < kTiesGrid ? nb : kTiesGrid;
        hipLaunchKernelGGL((k_merge_ties<DT, kTiesThreads, Src>), dim3((unsigned)gridT), dim3(kTiesThreads), 0, s,
                           src, base, mask, bt.d_off, bt.d_len, a.density, a.lambda, kmask, out, ctr, nb);
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
