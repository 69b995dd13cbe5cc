// Algorithm 1 (PlanGen) on the GPU, bit-exact with a literal sort + greedy.
//
// Every unit u = (g, i) gets the 64-bit key  (~bits(score) << 32) | uid
// with score = float(float(w_i*w_i) * S_u) >= +0, so ascending keys are the
// candidate order of Algorithm 1 (decreasing score, ties by increasing uid)
// and keys are unique.  The literal greedy takes every candidate before the
// first one whose running cost overflows B (the "cut" p), skips p, and then
// keeps scanning; after p only candidates cheaper than c_p can still fit.
//
// So no full sort is needed:
//   round r:  find the cut key of the current candidate set by a
//             cost-weighted MSD radix select (8 digit passes of 8 bits;
//             each pass builds a cost histogram of the candidates that match
//             the resolved key prefix, in LDS, then one wave scans it);
//             select every candidate below the cut; the candidates above the
//             cut that are cheaper than c_p form the next round's set (a
//             compact uid list), with the remaining budget.
//   A round whose candidates all fit selects them all and ends the plan.
// Each round strictly lowers the cost bound, so the number of rounds is at
// most the number of distinct block lengths of the layout.
//
// Round 0 (all units) runs as one launch per digit pass over the whole
// device; the later rounds, whose candidate lists are short, run together
// in one single-workgroup launch.  All control state lives on the device
// (PlanCtl); the host enqueues a fixed kernel sequence and kernels that are
// no longer needed return at once.
#include "device_common.h"
#include "mp_internal.h"

namespace mp {

// Workgroups of the round-0 kernels (at most).  Each workgroup ends a pass
// with device-scope atomic adds into the shared histogram, which serialize
// per address; 512 workgroups measured fastest (2048: the atomics dominate
// the first digit pass; 256: no faster).
constexpr int kPlanGrid = 512;

struct PlanCtl {
    unsigned long long brem[9];       // remaining budget before resolving digit d
    unsigned long long prefix[9];     // key prefix with digits < d resolved
    unsigned long long hist[3][256];  // rotating cost histograms of digit passes
    unsigned long long total0;        // candidate cost of the round (all-fit case)
    unsigned long long sel_cost;
    unsigned long long sel_count;
    unsigned long long digest_acc;
    unsigned long long stats[7];      // budget, cost, full, n_sel, n_units, digest, error
    unsigned int all_fit;
    unsigned int done;
    unsigned int list_n[2];
    unsigned int error;  // set if an internal invariant failed (reported by the host)
    // per-workgroup partial sums of the round-0 kernels (selected cost and
    // count of k_plan_mark, digest terms of k_plan_digest): one plain store
    // per workgroup, summed by the one-workgroup kernel that follows.  Many
    // workgroups adding to one device-scope word serialize at the memory
    // side (the L2 caches are per XCD), which cost tens of microseconds.
    unsigned long long part[3][kPlanGrid];
};

namespace {

constexpr int kT = 256;

// Plan options (the flags of mp_plan).
constexpr uint32_t kPlanPerByte = 1u;   // score per byte of cost
constexpr uint32_t kPlanSkipZero = 2u;  // units with a zero sum of squares are not candidates

// The unit's sort key; c is its cost in bytes.  Per byte: the fp32 score
// divided by c in fp64, rounded once to fp32.
__device__ inline unsigned long long unit_key(float S, float w, uint32_t uid, unsigned long long c, uint32_t flags)
{
    const float w2 = w * w;
    float sc = w2 * S;
    if (flags & kPlanPerByte)
        sc = (float)((double)sc / (double)c);
    return ((unsigned long long)(~__float_as_uint(sc)) << 32) | uid;
}

// Units that are not candidates: a zero statistic under the skip-zero
// option, and (tensor-level plans) tensors without elements, which have no
// block to select.
__device__ inline bool plan_skips(float S, unsigned long long c, uint32_t flags)
{
    return ((flags & kPlanSkipZero) && S == 0.0f) || c == 0ull;
}

// A unit's catalog statistic; the tensor-level plan (no block catalog,
// sumsq null) gives every unit 1, so it takes units by weight, then in uid
// order.
__device__ inline float plan_stat(const float* __restrict__ sumsq, uint32_t uid)
{
    return sumsq != nullptr ? sumsq[uid] : 1.0f;
}

// Wave-level resolution of one digit: h[256] holds the cost of the matching
// candidates per digit value.  Returns the smallest v with
// sum_{v' <= v} h[v'] > brem (v = -1 if the total fits), the cost below v,
// and the total.  Must be called by all 64 lanes of one wave.
__device__ inline void resolve_digit(const unsigned long long* h, unsigned long long brem, int lane,
                                     int* v_out, unsigned long long* below_out,
                                     unsigned long long* total_out)
{
    unsigned long long c[4];
    unsigned long long run = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        run += h[lane * 4 + q];
        c[q] = run;
    }
    unsigned long long incl = run;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const unsigned long long y = __shfl_up(incl, (unsigned)off);
        if (lane >= off)
            incl += y;
    }
    const unsigned long long excl = incl - run;
    const unsigned long long total = __shfl(incl, 63);
    int v = -1;
    unsigned long long below = 0;
    if (excl <= brem && incl > brem) {
        // c[] is non-decreasing and excl + c[3] > brem: q = first slot that overflows
        const unsigned long long room = brem - excl;
        const int q = (c[0] <= room) + (c[1] <= room) + (c[2] <= room);
        v = lane * 4 + q;
        below = excl + (q == 0 ? 0ull : (q == 1 ? c[0] : (q == 2 ? c[1] : c[2])));
    }
    // exactly one lane (or none) found the crossing
    const unsigned long long bal = __ballot(v >= 0);
    if (bal) {
        const int src = __ffsll((long long)bal) - 1;
        v = __shfl(v, src);
        below = __shfl(below, src);
    }
    *v_out = v;
    *below_out = below;
    *total_out = total;
}

struct CandSrc {
    // round 0: implicit (all units, one thread per block handling its K units)
    // later rounds: explicit list of uids
    const uint32_t* list;  // null in round 0
    const unsigned int* list_n;
    unsigned int cap;
};

__global__ __launch_bounds__(kT) void k_plan_init(PlanCtl* ctl, unsigned long long budget)
{
    const int t = threadIdx.x;
    for (int q = t; q < 3 * 256; q += kT)
        (&ctl->hist[0][0])[q] = 0ull;
    if (t == 0) {
        ctl->brem[0] = budget;
        ctl->prefix[0] = 0ull;
        ctl->total0 = 0ull;
        ctl->sel_cost = 0ull;
        ctl->sel_count = 0ull;
        ctl->digest_acc = 0ull;
        ctl->all_fit = 0u;
        ctl->done = 0u;
        ctl->list_n[0] = 0u;
        ctl->list_n[1] = 0u;
        ctl->error = 0u;
    }
}

// Digit pass d of the current round: resolve digit d-1 (every workgroup does
// it redundantly from the previous histogram; workgroup 0 publishes it), then
// histogram digit d of the candidates matching the resolved prefix.
__global__ __launch_bounds__(kT) void k_plan_hist(PlanCtl* ctl, int d, const float* __restrict__ sumsq,
                                                  Coeffs w, uint32_t flags, int K,
                                                  const uint32_t* __restrict__ blen, uint32_t esize, int64_t G,
                                                  CandSrc src)
{
    __shared__ unsigned long long lh[256];
    __shared__ unsigned long long s_prefix;
    __shared__ int s_stop;
    if (ctl->done || ctl->all_fit)
        return;
    const int t = threadIdx.x;
    const int lane = t & 63;
    if (t < 64) {
        unsigned long long prefix = 0ull, brem = ctl->brem[0];
        int stop = 0;
        if (d > 0) {
            int v;
            unsigned long long below, total;
            resolve_digit(ctl->hist[(d - 1) % 3], ctl->brem[d - 1], lane, &v, &below, &total);
            if (v < 0) {  // digit 0: every candidate fits; later digits: cannot happen
                stop = 1;
                if (blockIdx.x == 0 && lane == 0) {
                    if (d == 1) {
                        ctl->total0 = total;
                        ctl->all_fit = 1u;
                    } else {
                        ctl->error = 3u;
                    }
                }
            } else {
                prefix = ctl->prefix[d - 1] | ((unsigned long long)v << (56 - 8 * (d - 1)));
                brem = ctl->brem[d - 1] - below;
                if (blockIdx.x == 0 && lane == 0) {
                    ctl->prefix[d] = prefix;
                    ctl->brem[d] = brem;
                }
            }
        }
        if (lane == 0) {
            s_prefix = prefix;
            s_stop = stop;
        }
    }
    if (blockIdx.x == 0) {
        unsigned long long* hn = ctl->hist[(d + 1) % 3];
        for (int q = t; q < 256; q += kT)
            hn[q] = 0ull;
    }
    lh[t] = 0ull;
    __syncthreads();
    if (s_stop)
        return;
    const unsigned long long prefix = s_prefix;
    const int hi_shift = 64 - 8 * d;  // bits above the digit (d > 0)
    const int dg_shift = 56 - 8 * d;
    if (src.list == nullptr) {
        for (int64_t g = (int64_t)blockIdx.x * kT + t; g < G; g += (int64_t)gridDim.x * kT) {
            const unsigned long long c = (unsigned long long)blen[g] * esize;
            for (int i = 0; i < K; ++i) {
                const uint32_t uid = (uint32_t)(g * K + i);
                const float S = plan_stat(sumsq, uid);
                if (plan_skips(S, c, flags))
                    continue;
                const unsigned long long key = unit_key(S, w.v[i], uid, c, flags);
                if (d == 0 || ((key ^ prefix) >> hi_shift) == 0)
                    atomicAdd(&lh[(key >> dg_shift) & 255u], c);
            }
        }
    } else {
        // listed units are candidates already
        const unsigned int n = min(*src.list_n, src.cap);
        for (unsigned int q = blockIdx.x * kT + t; q < n; q += gridDim.x * kT) {
            const uint32_t uid = src.list[q];
            const uint32_t g = uid / (uint32_t)K, i = uid % (uint32_t)K;
            const unsigned long long c = (unsigned long long)blen[g] * esize;
            const unsigned long long key = unit_key(plan_stat(sumsq, uid), w.v[i], uid, c, flags);
            if (d == 0 || ((key ^ prefix) >> hi_shift) == 0)
                atomicAdd(&lh[(key >> dg_shift) & 255u], c);
        }
    }
    __syncthreads();
    if (lh[t])
        atomicAdd(&ctl->hist[d % 3][t], lh[t]);
}

// After digit pass 7: resolve the last digit (the cut key p), select the
// candidates below it, and collect the next round's candidates (above p,
// cheaper than c_p).  In the all-fit case select every candidate.
__global__ __launch_bounds__(kT) void k_plan_mark(PlanCtl* ctl, const float* __restrict__ sumsq, Coeffs w,
                                                  uint32_t flags, int K, const uint32_t* __restrict__ blen,
                                                  uint32_t esize, int64_t G, CandSrc src,
                                                  uint32_t* __restrict__ mask, uint32_t* __restrict__ next,
                                                  unsigned int* __restrict__ next_n, unsigned int next_cap)
{
    __shared__ unsigned long long s_keyp, s_cp;
    __shared__ int s_all;
    __shared__ unsigned long long s_cost[4], s_cnt[4];
    if (ctl->done)
        return;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    if (t < 64) {
        int all = (int)ctl->all_fit;
        unsigned long long keyp = 0ull, cp = 0ull;
        if (!all) {
            int v;
            unsigned long long below, total;
            resolve_digit(ctl->hist[7 % 3], ctl->brem[7], lane, &v, &below, &total);
            keyp = ctl->prefix[7] | (unsigned long long)(unsigned)(v < 0 ? 0 : v);
            const uint32_t gp = (uint32_t)keyp / (uint32_t)K;
            if (v < 0 || (int64_t)gp >= G) {  // cannot happen: the cut is a real unit
                if (lane == 0)
                    ctl->error = 1u;
                keyp = 0ull;  // select nothing more this round
                cp = 0ull;
            } else {
                cp = (unsigned long long)blen[gp] * esize;
            }
            if (blockIdx.x == 0 && lane == 0) {
                ctl->prefix[8] = keyp;
                ctl->brem[8] = ctl->brem[7] - below;
            }
        }
        if (lane == 0) {
            s_keyp = keyp;
            s_cp = cp;
            s_all = all;
        }
    }
    __syncthreads();
    const unsigned long long keyp = s_keyp, cp = s_cp;
    const int all = s_all;
    unsigned long long my_cost = 0ull, my_cnt = 0ull;
    if (src.list == nullptr) {
        for (int64_t g = (int64_t)blockIdx.x * kT + t; g < G; g += (int64_t)gridDim.x * kT) {
            const unsigned long long c = (unsigned long long)blen[g] * esize;
            uint32_t word = 0u;
            for (int i = 0; i < K; ++i) {
                const uint32_t uid = (uint32_t)(g * K + i);
                const float S = plan_stat(sumsq, uid);
                if (plan_skips(S, c, flags))
                    continue;
                const unsigned long long key = unit_key(S, w.v[i], uid, c, flags);
                if (all || key < keyp) {
                    word |= 1u << i;
                    my_cost += c;
                    my_cnt += 1;
                } else if (key > keyp && c < cp) {
                    const unsigned int slot = atomicAdd(next_n, 1u);
                    if (slot < next_cap)
                        next[slot] = uid;
                    else
                        ctl->error = 2u;
                }
            }
            mask[g] = word;
        }
    } else {
        const unsigned int n = min(*src.list_n, src.cap);
        for (unsigned int q = blockIdx.x * kT + t; q < n; q += gridDim.x * kT) {
            const uint32_t uid = src.list[q];
            const uint32_t g = uid / (uint32_t)K, i = uid % (uint32_t)K;
            const unsigned long long c = (unsigned long long)blen[g] * esize;
            const unsigned long long key = unit_key(plan_stat(sumsq, uid), w.v[i], uid, c, flags);
            if (all || key < keyp) {
                atomicOr(&mask[g], 1u << i);
                my_cost += c;
                my_cnt += 1;
            } else if (key > keyp && c < cp) {
                const unsigned int slot = atomicAdd(next_n, 1u);
                if (slot < next_cap)
                    next[slot] = uid;
                else
                    ctl->error = 2u;
            }
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        my_cost += __shfl_xor(my_cost, off);
        my_cnt += __shfl_xor(my_cnt, off);
    }
    if (lane == 0) {
        s_cost[wave] = my_cost;
        s_cnt[wave] = my_cnt;
    }
    __syncthreads();
    if (t == 0) {
        ctl->part[0][blockIdx.x] = s_cost[0] + s_cost[1] + s_cost[2] + s_cost[3];
        ctl->part[1][blockIdx.x] = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    }
}

// Sum of part[row][0 .. n) over one 256-thread workgroup (all threads call
// it; every thread gets the sum).  The loads are issued together.
__device__ inline unsigned long long block_sum_parts(const PlanCtl* ctl, int row, int n)
{
    __shared__ unsigned long long s[4];
    const int t = threadIdx.x;
    unsigned long long a = 0ull;
#pragma unroll
    for (int j = 0; j < (kPlanGrid + kT - 1) / kT; ++j) {
        const int q = j * kT + t;
        a += (q < n) ? ctl->part[row][q] : 0ull;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        a += __shfl_xor(a, off);
    __syncthreads();
    if ((t & 63) == 0)
        s[t >> 6] = a;
    __syncthreads();
    return s[0] + s[1] + s[2] + s[3];
}

// Close round r: carry the remaining budget, reset the digit state, and
// finish the plan when everything fit or no cheaper candidate is left.
__global__ __launch_bounds__(kT) void k_plan_advance(PlanCtl* ctl, int next_list, int reuse_list, int n_part)
{
    // takes in the selections of k_plan_mark's n_part workgroups
    const int t = threadIdx.x;
    if (ctl->done)
        return;
    const unsigned long long cs = block_sum_parts(ctl, 0, n_part);
    const unsigned long long cn = block_sum_parts(ctl, 1, n_part);
    for (int q = t; q < 3 * 256; q += kT)
        (&ctl->hist[0][0])[q] = 0ull;
    if (t != 0)
        return;
    ctl->sel_cost += cs;
    ctl->sel_count += cn;
    unsigned long long rem;
    if (ctl->all_fit) {
        rem = ctl->brem[0] - ctl->total0;
        ctl->done = 1u;
    } else {
        rem = ctl->brem[8];
        if (ctl->list_n[next_list] == 0u)
            ctl->done = 1u;
    }
    ctl->brem[0] = rem;
    ctl->prefix[0] = 0ull;
    ctl->all_fit = 0u;
    ctl->list_n[reuse_list] = 0u;
}

// Rounds r_begin .. r_end-1 (the later rounds, whose candidates are the
// short lists left by the round before) in one workgroup: the same digit
// passes, cut and selection as k_plan_hist / k_plan_mark / k_plan_advance,
// with the round state in LDS and barriers instead of launches.
__device__ inline uint32_t plan_list_load(const uint32_t* p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kT) void k_plan_rest(PlanCtl* ctl, const float* __restrict__ sumsq, Coeffs w,
                                                  uint32_t flags, int K,
                                                  const uint32_t* __restrict__ blen, uint32_t esize, int64_t G,
                                                  uint32_t* list0, uint32_t* list1, unsigned int cap,
                                                  uint32_t* __restrict__ mask, int r_begin, int r_end)
{
    __shared__ unsigned long long lh[256];
    __shared__ unsigned long long s_brem0, s_below, s_total;
    __shared__ unsigned long long s_cost[4], s_cnt[4];
    __shared__ unsigned int s_n, s_next_n, s_err;
    __shared__ int s_v, s_done;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (t == 0) {
        s_done = (int)ctl->done;
        s_brem0 = ctl->brem[0];
        s_n = ctl->list_n[r_begin & 1];
        s_err = 0u;
    }
    unsigned long long sel_cost = 0ull, sel_cnt = 0ull;  // this thread's selections
    for (int r = r_begin; r < r_end; ++r) {
        __syncthreads();
        if (s_done)
            break;
        const uint32_t* list = (r & 1) ? list1 : list0;
        uint32_t* next = (r & 1) ? list0 : list1;
        const unsigned int n = min(s_n, cap);
        const unsigned long long brem0 = s_brem0;
        unsigned long long prefix = 0ull, brem = brem0, total0 = 0ull;
        bool all = false;
        for (int d = 0; d < 8; ++d) {
            lh[t] = 0ull;
            if (t == 0)
                s_next_n = 0u;
            __syncthreads();
            const int hi_shift = 64 - 8 * d, dg_shift = 56 - 8 * d;
            for (unsigned int q = t; q < n; q += kT) {
                const uint32_t uid = plan_list_load(&list[q]);
                const uint32_t g = uid / (uint32_t)K, i = uid % (uint32_t)K;
                const unsigned long long c = (unsigned long long)blen[g] * esize;
                const unsigned long long key = unit_key(plan_stat(sumsq, uid), w.v[i], uid, c, flags);
                if (d == 0 || ((key ^ prefix) >> hi_shift) == 0)
                    atomicAdd(&lh[(key >> dg_shift) & 255u], c);
            }
            __syncthreads();
            if (wave == 0) {
                int v;
                unsigned long long below, total;
                resolve_digit(lh, brem, lane, &v, &below, &total);
                if (lane == 0) {
                    s_v = v;
                    s_below = below;
                    s_total = total;
                }
            }
            __syncthreads();
            const int v = s_v;
            if (v < 0) {  // digit 0: every candidate fits; later digits: cannot happen
                if (d == 0) {
                    all = true;
                    total0 = s_total;
                } else if (t == 0) {
                    s_err = 3u;
                }
                break;
            }
            prefix |= (unsigned long long)v << (56 - 8 * d);
            brem -= s_below;
        }
        // the cut key p = prefix; select below it, keep the cheaper ones above
        unsigned long long cp = 0ull;
        bool cut_ok = true;
        if (!all) {
            const uint32_t gp = (uint32_t)prefix / (uint32_t)K;
            if ((int64_t)gp >= G) {  // cannot happen: the cut is a real unit
                cut_ok = false;
                if (t == 0)
                    s_err = 1u;
            } else {
                cp = (unsigned long long)blen[gp] * esize;
            }
        }
        if (all || cut_ok) {
            for (unsigned int q = t; q < n; q += kT) {
                const uint32_t uid = plan_list_load(&list[q]);
                const uint32_t g = uid / (uint32_t)K, i = uid % (uint32_t)K;
                const unsigned long long c = (unsigned long long)blen[g] * esize;
                const unsigned long long key = unit_key(plan_stat(sumsq, uid), w.v[i], uid, c, flags);
                if (all || key < prefix) {
                    atomicOr(&mask[g], 1u << i);
                    sel_cost += c;
                    sel_cnt += 1;
                } else if (key > prefix && c < cp) {
                    const unsigned int slot = atomicAdd(&s_next_n, 1u);
                    if (slot < cap)
                        next[slot] = uid;
                    else
                        s_err = 2u;
                }
            }
        }
        __threadfence();  // the next list is in memory before the next round reads it
        __syncthreads();
        if (t == 0) {
            s_brem0 = all ? brem0 - total0 : brem;
            s_done = (all || !cut_ok || s_next_n == 0u) ? 1 : 0;
            s_n = s_next_n;
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        sel_cost += __shfl_xor(sel_cost, off);
        sel_cnt += __shfl_xor(sel_cnt, off);
    }
    __syncthreads();
    if (lane == 0) {
        s_cost[wave] = sel_cost;
        s_cnt[wave] = sel_cnt;
    }
    __syncthreads();
    if (t == 0) {
        const unsigned long long cs = s_cost[0] + s_cost[1] + s_cost[2] + s_cost[3];
        const unsigned long long cn = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
        if (cn) {
            atomicAdd(&ctl->sel_cost, cs);
            atomicAdd(&ctl->sel_count, cn);
        }
        if (s_err)
            ctl->error = s_err;
        ctl->done = 1u;
    }
}

__global__ __launch_bounds__(kT) void k_plan_digest(PlanCtl* ctl, const uint32_t* __restrict__ mask, int64_t G)
{
    __shared__ unsigned long long s[4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    unsigned long long acc = 0ull;
    for (int64_t g = (int64_t)blockIdx.x * kT + t; g < G; g += (int64_t)gridDim.x * kT)
        acc += mix64(((unsigned long long)g << 32) | mask[g]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        acc += __shfl_xor(acc, off);
    if (lane == 0)
        s[wave] = acc;
    __syncthreads();
    if (t == 0)
        ctl->part[2][blockIdx.x] = s[0] + s[1] + s[2] + s[3];
}

__global__ __launch_bounds__(kT) void k_plan_final(PlanCtl* ctl, unsigned long long budget, unsigned long long full,
                                                   unsigned long long n_units, int n_part)
{
    // takes in the digest terms of k_plan_digest's n_part workgroups
    const unsigned long long dg = block_sum_parts(ctl, 2, n_part);
    if (threadIdx.x != 0)
        return;
    ctl->digest_acc += dg;
    ctl->stats[0] = budget;
    ctl->stats[1] = ctl->sel_cost;
    ctl->stats[2] = full;
    ctl->stats[3] = ctl->sel_count;
    ctl->stats[4] = n_units;
    ctl->stats[5] = mix64(ctl->digest_acc ^ ctl->sel_cost);
    ctl->stats[6] = ctl->error;
}

}  // namespace

namespace {

// The plan's kernel sequence over G blocks with lengths blen[G] (elements),
// control block ctl and two candidate lists of cap uids each; `rounds`
// bounds the number of rounds (the distinct block lengths, or any larger
// number: the later rounds stop once the plan is done).
// Algorithm 1's selection over G "blocks" with lengths blen[G] (elements):
// control block ctl, two candidate lists of cap uids each; `rounds` bounds
// the number of rounds (the distinct lengths, or any larger number: the
// later rounds stop once the plan is done).  Writes mask[G] and the
// selected cost into ctl; stats come from one of the finals below.
void enqueue_select(PlanCtl* ctl, uint32_t* list0, uint32_t* list1, unsigned cap, const uint32_t* blen,
                    uint32_t es, int64_t G, int rounds, int K, const float* sumsq, const Coeffs& w,
                    uint32_t flags, uint64_t budget, uint32_t* mask, hipStream_t s)
{
    hipLaunchKernelGGL(k_plan_init, dim3(1), dim3(kT), 0, s, ctl, (unsigned long long)budget);
    if (G > 0) {
        const int64_t want = (G + kT - 1) / kT;
        const unsigned grid0 = (unsigned)std::min<int64_t>(want, kPlanGrid);
        // round 0 over every unit; its candidates for round 1 go to list1
        const CandSrc src{nullptr, nullptr, 0u};
        for (int d = 0; d < 8; ++d)
            hipLaunchKernelGGL(k_plan_hist, dim3(grid0), dim3(kT), 0, s, ctl, d, sumsq, w, flags, K, blen, es, G,
                               src);
        hipLaunchKernelGGL(k_plan_mark, dim3(grid0), dim3(kT), 0, s, ctl, sumsq, w, flags, K, blen, es, G, src,
                           mask, list1, &ctl->list_n[1], cap);
        hipLaunchKernelGGL(k_plan_advance, dim3(1), dim3(kT), 0, s, ctl, 1, 0, (int)grid0);
        if (rounds > 1)
            hipLaunchKernelGGL(k_plan_rest, dim3(1), dim3(kT), 0, s, ctl, sumsq, w, flags, K, blen, es, G, list0,
                               list1, cap, mask, 1, rounds);
    }
}

// Stats of a block-level plan: digest over mask[G], the units selected.
hipError_t enqueue_block_final(PlanCtl* ctl, const uint32_t* mask, int64_t G, int K, uint64_t budget,
                               uint64_t full_bytes, hipStream_t s)
{
    const int n_digest = G > 0 ? (int)std::min<int64_t>((G + kT - 1) / kT, kPlanGrid) : 0;
    if (G > 0)
        hipLaunchKernelGGL(k_plan_digest, dim3((unsigned)n_digest), dim3(kT), 0, s, ctl, mask, G);
    hipLaunchKernelGGL(k_plan_final, dim3(1), dim3(kT), 0, s, ctl, (unsigned long long)budget,
                       (unsigned long long)full_bytes, (unsigned long long)(G * K), n_digest);
    return hipGetLastError();
}

// Tensor-level plan: block g takes the selection word of its tensor t, the
// last one with g0[t] <= g (tensors without elements have no blocks); per
// workgroup, the selected block units and the digest terms.
__global__ __launch_bounds__(kT) void k_plan_expand(PlanCtl* ctl, const uint32_t* __restrict__ tmask,
                                                    const uint32_t* __restrict__ g0, int T, int64_t G,
                                                    uint32_t* __restrict__ mask)
{
    __shared__ unsigned long long s_c[4], s_d[4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    unsigned long long cnt = 0ull, dg = 0ull;
    for (int64_t g = (int64_t)blockIdx.x * kT + t; g < G; g += (int64_t)gridDim.x * kT) {
        int lo = 0, hi = T - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int64_t)g0[mid] <= g)
                lo = mid;
            else
                hi = mid - 1;
        }
        const uint32_t m = tmask[lo];
        mask[g] = m;
        cnt += (unsigned long long)__popc(m);
        dg += mix64(((unsigned long long)g << 32) | m);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        cnt += __shfl_xor(cnt, off);
        dg += __shfl_xor(dg, off);
    }
    if (lane == 0) {
        s_c[wave] = cnt;
        s_d[wave] = dg;
    }
    __syncthreads();
    if (t == 0) {
        ctl->part[1][blockIdx.x] = s_c[0] + s_c[1] + s_c[2] + s_c[3];
        ctl->part[2][blockIdx.x] = s_d[0] + s_d[1] + s_d[2] + s_d[3];
    }
}

__global__ __launch_bounds__(kT) void k_plan_final_tensors(PlanCtl* ctl, unsigned long long budget,
                                                           unsigned long long full, unsigned long long n_units,
                                                           int n_part)
{
    const unsigned long long cn = block_sum_parts(ctl, 1, n_part);
    const unsigned long long dg = block_sum_parts(ctl, 2, n_part);
    if (threadIdx.x != 0)
        return;
    ctl->stats[0] = budget;
    ctl->stats[1] = ctl->sel_cost;
    ctl->stats[2] = full;
    ctl->stats[3] = cn;
    ctl->stats[4] = n_units;
    ctl->stats[5] = mix64(dg ^ ctl->sel_cost);
    ctl->stats[6] = ctl->error;
}

// Stats of a tensor-level plan: expand tmask[T] to mask[G], then count and
// digest the block mask.
hipError_t enqueue_tensor_final(PlanCtl* ctl, const uint32_t* tmask, const uint32_t* g0, int T, int64_t G, int K,
                                uint64_t budget, uint64_t full_bytes, uint32_t* mask, hipStream_t s)
{
    const int n_part = G > 0 ? (int)std::min<int64_t>((G + kT - 1) / kT, kPlanGrid) : 0;
    if (G > 0)
        hipLaunchKernelGGL(k_plan_expand, dim3((unsigned)n_part), dim3(kT), 0, s, ctl, tmask, g0, T, G, mask);
    hipLaunchKernelGGL(k_plan_final_tensors, dim3(1), dim3(kT), 0, s, ctl, (unsigned long long)budget,
                       (unsigned long long)full_bytes, (unsigned long long)(G * K), n_part);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_plan(const BlockTable& bt, PlanScratch& ps, int K, const float* sumsq,
                       const Coeffs& w, uint32_t flags, uint64_t budget, uint64_t full_bytes, uint32_t* mask,
                       hipStream_t s)
{
    PlanCtl* ctl = ps.ctl;
    const uint32_t es = (uint32_t)bt.esize;
    hipError_t e;
    if (sumsq != nullptr) {
        enqueue_select(ctl, ps.list[0], ps.list[1], (unsigned)ps.list_cap, bt.d_len, es, bt.G, bt.n_distinct_len, K,
                       sumsq, w, flags, budget, mask, s);
        e = enqueue_block_final(ctl, mask, bt.G, K, budget, full_bytes, s);
    } else {
        // no block catalog: the tensor-level plan, each tensor one unit per expert
        const int64_t T = bt.n_tensors;
        enqueue_select(ctl, ps.list[0], ps.list[1], (unsigned)ps.list_cap, bt.d_tlen, es, T, bt.n_distinct_tlen, K,
                       nullptr, w, flags, budget, ps.tmask, s);
        e = enqueue_tensor_final(ctl, ps.tmask, bt.d_g0, (int)T, bt.G, K, budget, full_bytes, mask, s);
    }
    if (e != hipSuccess)
        return e;
    return hipMemcpyAsync(ps.h_stats, ctl->stats, sizeof(ctl->stats), hipMemcpyDeviceToHost, s);
}

// ---------------------------------------------------------------- plan without allocation
// The plan on a fixed device array instead of the cached workspace and
// block table: for callers that cannot allocate device memory.  The array
// holds, each at a 256-byte boundary: the control block, the layout's
// tensor sizes, the first block of every tensor, the block lengths and the
// two candidate lists.  Every call on a device shares that device's copy,
// and each call rebuilds everything it reads from it.
namespace {

constexpr size_t kStaticPlanBytes = size_t(16) << 20;

static __device__ __align__(256) unsigned char scratch[kStaticPlanBytes];

// The address of `scratch` on each device (0 until the first call there).
constexpr int kMaxDevices = 64;
void* g_scratch_dev[kMaxDevices] = {};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// One workgroup: g0[t] = first block of tensor t (blocks of the tensors
// before it), g0[T] = G; tlen[t] = elements of tensor t (below 2^32, checked
// by the host when the tensor-level plan needs them).
__global__ __launch_bounds__(kT) void k_static_g0(const int64_t* __restrict__ numel, int T, int64_t be,
                                                  uint32_t* __restrict__ g0, uint32_t* __restrict__ tlen)
{
    __shared__ unsigned long long s_w[kT / 64];
    __shared__ unsigned long long s_run;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (t == 0)
        s_run = 0ull;
    for (int base = 0; base < T; base += kT) {
        const int q = base + t;
        const unsigned long long nb = (q < T) ? (unsigned long long)((numel[q] + be - 1) / be) : 0ull;
        unsigned long long incl = nb;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const unsigned long long y = __shfl_up(incl, (unsigned)off);
            if (lane >= off)
                incl += y;
        }
        __syncthreads();  // s_run of the previous chunk is final; s_w is free
        if (lane == 63)
            s_w[wave] = incl;
        __syncthreads();
        unsigned long long before = s_run;
        for (int v = 0; v < wave; ++v)
            before += s_w[v];
        if (q < T) {
            g0[q] = (uint32_t)(before + incl - nb);
            tlen[q] = (uint32_t)numel[q];
        }
        __syncthreads();
        if (t == kT - 1)
            s_run = before + incl;
    }
    __syncthreads();
    if (t == 0)
        g0[T] = (uint32_t)s_run;
}

// blen[g] = elements of block g: the tensor t holding g is the last one
// with g0[t] <= g (tensors without elements have no blocks).
__global__ __launch_bounds__(kT) void k_static_blen(const int64_t* __restrict__ numel, const uint32_t* __restrict__ g0,
                                                    int T, int64_t be, int64_t G, uint32_t* __restrict__ blen)
{
    const int64_t g = (int64_t)blockIdx.x * kT + threadIdx.x;
    if (g >= G)
        return;
    int lo = 0, hi = T - 1;  // g0[lo] <= g holds for lo = 0
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((int64_t)g0[mid] <= g)
            lo = mid;
        else
            hi = mid - 1;
    }
    const int64_t left = numel[lo] - (g - (int64_t)g0[lo]) * be;
    blen[g] = (uint32_t)(left < be ? left : be);
}

}  // namespace

// Sizes of the parts of the fixed array a layout needs; the candidate lists
// hold K units per tensor, which covers both plans (a block-level plan's
// later rounds list only units of short blocks, at most one per tensor).
namespace {
struct StaticParts {
    size_t ctl, numel, g0, tlen, tmask, blen, list;
};
StaticParts static_parts(int64_t n_tensors, int64_t G, int K)
{
    const int64_t cap = (int64_t)K * std::max<int64_t>(n_tensors, 1);
    return {align256(sizeof(PlanCtl)), align256(sizeof(int64_t) * (size_t)n_tensors),
            align256(sizeof(uint32_t) * (size_t)(n_tensors + 1)), align256(sizeof(uint32_t) * (size_t)n_tensors),
            align256(sizeof(uint32_t) * (size_t)n_tensors), align256(sizeof(uint32_t) * (size_t)G),
            align256(sizeof(uint32_t) * (size_t)cap)};
}
}  // namespace

int64_t static_plan_bytes(int64_t n_tensors, int64_t G, int64_t n_short, int K)
{
    const StaticParts a = static_parts(n_tensors, G, K);
    return (int64_t)(a.ctl + a.numel + a.g0 + a.tlen + a.tmask + a.blen + 2 * a.list);
}

int64_t static_plan_limit() { return (int64_t)kStaticPlanBytes; }

hipError_t static_plan_scratch(void** ptr)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    if (g_scratch_dev[dev] == nullptr) {
        void* p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
            return e;
        if (p == nullptr)
            return hipErrorInvalidSymbol;
        g_scratch_dev[dev] = p;
    }
    *ptr = g_scratch_dev[dev];
    return hipSuccess;
}

hipError_t launch_plan_static(void* ws, const int64_t* numel, int32_t n_tensors, int64_t block_elems, uint32_t es,
                              int64_t G, int64_t n_short, int K, const float* sumsq, const Coeffs& w, uint32_t flags,
                              uint64_t budget, uint64_t full_bytes, uint32_t* mask, uint64_t* stats,
                              hipStream_t s)
{
    const StaticParts a = static_parts(n_tensors, G, K);
    const int64_t cap = (int64_t)K * std::max<int64_t>(n_tensors, 1);
    char* p = static_cast<char*>(ws);
    PlanCtl* ctl = reinterpret_cast<PlanCtl*>(p);
    p += a.ctl;
    int64_t* d_numel = reinterpret_cast<int64_t*>(p);
    p += a.numel;
    uint32_t* g0 = reinterpret_cast<uint32_t*>(p);
    p += a.g0;
    uint32_t* tlen = reinterpret_cast<uint32_t*>(p);
    p += a.tlen;
    uint32_t* tmask = reinterpret_cast<uint32_t*>(p);
    p += a.tmask;
    uint32_t* blen = reinterpret_cast<uint32_t*>(p);
    p += a.blen;
    uint32_t* list0 = reinterpret_cast<uint32_t*>(p);
    p += a.list;
    uint32_t* list1 = reinterpret_cast<uint32_t*>(p);
    hipError_t e;
    if (G > 0) {
        if ((e = hipMemcpyAsync(d_numel, numel, sizeof(int64_t) * (size_t)n_tensors, hipMemcpyHostToDevice, s)) !=
            hipSuccess)
            return e;
        hipLaunchKernelGGL(k_static_g0, dim3(1), dim3(kT), 0, s, d_numel, (int)n_tensors, block_elems, g0, tlen);
        if (sumsq != nullptr)
            hipLaunchKernelGGL(k_static_blen, dim3((unsigned)((G + kT - 1) / kT)), dim3(kT), 0, s, d_numel, g0,
                               (int)n_tensors, block_elems, G, blen);
    }
    if (sumsq != nullptr) {
        // n_short + 1 bounds the distinct block lengths, hence the rounds
        enqueue_select(ctl, list0, list1, (unsigned)cap, blen, es, G, (int)std::min<int64_t>(n_short + 1, 1 << 30), K,
                       sumsq, w, flags, budget, mask, s);
        e = enqueue_block_final(ctl, mask, G, K, budget, full_bytes, s);
    } else {
        // tensor-level plan; the number of tensors bounds its rounds
        const int64_t T = G > 0 ? n_tensors : 0;
        enqueue_select(ctl, list0, list1, (unsigned)cap, tlen, es, T, (int)std::max<int64_t>(T, 1), K, nullptr, w,
                       flags, budget, tmask, s);
        e = enqueue_tensor_final(ctl, tmask, g0, (int)n_tensors, G, K, budget, full_bytes, mask, s);
    }
    if (e != hipSuccess)
        return e;
    if ((e = hipMemcpyAsync(stats, ctl->stats, sizeof(ctl->stats), hipMemcpyDeviceToHost, s)) != hipSuccess)
        return e;
    return hipStreamSynchronize(s);
}

hipError_t plan_ctl_alloc(PlanCtl** ctl) { return ws_malloc((void**)ctl, sizeof(PlanCtl)); }

// ---------------------------------------------------------------- coverage
// Touched elements per (tensor, expert) of an access mask, for the run's
// manifest (Section 3: touched blocks and contributing experts):
// cov[t * K + i] = sum of the lengths of tensor t's blocks selecting expert
// i.  One thread per block; a wave whose selecting blocks all lie in one
// tensor (the usual case: blocks run in tensor order) adds one wave sum per
// expert, other waves add per block.
namespace {
__global__ __launch_bounds__(256) void k_zero_cov(unsigned long long* p, int64_t n)
{
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n; q += (int64_t)gridDim.x * 256)
        p[q] = 0ull;
}

__global__ __launch_bounds__(256) void k_coverage(const uint32_t* __restrict__ mask, const uint32_t* __restrict__ len,
                                                  const uint32_t* __restrict__ tensor, int64_t G, int K,
                                                  uint32_t kmask, unsigned long long* __restrict__ cov)
{
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool in = g < G;
    const uint32_t m = in ? (mask[g] & kmask) : 0u;
    const uint32_t t = in ? tensor[g] : 0u;
    const unsigned long long n = in ? len[g] : 0ull;
    const unsigned long long any = __ballot(m != 0u);
    if (any == 0ull)
        return;
    const uint32_t t0 = __shfl(t, __ffsll((long long)any) - 1);
    if (__ballot(m != 0u && t != t0) == 0ull) {
        for (int i = 0; i < K; ++i) {
            unsigned long long v = ((m >> i) & 1u) ? n : 0ull;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1)
                v += __shfl_xor(v, off);
            if ((threadIdx.x & 63) == 0 && v != 0ull)
                atomicAdd(&cov[(uint64_t)t0 * (uint32_t)K + (uint32_t)i], v);
        }
    } else {
        for (uint32_t mm = m; mm; mm &= mm - 1u)
            atomicAdd(&cov[(uint64_t)t * (uint32_t)K + (uint32_t)__builtin_ctz(mm)], n);
    }
}
}  // namespace

hipError_t launch_coverage(const BlockTable& bt, int K, const uint32_t* mask, unsigned long long* cov, hipStream_t s)
{
    const int64_t n = bt.n_tensors * K;
    if (n > 0)
        hipLaunchKernelGGL(k_zero_cov, dim3((unsigned)std::min<int64_t>((n + 255) / 256, 1024)), dim3(256), 0, s,
                           cov, n);
    if (bt.G > 0) {
        const uint32_t kmask = (K >= 32) ? 0xffffffffu : ((1u << K) - 1u);
        hipLaunchKernelGGL(k_coverage, dim3((unsigned)((bt.G + 255) / 256)), dim3(256), 0, s, mask, bt.d_len,
                           bt.d_tensor, bt.G, K, kmask, cov);
    }
    return hipGetLastError();
}

}  // namespace mp
