/*
 * oracle.c -- plain CPU oracle for budgeted weight-space merging.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  It shares no
 * code with the GPU library.  Each function follows the paper's definition
 * in the paper's order, plainly; readings of points the paper leaves open
 * are stated where they are used.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fopenmp -shared -fPIC
 * (no fast-math: every rounding below is the IEEE-754 one written).
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ */
/* element access                                                      */
/* ------------------------------------------------------------------ */

/* The dtype argument: bits 0-7 give the element type (0 fp32, 1 bf16);
 * bit 8 (ORC_DELTA) says the expert buffers hold the deltas
 * Delta_i = W_i - W_0 themselves (the executor's "explicit deltas" source,
 * Section 3) instead of fine-tuned weights.  Then d = fl32(Delta_i), read
 * without the base; the base still anchors the merged output. */
#define ORC_DELTA 0x100
static int32_t etype(int32_t dtype) { return dtype & 0xff; }
static int elem_bytes(int32_t dtype)
{
    if (dtype & ~(ORC_DELTA | 0xff))
        return 0;
    dtype = etype(dtype);
    return dtype == 0 ? 4 : (dtype == 1 ? 2 : 0);
}

static float bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* Round-to-nearest-even from fp32 to bfloat16 (inputs are finite). */
static uint16_t f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) /* inf / nan: keep, quiet nan */
        return (uint16_t)((u >> 16) | ((u & 0x007fffffu) ? 0x40u : 0u));
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

static float load(const void* p, int32_t dtype, int64_t j)
{
    if (etype(dtype) == 0)
        return ((const float*)p)[j];
    return bf16_to_f32(((const uint16_t*)p)[j]);
}

static void store(void* p, int32_t dtype, int64_t j, float v)
{
    if (etype(dtype) == 0)
        ((float*)p)[j] = v;
    else
        ((uint16_t*)p)[j] = f32_to_bf16(v);
}

/* Delta of expert buffer ex at element j: fl32(x_i - x_0) for weights (x0
 * is x_0 there), the stored delta itself under ORC_DELTA. */
static float delta_at(const void* ex, int32_t dtype, int64_t j, float x0)
{
    const float x = load(ex, dtype, j);
    return (dtype & ORC_DELTA) ? x : x - x0;
}

/* The same, reading x_0 from the base only where it is needed. */
static float delta_vs_base(const void* ex, const void* base, int32_t dtype, int64_t j)
{
    return (dtype & ORC_DELTA) ? load(ex, dtype, j) : load(ex, dtype, j) - load(base, dtype, j);
}

void orc_round_bf16(const float* x, uint16_t* y, int64_t n)
{
    for (int64_t j = 0; j < n; ++j)
        y[j] = f32_to_bf16(x[j]);
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the parallel loops that follow (n >= 1).  Every per-block
 * computation is sequential, so results do not depend on it. */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------ */
/* Section 2: the tensor set and its deterministic blocks.             */
/* Reading: each tensor is flattened row-major and cut into            */
/* consecutive blocks of block_elems elements; the last block of a     */
/* tensor may be shorter; blocks never cross tensors; blocks are       */
/* numbered in tensor order.  (Prop. 2 relies on the blocks covering    */
/* every parameter exactly once.)                                      */
/* ------------------------------------------------------------------ */

int64_t orc_num_blocks(int32_t n_tensors, const int64_t* numel, int64_t block_elems)
{
    if (n_tensors < 0 || block_elems <= 0)
        return -1;
    int64_t G = 0;
    for (int32_t t = 0; t < n_tensors; ++t) {
        if (numel[t] < 0)
            return -1;
        G += (numel[t] + block_elems - 1) / block_elems;
    }
    return G;
}

int orc_blocks(int32_t n_tensors, const int64_t* numel, int64_t block_elems,
               int64_t* off, int64_t* len, int32_t* tensor, int64_t* elem0)
{
    if (orc_num_blocks(n_tensors, numel, block_elems) < 0)
        return -1;
    int64_t g = 0, start = 0;
    for (int32_t t = 0; t < n_tensors; ++t) {
        for (int64_t e = 0; e < numel[t]; e += block_elems) {
            int64_t n = numel[t] - e;
            if (n > block_elems)
                n = block_elems;
            off[g] = start + e;
            len[g] = n;
            tensor[g] = t;
            elem0[g] = e;
            ++g;
        }
        start += numel[t];
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Catalog statistic (Section 2 and Section 3 "Catalog"): the squared   */
/* L2 norm of each expert delta block, Delta = M_i - M_0.              */
/* Reading of the summation order (the paper leaves it open; a fixed   */
/* order is what makes plans reproducible bit for bit): with V = 16 /   */
/* (bytes per element) elements per 16-byte chunk, 64 partial sums p_l; */
/* partial l takes chunks l, l+64, l+128, ... in turn, elements of a    */
/* chunk in order, p_l = fma(d, d, p_l) from +0; then for              */
/* s = 32,16,8,4,2,1 every p_l becomes p_l + p_(l xor s); the result   */
/* is p_0.  Deltas are fp32: d = float(x_i) - float(x_0).              */
/* ------------------------------------------------------------------ */

static float block_sumsq(const void* base, const void* ex, int32_t dtype, int64_t doff, int64_t n)
{
    const int V = 16 / elem_bytes(dtype);
    float p[64], q[64];
    for (int l = 0; l < 64; ++l)
        p[l] = 0.0f;
    int64_t R = (n + 64 * V - 1) / (64 * V);
    for (int l = 0; l < 64; ++l) {
        for (int64_t r = 0; r < R; ++r) {
            for (int e = 0; e < V; ++e) {
                int64_t j = (r * 64 + l) * V + e;
                if (j >= n)
                    continue;
                float d = delta_vs_base(ex, base, dtype, doff + j);
                p[l] = fmaf(d, d, p[l]);
            }
        }
    }
    for (int s = 32; s >= 1; s >>= 1) {
        for (int l = 0; l < 64; ++l)
            q[l] = p[l] + p[l ^ s];
        for (int l = 0; l < 64; ++l)
            p[l] = q[l];
    }
    return p[0];
}

int orc_index(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
              const void* base, const void* const* experts, int32_t K, float* sumsq)
{
    if (elem_bytes(dtype) == 0 || K < 1 || K > 32 || nb < 0)
        return -1;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t b = 0; b < nb; ++b)
        for (int32_t i = 0; i < K; ++i)
            sumsq[b * K + i] = block_sumsq(base, experts[i], dtype, doff[b], len[b]);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Algorithm 1 (PlanGen).                                              */
/*  candidates: every unit u = (g, i), uid = g*K + i;                  */
/*  score (Eq. 6 with Section 2's retained utility u = |alpha| ||D||):  */
/*      s = float(float(w_i * w_i) * S_u), ranking as |w_i| * ||D||;    */
/*  cost (Appendix A.1: stored byte length of the block):              */
/*      c = len(g) * bytes per element;                                */
/*  sort by decreasing score, ties by increasing uid (earlier          */
/*  tensor/block first, then lower expert);                            */
/*  greedy: take a candidate iff C + c <= B, and keep scanning.         */
/* Options (flags):                                                     */
/*  1 per byte: s = float(double(s) / double(c)), retained utility per */
/*    byte of expert read (Eq. 6's ratio of utility to cost);           */
/*  2 skip zero: a unit with S_u = 0 (its block is unchanged up to      */
/*    squares that underflow) is not a candidate.                       */
/* Digest (the "selected-block digest"; the hash is this reading):     */
/*  D = sum over blocks g of mix64((g << 32) | mask[g]) mod 2^64,       */
/*  digest = mix64(D xor C).                                           */
/* ------------------------------------------------------------------ */

uint64_t orc_mix64(uint64_t x)
{
    /* SplitMix64 output function (Steele, Lea, Flood 2014; Vigna): the  */
    /* value SplitMix64 returns when its state before the step is x.     */
    uint64_t z = x + 0x9e3779b97f4a7c15ull;
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

typedef struct {
    float score;
    uint32_t uid;
} cand_t;

static int cand_cmp(const void* pa, const void* pb)
{
    const cand_t* a = (const cand_t*)pa;
    const cand_t* b = (const cand_t*)pb;
    if (a->score > b->score)
        return -1;
    if (a->score < b->score)
        return 1;
    return (a->uid < b->uid) ? -1 : (a->uid > b->uid ? 1 : 0);
}

int orc_plan(int64_t G, const int64_t* len, int32_t dtype, int32_t K,
             const float* sumsq, const float* w, uint64_t budget, uint32_t flags,
             uint32_t* mask, uint64_t* stats)
{
    int s = elem_bytes(dtype);
    if (s == 0 || K < 1 || K > 32 || G < 0 || (flags & ~3u) != 0 || sumsq == NULL)
        return -1;
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return -1;
    int64_t nu = G * K;
    cand_t* q = (cand_t*)malloc(sizeof(cand_t) * (size_t)(nu > 0 ? nu : 1));
    if (!q)
        return -2;
    uint64_t full = 0;
    int64_t nq = 0; /* candidates */
    for (int64_t u = 0; u < nu; ++u) {
        int32_t i = (int32_t)(u % K);
        uint64_t c = (uint64_t)len[u / K] * (uint64_t)s;
        full += c;
        const float S = sumsq[u];
        if ((flags & 2u) && S == 0.0f)
            continue;
        float w2 = w[i] * w[i];
        float sc = w2 * S;
        if (flags & 1u)
            sc = (float)((double)sc / (double)c);
        q[nq].score = sc;
        q[nq].uid = (uint32_t)u;
        ++nq;
    }
    qsort(q, (size_t)nq, sizeof(cand_t), cand_cmp);

    for (int64_t g = 0; g < G; ++g)
        mask[g] = 0;
    uint64_t C = 0, nsel = 0;
    for (int64_t r = 0; r < nq; ++r) {
        uint32_t u = q[r].uid;
        uint64_t c = (uint64_t)len[u / K] * (uint64_t)s;
        if (C + c <= budget) {
            mask[u / K] |= 1u << (u % K);
            C += c;
            ++nsel;
        }
    }
    free(q);

    uint64_t D = 0;
    for (int64_t g = 0; g < G; ++g)
        D += orc_mix64(((uint64_t)g << 32) | (uint64_t)mask[g]);
    stats[0] = C;
    stats[1] = nsel;
    stats[2] = full;
    stats[3] = orc_mix64(D ^ C);
    stats[4] = (uint64_t)nu;
    return 0;
}

/* ------------------------------------------------------------------ */
/* Planning without block metadata (Section 3, Planner: a deterministic */
/* tensor-level fallback when block metadata are missing; Algorithm 1   */
/* with fallback scores).  Reading: a unit is (expert i, tensor t) with */
/* uid t*K + i; its cost is the tensor's stored bytes, numel_t * s; no   */
/* statistic is known, so every unit's statistic is 1 and its score is  */
/* fl32(w_i * w_i) (per byte: fl32(score / cost) in fp64); tensors       */
/* without elements are not candidates.  Algorithm 1 then runs over     */
/* these units unchanged: decreasing score, ties by uid (tensor, then    */
/* expert), take a unit iff C + c <= B, continue past the ones that do   */
/* not fit.  A selected unit sets expert i's bit in every block of      */
/* tensor t, so a tensor is never split.  Stats and digest are those of */
/* the resulting block mask (n_selected counts block units).  The skip-  */
/* zero option has nothing to skip (no statistic is zero).              */
/* ------------------------------------------------------------------ */
int orc_plan_tensors(int32_t n_tensors, const int64_t* numel, int64_t block_elems, int32_t dtype,
                     int32_t K, const float* w, uint64_t budget, uint32_t flags, uint32_t* mask,
                     uint64_t* stats)
{
    int s = elem_bytes(dtype);
    int64_t G = orc_num_blocks(n_tensors, numel, block_elems);
    if (s == 0 || K < 1 || K > 32 || G < 0 || (flags & ~3u) != 0)
        return -1;
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return -1;
    int64_t nu = (int64_t)n_tensors * K;
    cand_t* q = (cand_t*)malloc(sizeof(cand_t) * (size_t)(nu > 0 ? nu : 1));
    if (!q)
        return -2;
    uint64_t full = 0;
    int64_t nq = 0;
    for (int32_t t = 0; t < n_tensors; ++t) {
        const uint64_t c = (uint64_t)numel[t] * (uint64_t)s;
        full += c * (uint64_t)K;
        if (numel[t] == 0)
            continue;
        for (int32_t i = 0; i < K; ++i) {
            float sc = (w[i] * w[i]) * 1.0f;
            if (flags & 1u)
                sc = (float)((double)sc / (double)c);
            q[nq].score = sc;
            q[nq].uid = (uint32_t)((int64_t)t * K + i);
            ++nq;
        }
    }
    qsort(q, (size_t)nq, sizeof(cand_t), cand_cmp);
    /* per-tensor selection words, then the greedy of Algorithm 1 */
    uint32_t* tsel = (uint32_t*)calloc((size_t)(n_tensors > 0 ? n_tensors : 1), sizeof(uint32_t));
    if (!tsel) {
        free(q);
        return -2;
    }
    uint64_t C = 0;
    for (int64_t r = 0; r < nq; ++r) {
        const uint32_t u = q[r].uid;
        const int32_t t = (int32_t)(u / (uint32_t)K), i = (int32_t)(u % (uint32_t)K);
        const uint64_t c = (uint64_t)numel[t] * (uint64_t)s;
        if (C + c <= budget) {
            tsel[t] |= 1u << i;
            C += c;
        }
    }
    free(q);
    /* every block of tensor t takes the tensor's selection word */
    uint64_t nsel = 0, D = 0;
    int64_t g = 0;
    for (int32_t t = 0; t < n_tensors; ++t) {
        const int64_t nb = (numel[t] + block_elems - 1) / block_elems;
        for (int64_t j = 0; j < nb; ++j, ++g) {
            mask[g] = tsel[t];
            nsel += (uint64_t)__builtin_popcount(tsel[t]);
            D += orc_mix64(((uint64_t)g << 32) | (uint64_t)mask[g]);
        }
    }
    free(tsel);
    stats[0] = C;
    stats[1] = nsel;
    stats[2] = full;
    stats[3] = orc_mix64(D ^ C);
    stats[4] = (uint64_t)(G * K);
    return 0;
}

/* ------------------------------------------------------------------ */
/* AVG (Appendix A.1): Psi = sum_i alpha_i * A_i * Delta_i with fixed   */
/* alpha (no renormalisation over the selected experts); output        */
/* M_A = M_0 + Psi (Eq. 4).  Omitted experts contribute nothing and     */
/* are never read.  Accumulation: acc = +0, then for selected i in     */
/* increasing order acc = fma(alpha_i, d_i, acc); y = x_0 + acc;        */
/* round once to the checkpoint dtype.                                 */
/* ------------------------------------------------------------------ */

static int check_common(int32_t dtype, int32_t K, int64_t nb)
{
    return (elem_bytes(dtype) == 0 || K < 1 || K > 32 || nb < 0) ? -1 : 0;
}

int orc_merge_avg(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                  const void* base, const void* const* experts, int32_t K,
                  const uint32_t* mask, const float* alpha, void* out)
{
    if (check_common(dtype, K, nb))
        return -1;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t b = 0; b < nb; ++b) {
        for (int64_t j = doff[b]; j < doff[b] + len[b]; ++j) {
            float x0 = load(base, dtype, j);
            float acc = 0.0f;
            for (int32_t i = 0; i < K; ++i) {
                if (!((mask[b] >> i) & 1u))
                    continue;
                float d = delta_at(experts[i], dtype, j, x0);
                acc = fmaf(alpha[i], d, acc);
            }
            store(out, dtype, j, x0 + acc);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Selected-only AVG (Appendix A.1, the coefficient-drift variant):    */
/* the merge renormalises the coefficients over the experts selected   */
/* in each block.  For block b, s_b = sum of alpha_i over the selected */
/* i (fp32 adds from +0, increasing i); beta_i = alpha_i / s_b (IEEE   */
/* fp32 division) for a selected i and 0 otherwise; s_b = 0 gives      */
/* beta = 0, so such a block keeps the base.  Then as AVG:             */
/* acc = fma(beta_i, d_i, acc) over the selected i in increasing       */
/* order from +0, out = round(x0 + acc).                               */
/* ------------------------------------------------------------------ */
int orc_merge_avg_renorm(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                         const void* base, const void* const* experts, int32_t K,
                         const uint32_t* mask, const float* alpha, void* out)
{
    if (check_common(dtype, K, nb))
        return -1;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t b = 0; b < nb; ++b) {
        float s = 0.0f;
        for (int32_t i = 0; i < K; ++i)
            if ((mask[b] >> i) & 1u)
                s = s + alpha[i];
        float beta[32];
        for (int32_t i = 0; i < K; ++i)
            beta[i] = (((mask[b] >> i) & 1u) && s != 0.0f) ? alpha[i] / s : 0.0f;
        for (int64_t j = doff[b]; j < doff[b] + len[b]; ++j) {
            float x0 = load(base, dtype, j);
            float acc = 0.0f;
            for (int32_t i = 0; i < K; ++i) {
                if (!((mask[b] >> i) & 1u))
                    continue;
                float d = delta_at(experts[i], dtype, j, x0);
                acc = fmaf(beta[i], d, acc);
            }
            store(out, dtype, j, x0 + acc);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Sign election and disjoint mean (the second and third TIES steps of */
/* Appendix A.1), shared by TIES and DARE's sign-elect                  */
/* combine.  t[r*n + j] holds the (trimmed or dropped) delta of the    */
/* r-th selected expert, experts in increasing index order.            */
/*   P_j = sum of the positive t_rj, N_j = sum of the negative t_rj     */
/*   (each in fp32, adds from +0, increasing r), with their counts;     */
/*   gamma_j = +1 if fl32(P_j) > -fl32(N_j), -1 if fl32(P_j) <          */
/*   -fl32(N_j), 0 if they are equal.  The paper fixes no summation     */
/*   order; this compares the two rounded one-signed masses, which can  */
/*   differ from the sign of the exact sum: (1, -1, 2^-25) gives        */
/*   P = fl32(1 + 2^-25) = 1 = -N, so no sign, in every expert order;   */
/*   mean_j = P_j / count(+) if gamma = +1, N_j / count(-) if -1, else 0 */
/*   (the sum over the agreeing entries divided by their number);      */
/*   out_j = round(fma(lambda, mean_j, x0_j)).                          */
/* ------------------------------------------------------------------ */

static float sign_elect_mean(const float* t, int nsel, int64_t n, int64_t j)
{
    float P = 0.0f, N = 0.0f;
    int np = 0, nn = 0;
    for (int r = 0; r < nsel; ++r) {
        float v = t[(int64_t)r * n + j];
        if (v > 0.0f) {
            P = P + v;
            ++np;
        } else if (v < 0.0f) {
            N = N + v;
            ++nn;
        }
    }
    if (P > -N)
        return P / (float)np;
    if (P < -N)
        return N / (float)nn;
    return 0.0f;
}

/* ------------------------------------------------------------------ */
/* TIES (Appendix A.1: magnitude trim, sign election and the mean of    */
/* the entries agreeing with the elected sign, on the masked deltas).  */
/* Reading: trim is per (selected expert, block) -- Eq. 1 and Eq. 4     */
/* make the operator a function of that block's deltas only.  Keep     */
/* density rho: k = min(n, ceil(rho * n)) computed in fp64; tau = the   */
/* k-th largest |d| of the block (multiplicity counted); keep d_j iff   */
/* |d_j| >= tau and |d_j| > 0 (ties at tau are all kept, k = 0 keeps     */
/* nothing).  Then sign election and disjoint mean as above.           */
/* ------------------------------------------------------------------ */

int64_t orc_ties_k(int64_t n, double density)
{
    double kk = ceil(density * (double)n);
    int64_t k = (int64_t)kk;
    if (k > n)
        k = n;
    if (k < 0)
        k = 0;
    return k;
}

static int desc_float(const void* pa, const void* pb)
{
    float a = *(const float*)pa, b = *(const float*)pb;
    return (a > b) ? -1 : ((a < b) ? 1 : 0);
}

/* The trim threshold of one (expert, block) unit: m[0..n-1] holds |d|; the
 * result is the fp32 bit pattern of the k-th largest of them (multiplicity
 * counted), or all ones when k = 0: a NaN pattern, which no magnitude meets,
 * so nothing is kept (an infinite delta included).  m is sorted in place. */
static uint32_t kth_largest_pattern(float* m, int64_t n, int64_t k)
{
    if (k == 0)
        return 0xffffffffu;
    qsort(m, (size_t)n, sizeof(float), desc_float);
    float tau = m[k - 1];
    uint32_t u;
    memcpy(&u, &tau, sizeof u);
    return u;
}

static float pattern_float(uint32_t u)
{
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

int orc_merge_ties(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                   const void* base, const void* const* experts, int32_t K,
                   const uint32_t* mask, double density, float lambda, void* out)
{
    if (check_common(dtype, K, nb) || !(density >= 0.0 && density <= 1.0))
        return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < nb; ++b) {
        int64_t n = len[b], o = doff[b];
        int nsel = 0;
        for (int32_t i = 0; i < K; ++i)
            nsel += (mask[b] >> i) & 1u;
        float* t = (float*)malloc(sizeof(float) * (size_t)((nsel > 0 ? nsel : 1) * n + 1));
        float* m = (float*)malloc(sizeof(float) * (size_t)(n + 1));
        if (!t || !m) {
            free(t);
            free(m);
#pragma omp atomic write
            bad = 1;
            continue;
        }
        int64_t k = orc_ties_k(n, density);
        int r = 0;
        for (int32_t i = 0; i < K; ++i) {
            if (!((mask[b] >> i) & 1u))
                continue;
            float* ti = t + (int64_t)r * n;
            for (int64_t j = 0; j < n; ++j) {
                ti[j] = delta_vs_base(experts[i], base, dtype, o + j);
                m[j] = fabsf(ti[j]);
            }
            float tau = pattern_float(kth_largest_pattern(m, n, k));
            for (int64_t j = 0; j < n; ++j) {
                float a = fabsf(ti[j]);
                if (!(a >= tau && a > 0.0f))
                    ti[j] = 0.0f;
            }
            ++r;
        }
        for (int64_t j = 0; j < n; ++j) {
            float x0 = load(base, dtype, o + j);
            float mean = sign_elect_mean(t, nsel, n, j);
            store(out, dtype, o + j, fmaf(lambda, mean, x0));
        }
        free(t);
        free(m);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------------------ */
/* The TIES trim threshold depends only on the (expert, block) unit and */
/* the density, never on the access mask (Appendix A.1's trim is read  */
/* per unit, see above).  It can therefore be computed once per unit   */
/* and reused by merges at any budget.  tau[b*K + i] = the threshold   */
/* pattern of unit (block b, expert i) as kth_largest_pattern defines  */
/* it.                                                                 */
/* ------------------------------------------------------------------ */

int orc_ties_thresholds(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                        const void* base, const void* const* experts, int32_t K, double density,
                        uint32_t* tau)
{
    if (check_common(dtype, K, nb) || !(density >= 0.0 && density <= 1.0))
        return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < nb; ++b) {
        int64_t n = len[b], o = doff[b];
        float* m = (float*)malloc(sizeof(float) * (size_t)(n + 1));
        if (!m) {
#pragma omp atomic write
            bad = 1;
            continue;
        }
        int64_t k = orc_ties_k(n, density);
        for (int32_t i = 0; i < K; ++i) {
            for (int64_t j = 0; j < n; ++j)
                m[j] = fabsf(delta_vs_base(experts[i], base, dtype, o + j));
            tau[b * K + i] = kth_largest_pattern(m, n, k);
        }
        free(m);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------------------ */
/* TIES with a per-tensor trim scope (the original TIES granularity     */
/* applied per tensor, a variant of Appendix A.1's trim after masking). */
/* For expert i and tensor t the trim runs over the tensor's zero-      */
/* completed masked deltas: unselected blocks count as zeros and are    */
/* never read.  k = orc_ties_k(n_t, density) over the tensor's n_t      */
/* elements; tau = the k-th largest |d| pattern among them.  With m     */
/* selected elements and m < k the k-th largest is a completed zero, so */
/* tau = 0 (every nonzero selected delta is kept); k = 0 gives all ones */
/* (nothing kept).  Output tau_t[t * K + i].  The blocks of a tensor    */
/* are consecutive (the partition's order), tensor[b] their tensor id.  */
/* ------------------------------------------------------------------ */
int orc_ties_tensor_thresholds(int64_t nb, const int64_t* doff, const int64_t* len, const int32_t* tensor,
                               int32_t n_tensors, int32_t dtype, const void* base, const void* const* experts,
                               int32_t K, const uint32_t* mask, double density, uint32_t* tau_t)
{
    if (check_common(dtype, K, nb) || n_tensors < 0 || !(density >= 0.0 && density <= 1.0))
        return -1;
    int64_t* first = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_tensors + 1));
    int64_t* last = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_tensors + 1));
    if (!first || !last) {
        free(first);
        free(last);
        return -2;
    }
    for (int32_t t = 0; t < n_tensors; ++t)
        first[t] = last[t] = -1;
    for (int64_t b = 0; b < nb; ++b) {
        const int32_t t = tensor[b];
        if (t < 0 || t >= n_tensors || (last[t] >= 0 && last[t] != b - 1)) {
            free(first);
            free(last);
            return -1;  /* not the partition's consecutive order */
        }
        if (first[t] < 0)
            first[t] = b;
        last[t] = b;
    }
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t q = 0; q < (int64_t)n_tensors * K; ++q) {
        const int32_t t = (int32_t)(q / K), i = (int32_t)(q % K);
        int64_t n_t = 0, m = 0;
        for (int64_t b = first[t]; b >= 0 && b <= last[t]; ++b) {
            n_t += len[b];
            if ((mask[b] >> i) & 1u)
                m += len[b];
        }
        const int64_t k = orc_ties_k(n_t, density);
        if (k == 0) {
            tau_t[q] = 0xffffffffu;
            continue;
        }
        if (m < k) {
            tau_t[q] = 0u;
            continue;
        }
        float* mag = (float*)malloc(sizeof(float) * (size_t)m);
        if (!mag) {
#pragma omp atomic write
            bad = 1;
            continue;
        }
        int64_t c = 0;
        for (int64_t b = first[t]; b <= last[t]; ++b)
            if ((mask[b] >> i) & 1u)
                for (int64_t j = 0; j < len[b]; ++j)
                    mag[c++] = fabsf(delta_vs_base(experts[i], base, dtype, doff[b] + j));
        tau_t[q] = kth_largest_pattern(mag, m, k);
        free(mag);
    }
    free(first);
    free(last);
    return bad ? -2 : 0;
}

/* TIES with the thresholds given: d is kept iff |d| >= float(tau) and  */
/* |d| > 0, then the election and mean of sign_elect_mean.  With the    */
/* thresholds of orc_ties_thresholds this is orc_merge_ties exactly.    */
int orc_merge_ties_tau(int64_t nb, const int64_t* doff, const int64_t* len, int32_t dtype,
                       const void* base, const void* const* experts, int32_t K,
                       const uint32_t* mask, const uint32_t* tau, float lambda, void* out)
{
    if (check_common(dtype, K, nb))
        return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < nb; ++b) {
        int64_t n = len[b], o = doff[b];
        int nsel = 0;
        for (int32_t i = 0; i < K; ++i)
            nsel += (mask[b] >> i) & 1u;
        float* t = (float*)malloc(sizeof(float) * (size_t)((nsel > 0 ? nsel : 1) * n + 1));
        if (!t) {
#pragma omp atomic write
            bad = 1;
            continue;
        }
        int r = 0;
        for (int32_t i = 0; i < K; ++i) {
            if (!((mask[b] >> i) & 1u))
                continue;
            float th = pattern_float(tau[b * K + i]);
            float* ti = t + (int64_t)r * n;
            for (int64_t j = 0; j < n; ++j) {
                float d = delta_vs_base(experts[i], base, dtype, o + j);
                float a = fabsf(d);
                ti[j] = (a >= th && a > 0.0f) ? d : 0.0f;
            }
            ++r;
        }
        for (int64_t j = 0; j < n; ++j) {
            float x0 = load(base, dtype, o + j);
            store(out, dtype, o + j, fmaf(lambda, sign_elect_mean(t, nsel, n, j), x0));
        }
        free(t);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: */
/* As Easy as 1, 2, 3", SC 2011): ten rounds of                        */
/*   (hi0,lo0) = M0 * c0, (hi1,lo1) = M1 * c2 (32x32 -> 64 products),  */
/*   c = (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0),                      */
/* with the key bumped by the Weyl constants between rounds.           */
/* ------------------------------------------------------------------ */

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        uint64_t p0 = (uint64_t)M0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)M1 * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0;
        c1 = n1;
        c2 = n2;
        c3 = n3;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* ------------------------------------------------------------------ */
/* DARE (Appendix A.1: TIES-like combination after a random drop and   */
/* rescale whose randomness is fixed by a seed or a given mask omega). */
/* Reading: the drop decision for expert i, tensor t, element e of     */
/* that tensor comes from Philox4x32-10 with key (seed, i) and counter  */
/* (low32(e/8), high32(e/8), t, 0).  The four output words hold eight   */
/* 16-bit draws, the low half of a word before its high half: with      */
/* h = e mod 8, u = bits 16*(h mod 2) .. 16*(h mod 2)+15 of word h/2.   */
/* The element is dropped iff u < T with T = floor(p * 2^16) (fp64).    */
/* It depends only on (seed, i, t, e), never on the access mask.  Kept  */
/* deltas are rescaled: t = float(d * s) with s = float(1 / (1 - p))    */
/* (fp64 quotient).  Combine: linear -- acc = fma(alpha_i, t_i, acc)    */
/* over selected i increasing, out = round(fma(lambda, acc, x0)); or    */
/* sign-elect -- the TIES election and disjoint mean without a trim.   */
/* ------------------------------------------------------------------ */

int orc_merge_dare(int64_t nb, const int64_t* doff, const int64_t* len,
                   const int32_t* tensor, const int64_t* elem0, int32_t dtype,
                   const void* base, const void* const* experts, int32_t K,
                   const uint32_t* mask, double p, uint32_t seed, int32_t combine,
                   const float* alpha, float lambda, void* out)
{
    if (check_common(dtype, K, nb) || !(p >= 0.0 && p < 1.0) || (combine != 0 && combine != 1))
        return -1;
    const uint32_t T = (uint32_t)floor(p * 65536.0);
    const float scale = (float)(1.0 / (1.0 - p));
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < nb; ++b) {
        int64_t n = len[b], o = doff[b];
        int nsel = 0;
        for (int32_t i = 0; i < K; ++i)
            nsel += (mask[b] >> i) & 1u;
        float* t = (float*)malloc(sizeof(float) * (size_t)((nsel > 0 ? nsel : 1) * n + 1));
        if (!t) {
#pragma omp atomic write
            bad = 1;
            continue;
        }
        int r = 0;
        for (int32_t i = 0; i < K; ++i) {
            if (!((mask[b] >> i) & 1u))
                continue;
            for (int64_t j = 0; j < n; ++j) {
                uint64_t e = (uint64_t)elem0[b] + (uint64_t)j;
                uint64_t q = e >> 3;
                uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), (uint32_t)tensor[b], 0u};
                uint32_t key[2] = {seed, (uint32_t)i};
                uint32_t word[4];
                orc_philox4x32_10(ctr, key, word);
                uint32_t h = (uint32_t)(e & 7u);
                uint32_t u = (word[h >> 1] >> (16u * (h & 1u))) & 0xFFFFu;
                float d = delta_vs_base(experts[i], base, dtype, o + j);
                t[(int64_t)r * n + j] = (u < T) ? 0.0f : d * scale;
            }
            ++r;
        }
        for (int64_t j = 0; j < n; ++j) {
            float x0 = load(base, dtype, o + j);
            float y;
            if (combine == 0) {
                float acc = 0.0f;
                int rr = 0;
                for (int32_t i = 0; i < K; ++i) {
                    if (!((mask[b] >> i) & 1u))
                        continue;
                    acc = fmaf(alpha[i], t[(int64_t)rr * n + j], acc);
                    ++rr;
                }
                y = fmaf(lambda, acc, x0);
            } else {
                y = fmaf(lambda, sign_elect_mean(t, nsel, n, j), x0);
            }
            store(out, dtype, o + j, y);
        }
        free(t);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------------------ */
/* Low-rank adapters as a delta source                                 */
/* ------------------------------------------------------------------ */

/* Section 3 (Executor): the delta iterator may draw an expert's deltas from
 * LoRA-style adapters (Hu et al., 2022).  Tensor t, viewed as a rows x cols
 * row-major matrix, has the delta scale * B A with A (rank x cols) and B
 * (rows x rank), both row-major in the checkpoint dtype.  Reading (the paper
 * fixes no precision): y = fp32 rounding of the exact sum over k of
 * B[r][k] * A[k][c]; d = fl32(scale * y), stored in the checkpoint dtype.
 * Products of fp32 or bf16 values are exact in fp64 and are summed in fp64
 * in k order, which is the exact sum whenever it fits fp64's 53 bits.
 * out: rows * cols elements in the checkpoint dtype. */
int orc_lora_delta(int32_t dtype, int64_t rows, int64_t cols, int32_t rank, const void* A, const void* B,
                   float scale, void* out)
{
    if (elem_bytes(dtype) == 0 || (dtype & ORC_DELTA) || rows < 0 || cols < 0 || rank < 1)
        return -1;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t c = 0; c < cols; ++c) {
            double s = 0.0;
            for (int32_t k = 0; k < rank; ++k)
                s += (double)load(B, dtype, r * rank + k) * (double)load(A, dtype, (int64_t)k * cols + c);
            const float y = (float)s;
            store(out, dtype, r * cols + c, scale * y);
        }
    }
    return 0;
}
