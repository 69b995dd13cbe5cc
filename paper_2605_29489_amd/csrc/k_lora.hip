// Deltas drawn from low-rank adapters (the LoRA source of Section 3's delta
// iterator): for an adapted tensor viewed as a rows x cols row-major matrix,
// d = scale * (B A) with A (rank x cols) and B (rows x rank).  Two uses:
//   * the pull writes them into an explicit-delta checkpoint for the
//     selected units only (k_lora_pull on an operand-order copy of the
//     adapters made by k_lora_prep; the band kernel k_lora_band below when
//     a bf16 tensor's rows are not whole 16-byte chunks);
//   * the fused TIES merge (k_lora_ties, further down) folds them into the
//     merge without writing them.
// All compute the same 16 x 16 MFMA tiles in the same arrangement, so they
// give the same bits.
//
// The band kernel.  The contraction runs on the matrix cores.  One
// 256-thread workgroup takes a band of 64 rows of one tensor for one expert:
// it stages the band's B rows in LDS once, then walks the band's 128-column
// tiles, staging each tile's A columns transposed in LDS (16-byte loads of
// the next tile are in flight while the current one computes and stores).  Wave w owns rows
// w*16 .. w*16+15 and computes the tile transposed, D^T = A^T B^T, in eight
// 16 x 16 MFMA tiles along the columns:
//   MFMA rows    = output columns (operand from A)
//   MFMA columns = output rows    (operand from B)
// so that a lane's four accumulators are four consecutive columns of one
// output row: one 16-byte store each in fp32; in bf16 (columns a multiple of
// 8) the wave passes its rows through LDS so that lanes store 16 contiguous
// bytes and each store instruction writes whole row segments.  The rank is
// zero-padded to the MFMA depth (16 for bf16, 4 for fp32).  Column tiles
// with no selected element are neither loaded nor computed.
//
// A masked band pull computes only the rows that hold a selected element:
// k_lora_rows lists, per tensor and expert, the rows that meet a selected
// block, and the bands then take 64 listed rows each (bands past the list's
// end return at once).  Selected blocks are spread over a tensor's rows, so
// at a low budget most rows are skipped whole.
//
// Blocks of tensors without an adapter get zeros (k_lora_zero).
#include <type_traits>

#include "device_common.h"
#include "mp_internal.h"

namespace mp {

namespace {

constexpr int kTM = 64;   // tile rows (4 waves x 16)
constexpr int kTN = 128;  // tile columns (8 MFMA tiles of 16)
constexpr int kCT = kTN / 16;

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

// The band's descriptor: the last entry with tile0 <= x (wave-uniform search).
__device__ inline int find_desc(const LoraDesc* __restrict__ desc, int n, uint32_t x)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (desc[mid].tile0 <= x)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// A workgroup barrier that orders LDS only: unlike __syncthreads it does not
// wait for the wave's outstanding global loads and stores.
__device__ inline void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The rows of each adapted tensor that meet a selected block of expert i
// (blockIdx.y): workgroup d lists tensor d's in increasing order at
// rl[i * rows_total + r0 ..] and their count at rc[i * n_desc + d].
__global__ __launch_bounds__(256) void k_lora_rows(const LoraDesc* __restrict__ desc, int n_desc,
                                                   const uint32_t* __restrict__ mask, uint32_t block_elems,
                                                   uint32_t* __restrict__ rl, uint32_t* __restrict__ rc,
                                                   uint32_t rows_total)
{
    __shared__ uint32_t wcount[4];
    const int d = blockIdx.x, i = blockIdx.y;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const LoraDesc D = desc[d];
    uint32_t* out = rl + (uint64_t)i * rows_total + D.r0;
    uint32_t total = 0u;
    for (uint32_t r0 = 0; r0 < D.rows; r0 += 256) {
        const uint32_t r = r0 + (uint32_t)t;
        bool need = false;
        if (r < D.rows) {
            const uint32_t b0 = r * D.cols / block_elems;  // < numel < 2^32
            const uint32_t b1 = (r * D.cols + D.cols - 1) / block_elems;
            for (uint32_t b = b0; b <= b1 && !need; ++b)
                need = ((mask[D.g0 + b] >> i) & 1u) != 0u;
        }
        const unsigned long long bal = __ballot(need);
        if (lane == 0)
            wcount[wave] = (uint32_t)__popcll(bal);
        __syncthreads();
        uint32_t before = total;
        for (int w = 0; w < wave; ++w)
            before += wcount[w];
        const uint32_t pos =
            __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, before));
        if (need)
            out[pos] = r;
        total += wcount[0] + wcount[1] + wcount[2] + wcount[3];
        __syncthreads();  // wcount is rewritten by the next chunk
    }
    if (t == 0)
        rc[(uint64_t)i * n_desc + d] = total;
}

template <int DT>
__global__ __launch_bounds__(256, DT == 1 ? 4 : 2) void k_lora_band(const LoraDesc* __restrict__ desc, int n_desc,
                                                   ExpertPtrs ad, OutPtrs dl, const uint32_t* __restrict__ mask,
                                                   uint32_t block_elems, int aligned,
                                                   const uint32_t* __restrict__ rl, const uint32_t* __restrict__ rc,
                                                   uint32_t rows_total)
{
    using E = typename std::conditional<DT == 0, float, uint16_t>::type;
    constexpr int KS = DT == 0 ? 4 : 16;    // MFMA depth
    constexpr int CV = 16 / sizeof(E);      // elements per 16-byte chunk
    constexpr int RS = kMaxLoraRank + 4;    // LDS row stride in elements (breaks bank aliasing, keeps 8 B alignment)
    constexpr int APT = kMaxLoraRank * kTN / CV / 256;  // A chunks per thread at the largest rank
    __shared__ __align__(16) E As[kTN * RS];  // As[n * RS + k] = A[k][n0 + n]
    __shared__ __align__(16) E Bs[kTM * RS];  // Bs[m * RS + k] = B[rix[m]][k]
    constexpr int OS = kTN / 2 + 8;  // bf16 output strip row stride (16-byte aligned rows)
    __shared__ __align__(16) uint16_t Os[DT == 1 ? kTM * OS : 8];  // vector reads and writes
    __shared__ uint32_t flags[2][4];
    __shared__ uint32_t rix[kTM];  // the band's rows (rows: none)
    const int i = blockIdx.y;
    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int d = __builtin_amdgcn_readfirstlane(find_desc(desc, n_desc, blockIdx.x));
    const LoraDesc D = desc[d];
    const uint32_t m0 = (blockIdx.x - D.tile0) * kTM;  // the band's first (listed) row
    const uint32_t rows = D.rows, cols = D.cols, rank = D.rank;
    const uint32_t rp = (rank + KS - 1) / KS * KS;
    // a masked pull walks the listed rows; a full pull every row
    const uint32_t nrow = mask != nullptr ? rc[(uint64_t)i * n_desc + d] : rows;
    if (m0 >= nrow)
        return;  // past the list's end (workgroup-uniform, before any barrier)
    if (t < kTM) {
        // the list holds rows in increasing order, so a full list is the identity
        const uint32_t j = m0 + (uint32_t)t;
        rix[t] = (j >= nrow) ? rows : (nrow != rows ? rl[(uint64_t)i * rows_total + D.r0 + j] : j);
    }
    __syncthreads();
    const uint32_t row = rix[wave * 16 + (lane & 15)];
    const uint32_t cg = 4u * (uint32_t)(lane >> 4);  // the lane's first column inside each 16-column tile
    const E* __restrict__ A = static_cast<const E*>(ad.p[i]) + D.a_off;
    const E* __restrict__ B = static_cast<const E*>(ad.p[i]) + D.b_off;
    E* __restrict__ out = static_cast<E*>(dl.p[i]) + D.toff;
    const bool vec = D.vec != 0u && aligned != 0;  // A's rows are 16-byte aligned: chunked loads
    // the band's B rows, once
    for (uint32_t x = t; x < rp * kTM; x += 256) {
        const uint32_t m = x / rp, k = x % rp;
        const uint32_t rm = rix[m];
        Bs[m * RS + k] = (k < rank && rm < rows) ? B[(uint64_t)rm * rank + k] : E(0);
    }
    // A chunk c of a column tile: depth k = c / (kTN / CV), columns n = (c % (kTN / CV)) * CV ..
    auto load_a = [&](uint32_t n0, uint4 (&ra)[APT]) {
#pragma unroll
        for (int j = 0; j < APT; ++j) {
            const uint32_t c = (uint32_t)(j * 256 + t);
            const uint32_t k = c / (kTN / CV), n = (c % (kTN / CV)) * CV;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (k < rank && n0 + n < cols) {
                const E* src = A + (uint64_t)k * cols + n0 + n;
                if (vec) {
                    v = *reinterpret_cast<const uint4*>(src);
                } else {
                    E tmp[CV];
#pragma unroll
                    for (int q = 0; q < CV; ++q)
                        tmp[q] = (n0 + n + q < cols) ? src[q] : E(0);
                    v = *reinterpret_cast<const uint4*>(tmp);
                }
            }
            ra[j] = v;
        }
    };
    auto store_a = [&](const uint4 (&ra)[APT]) {
#pragma unroll
        for (int j = 0; j < APT; ++j) {
            const uint32_t c = (uint32_t)(j * 256 + t);
            const uint32_t k = c / (kTN / CV), n = (c % (kTN / CV)) * CV;
            if (k < rp) {
                const E* v = reinterpret_cast<const E*>(&ra[j]);
#pragma unroll
                for (int q = 0; q < CV; ++q)
                    As[(n + q) * RS + k] = v[q];
            }
        }
    };
    // The lane's column groups of a tile: c0 + 16 ct (ct < kCT), c0 = n0 + cg.
    // Element row * cols + c0 lies in block lb of the tensor, lr elements in;
    // tiles are selected in order, so (lb, lr) advances by kTN elements per
    // tile instead of being divided out again.  With blocks of at least 116
    // elements the lane's groups (within 116 elements) lie in block lb or
    // lb + 1; shorter blocks take the division per group.
    const bool two = block_elems >= 116u;
    uint32_t lb = 0u, lr = 0u;
    if (row < rows && two) {
        const uint32_t e = row * cols + cg;  // < numel < 2^32
        lb = e / block_elems;
        lr = e - lb * block_elems;
    }
    auto selection = [&](uint32_t n0) {
        uint32_t sel = 0u;
        const uint32_t c0 = n0 + cg;
        if (row < rows && c0 < cols) {
            if (mask == nullptr) {
#pragma unroll
                for (int ct = 0; ct < kCT; ++ct)
                    sel |= (c0 + ct * 16 < cols ? 1u : 0u) << ct;
            } else if (two) {
                // the lane's last group; a second mask word only if it crosses
                const uint32_t span = min((uint32_t)((kCT - 1) * 16), ((cols - 1) & ~3u) - c0);
                const uint32_t w0 = mask[D.g0 + lb];
                const uint32_t w1 = (lr + span >= block_elems) ? mask[D.g0 + lb + 1] : w0;
#pragma unroll
                for (int ct = 0; ct < kCT; ++ct) {
                    const uint32_t w = (lr + ct * 16 >= block_elems) ? w1 : w0;
                    sel |= (c0 + ct * 16 < cols ? ((w >> i) & 1u) : 0u) << ct;
                }
            } else {
#pragma unroll
                for (int ct = 0; ct < kCT; ++ct) {
                    const uint32_t col = c0 + ct * 16;
                    if (col < cols)
                        sel |= ((mask[D.g0 + (row * cols + col) / block_elems] >> i) & 1u) << ct;
                }
            }
        }
        if (two) {  // the next tile's first group
            lr += kTN;
            while (lr >= block_elems) {
                lr -= block_elems;
                ++lb;
            }
        }
        return sel;
    };
    // workgroup "any lane selected" through LDS, one flag word per wave,
    // double-buffered so that a flag is rewritten only two barriers later
    auto any_selected = [&](uint32_t sel, int parity) {
        const bool w = __ballot(sel != 0u) != 0ull;
        if (lane == 0)
            flags[parity][wave] = w ? 1u : 0u;
        lds_barrier();
        return (flags[parity][0] | flags[parity][1] | flags[parity][2] | flags[parity][3]) != 0u;
    };
    const int mr = wave * 16 + (lane & 15);  // the B operand row (an output row)
    const float scale = D.scale;
    uint4 ra[APT];
    uint32_t sel = selection(0);
    load_a(0, ra);
    bool any = any_selected(sel, 0);  // also orders the B staging before its first use
    for (uint32_t tn = 0; tn < D.tiles_n; ++tn) {
        const uint32_t n0 = tn * kTN, n1 = n0 + kTN;
        const bool more = tn + 1 < D.tiles_n;
        if (any) {
            store_a(ra);
            lds_barrier();
        }
        // the next tile's mask words and A chunks are issued before this
        // tile's stores, so waiting for them never waits for the stores
        const uint32_t sel_next = more ? selection(n1) : 0u;
        if (any) {
            float4_t acc[kCT];
#pragma unroll
            for (int ct = 0; ct < kCT; ++ct)
                acc[ct] = float4_t{0.f, 0.f, 0.f, 0.f};
            for (uint32_t k0 = 0; k0 < rp; k0 += KS) {
                if constexpr (DT == 1) {
                    const uint32_t kk = k0 + cg;  // lanes 16j.. hold depth 4j..4j+3
                    const short4_t b = *reinterpret_cast<const short4_t*>(&Bs[mr * RS + kk]);
#pragma unroll
                    for (int ct = 0; ct < kCT; ++ct) {
                        const short4_t a =
                            *reinterpret_cast<const short4_t*>(&As[(ct * 16 + (lane & 15)) * RS + kk]);
                        acc[ct] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc[ct], 0, 0, 0);
                    }
                } else {
                    const uint32_t kk = k0 + (uint32_t)(lane >> 4);  // lanes 16j.. hold depth j
                    const float b = Bs[mr * RS + kk];
#pragma unroll
                    for (int ct = 0; ct < kCT; ++ct) {
                        const float a = As[(ct * 16 + (lane & 15)) * RS + kk];
                        acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[ct], 0, 0, 0);
                    }
                }
            }
            if (more)
                load_a(n1, ra);
            // accumulator j of tile ct is output (row, n0 + ct*16 + cg + j)
            auto direct_store = [&]() {
#pragma unroll
                for (int ct = 0; ct < kCT; ++ct) {
                    if (!((sel >> ct) & 1u))
                        continue;
                    const uint64_t e = (uint64_t)row * cols + n0 + ct * 16 + cg;
                    const float y0 = scale * acc[ct][0], y1 = scale * acc[ct][1];
                    const float y2 = scale * acc[ct][2], y3 = scale * acc[ct][3];
                    if constexpr (DT == 1) {
                        *reinterpret_cast<uint2*>(out + e) =
                            make_uint2(Fmt<1>::pack2(y0, y1), Fmt<1>::pack2(y2, y3));
                    } else {
                        *reinterpret_cast<float4*>(out + e) = make_float4(y0, y1, y2, y3);
                    }
                }
            };
            if constexpr (DT == 1) {
                if ((cols & 7u) == 0u) {
                    // bf16 rows through the wave's own LDS strip, 64 columns at a
                    // time: each lane then stores 16 contiguous bytes and a store
                    // instruction writes 8 whole 128-byte row segments.  Only this
                    // wave touches its strip; its LDS operations run in order.
                    uint16_t* ow = &Os[wave * 16 * OS];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
#pragma unroll
                        for (int q = 0; q < kCT / 2; ++q) {
                            const int ct = h * (kCT / 2) + q;
                            const float y0 = scale * acc[ct][0], y1 = scale * acc[ct][1];
                            const float y2 = scale * acc[ct][2], y3 = scale * acc[ct][3];
                            *reinterpret_cast<uint2*>(&ow[(lane & 15) * OS + q * 16 + cg]) =
                                make_uint2(Fmt<1>::pack2(y0, y1), Fmt<1>::pack2(y2, y3));
                        }
#pragma unroll
                        for (int it = 0; it < 2; ++it) {
                            const int c = it * 64 + lane;  // 16 rows x 8 chunks of 8 columns
                            const int r = c >> 3, cc = (c & 7) * 8;
                            // the chunk's selection is the bit of its first four-column
                            // group, held by the lane of row r and that group (a chunk
                            // never straddles a block or the row end)
                            const uint32_t so = (uint32_t)__shfl((int)sel, r + 16 * ((cc & 15) >> 2));
                            if ((so >> (h * (kCT / 2) + (cc >> 4))) & 1u) {
                                const uint32_t e = rix[wave * 16 + r] * cols + n0 + h * 64 + cc;
                                *reinterpret_cast<uint4*>(out + e) = *reinterpret_cast<const uint4*>(&ow[r * OS + cc]);
                            }
                        }
                    }
                } else {
                    direct_store();
                }
            } else {
                direct_store();
            }
        } else if (more) {
            load_a(n1, ra);
        }
        // this barrier also ends every wave's reads of As for this tile
        any = any_selected(sel_next, (int)((tn + 1) & 1u));
        sel = sel_next;
    }
}

// Zeros in the selected blocks of tensors without an adapter.
__global__ __launch_bounds__(256) void k_lora_zero(const uint32_t* __restrict__ blocks,
                                                   const uint64_t* __restrict__ boff,
                                                   const uint32_t* __restrict__ blen, int esize, OutPtrs dl,
                                                   const uint32_t* __restrict__ mask)
{
    const uint32_t g = blocks[blockIdx.x];
    const int i = blockIdx.y;
    if (mask != nullptr && !((mask[g] >> i) & 1u))
        return;
    uint4* p = reinterpret_cast<uint4*>(static_cast<char*>(dl.p[i]) + boff[g] * (uint64_t)esize);
    const uint32_t nch = blen[g] * (uint32_t)esize / 16u;
    for (uint32_t c = threadIdx.x; c < nch; c += 256)
        p[c] = make_uint4(0u, 0u, 0u, 0u);
}

// ---------------------------------------------------------------- TIES from thresholds, fused
// The budgeted TIES merge with stored trim thresholds, drawing each delta
// from the adapters inside the merge: out = fma(lambda, mean, x0) with the
// sign election and disjoint mean over the selected units' kept deltas, each
// delta computed exactly as the pull computes it (the same matrix-core tile
// arrangement and summation, the same scaling and rounding to the dtype) and
// never written to memory.
//
// First k_lora_prep lays each adapter out in MFMA operand order, zero-padded
// to the depth RM: A^T (columns padded to a multiple of 64, RM values per
// column) and B (rows padded to a multiple of 16, RM values per row).  An
// operand is then one unconditional 8-byte (bf16) or 4-byte (fp32) load per
// lane, and no staging in LDS is needed.  Zero padding adds exact zero
// products, so the sums equal the pull's.
//
// k_lora_ties: one wave takes 16 rows of an adapted tensor (a quarter of a
// 64-row band) and walks its 64-column tiles, on its own (no workgroup
// barrier).  Per tile it issues the next tile's mask words and this tile's
// base chunks, then for each expert selected in some block the tile meets
// (a wave skips the experts none of its chunks selects), in increasing
// order:
//   * the expert's operands and thresholds arrive from a load issued while
//     the previous expert computed;
//   * it computes the 16 x 64 delta tile as D^T = A^T B^T in four 16 x 16
//     MFMA tiles, scales and rounds it to the dtype, and passes it through
//     its LDS strip so that each lane holds whole 16-byte chunks of one row;
//   * the lane folds its chunks into the TIES state (sums and counts of the
//     kept positive and negative deltas) with the unit's threshold; a chunk
//     whose block does not select the expert gets a NaN threshold, which
//     keeps nothing.
// Then the sign election and mean, and the output chunks are stored.  A
// chunk never straddles a block or a row: rows are a whole number of chunks
// (bf16 tensors need a multiple of 8 columns) and blocks a whole number of
// chunks.  The band's four waves run on one XCD and the bands are split
// into eight contiguous ranges, one per XCD, so that a tensor's operands are
// read into few L2s.
constexpr int kFN = 64;  // fused tile columns (four MFMA tiles of 16)

// Two deltas d0, d1 folded into their elements' TIES state with threshold
// tau: keep d iff d >= tau (positive) or -d >= tau (negative); ps sums the
// kept positive deltas, ns the kept negative ones, cpn counts them (low half
// positive, high half negative).  Eight instructions per delta, the positive
// test being the carry into the count's add (the compiler's own form takes
// ten).  Every lane mask is read at least three instructions after the
// compare that writes it (a VALU write of an SGPR needs two wait states
// before a VALU reads it).  c16 holds 0x10000.
__device__ inline void ties_fold2(float d0, float d1, float tau, uint32_t c16, float& ps0, float& ns0,
                                  uint32_t& cpn0, float& ps1, float& ns1, uint32_t& cpn1)
{
    uint64_t kp0, kn0, kp1, kn1, co;
    float t0, t1;
    asm("v_cmp_le_f32_e64 %[kp0], %[tau], %[d0]\n\t"
        "v_cmp_le_f32_e64 %[kn0], %[tau], -%[d0]\n\t"
        "v_cmp_le_f32_e64 %[kp1], %[tau], %[d1]\n\t"
        "v_cmp_le_f32_e64 %[kn1], %[tau], -%[d1]\n\t"
        "v_cndmask_b32_e64 %[t0], 0, %[d0], %[kp0]\n\t"
        "v_cndmask_b32_e64 %[t1], 0, %[d0], %[kn0]\n\t"
        "v_add_f32_e32 %[ps0], %[ps0], %[t0]\n\t"
        "v_add_f32_e32 %[ns0], %[ns0], %[t1]\n\t"
        "v_cndmask_b32_e64 %[t0], 0, %[d1], %[kp1]\n\t"
        "v_cndmask_b32_e64 %[t1], 0, %[d1], %[kn1]\n\t"
        "v_add_f32_e32 %[ps1], %[ps1], %[t0]\n\t"
        "v_add_f32_e32 %[ns1], %[ns1], %[t1]\n\t"
        "v_cndmask_b32_e64 %[t0], 0, %[c16], %[kn0]\n\t"
        "v_cndmask_b32_e64 %[t1], 0, %[c16], %[kn1]\n\t"
        "v_addc_co_u32_e64 %[cpn0], %[co], %[cpn0], %[t0], %[kp0]\n\t"
        "v_addc_co_u32_e64 %[cpn1], %[co], %[cpn1], %[t1], %[kp1]"
        : [ps0] "+v"(ps0), [ns0] "+v"(ns0), [cpn0] "+v"(cpn0), [ps1] "+v"(ps1), [ns1] "+v"(ns1),
          [cpn1] "+v"(cpn1), [kp0] "=&s"(kp0), [kn0] "=&s"(kn0), [kp1] "=&s"(kp1), [kn1] "=&s"(kn1),
          [co] "=&s"(co), [t0] "=&v"(t0), [t1] "=&v"(t1)
        : [d0] "v"(d0), [d1] "v"(d1), [tau] "v"(tau), [c16] "v"(c16));
}

// Workgroup z of (tensor, expert) lays out columns z*128 .. of A^T and rows
// z*128 .. of B.  A's 128-column slice is read in 16-byte row chunks and
// transposed through LDS, so that both the loads and the stores are
// contiguous across lanes.
constexpr int kPrepCols = 128;

template <int DT, int RM>
__global__ __launch_bounds__(256) void k_lora_prep(const LoraDesc* __restrict__ desc, ExpertPtrs ad, OutPtrs prep,
                                                   int aligned)
{
    using E = typename std::conditional<DT == 0, float, uint16_t>::type;
    constexpr int CV = 16 / sizeof(E);
    constexpr int RS = RM + CV;  // LDS row stride: rows stay 16-byte aligned
    constexpr int CPC = RM / CV; // chunks per A^T column (and per B row)
    __shared__ __align__(16) E T[kPrepCols * RS];
    const LoraDesc D = desc[blockIdx.x];
    const int i = blockIdx.y;
    const uint32_t t = threadIdx.x;
    const E* __restrict__ A = static_cast<const E*>(ad.p[i]) + D.a_off;
    const E* __restrict__ B = static_cast<const E*>(ad.p[i]) + D.b_off;
    E* __restrict__ at = static_cast<E*>(prep.p[i]) + D.at_off;
    E* __restrict__ bp = static_cast<E*>(prep.p[i]) + D.bp_off;
    const uint32_t colsp = (D.cols + kFN - 1) / kFN * kFN, rowsp = (D.rows + 15u) / 16u * 16u;
    const uint32_t c0 = blockIdx.z * kPrepCols;
    if (c0 < colsp) {
        // A[k][c0 + n .. + CV - 1] for k < RM (zeros past the rank and the columns)
        const bool vec = aligned != 0 && D.vec != 0u;
        for (uint32_t c = t; c < (uint32_t)(RM * kPrepCols / CV); c += 256) {
            const uint32_t k = c / (kPrepCols / CV), n = (c % (kPrepCols / CV)) * CV;
            E v[CV];
            if (vec && k < D.rank && c0 + n < D.cols) {
                *reinterpret_cast<uint4*>(v) = *reinterpret_cast<const uint4*>(A + (uint64_t)k * D.cols + c0 + n);
            } else {
#pragma unroll
                for (int q = 0; q < CV; ++q)
                    v[q] = (k < D.rank && c0 + n + q < D.cols) ? A[(uint64_t)k * D.cols + c0 + n + q] : E(0);
            }
#pragma unroll
            for (int q = 0; q < CV; ++q)
                T[(n + q) * RS + k] = v[q];
        }
        __syncthreads();
        const uint32_t ncol = min((uint32_t)kPrepCols, colsp - c0);
        for (uint32_t c = t; c < ncol * CPC; c += 256) {
            const uint32_t n = c / CPC, j = c % CPC;
            reinterpret_cast<uint4*>(at + (uint64_t)(c0 + n) * RM)[j] =
                *reinterpret_cast<const uint4*>(&T[n * RS + j * CV]);
        }
    }
    if (c0 < rowsp) {
        // B's rows c0 .. with RM values each (zeros past the rank and the rows)
        const uint32_t nrow = min((uint32_t)kPrepCols, rowsp - c0);
        if (aligned != 0 && D.rank == (uint32_t)RM && D.b_off % CV == 0) {
            const uint4* src = reinterpret_cast<const uint4*>(B + (uint64_t)c0 * RM);
            uint4* dst = reinterpret_cast<uint4*>(bp + (uint64_t)c0 * RM);
            for (uint32_t c = t; c < nrow * CPC; c += 256)
                dst[c] = (c0 + c / CPC < D.rows) ? src[c] : make_uint4(0u, 0u, 0u, 0u);
        } else {
            for (uint32_t c = t; c < nrow * RM; c += 256) {
                const uint32_t r = c0 + c / RM, k = c % RM;
                bp[(uint64_t)c0 * RM + c] = (k < D.rank && r < D.rows) ? B[(uint64_t)r * D.rank + k] : E(0);
            }
        }
    }
}

template <int DT, int RM>
__global__ __launch_bounds__(64, (DT == 1 && RM == 16) ? 4 : (DT == 0 && RM == 64) ? 1 : 2) void k_lora_ties(const LoraDesc* __restrict__ desc, int n_desc, uint32_t n_bands,
                                                  uint32_t bpx, ExpertPtrs prep, const void* __restrict__ base,
                                                  const uint32_t* __restrict__ mask,
                                                  const uint32_t* __restrict__ tau, int K, uint32_t kmask,
                                                  float lambda, uint32_t block_elems, void* __restrict__ out,
                                                  const uint32_t* __restrict__ zero, const uint64_t* __restrict__ zoff,
                                                  const uint32_t* __restrict__ zlen)
{
    using E = typename std::conditional<DT == 0, float, uint16_t>::type;
    constexpr int KS = DT == 0 ? 4 : 16;  // MFMA depth
    constexpr int CV = 16 / sizeof(E);    // elements per 16-byte chunk
    constexpr int NKS = RM / KS;          // MFMA depth steps
    constexpr int CPR = kFN / CV;         // chunks per strip row
    constexpr int NS = 16 * CPR / 64;     // chunk slots per lane
    constexpr int EL = NS * CV;           // elements per lane (16)
    constexpr int OSR = kFN + CV;         // strip row stride (elements; rows stay 16-byte aligned)
    constexpr int FC = kFN / 16;          // MFMA tiles per tile
    using AOp = typename std::conditional<DT == 0, float, short4_t>::type;
    __shared__ __align__(16) E ow[16 * OSR];
    if (blockIdx.x >= 32u * bpx) {
        // the workgroups past the bands take the blocks of tensors without an
        // adapter, where nothing is kept: fma(lambda, 0, x0), as the merge
        // over zero deltas writes it (they run last and fill the tail)
        constexpr int V = Fmt<DT>::V, ES = Fmt<DT>::esize;
        const uint32_t g = zero[blockIdx.x - 32u * bpx];
        const uint4* src = chunk_ptr(base, zoff[g], ES);
        uint4* dst = reinterpret_cast<uint4*>(static_cast<char*>(out) + zoff[g] * (uint64_t)ES);
        const uint32_t nch = zlen[g] / (uint32_t)V;
        for (uint32_t c0 = 0; c0 < nch; c0 += 4 * 64) {
            uint4 v[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t c = c0 + (uint32_t)(q * 64) + threadIdx.x;
                v[q] = c < nch ? ld16s(src + c) : make_uint4(0u, 0u, 0u, 0u);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t c = c0 + (uint32_t)(q * 64) + threadIdx.x;
                float x0[V], y[V];
                Fmt<DT>::unpack(v[q], x0);
#pragma unroll
                for (int e = 0; e < V; ++e)
                    y[e] = fmaf(lambda, 0.0f, x0[e]);
                if (c < nch)
                    st16s(dst + c, Fmt<DT>::pack(y));
            }
        }
        return;
    }
    // workgroup -> (band, quarter): XCD x = id mod 8 takes bands x*bpx ..
    const uint32_t id = blockIdx.x, xcd = id & 7u, j = id >> 3;
    const uint32_t band = xcd * bpx + (j >> 2);
    if (band >= n_bands)
        return;
    const int lane = threadIdx.x;
    const int d = __builtin_amdgcn_readfirstlane(find_desc(desc, n_desc, band));
    const LoraDesc D = desc[d];
    const uint32_t r0 = (band - D.tile0) * kTM + (j & 3u) * 16u;  // the wave's first row
    const uint32_t rows = D.rows, cols = D.cols;
    if (r0 >= rows)
        return;
    const uint32_t nrow = min(16u, rows - r0);
    const uint32_t tiles = (cols + kFN - 1) / kFN;
    const uint32_t nblk = (uint32_t)(((uint64_t)rows * cols + block_elems - 1) / block_elems);
    const float scale = D.scale;
    const uint32_t c16 = 0x10000u;  // a negative kept delta's count increment
    // the wave's rows of the base as a buffer: a load at an offset past them
    // returns zeros without reading (16 * cols * esize < 2^31, checked by
    // the host, so 2^31 is past them)
    const uint32_t wbytes = nrow * cols * (uint32_t)sizeof(E);
    const __amdgpu_buffer_rsrc_t rbase =
        block_rsrc(static_cast<const E*>(base) + D.toff + (uint64_t)r0 * cols, wbytes);
    E* __restrict__ xo = static_cast<E*>(out) + D.toff + (uint64_t)r0 * cols;
    const uint32_t* __restrict__ mk = mask + D.g0;
    const uint32_t* __restrict__ tk = tau + (uint64_t)D.g0 * (uint32_t)K;
    // operands: A^T column n0 + ct*16 + lane%16, depth k0 + (bf16) 4*(lane/16) .. +3
    // or (fp32) lane/16; B row r0 + lane%16, the same depths
    const uint32_t dk = DT == 1 ? 4u * (uint32_t)(lane >> 4) : (uint32_t)(lane >> 4);
    const uint64_t aoff = D.at_off + (uint64_t)(lane & 15) * RM + dk;
    const uint64_t boff = D.bp_off + (uint64_t)(r0 + (uint32_t)(lane & 15)) * RM + dk;
    // the lane's chunk slots: strip row srow, column scol; element e of the
    // tensor in block lb, lr elements in
    uint32_t srow[NS], scol[NS], lb[NS], lr[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q) {
        const int c = q * 64 + lane;
        srow[q] = (uint32_t)(c / CPR);
        scol[q] = (uint32_t)((c % CPR) * CV);
        const uint32_t e = (r0 + srow[q] < rows) ? (r0 + srow[q]) * cols + scol[q] : 0u;  // < numel < 2^32
        lb[q] = e / block_elems;
        lr[q] = e - lb[q] * block_elems;
    }
    auto chunk_ok = [&](int q, uint32_t n0) { return srow[q] < nrow && n0 + scol[q] < cols; };
    // mask words of a tile's chunks (zero for chunks outside the tensor)
    auto words = [&](uint32_t n0, const uint32_t (&b)[NS], uint32_t (&w)[NS]) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            const uint32_t v = mk[min(b[q], nblk - 1u)];
            w[q] = chunk_ok(q, n0) ? (v & kmask) : 0u;
        }
    };
    auto tile_set = [&](const uint32_t (&w)[NS]) {
        uint32_t o = 0u;
#pragma unroll
        for (int q = 0; q < NS; ++q)
            o |= w[q];
        return wave_or_u32(o);
    };
    struct Ops {
        AOp a[NKS][FC];
        AOp b[NKS];
        uint32_t t[NS];
    };
    // expert i's operands for the tile at column n0, and its thresholds for
    // the tile's blocks b
    auto load_ops = [&](int i, uint32_t n0, const uint32_t (&b)[NS], Ops& o) {
        const E* __restrict__ pa = static_cast<const E*>(prep.p[i]) + aoff + (uint64_t)n0 * RM;
        const E* __restrict__ pb = static_cast<const E*>(prep.p[i]) + boff;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
            for (int ct = 0; ct < FC; ++ct)
                o.a[ks][ct] = *reinterpret_cast<const AOp*>(pa + ct * 16 * RM + ks * KS);
            o.b[ks] = *reinterpret_cast<const AOp*>(pb + ks * KS);
        }
#pragma unroll
        for (int q = 0; q < NS; ++q)
            o.t[q] = tk[(uint64_t)min(b[q], nblk - 1u) * (uint32_t)K + (uint32_t)i];
    };
    uint32_t w[NS];
    words(0u, lb, w);
    uint32_t sel = tile_set(w);
    Ops pre;
    int pre_i = -1;       // the expert whose operands pre holds
    uint32_t pre_t = 0u;  // and their tile
    if (sel != 0u) {
        pre_i = __builtin_ctz(sel);
        load_ops(pre_i, 0u, lb, pre);
    }
    for (uint32_t tn = 0; tn < tiles; ++tn) {
        const uint32_t n0 = tn * kFN;
        const bool more = tn + 1 < tiles;
        // the next tile's blocks and mask words, then this tile's base chunks
        uint32_t lbn[NS], lrn[NS], wn[NS];
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            lbn[q] = lb[q];
            lrn[q] = lr[q] + kFN;
            while (lrn[q] >= block_elems) {
                lrn[q] -= block_elems;
                ++lbn[q];
            }
        }
        words(n0 + kFN, lbn, wn);  // all zero past the last tile (no chunk is inside)
        uint4 xr[NS];
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            const uint32_t off = chunk_ok(q, n0) ? (srow[q] * cols + n0 + scol[q]) * (uint32_t)sizeof(E) : 0x80000000u;
            xr[q] = bld16s(rbase, off);
        }
        float ps[EL], ns[EL];
        uint32_t cpn[EL];
        if (sel == 0u) {
#pragma unroll
            for (int e = 0; e < EL; ++e) {
                ps[e] = 0.0f;
                ns[e] = 0.0f;
                cpn[e] = 0u;
            }
        }
        // the first selected expert starts the state: 0 + t is t for every
        // t a kept or dropped delta contributes (kept ones are nonzero)
        bool first = true;
        uint32_t mm = sel;
        while (mm != 0u) {
            const int i = __builtin_ctz(mm);
            mm &= mm - 1u;
            if (pre_i != i || pre_t != tn)  // not prefetched (wave-uniform; not expected)
                load_ops(i, n0, lb, pre);
            const Ops cur = pre;
            // the following expert's operands, in flight while this one computes
            if (mm != 0u) {
                pre_i = __builtin_ctz(mm);
                pre_t = tn;
                load_ops(pre_i, n0, lb, pre);
            } else if (more) {
                const uint32_t sn = tile_set(wn);
                if (sn != 0u) {
                    pre_i = __builtin_ctz(sn);
                    pre_t = tn + 1;
                    load_ops(pre_i, n0 + kFN, lbn, pre);
                }
            }
            float4_t acc[FC];
#pragma unroll
            for (int ct = 0; ct < FC; ++ct)
                acc[ct] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
                for (int ct = 0; ct < FC; ++ct) {
                    if constexpr (DT == 1)
                        acc[ct] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(cur.a[ks][ct], cur.b[ks], acc[ct], 0, 0, 0);
                    else
                        acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur.a[ks][ct], cur.b[ks], acc[ct], 0, 0, 0);
                }
            }
            // the deltas as the pull stores them: scale * acc rounded to the
            // dtype; accumulator j of tile ct is column ct*16 + 4*(lane/16) + j
            // of strip row lane % 16 (the wave's LDS operations run in order)
            const uint32_t cg = 4u * (uint32_t)(lane >> 4);
#pragma unroll
            for (int ct = 0; ct < FC; ++ct) {
                const float y0 = scale * acc[ct][0], y1 = scale * acc[ct][1];
                const float y2 = scale * acc[ct][2], y3 = scale * acc[ct][3];
                E* p = &ow[(lane & 15) * OSR + ct * 16 + cg];
                if constexpr (DT == 1)
                    *reinterpret_cast<uint2*>(p) = make_uint2(Fmt<1>::pack2(y0, y1), Fmt<1>::pack2(y2, y3));
                else
                    *reinterpret_cast<float4*>(p) = make_float4(y0, y1, y2, y3);
            }
#pragma unroll
            for (int q = 0; q < NS; ++q) {
                const uint4 raw = *reinterpret_cast<const uint4*>(&ow[srow[q] * OSR + scol[q]]);
                float x[CV];
                Fmt<DT>::unpack(raw, x);
                // keep |d| >= tau (at least the smallest positive pattern); a
                // NaN threshold where the block does not select expert i
                const float tauf = __uint_as_float(((w[q] >> i) & 1u) ? max(cur.t[q], 1u) : 0x7fc00000u);
                if (first) {
#pragma unroll
                    for (int v = 0; v < CV; ++v) {
                        const int e = q * CV + v;
                        const bool kp = x[v] >= tauf, kn = -x[v] >= tauf;
                        ps[e] = kp ? x[v] : 0.0f;
                        ns[e] = kn ? x[v] : 0.0f;
                        cpn[e] = kp ? 1u : (kn ? 0x10000u : 0u);
                    }
                } else {
#pragma unroll
                    for (int v = 0; v < CV; v += 2) {
                        const int e = q * CV + v;
                        ties_fold2(x[v], x[v + 1], tauf, c16, ps[e], ns[e], cpn[e], ps[e + 1], ns[e + 1],
                                   cpn[e + 1]);
                    }
                }
            }
            first = false;
        }
        float mean[EL];
        ties_elect_mean<EL>(ps, ns, cpn, mean, lane);
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            float x0[CV], y[CV];
            Fmt<DT>::unpack(xr[q], x0);
#pragma unroll
            for (int v = 0; v < CV; ++v)
                y[v] = fmaf(lambda, mean[q * CV + v], x0[v]);
            if (chunk_ok(q, n0))
                st16s(reinterpret_cast<uint4*>(xo + (uint64_t)srow[q] * cols + n0 + scol[q]), Fmt<DT>::pack(y));
        }
        sel = tile_set(wn);
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            lb[q] = lbn[q];
            lr[q] = lrn[q];
            w[q] = wn[q];
        }
    }
}

// The pull of every unit on the operand-order copy (the full pull the
// catalog reads): one wave per 16 rows of a band and expert (blockIdx.y),
// 64-column tiles with the next tile's A operands in flight, the B operands
// held for the whole band, and the deltas stored as whole 16-byte chunks
// through the wave's LDS strip.  The same MFMA tiles as k_lora_band, so the
// same bits.  Workgroups past the bands write the zeros of tensors without
// an adapter.
template <int DT, int RM, bool MASKED>
__global__ __launch_bounds__(64) void k_lora_pull(const LoraDesc* __restrict__ desc, int n_desc, uint32_t n_bands,
                                                  uint32_t bpx, ExpertPtrs prep, OutPtrs dl,
                                                  const uint32_t* __restrict__ zero, const uint64_t* __restrict__ zoff,
                                                  const uint32_t* __restrict__ zlen,
                                                  const uint32_t* __restrict__ mask, uint32_t block_elems)
{
    using E = typename std::conditional<DT == 0, float, uint16_t>::type;
    constexpr int KS = DT == 0 ? 4 : 16;
    constexpr int CV = 16 / sizeof(E);
    constexpr int NKS = RM / KS;
    constexpr int CPR = kFN / CV;
    constexpr int NS = 16 * CPR / 64;
    constexpr int OSR = kFN + CV;
    constexpr int FC = kFN / 16;
    using AOp = typename std::conditional<DT == 0, float, short4_t>::type;
    __shared__ __align__(16) E ow[16 * OSR];
    const int i = blockIdx.y;
    const int lane = threadIdx.x;
    if (blockIdx.x >= 32u * bpx) {
        const uint32_t g = zero[blockIdx.x - 32u * bpx];
        if (MASKED && !((mask[g] >> i) & 1u))
            return;
        uint4* dst = reinterpret_cast<uint4*>(static_cast<char*>(dl.p[i]) + zoff[g] * (uint64_t)sizeof(E));
        const uint32_t nch = zlen[g] / (uint32_t)CV;
        for (uint32_t c = (uint32_t)lane; c < nch; c += 64)
            st16s(dst + c, make_uint4(0u, 0u, 0u, 0u));
        return;
    }
    const uint32_t id = blockIdx.x, xcd = id & 7u, j = id >> 3;
    const uint32_t band = xcd * bpx + (j >> 2);
    if (band >= n_bands)
        return;
    const int d = __builtin_amdgcn_readfirstlane(find_desc(desc, n_desc, band));
    const LoraDesc D = desc[d];
    const uint32_t r0 = (band - D.tile0) * kTM + (j & 3u) * 16u;
    const uint32_t rows = D.rows, cols = D.cols;
    if (r0 >= rows)
        return;
    const uint32_t nrow = min(16u, rows - r0);
    const uint32_t tiles = (cols + kFN - 1) / kFN;
    const float scale = D.scale;
    E* __restrict__ xo = static_cast<E*>(dl.p[i]) + D.toff + (uint64_t)r0 * cols;
    const uint32_t dk = DT == 1 ? 4u * (uint32_t)(lane >> 4) : (uint32_t)(lane >> 4);
    const E* __restrict__ pa = static_cast<const E*>(prep.p[i]) + D.at_off + (uint64_t)(lane & 15) * RM + dk;
    const E* __restrict__ pb = static_cast<const E*>(prep.p[i]) + D.bp_off + (uint64_t)(r0 + (uint32_t)(lane & 15)) * RM + dk;
    AOp b[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
        b[ks] = *reinterpret_cast<const AOp*>(pb + ks * KS);
    auto load_a = [&](uint32_t n0, AOp (&a)[NKS][FC]) {
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
            for (int ct = 0; ct < FC; ++ct)
                a[ks][ct] = *reinterpret_cast<const AOp*>(pa + (uint64_t)(n0 + ct * 16) * RM + ks * KS);
    };
    AOp pre[NKS][FC];
    load_a(0u, pre);
    const uint32_t cg = 4u * (uint32_t)(lane >> 4);
    // masked: the lane's chunk slots' blocks (tracked across tiles) and
    // whether expert i is selected there
    uint32_t lb[NS], lr[NS];
    const uint32_t nblk = (uint32_t)(((uint64_t)rows * cols + block_elems - 1) / block_elems);
    if (MASKED) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            const int c = q * 64 + lane;
            const uint32_t sr = (uint32_t)(c / CPR), sc = (uint32_t)((c % CPR) * CV);
            const uint32_t e = (sr < nrow) ? (r0 + sr) * cols + sc : 0u;  // < numel < 2^32
            lb[q] = e / block_elems;
            lr[q] = e - lb[q] * block_elems;
        }
    }
    for (uint32_t tn = 0; tn < tiles; ++tn) {
        const uint32_t n0 = tn * kFN;
        bool selq[NS];
        if (MASKED) {
            uint32_t any = 0u;
#pragma unroll
            for (int q = 0; q < NS; ++q) {
                const int c = q * 64 + lane;
                const uint32_t sr = (uint32_t)(c / CPR), sc = (uint32_t)((c % CPR) * CV);
                const uint32_t w = mask[D.g0 + min(lb[q], nblk - 1u)];  // clamped into the tensor
                selq[q] = sr < nrow && n0 + sc < cols && ((w >> i) & 1u);
                any |= selq[q] ? 1u : 0u;
            }
            // the next tile's blocks
#pragma unroll
            for (int q = 0; q < NS; ++q) {
                lr[q] += kFN;
                while (lr[q] >= block_elems) {
                    lr[q] -= block_elems;
                    ++lb[q];
                }
            }
            if (wave_or_u32(any) == 0u) {  // nothing selected in the wave's tile: no compute, no store
                if (tn + 1 < tiles)
                    load_a(n0 + kFN, pre);
                continue;
            }
        }
        AOp cur[NKS][FC];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
            for (int ct = 0; ct < FC; ++ct)
                cur[ks][ct] = pre[ks][ct];
        if (tn + 1 < tiles)
            load_a(n0 + kFN, pre);
        float4_t acc[FC];
#pragma unroll
        for (int ct = 0; ct < FC; ++ct)
            acc[ct] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
            for (int ct = 0; ct < FC; ++ct) {
                if constexpr (DT == 1)
                    acc[ct] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(cur[ks][ct], b[ks], acc[ct], 0, 0, 0);
                else
                    acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur[ks][ct], b[ks], acc[ct], 0, 0, 0);
            }
        }
#pragma unroll
        for (int ct = 0; ct < FC; ++ct) {
            const float y0 = scale * acc[ct][0], y1 = scale * acc[ct][1];
            const float y2 = scale * acc[ct][2], y3 = scale * acc[ct][3];
            E* p = &ow[(lane & 15) * OSR + ct * 16 + cg];
            if constexpr (DT == 1)
                *reinterpret_cast<uint2*>(p) = make_uint2(Fmt<1>::pack2(y0, y1), Fmt<1>::pack2(y2, y3));
            else
                *reinterpret_cast<float4*>(p) = make_float4(y0, y1, y2, y3);
        }
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            const int c = q * 64 + lane;
            const uint32_t sr = (uint32_t)(c / CPR), sc = (uint32_t)((c % CPR) * CV);
            const uint4 v = *reinterpret_cast<const uint4*>(&ow[sr * OSR + sc]);
            if (MASKED ? selq[q] : (sr < nrow && n0 + sc < cols))
                st16s(reinterpret_cast<uint4*>(xo + (uint64_t)sr * cols + n0 + sc), v);
        }
    }
}

}  // namespace

uint32_t lora_bands(uint32_t rows, uint32_t cols, uint32_t* tiles_n)
{
    *tiles_n = (cols + kTN - 1) / kTN;
    return (rows + kTM - 1) / kTM;
}

hipError_t launch_lora(const BlockTable& bt, const LoraTable& lt, const ExpertPtrs& ad, const OutPtrs& dl, int K,
                       const uint32_t* mask, hipStream_t s, const OutPtrs* prep)
{
    if (prep != nullptr) {
        // the pull on the operand-order copy
        const uint32_t bpx = (lt.n_tiles + 7u) / 8u;
        if (32u * bpx + lt.n_zero == 0u)
            return hipSuccess;
        int aligned = 1;
        for (int i = 0; i < K && lt.n_tiles > 0; ++i)
            if (reinterpret_cast<uintptr_t>(ad.p[i]) % 16 != 0)
                aligned = 0;
        const dim3 pgrid((unsigned)lt.n_desc, (unsigned)K, lt.prep_z), grid(32u * bpx + lt.n_zero, (unsigned)K);
        const uint32_t be = (uint32_t)bt.block_elems;
        ExpertPtrs pp{};
        for (int i = 0; i < K; ++i)
            pp.p[i] = prep->p[i];
#define MP_LORA_PULL(DTV, RMV)                                                                                     \
    do {                                                                                                           \
        if (lt.n_tiles > 0)                                                                                        \
            hipLaunchKernelGGL((k_lora_prep<DTV, RMV>), pgrid, dim3(256), 0, s, lt.d_desc, ad, *prep, aligned);    \
        if (mask != nullptr)                                                                                       \
            hipLaunchKernelGGL((k_lora_pull<DTV, RMV, true>), grid, dim3(64), 0, s, lt.d_desc, lt.n_desc,          \
                               lt.n_tiles, bpx, pp, dl, lt.d_zero, bt.d_off, bt.d_len, mask, be);                   \
        else                                                                                                       \
            hipLaunchKernelGGL((k_lora_pull<DTV, RMV, false>), grid, dim3(64), 0, s, lt.d_desc, lt.n_desc,         \
                               lt.n_tiles, bpx, pp, dl, lt.d_zero, bt.d_off, bt.d_len, mask, be);                   \
    } while (0)
        if (bt.dtype == 0) {
            if (lt.prep_rank == 16)
                MP_LORA_PULL(0, 16);
            else
                MP_LORA_PULL(0, kMaxLoraRank);
        } else {
            if (lt.prep_rank == 16)
                MP_LORA_PULL(1, 16);
            else
                MP_LORA_PULL(1, kMaxLoraRank);
        }
#undef MP_LORA_PULL
        return hipGetLastError();
    }
    if (lt.n_tiles > 0) {
        const dim3 grid((unsigned)lt.n_tiles, (unsigned)K);
        const uint32_t be = (uint32_t)bt.block_elems;
        int aligned = 1;  // every adapter buffer starts 16-byte aligned
        for (int i = 0; i < K; ++i)
            if (reinterpret_cast<uintptr_t>(ad.p[i]) % 16 != 0)
                aligned = 0;
        if (mask != nullptr)
            hipLaunchKernelGGL(k_lora_rows, dim3((unsigned)lt.n_desc, (unsigned)K), dim3(256), 0, s, lt.d_desc,
                               lt.n_desc, mask, be, lt.d_rl, lt.d_rc, lt.rows_total);
        if (bt.dtype == 0)
            hipLaunchKernelGGL(k_lora_band<0>, grid, dim3(256), 0, s, lt.d_desc, lt.n_desc, ad, dl, mask, be,
                               aligned, lt.d_rl, lt.d_rc, lt.rows_total);
        else
            hipLaunchKernelGGL(k_lora_band<1>, grid, dim3(256), 0, s, lt.d_desc, lt.n_desc, ad, dl, mask, be,
                               aligned, lt.d_rl, lt.d_rc, lt.rows_total);
    }
    if (lt.n_zero > 0)
        hipLaunchKernelGGL(k_lora_zero, dim3((unsigned)lt.n_zero, (unsigned)K), dim3(256), 0, s, lt.d_zero,
                           bt.d_off, bt.d_len, bt.esize, dl, mask);
    return hipGetLastError();
}


hipError_t launch_lora_ties(const BlockTable& bt, const LoraTable& lt, const ExpertPtrs& ad, const OutPtrs& prep,
                            int K, const void* base, const uint32_t* mask, const uint32_t* tau, float lambda,
                            void* out, hipStream_t s)
{
    const uint32_t kmask = (K >= 32) ? 0xffffffffu : ((1u << K) - 1u);
    const uint32_t be = (uint32_t)bt.block_elems;
    const uint32_t bpx = (lt.n_tiles + 7u) / 8u;  // bands per XCD
    if (32u * bpx + lt.n_zero == 0u)
        return hipSuccess;
    int aligned = 1;
    for (int i = 0; i < K && lt.n_tiles > 0; ++i)
        if (reinterpret_cast<uintptr_t>(ad.p[i]) % 16 != 0)
            aligned = 0;
    const dim3 pgrid((unsigned)lt.n_desc, (unsigned)K, lt.prep_z), grid(32u * bpx + lt.n_zero);
    ExpertPtrs pp{};
    for (int i = 0; i < K; ++i)
        pp.p[i] = prep.p[i];
#define MP_LORA_TIES(DTV, RMV)                                                                                     \
    do {                                                                                                           \
        if (lt.n_tiles > 0)                                                                                        \
            hipLaunchKernelGGL((k_lora_prep<DTV, RMV>), pgrid, dim3(256), 0, s, lt.d_desc, ad, prep, aligned);     \
        hipLaunchKernelGGL((k_lora_ties<DTV, RMV>), grid, dim3(64), 0, s, lt.d_desc, lt.n_desc, lt.n_tiles, bpx,  \
                           pp, base, mask, tau, K, kmask, lambda, be, out, lt.d_zero, bt.d_off, bt.d_len);         \
    } while (0)
    if (bt.dtype == 0) {
        if (lt.prep_rank == 16)
            MP_LORA_TIES(0, 16);
        else
            MP_LORA_TIES(0, kMaxLoraRank);
    } else {
        if (lt.prep_rank == 16)
            MP_LORA_TIES(1, 16);
        else
            MP_LORA_TIES(1, kMaxLoraRank);
    }
#undef MP_LORA_TIES
    return hipGetLastError();
}

}  // namespace mp
