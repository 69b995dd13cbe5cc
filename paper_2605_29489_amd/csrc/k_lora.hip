// Deltas drawn from low-rank adapters (the LoRA source of Section 3's delta
// iterator): for an adapted tensor viewed as a rows x cols row-major matrix,
// d = scale * (B A) with A (rank x cols) and B (rows x rank), written into
// an explicit-delta checkpoint for the selected units only.
//
// The contraction runs on the matrix cores.  One 256-thread workgroup takes
// a band of 64 rows of one tensor for one expert: it stages the band's B
// rows in LDS once, then walks the band's 128-column tiles, staging each
// tile's A columns transposed in LDS (16-byte loads of the next tile are in
// flight while the current one computes and stores).  Wave w owns rows
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
// A masked pull computes only the rows that hold a selected element:
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

}  // namespace

uint32_t lora_bands(uint32_t rows, uint32_t cols, uint32_t* tiles_n)
{
    *tiles_n = (cols + kTN - 1) / kTN;
    return (rows + kTM - 1) / kTM;
}

hipError_t launch_lora(const BlockTable& bt, const LoraTable& lt, const ExpertPtrs& ad, const OutPtrs& dl, int K,
                       const uint32_t* mask, hipStream_t s)
{
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

}  // namespace mp
