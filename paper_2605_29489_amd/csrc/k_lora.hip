// Deltas drawn from low-rank adapters (the LoRA source of Section 3's delta
// iterator): for an adapted tensor viewed as a rows x cols row-major matrix,
// d = scale * (B A) with A (rank x cols) and B (rows x rank), written into
// an explicit-delta checkpoint for the selected units only.
//
// The contraction runs on the matrix cores.  One 256-thread workgroup takes
// a 64-row x 128-column output tile of one tensor for one expert; wave w
// owns rows w*16 .. w*16+15 and computes the tile transposed, D^T = A^T B^T,
// in eight 16 x 16 MFMA tiles along the columns:
//   MFMA rows    = output columns (operand from A, staged transposed in LDS)
//   MFMA columns = output rows    (operand from B, staged row-major in LDS)
// so that a lane's four accumulators are four consecutive columns of one
// output row: one 8-byte (bf16) or 16-byte (fp32) store each.  The rank is
// zero-padded to the MFMA depth (16 for bf16, 4 for fp32).  A tile with no
// selected element returns before reading its adapters.
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

// The tile's descriptor: the last entry with tile0 <= x (wave-uniform search).
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

template <int DT>
__global__ __launch_bounds__(256) void k_lora_tile(const LoraDesc* __restrict__ desc, int n_desc,
                                                   ExpertPtrs ad, OutPtrs dl, const uint32_t* __restrict__ mask,
                                                   uint32_t block_elems)
{
    using E = typename std::conditional<DT == 0, float, uint16_t>::type;
    constexpr int KS = DT == 0 ? 4 : 16;  // MFMA depth
    constexpr int RS = kMaxLoraRank + 4;  // LDS row stride in elements (breaks bank aliasing, keeps 8 B alignment)
    __shared__ E As[kTN * RS];  // As[n * RS + k] = A[k][n0 + n]
    __shared__ E Bs[kTM * RS];  // Bs[m * RS + k] = B[m0 + m][k]
    const int i = blockIdx.y;
    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int d = __builtin_amdgcn_readfirstlane(find_desc(desc, n_desc, blockIdx.x));
    const LoraDesc D = desc[d];
    const uint32_t q = blockIdx.x - D.tile0;
    const uint32_t m0 = (q / D.tiles_n) * kTM, n0 = (q % D.tiles_n) * kTN;
    const uint32_t rows = D.rows, cols = D.cols, rank = D.rank;
    const uint32_t row = m0 + wave * 16 + (lane & 15);
    const uint32_t cg = 4u * (uint32_t)(lane >> 4);  // the lane's first column inside each 16-column tile
    // selection of the lane's four-column groups (a group never straddles a
    // block: block_elems and cols are multiples of 4)
    uint32_t sel = 0u;
    if (row < rows) {
#pragma unroll
        for (int ct = 0; ct < kCT; ++ct) {
            const uint32_t col = n0 + ct * 16 + cg;
            if (col < cols) {
                const uint32_t e = row * cols + col;  // < numel < 2^32
                const uint32_t g = D.g0 + e / block_elems;
                if (mask == nullptr || ((mask[g] >> i) & 1u))
                    sel |= 1u << ct;
            }
        }
    }
    if (!__syncthreads_or(sel != 0u))
        return;
    const uint32_t rp = (rank + KS - 1) / KS * KS;
    const E* __restrict__ A = static_cast<const E*>(ad.p[i]) + D.a_off;
    const E* __restrict__ B = static_cast<const E*>(ad.p[i]) + D.b_off;
    for (uint32_t x = t; x < rp * kTN; x += 256) {  // coalesced along A's columns
        const uint32_t k = x / kTN, n = x % kTN;
        As[n * RS + k] = (k < rank && n0 + n < cols) ? A[(uint64_t)k * cols + n0 + n] : E(0);
    }
    for (uint32_t x = t; x < rp * kTM; x += 256) {  // B's rows m0.. are contiguous
        const uint32_t m = x / rp, k = x % rp;
        Bs[m * RS + k] = (k < rank && m0 + m < rows) ? B[(uint64_t)(m0 + m) * rank + k] : E(0);
    }
    __syncthreads();
    const int mr = wave * 16 + (lane & 15);  // the B operand row (an output row)
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
                const short4_t a = *reinterpret_cast<const short4_t*>(&As[(ct * 16 + (lane & 15)) * RS + kk]);
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
    // accumulator j of tile ct is output (row, n0 + ct*16 + cg + j)
    const float scale = D.scale;
    E* __restrict__ out = static_cast<E*>(dl.p[i]) + D.toff;
#pragma unroll
    for (int ct = 0; ct < kCT; ++ct) {
        if (!((sel >> ct) & 1u))
            continue;
        const uint64_t e = (uint64_t)row * cols + n0 + ct * 16 + cg;
        const float y0 = scale * acc[ct][0], y1 = scale * acc[ct][1];
        const float y2 = scale * acc[ct][2], y3 = scale * acc[ct][3];
        if constexpr (DT == 1) {
            *reinterpret_cast<uint2*>(out + e) = make_uint2(Fmt<1>::pack2(y0, y1), Fmt<1>::pack2(y2, y3));
        } else {
            *reinterpret_cast<float4*>(out + e) = make_float4(y0, y1, y2, y3);
        }
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

uint32_t lora_tiles(uint32_t rows, uint32_t cols, uint32_t* tiles_n)
{
    *tiles_n = (cols + kTN - 1) / kTN;
    return ((rows + kTM - 1) / kTM) * *tiles_n;
}

hipError_t launch_lora(const BlockTable& bt, const LoraTable& lt, const ExpertPtrs& ad, const OutPtrs& dl, int K,
                       const uint32_t* mask, hipStream_t s)
{
    if (lt.n_tiles > 0) {
        const dim3 grid((unsigned)lt.n_tiles, (unsigned)K);
        if (bt.dtype == 0)
            hipLaunchKernelGGL(k_lora_tile<0>, grid, dim3(256), 0, s, lt.d_desc, lt.n_desc, ad, dl, mask,
                               (uint32_t)bt.block_elems);
        else
            hipLaunchKernelGGL(k_lora_tile<1>, grid, dim3(256), 0, s, lt.d_desc, lt.n_desc, ad, dl, mask,
                               (uint32_t)bt.block_elems);
    }
    if (lt.n_zero > 0)
        hipLaunchKernelGGL(k_lora_zero, dim3((unsigned)lt.n_zero, (unsigned)K), dim3(256), 0, s, lt.d_zero,
                           bt.d_off, bt.d_len, bt.esize, dl, mask);
    return hipGetLastError();
}

}  // namespace mp
