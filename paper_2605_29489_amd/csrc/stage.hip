// Experts in ordinary host memory (MP_HOST_PAGEABLE): the stage-and-merge
// pipeline of Algorithm 2.  The block sequence is cut into chunks.  For each
// chunk, host threads pack the blocks that the merge needs (the selected
// expert blocks; for the index, every expert block) into a pinned staging
// buffer, a side stream copies the packed bytes to a device buffer, and the
// merge (or index) kernels run over the chunk's blocks reading the staged
// copy.  Two buffers alternate, so packing chunk c+1 overlaps the copy of
// chunk c and the kernels of chunk c-1.  Only packed bytes cross PCIe: for a
// merge they are exactly the plan's cost Chat (Prop. 1); the byte offsets of
// the staged blocks are computed on the device from the mask.
#include <hip/hip_runtime.h>

#include <sys/uio.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <thread>
#include <vector>

#include "mp_internal.h"

namespace mp {

namespace {

constexpr int kStageMaxBlocks = 65536;  // blocks per chunk (bounds the offset table)
constexpr int kScanT = 1024;

// Byte offset, inside a staged merge chunk, of each block's first selected
// expert: the exclusive prefix over blocks b0 .. b0+nb-1 of
// popc(mask & kmask) * len * es (the selected experts of a block are packed
// together in increasing expert order).  One workgroup; nb <= kStageMaxBlocks.
__global__ __launch_bounds__(kScanT) void k_stage_offsets(const uint32_t* __restrict__ mask,
                                                          const uint32_t* __restrict__ blen, int64_t b0, int nb,
                                                          uint32_t kmask, uint32_t es, uint64_t* __restrict__ soff)
{
    constexpr int IPT = kStageMaxBlocks / kScanT;  // blocks per thread
    __shared__ unsigned long long wsum[kScanT / 64];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    auto size_of = [&](int b) -> unsigned long long {
        return (unsigned long long)__popc(mask[b0 + b] & kmask) * blen[b0 + b] * es;
    };
    unsigned long long tot = 0;
    for (int q = 0; q < IPT; ++q) {
        const int b = t * IPT + q;
        if (b < nb)
            tot += size_of(b);
    }
    unsigned long long incl = tot;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const unsigned long long y = __shfl_up(incl, (unsigned)off);
        if (lane >= off)
            incl += y;
    }
    if (lane == 63)
        wsum[wave] = incl;
    __syncthreads();
    unsigned long long run = incl - tot;
    for (int w = 0; w < wave; ++w)
        run += wsum[w];
    for (int q = 0; q < IPT; ++q) {
        const int b = t * IPT + q;
        if (b < nb) {
            soff[b] = run;
            run += size_of(b);
        }
    }
}

struct Stager {
    size_t bytes = 0;          // per buffer
    char* h[2] = {nullptr, nullptr};  // pinned host
    char* d[2] = {nullptr, nullptr};  // device
    uint64_t* soff[2] = {nullptr, nullptr};  // device [kStageMaxBlocks]
    hipStream_t side = nullptr;
    hipEvent_t copied[2] = {nullptr, nullptr};
    hipEvent_t consumed[2] = {nullptr, nullptr};
};

size_t g_stage_bytes = size_t(256) << 20;
std::map<int, std::unique_ptr<Stager>> g_stagers;

void free_stager(int dev, Stager& st)
{
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(dev);
    for (int k = 0; k < 2; ++k) {
        if (st.consumed[k])
            (void)hipEventSynchronize(st.consumed[k]);
        if (st.copied[k])
            (void)hipEventSynchronize(st.copied[k]);
    }
    for (int k = 0; k < 2; ++k) {
        ws_host_free(st.h[k]);
        ws_free(st.d[k]);
        ws_free(st.soff[k]);
        if (st.copied[k])
            (void)hipEventDestroy(st.copied[k]);
        if (st.consumed[k])
            (void)hipEventDestroy(st.consumed[k]);
    }
    if (st.side)
        (void)hipStreamDestroy(st.side);
    (void)hipSetDevice(cur);
    st = Stager{};
}

hipError_t get_stager(Stager** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    auto it = g_stagers.find(dev);
    if (it != g_stagers.end() && it->second->bytes == g_stage_bytes) {
        *out = it->second.get();
        return hipSuccess;
    }
    if (it != g_stagers.end()) {
        free_stager(dev, *it->second);
        g_stagers.erase(it);
    }
    auto st = std::make_unique<Stager>();
    st->bytes = g_stage_bytes;
    for (int k = 0; k < 2 && e == hipSuccess; ++k) {
        if ((e = ws_host_malloc((void**)&st->h[k], st->bytes)) != hipSuccess ||
            (e = ws_malloc((void**)&st->d[k], st->bytes)) != hipSuccess ||
            (e = ws_malloc((void**)&st->soff[k], sizeof(uint64_t) * kStageMaxBlocks)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&st->copied[k], hipEventDisableTiming)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&st->consumed[k], hipEventDisableTiming)) != hipSuccess)
            break;
    }
    if (e == hipSuccess)
        e = hipStreamCreateWithFlags(&st->side, hipStreamNonBlocking);
    if (e != hipSuccess) {
        free_stager(dev, *st);
        return e;
    }
    *out = st.get();
    g_stagers.emplace(dev, std::move(st));
    return hipSuccess;
}

// Runs fn(lo, hi) over [0, n) split into contiguous parts on host threads:
// up to 16 for copies from memory; for file reads (blocking I/O) up to 64,
// which keeps that many reads in flight.
template <class Fn>
void parallel_for(int64_t n, Fn fn, bool io = false)
{
    const int64_t cpu = io ? 64 : std::min<int64_t>(16, std::max(1u, std::thread::hardware_concurrency()));
    const int T = (int)std::max<int64_t>(1, std::min<int64_t>(cpu, n));
    if (T <= 1) {
        fn((int64_t)0, n);
        return;
    }
    std::vector<std::thread> th;
    th.reserve((size_t)T);
    for (int q = 0; q < T; ++q)
        th.emplace_back([=] { fn(n * q / T, n * (q + 1) / T); });
    for (auto& x : th)
        x.join();
}

// A view of blocks [b0, b0 + nb) of bt for the index launchers (which
// number blocks from 0).
BlockTable view_of(const BlockTable& bt, int64_t b0, int64_t nb)
{
    BlockTable v;
    v.device = bt.device;
    v.dtype = bt.dtype;
    v.esize = bt.esize;
    v.block_elems = bt.block_elems;
    v.G = nb;
    v.max_len = bt.max_len;
    v.d_off = bt.d_off + b0;
    v.d_len = bt.d_len + b0;
    v.d_tensor = bt.d_tensor + b0;
    v.d_elem0 = bt.d_elem0 + b0;
    return v;
}

}  // namespace

void set_stage_bytes(size_t bytes) { g_stage_bytes = bytes; }

namespace {
// Fault injection for tests: with MP_FAULT_PACK_CHUNK=n in the environment,
// the pack of chunk n of every staged call reports a failed read, as an
// unreadable expert file does.  -1 (unset): no fault.
int64_t fault_chunk()
{
    const char* v = std::getenv("MP_FAULT_PACK_CHUNK");
    if (v == nullptr || *v == '\0')
        return -1;
    char* end = nullptr;
    const long long n = std::strtoll(v, &end, 10);
    return (end != v && n >= 0) ? (int64_t)n : -1;
}
}  // namespace

void release_stagers()
{
    for (auto& kv : g_stagers)
        free_stager(kv.first, *kv.second);
    g_stagers.clear();
}

bool HostExperts::read(int i, void* dst, size_t pos, size_t n) const
{
    if (fd == nullptr) {
        std::memcpy(dst, static_cast<const char*>(ptr[i]) + pos, n);
        return true;
    }
    char* p = static_cast<char*>(dst);
    while (n > 0) {
        const ssize_t r = pread(fd[i], p, n, (off_t)pos);
        if (r < 0 && errno == EINTR)
            continue;
        if (r <= 0) {
            failed.store(1);
            return false;
        }
        p += r;
        pos += (size_t)r;
        n -= (size_t)r;
    }
    return true;
}

namespace {
// Reads the contiguous file range [pos, pos + sum of lengths) of fd into
// the buffers of iov (a run of consecutive selected blocks of one expert,
// each landing at its staging slot); false on an error or end of file.
bool read_run(int fd, struct iovec* iov, int cnt, size_t pos)
{
    while (cnt > 0) {
        const ssize_t r = preadv(fd, iov, std::min(cnt, IOV_MAX), (off_t)pos);
        if (r < 0 && errno == EINTR)
            continue;
        if (r <= 0)
            return false;
        pos += (size_t)r;
        size_t left = (size_t)r;
        while (cnt > 0 && left >= iov->iov_len) {  // drop the filled buffers
            left -= iov->iov_len;
            ++iov;
            --cnt;
        }
        if (cnt > 0 && left > 0) {  // a partly filled buffer
            iov->iov_base = static_cast<char*>(iov->iov_base) + left;
            iov->iov_len -= left;
        }
    }
    return true;
}
}  // namespace

hipError_t stage_index(const BlockTable& bt, const void* base, const HostExperts& experts, int K, bool ties,
                       double density, float* sumsq, uint32_t* tau, hipStream_t s, uint64_t* h2d, bool delta)
{
    *h2d = 0;
    if (bt.G == 0)
        return hipSuccess;
    Stager* st = nullptr;
    hipError_t e = get_stager(&st);
    if (e != hipSuccess)
        return e;
    const size_t es = (size_t)bt.esize;
    const size_t cap_elems = st->bytes / (es * (size_t)K);  // chunk elements per expert
    const int64_t fault = fault_chunk();
    int64_t g = 0;
    for (int c = 0; g < bt.G; ++c) {
        const int k = c & 1;
        const int64_t b0 = g;
        const uint64_t e0 = bt.h_off[(size_t)b0];
        while (g < bt.G && g - b0 < kStageMaxBlocks &&
               bt.h_off[(size_t)g] + bt.h_len[(size_t)g] - e0 <= cap_elems)
            ++g;
        if (g == b0)
            return hipErrorInvalidValue;  // a block larger than the staging buffer
        const int64_t nb = g - b0;
        const size_t chunk = (size_t)(bt.h_off[(size_t)(g - 1)] + bt.h_len[(size_t)(g - 1)] - e0) * es;
        if ((e = hipEventSynchronize(st->consumed[k])) != hipSuccess)
            return e;
        // pack: expert i's bytes of the chunk at i * chunk
        parallel_for((int64_t)K * 16, [&](int64_t lo, int64_t hi) {
            for (int64_t w = lo; w < hi; ++w) {
                const int i = (int)(w / 16), part = (int)(w % 16);
                const size_t a = chunk * part / 16, z = chunk * (part + 1) / 16;
                experts.read(i, st->h[k] + (size_t)i * chunk + a, e0 * es + a, z - a);
            }
        }, experts.fd != nullptr);
        if (c == fault)
            experts.failed.store(1);
        if (experts.failed.load())
            return hipErrorInvalidValue;
        const size_t bytes = chunk * (size_t)K;
        if ((e = hipMemcpyAsync(st->d[k], st->h[k], bytes, hipMemcpyHostToDevice, st->side)) != hipSuccess ||
            (e = hipEventRecord(st->copied[k], st->side)) != hipSuccess ||
            (e = hipStreamWaitEvent(s, st->copied[k], 0)) != hipSuccess)
            return e;
        ExpertPtrs ex{};
        for (int i = 0; i < K; ++i)  // chunk_ptr(ex.p[i], off) lands at the staged copy of element off
            ex.p[i] = reinterpret_cast<const void*>(reinterpret_cast<uintptr_t>(st->d[k]) + (uintptr_t)i * chunk -
                                                    (uintptr_t)(e0 * es));
        const BlockTable v = view_of(bt, b0, nb);
        float* sq = sumsq ? sumsq + b0 * K : nullptr;
        e = ties ? launch_index_ties(v, base, ex, K, density, sq, tau + b0 * K, s, delta)
                 : launch_index(v, base, ex, K, sq, s, delta);
        if (e != hipSuccess || (e = hipEventRecord(st->consumed[k], s)) != hipSuccess)
            return e;
        *h2d += bytes;
    }
    return hipSuccess;
}

hipError_t stage_merge(const BlockTable& bt, const MergeArgs& a, const void* base, const HostExperts& experts,
                       int K, const uint32_t* mask, void* out, unsigned long long* ctr, hipStream_t s,
                       uint64_t* h2d)
{
    *h2d = 0;
    if (bt.G == 0)
        return hipSuccess;
    Stager* st = nullptr;
    hipError_t e = get_stager(&st);
    if (e != hipSuccess)
        return e;
    const uint32_t kmask = (K >= 32) ? 0xffffffffu : ((1u << K) - 1u);
    const size_t es = (size_t)bt.esize;
    // the plan's mask on the host: which blocks to pack
    std::vector<uint32_t> hm((size_t)bt.G);
    if ((e = hipMemcpyAsync(hm.data(), mask, sizeof(uint32_t) * hm.size(), hipMemcpyDeviceToHost, s)) !=
            hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return e;
    auto size_of = [&](int64_t g) -> size_t {
        return (size_t)__builtin_popcount(hm[(size_t)g] & kmask) * bt.h_len[(size_t)g] * es;
    };
    std::vector<size_t> off;
    const int64_t fault = fault_chunk();
    int64_t g = 0;
    for (int c = 0; g < bt.G; ++c) {
        const int k = c & 1;
        const int64_t b0 = g;
        size_t bytes = 0;
        while (g < bt.G && g - b0 < kStageMaxBlocks && bytes + size_of(g) <= st->bytes)
            bytes += size_of(g++);
        if (g == b0)
            return hipErrorInvalidValue;  // one block's selected experts exceed the staging buffer
        const int64_t nb = g - b0;
        if ((e = hipEventSynchronize(st->consumed[k])) != hipSuccess)
            return e;
        if (bytes > 0) {
            off.assign((size_t)nb, 0);
            size_t run = 0;
            for (int64_t b = 0; b < nb; ++b) {
                off[(size_t)b] = run;
                run += size_of(b0 + b);
            }
            if (experts.fd == nullptr) {  // memory: one copy per selected block
                parallel_for(nb, [&](int64_t lo, int64_t hi) {
                    for (int64_t b = lo; b < hi; ++b) {
                        const int64_t gg = b0 + b;
                        const size_t n = (size_t)bt.h_len[(size_t)gg] * es;
                        uint32_t m = hm[(size_t)gg] & kmask;
                        size_t dst = off[(size_t)b];
                        while (m) {
                            const int i = __builtin_ctz(m);
                            m &= m - 1u;
                            experts.read(i, st->h[k] + dst, bt.h_off[(size_t)gg] * es, n);
                            dst += n;
                        }
                    }
                });
            } else {  // files: one vectored read per run of consecutive selected blocks of an expert
                struct Run {
                    int i;
                    int64_t b, e;  // blocks [b, e) of the chunk
                };
                std::vector<Run> runs;
                for (int i = 0; i < K; ++i) {
                    int64_t b = 0;
                    while (b < nb) {
                        while (b < nb && !((hm[(size_t)(b0 + b)] >> i) & 1u))
                            ++b;
                        const int64_t rb = b;
                        while (b < nb && ((hm[(size_t)(b0 + b)] >> i) & 1u))
                            ++b;
                        if (b > rb)
                            runs.push_back({i, rb, b});
                    }
                }
                parallel_for((int64_t)runs.size(), [&](int64_t lo, int64_t hi) {
                    std::vector<struct iovec> iov;
                    for (int64_t q = lo; q < hi; ++q) {
                        const Run& r = runs[(size_t)q];
                        iov.clear();
                        for (int64_t b = r.b; b < r.e; ++b) {
                            const int64_t gg = b0 + b;
                            const size_t n = (size_t)bt.h_len[(size_t)gg] * es;
                            // the expert's slot: after the block's lower selected experts
                            const uint32_t below = hm[(size_t)gg] & kmask & ((1u << r.i) - 1u);
                            iov.push_back({st->h[k] + off[(size_t)b] + (size_t)__builtin_popcount(below) * n, n});
                        }
                        if (!read_run(experts.fd[r.i], iov.data(), (int)iov.size(),
                                      bt.h_off[(size_t)(b0 + r.b)] * es))
                            experts.failed.store(1);
                    }
                }, true);
            }
            if (c == fault)
                experts.failed.store(1);
            if (experts.failed.load())
                return hipErrorInvalidValue;
            if ((e = hipMemcpyAsync(st->d[k], st->h[k], bytes, hipMemcpyHostToDevice, st->side)) != hipSuccess ||
                (e = hipEventRecord(st->copied[k], st->side)) != hipSuccess)
                return e;
        }
        hipLaunchKernelGGL(k_stage_offsets, dim3(1), dim3(kScanT), 0, s, mask, bt.d_len, b0, (int)nb, kmask,
                           (uint32_t)es, st->soff[k]);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        if (bytes > 0 && (e = hipStreamWaitEvent(s, st->copied[k], 0)) != hipSuccess)
            return e;
        if ((e = launch_merge_staged(bt, a, base, K, mask, out, ctr, s, st->d[k], st->soff[k], b0, nb)) !=
                hipSuccess ||
            (e = hipEventRecord(st->consumed[k], s)) != hipSuccess)
            return e;
        *h2d += bytes;
    }
    return hipSuccess;
}

}  // namespace mp
