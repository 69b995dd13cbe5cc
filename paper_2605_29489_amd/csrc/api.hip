// Host runtime behind include/mergepipe.h: argument validation, the cached
// per-(device, layout) block tables, per-device workspaces and dispatch to
// the kernel launchers.  Everything the paper's path computes runs in the
// kernels; this file only checks, allocates, copies tables and enqueues.
#include <hip/hip_runtime.h>

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <set>
#include <string>
#include <vector>

#include "mp_internal.h"

namespace mp {

hipError_t plan_ctl_alloc(PlanCtl** ctl);

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what)
{
    // an allocation that failed (or passed the workspace limit) is MP_E_NOMEM
    return fail(e == hipErrorOutOfMemory ? MP_E_NOMEM : MP_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ------------------------------------------------------------ workspaces
uint64_t g_ws_limit = 0;  // bytes; 0 = no limit
uint64_t g_ws_held = 0;
std::map<const void*, size_t> g_ws_sizes;

int ws_free_r(void* p)
{
    ws_free(p);
    return 0;
}
int ws_host_free_r(void* p)
{
    ws_host_free(p);
    return 0;
}

struct DeviceWs {
    PlanScratch plan;
    unsigned long long* counters = nullptr;  // [256]
    unsigned long long* h_counters = nullptr;  // pinned [256]
    unsigned long long* cov = nullptr;         // coverage counters, grown on demand
    int64_t cov_cap = 0;
    uint32_t* tt_hist = nullptr;               // tensor-scope TIES: digit histograms per (expert, tensor)
    uint4* tt_state = nullptr;                 //   and the select state per pair (+ the error word)
    int64_t tt_pairs = 0;
    uint32_t* h_tt_err = nullptr;              // pinned copy of the error word
};

std::mutex g_mu;
std::map<std::string, std::unique_ptr<BlockTable>> g_tables;
std::map<int, std::unique_ptr<DeviceWs>> g_ws;
struct LoraEntry {
    int device = -1;
    LoraTable t;
};
std::map<std::string, std::unique_ptr<LoraEntry>> g_loras;

void free_lora(LoraEntry& e)
{
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(e.device);
    (void)ws_free_r(e.t.d_desc);
    (void)ws_free_r(e.t.d_zero);
    (void)ws_free_r(e.t.d_rl);
    (void)ws_free_r(e.t.d_rc);
    (void)ws_free_r(e.t.d_prep);
    if (e.t.ev != nullptr)
        (void)hipEventDestroy(e.t.ev);
    (void)hipSetDevice(cur);
}

void free_table(BlockTable& bt)
{
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(bt.device);
    (void)ws_free_r(bt.d_off);
    (void)ws_free_r(bt.d_len);
    (void)ws_free_r(bt.d_tensor);
    (void)ws_free_r(bt.d_elem0);
    (void)ws_free_r(bt.d_chunk);
    (void)ws_free_r(bt.d_tnumel);
    (void)ws_free_r(bt.d_tlen);
    (void)ws_free_r(bt.d_g0);
    (void)hipSetDevice(cur);
}

void free_ws(int dev, DeviceWs& w)
{
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(dev);
    (void)ws_free_r(w.plan.ctl);
    (void)ws_free_r(w.plan.list[0]);
    (void)ws_free_r(w.plan.list[1]);
    (void)ws_free_r(w.plan.tmask);
    (void)ws_host_free_r(w.plan.h_stats);
    (void)ws_free_r(w.counters);
    (void)ws_host_free_r(w.h_counters);
    (void)ws_free_r(w.cov);
    (void)ws_free_r(w.tt_hist);
    (void)ws_free_r(w.tt_state);
    (void)ws_host_free_r(w.h_tt_err);
    (void)hipSetDevice(cur);
}

// ------------------------------------------------------------ layout
int validate_layout(const mp_layout* L, int* esize)
{
    if (L == nullptr)
        return fail(MP_E_ARG, "layout is NULL");
    if (L->dtype != MP_F32 && L->dtype != MP_BF16)
        return fail(MP_E_ARG, "layout.dtype %d is not MP_F32 or MP_BF16", L->dtype);
    if (L->n_tensors < 0)
        return fail(MP_E_ARG, "layout.n_tensors %d < 0", L->n_tensors);
    if (L->n_tensors > 0 && L->numel == nullptr)
        return fail(MP_E_ARG, "layout.numel is NULL");
    *esize = L->dtype == MP_F32 ? 4 : 2;
    const int64_t V = 16 / *esize;
    if (L->block_elems <= 0 || L->block_elems % V != 0)
        return fail(MP_E_ARG, "layout.block_elems %lld must be a positive multiple of %lld",
                    (long long)L->block_elems, (long long)V);
    if (L->block_elems > (int64_t)1 << 30)
        return fail(MP_E_ARG, "layout.block_elems %lld too large", (long long)L->block_elems);
    for (int32_t t = 0; t < L->n_tensors; ++t) {
        if (L->numel[t] < 0 || L->numel[t] % V != 0)
            return fail(MP_E_ARG, "layout.numel[%d] = %lld must be >= 0 and a multiple of %lld", t,
                        (long long)L->numel[t], (long long)V);
    }
    return MP_OK;
}

int64_t count_blocks(const mp_layout* L)
{
    int64_t G = 0;
    for (int32_t t = 0; t < L->n_tensors; ++t)
        G += (L->numel[t] + L->block_elems - 1) / L->block_elems;
    return G;
}

std::string layout_key(int dev, const mp_layout* L)
{
    std::string k;
    k.reserve(32 + 8 * (size_t)L->n_tensors);
    k.append(reinterpret_cast<const char*>(&dev), sizeof dev);
    k.append(reinterpret_cast<const char*>(&L->dtype), sizeof L->dtype);
    k.append(reinterpret_cast<const char*>(&L->block_elems), sizeof L->block_elems);
    if (L->n_tensors > 0)
        k.append(reinterpret_cast<const char*>(L->numel), sizeof(int64_t) * (size_t)L->n_tensors);
    return k;
}

// Looks up or builds the device block table of a validated layout.
int get_table(const mp_layout* L, int esize, BlockTable** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    const std::string key = layout_key(dev, L);
    auto it = g_tables.find(key);
    if (it != g_tables.end()) {
        *out = it->second.get();
        return MP_OK;
    }
    auto bt = std::make_unique<BlockTable>();
    bt->device = dev;
    bt->dtype = L->dtype;
    bt->esize = esize;
    bt->block_elems = L->block_elems;
    bt->n_tensors = L->n_tensors;
    bt->numel.assign(L->numel, L->numel + L->n_tensors);
    const int64_t G = count_blocks(L);
    bt->G = G;
    std::vector<uint32_t> tens((size_t)G);
    std::vector<uint64_t> e0((size_t)G);
    bt->h_off.resize((size_t)G);
    bt->h_len.resize((size_t)G);
    std::set<uint32_t> lens;
    int64_t g = 0, start = 0;
    for (int32_t t = 0; t < L->n_tensors; ++t) {
        for (int64_t x = 0; x < L->numel[t]; x += L->block_elems) {
            const int64_t n = std::min<int64_t>(L->block_elems, L->numel[t] - x);
            bt->h_off[(size_t)g] = (uint64_t)(start + x);
            bt->h_len[(size_t)g] = (uint32_t)n;
            tens[(size_t)g] = (uint32_t)t;
            e0[(size_t)g] = (uint64_t)x;
            lens.insert((uint32_t)n);
            bt->max_len = std::max<uint32_t>(bt->max_len, (uint32_t)n);
            if (n < L->block_elems)
                ++bt->n_short;
            ++g;
        }
        start += L->numel[t];
    }
    bt->P = start;
    bt->n_distinct_len = (int)lens.size();
    // runs of consecutive blocks of one tensor (the tensor-scope TIES passes)
    std::vector<uint4> chunks;
    std::vector<uint64_t> tnumel(L->numel, L->numel + L->n_tensors);
    for (int64_t a = 0; a < G;) {
        int64_t z = a + 1;
        while (z < G && z - a < kChunkBlocks && tens[(size_t)z] == tens[(size_t)a])
            ++z;
        chunks.push_back(make_uint4((uint32_t)a, (uint32_t)z, tens[(size_t)a], 0u));
        a = z;
    }
    bt->n_chunks = (int64_t)chunks.size();
    // the tensor-level plan's table
    std::vector<uint32_t> tlen((size_t)L->n_tensors), tg0((size_t)L->n_tensors + 1, 0);
    std::set<uint32_t> tl;
    for (int32_t t = 0; t < L->n_tensors; ++t) {
        if (L->numel[t] >= ((int64_t)1 << 32))
            bt->tlen_fits = false;
        tlen[(size_t)t] = (uint32_t)L->numel[t];
        tl.insert(tlen[(size_t)t]);
        tg0[(size_t)t + 1] = tg0[(size_t)t] + (uint32_t)((L->numel[t] + L->block_elems - 1) / L->block_elems);
    }
    bt->n_distinct_tlen = (int)tl.size();
    if (G > 0) {
        if ((e = ws_malloc((void**)&bt->d_off, sizeof(uint64_t) * (size_t)G)) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_len, sizeof(uint32_t) * (size_t)G)) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_tensor, sizeof(uint32_t) * (size_t)G)) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_elem0, sizeof(uint64_t) * (size_t)G)) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_chunk, sizeof(uint4) * chunks.size())) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_tnumel, sizeof(uint64_t) * tnumel.size())) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_tlen, sizeof(uint32_t) * tlen.size())) != hipSuccess ||
            (e = ws_malloc((void**)&bt->d_g0, sizeof(uint32_t) * tg0.size())) != hipSuccess) {
            free_table(*bt);
            return fail(MP_E_NOMEM, "block table allocation failed: %s", hipGetErrorString(e));
        }
        if ((e = hipMemcpy(bt->d_off, bt->h_off.data(), sizeof(uint64_t) * (size_t)G, hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_len, bt->h_len.data(), sizeof(uint32_t) * (size_t)G, hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_tensor, tens.data(), sizeof(uint32_t) * (size_t)G, hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_elem0, e0.data(), sizeof(uint64_t) * (size_t)G, hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_chunk, chunks.data(), sizeof(uint4) * chunks.size(), hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_tnumel, tnumel.data(), sizeof(uint64_t) * tnumel.size(), hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_tlen, tlen.data(), sizeof(uint32_t) * tlen.size(), hipMemcpyHostToDevice)) != hipSuccess ||
            (e = hipMemcpy(bt->d_g0, tg0.data(), sizeof(uint32_t) * tg0.size(), hipMemcpyHostToDevice)) != hipSuccess) {
            free_table(*bt);
            return hip_fail(e, "block table upload");
        }
    }
    *out = bt.get();
    g_tables.emplace(key, std::move(bt));
    return MP_OK;
}

int get_ws(DeviceWs** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    auto it = g_ws.find(dev);
    if (it != g_ws.end()) {
        *out = it->second.get();
        return MP_OK;
    }
    auto w = std::make_unique<DeviceWs>();
    if ((e = plan_ctl_alloc(&w->plan.ctl)) != hipSuccess ||
        (e = ws_host_malloc((void**)&w->plan.h_stats, sizeof(uint64_t) * 8)) != hipSuccess ||
        (e = ws_malloc((void**)&w->counters, sizeof(unsigned long long) * 256)) != hipSuccess ||
        (e = ws_host_malloc((void**)&w->h_counters, sizeof(unsigned long long) * 256)) != hipSuccess ||
        (e = ws_host_malloc((void**)&w->h_tt_err, sizeof(uint32_t))) != hipSuccess) {
        free_ws(dev, *w);
        return fail(MP_E_NOMEM, "workspace allocation failed: %s", hipGetErrorString(e));
    }
    *out = w.get();
    g_ws.emplace(dev, std::move(w));
    return MP_OK;
}

// Plan candidate lists hold at most K * (number of short blocks) entries
// after the first round: every later candidate is cheaper than a cut unit,
// hence shorter than block_elems, and each tensor has at most one short block.
int ensure_lists(PlanScratch& ps, int64_t need)
{
    if (ps.list_cap >= need)
        return MP_OK;
    (void)ws_free_r(ps.list[0]);
    (void)ws_free_r(ps.list[1]);
    ps.list[0] = ps.list[1] = nullptr;
    ps.list_cap = 0;
    const size_t bytes = sizeof(uint32_t) * (size_t)std::max<int64_t>(need, 1);
    hipError_t e;
    if ((e = ws_malloc((void**)&ps.list[0], bytes)) != hipSuccess ||
        (e = ws_malloc((void**)&ps.list[1], bytes)) != hipSuccess)
        return fail(MP_E_NOMEM, "plan list allocation failed: %s", hipGetErrorString(e));
    ps.list_cap = std::max<int64_t>(need, 1);
    return MP_OK;
}

// ------------------------------------------------------------ pointer checks
struct Range {
    const char* p;
    size_t n;
    const char* name;
};

int check_device_buffer(const void* p, size_t bytes, const char* name)
{
    if (p == nullptr)
        return fail(MP_E_ARG, "%s is NULL", name);
    if (bytes == 0)
        return MP_OK;
    int dev = 0;
    (void)hipGetDevice(&dev);
    hipPointerAttribute_t a;
    std::memset(&a, 0, sizeof a);
    hipError_t e = hipPointerGetAttributes(&a, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(MP_E_ARG, "%s is not a HIP allocation", name);
    }
    if (a.type != hipMemoryTypeDevice && !a.isManaged)
        return fail(MP_E_ARG, "%s is not device memory", name);
    if (a.type == hipMemoryTypeDevice && a.device != dev)
        return fail(MP_E_ARG, "%s lives on device %d, current device is %d", name, a.device, dev);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p);
    if (e == hipSuccess) {
        const char* b = static_cast<const char*>(base);
        const char* q = static_cast<const char*>(p);
        if (q < b || (size_t)(q - b) + bytes > size)
            return fail(MP_E_ARG, "%s: %zu bytes needed, allocation too small", name, bytes);
    } else {
        (void)hipGetLastError();
    }
    return MP_OK;
}

// Pinned host memory of at least `bytes` bytes from p; *dev receives the
// address at which device kernels read it (they then load over PCIe).
int check_pinned_buffer(const void* p, size_t bytes, const char* name, const void** dev)
{
    if (p == nullptr)
        return fail(MP_E_ARG, "%s is NULL", name);
    *dev = p;
    if (bytes == 0)
        return MP_OK;
    hipPointerAttribute_t a;
    std::memset(&a, 0, sizeof a);
    hipError_t e = hipPointerGetAttributes(&a, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(MP_E_ARG, "%s is not pinned host memory", name);
    }
    if (a.type != hipMemoryTypeHost)
        return fail(MP_E_ARG, "%s is not pinned host memory", name);
    void* base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(reinterpret_cast<hipDeviceptr_t*>(&base), &size,
                              reinterpret_cast<hipDeviceptr_t>(const_cast<void*>(p))) != hipSuccess ||
        base == nullptr) {
        (void)hipGetLastError();
        return fail(MP_E_ARG, "%s: the size of its pinned allocation is unknown", name);
    }
    const size_t used = (size_t)(static_cast<const char*>(p) - static_cast<const char*>(base));
    if (used > size || size - used < bytes)
        return fail(MP_E_ARG, "%s holds %zu bytes from the pointer, %zu needed", name,
                    used > size ? (size_t)0 : size - used, bytes);
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, const_cast<void*>(p), 0) == hipSuccess && d != nullptr)
        *dev = d;
    else
        (void)hipGetLastError();  // unified addressing: the host address is the device address
    return MP_OK;
}

// Host memory of any kind (pageable or pinned) for MP_HOST_PAGEABLE: the
// library reads it on the host only.  Device memory is refused; the size of
// an ordinary host allocation cannot be checked (the caller guarantees it).
int check_host_buffer(const void* p, const char* name)
{
    if (p == nullptr)
        return fail(MP_E_ARG, "%s is NULL", name);
    hipPointerAttribute_t a;
    std::memset(&a, 0, sizeof a);
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();  // unknown to HIP: ordinary host memory
        return MP_OK;
    }
    if (a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeArray)
        return fail(MP_E_ARG, "%s is device memory (use MP_DEVICE)", name);
    return MP_OK;
}

bool overlaps(const Range& a, const Range& b)
{
    return a.n && b.n && a.p < b.p + b.n && b.p < a.p + a.n;
}

struct Common {
    int esize = 0;
    BlockTable* bt = nullptr;
    DeviceWs* ws = nullptr;
    ExpertPtrs ex{};
    size_t ckpt_bytes = 0;
    std::vector<int> fds;  // MP_HOST_FILE: the opened expert files (closed with the call)
    ~Common()
    {
        for (int fd : fds)
            if (fd >= 0)
                (void)close(fd);
    }
};

// The experts of a staged call (MP_HOST_PAGEABLE memory or MP_HOST_FILE files).
void host_experts(const Common& c, const void* const* experts, HostExperts* hx)
{
    if (c.fds.empty())
        hx->ptr = experts;
    else
        hx->fd = c.fds.data();
}

bool staged(int32_t residency) { return residency == MP_HOST_PAGEABLE || residency == MP_HOST_FILE; }

// Validates the arguments every data entry point shares and resolves the
// block table / workspace.  `out` may be NULL (index).
int check_common(const mp_layout* L, const void* base, const void* const* experts, int32_t K,
                 int32_t residency, const void* out, Common* c)
{
    int rc = validate_layout(L, &c->esize);
    if (rc)
        return rc;
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    if (residency != MP_DEVICE && residency != MP_HOST_PINNED && residency != MP_HOST_PAGEABLE &&
        residency != MP_HOST_FILE)
        return fail(MP_E_ARG, "residency %d is not MP_DEVICE, MP_HOST_PINNED, MP_HOST_PAGEABLE or MP_HOST_FILE",
                    residency);
    const int64_t G = count_blocks(L);
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return fail(MP_E_ARG, "K * G = %lld does not fit 32-bit unit ids", (long long)(G * K));
    int64_t P = 0;
    for (int32_t t = 0; t < L->n_tensors; ++t)
        P += L->numel[t];
    c->ckpt_bytes = (size_t)P * (size_t)c->esize;
    if (experts == nullptr)
        return fail(MP_E_ARG, "experts is NULL");
    if ((rc = check_device_buffer(base, c->ckpt_bytes, "base")))
        return rc;
    std::vector<Range> ranges;
    ranges.push_back({static_cast<const char*>(base), c->ckpt_bytes, "base"});
    for (int i = 0; i < K; ++i) {
        char nm[32];
        std::snprintf(nm, sizeof nm, "experts[%d]", i);
        const void* dev = experts[i];
        if (residency == MP_HOST_FILE) {  // experts[i] is the path of a file holding the checkpoint
            if (experts[i] == nullptr)
                return fail(MP_E_ARG, "%s: path is NULL", nm);
            const char* path = static_cast<const char*>(experts[i]);
            const int fd = open(path, O_RDONLY | O_CLOEXEC);
            if (fd < 0)
                return fail(MP_E_IO, "%s: cannot open %s: %s", nm, path, std::strerror(errno));
            c->fds.push_back(fd);
            // only the selected blocks may be read (Prop. 1): no readahead of their neighbours
            (void)posix_fadvise(fd, 0, 0, POSIX_FADV_RANDOM);
            struct stat sb;
            if (fstat(fd, &sb) != 0 || (uint64_t)sb.st_size < (uint64_t)c->ckpt_bytes)
                return fail(MP_E_ARG, "%s: %s holds fewer than the checkpoint's %zu bytes", nm, path,
                            c->ckpt_bytes);
            c->ex.p[i] = nullptr;
            continue;
        }
        if (residency == MP_DEVICE)
            rc = check_device_buffer(experts[i], c->ckpt_bytes, nm);
        else if (residency == MP_HOST_PINNED)
            rc = check_pinned_buffer(experts[i], c->ckpt_bytes, nm, &dev);
        else
            rc = check_host_buffer(experts[i], nm);
        if (rc)
            return rc;
        c->ex.p[i] = dev;
        ranges.push_back({static_cast<const char*>(experts[i]), c->ckpt_bytes, "expert"});
    }
    if (out != nullptr) {
        if ((rc = check_device_buffer(out, c->ckpt_bytes, "out")))
            return rc;
        const Range o{static_cast<const char*>(out), c->ckpt_bytes, "out"};
        for (const Range& r : ranges)
            if (overlaps(o, r))
                return fail(MP_E_ARG, "out overlaps %s", r.name);
    }
    if ((rc = get_table(L, c->esize, &c->bt)))
        return rc;
    if ((rc = get_ws(&c->ws)))
        return rc;
    return MP_OK;
}

__global__ void k_zero_u64(unsigned long long* p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        p[i] = 0ull;
}

// Splits a residency argument into where the experts live and whether they
// hold explicit deltas (MP_EXPERTS_DELTA).
bool take_delta(int32_t* residency)
{
    const bool delta = (*residency & MP_EXPERTS_DELTA) != 0;
    *residency &= ~MP_EXPERTS_DELTA;
    return delta;
}

int run_merge(const mp_layout* L, const void* base, const void* const* experts, int32_t K,
              int32_t residency, const uint32_t* mask, void* out, mp_io_stats* io, hipStream_t s,
              MergeArgs a)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    a.bsub = take_delta(&residency) ? 0.0f : 1.0f;
    Common c;
    int rc = check_common(L, base, experts, K, residency, out, &c);
    if (rc)
        return rc;
    const BlockTable& bt = *c.bt;
    if ((rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)bt.G, "mask")))
        return rc;
    if (a.op == Op::TIES && bt.max_len > (uint32_t)kTiesMaxBlock)
        return fail(MP_E_UNSUPPORTED, "TIES supports blocks of at most %d elements", kTiesMaxBlock);
    if (a.op == Op::TIES_TAU && (rc = check_device_buffer(a.tau, sizeof(uint32_t) * (size_t)(bt.G * K), "tau")))
        return rc;
    unsigned long long* ctr = io ? c.ws->counters : nullptr;
    hipError_t e;
    if (ctr) {
        hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(256), 0, s, ctr, 256);
        if ((e = hipGetLastError()) != hipSuccess)
            return hip_fail(e, "counter reset");
    }
    mp_io_stats st{};
    uint64_t staged_bytes = 0;
    if (staged(residency)) {
        HostExperts hx;
        host_experts(c, experts, &hx);
        e = stage_merge(bt, a, base, hx, K, mask, out, ctr, s, &staged_bytes);
        if (hx.failed.load())
            return fail(MP_E_IO, "packing expert blocks failed (a failed file read, or MP_FAULT_PACK_CHUNK)");
        if (e != hipSuccess)
            return hip_fail(e, "staged merge");
    } else if ((e = launch_merge(bt, a, base, c.ex, K, mask, out, ctr, s)) != hipSuccess) {
        return hip_fail(e, "merge launch");
    }
    if (io) {
        if ((e = hipMemcpyAsync(c.ws->h_counters, ctr, sizeof(unsigned long long) * 256,
                                hipMemcpyDeviceToHost, s)) != hipSuccess)
            return hip_fail(e, "counter readback");
        if ((e = hipStreamSynchronize(s)) != hipSuccess)
            return hip_fail(e, "hipStreamSynchronize");
        unsigned long long sum = 0;
        for (int q = 0; q < 256; ++q) {  // slot (block mod 8) * 32 + expert
            st.expert_bytes_by_expert[q & 31] += c.ws->h_counters[q];
            sum += c.ws->h_counters[q];
        }
        st.expert_bytes = sum;
        if (residency == MP_HOST_PINNED)
            st.h2d_bytes = sum;  // expert blocks are read over PCIe, nothing else crosses it
        else if (staged(residency))
            st.h2d_bytes = staged_bytes;  // the packed selected blocks
        st.base_bytes = (uint64_t)bt.P * (uint64_t)bt.esize;
        st.out_bytes = st.base_bytes;
        *io = st;
    }
    return MP_OK;
}

}  // namespace

namespace {
hipError_t ws_take(void** p, size_t bytes, bool host)
{
    *p = nullptr;
    if (g_ws_limit != 0 && g_ws_held + bytes > g_ws_limit)
        return hipErrorOutOfMemory;
    const hipError_t e = host ? hipHostMalloc(p, bytes, hipHostMallocDefault) : hipMalloc(p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        return e;
    }
    g_ws_sizes[*p] = bytes;
    g_ws_held += bytes;
    return hipSuccess;
}
void ws_give(void* p, bool host)
{
    if (p == nullptr)
        return;
    auto it = g_ws_sizes.find(p);
    if (it != g_ws_sizes.end()) {
        g_ws_held -= it->second;
        g_ws_sizes.erase(it);
    }
    (void)(host ? hipHostFree(p) : hipFree(p));
}
}  // namespace

hipError_t ws_malloc(void** p, size_t bytes) { return ws_take(p, bytes, false); }
hipError_t ws_host_malloc(void** p, size_t bytes) { return ws_take(p, bytes, true); }
void ws_free(void* p) { ws_give(p, false); }
void ws_host_free(void* p) { ws_give(p, true); }

}  // namespace mp

using namespace mp;

extern "C" {

int mp_layout_blocks(const mp_layout* layout, int64_t* n_blocks)
{
    g_err.clear();
    int es = 0;
    int rc = validate_layout(layout, &es);
    if (rc)
        return rc;
    if (n_blocks == nullptr)
        return fail(MP_E_ARG, "n_blocks is NULL");
    *n_blocks = count_blocks(layout);
    return MP_OK;
}

int mp_index_blocks(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                    int32_t residency, float* sumsq, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    const bool delta = take_delta(&residency);
    Common c;
    int rc = check_common(layout, base, experts, K, residency, nullptr, &c);
    if (rc)
        return rc;
    const BlockTable& bt = *c.bt;
    if ((rc = check_device_buffer(sumsq, sizeof(float) * (size_t)(bt.G * K), "sumsq")))
        return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (staged(residency)) {
        uint64_t staged_bytes = 0;
        HostExperts hx;
        host_experts(c, experts, &hx);
        e = stage_index(bt, base, hx, K, false, 0.0, sumsq, nullptr, s, &staged_bytes, delta);
        if (hx.failed.load())
            return fail(MP_E_IO, "packing expert blocks failed (a failed file read, or MP_FAULT_PACK_CHUNK)");
    } else {
        e = launch_index(bt, base, c.ex, K, sumsq, s, delta);
    }
    if (e != hipSuccess)
        return hip_fail(e, "index launch");
    return MP_OK;
}

int mp_index_ties(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                  int32_t residency, double density, float* sumsq, uint32_t* tau, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    if (!(density >= 0.0 && density <= 1.0))
        return fail(MP_E_ARG, "density %g must be in [0, 1]", density);
    const bool delta = take_delta(&residency);
    Common c;
    int rc = check_common(layout, base, experts, K, residency, nullptr, &c);
    if (rc)
        return rc;
    const BlockTable& bt = *c.bt;
    if (bt.max_len > (uint32_t)kTiesMaxBlock)
        return fail(MP_E_UNSUPPORTED, "TIES supports blocks of at most %d elements", kTiesMaxBlock);
    if (sumsq != nullptr && (rc = check_device_buffer(sumsq, sizeof(float) * (size_t)(bt.G * K), "sumsq")))
        return rc;
    if ((rc = check_device_buffer(tau, sizeof(uint32_t) * (size_t)(bt.G * K), "tau")))
        return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (staged(residency)) {
        uint64_t staged_bytes = 0;
        HostExperts hx;
        host_experts(c, experts, &hx);
        e = stage_index(bt, base, hx, K, true, density, sumsq, tau, s, &staged_bytes, delta);
        if (hx.failed.load())
            return fail(MP_E_IO, "packing expert blocks failed (a failed file read, or MP_FAULT_PACK_CHUNK)");
    } else {
        e = launch_index_ties(bt, base, c.ex, K, density, sumsq, tau, s, delta);
    }
    if (e != hipSuccess)
        return hip_fail(e, "index launch");
    return MP_OK;
}

int mp_coverage(const mp_layout* layout, int32_t K, const uint32_t* mask, uint64_t* cov, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    int es = 0;
    int rc = validate_layout(layout, &es);
    if (rc)
        return rc;
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    if (cov == nullptr)
        return fail(MP_E_ARG, "cov is NULL");
    BlockTable* bt = nullptr;
    DeviceWs* ws = nullptr;
    if ((rc = get_table(layout, es, &bt)) || (rc = get_ws(&ws)))
        return rc;
    if ((rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)bt->G, "mask")))
        return rc;
    const int64_t n = bt->n_tensors * K;
    hipError_t e;
    if (n > ws->cov_cap) {
        (void)ws_free_r(ws->cov);
        ws->cov = nullptr;
        ws->cov_cap = 0;
        if ((e = ws_malloc((void**)&ws->cov, sizeof(unsigned long long) * (size_t)n)) != hipSuccess)
            return fail(MP_E_NOMEM, "coverage buffer: %s", hipGetErrorString(e));
        ws->cov_cap = n;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((e = launch_coverage(*bt, K, mask, ws->cov, s)) != hipSuccess)
        return hip_fail(e, "coverage launch");
    if (n > 0 && (e = hipMemcpyAsync(cov, ws->cov, sizeof(uint64_t) * (size_t)n, hipMemcpyDeviceToHost, s)) !=
                     hipSuccess)
        return hip_fail(e, "coverage readback");
    if ((e = hipStreamSynchronize(s)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    return MP_OK;
}

int mp_ties_tensor_thresholds(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                              int32_t residency, const uint32_t* mask, double density, uint32_t* tau,
                              void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    if (!(density >= 0.0 && density <= 1.0))
        return fail(MP_E_ARG, "density %g must be in [0, 1]", density);
    const bool delta = take_delta(&residency);
    if (staged(residency))
        return fail(MP_E_UNSUPPORTED, "tensor-scope thresholds need device or pinned experts");
    Common c;
    int rc = check_common(layout, base, experts, K, residency, nullptr, &c);
    if (rc)
        return rc;
    const BlockTable& bt = *c.bt;
    if ((rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)bt.G, "mask")))
        return rc;
    if ((rc = check_device_buffer(tau, sizeof(uint32_t) * (size_t)(bt.G * K), "tau")))
        return rc;
    const int64_t pairs = (int64_t)K * bt.n_tensors;
    hipError_t e;
    DeviceWs& ws = *c.ws;
    if (pairs > ws.tt_pairs) {
        (void)ws_free_r(ws.tt_hist);
        (void)ws_free_r(ws.tt_state);
        ws.tt_hist = nullptr;
        ws.tt_state = nullptr;
        ws.tt_pairs = 0;
        if ((e = ws_malloc((void**)&ws.tt_hist, sizeof(uint32_t) * 2048 * (size_t)pairs)) != hipSuccess ||
            (e = ws_malloc((void**)&ws.tt_state, sizeof(uint4) * (size_t)(pairs + 1))) != hipSuccess)
            return fail(MP_E_NOMEM, "tensor-scope TIES buffers: %s", hipGetErrorString(e));
        ws.tt_pairs = pairs;
    }
    // The scratch is shared by every call on this device: the call returns
    // only once its kernels are done (under the library lock), so a call on
    // another stream never finds it in use, and the error word is read here.
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (bt.G == 0)
        return MP_OK;  // no units: nothing to select
    const char* hook = std::getenv("MP_FAULT_TENSOR_NO_CUT");
    const bool force = hook != nullptr && hook[0] == '1';
    if ((e = launch_ties_tensor(bt, base, c.ex, K, mask, density, tau, ws.tt_hist, ws.tt_state, s, delta, force)) !=
        hipSuccess)
        return hip_fail(e, "tensor-scope thresholds launch");
    if ((e = hipMemcpyAsync(ws.h_tt_err, ws.tt_state + pairs, sizeof(uint32_t), hipMemcpyDeviceToHost, s)) !=
        hipSuccess)
        return hip_fail(e, "tensor-scope error word readback");
    if ((e = hipStreamSynchronize(s)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    if (*ws.h_tt_err != 0u)
        return fail(MP_E_HIP, "tensor-scope threshold kernels reported an internal error (no cut found)");
    return MP_OK;
}

int mp_plan(const mp_layout* layout, int32_t K, const float* sumsq, const float* w,
            uint64_t budget_bytes, uint32_t flags, uint32_t* mask, mp_plan_stats* stats, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    int es = 0;
    int rc = validate_layout(layout, &es);
    if (rc)
        return rc;
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    if ((flags & ~(uint32_t)(MP_PLAN_PER_BYTE | MP_PLAN_SKIP_ZERO)) != 0u)
        return fail(MP_E_UNSUPPORTED, "plan flags 0x%x not supported", flags);
    if (w == nullptr || stats == nullptr)
        return fail(MP_E_ARG, "w and stats must not be NULL");
    const int64_t G = count_blocks(layout);
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return fail(MP_E_ARG, "K * G does not fit 32-bit unit ids");
    Coeffs cw{};
    for (int i = 0; i < K; ++i) {
        if (!std::isfinite(w[i]))
            return fail(MP_E_ARG, "w[%d] is not finite", i);
        cw.v[i] = w[i];
    }
    // sumsq NULL: no catalog, the deterministic fallback ranking
    if (sumsq != nullptr && (rc = check_device_buffer(sumsq, sizeof(float) * (size_t)(G * K), "sumsq")))
        return rc;
    if ((rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)G, "mask")))
        return rc;
    BlockTable* bt = nullptr;
    DeviceWs* ws = nullptr;
    if ((rc = get_table(layout, es, &bt)) || (rc = get_ws(&ws)))
        return rc;
    if (sumsq == nullptr) {
        // tensor-level plan: a selection word per tensor, K units per tensor
        if (!bt->tlen_fits)
            return fail(MP_E_UNSUPPORTED, "the tensor-level plan needs tensors of fewer than 2^32 elements");
        if (bt->n_tensors > ws->plan.tmask_cap) {
            (void)ws_free_r(ws->plan.tmask);
            ws->plan.tmask = nullptr;
            ws->plan.tmask_cap = 0;
            hipError_t he = ws_malloc((void**)&ws->plan.tmask, sizeof(uint32_t) * (size_t)bt->n_tensors);
            if (he != hipSuccess)
                return fail(MP_E_NOMEM, "tensor selection words: %s", hipGetErrorString(he));
            ws->plan.tmask_cap = bt->n_tensors;
        }
    }
    const int64_t per_k = sumsq != nullptr ? bt->n_short : bt->n_tensors;
    if ((rc = ensure_lists(ws->plan, (int64_t)K * std::max<int64_t>(per_k, 1))))
        return rc;
    // the blocks partition the checkpoint: their lengths sum to P
    const uint64_t full = (uint64_t)bt->P * (uint64_t)es * (uint64_t)K;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = launch_plan(*bt, ws->plan, K, sumsq, cw, flags, budget_bytes, full, mask, s);
    if (e != hipSuccess)
        return hip_fail(e, "plan launch");
    if ((e = hipStreamSynchronize(s)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    const uint64_t* h = ws->plan.h_stats;
    stats->budget_bytes = h[0];
    stats->cost_bytes = h[1];
    stats->full_bytes = h[2];
    stats->n_selected = h[3];
    stats->n_units = h[4];
    stats->digest = h[5];
    if (h[6] != 0)
        return fail(MP_E_HIP, "plan kernels reported internal error %llu", (unsigned long long)h[6]);
    if (stats->cost_bytes > budget_bytes)
        return fail(MP_E_HIP, "plan cost %llu exceeds the budget %llu", (unsigned long long)stats->cost_bytes,
                    (unsigned long long)budget_bytes);
    return MP_OK;
}

int mp_plan_noalloc(const mp_layout* layout, int32_t K, const float* sumsq, const float* w,
                    uint64_t budget_bytes, uint32_t flags, uint32_t* mask, mp_plan_stats* stats, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    int es = 0;
    int rc = validate_layout(layout, &es);
    if (rc)
        return rc;
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    if ((flags & ~(uint32_t)(MP_PLAN_PER_BYTE | MP_PLAN_SKIP_ZERO)) != 0u)
        return fail(MP_E_UNSUPPORTED, "plan flags 0x%x not supported", flags);
    if (w == nullptr || stats == nullptr)
        return fail(MP_E_ARG, "w and stats must not be NULL");
    // the block partition's counts, on the host without allocating
    int64_t G = 0, n_short = 0, P = 0;
    for (int32_t t = 0; t < layout->n_tensors; ++t) {
        const int64_t n = layout->numel[t];
        G += (n + layout->block_elems - 1) / layout->block_elems;
        n_short += (n % layout->block_elems) != 0 ? 1 : 0;
        P += n;
    }
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return fail(MP_E_ARG, "K * G does not fit 32-bit unit ids");
    if (sumsq == nullptr)
        for (int32_t t = 0; t < layout->n_tensors; ++t)
            if (layout->numel[t] >= ((int64_t)1 << 32))
                return fail(MP_E_UNSUPPORTED, "the tensor-level plan needs tensors of fewer than 2^32 elements");
    const int64_t need = static_plan_bytes(layout->n_tensors, G, n_short, K);
    if (need > static_plan_limit())
        return fail(MP_E_UNSUPPORTED,
                    "the layout (%d tensors, %lld blocks, K = %d) needs %lld bytes of the fixed plan scratch, "
                    "whose size is %lld bytes; use mp_plan", layout->n_tensors, (long long)G, K,
                    (long long)need, (long long)static_plan_limit());
    Coeffs cw{};
    for (int i = 0; i < K; ++i) {
        if (!std::isfinite(w[i]))
            return fail(MP_E_ARG, "w[%d] is not finite", i);
        cw.v[i] = w[i];
    }
    if (sumsq != nullptr && (rc = check_device_buffer(sumsq, sizeof(float) * (size_t)(G * K), "sumsq")))
        return rc;
    if ((rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)G, "mask")))
        return rc;
    void* ws = nullptr;
    hipError_t e = static_plan_scratch(&ws);
    if (e != hipSuccess)
        return hip_fail(e, "address of the fixed plan scratch");
    const uint64_t full = (uint64_t)P * (uint64_t)es * (uint64_t)K;
    uint64_t h[7] = {0, 0, 0, 0, 0, 0, 0};
    e = launch_plan_static(ws, layout->numel, layout->n_tensors, layout->block_elems, (uint32_t)es, G, n_short, K,
                           sumsq, cw, flags, budget_bytes, full, mask, h, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return hip_fail(e, "plan (fixed scratch)");
    stats->budget_bytes = h[0];
    stats->cost_bytes = h[1];
    stats->full_bytes = h[2];
    stats->n_selected = h[3];
    stats->n_units = h[4];
    stats->digest = h[5];
    if (h[6] != 0)
        return fail(MP_E_HIP, "plan kernels reported internal error %llu", (unsigned long long)h[6]);
    if (stats->cost_bytes > budget_bytes)
        return fail(MP_E_HIP, "plan cost %llu exceeds the budget %llu", (unsigned long long)stats->cost_bytes,
                    (unsigned long long)budget_bytes);
    return MP_OK;
}

static int merge_additive(Op op, const mp_layout* layout, const void* base, const void* const* experts,
                          int32_t K, int32_t residency, const uint32_t* mask, const float* alpha, void* out,
                          mp_io_stats* io, void* stream)
{
    MergeArgs a;
    a.op = op;
    if (alpha == nullptr)
        return fail(MP_E_ARG, "alpha is NULL");
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    for (int i = 0; i < K; ++i) {
        if (!std::isfinite(alpha[i]))
            return fail(MP_E_ARG, "alpha[%d] is not finite", i);
        a.alpha.v[i] = alpha[i];
    }
    return run_merge(layout, base, experts, K, residency, mask, out, io, static_cast<hipStream_t>(stream), a);
}

int mp_merge_avg(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                 int32_t residency, const uint32_t* mask, const float* alpha, void* out,
                 mp_io_stats* io, void* stream)
{
    return merge_additive(Op::AVG, layout, base, experts, K, residency, mask, alpha, out, io, stream);
}

int mp_merge_avg_renorm(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                        int32_t residency, const uint32_t* mask, const float* alpha, void* out,
                        mp_io_stats* io, void* stream)
{
    return merge_additive(Op::AVG_RENORM, layout, base, experts, K, residency, mask, alpha, out, io, stream);
}

int mp_merge_ties(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                  int32_t residency, const uint32_t* mask, double density, float lambda, void* out,
                  mp_io_stats* io, void* stream)
{
    if (!(density >= 0.0 && density <= 1.0))
        return fail(MP_E_ARG, "density %g must be in [0, 1]", density);
    if (!std::isfinite(lambda))
        return fail(MP_E_ARG, "lambda is not finite");
    MergeArgs a;
    a.op = Op::TIES;
    a.density = density;
    a.lambda = lambda;
    return run_merge(layout, base, experts, K, residency, mask, out, io, static_cast<hipStream_t>(stream), a);
}

int mp_merge_ties_tau(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                      int32_t residency, const uint32_t* mask, const uint32_t* tau, float lambda, void* out,
                      mp_io_stats* io, void* stream)
{
    if (!std::isfinite(lambda))
        return fail(MP_E_ARG, "lambda is not finite");
    MergeArgs a;
    a.op = Op::TIES_TAU;
    a.lambda = lambda;
    a.tau = tau;
    return run_merge(layout, base, experts, K, residency, mask, out, io, static_cast<hipStream_t>(stream), a);
}

int mp_merge_dare(const mp_layout* layout, const void* base, const void* const* experts, int32_t K,
                  int32_t residency, const uint32_t* mask, double p, uint32_t seed, int32_t combine,
                  const float* alpha, float lambda, void* out, mp_io_stats* io, void* stream)
{
    if (!(p >= 0.0 && p < 1.0))
        return fail(MP_E_ARG, "p %g must be in [0, 1)", p);
    if (!std::isfinite(lambda))
        return fail(MP_E_ARG, "lambda is not finite");
    if (combine != MP_COMBINE_LINEAR && combine != MP_COMBINE_SIGN_ELECT)
        return fail(MP_E_ARG, "combine %d is not MP_COMBINE_LINEAR or MP_COMBINE_SIGN_ELECT", combine);
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    MergeArgs a;
    a.op = combine == MP_COMBINE_LINEAR ? Op::DARE_LINEAR : Op::DARE_SIGN;
    a.p = p;
    a.seed = seed;
    a.lambda = lambda;
    if (combine == MP_COMBINE_LINEAR) {
        if (alpha == nullptr)
            return fail(MP_E_ARG, "alpha is NULL");
        for (int i = 0; i < K; ++i) {
            if (!std::isfinite(alpha[i]))
                return fail(MP_E_ARG, "alpha[%d] is not finite", i);
            a.alpha.v[i] = alpha[i];
        }
    }
    return run_merge(layout, base, experts, K, residency, mask, out, io, static_cast<hipStream_t>(stream), a);
}

// Validates the adapter records against a validated layout (host only).
// *need receives the elements every adapter buffer must hold.
static int validate_loras(const mp_layout* L, const mp_lora_tensor* loras, int32_t n_lora, int64_t* need)
{
    if (n_lora < 0 || (n_lora > 0 && loras == nullptr))
        return fail(MP_E_ARG, "n_lora = %d with loras %s", n_lora, loras ? "set" : "NULL");
    if (n_lora > L->n_tensors)
        return fail(MP_E_ARG, "n_lora = %d exceeds the layout's %d tensors", n_lora, L->n_tensors);
    std::vector<char> adapted((size_t)L->n_tensors, 0);
    *need = 0;
    for (int32_t r = 0; r < n_lora; ++r) {
        const mp_lora_tensor& x = loras[r];
        if (x.tensor < 0 || x.tensor >= L->n_tensors)
            return fail(MP_E_ARG, "loras[%d].tensor = %d is not a tensor of the layout", r, x.tensor);
        if (adapted[(size_t)x.tensor])
            return fail(MP_E_ARG, "loras[%d]: tensor %d has two adapters", r, x.tensor);
        adapted[(size_t)x.tensor] = 1;
        if (x.rank < 1 || x.rank > kMaxLoraRank)
            return fail(MP_E_ARG, "loras[%d].rank = %d must be in [1, %d]", r, x.rank, kMaxLoraRank);
        const int64_t n = L->numel[x.tensor];
        // rows * cols == n without forming the product (no overflow)
        if (x.rows < 1 || x.cols < 1 || x.cols % 4 != 0 || n % x.rows != 0 || n / x.rows != x.cols)
            return fail(MP_E_ARG, "loras[%d]: %lld x %lld does not shape tensor %d (%lld elements; cols a multiple of 4)",
                        r, (long long)x.rows, (long long)x.cols, x.tensor, (long long)n);
        if (n >= ((int64_t)1 << 32))
            return fail(MP_E_UNSUPPORTED, "loras[%d]: tensor %d has 2^32 or more elements", r, x.tensor);
        if (x.a_off < 0 || x.b_off < 0 || x.a_off > ((int64_t)1 << 48) || x.b_off > ((int64_t)1 << 48) ||
            !std::isfinite(x.scale))
            return fail(MP_E_ARG, "loras[%d]: offset outside [0, 2^48] or non-finite scale", r);
        *need = std::max(*need, std::max(x.a_off + (int64_t)x.rank * x.cols, x.b_off + x.rows * (int64_t)x.rank));
    }
    return MP_OK;
}

// Looks up or builds the device table of validated adapter records.
static int get_lora_table(const mp_layout* L, const BlockTable& bt, const mp_lora_tensor* loras, int32_t n_lora,
                          LoraTable** out)
{
    std::vector<int64_t> toff((size_t)L->n_tensors + 1, 0), tg0((size_t)L->n_tensors + 1, 0);
    for (int32_t t = 0; t < L->n_tensors; ++t) {
        toff[(size_t)t + 1] = toff[(size_t)t] + L->numel[t];
        tg0[(size_t)t + 1] = tg0[(size_t)t] + (L->numel[t] + L->block_elems - 1) / L->block_elems;
    }
    std::vector<char> adapted((size_t)L->n_tensors, 0);
    for (int32_t r = 0; r < n_lora; ++r)
        adapted[(size_t)loras[r].tensor] = 1;
    std::string key = layout_key(bt.device, L);
    for (int32_t r = 0; r < n_lora; ++r) {  // field by field: the struct's padding bytes are not part of it
        const mp_lora_tensor& x = loras[r];
        uint32_t sc = 0;
        std::memcpy(&sc, &x.scale, sizeof sc);
        const int64_t f[7] = {x.tensor, x.rank, x.rows, x.cols, x.a_off, x.b_off, (int64_t)sc};
        key.append(reinterpret_cast<const char*>(f), sizeof f);
    }
    auto it = g_loras.find(key);
    if (it != g_loras.end()) {
        *out = &it->second->t;
        return MP_OK;
    }
    auto e = std::make_unique<LoraEntry>();
    e->device = bt.device;
    std::vector<LoraDesc> desc;
    uint64_t tiles = 0;
    for (int32_t r = 0; r < n_lora; ++r) {  // descriptors in layout order
        const mp_lora_tensor& x = loras[r];
        LoraDesc d{};
        d.toff = (uint64_t)toff[(size_t)x.tensor];
        d.a_off = (uint64_t)x.a_off;
        d.b_off = (uint64_t)x.b_off;
        d.rows = (uint32_t)x.rows;
        d.cols = (uint32_t)x.cols;
        d.rank = (uint32_t)x.rank;
        d.scale = x.scale;
        d.g0 = (uint32_t)tg0[(size_t)x.tensor];
        desc.push_back(d);
    }
    std::sort(desc.begin(), desc.end(), [](const LoraDesc& a, const LoraDesc& b) { return a.toff < b.toff; });
    uint64_t rows_total = 0;
    for (LoraDesc& d : desc) {
        d.r0 = (uint32_t)rows_total;
        rows_total += d.rows;
        if (rows_total >= ((uint64_t)1 << 31))
            return fail(MP_E_UNSUPPORTED, "adapted tensors hold 2^31 or more rows");
        d.tile0 = (uint32_t)tiles;
        tiles += lora_bands(d.rows, d.cols, &d.tiles_n);
        if (tiles >= ((uint64_t)1 << 31))
            return fail(MP_E_UNSUPPORTED, "adapted tensors need 2^31 or more row bands");
        const uint64_t cv = 16 / (uint64_t)bt.esize;  // elements per 16 bytes
        d.vec = (d.a_off % cv == 0 && d.cols % cv == 0) ? 1u : 0u;
        e->t.max_rank = std::max(e->t.max_rank, d.rank);
        e->t.max_cols = std::max(e->t.max_cols, d.cols);
        if (d.cols % cv != 0)
            e->t.rows_chunked = false;
    }
    // the fused merge's operand-order copy of one expert: per tensor A^T
    // (columns padded to 64) then B (rows padded to 16), prep_rank values each
    e->t.prep_rank = e->t.max_rank <= 16 ? 16u : (uint32_t)kMaxLoraRank;
    uint64_t prep = 0;
    for (LoraDesc& d : desc) {
        const uint64_t z = std::max((uint64_t)(d.cols + 63) / 64 * 64, (uint64_t)(d.rows + 15) / 16 * 16);
        e->t.prep_z = std::max(e->t.prep_z, (uint32_t)((z + 127) / 128));
        d.at_off = prep;
        prep += (uint64_t)(d.cols + 63) / 64 * 64 * e->t.prep_rank;
        d.bp_off = prep;
        prep += (uint64_t)(d.rows + 15) / 16 * 16 * e->t.prep_rank;
    }
    e->t.prep_elems = prep;
    std::vector<uint32_t> zero;
    for (int32_t t = 0; t < L->n_tensors; ++t)
        if (!adapted[(size_t)t])
            for (int64_t g = tg0[(size_t)t]; g < tg0[(size_t)t + 1]; ++g)
                zero.push_back((uint32_t)g);
    e->t.n_desc = (int)desc.size();
    e->t.n_tiles = (uint32_t)tiles;
    e->t.rows_total = (uint32_t)rows_total;
    e->t.n_zero = (uint32_t)zero.size();
    hipError_t he = hipSuccess;
    if ((!desc.empty() && ((he = ws_malloc((void**)&e->t.d_desc, sizeof(LoraDesc) * desc.size())) != hipSuccess ||
                           (he = hipMemcpy(e->t.d_desc, desc.data(), sizeof(LoraDesc) * desc.size(),
                                           hipMemcpyHostToDevice)) != hipSuccess)) ||
        (!zero.empty() && ((he = ws_malloc((void**)&e->t.d_zero, sizeof(uint32_t) * zero.size())) != hipSuccess ||
                           (he = hipMemcpy(e->t.d_zero, zero.data(), sizeof(uint32_t) * zero.size(),
                                           hipMemcpyHostToDevice)) != hipSuccess))) {
        free_lora(*e);
        return fail(MP_E_NOMEM, "adapter table: %s", hipGetErrorString(he));
    }
    *out = &e->t;
    g_loras.emplace(key, std::move(e));
    return MP_OK;
}

// The operand-order copies of a record table for K experts (grown on
// demand), with `s` ordered after the previous call that used the table's
// scratch (on any stream); the caller records lt->ev after its launches.
static int lora_prep(LoraTable* lt, int K, int es, hipStream_t s, OutPtrs* prep)
{
    hipError_t e;
    if (lt->ev == nullptr && (e = hipEventCreateWithFlags(&lt->ev, hipEventDisableTiming)) != hipSuccess)
        return hip_fail(e, "hipEventCreateWithFlags");
    if (lt->prep_k < K) {
        if (lt->d_prep != nullptr && (e = hipEventSynchronize(lt->ev)) != hipSuccess)
            return hip_fail(e, "hipEventSynchronize");
        (void)ws_free_r(lt->d_prep);
        lt->d_prep = nullptr;
        lt->prep_k = 0;
        if ((e = ws_malloc(&lt->d_prep, (size_t)K * lt->prep_elems * (size_t)es)) != hipSuccess)
            return fail(MP_E_NOMEM, "adapter operand copies (%zu bytes): %s",
                        (size_t)K * lt->prep_elems * (size_t)es, hipGetErrorString(e));
        lt->prep_k = K;
    }
    for (int i = 0; i < K; ++i)
        prep->p[i] = static_cast<char*>(lt->d_prep) + (size_t)i * lt->prep_elems * (size_t)es;
    if ((e = hipStreamWaitEvent(s, lt->ev, 0)) != hipSuccess)
        return hip_fail(e, "hipStreamWaitEvent");
    return MP_OK;
}

int mp_lora_materialize(const mp_layout* layout, const mp_lora_tensor* loras, int32_t n_lora,
                        const void* const* adapters, int32_t K, const uint32_t* mask, void* const* deltas,
                        void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    int es = 0;
    int rc = validate_layout(layout, &es);
    if (rc)
        return rc;
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    if ((n_lora > 0 && adapters == nullptr) || deltas == nullptr)
        return fail(MP_E_ARG, "adapters or deltas is NULL");
    const int64_t G = count_blocks(layout);
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return fail(MP_E_ARG, "K * G = %lld does not fit 32-bit unit ids", (long long)(G * K));
    int64_t need = 0;
    if ((rc = validate_loras(layout, loras, n_lora, &need)))
        return rc;
    BlockTable* bt = nullptr;
    LoraTable* lt = nullptr;
    if ((rc = get_table(layout, es, &bt)) || (rc = get_lora_table(layout, *bt, loras, n_lora, &lt)))
        return rc;
    const size_t ckpt = (size_t)bt->P * (size_t)es;
    std::vector<Range> ins, outs;
    ExpertPtrs ad{};
    OutPtrs dl{};
    for (int i = 0; i < K; ++i) {
        char nm[32];
        std::snprintf(nm, sizeof nm, "adapters[%d]", i);
        if (n_lora > 0) {
            if ((rc = check_device_buffer(adapters[i], (size_t)need * (size_t)es, nm)))
                return rc;
            ins.push_back({static_cast<const char*>(adapters[i]), (size_t)need * (size_t)es, "an adapter"});
        }
        ad.p[i] = n_lora > 0 ? adapters[i] : nullptr;
        std::snprintf(nm, sizeof nm, "deltas[%d]", i);
        if ((rc = check_device_buffer(deltas[i], ckpt, nm)))
            return rc;
        const Range o{static_cast<const char*>(deltas[i]), ckpt, "deltas"};
        for (const Range& r : ins)
            if (overlaps(o, r))
                return fail(MP_E_ARG, "deltas[%d] overlaps %s", i, r.name);
        for (const Range& r : outs)
            if (overlaps(o, r))
                return fail(MP_E_ARG, "deltas[%d] overlaps another delta buffer", i);
        outs.push_back(o);
        dl.p[i] = deltas[i];
    }
    for (const Range& o : outs)
        for (const Range& r : ins)
            if (overlaps(o, r))
                return fail(MP_E_ARG, "a delta buffer overlaps %s", r.name);
    if (mask != nullptr && (rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)G, "mask")))
        return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    // with every adapted tensor's rows whole 16-byte chunks the pull runs on
    // the operand-order copy (the table's scratch); otherwise masked pulls
    // use row lists (scratch too); either way ordered across streams
    const bool prepped = lt->n_tiles > 0 && lt->rows_chunked;
    const bool listed = mask != nullptr && lt->n_tiles > 0 && !prepped;
    if (listed) {
        // the row lists of a masked pull; calls with the same layout and
        // records share them, so each call's stream first waits for the
        // previous masked pull's kernels (on any stream)
        if (lt->ev == nullptr && (e = hipEventCreateWithFlags(&lt->ev, hipEventDisableTiming)) != hipSuccess)
            return hip_fail(e, "hipEventCreateWithFlags");
        if (lt->rl_k < K) {
            if (lt->d_rl != nullptr && (e = hipEventSynchronize(lt->ev)) != hipSuccess)  // its last reader is done
                return hip_fail(e, "hipEventSynchronize");
            (void)ws_free_r(lt->d_rl);
            (void)ws_free_r(lt->d_rc);
            lt->d_rl = nullptr;
            lt->d_rc = nullptr;
            lt->rl_k = 0;
            if ((e = ws_malloc((void**)&lt->d_rl, sizeof(uint32_t) * (size_t)K * lt->rows_total)) != hipSuccess ||
                (e = ws_malloc((void**)&lt->d_rc, sizeof(uint32_t) * (size_t)K * (size_t)lt->n_desc)) != hipSuccess)
                return fail(MP_E_NOMEM, "adapter row lists: %s", hipGetErrorString(e));
            lt->rl_k = K;
        }
        if ((e = hipStreamWaitEvent(s, lt->ev, 0)) != hipSuccess)
            return hip_fail(e, "hipStreamWaitEvent");
    }
    OutPtrs prep{};
    if (prepped && (rc = lora_prep(lt, K, es, s, &prep)))
        return rc;
    e = launch_lora(*bt, *lt, ad, dl, K, mask, s, prepped ? &prep : nullptr);
    if (e == hipSuccess && (listed || prepped))
        e = hipEventRecord(lt->ev, s);
    if (e != hipSuccess)
        return hip_fail(e, "adapter delta launch");
    return MP_OK;
}

int mp_lora_merge_ties_tau(const mp_layout* layout, const void* base, const mp_lora_tensor* loras, int32_t n_lora,
                           const void* const* adapters, int32_t K, const uint32_t* mask, const uint32_t* tau,
                           float lambda, void* out, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    int es = 0;
    int rc = validate_layout(layout, &es);
    if (rc)
        return rc;
    if (K < 1 || K > kMaxK)
        return fail(MP_E_ARG, "K = %d must be in [1, 32]", K);
    if (!std::isfinite(lambda))
        return fail(MP_E_ARG, "lambda is not finite");
    if (n_lora > 0 && adapters == nullptr)
        return fail(MP_E_ARG, "adapters is NULL");
    const int64_t G = count_blocks(layout);
    if ((uint64_t)G * (uint64_t)K >= (1ull << 32))
        return fail(MP_E_ARG, "K * G = %lld does not fit 32-bit unit ids", (long long)(G * K));
    int64_t need = 0;
    if ((rc = validate_loras(layout, loras, n_lora, &need)))
        return rc;
    BlockTable* bt = nullptr;
    LoraTable* lt = nullptr;
    if ((rc = get_table(layout, es, &bt)) || (rc = get_lora_table(layout, *bt, loras, n_lora, &lt)))
        return rc;
    if (!lt->rows_chunked)
        return fail(MP_E_UNSUPPORTED, "an adapted tensor's rows are not a whole number of 16-byte chunks "
                                      "(bf16 needs a multiple of 8 columns)");
    if ((uint64_t)16 * lt->max_cols * (uint64_t)es >= ((uint64_t)1 << 31))
        return fail(MP_E_UNSUPPORTED, "an adapted tensor has %u columns: 16 rows exceed 2 GiB", lt->max_cols);
    const size_t ckpt = (size_t)bt->P * (size_t)es;
    std::vector<Range> ins;
    if ((rc = check_device_buffer(base, ckpt, "base")))
        return rc;
    ins.push_back({static_cast<const char*>(base), ckpt, "base"});
    ExpertPtrs ad{};
    for (int i = 0; i < K && n_lora > 0; ++i) {
        char nm[32];
        std::snprintf(nm, sizeof nm, "adapters[%d]", i);
        if ((rc = check_device_buffer(adapters[i], (size_t)need * (size_t)es, nm)))
            return rc;
        ins.push_back({static_cast<const char*>(adapters[i]), (size_t)need * (size_t)es, "an adapter"});
        ad.p[i] = adapters[i];
    }
    if ((rc = check_device_buffer(mask, sizeof(uint32_t) * (size_t)G, "mask")) ||
        (rc = check_device_buffer(tau, sizeof(uint32_t) * (size_t)(G * K), "tau")) ||
        (rc = check_device_buffer(out, ckpt, "out")))
        return rc;
    ins.push_back({reinterpret_cast<const char*>(mask), sizeof(uint32_t) * (size_t)G, "mask"});
    ins.push_back({reinterpret_cast<const char*>(tau), sizeof(uint32_t) * (size_t)(G * K), "tau"});
    const Range o{static_cast<const char*>(out), ckpt, "out"};
    for (const Range& r : ins)
        if (overlaps(o, r))
            return fail(MP_E_ARG, "out overlaps %s", r.name);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    OutPtrs prep{};
    // the operand-order copies belong to the table: calls with the same
    // layout and records run one after the other, on whatever streams
    if (lt->n_tiles > 0 && (rc = lora_prep(lt, K, es, s, &prep)))
        return rc;
    e = launch_lora_ties(*bt, *lt, ad, prep, K, base, mask, tau, lambda, out, s);
    if (e == hipSuccess && lt->n_tiles > 0)
        e = hipEventRecord(lt->ev, s);
    if (e != hipSuccess)
        return hip_fail(e, "adapter TIES merge launch");
    return MP_OK;
}

const char* mp_last_error(void) { return g_err.c_str(); }

int mp_set_workspace_limit(uint64_t bytes)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    g_ws_limit = bytes;
    return MP_OK;
}

uint64_t mp_workspace_bytes(void)
{
    std::lock_guard<std::mutex> lock(g_mu);
    return g_ws_held;
}

int mp_stream_copy(const void* src, void* dst, uint64_t bytes, void* stream)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    if (bytes % 16 != 0)
        return fail(MP_E_ARG, "bytes = %llu must be a multiple of 16", (unsigned long long)bytes);
    if (bytes > (uint64_t(1) << 40))
        return fail(MP_E_ARG, "bytes = %llu exceeds 2^40", (unsigned long long)bytes);
    int rc;
    if ((rc = check_device_buffer(src, (size_t)bytes, "src")) || (rc = check_device_buffer(dst, (size_t)bytes, "dst")))
        return rc;
    const char* a = static_cast<const char*>(src);
    const char* b = static_cast<const char*>(dst);
    if (bytes != 0 && a < b + bytes && b < a + bytes)
        return fail(MP_E_ARG, "src and dst overlap");
    hipError_t e = launch_stream_copy(src, dst, bytes, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return hip_fail(e, "stream copy launch");
    return MP_OK;
}

int mp_set_stage_bytes(uint64_t bytes)
{
    std::lock_guard<std::mutex> lock(g_mu);
    g_err.clear();
    if (bytes < (uint64_t(1) << 20) || bytes > (uint64_t(4) << 30))
        return fail(MP_E_ARG, "staging size %llu must be in [1 MiB, 4 GiB]", (unsigned long long)bytes);
    set_stage_bytes((size_t)(bytes & ~uint64_t(255)));
    return MP_OK;
}

void mp_release(void)
{
    std::lock_guard<std::mutex> lock(g_mu);
    release_stagers();
    for (auto& kv : g_tables)
        free_table(*kv.second);
    g_tables.clear();
    for (auto& kv : g_loras)
        free_lora(*kv.second);
    g_loras.clear();
    for (auto& kv : g_ws)
        free_ws(kv.first, *kv.second);
    g_ws.clear();
}

}  // extern "C"
