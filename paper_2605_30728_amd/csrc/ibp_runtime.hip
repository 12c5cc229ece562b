// Device runtime of the library: handles, metadata upload, the PCIe staging pipeline
// and the C ABI entry points that enqueue the decompression kernels.
//
// Data layout in device memory (per handle):
//   d_meta    n_groups * 2 * row_bytes  Mask then Bitval per group, as in the stream
//   d_index   (n_groups + 1) u64        payload byte offset of every group (participation
//                                       scheme: (n_rows + 1) u64, of every row)
//   d_payload payload_bytes + slack     packed rows (IBP_OPEN_PAYLOAD_DEVICE only; with
//                                       IBP_OPEN_PAYLOAD_HOST_ZERO_COPY the kernels read
//                                       the pinned host copy through its device address;
//                                       with ..._ALIGNED that copy holds every row on a
//                                       128-byte boundary and d_index its offsets). The
//                                       device and zero-copy copies of a clustered stream
//                                       whose rows are mostly whole 128-byte lines start
//                                       every cluster on a line (line_aligned_clusters),
//                                       d_index then holding those offsets
// The kernels read a word's 64-bit window as two dwords at its bit offset, so every
// payload buffer the kernels see (device payload or staging) has kSlack readable bytes
// past its last packed byte.
//
// PCIe path (IBP_OPEN_PAYLOAD_HOST): the packed payload lives in library-owned pinned
// host memory. kStages device staging buffers rotate; for chunk k the side copy stream
// first waits until the kernel that last read buffer k%kStages has finished, copies the
// chunk in, and records an event that the caller's stream waits on before the decode
// kernel (the paper overlaps CPU memory reads with decoding, Sec. 4.3; here the overlap
// is between DMA of chunk k+1 and decode of chunk k). For gathers the host first packs
// the selected packed rows, their clusters and staged offsets into pinned staging
// (multi-threaded), which is the host half of the paper's lookup + transfer.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <functional>
#include <mutex>
#include <new>
#include <thread>
#include <unordered_map>
#include <utility>
#include <vector>

#include <hip/hip_runtime.h>

#include "ibp_device.hpp"
#include "ibp_internal.hpp"

namespace ibp {
namespace {

constexpr uint64_t kSlack = 256;                 // readable bytes past any payload end
constexpr uint64_t kStageBytes = 128ull << 20;   // one staging buffer (a whole compressed 128 MiB
                                                  // KV layer in one copy: 0.98 of CR x raw H2D,
                                                  // against 0.85 in two 64 MiB copies)
constexpr int kStages = 3;                        // staging buffers in rotation
constexpr int kIdSlots = 2;                       // host-id buffers in rotation
constexpr uint64_t kRowAlign = 128;               // PCIe line: row start of aligned zero-copy
constexpr uint64_t kMaxRuns = 4096;               // copy pieces of a line-aligned cluster layout
constexpr uint64_t kCountBytes = dev::kCountLines * dev::kCountStride * 8;   // cache counters
constexpr uint64_t kBlk = 256;                    // rows per host packing task (a chunk
                                                  // holds tens of them, for 16 threads)

// the host builds the compact metadata slots that the kernels read: one layout
static_assert(meta_slot_bytes(8, 1) == dev::meta_slot_bytes(8, 1) && meta_slot_bytes(8, 2) == dev::meta_slot_bytes(8, 2) &&
                  meta_slot_bytes(16, 4) == dev::meta_slot_bytes(16, 4) &&
                  meta_slot_bytes(16, 8) == dev::meta_slot_bytes(16, 8),
              "slot size");

uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Best-effort calls (cleanup, device restore) whose status is deliberately ignored.
inline void ignore(hipError_t) {}

// Host wait for an event by polling: the staging pipeline waits for copies that are
// normally about to finish, and polling resumes within microseconds where a blocking
// synchronize can sleep much longer.
hipError_t wait_event(hipEvent_t e) {
    for (;;) {
        const hipError_t r = hipEventQuery(e);
        if (r != hipErrorNotReady) return r;
        std::this_thread::yield();
    }
}

// Every device and pinned host allocation of the library goes through these, which keep
// the byte counts that ibp_memory_usage reports and honour the allocation test hook.
std::mutex g_mem_mu;
std::unordered_map<void *, std::pair<uint64_t, bool>> g_mem;   // address -> (bytes, pinned)
uint64_t g_dev_bytes = 0, g_pin_bytes = 0;

bool track(void *p, uint64_t bytes, bool pinned) {
    std::lock_guard<std::mutex> lock(g_mem_mu);
    try {
        g_mem.emplace(p, std::make_pair(bytes, pinned));
    } catch (...) {
        return false;
    }
    (pinned ? g_pin_bytes : g_dev_bytes) += bytes;
    return true;
}

void untrack(void *p) {
    std::lock_guard<std::mutex> lock(g_mem_mu);
    auto it = g_mem.find(p);
    if (it == g_mem.end()) return;
    (it->second.second ? g_pin_bytes : g_dev_bytes) -= it->second.first;
    g_mem.erase(it);
}

template <class T>
hipError_t dev_alloc(T **p, uint64_t bytes) {
    *p = nullptr;
    if (alloc_fails()) return hipErrorOutOfMemory;
    void *q = nullptr;
    hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess) return e;
    if (!track(q, bytes, false)) {
        ignore(hipFree(q));
        return hipErrorOutOfMemory;
    }
    *p = static_cast<T *>(q);
    return hipSuccess;
}

template <class T>
hipError_t pinned_alloc(T **p, uint64_t bytes, unsigned flags = hipHostMallocDefault) {
    *p = nullptr;
    if (alloc_fails()) return hipErrorOutOfMemory;
    void *q = nullptr;
    hipError_t e = hipHostMalloc(&q, bytes, flags);
    if (e != hipSuccess) return e;
    if (!track(q, bytes, true)) {
        ignore(hipHostFree(q));
        return hipErrorOutOfMemory;
    }
    *p = static_cast<T *>(q);
    return hipSuccess;
}

void dev_free(const void *p) {
    if (!p) return;
    untrack(const_cast<void *>(p));
    ignore(hipFree(const_cast<void *>(p)));
}

void pinned_free(const void *p) {
    if (!p) return;
    untrack(const_cast<void *>(p));
    ignore(hipHostFree(const_cast<void *>(p)));
}

}  // namespace
}  // namespace ibp

// Fixed device scratch of the allocation-free host-id gather: the row ids of one call are
// copied here and the gather kernel reads them from here. One copy per device, held until
// the process ends; every call on a device shares it (calls that overlap on one device
// race). Host code never uses this name as an address: it uses the per-device pointer
// that hipGetSymbolAddress returns (scratch_on_device).
constexpr uint64_t kScratchIds = 4ull << 20;   // 4,194,304 ids = 32 MiB
static __device__ __align__(256) int64_t scratch[kScratchIds];

namespace ibp {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int64_t *g_scratch_ptr[kMaxDevices] = {};
hipError_t g_scratch_err[kMaxDevices] = {};
bool g_scratch_done[kMaxDevices] = {};

// Device address of `scratch` on `device`, resolved once per device with that device
// current (each device holds its own copy of the array at its own address).
hipError_t scratch_on_device(int device, int64_t **ptr) {
    *ptr = nullptr;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_done[device]) {
        void *p = nullptr;
        g_scratch_err[device] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_ptr[device] = g_scratch_err[device] == hipSuccess ? static_cast<int64_t *>(p) : nullptr;
        g_scratch_done[device] = true;
    }
    *ptr = g_scratch_ptr[device];
    return g_scratch_err[device];
}

}  // namespace
}  // namespace ibp

using namespace ibp;

struct ibp_handle {
    int device = 0;
    uint32_t flags = 0;
    ibp_desc d{};
    dev::DevStream ds{};
    uint32_t *d_meta = nullptr;
    uint8_t *d_slots = nullptr;           // compact metadata of the row gathers (clustered, W <= 512)
    uint8_t *d_row_lines = nullptr;       // line-packed row offsets (participation, rows <= 1092 B)
    uint64_t *d_index = nullptr;
    uint8_t *d_payload = nullptr;
    const uint8_t *k_payload = nullptr;   // what the kernels read: d_payload or the pinned host payload
    unsigned long long *d_err = nullptr;
    int64_t *scratch_ids = nullptr;       // this device's `scratch` (allocation-free gather)
    hipError_t scratch_err = hipSuccess;
    // host ids of gathers over a device or zero-copy payload: two slots alternate, so the
    // ids of call k+1 are staged while the kernel of call k still reads slot k%2
    int64_t *h_ids[kIdSlots] = {}, *d_ids[kIdSlots] = {};
    uint64_t ids_cap[kIdSlots] = {};
    hipEvent_t ev_ids_free[kIdSlots] = {};
    bool ids_used[kIdSlots] = {};
    int next_ids = 0;
    // PCIe path
    uint8_t *h_payload = nullptr;
    std::vector<uint64_t> h_off;    // the stream's index: per group, or per row (participation)
    std::vector<uint32_t> h_rb;     // clustered scheme: packed row bytes of every group
    uint32_t max_rb = 0;            // largest packed row
    uint8_t *h_stage[kStages] = {};
    uint8_t *d_stage[kStages] = {};
    hipStream_t copy_stream = nullptr;
    hipEvent_t ev_copied[kStages] = {};
    hipEvent_t ev_free[kStages] = {};
    bool stage_used[kStages] = {};
    int next_stage = 0;
    std::vector<uint32_t> req_g, req_rb;   // per-request cluster and packed size (host gathers)
    std::vector<uint64_t> req_src;         // payload byte of every request's packed row
    std::vector<uint64_t> blk_off;         // packed bytes of every packing block (host gathers)
    std::vector<uint64_t> chunk_off;       // staged byte offset of every block of one chunk
    Pool *pool = nullptr;
    // 0: free, 1: a call is running, 2: closed. A closed handle keeps this struct (its
    // resources are freed), so later calls on it, a second ibp_close included, find the
    // state and return IBP_ESTATE instead of touching freed memory.
    std::atomic<int> busy{0};
    int n_caches = 0;                      // live caches built on this handle
    ibp_stats stats{};
    hipError_t sticky = hipSuccess;
};

// A static compressed row cache on the device (Sec. 5, cache compression): cached rows'
// packed bytes back to back in one device slab, and an open-addressing table from row id
// to slab entry. Misses are decoded from the handle's pinned payload, read in place.
struct ibp_cache {
    ibp_handle *h = nullptr;
    uint8_t *d_slab = nullptr;
    void *d_table = nullptr;
    unsigned long long *d_counts = nullptr;
    dev::CacheView view{};
    uint64_t rows = 0, slab_bytes = 0, slots = 0;
    bool destroyed = false;   // kept as a marker after ibp_cache_destroy (under the handle's call)
};

namespace {

// Marks a handle busy for one call and makes its device current for the call.
class CallScope {
public:
    explicit CallScope(ibp_handle *h) : h_(h) {
        if (!h_) return;
        int expected = 0;
        ok_ = h_->busy.compare_exchange_strong(expected, 1);
        closed_ = !ok_ && expected == 2;
        if (ok_) {
            ignore(hipGetDevice(&prev_));
            if (prev_ != h_->device) ignore(hipSetDevice(h_->device));
        }
    }
    ~CallScope() {
        if (!ok_) return;
        if (prev_ != h_->device) ignore(hipSetDevice(prev_));
        h_->busy.store(0);
    }
    bool ok() const { return ok_; }
    bool closed() const { return closed_; }

private:
    ibp_handle *h_;
    bool ok_ = false;
    bool closed_ = false;
    int prev_ = -1;
};

ibp_status hip_fail(ibp_handle *h, hipError_t e, const char *what) {
    if (h && h->sticky == hipSuccess) h->sticky = e;
    return fail(IBP_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define IBP_HIP(h, call)                                  \
    do {                                                  \
        hipError_t e_ = (call);                           \
        if (e_ != hipSuccess) return hip_fail(h, e_, #call); \
    } while (0)

ibp_status check_handle(ibp_handle *h, const CallScope &cs) {
    if (!h) return fail(IBP_EINVAL, "handle is null");
    if (!cs.ok()) return fail(IBP_ESTATE, cs.closed() ? "handle is closed" : "handle is in use by another thread");
    if (h->sticky != hipSuccess)
        return fail(IBP_EHIP, std::string("earlier HIP error on this handle: ") + hipGetErrorString(h->sticky));
    return IBP_OK;
}

// Frees everything a handle owns except the struct itself.
void release_handle(ibp_handle *h) {
    dev_free(h->d_meta);
    dev_free(h->d_slots);
    dev_free(h->d_row_lines);
    dev_free(h->d_index);
    dev_free(h->d_payload);
    dev_free(h->d_err);
    h->d_meta = nullptr;
    h->d_slots = nullptr;
    h->d_row_lines = nullptr;
    h->d_index = nullptr;
    h->d_payload = nullptr;
    h->d_err = nullptr;
    h->k_payload = nullptr;
    for (int j = 0; j < kIdSlots; ++j) {
        dev_free(h->d_ids[j]);
        pinned_free(h->h_ids[j]);
        if (h->ev_ids_free[j]) ignore(hipEventDestroy(h->ev_ids_free[j]));
        h->d_ids[j] = nullptr;
        h->h_ids[j] = nullptr;
        h->ev_ids_free[j] = nullptr;
        h->ids_cap[j] = 0;
    }
    pinned_free(h->h_payload);
    h->h_payload = nullptr;
    for (int b = 0; b < kStages; ++b) {
        pinned_free(h->h_stage[b]);
        dev_free(h->d_stage[b]);
        if (h->ev_copied[b]) ignore(hipEventDestroy(h->ev_copied[b]));
        if (h->ev_free[b]) ignore(hipEventDestroy(h->ev_free[b]));
        h->h_stage[b] = nullptr;
        h->d_stage[b] = nullptr;
        h->ev_copied[b] = nullptr;
        h->ev_free[b] = nullptr;
    }
    if (h->copy_stream) ignore(hipStreamDestroy(h->copy_stream));
    h->copy_stream = nullptr;
    delete h->pool;
    h->pool = nullptr;
    std::vector<uint64_t>().swap(h->h_off);
    std::vector<uint32_t>().swap(h->h_rb);
    std::vector<uint32_t>().swap(h->req_g);
    std::vector<uint32_t>().swap(h->req_rb);
    std::vector<uint64_t>().swap(h->req_src);
    std::vector<uint64_t>().swap(h->blk_off);
    std::vector<uint64_t>().swap(h->chunk_off);
}

void free_handle(ibp_handle *h) {
    if (!h) return;
    release_handle(h);
    delete h;
}

// Claim id slot j for n ids: its last kernel must have finished with it (host wait, needed
// anyway before the pinned half is rewritten), and the buffers must hold n ids.
ibp_status claim_ids(ibp_handle *h, int j, uint64_t n) {
    if (h->ids_used[j]) IBP_HIP(h, wait_event(h->ev_ids_free[j]));
    if (n <= h->ids_cap[j]) return IBP_OK;
    uint64_t cap = std::max<uint64_t>(n, 2 * h->ids_cap[j]);
    pinned_free(h->h_ids[j]);
    dev_free(h->d_ids[j]);
    h->h_ids[j] = nullptr;
    h->d_ids[j] = nullptr;
    h->ids_cap[j] = 0;
    if (pinned_alloc(&h->h_ids[j], cap * 8) != hipSuccess)
        return fail(IBP_ENOMEM, "pinned allocation for row ids failed");
    if (dev_alloc(&h->d_ids[j], cap * 8) != hipSuccess) {
        pinned_free(h->h_ids[j]);      // a failed call holds nothing new
        h->h_ids[j] = nullptr;
        return fail(IBP_ENOMEM, "device allocation for row ids failed");
    }
    h->ids_cap[j] = cap;
    return IBP_OK;
}

// The host payload of the PCIe placements (IBP_OPEN_PAYLOAD_HOST, _ZERO_COPY) in pinned
// memory; `aoff`/`runs` (zero-copy only) give the line-aligned cluster layout, else the
// stream's own byte layout is kept.
ibp_status setup_host_path(ibp_handle *h, const StreamView &v, const std::vector<uint64_t> *aoff,
                           const std::vector<uint64_t> &runs) {
    const ibp_desc &d = h->d;
    const uint64_t bytes = aoff ? (*aoff)[d.n_groups] : d.payload_bytes;
    if (pinned_alloc(&h->h_payload, bytes + kSlack) != hipSuccess)
        return fail(IBP_ENOMEM, "pinned allocation for the payload failed");
    const uint8_t *src = v.payload();
    uint8_t *dst = h->h_payload;
    if (!aoff) {
        h->pool->run(d.payload_bytes, 64ull << 20, [&](uint64_t lo, uint64_t hi) {
            std::memcpy(dst + lo, src + lo, hi - lo);
        });
    } else {
        // each stretch in one piece (its bytes keep their order), then the padding between
        // stretches zeroed
        for (size_t k = 0; k + 1 < runs.size(); ++k) {
            const uint64_t g0 = runs[k], g1 = runs[k + 1];
            const uint64_t s0 = v.off(g0), n = v.off(g1) - s0, d0 = (*aoff)[g0];
            h->pool->run(n, 64ull << 20, [&](uint64_t lo, uint64_t hi) {
                std::memcpy(dst + d0 + lo, src + s0 + lo, hi - lo);
            });
            const uint64_t next = g1 < d.n_groups ? (*aoff)[g1] : d0 + n;
            std::memset(dst + d0 + n, 0, next - (d0 + n));
        }
    }
    std::memset(dst + bytes, 0, kSlack);
    check_alloc();
    if (d.flags & IBP_STREAM_PARTICIPATION) {
        h->h_off.resize(d.n_rows + 1);
        for (uint64_t r = 0; r <= d.n_rows; ++r) h->h_off[r] = v.off(r);
        h->max_rb = d.row_bytes;        // a raw row
    } else {
        h->h_off.resize(d.n_groups + 1);
        h->h_rb.resize(d.n_groups);
        for (uint64_t g = 0; g <= d.n_groups; ++g) h->h_off[g] = aoff ? (*aoff)[g] : v.off(g);
        for (uint64_t g = 0; g < d.n_groups; ++g) {
            h->h_rb[g] = (uint32_t)((v.off(g + 1) - v.off(g)) / v.rows_in_group(g));
            h->max_rb = std::max(h->max_rb, h->h_rb[g]);
        }
    }
    if (h->flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY) return IBP_OK;   // no staging: kernels read in place
    if (d.n_groups > 0xFFFFFFFFull) return fail(IBP_EINVAL, "too many clusters for the PCIe path");
    // a staged chunk holds at least one whole row with its tables (gathers) or one packed
    // row (ranges), so every call can make progress without overrunning a stage
    if ((uint64_t)d.row_bytes + 72 > kStageBytes)
        return fail(IBP_EINVAL, "rows larger than a staging buffer need another placement");
    for (int b = 0; b < kStages; ++b) {
        if (pinned_alloc(&h->h_stage[b], kStageBytes + kSlack) != hipSuccess)
            return fail(IBP_ENOMEM, "pinned allocation for staging failed");
        if (dev_alloc(&h->d_stage[b], kStageBytes + kSlack) != hipSuccess)
            return fail(IBP_ENOMEM, "device allocation for staging failed");
        IBP_HIP(h, hipMemset(h->d_stage[b], 0, kStageBytes + kSlack));
        IBP_HIP(h, hipEventCreateWithFlags(&h->ev_copied[b], hipEventDisableTiming));
        IBP_HIP(h, hipEventCreateWithFlags(&h->ev_free[b], hipEventDisableTiming));
    }
    IBP_HIP(h, hipStreamCreateWithFlags(&h->copy_stream, hipStreamNonBlocking));
    return IBP_OK;
}

// Zero-copy payload with aligned rows: in the pinned copy every packed row of cluster g
// starts on a kRowAlign boundary (row stride roundup(rb_g, kRowAlign), zero padding), and
// the device index is replaced by the offsets of this layout. A GPU read of a row then
// touches ceil(rb_g / 128) PCIe lines; a row at an arbitrary byte offset touches up to one
// more.
ibp_status setup_aligned_host_payload(ibp_handle *h, const StreamView &v) {
    const ibp_desc &d = h->d;
    const uint64_t ng = d.n_groups;
    check_alloc();
    std::vector<uint64_t> aoff(ng + 1), rbs(ng);
    aoff[0] = 0;
    for (uint64_t g = 0; g < ng; ++g) {
        const uint64_t n = v.rows_in_group(g);
        rbs[g] = (v.off(g + 1) - v.off(g)) / n;
        aoff[g + 1] = aoff[g] + n * ((rbs[g] + kRowAlign - 1) / kRowAlign * kRowAlign);
    }
    if (pinned_alloc(&h->h_payload, aoff[ng] + kSlack) != hipSuccess)
        return fail(IBP_ENOMEM, "pinned allocation for the aligned payload failed");
    const uint8_t *src = v.payload();
    uint8_t *dst = h->h_payload;
    h->pool->run(ng, 256, [&](uint64_t lo, uint64_t hi) {
        for (uint64_t g = lo; g < hi; ++g) {
            const uint64_t n = v.rows_in_group(g), rb = rbs[g];
            const uint64_t stride = (rb + kRowAlign - 1) / kRowAlign * kRowAlign;
            for (uint64_t r = 0; r < n; ++r) {
                uint8_t *o = dst + aoff[g] + r * stride;
                std::memcpy(o, src + v.off(g) + r * rb, rb);
                std::memset(o + rb, 0, stride - rb);
            }
        }
    });
    std::memset(dst + aoff[ng], 0, kSlack);
    IBP_HIP(h, hipMemcpy(h->d_index, aoff.data(), 8 * (ng + 1), hipMemcpyHostToDevice));
    return IBP_OK;
}

// Claim staging buffer b for a new chunk: the previous copy out of its pinned half must
// have finished (host wait), and the next copy into its device half must wait for the
// kernel that last read it (device wait on the copy stream).
ibp_status claim_stage(ibp_handle *h, int b, bool host_side_too) {
    if (h->stage_used[b]) {
        if (host_side_too) IBP_HIP(h, wait_event(h->ev_copied[b]));
        IBP_HIP(h, hipStreamWaitEvent(h->copy_stream, h->ev_free[b], 0));
    }
    return IBP_OK;
}

// PCIe gather: the host packs the requested packed rows into pinned staging chunk by
// chunk, rotating kStages buffers, so that packing chunk k+1 overlaps the DMA of chunk k
// and the decode of chunk k-1. A chunk's staging is [cluster of each request (u32) |
// staged byte offset of each request and the end of the last (u32, nc + 1 entries) |
// the packed rows, byte-packed].
ibp_status gather_host_payload(ibp_handle *h, const int64_t *ids, uint64_t n, uint8_t *d_out, hipStream_t s) {
    const uint64_t L = h->d.row_bytes, G = h->d.group_rows;
    const uint64_t magic = dev::div_magic((uint32_t)G);
    // rows per chunk: as many as one staging buffer holds (8 B of tables + the largest packed
    // row each), in whole packing blocks. Consecutive calls overlap through the rotating
    // buffers (call k+1 packs while call k's chunk crosses PCIe); cutting a call into
    // smaller chunks measured slower, since every chunk costs a DMA and a launch.
    const uint64_t row_max = 8 + (uint64_t)h->max_rb;
    const uint64_t cap_rows = std::max<uint64_t>(1, (kStageBytes - 64) / row_max);
    const uint64_t per_chunk = cap_rows >= kBlk ? cap_rows / kBlk * kBlk : cap_rows;
    const uint64_t blk = std::min(kBlk, per_chunk);   // per_chunk is a multiple of blk
    // one pass over the ids: cluster and packed size of every request, and the packed
    // bytes of every block
    const uint64_t nblk_all = (n + blk - 1) / blk;
    // every host table of the call is sized here, before anything is enqueued
    check_alloc();
    h->req_g.resize(n);
    h->req_rb.resize(n);
    h->req_src.resize(n);
    h->blk_off.assign(nblk_all + 1, 0);
    h->chunk_off.resize((per_chunk + blk - 1) / blk + 1);
    uint32_t *rg = h->req_g.data(), *rrb = h->req_rb.data();
    uint64_t *rsrc = h->req_src.data();
    uint64_t *bs = h->blk_off.data();
    const uint32_t *grb = h->h_rb.data();
    const uint64_t *hoff = h->h_off.data();
    const bool part = h->d.flags & IBP_STREAM_PARTICIPATION;
    // the range check of every id rides on this pass (no extra serial pass over the ids);
    // the first bad position is reported before anything is enqueued
    const uint64_t n_rows = h->d.n_rows;
    std::atomic<uint64_t> first_bad{n};
    // Every request reads its cluster's (or row's) offset and size at random places in
    // host tables of tens of MB: prefetch them a few requests ahead, so that the misses
    // overlap instead of following one another.
    auto prefetch_meta = [&](uint64_t i) {
        const uint64_t id = (uint64_t)ids[i];
        if (id >= n_rows) return;
        if (part) {
            __builtin_prefetch(hoff + id);
            __builtin_prefetch(hoff + id + 1);
        } else {
            const uint64_t g = G == 1 ? id : (uint64_t)(((unsigned __int128)id * magic) >> 64);
            __builtin_prefetch(hoff + g);
            __builtin_prefetch(grb + g);
        }
    };
    h->pool->run(nblk_all, 1, [&](uint64_t lo, uint64_t hi) {
        constexpr uint64_t kAhead = 16;   // requests prefetched ahead
        for (uint64_t k = lo; k < hi; ++k) {
            uint64_t sum = 0;
            const uint64_t a = k * blk, e = std::min(n, a + blk);
            for (uint64_t i = a; i < std::min(e, a + kAhead); ++i) prefetch_meta(i);
            for (uint64_t i = a; i < e; ++i) {
                if (i + kAhead < e) prefetch_meta(i + kAhead);
                const uint64_t id = (uint64_t)ids[i];
                if (id >= n_rows) {   // negative ids wrap to large values
                    uint64_t cur = first_bad.load(std::memory_order_relaxed);
                    while (i < cur && !first_bad.compare_exchange_weak(cur, i, std::memory_order_relaxed)) {
                    }
                    rg[i] = 0;
                    rsrc[i] = 0;
                    rrb[i] = 0;
                    continue;
                }
                const uint64_t g = G == 1 ? id : (uint64_t)(((unsigned __int128)id * magic) >> 64);
                rg[i] = (uint32_t)g;
                if (part) {
                    rsrc[i] = hoff[id];
                    rrb[i] = (uint32_t)(hoff[id + 1] - hoff[id]);
                } else {
                    rsrc[i] = hoff[g] + (id - g * G) * grb[g];
                    rrb[i] = grb[g];
                }
                sum += rrb[i];
            }
            bs[k + 1] = sum;
        }
    });
    if (const uint64_t i = first_bad.load(); i < n)
        return fail(IBP_ERANGE, "row id " + std::to_string(ids[i]) + " at position " + std::to_string(i) +
                                    " is outside [0, " + std::to_string(n_rows) + ")");
    for (uint64_t i0 = 0; i0 < n; i0 += per_chunk) {
        const uint64_t nc = std::min(per_chunk, n - i0);
        const int b = h->next_stage;
        h->next_stage = (h->next_stage + 1) % kStages;
        ibp_status st = claim_stage(h, b, true);
        if (st != IBP_OK) return st;
        auto t0 = std::chrono::steady_clock::now();
        uint8_t *stg = h->h_stage[b];
        uint32_t *sg = reinterpret_cast<uint32_t *>(stg);
        uint32_t *soff = sg + nc;
        const uint64_t tables = 8 * nc + 4;
        uint8_t *pay = stg + tables;
        // staged offsets: an exclusive scan over this chunk's block sums, then every block
        // writes its tables and copies its rows (prefetching a few rows ahead, since each
        // row is a random read of ~rb bytes from host memory)
        const uint64_t k0 = i0 / blk, nblk = (nc + blk - 1) / blk;
        uint64_t *bo = h->chunk_off.data();   // sized for a whole chunk's blocks above
        bo[0] = 0;
        for (uint64_t k = 0; k < nblk; ++k) bo[k + 1] = bo[k] + bs[k0 + k + 1];
        const uint64_t total_pay = bo[nblk];
        soff[nc] = (uint32_t)total_pay;
        // Every block packs its rows into a small thread-local buffer (cache resident), then
        // streams the buffer to the pinned staging with non-temporal 16-byte stores: the
        // staging lines are neither read for ownership nor left dirty in the CPU caches for
        // the DMA engine to snoop (measured on the GNN minibatch: packing 0.55 -> 0.39 ms per
        // call, the staged leg 0.81 -> 0.94 of CR x raw H2D). Only each block's first and
        // last partial 16 bytes take plain stores.
        const uint8_t *src_base = h->h_payload;
        h->pool->run(nblk, 1, [&](uint64_t lo, uint64_t hi) {
            constexpr uint64_t kAhead = 24;              // rows prefetched ahead (random host reads)
            constexpr uint64_t kMaxBuffered = 1u << 20;  // larger blocks (very wide rows) store directly
            thread_local std::vector<uint8_t> buf;
            bool streamed = false;
            for (uint64_t k = lo; k < hi; ++k) {
                const uint64_t a = i0 + k * blk, e = std::min(i0 + nc, a + blk), bytes = bo[k + 1] - bo[k];
                auto src_of = [&](uint64_t i) { return src_base + rsrc[i]; };
                for (uint64_t i = a; i < std::min(e, a + kAhead); ++i) {
                    const uint8_t *p = src_of(i);
                    for (uint32_t c = 0; c < rrb[i]; c += 64) __builtin_prefetch(p + c);
                }
                uint8_t *const dst = pay + bo[k];
                uint8_t *wr = dst;
                if (bytes > 0 && bytes <= kMaxBuffered) {
                    try {
                        if (buf.size() < bytes) buf.resize(bytes);
                        wr = buf.data();
                    } catch (...) {
                        wr = dst;   // no buffer: plain stores
                    }
                }
                uint64_t o = 0;
                for (uint64_t i = a; i < e; ++i) {
                    if (i + kAhead < e) {
                        const uint8_t *p = src_of(i + kAhead);
                        for (uint32_t c = 0; c < rrb[i + kAhead]; c += 64) __builtin_prefetch(p + c);
                    }
                    sg[i - i0] = rg[i];
                    soff[i - i0] = (uint32_t)(bo[k] + o);
                    std::memcpy(wr + o, src_of(i), rrb[i]);
                    o += rrb[i];
                }
                if (wr != dst) {
                    typedef long long v2 __attribute__((vector_size(16)));
                    const uint64_t head = std::min<uint64_t>(bytes, (16 - ((uintptr_t)dst & 15)) & 15);
                    std::memcpy(dst, wr, head);
                    uint64_t q = head;
                    for (; q + 16 <= bytes; q += 16) {
                        v2 v;
                        std::memcpy(&v, wr + q, 16);
                        __builtin_nontemporal_store(v, reinterpret_cast<v2 *>(dst + q));
                    }
                    std::memcpy(dst + q, wr + q, bytes - q);
                    streamed = true;
                }
            }
            // non-temporal stores are weakly ordered: make them visible before the pool
            // reports the work done (and the DMA is enqueued)
            if (streamed) std::atomic_thread_fence(std::memory_order_seq_cst);
        });
        h->stats.host_pack_ns +=
            (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0).count();
        const uint64_t total = tables + total_pay;
        IBP_HIP(h, hipMemcpyAsync(h->d_stage[b], stg, total, hipMemcpyHostToDevice, h->copy_stream));
        IBP_HIP(h, hipEventRecord(h->ev_copied[b], h->copy_stream));
        IBP_HIP(h, hipStreamWaitEvent(s, h->ev_copied[b], 0));
        const uint8_t *dst = h->d_stage[b];
        IBP_HIP(h, dev::launch_gather(h->ds, dst + tables, nullptr, reinterpret_cast<const uint32_t *>(dst),
                                      reinterpret_cast<const uint32_t *>(dst) + nc, nc, d_out + i0 * L, h->d_err, s));
        IBP_HIP(h, hipEventRecord(h->ev_free[b], s));
        h->stage_used[b] = true;
        h->stats.h2d_bytes += total;
        h->stats.h2d_payload_bytes += total_pay;
    }
    return IBP_OK;
}

}  // namespace

extern "C" {

}  // extern "C"

namespace {

// The body of ibp_open. `h` and `prev` are the caller's, so that it can also clean up after
// an exception: h is the handle being built (null once freed here), prev the device that
// was current before (-1 once restored here).
ibp_status open_impl(const void *stream, uint64_t stream_bytes, int device, uint32_t flags, ibp_handle **out,
                     ibp_handle *&h, int &prev) {
    if (!out) return fail(IBP_EINVAL, "handle output is null");
    *out = nullptr;
    if (flags != IBP_OPEN_PAYLOAD_DEVICE && flags != IBP_OPEN_PAYLOAD_HOST &&
        flags != IBP_OPEN_PAYLOAD_HOST_ZERO_COPY && flags != IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED)
        return fail(IBP_EINVAL, "unknown open flags");
    StreamView v;
    ibp_status st = parse_stream(stream, stream_bytes, v);
    if (st != IBP_OK) return st;
    const ibp_desc &d = v.d;
    if (flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED && d.flags != 0)
        return fail(IBP_EINVAL, "aligned rows need a clustered-scheme stream (flags = 0)");
    if (d.group_rows > 1 && d.n_rows > ~0ull / d.group_rows)
        return fail(IBP_EINVAL, "n_rows * group_rows must stay below 2^64");
    if (2ull * d.row_bytes * 8 > 0xFFFFFFFFull) return fail(IBP_EINVAL, "row_bytes too large");
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device < 0 || device >= count)
        return fail(IBP_EINVAL, "no such HIP device");
    int cur = 0;
    ignore(hipGetDevice(&cur));
    if (hipSetDevice(device) != hipSuccess) return fail(IBP_EHIP, "hipSetDevice failed");
    prev = cur;
    int64_t *scratch_ids = nullptr;
    const hipError_t scratch_err = scratch_on_device(device, &scratch_ids);

    auto bail = [&](ibp_status s) {
        free_handle(h);
        h = nullptr;
        ignore(hipSetDevice(prev));
        prev = -1;
        return s;
    };
    if (alloc_fails() || !(h = new (std::nothrow) ibp_handle())) return bail(fail(IBP_ENOMEM, "host allocation failed"));
    h->device = device;
    h->flags = flags;
    h->scratch_ids = scratch_ids;
    h->scratch_err = scratch_err;
    h->d = d;
    check_alloc();
    h->pool = new Pool(std::min(16, online_cpus()));
    const uint64_t meta_bytes = d.n_groups * 2ull * d.row_bytes;
    const uint64_t n_index = (d.flags & IBP_STREAM_PARTICIPATION) ? d.n_rows + 1 : d.n_groups + 1;
    if (dev_alloc(&h->d_meta, std::max<uint64_t>(meta_bytes, 4)) != hipSuccess ||
        dev_alloc(&h->d_index, 8 * n_index) != hipSuccess || dev_alloc(&h->d_err, 8) != hipSuccess)
        return bail(fail(IBP_ENOMEM, "device allocation for metadata failed"));
    if (meta_bytes && hipMemcpy(h->d_meta, v.meta(), meta_bytes, hipMemcpyHostToDevice) != hipSuccess)
        return bail(fail(IBP_EHIP, "metadata upload failed"));
    // the payload copies the kernels read in place (device, zero-copy) start every cluster
    // on a 128-byte line when that keeps rows on whole lines (line_aligned_clusters)
    std::vector<uint64_t> aoff, runs;
    const bool line_al = (flags == IBP_OPEN_PAYLOAD_DEVICE || flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY) &&
                         line_aligned_clusters(v, kRowAlign, kMaxRuns, aoff, runs);
    if (hipMemcpy(h->d_index, line_al ? static_cast<const void *>(aoff.data()) : v.index_bytes(), 8 * n_index,
                  hipMemcpyHostToDevice) != hipSuccess ||
        hipMemset(h->d_err, 0, 8) != hipSuccess)
        return bail(fail(IBP_EHIP, "index upload failed"));
    const uint32_t W = d.row_bytes / 4;
    if (d.flags == 0 && W <= 512) {
        // the row gathers read a cluster's metadata for every row they decode: when every
        // cluster fits one, give each a compact slot as well
        const uint32_t K = (uint32_t)dev::words_per_lane(W);
        check_alloc();
        std::vector<uint8_t> slots;
        const uint32_t P = build_meta_slots(v.meta(), d.n_groups, W, K, *h->pool, slots);
        if (P) {
            if (dev_alloc(&h->d_slots, slots.size()) != hipSuccess)
                return bail(fail(IBP_ENOMEM, "device allocation for metadata failed"));
            if (hipMemcpy(h->d_slots, slots.data(), slots.size(), hipMemcpyHostToDevice) != hipSuccess)
                return bail(fail(IBP_EHIP, "metadata upload failed"));
            h->ds.slot_pairs = P;
            h->ds.slot_bytes = (uint32_t)meta_slot_bytes(P, K);
        }
    }
    if ((d.flags & IBP_STREAM_PARTICIPATION) && d.n_rows > 0 && d.n_rows <= ~0ull / dev::kRowLineRows &&
        (uint64_t)d.row_bytes * dev::kRowLineRows <= 0xFFFF) {
        // every row is at most row_bytes long (validated), so a line's 60 row ends fit u16
        check_alloc();
        std::vector<uint8_t> lines;
        if (build_row_lines(v.index_bytes(), d.n_rows, dev::kRowLineRows, *h->pool, lines)) {
            if (dev_alloc(&h->d_row_lines, lines.size()) != hipSuccess)
                return bail(fail(IBP_ENOMEM, "device allocation for metadata failed"));
            if (hipMemcpy(h->d_row_lines, lines.data(), lines.size(), hipMemcpyHostToDevice) != hipSuccess)
                return bail(fail(IBP_EHIP, "metadata upload failed"));
        }
    }
    if (flags == IBP_OPEN_PAYLOAD_DEVICE) {
        const uint64_t used = line_al ? aoff[d.n_groups] : d.payload_bytes;
        const uint64_t bytes = round_up(used + kSlack, 256);
        if (dev_alloc(&h->d_payload, bytes) != hipSuccess)
            return bail(fail(IBP_ENOMEM, "device allocation for the payload failed"));
        if (!line_al) {
            if (hipMemset(h->d_payload + d.payload_bytes, 0, bytes - d.payload_bytes) != hipSuccess ||
                (d.payload_bytes &&
                 hipMemcpy(h->d_payload, v.payload(), d.payload_bytes, hipMemcpyHostToDevice) != hipSuccess))
                return bail(fail(IBP_EHIP, "payload upload failed"));
        } else {
            // padding and slack zeroed, then every stretch of clusters in one copy
            if (hipMemset(h->d_payload, 0, bytes) != hipSuccess)
                return bail(fail(IBP_EHIP, "payload upload failed"));
            for (size_t k = 0; k + 1 < runs.size(); ++k) {
                const uint64_t s0 = v.off(runs[k]), n = v.off(runs[k + 1]) - s0;
                if (n && hipMemcpy(h->d_payload + aoff[runs[k]], v.payload() + s0, n, hipMemcpyHostToDevice) !=
                             hipSuccess)
                    return bail(fail(IBP_EHIP, "payload upload failed"));
            }
        }
        h->k_payload = h->d_payload;
    } else {
        st = flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED ? setup_aligned_host_payload(h, v)
                                                             : setup_host_path(h, v, line_al ? &aoff : nullptr, runs);
        if (st != IBP_OK) return bail(st);
        if (flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY || flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED) {
            void *dp = nullptr;
            if (hipHostGetDevicePointer(&dp, h->h_payload, 0) != hipSuccess || !dp)
                return bail(fail(IBP_EHIP, "pinned payload is not mapped for the device"));
            h->k_payload = static_cast<const uint8_t *>(dp);
        }
    }
    for (int j = 0; j < kIdSlots; ++j)
        if (hipEventCreateWithFlags(&h->ev_ids_free[j], hipEventDisableTiming) != hipSuccess)
            return bail(fail(IBP_EHIP, "event creation failed"));
    if (hipDeviceSynchronize() != hipSuccess) return bail(fail(IBP_EHIP, "upload did not complete"));
    h->ds.meta = h->d_meta;
    h->ds.slots = h->d_slots;
    h->ds.row_lines = h->d_row_lines;
    h->ds.rl_magic = dev::div_magic(dev::kRowLineRows);
    h->ds.index = h->d_index;
    h->ds.n_rows = d.n_rows;
    h->ds.n_groups = d.n_groups;
    h->ds.g_magic = dev::div_magic(d.group_rows);
    h->ds.part_m = (d.flags & IBP_STREAM_PARTICIPATION) ? d.chunk_bytes / 4 : 0;
    h->ds.row_align = flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED ? (uint32_t)kRowAlign : 0;
    h->ds.payload_host = flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY || flags == IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED;
    h->ds.W = d.row_bytes / 4;
    h->ds.G = d.group_rows;
    ignore(hipSetDevice(prev));
    prev = -1;
    *out = h;
    return IBP_OK;
}

}  // namespace

extern "C" {

ibp_status ibp_open(const void *stream, uint64_t stream_bytes, int device, uint32_t flags, ibp_handle **out) {
    clear_error();
    AllocTestScope scope;
    ibp_handle *h = nullptr;
    int prev = -1;
    const ibp_status st = guarded([&] { return open_impl(stream, stream_bytes, device, flags, out, h, prev); });
    if (st != IBP_OK) {
        if (h) free_handle(h);
        if (prev >= 0) ignore(hipSetDevice(prev));
        if (out) *out = nullptr;
    }
    return st;
}

ibp_status ibp_decompress(ibp_handle *h, uint64_t first_row, uint64_t n_rows, void *d_out, uint64_t out_cap,
                          void *stream) {
    clear_error();
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    const ibp_desc &d = h->d;
    if (first_row > d.n_rows || n_rows > d.n_rows - first_row)
        return fail(IBP_ERANGE, "row range outside the stream");
    if (n_rows == 0) return IBP_OK;
    if (!d_out) return fail(IBP_EINVAL, "output is null");
    if (out_cap / d.row_bytes < n_rows) return fail(IBP_ENOMEM, "output capacity too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint64_t L = d.row_bytes, G = d.group_rows;
    if (h->flags != IBP_OPEN_PAYLOAD_HOST) {
        IBP_HIP(h, dev::launch_decompress(h->ds, h->k_payload, 0, d_out, first_row, n_rows, s));
    } else {
        // chunks of consecutive rows whose packed bytes fit one staging buffer: the packed
        // rows of any row range are one contiguous byte range of the payload (clusters back
        // to back, rows of a cluster back to back), so exactly those bytes cross PCIe and
        // the kernel addresses them relative to the chunk's first byte
        const bool part = d.flags & IBP_STREAM_PARTICIPATION;
        auto row_byte = [&](uint64_t r) {
            if (part) return h->h_off[r];
            const uint64_t g = std::min(r / G, d.n_groups - 1);
            return h->h_off[g] + (r - g * G) * h->h_rb[g];
        };
        const uint64_t last = first_row + n_rows;
        uint64_t r = first_row;
        while (r < last) {
            const uint64_t byte0 = row_byte(r);
            // the furthest row end e <= last with row_byte(e) - byte0 <= kStageBytes
            uint64_t lo = r, hi = last;
            while (lo < hi) {
                const uint64_t mid = lo + (hi - lo + 1) / 2;
                if (row_byte(mid) - byte0 <= kStageBytes) lo = mid; else hi = mid - 1;
            }
            if (lo == r) return fail(IBP_EINVAL, "a packed row is larger than the staging buffer");
            const uint64_t e = lo, bytes = row_byte(e) - byte0;
            const int b = h->next_stage;
            h->next_stage = (h->next_stage + 1) % kStages;
            st = claim_stage(h, b, false);
            if (st != IBP_OK) return st;
            if (bytes)
                IBP_HIP(h, hipMemcpyAsync(h->d_stage[b], h->h_payload + byte0, bytes, hipMemcpyHostToDevice,
                                          h->copy_stream));
            IBP_HIP(h, hipEventRecord(h->ev_copied[b], h->copy_stream));
            IBP_HIP(h, hipStreamWaitEvent(s, h->ev_copied[b], 0));
            IBP_HIP(h, dev::launch_decompress(h->ds, h->d_stage[b], byte0,
                                              static_cast<uint8_t *>(d_out) + (r - first_row) * L, r, e - r, s));
            IBP_HIP(h, hipEventRecord(h->ev_free[b], s));
            h->stage_used[b] = true;
            h->stats.h2d_bytes += bytes;
            h->stats.h2d_payload_bytes += bytes;
            r = e;
        }
    }
    h->stats.calls += 1;
    h->stats.rows_out += n_rows;
    h->stats.out_bytes += n_rows * L;
    return IBP_OK;
}

}  // extern "C"

namespace {

ibp_status gather_impl(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids, void *d_out, uint64_t out_cap,
                       void *stream) {
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    const ibp_desc &d = h->d;
    if (n_ids == 0) return IBP_OK;
    if (!row_ids || !d_out) return fail(IBP_EINVAL, "row ids or output is null");
    if (out_cap / d.row_bytes < n_ids) return fail(IBP_ENOMEM, "output capacity too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint64_t L = d.row_bytes;
    if (h->flags != IBP_OPEN_PAYLOAD_HOST) {
        for (uint64_t i = 0; i < n_ids; ++i)
            if (row_ids[i] < 0 || (uint64_t)row_ids[i] >= d.n_rows)
                return fail(IBP_ERANGE, "row id " + std::to_string(row_ids[i]) + " at position " + std::to_string(i) +
                                            " is outside [0, " + std::to_string(d.n_rows) + ")");
        const int j = h->next_ids;
        st = claim_ids(h, j, n_ids);
        if (st != IBP_OK) return st;
        h->next_ids = (j + 1) % kIdSlots;
        std::memcpy(h->h_ids[j], row_ids, n_ids * 8);
        IBP_HIP(h, hipMemcpyAsync(h->d_ids[j], h->h_ids[j], n_ids * 8, hipMemcpyHostToDevice, s));
        IBP_HIP(h, dev::launch_gather(h->ds, h->k_payload, h->d_ids[j], nullptr, nullptr, n_ids, d_out, h->d_err, s));
        IBP_HIP(h, hipEventRecord(h->ev_ids_free[j], s));
        h->ids_used[j] = true;
        h->stats.h2d_bytes += n_ids * 8;
    } else {
        st = gather_host_payload(h, row_ids, n_ids, static_cast<uint8_t *>(d_out), s);
        if (st != IBP_OK) return st;
    }
    h->stats.calls += 1;
    h->stats.rows_out += n_ids;
    h->stats.out_bytes += n_ids * L;
    return IBP_OK;
}

}  // namespace

extern "C" {

ibp_status ibp_gather_decompress(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids, void *d_out,
                                 uint64_t out_cap, void *stream) {
    clear_error();
    AllocTestScope scope;
    return guarded([&] { return gather_impl(h, row_ids, n_ids, d_out, out_cap, stream); });
}

ibp_status ibp_gather_decompress_device(ibp_handle *h, const int64_t *d_row_ids, uint64_t n_ids, void *d_out,
                                        uint64_t out_cap, void *stream) {
    clear_error();
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    if (h->flags == IBP_OPEN_PAYLOAD_HOST)
        return fail(IBP_EINVAL, "device row ids need a handle whose kernels read the payload in place "
                                "(IBP_OPEN_PAYLOAD_DEVICE or IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)");
    if (n_ids == 0) return IBP_OK;
    if (!d_row_ids || !d_out) return fail(IBP_EINVAL, "row ids or output is null");
    if (out_cap / h->d.row_bytes < n_ids) return fail(IBP_ENOMEM, "output capacity too small");
    IBP_HIP(h, dev::launch_gather(h->ds, h->k_payload, d_row_ids, nullptr, nullptr, n_ids, d_out, h->d_err,
                                  static_cast<hipStream_t>(stream)));
    h->stats.calls += 1;
    h->stats.rows_out += n_ids;
    h->stats.out_bytes += n_ids * h->d.row_bytes;
    return IBP_OK;
}

ibp_status ibp_gather_decompress_noalloc(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids, void *d_out,
                                         uint64_t out_cap, void *stream) {
    clear_error();
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    if (h->flags == IBP_OPEN_PAYLOAD_HOST)
        return fail(IBP_EINVAL, "the allocation-free gather needs a handle whose kernels read the payload in place "
                                "(IBP_OPEN_PAYLOAD_DEVICE or IBP_OPEN_PAYLOAD_HOST_ZERO_COPY[_ALIGNED])");
    if (n_ids == 0) return IBP_OK;
    if (!row_ids || !d_out) return fail(IBP_EINVAL, "row ids or output is null");
    if (n_ids > kScratchIds) return fail(IBP_EINVAL, "n_ids exceeds the fixed scratch of 4194304 ids");
    const ibp_desc &d = h->d;
    if (out_cap / d.row_bytes < n_ids) return fail(IBP_ENOMEM, "output capacity too small");
    if (!h->scratch_ids)
        return fail(IBP_EHIP, std::string("device scratch is not available: ") + hipGetErrorString(h->scratch_err));
    for (uint64_t i = 0; i < n_ids; ++i)
        if (row_ids[i] < 0 || (uint64_t)row_ids[i] >= d.n_rows)
            return fail(IBP_ERANGE, "row id " + std::to_string(row_ids[i]) + " at position " + std::to_string(i) +
                                        " is outside [0, " + std::to_string(d.n_rows) + ")");
    hipStream_t s = static_cast<hipStream_t>(stream);
    IBP_HIP(h, hipMemcpyAsync(h->scratch_ids, row_ids, n_ids * 8, hipMemcpyHostToDevice, s));
    IBP_HIP(h, dev::launch_gather(h->ds, h->k_payload, h->scratch_ids, nullptr, nullptr, n_ids, d_out, h->d_err, s));
    h->stats.calls += 1;
    h->stats.rows_out += n_ids;
    h->stats.out_bytes += n_ids * d.row_bytes;
    h->stats.h2d_bytes += n_ids * 8;
    return IBP_OK;
}

ibp_status ibp_device_errors(ibp_handle *h, uint64_t *count) {
    clear_error();
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    if (!count) return fail(IBP_EINVAL, "count is null");
    IBP_HIP(h, hipDeviceSynchronize());
    unsigned long long c = 0;
    IBP_HIP(h, hipMemcpy(&c, h->d_err, 8, hipMemcpyDeviceToHost));
    IBP_HIP(h, hipMemset(h->d_err, 0, 8));
    IBP_HIP(h, hipDeviceSynchronize());
    *count = c;
    return IBP_OK;
}

ibp_status ibp_get_desc(ibp_handle *h, ibp_desc *d) {
    clear_error();
    if (!d) return fail(IBP_EINVAL, "null argument");
    CallScope cs(h);
    if (!h) return fail(IBP_EINVAL, "handle is null");
    if (!cs.ok()) return fail(IBP_ESTATE, cs.closed() ? "handle is closed" : "handle is in use by another thread");
    *d = h->d;
    return IBP_OK;
}

ibp_status ibp_get_stats(ibp_handle *h, ibp_stats *st) {
    clear_error();
    if (!st) return fail(IBP_EINVAL, "null argument");
    CallScope cs(h);
    if (!h) return fail(IBP_EINVAL, "handle is null");
    if (!cs.ok()) return fail(IBP_ESTATE, cs.closed() ? "handle is closed" : "handle is in use by another thread");
    *st = h->stats;
    st->gather_meta_bytes = h->d_slots ? h->ds.slot_bytes : 2ull * h->d.row_bytes;
    return IBP_OK;
}

ibp_status ibp_reset_stats(ibp_handle *h) {
    clear_error();
    CallScope cs(h);
    if (!h) return fail(IBP_EINVAL, "handle is null");
    if (!cs.ok()) return fail(IBP_ESTATE, cs.closed() ? "handle is closed" : "handle is in use by another thread");
    h->stats = ibp_stats{};
    return IBP_OK;
}

ibp_status ibp_close(ibp_handle *h) {
    clear_error();
    if (!h) return IBP_OK;
    int expected = 0;
    if (!h->busy.compare_exchange_strong(expected, 1))
        return fail(IBP_ESTATE, expected == 2 ? "handle is already closed" : "handle is in use by another thread");
    if (h->n_caches) {
        h->busy.store(0);
        return fail(IBP_ESTATE, "destroy the caches built on this handle first");
    }
    int prev = 0;
    ignore(hipGetDevice(&prev));
    ignore(hipSetDevice(h->device));
    hipError_t e = hipDeviceSynchronize();
    release_handle(h);
    ignore(hipSetDevice(prev));
    h->busy.store(2);   // the struct stays as the closed marker
    if (e != hipSuccess) return fail(IBP_EHIP, std::string("pending work failed: ") + hipGetErrorString(e));
    return IBP_OK;
}

ibp_status ibp_memory_usage(uint64_t *device_bytes, uint64_t *pinned_bytes) {
    clear_error();
    if (!device_bytes || !pinned_bytes) return fail(IBP_EINVAL, "null argument");
    std::lock_guard<std::mutex> lock(g_mem_mu);
    *device_bytes = g_dev_bytes;
    *pinned_bytes = g_pin_bytes;
    return IBP_OK;
}

// ---- compressed device cache ---------------------------------------------------

}  // extern "C"

namespace {

ibp_status cache_create_impl(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids, ibp_cache **out) {
    if (!out) return fail(IBP_EINVAL, "cache output is null");
    *out = nullptr;
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    const ibp_desc &d = h->d;
    if (h->flags != IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)
        return fail(IBP_EINVAL, "a cache needs a handle opened with IBP_OPEN_PAYLOAD_HOST_ZERO_COPY (misses are read "
                                "from the pinned payload in place)");
    if (d.flags != 0) return fail(IBP_EINVAL, "the cache holds clustered-scheme streams (flags = 0)");
    if (d.row_bytes / 4 > 512) return fail(IBP_EINVAL, "the cache supports rows of at most 2048 bytes");
    if (n_ids && !row_ids) return fail(IBP_EINVAL, "row ids are null");
    for (uint64_t i = 0; i < n_ids; ++i)
        if (row_ids[i] < 0 || (uint64_t)row_ids[i] >= d.n_rows)
            return fail(IBP_ERANGE, "row id " + std::to_string(row_ids[i]) + " at position " + std::to_string(i) +
                                        " is outside [0, " + std::to_string(d.n_rows) + ")");
    check_alloc();
    std::vector<int64_t> ids(row_ids, row_ids + n_ids);
    std::sort(ids.begin(), ids.end());
    ids.erase(std::unique(ids.begin(), ids.end()), ids.end());
    const uint64_t n = ids.size(), G = d.group_rows;
    // slab: the cached rows' packed bytes back to back, in id order
    std::vector<uint64_t> src(n), dst(n + 1);
    dst[0] = 0;
    for (uint64_t i = 0; i < n; ++i) {
        const uint64_t id = (uint64_t)ids[i], g = id / G;
        src[i] = h->h_off[g] + (id - g * G) * h->h_rb[g];
        dst[i + 1] = dst[i] + h->h_rb[g];
    }
    if (dst[n] >= (1ull << 40)) return fail(IBP_EINVAL, "cached rows exceed the 40-bit slab offset");
    uint32_t log2cap = 6;
    while ((1ull << log2cap) < 2 * n) ++log2cap;
    const uint64_t cap = 1ull << log2cap;
    struct Slot {
        uint64_t key, val;
    };
    std::vector<uint8_t> slab;
    std::vector<Slot> table;
    try {
        check_alloc();
        slab.assign(dst[n] + kSlack, 0);
        table.assign(cap, Slot{0, 0});
    } catch (const std::bad_alloc &) {
        return fail(IBP_ENOMEM, "host allocation for the cache failed");
    }
    h->pool->run(n, 4096, [&](uint64_t lo, uint64_t hi) {
        for (uint64_t i = lo; i < hi; ++i) std::memcpy(slab.data() + dst[i], h->h_payload + src[i], dst[i + 1] - dst[i]);
    });
    for (uint64_t i = 0; i < n; ++i) {
        const uint64_t id = (uint64_t)ids[i];
        uint64_t k = (id * 0x9E3779B97F4A7C15ull) >> (64 - log2cap);
        while (table[k].key != 0) k = (k + 1) & (cap - 1);
        // entry: slab byte offset (bits 0-39), slab 0 (bits 40-42), compressed form (bit 43)
        table[k] = Slot{id + 1, dst[i] | (1ull << 43)};
    }
    auto *c = alloc_fails() ? nullptr : new (std::nothrow) ibp_cache();
    if (!c) return fail(IBP_ENOMEM, "host allocation failed");
    auto bail = [&](ibp_status e) {
        dev_free(c->d_slab);
        dev_free(c->d_table);
        dev_free(c->d_counts);
        delete c;
        return e;
    };
    if (dev_alloc(&c->d_slab, slab.size()) != hipSuccess || dev_alloc(&c->d_table, cap * sizeof(Slot)) != hipSuccess ||
        dev_alloc(&c->d_counts, kCountBytes) != hipSuccess)
        return bail(fail(IBP_ENOMEM, "device allocation for the cache failed"));
    if (hipMemcpy(c->d_slab, slab.data(), slab.size(), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(c->d_table, table.data(), cap * sizeof(Slot), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemset(c->d_counts, 0, kCountBytes) != hipSuccess)
        return bail(fail(IBP_EHIP, "cache upload failed"));
    c->h = h;
    c->rows = n;
    c->slab_bytes = dst[n];
    c->slots = cap;
    c->view.table = c->d_table;
    c->view.slab = c->d_slab;
    c->view.host_payload = h->k_payload;
    c->view.counts = c->d_counts;
    c->view.mask = cap - 1;
    c->view.log2cap = log2cap;
    ++h->n_caches;
    *out = c;
    return IBP_OK;
}

}  // namespace

extern "C" {

ibp_status ibp_cache_create(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids, ibp_cache **out) {
    clear_error();
    AllocTestScope scope;
    return guarded([&] { return cache_create_impl(h, row_ids, n_ids, out); });
}

ibp_status ibp_cache_gather(ibp_cache *c, const int64_t *d_row_ids, uint64_t n_ids, void *d_out, uint64_t out_cap,
                            void *stream) {
    clear_error();
    if (!c) return fail(IBP_EINVAL, "cache is null");
    ibp_handle *h = c->h;
    CallScope cs(h);
    ibp_status st = check_handle(h, cs);
    if (st != IBP_OK) return st;
    if (c->destroyed) return fail(IBP_ESTATE, "cache is destroyed");
    if (n_ids == 0) return IBP_OK;
    if (!d_row_ids || !d_out) return fail(IBP_EINVAL, "row ids or output is null");
    if (out_cap / h->d.row_bytes < n_ids) return fail(IBP_ENOMEM, "output capacity too small");
    IBP_HIP(h, dev::launch_cache_gather(h->ds, c->view, d_row_ids, n_ids, d_out, h->d_err,
                                        static_cast<hipStream_t>(stream)));
    h->stats.calls += 1;
    h->stats.rows_out += n_ids;
    h->stats.out_bytes += n_ids * h->d.row_bytes;
    return IBP_OK;
}

ibp_status ibp_cache_get_stats(ibp_cache *c, ibp_cache_stats *st) {
    clear_error();
    if (!c || !st) return fail(IBP_EINVAL, "cache or stats is null");
    CallScope cs(c->h);
    ibp_status s = check_handle(c->h, cs);
    if (s != IBP_OK) return s;
    if (c->destroyed) return fail(IBP_ESTATE, "cache is destroyed");
    unsigned long long counts[dev::kCountLines * dev::kCountStride];
    IBP_HIP(c->h, hipDeviceSynchronize());
    IBP_HIP(c->h, hipMemcpy(counts, c->d_counts, kCountBytes, hipMemcpyDeviceToHost));
    st->rows = c->rows;
    st->slab_bytes = c->slab_bytes;
    st->table_slots = c->slots;
    st->hits = st->misses = 0;
    for (uint32_t k = 0; k < dev::kCountLines; ++k) {
        st->hits += counts[k * dev::kCountStride];
        st->misses += counts[k * dev::kCountStride + 1];
    }
    return IBP_OK;
}

ibp_status ibp_cache_reset_stats(ibp_cache *c) {
    clear_error();
    if (!c) return fail(IBP_EINVAL, "cache is null");
    CallScope cs(c->h);
    ibp_status s = check_handle(c->h, cs);
    if (s != IBP_OK) return s;
    if (c->destroyed) return fail(IBP_ESTATE, "cache is destroyed");
    IBP_HIP(c->h, hipDeviceSynchronize());
    IBP_HIP(c->h, hipMemset(c->d_counts, 0, kCountBytes));
    return IBP_OK;
}

ibp_status ibp_cache_destroy(ibp_cache *c) {
    clear_error();
    if (!c) return IBP_OK;
    ibp_handle *h = c->h;
    CallScope cs(h);
    if (!cs.ok())
        return fail(IBP_ESTATE, cs.closed() ? "the cache's handle is closed" : "the cache's handle is in use by another thread");
    if (c->destroyed) return fail(IBP_ESTATE, "cache is already destroyed");
    hipError_t e = hipDeviceSynchronize();
    dev_free(c->d_slab);
    dev_free(c->d_table);
    dev_free(c->d_counts);
    c->d_slab = nullptr;
    c->d_table = nullptr;
    c->d_counts = nullptr;
    --h->n_caches;
    c->destroyed = true;   // the struct stays as the destroyed marker
    if (e != hipSuccess) return fail(IBP_EHIP, std::string("pending work failed: ") + hipGetErrorString(e));
    return IBP_OK;
}

}  // extern "C"
