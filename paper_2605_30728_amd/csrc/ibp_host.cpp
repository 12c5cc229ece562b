// Host half of the library: stream validation and the multi-threaded compressors.
//
// ibp_compress_ex adds the paper's thresholded scheme (Sec. 4.1-4.2 with T < n): per-bit
// counters over the counted rows of each cluster (split over threads when there are few,
// large clusters, e.g. one global Mask), one participation bit per chunk, a raw row
// when nothing would be saved, and a u64 offset per row.
//
// Compression follows the paper's Sec. 4.1-4.2 with clustered metadata (Sec. 6.5):
// for each cluster of G consecutive rows, Mask = the bits on which every row agrees
// and Bitval = their values (zero elsewhere); each row then keeps only its variant
// bits, in ascending bit order, byte-aligned, with the Fig. 4 size rule
// rb = L - floor(popcount(Mask)/8) and no participation bits.
//
// The invariant bits are found with AND/OR reductions (a bit is invariant iff the AND
// and the OR of the cluster agree on it), and rows are packed run by run: each 32-bit
// word's variant positions are decomposed once per cluster into runs of consecutive
// bits, so packing a word costs one shift-and-mask per run.
#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <new>
#include <thread>
#include <vector>

#include <unistd.h>

#include "ibp_internal.hpp"

namespace ibp {

namespace {
thread_local std::string g_last_error;
thread_local int g_alloc_depth = 0;          // nested AllocTestScopes on this thread
thread_local long long g_alloc_countdown = 0; // allocations left before the injected failure

inline uint32_t load_u32(const uint8_t *p) {
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}
inline uint64_t load_u64(const uint8_t *p) {
    uint64_t v;
    std::memcpy(&v, p, 8);
    return v;
}
inline void store_u32(uint8_t *p, uint32_t v) { std::memcpy(p, &v, 4); }
inline void store_u64(uint8_t *p, uint64_t v) { std::memcpy(p, &v, 8); }

bool mul_overflows(uint64_t a, uint64_t b, uint64_t *r) { return __builtin_mul_overflow(a, b, r); }
bool add_overflows(uint64_t a, uint64_t b, uint64_t *r) { return __builtin_add_overflow(a, b, r); }

// Run `fn(item)` for item in [0, n) on up to `threads` threads, in blocks.
template <class F>
void parallel_for(uint64_t n, int threads, uint64_t block, F fn) {
    if (n == 0) return;
    uint64_t blocks = (n + block - 1) / block;
    int t = (int)std::min<uint64_t>((uint64_t)std::max(threads, 1), blocks);
    if (t <= 1) {
        for (uint64_t i = 0; i < n; ++i) fn(i);
        return;
    }
    std::atomic<uint64_t> next{0};
    auto worker = [&]() {
        for (;;) {
            uint64_t b = next.fetch_add(1, std::memory_order_relaxed);
            if (b >= blocks) break;
            uint64_t lo = b * block, hi = std::min(n, lo + block);
            for (uint64_t i = lo; i < hi; ++i) fn(i);
        }
    };
    std::vector<std::thread> pool;
    pool.reserve(t - 1);
    for (int i = 0; i < t - 1; ++i) pool.emplace_back(worker);
    worker();
    for (auto &th : pool) th.join();
}

// A run of consecutive variant bits inside one 32-bit word.
struct Run {
    uint8_t lo, len;
};

// Decompose ~mask into runs (ascending); returns the count (at most 16).
inline int variant_runs(uint32_t mask, Run *runs) {
    uint32_t v = ~mask;
    int n = 0;
    while (v) {
        uint32_t low = v & (0u - v);
        uint32_t t = v + low;               // carries through the lowest run
        uint32_t run = v & ~t;
        v &= t;
        runs[n].lo = (uint8_t)__builtin_ctz(run);
        runs[n].len = (uint8_t)__builtin_popcount(run);
        ++n;
    }
    return n;
}

}  // namespace

AllocTestScope::AllocTestScope() : outer_(g_alloc_depth++ == 0) {
    if (!outer_) return;
    const char *e = std::getenv("IBP_TEST_FAIL_ALLOC");
    g_alloc_countdown = e ? std::atoll(e) : 0;
}

AllocTestScope::~AllocTestScope() {
    --g_alloc_depth;
    if (outer_) g_alloc_countdown = 0;
}

bool alloc_fails() { return g_alloc_countdown > 0 && --g_alloc_countdown == 0; }

void check_alloc() {
    if (alloc_fails()) throw std::bad_alloc();
}

ibp_status fail(ibp_status s, const std::string &msg) {
    g_last_error = msg;
    return s;
}
void clear_error() { g_last_error.clear(); }

int online_cpus() {
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

uint64_t StreamView::off(uint64_t g) const { return load_u64(index_bytes() + 8 * g); }

uint64_t StreamView::rows_in_group(uint64_t g) const {
    uint64_t start = g * d.group_rows;
    uint64_t end = std::min<uint64_t>(start + d.group_rows, d.n_rows);
    return end - start;
}

namespace {

// Mask bits of chunk c of a row (m words per chunk) under a cluster's Mask.
inline uint32_t chunk_mask_bits(const uint8_t *mask, uint32_t m, uint64_t c) {
    uint32_t n = 0;
    for (uint32_t j = 0; j < m; ++j) n += (uint32_t)__builtin_popcount(load_u32(mask + 4 * (c * m + j)));
    return n;
}

// Validation of a participation-scheme stream past its header: Bitval only under Mask,
// a monotone per-row index inside the stream, and every row's size either row_bytes
// (raw) or the size its participation bits give.
ibp_status validate_participation(StreamView &v, uint64_t stream_bytes) {
    ibp_desc &d = v.d;
    const uint32_t L = d.row_bytes, W = L / 4, m = d.chunk_bytes / 4, C = W / m;
    std::atomic<uint64_t> bad{UINT64_MAX};
    auto flag = [&](uint64_t i) {
        uint64_t cur = bad.load();
        while (i < cur && !bad.compare_exchange_weak(cur, i)) {}
    };
    parallel_for(d.n_groups, d.n_groups > 4096 ? online_cpus() : 1, 4096, [&](uint64_t g) {
        const uint8_t *mk = v.meta() + g * 2ull * L;
        uint32_t stray = 0;
        for (uint32_t w = 0; w < W; ++w) stray |= load_u32(mk + L + 4 * w) & ~load_u32(mk + 4 * w);
        if (stray) flag(g);
    });
    if (bad.load() != UINT64_MAX)
        return fail(IBP_ECORRUPT, "Bitval set outside Mask in group " + std::to_string(bad.load()));
    // the index must be monotone before any row is read through it
    parallel_for(d.n_rows, d.n_rows > 65536 ? online_cpus() : 1, 65536, [&](uint64_t i) {
        if (v.off(i + 1) < v.off(i)) flag(i);
    });
    if (bad.load() != UINT64_MAX)
        return fail(IBP_ECORRUPT, "row index decreases at row " + std::to_string(bad.load()));
    d.payload_bytes = v.off(d.n_rows);
    uint64_t end;
    if (add_overflows(d.payload_off, d.payload_bytes, &end) || end > stream_bytes)
        return fail(IBP_ECORRUPT, "stream truncated inside the payload");
    d.stream_bytes = end;
    const uint8_t *pay = v.payload();
    parallel_for(d.n_rows, d.n_rows > 65536 ? online_cpus() : 1, 16384, [&](uint64_t i) {
        const uint64_t o = v.off(i), size = v.off(i + 1) - o;
        if (size == L) return;                        // raw row
        if (size > L || size * 8 < C) {
            flag(i);
            return;
        }
        const uint8_t *mk = v.meta() + (i / d.group_rows) * 2ull * L;
        uint64_t saved = 0;
        for (uint32_t c = 0; c < C; ++c)
            if ((pay[o + c / 8] >> (c % 8)) & 1) saved += chunk_mask_bits(mk, m, c);
        if (saved < (uint64_t)C + 8 || size != L - (saved - C) / 8) flag(i);
    });
    if (bad.load() != UINT64_MAX)
        return fail(IBP_ECORRUPT, "row " + std::to_string(bad.load()) +
                                      ": size does not match its participation bits");
    return IBP_OK;
}

}  // namespace

ibp_status parse_stream(const void *stream, uint64_t stream_bytes, StreamView &v) {
    if (!stream) return fail(IBP_EINVAL, "stream is null");
    const uint8_t *s = static_cast<const uint8_t *>(stream);
    if (stream_bytes < kHeaderBytes) return fail(IBP_ECORRUPT, "stream shorter than its header");
    if (std::memcmp(s, kMagic, 4) != 0) return fail(IBP_ECORRUPT, "bad magic");
    if (load_u32(s + 4) != kVersion) return fail(IBP_ECORRUPT, "unsupported stream version");
    ibp_desc d{};
    d.row_bytes = load_u32(s + 8);
    d.group_rows = load_u32(s + 12);
    d.n_rows = load_u64(s + 16);
    d.n_groups = load_u64(s + 24);
    const uint32_t flags = load_u32(s + 32), chunk = load_u32(s + 36);
    d.meta_off = load_u64(s + 40);
    d.index_off = load_u64(s + 48);
    d.payload_off = load_u64(s + 56);
    if (d.row_bytes == 0 || d.row_bytes % 4 != 0) return fail(IBP_ECORRUPT, "bad row_bytes");
    if (d.group_rows == 0) return fail(IBP_ECORRUPT, "bad group_rows");
    const bool part = flags == IBP_STREAM_PARTICIPATION;
    if (flags == 0) {
        if (chunk != 0) return fail(IBP_ECORRUPT, "chunk_bytes set without the participation flag");
    } else if (part) {
        if (chunk == 0 || chunk % 4 != 0 || d.row_bytes % chunk != 0)
            return fail(IBP_ECORRUPT, "bad chunk_bytes");
    } else {
        return fail(IBP_ECORRUPT, "unsupported flags");
    }
    d.flags = flags;
    d.chunk_bytes = chunk;
    if (d.n_groups != d.n_rows / d.group_rows + (d.n_rows % d.group_rows != 0))
        return fail(IBP_ECORRUPT, "n_groups inconsistent with n_rows and group_rows");
    const uint64_t n_index = part ? d.n_rows + 1 : d.n_groups + 1;
    uint64_t meta_bytes, index_bytes, idx_off, pay_off;
    if (mul_overflows(d.n_groups, 2ull * d.row_bytes, &meta_bytes) ||
        add_overflows(kHeaderBytes, meta_bytes, &idx_off) ||
        mul_overflows(n_index, 8, &index_bytes) ||
        add_overflows(idx_off, index_bytes, &pay_off))
        return fail(IBP_ECORRUPT, "section sizes overflow");
    if (d.meta_off != kHeaderBytes || d.index_off != idx_off || d.payload_off != pay_off)
        return fail(IBP_ECORRUPT, "section offsets inconsistent");
    if (stream_bytes < d.payload_off) return fail(IBP_ECORRUPT, "stream truncated before payload");
    v.base = s;
    v.d = d;
    if (v.off(0) != 0) return fail(IBP_ECORRUPT, "index does not start at 0");
    if (part) return validate_participation(v, stream_bytes);
    const uint32_t L = d.row_bytes, W = L / 4;
    // per group: Bitval only under Mask, and the index step matches the size rule
    std::atomic<uint64_t> bad_group{UINT64_MAX};
    std::atomic<int> bad_kind{0};
    parallel_for(d.n_groups, d.n_groups > 4096 ? online_cpus() : 1, 4096, [&](uint64_t g) {
        const uint8_t *m = v.meta() + g * 2ull * L;
        const uint8_t *b = m + L;
        uint64_t P = 0;
        uint32_t stray = 0;
        for (uint32_t w = 0; w < W; ++w) {
            uint32_t mw = load_u32(m + 4 * w), bw = load_u32(b + 4 * w);
            P += (uint64_t)__builtin_popcount(mw);
            stray |= bw & ~mw;
        }
        uint64_t rb = packed_row_bytes(L, P);
        uint64_t o0 = v.off(g), o1 = v.off(g + 1);
        int kind = 0;
        if (stray) kind = 1;
        else if (o1 < o0 || o1 - o0 != v.rows_in_group(g) * rb) kind = 2;
        if (kind) {
            uint64_t cur = bad_group.load();
            while (g < cur && !bad_group.compare_exchange_weak(cur, g)) {}
            bad_kind.store(kind);
        }
    });
    if (bad_group.load() != UINT64_MAX) {
        std::string which = std::to_string(bad_group.load());
        if (bad_kind.load() == 1) return fail(IBP_ECORRUPT, "Bitval set outside Mask in group " + which);
        return fail(IBP_ECORRUPT, "index step does not match the Mask of group " + which);
    }
    d.payload_bytes = v.off(d.n_groups);
    uint64_t end;
    if (add_overflows(d.payload_off, d.payload_bytes, &end) || end > stream_bytes)
        return fail(IBP_ECORRUPT, "stream truncated inside the payload");
    d.stream_bytes = end;
    v.d = d;
    return IBP_OK;
}

}  // namespace ibp

using namespace ibp;

extern "C" {

const char *ibp_last_error(void) { return g_last_error.c_str(); }

const char *ibp_version(void) { return "ibp-mi355x 1 (stream format 1)"; }

ibp_status ibp_compress_bound(uint64_t n_rows, uint32_t row_bytes, uint32_t group_rows,
                              uint64_t *bound) {
    clear_error();
    if (!bound) return fail(IBP_EINVAL, "bound is null");
    if (row_bytes == 0 || row_bytes % 4 != 0)
        return fail(IBP_EINVAL, "row_bytes must be a positive multiple of 4");
    if (group_rows == 0) return fail(IBP_EINVAL, "group_rows must be >= 1");
    uint64_t ng = n_rows / group_rows + (n_rows % group_rows != 0);
    uint64_t meta, raw, idx, t;
    if (mul_overflows(ng, 2ull * row_bytes, &meta) || mul_overflows(n_rows, row_bytes, &raw) ||
        mul_overflows(ng + 1, 8, &idx) || add_overflows(meta, raw, &t) || add_overflows(t, idx, &t) ||
        add_overflows(t, kHeaderBytes, &t))
        return fail(IBP_EINVAL, "stream size overflows 64 bits");
    *bound = t;
    return IBP_OK;
}

}  // extern "C"

namespace {

ibp_status compress_clustered(const void *rows, uint64_t n_rows, uint32_t row_bytes, uint32_t group_rows,
                              int n_threads, void *out, uint64_t out_cap, uint64_t *out_bytes) {
    if (!out_bytes) return fail(IBP_EINVAL, "out_bytes is null");
    uint64_t bound;
    ibp_status st = ibp_compress_bound(n_rows, row_bytes, group_rows, &bound);
    if (st != IBP_OK) return st;
    if (n_rows > 0 && !rows) return fail(IBP_EINVAL, "rows is null");
    const uint8_t *src = static_cast<const uint8_t *>(rows);
    const uint32_t L = row_bytes, W = L / 4, G = group_rows;
    const uint64_t ng = n_rows / G + (n_rows % G != 0);
    const int threads = n_threads > 0 ? n_threads : online_cpus();
    const uint64_t meta_off = kHeaderBytes, index_off = meta_off + ng * 2ull * L,
                   payload_off = index_off + 8 * (ng + 1);

    // Pass 1: per cluster, Mask/Bitval by AND/OR reduction and the packed row size.
    std::vector<uint32_t> meta;
    std::vector<uint64_t> rb;
    try {
        check_alloc();
        meta.resize(ng * 2ull * W);
        rb.resize(ng);
    } catch (const std::bad_alloc &) {
        return fail(IBP_ENOMEM, "host allocation for cluster metadata failed");
    }
    auto rows_of = [&](uint64_t g) { return std::min<uint64_t>(G, n_rows - g * G); };
    parallel_for(ng, threads, std::max<uint64_t>(1, 65536 / std::max<uint64_t>(1, (uint64_t)G * L / 64)),
                 [&](uint64_t g) {
        uint32_t *m = &meta[g * 2ull * W];
        uint32_t *b = m + W;
        const uint8_t *grp = src + g * (uint64_t)G * L;
        uint64_t n = rows_of(g);
        for (uint32_t w = 0; w < W; ++w) {
            m[w] = 0;           // running OR
            b[w] = 0xFFFFFFFFu; // running AND
        }
        for (uint64_t r = 0; r < n; ++r) {
            const uint8_t *row = grp + r * L;
            for (uint32_t w = 0; w < W; ++w) {
                uint32_t x = load_u32(row + 4 * w);
                m[w] |= x;
                b[w] &= x;
            }
        }
        uint64_t P = 0;
        for (uint32_t w = 0; w < W; ++w) {
            m[w] = ~(m[w] ^ b[w]);   // agree in every row <=> AND == OR
            P += (uint64_t)__builtin_popcount(m[w]);
        }
        rb[g] = packed_row_bytes(L, P);
    });

    uint64_t payload = 0;
    for (uint64_t g = 0; g < ng; ++g) payload += rows_of(g) * rb[g];
    const uint64_t total = payload_off + payload;
    *out_bytes = total;
    if (total > out_cap) return fail(IBP_ENOMEM, "output capacity smaller than the stream");
    if (!out) return fail(IBP_EINVAL, "out is null");
    uint8_t *dst = static_cast<uint8_t *>(out);
    // allocated before the first byte of the output is written, so a failure writes nothing
    check_alloc();
    std::vector<uint64_t> off(ng + 1);

    std::memset(dst, 0, kHeaderBytes);
    std::memcpy(dst, kMagic, 4);
    store_u32(dst + 4, kVersion);
    store_u32(dst + 8, L);
    store_u32(dst + 12, G);
    store_u64(dst + 16, n_rows);
    store_u64(dst + 24, ng);
    store_u64(dst + 40, meta_off);
    store_u64(dst + 48, index_off);
    store_u64(dst + 56, payload_off);
    if (ng) std::memcpy(dst + meta_off, meta.data(), ng * 2ull * L);
    off[0] = 0;
    for (uint64_t g = 0; g < ng; ++g) off[g + 1] = off[g] + rows_of(g) * rb[g];
    for (uint64_t g = 0; g <= ng; ++g) store_u64(dst + index_off + 8 * g, off[g]);

    // Pass 2: pack every row's variant bits, run by run, through a 64-bit accumulator.
    uint8_t *pay = dst + payload_off;
    parallel_for(ng, threads, std::max<uint64_t>(1, 65536 / std::max<uint64_t>(1, (uint64_t)G * L / 64)),
                 [&](uint64_t g) {
        thread_local std::vector<Run> runs;
        thread_local std::vector<uint32_t> first;
        runs.resize(16ull * W);
        first.resize(W + 1);
        const uint32_t *m = &meta[g * 2ull * W];
        uint32_t nr = 0;
        for (uint32_t w = 0; w < W; ++w) {
            first[w] = nr;
            nr += (uint32_t)variant_runs(m[w], &runs[nr]);
        }
        first[W] = nr;
        const uint8_t *grp = src + g * (uint64_t)G * L;
        uint64_t n = rows_of(g);
        for (uint64_t r = 0; r < n; ++r) {
            const uint8_t *row = grp + r * L;
            uint8_t *o = pay + off[g] + r * rb[g];
            uint64_t acc = 0;
            uint32_t nacc = 0;
            for (uint32_t w = 0; w < W; ++w) {
                uint64_t x = load_u32(row + 4 * w);
                for (uint32_t k = first[w]; k < first[w + 1]; ++k) {
                    uint64_t bits = (x >> runs[k].lo) & ((1ull << runs[k].len) - 1);
                    acc |= bits << nacc;
                    nacc += runs[k].len;
                    if (nacc >= 32) {
                        store_u32(o, (uint32_t)acc);
                        o += 4;
                        acc >>= 32;
                        nacc -= 32;
                    }
                }
            }
            for (uint32_t k = 0; k < (nacc + 7) / 8; ++k) o[k] = (uint8_t)(acc >> (8 * k));
        }
    });
    return IBP_OK;
}

ibp_status compress_participation(const void *rows, uint64_t n_rows, uint32_t row_bytes, const ibp_params *p,
                                  int n_threads, void *out, uint64_t out_cap, uint64_t *out_bytes) {
    if (!p) return fail(IBP_EINVAL, "params is null");
    if (!out_bytes) return fail(IBP_EINVAL, "out_bytes is null");
    if (p->threshold_den == 0 || p->threshold_num > p->threshold_den ||
        2ull * p->threshold_num <= (uint64_t)p->threshold_den)
        return fail(IBP_EINVAL, "threshold must satisfy den/2 < num <= den");
    if (p->sample_every == 0) return fail(IBP_EINVAL, "sample_every must be >= 1");
    if (p->chunk_bytes == 0) {
        if (p->threshold_num != p->threshold_den || p->sample_every != 1)
            return fail(IBP_EINVAL, "a threshold below 1 or a sampled Mask needs participation bits");
        return compress_clustered(rows, n_rows, row_bytes, p->group_rows, n_threads, out, out_cap, out_bytes);
    }
    if (row_bytes == 0 || row_bytes % 4 != 0)
        return fail(IBP_EINVAL, "row_bytes must be a positive multiple of 4");
    if (p->group_rows == 0) return fail(IBP_EINVAL, "group_rows must be >= 1");
    if (p->chunk_bytes % 4 != 0 || row_bytes % p->chunk_bytes != 0)
        return fail(IBP_EINVAL, "chunk_bytes must be a multiple of 4 dividing row_bytes");
    if (n_rows > 0 && !rows) return fail(IBP_EINVAL, "rows is null");
    const uint8_t *src = static_cast<const uint8_t *>(rows);
    const uint32_t L = row_bytes, W = L / 4, G = p->group_rows, m = p->chunk_bytes / 4, C = W / m;
    const uint32_t every = p->sample_every;
    const uint64_t ng = n_rows / G + (n_rows % G != 0);
    const int threads = n_threads > 0 ? n_threads : online_cpus();
    uint64_t meta_bytes, idx_bytes, raw, t;
    if (mul_overflows(ng, 2ull * L, &meta_bytes) || mul_overflows(n_rows + 1, 8, &idx_bytes) ||
        mul_overflows(n_rows, L, &raw) || add_overflows(meta_bytes, idx_bytes, &t) ||
        add_overflows(t, raw, &t) || add_overflows(t, kHeaderBytes, &t))
        return fail(IBP_EINVAL, "stream size overflows 64 bits");
    const uint64_t meta_off = kHeaderBytes, index_off = meta_off + meta_bytes, payload_off = index_off + idx_bytes;
    auto rows_of = [&](uint64_t g) { return std::min<uint64_t>(G, n_rows - g * G); };

    // Pass 1: per cluster, per-bit counters over the counted rows, then the threshold rule.
    std::vector<uint32_t> meta;
    std::vector<uint32_t> size;
    try {
        check_alloc();
        meta.resize(ng * 2ull * W);
        size.resize(n_rows);
    } catch (const std::bad_alloc &) {
        return fail(IBP_ENOMEM, "host allocation for metadata failed");
    }
    // Adds, for every bit position of the row, how many of the counted rows r0, r0 + every,
    // ... (< r1) have that bit set. The counts are kept bit-sliced while rows stream in:
    // plane k holds bit k of every counter (one u32 of 32 counters per word), so adding a
    // row is a ripple-carry add of its words into the planes, word-parallel (and vectorised
    // over the words) instead of an increment per set bit; the carry usually dies within a
    // few planes. The planes are flushed into cnt every 255 rows, before an 8-bit count can
    // overflow.
    auto count_rows = [&](const uint8_t *grp, uint64_t r0, uint64_t r1, uint64_t *cnt) {
        // local copies: the planes are u32 stores, which the compiler cannot otherwise prove
        // leave the captured sizes alone (it would reload them and not vectorise)
        const uint32_t nw = W;
        const uint64_t row_len = L, step = every;
        std::vector<uint32_t> planes(8ull * nw, 0u), carry(nw);
        uint32_t pending = 0;
        auto flush = [&]() {
            // counts are at most `pending`, so planes from its bit width up are still zero
            const uint32_t kmax = 32u - (uint32_t)__builtin_clz(pending);
            for (uint32_t w = 0; w < nw; ++w)
                for (uint32_t b = 0; b < 32; ++b) {
                    uint64_t c = 0;
                    for (uint32_t k = 0; k < kmax; ++k) c |= (uint64_t)((planes[(uint64_t)k * nw + w] >> b) & 1u) << k;
                    cnt[32ull * w + b] += c;
                }
            std::fill(planes.begin(), planes.end(), 0u);
            pending = 0;
        };
        uint32_t *cy = carry.data();
        for (uint64_t r = r0; r < r1; r += step) {
            const uint8_t *row = grp + r * row_len;
            for (uint32_t w = 0; w < nw; ++w) cy[w] = load_u32(row + 4 * w);
            for (uint32_t k = 0; k < 8; ++k) {
                uint32_t *pl = &planes[(uint64_t)k * nw], any = 0;
                for (uint32_t w = 0; w < nw; ++w) {
                    const uint32_t t = pl[w] & cy[w];
                    pl[w] ^= cy[w];
                    cy[w] = t;
                    any |= t;
                }
                if (!any) break;
            }
            if (++pending == 255) flush();
        }
        if (pending) flush();
    };
    auto finish_masks = [&](uint64_t g, const uint64_t *cnt) {
        const uint64_t n = (rows_of(g) + every - 1) / every;
        uint32_t *mk = &meta[g * 2ull * W];
        uint32_t *bv = mk + W;
        const unsigned __int128 need = (unsigned __int128)p->threshold_num * n;
        for (uint32_t w = 0; w < W; ++w) {
            uint32_t mw = 0, bw = 0;
            for (uint32_t b = 0; b < 32; ++b) {
                const uint64_t c = cnt[32ull * w + b];
                if ((unsigned __int128)c * p->threshold_den >= need) {
                    mw |= 1u << b;
                    bw |= 1u << b;
                } else if ((unsigned __int128)(n - c) * p->threshold_den >= need) {
                    mw |= 1u << b;
                }
            }
            mk[w] = mw;
            bv[w] = bw;
        }
    };
    if (ng >= 4ull * (uint64_t)threads || ng == 0) {
        parallel_for(ng, threads, 1, [&](uint64_t g) {
            std::vector<uint64_t> cnt(32ull * W, 0);
            count_rows(src + g * (uint64_t)G * L, 0, rows_of(g), cnt.data());
            finish_masks(g, cnt.data());
        });
    } else {
        // few, large clusters (a global Mask): split each cluster's counted rows
        check_alloc();
        std::vector<uint64_t> part_cnt((size_t)threads * 32ull * W);
        for (uint64_t g = 0; g < ng; ++g) {
            const uint64_t n = rows_of(g), counted = (n + every - 1) / every;
            std::fill(part_cnt.begin(), part_cnt.end(), 0);
            parallel_for((uint64_t)threads, threads, 1, [&](uint64_t k) {
                const uint64_t a = counted * k / threads, b = counted * (k + 1) / threads;
                count_rows(src + g * (uint64_t)G * L, a * every, std::min(n, b * every), &part_cnt[k * 32ull * W]);
            });
            for (int k = 1; k < threads; ++k)
                for (uint64_t j = 0; j < 32ull * W; ++j) part_cnt[j] += part_cnt[(uint64_t)k * 32ull * W + j];
            finish_masks(g, part_cnt.data());
        }
    }

    // Row blocks that never straddle a cluster, for passes 2 and 3.
    const uint64_t blk = std::min<uint64_t>(G, 4096), bpc = (G + blk - 1) / blk;
    auto block_rows = [&](uint64_t k, uint64_t &g, uint64_t &r0, uint64_t &r1) {
        g = k / bpc;
        r0 = g * G + (k % bpc) * blk;
        r1 = std::min(std::min(r0 + blk, g * G + G), n_rows);
    };
    auto chunk_ok = [&](const uint32_t *mk, const uint8_t *row, uint32_t c) {
        const uint32_t *bv = mk + W;
        for (uint32_t j = 0; j < m; ++j) {
            const uint32_t w = c * m + j;
            if ((load_u32(row + 4 * w) & mk[w]) != bv[w]) return false;
        }
        return true;
    };

    // Pass 2: the size of every row (participation bits + kept bits, or raw).
    parallel_for(ng * bpc, threads, 1, [&](uint64_t k) {
        uint64_t g, r0, r1;
        block_rows(k, g, r0, r1);
        const uint32_t *mk = &meta[g * 2ull * W];
        std::vector<uint32_t> cbits(C);
        for (uint32_t c = 0; c < C; ++c) {
            uint32_t n = 0;
            for (uint32_t j = 0; j < m; ++j) n += (uint32_t)__builtin_popcount(mk[c * m + j]);
            cbits[c] = n;
        }
        for (uint64_t r = r0; r < r1; ++r) {
            const uint8_t *row = src + r * L;
            uint64_t saved = 0;
            for (uint32_t c = 0; c < C; ++c)
                if (chunk_ok(mk, row, c)) saved += cbits[c];
            size[r] = saved >= (uint64_t)C + 8 ? (uint32_t)(L - (saved - C) / 8) : L;
        }
    });
    uint64_t payload = 0;
    for (uint64_t r = 0; r < n_rows; ++r) payload += size[r];
    const uint64_t total = payload_off + payload;
    *out_bytes = total;
    if (total > out_cap) return fail(IBP_ENOMEM, "output capacity smaller than the stream");
    if (!out) return fail(IBP_EINVAL, "out is null");
    uint8_t *dst = static_cast<uint8_t *>(out);

    std::memset(dst, 0, kHeaderBytes);
    std::memcpy(dst, kMagic, 4);
    store_u32(dst + 4, kVersion);
    store_u32(dst + 8, L);
    store_u32(dst + 12, G);
    store_u64(dst + 16, n_rows);
    store_u64(dst + 24, ng);
    store_u32(dst + 32, IBP_STREAM_PARTICIPATION);
    store_u32(dst + 36, p->chunk_bytes);
    store_u64(dst + 40, meta_off);
    store_u64(dst + 48, index_off);
    store_u64(dst + 56, payload_off);
    if (ng) std::memcpy(dst + meta_off, meta.data(), ng * 2ull * L);
    uint64_t o = 0;
    for (uint64_t r = 0; r < n_rows; ++r) {
        store_u64(dst + index_off + 8 * r, o);
        o += size[r];
    }
    store_u64(dst + index_off + 8 * n_rows, o);

    // Pass 3: encode every row: participation bits, then per chunk either the variant
    // bits (run by run, as in the clustered scheme) or all of its bits.
    uint8_t *pay = dst + payload_off;
    parallel_for(ng * bpc, threads, 1, [&](uint64_t k) {
        uint64_t g, r0, r1;
        block_rows(k, g, r0, r1);
        if (r0 >= r1) return;
        const uint32_t *mk = &meta[g * 2ull * W];
        std::vector<Run> runs(16ull * W);
        std::vector<uint32_t> first(W + 1);
        uint32_t nr = 0;
        for (uint32_t w = 0; w < W; ++w) {
            first[w] = nr;
            nr += (uint32_t)variant_runs(mk[w], &runs[nr]);
        }
        first[W] = nr;
        std::vector<uint8_t> ok(C);
        for (uint64_t r = r0; r < r1; ++r) {
            const uint8_t *row = src + r * L;
            uint8_t *dp = pay + load_u64(dst + index_off + 8 * r);
            if (size[r] == L) {
                std::memcpy(dp, row, L);
                continue;
            }
            uint64_t acc = 0;
            uint32_t nacc = 0;
            auto put = [&](uint64_t bits, uint32_t len) {
                acc |= bits << nacc;
                nacc += len;
                if (nacc >= 32) {
                    store_u32(dp, (uint32_t)acc);
                    dp += 4;
                    acc >>= 32;
                    nacc -= 32;
                }
            };
            // the participation bits, up to 32 per put
            for (uint32_t c0 = 0; c0 < C; c0 += 32) {
                const uint32_t nb = std::min<uint32_t>(32, C - c0);
                uint64_t bits = 0;
                for (uint32_t c = 0; c < nb; ++c) {
                    ok[c0 + c] = chunk_ok(mk, row, c0 + c);
                    bits |= (uint64_t)ok[c0 + c] << c;
                }
                put(bits, nb);
            }
            // then every word: all 32 bits of a raw chunk, or its variant bits gathered run
            // by run into one field of popcount(~Mask) bits
            for (uint32_t c = 0; c < C; ++c) {
                for (uint32_t j = 0; j < m; ++j) {
                    const uint32_t w = c * m + j;
                    const uint64_t x = load_u32(row + 4 * w);
                    if (!ok[c]) {
                        put(x, 32);
                        continue;
                    }
                    uint64_t packed = 0;
                    uint32_t width = 0;
                    for (uint32_t q = first[w]; q < first[w + 1]; ++q) {
                        packed |= ((x >> runs[q].lo) & ((1ull << runs[q].len) - 1)) << width;
                        width += runs[q].len;
                    }
                    if (width) put(packed, width);
                }
            }
            for (uint32_t b = 0; b < (nacc + 7) / 8; ++b) dp[b] = (uint8_t)(acc >> (8 * b));
        }
    });
    return IBP_OK;
}

}  // namespace

extern "C" {

ibp_status ibp_compress(const void *rows, uint64_t n_rows, uint32_t row_bytes, uint32_t group_rows,
                        int n_threads, void *out, uint64_t out_cap, uint64_t *out_bytes) {
    clear_error();
    AllocTestScope scope;
    return guarded([&] {
        return compress_clustered(rows, n_rows, row_bytes, group_rows, n_threads, out, out_cap, out_bytes);
    });
}

ibp_status ibp_compress_ex(const void *rows, uint64_t n_rows, uint32_t row_bytes, const ibp_params *p,
                           int n_threads, void *out, uint64_t out_cap, uint64_t *out_bytes) {
    clear_error();
    AllocTestScope scope;
    return guarded([&] {
        return compress_participation(rows, n_rows, row_bytes, p, n_threads, out, out_cap, out_bytes);
    });
}

ibp_status ibp_describe(const void *stream, uint64_t stream_bytes, ibp_desc *d) {
    clear_error();
    if (!d) return fail(IBP_EINVAL, "desc is null");
    StreamView v;
    ibp_status st = parse_stream(stream, stream_bytes, v);
    if (st != IBP_OK) return st;
    *d = v.d;
    return IBP_OK;
}

}  // extern "C"
