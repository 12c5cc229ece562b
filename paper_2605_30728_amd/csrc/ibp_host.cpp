// Host half of the library: stream validation and the multi-threaded compressor.
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
#include <cstring>
#include <new>
#include <thread>
#include <vector>

#include <unistd.h>

#include "ibp_internal.hpp"

namespace ibp {

namespace {
thread_local std::string g_last_error;

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
    uint32_t flags = load_u32(s + 32), reserved = load_u32(s + 36);
    d.meta_off = load_u64(s + 40);
    d.index_off = load_u64(s + 48);
    d.payload_off = load_u64(s + 56);
    if (d.row_bytes == 0 || d.row_bytes % 4 != 0) return fail(IBP_ECORRUPT, "bad row_bytes");
    if (d.group_rows == 0) return fail(IBP_ECORRUPT, "bad group_rows");
    if (flags != 0 || reserved != 0) return fail(IBP_ECORRUPT, "unsupported flags");
    if (d.n_groups != d.n_rows / d.group_rows + (d.n_rows % d.group_rows != 0))
        return fail(IBP_ECORRUPT, "n_groups inconsistent with n_rows and group_rows");
    uint64_t meta_bytes, index_bytes, idx_off, pay_off;
    if (mul_overflows(d.n_groups, 2ull * d.row_bytes, &meta_bytes) ||
        add_overflows(kHeaderBytes, meta_bytes, &idx_off) ||
        mul_overflows(d.n_groups + 1, 8, &index_bytes) ||
        add_overflows(idx_off, index_bytes, &pay_off))
        return fail(IBP_ECORRUPT, "section sizes overflow");
    if (d.meta_off != kHeaderBytes || d.index_off != idx_off || d.payload_off != pay_off)
        return fail(IBP_ECORRUPT, "section offsets inconsistent");
    if (stream_bytes < d.payload_off) return fail(IBP_ECORRUPT, "stream truncated before payload");
    v.base = s;
    v.d = d;
    const uint32_t L = d.row_bytes, W = L / 4;
    if (v.off(0) != 0) return fail(IBP_ECORRUPT, "index does not start at 0");
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

ibp_status ibp_compress(const void *rows, uint64_t n_rows, uint32_t row_bytes, uint32_t group_rows,
                        int n_threads, void *out, uint64_t out_cap, uint64_t *out_bytes) {
    clear_error();
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
    std::vector<uint64_t> off(ng + 1);
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
