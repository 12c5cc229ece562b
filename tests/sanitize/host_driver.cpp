// Test driver for the CPU sanitizer build (AddressSanitizer, LeakSanitizer and
// UndefinedBehaviorSanitizer): the library's host half (stream compressors and
// validation, the compact metadata-slot builder, the worker pool) and the CPU oracle,
// linked into one executable with no GPU code, run over seeded cases:
//   - both compressors against the oracle's streams, byte for byte, for both schemes and
//     1 and 4 threads, including empty inputs, 1-row clusters, tail clusters and rows of
//     one word up to 513 words;
//   - the oracle decoding every row of the library's stream back to the input;
//   - for a seeded quarter of the cases, ibp_describe over every single-byte corruption of
//     the header and of the index's first 256 bytes, a sample of corruptions elsewhere,
//     and truncations (any status, no invalid access; truncations must be refused);
//   - two seeded variants of the thresholded scheme (chunk size, threshold, sampling) per
//     clustered case;
//   - the metadata slots expanded back to each word's Mask/Bitval;
//   - the pool covering every index exactly once for several sizes and block sizes;
//   - the allocation-failure hook (IBP_TEST_FAIL_ALLOC): IBP_ENOMEM, the output untouched,
//     and no leak (LeakSanitizer at exit).
// Exit status 0 and "host sanitize ok" on success; the sanitizers abort on any finding.
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "ibp_internal.hpp"

extern "C" {
int ibpo_compress(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G, uint8_t *out, uint64_t cap,
                  uint64_t *out_bytes);
uint64_t ibpo_stream_bytes(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G);
int ibpo_decode_rows(const uint8_t *stream, uint64_t stream_bytes, const int64_t *ids, uint64_t n_ids,
                     uint8_t *out);
uint64_t ibpo_part_stream_bytes(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G, uint32_t CS,
                                uint32_t num, uint32_t den, uint32_t every);
int ibpo_part_compress(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G, uint32_t CS, uint32_t num,
                       uint32_t den, uint32_t every, uint8_t *out, uint64_t cap, uint64_t *out_bytes);
int ibpo_part_decode_rows(const uint8_t *stream, uint64_t stream_bytes, const int64_t *ids, uint64_t n_ids,
                          uint8_t *out);
}

namespace {

int g_fail = 0;
#define CHECK(cond, ...)                                      \
    do {                                                      \
        if (!(cond)) {                                        \
            std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            std::fprintf(stderr, __VA_ARGS__);                \
            std::fprintf(stderr, "\n");                       \
            ++g_fail;                                         \
        }                                                     \
    } while (0)

struct Rng {
    uint64_t s;
    uint64_t next() {
        uint64_t z = (s += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
};

// Rows with some structure: kind 0 uniform bytes, 1 a shared base with a few varying bits
// per word, 2 mostly zero words, 3 identical rows.
std::vector<uint8_t> make_rows(uint64_t n, uint32_t L, int kind, uint64_t seed) {
    Rng r{seed};
    std::vector<uint8_t> v(n * L);
    std::vector<uint32_t> base(L / 4), vary(L / 4);
    for (auto &b : base) b = (uint32_t)r.next();
    for (auto &m : vary) m = (uint32_t)r.next() & (uint32_t)r.next() & 0x0F0F0FFFu;
    for (uint64_t i = 0; i < n; ++i)
        for (uint32_t w = 0; w < L / 4; ++w) {
            uint32_t x;
            switch (kind) {
            case 0: x = (uint32_t)r.next(); break;
            case 1: x = (base[w] & ~vary[w]) | ((uint32_t)r.next() & vary[w]); break;
            case 2: x = (r.next() % 8 == 0) ? (uint32_t)r.next() : 0u; break;
            default: x = base[w]; break;
            }
            std::memcpy(&v[i * L + 4ull * w], &x, 4);
        }
    return v;
}

std::vector<uint8_t> lib_stream(const std::vector<uint8_t> &rows, uint64_t n, uint32_t L, const ibp_params &p,
                                int threads) {
    uint64_t size = 0;
    ibp_status st = ibp_compress_ex(rows.data(), n, L, &p, threads, nullptr, 0, &size);
    CHECK(st == IBP_ENOMEM || (st == IBP_OK && size == 0), "size query status %d", (int)st);
    std::vector<uint8_t> s(size + 1, 0xEE);
    st = ibp_compress_ex(rows.data(), n, L, &p, threads, s.data(), size, &size);
    CHECK(st == IBP_OK, "compress status %d: %s", (int)st, ibp_last_error());
    CHECK(s[size] == 0xEE, "wrote past the stream");
    s.resize(size);
    return s;
}

std::vector<uint8_t> oracle_stream(const std::vector<uint8_t> &rows, uint64_t n, uint32_t L, const ibp_params &p) {
    const uint8_t *src = n ? rows.data() : nullptr;
    std::vector<uint8_t> s;
    uint64_t got = 0;
    if (p.chunk_bytes == 0) {
        s.resize(ibpo_stream_bytes(src, n, L, p.group_rows));
        CHECK(ibpo_compress(src, n, L, p.group_rows, s.data(), s.size(), &got) == 0, "oracle compress");
    } else {
        s.resize(ibpo_part_stream_bytes(src, n, L, p.group_rows, p.chunk_bytes, p.threshold_num, p.threshold_den,
                                        p.sample_every));
        CHECK(ibpo_part_compress(src, n, L, p.group_rows, p.chunk_bytes, p.threshold_num, p.threshold_den,
                                 p.sample_every, s.data(), s.size(), &got) == 0,
              "oracle part compress");
    }
    CHECK(got == s.size(), "oracle size");
    return s;
}

void check_slots(const std::vector<uint8_t> &stream, ibp::Pool &pool) {
    ibp_desc d{};
    if (ibp_describe(stream.data(), stream.size(), &d) != IBP_OK || d.flags != 0 || d.n_groups == 0) return;
    const uint32_t W = d.row_bytes / 4;
    if (W > 512) return;
    const uint32_t K = W <= 64 ? 1 : W <= 128 ? 2 : W <= 256 ? 4 : 8;
    std::vector<uint8_t> slots;
    const uint8_t *meta = stream.data() + d.meta_off;
    const uint32_t P = ibp::build_meta_slots(meta, d.n_groups, W, K, pool, slots);
    if (!P) return;
    const uint64_t S = ibp::meta_slot_bytes(P, K);
    CHECK(slots.size() >= d.n_groups * S, "slot area");
    for (uint64_t g = 0; g < d.n_groups; ++g) {
        const uint8_t *slot = slots.data() + g * S, *mg = meta + g * 8ull * W;
        for (uint32_t w = 0; w < W; ++w) {
            const uint32_t l = w % 64, j = w / 64;
            const uint64_t bit = 4ull * (K * l + j);
            const uint32_t k = (slot[8ull * P + (bit >> 3)] >> (bit & 7)) & 15u;
            CHECK(k < P, "pair index");
            CHECK(std::memcmp(slot + 8ull * k, mg + 4ull * w, 4) == 0, "slot Mask g=%llu w=%u", (unsigned long long)g, w);
            CHECK(std::memcmp(slot + 8ull * k + 4, mg + 4ull * (W + w), 4) == 0, "slot Bitval");
        }
    }
}

// The line-packed row offsets of a participation stream give back every row's span of
// the per-row index, for the kernels' block of 60 rows and for short blocks that make
// small streams span several lines.
void check_row_lines(const std::vector<uint8_t> &stream, ibp::Pool &pool) {
    ibp_desc d{};
    if (ibp_describe(stream.data(), stream.size(), &d) != IBP_OK || d.flags == 0) return;
    const uint8_t *index = stream.data() + d.index_off;
    auto off = [&](uint64_t r) {
        uint64_t v;
        std::memcpy(&v, index + 8 * r, 8);
        return v;
    };
    std::vector<uint8_t> lines;
    CHECK(!ibp::build_row_lines(index, d.n_rows, 61, pool, lines), "61 rows do not fit a line");
    for (uint32_t R : {1u, 3u, 60u}) {
        const bool fits = (uint64_t)R * d.row_bytes <= 0xFFFF;
        const bool built = ibp::build_row_lines(index, d.n_rows, R, pool, lines);
        if (!built) {
            CHECK(!fits, "row lines refused although R * row_bytes fits 16 bits");
            continue;
        }
        CHECK(lines.size() >= (d.n_rows + R - 1) / R * 128, "row line area");
        for (uint64_t r = 0; r < d.n_rows; ++r) {
            const uint8_t *ln = lines.data() + (r / R) * 128;
            const uint32_t k = (uint32_t)(r % R);
            uint64_t base;
            uint16_t e0 = 0, e1;
            std::memcpy(&base, ln, 8);
            if (k) std::memcpy(&e0, ln + 8 + 2ull * (k - 1), 2);
            std::memcpy(&e1, ln + 8 + 2ull * k, 2);
            CHECK(base + e0 == off(r) && base + e1 == off(r + 1), "row line span r=%llu R=%u",
                  (unsigned long long)r, R);
        }
    }
}

// The line-aligned cluster layout: every cluster starts on a line, each has room for its
// packed rows, the last ends right after its rows, and the copy pieces cover the clusters
// in order, each keeping one shift from the stream's offsets. Small lines make the small
// streams here engage it; a limit of one piece exercises the refusal.
void check_line_layout(const std::vector<uint8_t> &stream) {
    ibp::StreamView v;
    if (ibp::parse_stream(stream.data(), stream.size(), v) != IBP_OK || v.d.flags != 0 || v.d.n_groups == 0) return;
    const uint64_t ng = v.d.n_groups;
    for (uint64_t line : {4ull, 16ull, 128ull}) {
        uint64_t whole = 0;
        for (uint64_t g = 0; g < ng; ++g)
            if ((v.off(g + 1) - v.off(g)) / v.rows_in_group(g) % line == 0) ++whole;
        std::vector<uint64_t> aoff, runs;
        const bool on = ibp::line_aligned_clusters(v, line, 1u << 20, aoff, runs);
        CHECK(on == (2 * whole >= ng), "line layout engaged iff half the clusters have whole-line rows");
        if (!on) continue;
        CHECK(aoff.size() == ng + 1 && aoff[0] == 0 && runs.front() == 0 && runs.back() == ng, "layout shape");
        for (uint64_t g = 0; g < ng; ++g) {
            const uint64_t size = v.off(g + 1) - v.off(g);
            CHECK(aoff[g] % line == 0, "cluster %llu not on a line", (unsigned long long)g);
            if (g + 1 < ng)
                CHECK(aoff[g + 1] == (aoff[g] + size + line - 1) / line * line, "cluster %llu end", (unsigned long long)g);
            else
                CHECK(aoff[g + 1] == aoff[g] + size, "last cluster end");
        }
        for (size_t k = 0; k + 1 < runs.size(); ++k) {
            CHECK(runs[k] < runs[k + 1], "pieces in order");
            for (uint64_t g = runs[k]; g < runs[k + 1]; ++g)
                CHECK(aoff[g] - v.off(g) == aoff[runs[k]] - v.off(runs[k]), "one shift per piece");
            if (k > 0)
                CHECK(aoff[runs[k]] - v.off(runs[k]) != aoff[runs[k] - 1] - v.off(runs[k] - 1), "piece boundary");
        }
        if (runs.size() > 2) CHECK(!ibp::line_aligned_clusters(v, line, 1, aoff, runs), "piece limit");
    }
}

void corrupt_describe(const std::vector<uint8_t> &stream, Rng &r) {
    ibp_desc d{};
    if (ibp_describe(stream.data(), stream.size(), &d) != IBP_OK) return;
    std::vector<uint8_t> c;
    // every byte of the header and of the index (bounded), and a sample elsewhere
    std::vector<uint64_t> at;
    for (uint64_t i = 0; i < std::min<uint64_t>(64, stream.size()); ++i) at.push_back(i);
    for (uint64_t i = d.index_off; i < std::min<uint64_t>(d.payload_off, d.index_off + 256); ++i) at.push_back(i);
    for (int k = 0; k < 64 && !stream.empty(); ++k) at.push_back(r.next() % stream.size());
    for (uint64_t i : at) {
        c = stream;
        c[i] ^= (uint8_t)(1u << (r.next() % 8));
        ibp_desc e{};
        (void)ibp_describe(c.data(), c.size(), &e);
        c[i] = 0xFF;
        (void)ibp_describe(c.data(), c.size(), &e);
    }
    for (uint64_t cut : {uint64_t(0), uint64_t(1), uint64_t(63), uint64_t(64), d.index_off, d.payload_off,
                         stream.size() - 1}) {
        if (cut > stream.size()) continue;
        // a truncated copy of its own, so that any read past `cut` leaves the allocation
        std::vector<uint8_t> t(stream.begin(), stream.begin() + cut);
        ibp_desc e{};
        const ibp_status st = ibp_describe(cut ? t.data() : nullptr, cut, &e);
        CHECK(cut == stream.size() || st != IBP_OK, "truncation to %llu accepted", (unsigned long long)cut);
    }
}

void roundtrip(const std::vector<uint8_t> &rows, uint64_t n, uint32_t L, const std::vector<uint8_t> &s, bool part) {
    if (!n) return;
    std::vector<int64_t> ids(n);
    for (uint64_t i = 0; i < n; ++i) ids[i] = (int64_t)(n - 1 - i);
    std::vector<uint8_t> out(n * L);
    const int rc = part ? ibpo_part_decode_rows(s.data(), s.size(), ids.data(), n, out.data())
                        : ibpo_decode_rows(s.data(), s.size(), ids.data(), n, out.data());
    CHECK(rc == 0, "oracle decode of the library stream");
    for (uint64_t i = 0; i < n; ++i)
        CHECK(std::memcmp(&out[i * L], &rows[(n - 1 - i) * L], L) == 0, "round trip row %llu", (unsigned long long)i);
}

void pool_cover() {
    for (int threads : {1, 3, 8}) {
        ibp::Pool pool(threads);
        for (uint64_t n : {0ull, 1ull, 7ull, 1000ull, 65537ull})
            for (uint64_t blk : {1ull, 3ull, 1024ull}) {
                std::vector<std::atomic<int>> hit(n);
                for (auto &h : hit) h.store(0);
                pool.run(n, blk, [&](uint64_t lo, uint64_t hi) {
                    for (uint64_t i = lo; i < hi; ++i) hit[i].fetch_add(1);
                });
                for (uint64_t i = 0; i < n; ++i) CHECK(hit[i].load() == 1, "pool index %llu", (unsigned long long)i);
            }
    }
}

void alloc_failures() {
    const uint64_t n = 300;
    const uint32_t L = 64;
    auto rows = make_rows(n, L, 1, 99);
    for (int part = 0; part < 2; ++part) {
        ibp_params p{part ? 300u : 16u, part ? 8u : 0u, part ? 4u : 1u, part ? 5u : 1u, 1u};
        const auto want = oracle_stream(rows, n, L, p);
        int fails = 0;
        for (int k = 1; k < 12; ++k) {
            char v[16];
            std::snprintf(v, sizeof v, "%d", k);
            setenv("IBP_TEST_FAIL_ALLOC", v, 1);
            std::vector<uint8_t> out(want.size(), 0xAB);
            uint64_t got = 0;
            const ibp_status st = ibp_compress_ex(rows.data(), n, L, &p, 2, out.data(), out.size(), &got);
            unsetenv("IBP_TEST_FAIL_ALLOC");
            if (st == IBP_OK) {
                CHECK(out == want, "stream after the injected failures");
                break;
            }
            CHECK(st == IBP_ENOMEM, "injected failure status %d", (int)st);
            bool untouched = true;
            for (uint8_t b : out) untouched &= b == 0xAB;
            CHECK(untouched, "output written by a failed call (k=%d)", k);
            ++fails;
        }
        CHECK(fails >= 2, "allocations seen: %d", fails);
    }
}

}  // namespace

int main() {
    Rng r{2024};
    ibp::Pool pool(4);
    int cases = 0;
    const uint32_t widths[] = {4, 12, 64, 400, 2052};
    const uint64_t counts[] = {0, 1, 5, 37, 300};
    for (uint32_t L : widths)
        for (uint64_t n : counts)
            for (int kind = 0; kind < 4; ++kind) {
                auto rows = make_rows(n, L, kind, r.next());
                for (uint32_t G : {1u, 3u, 32u, (uint32_t)n + 5}) {
                    ibp_params p{G, 0, 1, 1, 1};
                    const auto want = oracle_stream(rows, n, L, p);
                    for (int threads : {1, 4}) {
                        const auto got = lib_stream(rows, n, L, p, threads);
                        CHECK(got == want, "clustered stream L=%u n=%llu kind=%d G=%u t=%d", L, (unsigned long long)n,
                              kind, G, threads);
                    }
                    roundtrip(rows, n, L, want, false);
                    check_slots(want, pool);
                    check_line_layout(want);
                    if (r.next() % 4 == 0) corrupt_describe(want, r);
                    ++cases;
                    // two seeded variants of the thresholded scheme per case
                    const uint32_t chunks[] = {4u, 8u, L};
                    const std::pair<uint32_t, uint32_t> ths[] = {{4, 5}, {9, 10}, {1, 1}};
                    for (int v = 0; v < 2; ++v) {
                        const uint32_t CS = chunks[r.next() % 3];
                        if (L % CS) continue;
                        const auto th = ths[r.next() % 3];
                        const uint32_t every = 1 + 2 * (uint32_t)(r.next() % 2);
                        ibp_params q{G, CS, th.first, th.second, every};
                        const auto pw = oracle_stream(rows, n, L, q);
                        const auto pg = lib_stream(rows, n, L, q, 1 + (int)(r.next() % 4));
                        CHECK(pg == pw, "participation stream L=%u n=%llu kind=%d G=%u CS=%u T=%u/%u every=%u", L,
                              (unsigned long long)n, kind, G, CS, th.first, th.second, every);
                        roundtrip(rows, n, L, pw, true);
                        check_row_lines(pw, pool);
                        if (r.next() % 4 == 0) corrupt_describe(pw, r);
                        ++cases;
                    }
                }
            }
    pool_cover();
    alloc_failures();
    if (g_fail) {
        std::fprintf(stderr, "host sanitize: %d failure(s)\n", g_fail);
        return 1;
    }
    std::printf("host sanitize ok: %d stream cases\n", cases);
    return 0;
}
