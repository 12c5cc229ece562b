// Compact device form of the clustered scheme's Mask/Bitval words, read by the row
// gathers (the kernel side is load_row_meta / expand_row_meta in ibp_wave.hpp).
//
// A cluster stores one (Mask_w, Bitval_w) pair per 32-bit word w (the Mask and Bitval of
// Sec. 4.1, one pair per cluster as in the clustered compression of Sec. 6.5). The words of
// a row repeat few distinct pairs (columns of one feature table share their invariant
// exponent and mantissa bits), and a gather reads a cluster's metadata for every row it
// decodes. So every cluster also gets a fixed-size slot, at g * slot bytes of the slot
// area, holding
//
//   pairs   P x {u32 Mask, u32 Bitval}: the cluster's distinct pairs in order of first
//           appearance (unused entries zero); P = 8, or 16 when some cluster of the
//           stream has more than 8
//   index   32*K bytes: a 4-bit pair index per word, laid out for the wave that decodes
//           the row: lane l owns words l, l+64, ..., l+64*(K-1) and their K indices sit
//           together in bits [4*K*l, 4*K*l + 4*K) of the area (index j in bits 4j..4j+3
//           of that field), so a lane fetches all of its indices with one load
//
// padded to whole 128-byte lines. Words past the row's end (lanes of the last tile) take
// index 0. A slot's address follows from the cluster number alone, so its loads need
// nothing but the row id; at K <= 2 and P = 8 a slot is one 128-byte line, against 8W
// bytes of raw metadata. The kernels read slots only when every cluster of the stream
// fits one (a per-row choice of form would cost every row a branch); a stream with a
// cluster of more than 16 pairs gets no slots and the raw words are read.
//
// The payload copies the kernels read in place may also start every cluster on a 128-byte
// line (line_aligned_clusters), so that one cluster of odd-sized rows does not shift the
// rows of whole lines after it across line boundaries.
//
// The participation scheme's per-row index gets a line-packed copy as well
// (build_row_lines): a gather request then reads one 128-byte line holding its row's
// offset and end instead of two u64 index entries, and the sparse requests of a batch
// share those lines 7.5 times as often.
#include <algorithm>
#include <atomic>
#include <cstring>

#include "ibp_internal.hpp"

namespace ibp {

namespace {

constexpr uint32_t kMaxPairs = 16;   // 4-bit indices

inline uint32_t rd32(const uint8_t *p) {
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}

// Distinct (Mask, Bitval) pairs of the cluster at mg, in order of first appearance, and
// each word's pair index; stops (returning kMaxPairs + 1) at the first pair beyond
// kMaxPairs.
uint32_t cluster_pairs(const uint8_t *mg, uint32_t W, uint32_t *pm, uint32_t *pb, uint8_t *word_pair) {
    uint32_t n = 0;
    for (uint32_t w = 0; w < W; ++w) {
        const uint32_t m = rd32(mg + 4ull * w), b = rd32(mg + 4ull * (W + w));
        uint32_t k = 0;
        while (k < n && (pm[k] != m || pb[k] != b)) ++k;
        if (k == n) {
            if (n == kMaxPairs) return kMaxPairs + 1;
            pm[n] = m;
            pb[n] = b;
            ++n;
        }
        if (word_pair) word_pair[w] = (uint8_t)k;
    }
    return n;
}

}  // namespace

uint32_t build_meta_slots(const uint8_t *meta, uint64_t n_groups, uint32_t W, uint32_t K, Pool &pool,
                          std::vector<uint8_t> &slots) {
    const uint64_t raw = 8ull * W;
    // pass 1: the most distinct pairs of any cluster
    std::atomic<uint32_t> most{0};
    pool.run(n_groups, 1024, [&](uint64_t lo, uint64_t hi) {
        uint32_t pm[kMaxPairs], pb[kMaxPairs], m = 0;
        for (uint64_t g = lo; g < hi && m <= kMaxPairs; ++g)
            m = std::max(m, cluster_pairs(meta + g * raw, W, pm, pb, nullptr));
        uint32_t cur = most.load(std::memory_order_relaxed);
        while (m > cur && !most.compare_exchange_weak(cur, m, std::memory_order_relaxed)) {
        }
    });
    const uint32_t P = most.load() <= 8 ? 8u : most.load() <= kMaxPairs ? kMaxPairs : 0u;
    if (!P) {
        slots.clear();
        return 0;
    }
    const uint64_t S = meta_slot_bytes(P, K);
    slots.assign(std::max<uint64_t>(n_groups * S, 8), 0);
    // pass 2: the slots
    pool.run(n_groups, 1024, [&](uint64_t lo, uint64_t hi) {
        std::vector<uint8_t> word_pair(W);
        uint32_t pm[kMaxPairs], pb[kMaxPairs];
        for (uint64_t g = lo; g < hi; ++g) {
            uint8_t *slot = slots.data() + g * S;
            const uint32_t n = cluster_pairs(meta + g * raw, W, pm, pb, word_pair.data());
            for (uint32_t k = 0; k < n; ++k) {
                std::memcpy(slot + 8ull * k, &pm[k], 4);
                std::memcpy(slot + 8ull * k + 4, &pb[k], 4);
            }
            uint8_t *idx = slot + 8ull * P;
            for (uint32_t l = 0; l < 64; ++l)
                for (uint32_t j = 0; j < K; ++j) {
                    const uint32_t w = l + 64 * j;
                    const uint32_t k = w < W ? word_pair[w] : 0u;
                    const uint64_t bit = 4ull * (K * l + j);
                    idx[bit >> 3] |= (uint8_t)(k << (bit & 7));
                }
        }
    });
    return P;
}

bool line_aligned_clusters(const StreamView &v, uint64_t line, uint64_t max_runs, std::vector<uint64_t> &aoff,
                           std::vector<uint64_t> &runs) {
    const ibp_desc &d = v.d;
    const uint64_t ng = d.n_groups;
    if (d.flags != 0 || ng == 0 || line == 0) return false;
    uint64_t whole = 0;
    for (uint64_t g = 0; g < ng; ++g)
        if ((v.off(g + 1) - v.off(g)) / v.rows_in_group(g) % line == 0) ++whole;
    if (2 * whole < ng) return false;
    check_alloc();
    aoff.assign(ng + 1, 0);
    runs.assign(1, 0);
    for (uint64_t g = 0; g < ng; ++g) {
        const uint64_t end = aoff[g] + (v.off(g + 1) - v.off(g));
        aoff[g + 1] = g + 1 < ng ? (end + line - 1) / line * line : end;
        if (g + 1 < ng && aoff[g + 1] - v.off(g + 1) != aoff[g] - v.off(g)) {
            runs.push_back(g + 1);
            if (runs.size() > max_runs) return false;
        }
    }
    runs.push_back(ng);
    return true;
}

bool build_row_lines(const uint8_t *index_bytes, uint64_t n_rows, uint32_t R, Pool &pool,
                     std::vector<uint8_t> &lines) {
    if (R == 0 || 8ull + 2ull * R > 128) {
        lines.clear();
        return false;
    }
    auto off = [&](uint64_t r) {
        uint64_t v;
        std::memcpy(&v, index_bytes + 8 * r, 8);
        return v;
    };
    const uint64_t n_lines = (n_rows + R - 1) / R;
    lines.assign(std::max<uint64_t>(n_lines * 128, 8), 0);
    std::atomic<bool> fits{true};
    pool.run(n_lines, 4096, [&](uint64_t lo, uint64_t hi) {
        for (uint64_t j = lo; j < hi; ++j) {
            uint8_t *ln = lines.data() + j * 128;
            const uint64_t r0 = j * R, base = off(r0);
            std::memcpy(ln, &base, 8);
            for (uint32_t k = 1; k <= R; ++k) {
                const uint64_t d = off(std::min<uint64_t>(r0 + k, n_rows)) - base;
                if (d > 0xFFFF) fits.store(false, std::memory_order_relaxed);
                const uint16_t v = (uint16_t)d;
                std::memcpy(ln + 8 + 2ull * (k - 1), &v, 2);
            }
        }
    });
    if (!fits.load()) lines.clear();
    return fits.load();
}

}  // namespace ibp
