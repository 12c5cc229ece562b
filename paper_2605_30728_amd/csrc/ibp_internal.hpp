// Internal declarations shared by the host and device halves of the library.
#pragma once

#include <cstddef>
#include <cstdint>
#include <exception>
#include <functional>
#include <new>
#include <string>
#include <vector>

#include "ibp.h"

namespace ibp {

constexpr uint32_t kHeaderBytes = 64;
constexpr uint32_t kVersion = 1;
constexpr char kMagic[4] = {'I', 'B', 'P', '1'};

// Parsed, validated view of a version-1 stream.
struct StreamView {
    const uint8_t *base = nullptr;
    ibp_desc d{};
    const uint8_t *meta() const { return base + d.meta_off; }
    const uint8_t *index_bytes() const { return base + d.index_off; }
    const uint8_t *payload() const { return base + d.payload_off; }
    uint64_t off(uint64_t g) const;            // index entry g (unaligned-safe read)
    uint64_t rows_in_group(uint64_t g) const;
};

// Thread-local error message plumbing.
ibp_status fail(ibp_status s, const std::string &msg);
void clear_error();

// Runs an entry point's body and turns a C++ exception into a status, so that none crosses
// the C ABI: std::bad_alloc is IBP_ENOMEM, anything else IBP_EINVAL.
template <class F>
ibp_status guarded(F &&body) noexcept {
    try {
        return body();
    } catch (const std::bad_alloc &) {
        return fail(IBP_ENOMEM, "host allocation failed");
    } catch (const std::exception &e) {
        return fail(IBP_EINVAL, e.what());
    } catch (...) {
        return fail(IBP_EINVAL, "unexpected error");
    }
}

// Test hook for allocation failures: while the environment variable IBP_TEST_FAIL_ALLOC
// holds a number n >= 1, the n-th allocation made by one call of an allocating entry point
// (counted from 1 within that call) fails as if memory were exhausted. An AllocTestScope
// at the top of the entry point reads the variable; nested scopes keep the outer count.
class AllocTestScope {
public:
    AllocTestScope();
    ~AllocTestScope();
    AllocTestScope(const AllocTestScope &) = delete;
    AllocTestScope &operator=(const AllocTestScope &) = delete;

private:
    bool outer_;
};
bool alloc_fails();     // counts one allocation; true when it is the one to fail
void check_alloc();     // counts one allocation; throws std::bad_alloc when it is to fail

// Validate `stream` and fill `v`; on failure sets the error message.
ibp_status parse_stream(const void *stream, uint64_t stream_bytes, StreamView &v);

// Bytes of one packed row of a group whose Mask has P set bits.
inline uint64_t packed_row_bytes(uint32_t row_bytes, uint64_t mask_popcount) {
    return (uint64_t)row_bytes - mask_popcount / 8;
}

int online_cpus();

// Persistent worker pool (threads - 1 workers plus the calling thread).
class Pool {
public:
    explicit Pool(int threads);
    ~Pool();
    Pool(const Pool &) = delete;
    Pool &operator=(const Pool &) = delete;
    int size() const;
    // Run fn(lo, hi) over [0, n) in blocks of `block` on every worker and the caller;
    // returns once every block has run. One caller at a time.
    void run(uint64_t n, uint64_t block, const std::function<void(uint64_t, uint64_t)> &fn);

private:
    struct State;
    State *st_;
};

// Compact device metadata of the clustered scheme's row gathers (ibp_meta_slots.cpp): a
// fixed-size slot per cluster, cluster g at g * slot bytes, with its distinct (Mask, Bitval)
// pairs (room for 8, or for 16 when some cluster has more than 8) and a 4-bit pair index per
// word, laid out for lanes owning K words each. Returns the pairs per slot (8 or 16), or 0
// when some cluster has more than 16 distinct pairs (no slots).
constexpr uint64_t meta_slot_bytes(uint32_t pairs, uint32_t K) { return (8ull * pairs + 32ull * K + 127) / 128 * 128; }
uint32_t build_meta_slots(const uint8_t *meta, uint64_t n_groups, uint32_t W, uint32_t K, Pool &pool,
                          std::vector<uint8_t> &slots);

// Line-packed row offsets of a participation-scheme stream (ibp_meta_slots.cpp), from its
// per-row index off[0..n_rows] (unaligned u64s at index_bytes): one 128-byte line per R
// rows, line j holding off[jR] (u64) and then off[min(jR + k, n_rows)] - off[jR] for
// k = 1..R (u16). Returns false (lines cleared) when a difference does not fit 16 bits
// or 8 + 2R > 128.
bool build_row_lines(const uint8_t *index_bytes, uint64_t n_rows, uint32_t R, Pool &pool,
                     std::vector<uint8_t> &lines);

// Line-aligned cluster layout of a clustered stream's payload (ibp_meta_slots.cpp), for the
// copies the kernels read in place (device payload, zero-copy pinned payload): every cluster
// starts on a `line`-byte boundary, rows of a cluster back to back as in the stream. A
// cluster whose rows are whole lines (rb a multiple of `line`) then keeps every row on whole
// lines: in the stream one cluster of 255-byte rows shifts all later rows by 64 bytes, and a
// 256-byte row 64 bytes off a 128-byte line costs three line fetches instead of two. aoff
// receives the aligned cluster offsets (n_groups + 1); runs the first cluster of every
// stretch that keeps one shift from the stream's offsets (copied as one piece), then
// n_groups. Returns false when fewer than half the clusters have rows of whole lines (the
// padding would buy nothing), when the copy would take more than max_runs pieces, or for
// a thresholded stream.
bool line_aligned_clusters(const StreamView &v, uint64_t line, uint64_t max_runs, std::vector<uint64_t> &aoff,
                           std::vector<uint64_t> &runs);

}  // namespace ibp
