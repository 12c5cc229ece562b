// Launchers of the gfx950 decompression kernels (ibp_kernels.hip).
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

namespace ibp {
namespace dev {

// What the kernels need to know about a stream resident on the device.
struct DevStream {
    const uint32_t *meta;    // per group: Mask[W] then Bitval[W] (32-bit words)
    const uint64_t *index;   // clustered scheme: off[0..n_groups] (payload byte offset of
                             // each group); participation scheme: off[0..n_rows] (of each row)
    uint64_t n_rows;
    uint64_t n_groups;
    uint64_t g_magic;        // ceil(2^64 / G) for G >= 2: id / G = mulhi(id, g_magic)
    uint32_t W;              // 32-bit words per row
    uint32_t G;              // rows per group
    uint32_t part_m;         // participation scheme: words per chunk; 0 = clustered scheme
    uint32_t row_align;      // clustered scheme: rows of a cluster start every
                             // roundup(rb, row_align) bytes (0: every rb bytes, no padding)
    uint32_t payload_host;   // 1: the kernels read the payload in pinned host memory over
                             // PCIe (zero-copy placements), 0: device memory (payload or stage)
    // clustered scheme, W <= 512, every cluster with at most 16 distinct (Mask, Bitval)
    // pairs: the row gathers' compact metadata, one slot of slot_bytes per cluster holding
    // slot_pairs (8 or 16) pairs and the 4-bit word indices (see load_row_meta); slots
    // null: they read `meta`
    const uint8_t *slots;
    uint32_t slot_pairs;
    uint32_t slot_bytes;
    // participation scheme, rows of at most 65535 / kRowLineRows bytes: the row offsets
    // line-packed, one 128-byte line per kRowLineRows rows (see row_span); null: the
    // kernels read `index`
    const uint8_t *row_lines;
    uint64_t rl_magic;       // div_magic(kRowLineRows)
};

// Rows per line of DevStream::row_lines: line j holds the u64 payload offset of row
// j * kRowLineRows, then for k = 1 .. kRowLineRows the u16 offset of row j * kRowLineRows + k
// (of the payload end past the last row) relative to it: 8 + 2 * 60 = 128 bytes.
inline constexpr uint32_t kRowLineRows = 60;

uint64_t div_magic(uint32_t G);

// Words per lane (K) of the tile that decodes a row of W words in one wave: lane l owns
// words l, l + 64, ..., l + 64(K - 1). Rows wider than 512 words are decoded tile by tile
// with K = 8.
inline int words_per_lane(uint32_t W) { return W <= 64 ? 1 : W <= 128 ? 2 : W <= 256 ? 4 : 8; }

// Bytes of a compact metadata slot holding `pairs` (Mask, Bitval) u32 pairs and the 4-bit
// pair indices of rows decoded with K words per lane (32K bytes), padded to 128-byte lines.
inline constexpr uint32_t meta_slot_bytes(uint32_t pairs, uint32_t K) { return (8 * pairs + 32 * K + 127) / 128 * 128; }

// Rows [first, first + n) into out (row-major). Packed row r of group g is read at byte
// off[g] - pay_base + (r - g*G) * rb_g of `payload` (participation scheme: at byte
// off[r] - pay_base, off[r+1] - off[r] bytes), which must be readable for 8 bytes past
// the last packed byte.
hipError_t launch_decompress(const DevStream &s, const uint8_t *payload, uint64_t pay_base,
                             void *out, uint64_t first, uint64_t n, hipStream_t stream);

// out[i] = row i of n requests. Device payload (sg == soff == null): request i is row
// ids[i], read at off[g] + r*rb_g (participation scheme: off[id]) of the device-resident
// payload; ids outside [0, n_rows) give a zero row and one increment of *err.
// Host-packed staging (ids null): request i belongs to cluster sg[i] (validated on the
// host) and its packed bytes are [soff[i], soff[i+1]) of `payload` (soff has n + 1
// entries). Either payload is readable 8 bytes past its last byte.
hipError_t launch_gather(const DevStream &s, const uint8_t *payload, const int64_t *ids,
                         const uint32_t *sg, const uint32_t *soff, uint64_t n, void *out,
                         unsigned long long *err, hipStream_t stream);

// Hit / miss counters of a cache: kCountLines pairs, one per 128-byte line.
inline constexpr uint32_t kCountLines = 64;
inline constexpr uint32_t kCountStride = 16;   // u64 per line

// A compressed row cache resident on the device (see ibp_cache_kernels.hip).
struct CacheView {
    const void *table;               // 2^log2cap slots of {u64 key = id + 1 (0 empty), u64 entry}
    const uint8_t *slab;             // cached packed rows (readable 8 bytes past the last)
    const uint8_t *host_payload;     // device address of the pinned payload (misses)
    unsigned long long *counts;      // kCountLines x [hits, misses, unused...]
    uint64_t mask;                   // 2^log2cap - 1
    uint32_t log2cap;
};

// out[i] = row ids[i] for a clustered-scheme stream of at most 512 words per row: rows
// found in the cache table are decoded from the slab, the others from the pinned host
// payload; ids outside [0, n_rows) give a zero row and one increment of *err.
hipError_t launch_cache_gather(const DevStream &s, const CacheView &c, const int64_t *ids, uint64_t n, void *out,
                               unsigned long long *err, hipStream_t stream);

}  // namespace dev
}  // namespace ibp
