/*
 * ibp.h -- C ABI of the MI355X (gfx950) Invariant Bit Packing library.
 *
 * Invariant Bit Packing (arxiv 2605.30728, Sec. 4) stores, for each cluster of rows,
 * the bit positions on which every row agrees once (Mask, and their values in Bitval)
 * and packs only the remaining, variant bits of each row. This library uses clusters
 * of `group_rows` consecutive rows (the clustered form of Sec. 6.5 with the threshold
 * T equal to the cluster size, so a bit is invariant exactly when every row of the
 * cluster agrees on it). Decompression rebuilds each 32-bit word of a row as
 *     word = Bitval_w | deposit(next popcount(~Mask_w) packed bits, ~Mask_w)
 * on the GPU (Sec. 4.3), fused with a row gather for embedding / feature lookups.
 *
 * Conventions for every call:
 *   - Return value: an ibp_status; IBP_OK (0) on success. On any other value the call
 *     wrote nothing to its outputs and enqueued nothing, and ibp_last_error() gives a
 *     message (thread-local, valid until the next call on the same thread).
 *   - Rows are opaque little-endian bytes (any element type); row_bytes must be a
 *     positive multiple of 4 (32-bit chunks, the paper's 4-byte chunk size).
 *   - Row ids are int64; an id outside [0, n_rows) is IBP_ERANGE (host ids).
 *   - `stream` arguments are HIP streams (hipStream_t) passed as void*; NULL means
 *     the device's null stream. Device work is asynchronous: results in device
 *     memory are valid once that stream reaches the point where the call enqueued.
 *   - A handle may be used by one host thread at a time (IBP_ESTATE otherwise).
 *     Distinct handles are independent.
 *
 * Compressed stream layout (version 1, little-endian, no implicit padding):
 *   [0,64)   header: "IBP1", u32 version=1, u32 row_bytes, u32 group_rows,
 *            u64 n_rows, u64 n_groups=ceil(n_rows/group_rows), u32 flags,
 *            u32 chunk_bytes, u64 meta_off=64, u64 index_off, u64 payload_off
 *   meta     per group g: Mask_g[row_bytes] then Bitval_g[row_bytes]
 *
 * flags = 0, chunk_bytes = 0 -- the clustered scheme (T = cluster size):
 *   index    u64 off[0..n_groups], off[0]=0, off[g+1]=off[g]+n_g*rb_g where
 *            rb_g = row_bytes - floor(popcount(Mask_g)/8) (Fig. 4 size rule with no
 *            participation bits: under T = cluster size every chunk matches Bitval)
 *   payload  packed rows back to back: row r of group g starts at
 *            payload_off + off[g] + r*rb_g; packed bit k is bit k%8 of byte k/8 and
 *            holds the k-th variant bit of the row in ascending bit position
 *            (row bit p = bit p%8 of byte p/8); padding bits are zero.
 *
 * flags = 1 (IBP_STREAM_PARTICIPATION) -- the thresholded scheme of Sec. 4.1-4.2:
 *   Mask/Bitval from a threshold T < n (rows may disagree with Bitval), the row cut
 *   into chunks of chunk_bytes (a multiple of 4 dividing row_bytes), one
 *   participation bit per chunk:
 *   index    u64 off[0..n_rows], off[0]=0: row i occupies [off[i], off[i+1]) of the
 *            payload (rows back to back)
 *   payload  a row of size row_bytes is stored raw (no byte would be saved); any other
 *            row is: bit c (c < C = row_bytes/chunk_bytes) = 1 when chunk c is
 *            compressed (chunk AND Mask == Bitval), then chunk by chunk the row's
 *            bits in ascending position, leaving out the Mask bits of compressed
 *            chunks; size = row_bytes - floor((S - C)/8) where S is the number of
 *            Mask bits of its compressed chunks (S - C >= 8 for such a row).
 */
#ifndef IBP_H
#define IBP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Test hook (every allocating call: ibp_compress, ibp_compress_ex, ibp_open,
 * ibp_gather_decompress, ibp_cache_create): while the environment variable
 * IBP_TEST_FAIL_ALLOC holds a number n >= 1, the n-th allocation that one such call makes
 * (host, pinned or device, counted from 1 within the call) fails as if memory were
 * exhausted. The call then returns IBP_ENOMEM, has written nothing to its outputs and
 * holds nothing more than before (ibp_memory_usage).
 */

typedef enum {
    IBP_OK = 0,
    IBP_EINVAL = 1,    /* a bad argument (null pointer, size, alignment, flag) */
    IBP_ERANGE = 2,    /* a row id or row range outside the stream */
    IBP_ENOMEM = 3,    /* host or device allocation failed, or an output is too small */
    IBP_ECORRUPT = 4,  /* the stream failed validation */
    IBP_EHIP = 5,      /* a HIP runtime error (sticky on a handle once seen) */
    IBP_ESTATE = 6     /* the handle is in use by another thread, or closed */
} ibp_status;

typedef struct ibp_handle ibp_handle;   /* opaque, owned by the library */

typedef struct {
    uint64_t n_rows;
    uint64_t n_groups;
    uint64_t meta_off;       /* byte offsets inside the stream */
    uint64_t index_off;
    uint64_t payload_off;
    uint64_t payload_bytes;  /* off[n_groups] */
    uint64_t stream_bytes;   /* payload_off + payload_bytes */
    uint32_t row_bytes;
    uint32_t group_rows;
    uint32_t flags;          /* 0 or IBP_STREAM_PARTICIPATION */
    uint32_t chunk_bytes;    /* participation chunk bytes (0 for the clustered scheme) */
} ibp_desc;

/* Stream flags. */
enum { IBP_STREAM_PARTICIPATION = 1 };

/* Compression parameters of ibp_compress_ex. */
typedef struct {
    uint32_t group_rows;     /* rows per cluster (>= n_rows: one Mask for all rows) */
    uint32_t chunk_bytes;    /* 0: the clustered scheme, no participation bits (then
                                threshold_num must equal threshold_den and
                                sample_every be 1); else the participation chunk size,
                                a multiple of 4 dividing row_bytes */
    uint32_t threshold_num;  /* T = threshold_num / threshold_den of the counted rows; */
    uint32_t threshold_den;  /*   require threshold_den/2 < threshold_num <= threshold_den */
    uint32_t sample_every;   /* count rows 0, k, 2k, ... of each cluster (1 = all rows) */
} ibp_params;

typedef struct {
    uint64_t calls;          /* decompress / gather calls that enqueued work */
    uint64_t rows_out;       /* rows written to device outputs */
    uint64_t out_bytes;      /* bytes written to device outputs */
    uint64_t h2d_bytes;      /* bytes the calls moved host-to-device (ids, tables, payload) */
    uint64_t h2d_payload_bytes; /* of which packed payload bytes */
    uint64_t host_pack_ns;   /* host time spent gathering packed rows into staging */
    uint64_t gather_meta_bytes; /* device metadata a row gather reads per cluster it
                                touches: a compact slot when the stream uses the clustered
                                scheme, rows of at most 2048 bytes and every cluster
                                repeats at most 16 distinct (Mask, Bitval) pairs over its
                                words (128 bytes at up to 512-byte rows and 8 pairs), else
                                the 2 * row_bytes of Mask and Bitval. A property of the
                                handle: ibp_reset_stats leaves it */
} ibp_stats;

/* Open flags: where the packed payload lives after ibp_open. */
enum {
    IBP_OPEN_PAYLOAD_DEVICE = 0, /* copied to device memory (HBM) once, at open */
    IBP_OPEN_PAYLOAD_HOST = 1,   /* kept in library-owned pinned host memory; every call
                                    moves the needed packed bytes over PCIe through
                                    rotating 128 MiB staging buffers on a side stream (the
                                    host packs the rows of a gather); rows of at most
                                    128 MiB - 72 bytes */
    IBP_OPEN_PAYLOAD_HOST_ZERO_COPY = 2, /* kept in library-owned pinned host memory and read
                                    by the decode kernels themselves over PCIe
                                    (GPU-initiated transfers, Sec. 4.4): no host packing,
                                    no staging copies */
    IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED = 3 /* as ZERO_COPY, but the pinned copy starts
                                    every packed row on a 128-byte boundary (each row padded
                                    to a multiple of 128 bytes), so reading a row over PCIe
                                    touches ceil(rb/128) 128-byte lines instead of up to one
                                    more (Sec. 4.4 aligned transfers, applied to the layout);
                                    costs host memory; clustered-scheme streams only */
};

/*
 * ibp_compress_bound -- an upper bound on the stream size of n_rows rows: the header,
 * metadata and index plus every row at its raw size, since the Fig. 4 size rule never
 * stores a row in more than its raw bytes (Sec. 4.2: a row that would save nothing is kept
 * uncompressed, so the data never grows). Host only.
 * Errors: IBP_EINVAL for a null `bound`, row_bytes not a positive multiple of 4,
 * group_rows == 0, or a size that overflows 64 bits.
 */
ibp_status ibp_compress_bound(uint64_t n_rows, uint32_t row_bytes, uint32_t group_rows,
                              uint64_t *bound);

/*
 * ibp_compress -- compress n_rows rows (row-major, row_bytes each, at `rows`) in
 * clusters of group_rows consecutive rows: per cluster, Mask/Bitval of the bits every
 * row agrees on (Sec. 4.1 with T = cluster size), then each row's variant bits packed
 * in ascending order (Sec. 4.2), into the version-1 stream above. Host only,
 * synchronous, re-entrant. n_threads <= 0 uses every online CPU. The caller owns
 * `rows` and `out`; *out_bytes receives the stream size (also when out_cap is too
 * small, in which case IBP_ENOMEM is returned and `out` is untouched). The stream is
 * a pure function of (rows, n_rows, row_bytes, group_rows).
 * Errors: IBP_EINVAL (null pointers with n_rows > 0, bad row_bytes or group_rows),
 * IBP_ENOMEM (out_cap too small or a host allocation failed).
 */
ibp_status ibp_compress(const void *rows, uint64_t n_rows, uint32_t row_bytes,
                        uint32_t group_rows, int n_threads, void *out, uint64_t out_cap,
                        uint64_t *out_bytes);

/*
 * ibp_compress_ex -- compress with explicit parameters: the clustered scheme above
 * (chunk_bytes = 0, same stream as ibp_compress) or the thresholded scheme with
 * participation bits (Sec. 4.1-4.2): per cluster, bit p is invariant 1 when at least
 * T of the counted rows have it set and invariant 0 when at least T have it clear
 * (T = threshold_num/threshold_den of the counted rows, inclusive), then every row is
 * encoded chunk by chunk as in the flags = 1 layout, or stored raw when it would save
 * no byte. Host only, synchronous, re-entrant; n_threads <= 0 uses every online CPU.
 * Call with out_cap = 0 to learn the size (*out_bytes, IBP_ENOMEM). The stream is a
 * pure function of (rows, n_rows, row_bytes, *params).
 * Errors: IBP_EINVAL (null pointers with n_rows > 0, bad row_bytes or parameters),
 * IBP_ENOMEM (out_cap too small or a host allocation failed).
 */
ibp_status ibp_compress_ex(const void *rows, uint64_t n_rows, uint32_t row_bytes,
                           const ibp_params *params, int n_threads, void *out,
                           uint64_t out_cap, uint64_t *out_bytes);

/*
 * ibp_describe -- validate a stream and fill *d. The sections mean what Sec. 4.1-4.2 and
 * Sec. 6.5 define (per-cluster Mask/Bitval, packed rows, the size rule); the container
 * around them is this library's (the paper prints none), as laid out above. Host only.
 * Validation covers the
 * header fields, the section offsets, Bitval being zero wherever Mask is zero, a
 * monotone index with off[0] = 0 and off[g+1] - off[g] = n_g * rb_g (clustered
 * scheme) or every row's size agreeing with its participation bits (flags = 1), and
 * the stream being at least payload_off + the last index entry bytes long.
 * Errors: IBP_EINVAL (null pointers), IBP_ECORRUPT (any validation failure).
 */
ibp_status ibp_describe(const void *stream, uint64_t stream_bytes, ibp_desc *d);

/*
 * ibp_open -- validate `stream` (as ibp_describe) and load it for decompression on
 * HIP device `device`: the metadata and index are copied to device memory once and
 * serve every later decompression (Sec. 4: the invariant-bit metadata lives in GPU
 * memory for the whole dataset), and the payload goes to device memory or stays in
 * library-owned pinned host memory to be read over PCIe on demand (Sec. 5, PCIe transfer
 * compression; Sec. 4.4), see the flags. Derived device copies are added where they
 * serve the gathers: compact per-cluster metadata slots (clustered streams, rows of at
 * most 2 KiB) and the per-row offsets packed 60 rows to a 128-byte line (thresholded
 * streams, rows of at most 1,092 bytes); ibp_memory_usage reports the total. The payload
 * copies the kernels read in place (device, zero-copy) of a clustered stream whose rows
 * are mostly whole 128-byte lines start every cluster on a line (at most 127 bytes of
 * padding per cluster), so one cluster of odd-sized rows does not shift later rows off
 * the lines.
 * The stream buffer is not referenced after ibp_open returns. *h receives a handle
 * owned by the library until ibp_close.
 * Errors: IBP_EINVAL, IBP_ECORRUPT, IBP_ENOMEM, IBP_EHIP.
 */
ibp_status ibp_open(const void *stream, uint64_t stream_bytes, int device, uint32_t flags,
                    ibp_handle **h);

/*
 * ibp_decompress -- decompress rows [first_row, first_row + n_rows) into d_out
 * (device memory, n_rows * row_bytes bytes, row-major), on `stream`. This is the
 * drop-in replacement for a host-to-device copy of those rows (Sec. 4.3 and the
 * Python decompress of the paper's library). With IBP_OPEN_PAYLOAD_HOST the packed
 * bytes cross PCIe in chunks, each copy overlapping the previous chunk's decode.
 * Errors: IBP_EINVAL (null handle/output with n_rows > 0), IBP_ERANGE (range outside
 * the stream), IBP_ENOMEM (out_cap < n_rows * row_bytes), IBP_EHIP, IBP_ESTATE.
 */
ibp_status ibp_decompress(ibp_handle *h, uint64_t first_row, uint64_t n_rows, void *d_out,
                          uint64_t out_cap, void *stream);

/*
 * ibp_gather_decompress -- d_out[i] = row(row_ids[i]) for i < n_ids, with row_ids in
 * host memory (read before the call returns; duplicates allowed) and d_out in device
 * memory (n_ids * row_bytes bytes). This is the one-call lookup + transfer +
 * decompress of the paper's embedding integration (Sec. 6.3) and GNN feature
 * gathering. With IBP_OPEN_PAYLOAD_HOST the host packs the selected packed rows into
 * pinned staging, which crosses PCIe chunk by chunk overlapped with the decode.
 * Errors: IBP_EINVAL, IBP_ERANGE (an id out of range; nothing is enqueued),
 * IBP_ENOMEM (out_cap too small), IBP_EHIP, IBP_ESTATE.
 */
ibp_status ibp_gather_decompress(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids,
                                 void *d_out, uint64_t out_cap, void *stream);

/*
 * ibp_gather_decompress_device -- as ibp_gather_decompress, with the row ids already
 * in device memory (d_row_ids, n_ids int64 values), for a handle whose payload is in
 * device memory (IBP_OPEN_PAYLOAD_DEVICE: every input is resident in HBM and the call
 * only enqueues the gather kernel) or read in place from pinned host memory
 * (IBP_OPEN_PAYLOAD_HOST_ZERO_COPY or _ALIGNED). Ids cannot be checked on the host: a row
 * whose id is out of range is written as zeros and counted in a device-side error
 * counter that ibp_device_errors() reads.
 * Errors: IBP_EINVAL (null pointers with n_ids > 0, or a handle opened with
 * IBP_OPEN_PAYLOAD_HOST),
 * IBP_ENOMEM (out_cap too small), IBP_EHIP, IBP_ESTATE.
 */
ibp_status ibp_gather_decompress_device(ibp_handle *h, const int64_t *d_row_ids,
                                        uint64_t n_ids, void *d_out, uint64_t out_cap,
                                        void *stream);

/*
 * ibp_gather_decompress_noalloc -- as ibp_gather_decompress (host row ids), for callers
 * that cannot allocate memory during the call: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc. It calls no hipMalloc, hipFree or other
 * allocating routine: the ids are copied (hipMemcpyAsync on `stream`) into a fixed device
 * scratch array of the library, 4,194,304 int64 ids (32 MiB) per device, which each
 * device holds from the first ibp_open on it until the process ends, and the gather
 * kernel reads them there. For a handle opened with IBP_OPEN_PAYLOAD_DEVICE or
 * IBP_OPEN_PAYLOAD_HOST_ZERO_COPY[_ALIGNED]. The ids are range-checked on the host first
 * (nothing is enqueued on IBP_ERANGE). From pageable host memory the HIP runtime has read
 * row_ids when the call returns; from pinned host memory the copy is asynchronous and
 * row_ids must stay unchanged until `stream` reaches this call. Every call on a device
 * shares that device's scratch and leaves its ids there: calls in a row on one stream
 * are ordered, but calls that overlap on one device (other streams, other threads or
 * handles) race and may decode each other's ids.
 * Errors: IBP_EINVAL (null pointers with n_ids > 0, n_ids above 4,194,304, or a handle
 * opened with IBP_OPEN_PAYLOAD_HOST), IBP_ERANGE, IBP_ENOMEM (out_cap too small),
 * IBP_EHIP, IBP_ESTATE.
 */
ibp_status ibp_gather_decompress_noalloc(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids,
                                         void *d_out, uint64_t out_cap, void *stream);

/*
 * ibp_device_errors -- synchronize the device and return (in *count) how many
 * out-of-range device ids the gather kernels met since ibp_open or the last call of
 * this function, then reset the counter. Library plumbing: the paper defines no device
 * error reporting. An asynchronous failure of an enqueued kernel or copy (a fault, not an
 * id out of range) is reported by the HIP runtime at the next synchronizing call: this
 * one (IBP_EHIP, then sticky on the handle), ibp_close, ibp_cache_get_stats, or a
 * synchronize of the caller's own.
 * Errors: IBP_EINVAL, IBP_EHIP, IBP_ESTATE.
 */
ibp_status ibp_device_errors(ibp_handle *h, uint64_t *count);

/*
 * ibp_get_desc / ibp_get_stats / ibp_reset_stats -- a copy of the handle's description,
 * a copy of its counters, and a reset of the counters. The counters report the bytes the
 * calls moved host-to-device, which the paper's evaluation normalises by (Sec. 6.1: the
 * compressed bytes moved over PCIe, as in its no-decode mock system); the calls
 * themselves are library plumbing. They take the handle like every other call: IBP_ESTATE
 * while another thread's call runs on it, or once it is closed.
 * Errors: IBP_EINVAL (null pointers), IBP_ESTATE.
 */
ibp_status ibp_get_desc(ibp_handle *h, ibp_desc *d);
ibp_status ibp_get_stats(ibp_handle *h, ibp_stats *st);
ibp_status ibp_reset_stats(ibp_handle *h);

/*
 * ibp_close -- wait for the handle's outstanding work, free everything it owns and mark
 * it closed. Library plumbing (the paper defines no such call). NULL is accepted (IBP_OK).
 * The handle's small descriptor (well under 1 KiB) stays allocated as a closed marker
 * until the process ends, so that a second ibp_close, or any other call on the closed
 * handle, returns IBP_ESTATE and does nothing. IBP_ESTATE also while another thread's
 * call runs on the handle, or while caches built on it exist (the handle stays open).
 * IBP_EHIP when outstanding work failed (the handle is closed all the same).
 */
ibp_status ibp_close(ibp_handle *h);

/*
 * ibp_memory_usage -- bytes of device memory and of pinned host memory the library
 * holds right now, over every open handle and cache (metadata, payload copies, staging,
 * id buffers, cache slabs and tables; not the fixed scratch array of
 * ibp_gather_decompress_noalloc, which is part of the loaded code object). Library
 * plumbing for memory accounting and leak checks; the paper defines no such call.
 * Errors: IBP_EINVAL (null pointers).
 */
ibp_status ibp_memory_usage(uint64_t *device_bytes, uint64_t *pinned_bytes);

/*
 * Compressed device-resident row cache (Sec. 5, cache compression). A static set of
 * rows is kept on the device in packed form, back to back in one data slab, so a slab of
 * B bytes holds about CR times more rows than an uncompressed cache; a lookup table
 * maps a row id to a 64-bit entry: slab byte offset (bits 0-39), slab id (bits 40-42,
 * always 0 on one GPU), compressed-form flag (bit 43; set for every row of a
 * clustered-scheme stream), bits 44-63 spare. A cache gather decodes hits from the slab
 * in HBM and misses from the handle's pinned payload, read in place over PCIe, in one
 * kernel. The cache keeps the handle's metadata on the device as its decode state.
 */
typedef struct ibp_cache ibp_cache;   /* opaque, owned by the library */

typedef struct {
    uint64_t rows;           /* distinct rows held */
    uint64_t slab_bytes;     /* packed bytes held (the slab) */
    uint64_t table_slots;    /* lookup table slots (16 bytes each) */
    uint64_t hits;           /* requests served from the slab since creation or reset */
    uint64_t misses;         /* requests served from host memory */
} ibp_cache_stats;

/*
 * ibp_cache_create -- build a cache holding rows row_ids[0..n_ids) (host memory, read
 * before the call returns; duplicates are held once), packed back to back in one slab
 * and mapped by a table of entries as Sec. 5 (cache compression) lays out, of a handle
 * opened with
 * IBP_OPEN_PAYLOAD_HOST_ZERO_COPY on a clustered-scheme stream (flags = 0) of at most
 * 2048-byte rows. Synchronous. The handle must outlive the cache (ibp_close returns
 * IBP_ESTATE while caches exist).
 * Errors: IBP_EINVAL (null pointers, another placement or scheme, rows too wide),
 * IBP_ERANGE (an id out of range), IBP_ENOMEM, IBP_EHIP, IBP_ESTATE.
 */
ibp_status ibp_cache_create(ibp_handle *h, const int64_t *row_ids, uint64_t n_ids, ibp_cache **c);

/*
 * ibp_cache_gather -- d_out[i] = row(d_row_ids[i]) for i < n_ids (device ids, device
 * output of n_ids * row_bytes bytes) on `stream`; hits are decoded from the slab, misses
 * from host memory (Sec. 5: a cache access finds the slab and offset of a tensor and its
 * compressed flag in the hashmap entry, and decompresses it or reads it). An id out of
 * range gives a zero row and counts in ibp_device_errors() of the handle.
 * Errors: IBP_EINVAL, IBP_ENOMEM (out_cap too small), IBP_EHIP, IBP_ESTATE (also on a
 * destroyed cache).
 */
ibp_status ibp_cache_gather(ibp_cache *c, const int64_t *d_row_ids, uint64_t n_ids, void *d_out,
                            uint64_t out_cap, void *stream);

/* ibp_cache_get_stats -- synchronize the device and copy the cache's sizes and counters
 * (the hit rate the paper's cache compression raises, Sec. 5). IBP_ESTATE on a destroyed
 * cache. */
ibp_status ibp_cache_get_stats(ibp_cache *c, ibp_cache_stats *st);
/* ibp_cache_reset_stats -- synchronize the device and zero the hit / miss counters.
 * IBP_ESTATE on a destroyed cache. */
ibp_status ibp_cache_reset_stats(ibp_cache *c);
/* ibp_cache_destroy -- wait for outstanding work and free the cache's device memory.
 * Library plumbing. NULL is accepted. The cache's small descriptor stays allocated as a
 * destroyed marker, so a second ibp_cache_destroy (or any call on it) returns IBP_ESTATE. */
ibp_status ibp_cache_destroy(ibp_cache *c);

/* ibp_last_error -- message of the last failed call on this thread ("" if none).
 * Library plumbing (the paper defines no error reporting). */
const char *ibp_last_error(void);

/* ibp_version -- library/stream format version string. Library plumbing. */
const char *ibp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* IBP_H */
