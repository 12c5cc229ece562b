/*
 * ibp_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded, bit-serial CPU oracle of Invariant Bit Packing
 * (IBP) with clustered metadata: one Mask/Bitval pair per cluster of G consecutive
 * rows, a bit being invariant only when every row of the cluster agrees on it.
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may load or
 * call this code. The product library never does, and this file shares no code,
 * header, table or helper with it.
 *
 * What each step follows in the paper (arxiv 2605.30728):
 *   - ibpo_group_masks: Sec. 4.1 "Preprocessing" -- one counter per bit position,
 *     incremented for every set bit of every tensor; a counter at the upper
 *     threshold gives Mask 1 / Bitval 1, at the lower threshold Mask 1 / Bitval 0,
 *     anything else Mask 0 / Bitval 0 (Bitval bits under Mask 0 are kept 0). The
 *     threshold is T = n_g, the clustered form of Sec. 6.5 "Clustered Compression"
 *     with each cluster being G consecutive rows, so a bit is invariant exactly when
 *     its counter is 0 or n_g (inclusive reading of the threshold inequalities).
 *   - ibpo_packed_row_bytes: Sec. 4.2 "Compression", Fig. 4 size rule, with zero
 *     participation bits (under T = n_g every chunk matches Bitval, so the flag is
 *     always 1 and carries no information) and byte-aligned tensors:
 *     bytes = L - floor(popcount(Mask) / 8) = ceil((8L - popcount(Mask)) / 8).
 *   - ibpo_pack_row: Sec. 4.2 -- the invariant bits are removed and the remaining
 *     bits shifted together. Reading of the unspecified bit order: row bit p is bit
 *     (p mod 8) of byte floor(p / 8); the kept bits are emitted in ascending p and
 *     packed bit k goes to bit (k mod 8) of byte floor(k / 8); padding bits are 0.
 *   - ibpo_unpack_row: Sec. 4.3 "Decompression" -- rebuild the tensor by reinserting
 *     the removed bits: a Mask-1 position takes the Bitval bit, a Mask-0 position
 *     takes the next packed bit.
 *   - ibpo_compress / ibpo_decode_rows: the stream container (64-byte header, per
 *     group Mask then Bitval, a u64 offset index, then the packed rows back to back
 *     with no padding between rows, as the paper keeps tensors byte-aligned).
 *
 *
 * The thresholded scheme with participation bits (the paper's primary form, Sec. 4.1
 * and 4.2 with T < N), in the same container with header flag bit 0 set:
 *   - ibpo_thr_masks: Sec. 4.1 with a threshold T = (num/den) * n over the counters
 *     of the cluster's rows (or of every k-th row, a sampled Mask): counter >= T
 *     gives Mask 1 / Bitval 1, else n - counter >= T gives Mask 1 / Bitval 0, else
 *     Mask 0 / Bitval 0 (inclusive inequalities; 2 num > den so at most one holds).
 *   - ibpo_part_row_bytes: Sec. 4.2 and Fig. 4 -- a chunk of CS bytes is compressible
 *     when chunk AND Mask equals Bitval on all its bits; bits saved = the Mask bits of
 *     the compressible chunks; with one participation bit per chunk the bytes saved
 *     are floor((saved - chunks) / 8); a row that saves no byte is stored raw (L bytes,
 *     no participation bits), any other row takes L - bytes saved.
 *   - ibpo_part_pack_row: Sec. 4.2 -- the participation bits first (bit c set when
 *     chunk c is compressed), then chunk by chunk the row's bits in ascending order,
 *     skipping the Mask bits of compressed chunks; LSB-first, zero padding.
 *   - ibpo_part_unpack_row: Sec. 4.3 -- the reverse walk; a raw row is copied.
 *   - rows are addressed by a u64 offset per row (the paper keeps in-place slots and a
 *     compressed/raw bitmask, Sec. 5; here a row's size both locates it and tells a
 *     raw row, size L, from a compressed one, size < L).
 *
 * Parity status: every function here is pinned by tests (brute force on tiny
 * inputs, closed forms, identities and hand-derived worked examples).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define IBPO_HEADER_BYTES 64u

/* ---- bit access on little-endian byte strings ---------------------------- */

static int get_bit(const uint8_t *bytes, uint64_t p)
{
    return (bytes[p / 8] >> (p % 8)) & 1;
}

static void set_bit(uint8_t *bytes, uint64_t p, int v)
{
    if (v)
        bytes[p / 8] = (uint8_t)(bytes[p / 8] | (1u << (p % 8)));
    else
        bytes[p / 8] = (uint8_t)(bytes[p / 8] & ~(1u << (p % 8)));
}

static void put_u32(uint8_t *dst, uint32_t v)
{
    for (int i = 0; i < 4; ++i)
        dst[i] = (uint8_t)(v >> (8 * i));
}

static void put_u64(uint8_t *dst, uint64_t v)
{
    for (int i = 0; i < 8; ++i)
        dst[i] = (uint8_t)(v >> (8 * i));
}

static uint32_t get_u32(const uint8_t *src)
{
    uint32_t v = 0;
    for (int i = 0; i < 4; ++i)
        v |= (uint32_t)src[i] << (8 * i);
    return v;
}

static uint64_t get_u64(const uint8_t *src)
{
    uint64_t v = 0;
    for (int i = 0; i < 8; ++i)
        v |= (uint64_t)src[i] << (8 * i);
    return v;
}

/* ---- Sec. 4.1: Mask / Bitval of one cluster by per-bit counters ----------- */

void ibpo_group_masks(const uint8_t *rows, uint64_t n, uint32_t L,
                      uint8_t *mask, uint8_t *bitval)
{
    uint64_t nbits = 8ull * L;
    uint64_t *counter = (uint64_t *)calloc(nbits, sizeof(uint64_t));
    for (uint64_t i = 0; i < n; ++i)
        for (uint64_t p = 0; p < nbits; ++p)
            counter[p] += (uint64_t)get_bit(rows + i * L, p);
    memset(mask, 0, L);
    memset(bitval, 0, L);
    for (uint64_t p = 0; p < nbits; ++p) {
        if (counter[p] >= n) {          /* set in every row: invariant 1 */
            set_bit(mask, p, 1);
            set_bit(bitval, p, 1);
        } else if (counter[p] == 0) {   /* clear in every row: invariant 0 */
            set_bit(mask, p, 1);
        }                               /* else variant: Mask 0, Bitval 0 */
    }
    free(counter);
}

/* ---- Fig. 4 size rule, no participation bits ------------------------------ */

uint64_t ibpo_packed_row_bytes(const uint8_t *mask, uint32_t L)
{
    uint64_t saved = 0;
    for (uint64_t p = 0; p < 8ull * L; ++p)
        saved += (uint64_t)get_bit(mask, p);
    return (uint64_t)L - saved / 8;
}

/* ---- Sec. 4.2: remove the invariant bits and shift the rest together ------- */

void ibpo_pack_row(const uint8_t *row, const uint8_t *mask, uint32_t L, uint8_t *out)
{
    uint64_t rb = ibpo_packed_row_bytes(mask, L);
    memset(out, 0, rb);
    uint64_t k = 0;
    for (uint64_t p = 0; p < 8ull * L; ++p) {
        if (!get_bit(mask, p)) {
            set_bit(out, k, get_bit(row, p));
            ++k;
        }
    }
}

/* ---- Sec. 4.3: reinsert the removed bits ----------------------------------- */

void ibpo_unpack_row(const uint8_t *packed, const uint8_t *mask, const uint8_t *bitval,
                     uint32_t L, uint8_t *row)
{
    memset(row, 0, L);
    uint64_t k = 0;
    for (uint64_t p = 0; p < 8ull * L; ++p) {
        if (get_bit(mask, p)) {
            set_bit(row, p, get_bit(bitval, p));
        } else {
            set_bit(row, p, get_bit(packed, k));
            ++k;
        }
    }
}

/* ---- the stream container -------------------------------------------------- */

static uint64_t n_groups_of(uint64_t n_rows, uint32_t G)
{
    return (n_rows + G - 1) / G;
}

static uint64_t rows_in_group(uint64_t g, uint64_t n_rows, uint32_t G)
{
    uint64_t start = g * G;
    uint64_t end = start + G;
    if (end > n_rows)
        end = n_rows;
    return end - start;
}

/* Total stream bytes for these rows; 0 on bad arguments. */
uint64_t ibpo_stream_bytes(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G)
{
    if (L == 0 || L % 4 != 0 || G == 0)
        return 0;
    uint64_t ng = n_groups_of(n_rows, G);
    uint64_t total = IBPO_HEADER_BYTES + ng * 2ull * L + 8ull * (ng + 1);
    uint8_t *mask = (uint8_t *)malloc(L);
    uint8_t *bitval = (uint8_t *)malloc(L);
    for (uint64_t g = 0; g < ng; ++g) {
        uint64_t n = rows_in_group(g, n_rows, G);
        ibpo_group_masks(rows + g * G * (uint64_t)L, n, L, mask, bitval);
        total += n * ibpo_packed_row_bytes(mask, L);
    }
    free(mask);
    free(bitval);
    return total;
}

/*
 * Compress n_rows rows of L bytes in clusters of G rows. Returns 0 on success,
 * 1 on bad arguments, 2 if cap is too small. *out_bytes receives the size.
 */
int ibpo_compress(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G,
                  uint8_t *out, uint64_t cap, uint64_t *out_bytes)
{
    if (L == 0 || L % 4 != 0 || G == 0)
        return 1;
    uint64_t total = ibpo_stream_bytes(rows, n_rows, L, G);
    *out_bytes = total;
    if (total > cap)
        return 2;
    uint64_t ng = n_groups_of(n_rows, G);
    uint64_t meta_off = IBPO_HEADER_BYTES;
    uint64_t index_off = meta_off + ng * 2ull * L;
    uint64_t payload_off = index_off + 8ull * (ng + 1);

    memset(out, 0, IBPO_HEADER_BYTES);
    memcpy(out, "IBP1", 4);
    put_u32(out + 4, 1);
    put_u32(out + 8, L);
    put_u32(out + 12, G);
    put_u64(out + 16, n_rows);
    put_u64(out + 24, ng);
    put_u32(out + 32, 0);
    put_u32(out + 36, 0);
    put_u64(out + 40, meta_off);
    put_u64(out + 48, index_off);
    put_u64(out + 56, payload_off);

    uint64_t off = 0;
    for (uint64_t g = 0; g < ng; ++g) {
        uint64_t n = rows_in_group(g, n_rows, G);
        const uint8_t *grows = rows + g * G * (uint64_t)L;
        uint8_t *mask = out + meta_off + g * 2ull * L;
        uint8_t *bitval = mask + L;
        ibpo_group_masks(grows, n, L, mask, bitval);
        uint64_t rb = ibpo_packed_row_bytes(mask, L);
        put_u64(out + index_off + 8 * g, off);
        for (uint64_t r = 0; r < n; ++r)
            ibpo_pack_row(grows + r * L, mask, L, out + payload_off + off + r * rb);
        off += n * rb;
    }
    put_u64(out + index_off + 8 * ng, off);
    return 0;
}

/*
 * Decode rows ids[0..n_ids) of a stream into out (n_ids * L bytes).
 * Returns 0 on success, 1 on a malformed header, 2 on an id out of range.
 */
int ibpo_decode_rows(const uint8_t *stream, uint64_t stream_bytes,
                     const int64_t *ids, uint64_t n_ids, uint8_t *out)
{
    if (stream_bytes < IBPO_HEADER_BYTES || memcmp(stream, "IBP1", 4) != 0 ||
        get_u32(stream + 4) != 1)
        return 1;
    uint32_t L = get_u32(stream + 8);
    uint32_t G = get_u32(stream + 12);
    uint64_t n_rows = get_u64(stream + 16);
    uint64_t meta_off = get_u64(stream + 40);
    uint64_t index_off = get_u64(stream + 48);
    uint64_t payload_off = get_u64(stream + 56);
    if (L == 0 || G == 0)
        return 1;
    for (uint64_t i = 0; i < n_ids; ++i) {
        if (ids[i] < 0 || (uint64_t)ids[i] >= n_rows)
            return 2;
        uint64_t id = (uint64_t)ids[i];
        uint64_t g = id / G;
        uint64_t r = id % G;
        const uint8_t *mask = stream + meta_off + g * 2ull * L;
        const uint8_t *bitval = mask + L;
        uint64_t rb = ibpo_packed_row_bytes(mask, L);
        uint64_t off = get_u64(stream + index_off + 8 * g);
        ibpo_unpack_row(stream + payload_off + off + r * rb, mask, bitval, L, out + i * L);
    }
    return 0;
}


/* ======================= thresholded scheme with participation bits ========== */

#define IBPO_FLAG_PARTICIPATION 1u

/* Sec. 4.1 with T = (num/den) * n, over rows 0, every, 2*every, ... of the cluster. */
void ibpo_thr_masks(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t num,
                    uint32_t den, uint32_t every, uint8_t *mask, uint8_t *bitval)
{
    uint64_t nbits = 8ull * L;
    uint64_t *counter = (uint64_t *)calloc(nbits, sizeof(uint64_t));
    uint64_t n = 0;
    for (uint64_t i = 0; i < n_rows; i += every) {
        for (uint64_t p = 0; p < nbits; ++p)
            counter[p] += (uint64_t)get_bit(rows + i * L, p);
        ++n;
    }
    memset(mask, 0, L);
    memset(bitval, 0, L);
    for (uint64_t p = 0; p < nbits; ++p) {
        /* counter >= T  <=>  counter * den >= num * n (exact in integers) */
        if (counter[p] * den >= (uint64_t)num * n) {
            set_bit(mask, p, 1);
            set_bit(bitval, p, 1);
        } else if ((n - counter[p]) * den >= (uint64_t)num * n) {
            set_bit(mask, p, 1);
        }
    }
    free(counter);
}

/* Is chunk c (CS bytes) of the row compressible: row AND Mask == Bitval on it? */
static int chunk_matches(const uint8_t *row, const uint8_t *mask, const uint8_t *bitval,
                         uint32_t CS, uint64_t c)
{
    for (uint64_t p = 8ull * CS * c; p < 8ull * CS * (c + 1); ++p)
        if (get_bit(mask, p) && get_bit(row, p) != get_bit(bitval, p))
            return 0;
    return 1;
}

/* Bytes of one row in the participation scheme (L when stored raw). */
uint64_t ibpo_part_row_bytes(const uint8_t *row, const uint8_t *mask, const uint8_t *bitval,
                             uint32_t L, uint32_t CS)
{
    uint64_t chunks = L / CS;
    uint64_t saved = 0;
    for (uint64_t c = 0; c < chunks; ++c) {
        if (!chunk_matches(row, mask, bitval, CS, c))
            continue;
        for (uint64_t p = 8ull * CS * c; p < 8ull * CS * (c + 1); ++p)
            saved += (uint64_t)get_bit(mask, p);
    }
    if (saved < chunks + 8)       /* bytes saved = floor((saved - chunks) / 8) <= 0 */
        return L;
    return (uint64_t)L - (saved - chunks) / 8;
}

void ibpo_part_pack_row(const uint8_t *row, const uint8_t *mask, const uint8_t *bitval,
                        uint32_t L, uint32_t CS, uint8_t *out)
{
    uint64_t size = ibpo_part_row_bytes(row, mask, bitval, L, CS);
    if (size == L) {
        memcpy(out, row, L);
        return;
    }
    uint64_t chunks = L / CS;
    memset(out, 0, size);
    uint64_t k = 0;
    for (uint64_t c = 0; c < chunks; ++c)
        set_bit(out, k++, chunk_matches(row, mask, bitval, CS, c));
    for (uint64_t c = 0; c < chunks; ++c) {
        int comp = chunk_matches(row, mask, bitval, CS, c);
        for (uint64_t p = 8ull * CS * c; p < 8ull * CS * (c + 1); ++p) {
            if (comp && get_bit(mask, p))
                continue;
            set_bit(out, k++, get_bit(row, p));
        }
    }
}

void ibpo_part_unpack_row(const uint8_t *packed, uint64_t size, const uint8_t *mask,
                          const uint8_t *bitval, uint32_t L, uint32_t CS, uint8_t *row)
{
    if (size == L) {
        memcpy(row, packed, L);
        return;
    }
    uint64_t chunks = L / CS;
    memset(row, 0, L);
    uint64_t k = chunks;
    for (uint64_t c = 0; c < chunks; ++c) {
        int comp = get_bit(packed, c);
        for (uint64_t p = 8ull * CS * c; p < 8ull * CS * (c + 1); ++p) {
            if (comp && get_bit(mask, p))
                set_bit(row, p, get_bit(bitval, p));
            else
                set_bit(row, p, get_bit(packed, k++));
        }
    }
}

static int part_args_ok(uint32_t L, uint32_t G, uint32_t CS, uint32_t num, uint32_t den,
                        uint32_t every)
{
    return L != 0 && L % 4 == 0 && G != 0 && CS != 0 && CS % 4 == 0 && L % CS == 0 &&
           den != 0 && num <= den && 2ull * num > den && every != 0;
}

/* Stream bytes of the participation scheme; 0 on bad arguments. */
uint64_t ibpo_part_stream_bytes(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G,
                                uint32_t CS, uint32_t num, uint32_t den, uint32_t every)
{
    if (!part_args_ok(L, G, CS, num, den, every))
        return 0;
    uint64_t ng = n_groups_of(n_rows, G);
    uint64_t total = IBPO_HEADER_BYTES + ng * 2ull * L + 8ull * (n_rows + 1);
    uint8_t *mask = (uint8_t *)malloc(L);
    uint8_t *bitval = (uint8_t *)malloc(L);
    for (uint64_t g = 0; g < ng; ++g) {
        uint64_t n = rows_in_group(g, n_rows, G);
        const uint8_t *grows = rows + g * G * (uint64_t)L;
        ibpo_thr_masks(grows, n, L, num, den, every, mask, bitval);
        for (uint64_t r = 0; r < n; ++r)
            total += ibpo_part_row_bytes(grows + r * L, mask, bitval, L, CS);
    }
    free(mask);
    free(bitval);
    return total;
}

/*
 * Compress in the participation scheme: header flags = 1 and the chunk bytes in the
 * header word at offset 36, per cluster Mask then Bitval, a u64 offset per row
 * (n_rows + 1 entries), then the rows back to back. Returns 0, 1 (bad arguments)
 * or 2 (cap too small).
 */
int ibpo_part_compress(const uint8_t *rows, uint64_t n_rows, uint32_t L, uint32_t G,
                       uint32_t CS, uint32_t num, uint32_t den, uint32_t every,
                       uint8_t *out, uint64_t cap, uint64_t *out_bytes)
{
    if (!part_args_ok(L, G, CS, num, den, every))
        return 1;
    uint64_t total = ibpo_part_stream_bytes(rows, n_rows, L, G, CS, num, den, every);
    *out_bytes = total;
    if (total > cap)
        return 2;
    uint64_t ng = n_groups_of(n_rows, G);
    uint64_t meta_off = IBPO_HEADER_BYTES;
    uint64_t index_off = meta_off + ng * 2ull * L;
    uint64_t payload_off = index_off + 8ull * (n_rows + 1);

    memset(out, 0, IBPO_HEADER_BYTES);
    memcpy(out, "IBP1", 4);
    put_u32(out + 4, 1);
    put_u32(out + 8, L);
    put_u32(out + 12, G);
    put_u64(out + 16, n_rows);
    put_u64(out + 24, ng);
    put_u32(out + 32, IBPO_FLAG_PARTICIPATION);
    put_u32(out + 36, CS);
    put_u64(out + 40, meta_off);
    put_u64(out + 48, index_off);
    put_u64(out + 56, payload_off);

    uint64_t off = 0;
    for (uint64_t g = 0; g < ng; ++g) {
        uint64_t n = rows_in_group(g, n_rows, G);
        const uint8_t *grows = rows + g * G * (uint64_t)L;
        uint8_t *mask = out + meta_off + g * 2ull * L;
        uint8_t *bitval = mask + L;
        ibpo_thr_masks(grows, n, L, num, den, every, mask, bitval);
        for (uint64_t r = 0; r < n; ++r) {
            put_u64(out + index_off + 8 * (g * (uint64_t)G + r), off);
            ibpo_part_pack_row(grows + r * L, mask, bitval, L, CS, out + payload_off + off);
            off += ibpo_part_row_bytes(grows + r * L, mask, bitval, L, CS);
        }
    }
    put_u64(out + index_off + 8 * n_rows, off);
    return 0;
}

/* Decode rows of a participation-scheme stream. Returns 0, 1 (malformed) or 2 (range). */
int ibpo_part_decode_rows(const uint8_t *stream, uint64_t stream_bytes,
                          const int64_t *ids, uint64_t n_ids, uint8_t *out)
{
    if (stream_bytes < IBPO_HEADER_BYTES || memcmp(stream, "IBP1", 4) != 0 ||
        get_u32(stream + 4) != 1 || get_u32(stream + 32) != IBPO_FLAG_PARTICIPATION)
        return 1;
    uint32_t L = get_u32(stream + 8);
    uint32_t G = get_u32(stream + 12);
    uint64_t n_rows = get_u64(stream + 16);
    uint32_t CS = get_u32(stream + 36);
    uint64_t meta_off = get_u64(stream + 40);
    uint64_t index_off = get_u64(stream + 48);
    uint64_t payload_off = get_u64(stream + 56);
    if (L == 0 || G == 0 || CS == 0 || L % CS != 0)
        return 1;
    for (uint64_t i = 0; i < n_ids; ++i) {
        if (ids[i] < 0 || (uint64_t)ids[i] >= n_rows)
            return 2;
        uint64_t id = (uint64_t)ids[i];
        uint64_t g = id / G;
        const uint8_t *mask = stream + meta_off + g * 2ull * L;
        const uint8_t *bitval = mask + L;
        uint64_t o0 = get_u64(stream + index_off + 8 * id);
        uint64_t o1 = get_u64(stream + index_off + 8 * (id + 1));
        ibpo_part_unpack_row(stream + payload_off + o0, o1 - o0, mask, bitval, L, CS, out + i * L);
    }
    return 0;
}
