// gfx950 decompression kernels of Invariant Bit Packing.
//
// The paper decodes one tensor per warp (Sec. 4.3): each thread takes a chunk, counts
// the unset Mask bits of its chunk, an exclusive scan over the warp gives every chunk's
// starting bit, and each thread then pulls its bits out of a shared workspace. The
// kernels here keep that structure, shaped for CDNA4 wave64 and for clusters of rows
// sharing one Mask/Bitval:
//
//   * one wave owns a cluster (decompress) or a segment of requested rows (gather);
//     lane t owns the 32-bit words t, t+64, t+128, ... of a row, so every output store
//     of the wave is 64 consecutive dwords (256 B, fully coalesced);
//   * per cluster, each lane loads Mask/Bitval for its words, counts n_w =
//     popcount(~Mask_w), and a wave inclusive scan built from DPP row shifts and row
//     broadcasts turns the counts into bit offsets S_w inside a packed row. Under the
//     cluster threshold T = cluster size the offsets depend only on the Mask, so they
//     are computed once per cluster and reused for all of its rows;
//   * per cluster, each word's variant positions (~Mask_w) are split into runs of
//     consecutive bits; a run is placed by one funnel rotate (v_alignbit) and one
//     and-or, so rebuilding a word is: funnel-shift its 32-bit window out of two
//     packed dwords, then Bitval_w | sum over runs of (rotr(x, r_k) & run_k). Words
//     with more runs than the register budget take a generic bit-run loop;
//   * packed rows are byte-aligned and of any length, so a word's window is read as
//     two dwords at its bit offset and funnel-shifted (v_alignbit_b32), never with
//     sub-dword loads. No MFMA anywhere: nothing here is a contraction.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "ibp_device.hpp"
#include "ibp_wave.hpp"

namespace ibp {
namespace dev {

namespace {


// Per-wave decode state for one tile of a row (64*K words) of one cluster.
template <int K, int MAXR>
struct Tile {
    uint32_t bv[K];          // Bitval of the lane's words
    uint32_t nm[K];          // ~Mask: the variant positions
    uint32_t s[K];           // bit offset of the word inside the packed row
    uint32_t pk[K];          // packed width popcount(~Mask) (0 past the row's end)
    uint32_t rot[K][MAXR];   // rotate-right amount that lands run k at its position
    uint32_t rm[K][MAXR];    // run k's bits in place
    uint32_t bits;           // packed bits of this tile (wave-uniform)
    int nr;                  // runs applied per word (uniform); -1 = generic loop
};

template <int K, int MAXR>
__device__ __forceinline__ void tile_setup(Tile<K, MAXR> &t, const uint32_t *__restrict__ mg,
                                           uint32_t W, uint32_t w0, uint32_t carry) {
    const uint32_t l = lane_id();
    uint32_t c = carry;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const uint32_t w = w0 + l + kWave * j;
        uint32_t m = 0xFFFFFFFFu, b = 0u;
        if (w < W) {
            m = mg[w];
            b = mg[W + w];
        }
        t.nm[j] = ~m;
        t.bv[j] = b;
        const uint32_t n = (uint32_t)__builtin_popcount(~m);
        t.pk[j] = n;
        const uint32_t inc = wave_incl_scan(n);
        t.s[j] = c + inc - n;
        c += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
    }
    t.bits = c - carry;

    int cnt_max = 0;
    bool rest = false;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        uint32_t v = t.nm[j];
        uint32_t so = 0;
        int cnt = 0;
#pragma unroll
        for (int k = 0; k < MAXR; ++k) {
            const uint32_t low = v & (0u - v);
            const uint32_t tt = v + low;      // carries through the lowest run
            const uint32_t run = v & ~tt;
            v &= tt;
            const uint32_t lo = (uint32_t)__builtin_ctz(run | 0x80000000u);
            t.rot[j][k] = (so - lo) & 31u;
            t.rm[j][k] = run;
            so += (uint32_t)__builtin_popcount(run);
            cnt += run != 0u;
        }
        cnt_max = cnt > cnt_max ? cnt : cnt_max;
        rest = rest || v != 0u;
    }
    if (__any(rest)) {
        t.nr = -1;
    } else {
        int nr = 0;
#pragma unroll
        for (int k = 0; k < MAXR; ++k)
            if (__any(cnt_max > k)) nr = k + 1;
        t.nr = nr;
    }
}

// Rebuild one word from its 32-bit window x: Bitval | the NR runs of variant bits.
template <int NR, int K, int MAXR>
__device__ __forceinline__ uint32_t word_fast(const Tile<K, MAXR> &t, int j, uint32_t x) {
    uint32_t acc = t.bv[j];
#pragma unroll
    for (int k = 0; k < NR; ++k) acc |= __builtin_amdgcn_alignbit(x, x, t.rot[j][k]) & t.rm[j][k];
    return acc;
}

// Generic rebuild for any Mask: walk the runs of ~Mask from the lowest bit up.
__device__ __forceinline__ uint32_t word_generic(uint32_t bv, uint32_t nm, uint32_t x) {
    uint32_t acc = bv, v = nm;
    while (v) {
        const uint32_t low = v & (0u - v);
        const uint32_t tt = v + low;
        const uint32_t run = v & ~tt;
        v &= tt;
        acc |= (x << __builtin_ctz(run)) & run;
        x = __builtin_amdgcn_alignbit(0u, x, (uint32_t)__builtin_popcount(run));
    }
    return acc;
}

// Decode RB rows of one cluster. `at.byte(i)` is the payload byte where row i's packed
// bits start and `at.out(i)` the row's output; both are wave-uniform. All loads of the
// batch are issued before any word is rebuilt, so RB*K loads are in flight per wave.
// NR >= 0 applies NR precomputed runs per word; NR < 0 takes the generic loop.
template <int NR, int RB, int K, int MAXR, class At>
__device__ __forceinline__ void decode_batch(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                             const At &at, uint32_t W, uint32_t w0) {
    const uint32_t l = lane_id();
    uint32_t d0[RB][K], d1[RB][K], b[RB][K];
#pragma unroll
    for (int i = 0; i < RB; ++i) {
        const uint64_t rbyte = at.byte(i);
        const uint32_t *__restrict__ p = pay32 + (rbyte >> 2);
        const uint32_t bit0 = ((uint32_t)rbyte & 3u) * 8u;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            b[i][j] = bit0 + t.s[j];
            if constexpr (At::kSplit) {
                load_window(p, b[i][j] >> 5, d0[i][j], d1[i][j]);
            } else {
                d0[i][j] = p[b[i][j] >> 5];
                d1[i][j] = p[(b[i][j] >> 5) + 1];
            }
        }
    }
#pragma unroll
    for (int i = 0; i < RB; ++i) {
        uint32_t *__restrict__ o = at.out(i);
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t x = __builtin_amdgcn_alignbit(d1[i][j], d0[i][j], b[i][j]);
            uint32_t v;
            if constexpr (NR >= 0) v = word_fast<NR>(t, j, x);
            else v = word_generic(t.bv[j], t.nm[j], x);
            const uint32_t w = w0 + l + kWave * j;
            if (w < W) o[w] = v;   // plain store: streamed output, measured 7% faster than non-temporal
        }
    }
}

// Decode rows [0, n) of one cluster with the run count fixed at compile time.
template <int NR, int K, int MAXR, class At>
__device__ __forceinline__ void decode_rows_nr(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                               uint32_t n, const At &at, uint32_t W, uint32_t w0) {
    constexpr int RB = K <= 1 ? 8 : (K <= 2 ? 4 : (K <= 4 ? 2 : 1));
    uint32_t k = 0;
    for (; k + RB <= n; k += RB) decode_batch<NR, RB>(t, pay32, at.shifted(k), W, w0);
    for (; k < n; ++k) decode_batch<NR, 1>(t, pay32, at.shifted(k), W, w0);
}

template <int K, int MAXR, class At>
__device__ __forceinline__ void decode_rows(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                            uint32_t n, const At &at, uint32_t W, uint32_t w0) {
    switch (t.nr) {   // wave-uniform
    case 0: decode_rows_nr<0>(t, pay32, n, at, W, w0); break;
    case 1: decode_rows_nr<1>(t, pay32, n, at, W, w0); break;
    case 2: if constexpr (MAXR >= 2) decode_rows_nr<2>(t, pay32, n, at, W, w0); break;
    case 3: if constexpr (MAXR >= 3) decode_rows_nr<3>(t, pay32, n, at, W, w0); break;
    case 4: if constexpr (MAXR >= 4) decode_rows_nr<4>(t, pay32, n, at, W, w0); break;
    default: decode_rows_nr<-1>(t, pay32, n, at, W, w0); break;
    }
}

// Rows of a contiguous slice: row i at byte base + i*rb, output out0 + i*W. SPLIT: each
// window as two dword loads (payload in device memory); else one 8-byte load (payload in
// pinned host memory: its reads bypass the L2, so two loads would send each line over
// PCIe twice; measured on a zero-copy KV layer, 0.94 merged against 0.89 split of CR x raw).
template <bool SPLIT>
struct SliceAt {
    static constexpr bool kSplit = SPLIT;
    uint64_t base, rb;
    uint32_t *out0;
    uint32_t W;
    __device__ uint64_t byte(int i) const { return base + (uint64_t)i * rb; }
    __device__ uint32_t *out(int i) const { return out0 + (uint64_t)i * W; }
    __device__ SliceAt shifted(uint32_t k) const { return {base + k * rb, rb, out0 + (uint64_t)k * W, W}; }
};

// Rows of a run of gathered ids from one cluster: the row index inside the cluster
// (or the staged byte offset) of request i0+i sits in lane i0+i of `rloc`.
struct GatherAt {
    static constexpr bool kSplit = false;
    uint64_t base, rb;       // cluster payload byte and packed row bytes (device payload)
    uint32_t *seg_out;       // output row of request 0 of the wave's segment
    uint32_t W;
    uint32_t i0;             // first request of this run, relative to the segment
    uint32_t rloc;           // per lane: row inside the cluster, or staged byte offset
    bool staged;
    __device__ uint64_t byte(int i) const {
        const uint32_t v = (uint32_t)__builtin_amdgcn_readlane((int)rloc, (int)(i0 + i));
        return staged ? (uint64_t)v : base + (uint64_t)v * rb;
    }
    __device__ uint32_t *out(int i) const { return seg_out + (uint64_t)(i0 + i) * W; }
    __device__ GatherAt shifted(uint32_t k) const {
        GatherAt a = *this;
        a.i0 += k;
        return a;
    }
};

// Packed bits of a full row of the cluster whose metadata starts at mg.
__device__ __forceinline__ uint32_t row_bits(const uint32_t *__restrict__ mg, uint32_t W) {
    uint32_t n = 0;
    for (uint32_t w = lane_id(); w < W; w += kWave) n += (uint32_t)__builtin_popcount(~mg[w]);
    return wave_sum(n);
}

// Decode n rows of a cluster whose rows span several tiles: tile by tile, each tile's
// setup carrying the bit offset of the tiles before it.
template <int K, int MAXR, class At>
__device__ __forceinline__ void decode_rows_tiled(const uint32_t *__restrict__ mg,
                                                  const uint32_t *__restrict__ pay32, uint32_t n,
                                                  const At &at, uint32_t W) {
    uint32_t carry = 0;
    for (uint32_t w0 = 0; w0 < W; w0 += kWave * K) {
        Tile<K, MAXR> t;
        tile_setup(t, mg, W, w0, carry);
        decode_rows(t, pay32, n, at, W, w0);
        carry += t.bits;
    }
}


// One wave per unit = (cluster, slice of at most rpu rows of it).
template <int K, int MAXR, bool SPLIT>
__global__ __launch_bounds__(kBlock) void k_decompress(DevStream s, const uint32_t *__restrict__ pay32,
                                                        uint64_t pay_base, uint32_t *__restrict__ out,
                                                        uint64_t first, uint64_t n, uint64_t g0,
                                                        uint64_t n_units, uint32_t upg, uint32_t rpu) {
    const uint64_t unit = wave_slot();
    if (unit >= n_units) return;
    const uint64_t g = g0 + unit / upg;
    const uint64_t gstart = g * s.G;
    uint64_t r_lo = gstart + (unit % upg) * (uint64_t)rpu;
    uint64_t r_hi = min(r_lo + rpu, min(gstart + s.G, s.n_rows));
    r_lo = max(r_lo, first);
    r_hi = min(r_hi, first + n);
    if (r_lo >= r_hi) return;
    const uint32_t W = s.W;
    const uint32_t *__restrict__ mg = s.meta + g * 2ull * W;
    const uint64_t base = s.index[g] - pay_base;
    const uint32_t rows = (uint32_t)(r_hi - r_lo);
    if (W <= (uint32_t)(kWave * K)) {
        Tile<K, MAXR> t;
        tile_setup(t, mg, W, 0, 0);
        const uint64_t rb = row_stride((t.bits + 7u) >> 3, s.row_align);
        const SliceAt<SPLIT> at{base + (r_lo - gstart) * rb, rb, out + (r_lo - first) * W, W};
        decode_rows(t, pay32, rows, at, W, 0);
    } else {
        const uint64_t rb = row_stride((row_bits(mg, W) + 7u) >> 3, s.row_align);
        const SliceAt<SPLIT> at{base + (r_lo - gstart) * rb, rb, out + (r_lo - first) * W, W};
        decode_rows_tiled<K, MAXR>(mg, pay32, rows, at, W);
    }
}

// Gather of rows wider than one tile (W > 512 words). One wave per segment of up to 64
// requests; lane i loads request i's id; runs of consecutive requests that fall in the
// same cluster (sorted ids) share one setup, and each row is decoded tile by tile.
template <int K, int MAXR, bool STAGED>
__global__ __launch_bounds__(kBlock) void k_gather_tiled(DevStream s, const uint32_t *__restrict__ pay32,
                                                    const int64_t *__restrict__ ids,
                                                    const uint32_t *__restrict__ sg,
                                                    const uint32_t *__restrict__ soff, uint64_t n,
                                                    uint32_t *__restrict__ out, uint32_t seg,
                                                    unsigned long long *err) {
    const uint64_t i0 = wave_slot() * seg;
    if (i0 >= n) return;
    const uint32_t cnt = (uint32_t)min((uint64_t)seg, n - i0);
    const uint32_t l = lane_id();
    const uint32_t W = s.W;
    bool valid;
    uint64_t g_l;
    uint32_t r_l = 0, so = 0;
    if constexpr (STAGED) {
        valid = l < cnt;
        g_l = valid ? sg[i0 + l] : 0u;
        so = valid ? soff[i0 + l] : 0u;
    } else {
        const int64_t id = l < cnt ? ids[i0 + l] : -1;
        valid = l < cnt && id >= 0 && (uint64_t)id < s.n_rows;
        const uint64_t uid = valid ? (uint64_t)id : 0;
        g_l = s.G == 1 ? uid : __umul64hi(uid, s.g_magic);
        r_l = (uint32_t)(uid - g_l * s.G);
    }
    const uint64_t bad = __ballot(l < cnt && !valid);
    uint32_t *__restrict__ out_seg = out + i0 * W;
    if (bad) {
        // zero the rows of out-of-range ids and count them
        for (uint32_t i = 0; i < cnt; ++i) {
            if ((bad >> i) & 1ull) {
                for (uint32_t w = l; w < W; w += kWave) out_seg[(uint64_t)i * W + w] = 0u;
            }
        }
        if (l == 0) atomicAdd(err, (unsigned long long)__popcll(bad));
    }
    const uint32_t g_lo = (uint32_t)g_l, g_hi = (uint32_t)(g_l >> 32);
    uint32_t i = 0;
    while (i < cnt) {
        if ((bad >> i) & 1ull) {
            ++i;
            continue;
        }
        const uint32_t gl = (uint32_t)__builtin_amdgcn_readlane((int)g_lo, (int)i);
        const uint32_t gh = (uint32_t)__builtin_amdgcn_readlane((int)g_hi, (int)i);
        const uint64_t g = ((uint64_t)gh << 32) | gl;
        // end of the run: first later request in another cluster, invalid, or past cnt
        const uint64_t other = __ballot(l >= cnt || !valid || g_lo != gl || g_hi != gh);
        const uint64_t later = other & ~((2ull << i) - 1ull);
        const uint32_t end = later ? (uint32_t)__builtin_ctzll(later) : cnt;
        const uint32_t *__restrict__ mg = s.meta + g * 2ull * W;
        GatherAt at{0, 0, out_seg, W, i, STAGED ? so : r_l, STAGED};
        if (W <= (uint32_t)(kWave * K)) {
            Tile<K, MAXR> t;
            tile_setup(t, mg, W, 0, 0);
            at.rb = row_stride((t.bits + 7u) >> 3, s.row_align);
            if constexpr (!STAGED) at.base = s.index[g];
            decode_rows(t, pay32, end - i, at, W, 0);
        } else {
            at.rb = row_stride((row_bits(mg, W) + 7u) >> 3, s.row_align);
            if constexpr (!STAGED) at.base = s.index[g];
            decode_rows_tiled<K, MAXR>(mg, pay32, end - i, at, W);
        }
        i = end;
    }
}

// Gather of rows that fit one tile (W <= 64*K), built for memory-level parallelism.
// A wave owns `seg` requests (lane i loads request i's id and cluster offset, once) and
// decodes them RB rows at a time, each row independently: its cluster's metadata (compact
// slot or Mask/Bitval words), a wave scan of popcount(~Mask) for the bit offsets, then its
// packed windows. All metadata loads of a batch leave together, then all its window loads;
// a row in its predecessor's cluster (also the previous batch's last row) loads no
// metadata and reuses that row's setup.
// One batch per wave measured fastest at the gathers' sizes: prefetching the next batch's
// metadata during the current batch's windows keeps its registers live through the
// rebuild, and the lost occupancy costs more than the overlap gains. Rows are rebuilt with
// the holes deposit: with a setup per row, precomputed runs would cost more than they
// save.
template <int K, int RB, bool STAGED, int FORM>
__global__ __launch_bounds__(kBlock) void k_gather_rows(DevStream s, const uint32_t *__restrict__ pay32,
                                                         const int64_t *__restrict__ ids,
                                                         const uint32_t *__restrict__ sg,
                                                         const uint32_t *__restrict__ soff, uint64_t n,
                                                         uint32_t *__restrict__ out, uint32_t seg,
                                                         unsigned long long *err) {
    const uint64_t slot = (uint64_t)xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock +
                          (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
    const uint64_t i0 = slot * seg;
    if (i0 >= n) return;
    const uint32_t cnt = (uint32_t)min((uint64_t)seg, n - i0);
    const uint32_t l = lane_id();
    const uint32_t W = s.W;
    // lane l < cnt holds request l: its cluster g_l and row r_l inside the cluster (or,
    // for staged rows, the byte offset `so` of its packed bits)
    bool valid;
    uint64_t g_l;
    uint32_t r_l = 0, so = 0;
    if constexpr (STAGED) {
        valid = l < cnt;
        g_l = valid ? sg[i0 + l] : 0u;
        so = valid ? soff[i0 + l] : 0u;
    } else {
        const int64_t id = l < cnt ? ids[i0 + l] : -1;
        valid = l < cnt && id >= 0 && (uint64_t)id < s.n_rows;
        const uint64_t uid = valid ? (uint64_t)id : 0;
        g_l = s.G == 1 ? uid : __umul64hi(uid, s.g_magic);
        r_l = (uint32_t)(uid - g_l * s.G);
    }
    const uint32_t g_lo = (uint32_t)g_l, g_hi = (uint32_t)(g_l >> 32);
    // each lane fetches its request's cluster offset once, so rows never wait on an
    // index load of their own
    uint64_t off_l = 0;
    if constexpr (!STAGED) off_l = s.index[g_l];
    const uint32_t off_lo = (uint32_t)off_l, off_hi = (uint32_t)(off_l >> 32);
    const uint64_t bad = __ballot(l < cnt && !valid);
    const uint64_t okm = __ballot(l < cnt && valid);   // requests whose rows are stored
    // requests whose cluster is the previous request's (sorted ids put them together)
    const uint32_t prev = (l ? l - 1u : 0u) * 4u;
    const uint32_t pg_lo = (uint32_t)__builtin_amdgcn_ds_bpermute((int)prev, (int)g_lo);
    const uint32_t pg_hi = (uint32_t)__builtin_amdgcn_ds_bpermute((int)prev, (int)g_hi);
    const uint64_t samep = __ballot(l > 0 && pg_lo == g_lo && pg_hi == g_hi);
    uint32_t *__restrict__ out_seg = out + i0 * W;
    if (bad) {
        for (uint32_t i = 0; i < cnt; ++i)
            if ((bad >> i) & 1ull)
                for (uint32_t w = l; w < W; w += kWave) out_seg[(uint64_t)i * W + w] = 0u;
        if (l == 0) atomicAdd(err, (unsigned long long)__popcll(bad));
    }
    auto rd64 = [](uint32_t lo, uint32_t hi, uint32_t i) -> uint64_t {
        return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, (int)i) << 32) |
               (uint32_t)__builtin_amdgcn_readlane((int)lo, (int)i);
    };
    // request slot i of the segment; slots past the end repeat the last request (their
    // loads stay in bounds and their stores are skipped)
    auto slot_of = [&](uint32_t i) { return i < cnt ? i : cnt - 1; };
    const uint32_t nb = (cnt + RB - 1) / RB;
    // rebuilt words of the previous batch: stored once the next batch's metadata loads have
    // left, so waiting for that metadata never waits for those stores
    uint32_t pv[RB][K];
    uint32_t pbase = 0;
    bool pending = false;
    auto store_pending = [&]() {
        if (!pending) return;
#pragma unroll
        for (int u = 0; u < RB; ++u) {
            const uint32_t i = pbase + u;
            const bool row_ok = (okm >> (i & 63)) & 1ull;
            uint32_t *__restrict__ orow = out_seg + (uint64_t)i * W;
#pragma unroll
            for (int j = 0; j < K; ++j) {
                const uint32_t w = l + kWave * j;
                if (row_ok && w < W) store_out(&orow[w], pv[u][j]);
            }
        }
        pending = false;
    };
    // the setup of the previous batch's last row, for a batch whose first row shares its
    // cluster (sorted ids often continue a cluster across the batch boundary)
    uint32_t c_nm[K] = {}, c_bv[K] = {}, c_ofs[K] = {}, c_nh = 0, c_tot = 0;
    for (uint32_t bb = 0; bb < nb; ++bb) {
        const uint32_t base_i = bb * RB;
        RowMeta<K, FORM> meta[RB];
        // a row whose cluster is its predecessor's in the batch reuses that row's setup
        // below, so only the batch's first row of each cluster loads the metadata
#pragma unroll
        for (int u = 0; u < RB; ++u) {
            // base_i + u > 0: samep's bit compares the request with the one before it, which
            // for u = 0 is the previous batch's last row
            const bool same = base_i + u > 0 && (base_i + u >= cnt || ((samep >> ((base_i + u) & 63)) & 1ull));
            if (same) {
#pragma unroll
                for (int k = 0; k < (int)(sizeof(meta[u].v) / sizeof(meta[u].v[0])); ++k) meta[u].v[k] = 0u;
                continue;
            }
            const uint64_t g = rd64(g_lo, g_hi, slot_of(base_i + u));
            load_row_meta<K, FORM>(meta[u], s.meta + g * 2ull * W, s.slots + g * s.slot_bytes, s.slot_pairs, W);
        }
        store_pending();
#pragma unroll
        for (int u = 0; u < RB; ++u) hold_row_meta(meta[u]);
        // per row: variant positions, Bitval, bit offsets of the words inside the packed
        // row (without the row's byte misalignment bit0), hole iterations, packed bits
        uint32_t nm[RB][K], bv[RB][K], ofs[RB][K], d0[RB][K], d1[RB][K], nh[RB], tot[RB], bit0[RB];
#pragma unroll
        for (int u = 0; u < RB; ++u) {
            const int up = u > 0 ? u - 1 : 0;
            const uint32_t i = slot_of(base_i + u);
            // sorted ids put rows of one cluster next to each other: a row whose cluster
            // is its predecessor's reuses that row's offsets and hole count (uniform branch;
            // slots past the end repeat the last request, so they always do)
            const bool same = base_i + u > 0 && (base_i + u >= cnt || ((samep >> ((base_i + u) & 63)) & 1ull));
            if (same && u == 0) {
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    nm[u][j] = c_nm[j];
                    bv[u][j] = c_bv[j];
                    ofs[u][j] = c_ofs[j];
                }
                nh[u] = c_nh;
                tot[u] = c_tot;
            } else if (same) {
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    nm[u][j] = nm[up][j];
                    bv[u][j] = bv[up][j];
                    ofs[u][j] = ofs[up][j];
                }
                nh[u] = nh[up];
                tot[u] = tot[up];
            } else {
                uint32_t cntw[K], runs = 0, mw[K], bw[K];
                expand_row_meta(meta[u], mw, bw);
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    const bool in_row = l + kWave * j < W;
                    nm[u][j] = in_row ? ~mw[j] : 0u;
                    bv[u][j] = in_row ? bw[j] : 0u;
                    cntw[j] = (uint32_t)__builtin_popcount(nm[u][j]);
                    if constexpr (FORM == kMetaRaw) runs = max(runs, run_count(nm[u][j]));
                }
                tot[u] = row_offsets<K>(cntw, ofs[u]);
                uint32_t max_runs;
                if constexpr (FORM == kMetaSlots) max_runs = slot_max_runs(meta[u], s.slot_pairs);
                else max_runs = wave_max(runs);
                nh[u] = max_runs ? max_runs - 1u : 0u;
            }
            const uint64_t rb = row_stride((tot[u] + 7u) >> 3, s.row_align);
            uint64_t rbyte;
            if constexpr (STAGED) rbyte = (uint32_t)__builtin_amdgcn_readlane((int)so, (int)i);
            else {
                const uint64_t off = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)off_hi, (int)i) << 32) |
                                     (uint32_t)__builtin_amdgcn_readlane((int)off_lo, (int)i);
                rbyte = off + (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)r_l, (int)i) * rb;
            }
            bit0[u] = ((uint32_t)rbyte & 3u) * 8u;
            const __amdgpu_buffer_rsrc_t rr = row_rsrc(pay32 + (rbyte >> 2), ((bit0[u] + tot[u] + 31u) >> 5) * 4u);
#pragma unroll
            for (int j = 0; j < K; ++j) {
                load_window(rr, (ofs[u][j] + bit0[u]) >> 5, d0[u][j], d1[u][j]);
            }
        }
        uint32_t x[RB][K];
#pragma unroll
        for (int u = 0; u < RB; ++u)
#pragma unroll
            for (int j = 0; j < K; ++j)
                x[u][j] = __builtin_amdgcn_alignbit(d1[u][j], d0[u][j], ofs[u][j] + bit0[u]);
#pragma unroll
        for (int u = 0; u < RB; ++u)
#pragma unroll
            for (int j = 0; j < K; ++j) pv[u][j] = word_deposit(bv[u][j], nm[u][j], x[u][j], nh[u]);
#pragma unroll
        for (int j = 0; j < K; ++j) {
            c_nm[j] = nm[RB - 1][j];
            c_bv[j] = bv[RB - 1][j];
            c_ofs[j] = ofs[RB - 1][j];
        }
        c_nh = nh[RB - 1];
        c_tot = tot[RB - 1];
        pbase = base_i;
        pending = true;
    }
    store_pending();
}

// ---- the thresholded scheme with participation bits (stream flags = 1) ----------
//
// A row is either raw (row_bytes long) or: C participation bits, then chunk by chunk
// the row's bits, without the Mask bits of the compressed chunks. Which chunks are
// compressed differs from row to row, so the word offsets are a scan per row: word w's
// width is popcount(~Mask_w) when its chunk is compressed and 32 otherwise. The
// cluster's tile (Mask/Bitval, precomputed runs) is set up once and kept while
// consecutive rows share the cluster (with one global Mask, once per wave).

enum { kSrcRange = 0, kSrcIds = 1, kSrcStaged = 2 };

// Decode one tile (words [w0, w0 + 64K)) of one participation-scheme row whose bytes
// start at byte `rbyte` of pay32; `start` is the bit of the row where this tile's first
// word begins. Returns the tile's bits.
template <int NR, int K, int MAXR>
__device__ __forceinline__ uint32_t part_tile(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                              uint64_t rbyte, bool raw, uint32_t m, uint32_t start,
                                              uint32_t W, uint32_t w0, uint32_t *__restrict__ orow) {
    const uint32_t l = lane_id();
    const uint32_t *__restrict__ p = pay32 + (rbyte >> 2);
    const uint32_t bit0 = ((uint32_t)rbyte & 3u) * 8u;
    // the participation bits of this tile's chunks: dwords dbase .. dbase + nd - 1 of
    // the row's bit string, dword q in lane q - dbase
    const uint32_t w_end = min(W, w0 + (uint32_t)(kWave * K));
    const uint32_t dbase = (w0 / m) >> 5;
    const uint32_t nd = (((w_end - 1) / m) >> 5) - dbase + 1;
    uint32_t pd = 0;
    if (!raw && l < nd) {
        const uint32_t q = dbase + l;
        pd = __builtin_amdgcn_alignbit(p[q + 1], p[q], bit0);
    }
    uint32_t width[K], pb[K];
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const uint32_t w = w0 + l + kWave * j;
        const uint32_t c = (w < W ? w : w0) / m;
        const uint32_t dw = (uint32_t)__builtin_amdgcn_ds_bpermute((int)((((c >> 5) - dbase) & 63u) * 4u), (int)pd);
        pb[j] = raw ? 0u : (dw >> (c & 31u)) & 1u;
        width[j] = w < W ? (pb[j] ? (uint32_t)__builtin_popcount(t.nm[j]) : 32u) : 0u;
    }
    uint32_t ofs[K];
    uint32_t c = 0;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const uint32_t inc = wave_incl_scan(width[j]);
        ofs[j] = c + inc - width[j];
        c += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
    }
    uint32_t d0[K], d1[K], b[K];
#pragma unroll
    for (int j = 0; j < K; ++j) {
        b[j] = bit0 + start + ofs[j];
        d0[j] = p[b[j] >> 5];
        d1[j] = p[(b[j] >> 5) + 1];
    }
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const uint32_t x = __builtin_amdgcn_alignbit(d1[j], d0[j], b[j]);
        uint32_t v;
        if constexpr (NR >= 0) v = word_fast<NR>(t, j, x);
        else v = word_generic(t.bv[j], t.nm[j], x);
        v = pb[j] ? v : x;
        const uint32_t w = w0 + l + kWave * j;
        if (w < W) orow[w] = v;
    }
    return c;
}

template <int K, int MAXR>
__device__ __forceinline__ uint32_t part_tile_any(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                                  uint64_t rbyte, bool raw, uint32_t m, uint32_t start,
                                                  uint32_t W, uint32_t w0, uint32_t *__restrict__ orow) {
    switch (t.nr) {   // wave-uniform
    case 0: return part_tile<0>(t, pay32, rbyte, raw, m, start, W, w0, orow);
    case 1: return part_tile<1>(t, pay32, rbyte, raw, m, start, W, w0, orow);
    case 2: if constexpr (MAXR >= 2) return part_tile<2>(t, pay32, rbyte, raw, m, start, W, w0, orow); break;
    case 3: if constexpr (MAXR >= 3) return part_tile<3>(t, pay32, rbyte, raw, m, start, W, w0, orow); break;
    case 4: if constexpr (MAXR >= 4) return part_tile<4>(t, pay32, rbyte, raw, m, start, W, w0, orow); break;
    default: break;
    }
    return part_tile<-1>(t, pay32, rbyte, raw, m, start, W, w0, orow);
}

// Payload byte span [o0, o1) of row r of a participation-scheme stream. With line-packed
// offsets a request reads one 128-byte line (its 60-row block's base offset and the u16
// ends of the block's rows) instead of two u64 entries in the per-row index: sparse
// requests then share lines 7.5 times more often.
__device__ __forceinline__ void row_span(const DevStream &s, uint64_t r, uint64_t &o0, uint64_t &o1) {
    if (s.row_lines) {
        const uint64_t j = __umul64hi(r, s.rl_magic);
        const uint32_t k = (uint32_t)(r - j * kRowLineRows);
        const uint8_t *__restrict__ ln = s.row_lines + j * 128ull;
        const uint64_t base = *reinterpret_cast<const uint64_t *>(ln);
        const uint16_t *__restrict__ ends = reinterpret_cast<const uint16_t *>(ln + 8);
        const uint32_t start = ends[k ? k - 1u : 0u];
        o0 = base + (k ? start : 0u);
        o1 = base + ends[k];
    } else {
        o0 = s.index[r];
        o1 = s.index[r + 1];
    }
}

// One wave decodes `per_wave` consecutive work items (rows of a range, requests of a
// gather), one row at a time.
template <int K, int MAXR, int SRC>
__global__ __launch_bounds__(kBlock) void k_part_rows(DevStream s, const uint32_t *__restrict__ pay32,
                                                       uint64_t pay_base, const int64_t *__restrict__ ids,
                                                       const uint32_t *__restrict__ sg,
                                                       const uint32_t *__restrict__ soff, uint64_t first,
                                                       uint64_t n, uint32_t *__restrict__ out, uint32_t per_wave,
                                                       unsigned long long *err) {
    const uint64_t i0 = wave_slot() * per_wave;
    if (i0 >= n) return;
    const uint32_t cnt = (uint32_t)min((uint64_t)per_wave, n - i0);
    const uint32_t l = lane_id();
    const uint32_t W = s.W, m = s.part_m, C = W / m;
    const bool one_tile = W <= (uint32_t)(kWave * K);
    uint64_t cached_g = ~0ull;
    Tile<K, MAXR> t;
    for (uint32_t k = 0; k < cnt; ++k) {
        const uint64_t i = i0 + k;
        uint32_t *__restrict__ orow = out + i * W;
        uint64_t g, rbyte, size;
        if constexpr (SRC == kSrcStaged) {
            g = sg[i];
            rbyte = soff[i];
            size = soff[i + 1] - soff[i];
        } else {
            uint64_t r;
            if constexpr (SRC == kSrcIds) {
                const int64_t id = ids[i];
                if (id < 0 || (uint64_t)id >= s.n_rows) {
                    for (uint32_t w = l; w < W; w += kWave) orow[w] = 0u;
                    if (l == 0) atomicAdd(err, 1ull);
                    continue;
                }
                r = (uint64_t)id;
            } else {
                r = first + i;
            }
            g = s.G == 1 ? r : __umul64hi(r, s.g_magic);
            uint64_t o0, o1;
            row_span(s, r, o0, o1);
            rbyte = o0 - pay_base;
            size = o1 - o0;
        }
        const bool raw = size == 4ull * W;
        const uint32_t *__restrict__ mg = s.meta + g * 2ull * W;
        if (one_tile) {
            if (g != cached_g) {
                tile_setup(t, mg, W, 0, 0);
                cached_g = g;
            }
            part_tile_any(t, pay32, rbyte, raw, m, raw ? 0u : C, W, 0, orow);
        } else {
            uint32_t start = raw ? 0u : C;
            for (uint32_t w0 = 0; w0 < W; w0 += kWave * K) {
                tile_setup(t, mg, W, w0, 0);
                start += part_tile_any(t, pay32, rbyte, raw, m, start, W, w0, orow);
            }
            cached_g = ~0ull;
        }
    }
}

// RB participation-scheme rows of one cluster (tile t), one tile each (W <= 64K), in two
// stages. part_batch_load: the participation bits of all RB rows (loaded together, or
// prefetched with the lookup), then every row's widths, scan and two-dword windows.
// part_batch_rebuild: the rebuilt words. With deferred stores the caller stores the
// previous batch between the two, so those stores leave after this batch's window loads
// and the compiler never waits for them before reusing registers. Loads are unconditional with clamped addresses
// (inside the row or the readable slack), so no exec-masked load makes earlier loads drain.
//
// Everything a batch knows about its rows is wave-uniform and read on demand from the
// lanes of the lookup (lane i holds item i): a row's first data bit and prefetched
// participation dwords by readlane, whether it is raw or to be stored from bit masks. A
// row's chunk bit becomes an all-ones or all-zeros lane mask (a sign-extended bit-field
// extract), which then selects the word's width and its rebuilt or raw value by bitfield
// insert, with no compare and no branch per row. PRE: 0 = the participation dwords are
// loaded per batch, 1 or 2 = that many dwords were prefetched (at most 32 or 64 chunks).
template <int RB, int K>
struct PartLoads {
    uint32_t d0[RB][K], d1[RB][K];
    uint32_t bs[RB][K];   // bits 0-4: the window's shift; bits 5-31: all ones when the chunk is compressed
};

__device__ __forceinline__ uint64_t lane_u64(uint64_t v, uint32_t i) {
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), (int)i) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, (int)i);
}

// m ? a : b, bit by bit, in one instruction (written out, the compiler splits it into a
// not, an and and an and-or, and keeps every row's inverted mask live)
__device__ __forceinline__ uint32_t bit_select(uint32_t m, uint32_t a, uint32_t b) {
    uint32_t r;
    asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "v"(a), "v"(b));
    return r;
}

template <int RB, int PRE, int K, int MAXR>
__device__ __forceinline__ void part_batch_load(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                                uint64_t bit_l, const uint32_t (&pdw)[2], uint32_t i,
                                                uint32_t last, uint64_t rawm, uint32_t m, uint32_t C, uint32_t W,
                                                const uint32_t (&full)[K], PartLoads<RB, K> &ld) {
    const uint32_t l = lane_id();
    uint32_t pd[RB];
    if constexpr (PRE == 0) {
        const uint32_t nd = (((W - 1) / m) >> 5) + 1;
        const uint32_t ql = min(l, nd - 1);
#pragma unroll
        for (int u = 0; u < RB; ++u) {
            const uint32_t iu = min(i + u, last);
            const uint32_t raw = (uint32_t)(rawm >> iu) & 1u;
            const uint64_t pbit = lane_u64(bit_l, iu) - (raw ? 0u : C);   // the row's first bit
            const uint32_t *__restrict__ p = pay32 + (pbit >> 5);
            const uint32_t d = __builtin_amdgcn_alignbit(p[ql + 1], p[ql], (uint32_t)pbit & 31u);
            pd[u] = d & (raw - 1u);   // raw rows: no chunk is compressed
        }
    }
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        const uint32_t iu = min(i + u, last);
        const uint64_t rbit = lane_u64(bit_l, iu);
        uint32_t d_lo = 0, d_hi = 0;
        if constexpr (PRE >= 1) d_lo = (uint32_t)__builtin_amdgcn_readlane((int)pdw[0], (int)iu);
        if constexpr (PRE >= 2) d_hi = (uint32_t)__builtin_amdgcn_readlane((int)pdw[1], (int)iu);
        uint32_t width[K], sel[K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t w = l + kWave * j;
            const uint32_t c = (w < W ? w : 0u) / m;
            uint32_t dw;
            if constexpr (PRE == 0) dw = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(((c >> 5) & 63u) * 4u), (int)pd[u]);
            else if constexpr (PRE == 1) dw = d_lo;
            else dw = (c >> 5) ? d_hi : d_lo;
            sel[j] = (uint32_t)__builtin_amdgcn_sbfe((int)dw, c & 31u, 1u);   // 0 or ~0
            width[j] = bit_select(sel[j], t.pk[j], full[j]);
        }
        const uint32_t *__restrict__ p = pay32 + (rbit >> 5);
        uint32_t c = (uint32_t)rbit & 31u;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t inc = wave_incl_scan(width[j]);
            const uint32_t b = c + inc - width[j];
            if (j + 1 < K) c += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
            ld.d0[u][j] = p[b >> 5];
            ld.d1[u][j] = p[(b >> 5) + 1];
            ld.bs[u][j] = bit_select(31u, b, sel[j]);
        }
    }
}

template <int NR, int RB, int K, int MAXR>
__device__ __forceinline__ void part_batch_rebuild(const Tile<K, MAXR> &t, const PartLoads<RB, K> &ld,
                                                   uint32_t (&v)[RB][K]) {
#pragma unroll
    for (int u = 0; u < RB; ++u) {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t x = __builtin_amdgcn_alignbit(ld.d1[u][j], ld.d0[u][j], ld.bs[u][j]);
            uint32_t y;
            if constexpr (NR >= 0) y = word_fast<NR>(t, j, x);
            else y = word_generic(t.bv[j], t.nm[j], x);
            v[u][j] = bit_select((uint32_t)((int32_t)ld.bs[u][j] >> 31), y, x);
        }
    }
}

// Rebuilt words of RB rows waiting to be stored: rows row0 .. row0 + RB - 1 of the wave's
// output, row row0 + u stored when bit u of `ok` is set (both wave-uniform).
template <int RB, int K>
struct PartPending {
    uint32_t v[RB][K];
    uint32_t row0 = 0;
    uint32_t ok = 0;
};

template <int RB, int K>
__device__ __forceinline__ void part_store(PartPending<RB, K> &pp, uint32_t *__restrict__ out_seg, uint32_t W) {
    if (!pp.ok) return;
    const uint32_t l = lane_id();
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        if (!((pp.ok >> u) & 1u)) continue;
        uint32_t *__restrict__ orow = out_seg + (uint64_t)(pp.row0 + u) * W;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t w = l + kWave * j;
            if (w < W) store_out(&orow[w], pp.v[u][j]);
        }
    }
    pp.ok = 0;
}

// One batch: its loads, then (DEFER) the previous batch's stores, its rebuild, and
// (otherwise) its own stores. The run count is a template parameter of the whole step, so
// each variant keeps only its own registers live.
template <int NR, int RB, int PRE, bool DEFER, int K, int MAXR>
__device__ __forceinline__ void part_batch_step(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                                uint64_t bit_l, const uint32_t (&pdw)[2], uint32_t i,
                                                uint32_t last, uint64_t rawm, uint32_t ok, uint32_t m, uint32_t C,
                                                uint32_t W, const uint32_t (&full)[K], uint32_t *__restrict__ out_seg,
                                                PartPending<RB, K> &pend) {
    PartLoads<RB, K> ld;
    part_batch_load<RB, PRE>(t, pay32, bit_l, pdw, i, last, rawm, m, C, W, full, ld);
    if constexpr (DEFER) part_store(pend, out_seg, W);
    part_batch_rebuild<NR>(t, ld, pend.v);
    pend.row0 = i;
    pend.ok = ok;
    if constexpr (!DEFER) part_store(pend, out_seg, W);
}

template <int RB, int PRE, bool DEFER, int K, int MAXR>
__device__ __forceinline__ void part_batch_step_any(const Tile<K, MAXR> &t, const uint32_t *__restrict__ pay32,
                                                    uint64_t bit_l, const uint32_t (&pdw)[2], uint32_t i,
                                                    uint32_t last, uint64_t rawm, uint32_t ok, uint32_t m,
                                                    uint32_t C, uint32_t W, const uint32_t (&full)[K],
                                                    uint32_t *__restrict__ out_seg, PartPending<RB, K> &pend) {
#define IBP_PART_STEP(NR) \
    part_batch_step<NR, RB, PRE, DEFER>(t, pay32, bit_l, pdw, i, last, rawm, ok, m, C, W, full, out_seg, pend)
    switch (t.nr) {   // wave-uniform
    case 0: IBP_PART_STEP(0); return;
    case 1: IBP_PART_STEP(1); return;
    case 2: if constexpr (MAXR >= 2) { IBP_PART_STEP(2); return; } break;
    case 3: if constexpr (MAXR >= 3) { IBP_PART_STEP(3); return; } break;
    case 4: if constexpr (MAXR >= 4) { IBP_PART_STEP(4); return; } break;
    default: break;
    }
    IBP_PART_STEP(-1);
#undef IBP_PART_STEP
}

// RB participation-scheme rows of a batch whose rows lie in different clusters (a gather
// under per-cluster Masks). Every row's Mask/Bitval words are loaded together, then each row
// takes the same widths, scan and windows as a batch of one cluster, and its compressed
// words are rebuilt with the holes deposit: a setup of runs per row would cost more than it
// saves. Stores are immediate (this path keeps no words pending).
template <int RB, int PRE, int K>
__device__ __forceinline__ void part_mixed_batch(const DevStream &s, const uint32_t *__restrict__ pay32,
                                                 uint64_t g_l, uint64_t bit_l, const uint32_t (&pdw)[2],
                                                 uint32_t i, uint32_t last, uint64_t rawm, uint32_t ok, uint32_t m,
                                                 uint32_t C, uint32_t W, const uint32_t (&full)[K],
                                                 uint32_t *__restrict__ out_seg) {
    const uint32_t l = lane_id();
    uint32_t nm[RB][K], bv[RB][K];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        const uint32_t *__restrict__ mg = s.meta + lane_u64(g_l, min(i + u, last)) * 2ull * W;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t w = l + kWave * j, wc = w < W ? w : 0u;
            nm[u][j] = mg[wc];
            bv[u][j] = mg[W + wc];
        }
    }
    uint32_t pd[RB];
    if constexpr (PRE == 0) {
        const uint32_t nd = (((W - 1) / m) >> 5) + 1;
        const uint32_t ql = min(l, nd - 1);
#pragma unroll
        for (int u = 0; u < RB; ++u) {
            const uint32_t iu = min(i + u, last);
            const uint32_t raw = (uint32_t)(rawm >> iu) & 1u;
            const uint64_t pbit = lane_u64(bit_l, iu) - (raw ? 0u : C);
            const uint32_t *__restrict__ p = pay32 + (pbit >> 5);
            pd[u] = __builtin_amdgcn_alignbit(p[ql + 1], p[ql], (uint32_t)pbit & 31u) & (raw - 1u);
        }
    }
    uint32_t d0[RB][K], d1[RB][K], bs[RB][K], nh[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        const uint32_t iu = min(i + u, last);
        const uint64_t rbit = lane_u64(bit_l, iu);
        uint32_t d_lo = 0, d_hi = 0;
        if constexpr (PRE >= 1) d_lo = (uint32_t)__builtin_amdgcn_readlane((int)pdw[0], (int)iu);
        if constexpr (PRE >= 2) d_hi = (uint32_t)__builtin_amdgcn_readlane((int)pdw[1], (int)iu);
        uint32_t width[K], sel[K], runs = 0;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t w = l + kWave * j;
            const uint32_t c = (w < W ? w : 0u) / m;
            uint32_t dw;
            if constexpr (PRE == 0) dw = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(((c >> 5) & 63u) * 4u), (int)pd[u]);
            else if constexpr (PRE == 1) dw = d_lo;
            else dw = (c >> 5) ? d_hi : d_lo;
            sel[j] = (uint32_t)__builtin_amdgcn_sbfe((int)dw, c & 31u, 1u);
            nm[u][j] = w < W ? ~nm[u][j] : 0u;   // the variant positions
            bv[u][j] = w < W ? bv[u][j] : 0u;
            width[j] = bit_select(sel[j], (uint32_t)__builtin_popcount(nm[u][j]), full[j]);
            runs = max(runs, run_count(nm[u][j]));
        }
        const uint32_t *__restrict__ p = pay32 + (rbit >> 5);
        uint32_t c = (uint32_t)rbit & 31u;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t inc = wave_incl_scan(width[j]);
            const uint32_t b = c + inc - width[j];
            if (j + 1 < K) c += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
            d0[u][j] = p[b >> 5];
            d1[u][j] = p[(b >> 5) + 1];
            bs[u][j] = bit_select(31u, b, sel[j]);
        }
        const uint32_t most = wave_max(runs);
        nh[u] = most ? most - 1u : 0u;
    }
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        if (!((ok >> u) & 1u)) continue;
        uint32_t *__restrict__ orow = out_seg + (uint64_t)(i + u) * W;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t x = __builtin_amdgcn_alignbit(d1[u][j], d0[u][j], bs[u][j]);
            const uint32_t y = word_deposit(bv[u][j], nm[u][j], x, nh[u]);
            const uint32_t v = bit_select((uint32_t)((int32_t)bs[u][j] >> 31), y, x);
            const uint32_t w = l + kWave * j;
            if (w < W) store_out(&orow[w], v);
        }
    }
}

// Participation-scheme rows that fit one tile (W <= 64K), in batches of RB rows. With
// DEFER (two batches per wave) each batch's stores wait until the next batch's window
// loads have left; otherwise a batch stores at once and keeps fewer registers. A wave owns
// `seg` (<= 64) work items; lane i < seg first locates item i (its cluster, the first data
// bit of its row and its size). A batch whose rows share a cluster (always under one global
// Mask, ONE) is decoded with that cluster's tile; a batch of rows from different clusters
// loads each row's Mask/Bitval words (part_mixed_batch).
template <int K, int MAXR, int RB, int SRC, int PRE, bool DEFER, bool ONE>
__global__ __launch_bounds__(kBlock, (ONE && (K == 1 || (K == 2 && PRE != 0))) ? 8 : 1) void k_part_batched(DevStream s, const uint32_t *__restrict__ pay32,
                                                          uint64_t pay_base, const int64_t *__restrict__ ids,
                                                          const uint32_t *__restrict__ sg,
                                                          const uint32_t *__restrict__ soff, uint64_t first,
                                                          uint64_t n, uint32_t *__restrict__ out, uint32_t seg,
                                                          unsigned long long *err) {
    const uint64_t i0 = wave_slot() * seg;
    if (i0 >= n) return;
    const uint32_t cnt = (uint32_t)min((uint64_t)seg, n - i0);
    const uint32_t l = lane_id();
    const uint32_t W = s.W, m = s.part_m, C = W / m;
    const uint32_t li = l < cnt ? l : cnt - 1;      // lanes past the end repeat the last item
    uint64_t g_l, byte_l, size_l;
    bool valid = true;
    if constexpr (SRC == kSrcStaged) {
        g_l = sg[i0 + li];
        byte_l = soff[i0 + li];
        size_l = soff[i0 + li + 1] - byte_l;
    } else {
        uint64_t r;
        if constexpr (SRC == kSrcIds) {
            const int64_t id = ids[i0 + li];
            valid = id >= 0 && (uint64_t)id < s.n_rows;
            r = valid ? (uint64_t)id : 0u;
        } else {
            r = first + i0 + li;
        }
        g_l = s.G == 1 ? r : __umul64hi(r, s.g_magic);
        uint64_t o0, o1;
        row_span(s, r, o0, o1);
        byte_l = o0 - pay_base;
        size_l = o1 - o0;
    }
    // few chunks: each lane fetches its own row's participation dwords now, in one round
    // trip for the whole segment
    uint32_t pdw[2] = {0u, 0u};
    if constexpr (PRE >= 1) {
        const uint32_t *__restrict__ p = pay32 + (byte_l >> 2);
        const uint32_t b0 = ((uint32_t)byte_l & 3u) * 8u;
        const uint32_t q0 = p[0], q1 = p[1];
        pdw[0] = __builtin_amdgcn_alignbit(q1, q0, b0);
        if constexpr (PRE >= 2) pdw[1] = __builtin_amdgcn_alignbit(p[2], q1, b0);
    }
    // the wave's items as bit masks: bad ids, raw rows, rows to store, and rows that share
    // the previous item's cluster (lanes past the end repeat the last item, so they do)
    const bool raw_l = size_l == 4ull * W;
    const uint64_t bad = __ballot(l < cnt && !valid);
    const uint64_t rawm = __ballot(raw_l);
    // each item's first data bit in the payload, past its participation bits; a raw row
    // has no compressed chunk
    const uint64_t bit_l = byte_l * 8u + (raw_l ? 0u : C);
    if (raw_l) pdw[0] = pdw[1] = 0u;
    const uint64_t okm = __ballot(l < cnt && valid);
    uint64_t samep = ~0ull;
    if constexpr (!ONE) {
        const uint32_t src = (l ? l - 1u : 0u) * 4u;
        const uint32_t gp_lo = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, (int)(uint32_t)g_l);
        const uint32_t gp_hi = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, (int)(uint32_t)(g_l >> 32));
        samep = __ballot((((uint64_t)gp_hi << 32) | gp_lo) == g_l);
    }
    uint32_t *__restrict__ out_seg = out + i0 * W;
    if (bad) {
        for (uint32_t i = 0; i < cnt; ++i)
            if ((bad >> i) & 1ull)
                for (uint32_t w = l; w < W; w += kWave) out_seg[(uint64_t)i * W + w] = 0u;
        if (l == 0) atomicAdd(err, (unsigned long long)__popcll(bad));
    }
    uint32_t full[K];   // a word's width when its chunk is stored raw (0 past the row's end)
#pragma unroll
    for (int j = 0; j < K; ++j) full[j] = l + kWave * j < W ? 32u : 0u;
    Tile<K, MAXR> t;
    PartPending<RB, K> pend;
    if constexpr (ONE) {
        // one cluster for the whole stream (the scheme's single global Mask)
        tile_setup(t, s.meta, W, 0, 0);
        for (uint32_t i = 0; i < cnt; i += RB) {
            const uint32_t ok = (uint32_t)(okm >> i) & ((1u << RB) - 1u);
            part_batch_step_any<RB, PRE, DEFER>(t, pay32, bit_l, pdw, i, cnt - 1, rawm, ok, m, C, W, full,
                                                out_seg, pend);
        }
        part_store(pend, out_seg, W);
        return;
    }
    constexpr uint64_t kTail = (1ull << (RB - 1)) - 1ull;   // rows 1 .. RB-1 of a batch
    uint64_t cached_g = ~0ull;
    for (uint32_t i = 0; i < cnt; i += RB) {
        const uint64_t g0 = lane_u64(g_l, i);
        const uint32_t ok = (uint32_t)(okm >> i) & ((1u << RB) - 1u);
        const uint64_t tail = RB > 1 ? kTail << (i + 1) : 0ull;   // i + RB <= seg <= 64
        if ((samep & tail) == tail) {
            if (g0 != cached_g) {
                part_store(pend, out_seg, W);
                tile_setup(t, s.meta + g0 * 2ull * W, W, 0, 0);
                cached_g = g0;
            }
            part_batch_step_any<RB, PRE, DEFER>(t, pay32, bit_l, pdw, i, cnt - 1, rawm, ok, m, C, W, full,
                                                out_seg, pend);
        } else {
            part_store(pend, out_seg, W);
            // in halves: the per-row metadata would otherwise cost this kernel occupancy
            constexpr int H = RB > 1 ? RB / 2 : 1;
#pragma unroll
            for (int h = 0; h < RB; h += H)
                part_mixed_batch<H, PRE>(s, pay32, g_l, bit_l, pdw, i + h, cnt - 1, rawm, (ok >> h) & ((1u << H) - 1u),
                                         m, C, W, full, out_seg);
        }
    }
    part_store(pend, out_seg, W);
}

template <int K, int MAXR>
hipError_t launch_part_k(const DevStream &s, const uint32_t *p, uint64_t pay_base, const int64_t *ids,
                         const uint32_t *sg, const uint32_t *soff, uint64_t first, uint64_t n, uint32_t *o,
                         unsigned long long *err, hipStream_t stream) {
    if (s.W <= (uint32_t)(kWave * K)) {
        // rows of one tile: batches of RB rows, 1-2 batches per wave (2 when there is work
        // for ~16k waves; measured on the KV layer: 4 batches 57.6 us, 2 batches 54.1, 8
        // batches 64.4: a wave's lookup and its batches are dependent round trips, and more
        // waves in flight hide them better than more batches per wave)
        constexpr int RB = K <= 1 ? 8 : (K <= 2 ? 4 : (K <= 4 ? 2 : 1));
        const uint32_t nb = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(2, n / (16384ull * RB)));
        const uint32_t seg = RB * nb;
        if (seg > (uint32_t)kWave) return hipErrorInvalidValue;   // lane i holds item i
        const uint64_t waves = (n + seg - 1) / seg;
        const dim3 grid((unsigned)((waves + kWavesPerBlock - 1) / kWavesPerBlock)), block(kBlock);
        // participation dwords prefetched with the lookup: 1 for at most 32 chunks, 2 for
        // at most 64, else loaded per batch
        const uint32_t chunks = s.W / s.part_m;
        const int pre = chunks <= 32u ? 1 : (chunks <= 64u ? 2 : 0);
        if (K == 1 && pre == 0) return hipErrorInvalidValue;   // W <= 64 words: at most 64 chunks
        const bool one = (uint64_t)s.G >= s.n_rows;   // a single cluster
        auto go = [&](auto pre_tag, auto defer_tag) {
            constexpr int P = decltype(pre_tag)::value;
            constexpr bool D = decltype(defer_tag)::value;
            auto go_one = [&](auto one_tag) {
                constexpr bool O = decltype(one_tag)::value;
                if (ids)
                    hipLaunchKernelGGL((k_part_batched<K, MAXR, RB, kSrcIds, P, D, O>), grid, block, 0, stream, s,
                                       p, pay_base, ids, sg, soff, first, n, o, seg, err);
                else if (sg)
                    hipLaunchKernelGGL((k_part_batched<K, MAXR, RB, kSrcStaged, P, D, O>), grid, block, 0, stream,
                                       s, p, pay_base, ids, sg, soff, first, n, o, seg, err);
                else
                    hipLaunchKernelGGL((k_part_batched<K, MAXR, RB, kSrcRange, P, D, O>), grid, block, 0, stream,
                                       s, p, pay_base, ids, sg, soff, first, n, o, seg, err);
            };
            if (one) go_one(std::true_type{});
            else go_one(std::false_type{});
        };
        auto go_pre = [&](auto defer_tag) {
            if (pre == 1) go(std::integral_constant<int, 1>{}, defer_tag);
            else if (pre == 2) go(std::integral_constant<int, 2>{}, defer_tag);
            else if constexpr (K > 1) go(std::integral_constant<int, 0>{}, defer_tag);   // K = 1: at most 64 chunks
        };
        // deferred stores, measured: the KV layer (K = 1) 4% faster, 1 KB rows read in place
        // from host memory (K = 4) 5-25% faster; at K = 2 their registers cost a wave per
        // SIMD and the GNN gather ran 15% slower
        if constexpr (K != 2) {
            if (nb > 1) go_pre(std::true_type{});
            else go_pre(std::false_type{});
        } else {
            go_pre(std::false_type{});
        }
        return hipGetLastError();
    }
    // rows of several tiles (only at eight words per lane): one row at a time per wave
    if constexpr (K == 8) {
        const uint32_t per_wave = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(16, n / 16384));
        const uint64_t waves = (n + per_wave - 1) / per_wave;
        const dim3 grid((unsigned)((waves + kWavesPerBlock - 1) / kWavesPerBlock)), block(kBlock);
        if (ids)
            hipLaunchKernelGGL((k_part_rows<K, MAXR, kSrcIds>), grid, block, 0, stream, s, p, pay_base, ids, sg, soff,
                               first, n, o, per_wave, err);
        else if (sg)
            hipLaunchKernelGGL((k_part_rows<K, MAXR, kSrcStaged>), grid, block, 0, stream, s, p, pay_base, ids, sg,
                               soff, first, n, o, per_wave, err);
        else
            hipLaunchKernelGGL((k_part_rows<K, MAXR, kSrcRange>), grid, block, 0, stream, s, p, pay_base, ids, sg,
                               soff, first, n, o, per_wave, err);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}


// Compute units of the current device (cached per device; concurrent first calls store
// the same value).
uint32_t compute_units() {
    static std::atomic<uint32_t> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    uint32_t cu = cached[dev].load(std::memory_order_relaxed);
    if (!cu) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cu = (uint32_t)v;
        cached[dev].store(cu, std::memory_order_relaxed);
    }
    return cu;
}

}  // namespace

uint64_t div_magic(uint32_t G) {
    if (G <= 1) return 0;
    // ceil(2^64 / G) = floor((2^64 - 1) / G) + 1 for every G >= 2. With magic =
    // 2^64/G + e (0 <= e < 1), mulhi(id, magic) = floor(id/G + id*e/2^64) equals
    // floor(id/G) whenever id * G < 2^64, which ibp_open checks.
    return ~0ull / G + 1;
}

hipError_t launch_part(const DevStream &s_in, const uint8_t *payload, uint64_t pay_base, const int64_t *ids,
                       const uint32_t *sg, const uint32_t *soff, uint64_t first, uint64_t n, void *out,
                       unsigned long long *err, hipStream_t stream) {
    const auto *p = reinterpret_cast<const uint32_t *>(payload);
    auto *o = static_cast<uint32_t *>(out);
    // line-packed row offsets only for gathers with more than one request per line's worth
    // of rows on average: ranges read the per-row index contiguously, and sparser requests
    // touch a line each either way (measured: the KV layer and the DLRM lookups 1-2%
    // slower through the lines, the GNN minibatch even)
    DevStream s = s_in;
    if (!ids || n * kRowLineRows < s.n_rows) s.row_lines = nullptr;
    switch (words_per_lane(s.W)) {
    case 1: return launch_part_k<1, 4>(s, p, pay_base, ids, sg, soff, first, n, o, err, stream);
    case 2: return launch_part_k<2, 4>(s, p, pay_base, ids, sg, soff, first, n, o, err, stream);
    case 4: return launch_part_k<4, 2>(s, p, pay_base, ids, sg, soff, first, n, o, err, stream);
    default: return launch_part_k<8, 1>(s, p, pay_base, ids, sg, soff, first, n, o, err, stream);
    }
}

hipError_t launch_decompress(const DevStream &s, const uint8_t *payload, uint64_t pay_base, void *out,
                             uint64_t first, uint64_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (s.part_m) return launch_part(s, payload, pay_base, nullptr, nullptr, nullptr, first, n, out, nullptr, stream);
    const uint64_t g0 = first / s.G, g1 = (first + n - 1) / s.G;
    // rows per wave: a whole cluster (at most 64 rows), halved while the launch would have
    // fewer than ~16k waves (2 per wave slot of the chip), down to one batch of rows;
    // every slice repeats its cluster's setup, which is small next to its rows
    const int k = words_per_lane(s.W);
    const uint32_t min_rows = k == 1 ? 8 : (k == 2 ? 4 : (k == 4 ? 2 : 1));
    uint32_t rpu = s.G <= 64 ? s.G : 64;
    while (rpu > min_rows && (g1 - g0 + 1) * ((s.G + rpu - 1) / rpu) < 16384) rpu = (rpu + 1) / 2;
    const uint32_t upg = (s.G + rpu - 1) / rpu;
    const uint64_t n_units = (g1 - g0 + 1) * upg;
    const uint64_t blocks = (n_units + kWavesPerBlock - 1) / kWavesPerBlock;
    const auto *p = reinterpret_cast<const uint32_t *>(payload);
    auto *o = static_cast<uint32_t *>(out);
    dim3 grid((unsigned)blocks), block(kBlock);
    auto go = [&](auto kk, auto mr, auto split) {
        constexpr int KK = decltype(kk)::value, MR = decltype(mr)::value;
        constexpr bool SP = decltype(split)::value;
        hipLaunchKernelGGL((k_decompress<KK, MR, SP>), grid, block, 0, stream, s, p, pay_base, o, first, n, g0,
                           n_units, upg, rpu);
    };
    // two dword loads per window from device memory, one 8-byte load from pinned host memory
    auto launch = [&](auto kk, auto mr) {
        if (s.payload_host) go(kk, mr, std::false_type{});
        else go(kk, mr, std::true_type{});
    };
    switch (k) {
    case 1: launch(std::integral_constant<int, 1>{}, std::integral_constant<int, 4>{}); break;
    case 2: launch(std::integral_constant<int, 2>{}, std::integral_constant<int, 4>{}); break;
    case 4: launch(std::integral_constant<int, 4>{}, std::integral_constant<int, 2>{}); break;
    default: launch(std::integral_constant<int, 8>{}, std::integral_constant<int, 1>{}); break;
    }
    return hipGetLastError();
}

hipError_t launch_gather(const DevStream &s, const uint8_t *payload, const int64_t *ids, const uint32_t *sg,
                         const uint32_t *soff, uint64_t n, void *out, unsigned long long *err, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (s.part_m) return launch_part(s, payload, 0, ids, sg, soff, 0, n, out, err, stream);
    const auto *p = reinterpret_cast<const uint32_t *>(payload);
    auto *o = static_cast<uint32_t *>(out);
    const int k = words_per_lane(s.W);
    if (s.W > 512) {
        const uint32_t seg = 16;
        const uint64_t blocks = ((n + seg - 1) / seg + kWavesPerBlock - 1) / kWavesPerBlock;
        if (soff)
            hipLaunchKernelGGL((k_gather_tiled<8, 1, true>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, s, p,
                               ids, sg, soff, n, o, seg, err);
        else
            hipLaunchKernelGGL((k_gather_tiled<8, 1, false>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, s, p,
                               ids, sg, soff, n, o, seg, err);
        return hipGetLastError();
    }
    // Batches of RB rows (RB = 4 at K = 2 keeps 8 waves per SIMD; larger batches cost
    // occupancy, smaller ones memory-level parallelism). A wave takes one batch, or two or
    // four while that still leaves at least two waves per wave slot of the chip: measured
    // on the gathers, 2 batches per wave gain 1% on the 164k-row GNN minibatch and 4 gain
    // 7% on the 3.69M-row one (fewer waves to launch), while the 53k DLRM lookups, with
    // fewer waves than slots to begin with, lose 6-60% with more than one.
    const int rb_sel = k == 1 ? 8 : (k == 2 ? 4 : (k == 4 ? 2 : 1));
    const uint64_t min_waves = 2ull * compute_units() * 4 * 8;
    uint32_t nb = 1;
    while (nb < 4 && n / ((uint64_t)rb_sel * nb * 2) >= min_waves) nb *= 2;
    const uint32_t seg = (uint32_t)rb_sel * nb;
    if (seg > (uint32_t)kWave) return hipErrorInvalidValue;   // lane i holds request i
    const uint64_t blocks = ((n + seg - 1) / seg + kWavesPerBlock - 1) / kWavesPerBlock;
    dim3 grid((unsigned)blocks), block(kBlock);
    auto go = [&](auto kk, auto rb) {
        constexpr int KK = decltype(kk)::value, R = decltype(rb)::value;
        if (soff) {
            if (s.slots) hipLaunchKernelGGL((k_gather_rows<KK, R, true, kMetaSlots>), grid, block, 0, stream, s, p, ids, sg, soff, n, o, seg, err);
            else hipLaunchKernelGGL((k_gather_rows<KK, R, true, kMetaRaw>), grid, block, 0, stream, s, p, ids, sg, soff, n, o, seg, err);
        } else {
            if (s.slots) hipLaunchKernelGGL((k_gather_rows<KK, R, false, kMetaSlots>), grid, block, 0, stream, s, p, ids, sg, soff, n, o, seg, err);
            else hipLaunchKernelGGL((k_gather_rows<KK, R, false, kMetaRaw>), grid, block, 0, stream, s, p, ids, sg, soff, n, o, seg, err);
        }
    };
#define IBP_GATHER_ROWS(KK, RB) go(std::integral_constant<int, KK>{}, std::integral_constant<int, RB>{})
    switch (k) {
    case 1: IBP_GATHER_ROWS(1, 8); break;
    case 2: IBP_GATHER_ROWS(2, 4); break;
    case 4: IBP_GATHER_ROWS(4, 2); break;
    default: IBP_GATHER_ROWS(8, 1); break;
    }
#undef IBP_GATHER_ROWS
    return hipGetLastError();
}

}  // namespace dev
}  // namespace ibp
