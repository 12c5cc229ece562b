// gfx950 kernel of the compressed device-resident row cache (the paper's cache
// compression, Sec. 5): a static set of rows is kept, in packed form, back to back in a
// device slab; a lookup table maps a row id to a 64-bit entry (slab byte offset in bits
// 0-39, slab id in bits 40-42, compressed-form flag in bit 43). A gather resolves every
// requested id against the table: hits are decoded from the slab in HBM, misses from the
// stream's payload in pinned host memory, read in place over PCIe.
//
// The decode is the clustered-scheme gather: one wave per batch of RB requests, each row
// decoded on its own (its cluster's Mask/Bitval, a scan of popcount(~Mask), the holes
// deposit), all loads of the batch issued before any word is rebuilt. The only change is
// that a row's packed bytes are located by an absolute address chosen per request.
#include <type_traits>

#include "ibp_device.hpp"
#include "ibp_wave.hpp"

namespace ibp {
namespace dev {

namespace {

struct Slot {
    uint64_t key;   // row id + 1; 0 = empty
    uint64_t val;   // cache entry
};

template <int K, int RB, int FORM>
__global__ __launch_bounds__(kBlock) void k_cache_gather(DevStream s, CacheView c, const int64_t *__restrict__ ids,
                                                          uint64_t n, uint32_t *__restrict__ out,
                                                          unsigned long long *err) {
    const uint64_t slot = (uint64_t)xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock +
                          (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
    const uint64_t i0 = slot * RB;
    if (i0 >= n) return;
    const uint32_t cnt = (uint32_t)min((uint64_t)RB, n - i0);
    const uint32_t l = lane_id();
    const uint32_t W = s.W;
    // lane l < cnt resolves request l: cluster, row inside it, and where its bytes are
    const int64_t id = l < cnt ? ids[i0 + l] : -1;
    const bool valid = l < cnt && id >= 0 && (uint64_t)id < s.n_rows;
    const uint64_t uid = valid ? (uint64_t)id : 0;
    const uint64_t g_l = s.G == 1 ? uid : __umul64hi(uid, s.g_magic);
    const uint32_t r_l = (uint32_t)(uid - g_l * s.G);
    bool hit = false;
    uint64_t val = 0;
    if (valid) {
        const Slot *__restrict__ tab = reinterpret_cast<const Slot *>(c.table);
        const uint64_t key = uid + 1;
        uint64_t h = (uid * 0x9E3779B97F4A7C15ull) >> (64 - c.log2cap);
        // the table is at most half full, so an empty slot ends every probe sequence
        for (uint64_t k = 0; k <= c.mask; ++k) {
            const Slot e = tab[h];
            if (e.key == key) {
                hit = true;
                val = e.val;
                break;
            }
            if (e.key == 0) break;
            h = (h + 1) & c.mask;
        }
    }
    // byte address of the row's packed bits: the slab entry for a hit; for a miss the
    // cluster's payload offset, to which the row's index times its packed size is added
    // once the size is known from the Mask
    const uint64_t off_l = hit ? (val & 0xFFFFFFFFFFull) : s.index[g_l];
    const uint32_t mul_l = hit ? 0u : r_l;
    const uint64_t nhit = __ballot(valid && hit), nmiss = __ballot(valid && !hit);
    const uint64_t bad = __ballot(l < cnt && !valid);
    if (l == 0) {
        // counters spread over kCountLines 128-byte lines so that waves do not all
        // contend for one address
        unsigned long long *cnt = c.counts + (blockIdx.x % kCountLines) * kCountStride;
        if (nhit) atomicAdd(cnt, (unsigned long long)__popcll(nhit));
        if (nmiss) atomicAdd(cnt + 1, (unsigned long long)__popcll(nmiss));
        if (bad) atomicAdd(err, (unsigned long long)__popcll(bad));
    }
    uint32_t *__restrict__ out_seg = out + i0 * W;
    if (bad) {
        for (uint32_t i = 0; i < cnt; ++i)
            if ((bad >> i) & 1ull)
                for (uint32_t w = l; w < W; w += kWave) out_seg[(uint64_t)i * W + w] = 0u;
    }
    auto rd64 = [](uint64_t v, uint32_t i) -> uint64_t {
        return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), (int)i) << 32) |
               (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, (int)i);
    };
    auto slot_of = [&](uint32_t i) { return i < cnt ? i : cnt - 1; };
    RowMeta<K, FORM> meta[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        const uint64_t g = rd64(g_l, slot_of(u));
        load_row_meta<K, FORM>(meta[u], s.meta + g * 2ull * W, s.slots + g * s.slot_bytes, s.slot_pairs, W);
    }
#pragma unroll
    for (int u = 0; u < RB; ++u) hold_row_meta(meta[u]);
    uint32_t nm[RB][K], bv[RB][K], ofs[RB][K], d0[RB][K], d1[RB][K], nh[RB], bit0[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        const uint32_t i = slot_of(u);
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
        const uint32_t tot = row_offsets<K>(cntw, ofs[u]);
        uint32_t max_runs;
        if constexpr (FORM == kMetaSlots) max_runs = slot_max_runs(meta[u], s.slot_pairs);
        else max_runs = wave_max(runs);
        nh[u] = max_runs ? max_runs - 1u : 0u;
        const uint64_t rb = (tot + 7u) >> 3;
        // a select of the two buffers, not an integer address, keeps the loads global
        // (not flat) and the choice free of branches
        const uint8_t *__restrict__ buf = ((nhit >> i) & 1ull) ? c.slab : c.host_payload;
        const uint64_t addr = rd64(off_l, i) + (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)mul_l, (int)i) * rb;
        const uint32_t *__restrict__ p = reinterpret_cast<const uint32_t *>(buf + (addr & ~3ull));
        bit0[u] = ((uint32_t)addr & 3u) * 8u;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t q = (ofs[u][j] + bit0[u]) >> 5;
            d0[u][j] = p[q];
            d1[u][j] = p[q + 1];
        }
    }
#pragma unroll
    for (int u = 0; u < RB; ++u) {
        const uint32_t i = u;
        const bool row_ok = i < cnt && !((bad >> i) & 1ull);
        uint32_t *__restrict__ orow = out_seg + (uint64_t)slot_of(i) * W;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t x = __builtin_amdgcn_alignbit(d1[u][j], d0[u][j], ofs[u][j] + bit0[u]);
            const uint32_t v = word_deposit(bv[u][j], nm[u][j], x, nh[u]);
            const uint32_t w = l + kWave * j;
            if (row_ok && w < W) store_out(&orow[w], v);
        }
    }
}

}  // namespace

hipError_t launch_cache_gather(const DevStream &s, const CacheView &c, const int64_t *ids, uint64_t n, void *out,
                               unsigned long long *err, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    auto *o = static_cast<uint32_t *>(out);
    auto grid = [&](uint64_t rb) { return dim3((unsigned)(((n + rb - 1) / rb + kWavesPerBlock - 1) / kWavesPerBlock)); };
    auto go = [&](auto kk, auto rb) {
        constexpr int KK = decltype(kk)::value, R = decltype(rb)::value;
        if (s.slots) hipLaunchKernelGGL((k_cache_gather<KK, R, kMetaSlots>), grid(R), dim3(kBlock), 0, stream, s, c, ids, n, o, err);
        else hipLaunchKernelGGL((k_cache_gather<KK, R, kMetaRaw>), grid(R), dim3(kBlock), 0, stream, s, c, ids, n, o, err);
    };
    if (s.W <= 64) go(std::integral_constant<int, 1>{}, std::integral_constant<int, 8>{});
    else if (s.W <= 128) go(std::integral_constant<int, 2>{}, std::integral_constant<int, 4>{});
    else if (s.W <= 256) go(std::integral_constant<int, 4>{}, std::integral_constant<int, 2>{});
    else if (s.W <= 512) go(std::integral_constant<int, 8>{}, std::integral_constant<int, 1>{});
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace dev
}  // namespace ibp
