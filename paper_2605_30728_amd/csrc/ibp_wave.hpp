// Wave64 building blocks shared by the gfx950 decode kernels: lane/wave indexing, DPP
// scans and reductions, per-row offsets, the holes deposit and the XCD-aware block order.
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

#include "ibp_device.hpp"

namespace ibp {
namespace dev {

inline constexpr int kWave = 64;
inline constexpr int kWavesPerBlock = 4;
inline constexpr int kBlock = kWave * kWavesPerBlock;

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// Inclusive prefix sum over the 64 lanes of a wave: row_shr 1/2/4/8 scan each row of
// 16 lanes, row_bcast:15 carries rows 0->1 and 2->3, row_bcast:31 carries rows 0-1
// into rows 2-3. Disabled or out-of-row sources contribute 0 (old value 0).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
    int x = (int)v;
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
    return (uint32_t)x;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(v), 63);
}

// Distance between consecutive packed rows of a cluster: the packed size, or the packed
// size rounded up to `align` bytes (a power of two) when rows start on aligned slots.
__device__ __forceinline__ uint64_t row_stride(uint64_t rb, uint32_t align) {
    return align ? (rb + align - 1) & ~(uint64_t)(align - 1) : rb;
}

__device__ __forceinline__ uint64_t wave_slot() {
    return (uint64_t)blockIdx.x * kWavesPerBlock +
           (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

// How the row gathers read a cluster's Mask/Bitval words: the raw words, or the
// cluster's compact slot (P = 8 or 16 {Mask, Bitval} u32 pairs, then the 4-bit pair
// indices, lane l's K indices in bits [4Kl, 4Kl + 4K)), used when every cluster of the
// stream fits one.
enum { kMetaRaw = 0, kMetaSlots = 1 };

// A row's metadata as loaded: raw v[2j] = Mask, v[2j+1] = Bitval of word l + 64j; slots
// v[0], v[1] = pair l mod P, v[2] = the lane's index bits.
template <int K, int FORM>
struct RowMeta {
    uint32_t v[FORM == kMetaSlots ? 3 : 2 * K];
};

// Issue a row's metadata loads (every address inside the slot or clamped inside the row,
// so none is exec-masked).
template <int K, int FORM>
__device__ __forceinline__ void load_row_meta(RowMeta<K, FORM> &r, const uint32_t *__restrict__ mg,
                                              const uint8_t *__restrict__ slot, uint32_t P, uint32_t W) {
    const uint32_t l = lane_id();
    if constexpr (FORM == kMetaSlots) {
        const uint2 p = reinterpret_cast<const uint2 *>(slot)[l & (P - 1)];
        r.v[0] = p.x;
        r.v[1] = p.y;
        const uint8_t *__restrict__ idx = slot + 8 * P;
        if constexpr (K == 1) r.v[2] = idx[l >> 1];
        else if constexpr (K == 2) r.v[2] = idx[l];
        else if constexpr (K == 4) r.v[2] = reinterpret_cast<const uint16_t *>(idx)[l];
        else r.v[2] = reinterpret_cast<const uint32_t *>(idx)[l];
    } else {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint32_t w = min(l + kWave * j, W - 1);
            r.v[2 * j] = mg[w];
            r.v[2 * j + 1] = mg[W + w];
        }
    }
}

// Makes the loaded words values needed at this point of the program, so the compiler
// can neither sink the loads into the branches that use them nor interleave them with
// the arithmetic of earlier rows: a batch's loads all leave before the first one is
// waited for, and the batch pays one memory round trip instead of one per row.
template <int K, int FORM>
__device__ __forceinline__ void hold_row_meta(RowMeta<K, FORM> &r) {
#pragma unroll
    for (int k = 0; k < (int)(sizeof(r.v) / sizeof(r.v[0])); ++k) asm volatile("" : "+v"(r.v[k]));
}

// The lane's K Mask and Bitval words; from a slot, each word takes its pair from the
// lane that holds it (ds_bpermute).
template <int K, int FORM>
__device__ __forceinline__ void expand_row_meta(const RowMeta<K, FORM> &r, uint32_t (&m)[K], uint32_t (&b)[K]) {
    if constexpr (FORM == kMetaSlots) {
        const uint32_t bits = K == 1 ? r.v[2] >> ((lane_id() & 1u) * 4u) : r.v[2];
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const int a = (int)(((bits >> (4 * j)) & 15u) * 4u);
            m[j] = (uint32_t)__builtin_amdgcn_ds_bpermute(a, (int)r.v[0]);
            b[j] = (uint32_t)__builtin_amdgcn_ds_bpermute(a, (int)r.v[1]);
        }
    } else {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            m[j] = r.v[2 * j];
            b[j] = r.v[2 * j + 1];
        }
    }
}

// A buffer resource over the dwords of one packed row (from `p`, `bytes` of them, a
// multiple of 4): a buffer load at a byte offset at or past `bytes` returns 0 without
// touching memory (the buffer range check), so a row's window loads, which read each
// word's two dwords and for lanes past the row's last word the dword after it, never
// fetch the line after the row's last packed dword. 0x00020000 is the gfx9 descriptor's
// fourth dword for raw 32-bit buffer loads.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const uint32_t *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t *>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint32_t row_dword(__amdgpu_buffer_rsrc_t r, uint32_t q) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)(q * 4u), 0, 0);
}

// A word's 64-bit window as two dword loads (dwords q and q + 1 of p). The compiler would
// merge them into one 8-byte load, which is misaligned for every odd q; an opaque second
// index keeps them two 4-byte loads. Measured: the 111M-row gather 830 -> 695 us, the bf16
// KV layer decompress 46.3 -> 43.0 us; the thresholded kernels keep the merged load (their
// KV layer measured 5% slower split, their gathers no faster).
__device__ __forceinline__ void load_window(const uint32_t *__restrict__ p, uint32_t q, uint32_t &d0, uint32_t &d1) {
    uint32_t q1 = q + 1u;
    asm volatile("" : "+v"(q1));
    d0 = p[q];
    d1 = p[q1];
}
__device__ __forceinline__ void load_window(__amdgpu_buffer_rsrc_t r, uint32_t q, uint32_t &d0, uint32_t &d1) {
    uint32_t q1 = q + 1u;
    asm volatile("" : "+v"(q1));
    d0 = row_dword(r, q);
    d1 = row_dword(r, q1);
}

// Store of a gathered output word that no later step of the kernel reads: marked
// non-temporal, so a gather's output stream does not evict the metadata slots and packed
// rows that neighbouring requests are about to read from L2 (measured: 7% on 53k Zipf
// lookups, whose hot rows repeat across waves; the contiguous decompress keeps plain
// stores, which measured 7% faster there).
__device__ __forceinline__ void store_out(uint32_t *p, uint32_t v) { __builtin_nontemporal_store(v, p); }

// Maximum over the 64 lanes of a wave (DPP, as the scan), result in every lane's SGPR.
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
    int x = (int)v;
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false));  // row_shr:1
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false));  // row_shr:2
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false));  // row_shr:4
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false));  // row_shr:8
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false));  // row_bcast:15
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false));  // row_bcast:31
    return (uint32_t)__builtin_amdgcn_readlane(x, 63);
}

// Deposit by holes. The variant positions nm of a word span [lo, hi]; inside that span
// the invariant positions form "holes" (runs of invariant bits). Shifting the packed
// bits x up to lo places them contiguously; opening a gap of the right width at every
// hole, lowest first (bits at and above the hole move up by its width), puts each bit on
// its variant position, and Bitval fills the rest. A word with r runs of variant bits
// has r - 1 holes.
__device__ __forceinline__ uint32_t run_count(uint32_t v) { return (uint32_t)__builtin_popcount(v & ~(v << 1)); }

// Most runs of variant bits in any word of a row, from its slot of P (8 or 16) pairs: lane
// l holds pair l mod P, so lanes 0 .. P-1 hold every pair of the cluster (unused entries
// have Mask 0, one run, which never raises a row's hole count above that of its words).
template <int K>
__device__ __forceinline__ uint32_t slot_max_runs(const RowMeta<K, kMetaSlots> &r, uint32_t P) {
    int x = (int)run_count(~r.v[0]);
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false));  // row_shr:1
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false));  // row_shr:2
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false));  // row_shr:4
    if (P > 8) x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false));  // row_shr:8
    return (uint32_t)__builtin_amdgcn_readlane(x, (int)P - 1);
}

// nh is wave-uniform and at least the word's own hole count; extra iterations find no
// hole (below = all but bit 31, width 0) and leave y as it is.
__device__ __forceinline__ uint32_t word_deposit(uint32_t bv, uint32_t nm, uint32_t x, uint32_t nh) {
    const uint32_t lo = (uint32_t)__builtin_ctz(nm | 0x80000000u);
    // span [lo, hi] (nm = 0 gives garbage that the final select discards)
    const uint32_t span = (0xFFFFFFFFu >> __builtin_clz(nm | 1u)) & (0xFFFFFFFFu << lo);
    uint32_t holes = span & ~nm;   // never holds bit 31: the top of the span is variant
    uint32_t y = x << lo;
    for (uint32_t k = 0; k < nh; ++k) {
        const uint32_t pos = (uint32_t)__builtin_ctz(holes | 0x80000000u);
        const uint32_t t = holes + (1u << pos);      // carries through the lowest hole
        const uint32_t width = (uint32_t)__builtin_popcount(holes & ~t);
        holes &= t;
        const uint32_t below = (1u << pos) - 1u;
        y = (y & below) | ((y << width) & ~below);
    }
    return (nm & y) | (~nm & bv);
}

// Exclusive bit offsets of the lane's words inside a packed row (word order t + 64*j)
// and the row's total packed bits. Two strides share one wave scan: every count is at
// most 32, so every prefix is at most 2048 and fits a 16-bit field.
template <int K>
__device__ __forceinline__ uint32_t row_offsets(const uint32_t (&n)[K], uint32_t (&s)[K]) {
    uint32_t c = 0;
#pragma unroll
    for (int j = 0; j < K; j += 2) {
        if (j + 1 < K) {
            const uint32_t v = n[j] | (n[j + 1] << 16);
            const uint32_t inc = wave_incl_scan(v);
            const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
            s[j] = c + (inc & 0xFFFFu) - n[j];
            c += tot & 0xFFFFu;
            s[j + 1] = c + (inc >> 16) - n[j + 1];
            c += tot >> 16;
        } else {
            const uint32_t inc = wave_incl_scan(n[j]);
            s[j] = c + inc - n[j];
            c += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
        }
    }
    return c;
}

// Blocks are dealt to the 8 XCDs round-robin; renumber them so that consecutive
// logical blocks (neighbouring sorted ids, which share clusters) run on one XCD and
// share its L2. A bijection on [0, nblocks) for any nblocks.
__device__ __forceinline__ uint32_t xcd_block(uint32_t b, uint32_t nblocks) {
    constexpr uint32_t kXcd = 8;
    const uint32_t xcd = b % kXcd, idx = b / kXcd;
    const uint32_t per = nblocks / kXcd, extra = nblocks % kXcd;
    return xcd * per + min(xcd, extra) + idx;
}

}  // namespace dev
}  // namespace ibp
