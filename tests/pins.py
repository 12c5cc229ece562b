"""Pins of the CPU oracle: checks against things other than the oracle itself.

Each check takes an oracle object (oracle.OracleLib) so that the same pins can be
run against builds of the oracle with a planted mistake (test_oracle_pins.py). The
pins come from the paper's definitions and from mathematics, never from the GPU path:
  * hand-derived worked examples (tests/golden/worked_examples.txt);
  * brute force on tiny inputs: invariance as pairwise agreement of every row
    (a different formulation from the oracle's per-bit counters), packing by
    enumerating the variant positions;
  * closed forms: stream bytes = 64 + n_groups*(2L + 8) + 8 + sum_g n_g*ceil((8L-P_g)/8);
  * identities: identical rows pack to 0 bytes, clusters of one row pack to 0 bytes,
    a cluster with an all-zero Mask packs every row to exactly its raw bytes;
  * the bound the first synthetic workload must meet (sign bit, bit 30 and
    mantissa bits 15..0 are invariant in every cluster, so a row packs to <= 224 B).

The thresholded scheme with participation bits is pinned the same way: hand-derived
examples (tests/golden/participation_examples.txt), brute force with exact rational
thresholds and whole-chunk integer comparisons, its reduction to the clustered scheme
at T = n, sampling as counting over the sampled rows only, and a closed form.
"""
from fractions import Fraction
import os

import numpy as np

from workloads import CONFIGS, gen_rows, structured_rows

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_examples.txt")
GOLDEN_PART = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "participation_examples.txt")
HEADER = 64


def parse_golden(path=GOLDEN):
    examples, cur = [], None
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        tok = line.split()
        if tok[0] == "name":
            cur = {"name": tok[1], "rows": [], "mask": {}, "bitval": {}, "rb": {}, "packed": {}}
        elif tok[0] in ("L", "G"):
            cur[tok[0]] = int(tok[1])
        elif tok[0] == "row":
            cur["rows"].append(bytes.fromhex(tok[1]))
        elif tok[0] in ("mask", "bitval"):
            cur[tok[0]][int(tok[1])] = bytes.fromhex(tok[2])
        elif tok[0] == "rb":
            cur["rb"][int(tok[1])] = int(tok[2])
        elif tok[0] == "packed":
            cur["packed"][int(tok[1])] = b"" if tok[2] == "-" else bytes.fromhex(tok[2])
        elif tok[0] == "stream":
            cur["stream"] = bytes.fromhex("".join(tok[1:]))
        elif tok[0] == "end":
            examples.append(cur)
            cur = None
    return examples


# ------------------------------------------------------------ brute force helpers

def bits_of(row):
    """Row bit p = bit p%8 of byte p//8."""
    return [(row[p // 8] >> (p % 8)) & 1 for p in range(8 * len(row))]


def brute_masks(rows):
    """Invariance as pairwise agreement: bit p is invariant iff every pair of rows agrees."""
    rb = [bits_of(bytes(r)) for r in rows]
    nbits = len(rb[0])
    mask, bitval = [0] * nbits, [0] * nbits
    for p in range(nbits):
        if all(rb[i][p] == rb[j][p] for i in range(len(rb)) for j in range(len(rb))):
            mask[p] = 1
            bitval[p] = rb[0][p]
    return _to_bytes(mask), _to_bytes(bitval)


def _to_bytes(bits):
    out = bytearray((len(bits) + 7) // 8)
    for k, b in enumerate(bits):
        if b:
            out[k // 8] |= 1 << (k % 8)
    return bytes(out)


def brute_pack(row, mask):
    """Packed row by enumerating the Mask-0 positions in ascending order."""
    rbits, mbits = bits_of(bytes(row)), bits_of(bytes(mask))
    kept = [rbits[p] for p in range(len(rbits)) if not mbits[p]]
    return _to_bytes(kept)


def np_masks(rows):
    """Mask/Bitval by AND/OR over the rows (numpy), a third formulation for big inputs."""
    a = np.bitwise_and.reduce(rows, axis=0)
    o = np.bitwise_or.reduce(rows, axis=0)
    return (~(a ^ o)).astype(np.uint8), a.astype(np.uint8)


def popcount_bytes(b):
    return int(np.unpackbits(np.frombuffer(bytes(b), np.uint8)).sum())


def closed_form_bytes(rows, G):
    n, L = rows.shape
    ng = (n + G - 1) // G
    total = HEADER + ng * (2 * L + 8) + 8
    for g in range(ng):
        grp = rows[g * G:(g + 1) * G]
        m, _ = np_masks(grp)
        P = popcount_bytes(m)
        total += grp.shape[0] * ((8 * L - P + 7) // 8)
    return total


# ------------------------------------------------------------------------ the pins

def pin_worked_examples(orc):
    for ex in parse_golden():
        L, G = ex["L"], ex["G"]
        rows = np.frombuffer(b"".join(ex["rows"]), np.uint8).reshape(-1, L)
        n = rows.shape[0]
        for g in range((n + G - 1) // G):
            m, v = orc.group_masks(rows[g * G:(g + 1) * G])
            assert bytes(m) == ex["mask"][g], (ex["name"], "mask", g)
            assert bytes(v) == ex["bitval"][g], (ex["name"], "bitval", g)
            assert orc.packed_row_bytes(m) == ex["rb"][g], (ex["name"], "rb", g)
            for r in range(g * G, min(n, (g + 1) * G)):
                assert bytes(orc.pack_row(rows[r], m)) == ex["packed"][r], (ex["name"], "packed", r)
                got = orc.unpack_row(np.frombuffer(ex["packed"][r], np.uint8), m, v)
                assert bytes(got) == bytes(rows[r]), (ex["name"], "unpack", r)
        s = orc.compress(rows, G)
        assert bytes(s) == ex["stream"], (ex["name"], "stream")
        dec = orc.decompress(np.frombuffer(ex["stream"], np.uint8), n, L)
        assert np.array_equal(dec, rows), (ex["name"], "decode")


def pin_bruteforce_random(orc, trials=60, seed=1):
    rng = np.random.default_rng(seed)
    for t in range(trials):
        L = int(rng.choice([4, 8, 12]))
        n = int(rng.integers(1, 7))
        base = rng.integers(0, 256, size=L, dtype=np.uint8)
        # flip a few random bits per row so that masks have structure
        rows = np.tile(base, (n, 1))
        for i in range(n):
            for _ in range(int(rng.integers(0, 6))):
                p = int(rng.integers(0, 8 * L))
                rows[i, p // 8] ^= np.uint8(1 << (p % 8))
        m, v = orc.group_masks(rows)
        bm, bv = brute_masks(rows)
        assert bytes(m) == bm and bytes(v) == bv, ("masks", t)
        for i in range(n):
            packed = orc.pack_row(rows[i], m)
            assert bytes(packed) == brute_pack(rows[i], bm), ("pack", t, i)
            assert bytes(orc.unpack_row(packed, m, v)) == bytes(rows[i]), ("unpack", t, i)


def pin_exhaustive_alphabet(orc):
    """Every triple of rows drawn from a 16-word alphabet of one 32-bit word."""
    alphabet = np.array([0x00000000, 0xFFFFFFFF, 0x80000000, 0x00000001, 0x7FFFFFFF,
                         0x55555555, 0xAAAAAAAA, 0x3F800000, 0xBF800000, 0x7FC00000,
                         0x00800000, 0x0000FFFF, 0xFFFF0000, 0x12345678, 0x00010000,
                         0x40490FDB], dtype=np.uint32)
    idx = np.array(np.meshgrid(np.arange(16), np.arange(16), np.arange(16), indexing="ij")).reshape(3, -1).T
    for a, b, c in idx:
        rows = alphabet[[a, b, c]].reshape(3, 1).view(np.uint8).reshape(3, 4)
        m, v = orc.group_masks(rows)
        bm, bv = brute_masks(rows)
        assert bytes(m) == bm and bytes(v) == bv, ("masks", a, b, c)
        for i in range(3):
            packed = orc.pack_row(rows[i], m)
            assert bytes(packed) == brute_pack(rows[i], bm), ("pack", a, b, c, i)
            assert bytes(orc.unpack_row(packed, m, v)) == bytes(rows[i]), ("unpack", a, b, c, i)


def pin_zero_mask_is_identity(orc):
    """Uniform random bytes: almost every cluster has Mask = 0 and then each packed
    row must be exactly the raw row (this fixes the bit order and the word order)."""
    rows = structured_rows("random", 256, 64, seed=3)
    s = orc.compress(rows, 32)
    L, G = 64, 32
    ng = 256 // G
    index_off = HEADER + ng * 2 * L
    payload_off = index_off + 8 * (ng + 1)
    seen = 0
    for g in range(ng):
        m = s[HEADER + g * 2 * L:HEADER + g * 2 * L + L]
        if m.any():
            continue
        seen += 1
        off = int(s[index_off + 8 * g:index_off + 8 * g + 8].view(np.uint64)[0])
        pay = s[payload_off + off:payload_off + off + G * L].reshape(G, L)
        assert np.array_equal(pay, rows[g * G:(g + 1) * G]), ("identity", g)
    assert seen >= ng // 2, "expected most clusters of random rows to have Mask = 0"


def pin_identical_and_single_rows(orc):
    for L in (4, 20, 64):
        rows = structured_rows("identical", 10, L, seed=L)
        s = orc.compress(rows, 4)
        ng = 3
        assert s.size == HEADER + ng * (2 * L + 8) + 8, ("identical size", L)
        m, v = orc.group_masks(rows)
        assert bytes(m) == b"\xff" * L and bytes(v) == bytes(rows[0]), ("identical masks", L)
        assert orc.packed_row_bytes(m) == 0
        assert np.array_equal(orc.decompress(s, 10, L), rows)
        # clusters of one row: every bit is invariant, nothing is packed
        r = structured_rows("random", 7, L, seed=L + 1)
        s1 = orc.compress(r, 1)
        assert s1.size == HEADER + 7 * (2 * L + 8) + 8, ("G=1 size", L)
        assert np.array_equal(orc.decompress(s1, 7, L), r)
    z = structured_rows("zeros", 5, 8)
    m, v = orc.group_masks(z)
    assert bytes(m) == b"\xff" * 8 and bytes(v) == b"\x00" * 8
    o = structured_rows("ones", 5, 8)
    m, v = orc.group_masks(o)
    assert bytes(m) == b"\xff" * 8 and bytes(v) == b"\xff" * 8


def pin_closed_form_and_round_trip(orc):
    cases = [("random", 37, 12, 5), ("floats", 100, 64, 32), ("specials", 70, 16, 7),
             ("sparse", 65, 400, 32), ("smallint", 33, 8, 32), ("alternating", 40, 24, 8),
             ("onebit", 50, 36, 10), ("zeros", 3, 4, 2), ("floats", 1, 4, 32),
             ("floats", 64, 4, 64), ("random", 9, 4, 3)]
    for kind, n, L, G in cases:
        rows = structured_rows(kind, n, L, seed=n + L)
        s = orc.compress(rows, G)
        assert s.size == closed_form_bytes(rows, G), ("closed form", kind, n, L, G)
        assert bytes(s[:4]) == b"IBP1"
        hdr = s[:64]
        assert int(hdr[8:12].view(np.uint32)[0]) == L and int(hdr[12:16].view(np.uint32)[0]) == G
        assert int(hdr[16:24].view(np.uint64)[0]) == n
        dec = orc.decompress(s, n, L)
        assert np.array_equal(dec, rows), ("round trip", kind, n, L, G)
        # decode in a scrambled order with repeats
        ids = np.random.default_rng(n).integers(0, n, size=2 * n)
        assert np.array_equal(orc.decode_rows(s, ids, L), rows[ids]), ("gather", kind)


def pin_tiny_gnn_bound(orc):
    """The first synthetic workload (values k/256 or +0.0): sign bit, bit 30 and
    mantissa bits 15..0 are invariant in every cluster, so a row packs to <= 224 B."""
    cfg = CONFIGS["tiny_gnn"]
    rows = gen_rows(cfg, 0, 1024)
    G, L = cfg.group_rows, cfg.row_bytes
    want = np.zeros(L, np.uint8).view(np.uint32)
    want[:] = 0xC000FFFF
    want = want.view(np.uint8)
    for g in range(1024 // G):
        m, v = orc.group_masks(rows[g * G:(g + 1) * G])
        assert np.array_equal(m & want, want), ("expected invariant bits", g)
        assert not (v & want).any(), ("those invariant bits are 0", g)
        assert orc.packed_row_bytes(m) <= 224, g


# ------------------------------------------ thresholded scheme, participation bits

def parse_golden_part(path=GOLDEN_PART):
    examples, cur = [], None
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        tok = line.split()
        if tok[0] == "name":
            cur = {"name": tok[1], "rows": [], "size": {}, "packed": {}}
        elif tok[0] in ("L", "G", "chunk"):
            cur[tok[0]] = int(tok[1])
        elif tok[0] == "threshold":
            cur["threshold"] = (int(tok[1]), int(tok[2]))
        elif tok[0] == "row":
            cur["rows"].append(bytes.fromhex(tok[1]))
        elif tok[0] in ("mask", "bitval"):
            cur[tok[0]] = bytes.fromhex(tok[1])
        elif tok[0] == "size":
            cur["size"][int(tok[1])] = int(tok[2])
        elif tok[0] == "packed":
            cur["packed"][int(tok[1])] = bytes.fromhex(tok[2])
        elif tok[0] == "stream":
            cur["stream"] = bytes.fromhex("".join(tok[1:]))
        elif tok[0] == "end":
            examples.append(cur)
            cur = None
    return examples


def brute_thr_masks(rows, num, den, every=1):
    """Mask/Bitval as exact fractions of the counted rows agreeing on each bit."""
    counted = [bits_of(bytes(r)) for r in rows[::every]]
    n, t = len(counted), Fraction(num, den)
    nbits = len(counted[0])
    mask, bitval = [0] * nbits, [0] * nbits
    for p in range(nbits):
        ones = Fraction(sum(b[p] for b in counted), n)
        if ones >= t:
            mask[p], bitval[p] = 1, 1
        elif 1 - ones >= t:
            mask[p] = 1
    return _to_bytes(mask), _to_bytes(bitval)


def brute_part_pack(row, mask, bitval, cs):
    """The participation-scheme encoding of one row, chunk by chunk with whole-chunk
    integer comparisons; returns the packed bytes (the raw row when nothing is saved)."""
    row, mask, bitval = bytes(row), bytes(mask), bytes(bitval)
    L = len(row)
    chunks = L // cs
    comp, saved = [], 0
    for c in range(chunks):
        x = int.from_bytes(row[c * cs:(c + 1) * cs], "little")
        m = int.from_bytes(mask[c * cs:(c + 1) * cs], "little")
        b = int.from_bytes(bitval[c * cs:(c + 1) * cs], "little")
        ok = (x & m) == b
        comp.append(ok)
        saved += bin(m).count("1") if ok else 0
    if saved - chunks < 8:
        return row
    out = [1 if ok else 0 for ok in comp]
    for c in range(chunks):
        x = int.from_bytes(row[c * cs:(c + 1) * cs], "little")
        m = int.from_bytes(mask[c * cs:(c + 1) * cs], "little")
        for q in range(8 * cs):
            if comp[c] and (m >> q) & 1:
                continue
            out.append((x >> q) & 1)
    size = L - (saved - chunks) // 8
    packed = _to_bytes(out)
    return packed + bytes(size - len(packed))


def part_closed_form_bytes(rows, G, cs, num, den, every):
    n, L = rows.shape
    ng = (n + G - 1) // G
    total = HEADER + ng * 2 * L + 8 * (n + 1)
    for g in range(ng):
        grp = rows[g * G:(g + 1) * G]
        m, v = brute_thr_masks(grp, num, den, every) if L <= 16 else _np_thr_masks(grp, num, den, every)
        for r in grp:
            total += len(brute_part_pack(r, m, v, cs))
    return total


def _np_thr_masks(rows, num, den, every):
    """numpy form of the threshold rule for wider rows (exact integer comparisons)."""
    sel = rows[::every]
    n = sel.shape[0]
    cnt = np.unpackbits(sel, axis=1, bitorder="little").sum(axis=0).astype(np.int64)
    one = cnt * den >= num * n
    zero = ~one & ((n - cnt) * den >= num * n)
    return (bytes(np.packbits(one | zero, bitorder="little")),
            bytes(np.packbits(one, bitorder="little")))


def pin_part_worked_examples(orc):
    for ex in parse_golden_part():
        L, G, cs, (num, den) = ex["L"], ex["G"], ex["chunk"], ex["threshold"]
        rows = np.frombuffer(b"".join(ex["rows"]), np.uint8).reshape(-1, L)
        m, v = orc.thr_masks(rows, num, den)
        assert bytes(m) == ex["mask"] and bytes(v) == ex["bitval"], (ex["name"], "masks")
        for r in range(rows.shape[0]):
            assert orc.part_row_bytes(rows[r], m, v, cs) == ex["size"][r], (ex["name"], "size", r)
            assert bytes(orc.part_pack_row(rows[r], m, v, cs)) == ex["packed"][r], (ex["name"], "packed", r)
            got = orc.part_unpack_row(np.frombuffer(ex["packed"][r], np.uint8), m, v, cs)
            assert bytes(got) == bytes(rows[r]), (ex["name"], "unpack", r)
        s = orc.compress(rows, G, chunk_bytes=cs, threshold=(num, den))
        assert bytes(s) == ex["stream"], (ex["name"], "stream")
        assert np.array_equal(orc.decompress(s, rows.shape[0], L), rows), (ex["name"], "decode")


def pin_part_bruteforce(orc, trials=80, seed=5):
    """Random small clusters with structure, random thresholds, chunk sizes and sampling."""
    rng = np.random.default_rng(seed)
    for t in range(trials):
        cs = int(rng.choice([4, 8]))
        L = cs * int(rng.integers(1, 4))
        n = int(rng.integers(1, 12))
        base = rng.integers(0, 256, size=L, dtype=np.uint8)
        rows = np.tile(base, (n, 1))
        for i in range(n):
            for _ in range(int(rng.integers(0, 10))):
                p = int(rng.integers(0, 8 * L))
                rows[i, p // 8] ^= np.uint8(1 << (p % 8))
        den = int(rng.integers(2, 11))
        num = int(rng.integers(den // 2 + 1, den + 1))
        every = int(rng.choice([1, 1, 2, 3]))
        m, v = orc.thr_masks(rows, num, den, every)
        bm, bv = brute_thr_masks(rows, num, den, every)
        assert bytes(m) == bm and bytes(v) == bv, ("thr masks", t)
        for i in range(n):
            want = brute_part_pack(rows[i], bm, bv, cs)
            got = orc.part_pack_row(rows[i], m, v, cs)
            assert orc.part_row_bytes(rows[i], m, v, cs) == len(want), ("size", t, i)
            assert bytes(got) == want, ("pack", t, i)
            assert bytes(orc.part_unpack_row(got, m, v, cs)) == bytes(rows[i]), ("unpack", t, i)


def pin_part_random_metadata(orc, trials=200, seed=6):
    """Any Mask/Bitval (Bitval inside Mask), not only ones derived from the rows: the
    encoding and the raw fallback must still round-trip and match brute force."""
    rng = np.random.default_rng(seed)
    for t in range(trials):
        cs = int(rng.choice([4, 8, 12]))
        L = cs * int(rng.integers(1, 3))
        row = rng.integers(0, 256, size=L, dtype=np.uint8)
        mask = rng.integers(0, 256, size=L, dtype=np.uint8) | (0xFF if t % 3 == 0 else 0)
        mask = mask.astype(np.uint8)
        bitval = (rng.integers(0, 256, size=L, dtype=np.uint8) & mask).astype(np.uint8)
        if t % 2 == 0:      # make most chunks match
            bitval = (row & mask).astype(np.uint8)
            j = int(rng.integers(0, L))
            bitval[j] ^= mask[j] & np.uint8(1 << int(rng.integers(0, 8)))
        want = brute_part_pack(row, mask, bitval, cs)
        got = orc.part_pack_row(row, mask, bitval, cs)
        assert bytes(got) == want, ("pack", t)
        assert bytes(orc.part_unpack_row(got, mask, bitval, cs)) == bytes(row), ("unpack", t)


def pin_part_raw_fallback_boundary(orc):
    """A row of C chunks that saves `saved` Mask bits is stored raw exactly while
    saved - C < 8 (bytes saved = floor((saved - C) / 8) <= 0): sweep saved across that
    boundary with every chunk compressible, for several chunk counts."""
    rng = np.random.default_rng(11)
    for L, cs in [(32, 4), (64, 8), (16, 4), (48, 4)]:
        chunks = L // cs
        for saved in range(0, min(8 * L, chunks + 20)):
            row = rng.integers(0, 256, size=L, dtype=np.uint8)
            pos = rng.permutation(8 * L)[:saved]
            mbits = np.zeros(8 * L, np.uint8)
            mbits[pos] = 1
            mask = np.packbits(mbits, bitorder="little")
            bitval = (row & mask).astype(np.uint8)          # every chunk compressible
            size = orc.part_row_bytes(row, mask, bitval, cs)
            want = L if saved - chunks < 8 else L - (saved - chunks) // 8
            assert size == want, (L, cs, saved, size, want)
            got = orc.part_pack_row(row, mask, bitval, cs)
            assert bytes(got) == brute_part_pack(row, mask, bitval, cs), (L, cs, saved)
            assert bytes(orc.part_unpack_row(got, mask, bitval, cs)) == bytes(row), (L, cs, saved)


def pin_part_reduces_to_clustered(orc):
    """At T = n every counted row agrees on every Mask bit, so every chunk participates:
    the masks equal the clustered scheme's, each row's part bits are all 1, and the bits
    after them are the clustered scheme's packed bits."""
    for kind, n, L, G, cs in [("floats", 64, 64, 32, 4), ("sparse", 40, 128, 16, 8), ("smallint", 33, 16, 32, 4),
                              ("onebit", 20, 24, 10, 8)]:
        rows = structured_rows(kind, n, L, seed=n * L)
        for g in range((n + G - 1) // G):
            grp = rows[g * G:(g + 1) * G]
            m1, v1 = orc.group_masks(grp)
            m2, v2 = orc.thr_masks(grp, 1, 1, 1)
            assert bytes(m1) == bytes(m2) and bytes(v1) == bytes(v2), (kind, g)
            chunks = L // cs
            for r in grp:
                pk = orc.part_pack_row(r, m2, v2, cs)
                if pk.size == L and (8 * L - popcount_bytes(m1)) + chunks > 8 * L - 8:
                    continue      # nothing saved: stored raw
                bits = np.unpackbits(pk, bitorder="little")
                assert bits[:chunks].all(), (kind, "part bits")
                v1bits = np.unpackbits(orc.pack_row(r, m1), bitorder="little")[:8 * L - popcount_bytes(m1)]
                assert np.array_equal(bits[chunks:chunks + v1bits.size], v1bits), (kind, "payload")


def pin_part_sampling_and_closed_form(orc):
    """Sampled masks count only rows 0, k, 2k, ... of each cluster; stream size by the
    closed form 64 + n_groups * 2L + 8 (n + 1) + sum of row sizes; round trips."""
    cases = [("floats", 70, 16, 32, 4, (4, 5), 1), ("sparse", 50, 32, 64, 8, (3, 4), 2),
             ("random", 21, 8, 7, 4, (9, 10), 1), ("specials", 40, 16, 40, 8, (7, 10), 3),
             ("smallint", 33, 12, 11, 4, (1, 1), 1), ("floats", 1, 8, 4, 8, (4, 5), 1)]
    for kind, n, L, G, cs, (num, den), every in cases:
        rows = structured_rows(kind, n, L, seed=n + 7 * L)
        for g in range((n + G - 1) // G):
            grp = rows[g * G:(g + 1) * G]
            m, v = orc.thr_masks(grp, num, den, every)
            ms, vs = orc.thr_masks(np.ascontiguousarray(grp[::every]), num, den, 1)
            assert bytes(m) == bytes(ms) and bytes(v) == bytes(vs), ("sampling", kind, g)
        s = orc.compress(rows, G, chunk_bytes=cs, threshold=(num, den), sample_every=every)
        assert s.size == part_closed_form_bytes(rows, G, cs, num, den, every), ("closed form", kind)
        assert int(s[32:36].view(np.uint32)[0]) == 1 and int(s[36:40].view(np.uint32)[0]) == cs
        assert np.array_equal(orc.decompress(s, n, L), rows), ("round trip", kind)
        ids = np.random.default_rng(n).integers(0, n, size=2 * n)
        assert np.array_equal(orc.decode_rows(s, ids, L), rows[ids]), ("gather", kind)


ALL_PINS = [pin_worked_examples, pin_bruteforce_random, pin_exhaustive_alphabet,
            pin_zero_mask_is_identity, pin_identical_and_single_rows,
            pin_closed_form_and_round_trip, pin_tiny_gnn_bound,
            pin_part_worked_examples, pin_part_bruteforce, pin_part_random_metadata,
            pin_part_raw_fallback_boundary, pin_part_reduces_to_clustered,
            pin_part_sampling_and_closed_form]
