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
"""
import os

import numpy as np

from workloads import CONFIGS, gen_rows, structured_rows

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_examples.txt")
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


ALL_PINS = [pin_worked_examples, pin_bruteforce_random, pin_exhaustive_alphabet,
            pin_zero_mask_is_identity, pin_identical_and_single_rows,
            pin_closed_form_and_round_trip, pin_tiny_gnn_bound]
