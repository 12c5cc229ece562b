"""TEST INFRASTRUCTURE ONLY: the CPU oracle of Invariant Bit Packing.

A plain, slow, single-threaded implementation written from the paper (Sec. 4.1-4.3
and Sec. 6.5): the clustered scheme with T = cluster size, and the thresholded scheme
with participation bits and raw fallback. It is used to check the library. Only
tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may import it; the
product package never does.

The arithmetic lives in ibp_oracle.c (bit-serial C); this module only marshals
numpy arrays into it. `OracleLib(path)` wraps any build of that file, so tests can
also load variants with a planted mistake and check that the pins catch them.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_u8p = ctypes.POINTER(ctypes.c_uint8)


def _u8(a):
    if a.size == 0:
        a = np.zeros(1, np.uint8)
    return a.ctypes.data_as(_u8p)


def _as_rows(rows):
    a = np.ascontiguousarray(rows)
    if a.ndim != 2:
        raise ValueError("rows must be 2-D (n_rows, bytes or elements)")
    n = a.shape[0]
    L = a.shape[1] * a.itemsize
    b = a.view(np.uint8).reshape(n, L) if n else np.zeros((0, L), np.uint8)
    return b, n, L


class OracleLib:
    """ctypes view of one build of ibp_oracle.c."""

    def __init__(self, path=None):
        if path is None:
            path = _build.LIB
            if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
                _build.build()
        lib = ctypes.CDLL(path)
        u64, u32 = ctypes.c_uint64, ctypes.c_uint32
        lib.ibpo_group_masks.argtypes = [_u8p, u64, u32, _u8p, _u8p]
        lib.ibpo_group_masks.restype = None
        lib.ibpo_packed_row_bytes.argtypes = [_u8p, u32]
        lib.ibpo_packed_row_bytes.restype = u64
        lib.ibpo_pack_row.argtypes = [_u8p, _u8p, u32, _u8p]
        lib.ibpo_pack_row.restype = None
        lib.ibpo_unpack_row.argtypes = [_u8p, _u8p, _u8p, u32, _u8p]
        lib.ibpo_unpack_row.restype = None
        lib.ibpo_stream_bytes.argtypes = [_u8p, u64, u32, u32]
        lib.ibpo_stream_bytes.restype = u64
        lib.ibpo_compress.argtypes = [_u8p, u64, u32, u32, _u8p, u64, ctypes.POINTER(u64)]
        lib.ibpo_compress.restype = ctypes.c_int
        lib.ibpo_decode_rows.argtypes = [_u8p, u64, ctypes.POINTER(ctypes.c_int64), u64, _u8p]
        lib.ibpo_decode_rows.restype = ctypes.c_int
        lib.ibpo_thr_masks.argtypes = [_u8p, u64, u32, u32, u32, u32, _u8p, _u8p]
        lib.ibpo_thr_masks.restype = None
        lib.ibpo_part_row_bytes.argtypes = [_u8p, _u8p, _u8p, u32, u32]
        lib.ibpo_part_row_bytes.restype = u64
        lib.ibpo_part_pack_row.argtypes = [_u8p, _u8p, _u8p, u32, u32, _u8p]
        lib.ibpo_part_pack_row.restype = None
        lib.ibpo_part_unpack_row.argtypes = [_u8p, u64, _u8p, _u8p, u32, u32, _u8p]
        lib.ibpo_part_unpack_row.restype = None
        lib.ibpo_part_stream_bytes.argtypes = [_u8p, u64, u32, u32, u32, u32, u32, u32]
        lib.ibpo_part_stream_bytes.restype = u64
        lib.ibpo_part_compress.argtypes = [_u8p, u64, u32, u32, u32, u32, u32, u32, _u8p, u64,
                                           ctypes.POINTER(u64)]
        lib.ibpo_part_compress.restype = ctypes.c_int
        lib.ibpo_part_decode_rows.argtypes = [_u8p, u64, ctypes.POINTER(ctypes.c_int64), u64, _u8p]
        lib.ibpo_part_decode_rows.restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def group_masks(self, rows):
        """Mask and Bitval (uint8, L bytes each) of one cluster of rows (Sec. 4.1, T = n)."""
        b, n, L = _as_rows(rows)
        m = np.zeros(L, np.uint8)
        v = np.zeros(L, np.uint8)
        self.lib.ibpo_group_masks(_u8(b), n, L, _u8(m), _u8(v))
        return m, v

    def packed_row_bytes(self, mask):
        """Bytes of one packed row under this Mask (Fig. 4 size rule, no participation bits)."""
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        return int(self.lib.ibpo_packed_row_bytes(_u8(m), m.size))

    def pack_row(self, row, mask):
        """Packed bytes of one row: its Mask-0 bits in ascending order (Sec. 4.2)."""
        r = np.ascontiguousarray(row).view(np.uint8).reshape(-1)
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        out = np.zeros(self.packed_row_bytes(m), np.uint8)
        self.lib.ibpo_pack_row(_u8(r), _u8(m), m.size, _u8(out))
        return out

    def unpack_row(self, packed, mask, bitval):
        """One row rebuilt from its packed bits and its cluster's Mask/Bitval (Sec. 4.3)."""
        p = np.ascontiguousarray(packed, dtype=np.uint8)
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        v = np.ascontiguousarray(bitval, dtype=np.uint8)
        out = np.zeros(m.size, np.uint8)
        self.lib.ibpo_unpack_row(_u8(p), _u8(m), _u8(v), m.size, _u8(out))
        return out

    def stream_bytes(self, rows, group_rows):
        b, n, L = _as_rows(rows)
        return int(self.lib.ibpo_stream_bytes(_u8(b), n, L, group_rows))

    # ---- thresholded scheme with participation bits (Sec. 4.1-4.2, T < N)

    def thr_masks(self, rows, num, den, every=1):
        """Mask and Bitval of one cluster under T = (num/den) * n over every k-th row."""
        b, n, L = _as_rows(rows)
        m = np.zeros(L, np.uint8)
        v = np.zeros(L, np.uint8)
        self.lib.ibpo_thr_masks(_u8(b), n, L, num, den, every, _u8(m), _u8(v))
        return m, v

    def part_row_bytes(self, row, mask, bitval, chunk_bytes):
        r = np.ascontiguousarray(row).view(np.uint8).reshape(-1)
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        v = np.ascontiguousarray(bitval, dtype=np.uint8)
        return int(self.lib.ibpo_part_row_bytes(_u8(r), _u8(m), _u8(v), m.size, chunk_bytes))

    def part_pack_row(self, row, mask, bitval, chunk_bytes):
        r = np.ascontiguousarray(row).view(np.uint8).reshape(-1)
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        v = np.ascontiguousarray(bitval, dtype=np.uint8)
        out = np.zeros(self.part_row_bytes(r, m, v, chunk_bytes), np.uint8)
        self.lib.ibpo_part_pack_row(_u8(r), _u8(m), _u8(v), m.size, chunk_bytes, _u8(out))
        return out

    def part_unpack_row(self, packed, mask, bitval, chunk_bytes):
        p = np.ascontiguousarray(packed, dtype=np.uint8)
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        v = np.ascontiguousarray(bitval, dtype=np.uint8)
        out = np.zeros(m.size, np.uint8)
        self.lib.ibpo_part_unpack_row(_u8(p), p.size, _u8(m), _u8(v), m.size, chunk_bytes, _u8(out))
        return out

    def compress(self, rows, group_rows, chunk_bytes=0, threshold=(1, 1), sample_every=1):
        """The whole compressed stream (numpy uint8) of rows in clusters of group_rows.

        chunk_bytes = 0: the clustered scheme with T = cluster size and no participation
        bits (threshold must be (1, 1), every row counted). chunk_bytes > 0: the
        thresholded scheme, T = threshold[0] / threshold[1] of the counted rows, one
        participation bit per chunk, counters over every sample_every-th row."""
        if chunk_bytes:
            return self._part_compress(rows, group_rows, chunk_bytes, threshold, sample_every)
        if tuple(threshold) != (1, 1) or sample_every != 1:
            raise ValueError("a threshold below 1 or a sampled Mask needs participation bits (chunk_bytes > 0)")
        b, n, L = _as_rows(rows)
        size = self.lib.ibpo_stream_bytes(_u8(b), n, L, group_rows)
        if size == 0:
            raise ValueError("row bytes must be a positive multiple of 4 and G >= 1")
        out = np.zeros(size, np.uint8)
        got = ctypes.c_uint64(0)
        rc = self.lib.ibpo_compress(_u8(b), n, L, group_rows, _u8(out), size, ctypes.byref(got))
        if rc != 0:
            raise RuntimeError(f"ibpo_compress failed with {rc}")
        return out

    def _part_compress(self, rows, group_rows, chunk_bytes, threshold, sample_every):
        b, n, L = _as_rows(rows)
        num, den = threshold
        size = self.lib.ibpo_part_stream_bytes(_u8(b), n, L, group_rows, chunk_bytes, num, den, sample_every)
        if size == 0:
            raise ValueError("bad arguments for the participation scheme")
        out = np.zeros(size, np.uint8)
        got = ctypes.c_uint64(0)
        rc = self.lib.ibpo_part_compress(_u8(b), n, L, group_rows, chunk_bytes, num, den, sample_every,
                                         _u8(out), size, ctypes.byref(got))
        if rc != 0:
            raise RuntimeError(f"ibpo_part_compress failed with {rc}")
        return out

    def decode_rows(self, stream, ids, row_bytes):
        """Rows `ids` of a stream decoded bit by bit: uint8 array (n_ids, row_bytes)."""
        s = np.ascontiguousarray(stream, dtype=np.uint8)
        i = np.ascontiguousarray(ids, dtype=np.int64)
        out = np.zeros((i.size, row_bytes), np.uint8)
        part = s.size >= 64 and int(s[32:36].view(np.uint32)[0]) == 1
        fn = self.lib.ibpo_part_decode_rows if part else self.lib.ibpo_decode_rows
        rc = fn(_u8(s), s.size, i.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), i.size, _u8(out))
        if rc != 0:
            raise ValueError(f"ibpo_decode_rows failed with {rc}")
        return out

    def decompress(self, stream, n_rows, row_bytes):
        """All rows of a stream."""
        return self.decode_rows(stream, np.arange(n_rows, dtype=np.int64), row_bytes)


_default = None


def default():
    global _default
    if _default is None:
        _default = OracleLib()
    return _default


def group_masks(rows):
    return default().group_masks(rows)


def packed_row_bytes(mask):
    return default().packed_row_bytes(mask)


def pack_row(row, mask):
    return default().pack_row(row, mask)


def unpack_row(packed, mask, bitval):
    return default().unpack_row(packed, mask, bitval)


def stream_bytes(rows, group_rows):
    return default().stream_bytes(rows, group_rows)


def compress(rows, group_rows, chunk_bytes=0, threshold=(1, 1), sample_every=1):
    return default().compress(rows, group_rows, chunk_bytes, threshold, sample_every)


def thr_masks(rows, num, den, every=1):
    return default().thr_masks(rows, num, den, every)


def part_row_bytes(row, mask, bitval, chunk_bytes):
    return default().part_row_bytes(row, mask, bitval, chunk_bytes)


def part_pack_row(row, mask, bitval, chunk_bytes):
    return default().part_pack_row(row, mask, bitval, chunk_bytes)


def part_unpack_row(packed, mask, bitval, chunk_bytes):
    return default().part_unpack_row(packed, mask, bitval, chunk_bytes)


def decode_rows(stream, ids, row_bytes):
    return default().decode_rows(stream, ids, row_bytes)


def decompress(stream, n_rows, row_bytes):
    return default().decompress(stream, n_rows, row_bytes)
