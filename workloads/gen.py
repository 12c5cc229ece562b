"""Seeded generators for the five synthetic workloads and for test inputs.

Conventions (so any row range can be regenerated on its own):
  * numpy Generator(PCG64) seeded with SeedSequence(seed, spawn_key=(purpose, chunk));
  * rows are drawn in chunks of CHUNK_ROWS = 2**20 rows, chunk c covering rows
    [c * CHUNK_ROWS, (c + 1) * CHUNK_ROWS);
  * purposes: 0 = row values, 1 = batch ids, 2 = outlier channels, 3 = table permutations,
    4 = fixed-bit patterns of the decompression microbenchmark.

The workloads stand in for the paper's datasets, which are not available here:
OGB-Products-like GNN features, Criteo-like DLRM embedding tables, an LLM KV cache
in bfloat16, and a papers100M-like large feature table (the paper's Sec. 6 workloads).
Only shapes, sizes and value structure are imitated.
"""
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
import os

import numpy as np

CHUNK_ROWS = 1 << 20
P_VALUES, P_IDS, P_OUTLIERS, P_PERM, P_MICRO = 0, 1, 2, 3, 4


def chunk_rng(seed, purpose, chunk):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(purpose, chunk))))


@dataclass(frozen=True)
class Config:
    key: str
    title: str
    n_rows: int
    row_bytes: int
    group_rows: int
    dtype: str              # element type of a row, for documentation and views
    elems: int              # elements per row
    extra: dict = field(default_factory=dict, hash=False, compare=False)


CONFIGS = {
    "tiny_gnn": Config("tiny_gnn", "tiny GNN features 4,096 x 128 fp32, G=32",
                       4096, 512, 32, "float32", 128),
    "gnn_gather": Config("gnn_gather", "GNN minibatch gather 2.4M x 100 fp32, G=32, fanout (15,10)",
                         2_400_000, 400, 32, "float32", 100,
                         {"seeds": 1024, "fanouts": (15, 10)}),
    "dlrm": Config("dlrm", "DLRM lookup 26 x 4M x 128 fp32, G=32, batch 2,048, Zipf 1.05",
                   26 * 4_000_000, 512, 32, "float32", 128,
                   {"tables": 26, "rows_per_table": 4_000_000, "batch": 2048, "zipf_s": 1.05}),
    "kv_bf16": Config("kv_bf16", "LLM KV cache 32 layers x [K,V] x 8 heads x 32,768 tokens x 128 bf16, G=32",
                      32 * 2 * 8 * 32768, 256, 32, "bfloat16", 128,
                      {"layers": 32, "heads": 8, "tokens": 32768, "rows_per_layer": 2 * 8 * 32768}),
    "big_gnn": Config("big_gnn", "large GNN features 111M x 128 fp32, G=64, fanout (15,10,5)",
                      111_000_000, 512, 64, "float32", 128,
                      {"seeds": 4096, "fanouts": (15, 10, 5)}),
}


# ---------------------------------------------------------------- row values

def _round_fp32_mantissa(x, keep_bits):
    """Round fp32 values to keep_bits explicit mantissa bits, ties to even."""
    u = x.view(np.uint32)
    drop = 23 - keep_bits
    half = np.uint32((1 << (drop - 1)) - 1)
    lsb = (u >> np.uint32(drop)) & np.uint32(1)
    u = (u + half + lsb) & np.uint32(~((1 << drop) - 1) & 0xFFFFFFFF)
    return u.view(np.float32)


def _fp32_to_bf16_bits(x):
    """bfloat16 bit patterns of fp32 values, round to nearest even (finite inputs)."""
    u = x.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def _chunk_values(cfg, seed, chunk, n):
    """Values of rows [chunk*CHUNK_ROWS, chunk*CHUNK_ROWS + n) as a (n, row_bytes) uint8 array."""
    rng = chunk_rng(seed, P_VALUES, chunk)
    e = cfg.elems
    if cfg.key == "tiny_gnn":
        k = rng.integers(0, 256, size=(n, e))
        z = rng.random((n, e)) < 0.5
        v = np.where(z, 0.0, k / 256.0).astype(np.float32)
    elif cfg.key == "gnn_gather":
        v = _round_fp32_mantissa(rng.standard_normal((n, e), dtype=np.float32), 8)
    elif cfg.key == "dlrm":
        u = rng.uniform(-0.05, 0.05, size=(n, e))
        v = (np.rint(u * 4096.0) / 4096.0).astype(np.float32)
    elif cfg.key == "kv_bf16":
        x = rng.standard_normal((n, e), dtype=np.float32) * np.float32(0.5)
        tokens = cfg.extra["tokens"]
        first = chunk * CHUNK_ROWS
        # rows are ordered [layer][K,V][head][token]; each (layer, K/V, head) run of
        # `tokens` rows gets 2 seeded outlier channels scaled by 20
        r = first
        while r < first + n:
            head_run = r // tokens                     # = (layer*2 + kv)*heads + head
            end = min((head_run + 1) * tokens, first + n)
            ch = chunk_rng(seed, P_OUTLIERS, head_run).choice(e, 2, replace=False)
            x[r - first:end - first, ch] *= np.float32(20.0)
            r = end
        v = _fp32_to_bf16_bits(x)
    elif cfg.key == "big_gnn":
        z = rng.random((n, e)) < 0.7
        u = rng.random((n, e))
        v = np.where(z, 0.0, np.rint(u * 1024.0) / 1024.0).astype(np.float32)
    else:
        raise KeyError(cfg.key)
    return np.ascontiguousarray(v).view(np.uint8).reshape(n, cfg.row_bytes)


def gen_rows(cfg, start, stop, seed=0):
    """Rows [start, stop) of a workload as a (stop-start, row_bytes) uint8 array."""
    out = np.empty((stop - start, cfg.row_bytes), np.uint8)
    c0, c1 = start // CHUNK_ROWS, (stop - 1) // CHUNK_ROWS if stop > start else -1
    for c in range(c0, c1 + 1):
        lo = c * CHUNK_ROWS
        n = min(CHUNK_ROWS, cfg.n_rows - lo)
        vals = _chunk_values(cfg, seed, c, n)
        a, b = max(start, lo), min(stop, lo + n)
        out[a - start:b - start] = vals[a - lo:b - lo]
    return out


def gen_all_rows(cfg, seed=0, n_rows=None, threads=None, out=None):
    """All rows (or the first n_rows) of a workload, chunks drawn in parallel."""
    n_rows = cfg.n_rows if n_rows is None else n_rows
    if out is None:
        out = np.empty((n_rows, cfg.row_bytes), np.uint8)
    n_chunks = (n_rows + CHUNK_ROWS - 1) // CHUNK_ROWS
    threads = threads or min(16, os.cpu_count() or 1)

    def one(c):
        lo = c * CHUNK_ROWS
        n = min(CHUNK_ROWS, n_rows - lo)
        out[lo:lo + n] = _chunk_values(cfg, seed, c, min(CHUNK_ROWS, cfg.n_rows - lo))[:n]

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(one, range(n_chunks)))
    return out


# ---------------------------------------------------------------- batch ids

def gnn_batch_ids(n_rows, n_seeds, fanouts, seed=0, batch_index=0):
    """Sorted unique row ids of a GNN minibatch: seeds drawn without replacement,
    then each hop draws `fanout` uniform neighbours (with replacement) per node of
    the previous hop's draws; the union is de-duplicated and sorted."""
    rng = chunk_rng(seed, P_IDS, batch_index)
    seeds = rng.choice(n_rows, n_seeds, replace=False)
    parts = [seeds]
    frontier = n_seeds
    for f in fanouts:
        frontier *= f
        parts.append(rng.integers(0, n_rows, size=frontier))
    return np.unique(np.concatenate(parts)).astype(np.int64)


_ZIPF_CDF = {}


def dlrm_batch_ids(tables, rows_per_table, batch, s, seed=0, batch_index=0):
    """Row ids of a DLRM batch in [sample][table] order: per table, a bounded
    Zipf(s) rank over [1, rows_per_table] by inverse CDF, mapped to a row by a
    seeded per-table permutation; global id = table * rows_per_table + row."""
    key = (rows_per_table, s)
    if key not in _ZIPF_CDF:
        w = np.arange(1, rows_per_table + 1, dtype=np.float64) ** (-s)
        c = np.cumsum(w)
        _ZIPF_CDF[key] = c / c[-1]
    cdf = _ZIPF_CDF[key]
    rng = chunk_rng(seed, P_IDS, batch_index)
    ids = np.empty((batch, tables), np.int64)
    for t in range(tables):
        u = rng.random(batch)
        rank0 = np.minimum(np.searchsorted(cdf, u, side="left"), rows_per_table - 1)
        perm = chunk_rng(seed, P_PERM, t).permutation(rows_per_table)
        ids[:, t] = t * rows_per_table + perm[rank0]
    return ids.reshape(-1)


def dlrm_hot_order(tables, rows_per_table, seed=0, n=None):
    """The first n row ids of the DLRM tables in popularity order (rank 0 of every
    table, then rank 1, ...), through the same per-table permutations as
    dlrm_batch_ids: the order in which a static cache would be filled from a long
    profiling pass."""
    n = tables * rows_per_table if n is None else n
    ranks = (n + tables - 1) // tables
    cols = [t * rows_per_table + chunk_rng(seed, P_PERM, t).permutation(rows_per_table)[:ranks]
            for t in range(tables)]
    return np.stack(cols, axis=1).reshape(-1)[:n]


# ---------------------------------------------------------------- test inputs

_KINDS = ("random", "identical", "zeros", "ones", "onebit", "alternating", "floats",
          "specials", "sparse", "smallint")


def structured_rows(kind, n_rows, row_bytes, seed=0):
    """Small row sets with a chosen bit structure, for tests.

    kinds: 'random' (uniform bytes), 'identical', 'zeros', 'ones', 'onebit'
    (rows differ from a base row in one random bit), 'alternating' (only odd bit
    positions vary), 'floats' (fp32 N(0,1) with 8 mantissa bits), 'specials'
    (fp32 NaN payloads, +-0.0, denormals, infinities mixed with normals),
    'sparse' (fp32 with 90% zeros), 'smallint' (uint32 in [0, 16)).
    """
    rng = chunk_rng(seed, P_VALUES, 1000 + _KINDS.index(kind))
    shape = (n_rows, row_bytes)
    if kind == "random":
        return rng.integers(0, 256, size=shape, dtype=np.uint8)
    if kind == "identical":
        base = rng.integers(0, 256, size=row_bytes, dtype=np.uint8)
        return np.tile(base, (n_rows, 1))
    if kind == "zeros":
        return np.zeros(shape, np.uint8)
    if kind == "ones":
        return np.full(shape, 0xFF, np.uint8)
    if kind == "onebit":
        base = rng.integers(0, 256, size=row_bytes, dtype=np.uint8)
        rows = np.tile(base, (n_rows, 1))
        for i in range(n_rows):
            p = int(rng.integers(0, 8 * row_bytes))
            rows[i, p // 8] ^= np.uint8(1 << (p % 8))
        return rows
    if kind == "alternating":
        base = rng.integers(0, 256, size=row_bytes, dtype=np.uint8)
        noise = rng.integers(0, 256, size=shape, dtype=np.uint8)
        return ((base & np.uint8(0x55)) | (noise & np.uint8(0xAA))).astype(np.uint8)
    assert row_bytes % 4 == 0
    e = row_bytes // 4
    if kind == "floats":
        v = _round_fp32_mantissa(rng.standard_normal((n_rows, e), dtype=np.float32), 8)
        return v.view(np.uint8).reshape(shape)
    if kind == "specials":
        pool = np.array([0x00000000, 0x80000000, 0x7FC00000, 0x7FC00001, 0xFFC12345,
                         0x7F800000, 0xFF800000, 0x00000001, 0x007FFFFF, 0x80000001,
                         0x3F800000, 0xBF800000], dtype=np.uint32)
        u = pool[rng.integers(0, pool.size, size=(n_rows, e))]
        return u.view(np.uint8).reshape(shape)
    if kind == "sparse":
        z = rng.random((n_rows, e)) < 0.9
        v = np.where(z, 0.0, rng.random((n_rows, e))).astype(np.float32)
        return v.view(np.uint8).reshape(shape)
    if kind == "smallint":
        return rng.integers(0, 16, size=(n_rows, e), dtype=np.uint32).view(np.uint8).reshape(shape)
    raise KeyError(kind)


# ---------------------------------------------------------------- microbenchmark inputs

def micro_rows(n_rows, row_bytes, fixed_fraction, seed=0, threads=None):
    """Tensors for the decompression-overhead microbenchmark (the paper's Sec. 6.1
    microbenchmark with synthetic metadata): n_rows tensors of row_bytes bytes in which
    a seeded set of round(fixed_fraction * 8 * row_bytes) bit positions holds the same
    seeded value in every tensor and every other bit is uniformly random. The fixed
    positions are drawn once for the whole set, so every cluster of rows shares them.
    """
    n_bits = 8 * row_bytes
    k = int(round(fixed_fraction * n_bits))
    rng = chunk_rng(seed, P_MICRO, row_bytes)
    pos = rng.permutation(n_bits)[:k]
    fixed = np.zeros(n_bits, np.uint8)
    fixed[pos] = 1
    value = fixed & rng.integers(0, 2, size=n_bits, dtype=np.uint8)
    keep = np.packbits(fixed, bitorder="little")          # bit p of the row = bit p%8 of byte p/8
    val = np.packbits(value, bitorder="little")
    out = np.empty((n_rows, row_bytes), np.uint8)

    def fill(c):
        a, b = c * CHUNK_ROWS, min(n_rows, (c + 1) * CHUNK_ROWS)
        r = chunk_rng(seed, P_MICRO, (row_bytes << 20) + 1 + c).integers(0, 256, size=(b - a, row_bytes), dtype=np.uint8)
        out[a:b] = (r & ~keep) | val

    n_chunks = (n_rows + CHUNK_ROWS - 1) // CHUNK_ROWS
    with ThreadPoolExecutor(threads or min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(fill, range(n_chunks)))
    return out
