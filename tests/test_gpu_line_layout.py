"""GPU parity of the line-aligned cluster layout: the device and zero-copy copies of a
clustered stream whose rows are mostly whole 128-byte lines start every cluster on a
line, so that a cluster of 255-byte rows does not shift every later row off the lines.
The stream mixes clusters of 256-byte rows with clusters of 255-byte rows (one word with
8 more invariant bits) and a ragged last cluster; gathers (host and device ids),
decompressed ranges and the compressed cache are compared with the CPU oracle."""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp

pytestmark = pytest.mark.gpu

G, W = 32, 128
L = 4 * W


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    ibp.lib()
    return t


def mixed_rows(n_clusters, odd_every, tail, seed):
    """Clusters of G rows whose words keep 16 invariant bits (bits 0-13, 30, 31), so rows
    pack to 256 bytes; every odd_every-th cluster keeps 8 more in word 5 (255 bytes)."""
    rng = np.random.default_rng(seed)
    n = n_clusters * G + tail
    out = np.empty((n, W), np.uint32)
    base = np.uint32(0xC0003FFF)
    for c in range((n + G - 1) // G):
        r0, r1 = c * G, min(n, (c + 1) * G)
        mask = np.full(W, base, np.uint32)
        if c % odd_every == odd_every - 1:
            mask[5] |= np.uint32(0x003FC000)
        fixed = rng.integers(0, 2 ** 32, size=W, dtype=np.uint64).astype(np.uint32)
        noise = rng.integers(0, 2 ** 32, size=(r1 - r0, W), dtype=np.uint64).astype(np.uint32)
        out[r0:r1] = (fixed & mask) | (noise & ~mask)
    return out.view(np.uint8).reshape(n, L)


def packed_sizes(stream):
    d = oracle.describe(stream) if hasattr(oracle, "describe") else ibp.ibp_describe(stream)
    idx = stream[d["index_off"]:d["index_off"] + 8 * (d["n_groups"] + 1)].view(np.uint64).astype(np.int64)
    per = np.full(d["n_groups"], G, np.int64)
    per[-1] = d["n_rows"] - G * (d["n_groups"] - 1)
    return np.diff(idx) // per


@pytest.mark.parametrize("odd_every,tail", [(7, 5), (2, 0), (40, 17)])
@pytest.mark.parametrize("flags", ["device", "zero_copy"])
def test_line_aligned_clusters(torch, odd_every, tail, flags):
    rows = mixed_rows(60, odd_every, tail, seed=odd_every * 100 + tail)
    n = rows.shape[0]
    stream = oracle.compress(rows, G)
    rb = packed_sizes(stream)
    full = rb[:-1] if tail else rb
    assert (full == 256).sum() >= full.size // 2 and (full == 255).any(), np.unique(rb)
    rng = np.random.default_rng(n)
    ids = np.concatenate([rng.integers(0, n, size=2 * n), np.sort(rng.choice(n, n // 2, replace=False)),
                          [0, n - 1]]).astype(np.int64)
    want = oracle.decode_rows(stream, ids, L)
    assert np.array_equal(want, rows[ids])
    say(f"[line layout] odd_every={odd_every} tail={tail} flags={flags} n={n} sizes={sorted(set(rb.tolist()))}")
    f = ibp.IBP_OPEN_PAYLOAD_DEVICE if flags == "device" else ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY
    with ibp.ibp_open(stream, 0, f) as h:
        out = torch.full((ids.size * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")
        ibp.ibp_gather_decompress(h, ids, out, out_cap=ids.size * L)
        torch.cuda.synchronize()
        assert np.array_equal(out[:ids.size * L].cpu().numpy().reshape(-1, L), want)
        assert (out[ids.size * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
        out.fill_(0xA5)
        ibp.ibp_gather_decompress_device(h, torch.from_numpy(ids).cuda(), out, out_cap=ids.size * L)
        torch.cuda.synchronize()
        assert np.array_equal(out[:ids.size * L].cpu().numpy().reshape(-1, L), want)
        # ranges: the whole tensor, and ranges cut inside clusters on both sides of odd ones
        for first, cnt in [(0, n), (G * (odd_every - 1) + 3, 2 * G + 7), (n - 9, 9), (1, n - 2)]:
            first, cnt = min(first, n - 1), min(cnt, n - min(first, n - 1))
            out.fill_(0xA5)
            ibp.ibp_decompress(h, first, cnt, out, out_cap=cnt * L)
            torch.cuda.synchronize()
            assert np.array_equal(out[:cnt * L].cpu().numpy().reshape(-1, L), rows[first:first + cnt]), (first, cnt)
            assert (out[cnt * L:cnt * L + 256].cpu().numpy() == 0xA5).all()
        if flags == "zero_copy":
            # cached rows come from the slab, misses from the pinned payload in place
            with ibp.ibp_cache_create(h, np.arange(0, n, 3)) as c:
                out.fill_(0xA5)
                ibp.ibp_cache_gather(c, torch.from_numpy(ids).cuda(), out, out_cap=ids.size * L)
                torch.cuda.synchronize()
                assert np.array_equal(out[:ids.size * L].cpu().numpy().reshape(-1, L), want)
        assert ibp.ibp_device_errors(h) == 0
