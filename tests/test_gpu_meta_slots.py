"""GPU parity of the row gathers across the forms of cluster metadata they read: compact
slots with room for 8 pairs (every cluster's words repeat at most 8 distinct (Mask,
Bitval) pairs), for 16 (some cluster has 9-16), and the raw Mask/Bitval words (some
cluster has more). Clusters are drawn with a chosen number of distinct pairs, up to each
boundary and across it, for every tile width (1, 2, 4 and 8 words per lane) and a ragged
last cluster; expected rows come from the CPU oracle."""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp

pytestmark = pytest.mark.gpu

SETS = {"fit": [1, 2, 7, 8, 3], "fit16": [1, 9, 16, 12, 3], "mixed": [1, 2, 7, 8, 9, 16, 40]}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    ibp.lib()
    return t


def pair_rows(W, G, n, seed, pairs):
    """Rows of 32-bit words whose cluster c (rows cG .. cG+G-1) repeats pairs[c % len]
    distinct (Mask, Bitval) pairs (capped at W): word w of the cluster follows pattern
    w mod p, a random invariant mask and value, random bits elsewhere (none in a ragged
    last cluster, whose few rows would agree on random bits)."""
    rng = np.random.default_rng(seed)
    out = np.empty((n, W), np.uint32)
    for c in range((n + G - 1) // G):
        r0, r1 = c * G, min(n, (c + 1) * G)
        p = min(pairs[c % len(pairs)], W)
        masks = rng.integers(0, 2 ** 32, size=p, dtype=np.uint64).astype(np.uint32)
        masks[0] = 0xFFFFFFFF if p > 1 else masks[0]      # one fully invariant pattern
        vals = rng.integers(0, 2 ** 32, size=p, dtype=np.uint64).astype(np.uint32)
        # distinct patterns: a distinct invariant value in the low byte when masks repeat
        masks |= np.uint32(0xFF)
        if r1 - r0 < G:
            masks[:] = 0xFFFFFFFF
        vals = (vals & np.uint32(0xFFFFFF00)) | np.arange(p, dtype=np.uint32)
        pat = np.arange(W) % p
        noise = rng.integers(0, 2 ** 32, size=(r1 - r0, W), dtype=np.uint64).astype(np.uint32)
        out[r0:r1] = (vals[pat] & masks[pat]) | (noise & ~masks[pat])
    return out.view(np.uint8).reshape(n, 4 * W)


def distinct_pairs(rows, G, W):
    u = rows.view(np.uint32).reshape(-1, W)
    counts = []
    for c in range((u.shape[0] + G - 1) // G):
        blk = u[c * G:(c + 1) * G]
        a, o = np.bitwise_and.reduce(blk, 0), np.bitwise_or.reduce(blk, 0)
        m = ~(a ^ o)
        counts.append(len(set(zip(m.tolist(), (a & m).tolist()))))
    return counts


@pytest.mark.parametrize("W", [16, 64, 100, 128, 200, 256, 500, 512])
@pytest.mark.parametrize("mode", ["device_ids", "host_ids", "host_payload", "zero_copy", "cache"])
@pytest.mark.parametrize("pairs", ["fit", "fit16", "mixed"])
def test_gather_both_metadata_forms(torch, W, mode, pairs):
    G = 32
    n = G * len(SETS[pairs]) * 2 + 5
    L = 4 * W
    rows = pair_rows(W, G, n, seed=W, pairs=SETS[pairs])
    counts = distinct_pairs(rows, G, W)
    if pairs == "fit":
        assert max(counts) <= 8 and 8 in counts, counts
    elif pairs == "fit16":
        assert max(counts) == 16 and 9 in counts, counts
    else:
        assert 8 in counts and 9 in counts and (W <= 16 or max(counts) > 16), counts
    room = 8 if max(counts) <= 8 else 16 if max(counts) <= 16 else None
    stream = oracle.compress(rows, G)
    rng = np.random.default_rng(W + 1)
    ids = np.concatenate([np.sort(rng.integers(0, n, size=3 * n)), rng.integers(0, n, size=n),
                          np.arange(n), [n - 1, 0]]).astype(np.int64)
    want = oracle.decode_rows(stream, ids, L)
    assert np.array_equal(want, rows[ids])
    say(f"[meta forms] W={W} mode={mode} n={n} ids={ids.size} pairs={sorted(set(counts))}")
    flags = {"device_ids": ibp.IBP_OPEN_PAYLOAD_DEVICE, "host_ids": ibp.IBP_OPEN_PAYLOAD_DEVICE,
             "host_payload": ibp.IBP_OPEN_PAYLOAD_HOST, "zero_copy": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY,
             "cache": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY}[mode]
    out = torch.full((ids.size * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")
    d_ids = torch.from_numpy(ids).cuda()
    with ibp.ibp_open(stream, 0, flags) as h:
        # slots (8 or 16 pairs of 8 bytes and 32K bytes of indices, in 128-byte lines)
        # only when every cluster fits one
        k = 1 if W <= 64 else 2 if W <= 128 else 4 if W <= 256 else 8
        want_meta = 2 * L if room is None else (8 * room + 32 * k + 127) // 128 * 128
        assert ibp.ibp_get_stats(h)["gather_meta_bytes"] == want_meta
        if mode == "cache":
            with ibp.ibp_cache_create(h, np.arange(0, n, 3)) as c:
                ibp.ibp_cache_gather(c, d_ids, out, out_cap=ids.size * L)
                torch.cuda.synchronize()
        elif mode in ("device_ids", "zero_copy"):
            ibp.ibp_gather_decompress_device(h, d_ids, out, out_cap=ids.size * L)
        else:
            ibp.ibp_gather_decompress(h, ids, out, out_cap=ids.size * L)
        torch.cuda.synchronize()
        assert ibp.ibp_device_errors(h) == 0
    got = out[:ids.size * L].cpu().numpy().reshape(ids.size, L)
    assert (out[ids.size * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
    assert np.array_equal(got, want)


@pytest.mark.parametrize("W", [16, 64, 100, 128, 200, 256, 500, 512])
@pytest.mark.parametrize("mode", ["device_ids", "host_ids", "host_payload", "zero_copy"])
@pytest.mark.parametrize("pairs", ["fit", "fit16", "mixed"])
def test_participation_gather_both_metadata_forms(torch, W, mode, pairs):
    """The thresholded scheme under per-cluster Masks over the same clusters: batches whose
    rows lie in different clusters read every row's raw Mask/Bitval words (no slots for
    this scheme; the slot's pair expansion measured slower there). With T = n (threshold
    1/1) the per-cluster Masks are the clustered scheme's, so the same rows give the same
    pair counts."""
    G = 32
    n = G * len(SETS[pairs]) * 2 + 5
    L = 4 * W
    rows = pair_rows(W, G, n, seed=W + 7, pairs=SETS[pairs])
    counts = distinct_pairs(rows, G, W)
    stream = oracle.compress(rows, G, chunk_bytes=4, threshold=(1, 1))
    rng = np.random.default_rng(W + 3)
    # unsorted ids put rows of different clusters into one batch; the sorted run and the
    # full range give batches of one cluster too
    ids = np.concatenate([rng.integers(0, n, size=3 * n), np.sort(rng.integers(0, n, size=n)),
                          np.arange(n), [n - 1, 0]]).astype(np.int64)
    want = oracle.decode_rows(stream, ids, L)
    assert np.array_equal(want, rows[ids])
    say(f"[part meta forms] W={W} mode={mode} n={n} ids={ids.size} pairs={sorted(set(counts))}")
    flags = {"device_ids": ibp.IBP_OPEN_PAYLOAD_DEVICE, "host_ids": ibp.IBP_OPEN_PAYLOAD_DEVICE,
             "host_payload": ibp.IBP_OPEN_PAYLOAD_HOST, "zero_copy": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY}[mode]
    out = torch.full((ids.size * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")
    with ibp.ibp_open(stream, 0, flags) as h:
        assert ibp.ibp_get_stats(h)["gather_meta_bytes"] == 2 * L
        if mode in ("device_ids", "zero_copy"):
            ibp.ibp_gather_decompress_device(h, torch.from_numpy(ids).cuda(), out, out_cap=ids.size * L)
        else:
            ibp.ibp_gather_decompress(h, ids, out, out_cap=ids.size * L)
        torch.cuda.synchronize()
        assert ibp.ibp_device_errors(h) == 0
    got = out[:ids.size * L].cpu().numpy().reshape(ids.size, L)
    assert (out[ids.size * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
    assert np.array_equal(got, want)
