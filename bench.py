#!/usr/bin/env python3
"""Benchmark of the IBP decompression hot path on one MI355X.

Workload (default): the GNN minibatch gather -- 2,400,000 rows x 100 fp32 features
(values N(0,1) rounded to 8 mantissa bits), clusters of 32 rows, minibatches of 1,024
seed rows with a 2-hop (15, 10) uniform fanout (about 164k unique sorted row ids). The
compressed stream and every batch's ids are resident in HBM before timing starts; one
step = one ibp_gather_decompress_device call over one minibatch (a different batch per
step). `value` is decompressed output bytes per second of the timed steps.

Also reported on the same JSON line:
  roofline      the gather kernel's algorithmic HBM bytes per launch (ids + packed rows
                read + rows written + Mask/Bitval/index once per distinct cluster) over
                its average duration from HIP events, against 8 TB/s;
  cpu_baseline  the CPU oracle (single thread, bit-serial) decoding a bounded sample of
                one minibatch, in the same unit;
  e2e           the PCIe-inclusive paths (payload in pinned host memory): the same gather
                with host packing + staged DMA and with GPU-initiated zero-copy reads, and
                8 layers of the bf16 KV workload streamed both ways; effective output GB/s
                next to raw pinned H2D GB/s and the compression ratio of the bytes needed.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decompressed GB/s (HBM roofline %) + effective H2D GB/s vs raw PCIe"
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2605_30728_amd", "csrc", "ibp_kernels.hip")
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "k_gather_rows_gnn_gather.md")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(ids, G, L, rb_of_group):
    """HBM bytes one gather launch must move: ids, packed rows, output rows, and the
    Mask/Bitval + index entry of every distinct cluster touched."""
    g = ids // G
    distinct = np.unique(g).size
    return int(ids.size * 8 + rb_of_group[g].sum() + ids.size * L + distinct * (2 * L + 8))


def measured_traffic():
    """HBM bytes per gather launch from the committed rocprofv3 counter summary, or None
    when the kernel source has changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    text = open(TRAFFIC_PROFILE).read()
    m_hash = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    m_bytes = re.search(r"traffic_bytes_per_launch:\s*(\d+)", text)
    if not m_hash or not m_bytes:
        return None
    if hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest() != m_hash.group(1):
        return None
    return int(m_bytes.group(1))


def d2d_copy_gbs(torch, nbytes=1 << 30, reps=5):
    """Plain device-to-device copy of nbytes (read + write GB/s): the achievable line, and
    the known-size kernel that scales the FETCH_SIZE / WRITE_SIZE counters."""
    a = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes * reps / (s.elapsed_time(e) * 1e-3) / 1e9
    del a, b
    return gbs


def raw_h2d_gbs(torch, nbytes, reps=5):
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    e.record()
    torch.cuda.synchronize()
    return nbytes * reps / (s.elapsed_time(e) * 1e-3) / 1e9


def pcie_legs(torch, ibp, stream, rows, timed, warm, L, G, rb_of_group):
    """The PCIe-inclusive legs (never `value`): the same minibatch gather with the payload
    in pinned host memory, (a) host-packed rows through rotating staging + DMA and
    (b) GPU-initiated zero-copy reads by the gather kernel; and (c) streaming the layers
    of the bf16 KV workload through ibp_decompress both ways. Effective GB/s = output bytes
    / wall time; compared with raw pinned H2D and the ratio of output bytes to the packed
    bytes the path needs (packed rows + 8 B of per-row tables for gathers)."""
    from workloads import CONFIGS, gen_rows
    raw = raw_h2d_gbs(torch, 1 << 30)
    out = torch.empty(max(b.size for b in timed + warm) * L, dtype=torch.uint8, device="cuda")
    packed = sum(int(rb_of_group[b // G].sum()) + 8 * b.size for b in timed)
    out_total = sum(b.size * L for b in timed)
    cr = out_total / packed
    res = {"raw_h2d_GBps_1GiB": round(raw, 2), "steps": len(timed)}
    for mode, flags in (("gather_host_pack", ibp.IBP_OPEN_PAYLOAD_HOST),
                        ("gather_zero_copy", ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)):
        h = ibp.ibp_open(stream, 0, flags)
        for b in warm:
            ibp.ibp_gather_decompress(h, b, out)
        torch.cuda.synchronize()
        ibp.ibp_reset_stats(h)
        t = time.perf_counter()
        for b in timed:
            ibp.ibp_gather_decompress(h, b, out)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        st = ibp.ibp_get_stats(h)
        got = out[:timed[-1].size * L].cpu().numpy().reshape(-1, L)
        assert np.array_equal(got, rows[timed[-1]]), mode
        ibp.ibp_close(h)
        eff = out_total / dt / 1e9
        res[mode] = {"effective_GBps": round(eff, 2), "cr": round(cr, 3),
                     "effective_over_cr_raw": round(eff / (cr * raw), 3),
                     "host_pack_ms_per_batch": round(st["host_pack_ns"] / len(timed) / 1e6, 3)}
        log(f"[bench] e2e {mode}: {eff:.1f} GB/s effective ({eff / (cr * raw):.2f} of CR x raw)")
    kv = CONFIGS["kv_bf16"]
    n = kv.extra["rows_per_layer"]
    layers = 8
    krows = gen_rows(kv, 0, layers * n)
    ks = ibp.ibp_compress(krows, kv.group_rows)
    kcr = layers * n * kv.row_bytes / ibp.ibp_describe(ks)["payload_bytes"]
    kout = torch.empty(n * kv.row_bytes, dtype=torch.uint8, device="cuda")
    for mode, flags in (("kv_stream_staged_dma", ibp.IBP_OPEN_PAYLOAD_HOST),
                        ("kv_stream_zero_copy", ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)):
        h = ibp.ibp_open(ks, 0, flags)
        ibp.ibp_decompress(h, 0, n, kout)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for layer in range(layers):
            ibp.ibp_decompress(h, layer * n, n, kout)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        assert np.array_equal(kout.cpu().numpy().reshape(-1, kv.row_bytes), krows[(layers - 1) * n:]), mode
        ibp.ibp_close(h)
        eff = layers * n * kv.row_bytes / dt / 1e9
        res[mode] = {"effective_GBps": round(eff, 2), "cr": round(kcr, 3),
                     "effective_over_cr_raw": round(eff / (kcr * raw), 3), "layers": layers}
        log(f"[bench] e2e {mode}: {eff:.1f} GB/s effective ({eff / (kcr * raw):.2f} of CR x raw)")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-e2e", action="store_true")
    ap.add_argument("--e2e-steps", type=int, default=20)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(clusters shard by row range with no exchange between GPUs)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2605_30728_amd as ibp
    from workloads import CONFIGS, gen_all_rows, gnn_batch_ids

    cfg = CONFIGS["gnn_gather"]
    G, L = cfg.group_rows, cfg.row_bytes
    K, Wm = args.steps, args.warmup
    t = time.time()
    rows = gen_all_rows(cfg)
    log(f"[bench] generated {cfg.n_rows} x {L} B rows in {time.time() - t:.1f}s")
    t = time.time()
    threads = min(16, os.cpu_count() or 1)
    stream = ibp.ibp_compress(rows, G, n_threads=threads)
    compress_s = time.time() - t
    d = ibp.ibp_describe(stream)
    index = stream[d["index_off"]:d["index_off"] + 8 * (d["n_groups"] + 1)].view(np.uint64).astype(np.int64)
    n_in_group = np.full(d["n_groups"], G, np.int64)
    n_in_group[-1] = cfg.n_rows - G * (d["n_groups"] - 1)
    rb_of_group = np.diff(index) // n_in_group
    log(f"[bench] compressed in {compress_s:.2f}s ({threads} threads): payload {d['payload_bytes'] / 1e6:.1f} MB, "
        f"stream {d['stream_bytes'] / 1e6:.1f} MB, raw {cfg.n_rows * L / 1e6:.1f} MB")

    batches = [gnn_batch_ids(cfg.n_rows, cfg.extra["seeds"], cfg.extra["fanouts"], batch_index=b)
               for b in range(Wm + K)]
    d_batches = [torch.from_numpy(b).cuda() for b in batches]
    max_n = max(b.size for b in batches)
    out = torch.empty(max_n * L, dtype=torch.uint8, device="cuda")
    alg = [algorithmic_bytes(b, G, L, rb_of_group) for b in batches]

    h = ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE)
    log(f"[bench] opened on cuda:0; warmup {Wm} steps, timing {K} steps")
    for b in range(Wm):
        ibp.ibp_gather_decompress_device(h, d_batches[b], out)
    torch.cuda.synchronize()

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        ev[k][0].record()
        ibp.ibp_gather_decompress_device(h, d_batches[Wm + k], out)
        ev[k][1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    out_bytes = sum(batches[Wm + k].size * L for k in range(K))
    kern_ms = float(np.mean([s.elapsed_time(e) for s, e in ev]))
    alg_avg = float(np.mean(alg[Wm:]))
    achieved = alg_avg / (kern_ms * 1e-3) / 1e9
    value = out_bytes / wall / 1e9
    # correctness of the last timed batch against the original rows
    last = batches[Wm + K - 1]
    got = out[:last.size * L].cpu().numpy().reshape(last.size, L)
    if not np.array_equal(got, rows[last]):
        log("[bench] ERROR: gathered rows differ from the originals")
        sys.exit(1)
    assert ibp.ibp_device_errors(h) == 0
    copy_gbs = d2d_copy_gbs(torch)
    traffic = measured_traffic()
    log(f"[bench] {K} steps in {wall * 1e3:.2f} ms: {value:.1f} GB/s decompressed; kernel {kern_ms * 1e3:.1f} us "
        f"avg, {achieved:.0f} GB/s algorithmic ({achieved / HBM_PEAK_GBS:.1%} of HBM peak); "
        f"plain 1 GiB d2d copy {copy_gbs:.0f} GB/s")

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        ids = batches[Wm]
        probe = ids[:400]
        t = time.perf_counter()
        oracle.decode_rows(stream, probe, L)
        per_row = (time.perf_counter() - t) / probe.size
        m = int(min(ids.size, max(probe.size, args.cpu_seconds / per_row)))
        t = time.perf_counter()
        ref = oracle.decode_rows(stream, ids[:m], L)
        cpu_s = time.perf_counter() - t
        assert np.array_equal(ref, rows[ids[:m]])
        cpu = {"value": round(m * L / cpu_s / 1e9, 6), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"bit-serial oracle decode of the first {m} of {ids.size} rows of one minibatch "
                         f"({cpu_s:.1f} s, 1 thread)"}
        log(f"[bench] cpu oracle: {cpu['value'] * 1e3:.2f} MB/s over {m} rows")

    e2e = None
    if not args.no_e2e:
        e2e = pcie_legs(torch, ibp, stream, rows, batches[Wm:Wm + args.e2e_steps], batches[:3], L, G,
                        rb_of_group)
    ibp.ibp_close(h)

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": Wm,
        "ms_per_step": round(wall * 1e3 / K, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": "gnn_gather: 2.4M x 100 fp32 rows (N(0,1), 8 mantissa bits), G=32, "
                               "1,024 seeds, fanout (15,10), device-resident stream and ids",
                   "rows": cfg.n_rows, "row_bytes": L, "group_rows": G,
                   "batch_rows_avg": round(float(np.mean([b.size for b in batches[Wm:]])), 1),
                   "payload_cr": round(cfg.n_rows * L / d["payload_bytes"], 3),
                   "stream_cr": round(cfg.n_rows * L / d["stream_bytes"], 3)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": "k_gather_rows<2,4>", "kernel_us": round(kern_ms * 1e3, 2),
                     "algorithmic_bytes_per_launch": int(alg_avg),
                     "d2d_copy_GBps": round(copy_gbs, 1)},
        "cpu_baseline": cpu,
        "e2e": e2e,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
