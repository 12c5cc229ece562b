#!/usr/bin/env python3
"""Benchmark of the IBP decompression hot path on one MI355X.

Headline workload (the default run): the large GNN feature gather -- 111,000,000 rows x
128 fp32 features (70% zeros, the rest U(0,1) in 1/1024 steps), clusters of 64 rows,
minibatches of 4,096 seed rows with a 3-hop (15, 10, 5) uniform fanout (about 3.69M unique
sorted row ids). The compressed stream and every batch's ids are resident in HBM before
timing starts; one step = one ibp_gather_decompress_device call over one minibatch (a
different batch each step). `value` is decompressed output bytes per second over the
timed steps.

The default run then measures the other four workloads the same way (without the CPU
oracle leg, with at least 200 timed steps each) and reports them under `other_configs`,
within --budget-s of wall time:
`tiny_gnn` (one step = the whole 4,096 x 128 fp32 tensor), `gnn_gather` (2.4M x 100 fp32,
2-hop minibatches of ~164k rows), `kv_bf16` (one step = one 128 MiB layer of the bf16 KV
cache through ibp_decompress) and `dlrm` (26 tables x 4M x 128 fp32, batches of 2,048 x 26
Zipf lookups). `--workload W` measures only W, as the headline.

Also reported on the same JSON line:
  roofline      the step kernel's algorithmic HBM bytes per launch over its average
                duration (HIP events around the timed steps, over K), against 8 TB/s,
                plus the median and minimum of single event-bracketed launches taken
                after the timed region; `traffic` comes from the
                committed rocprofv3 counter summary of that kernel on that workload while
                the kernel source is unchanged (else null); plus a plain 1 GiB device copy;
  cpu_baseline  the CPU oracle (single thread, bit-serial) decoding the rows of whole steps
                for about --cpu-seconds, in the same unit, plus an oracle compress sample
                and the library's multi-threaded host compressor rate (context);
  uncompressed_device  the same steps over the rows stored uncompressed (a stream whose
                Masks are all 0, decoded by the same kernels): the uncompressed baseline;
  plain_gather  (gathers) the same ids through torch.index_select over the uncompressed
                rows in HBM: the achievable line of the access pattern, for context;
  e2e           the PCIe-inclusive paths (payload in pinned host memory): host-packed
                staging + DMA, GPU-initiated zero-copy reads, and zero-copy reads of a
                pinned copy whose rows start on 128-byte boundaries; effective output GB/s
                next to raw pinned H2D GB/s and the compression ratio of the bytes needed,
                the speedup over moving the uncompressed rows the same way (the paper's
                normalisation to uncompressed transfers, its Tab. 1), and the paper's mock
                system (the same compressed bytes moved by one DMA per step and the rows
                written, no decode; Sec. 6.1) as the ideal the path is compared with.

`--micro` runs the paper's decompression-overhead microbenchmark instead (tensors of
256 B / 1 KB / 4 KB at 10-90% space savings, PCIe paths normalised to the mock system)
and prints one JSON line holding every point. `--cache` compares the compressed device
cache with an uncompressed one of the same slab bytes (and no cache) on a gather workload.
"""
import argparse
import gc
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
# the sources the profiled kernels are compiled from, and the runtime and layout builders
# that lay out the data they read (a profile's counters stand only while these hash to the
# value recorded with them)
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2605_30728_amd", "csrc", f)
                  for f in ("ibp_kernels.hip", "ibp_cache_kernels.hip", "ibp_wave.hpp", "ibp_device.hpp",
                            "ibp_runtime.hip", "ibp_meta_slots.cpp")]


def code_sha256(texts):
    """sha256 of C/HIP source texts' code: comments, trailing blanks and empty lines are
    dropped first, so that editing a comment does not retire the counters taken on the code."""
    h = hashlib.sha256()
    for text in texts:
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for line in text.splitlines():
            code = re.sub(r"//.*", "", line).rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()


def kernel_sources_sha256():
    return code_sha256(open(path).read() for path in KERNEL_SOURCES)
GATHERS = ("gnn_gather", "dlrm", "big_gnn")
HEADLINE = "big_gnn"        # the largest configuration that fits one GPU
OTHERS = ("tiny_gnn", "gnn_gather", "kv_bf16", "dlrm")
# seconds a workload usually takes end to end in the default run (drawing, compressing,
# every leg), so the run stops starting new ones before the budget runs out
BUDGET_NEEDS = {"tiny_gnn": 15, "gnn_gather": 40, "kv_bf16": 60, "dlrm": 150}
STREAMS = ("kv_bf16", "tiny_gnn")
DESCRIPTIONS = {
    "gnn_gather": "gnn_gather: 2.4M x 100 fp32 rows (N(0,1), 8 mantissa bits), G=32, 1,024 seeds, "
                  "fanout (15,10), device-resident stream and ids",
    "dlrm": "dlrm: 26 tables x 4M x 128 fp32 (U(-0.05,0.05) in 1/4096 steps), G=32, batch 2,048 x 26 "
            "Zipf(1.05) lookups, device-resident stream and ids",
    "big_gnn": "big_gnn: 111M x 128 fp32 (70% zeros, else U(0,1) in 1/1024 steps), G=64, 4,096 seeds, "
               "fanout (15,10,5), device-resident stream and ids",
    "kv_bf16": "kv_bf16: 32 layers x [K,V] x 8 heads x 32,768 tokens x 128 bf16, G=32 tokens, one layer "
               "(524,288 rows) per step, device-resident stream",
    "tiny_gnn": "tiny_gnn: 4,096 x 128 fp32 (k/256, 50% zeros), G=32, all rows per step, device-resident stream",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def wk_for(W):
    return 1 if W <= 64 else 2 if W <= 128 else 4 if W <= 256 else 8


def kernel_name(workload, W, part=False):
    k = wk_for(W)
    if part:
        maxr = {1: 4, 2: 4, 4: 2, 8: 1}[k]
        src = 'ids' if workload in GATHERS else 'range'
        if W <= 512:
            return f"k_part_batched<{k},{maxr},{ {1: 8, 2: 4, 4: 2, 8: 1}[k] },{src}>"
        return f"k_part_rows<{k},{maxr},{src}>"
    if workload in GATHERS:
        rb = {1: 8, 2: 4, 4: 2, 8: 1}[k]
        return f"k_gather_rows<{k},{rb}>" if W <= 512 else "k_gather_tiled"
    return f"k_decompress<{k},{ {1: 4, 2: 4, 4: 2, 8: 1}[k] },true>"   # device payload: split window loads


def measured_traffic(workload, part=False):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this workload,
    or None when the kernel source has changed since the counters were taken."""
    kind = "k_part_batched" if part else "k_gather_rows" if workload in GATHERS else "k_decompress"
    path = os.path.join(ROOT, "profiles", f"{kind}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    m_bytes = re.search(r"traffic_bytes_per_launch:\s*(\d+)", text)
    if not m_hash or not m_bytes:
        return None
    if kernel_sources_sha256() != m_hash.group(1):
        return None
    return int(m_bytes.group(1))


def plain_gather(torch, rows, steps, Wm, K, L):
    """The achievable line of the gather's access pattern: the same steps as a plain row
    gather of the uncompressed rows resident in HBM (torch.index_select, a library kernel,
    not the product path): its output GB/s and its read + write GB/s."""
    table = torch.from_numpy(rows).cuda()
    d_units = [torch.from_numpy(u).cuda() for u in steps.units]
    out = torch.empty((max(steps.rows), L), dtype=torch.uint8, device="cuda")

    def step(k):
        u = d_units[k % len(steps)]
        torch.index_select(table, 0, u, out=out[:u.numel()])
    d2d_copy_gbs(torch)   # as before every timed device measurement
    for k in range(Wm):
        step(k)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        step(Wm + k)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    out_bytes = sum(steps.rows[(Wm + k) % len(steps)] * L for k in range(K))
    last = (Wm + K - 1) % len(steps)
    ok = np.array_equal(out[:steps.rows[last]].cpu().numpy(), rows[steps.row_ids(last)])
    del table, out, d_units
    torch.cuda.empty_cache()
    if not ok:
        log("[bench] ERROR: plain gather differs from the rows")
        sys.exit(1)
    gbs = out_bytes / dt / 1e9
    log(f"[bench] plain uncompressed row gather (torch.index_select, same ids): {gbs:.1f} GB/s out, "
        f"{2 * gbs:.0f} GB/s read+write")
    return {"GBps": round(gbs, 2), "read_write_GBps": round(2 * gbs, 1), "op": "torch.index_select"}


def d2d_copy_gbs(torch, nbytes=1 << 30, seconds=0.25):
    """Plain device-to-device copies of nbytes for about `seconds` (read + write GB/s of the
    median copy): the achievable line, and the known-size kernel that scales the FETCH_SIZE /
    WRITE_SIZE counters. Each timed device measurement runs it first. After an idle spell
    (a handle's upload crosses PCIe while the compute units idle) the next ~20 launches of
    the 111M-row gather run up to 20% slower than at steady state; with these copies first,
    the ramp is about half as deep (measured in the default run's traces)."""
    a = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    # back to back, 20 copies between host waits, an event between consecutive copies
    ms = []
    t0 = time.perf_counter()
    while not ms or time.perf_counter() - t0 < seconds:
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(21)]
        ev[0].record()
        for i in range(20):
            b.copy_(a)
            ev[i + 1].record()
        ev[-1].synchronize()
        ms += [ev[i].elapsed_time(ev[i + 1]) for i in range(20)]
    gbs = 2 * nbytes / (float(np.median(ms)) * 1e-3) / 1e9
    del a, b   # back to torch's cache, not freed, so the timed steps follow at once
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


def identity_stream(rows, G):
    """A valid stream holding the rows uncompressed: every cluster's Mask and Bitval are 0,
    so each packed row is exactly the raw row (the stream format's raw case). Run through
    the same placements and kernels it is the uncompressed-transfer baseline."""
    n, L = rows.shape
    ng = (n + G - 1) // G
    meta_off, index_off = 64, 64 + ng * 2 * L
    payload_off = index_off + 8 * (ng + 1)
    s = np.zeros(payload_off + n * L, np.uint8)
    hdr = s[:64]
    hdr[:4] = np.frombuffer(b"IBP1", np.uint8)
    hdr[4:16] = np.array([1, L, G], np.uint32).view(np.uint8)
    hdr[16:32] = np.array([n, ng], np.uint64).view(np.uint8)
    hdr[40:64] = np.array([meta_off, index_off, payload_off], np.uint64).view(np.uint8)
    rows_per = np.full(ng, G, np.uint64)
    rows_per[-1] = n - G * (ng - 1)
    idx = np.zeros(ng + 1, np.uint64)
    np.cumsum(rows_per * np.uint64(L), out=idx[1:])
    s[index_off:payload_off] = idx.view(np.uint8)
    s[payload_off:] = rows.reshape(-1)
    return s


def host_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": len(os.sched_getaffinity(0))}


class Layout:
    """Packed sizes and addressing of a stream, for the algorithmic byte counts: the
    clustered scheme (a u64 offset per cluster, one packed size per cluster) or the
    participation scheme (a u64 offset per row, sizes per row)."""

    def __init__(self, stream, d):
        self.L, self.G = d["row_bytes"], d["group_rows"]
        self.part = d["flags"] == 1
        n_index = d["n_rows"] + 1 if self.part else d["n_groups"] + 1
        self.index = stream[d["index_off"]:d["index_off"] + 8 * n_index].view(np.uint64).astype(np.int64)
        if self.part:
            self.row_size = np.diff(self.index)
        else:
            n_in_group = np.full(d["n_groups"], self.G, np.int64)
            n_in_group[-1] = d["n_rows"] - self.G * (d["n_groups"] - 1)
            self.rb_of_group = np.diff(self.index) // n_in_group

    def sizes(self, ids):
        return self.row_size[ids] if self.part else self.rb_of_group[ids // self.G]

    def range_bytes(self, f, n):
        if self.part:
            return int(self.index[f + n] - self.index[f])
        return int(self.index[(f + n - 1) // self.G + 1] - self.index[f // self.G])

    def gather_alg(self, ids):
        """ids, packed rows read, rows written, and per touched cluster its Mask/Bitval
        (plus its index entry; per row two index entries in the participation scheme).
        The Mask/Bitval count is the format's 2 * row_bytes even where the kernels read a
        cluster's compact slot instead (fewer bytes)."""
        clusters = np.unique(ids // self.G).size
        idx = 16 * ids.size if self.part else 8 * clusters
        return int(ids.size * 8 + self.sizes(ids).sum() + ids.size * self.L + clusters * 2 * self.L + idx)

    def range_alg(self, f, n):
        g0, g1 = f // self.G, (f + n - 1) // self.G + 1
        idx = 8 * (n + 1) if self.part else 8 * (g1 - g0)
        return int(self.range_bytes(f, n) + n * self.L + (g1 - g0) * 2 * self.L + idx)


class Steps:
    """The per-step units of a workload: row-id batches (gathers) or row ranges (streams),
    with the algorithmic HBM bytes one launch over each must move."""

    def __init__(self, workload, cfg, n_steps, layout):
        from workloads import dlrm_batch_ids, gnn_batch_ids
        self.workload, self.cfg = workload, cfg
        if workload in GATHERS:
            distinct = min(n_steps, {"gnn_gather": 64, "dlrm": 8, "big_gnn": 8}[workload])
            x = cfg.extra
            if workload == "dlrm":
                self.units = [dlrm_batch_ids(x["tables"], x["rows_per_table"], x["batch"], x["zipf_s"], batch_index=b)
                              for b in range(distinct)]
            else:
                self.units = [gnn_batch_ids(cfg.n_rows, x["seeds"], x["fanouts"], batch_index=b)
                              for b in range(distinct)]
            self.alg = [layout.gather_alg(u) for u in self.units]
            self.rows = [u.size for u in self.units]
        else:
            per = cfg.extra["rows_per_layer"] if workload == "kv_bf16" else cfg.n_rows
            self.units = [(f, per) for f in range(0, cfg.n_rows, per)]
            self.alg = [layout.range_alg(f, n) for f, n in self.units]
            self.rows = [n for _, n in self.units]

    def __len__(self):
        return len(self.units)

    def row_ids(self, k):
        u = self.units[k % len(self)]
        return u if self.workload in GATHERS else np.arange(u[0], u[0] + u[1], dtype=np.int64)


def cpu_baseline(stream, rows, steps, last, L, G, seconds, compress_kw=None):
    """The oracle on this host's cores (one thread): decode of exactly the rows of whole
    steps, starting with the step the GPU ran last, until about `seconds` have passed; then
    compress of whole clusters spread evenly over the tensor, at least 1% of them and more
    while a third of that time allows (with the stream's own scheme: compress_kw holds the
    participation-scheme parameters)."""
    kw = compress_kw or {}
    import oracle
    t0 = time.perf_counter()
    done_rows, done_steps, k = 0, 0, last
    while True:
        ids = steps.row_ids(k)
        ref = oracle.decode_rows(stream, ids, L)
        assert np.array_equal(ref, rows[ids]), "oracle decode"
        done_rows += ids.size
        done_steps += 1
        k = (k + 1) % len(steps)
        if time.perf_counter() - t0 >= seconds or done_steps >= 4 * len(steps):
            break
    dec_s = time.perf_counter() - t0
    # compress: whole clusters spread evenly over the tensor (every k-th), as many as a third
    # of the time budget allows and at least 1% of them; clusters compress independently
    # (the thresholded scheme's sampled global Mask is drawn from these rows only)
    n_groups = (rows.shape[0] + G - 1) // G
    t = time.perf_counter()
    oracle.compress(rows[:G], G, **kw)
    per_group = max(time.perf_counter() - t, 1e-6)
    ng = int(min(n_groups, max(1, seconds / 3 / per_group, -(-n_groups // 100))))
    step = max(1, n_groups // ng)
    picked = np.arange(0, n_groups, step)[:ng]
    sel = np.concatenate([np.arange(g * G, min((g + 1) * G, rows.shape[0])) for g in picked]) \
        if step > 1 else np.arange(min(rows.shape[0], ng * G))
    sample = rows[sel]
    m = sample.shape[0]
    t = time.perf_counter()
    oracle.compress(sample, G, **kw)
    comp_s = time.perf_counter() - t
    del sample
    log(f"[bench] cpu oracle: decode {done_rows * L / dec_s / 1e6:.1f} MB/s over {done_steps} step(s); "
        f"compress {m * L / comp_s / 1e6:.1f} MB/s over {ng} of {n_groups} clusters")
    return {"value": round(done_rows * L / dec_s / 1e9, 6), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"bit-serial oracle decode of the rows of {done_steps} whole step(s) "
                      f"({done_rows} rows, {dec_s:.1f} s, 1 thread)",
            "compress": {"GBps": round(m * L / comp_s / 1e9, 6),
                         "sample": (f"all {n_groups} clusters" if ng == n_groups else
                                    f"{ng} of {n_groups} clusters, one in every {step}") +
                                   f" ({m} rows, {comp_s:.1f} s, 1 thread)"},
            "host": host_info()}


def pcie_legs(torch, ibp, args, stream, ident, rows, steps, L, layout):
    """The PCIe-inclusive legs (never `value`): the same steps with the payload in pinned
    host memory, (a) through host-packed staging + DMA on a side stream (host packing of
    the requested rows for gathers, whole cluster ranges for streams) and (b) read by the
    decode kernels themselves (GPU-initiated zero-copy). Effective GB/s = output bytes /
    wall time of the median timed block (up to five blocks of the same steps); cr = output bytes / packed bytes the path needs (packed rows, plus 8 B of
    per-row tables for gathers)."""
    raw = raw_h2d_gbs(torch, 1 << 30)
    # up to --e2e-steps, at most 4 passes over the workload's distinct steps; steps that
    # write little repeat until the timed steps write 256 MiB, so that per-call host costs
    # of a few microseconds do not decide a small workload's rate
    n_e2e = min(args.e2e_steps, max(len(steps), 1) * 4)
    avg_out = sum(steps.rows) * L / max(len(steps), 1)
    n_e2e = max(n_e2e, min(4096, -(-(256 << 20) // max(int(avg_out), 1))))
    sel = [k % len(steps) for k in range(n_e2e)]
    out = torch.empty(max(steps.rows) * L, dtype=torch.uint8, device="cuda")
    out_total = sum(steps.rows[k] * L for k in sel)
    needs = {}
    for k in set(sel):
        if steps.workload in GATHERS:
            needs[k] = int(layout.sizes(steps.units[k]).sum()) + 8 * steps.rows[k]
        else:
            f, n = steps.units[k]
            needs[k] = layout.range_bytes(f, n)
    need = sum(needs[k] for k in sel)
    cr = out_total / need

    def mock_step(k):
        dev_buf[:needs[k]].copy_(host_buf[:needs[k]], non_blocking=True)
        out[:steps.rows[k] * L].fill_(0)
    res = {"raw_h2d_GBps_1GiB": round(raw, 2), "steps": n_e2e, "cr": round(cr, 3)}

    def run(h, k):
        if steps.workload in GATHERS:
            ibp.ibp_gather_decompress(h, steps.units[k], out)
        else:
            f, n = steps.units[k]
            ibp.ibp_decompress(h, f, n, out)

    def warm(fn):
        # untimed steps for at least 10 steps and 0.25 s: the first tens of milliseconds
        # after opening a handle (or allocating pinned buffers) run slower, with the host
        # threads and the copy path warming up; ten steps of a small workload last a few
        # milliseconds, well inside that window
        t, done = time.perf_counter(), 0
        while done < 10 or (time.perf_counter() - t < 0.25 and done < 20000):
            fn(sel[done % len(sel)])
            done += 1
            if done % 10 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()

    def blocks(fn):
        # the timed steps, as several blocks: a host stall of a few milliseconds (a packing
        # thread descheduled mid-task) lands in about one block in ten, so the rate is the
        # median block's; the slowest block is reported beside it
        dts = []
        for _ in range(E2E_BLOCKS):
            t = time.perf_counter()
            for k in sel:
                fn(k)
            torch.cuda.synchronize()
            dts.append(time.perf_counter() - t)
            if sum(dts) > 3.0:
                break
        return float(np.median(dts)), dts

    def leg(src, flags, check):
        h = ibp.ibp_open(src, 0, flags)
        warm(lambda k: run(h, k))
        ibp.ibp_reset_stats(h)
        dt, dts = blocks(lambda k: run(h, k))
        st = ibp.ibp_get_stats(h)
        st["dts"] = dts
        last = sel[-1]
        got = out[:steps.rows[last] * L].cpu().numpy().reshape(-1, L)
        assert np.array_equal(got, rows[steps.row_ids(last)]), check
        ibp.ibp_close(h)
        return dt, st

    # the paper's mock system: the same compressed bytes cross PCIe (one pinned DMA per step)
    # and the uncompressed rows are written, with no decode
    host_buf = torch.empty(max(needs.values()), dtype=torch.uint8, pin_memory=True)
    dev_buf = torch.empty(max(needs.values()), dtype=torch.uint8, device="cuda")
    warm(mock_step)
    dt_mock, dts_mock = blocks(mock_step)
    res["mock"] = {"GBps": round(out_total / dt_mock / 1e9, 2),
                   "raw_h2d_GBps_batch": round(need / dt_mock / 1e9, 2),
                   "blocks_GBps": [round(out_total / x / 1e9, 2) for x in dts_mock]}
    log(f"[bench] e2e mock (compressed bytes moved, rows written, no decode): {out_total / dt_mock / 1e9:.1f} GB/s; "
        f"raw H2D at the batch's size {need / dt_mock / 1e9:.1f} GB/s")
    del host_buf, dev_buf
    modes = [("staged_dma", ibp.IBP_OPEN_PAYLOAD_HOST), ("zero_copy", ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)]
    if not layout.part:
        modes.append(("zero_copy_aligned", ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED))
    for mode, flags in modes:
        dt, st = leg(stream, flags, mode)
        dt_raw, _ = leg(ident, flags, mode + " uncompressed")
        eff = out_total / dt / 1e9
        res[mode] = {"effective_GBps": round(eff, 2), "effective_over_cr_raw": round(eff / (cr * raw), 3),
                     "effective_over_cr_minus_0p1_raw": round(eff / ((cr - 0.1) * raw), 3),
                     "effective_over_mock": round(dt_mock / dt, 3),
                     "uncompressed_GBps": round(out_total / dt_raw / 1e9, 2),
                     "speedup_vs_uncompressed": round(dt_raw / dt, 3),
                     "blocks_GBps": [round(out_total / x / 1e9, 2) for x in st["dts"]],
                     "host_pack_ms_per_step": round(st["host_pack_ns"] / (n_e2e * len(st["dts"])) / 1e6, 3)}
        log(f"[bench] e2e {mode}: {eff:.1f} GB/s effective ({eff / (cr * raw):.2f} of CR x raw, "
            f"raw {raw:.1f} GB/s, CR {cr:.2f}); uncompressed rows through the same path "
            f"{out_total / dt_raw / 1e9:.1f} GB/s -> speedup {dt_raw / dt:.2f}x")
    return res


E2E_BLOCKS = 5   # timed blocks of the PCIe legs (fewer once they pass 3 s)

MICRO_SIZES = (256, 1024, 4096)
MICRO_SAVINGS = (0.1, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.9)


def micro(args):
    """The paper's decompression-overhead microbenchmark (Sec. 6.1, Fig. decompression_micro):
    for tensors of 256 B, 1 KB and 4 KB and target space savings of 10-90%, n tensors
    with that many fixed bits (clusters of 32 tensors) sit compressed in pinned host
    memory; one step transfers and decompresses all of them into HBM (ibp_decompress over
    the whole set). Throughput is normalised to the mock system: one DMA of the same
    compressed bytes plus a write of the uncompressed tensors, with no decode."""
    import torch
    import paper_2605_30728_amd as ibp
    from workloads import micro_rows
    n, iters, G = args.micro_tensors, args.micro_iters, 32
    raw = raw_h2d_gbs(torch, 1 << 30)

    def timed(fn):
        # median over iterations of the time between completions (each iteration is
        # enqueued behind the previous one), so a host stall in one iteration does not
        # decide the point
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(iters + 1)]
        ev[0].record()
        for k in range(iters):
            fn()
            ev[k + 1].record()
        torch.cuda.synchronize()
        return float(np.median([ev[k].elapsed_time(ev[k + 1]) for k in range(iters)])) * 1e-3

    part = args.scheme == "participation"
    num, den = (int(x) for x in args.threshold.split("/"))

    def point(L, target, out):
        rows = micro_rows(n, L, target)
        if part:   # one global Mask, participation bits per chunk (the paper's own scheme)
            stream = ibp.ibp_compress_ex(rows, n, args.chunk_bytes, (num, den), args.sample_every)
        else:
            stream = ibp.ibp_compress(rows, G)
        d = ibp.ibp_describe(stream)
        pay = max(d["payload_bytes"], 1)
        ref = torch.from_numpy(rows.reshape(-1)).cuda()
        host_buf = torch.empty(pay, dtype=torch.uint8, pin_memory=True)
        dev_buf = torch.empty(pay, dtype=torch.uint8, device="cuda")

        def mock():
            dev_buf.copy_(host_buf, non_blocking=True)
            out.fill_(0)
        t_mock = timed(mock)
        del host_buf, dev_buf
        pt = {"tensor_bytes": L, "target_savings": target,
              "savings": round(1 - d["payload_bytes"] / (n * L), 4),
              "mock_GBps": round(n * L / t_mock / 1e9, 2)}
        for mode, flags in (("zero_copy", ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY),
                            ("staged_dma", ibp.IBP_OPEN_PAYLOAD_HOST)):
            h = ibp.ibp_open(stream, 0, flags)
            dt = timed(lambda: ibp.ibp_decompress(h, 0, n, out))
            ok = bool(torch.equal(out, ref))
            ibp.ibp_close(h)
            if not ok:
                log(f"[micro] ERROR: {mode} L={L} savings={target}: output differs from the tensors")
                sys.exit(1)
            pt[mode] = {"GBps": round(n * L / dt / 1e9, 2), "frac_of_mock": round(t_mock / dt, 3)}
        return pt

    sizes = [int(x) for x in args.micro_sizes.split(",")]
    savings = [float(x) for x in args.micro_savings.split(",")]
    points = []
    for L in sizes:
        out = torch.empty(n * L, dtype=torch.uint8, device="cuda")
        if L == sizes[0]:
            point(L, savings[0], out)      # warm-up pass (first pinned buffers, first launches)
        for target in savings:
            pt = point(L, target, out)
            log(f"[micro] {L:5d} B, savings {pt['savings']:.3f}: mock {pt['mock_GBps']:.1f} GB/s; "
                f"zero-copy {pt['zero_copy']['GBps']:.1f} ({pt['zero_copy']['frac_of_mock']:.2f} of mock); "
                f"staged {pt['staged_dma']['GBps']:.1f} ({pt['staged_dma']['frac_of_mock']:.2f})")
            points.append(pt)
        del out
    print(json.dumps({"metric": "decompression throughput relative to the no-decode mock system",
                      "unit": "fraction of mock", "n_gpus": 1, "tensors": n, "iterations": iters,
                      "scheme": ({"name": "participation", "chunk_bytes": args.chunk_bytes,
                                  "threshold": args.threshold, "mask_rows": n} if part else
                                 {"name": "clustered", "group_rows": G}),
                      "raw_h2d_GBps_1GiB": round(raw, 2), "data": "synthetic",
                      "points": points}), flush=True)


def cache_bench(args):
    """The compressed device cache (Sec. 5, cache compression) on a gather workload: a slab
    of --cache-frac of the table's raw bytes is filled with the most popular rows (DLRM:
    by Zipf rank; GNN: most frequent in a profiling pass over batches other than the
    timed ones), in packed form (about CR times more rows) or uncompressed (rows of a
    stream whose Masks are all 0); the
    timed steps gather through ibp_cache_gather, hits decoded from HBM and misses from
    pinned host memory read in place. Also the same steps with no cache."""
    import torch
    import paper_2605_30728_amd as ibp
    from workloads import CONFIGS, gen_all_rows, gnn_batch_ids
    wl = args.workload
    if wl not in GATHERS:
        log("--cache needs a gather workload")
        sys.exit(2)
    cfg = CONFIGS[wl]
    G, L = cfg.group_rows, cfg.row_bytes
    K, Wm = args.steps, args.warmup
    rows = gen_all_rows(cfg)
    stream = ibp.ibp_compress(rows, G, n_threads=min(16, os.cpu_count() or 1))
    d = ibp.ibp_describe(stream)
    layout = Layout(stream, d)
    steps = Steps(wl, cfg, Wm + K, layout)
    x = cfg.extra
    budget = int(args.cache_frac * cfg.n_rows * L)
    if wl == "dlrm":
        # Zipf popularity is known: fill in rank order (what a long profiling pass gives)
        from workloads import dlrm_hot_order
        order = dlrm_hot_order(x["tables"], x["rows_per_table"], n=min(cfg.n_rows, 8 * budget // L))
    else:
        prof = range(1000, 1000 + args.cache_profile_batches)
        prof_ids = [gnn_batch_ids(cfg.n_rows, x["seeds"], x["fanouts"], batch_index=b) for b in prof]
        counts = np.bincount(np.concatenate(prof_ids), minlength=cfg.n_rows)
        order = np.argsort(-counts, kind="stable")
    csum = np.cumsum(layout.sizes(order))
    n_comp = int(np.searchsorted(csum, budget, side="right"))
    n_raw = budget // L
    log(f"[cache] {wl}: slab budget {budget / 1e6:.1f} MB = {n_comp} packed rows or {n_raw} raw rows")
    d_units = [torch.from_numpy(u).cuda() for u in steps.units]
    out = torch.empty(max(steps.rows) * L, dtype=torch.uint8, device="cuda")
    out_bytes = sum(steps.rows[(Wm + k) % len(steps)] * L for k in range(K))
    last = (Wm + K - 1) % len(steps)

    def timed(fn):
        for k in range(Wm):
            fn(k)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for k in range(K):
            fn(Wm + k)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        got = out[:steps.rows[last] * L].cpu().numpy().reshape(-1, L)
        assert np.array_equal(got, rows[steps.row_ids(last)]), "cache gather output"
        return out_bytes / dt / 1e9

    res = {}
    for name, src, n_cached in (("compressed", stream, n_comp), ("uncompressed", None, n_raw)):
        if src is None:
            src = identity_stream(rows, G)
        h = ibp.ibp_open(src, 0, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)
        del src
        c = ibp.ibp_cache_create(h, order[:n_cached])
        gbs = timed(lambda k: ibp.ibp_cache_gather(c, d_units[k % len(steps)], out))
        st = ibp.ibp_cache_get_stats(c)
        hit = st["hits"] / max(1, st["hits"] + st["misses"])
        res[name] = {"GBps": round(gbs, 2), "hit_rate": round(hit, 4), "rows_cached": st["rows"],
                     "slab_bytes": st["slab_bytes"]}
        log(f"[cache] {name}: {st['rows']} rows in {st['slab_bytes'] / 1e6:.1f} MB, hit rate {hit:.3f}, "
            f"{gbs:.1f} GB/s decompressed")
        if name == "compressed":
            gbs0 = timed(lambda k: ibp.ibp_gather_decompress_device(h, d_units[k % len(steps)], out))
            res["no_cache"] = {"GBps": round(gbs0, 2), "hit_rate": 0.0}
            log(f"[cache] no cache (zero-copy gather): {gbs0:.1f} GB/s")
        ibp.ibp_cache_destroy(c)
        ibp.ibp_close(h)
    print(json.dumps({"metric": "compressed device cache: decompressed GB/s and hit rate at equal slab bytes",
                      "value": res["compressed"]["GBps"], "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": Wm,
                      "data": "synthetic", "config": {"workload": DESCRIPTIONS[wl], "cache_frac": args.cache_frac,
                                                      "slab_budget_bytes": budget,
                                                      "profile_batches": args.cache_profile_batches},
                      "variants": res}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None, choices=list(GATHERS + STREAMS),
                    help="measure only this workload (default: the 111M-row GNN gather as the headline, "
                         "then the other four under other_configs)")
    ap.add_argument("--budget-s", type=float, default=480.0,
                    help="wall-clock budget of the default run: a further workload starts only while "
                         "its usual time is left")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-e2e", action="store_true")
    ap.add_argument("--e2e-steps", type=int, default=40)
    ap.add_argument("--scheme", default="clustered", choices=["clustered", "participation"],
                    help="clustered: Mask/Bitval per cluster of the workload's G rows with T = G (the default); "
                         "participation: the thresholded scheme with participation bits")
    ap.add_argument("--chunk-bytes", type=int, default=8, help="participation scheme: chunk bytes")
    ap.add_argument("--threshold", default="4/5", help="participation scheme: T/N as num/den")
    ap.add_argument("--mask-rows", type=int, default=0,
                    help="participation scheme: rows per Mask (0 = one global Mask for all rows)")
    ap.add_argument("--sample-every", type=int, default=1, help="participation scheme: count every k-th row")
    ap.add_argument("--cache", action="store_true",
                    help="run the compressed device cache comparison on a gather workload instead")
    ap.add_argument("--cache-frac", type=float, default=0.05, help="slab bytes as a fraction of the raw table")
    ap.add_argument("--cache-profile-batches", type=int, default=32)
    ap.add_argument("--micro", action="store_true",
                    help="run the decompression-overhead microbenchmark instead (one JSON line with every point)")
    ap.add_argument("--micro-tensors", type=int, default=100000)
    ap.add_argument("--micro-iters", type=int, default=100)
    ap.add_argument("--micro-sizes", default=",".join(map(str, MICRO_SIZES)),
                    help="comma-separated tensor sizes in bytes")
    ap.add_argument("--micro-savings", default=",".join(map(str, MICRO_SAVINGS)),
                    help="comma-separated target space savings")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(clusters shard by row range with no exchange between GPUs)", file=sys.stderr)
        sys.exit(2)
    if args.micro:
        micro(args)
        return
    if args.cache:
        cache_bench(args)
        return

    if args.workload:
        line = run_workload(args, args.workload, args.steps, args.warmup)
    else:
        t_start = time.time()
        line = run_workload(args, HEADLINE, args.steps, args.warmup)
        others = {}
        for wl in OTHERS:
            left = args.budget_s - (time.time() - t_start)
            if left < BUDGET_NEEDS[wl]:
                others[wl] = {"skipped": f"time budget ({left:.0f} s left of --budget-s {args.budget_s:.0f})"}
                log(f"[bench] {wl}: skipped, {left:.0f} s left")
                continue
            # the previous workload's host and pinned memory (over 100 GB after the headline)
            # is handed back to the system first: while that runs, host-bound legs measured
            # several times slower (the 2 MiB tensor's staged copies: 9-23 GB/s against ~60)
            gc.collect()
            time.sleep(3.0)
            # at least 200 timed steps: the short lookups of the DLRM batches need that many
            # to reach their steady state (20 steps read ~60% slower), and they cost ~5 ms
            k_w, w_w = max(args.steps, 200), max(args.warmup, 20)
            r = run_workload(args, wl, k_w, w_w, with_cpu=False)
            others[wl] = {"steps": k_w, "warmup": w_w,
                          **{k: r[k] for k in ("value", "unit", "ms_per_step", "config", "roofline",
                                               "uncompressed_device", "plain_gather", "e2e")}}
        line["other_configs"] = others
        line["bench_wall_s"] = round(time.time() - t_start, 1)
    print(json.dumps(line), flush=True)


def run_workload(args, wl, K, Wm, with_cpu=True):
    """One workload's bench line (a dict): the device-resident steps, the uncompressed
    and plain-gather baselines, the CPU oracle (when with_cpu) and the PCIe legs."""
    import gc
    import torch
    import paper_2605_30728_amd as ibp
    from workloads import CONFIGS, gen_all_rows

    cfg = CONFIGS[wl]
    G, L, W = cfg.group_rows, cfg.row_bytes, cfg.row_bytes // 4
    t = time.time()
    rows = gen_all_rows(cfg)
    log(f"[bench] {wl}: generated {cfg.n_rows} x {L} B rows in {time.time() - t:.1f}s")
    t = time.time()
    threads = min(16, os.cpu_count() or 1)
    part = args.scheme == "participation"
    if part:
        num, den = (int(x) for x in args.threshold.split("/"))
        mask_rows = args.mask_rows or cfg.n_rows
        stream = ibp.ibp_compress_ex(rows, mask_rows, args.chunk_bytes, (num, den), args.sample_every,
                                     n_threads=threads)
    else:
        stream = ibp.ibp_compress(rows, G, n_threads=threads)
    compress_s = time.time() - t
    d = ibp.ibp_describe(stream)
    layout = Layout(stream, d)
    log(f"[bench] compressed in {compress_s:.2f}s ({threads} threads): payload {d['payload_bytes'] / 1e6:.1f} MB, "
        f"stream {d['stream_bytes'] / 1e6:.1f} MB, raw {cfg.n_rows * L / 1e6:.1f} MB")

    h = ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE)
    gather_meta = ibp.ibp_get_stats(h)["gather_meta_bytes"]
    steps = Steps(wl, cfg, Wm + K, layout)
    out = torch.empty(max(steps.rows) * L, dtype=torch.uint8, device="cuda")
    if wl in GATHERS:
        d_units = [torch.from_numpy(u).cuda() for u in steps.units]

        def step(k):
            ibp.ibp_gather_decompress_device(h, d_units[k % len(steps)], out)
    else:
        def step(k):
            f, n = steps.units[k % len(steps)]
            ibp.ibp_decompress(h, f, n, out)
    log(f"[bench] opened on cuda:0; {len(steps)} distinct step inputs; warmup {Wm} steps, timing {K} steps")
    # the device-copy line, measured first: it also takes the GPU out of the idle state the
    # upload leaves it in (d2d_copy_gbs)
    copy_gbs = d2d_copy_gbs(torch)
    for k in range(Wm):
        step(k)
    torch.cuda.synchronize()

    # the timed region: K steps back to back, one HIP event pair around them on the stream
    # the kernels run on; the average launch is the elapsed time over K (dispatch gaps
    # between launches included)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for k in range(K):
        step(Wm + k)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = e0.elapsed_time(e1) / K
    out_bytes = sum(steps.rows[(Wm + k) % len(steps)] * L for k in range(K))
    alg_avg = float(np.mean([steps.alg[(Wm + k) % len(steps)] for k in range(K)]))
    achieved = alg_avg / (kern_ms * 1e-3) / 1e9
    value = out_bytes / wall / 1e9
    last = (Wm + K - 1) % len(steps)
    got = out[:steps.rows[last] * L].cpu().numpy().reshape(-1, L)
    if not np.array_equal(got, rows[steps.row_ids(last)]):
        log("[bench] ERROR: decompressed rows differ from the originals")
        sys.exit(1)
    assert ibp.ibp_device_errors(h) == 0
    # the spread of single launches, after the timed region: each launch between its own
    # pair of events (which adds the event packets to every launch)
    nb = min(K, 100)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nb)]
    for k in range(nb):
        ev[k][0].record()
        step(Wm + k)
        ev[k][1].record()
    torch.cuda.synchronize()
    kern_all = np.array([a.elapsed_time(b) for a, b in ev])
    ibp.ibp_close(h)
    # the same steps over the rows stored uncompressed (Mask = 0 everywhere), same kernels
    ident = identity_stream(rows, G)
    hu = ibp.ibp_open(ident, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE)
    h = hu
    d2d_copy_gbs(torch)   # as before every timed device measurement
    for k in range(Wm):
        step(k)
    torch.cuda.synchronize()
    t0u = time.perf_counter()
    for k in range(K):
        step(Wm + k)
    torch.cuda.synchronize()
    wall_u = time.perf_counter() - t0u
    got = out[:steps.rows[last] * L].cpu().numpy().reshape(-1, L)
    assert np.array_equal(got, rows[steps.row_ids(last)]), "uncompressed baseline"
    ibp.ibp_close(hu)
    log(f"[bench] same steps over uncompressed rows (device-resident): {out_bytes / wall_u / 1e9:.1f} GB/s "
        f"-> compressed is {wall_u / wall:.2f}x the uncompressed speed")
    plain = plain_gather(torch, rows, steps, Wm, K, L) if wl in GATHERS else None
    traffic = measured_traffic(wl, part)
    log(f"[bench] {K} steps in {wall * 1e3:.2f} ms: {value:.1f} GB/s decompressed; kernel {kern_ms * 1e3:.1f} us "
        f"avg, {achieved:.0f} GB/s algorithmic ({achieved / HBM_PEAK_GBS:.1%} of HBM peak); "
        f"plain 1 GiB d2d copy {copy_gbs:.0f} GB/s")

    cpu = None
    if with_cpu and not args.no_cpu_baseline:
        kw = ({"chunk_bytes": args.chunk_bytes, "threshold": (num, den), "sample_every": args.sample_every}
              if part else None)
        cpu = cpu_baseline(stream, rows, steps, last, L, G, args.cpu_seconds, kw)
        cpu["host_compressor"] = {"GBps": round(cfg.n_rows * L / compress_s / 1e9, 3), "threads": threads}

    e2e = None
    if not args.no_e2e:
        e2e = pcie_legs(torch, ibp, args, stream, ident, rows, steps, L, layout)

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": Wm,
        "ms_per_step": round(wall * 1e3 / K, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": DESCRIPTIONS[wl], "rows": cfg.n_rows, "row_bytes": L, "group_rows": G,
                   "rows_per_step_avg": round(float(np.mean(steps.rows)), 1),
                   "scheme": ({"name": "participation", "chunk_bytes": args.chunk_bytes,
                               "threshold": args.threshold, "mask_rows": args.mask_rows or cfg.n_rows,
                               "sample_every": args.sample_every} if part else
                              {"name": "clustered", "group_rows": G}),
                   "payload_cr": round(cfg.n_rows * L / d["payload_bytes"], 3),
                   "stream_cr": round(cfg.n_rows * L / d["stream_bytes"], 3)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": kernel_name(wl, W, part), "kernel_us": round(kern_ms * 1e3, 2),
                     "kernel_us_bracketed_median": round(float(np.median(kern_all)) * 1e3, 2),
                     "kernel_us_bracketed_min": round(float(kern_all.min()) * 1e3, 2),
                     "algorithmic_bytes_per_launch": int(alg_avg), "d2d_copy_GBps": round(copy_gbs, 1),
                     "gather_meta_bytes_per_cluster": gather_meta if wl in GATHERS else None},
        "uncompressed_device": {"GBps": round(out_bytes / wall_u / 1e9, 2),
                                "speedup_of_compressed": round(wall_u / wall, 3)},
        "plain_gather": plain,
        "cpu_baseline": cpu,
        "e2e": e2e,
    }
    del rows, stream, ident, out
    if wl in GATHERS:
        del d_units
    gc.collect()
    torch.cuda.empty_cache()
    return line




if __name__ == "__main__":
    main()
