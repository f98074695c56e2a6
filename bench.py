#!/usr/bin/env python3
"""Decode-attention benchmark on one MI355X: µs per decode step and achieved HBM GB/s.

One step is the whole hot path on one batch: the retained sets from the
eviction policy, then split-K GQA attention over the retained K/V with the
log-sum-exp merge, on synthetic inputs already resident in HBM.  The step's
value times the single-launch murmur_decode_step (retained-set outputs
written); murmur_evict_compact followed by murmur_decode_attn is timed beside
it (step_two_launches_us).  Default workload: 12 chunks of 300 s (2250 speech tokens, 32
prompt tokens, 600-1200 output tokens), speech window 562 with delay 512,
output window 256, 1 layer, GQA 28/4, head_dim 128, bf16.

Timing:
  * value / ms_per_step: K steps captured once into a HIP graph and replayed,
    bracketed by device synchronisation and HIP events on the replay stream;
  * roofline.achieved: algorithmic bytes of one decode_attn launch divided by
    its duration: the marginal cost of a launch in a replayed graph of
    back-to-back launches (graphs of N and 2N launches between HIP events on
    the stream they are launched on, the difference over N), which leaves out
    the graph's fixed start; the plain mean over K launches is reported as
    decode_attn_graph_mean_us;
    decode_attn_per_step_us: the same per timed step (a graph of launches over
    that step's retained set), median and p90 over the steps; per-launch event
    brackets, which also count each launch's dispatch latency, are reported
    alongside;
  * cold reads: every launch reads the next replica of the KV cache (the
    replicas hold more than 2 x 256 MB), and an untimed 512 MB read before
    each timed replay evicts what the warm-up replay left in the 256 MB
    Infinity Cache, so K/V come from HBM;
  * read_ceiling: the fastest of 105 configurations of a plain streaming read
    (murmur_read_probe) over the same byte count, timed the same way.
cpu_baseline: the fp64 oracle timed on this host's cores on a bounded number
of steps of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

METRIC = "decode-attn µs/step + achieved HBM GB/s (% peak), 12×300s chunks w/ eviction"
HBM_PEAK_GBPS = 8000.0
MALL_BYTES = 256 << 20

DESCRIPTIONS = {
    "c1": "tiny: 1 layer, batch 1, 32 prompt + 450 speech + 64 output tokens, speech window 128, output window 32",
    "c2": "12 x 300 s chunks, dense: 1 layer, 32 prompt + 2250 speech + U{600..1200} output tokens, no eviction",
    "c3": "12 x 300 s chunks with eviction: 1 layer, 32 prompt + 2250 speech + U{600..1200} output tokens, "
          "speech window 562 (delay 512), output window 256, 5% planted keys",
    "c4_dense": "single-pass hour, dense: 1 layer, batch 1, 32 prompt + 27000 speech + 8000 output tokens",
    "c4_evict": "single-pass hour with eviction: speech window 2048 (delay 512), output window 512",
    "c5": "28 layers x 12 chunks: speech U{1800..2250}, output U{300..1200}, speech window L_s/4 (delay 512), "
          "output window 256, all layers in one launch",
    "c5_layers": "c5 with its first 4 layers dense and the eviction policy on the other 24 (per-layer policies)",
}


ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2606_01483_amd", "csrc")
# The device code and the host code that plans its launches (split counts, workspace layout): what the
# committed traffic figures depend on.
KERNEL_SOURCES = tuple(os.path.join(CSRC, f) for f in ("kernels.hip", "api.cpp", "internal.h", "policy.h"))


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_code_text(source: str) -> str:
    """The kernel source without its comments, whitespace runs collapsed: what the counters depend on."""
    import re
    source = re.sub(r"/\*.*?\*/", " ", source, flags=re.S)
    source = re.sub(r"//[^\n]*", " ", source)
    return " ".join(source.split())


def kernel_source_hash(paths=KERNEL_SOURCES) -> str:
    """First 16 hex digits of the sha256 of the kernel and launch-planning code (comments and whitespace do
    not count)."""
    import hashlib
    h = hashlib.sha256()
    for path in paths:
        h.update(kernel_code_text(open(path).read()).encode())
        h.update(b"\0")
    return h.hexdigest()[:16]


def committed_traffic(config: str) -> float | None:
    """HBM bytes per decode_attn launch from the committed rocprofv3 counter summary of this workload,
    or None if there is none or the kernel or launch-planning code has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"decode_attn_{config}_traffic.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.lstrip().startswith("#"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def summarize_trace(directory: str, top: int = 10) -> str:
    """Markdown tables of a rocprofv3 --kernel-trace --stats run: per kernel, calls and durations (the
    instantiations of the read probe folded into one row), then the median and p90 of each kernel's
    dispatch durations, from the run's *kernel_trace.csv."""
    import csv
    import glob
    path = sorted(glob.glob(os.path.join(directory, "**", "*kernel_trace.csv"), recursive=True))[0]
    dur: dict[str, list[int]] = {}
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"]
        if "read_probe_kernel<" in name:
            name = "murmur::read_probe_kernel (every configuration of the sweep)"
        dur.setdefault(name, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    total = sum(sum(d) for d in dur.values())
    rows = sorted(dur.items(), key=lambda kv: -sum(kv[1]))[:top]
    short = lambda n: n if len(n) <= 72 else n[:69] + "..."
    out = ["| Kernel | Calls | Total ns | Average ns | % | Min ns | Max ns | Median ns | p90 ns |",
           "|---|---|---|---|---|---|---|---|---|"]
    for name, d in rows:
        a = np.array(d, dtype=np.float64)
        out.append(f"| {short(name)} | {len(a)} | {int(a.sum())} | {a.mean():.0f} | {100 * a.sum() / total:.2f} | "
                   f"{int(a.min())} | {int(a.max())} | {np.median(a):.0f} | {np.percentile(a, 90):.0f} |")
    return "\n".join(out)


def _pmc_per_dispatch(directory: str, name_part: str) -> tuple[float, int]:
    """Mean counter value (KiB) per dispatch of the kernels whose name contains name_part."""
    import csv
    import glob
    path = sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True))[0]
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path)) if name_part in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no dispatch of a kernel named like {name_part!r} in {path}")
    return sum(vals) / len(vals), len(vals)


def summarize_pmc(config: str, kernel: str, fetch_dir: str, write_dir: str, copy_fetch_dir: str,
                  copy_write_dir: str, copy_mib: int, alg_bytes: int) -> str:
    """Body of profiles/decode_attn_<config>_traffic.txt: FETCH_SIZE and WRITE_SIZE per dispatch of
    `kernel`, each scaled by what the same counter reads for a plain device copy of copy_mib MiB."""
    f_kib, nf = _pmc_per_dispatch(fetch_dir, kernel)
    w_kib, nw = _pmc_per_dispatch(write_dir, kernel)
    cf_kib, _ = _pmc_per_dispatch(copy_fetch_dir, "copyBuffer")
    cw_kib, _ = _pmc_per_dispatch(copy_write_dir, "copyBuffer")
    f_scale, w_scale = copy_mib * 1024 / cf_kib, copy_mib * 1024 / cw_kib
    traffic = (f_kib * f_scale + w_kib * w_scale) * 1024
    return "\n".join([
        f"# Scale factors: a plain {copy_mib} MiB device copy (__amd_rocclr_copyBuffer) reads FETCH_SIZE "
        f"{cf_kib:.1f} KiB and WRITE_SIZE {cw_kib:.1f} KiB per dispatch,",
        f"# so FETCH_SIZE is scaled by {f_scale:.4f} and WRITE_SIZE by {w_scale:.4f}.",
        f"# {kernel}: FETCH_SIZE mean {f_kib:.1f} KiB over {nf} dispatches, WRITE_SIZE mean {w_kib:.1f} KiB over {nw}.",
        f"kernel: {kernel}", f"workload: {config}", f"fetch_kib_per_dispatch: {f_kib:.1f}",
        f"write_kib_per_dispatch: {w_kib:.1f}", f"fetch_scale: {f_scale:.4f}", f"write_scale: {w_scale:.4f}",
        f"algorithmic_bytes_per_launch: {alg_bytes}", f"traffic_bytes_per_launch: {traffic:.0f}",
        f"traffic_over_algorithmic: {traffic / alg_bytes:.3f}", f"kernel_source_sha256_16: {kernel_source_hash()}",
    ])


def copy_reference(mbytes: int, reps: int) -> dict:
    """A plain device copy of known size, the reference for scaling the PMC byte counters."""
    import torch
    n = mbytes << 20
    x = torch.ones(n, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    return {"copy_reference_bytes_read": n, "copy_reference_bytes_written": n, "launches": reps}


def cpu_baseline(wl, budget_s: float, threads: int) -> dict:
    import oracle
    oracle.build()
    qs = [wl.q(s) for s in range(wl.steps)]
    t0 = time.perf_counter()
    n = 0
    per_layer = wl.policy.ndim == 3
    while True:
        s = n % wl.steps
        if per_layer:  # the retained set of each layer's policy, attended layer by layer
            for layer in range(wl.n_layers):
                idx, cnt = oracle.retained(wl.seg(s), wl.policy[layer])
                sl = slice(layer, layer + 1)
                oracle.attend(qs[s][sl], wl.k[sl], wl.v[sl], idx, cnt, scale=wl.scale, n_threads=threads)
        else:
            idx, cnt = oracle.retained(wl.seg(s), wl.policy)
            oracle.attend(qs[s], wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=threads)
        n += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": dt / n * 1e6, "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": f"{n} decode step(s) of workload {wl.name} (all {wl.batch} sequences, {wl.n_layers} layer(s), "
                      f"{wl.hq} heads), retained set + fp64 attention, {threads} threads, {dt:.1f} s wall"}


PROBE_WORKGROUPS = (256, 512, 1024, 2048, 4096)
PROBE_THREADS = (256, 512, 1024)
PROBE_DEPTHS = (2, 4, 8, 16)


def probe_configs() -> list[tuple[str, int, int, int]]:
    """(load type, workgroups, threads, loads in flight per thread) of the read-ceiling sweep; the
    direct-to-LDS probe is limited to 64 KiB of LDS per workgroup."""
    out = []
    for mode in ("registers", "lds"):
        for wg in PROBE_WORKGROUPS:
            for t in PROBE_THREADS:
                for d in PROBE_DEPTHS:
                    if mode == "lds" and (t // 64) * d > 64:
                        continue
                    out.append((mode, wg, t, d))
    return out


def read_sweep(nbytes: int, steps: int, capture, time_graph, configs=None) -> list[dict]:
    """murmur_read_probe (a plain read-only streaming kernel) over every configuration of the sweep:
    per configuration, the marginal per-launch time (marginal_us, n = max(steps, 64)) of launches over
    nbytes each, every launch reading the next of enough regions to defeat the 256 MB Infinity Cache;
    and a graph of 8 launches over 1 GiB (two alternating regions; a replay's fixed start is negligible
    beside them)."""
    import torch
    from paper_2606_01483_amd import murmur as M
    nbytes = max(16, nbytes // 16 * 16)
    regions = max(2, math.ceil(2.2 * MALL_BYTES / nbytes))
    configs = configs or probe_configs()
    sink = torch.zeros(max(PROBE_WORKGROUPS), dtype=torch.int32, device="cuda")
    modes = {"registers": M.MURMUR_PROBE_REGISTERS, "lds": M.MURMUR_PROBE_LDS}
    log(f"read-ceiling sweep: {len(configs)} configurations, {nbytes / 1e6:.1f} MB x {regions} regions and 1 GiB")
    out = []
    buf = torch.empty(regions * nbytes, dtype=torch.uint8, device="cuda")
    n = max(steps, 64)
    for mode, wg, t, d in configs:
        us, _ = marginal_us(lambda i: M.murmur_read_probe(buf[(i % regions) * nbytes:], nbytes, wg, sink, t, d,
                                                          modes[mode]), n, capture, time_graph)
        out.append({"mode": mode, "workgroups": wg, "threads": t, "depth": d, "bytes": nbytes, "us": round(us, 3),
                    "GBps": round(nbytes / us / 1e3, 1)})
    del buf
    gib = 1 << 30
    big = torch.empty(2 * gib, dtype=torch.uint8, device="cuda")
    for r, (mode, wg, t, d) in zip(out, configs):
        graph = capture(lambda: [M.murmur_read_probe(big[(i % 2) * gib:], gib, wg, sink, t, d, modes[mode])
                                 for i in range(8)])
        us = time_graph(graph) / 8
        r["us_1GiB"], r["GBps_1GiB"] = round(us, 3), round(gib / us / 1e3, 1)
        del graph
    del big
    torch.cuda.empty_cache()
    return out


def read_ceiling(nbytes: int, steps: int, capture, time_graph) -> dict:
    """The practical read ceiling: the fastest configuration of the read_sweep at the attention launch's
    byte count, and the fastest at 1 GiB."""
    sweep = read_sweep(nbytes, steps, capture, time_graph)
    best = max(sweep, key=lambda r: r["GBps"])
    best_gib = max(sweep, key=lambda r: r["GBps_1GiB"])
    key = lambda r: f"{r['mode']}, {r['workgroups']} workgroups x {r['threads']} threads, depth {r['depth']}"
    return {"bytes": best["bytes"], "us": best["us"], "GBps": best["GBps"], "config": key(best),
            "us_1GiB": best_gib["us_1GiB"], "GBps_1GiB": best_gib["GBps_1GiB"], "config_1GiB": key(best_gib),
            "configurations": len(sweep),
            "GBps_default_probe": next(r["GBps"] for r in sweep if (r["mode"], r["workgroups"], r["threads"],
                                                                    r["depth"]) == ("registers", 256, 256, 8))}


def sweep_table(rows: list[dict]) -> str:
    out = ["| Load type | Workgroups | Threads | Depth | µs (attention bytes) | GB/s | µs (1 GiB) | GB/s (1 GiB) |",
           "|---|---|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -r["GBps"]):
        out.append(f"| {r['mode']} | {r['workgroups']} | {r['threads']} | {r['depth']} | {r['us']:.3f} | "
                   f"{r['GBps']:.0f} | {r['us_1GiB']:.1f} | {r['GBps_1GiB']:.0f} |")
    return "\n".join(out)


def oracle_parity(wl, db, i: int) -> dict:
    """CPU-baseline leg: the fused step's bf16 output for step i (all layers, sequences and heads) against the
    fp64 oracle: the largest error relative to max(|ref|, rms of the 128-wide row), and the same after
    subtracting half a bf16 ulp of the reference (what the bf16 store alone may add)."""
    import torch
    import oracle
    db.step_fused(i, 0)
    torch.cuda.synchronize()
    y = db.out.float().cpu().numpy().astype(np.float64)
    lse = db.lse.cpu().numpy().astype(np.float64)
    s = db.steps[i]
    seg, q = wl.seg(s), wl.q(s)
    if wl.policy.ndim == 3:
        parts = []
        for layer in range(wl.n_layers):
            idx, cnt = oracle.retained(seg, wl.policy[layer])
            sl = slice(layer, layer + 1)
            parts.append(oracle.attend(q[sl], wl.k[sl], wl.v[sl], idx, cnt, scale=wl.scale, n_threads=16))
        ref, ref_lse = np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])
    else:
        idx, cnt = oracle.retained(seg, wl.policy)
        ref, ref_lse = oracle.attend(q, wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
    denom = np.maximum(np.abs(ref), np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True)))
    half_ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 8)
    err = np.abs(y - ref)
    return {"step": int(s), "max_rel_err_bf16_out": float(np.max(err / denom)),
            "max_rel_err_beyond_bf16_rounding": float(np.max((err - half_ulp) / denom)),
            "lse_max_err": float(np.max(np.abs(lse - ref_lse) / np.maximum(1.0, np.abs(ref_lse)))),
            "tolerance": 2e-3}


def replicas_for(wl, kv_step: list[int]) -> int:
    """KV replicas to rotate over so that consecutive steps read more than 2.2 x the Infinity Cache
    (at most 24 GB of replicas)."""
    replicas = max(1, math.ceil(2.2 * MALL_BYTES / min(kv_step)))
    return min(replicas, max(1, (24 << 30) // (wl.k.nbytes * 2)))


def ring_capacity(wl, n_steps: int) -> int:
    """Ring rows for a workload: its largest output window, or, where output eviction is off, every
    output token the measured steps generate beyond the sinks."""
    from paper_2606_01483_amd.decode import layer_policies
    cap = 1
    last_j = wl.seg(n_steps - 1)[:, 3]
    for pol in layer_policies(wl):
        for b in range(wl.batch):
            w_o, n_so = int(pol[b, 3]), int(pol[b, 4])
            cap = max(cap, w_o if w_o >= 1 else int(last_j[b]) - n_so)
    return cap


def ring_timing(wl, n_steps: int, steps: int, warmup: int, replicas: int, split_len: int, capture,
                time_graph) -> dict:
    """The same steps on ring storage (murmur_decode_step_ring: retained set, attention and the append
    of the current token in one launch), timed as a replayed graph, with the storage it needs."""
    from paper_2606_01483_amd import murmur as M
    from paper_2606_01483_amd.decode import RingBatch
    cap = ring_capacity(wl, n_steps)
    log(f"ring storage: {cap} output rows, {replicas} replica(s)")
    rb = RingBatch(wl, cap, replicas=replicas, split_len=split_len if split_len >= 0 else 0,
                   steps=list(range(n_steps)))
    for i in range(warmup):
        rb.step(i % n_steps, i % replicas)
    graph = capture(lambda: [rb.step(i % n_steps, i % replicas) for i in range(steps)])
    ring_us = time_graph(graph) / steps
    if M.murmur_device_error() != 0:
        raise RuntimeError("device error during the timed ring steps")
    last = wl.seg(n_steps - 1)
    linear_rows = int(last.sum(axis=1).max())  # rows per sequence of the sequence-ordered cache at the last step
    per_row = wl.n_layers * wl.batch * wl.hkv * wl.head_dim * 2 * 2
    return {"step_us": round(ring_us, 3), "out_capacity": cap, "rows_per_sequence": rb.rows,
            "rows_per_sequence_linear": linear_rows, "kv_resident_bytes": rb.rows * per_row,
            "kv_resident_bytes_linear": linear_rows * per_row}


def paged_timing(wl, n_steps: int, steps: int, warmup: int, replicas: int, split_len: int, capture,
                 time_graph, block_size: int = 16) -> dict:
    """The same steps on a paged cache (blocks of 16 rows in one pool, [block][slot][kv head][D], a random block
    table): murmur_evict_compact_paged + murmur_decode_attn over the pool's rows, and the attention alone."""
    from paper_2606_01483_amd import murmur as M
    from paper_2606_01483_amd.decode import PagedBatch
    log(f"paged cache: blocks of {block_size}, {replicas} replica(s)")
    pb = PagedBatch(wl, block_size, replicas=replicas, split_len=split_len, steps=list(range(n_steps)))
    for i in range(warmup):
        pb.step(i % n_steps, i % replicas)
    graph = capture(lambda: [pb.step(i % n_steps, i % replicas) for i in range(steps)])
    step_us = time_graph(graph) / steps
    pb.evict(0)
    graph = capture(lambda: [pb.attend(0, i % replicas) for i in range(steps)])
    attn_us = time_graph(graph) / steps
    if M.murmur_device_error() != 0:
        raise RuntimeError("device error during the timed paged steps")
    res = {"block_size": block_size, "pool_layout": "block, slot, kv head, head dim",
           "step_two_launches_us": round(step_us, 3), "decode_attn_us": round(attn_us, 3)}
    res.update(device_manager_timing(wl, n_steps, block_size, split_len))
    return res


def device_manager_timing(wl, n_steps: int, block_size: int, split_len: int) -> dict:
    """The same decode on a paged cache whose block manager runs on the device: murmur_paged_step (free the
    blocks no later step reads, take a block for the current token, write its K/V) alone, and the whole
    three-launch step, each over all steps captured into one graph and replayed from the starting state.  One
    copy of the cache (its state changes with every step), so the attention here reads warm data."""
    import torch
    from paper_2606_01483_amd import murmur as M
    from paper_2606_01483_amd.decode import DevicePagedBatch
    log("device block manager: graphs of paged steps")
    lens = wl.seg(n_steps - 1).sum(axis=1)
    dp = DevicePagedBatch(wl, block_size, int((-(-lens // block_size)).sum()) + wl.batch,
                          out_dtype=M.MURMUR_DTYPE_BF16, split_len=split_len)
    start = dp.state()
    stream = torch.cuda.current_stream()

    def per_step_us(fn) -> float:
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        dp.restore(start)
        cap.wait_stream(stream)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap):
            for i in range(n_steps):
                fn(i)
        best = None
        for _ in range(3):  # the first replay warms up
            dp.restore(start)
            torch.cuda.synchronize()
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            graph.replay()
            t1.record(stream)
            torch.cuda.synchronize()
            us = t0.elapsed_time(t1) * 1e3 / n_steps
            best = us if best is None else min(best, us)
        return best

    manager_us = per_step_us(dp.manage)
    step_us = per_step_us(dp.step)
    if M.murmur_device_error() != 0:
        raise RuntimeError("device error during the device block manager timing")
    return {"device_manager_us": round(manager_us, 3), "device_managed_step_us_warm": round(step_us, 3)}


def recycled_blocks(seg0, policy, block_size: int = 16, n_outputs: int = 2700) -> dict:
    """Host-only: blocks of `block_size` positions the sequences hold over a decode from their layout to
    n_outputs output tokens when every block no later step retains goes back to the pool before each step
    (murmur_freeable_blocks_host), against the blocks they hold at the end without freeing."""
    from paper_2606_01483_amd import murmur as M
    seg0 = np.asarray(seg0, dtype=np.int32).reshape(-1, 4)
    pol = np.ascontiguousarray(policy, dtype=np.int32)
    B = seg0.shape[0]
    peak = 0
    for j in range(1, n_outputs + 1):
        seg = seg0.copy()
        seg[:, 3] = j
        held = -(-seg.sum(axis=1) // block_size)  # logical blocks up to the current token
        fb = M.murmur_freeable_blocks_host(seg, pol, block_size, 1 if pol.ndim == 2 else 0)
        peak = max(peak, int((held - fb[:, :, 1].sum(axis=1)).sum()))
    seg = seg0.copy()
    seg[:, 3] = n_outputs
    return {"block_size": block_size, "outputs": n_outputs, "peak_blocks": peak,
            "blocks_without_freeing": int((-(-seg.sum(axis=1) // block_size)).sum())}


def graph_tools(stream):
    """capture(fn): fn's launches captured into a HIP graph on a side stream, replayed once to warm up;
    time_graph(graph): µs of one replay, between HIP events recorded on `stream` around it.  Before the timed
    replay two plain reads of 512 MB (twice the Infinity Cache) run untimed, so that no data of the warm-up
    replay is still cached when the timed one starts; they are queued with the replay, so the GPU is busy
    while the host submits it and the start event is followed by the replay's first kernel at once."""
    import torch
    from paper_2606_01483_amd import murmur as M
    flush_bytes = 2 * MALL_BYTES
    flush_buf = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda")
    flush_sink = torch.zeros(1024, dtype=torch.int32, device="cuda")

    def capture(fn):
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap):
            fn()
        torch.cuda.synchronize()
        graph.replay()  # warm replay
        torch.cuda.synchronize()
        return graph

    def time_graph(graph) -> float:
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        # The flush reads run while the host submits the replay (no synchronisation in between), so the
        # replay's kernels follow the start event at once: the host's submission latency stays outside.
        for _ in range(2):
            M.murmur_read_probe(flush_buf, flush_bytes, 1024, flush_sink, 256, 8, M.MURMUR_PROBE_REGISTERS, stream)
        t0.record(stream)
        graph.replay()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) * 1e3

    return capture, time_graph


def marginal_us(launch, n: int, capture, time_graph) -> tuple[float, float]:
    """Per-launch time of back-to-back launches without the graph's fixed start cost: replayed graphs of n and
    of 2n launches (launch(i) issues the i-th), (t(2n) - t(n)) / n; and the plain mean t(n) / n beside it."""
    g1 = capture(lambda: [launch(i) for i in range(n)])
    t1 = time_graph(g1)
    del g1
    g2 = capture(lambda: [launch(i) for i in range(2 * n)])
    t2 = time_graph(g2)
    del g2
    return (t2 - t1) / n, t1 / n


def per_step_attn(db, steps: list[int], replicas: int, capture, time_graph) -> dict:
    """decode_attn duration step by step: per distinct step, its retained set, then the marginal per-launch
    time (marginal_us) of back-to-back launches over it, each on the next KV replica (the replicas together
    hold more than twice the Infinity Cache), n = max(replicas, 32); the median, p90, mean, min and max over
    the steps."""
    per = []
    n = max(replicas, 32)
    for s in sorted(set(steps)):
        db.evict(s)
        per.append(marginal_us(lambda r: db.attend(s, r % replicas), n, capture, time_graph)[0])
    a = np.array(per)
    return {"steps": len(per), "launches_per_step": n, "median": round(float(np.median(a)), 3),
            "p90": round(float(np.percentile(a, 90)), 3), "mean": round(float(a.mean()), 3),
            "min": round(float(a.min()), 3), "max": round(float(a.max()), 3)}


def run(config: str, steps: int, warmup: int, replicas: int | None, cpu: bool, cpu_budget: float,
        split_len: int, use_ranges: bool, with_ring: bool = True) -> dict:
    import torch
    from paper_2606_01483_amd import murmur as M
    from paper_2606_01483_amd import workloads as W
    from paper_2606_01483_amd.decode import DecodeBatch, retained_counts

    torch.cuda.init()
    M.lib()
    lay = W.layout(config)
    n_steps = max(lay.steps, steps)
    log(f"workload {config}: drawing inputs ({n_steps} steps)")
    wl = W.make(config, steps=n_steps)
    counts = [retained_counts(wl, s) for s in range(n_steps)]  # [NL, B] per step
    kv_step = [int(c.sum()) * wl.hkv * 2 * wl.head_dim * 2 for c in counts]
    if replicas is None:
        replicas = replicas_for(wl, kv_step)
    log(f"uploading: {replicas} KV replica(s) of {wl.k.nbytes * 2 / 1e6:.1f} MB")
    db = DecodeBatch(wl, replicas=replicas, out_dtype=M.MURMUR_DTYPE_BF16, split_len=split_len,
                     use_ranges=use_ranges, steps=list(range(n_steps)))
    stream = torch.cuda.current_stream()

    order = [i % n_steps for i in range(steps)]
    rep = [i % replicas for i in range(steps)]
    # Per-layer policies run on the fused step only: it is then also the kernel the roofline is taken on.
    two_launch = not db.per_layer

    for i in range(warmup):
        if two_launch:
            db.step(i % n_steps, i % replicas)
        db.step_fused(i % n_steps, i % replicas)
    torch.cuda.synchronize()
    if M.murmur_device_error() != 0:
        raise RuntimeError("device error during warm-up")

    bracket_us = None
    if two_launch:
        # Per-launch event brackets (diagnostic: they include each launch's dispatch latency).
        log("timing decode_attn launches with HIP event brackets")
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for i in range(steps):
            db.evict(order[i])
            evs[i][0].record(stream)
            db.attend(order[i], rep[i])
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        bracket_us = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])

    capture, time_graph = graph_tools(stream)

    # Whole steps, captured once into a graph and replayed: the single-launch murmur_decode_step (the
    # step's value, retained-set outputs written), and murmur_evict_compact + murmur_decode_attn.
    log("timing the fused steps as a replayed HIP graph")
    fused_graph = capture(lambda: [db.step_fused(order[i], rep[i]) for i in range(steps)])
    step_us = time_graph(fused_graph) / steps
    if M.murmur_device_error() != 0:
        raise RuntimeError("device error during the timed fused steps")
    io = db.io_bytes()
    if two_launch:
        log("timing the two-launch steps as a replayed HIP graph")
        step_graph = capture(lambda: [db.step(order[i], rep[i]) for i in range(steps)])
        two_launch_us = time_graph(step_graph) / steps
        if M.murmur_device_error() != 0:
            raise RuntimeError("device error during the timed steps")

        # decode_attn alone: the same launches back to back (retained set of the first timed step, each
        # launch reading the next KV replica).  The kernel's duration is the marginal cost of a launch in
        # such a graph (graphs of n and 2n launches, n = max(steps, 64)): a replay also pays a fixed start
        # (about 10 us here), which the mean over the K timed launches carries divided by K.
        log("timing decode_attn launches as replayed HIP graphs")
        db.evict(order[0])
        n_attn = max(steps, 64)
        attn_us, _ = marginal_us(lambda i: db.attend(order[i % steps], i % replicas), n_attn, capture, time_graph)
        attn_graph = capture(lambda: [db.attend(order[i], rep[i]) for i in range(steps)])
        attn_graph_mean_us = time_graph(attn_graph) / steps
        del attn_graph
        if M.murmur_device_error() != 0:
            raise RuntimeError("device error during the timed decode_attn launches")
        alg_bytes = float(kv_step[order[0]] + io)  # every launch of the decode_attn graph reads this set
        log("timing decode_attn step by step")
        attn_per_step = per_step_attn(db, order, replicas, capture, time_graph)
        if M.murmur_device_error() != 0:
            raise RuntimeError("device error during the per-step decode_attn launches")
    else:
        two_launch_us = None
        attn_us = step_us
        attn_graph_mean_us = step_us
        attn_per_step = None
        alg_bytes = float(np.mean([kv_step[o] for o in order]) + io)

    ceiling = read_ceiling(int(alg_bytes), steps, capture, time_graph)

    ring = None
    if with_ring:
        ring = ring_timing(wl, n_steps, steps, warmup, replicas_for(wl, kv_step), split_len, capture, time_graph)
    paged = None
    if with_ring and two_launch and split_len >= 0:
        paged = paged_timing(wl, n_steps, steps, warmup, replicas_for(wl, kv_step), split_len, capture, time_graph)

    achieved = float(alg_bytes / (attn_us * 1e-6) / 1e9)
    res = {
        "metric": METRIC,
        "value": round(step_us, 3),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(step_us / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{config}: {DESCRIPTIONS[config]}", "batch": wl.batch, "layers": wl.n_layers,
                   "q_heads": wl.hq, "kv_heads": wl.hkv, "head_dim": wl.head_dim,
                   "retained_per_step": int(np.mean([int(counts[o].sum()) for o in order]) / wl.n_layers),
                   "kv_replicas": replicas, "selection": "ranges" if use_ranges else "index list",
                   "split_len": db.split_len or "auto"},
        "step_two_launches_us": round(two_launch_us, 3) if two_launch else None,
        "decode_attn_us": round(attn_us, 3),
        "decode_attn_graph_mean_us": round(attn_graph_mean_us, 3),
        "decode_attn_per_step_us": attn_per_step,
        "decode_attn_event_bracket_us": None if bracket_us is None else {
            "mean": round(float(bracket_us.mean()), 3), "median": round(float(np.median(bracket_us)), 3),
            "p90": round(float(np.percentile(bracket_us, 90)), 3)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": committed_traffic(config),
                     "kernel": "decode_attn" if two_launch else "decode_step (fused; per-layer policies)",
                     "alg_bytes_per_launch": int(alg_bytes)},
    }
    res["read_ceiling"] = ceiling
    res["roofline"]["frac_of_read_ceiling"] = round(achieved / ceiling["GBps"], 4)
    if ring is not None:
        res["ring"] = ring
    if paged is not None:
        res["paged"] = paged
        if np.ndim(wl.policy) < 3:
            res["paged"]["recycled_to_2700_outputs"] = recycled_blocks(wl.seg0 * np.array([1, 1, 1, 0]), wl.policy)
    if cpu:
        threads = max(1, min(16, len(os.sched_getaffinity(0))))
        log(f"timing the fp64 oracle on {threads} host threads")
        res["cpu_baseline"] = cpu_baseline(wl, cpu_budget, threads)
        log("timing the fp64 oracle on one host thread")
        one = cpu_baseline(wl, max(1.0, cpu_budget / 3), 1)
        res["cpu_baseline"]["single_thread"] = {"value": one["value"], "unit": one["unit"], "sample": one["sample"]}
        log("checking one timed step against the oracle")
        res["cpu_baseline"]["parity"] = oracle_parity(wl, db, order[0])
    return res


def ablation(samples: int, reps: int, split_len: int) -> list[dict]:
    """Decode-attention time of every eviction preset of the paper's ablations over a whole decode of
    2700 output tokens (batch 16, 300 s chunks): the fused step is timed at `samples` evenly spaced
    steps (a graph of `reps` launches per step, each on the next KV replica) and averaged, next to the
    exact ratio of dense to retained positions summed over all 2700 steps."""
    import torch
    from paper_2606_01483_amd import murmur as M
    from paper_2606_01483_amd import workloads as W
    from paper_2606_01483_amd.decode import DecodeBatch

    torch.cuda.init()
    M.lib()
    log("ablation: drawing the 16-chunk cache")
    base = W.ablation_workload("full")
    T = base.steps
    sample_steps = sorted({int(round(k * (T - 1) / (samples - 1))) for k in range(samples)})
    dense = np.array([int(base.seg(s)[:, :4].sum()) for s in range(T)], dtype=np.float64)
    out = []
    full_us = None
    for name, pol in W.ABLATION_PRESETS.items():
        wl = W.with_policy(base, pol)
        kept = np.array([int(M.murmur_retained_count_host(wl.seg(s), wl.policy, 1)[0].sum()) for s in range(T)],
                        dtype=np.float64)
        kv_min = int(kept[sample_steps].min()) * wl.hkv * 2 * wl.head_dim * 2
        replicas = min(max(1, math.ceil(2.2 * MALL_BYTES / kv_min)), max(1, (24 << 30) // (wl.k.nbytes * 2)))
        log(f"ablation {name}: {replicas} replica(s)")
        db = DecodeBatch(wl, replicas=replicas, split_len=split_len, steps=sample_steps)
        stream = torch.cuda.current_stream()
        per_step = []
        for i in range(len(sample_steps)):
            for r in range(2):
                db.step_fused(i, r % replicas, outputs=False)
            graph = torch.cuda.CUDAGraph()
            cap = torch.cuda.Stream()
            cap.wait_stream(stream)
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=cap):
                for r in range(reps):
                    db.step_fused(i, r % replicas, outputs=False)
            torch.cuda.synchronize()
            graph.replay()
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            t0.record(stream)
            graph.replay()
            t1.record(stream)
            torch.cuda.synchronize()
            per_step.append(t0.elapsed_time(t1) * 1e3 / reps)
            del graph
        if M.murmur_device_error() != 0:
            raise RuntimeError(f"device error in ablation preset {name}")
        us = float(np.mean(per_step))
        if full_us is None:
            full_us = us
        out.append({"preset": name, "policy": list(map(int, pol)), "batch": wl.batch, "outputs": T,
                    "sample_steps": len(sample_steps), "attn_step_us_mean": round(us, 3),
                    "attn_step_us_first_last": [round(per_step[0], 3), round(per_step[-1], 3)],
                    "kept_fraction_mean": round(float(np.mean(kept / dense)), 4),
                    "kept_fraction_last": round(float(kept[-1] / dense[-1]), 4),
                    "dense_over_kept_positions": round(float(dense.sum() / kept.sum()), 4),
                    "measured_speedup_vs_full": round(full_us / us, 4)})
        print(json.dumps(out[-1]), flush=True)
        del db
        torch.cuda.empty_cache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c3", help="workload: c1, c2, c3, c4_dense, c4_evict, c5, c5_layers")
    ap.add_argument("--replicas", type=int, default=None, help="KV cache replicas to rotate over (default: auto)")
    ap.add_argument("--split-len", type=int, default=0)
    ap.add_argument("--index-list", action="store_true", help="attend from the index list instead of ranges")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ring", action="store_true", help="skip the ring-storage timing")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle timing")
    ap.add_argument("--all", action="store_true", help="one JSON line per workload (c1 .. c5), no CPU baseline")
    ap.add_argument("--ablation", action="store_true",
                    help="one JSON line per eviction preset of the paper's ablations (batch 16, 2700 outputs)")
    ap.add_argument("--ablation-samples", type=int, default=12)
    ap.add_argument("--copy-reference", type=int, default=0, metavar="MB",
                    help="only run plain device copies of this many MiB (PMC counter reference)")
    ap.add_argument("--summarize-trace", metavar="DIR", help="print the kernel table of a rocprofv3 --stats run")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="print the traffic summary from four rocprofv3 --pmc runs")
    ap.add_argument("--pmc-kernel", default="decode_attn_wide_kernel<1>", help="kernel name part for --summarize-pmc")
    ap.add_argument("--copy-mib", type=int, default=256, help="copy size of the --copy-reference runs")
    ap.add_argument("--alg-bytes", type=int, default=0, help="algorithmic bytes per launch (bench JSON)")
    ap.add_argument("--read-sweep", type=int, default=0, metavar="BYTES",
                    help="only run the read-ceiling sweep at this byte count (and 1 GiB), print a markdown table")
    args = ap.parse_args()
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return 0
    if args.summarize_pmc:
        print(summarize_pmc(args.config, args.pmc_kernel, *args.summarize_pmc, args.copy_mib, args.alg_bytes))
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this decode path has no multi-GPU mode (got --gpus {args.gpus})",
              file=sys.stderr)
        return 2
    if args.ablation:
        ablation(args.ablation_samples, max(4, args.steps // 4), args.split_len)
        return 0
    if args.copy_reference:
        print(json.dumps(copy_reference(args.copy_reference, 8)), flush=True)
        return 0
    if args.read_sweep:
        import torch
        from paper_2606_01483_amd import murmur as M
        torch.cuda.init()
        M.lib()
        rows = read_sweep(args.read_sweep, args.steps, *graph_tools(torch.cuda.current_stream()))
        print(sweep_table(rows), flush=True)
        print(json.dumps(rows), flush=True)
        return 0
    if args.all:
        from paper_2606_01483_amd import workloads as W
        for cfg in W.CONFIGS:
            res = run(cfg, args.steps, args.warmup, None, False, 0.0, args.split_len, not args.index_list,
                      not args.no_ring)
            print(json.dumps(res), flush=True)
        return 0
    res = run(args.config, args.steps, args.warmup, args.replicas, not args.no_cpu_baseline, args.cpu_budget,
              args.split_len, not args.index_list, not args.no_ring)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
