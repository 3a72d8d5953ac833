#!/usr/bin/env python3
"""Benchmark: split paged decode attention + merge on one MI355X.

One step = every partition's ``bana_decode_attn_partial`` call plus the
``bana_merge_partials`` call for one decode token of every sequence (one
layer), on inputs already resident in HBM.  The same step through the fused
entry point (``bana_decode_attn_fused``: all partitions and the merge in one
launch) is timed as well and reported under ``fused_path``.  Default workload: the
Llama-3-8B-shaped layer (batch 64, 32 query / 8 KV heads, head_dim 128,
block 16, seq_len 4096, last 30 % of each sequence's blocks migrated ->
2 partitions) over a 20 % oversized, randomly permuted block pool.

Prints ONE JSON line.  ``value`` is the KV-read bandwidth of the whole step
(K+V bytes of all covered tokens / step time); ``tokens_per_s`` is decode
tokens (sequences) per second for the layer.  Every time is the median of K
repetitions, each timed alone by HIP events on its stream after a cache scrub
(512 MiB written, then read back; ``timing`` gives p10 / p90); ``warm_back_to_back``
is the same step run K times back to back with warm caches, by the host
clock.  ``gather_read_ceiling`` reads the same
tiles with no arithmetic (the access pattern's practical ceiling);
``stream_read_ceiling`` reads both block pools front to back (HBM's
streaming-read ceiling on this GPU).
``roofline`` reports the partial-attention kernel against the 8 TB/s HBM
peak, timed with HIP events on the stream it runs on, with the HBM bytes of
the committed counter summary when it matches the kernel sources.
``migration`` times the KV-block copy of the migrated partition;
``head_split`` times the head-split form of the method (each half of the kv
heads over whole sequences, one ``bana_decode_attn_heads`` call each).
``cpu_baseline`` times the fp64 CPU oracle on the same workload on this host
(all cores, plus a single-core sample).
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
METRIC = "KV-read GB/s (% of HBM peak) and decode tokens/s, split paged attention"


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="llama3_8b", choices=["tiny", "llama3_8b", "long", "mixed", "fine", "mha13b"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target CPU time of the oracle baseline")
    ap.add_argument("--waves", type=int, default=0, help="waves-per-workgroup hint (0 = library plan)")
    ap.add_argument("--chunks", type=int, default=0, help="chunks-per-range hint (0 = library plan)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (for scaling HBM byte counters)")
    ap.add_argument("--profile-regions", action="store_true",
                    help="for profiler runs: each call type in a region of its own (K scrubbed repetitions), "
                         "regions separated by sentinel launches; prints the region list instead of timings")
    return ap.parse_args()


def _workload_desc(w):
    nb = (w.kv_end - w.kv_begin).astype(np.int64)
    return {
        "workload": w.name,
        "batch": w.batch,
        "num_q_heads": w.num_q_heads,
        "num_kv_heads": w.num_kv_heads,
        "head_dim": 128,
        "block_size": 16,
        "seq_len_mean": float(np.mean(w.seq_lens)),
        "partitions": w.n_parts,
        "tokens_per_partition": [int(x) for x in nb.sum(axis=1)],
        "pool_blocks": w.num_blocks,
        "seed": w.seed,
    }


def _partial_algorithmic_bytes(w, p):
    """Bytes one partial launch must move: K/V of covered tokens, q, table entries, fp32 out + lse."""
    toks = int(np.sum(w.kv_end[p].astype(np.int64) - w.kv_begin[p]))
    kv = toks * w.num_kv_heads * 128 * 2 * 2
    blocks = 0
    for b in range(w.batch):
        t0, t1 = int(w.kv_begin[p, b]), int(w.kv_end[p, b])
        if t1 > t0:
            blocks += (t1 - 1) // 16 - t0 // 16 + 1
    q = w.batch * w.num_q_heads * 128 * 2
    out = w.batch * w.num_q_heads * (128 + 1) * 4
    return kv + q + blocks * 4 + w.batch * 8 + out, kv


KERNEL_SOURCES = ("paper_2510_13223_amd/csrc/attn_partial.hip", "paper_2510_13223_amd/csrc/paged_addr.h",
                  "paper_2510_13223_amd/csrc/kernels.h", "paper_2510_13223_amd/csrc/bana_api.cpp")
TRAFFIC_PROFILE = "profiles/hbm_bytes_{workload}.md"


def _kernel_source_sha256() -> str:
    import hashlib

    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _measured_traffic(workload: str):
    """HBM bytes per partial launch from the committed FETCH_SIZE / WRITE_SIZE summary.

    Returned only when that summary was taken on the same workload and on the
    kernel sources as they are now (sha256 over the kernel's source files);
    otherwise None.
    """
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), TRAFFIC_PROFILE.format(workload=workload))
    try:
        fields = {}
        for line in open(path):
            if ":" in line and line.startswith("- "):
                k, v = line[2:].split(":", 1)
                fields[k.strip()] = v.strip().strip("`")
        if fields.get("workload") != workload or fields.get("kernel_source_sha256") != _kernel_source_sha256():
            return None
        return float(fields["fetch_bytes_per_launch"]) + float(fields["write_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def _cpu_baseline(w, target_s):
    import oracle  # CPU baseline leg only

    threads = len(os.sched_getaffinity(0))
    reps = 0
    t_start = time.perf_counter()
    while True:
        outs, lses = oracle.workload_partials(w, threads=threads)
        oracle.merge(outs, lses)
        reps += 1
        el = time.perf_counter() - t_start
        if el >= target_s or el / reps * (reps + 1) > 3 * target_s:
            break
    per_step = el / reps
    kv = w.kv_bytes()
    # One core: a prefix of the batch (whole sequences, all partitions), sized to about a tenth of target_s.
    per_seq = per_step * threads / w.batch  # rough single-core seconds per sequence
    n_single = int(max(1, min(w.batch, 0.1 * target_s / max(per_seq, 1e-9))))
    seqs = list(range(n_single))
    t_start = time.perf_counter()
    o1, l1 = oracle.workload_partials(w, seqs=seqs, threads=1)
    oracle.merge(o1, l1)
    t1 = time.perf_counter() - t_start
    n1 = n_single
    kv1 = int(np.sum(w.kv_end[:, :n1].astype(np.int64) - w.kv_begin[:, :n1])) * w.num_kv_heads * 128 * 2 * 2
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": kv / per_step / 1e9,
        "unit": "GB/s",
        "tokens_per_s": w.batch / per_step,
        "cores": threads,
        "kind": "oracle",
        "sample": f"full {w.name} step (all {w.n_parts} partitions of {w.batch} sequences + merge), "
                  f"fp64, {reps} repetitions in {el:.1f} s",
        "cpu_model": model,
        "s_per_step": per_step,
        "single_core": {
            "value": kv1 / t1 / 1e9,
            "unit": "GB/s",
            "cores": 1,
            "sample": f"first {n1} of {w.batch} sequences (all partitions + merge), fp64, {t1:.2f} s",
        },
    }


SENTINEL_BYTES = 4096  # sentinel launch: bana_debug_stream_read of 4 KiB by (region + 1) workgroups


def _profile_regions(args, w, dw, stream, h, torch, bana, workloads):
    """Profiler mode: every call type of the step (each partition's partial call, the merge, the
    fused call, the migration of the last partition, each head half, the gather read) runs K times
    in a region of its own, each repetition after a cache scrub (512 MiB written, then read back by
    2048 workgroups), regions separated by a sentinel launch of bana_debug_stream_read over 4 KiB
    with region + 1 workgroups, so a profiler's dispatch list splits into regions by kernel name
    and grid size alone.  Prints one JSON line naming the regions in order."""
    import numpy as np

    dev = dw.q.device
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    scrub_sink = torch.empty(2048, dtype=torch.int32, device=dev)
    sent_buf = torch.zeros(SENTINEL_BYTES, dtype=torch.uint8, device=dev)
    regions = [(f"partition {p}", (lambda p=p: dw.partial(p, h))) for p in range(w.n_parts)]
    regions += [("merge", lambda: dw.merge(h)), ("fused", lambda: dw.fused(h))]
    mig = workloads.make_migration(w, w.n_parts - 1, seed=1)
    to_dev = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    d_k, d_v = to_dev(mig.dst_k), to_dev(mig.dst_v)
    d_t, m_b, m_e = (torch.from_numpy(x).to(dev) for x in (mig.dst_table, mig.blk_begin, mig.blk_end))
    hint = int(np.max(mig.blk_end - mig.blk_begin)) * 16
    regions.append(("migration", lambda: bana.bana_migrate_kv_blocks(
        dw.k_cache, dw.v_cache, dw.block_table, d_k, d_v, d_t, m_b, m_e, stream=stream, max_range_tokens=hint)))
    lens = w.seq_lens.astype(np.int64)
    hs_dims = bana.make_dims(w.batch, w.num_q_heads, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks,
                             max_range_tokens=int(lens.max()), total_range_tokens=int(lens.sum()),
                             nonempty_ranges=int(np.count_nonzero(lens)))
    zeros = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    hs_out = torch.empty((w.batch, w.num_q_heads, 128), dtype=torch.float32, device=dev)
    hs_lse = torch.empty((w.batch, w.num_q_heads), dtype=torch.float32, device=dev)
    half = max(1, w.num_kv_heads // 2)
    for g0, g1 in ((0, half), (half, w.num_kv_heads)):
        if g0 == g1:
            continue
        n = bana.bana_decode_attn_workspace_bytes(bana.head_range_dims(hs_dims, g0, g1))
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device=dev)
        regions.append((f"heads {g0}-{g1}", (lambda g0=g0, g1=g1, ws=ws: bana.bana_decode_attn_heads(
            dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, zeros, dw.seq_lens, g0, g1, hs_out, hs_lse,
            workspace=ws, stream=stream, dims=hs_dims))))
    sink = torch.empty((w.batch, w.num_kv_heads), dtype=torch.int32, device=dev)
    regions.append(("gather read", lambda: bana.bana_debug_gather_read(
        dw.k_cache, dw.v_cache, dw.block_table, dw.kv_begin, dw.kv_end, sink, stream=stream)))
    with torch.cuda.stream(stream):
        for i, (name, fn) in enumerate(regions):
            bana.bana_debug_stream_read(sent_buf, scrub_sink[:i + 1], stream=stream)
            for k in range(args.steps):
                scrub.fill_(k & 0xFF)
                bana.bana_debug_stream_read(scrub, scrub_sink, stream=stream)
                fn()
            stream.synchronize()
            print(f"[bench] region {i}: {name}", file=sys.stderr, flush=True)
        bana.bana_debug_stream_read(sent_buf, scrub_sink[:len(regions) + 1], stream=stream)
    if args.copy_calibration:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"metric": METRIC, "profile_regions": [r[0] for r in regions], "steps": args.steps,
                      "config": _workload_desc(w), "copy_calibration_bytes": (1 << 30) if args.copy_calibration
                      else 0}), flush=True)


def main():
    args = _parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the method's partitions would shard across GPUs with one point-to-point exchange per step).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2510_13223_amd import workloads
    from paper_2510_13223_amd.runner import DeviceWorkload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.time()
    w = workloads.make_config(args.config, args.seed)
    print(f"[bench] generated {w.name} in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    dw = DeviceWorkload(w, device=dev, waves_hint=args.waves, chunks_hint=args.chunks)
    stream = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            dw.step(stream)
    stream.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    P = w.n_parts
    h = ctypes.c_void_p(stream.cuda_stream)
    from paper_2510_13223_amd import bana

    if args.profile_regions:
        _profile_regions(args, w, dw, stream, h, torch, bana, workloads)
        return

    # Every timed figure below is taken the same way: HIP events recorded on the stream the work
    # runs on, around each repetition alone, with a cache scrub between repetitions (outside the
    # events); the figure is the median over the K repetitions, with p10 / p90 beside it.  The
    # scrub writes a 512 MiB buffer, so neither L2 nor the 256 MB last-level cache holds K/V from
    # the previous repetition, then reads it back, so no dirty scrub line is left to be written
    # back inside the timed region (measured on MI355X: a write alone adds up to 60 us of
    # write-back to the fine workload's step).
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    scrub_sink = torch.empty(2048, dtype=torch.int32, device=dev)

    def scrub_caches(k):
        scrub.fill_(k & 0xFF)
        bana.bana_debug_stream_read(scrub, scrub_sink, stream=stream)

    def timed_cold(fn, inner=None):
        """Event-timed repetitions of fn with a scrub before each; returns us per repetition
        (and, when ``inner`` is given, the us between the two events fn passes to ``inner``)."""
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            for k in range(args.steps):
                scrub_caches(k)
                ev[k][0].record(stream)
                fn()
                ev[k][1].record(stream)
        stream.synchronize()
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) * 1e3 for a, b in ev])

    def stats(us):
        return {"median_us": round(float(np.median(us)), 2), "p10_us": round(float(np.percentile(us, 10)), 2),
                "p90_us": round(float(np.percentile(us, 90)), 2), "mean_us": round(float(np.mean(us)), 2)}

    # Timed region 1 (the headline): exactly K steps, each timed alone by events after a cache scrub,
    # synchronised on both sides of the region.
    step_us = timed_cold(lambda: dw.step_on(h))
    t_step = float(np.median(step_us)) / 1e6
    print(f"[bench] timed {args.steps} steps (cold caches): median {t_step * 1e6:.1f} us/step", file=sys.stderr,
          flush=True)

    # Side figure: the same K steps back to back with warm caches, host clock synchronised on both sides.
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for _ in range(args.steps):
        dw.step_on(h)
    stream.synchronize()
    torch.cuda.synchronize()
    warm_ms = (time.perf_counter() - wall0) * 1e3 / args.steps
    print(f"[bench] back to back: {warm_ms * 1e3:.1f} us/step", file=sys.stderr, flush=True)

    # Practical ceiling of the access pattern: the same K/V tiles read through the same
    # table walk with no arithmetic (bana_debug_gather_read over all partitions).
    sink = torch.empty((w.batch, w.num_kv_heads), dtype=torch.int32, device=dev)

    def gather():
        bana.bana_debug_gather_read(dw.k_cache, dw.v_cache, dw.block_table, dw.kv_begin, dw.kv_end, sink,
                                    stream=stream)

    for _ in range(args.warmup):
        gather()
    gather_s = float(np.median(timed_cold(gather))) / 1e6
    print(f"[bench] gather-read ceiling: {gather_s * 1e6:.1f} us", file=sys.stderr, flush=True)

    # Streaming ceiling of HBM reads: both pools read front to back (bana_debug_stream_read,
    # 2048 workgroups of 256 threads = 32 resident wavefronts per CU).
    stream_sink = torch.empty(2048, dtype=torch.int32, device=dev)
    pool_bytes = 2 * dw.k_cache.numel() * dw.k_cache.element_size()

    def stream_read():
        bana.bana_debug_stream_read(dw.k_cache, stream_sink, stream=stream)
        bana.bana_debug_stream_read(dw.v_cache, stream_sink, stream=stream)

    for _ in range(args.warmup):
        stream_read()
    stream_s = float(np.median(timed_cold(stream_read))) / 1e6
    print(f"[bench] stream-read ceiling: {stream_s * 1e6:.1f} us for {pool_bytes} B", file=sys.stderr, flush=True)

    # Timed region 2: the same K steps, scrubbed, with HIP events on the kernel's stream (a) around
    # each step's back-to-back partial-attention launches (the merge after the second event): the
    # kernel's mean launch duration for the roofline; (b) around every single launch, for the split
    # by partition (those records add a little time per launch).
    ev_all = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(P)]
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for k in range(args.steps):
            scrub_caches(k)
            ev_all[k][0].record(stream)
            for p in range(P):
                dw.partial(p, h)
            ev_all[k][1].record(stream)
            dw.merge(h)
        for k in range(args.steps):
            scrub_caches(k)
            for p in range(P):
                ev[k][p][0].record(stream)
                dw.partial(p, h)
                ev[k][p][1].record(stream)
            dw.merge(h)
    stream.synchronize()
    torch.cuda.synchronize()

    # Timed region 3: the same step through the fused entry point (every partition and the
    # merge in one launch).
    for _ in range(args.warmup):
        dw.fused(h)
    fused_us = timed_cold(lambda: dw.fused(h))
    fused_ms = float(np.median(fused_us)) / 1e3
    print(f"[bench] fused path: {fused_ms * 1e3:.1f} us/step", file=sys.stderr, flush=True)

    # Timed region 4: KV-block migration of the last (migrated) partition into a second pool.
    mig = workloads.make_migration(w, P - 1, seed=1)
    mig_blocks = int(np.sum(mig.blk_end - mig.blk_begin))
    d_k = torch.from_numpy(mig.dst_k.view(np.int16)).view(torch.bfloat16).to(dev)
    d_v = torch.from_numpy(mig.dst_v.view(np.int16)).view(torch.bfloat16).to(dev)
    d_t = torch.from_numpy(mig.dst_table).to(dev)
    m_b = torch.from_numpy(mig.blk_begin).to(dev)
    m_e = torch.from_numpy(mig.blk_end).to(dev)
    mig_hint = int(np.max(mig.blk_end - mig.blk_begin)) * 16

    def migrate():
        bana.bana_migrate_kv_blocks(dw.k_cache, dw.v_cache, dw.block_table, d_k, d_v, d_t, m_b, m_e, stream=stream,
                                    max_range_tokens=mig_hint)

    for _ in range(args.warmup):
        migrate()
    mig_ms = float(np.median(timed_cold(migrate))) / 1e3
    mig_bytes = mig_blocks * w.num_kv_heads * 8192  # K + V tiles of every migrated block, read once and written once
    del d_k, d_v
    print(f"[bench] migration: {mig_ms * 1e3:.1f} us for {mig_bytes / 1e6:.1f} MB", file=sys.stderr, flush=True)

    # Timed region 5: the head split (the cache split along kv heads instead of tokens): each half of
    # the kv heads over whole sequences, one bana_decode_attn_heads call each.
    hs_begin = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    hs_end = dw.seq_lens
    lens_all = w.seq_lens.astype(np.int64)
    hs_dims = bana.make_dims(w.batch, w.num_q_heads, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks,
                             max_range_tokens=int(lens_all.max()), total_range_tokens=int(lens_all.sum()))
    hs_out = torch.empty((w.batch, w.num_q_heads, 128), dtype=torch.float32, device=dev)
    hs_lse = torch.empty((w.batch, w.num_q_heads), dtype=torch.float32, device=dev)
    half = w.num_kv_heads // 2
    hs_ranges = [(0, half), (half, w.num_kv_heads)] if half > 0 else [(0, w.num_kv_heads)]
    hs_ws = []
    for g0, g1 in hs_ranges:
        nbytes = bana.bana_decode_attn_workspace_bytes(bana.head_range_dims(hs_dims, g0, g1))
        hs_ws.append(torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev))

    def head_call(i):
        g0, g1 = hs_ranges[i]
        bana.bana_decode_attn_heads(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, hs_begin, hs_end,
                                    g0, g1, hs_out, hs_lse, workspace=hs_ws[i], stream=stream, dims=hs_dims)

    for _ in range(args.warmup):
        for i in range(len(hs_ranges)):
            head_call(i)
    hs_us = [float(np.median(timed_cold(lambda i=i: head_call(i)))) for i in range(len(hs_ranges))]
    hs_bytes = [int(lens_all.sum()) * (g1 - g0) * 128 * 2 * 2 for g0, g1 in hs_ranges]
    print(f"[bench] head split: {[round(x, 1) for x in hs_us]} us", file=sys.stderr, flush=True)
    del scrub

    kv_bytes = w.kv_bytes()
    ms_per_step = t_step * 1e3
    # Partial-attention kernel: algorithmic bytes over its own launch durations.
    alg = [_partial_algorithmic_bytes(w, p) for p in range(P)]
    dur_ms = np.array([[ev[k][p][0].elapsed_time(ev[k][p][1]) for p in range(P)] for k in range(args.steps)])
    step_partials_ms = np.array([a.elapsed_time(b) for a, b in ev_all])
    mean_dur_s = float(step_partials_ms.mean()) / P / 1e3
    mean_bytes = float(np.mean([a[0] for a in alg]))
    achieved = mean_bytes / mean_dur_s / 1e9
    partial_kv_gbs = float(np.sum([a[1] for a in alg])) / (float(step_partials_ms.mean()) / 1e3) / 1e9

    single = all(bana.bana_decode_attn_workspace_bytes(d) == 0 for d in dw.dims)
    roofline_kernel = ("partial_attn_kernel" if single else
                       "bana_decode_attn_partial call (attention kernel + chunk or piece merge)")
    line = {
        "metric": METRIC,
        "value": round(kv_bytes / t_step / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": _workload_desc(w),
        "timing": {
            "method": "HIP events around each step alone on its stream; between steps (outside the events) "
                      "a 512 MiB scrub written then read back; value and ms_per_step from the median",
            **stats(step_us),
        },
        "frac_of_hbm_peak": round(kv_bytes / t_step / 1e9 / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(w.batch / t_step, 1),
        "tokens_per_s_32_layers": round(w.batch / (32 * t_step), 1),
        "kv_bytes_per_step": kv_bytes,
        "warm_back_to_back": {
            "method": "K steps back to back with warm caches, host clock synchronised on both sides",
            "ms_per_step": round(warm_ms, 5),
            "value": round(kv_bytes / (warm_ms / 1e3) / 1e9, 2),
            "unit": "GB/s",
        },
        "fused_path": {
            "entry_point": "bana_decode_attn_fused",
            "ms_per_step": round(fused_ms, 5),
            **stats(fused_us),
            "value": round(kv_bytes / (fused_ms / 1e3) / 1e9, 2),
            "unit": "GB/s",
            "frac_of_hbm_peak": round(kv_bytes / (fused_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
            "tokens_per_s": round(w.batch / (fused_ms / 1e3), 1),
        },
        "partial_kernels_kv_gbs": round(partial_kv_gbs, 2),
        "gather_read_ceiling": {
            "entry_point": "bana_debug_gather_read",
            "what": "the step's K/V tiles read through the block table with the attention kernel's load shapes, "
                    "no arithmetic",
            # one workgroup of 8 wavefronts per (sequence, kv head): a ceiling only when those fill one round
            "comparable": w.batch * w.num_kv_heads >= 512,
            "us": round(gather_s * 1e6, 2),
            "value": round(kv_bytes / gather_s / 1e9, 2),
            "unit": "GB/s",
            "frac_of_hbm_peak": round(kv_bytes / gather_s / 1e9 / HBM_PEAK_GBS, 4),
        },
        "stream_read_ceiling": {
            "entry_point": "bana_debug_stream_read",
            "what": "both block pools read front to back (two launches), 16-byte non-temporal loads, "
                    "32 wavefronts per CU, no arithmetic",
            "comparable": pool_bytes >= (256 << 20),
            "bytes": pool_bytes,
            "us": round(stream_s * 1e6, 2),
            "value": round(pool_bytes / stream_s / 1e9, 2),
            "unit": "GB/s",
            "frac_of_hbm_peak": round(pool_bytes / stream_s / 1e9 / HBM_PEAK_GBS, 4),
        },
        "head_split": {
            "entry_point": "bana_decode_attn_heads",
            "what": "the cache split along kv heads: each range of kv heads over whole sequences, one call each "
                    "(what each device of a head split computes), HIP events around each call",
            "kv_heads": [list(r) for r in hs_ranges],
            "us_per_call": [round(x, 2) for x in hs_us],
            "kv_bytes_per_call": hs_bytes,
            "value": round(sum(hs_bytes) / (sum(hs_us) * 1e-6) / 1e9, 2),
            "unit": "GB/s",
            "frac_of_hbm_peak": round(sum(hs_bytes) / (sum(hs_us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        },
        "migration": {
            "entry_point": "bana_migrate_kv_blocks",
            "partition": P - 1,
            "blocks": mig_blocks,
            "bytes_moved": mig_bytes,
            "ms": round(mig_ms, 5),
            "copy_gbs": round(mig_bytes / (mig_ms / 1e3) / 1e9, 2),
            "hbm_gbs": round(2 * mig_bytes / (mig_ms / 1e3) / 1e9, 2),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": roofline_kernel,
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": _measured_traffic(w.name),
            "algorithmic_bytes_per_launch": int(mean_bytes),
            "mean_launch_us": round(mean_dur_s * 1e6, 2),
            "launch_us_per_partition": [round(float(x) * 1e3, 2) for x in dur_ms.mean(axis=0)],
            "launch_timing": "mean launch = HIP events around each step's back-to-back partial launches / "
                             "partitions (scrubbed steps); per-partition split from events around every launch",
        },
    }
    if args.copy_calibration:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = n
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        line["cpu_baseline"] = _cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
