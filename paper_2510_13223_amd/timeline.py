"""Wavefront timelines of the attention launches (the BANA_WAVE_TIMELINE measurement build).

    python -m paper_2510_13223_amd.timeline [--md PATH] [--reps N] workload:partition ...

Runs each listed partition call once per repetition, after a cache scrub (512 MiB written, then read
back), with ``libbana_timeline.so`` -- the product kernels plus one clock reading per wavefront at
entry, schedule ready, first KV block consumed and exit -- and summarises when the wavefronts start,
get their first block and finish, overall and by dispatch quartile (slot order: workgroups are
dispatched in index order).  Orchestration and statistics only; the kernels are the library's.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import sys
from typing import Dict, List

import numpy as np
import torch

from . import bana
from . import workloads as W
from .runner import DeviceWorkload

TICK_US = 0.01  # the clock runs at 100 MHz
UNSET = np.uint64(0xFFFFFFFFFFFFFFFF)


def summarize(t: np.ndarray) -> Dict[str, float]:
    """Statistics of one launch's slots (uint64 [n, 4]); times in us from the earliest entry."""
    used = t[:, 0] != UNSET
    t = t[used]
    n = len(t)
    if n == 0:
        raise ValueError("no wavefront recorded an entry")
    t0 = t[:, 0].min()
    rel = lambda col: (t[:, col] - t0).astype(np.float64) * TICK_US
    entry, ready, exit_ = rel(0), rel(1), rel(3)
    has_first = t[:, 2] != UNSET
    first = np.where(has_first, (t[:, 2] - np.minimum(t[:, 2], t0)).astype(np.float64) * TICK_US, np.nan)
    done = t[:, 3] != UNSET
    q = lambda x, p: float(np.nanpercentile(x, p)) if np.isfinite(x).any() else float("nan")
    s = {
        "waves": n,
        "span_us": float(exit_[done].max()) if done.any() else float("nan"),
        "entry_spread_us": float(entry.max()),
        "ready_after_entry_p50_us": q(ready - entry, 50),
        "first_block_after_entry_p10_us": q(first - entry, 10),
        "first_block_after_entry_p50_us": q(first - entry, 50),
        "first_block_after_entry_p90_us": q(first - entry, 90),
        "exit_p10_us": q(exit_[done], 10),
        "exit_p50_us": q(exit_[done], 50),
        "exit_p90_us": q(exit_[done], 90),
    }
    quarters = np.array_split(np.arange(n), 4)  # slots in dispatch order
    for i, idx in enumerate(quarters):
        s[f"q{i}_first_block_p50_us"] = q((first - entry)[idx], 50)
        s[f"q{i}_exit_p50_us"] = q(np.where(done[idx], exit_[idx], np.nan), 50)
    return s


def run(cases: List[str], reps: int) -> List[Dict]:
    side = bana.load(bana.TIMELINE_LIB_PATH)
    dev = torch.device("cuda:0")
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    sink = torch.empty(2048, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream(device=dev)
    h = ctypes.c_void_p(stream.cuda_stream)
    by_workload: Dict[str, List[int]] = {}
    for c in cases:
        name, part = c.split(":")
        by_workload.setdefault(name, []).append(int(part))
    rows = []
    for name, parts in by_workload.items():
        w = W.make_config(name, 0)
        dw = DeviceWorkload(w, device=dev)
        for p in parts:
            runs = []
            for r in range(reps):
                with torch.cuda.stream(stream):
                    scrub.fill_(r & 255)
                    bana.bana_debug_stream_read(scrub, sink, stream=stream)
                bana.bana_debug_wave_timeline_clear(stream, library=side)
                st = side.bana_decode_attn_partial(*dw._partial_args[p], h)
                if st != bana.BANA_OK:
                    raise bana.BanaError(st, "bana_decode_attn_partial (timeline build)")
                t = bana.bana_debug_wave_timeline_read(bana.TIMELINE_SLOTS, stream, library=side)
                runs.append(summarize(t))
            med = {k: float(np.median([x[k] for x in runs])) for k in runs[0]}
            med.update(workload=name, partition=p, reps=reps)
            print(json.dumps(med), flush=True)
            rows.append(med)
        del dw
        torch.cuda.empty_cache()
    return rows


def markdown(rows: List[Dict], command: str) -> str:
    out = ["# Wavefront timelines of the partial-attention launches", "",
           "Command (repository root on one MI355X):", "", f"    {command}", "",
           "One call per repetition after a cache scrub, with the timeline build of the library (same kernels; "
           "each wavefront's lane 0 stores clock readings at entry, schedule ready, first KV block consumed and "
           "exit). Times in us from the launch's earliest wavefront entry, medians over the repetitions. "
           "The readings themselves (one store or atomic per mark) lengthen each launch by a few percent.", "",
           "| Call | Waves | Span | Entry spread | Ready (p50) | First block p10 / p50 / p90 | "
           "Exit p10 / p50 / p90 |",
           "|:--|--:|--:|--:|--:|--:|--:|"]
    for r in rows:
        out.append(f"| {r['workload']} partition {r['partition']} | {int(r['waves'])} | {r['span_us']:.1f} | "
                   f"{r['entry_spread_us']:.1f} | {r['ready_after_entry_p50_us']:.2f} | "
                   f"{r['first_block_after_entry_p10_us']:.1f} / {r['first_block_after_entry_p50_us']:.1f} / "
                   f"{r['first_block_after_entry_p90_us']:.1f} | {r['exit_p10_us']:.1f} / {r['exit_p50_us']:.1f} / "
                   f"{r['exit_p90_us']:.1f} |")
    out += ["", "By dispatch quarter (wavefront slots in index order; first block after entry, p50 / exit, p50):", "",
            "| Call | 1st quarter | 2nd | 3rd | 4th |", "|:--|--:|--:|--:|--:|"]
    for r in rows:
        cells = [f"{r[f'q{i}_first_block_p50_us']:.1f} / {r[f'q{i}_exit_p50_us']:.1f}" for i in range(4)]
        out.append(f"| {r['workload']} partition {r['partition']} | " + " | ".join(cells) + " |")
    return "\n".join(out) + "\n"


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("cases", nargs="+", help="workload:partition, e.g. fine:0")
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--md", default=None, help="write a markdown summary here")
    args = ap.parse_args(argv)
    rows = run(args.cases, args.reps)
    if args.md:
        cmd = "python -u -m paper_2510_13223_amd.timeline " + " ".join(
            (["--reps", str(args.reps)] if args.reps != 3 else []) + ["--md", args.md] + args.cases)
        with open(args.md, "w") as f:
            f.write(markdown(rows, cmd))


if __name__ == "__main__":
    main(sys.argv[1:])
