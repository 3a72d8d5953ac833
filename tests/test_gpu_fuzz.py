"""Seeded random-shape fuzz of the partial, merge and fused calls against the fp64 oracle (GPU).

Each case draws a workload shape (1-400 sequences, GQA groups 1-16, 1-6 ranges per sequence, some
sequences with overlapping or gapped ranges), lengths from one of four mixes (many short; few long;
log-normal with a heavy tail; one long among many tiny) and random launch hints (waves, chunks, plan,
dispatch order, no workspace, no range hints), runs every partition's call, the merge and the fused
call, and checks them against the oracle's partials and their merge (which, unlike unsplit
attention, also covers overlapping ranges).  On one random partition it also runs, each with some
probability: the head-split call over a random kv-head range (its rows against the oracle, every
other row untouched), the no-allocation call (bit for bit the workspace call's result when that ran
with a workspace, else against the oracle; a plan beyond the static scratch must be refused), the
block migration of that partition (bit for bit the oracle's copy), and the fused call with 0-8
random side copies (bit for bit the fused call with the chunked launch; every copy byte for byte).  By default a few cases run;
``BANA_FUZZ_SECONDS=<s>`` runs cases for that long instead (``BANA_FUZZ_SEED`` picks the stream).
"""

import math
import os
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2510_13223_amd import bana, workloads as W
from paper_2510_13223_amd.runner import DeviceWorkload

from test_gpu_parity import _check_lse, _check_out, _log, _migrate_and_check

pytestmark = pytest.mark.gpu


def _case(seed, case):
    rng = np.random.default_rng(777000 + seed * 100000 + case)
    kind = int(rng.integers(0, 4))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    Hq = Hkv * int(rng.choice([1, 2, 3, 4, 5, 8, 16]))
    n_parts = int(rng.integers(1, 7))
    if kind == 0:  # many short sequences
        B = int(rng.integers(1, 400))
        lens = rng.integers(1, 300, size=B)
    elif kind == 1:  # few long ones
        B = int(rng.integers(1, 6))
        lens = rng.integers(1, 20000, size=B)
    elif kind == 2:  # log-normal with a heavy tail
        B = int(rng.integers(2, 200))
        lens = np.clip(np.rint(np.exp(rng.normal(np.log(200), 1.3, size=B))), 1, 12000)
    else:  # one long among many tiny
        B = int(rng.integers(2, 300))
        lens = rng.integers(1, 40, size=B)
        lens[int(rng.integers(0, B))] = int(rng.integers(2000, 16000))
    lens = [int(x) for x in lens]
    ranges = [[] for _ in range(n_parts)]
    for L in lens:
        if rng.random() < 0.15:  # independent ranges: overlapping or leaving gaps
            for p in range(n_parts):
                a = int(rng.integers(0, L + 1))
                ranges[p].append((a, int(rng.integers(a, L + 1))))
        else:
            cuts = np.sort(rng.integers(0, L + 1, size=n_parts - 1)).tolist()
            edges = [0] + cuts + [L]
            for p in range(n_parts):
                ranges[p].append((edges[p], edges[p + 1]))
    kw = dict(waves_hint=int(rng.choice([0, 0, 0, 1, 2, 4, 8])), chunks_hint=int(rng.choice([0, 0, 0, 1, 2, 3, 7])),
              plan_hint=int(rng.choice([0, 0, 1, 2])), order_hints=bool(rng.integers(0, 2)),
              use_workspace=bool(rng.integers(0, 5) > 0), range_hints=bool(rng.integers(0, 5) > 0))
    w = W.make_custom(880000 + case, B, Hq, Hkv, lens, ranges, q_scale=1 / math.sqrt(128))
    return w, kw, f"fuzz {seed}:{case} kind={kind} B={B} Hq={Hq} Hkv={Hkv} parts={n_parts} maxL={max(lens)} {kw}"


def _extras(w, kw, dw, ro, rl, rng):
    B, Hq, Hkv = w.batch, w.num_q_heads, w.num_kv_heads
    G = Hq // Hkv
    p = int(rng.integers(0, w.n_parts))
    if Hkv > 1 and rng.random() < 0.5:
        g0 = int(rng.integers(0, Hkv))
        g1 = int(rng.integers(g0 + 1, Hkv + 1))
        sub = bana.head_range_dims(dw.dims[p], g0, g1)
        ws = torch.empty(max(256, bana.bana_decode_attn_workspace_bytes(sub)), dtype=torch.uint8, device="cuda")
        o = torch.full((B, Hq, 128), float("nan"), device="cuda")
        l = torch.full((B, Hq), float("nan"), device="cuda")
        bana.bana_decode_attn_heads(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin[p],
                                    dw.kv_end[p], g0, g1, o, l, workspace=ws, dims=dw.dims[p])
        o, l = o.cpu().numpy(), l.cpu().numpy()
        hs = slice(g0 * G, g1 * G)
        fin = np.isfinite(rl[p][:, hs])
        _check_out(o[:, hs][fin], ro[p][:, hs][fin], "head range out")
        assert np.all(o[:, hs][~fin] == 0.0)
        _check_lse(l[:, hs], rl[p][:, hs], "head range lse")
        assert np.all(np.isnan(o[:, :g0 * G])) and np.all(np.isnan(o[:, g1 * G:]))
    if rng.random() < 0.5:
        o = torch.full((B, Hq, 128), float("nan"), device="cuda")
        l = torch.full((B, Hq), float("nan"), device="cuda")
        try:
            bana.bana_decode_attn_partial_noalloc(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens,
                                                  dw.kv_begin[p], dw.kv_end[p], o, l, dims=dw.dims[p])
        except bana.BanaError as e:
            assert e.status == bana.BANA_ERR_UNSUPPORTED
            assert bana.bana_decode_attn_workspace_bytes(dw.dims[p]) > bana.STATIC_SCRATCH_BYTES
        else:
            torch.cuda.synchronize()
            if kw["use_workspace"]:
                assert torch.equal(o.view(torch.int32), dw.out_partials[p].view(torch.int32))
                assert torch.equal(l.view(torch.int32), dw.lses[p].view(torch.int32))
            else:
                on, ln = o.cpu().numpy(), l.cpu().numpy()
                _check_out(on[np.isfinite(rl[p])], ro[p][np.isfinite(rl[p])], "noalloc out_partial")
                _check_lse(ln, rl[p], "noalloc lse")
    if rng.random() < 0.3:
        _migrate_and_check(w, p, seed=int(rng.integers(0, 1 << 30)), hint=bool(rng.integers(0, 2)))
    if rng.random() < 0.3:
        _fused_copies(w, kw, dw, rng)


def _fused_copies(w, kw, dw, rng):
    """The fused call with 0-8 random side copies equals the fused call with the chunked launch bit for
    bit, and every copy arrives byte for byte."""
    B, Hq = w.batch, w.num_q_heads
    fd = bana.bana_dims.from_buffer_copy(dw.fused_dims)
    fd.plan_hint = 1
    ws = None
    if kw["use_workspace"]:
        ws = torch.empty(max(256, bana.bana_decode_attn_workspace_bytes(fd)), dtype=torch.uint8, device="cuda")
    ref_o = torch.empty((B, Hq, 128), device="cuda")
    ref_l = torch.empty((B, Hq), device="cuda")
    bana.bana_decode_attn_fused(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin, dw.kv_end,
                                ref_o, ref_l, workspace=ws, dims=fd)
    g = torch.Generator().manual_seed(int(rng.integers(0, 1 << 30)))
    copies, checks = [], []
    for _ in range(int(rng.integers(0, 9))):
        n = 4 * int(rng.integers(0, 1 << 17))  # int32 words: 0 to 2 MiB, a multiple of 16 bytes
        kind = int(rng.integers(0, 3))
        src = torch.randint(-2**31, 2**31 - 1, (n,), dtype=torch.int32, generator=g)
        if n == 0:
            src, dst = src.cuda(), torch.empty(0, dtype=torch.int32, device="cuda")
        elif kind == 0:  # pinned host -> device
            src, dst = src.pin_memory(), torch.zeros(n, dtype=torch.int32, device="cuda")
        elif kind == 1:  # device -> pinned host
            src, dst = src.cuda(), torch.zeros(n, dtype=torch.int32).pin_memory()
        else:  # device -> device
            src, dst = src.cuda(), torch.zeros(n, dtype=torch.int32, device="cuda")
        copies.append((dst, src))
        checks.append((dst, src))
    o = torch.full((B, Hq, 128), float("nan"), device="cuda")
    l = torch.full((B, Hq), float("nan"), device="cuda")
    bana.bana_decode_attn_fused_copies(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin,
                                       dw.kv_end, o, l, copies=copies, workspace=ws, dims=dw.fused_dims)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int32), ref_o.view(torch.int32))
    assert torch.equal(l.view(torch.int32), ref_l.view(torch.int32))
    for dst, src in checks:
        assert torch.equal(dst.cpu(), src.cpu())


def _check(w, kw, extras_rng=None):
    dw = DeviceWorkload(w, **kw)
    op, lp, out, lse_out = dw.results()
    ro, rl = oracle.workload_partials(w)
    for p in range(w.n_parts):
        _check_out(op[p][np.isfinite(rl[p])], ro[p][np.isfinite(rl[p])], f"part {p} out_partial")
        assert np.all(op[p][np.isneginf(rl[p])] == 0.0), "empty partition must give out_partial = 0"
        _check_lse(lp[p], rl[p], f"part {p}")
    mo, ml = oracle.merge(ro, rl)
    fin = np.isfinite(ml)
    _check_out(out[fin], mo[fin], "merged out")
    assert np.all(out[~fin] == 0.0)
    _check_lse(lse_out, ml, "merged lse")
    fo, fl = dw.fused_results()
    _check_out(fo[fin], mo[fin], "fused out")
    _check_lse(fl, ml, "fused lse")
    if extras_rng is not None:
        _extras(w, kw, dw, ro, rl, extras_rng)


def test_random_shape_fuzz():
    seed = int(os.environ.get("BANA_FUZZ_SEED", "0"))
    seconds = float(os.environ.get("BANA_FUZZ_SECONDS", "0"))
    t_end = time.time() + seconds
    case = 0
    while case < 16 or time.time() < t_end:
        w, kw, tag = _case(seed, case)
        _log(tag)
        _check(w, kw, np.random.default_rng(555000 + seed * 100000 + case))
        torch.cuda.empty_cache()
        case += 1
    _log(f"fuzz: {case} cases passed")
