"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Tolerances (fp32 outputs of bf16-in / fp32-accumulate kernels), over each
config's whole output tensor: max-abs error <= 2e-3 and relative L2 error
<= 1e-3 for every partition's out_partial and for the merged out; |dlse| <=
1e-4 on finite entries, and -inf exactly where a partition is empty.
Indexing and coverage are checked bit-exactly: the exported K rows equal the
oracle's, zero keys give round(exp(lse)) == range length, and a dominant key
returns its value row exactly.
"""

import ctypes
import dataclasses
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2510_13223_amd import bana, workloads as W
from paper_2510_13223_amd.runner import DeviceWorkload

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3
LSE_ABS = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bana.lib()  # raises if the HIP library is missing: there is no fallback
    yield


_CACHE = {}


def _workload(name, seed=0):
    key = (name, seed)
    if key not in _CACHE:
        if len(_CACHE) >= 2:
            _CACHE.clear()
        _CACHE[key] = W.make_config(name, seed)
    return _CACHE[key]


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _check_out(gpu, ref, what):
    gpu = gpu.astype(np.float64)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    diff = gpu - ref
    max_abs = float(np.max(np.abs(diff))) if diff.size else 0.0
    rel = float(np.linalg.norm(diff) / max(np.linalg.norm(ref), 1e-300)) if diff.size else 0.0
    assert max_abs <= MAX_ABS, f"{what}: max-abs {max_abs:.3e}"
    assert rel <= REL_L2, f"{what}: rel-L2 {rel:.3e}"
    return max_abs, rel


def _check_lse(gpu, ref, what):
    gpu = gpu.astype(np.float64)
    ninf = np.isneginf(ref)
    assert np.array_equal(np.isneginf(gpu), ninf), f"{what}: -inf pattern differs"
    fin = ~ninf
    assert np.all(np.isfinite(gpu[fin])), f"{what}: non-finite lse"
    err = float(np.max(np.abs(gpu[fin] - ref[fin]))) if fin.any() else 0.0
    assert err <= LSE_ABS, f"{what}: lse max-abs {err:.3e}"
    return err


def _full_parity(w, **kw):
    _log(f"[parity] {w.name} seed={w.seed} B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} parts={w.n_parts} {kw}")
    dw = DeviceWorkload(w, **kw)
    op, lp, out, lse_out = dw.results()
    ro, rl = oracle.workload_partials(w)
    for p in range(w.n_parts):
        _check_out(op[p][np.isfinite(rl[p])], ro[p][np.isfinite(rl[p])], f"{w.name} part {p} out_partial")
        assert np.all(op[p][np.isneginf(rl[p])] == 0.0), "empty partition must give out_partial = 0"
        _check_lse(lp[p], rl[p], f"{w.name} part {p}")
    mo, ml = oracle.merge(ro, rl)
    uo, ul = oracle.workload_unsplit(w)
    np.testing.assert_allclose(mo, uo, rtol=0, atol=1e-10)  # oracle's own merge == unsplit
    stats = _check_out(out, uo, f"{w.name} merged out")
    _check_lse(lse_out, ul, f"{w.name} merged lse")
    fo, fl = dw.fused_results()
    fstats = _check_out(fo, mo, f"{w.name} fused out")
    _check_lse(fl, ml, f"{w.name} fused lse")
    _log(f"  merged max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e}; fused max-abs {fstats[0]:.2e} rel-L2 {fstats[1]:.2e}")
    return dw


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_parity(seed):
    _full_parity(_workload("tiny", seed))


@pytest.mark.parametrize("name", ["llama3_8b", "long", "mixed", "fine", "mha13b"])
def test_config_parity(name):
    _full_parity(_workload(name))


@pytest.mark.parametrize("waves,chunks", [(1, 1), (2, 3), (4, 1), (8, 2), (1, 7), (8, 16)])
def test_launch_plans_agree(waves, chunks):
    """Every launch shape (waves per workgroup, chunks per range) meets the same bar."""
    w = _workload("tiny", 1)
    _full_parity(w, waves_hint=waves, chunks_hint=chunks)


def test_without_workspace_runs_unsplit():
    w = _workload("tiny", 2)
    _full_parity(w, use_workspace=False, range_hints=False)
    _full_parity(w, use_workspace=False, plan_hint=2)  # the balanced launch needs workspace: runs unsplit


@pytest.mark.parametrize("seed,plan", [(0, 1), (1, 1), (0, 2), (1, 2), (2, 2)])
def test_forced_launch_shapes(seed, plan):
    """The chunked (1) and the balanced (2) launch on the tiny workload; balanced there has fewer
    blocks than wavefronts (one block per wavefront, most wavefronts idle)."""
    _full_parity(_workload("tiny", seed), plan_hint=plan)


@pytest.mark.parametrize("name", ["long", "mixed"])
def test_chunked_launch_on_uneven_workloads(name):
    """long and mixed pick the balanced launch by themselves; the chunked one must still meet the bar."""
    _full_parity(_workload(name), plan_hint=1)


@pytest.mark.parametrize("B,every", [(64, 13), (300, 97)])
def test_balanced_launch_with_runs_of_empty_sequences(B, every):
    """Only every `every`-th sequence has tokens in partition 0 (runs of empty sequences between
    pieces), one sequence is long, range ends are ragged.  With 64 sequences the balanced launch runs
    (one sequence per lane of its schedule); with 300 the hint falls back to the chunked launch."""
    rng = np.random.default_rng(B)
    lens = rng.integers(1, 400, size=B)
    lens[B // 2] = 5000
    ranges = [[], []]
    for b in range(B):
        L = int(lens[b])
        cut = int(rng.integers(1, L + 1)) if (b % every == 3 or b == B // 2) else 0
        ranges[0].append((0, cut))
        ranges[1].append((cut, L))
    w = W.make_custom(21, B, 8, 2, lens, ranges, q_scale=1 / math.sqrt(128))
    _full_parity(w, plan_hint=2)


@pytest.mark.parametrize("name,plan", [("tiny", 0), ("tiny", 2), ("mixed", 0)])
def test_run_to_run_bit_determinism(name, plan):
    w = _workload(name, 0)
    dw = DeviceWorkload(w, plan_hint=plan)
    a = dw.results() + dw.fused_results()
    dw.step()
    dw.fused(__import__("ctypes").c_void_p(torch.cuda.current_stream().cuda_stream))
    b = dw.results() + dw.fused_results()
    for x, y in zip(a, b):
        assert np.array_equal(x, y, equal_nan=True)


@pytest.mark.parametrize("plan", [0, 2])
def test_physical_block_permutation_bit_identical(plan):
    w = _workload("tiny", 0)
    a = DeviceWorkload(w, plan_hint=plan).results()
    b = DeviceWorkload(W.permute_physical(w, 3), plan_hint=plan).results()
    for x, y in zip(a, b):
        assert np.array_equal(x, y, equal_nan=True)


def test_debug_rows_bit_exact():
    for name in ("tiny", "mixed"):
        w = _workload(name)
        _log(f"[rows] {name}")
        dw = DeviceWorkload(w)
        for p in range(w.n_parts):
            rows = torch.empty((w.batch, w.num_kv_heads, w.max_blocks_per_seq * 16), dtype=torch.int64, device="cuda")
            bana.bana_debug_kv_rows(dw.block_table, dw.kv_begin[p], dw.kv_end[p], w.num_blocks, w.num_kv_heads, rows)
            ref = oracle.kv_rows(w.block_table, w.num_blocks, w.num_kv_heads, w.kv_begin[p], w.kv_end[p])
            np.testing.assert_array_equal(rows.cpu().numpy(), ref)


def _aim_dominant(w, part, seed):
    """Per (b, g): one key in the partition aimed along head g*G's query so it wins by > 110."""
    rng = np.random.default_rng(seed)
    G = w.group
    chosen = {}
    for b in range(w.batch):
        t0, t1 = int(w.kv_begin[part, b]), int(w.kv_end[part, b])
        if t1 <= t0:
            continue
        for g in range(w.num_kv_heads):
            t = int(rng.integers(t0, t1))
            qf = W.bf16_bits_to_f32(w.q[b, g * G]).astype(np.float32)
            scale = np.float32(300.0 / float(qf @ qf))
            blk = w.block_table[b, t // 16]
            W.set_k_row(w.k_cache, blk, g, t % 16, W.f32_to_bf16_bits(qf * scale))
            chosen[(b, g)] = t
    return chosen


@pytest.mark.parametrize("waves,chunks,plan", [(0, 0, 0), (1, 1, 0), (8, 3, 0), (0, 0, 2)])
def test_dominant_key_returns_value_row_exactly(waves, chunks, plan):
    w = W.make_config("tiny", 3)
    chosen = {part: _aim_dominant(w, part, 10 + part) for part in range(w.n_parts)}
    _log(f"[dominant] waves={waves} chunks={chunks} plan={plan}")
    op, lp, _, _ = DeviceWorkload(w, waves_hint=waves, chunks_hint=chunks, plan_hint=plan).results()
    for part, picks in chosen.items():
        for (b, g), t in picks.items():
            blk = w.block_table[b, t // 16]
            v = W.bf16_bits_to_f32(w.v_cache[blk, g, :, t % 16])
            assert np.array_equal(op[part, b, g * w.group], v), (part, b, g, t)


def test_zero_keys_pin_coverage_counts():
    for name, kw in (("tiny", {}), ("tiny", dict(waves_hint=4, chunks_hint=5)), ("tiny", dict(plan_hint=2)),
                     ("mixed", {})):
        w = W.make_config(name, 0)
        finite = np.isfinite(W.bf16_bits_to_f32(w.k_cache))
        w.k_cache[finite] = 0
        _log(f"[coverage] {name} {kw}")
        dw = DeviceWorkload(w, **kw)
        op, lp, out, lse_out = dw.results()
        n = (w.kv_end - w.kv_begin).astype(np.float64)[:, :, None].repeat(w.num_q_heads, 2)
        live = n > 0
        assert np.array_equal(np.rint(np.exp(lp[live].astype(np.float64))), n[live])
        assert np.all(np.isneginf(lp[~live]))
        L = w.seq_lens.astype(np.float64)[:, None].repeat(w.num_q_heads, 1)
        assert np.array_equal(np.rint(np.exp(lse_out.astype(np.float64))), L)
        fo, fl = dw.fused_results()
        assert np.array_equal(np.rint(np.exp(fl.astype(np.float64))), L)


def test_single_key_and_non_aligned_ranges():
    lens = [37, 64, 300, 17, 1]
    ranges = [
        [(17, 18), (63, 64), (5, 299), (0, 17), (0, 0)],
        [(0, 17), (0, 63), (299, 300), (17, 17), (0, 1)],
        [(18, 37), (0, 0), (0, 5), (0, 0), (1, 1)],
    ]
    w = W.make_custom(4, 5, 8, 2, lens, ranges, q_scale=1 / math.sqrt(128))
    dw = _full_parity(w)
    op, _, _, _ = dw.results()
    for part, b, t in ((0, 0, 17), (0, 1, 63), (1, 2, 299), (1, 4, 0)):
        for h in range(8):
            blk = w.block_table[b, t // 16]
            v = W.bf16_bits_to_f32(w.v_cache[blk, h // 4, :, t % 16])
            assert np.array_equal(op[part, b, h], v)


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 4), (32, 2), (12, 4)])
def test_other_gqa_groups(Hq, Hkv):
    rng = np.random.default_rng(Hq * 100 + Hkv)
    lens = rng.integers(1, 700, size=6)
    ranges = [[], []]
    for L in lens:
        cut = int(rng.integers(0, L + 1))
        ranges[0].append((0, cut))
        ranges[1].append((cut, int(L)))
    w = W.make_custom(11, 6, Hq, Hkv, lens, ranges, q_scale=1 / math.sqrt(128))
    _full_parity(w)


def test_scaled_query_reading_llama_shape():
    """Alternative reading with a 1/sqrt(128) softmax scale folded into q (config-2 shape, 8 sequences)."""
    lens = [4096] * 8
    ranges = [[(0, 179 * 16)] * 8, [(179 * 16, 4096)] * 8]
    w = W.make_custom(2, 8, 32, 8, lens, ranges, max_blocks_per_seq=256, q_scale=1 / math.sqrt(128))
    _full_parity(w)


def _fused_vs_oracle(w, **kw):
    dw = DeviceWorkload(w, **kw)
    fo, fl = dw.fused_results()
    ro, rl = oracle.workload_partials(w)
    mo, ml = oracle.merge(ro, rl)
    fin = np.isfinite(ml)
    _check_out(fo[fin], mo[fin], "fused out")
    assert np.all(fo[~fin] == 0.0)
    _check_lse(fl, ml, "fused lse")


def test_fused_overlapping_empty_and_many_ranges():
    """Overlapping ranges count twice (as merging their partials would), empty ranges add nothing,
    and up to 64 ranges per sequence are accepted."""
    rng = np.random.default_rng(21)
    lens = [700, 333, 1, 64, 0 + 17]
    P = 64
    ranges = []
    for p in range(P):
        row = []
        for L in lens:
            a, b = sorted(int(x) for x in rng.integers(0, L + 1, size=2))
            row.append((a, b) if p % 7 else (a, a))  # every 7th range empty
        ranges.append(row)
    w = W.make_custom(5, len(lens), 8, 2, lens, ranges, q_scale=1 / math.sqrt(128))
    _log("[fused] 64 overlapping ranges")
    for kw in ({}, dict(waves_hint=8, chunks_hint=3), dict(waves_hint=1, chunks_hint=1), dict(plan_hint=2)):
        _fused_vs_oracle(w, **kw)


def test_fused_dominant_key_and_all_empty():
    w = W.make_config("tiny", 3)
    chosen = _aim_dominant(w, 1, 11)
    # tokens of partition 1 listed twice: the dominant key still wins alone
    w2 = dataclasses.replace(w, kv_begin=np.concatenate([w.kv_begin, w.kv_begin[1:]]),
                               kv_end=np.concatenate([w.kv_end, w.kv_end[1:]]))
    fo, fl = DeviceWorkload(w2).fused_results()
    for (b, g), t in chosen.items():
        blk = w.block_table[b, t // 16]
        assert np.array_equal(fo[b, g * w.group], W.bf16_bits_to_f32(w.v_cache[blk, g, :, t % 16]))
    empty = dataclasses.replace(w, kv_begin=w.kv_end.copy())
    for plan in (0, 2):  # chunked, balanced (no blocks at all: every wavefront idle, every row empty)
        dw = DeviceWorkload(empty, plan_hint=plan)
        op, lp, out, lse_out = dw.results()
        fo, fl = dw.fused_results()
        assert np.all(fo == 0.0) and np.all(np.isneginf(fl))
        assert np.all(out == 0.0) and np.all(np.isneginf(lse_out))
        assert np.all(op == 0.0) and np.all(np.isneginf(lp))


# (parts, batch, heads): the few-part kernel, and the many-part kernel with 1, 2, 4 and 8 thread
# groups per row, including more than 32 parts per group (several lse rounds per lane).
# Many rows take one thread group per row, streaming one part per round: up to 32 parts (one lse
# round per lane), more than 32, and a row count that leaves the last workgroup partly filled.
@pytest.mark.parametrize("n,B,Hq", [(2, 7, 8), (4, 3, 8), (5, 7, 8), (9, 7, 8), (20, 3, 8), (70, 2, 8),
                                    (300, 2, 8), (40, 128, 32), (6, 1, 1), (16, 128, 32), (12, 4099, 1)])
def test_merge_matches_oracle_merge(n, B, Hq):
    rng = np.random.default_rng(n * 1000 + B)
    outs = rng.standard_normal((n, B, Hq, 128)).astype(np.float32)
    lses = (rng.standard_normal((n, B, Hq)) * 20).astype(np.float32)
    lses[rng.random((n, B, Hq)) < 0.3] = -np.inf
    lses[:, 0, 0] = -np.inf  # an all-empty row
    if B * Hq > 1:
        lses[: n // 2, -1, -1] = -np.inf  # a row whose first half of parts (whole thread groups) is empty
        lses[n // 2:, -1, -1] = 80.0 * np.arange(n - n // 2)  # live parts far apart: most weights underflow
    outs[np.isneginf(lses)] = np.nan  # rows of empty parts are never read
    d_out = torch.empty((B, Hq, 128), dtype=torch.float32, device="cuda")
    d_lse = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    bana.bana_merge_partials(torch.from_numpy(outs).cuda(), torch.from_numpy(lses).cuda(), d_out, d_lse)
    ro, rl = oracle.merge(outs.astype(np.float64), lses.astype(np.float64))
    torch.cuda.synchronize()
    np.testing.assert_allclose(d_out.cpu().numpy(), ro, rtol=0, atol=1e-5)
    got = d_lse.cpu().numpy()
    assert np.array_equal(np.isneginf(got), np.isneginf(rl))
    np.testing.assert_allclose(got[np.isfinite(rl)], rl[np.isfinite(rl)], rtol=0, atol=1e-5)
    assert np.all(d_out.cpu().numpy()[0, 0] == 0)


def test_non_default_stream_and_binding_checks():
    w = _workload("tiny", 0)
    ref = DeviceWorkload(w).results()
    dw = DeviceWorkload(w)
    dw.out.zero_()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        dw.step(s)
    s.synchronize()
    got = dw.results()
    for x, y in zip(ref, got):
        assert np.array_equal(x, y, equal_nan=True)
    with pytest.raises(TypeError):
        bana.bana_decode_attn_partial(dw.q.float(), dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens,
                                      dw.kv_begin[0], dw.kv_end[0], dw.out_partials[0], dw.lses[0])
    # caller-built dims that do not describe the tensors are refused before any launch
    bad = bana.make_dims(w.batch, w.num_q_heads, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks * 4)
    with pytest.raises(ValueError):
        bana.bana_decode_attn_partial(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin[0],
                                      dw.kv_end[0], dw.out_partials[0], dw.lses[0], dims=bad)
    with pytest.raises(ValueError):
        bana.bana_decode_attn_fused(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin,
                                    dw.kv_end, dw.fused_out, dw.fused_lse, dims=bad)
    # host memory where device memory is expected is refused before any launch
    with pytest.raises(ValueError):
        bana.bana_decode_attn_partial(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin[0],
                                      dw.kv_end[0], dw.out_partials[0].cpu(), dw.lses[0])
    with pytest.raises(ValueError):
        bana.bana_decode_attn_partial(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin[0],
                                      dw.kv_end[0], dw.out_partials[0], dw.lses[0],
                                      workspace=torch.empty(1 << 20, dtype=torch.uint8))


@pytest.mark.parametrize("name,part", [("tiny", 0), ("tiny", 1), ("llama3_8b", 1), ("mixed", 1)])
def test_migration_bit_exact_and_attention_unchanged(name, part):
    """bana_migrate_kv_blocks equals the oracle's block copy bit for bit, leaves other destination
    blocks untouched, and attention over the migrated partition is bit-identical afterwards."""
    w = _workload(name)
    m = W.make_migration(w, part, seed=4)
    _log(f"[migrate] {name} part {part}: {int(np.sum(m.blk_end - m.blk_begin))} blocks")
    dw = DeviceWorkload(w)
    dk = torch.from_numpy(m.dst_k.view(np.int16)).view(torch.bfloat16).cuda()
    dv = torch.from_numpy(m.dst_v.view(np.int16)).view(torch.bfloat16).cuda()
    dt = torch.from_numpy(m.dst_table).cuda()
    bb = torch.from_numpy(m.blk_begin).cuda()
    be = torch.from_numpy(m.blk_end).cuda()
    bana.bana_migrate_kv_blocks(dw.k_cache, dw.v_cache, dw.block_table, dk, dv, dt, bb, be)
    ek, ev = oracle.migrate(w.k_cache, w.v_cache, w.block_table, m.dst_k, m.dst_v, m.dst_table, m.blk_begin,
                            m.blk_end)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dk.cpu().view(torch.int16).numpy().view(np.uint16), ek)
    np.testing.assert_array_equal(dv.cpu().view(torch.int16).numpy().view(np.uint16), ev)
    # attention over the partition through the destination pool and table
    B, Hq = w.batch, w.num_q_heads
    o1 = torch.empty((B, Hq, 128), dtype=torch.float32, device="cuda")
    l1 = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    d2 = bana.bana_dims.from_buffer_copy(dw.dims[part])  # the same plan, over the destination pool
    d2.num_blocks = m.num_blocks
    bana.bana_decode_attn_partial(dw.q, dk, dv, dt, dw.seq_lens, dw.kv_begin[part], dw.kv_end[part], o1, l1,
                                  workspace=dw.workspace, dims=d2)
    op, lp, _, _ = dw.results()
    assert np.array_equal(o1.cpu().numpy(), op[part], equal_nan=True)
    assert np.array_equal(l1.cpu().numpy(), lp[part], equal_nan=True)


@pytest.mark.parametrize("name,part,split", [("tiny", 0, 1), ("llama3_8b", 0, 3), ("long", 0, 5), ("mixed", 1, 4)])
def test_head_split_equals_the_call_on_a_cache_of_those_heads(name, part, split):
    """Head partitions (the literal head-dimension split): a kv-head range call gives, bit for bit, what
    the partial call gives on a cache holding only those heads (the device they migrate to), writes
    only its own rows, and complementary ranges together match the oracle; with a fixed launch shape
    they concatenate to the unsplit call bit for bit."""
    w = _workload(name)
    dw = DeviceWorkload(w)
    B, Hq, Hkv, G = w.batch, w.num_q_heads, w.num_kv_heads, w.group
    out = torch.full((B, Hq, 128), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device="cuda")
    begin, end = dw.kv_begin[part], dw.kv_end[part]
    for g0, g1 in ((0, split), (split, Hkv)):
        _log(f"[heads] {name} part {part} kv heads [{g0}, {g1})")
        sub = bana.head_range_dims(dw.dims[part], g0, g1)
        ws = torch.empty(max(256, bana.bana_decode_attn_workspace_bytes(sub)), dtype=torch.uint8, device="cuda")
        bana.bana_decode_attn_heads(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, begin, end, g0, g1,
                                    out, lse, workspace=ws, dims=dw.dims[part])
        if g0 == 0:
            o = out.cpu().numpy()
            assert np.all(np.isnan(o[:, g1 * G:])) and np.all(np.isnan(lse.cpu().numpy()[:, g1 * G:]))
        q_s = dw.q[:, g0 * G:g1 * G].contiguous()
        k_s = dw.k_cache[:, g0:g1].contiguous()
        v_s = dw.v_cache[:, g0:g1].contiguous()
        o_s = torch.empty((B, (g1 - g0) * G, 128), dtype=torch.float32, device="cuda")
        l_s = torch.empty((B, (g1 - g0) * G), dtype=torch.float32, device="cuda")
        ws2 = torch.empty_like(ws)
        bana.bana_decode_attn_partial(q_s, k_s, v_s, dw.block_table, dw.seq_lens, begin, end, o_s, l_s,
                                      workspace=ws2, dims=sub)
        assert np.array_equal(out[:, g0 * G:g1 * G].cpu().numpy(), o_s.cpu().numpy())
        assert np.array_equal(lse[:, g0 * G:g1 * G].cpu().numpy(), l_s.cpu().numpy())
    ro, rl = oracle.workload_partials(w)
    fin = np.isfinite(rl[part])
    o, l = out.cpu().numpy(), lse.cpu().numpy()
    _check_out(o[fin], ro[part][fin], f"{name} head-split out")
    assert np.all(o[~fin] == 0.0)
    _check_lse(l, rl[part], f"{name} head-split lse")

    # With the launch shape fixed by the hints, the plan no longer depends on the number of heads:
    # complementary head ranges then concatenate to the unsplit call bit for bit.
    lens = w.kv_end[part].astype(np.int64) - w.kv_begin[part]
    fixed = bana.make_dims(B, Hq, Hkv, w.max_blocks_per_seq, w.num_blocks, max_range_tokens=int(lens.max()),
                           total_range_tokens=int(lens.sum()), waves_hint=4, chunks_hint=3)
    ws = torch.empty(max(256, bana.bana_decode_attn_workspace_bytes(fixed)), dtype=torch.uint8, device="cuda")
    full_o = torch.empty((B, Hq, 128), dtype=torch.float32, device="cuda")
    full_l = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    bana.bana_decode_attn_partial(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, begin, end, full_o,
                                  full_l, workspace=ws, dims=fixed)
    out.fill_(float("nan"))
    lse.fill_(float("nan"))
    for g0, g1 in ((0, split), (split, Hkv)):
        bana.bana_decode_attn_heads(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, begin, end, g0, g1,
                                    out, lse, workspace=ws, dims=fixed)
    assert np.array_equal(out.cpu().numpy(), full_o.cpu().numpy())
    assert np.array_equal(lse.cpu().numpy(), full_l.cpu().numpy())


def test_hip_graph_capture_and_replay():
    """The library calls are capturable (no allocation, no synchronisation, no memset): a captured
    split step and a captured fused step replay bit-identically to eager execution, several times,
    with other device work in between."""
    w = _workload("tiny", 1)
    dw = DeviceWorkload(w)
    ref = dw.results()
    dw.fused(__import__("ctypes").c_void_p(torch.cuda.current_stream().cuda_stream))
    ref_fused = dw.fused_results()
    g_split, g_fused = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_split):
        dw.step()
    with torch.cuda.graph(g_fused):
        dw.fused(__import__("ctypes").c_void_p(torch.cuda.current_stream().cuda_stream))
    scratch = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        dw.out.fill_(float("nan"))
        dw.out_partials.fill_(float("nan"))
        dw.fused_out.fill_(float("nan"))
        scratch.add_(1.0)
        g_split.replay()
        torch.cuda.synchronize()
        for x, y in zip(ref, dw.results()):
            assert np.array_equal(x, y, equal_nan=True), rep
        g_fused.replay()
        torch.cuda.synchronize()
        for x, y in zip(ref_fused, dw.fused_results()):
            assert np.array_equal(x, y, equal_nan=True), rep


def test_layer_pipeline_matches_serial_and_oracle():
    """Three-stream layer pipeline (fetch layer i+1 / attend layer i / store layer i-1): the same
    per-layer results as running the stages one after the other, bit for bit; each layer's result
    matches the oracle on that layer's KV; stored blocks arrive intact."""
    from paper_2510_13223_amd.pipeline import LayerPipeline

    w = W.make_config("tiny", 2)
    st = W.make_layer_store(w, num_layers=5, fetch_tokens=100, store_tokens=64, seed=3)
    pipe = LayerPipeline(st)
    _log("[pipeline] tiny, 5 layers")
    pipe.run_serial()
    so, sl = pipe.outputs()
    ss = pipe.stored()
    pipe.out.fill_(float("nan"))
    pipe.run_pipelined(timing=True)
    po, pl = pipe.outputs()
    ps = pipe.stored()
    assert np.array_equal(so, po) and np.array_equal(sl, pl)
    # one launch per layer, the transfers carried by the attention launches
    for t in pipe.host_store_k + pipe.host_store_v:
        t.zero_()
    pipe.out.fill_(float("nan"))
    pipe.run_fused()
    fo, fl = pipe.outputs()
    fs = pipe.stored()
    assert np.array_equal(so, fo) and np.array_equal(sl, fl)
    for layer in range(st.num_layers):
        assert np.array_equal(fs[layer][0], ss[layer][0]) and np.array_equal(fs[layer][1], ss[layer][1])
    fb, sb = st.fetch_blocks, st.store_blocks
    for layer in range(st.num_layers):
        uo, ul = oracle.workload_unsplit(W.layer_view(st, layer))
        _check_out(po[layer], uo, f"layer {layer} out")
        _check_lse(pl[layer], ul, f"layer {layer} lse")
        for got in (ss[layer], ps[layer]):
            assert np.array_equal(got[0], st.w.k_cache[fb:fb + sb])
            assert np.array_equal(got[1], st.w.v_cache[fb:fb + sb])
    assert pipe.stage_ms.shape == (st.num_layers, 3)
    # layers see different fetched prefixes, so their outputs differ
    assert not np.array_equal(po[0], po[1])


def test_pool_beyond_4gib_uses_64bit_offsets():
    """Blocks placed beyond 2^31 bf16 elements of a pool (a 4.6 GB pool per cache) attend, migrate
    and export addresses exactly as the same blocks in a compact pool."""
    lens = [500, 333, 1000, 17]
    ranges = [[(0, 256), (0, 100), (0, 500), (0, 17)], [(256, 500), (100, 333), (500, 1000), (17, 17)]]
    w = W.make_custom(7, 4, 32, 8, lens, ranges, q_scale=1 / math.sqrt(128))
    base = 135000  # 135000 blocks x 8 kv heads x 2048 elements > 2^31
    big_nb = base + w.num_blocks
    _log(f"[64-bit] pools of {big_nb} blocks ({big_nb * 8 * 4096 / 1e9:.1f} GB each)")
    small = DeviceWorkload(w)
    ref = small.results()
    big_k = torch.full((big_nb,) + tuple(small.k_cache.shape[1:]), float("nan"), dtype=torch.bfloat16, device="cuda")
    big_v = torch.full((big_nb,) + tuple(small.v_cache.shape[1:]), float("nan"), dtype=torch.bfloat16, device="cuda")
    big_k[base:] = small.k_cache
    big_v[base:] = small.v_cache
    table = torch.where(small.block_table >= 0, small.block_table + base, small.block_table).contiguous()
    B, Hq = w.batch, w.num_q_heads
    for p in range(w.n_parts):
        o = torch.empty((B, Hq, 128), dtype=torch.float32, device="cuda")
        l = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
        d = bana.bana_dims.from_buffer_copy(small.dims[p])  # the same plan, over the big pools
        d.num_blocks = big_nb
        bana.bana_decode_attn_partial(small.q, big_k, big_v, table, small.seq_lens, small.kv_begin[p],
                                      small.kv_end[p], o, l, workspace=small.workspace, dims=d)
        assert np.array_equal(o.cpu().numpy(), ref[0][p]) and np.array_equal(l.cpu().numpy(), ref[1][p])
        rows = torch.empty((B, 8, w.max_blocks_per_seq * 16), dtype=torch.int64, device="cuda")
        bana.bana_debug_kv_rows(table, small.kv_begin[p], small.kv_end[p], big_nb, 8, rows)
        expect = oracle.kv_rows(table.cpu().numpy(), big_nb, 8, w.kv_begin[p], w.kv_end[p])
        assert expect.max() > 2 ** 31 // 128
        np.testing.assert_array_equal(rows.cpu().numpy(), expect)
    # migrate the blocks of partition 1 from the far end of the big pools into a compact pool
    m = W.make_migration(w, 1, seed=2)
    dk = torch.from_numpy(m.dst_k.view(np.int16)).view(torch.bfloat16).cuda()
    dv = torch.from_numpy(m.dst_v.view(np.int16)).view(torch.bfloat16).cuda()
    bana.bana_migrate_kv_blocks(big_k, big_v, table, dk, dv, torch.from_numpy(m.dst_table).cuda(),
                                torch.from_numpy(m.blk_begin).cuda(), torch.from_numpy(m.blk_end).cuda())
    ek, ev = oracle.migrate(w.k_cache, w.v_cache, w.block_table, m.dst_k, m.dst_v, m.dst_table, m.blk_begin,
                            m.blk_end)
    np.testing.assert_array_equal(dk.cpu().view(torch.int16).numpy().view(np.uint16), ek)
    np.testing.assert_array_equal(dv.cpu().view(torch.int16).numpy().view(np.uint16), ev)
    del big_k, big_v
    torch.cuda.empty_cache()


def test_million_sequences_at_the_launch_size_limits():
    """2^20 sequences x 8 kv heads (G = 1) with uneven ranges: the plan asks for 8 wavefronts per
    (sequence, kv head), which would pass 2^32 work-items in one launch, so the planner halves them;
    the per-partition call, a two-range fused call and the merge run at this size, and sampled rows
    (the two long sequences and 254 others) match the oracle."""
    B, H = 1 << 20, 8
    lens = np.full(B, 16, dtype=np.int32)
    rng = np.random.default_rng(11)
    lens[rng.integers(0, B, size=B // 8)] = 5  # ragged single blocks
    lens[12345], lens[B - 1] = 1024, 1000        # longest / mean > 1.25: uneven, 64 blocks
    _log(f"[1M] drawing B={B} H={H}")
    w = W.make_shared_pool(3, B, H, H, lens, pool_blocks=4096, q_scale=1 / math.sqrt(128))
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).view(dt)).cuda()
    q = dev(w.q, np.int16).view(torch.bfloat16)
    k = dev(w.k_cache, np.int16).view(torch.bfloat16)
    v = dev(w.v_cache, np.int16).view(torch.bfloat16)
    table, sl = dev(w.block_table, np.int32), dev(w.seq_lens, np.int32)
    begin, end = dev(w.kv_begin[0], np.int32), dev(w.kv_end[0], np.int32)
    dims = bana.make_dims(B, H, H, w.max_blocks_per_seq, w.num_blocks, max_range_tokens=int(lens.max()),
                          total_range_tokens=int(lens.astype(np.int64).sum()))
    ws_bytes = bana.bana_decode_attn_workspace_bytes(dims)
    ws = torch.empty(max(256, ws_bytes), dtype=torch.uint8, device="cuda")
    out = torch.empty((B, H, 128), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, H), dtype=torch.float32, device="cuda")
    _log("[1M] partial call")
    bana.bana_decode_attn_partial(q, k, v, table, sl, begin, end, out, lse, workspace=ws, dims=dims)
    # two ranges per sequence: [0, L/2) and [L/2, L) (the first empty for one-token halves)
    half = (lens // 2).astype(np.int32)
    b2 = np.stack([np.zeros(B, np.int32), half])
    e2 = np.stack([half, lens])
    fo = torch.empty_like(out)
    fl = torch.empty_like(lse)
    _log("[1M] fused call")
    bana.bana_decode_attn_fused(q, k, v, table, sl, dev(b2, np.int32), dev(e2, np.int32), fo, fl, workspace=ws,
                                dims=dims)
    _log("[1M] merge of the two results")
    mo = torch.empty_like(out)
    ml = torch.empty_like(lse)
    bana.bana_merge_partials(torch.stack([out, fo]), torch.stack([lse, fl]), mo, ml)
    torch.cuda.synchronize()
    seqs = np.unique(np.concatenate([[0, 12345, B - 1], rng.integers(0, B, size=253)]))
    sub = W.subset(w, seqs)
    ro, rl = oracle.workload_partials(sub)
    idx = torch.from_numpy(seqs).cuda()
    _check_out(out[idx].cpu().numpy(), ro[0], "1M partial out")
    _check_lse(lse[idx].cpu().numpy(), rl[0], "1M partial lse")
    _check_out(fo[idx].cpu().numpy(), ro[0], "1M fused out")
    _check_lse(fl[idx].cpu().numpy(), rl[0], "1M fused lse")
    # merging a result with itself keeps the output and adds ln 2 to the lse
    _check_out(mo[idx].cpu().numpy(), ro[0], "1M self-merge out")
    _check_lse(ml[idx].cpu().numpy(), rl[0] + math.log(2.0), "1M self-merge lse")
    del q, k, v, out, fo, mo, ws
    torch.cuda.empty_cache()


def test_validate_ranges_codes():
    w = _workload("tiny", 0)
    dw = DeviceWorkload(w)
    res = torch.empty(1, dtype=torch.int32, device="cuda")

    def check(table, lens, begin, end, nb=w.num_blocks):
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
        bana.bana_validate_ranges(t(table), t(lens), t(begin), t(end), nb, res)
        torch.cuda.synchronize()
        return int(res.item())

    tb, L, b0, e0 = w.block_table, w.seq_lens, w.kv_begin, w.kv_end
    assert check(tb, L, b0, e0) == 0
    assert check(tb, L, b0[0], e0[0]) == 0
    bad = b0.copy(); bad[1, 2] = e0[1, 2] + 1
    assert check(tb, L, bad, e0) == 1
    bad = b0.copy(); bad[0, 0] = -3
    assert check(tb, L, bad, e0) == 1
    bad = e0.copy(); bad[1, 3] = L[3] + 5
    assert check(tb, L, b0, bad) == 2
    lens = L.copy(); lens[0] = w.max_blocks_per_seq * 16 + 1
    assert check(tb, lens, b0, e0) == 3
    tbl = tb.copy(); tbl[2, 3] = -1
    assert check(tbl, L, b0, e0) == 4
    tbl = tb.copy(); tbl[1, 0] = w.num_blocks
    assert check(tbl, L, b0, e0) == 4
    bad = b0.copy(); bad[0, 0] = e0[0, 0] + 1  # sequence 0 breaks rule 1, sequence 1's table rule 4
    assert check(tbl, L, bad, e0) == 4  # the highest code wins
    # entries past a range are never read: poison them, still valid
    tbl = tb.copy()
    for b in range(w.batch):
        tbl[b, (L[b] + 15) // 16:] = 1 << 30
    assert check(tbl, L, b0, e0) == 0
    for name in ("llama3_8b", "mixed"):
        ww = _workload(name)
        assert check(ww.block_table, ww.seq_lens, ww.kv_begin, ww.kv_end, ww.num_blocks) == 0


@pytest.mark.parametrize("name", ["tiny", "mixed"])
def test_dispatch_order_hint_does_not_change_results(name):
    """Sequences dispatched longest-first (seq_order hint) or in natural order: bit-identical results."""
    w = _workload(name)
    a = DeviceWorkload(w, order_hints=True)
    b = DeviceWorkload(w, order_hints=False)
    for x, y in zip(a.results(), b.results()):
        assert np.array_equal(x, y, equal_nan=True)
    for x, y in zip(a.fused_results(), b.fused_results()):
        assert np.array_equal(x, y, equal_nan=True)


def _gather_xor_ref(w, begin, end):
    """Host XOR of the 32-bit words of every covered K and V tile, per (sequence, kv head)."""
    ref = np.zeros((w.batch, w.num_kv_heads), dtype=np.uint32)
    for b in range(w.batch):
        blks = []
        for p in range(begin.shape[0]):
            t0, t1 = int(begin[p, b]), int(end[p, b])
            if t1 > t0:
                blks.extend(int(w.block_table[b, j]) for j in range(t0 // 16, (t1 - 1) // 16 + 1))
        if not blks:
            continue
        idx = np.array(blks, dtype=np.int64)
        for g in range(w.num_kv_heads):
            kw = np.ascontiguousarray(w.k_cache[idx, g]).reshape(len(idx), -1).view(np.uint32)
            vw = np.ascontiguousarray(w.v_cache[idx, g]).reshape(len(idx), -1).view(np.uint32)
            ref[b, g] = np.bitwise_xor.reduce(kw, axis=None) ^ np.bitwise_xor.reduce(vw, axis=None)
    return ref


@pytest.mark.parametrize("seed", [0, 1])
def test_gather_read_covers_exactly_the_attention_tiles(seed):
    w = _workload("tiny", seed)
    _log(f"[gather] tiny seed={seed}")
    dw = DeviceWorkload(w)
    # The workload's partitions, plus an extra set: an empty range, a range inside one block,
    # and a range that overlaps partition 0 (its shared blocks are read twice and cancel).
    extra_b = np.zeros((3, w.batch), dtype=np.int32)
    extra_e = np.zeros((3, w.batch), dtype=np.int32)
    for b in range(w.batch):
        L = int(w.seq_lens[b])
        extra_b[1, b], extra_e[1, b] = 17, 20
        extra_b[2, b], extra_e[2, b] = 5, min(L, 300)
    for begin, end in ((w.kv_begin, w.kv_end), (extra_b, extra_e)):
        sink = torch.zeros((w.batch, w.num_kv_heads), dtype=torch.int32, device="cuda")
        bana.bana_debug_gather_read(dw.k_cache, dw.v_cache, dw.block_table, torch.from_numpy(begin).cuda(),
                                    torch.from_numpy(end).cuda(), sink)
        got = sink.cpu().numpy().view(np.uint32)
        np.testing.assert_array_equal(got, _gather_xor_ref(w, begin, end))


def test_hooks_stride_past_their_grid():
    """The validation and gather kernels stride over sequences / (sequence, kv head) pairs when there are
    more than their grids hold (65,536 sequences; 2^20 pairs): every sequence is still checked and every
    pair read."""
    rng = np.random.default_rng(7)
    B, Hkv, nb = 140_000, 8, 512  # 1.12 M pairs
    _log(f"[hooks] B={B} Hkv={Hkv} pool={nb}")
    k = rng.integers(0, 1 << 16, size=(nb, Hkv, 16, 16, 8), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=(nb, Hkv, 128, 16), dtype=np.uint16)
    table = rng.integers(0, nb, size=(B, 1), dtype=np.int32)
    end = rng.integers(0, 17, size=(1, B), dtype=np.int32)  # 0..16 tokens of the one block; 0 = empty
    begin = np.zeros((1, B), dtype=np.int32)
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).view(dt)).cuda()
    sink = torch.zeros((B, Hkv), dtype=torch.int32, device="cuda")
    bana.bana_debug_gather_read(dev(k, np.int16).view(torch.bfloat16), dev(v, np.int16).view(torch.bfloat16),
                                dev(table, np.int32), dev(begin, np.int32), dev(end, np.int32), sink)
    tile_x = (np.bitwise_xor.reduce(k.reshape(nb, Hkv, -1).view(np.uint32), axis=2)
              ^ np.bitwise_xor.reduce(v.reshape(nb, Hkv, -1).view(np.uint32), axis=2))
    ref = np.where((end[0] > 0)[:, None], tile_x[table[:, 0]], np.uint32(0))
    np.testing.assert_array_equal(sink.cpu().numpy().view(np.uint32), ref)

    res = torch.empty(1, dtype=torch.int32, device="cuda")
    Bv = 70_000
    lens = np.full(Bv, 16, dtype=np.int32)
    tb = table[:Bv].copy()

    def check(tbl, e):
        bana.bana_validate_ranges(dev(tbl, np.int32), dev(lens, np.int32), dev(np.zeros(Bv, np.int32), np.int32),
                                  dev(e, np.int32), nb, res)
        torch.cuda.synchronize()
        return int(res.item())

    e = np.full(Bv, 16, dtype=np.int32)
    assert check(tb, e) == 0
    e2 = e.copy(); e2[Bv - 1] = 17  # the last sequence, beyond the grid's first pass
    assert check(tb, e2) == 2
    tb2 = tb.copy(); tb2[Bv - 2, 0] = nb
    assert check(tb2, e) == 4


@pytest.mark.parametrize("nbytes,groups", [(16, 1), (4096 + 16, 7), ((1 << 20) + 48, 2048), (64 << 20, 2048)])
def test_stream_read_folds_every_word(nbytes, groups):
    """The streaming-read hook reads every 16-byte unit once: sink[w] is the XOR of the units
    w*256 + t + i*groups*256, so their XOR is the XOR of the whole buffer."""
    _log(f"[stream-read] bytes={nbytes} groups={groups}")
    rng = np.random.default_rng(nbytes)
    words = rng.integers(0, 1 << 32, size=nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).cuda()
    sink = torch.full((groups,), -1, dtype=torch.int32, device="cuda")
    bana.bana_debug_stream_read(buf, sink)
    got = sink.cpu().numpy().view(np.uint32)
    unit_x = np.bitwise_xor.reduce(words.reshape(-1, 4), axis=1)
    grp = (np.arange(unit_x.size) // 256) % groups
    ref = np.zeros(groups, dtype=np.uint32)
    np.bitwise_xor.at(ref, grp, unit_x)
    np.testing.assert_array_equal(got, ref)


def test_copy_binding_device_and_pinned_host():
    """bana_copy_async through its checked binding: device to device, pinned host to device and back,
    bit for bit, at a size that leaves a ragged last workgroup."""
    n = (3 << 20) + 16
    rng = np.random.default_rng(3)
    host = torch.from_numpy(rng.integers(0, 256, size=n, dtype=np.uint8)).pin_memory()
    dev_a = torch.empty(n, dtype=torch.uint8, device="cuda")
    dev_b = torch.empty(n, dtype=torch.uint8, device="cuda")
    back = torch.empty(n, dtype=torch.uint8).pin_memory()
    s = torch.cuda.Stream()
    bana.bana_copy_async(dev_a, host, stream=s)
    bana.bana_copy_async(dev_b, dev_a, stream=s)
    bana.bana_copy_async(back, dev_b, stream=s)
    s.synchronize()
    assert torch.equal(back, host)
    with pytest.raises(ValueError):
        bana.bana_copy_async(dev_a[:16], dev_b[:32])
    with pytest.raises(ValueError):
        bana.bana_copy_async(dev_a, torch.zeros(n, dtype=torch.uint8))  # pageable host memory


def test_plain_c_caller_through_the_abi():
    """A C program (tests/c/abi_roundtrip.c: hipMalloc'd buffers, its own stream, no Python or torch)
    runs the per-partition calls, the merge and the fused call and checks them against the oracle."""
    import os
    import subprocess

    here = os.path.dirname(os.path.abspath(__file__))
    exe = os.path.join(here, "c", "abi_roundtrip")
    if not os.path.exists(exe):  # normally built by __graft_entry__.build(); gcc takes a second
        import importlib.util

        oracle._load()  # builds liboracle.so if it is missing
        spec = importlib.util.spec_from_file_location("abi_roundtrip_build", os.path.join(here, "c", "build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()
    _log("[c-abi] running tests/c/abi_roundtrip")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    _log(r.stdout.strip())
    assert r.returncode == 0, r.stdout + r.stderr


@pytest.mark.parametrize("case", range(12))
def test_random_shapes_every_launch_shape(case):
    """Seeded random small workloads (batch, GQA group, lengths, 1-5 ranges per sequence with empty,
    one-token and ragged ranges) through the automatic, chunked and balanced plans, per-partition and
    fused, against the oracle."""
    rng = np.random.default_rng(1000 + case)
    B = int(rng.integers(1, 13))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    Hq = Hkv * int(rng.choice([1, 2, 4, 8, 16]))
    n_parts = int(rng.integers(1, 6))
    lens = [int(x) for x in rng.integers(1, 2500, size=B)]
    ranges = [[] for _ in range(n_parts)]
    for L in lens:
        cuts = np.sort(rng.integers(0, L + 1, size=n_parts - 1)).tolist()
        edges = [0] + cuts + [L]
        for p in range(n_parts):
            ranges[p].append((edges[p], edges[p + 1]))
    w = W.make_custom(50 + case, B, Hq, Hkv, lens, ranges, q_scale=1 / math.sqrt(128))
    _log(f"[random {case}] B={B} Hq={Hq} Hkv={Hkv} parts={n_parts}")
    for plan in (0, 1, 2):
        _full_parity(w, plan_hint=plan)


@pytest.mark.parametrize("case", range(24))
def test_random_launch_hints_and_head_ranges(case):
    """Seeded random small workloads (up to 40 sequences, G up to 16, 1-6 ranges each) under random
    launch hints (waves, chunks, plan, dispatch order, no workspace, no range hints), per-partition,
    merged and fused against the oracle, plus a random kv-head range of partition 0."""
    rng = np.random.default_rng(50000 + case)
    B = int(rng.integers(1, 41))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    Hq = Hkv * int(rng.choice([1, 2, 3, 4, 8, 16]))
    n_parts = int(rng.integers(1, 7))
    maxL = int(rng.choice([64, 600, 5000]))
    lens = [int(x) for x in rng.integers(1, maxL + 1, size=B)]
    ranges = [[] for _ in range(n_parts)]
    for L in lens:
        cuts = np.sort(rng.integers(0, L + 1, size=n_parts - 1)).tolist()
        edges = [0] + cuts + [L]
        for p in range(n_parts):
            ranges[p].append((edges[p], edges[p + 1]))
    w = W.make_custom(70000 + case, B, Hq, Hkv, lens, ranges, q_scale=1 / math.sqrt(128))
    kw = dict(waves_hint=int(rng.choice([0, 0, 1, 2, 4, 8])), chunks_hint=int(rng.choice([0, 0, 1, 2, 3, 5, 9])),
              plan_hint=int(rng.choice([0, 0, 1, 2])), order_hints=bool(rng.integers(0, 2)),
              use_workspace=bool(rng.integers(0, 4) > 0), range_hints=bool(rng.integers(0, 4) > 0))
    _log(f"[hints {case}] B={B} Hq={Hq} Hkv={Hkv} parts={n_parts} maxL={maxL} {kw}")
    dw = _full_parity(w, **kw)
    if Hkv > 1:
        ro, rl = oracle.workload_partials(w)
        g0 = int(rng.integers(0, Hkv))
        g1 = int(rng.integers(g0 + 1, Hkv + 1))
        G = Hq // Hkv
        sub = bana.head_range_dims(dw.dims[0], g0, g1)
        ws = torch.empty(max(256, bana.bana_decode_attn_workspace_bytes(sub)), dtype=torch.uint8, device="cuda")
        o = torch.full((B, Hq, 128), float("nan"), device="cuda")
        l = torch.full((B, Hq), float("nan"), device="cuda")
        bana.bana_decode_attn_heads(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin[0],
                                    dw.kv_end[0], g0, g1, o, l, workspace=ws, dims=dw.dims[0])
        o, l = o.cpu().numpy(), l.cpu().numpy()
        hs = slice(g0 * G, g1 * G)
        fin = np.isfinite(rl[0][:, hs])
        _check_out(o[:, hs][fin], ro[0][:, hs][fin], "head range out")
        assert np.all(o[:, hs][~fin] == 0.0)
        _check_lse(l[:, hs], rl[0][:, hs], "head range lse")
        assert np.all(np.isnan(o[:, :g0 * G])) and np.all(np.isnan(o[:, g1 * G:]))


def test_forced_balanced_launch_on_mixed():
    """The balanced launch over all 256 sequences of the mixed workload (the schedule's prefix sums
    span four 64-lane strides), per partition and fused, against the oracle."""
    _full_parity(_workload("mixed"), plan_hint=2)


@pytest.mark.parametrize("case", range(8))
def test_random_shapes_many_sequences(case):
    """Seeded random workloads of 65-300 sequences with uneven, empty and ragged ranges through the
    automatic, chunked and balanced plans (the balanced schedule beyond one 64-lane stride)."""
    rng = np.random.default_rng(90000 + case)
    B = int(rng.integers(65, 301))
    Hkv = int(rng.choice([1, 2, 4]))
    Hq = Hkv * int(rng.choice([1, 4, 8]))
    n_parts = int(rng.integers(1, 4))
    lens = [int(x) for x in np.clip(np.rint(np.exp(rng.normal(np.log(300.0), 1.0, size=B))), 1, 4000)]
    ranges = [[] for _ in range(n_parts)]
    for L in lens:
        cuts = np.sort(rng.integers(0, L + 1, size=n_parts - 1)).tolist()
        edges = [0] + cuts + [L]
        for p in range(n_parts):
            ranges[p].append((edges[p], edges[p + 1]))
    w = W.make_custom(91000 + case, B, Hq, Hkv, lens, ranges, q_scale=1 / math.sqrt(128))
    _log(f"[many {case}] B={B} Hq={Hq} Hkv={Hkv} parts={n_parts}")
    for plan in (0, 1, 2):
        _full_parity(w, plan_hint=plan)


def test_balanced_piece_merge_many_rows_many_pieces():
    """A balanced launch over 5,120 merged rows in which one sequence spans ~170 intervals (the piece
    merge with two thread groups per row) and the rest fit in one or two, against the oracle."""
    rng = np.random.default_rng(4242)
    B = 160
    lens = [int(x) for x in rng.integers(1, 65, size=B)]
    lens[37] = 8000
    cuts = [L // 3 if b == 37 else int(rng.integers(0, L + 1)) for b, L in enumerate(lens)]
    ranges = [[(0, c) for c in cuts], [(c, L) for c, L in zip(cuts, lens)]]
    w = W.make_custom(4242, B, 32, 8, lens, ranges, q_scale=1 / math.sqrt(128))
    for plan in (2, 0):
        _full_parity(w, plan_hint=plan)


@pytest.mark.parametrize("B", [2048, 2049])
def test_balanced_launch_at_its_batch_limit(B):
    """2048 sequences (the balanced schedule's limit: four per thread of the LDS scan) run the
    balanced launch; 2049 fall back to the chunked launch.  Both against the oracle."""
    rng = np.random.default_rng(B)
    lens = [int(x) for x in rng.integers(1, 97, size=B)]
    lens[5] = 3000
    cuts = [int(rng.integers(0, L + 1)) if b % 7 else L for b, L in enumerate(lens)]  # every 7th: 2nd part empty
    ranges = [[(0, c) for c in cuts], [(c, L) for c, L in zip(cuts, lens)]]
    w = W.make_custom(B, B, 4, 1, lens, ranges, q_scale=1 / math.sqrt(128))
    dw = _full_parity(w, plan_hint=2)
    # The balanced plan has a workspace layout of its own: the forced-balanced dims size differently
    # from the forced-chunked ones exactly when the balanced launch runs.
    chunked = bana.bana_dims.from_buffer_copy(dw.dims[0])
    chunked.plan_hint = 1
    balanced_ran = bana.bana_decode_attn_workspace_bytes(dw.dims[0]) != bana.bana_decode_attn_workspace_bytes(chunked)
    assert balanced_ran == (B <= 2048)


def _migrate_and_check(w, part, seed, hint=True):
    m = W.make_migration(w, part, seed=seed)
    dk = torch.from_numpy(m.dst_k.view(np.int16)).view(torch.bfloat16).cuda()
    dv = torch.from_numpy(m.dst_v.view(np.int16)).view(torch.bfloat16).cuda()
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    hint_tokens = int(np.max(m.blk_end - m.blk_begin)) * 16 if hint else 0
    bana.bana_migrate_kv_blocks(bf(w.k_cache), bf(w.v_cache), i32(w.block_table), dk, dv, i32(m.dst_table),
                                i32(m.blk_begin), i32(m.blk_end), max_range_tokens=hint_tokens)
    ek, ev = oracle.migrate(w.k_cache, w.v_cache, w.block_table, m.dst_k, m.dst_v, m.dst_table, m.blk_begin,
                            m.blk_end)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dk.cpu().view(torch.int16).numpy().view(np.uint16), ek)
    np.testing.assert_array_equal(dv.cpu().view(torch.int16).numpy().view(np.uint16), ev)


@pytest.mark.parametrize("case", range(10))
def test_migration_random_batches_bit_exact(case):
    """The flat migration (blocks of all sequences in one list, split evenly over the workgroups)
    on seeded random batches of 1-300 sequences, 1-8 kv heads, many empty ranges, against the
    oracle's copy bit for bit (every destination block outside the list keeps its sentinel)."""
    rng = np.random.default_rng(120000 + case)
    B = int(rng.integers(1, 301))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    lens = [int(x) for x in rng.integers(1, 700, size=B)]
    cuts = [int(rng.integers(0, L + 1)) if rng.random() < 0.6 else L for L in lens]
    ranges = [[(0, c) for c in cuts], [(c, L) for c, L in zip(cuts, lens)]]
    w = W.make_custom(121000 + case, B, Hkv, Hkv, lens, ranges)
    _log(f"[migrate random {case}] B={B} Hkv={Hkv}")
    _migrate_and_check(w, 1, seed=case, hint=bool(case % 2))


def test_migration_beyond_the_flat_batch_limit():
    """5000 sequences (above the flat list's 4096): the per-sequence grid, bit for bit."""
    B = 5000
    rng = np.random.default_rng(5000)
    lens = [int(x) for x in rng.integers(1, 80, size=B)]
    cuts = [int(rng.integers(0, L + 1)) for L in lens]
    w = W.make_custom(5000, B, 2, 2, lens, [[(0, c) for c in cuts], [(c, L) for c, L in zip(cuts, lens)]])
    _migrate_and_check(w, 1, seed=1)


def _raw_step(L, dw, h):
    """Every partition, the merge and the fused call of a prepared workload through library L."""
    for p in range(dw.w.n_parts):
        assert L.bana_decode_attn_partial(*dw._partial_args[p], h) == bana.BANA_OK
    assert L.bana_merge_partials(*dw._merge_args, h) == bana.BANA_OK
    assert L.bana_decode_attn_fused(*dw._fused_args, h) == bana.BANA_OK


@pytest.mark.parametrize("name,plan", [("tiny", 0), ("tiny", 2), ("fine", 0), ("llama3_8b", 0), ("mixed", 0)])
def test_lds_race_check_build_bit_identical(name, plan):
    """The LDS race-check build (odd wavefronts sleep before every LDS write that other wavefronts
    read back, and one more barrier precedes every read-back) gives the product build's results bit
    for bit: the cross-wave combine of the chunked launch (llama3_8b, mixed), the balanced launch's
    prefix scan and the piece merge's thread-group combine (tiny forced balanced, mixed's migrated
    partition), and the flat migration's scan."""
    side = bana.load(bana.RACECHECK_LIB_PATH)
    with open(bana.RACECHECK_LIB_PATH, "rb") as f1, open(bana.LIB_PATH, "rb") as f2:
        assert f1.read() != f2.read(), "the race-check build must differ from the product build"
    w = _workload(name)
    dw = DeviceWorkload(w, plan_hint=plan)
    h = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    outs = (dw.out_partials, dw.lses, dw.out, dw.lse_out, dw.fused_out, dw.fused_lse)
    _raw_step(bana.lib(), dw, h)
    ref = [t.clone() for t in outs]
    for t in outs:
        t.fill_(float("nan"))
    _raw_step(side, dw, h)
    torch.cuda.synchronize()
    for a, b in zip(outs, ref):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    # the flat migration of the last partition
    m = W.make_migration(w, w.n_parts - 1, seed=3)
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    dst = []
    for L in (bana.lib(), side):
        dk = torch.from_numpy(m.dst_k.view(np.int16)).view(torch.bfloat16).cuda()
        dv = torch.from_numpy(m.dst_v.view(np.int16)).view(torch.bfloat16).cuda()
        dt, mb, me = i32(m.dst_table), i32(m.blk_begin), i32(m.blk_end)
        d = bana.bana_dims(w.batch, w.num_kv_heads, w.num_kv_heads, 128, 16, w.max_blocks_per_seq, w.num_blocks,
                           0, 0, 0, 0, 0, None, 0)
        vp = lambda t: ctypes.c_void_p(t.data_ptr())
        assert L.bana_migrate_kv_blocks(ctypes.byref(d), vp(dw.k_cache), vp(dw.v_cache), vp(dw.block_table), vp(dk),
                                        vp(dv), vp(dt), m.num_blocks, vp(mb), vp(me), h) == bana.BANA_OK
        torch.cuda.synchronize()
        dst.append((dk, dv))
    assert torch.equal(dst[0][0].view(torch.int16), dst[1][0].view(torch.int16))
    assert torch.equal(dst[0][1].view(torch.int16), dst[1][1].view(torch.int16))


@pytest.mark.parametrize("name,plan", [("tiny", 0), ("tiny", 2), ("mixed", 0)])
def test_wave_timeline_build_bit_identical_and_ordered(name, plan):
    """The wavefront-timeline build gives the product build's results bit for bit (chunked launch;
    balanced launch with its piece merge; mixed's four dispatch rounds and its balanced migrated
    partition), and its clock readings are ordered: entry <= schedule ready <= first block <= exit
    for every wavefront of the last call that recorded them."""
    from paper_2510_13223_amd import timeline

    side = bana.load(bana.TIMELINE_LIB_PATH)
    w = _workload(name)
    dw = DeviceWorkload(w, plan_hint=plan)
    h = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    outs = (dw.out_partials, dw.lses, dw.out, dw.lse_out, dw.fused_out, dw.fused_lse)
    _raw_step(bana.lib(), dw, h)
    ref = [t.clone() for t in outs]
    for t in outs:
        t.fill_(float("nan"))
    _raw_step(side, dw, h)
    torch.cuda.synchronize()
    for a, b in zip(outs, ref):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    for p in range(w.n_parts):
        bana.bana_debug_wave_timeline_clear(library=side)
        assert side.bana_decode_attn_partial(*dw._partial_args[p], h) == bana.BANA_OK
        t = bana.bana_debug_wave_timeline_read(bana.TIMELINE_SLOTS, library=side)
        used = t[:, 0] != timeline.UNSET
        assert used.sum() > 0
        t = t[used]
        assert np.all(t[:, 1] != timeline.UNSET) and np.all(t[:, 0] <= t[:, 1])
        done = t[:, 3] != timeline.UNSET
        assert done.sum() > 0 and np.all(t[done, 1] <= t[done, 3])
        first = t[:, 2] != timeline.UNSET
        assert first.sum() > 0 and np.all(t[first, 1] <= t[first, 2])
        assert np.all(t[first & done, 2] <= t[first & done, 3])
        s = timeline.summarize(t)
        assert s["waves"] == len(t) and 0 < s["span_us"] < 1e5


@pytest.mark.parametrize("name", ["tiny", "llama3_8b"])
def test_fused_copies_equal_the_fused_call_and_copy_exactly(name):
    """bana_decode_attn_fused_copies: the attention equals bana_decode_attn_fused with the chunked
    launch bit for bit, and its side copies (pinned host -> device, device -> pinned host, device ->
    device, ragged sizes, a zero-byte copy) arrive byte for byte."""
    w = _workload(name)
    dw = DeviceWorkload(w, plan_hint=1, waves_hint=4)
    B, Hq = w.batch, w.num_q_heads
    ref_o = torch.empty((B, Hq, 128), device="cuda")
    ref_l = torch.empty((B, Hq), device="cuda")
    bana.bana_decode_attn_fused(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin, dw.kv_end,
                                ref_o, ref_l, workspace=dw.workspace, dims=dw.fused_dims)
    g = torch.Generator().manual_seed(7)
    host_src = torch.randint(-2**31, 2**31 - 1, (((3 << 20) + 48) // 4,), dtype=torch.int32, generator=g).pin_memory()
    dev_src = torch.randint(-2**31, 2**31 - 1, (((1 << 20) + 16) // 4,), dtype=torch.int32, generator=g).cuda()
    dev_dst = torch.zeros_like(host_src, device="cuda")
    host_dst = torch.zeros_like(dev_src, device="cpu").pin_memory()
    dev_dst2 = torch.zeros_like(dev_src)
    empty = torch.empty(0, dtype=torch.int32, device="cuda")
    o = torch.full((B, Hq, 128), float("nan"), device="cuda")
    l = torch.full((B, Hq), float("nan"), device="cuda")
    bana.bana_decode_attn_fused_copies(dw.q, dw.k_cache, dw.v_cache, dw.block_table, dw.seq_lens, dw.kv_begin,
                                       dw.kv_end, o, l, copies=[(dev_dst, host_src), (host_dst, dev_src),
                                                                (dev_dst2, dev_src), (empty, empty)],
                                       workspace=dw.workspace, dims=dw.fused_dims)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int32), ref_o.view(torch.int32))
    assert torch.equal(l.view(torch.int32), ref_l.view(torch.int32))
    assert torch.equal(dev_dst.cpu(), host_src)
    assert torch.equal(host_dst, dev_src.cpu())
    assert torch.equal(dev_dst2, dev_src)
