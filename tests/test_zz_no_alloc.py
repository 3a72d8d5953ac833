"""bana_decode_attn_partial_noalloc (the library's static device scratch in place of a caller
workspace) against bana_decode_attn_partial with a workspace of its own, through the C ABI.

Both run the same plan and kernels, so the outputs must agree bit for bit; each is also held to
the fp64 oracle's tolerances (max-abs 2e-3, rel-L2 1e-3, |dlse| 1e-4, -inf exactly where a range
is empty).  The calls come in a row on one device -- a balanced launch first, then a smaller
input through the chunked launch, then the first input again -- so each later call runs over
the scratch contents the previous one left there.
"""

import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2510_13223_amd import bana, workloads as W

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


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _uneven_workload(seed, B, Hq, Hkv, max_len):
    """One range per sequence, uneven lengths, some empty and some not block-aligned."""
    rng = np.random.default_rng(seed)
    lens = [int(x) for x in rng.integers(1, max_len + 1, size=B)]
    lens[0] = max_len  # one long range sets the spread
    ranges = []
    for b, L in enumerate(lens):
        if b % 5 == 3:
            ranges.append((L // 2, L // 2))  # empty
        else:
            t0 = int(rng.integers(0, L // 3 + 1))
            ranges.append((t0, L))
    return W.make_custom(seed, B, Hq, Hkv, lens, [ranges], q_scale=1 / math.sqrt(128))


class _Case:
    def __init__(self, w, **hints):
        dev = torch.device("cuda")
        bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
        self.w = w
        self.q, self.k, self.v = bf(w.q), bf(w.k_cache), bf(w.v_cache)
        self.table, self.lens = i32(w.block_table), i32(w.seq_lens)
        self.begin, self.end = i32(w.kv_begin[0]), i32(w.kv_end[0])
        lens = w.kv_end[0].astype(np.int64) - w.kv_begin[0]
        self.dims = bana.make_dims(w.batch, w.num_q_heads, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks,
                                   max_range_tokens=int(lens.max()), total_range_tokens=int(lens.sum()), **hints)
        self.need = bana.bana_decode_attn_workspace_bytes(self.dims)
        self.hints = hints

    def outputs(self):
        B, Hq = self.w.batch, self.w.num_q_heads
        return (torch.full((B, Hq, 128), float("nan"), device="cuda"),
                torch.full((B, Hq), float("nan"), device="cuda"))

    def with_workspace(self):
        o, l = self.outputs()
        ws = torch.empty(self.need, dtype=torch.uint8, device="cuda")
        bana.bana_decode_attn_partial(self.q, self.k, self.v, self.table, self.lens, self.begin, self.end, o, l,
                                      workspace=ws, dims=self.dims)
        torch.cuda.synchronize()
        return o, l

    def noalloc(self):
        o, l = self.outputs()
        bana.bana_decode_attn_partial_noalloc(self.q, self.k, self.v, self.table, self.lens, self.begin, self.end,
                                              o, l, dims=self.dims)
        torch.cuda.synchronize()
        return o, l


def _same_bits(a, b):
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def _check_oracle(w, o, l, what):
    ro, rl = oracle.workload_partials(w)
    ro, rl = ro[0], rl[0]
    o, l = o.cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64)
    fin = np.isfinite(rl)
    assert np.array_equal(np.isneginf(l), ~fin), f"{what}: -inf pattern differs"
    assert np.all(o[~fin] == 0.0), f"{what}: empty range must give out = 0"
    d = o[fin] - ro[fin]
    max_abs = float(np.max(np.abs(d)))
    rel = float(np.linalg.norm(d) / np.linalg.norm(ro[fin]))
    lse_err = float(np.max(np.abs(l[fin] - rl[fin])))
    assert max_abs <= MAX_ABS and rel <= REL_L2 and lse_err <= LSE_ABS, (what, max_abs, rel, lse_err)
    _log(f"  {what}: max-abs {max_abs:.2e} rel-L2 {rel:.2e} lse {lse_err:.2e}")


def test_noalloc_matches_the_workspace_call_on_consecutive_calls():
    # Call 1: a balanced launch (piece partials + prefix sums in the scratch).
    big = _Case(_uneven_workload(7, 12, 8, 2, 9000), plan_hint=2)
    # Call 2, a smaller input: the chunked launch with 4 chunks per range (chunk partials).
    small = _Case(_uneven_workload(8, 5, 8, 2, 3000), waves_hint=2, chunks_hint=4)
    for c in (big, small):
        assert 0 < c.need <= bana.STATIC_SCRATCH_BYTES, c.need
    assert small.need < big.need
    for i, c in enumerate((big, small, big)):
        _log(f"[noalloc call {i}] B={c.w.batch} Hq={c.w.num_q_heads} Hkv={c.w.num_kv_heads} {c.hints} "
             f"scratch use {c.need} B")
        ro, rl = c.with_workspace()
        o, l = c.noalloc()
        assert _same_bits(o, ro) and _same_bits(l, rl), f"call {i}: differs from the workspace call"
        _check_oracle(c.w, o, l, f"call {i}")


def test_noalloc_refuses_plans_beyond_the_static_scratch():
    c = _Case(_uneven_workload(9, 64, 32, 8, 400), waves_hint=1, chunks_hint=256)
    assert c.need > bana.STATIC_SCRATCH_BYTES
    o, l = c.outputs()
    with pytest.raises(bana.BanaError) as e:
        bana.bana_decode_attn_partial_noalloc(c.q, c.k, c.v, c.table, c.lens, c.begin, c.end, o, l, dims=c.dims)
    assert e.value.status == bana.BANA_ERR_UNSUPPORTED
    assert str(bana.STATIC_SCRATCH_BYTES) in bana.lib().bana_last_error().decode()
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(o)) and torch.all(torch.isnan(l)), "a refused call must launch nothing"
