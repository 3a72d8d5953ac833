"""CPU checks of libbana.so: it loads, exports every declared symbol, and rejects
bad arguments on the host before any HIP call (no compute call needs a GPU)."""

import ctypes
import os
import re

import pytest

from paper_2510_13223_amd import bana

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bana.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bana_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bana.LIB_PATH):
        from paper_2510_13223_amd import build
        build.build()
    return bana.lib()


def test_header_declares_the_boundary():
    names = _declared_functions()
    for n in ("bana_decode_attn_partial", "bana_merge_partials", "bana_decode_attn_workspace_bytes",
              "bana_status_string", "bana_last_error", "bana_debug_kv_rows"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in _declared_functions():
        assert hasattr(lib, n), n


def test_status_strings(lib):
    assert lib.bana_status_string(0) == b"ok"
    assert lib.bana_status_string(-1) == b"invalid argument"
    assert lib.bana_status_string(-2) == b"unsupported configuration"
    assert lib.bana_status_string(-3) == b"device error"
    assert lib.bana_last_error() == b""


def _dims(**kw):
    base = dict(batch=4, num_q_heads=8, num_kv_heads=2, max_blocks_per_seq=64, num_blocks=100)
    base.update(kw)
    d = bana.make_dims(base["batch"], base["num_q_heads"], base["num_kv_heads"], base["max_blocks_per_seq"],
                       base["num_blocks"])
    for k in ("head_dim", "block_size", "plan_hint", "waves_hint", "chunks_hint", "max_range_tokens"):
        if k in kw:
            setattr(d, k, kw[k])
    return d


FAKE = ctypes.c_void_p(0x100000)  # 16-byte aligned, never dereferenced: every case below fails validation


def _partial(lib, d, ptrs=None, ws=None, ws_bytes=0):
    p = ptrs or [FAKE] * 9
    return lib.bana_decode_attn_partial(ctypes.byref(d) if d is not None else None, *p, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(batch=0), -1), (dict(num_q_heads=-8), -1), (dict(num_kv_heads=3), -1), (dict(num_blocks=0), -1),
    (dict(max_blocks_per_seq=0), -1), (dict(plan_hint=3), -1), (dict(plan_hint=-1), -1), (dict(waves_hint=3), -1), (dict(chunks_hint=-1), -1),
    (dict(max_range_tokens=-5), -1),
    (dict(head_dim=64), -2), (dict(block_size=32), -2), (dict(num_q_heads=34, num_kv_heads=2), -2),
])
def test_partial_rejects_bad_dims(lib, kw, expect):
    assert _partial(lib, _dims(**kw)) == expect
    assert lib.bana_decode_attn_workspace_bytes(ctypes.byref(_dims(**kw))) == 0


def test_partial_rejects_null_and_misaligned(lib):
    assert _partial(lib, None) == -1
    for i in range(9):
        ptrs = [FAKE] * 9
        ptrs[i] = None
        assert _partial(lib, _dims(), ptrs) == -1, i
    for i in (0, 1, 2, 7):  # q, k_cache, v_cache, out_partial must be 16-byte aligned
        ptrs = [FAKE] * 9
        ptrs[i] = ctypes.c_void_p(0x100008)
        assert _partial(lib, _dims(), ptrs) == -1, i
    assert _partial(lib, _dims(), None, ctypes.c_void_p(0x100004), 4096) == -1


def test_merge_rejects_bad_arguments(lib):
    d = _dims()
    assert lib.bana_merge_partials(ctypes.byref(d), FAKE, FAKE, 0, FAKE, None, None) == -1
    assert lib.bana_merge_partials(ctypes.byref(d), None, FAKE, 2, FAKE, None, None) == -1
    assert lib.bana_merge_partials(ctypes.byref(d), FAKE, None, 2, FAKE, None, None) == -1
    assert lib.bana_merge_partials(ctypes.byref(d), FAKE, FAKE, 2, None, None, None) == -1
    assert lib.bana_merge_partials(ctypes.byref(d), ctypes.c_void_p(0x100004), FAKE, 2, FAKE, None, None) == -1
    assert lib.bana_merge_partials(ctypes.byref(_dims(head_dim=96)), FAKE, FAKE, 2, FAKE, None, None) == -2
    assert lib.bana_merge_partials(ctypes.byref(_dims(batch=0)), FAKE, FAKE, 2, FAKE, None, None) == -1
    assert lib.bana_merge_partials(None, FAKE, FAKE, 2, FAKE, None, None) == -1
    assert lib.bana_debug_kv_rows(ctypes.byref(d), None, FAKE, FAKE, FAKE, None) == -1


def test_fused_rejects_bad_arguments(lib):
    d = _dims()

    def fused(dd, n, ptrs=None):
        p = ptrs or [FAKE] * 7
        return lib.bana_decode_attn_fused(ctypes.byref(dd) if dd is not None else None, *p, n, FAKE, FAKE, None, 0,
                                          None)

    assert fused(d, 0) == -1
    assert fused(d, -3) == -1
    assert fused(d, 65) == -2
    assert fused(None, 2) == -1
    assert fused(_dims(head_dim=64), 2) == -2
    for i in range(7):
        ptrs = [FAKE] * 7
        ptrs[i] = None
        assert fused(d, 2, ptrs) == -1, i
    assert lib.bana_decode_attn_fused(ctypes.byref(d), *[FAKE] * 7, 2, FAKE, None, None, 0, None) == -1


def test_migrate_rejects_bad_arguments(lib):
    d = _dims()
    args = [FAKE] * 6
    assert lib.bana_migrate_kv_blocks(ctypes.byref(d), *args, 0, FAKE, FAKE, None) == -1
    for i in range(6):
        a = list(args)
        a[i] = None
        assert lib.bana_migrate_kv_blocks(ctypes.byref(d), *a, 10, FAKE, FAKE, None) == -1, i
    for i in (0, 1, 3, 4):
        a = list(args)
        a[i] = ctypes.c_void_p(0x100008)
        assert lib.bana_migrate_kv_blocks(ctypes.byref(d), *a, 10, FAKE, FAKE, None) == -1, i
    assert lib.bana_migrate_kv_blocks(ctypes.byref(d), *args, 10, None, FAKE, None) == -1
    assert lib.bana_migrate_kv_blocks(ctypes.byref(_dims(block_size=8)), *args, 10, FAKE, FAKE, None) == -2
    assert lib.bana_migrate_kv_blocks(ctypes.byref(_dims(batch=70000)), *args, 10, FAKE, FAKE, None) == -2


def test_heads_rejects_bad_ranges(lib):
    d = _dims()  # 2 kv heads

    def heads(h0, h1, dd=d):
        return lib.bana_decode_attn_heads(ctypes.byref(dd), *[FAKE] * 7, h0, h1, FAKE, FAKE, None, 0, None)

    assert heads(-1, 1) == -1
    assert heads(0, 3) == -1
    assert heads(2, 1) == -1
    assert heads(1, 1) == 0  # empty head range: nothing to do, no launch
    assert heads(0, 2, _dims(head_dim=64)) == -2
    assert lib.bana_decode_attn_heads(ctypes.byref(d), *[FAKE] * 7, 0, 2, None, FAKE, None, 0, None) == -1


def test_validate_rejects_bad_arguments(lib):
    d = _dims()
    assert lib.bana_validate_ranges(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 0, FAKE, None) == -1
    for i in range(5):
        a = [FAKE] * 5
        a[i] = None
        assert lib.bana_validate_ranges(ctypes.byref(d), *a[:4], 1, a[4], None) == -1, i
    assert lib.bana_validate_ranges(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 70000, FAKE, None) == -2


def test_copy_rejects_bad_arguments(lib):
    assert lib.bana_copy_async(None, FAKE, 64, None) == -1
    assert lib.bana_copy_async(FAKE, None, 64, None) == -1
    assert lib.bana_copy_async(FAKE, FAKE, 24, None) == -1
    assert lib.bana_copy_async(ctypes.c_void_p(0x100008), FAKE, 64, None) == -1


def test_negative_total_hint_rejected(lib):
    d = _dims()
    d.total_range_tokens = -1
    assert _partial(lib, d) == -1


def test_workspace_sizing_follows_the_plan(lib):
    # 64 sequences x 8 kv heads fill the GPU with one chunk per (sequence, kv head): no workspace
    d = bana.make_dims(64, 32, 8, 256, 19661, max_range_tokens=2864)
    assert lib.bana_decode_attn_workspace_bytes(ctypes.byref(d)) == 0
    # 8 sequences x 8 kv heads of long ranges: split into chunks, one fp32 row + lse per chunk row
    d = bana.make_dims(8, 32, 8, 8192, 50000, max_range_tokens=60000)
    ws = lib.bana_decode_attn_workspace_bytes(ctypes.byref(d))
    assert ws > 0 and ws % 256 == 0
    nc = round(ws / (8 * 32 * 129 * 4))
    assert nc >= 2 and ws >= nc * 8 * 32 * 129 * 4
    # an explicit chunk hint sizes the workspace exactly
    d = bana.make_dims(8, 32, 8, 8192, 50000, chunks_hint=4)
    assert lib.bana_decode_attn_workspace_bytes(ctypes.byref(d)) == (4 * 8 * 32 * 129 * 4 + 255) // 256 * 256


def test_gather_read_rejects_bad_arguments(lib):
    d = _dims()
    args = [FAKE] * 5
    assert lib.bana_debug_gather_read(ctypes.byref(d), *args, 0, FAKE, None) == -1
    assert lib.bana_debug_gather_read(None, *args, 1, FAKE, None) == -1
    for i in range(5):
        a = list(args)
        a[i] = None
        assert lib.bana_debug_gather_read(ctypes.byref(d), *a, 1, FAKE, None) == -1, i
    assert lib.bana_debug_gather_read(ctypes.byref(d), *args, 1, None, None) == -1
    assert lib.bana_debug_gather_read(ctypes.byref(d), ctypes.c_void_p(0x100008), *args[1:], 1, FAKE, None) == -1
    assert lib.bana_debug_gather_read(ctypes.byref(_dims(head_dim=64)), *args, 1, FAKE, None) == -2


def test_stream_read_rejects_bad_arguments(lib):
    assert lib.bana_debug_stream_read(None, 4096, 8, FAKE, None) == -1
    assert lib.bana_debug_stream_read(FAKE, 4096, 8, None, None) == -1
    assert lib.bana_debug_stream_read(FAKE, 4100, 8, FAKE, None) == -1
    assert lib.bana_debug_stream_read(ctypes.c_void_p(0x100008), 4096, 8, FAKE, None) == -1
    assert lib.bana_debug_stream_read(FAKE, 4096, 0, FAKE, None) == -1
    assert lib.bana_debug_stream_read(FAKE, 4096, 65537, FAKE, None) == -1


def test_sizes_beyond_32_bit_indices_are_unsupported(lib):
    big = _dims(batch=1 << 20, num_q_heads=4096, num_kv_heads=4096, max_blocks_per_seq=1)
    assert _partial(lib, big) == -2
    assert lib.bana_merge_partials(ctypes.byref(big), FAKE, FAKE, 2, FAKE, None, None) == -2
    assert _partial(lib, _dims(batch=1 << 16, max_blocks_per_seq=1 << 16)) == -2
    assert _partial(lib, _dims(batch=1, max_blocks_per_seq=1 << 28)) == -2
    # a launch counts work-items in 32 bits: batch x num_q_heads stays below 2^26
    at = _dims(batch=1 << 20, num_q_heads=64, num_kv_heads=8)
    below = _dims(batch=(1 << 20) - 1, num_q_heads=64, num_kv_heads=8)
    assert _partial(lib, at) == -2
    assert lib.bana_merge_partials(ctypes.byref(at), FAKE, FAKE, 2, FAKE, None, None) == -2
    # just below the limit the dims pass, and n_parts = 0 is the error reported
    assert lib.bana_merge_partials(ctypes.byref(below), FAKE, FAKE, 0, FAKE, None, None) == -1
    # fused: a sequence's blocks over all its ranges are counted in 32 bits
    wide = _dims(batch=1, max_blocks_per_seq=1 << 26)
    assert lib.bana_decode_attn_fused(ctypes.byref(wide), *[FAKE] * 7, 64, FAKE, FAKE, None, 0, None) == -2


def _balanced_bytes(B, Hq, Hkv):
    K = max(1, 2048 // (8 * Hkv)) * 8  # 2048 wavefronts over the kv heads, 8 per workgroup
    pieces = (K + B) * Hq
    lse = (pieces * 128 * 4 + 255) // 256 * 256
    prefix = (lse + pieces * 4 + 255) // 256 * 256
    return (prefix + (B + 1) * 4 + 255) // 256 * 256


def test_plan_choice_between_chunked_and_balanced(lib):
    """The balanced launch is chosen for an uneven spread over few active (sequence, kv head) pairs,
    and only there; its workspace holds K + B piece rows per query head and the prefix sums."""
    def ws(B, Hq, Hkv, max_tok, total_tok, **kw):
        d = bana.make_dims(B, Hq, Hkv, 8192, 100000, max_range_tokens=max_tok, total_range_tokens=total_tok, **kw)
        return lib.bana_decode_attn_workspace_bytes(ctypes.byref(d))

    # 8 sequences, longest 3 x the mean (a long-context partition): balanced
    assert ws(8, 32, 8, 77000, 8 * 25000) == _balanced_bytes(8, 32, 8)
    # a 1.3 x spread (long's fused call): balanced
    assert ws(8, 32, 8, 100000, 8 * 77000) == _balanced_bytes(8, 32, 8)
    # a 1.2 x spread: chunked (chunk partials [nc][B][Hq])
    w = ws(8, 32, 8, 92000, 8 * 77000)
    rows = 8 * 32
    assert w != _balanced_bytes(8, 32, 8)
    assert any(w == (nc * rows * 129 * 4 + 255) // 256 * 256 for nc in range(2, 257))
    # many pairs (256 sequences x 8 kv heads), heavy tail: chunked, never balanced
    assert ws(256, 32, 8, 7568, 256 * 1400) != _balanced_bytes(256, 32, 8)
    # 256 sequences x 4 kv heads (a head half of the same): 1024 pairs, balanced
    assert ws(256, 16, 4, 7568, 256 * 1400) == _balanced_bytes(256, 16, 4)
    # 256 sequences of which 61 have a range (a migrated partition): the active pairs decide
    assert ws(256, 32, 8, 14000, 61 * 1400, nonempty_ranges=61) == _balanced_bytes(256, 32, 8)
    assert ws(256, 32, 8, 14000, 61 * 1400) != _balanced_bytes(256, 32, 8)
    # batch up to 2048 takes the balanced hint; above, it falls back to the chunked plan
    assert ws(100, 8, 2, 5000, 100 * 300, plan_hint=2) == _balanced_bytes(100, 8, 2)
    assert ws(2048, 8, 2, 300, 2048 * 100, plan_hint=2) == _balanced_bytes(2048, 8, 2)
    assert ws(2049, 8, 2, 300, 2049 * 100, plan_hint=2) != _balanced_bytes(2049, 8, 2)
    # plan_hint 2 forces it, plan_hint 1 forbids it
    assert ws(4, 8, 2, 1000, 4 * 900, plan_hint=2) == _balanced_bytes(4, 8, 2)
    assert ws(8, 32, 8, 77000, 8 * 25000, plan_hint=1) != _balanced_bytes(8, 32, 8)
    # too few blocks for one round of wavefronts: no balanced launch without the hint
    assert ws(4, 8, 2, 1000, 4 * 300) != _balanced_bytes(4, 8, 2)
    # a table too wide for the balanced schedule's 32-bit block counts (batch x 64 ranges x width):
    # the hint falls back to the chunked plan
    wide = bana.make_dims(4, 8, 2, 1 << 23, 100000, max_range_tokens=1000, total_range_tokens=4 * 900, plan_hint=2)
    assert lib.bana_decode_attn_workspace_bytes(ctypes.byref(wide)) != _balanced_bytes(4, 8, 2)
    narrow = bana.make_dims(4, 8, 2, (1 << 23) - 1, 100000, max_range_tokens=1000, total_range_tokens=4 * 900,
                            plan_hint=2)
    assert lib.bana_decode_attn_workspace_bytes(ctypes.byref(narrow)) == _balanced_bytes(4, 8, 2)


def _c_build_module():
    import importlib.util

    spec = importlib.util.spec_from_file_location("abi_roundtrip_build", os.path.join(ROOT, "tests", "c", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_plain_c_caller_builds_against_the_header(lib):
    """The C ABI is usable from C: a program including only include/bana.h (and HIP's runtime API)
    compiles with -Wall and links libbana.so; tests/test_gpu_parity.py runs it on the GPU."""
    import oracle

    if not os.path.exists(oracle.LIB_PATH):
        oracle.build()
    path = _c_build_module().build()
    assert os.access(path, os.X_OK)


def test_noalloc_checks_arguments_and_refuses_plans_beyond_the_static_scratch(lib):
    def noalloc(dd, ptrs=None):
        p = ptrs or [FAKE] * 9
        return lib.bana_decode_attn_partial_noalloc(ctypes.byref(dd) if dd is not None else None, *p, None)

    assert noalloc(None) == -1
    assert noalloc(_dims(head_dim=64)) == -2
    for i in range(9):
        ptrs = [FAKE] * 9
        ptrs[i] = None
        assert noalloc(_dims(), ptrs) == -1, i
    ptrs = [FAKE] * 9
    ptrs[0] = ctypes.c_void_p(0x100008)
    assert noalloc(_dims(), ptrs) == -1
    # 256 chunk partials of 64 x 32 rows need far more than the static scratch: refused before any HIP call.
    d = _dims(batch=64, num_q_heads=32, num_kv_heads=8, chunks_hint=256, waves_hint=1)
    need = lib.bana_decode_attn_workspace_bytes(ctypes.byref(d))
    assert need > bana.STATIC_SCRATCH_BYTES
    assert noalloc(d) == -2
    msg = lib.bana_last_error().decode()
    assert msg.startswith("bana_decode_attn_partial_noalloc:")
    assert str(need) in msg and str(bana.STATIC_SCRATCH_BYTES) in msg


def test_static_scratch_size_matches_the_header():
    text = open(HEADER).read()
    m = re.search(r"#define BANA_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == bana.STATIC_SCRATCH_BYTES


def test_fused_copies_rejects_bad_arguments(lib):
    d = _dims()

    def call(n_copies, copies=None, n_parts=2, dd=d):
        arr = copies if copies is not None else (bana.bana_copy * 1)(bana.bana_copy(0x200000, 0x300000, 64))
        return lib.bana_decode_attn_fused_copies(ctypes.byref(dd) if dd is not None else None, *[FAKE] * 7, n_parts,
                                                 FAKE, FAKE, None, 0, arr, n_copies, None)

    assert call(1, n_parts=0) == -1
    assert call(-1) == -1
    assert call(9, (bana.bana_copy * 9)()) == -2
    assert call(1, dd=None) == -1
    assert call(1, dd=_dims(head_dim=64)) == -2
    assert lib.bana_decode_attn_fused_copies(ctypes.byref(d), *[FAKE] * 7, 2, FAKE, FAKE, None, 0, None, 1,
                                             None) == -1
    for bad in (bana.bana_copy(0, 0x300000, 64), bana.bana_copy(0x200000, 0, 64),
                bana.bana_copy(0x200008, 0x300000, 64), bana.bana_copy(0x200000, 0x300004, 64),
                bana.bana_copy(0x200000, 0x300000, 24)):
        assert call(1, (bana.bana_copy * 1)(bad)) == -1
    # a zero-byte copy is skipped, whatever its pointers; the call then fails only on n_parts
    assert call(1, (bana.bana_copy * 1)(bana.bana_copy(0, 0, 0)), n_parts=0) == -1


def test_wave_timeline_hooks_are_unsupported_in_the_product_build(lib):
    """The timeline entry points exist in every build; only the measurement build
    (libbana_timeline.so) implements them.  The product build refuses before any HIP call."""
    import numpy as np

    out = np.zeros((4, 4), dtype=np.uint64)
    assert lib.bana_debug_wave_timeline_clear(None) == bana.BANA_ERR_UNSUPPORTED
    assert lib.bana_debug_wave_timeline_read(out.ctypes.data_as(ctypes.c_void_p), 4, None) == bana.BANA_ERR_UNSUPPORTED
    assert lib.bana_debug_wave_timeline_read(None, 4, None) == bana.BANA_ERR_INVALID
    assert lib.bana_debug_wave_timeline_read(out.ctypes.data_as(ctypes.c_void_p), bana.TIMELINE_SLOTS + 1,
                                             None) == bana.BANA_ERR_INVALID
    with pytest.raises(bana.BanaError):
        bana.bana_debug_wave_timeline_read(4, stream=0)
    # the header's slot count and the binding's agree
    text = open(HEADER).read()
    assert re.search(r"#define BANA_TIMELINE_SLOTS \(1 << 18\)", text) and bana.TIMELINE_SLOTS == 1 << 18
