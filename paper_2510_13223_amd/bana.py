"""Python binding of libbana.so (ctypes).

Argument marshalling only: every function checks tensor dtypes, shapes,
devices and contiguity, then passes raw device pointers and the HIP stream
handle to the C ABI declared in ``include/bana.h``.  All arithmetic runs in
the library's HIP kernels; there is no fallback path, and a missing library
raises.  PyTorch only provides device memory and streams.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("BANA_LIBRARY") or os.path.join(_PKG, "libbana.so")
RACECHECK_LIB_PATH = os.path.join(_PKG, "libbana_racecheck.so")
TIMELINE_LIB_PATH = os.path.join(_PKG, "libbana_timeline.so")
TIMELINE_SLOTS = 1 << 18  # BANA_TIMELINE_SLOTS

HEAD_DIM = 128
BLOCK_SIZE = 16

BANA_OK = 0
BANA_ERR_INVALID = -1
BANA_ERR_UNSUPPORTED = -2
BANA_ERR_DEVICE = -3


class bana_dims(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("num_blocks", ctypes.c_int64),
        ("max_range_tokens", ctypes.c_int32),
        ("waves_hint", ctypes.c_int32),
        ("chunks_hint", ctypes.c_int32),
        ("plan_hint", ctypes.c_int32),
        ("total_range_tokens", ctypes.c_int64),
        ("seq_order", ctypes.c_void_p),
        ("nonempty_ranges", ctypes.c_int32),
    ]


class bana_copy(ctypes.Structure):
    _fields_ = [("dst", ctypes.c_void_p), ("src", ctypes.c_void_p), ("bytes", ctypes.c_size_t)]


class BanaError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str = ""):
        self.status = status
        if not detail and status == BANA_ERR_DEVICE:
            detail = lib().bana_last_error().decode()
        msg = f"{what}: {lib().bana_status_string(status).decode()} ({status})"
        super().__init__(msg + (f": {detail}" if detail else ""))


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libbana.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        _lib = load(LIB_PATH)
    return _lib


def load(path: str) -> ctypes.CDLL:
    """A build of the library at ``path`` with the C ABI's argument types set (raises if missing).
    Loaded with local symbol scope, so a second build (the LDS race-check one) keeps its own code."""
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2510_13223_amd.build`")
    L = ctypes.CDLL(path, mode=os.RTLD_LOCAL | os.RTLD_NOW)
    P = ctypes.c_void_p
    D = ctypes.POINTER(bana_dims)
    L.bana_decode_attn_partial.argtypes = [D, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    L.bana_decode_attn_partial.restype = ctypes.c_int
    L.bana_decode_attn_partial_noalloc.argtypes = [D, P, P, P, P, P, P, P, P, P, P]
    L.bana_decode_attn_partial_noalloc.restype = ctypes.c_int
    L.bana_decode_attn_workspace_bytes.argtypes = [D]
    L.bana_decode_attn_workspace_bytes.restype = ctypes.c_size_t
    L.bana_decode_attn_fused.argtypes = [D, P, P, P, P, P, P, P, ctypes.c_int32, P, P, P, ctypes.c_size_t, P]
    L.bana_decode_attn_fused.restype = ctypes.c_int
    L.bana_decode_attn_fused_copies.argtypes = [D, P, P, P, P, P, P, P, ctypes.c_int32, P, P, P, ctypes.c_size_t,
                                                ctypes.POINTER(bana_copy), ctypes.c_int32, P]
    L.bana_decode_attn_fused_copies.restype = ctypes.c_int
    L.bana_merge_partials.argtypes = [D, P, P, ctypes.c_int32, P, P, P]
    L.bana_merge_partials.restype = ctypes.c_int
    L.bana_status_string.argtypes = [ctypes.c_int]
    L.bana_status_string.restype = ctypes.c_char_p
    L.bana_last_error.argtypes = []
    L.bana_last_error.restype = ctypes.c_char_p
    L.bana_decode_attn_heads.argtypes = [D, P, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32, P, P, P,
                                         ctypes.c_size_t, P]
    L.bana_decode_attn_heads.restype = ctypes.c_int
    L.bana_migrate_kv_blocks.argtypes = [D, P, P, P, P, P, P, ctypes.c_int64, P, P, P]
    L.bana_migrate_kv_blocks.restype = ctypes.c_int
    L.bana_validate_ranges.argtypes = [D, P, P, P, P, ctypes.c_int32, P, P]
    L.bana_validate_ranges.restype = ctypes.c_int
    L.bana_copy_async.argtypes = [P, P, ctypes.c_size_t, P]
    L.bana_copy_async.restype = ctypes.c_int
    L.bana_debug_kv_rows.argtypes = [D, P, P, P, P, P]
    L.bana_debug_kv_rows.restype = ctypes.c_int
    L.bana_debug_gather_read.argtypes = [D, P, P, P, P, P, ctypes.c_int32, P, P]
    L.bana_debug_gather_read.restype = ctypes.c_int
    L.bana_debug_stream_read.argtypes = [P, ctypes.c_size_t, ctypes.c_int32, P, P]
    L.bana_debug_stream_read.restype = ctypes.c_int
    L.bana_debug_wave_timeline_clear.argtypes = [P]
    L.bana_debug_wave_timeline_clear.restype = ctypes.c_int
    L.bana_debug_wave_timeline_read.argtypes = [P, ctypes.c_size_t, P]
    L.bana_debug_wave_timeline_read.restype = ctypes.c_int
    return L


def make_dims(batch: int, num_q_heads: int, num_kv_heads: int, max_blocks_per_seq: int, num_blocks: int,
              max_range_tokens: int = 0, waves_hint: int = 0, chunks_hint: int = 0,
              total_range_tokens: int = 0, seq_order: Optional[torch.Tensor] = None,
              plan_hint: int = 0, nonempty_ranges: int = 0) -> bana_dims:
    """Dims for a call; ``seq_order`` (device int32 [batch], kept alive by the caller) is a dispatch hint,
    ``plan_hint`` 0 / 1 / 2 = library's choice / chunked launch / balanced launch, ``nonempty_ranges``
    the number of sequences with a non-empty range (0 = unknown)."""
    if seq_order is not None:
        _need(seq_order, "seq_order", torch.int32, (batch,))
    return bana_dims(batch, num_q_heads, num_kv_heads, HEAD_DIM, BLOCK_SIZE, max_blocks_per_seq, num_blocks,
                     max_range_tokens, waves_hint, chunks_hint, plan_hint, total_range_tokens,
                     None if seq_order is None else seq_order.data_ptr(), nonempty_ranges)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor, got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _check_dims(dims: bana_dims, q: torch.Tensor, k_cache: torch.Tensor, block_table: torch.Tensor) -> None:
    """Caller-built dims must describe the tensors passed with them (the kernels index by the dims)."""
    B, Hq, D = q.shape
    nb, Hkv = k_cache.shape[0], k_cache.shape[1]
    got = (dims.batch, dims.num_q_heads, dims.num_kv_heads, dims.head_dim, dims.max_blocks_per_seq, dims.num_blocks)
    want = (B, Hq, Hkv, D, block_table.shape[1], nb)
    if got != want:
        raise ValueError(f"dims (batch, Hq, Hkv, head_dim, max_blocks_per_seq, num_blocks) = {got} "
                         f"do not match the tensors {want}")


def dims_for(q: torch.Tensor, k_cache: torch.Tensor, block_table: torch.Tensor, max_range_tokens: int = 0,
             waves_hint: int = 0, chunks_hint: int = 0, total_range_tokens: int = 0) -> bana_dims:
    B, Hq, D = q.shape
    nb, Hkv, _, bs, _ = k_cache.shape
    return bana_dims(B, Hq, Hkv, D, bs, block_table.shape[1], nb, max_range_tokens, waves_hint, chunks_hint, 0,
                     total_range_tokens)


def bana_decode_attn_workspace_bytes(dims: bana_dims) -> int:
    return int(lib().bana_decode_attn_workspace_bytes(ctypes.byref(dims)))


def head_range_dims(dims: bana_dims, kv_head_begin: int, kv_head_end: int) -> bana_dims:
    """Dims of the sub-problem of kv heads [kv_head_begin, kv_head_end): what bana_decode_attn_heads
    plans for, and what sizes its workspace."""
    G = dims.num_q_heads // dims.num_kv_heads
    sub = bana_dims.from_buffer_copy(dims)
    sub.num_kv_heads = kv_head_end - kv_head_begin
    sub.num_q_heads = G * (kv_head_end - kv_head_begin)
    return sub


def bana_decode_attn_partial(q, k_cache, v_cache, block_table, seq_lens, kv_range_begin, kv_range_end,
                             out_partial, lse, workspace: Optional[torch.Tensor] = None, stream=None,
                             dims: Optional[bana_dims] = None, max_range_tokens: int = 0) -> None:
    """Partial attention of one partition; see ``bana_decode_attn_partial`` in include/bana.h."""
    B, Hq, D = _check_attn_inputs(q, k_cache, v_cache, block_table, seq_lens)
    _need(kv_range_begin, "kv_range_begin", torch.int32, (B,))
    _need(kv_range_end, "kv_range_end", torch.int32, (B,))
    _need(out_partial, "out_partial", torch.float32, (B, Hq, D))
    _need(lse, "lse", torch.float32, (B, Hq))
    _same_device(q, kv_range_begin, kv_range_end, out_partial, lse, workspace)
    ws_bytes = 0
    if workspace is not None:
        _need(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    if dims is None:
        dims = dims_for(q, k_cache, block_table, max_range_tokens)
    _check_dims(dims, q, k_cache, block_table)
    st = lib().bana_decode_attn_partial(
        ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
        _ptr(kv_range_begin), _ptr(kv_range_end), _ptr(out_partial), _ptr(lse), _ptr(workspace), ws_bytes,
        _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_decode_attn_partial")


STATIC_SCRATCH_BYTES = 64 << 20  # BANA_STATIC_SCRATCH_BYTES


def bana_decode_attn_partial_noalloc(q, k_cache, v_cache, block_table, seq_lens, kv_range_begin, kv_range_end,
                                     out_partial, lse, stream=None, dims: Optional[bana_dims] = None,
                                     max_range_tokens: int = 0) -> None:
    """``bana_decode_attn_partial`` with the library's static device scratch in place of a workspace
    (for callers that cannot allocate); see ``bana_decode_attn_partial_noalloc`` in include/bana.h.
    Calls that may overlap on one device share that scratch and must be serialised."""
    B, Hq, D = _check_attn_inputs(q, k_cache, v_cache, block_table, seq_lens)
    _need(kv_range_begin, "kv_range_begin", torch.int32, (B,))
    _need(kv_range_end, "kv_range_end", torch.int32, (B,))
    _need(out_partial, "out_partial", torch.float32, (B, Hq, D))
    _need(lse, "lse", torch.float32, (B, Hq))
    _same_device(q, kv_range_begin, kv_range_end, out_partial, lse)
    if dims is None:
        dims = dims_for(q, k_cache, block_table, max_range_tokens)
    _check_dims(dims, q, k_cache, block_table)
    st = lib().bana_decode_attn_partial_noalloc(
        ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
        _ptr(kv_range_begin), _ptr(kv_range_end), _ptr(out_partial), _ptr(lse), _stream(stream))
    if st != BANA_OK:
        text = lib().bana_last_error().decode()
        raise BanaError(st, "bana_decode_attn_partial_noalloc",
                        text if text.startswith("bana_decode_attn_partial_noalloc:") else "")


def _check_attn_inputs(q, k_cache, v_cache, block_table, seq_lens):
    if q.dim() != 3 or k_cache.dim() != 5:
        raise ValueError("q must be [B, Hq, D] and k_cache [num_blocks, Hkv, D / 8, block_size, 8]")
    B, Hq, D = q.shape
    nb, Hkv, _, bs, _ = k_cache.shape
    _need(q, "q", torch.bfloat16)
    _need(k_cache, "k_cache", torch.bfloat16, (nb, Hkv, D // 8, bs, 8))
    _need(v_cache, "v_cache", torch.bfloat16, (nb, Hkv, D, bs))
    _need(block_table, "block_table", torch.int32)
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B, max_blocks_per_seq]")
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    _same_device(q, k_cache, v_cache, block_table, seq_lens)
    return B, Hq, D


def _same_device(*tensors) -> None:
    """Every tensor of a call on one device, the current one (the library launches there)."""
    devs = {t.device for t in tensors if t is not None}
    if len(devs) != 1:
        raise ValueError(f"tensors of one call are on several devices: {sorted(map(str, devs))}")
    dev = devs.pop()
    if dev.index is not None and dev.index != torch.cuda.current_device():
        raise ValueError(f"tensors are on {dev}, but the current device is cuda:{torch.cuda.current_device()}")


def bana_decode_attn_fused(q, k_cache, v_cache, block_table, seq_lens, kv_range_begin, kv_range_end, out, lse_out,
                           workspace: Optional[torch.Tensor] = None, stream=None,
                           dims: Optional[bana_dims] = None) -> None:
    """All partitions ``kv_range_begin/end [n_parts, B]`` and their merge in one launch; see include/bana.h."""
    B, Hq, D = _check_attn_inputs(q, k_cache, v_cache, block_table, seq_lens)
    if kv_range_begin.dim() != 2 or kv_range_begin.shape[1] != B:
        raise ValueError("kv_range_begin must be [n_parts, B]")
    n = kv_range_begin.shape[0]
    _need(kv_range_begin, "kv_range_begin", torch.int32, (n, B))
    _need(kv_range_end, "kv_range_end", torch.int32, (n, B))
    _need(out, "out", torch.float32, (B, Hq, D))
    _need(lse_out, "lse_out", torch.float32, (B, Hq))
    _same_device(q, kv_range_begin, kv_range_end, out, lse_out, workspace)
    ws_bytes = 0
    if workspace is not None:
        _need(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    if dims is None:
        dims = dims_for(q, k_cache, block_table)
    _check_dims(dims, q, k_cache, block_table)
    st = lib().bana_decode_attn_fused(
        ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
        _ptr(kv_range_begin), _ptr(kv_range_end), n, _ptr(out), _ptr(lse_out), _ptr(workspace), ws_bytes,
        _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_decode_attn_fused")


def copy_list(copies) -> "ctypes.Array":
    """A bana_copy array from (dst tensor, src tensor) pairs (each contiguous, device or pinned host
    memory, the same number of bytes, a multiple of 16)."""
    arr = (bana_copy * len(copies))()
    for i, (dst, src) in enumerate(copies):
        for t, name in ((dst, "dst"), (src, "src")):
            if not isinstance(t, torch.Tensor) or not t.is_contiguous():
                raise ValueError(f"copy {i}: {name} must be a contiguous tensor")
            if t.device.type != "cuda" and not t.is_pinned():
                raise ValueError(f"copy {i}: {name} must be device or pinned host memory")
        nbytes = src.numel() * src.element_size()
        if dst.numel() * dst.element_size() != nbytes:
            raise ValueError(f"copy {i}: dst and src differ in size")
        arr[i] = bana_copy(dst.data_ptr(), src.data_ptr(), nbytes)
    return arr


def bana_decode_attn_fused_copies(q, k_cache, v_cache, block_table, seq_lens, kv_range_begin, kv_range_end, out,
                                  lse_out, copies=(), workspace: Optional[torch.Tensor] = None, stream=None,
                                  dims: Optional[bana_dims] = None) -> None:
    """The fused call with up to 8 (dst, src) copies carried by the same launch; see include/bana.h."""
    B, Hq, D = _check_attn_inputs(q, k_cache, v_cache, block_table, seq_lens)
    if kv_range_begin.dim() != 2 or kv_range_begin.shape[1] != B:
        raise ValueError("kv_range_begin must be [n_parts, B]")
    n = kv_range_begin.shape[0]
    _need(kv_range_begin, "kv_range_begin", torch.int32, (n, B))
    _need(kv_range_end, "kv_range_end", torch.int32, (n, B))
    _need(out, "out", torch.float32, (B, Hq, D))
    _need(lse_out, "lse_out", torch.float32, (B, Hq))
    _same_device(q, kv_range_begin, kv_range_end, out, lse_out, workspace)
    ws_bytes = 0
    if workspace is not None:
        _need(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    if dims is None:
        dims = dims_for(q, k_cache, block_table)
    _check_dims(dims, q, k_cache, block_table)
    arr = copy_list(list(copies))
    st = lib().bana_decode_attn_fused_copies(
        ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
        _ptr(kv_range_begin), _ptr(kv_range_end), n, _ptr(out), _ptr(lse_out), _ptr(workspace), ws_bytes, arr,
        len(arr), _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_decode_attn_fused_copies")


def bana_decode_attn_heads(q, k_cache, v_cache, block_table, seq_lens, kv_range_begin, kv_range_end,
                           kv_head_begin: int, kv_head_end: int, out, lse, workspace: Optional[torch.Tensor] = None,
                           stream=None, dims: Optional[bana_dims] = None) -> None:
    """Head-split partition: the kv heads [kv_head_begin, kv_head_end) only; see include/bana.h.

    The workspace is sized by ``bana_decode_attn_workspace_bytes(head_range_dims(dims, begin, end))``.
    """
    B, Hq, D = _check_attn_inputs(q, k_cache, v_cache, block_table, seq_lens)
    _need(kv_range_begin, "kv_range_begin", torch.int32, (B,))
    _need(kv_range_end, "kv_range_end", torch.int32, (B,))
    _need(out, "out", torch.float32, (B, Hq, D))
    _need(lse, "lse", torch.float32, (B, Hq))
    _same_device(q, kv_range_begin, kv_range_end, out, lse, workspace)
    ws_bytes = 0
    if workspace is not None:
        _need(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    if dims is None:
        dims = dims_for(q, k_cache, block_table)
    _check_dims(dims, q, k_cache, block_table)
    st = lib().bana_decode_attn_heads(
        ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
        _ptr(kv_range_begin), _ptr(kv_range_end), int(kv_head_begin), int(kv_head_end), _ptr(out), _ptr(lse),
        _ptr(workspace), ws_bytes, _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_decode_attn_heads")


def bana_merge_partials(out_partials, lses, out, lse_out: Optional[torch.Tensor] = None, stream=None) -> None:
    """Log-sum-exp merge of ``out_partials [n_parts, B, Hq, D]`` / ``lses [n_parts, B, Hq]``."""
    if out_partials.dim() != 4:
        raise ValueError("out_partials must be [n_parts, B, Hq, D]")
    n, B, Hq, D = out_partials.shape
    _need(out_partials, "out_partials", torch.float32)
    _need(lses, "lses", torch.float32, (n, B, Hq))
    _need(out, "out", torch.float32, (B, Hq, D))
    if lse_out is not None:
        _need(lse_out, "lse_out", torch.float32, (B, Hq))
    _same_device(out_partials, lses, out, lse_out)
    dims = bana_dims(B, Hq, 1, D, BLOCK_SIZE, 1, 1, 0, 0, 0, 0, 0)
    st = lib().bana_merge_partials(ctypes.byref(dims), _ptr(out_partials), _ptr(lses), n, _ptr(out), _ptr(lse_out),
                                   _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_merge_partials")


def bana_migrate_kv_blocks(src_k, src_v, src_table, dst_k, dst_v, dst_table, blk_begin, blk_end, stream=None,
                           max_range_tokens: int = 0) -> None:
    """Copy the K/V tiles of logical blocks [blk_begin, blk_end) between pools; see include/bana.h."""
    if src_k.dim() != 5 or dst_k.dim() != 5:
        raise ValueError("k pools must be [num_blocks, Hkv, D / 8, block_size, 8]")
    nb, Hkv, _, bs, _ = src_k.shape
    nbd = dst_k.shape[0]
    B, mb = src_table.shape
    _need(src_k, "src_k", torch.bfloat16, (nb, Hkv, HEAD_DIM // 8, bs, 8))
    _need(src_v, "src_v", torch.bfloat16, (nb, Hkv, HEAD_DIM, bs))
    _need(dst_k, "dst_k", torch.bfloat16, (nbd, Hkv, HEAD_DIM // 8, bs, 8))
    _need(dst_v, "dst_v", torch.bfloat16, (nbd, Hkv, HEAD_DIM, bs))
    _need(src_table, "src_table", torch.int32, (B, mb))
    _need(dst_table, "dst_table", torch.int32, (B, mb))
    _need(blk_begin, "blk_begin", torch.int32, (B,))
    _need(blk_end, "blk_end", torch.int32, (B,))
    _same_device(src_k, src_v, src_table, dst_k, dst_v, dst_table, blk_begin, blk_end)
    dims = bana_dims(B, Hkv, Hkv, HEAD_DIM, bs, mb, nb, max_range_tokens, 0, 0, 0, 0)
    st = lib().bana_migrate_kv_blocks(ctypes.byref(dims), _ptr(src_k), _ptr(src_v), _ptr(src_table), _ptr(dst_k),
                                      _ptr(dst_v), _ptr(dst_table), nbd, _ptr(blk_begin), _ptr(blk_end),
                                      _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_migrate_kv_blocks")


def bana_validate_ranges(block_table, seq_lens, kv_range_begin, kv_range_end, num_blocks: int, result,
                         stream=None) -> None:
    """Device-side precondition check; ``result`` (int32 [1]) receives 0 or a rule code (include/bana.h)."""
    B, mb = block_table.shape
    if kv_range_begin.dim() == 1:
        kv_range_begin, kv_range_end = kv_range_begin[None], kv_range_end[None]
    n = kv_range_begin.shape[0]
    _need(block_table, "block_table", torch.int32)
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    _need(kv_range_begin, "kv_range_begin", torch.int32, (n, B))
    _need(kv_range_end, "kv_range_end", torch.int32, (n, B))
    _need(result, "result", torch.int32, (1,))
    _same_device(block_table, seq_lens, kv_range_begin, kv_range_end, result)
    dims = bana_dims(B, 1, 1, HEAD_DIM, BLOCK_SIZE, mb, num_blocks, 0, 0, 0, 0, 0)
    st = lib().bana_validate_ranges(ctypes.byref(dims), _ptr(block_table), _ptr(seq_lens), _ptr(kv_range_begin),
                                    _ptr(kv_range_end), n, _ptr(result), _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_validate_ranges")


def bana_debug_kv_rows(block_table, kv_range_begin, kv_range_end, num_blocks: int, num_kv_heads: int, rows_out,
                       stream=None) -> None:
    """K rows the partial kernel reads per (b, g, t); see include/bana.h."""
    B, mb = block_table.shape
    _need(block_table, "block_table", torch.int32)
    _need(kv_range_begin, "kv_range_begin", torch.int32, (B,))
    _need(kv_range_end, "kv_range_end", torch.int32, (B,))
    _need(rows_out, "rows_out", torch.int64, (B, num_kv_heads, mb * BLOCK_SIZE))
    _same_device(block_table, kv_range_begin, kv_range_end, rows_out)
    dims = bana_dims(B, num_kv_heads, num_kv_heads, HEAD_DIM, BLOCK_SIZE, mb, num_blocks, 0, 0, 0, 0, 0)
    st = lib().bana_debug_kv_rows(ctypes.byref(dims), _ptr(block_table), _ptr(kv_range_begin), _ptr(kv_range_end),
                                  _ptr(rows_out), _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_debug_kv_rows")


def bana_debug_gather_read(k_cache, v_cache, block_table, kv_range_begin, kv_range_end, sink, stream=None) -> None:
    """K/V read of the ranges ``[n_parts, B]`` with no arithmetic; ``sink`` uint32 as int32 [B, Hkv].

    See ``bana_debug_gather_read`` in include/bana.h (sink[b][g] is the XOR of
    the 32-bit words of every covered K and V tile of (b, g)).
    """
    nb, Hkv, D8, bs, _ = k_cache.shape
    _need(k_cache, "k_cache", torch.bfloat16, (nb, Hkv, D8, bs, 8))
    _need(v_cache, "v_cache", torch.bfloat16, (nb, Hkv, D8 * 8, bs))
    _need(block_table, "block_table", torch.int32)
    B, mb = block_table.shape
    if kv_range_begin.dim() != 2 or kv_range_begin.shape[1] != B:
        raise ValueError("kv_range_begin must be [n_parts, B]")
    n = kv_range_begin.shape[0]
    _need(kv_range_begin, "kv_range_begin", torch.int32, (n, B))
    _need(kv_range_end, "kv_range_end", torch.int32, (n, B))
    _need(sink, "sink", torch.int32, (B, Hkv))
    _same_device(k_cache, v_cache, block_table, kv_range_begin, kv_range_end, sink)
    dims = bana_dims(B, Hkv, Hkv, D8 * 8, bs, mb, nb, 0, 0, 0, 0, 0)
    st = lib().bana_debug_gather_read(ctypes.byref(dims), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                      _ptr(kv_range_begin), _ptr(kv_range_end), n, _ptr(sink), _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_debug_gather_read")


def bana_debug_stream_read(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """Front-to-back read of the bytes of ``buf`` (contiguous device tensor, size a multiple of 16) by
    ``sink.numel()`` workgroups; ``sink`` uint32 as int32 [n_groups].

    See ``bana_debug_stream_read`` in include/bana.h (the XOR of the sink words is the XOR of the
    buffer's 32-bit words).
    """
    if not isinstance(buf, torch.Tensor) or buf.device.type != "cuda" or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    _need(sink, "sink", torch.int32)
    _same_device(buf, sink)
    nbytes = buf.numel() * buf.element_size()
    st = lib().bana_debug_stream_read(_ptr(buf), nbytes, sink.numel(), _ptr(sink), _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_debug_stream_read")


def bana_copy_async(dst: torch.Tensor, src: torch.Tensor, stream=None) -> None:
    """Stream-ordered copy of all bytes of ``src`` into ``dst`` by the library's copy kernel.

    Both contiguous, the same number of bytes (a multiple of 16), on the device or in pinned host
    memory; see ``bana_copy_async`` in include/bana.h.
    """
    for t, name in ((dst, "dst"), (src, "src")):
        if not isinstance(t, torch.Tensor) or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous tensor")
        if t.device.type != "cuda" and not t.is_pinned():
            raise ValueError(f"{name} must be device or pinned host memory")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("dst and src differ in size")
    st = lib().bana_copy_async(_ptr(dst), _ptr(src), nbytes, _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_copy_async")


def bana_debug_wave_timeline_clear(stream=None, library: Optional[ctypes.CDLL] = None) -> None:
    """Reset the wavefront timeline of the timeline build (``library``, default the loaded one).

    See ``bana_debug_wave_timeline_clear`` in include/bana.h; raises BanaError (BANA_ERR_UNSUPPORTED)
    on the product build.
    """
    st = (library or lib()).bana_debug_wave_timeline_clear(_stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_debug_wave_timeline_clear")


def bana_debug_wave_timeline_read(n_slots: int, stream=None, library: Optional[ctypes.CDLL] = None):
    """Slots [0, n_slots) of the wavefront timeline as a uint64 numpy array [n_slots, 4] (clock ticks
    of 10 ns: entry, schedule ready, first block, exit; UINT64_MAX where nothing was written)."""
    import numpy as np

    out = np.empty((n_slots, 4), dtype=np.uint64)
    st = (library or lib()).bana_debug_wave_timeline_read(out.ctypes.data_as(ctypes.c_void_p), n_slots,
                                                         _stream(stream))
    if st != BANA_OK:
        raise BanaError(st, "bana_debug_wave_timeline_read")
    return out
