"""fp64 CPU oracle for split paged decode attention.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; the product path never imports it.
The arithmetic lives in ``oracle.c`` (plain fp64 loops, OpenMP over
(sequence, head)); this module only marshals NumPy arrays into it.  Every
function follows Sec. 4.1(2) of the paper (attention-level migration: per
partition S = Q K^T, A = exp S, l = sum A, O = A / l . V, and the final
combine O = O^(1) + O^(2)), read as documented in ``oracle.c``.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")

HEAD_DIM = 128
BLOCK_SIZE = 16

_lib = None


def build(verbose: bool = False) -> str:
    """Compile oracle.c with gcc (-O2, OpenMP, no -ffast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", SRC_PATH, "-o", LIB_PATH + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # ORACLE_LIB points the tests at a deliberately broken copy of the oracle
    # (tests/test_oracle_mutants.py checks that the pins reject each one).
    path = os.environ.get("ORACLE_LIB", LIB_PATH)
    if path == LIB_PATH and not os.path.exists(LIB_PATH):
        build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int, ctypes.c_int64
    lib.oracle_partial.argtypes = [i32, i32, i32, i32, i32, i32, i64, P, P, P, P, P, P, P, P, i32, P, P, i32]
    lib.oracle_partial.restype = i32
    lib.oracle_merge.argtypes = [i32, i64, i32, P, P, P, P]
    lib.oracle_merge.restype = i32
    lib.oracle_kv_rows.argtypes = [i32, i32, i32, i32, i64, P, P, P, P]
    lib.oracle_kv_rows.restype = i32
    _lib = lib
    return lib


def _c(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def partial(q, k_cache, v_cache, block_table, seq_lens, kv_begin, kv_end,
            seqs: Optional[Sequence[int]] = None, threads: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Partial attention of one partition (out [n, Hq, D] fp64, lse [n, Hq] fp64).

    ``seqs`` selects sequences (default: all, in order); rows of the result
    follow that order.
    """
    lib = _load()
    q = _c(q, np.uint16)
    k_cache = _c(k_cache, np.uint16)
    v_cache = _c(v_cache, np.uint16)
    block_table = _c(block_table, np.int32)
    seq_lens = _c(seq_lens, np.int32)
    kv_begin = _c(kv_begin, np.int32)
    kv_end = _c(kv_end, np.int32)
    B, Hq, D = q.shape
    nb, Hkv, nchunk, bs, x = k_cache.shape
    assert nchunk * x == D and x == 8 and v_cache.shape == (nb, Hkv, D, bs)
    sel = None if seqs is None else _c(np.asarray(seqs), np.int32)
    n = B if sel is None else len(sel)
    out = np.zeros((n, Hq, D), dtype=np.float64)
    lse = np.zeros((n, Hq), dtype=np.float64)
    rc = lib.oracle_partial(B, Hq, Hkv, D, bs, block_table.shape[1], nb, _p(q), _p(k_cache), _p(v_cache),
                            _p(block_table), _p(seq_lens), _p(kv_begin), _p(kv_end), _p(sel), n,
                            _p(out), _p(lse), int(threads))
    if rc != 0:
        raise ValueError(f"oracle_partial rejected its inputs (code {rc})")
    return out, lse


def merge(outs: np.ndarray, lses: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Log-sum-exp merge of ``outs [n_parts, ..., D]`` with ``lses [n_parts, ...]``."""
    lib = _load()
    outs = _c(outs, np.float64)
    lses = _c(lses, np.float64)
    n_parts = outs.shape[0]
    D = outs.shape[-1]
    rows = int(np.prod(outs.shape[1:-1], dtype=np.int64))
    assert lses.shape == outs.shape[:-1]
    out = np.zeros(outs.shape[1:], dtype=np.float64)
    lse = np.zeros(lses.shape[1:], dtype=np.float64)
    rc = lib.oracle_merge(n_parts, rows, D, _p(outs), _p(lses), _p(out), _p(lse))
    if rc != 0:
        raise ValueError(f"oracle_merge rejected its inputs (code {rc})")
    return out, lse


def kv_rows(block_table, num_blocks: int, num_kv_heads: int, kv_begin, kv_end) -> np.ndarray:
    """K-row index per (b, g, logical token) of the table's span; -1 outside the range."""
    lib = _load()
    block_table = _c(block_table, np.int32)
    B, mb = block_table.shape
    rows = np.empty((B, num_kv_heads, mb * BLOCK_SIZE), dtype=np.int64)
    rc = lib.oracle_kv_rows(B, num_kv_heads, BLOCK_SIZE, mb, int(num_blocks), _p(block_table),
                            _p(_c(kv_begin, np.int32)), _p(_c(kv_end, np.int32)), _p(rows))
    if rc != 0:
        raise ValueError(f"oracle_kv_rows rejected its inputs (code {rc})")
    return rows


def workload_partials(w, seqs=None, threads: int = 0):
    """All partitions of a ``workloads.Workload``: (outs [P, n, Hq, D], lses [P, n, Hq])."""
    outs, lses = [], []
    for p in range(w.n_parts):
        o, l = partial(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.kv_begin[p], w.kv_end[p],
                       seqs=seqs, threads=threads)
        outs.append(o)
        lses.append(l)
    return np.stack(outs), np.stack(lses)


def workload_unsplit(w, seqs=None, threads: int = 0):
    """Attention over [0, seq_len) of every (selected) sequence, no split."""
    return partial(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, np.zeros_like(w.seq_lens),
                   w.seq_lens, seqs=seqs, threads=threads)


def migrate(src_k, src_v, src_table, dst_k, dst_v, dst_table, blk_begin, blk_end):
    """KV-block migration written out (Sec. 4.1(2), the KV transfer of attention-level migration):
    copies of the destination pools in which, for every sequence b and logical block j in
    [blk_begin[b], blk_end[b]), block dst_table[b][j] holds the K/V tiles (all kv heads) of source
    block src_table[b][j].  Returns (dst_k, dst_v)."""
    dk = np.array(dst_k, copy=True)
    dv = np.array(dst_v, copy=True)
    for b in range(len(blk_begin)):
        for j in range(int(blk_begin[b]), int(blk_end[b])):
            dk[dst_table[b][j]] = src_k[src_table[b][j]]
            dv[dst_table[b][j]] = src_v[src_table[b][j]]
    return dk, dv
