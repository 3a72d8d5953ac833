"""Seeded synthetic inputs for split paged decode attention.

This module only *draws* inputs; it contains none of the attention
arithmetic, so both the fp64 oracle and the HIP path can be fed from it
without sharing any of the method's code.

What is generated (all host NumPy arrays; bf16 values are carried as their
uint16 bit patterns because NumPy has no bfloat16):

* ``q``            uint16 [B, Hq, D]                      bf16 query of the decode step
* ``k_cache``      uint16 [num_blocks, Hkv, D/8, bs, 8]    bf16 keys; per (block, kv-head) tile, 16-byte
                                                          chunks of 8 dims, chunk-major then token
* ``v_cache``      uint16 [num_blocks, Hkv, D, bs]         bf16 values, dim-major tile per (block, kv-head)
* ``block_table``  int32  [B, max_blocks_per_seq]          logical block -> physical block, -1 when unused
* ``seq_lens``     int32  [B]                              tokens in the cache, current token included
* ``kv_begin``     int32  [n_parts, B]                     partition p of sequence b covers tokens
* ``kv_end``       int32  [n_parts, B]                     [kv_begin[p, b], kv_end[p, b])

The paged, block-level KV layout is the one the serving system builds on
(block-level KV management, Related Work); the split of each sequence's
blocks into a local partition and migrated partitions follows the
attention-level migration of Sec. 4.1(2) read as a split along token blocks.

Recipe (every draw comes from its own PCG64 stream keyed by
``(seed, config id, stream id[, chunk])`` so the arrays do not depend on the
number of threads used):

* Q, K, V ~ N(0, 1) in float32, rounded to bf16 round-to-nearest-even.
  ``tiny`` scales Q by 1/sqrt(128) before rounding; ``fine`` adds one
  N(0, 4) bias vector per kv-head to every key before rounding.
* Physical blocks: a pool of ceil(1.2 * sum_b n_b) blocks, assigned by one
  random permutation in logical (sequence, block) order.  Blocks no sequence
  uses, and the slots of a sequence's last block past ``seq_len``, hold a
  quiet-NaN bf16 poison pattern, so any read outside the covered tokens shows
  up as NaN.  Table entries past a sequence's last block are -1.
"""

from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np

HEAD_DIM = 128
BLOCK_SIZE = 16
K_CHUNK = 8  # bf16 elements per 16-byte key chunk
BF16_NAN = np.uint16(0x7FC0)

# Stream ids for independent PCG64 streams.
_S_LENS, _S_SPLIT, _S_PERM, _S_Q, _S_K, _S_V, _S_BIAS = range(7)

_CHUNK_BLOCKS = 2048  # logical blocks per generation chunk


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round-to-nearest-even; NaN stays a quiet NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounded = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded[nan] = BF16_NAN
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact widening)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, cfg_id: int, stream: int, chunk: int = -1) -> np.random.Generator:
    key = [int(seed), int(cfg_id), int(stream)]
    if chunk >= 0:
        key.append(int(chunk))
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    q: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    block_table: np.ndarray
    seq_lens: np.ndarray
    kv_begin: np.ndarray
    kv_end: np.ndarray
    max_range_tokens: int

    @property
    def batch(self) -> int:
        return int(self.q.shape[0])

    @property
    def n_parts(self) -> int:
        return int(self.kv_begin.shape[0])

    @property
    def num_blocks(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def kv_bytes(self, part: Optional[int] = None) -> int:
        """Algorithmic K+V bytes the covered tokens occupy (each read once)."""
        per_tok = self.num_kv_heads * HEAD_DIM * 2 * 2
        if part is None:
            toks = int(np.sum(self.kv_end.astype(np.int64) - self.kv_begin))
        else:
            toks = int(np.sum(self.kv_end[part].astype(np.int64) - self.kv_begin[part]))
        return toks * per_tok


# ---------------------------------------------------------------------------
# Sequence lengths and partition ranges for the five serving-shaped workloads
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Config:
    cfg_id: int
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    max_seq_len: int  # table width = max_seq_len / 16
    q_scale: float = 1.0
    key_bias_std: float = 0.0


CONFIGS: Dict[str, Config] = {
    "tiny": Config(1, "tiny", 4, 8, 2, 1024, q_scale=1.0 / math.sqrt(128.0)),
    "llama3_8b": Config(2, "llama3_8b", 64, 32, 8, 4096),
    "long": Config(3, "long", 8, 32, 8, 131072),
    "mixed": Config(4, "mixed", 256, 32, 8, 16384),
    "fine": Config(5, "fine", 512, 64, 8, 2048, key_bias_std=2.0),
    # Multi-head (G = 1) layer with the public LLaMA-13B / OPT-13B head layout (40 heads x 128), the
    # models the paper evaluates; 2048-token contexts, last 30 % of the blocks migrated.
    "mha13b": Config(6, "mha13b", 32, 40, 40, 2048),
}


def _nblk(L: int) -> int:
    return (L + BLOCK_SIZE - 1) // BLOCK_SIZE


def _split_at_block(L: int, j: int) -> List[Tuple[int, int]]:
    cut = j * BLOCK_SIZE
    return [(0, cut), (cut, L)]


def _lens_and_ranges(cfg: Config, seed: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    rl = _rng(seed, cfg.cfg_id, _S_LENS)
    rs = _rng(seed, cfg.cfg_id, _S_SPLIT)
    B = cfg.batch
    if cfg.name == "tiny":
        lens = rl.integers(256, 1024, size=B, endpoint=True)
        parts = []
        for L in lens:
            nb = _nblk(int(L))
            j = int(rs.integers(1, nb - 1, endpoint=True))
            parts.append(_split_at_block(int(L), j))
    elif cfg.name in ("llama3_8b", "mha13b"):
        L = cfg.max_seq_len
        lens = np.full(B, L)
        nb = L // BLOCK_SIZE
        migrated = int(round(0.3 * nb))
        parts = [_split_at_block(L, nb - migrated) for _ in range(B)]
    elif cfg.name == "long":
        lens = rl.integers(32768, 131072, size=B, endpoint=True)
        parts = []
        for L in lens:
            nb = _nblk(int(L))
            w = rs.dirichlet(np.ones(4)) * nb
            sizes = np.floor(w).astype(np.int64)
            rem = nb - int(sizes.sum())
            order = np.argsort(-(w - sizes), kind="stable")
            sizes[order[:rem]] += 1
            cum = np.concatenate([[0], np.cumsum(sizes)])
            parts.append([(int(min(cum[p] * BLOCK_SIZE, L)), int(min(cum[p + 1] * BLOCK_SIZE, L))) for p in range(4)])
    elif cfg.name == "mixed":
        z = rl.standard_normal(B)
        lens = np.clip(np.rint(np.exp(math.log(1024.0) + z)), 16, 16384).astype(np.int64)
        parts = []
        for L in lens:
            L = int(L)
            if L > 2048:
                nb = _nblk(L)
                j = int(rs.integers(1, nb - 1, endpoint=True))
                parts.append(_split_at_block(L, j))
            else:
                parts.append([(0, L), (L, L)])
    elif cfg.name == "fine":
        lens = np.full(B, 2048)
        step = 128
        parts = [[(p * step, (p + 1) * step) for p in range(16)] for _ in range(B)]
    else:  # pragma: no cover
        raise KeyError(cfg.name)
    lens = np.asarray(lens, dtype=np.int32)
    n_parts = len(parts[0])
    begin = np.array([[parts[b][p][0] for b in range(B)] for p in range(n_parts)], dtype=np.int32)
    end = np.array([[parts[b][p][1] for b in range(B)] for p in range(n_parts)], dtype=np.int32)
    return lens, begin, end


# ---------------------------------------------------------------------------
# Pool / table / tensor generation
# ---------------------------------------------------------------------------

def _gen_normal_bf16(seed, cfg_id, stream, chunk, shape, scale=1.0, bias=None):
    g = _rng(seed, cfg_id, stream, chunk)
    x = g.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    if bias is not None:
        x += bias
    return f32_to_bf16_bits(x)


def build_workload(
    name: str,
    seed: int,
    batch: int,
    num_q_heads: int,
    num_kv_heads: int,
    seq_lens: np.ndarray,
    kv_begin: np.ndarray,
    kv_end: np.ndarray,
    max_blocks_per_seq: int,
    cfg_id: int = 99,
    q_scale: float = 1.0,
    key_bias_std: float = 0.0,
    pool_factor: float = 1.2,
    threads: Optional[int] = None,
    kv_fill: Optional[Callable[[int, np.ndarray], None]] = None,
) -> Workload:
    """Draw Q, the paged K/V pools and the block table for given lengths and ranges."""
    B, Hq, Hkv, D, bs = batch, num_q_heads, num_kv_heads, HEAD_DIM, BLOCK_SIZE
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    nbs = np.array([_nblk(int(L)) for L in seq_lens], dtype=np.int64)
    if np.any(nbs > max_blocks_per_seq):
        raise ValueError("sequence longer than the block table")
    n_used = int(nbs.sum())
    num_blocks = max(1, int(math.ceil(pool_factor * n_used)))

    perm = _rng(seed, cfg_id, _S_PERM).permutation(num_blocks).astype(np.int64)
    phys_of_logical = perm[:n_used]  # logical block i (in (b, j) order) -> physical block

    table = np.full((B, max_blocks_per_seq), -1, dtype=np.int32)
    owner_seq = np.empty(n_used, dtype=np.int64)
    owner_blk = np.empty(n_used, dtype=np.int64)
    pos = 0
    for b in range(B):
        nb = int(nbs[b])
        table[b, :nb] = phys_of_logical[pos:pos + nb]
        owner_seq[pos:pos + nb] = b
        owner_blk[pos:pos + nb] = np.arange(nb)
        pos += nb

    bias = None
    if key_bias_std:
        bias = (_rng(seed, cfg_id, _S_BIAS).standard_normal((Hkv, D), dtype=np.float32) * np.float32(key_bias_std))

    q = _gen_normal_bf16(seed, cfg_id, _S_Q, -1, (B, Hq, D), scale=q_scale)

    k_cache = np.empty((num_blocks, Hkv, D // K_CHUNK, bs, K_CHUNK), dtype=np.uint16)
    v_cache = np.empty((num_blocks, Hkv, D, bs), dtype=np.uint16)
    used = np.zeros(num_blocks, dtype=bool)
    used[phys_of_logical] = True
    k_cache[~used] = BF16_NAN
    v_cache[~used] = BF16_NAN

    n_chunks = (n_used + _CHUNK_BLOCKS - 1) // _CHUNK_BLOCKS

    def do_chunk(c: int) -> None:
        lo, hi = c * _CHUNK_BLOCKS, min(n_used, (c + 1) * _CHUNK_BLOCKS)
        n = hi - lo
        kb = None if bias is None else bias[None, :, None, :]
        kk = _gen_normal_bf16(seed, cfg_id, _S_K, c, (n, Hkv, bs, D), bias=kb)
        vv = _gen_normal_bf16(seed, cfg_id, _S_V, c, (n, Hkv, bs, D))
        # Poison the slots past seq_len in each sequence's last block.
        last_len = seq_lens[owner_seq[lo:hi]] - owner_blk[lo:hi] * bs
        tail = np.arange(bs)[None, :] >= last_len[:, None]  # [n, bs]
        if tail.any():
            kk.transpose(0, 2, 1, 3)[tail] = BF16_NAN
            vv.transpose(0, 2, 1, 3)[tail] = BF16_NAN
        phys = phys_of_logical[lo:hi]
        k_cache[phys] = kk.reshape(n, Hkv, bs, D // K_CHUNK, K_CHUNK).transpose(0, 1, 3, 2, 4)
        v_cache[phys] = vv.transpose(0, 1, 3, 2)

    nthr = threads or min(16, os.cpu_count() or 1)
    if n_chunks > 1 and nthr > 1:
        with ThreadPoolExecutor(max_workers=nthr) as ex:
            list(ex.map(do_chunk, range(n_chunks)))
    else:
        for c in range(n_chunks):
            do_chunk(c)

    kv_begin = np.asarray(kv_begin, dtype=np.int32)
    kv_end = np.asarray(kv_end, dtype=np.int32)
    max_range = int(np.max(kv_end.astype(np.int64) - kv_begin)) if kv_begin.size else 0
    return Workload(name, seed, Hq, Hkv, q, k_cache, v_cache, table, seq_lens, kv_begin, kv_end, max_range)


def make_config(name: str, seed: int = 0, threads: Optional[int] = None) -> Workload:
    """One of the five serving-shaped workloads: tiny, llama3_8b, long, mixed, fine."""
    cfg = CONFIGS[name]
    lens, begin, end = _lens_and_ranges(cfg, seed)
    return build_workload(
        cfg.name, seed, cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, lens, begin, end,
        cfg.max_seq_len // BLOCK_SIZE, cfg_id=cfg.cfg_id, q_scale=cfg.q_scale,
        key_bias_std=cfg.key_bias_std, threads=threads)


def make_custom(
    seed: int,
    batch: int,
    num_q_heads: int,
    num_kv_heads: int,
    seq_lens,
    ranges,
    max_blocks_per_seq: Optional[int] = None,
    q_scale: float = 1.0,
    key_bias_std: float = 0.0,
    pool_factor: float = 1.2,
) -> Workload:
    """Small hand-shaped workload. ``ranges[p][b] = (begin, end)``."""
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    mb = max_blocks_per_seq or max(1, max(_nblk(int(L)) for L in seq_lens))
    begin = np.array([[r[0] for r in part] for part in ranges], dtype=np.int32)
    end = np.array([[r[1] for r in part] for part in ranges], dtype=np.int32)
    return build_workload("custom", seed, batch, num_q_heads, num_kv_heads, seq_lens, begin, end, mb,
                          cfg_id=100, q_scale=q_scale, key_bias_std=key_bias_std, pool_factor=pool_factor)


def make_shared_pool(seed: int, batch: int, num_q_heads: int, num_kv_heads: int, seq_lens, pool_blocks: int,
                     q_bank: int = 65536, q_scale: float = 1.0) -> Workload:
    """Very large batches over a small pool: every logical block of every sequence maps to a block
    drawn uniformly from ``pool_blocks`` physical blocks (blocks are shared between sequences, as
    with shared prefixes), and each (sequence, head) query row is one of ``q_bank`` N(0, 1) rows
    drawn once.  One partition [0, seq_len) per sequence.  Host memory stays near the size of q
    itself, so batches of a million sequences can be drawn in seconds."""
    cfg_id = 101
    B, Hq, Hkv, D, bs = batch, num_q_heads, num_kv_heads, HEAD_DIM, BLOCK_SIZE
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    nbs = (seq_lens.astype(np.int64) + bs - 1) // bs
    mb = max(1, int(nbs.max()))
    g = _rng(seed, cfg_id, _S_PERM)
    table = g.integers(0, pool_blocks, size=(B, mb), dtype=np.int32)
    table[np.arange(mb)[None, :] >= nbs[:, None]] = -1
    bank = _gen_normal_bf16(seed, cfg_id, _S_Q, -1, (q_bank, D), scale=q_scale)
    pick = _rng(seed, cfg_id, _S_SPLIT).integers(0, q_bank, size=B * Hq)
    q = bank[pick].reshape(B, Hq, D)
    kk = _gen_normal_bf16(seed, cfg_id, _S_K, 0, (pool_blocks, Hkv, bs, D))
    vv = _gen_normal_bf16(seed, cfg_id, _S_V, 0, (pool_blocks, Hkv, bs, D))
    k_cache = np.ascontiguousarray(kk.reshape(pool_blocks, Hkv, bs, D // K_CHUNK, K_CHUNK).transpose(0, 1, 3, 2, 4))
    v_cache = np.ascontiguousarray(vv.transpose(0, 1, 3, 2))
    begin = np.zeros((1, B), dtype=np.int32)
    end = seq_lens[None, :].copy()
    return Workload("shared_pool", seed, Hq, Hkv, q, k_cache, v_cache, table, seq_lens, begin, end,
                    int(seq_lens.max()))


def subset(w: Workload, seqs) -> Workload:
    """The sequences ``seqs`` of a workload (same pools): results per sequence do not depend on the
    other sequences of a batch, so a subset checks sampled rows of a large batch."""
    seqs = np.asarray(seqs, dtype=np.int64)
    return dataclasses.replace(w, q=np.ascontiguousarray(w.q[seqs]), block_table=np.ascontiguousarray(w.block_table[seqs]),
                               seq_lens=np.ascontiguousarray(w.seq_lens[seqs]),
                               kv_begin=np.ascontiguousarray(w.kv_begin[:, seqs]),
                               kv_end=np.ascontiguousarray(w.kv_end[:, seqs]))


def permute_physical(w: Workload, seed: int) -> Workload:
    """Same logical content under a different physical block placement."""
    g = _rng(seed, 1000, _S_PERM)
    perm = g.permutation(w.num_blocks)  # old physical p -> new physical perm[p]
    k2 = np.empty_like(w.k_cache)
    v2 = np.empty_like(w.v_cache)
    k2[perm] = w.k_cache
    v2[perm] = w.v_cache
    t2 = np.where(w.block_table >= 0, perm[np.maximum(w.block_table, 0)], -1).astype(np.int32)
    return dataclasses.replace(w, k_cache=k2, v_cache=v2, block_table=t2)


def k_token_major(k_cache: np.ndarray) -> np.ndarray:
    """Copy of a key pool as [num_blocks, Hkv, bs, D] (token-major rows)."""
    nb, Hkv, nc, bs, x = k_cache.shape
    return np.ascontiguousarray(k_cache.transpose(0, 1, 3, 2, 4)).reshape(nb, Hkv, bs, nc * x)


def get_k_row(k_cache: np.ndarray, blk: int, g: int, slot: int) -> np.ndarray:
    """The D bf16 key bits of slot `slot` of tile (blk, g)."""
    return k_cache[blk, g, :, slot, :].reshape(-1).copy()


def set_k_row(k_cache: np.ndarray, blk: int, g: int, slot: int, bits: np.ndarray) -> None:
    """Overwrite the key of slot `slot` of tile (blk, g) with D bf16 bit patterns."""
    nc, x = k_cache.shape[2], k_cache.shape[4]
    k_cache[blk, g, :, slot, :] = np.asarray(bits, dtype=np.uint16).reshape(nc, x)


def unsplit_ranges(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """The single partition [0, seq_len) per sequence."""
    return np.zeros((1, w.batch), dtype=np.int32), w.seq_lens[None, :].astype(np.int32).copy()


@dataclasses.dataclass
class Migration:
    """Destination pools and table for moving partition `part`'s blocks to another pool."""
    dst_k: np.ndarray
    dst_v: np.ndarray
    dst_table: np.ndarray
    blk_begin: np.ndarray
    blk_end: np.ndarray

    @property
    def num_blocks(self) -> int:
        return int(self.dst_k.shape[0])


SENTINEL = np.uint16(0x7FC1)  # a NaN pattern distinct from the generator's poison


def make_migration(w: Workload, part: int, seed: int = 0, pool_factor: float = 1.2) -> Migration:
    """Blocks overlapping partition `part` of every sequence, each given a random block of a new
    pool (pre-filled with a sentinel NaN pattern); other table entries are -1."""
    t0 = w.kv_begin[part].astype(np.int64)
    t1 = w.kv_end[part].astype(np.int64)
    begin = np.where(t1 > t0, t0 // BLOCK_SIZE, 0).astype(np.int32)
    end = np.where(t1 > t0, (t1 + BLOCK_SIZE - 1) // BLOCK_SIZE, 0).astype(np.int32)
    n = int(np.sum(end - begin))
    nb = max(1, int(math.ceil(pool_factor * n)))
    perm = _rng(seed, 2000, _S_PERM).permutation(nb)
    table = np.full_like(w.block_table, -1)
    pos = 0
    for b in range(w.batch):
        k = int(end[b] - begin[b])
        table[b, begin[b]:end[b]] = perm[pos:pos + k]
        pos += k
    dk = np.full((nb,) + w.k_cache.shape[1:], SENTINEL, dtype=np.uint16)
    dv = np.full((nb,) + w.v_cache.shape[1:], SENTINEL, dtype=np.uint16)
    return Migration(dk, dv, table, begin, end)


@dataclasses.dataclass
class LayerStore:
    """Host-side KV store for a layer-wise pipeline over a workload.

    The first `fetch_blocks` logical blocks of sequence 0 are prefix-cache hits
    held in the store (fetched host-to-device before each layer's attention);
    the `store_blocks` blocks after them are newly computed and stored back
    device-to-host after the layer.  The workload is re-placed so both groups
    are contiguous physical runs (fetch: blocks [0, fetch_blocks), store: the
    next `store_blocks`), one copy each per pool.  Every layer has its own
    fetched contents.
    """
    w: Workload
    num_layers: int
    fetch_blocks: int
    store_blocks: int
    fetch_k: np.ndarray  # [layers, fetch_blocks, Hkv, D/8, bs, 8]
    fetch_v: np.ndarray  # [layers, fetch_blocks, Hkv, D, bs]


def make_layer_store(w: Workload, num_layers: int, fetch_tokens: int, store_tokens: int, seed: int = 0) -> LayerStore:
    fb = (fetch_tokens + BLOCK_SIZE - 1) // BLOCK_SIZE
    sb = (store_tokens + BLOCK_SIZE - 1) // BLOCK_SIZE
    if fb + sb > int(np.sum(w.block_table[0] >= 0)):
        raise ValueError("sequence 0 is shorter than the fetched + stored blocks")
    # Physical permutation moving sequence 0's blocks 0 .. fb + sb - 1 to physical blocks 0 .. fb + sb - 1.
    want = w.block_table[0, :fb + sb].astype(np.int64)
    others = np.setdiff1d(np.arange(w.num_blocks), want, assume_unique=False)
    order = np.concatenate([want, others])  # new physical i holds old physical order[i]
    perm = np.empty(w.num_blocks, dtype=np.int64)
    perm[order] = np.arange(w.num_blocks)
    k2 = w.k_cache[order]
    v2 = w.v_cache[order]
    t2 = np.where(w.block_table >= 0, perm[np.maximum(w.block_table, 0)], -1).astype(np.int32)
    w2 = dataclasses.replace(w, k_cache=k2, v_cache=v2, block_table=t2)
    Hkv = w.num_kv_heads
    fk = np.empty((num_layers, fb) + w.k_cache.shape[1:], dtype=np.uint16)
    fv = np.empty((num_layers, fb) + w.v_cache.shape[1:], dtype=np.uint16)
    for layer in range(num_layers):
        kk = _gen_normal_bf16(seed, 3000 + layer, _S_K, -1, (fb, Hkv, BLOCK_SIZE, HEAD_DIM))
        fk[layer] = kk.reshape(fb, Hkv, BLOCK_SIZE, HEAD_DIM // K_CHUNK, K_CHUNK).transpose(0, 1, 3, 2, 4)
        fv[layer] = _gen_normal_bf16(seed, 3000 + layer, _S_V, -1, (fb, Hkv, BLOCK_SIZE, HEAD_DIM)).transpose(0, 1, 3, 2)
    return LayerStore(w2, num_layers, fb, sb, fk, fv)


def layer_view(store: LayerStore, layer: int) -> Workload:
    """The workload as layer `layer` sees it: its fetched prefix blocks in place."""
    k = store.w.k_cache.copy()
    v = store.w.v_cache.copy()
    k[:store.fetch_blocks] = store.fetch_k[layer]
    v[:store.fetch_blocks] = store.fetch_v[layer]
    return dataclasses.replace(store.w, k_cache=k, v_cache=v)
