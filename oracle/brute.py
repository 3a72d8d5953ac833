"""Per-token brute force in pure Python for tiny inputs (test infrastructure only).

Independent of ``oracle.c``: it walks the block table token by token, builds
the softmax weights exp(s_t) / sum exp(s_t) directly (no running maximum,
no log-sum-exp; fine for the small score magnitudes it is used on), and sums
the partitions' probability mass and weighted values exactly as Sec. 4.1(2)
of the paper accumulates A and l across partitions, with l^(2) = l^(1) + sum A^(2).
"""

from __future__ import annotations

import math
import struct


def _bf16(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def attention(q, k_cache, v_cache, block_table, seq_lens, ranges, b: int, h: int, num_kv_heads: int):
    """Exact attention of query head h of sequence b over the union of ``ranges``.

    ``ranges`` is a list of (begin, end) partitions.  Returns (out list of D
    floats, ln of the total denominator).  Sums run partition by partition
    and carry the denominator l across partitions like the paper's l^(2).
    """
    Hq = len(q[b])
    G = Hq // num_kv_heads
    g = h // G
    D = len(q[b][h])
    bs = len(v_cache[0][0][0])
    qv = [_bf16(x) for x in q[b][h]]
    num = [0.0] * D
    l = 0.0
    for (t0, t1) in ranges:
        for t in range(t0, t1):
            blk = int(block_table[b][t // bs])
            slot = t % bs
            kt = k_cache[blk][g]  # [D/8][bs][8]
            s = 0.0
            for d in range(D):
                s += qv[d] * _bf16(kt[d // 8][slot][d % 8])
            a = math.exp(s)
            l += a
            vt = v_cache[blk][g]
            for d in range(D):
                num[d] += a * _bf16(vt[d][slot])
    if l == 0.0:
        return [0.0] * D, -math.inf
    return [x / l for x in num], math.log(l)
