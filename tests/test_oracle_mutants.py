"""The oracle's pins reject plausible mistakes.

Each case plants one mistake in a copy of ``oracle/oracle.c`` (a dropped
term, a wrong sign, index or layout, a transposed operand), compiles it on
the CPU and runs the pin suite against it in a child process; the suite must
fail.  The real oracle is never modified.
"""

import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    ("no max in the weights", "double w = exp(s[t - t0] - m);", "double w = exp(s[t - t0]);"),
    ("flipped exponent sign", "double w = exp(s[t - t0] - m);", "double w = exp(m - s[t - t0]);"),
    ("gqa head mapping", "const int g = h / G;", "const int g = h % Hkv;"),
    ("token-major key tile", "kt[((d / 8) * bs + slot) * 8 + d % 8]", "kt[slot * D + d]"),
    ("transposed value tile", "vt[(int64_t)d * bs + slot]", "vt[(int64_t)slot * D + d]"),
    ("missing normalisation", "for (int d = 0; d < D; ++d) o[d] /= l;", ""),
    ("lse in base 2", "lse[(int64_t)i * Hq + h] = m + log(l);", "lse[(int64_t)i * Hq + h] = m + log2(l);"),
    ("lse without the max", "lse[(int64_t)i * Hq + h] = m + log(l);", "lse[(int64_t)i * Hq + h] = log(l);"),
    ("range misses its first token", "for (int t = t0; t < t1; ++t) {\n        int64_t blk = phys_block(block_table, max_blocks, num_blocks, bs, b, t);\n        const uint16_t* vt",
     "for (int t = t0 + 1; t < t1; ++t) {\n        int64_t blk = phys_block(block_table, max_blocks, num_blocks, bs, b, t);\n        const uint16_t* vt"),
    ("wrong slot in the block", "const int slot = t % bs;\n        double acc", "const int slot = (t + 1) % bs;\n        double acc"),
    ("merge without the max shift", "lse_out[r] = M + log(wsum);", "lse_out[r] = log(wsum);"),
    ("merge reads empty parts", "      if (v == -INFINITY) continue;\n      double w = exp(v - M);", "      double w = exp(v - M);"),
    ("merge weights unnormalised", "for (int d = 0; d < D; ++d) o[d] /= wsum;", ""),
    ("empty partition lse zero", "        lse[(int64_t)i * Hq + h] = -INFINITY;\n        continue;", "        lse[(int64_t)i * Hq + h] = 0.0;\n        continue;"),
    ("address export: head-major tile index", "*r = blk < 0 ? -2 : (blk * Hkv + g) * bs + t % bs;",
     "*r = blk < 0 ? -2 : (g * num_blocks + blk) * bs + t % bs;"),
    ("address export: reversed slot", "*r = blk < 0 ? -2 : (blk * Hkv + g) * bs + t % bs;",
     "*r = blk < 0 ? -2 : (blk * Hkv + g) * bs + (bs - 1 - t % bs);"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(tmp_path, name, old, new):
    src = open(oracle.SRC_PATH).read()
    assert src.count(old) >= 1, f"mutation site not found: {name}"
    c_path = tmp_path / "mutant.c"
    so_path = tmp_path / "libmutant.so"
    c_path.write_text(src.replace(old, new, 1))
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", str(c_path), "-o", str(so_path),
                           "-lm"])
    env = dict(os.environ, ORACLE_LIB=str(so_path), OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant '{name}' survived every pin:\n{r.stdout[-2000:]}"
