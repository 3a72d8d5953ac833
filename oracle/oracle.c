/*
 * oracle.c -- plain, slow fp64 CPU reference for split paged decode attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header or table with the
 * HIP library: the cache layouts below are re-stated from the interface
 * contract, not included from it.
 *
 * What it computes (paper: Sec. 4.1(2), "Attention-level migration",
 * partition equations for S, A, l, O and the final sum O = O1 + O2):
 * the KV cache of every sequence is split into token-block partitions; each
 * partition j yields the softmax-normalised partial output O^(j) over its own
 * keys together with its log-sum-exp, and the partials are combined into the
 * exact softmax attention over all keys.  Readings taken where the printed
 * equations are garbled:
 *   - the split runs along token blocks of one sequence (the stage names
 *     "Atten for Local Seq" / "Atten for Offload Seq" and the running
 *     denominator l^(2) = l^(1) + sum A^(2) only make sense that way);
 *   - scores are the unscaled products q.k (the S = Q K^T equation carries no
 *     1/sqrt(d)); a caller that wants the scale pre-scales q;
 *   - the exponential is evaluated max-subtracted (same value, finite range);
 *   - each partial carries lse = ln(sum_t exp(s_t)) instead of the bare
 *     denominator l, and the combine is the symmetric log-sum-exp merge,
 *     which equals the paper's exchange of l^(1) / O^(1) with l = exp(lse);
 *   - an empty partition yields out = 0, lse = -inf and is skipped by the
 *     merge; an all-empty merge yields out = 0, lse = -inf.
 *
 * Data (interface contract; bf16 values are uint16 bit patterns, widened
 * exactly to double):
 *   q            [B][Hq][D]
 *   k_cache      [num_blocks][Hkv][D/8][bs][8]  per (block, kv-head) tile: 16-byte chunks of 8 dims,
 *                                              chunk-major, then token
 *   v_cache      [num_blocks][Hkv][D][bs]   dim-major tile per (block, kv-head)
 *   block_table  [B][max_blocks_per_seq]    logical block -> physical block
 *   query head h reads kv head g = h / (Hq / Hkv).
 *   Logical token t of sequence b lives in physical block
 *   block_table[b][t / bs], slot t % bs.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_to_f64(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Physical block holding logical token t of sequence b, or -1 if the table
 * does not map it to a block of the pool. */
static int64_t phys_block(const int32_t* block_table, int max_blocks, int64_t num_blocks, int bs, int b, int t) {
  int j = t / bs;
  if (j < 0 || j >= max_blocks) return -1;
  int64_t blk = block_table[(int64_t)b * max_blocks + j];
  if (blk < 0 || blk >= num_blocks) return -1;
  return blk;
}

/*
 * One partition for a set of sequences.  For every selected sequence b and
 * query head h, over the tokens T = [kv_begin[b], kv_end[b]):
 *   s_t   = sum_d q[b,h,d] * K[t,d]                       (Sec. 4.1(2), S = Q K^T)
 *   m     = max_t s_t,  w_t = exp(s_t - m),  l = sum_t w_t (A = exp S, l = sum A)
 *   out   = sum_t w_t V[t,:] / l                          (O = A / l . V)
 *   lse   = m + ln l
 * An empty T gives out = 0 and lse = -inf.
 *
 * seqs / n_seqs select which sequences to compute (NULL: all B, in order);
 * out is [n_seqs][Hq][D] and lse is [n_seqs][Hq], in the order of seqs.
 * Returns 0, or -1 for bad dimensions / ranges, or -2 when a covered token
 * maps to no valid physical block.
 */
int oracle_partial(int B, int Hq, int Hkv, int D, int bs, int max_blocks, int64_t num_blocks,
                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                   const int32_t* block_table, const int32_t* seq_lens,
                   const int32_t* kv_begin, const int32_t* kv_end,
                   const int32_t* seqs, int n_seqs, double* out, double* lse, int nthreads) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || D % 8 != 0 || bs <= 0 || max_blocks <= 0 || Hq % Hkv != 0)
    return -1;
  if (seqs == NULL) n_seqs = B;
  const int G = Hq / Hkv;
  for (int i = 0; i < n_seqs; ++i) {
    int b = seqs ? seqs[i] : i;
    if (b < 0 || b >= B) return -1;
    if (kv_begin[b] < 0 || kv_begin[b] > kv_end[b] || kv_end[b] > seq_lens[b]) return -1;
    for (int t = kv_begin[b]; t < kv_end[b]; t += 1)
      if (phys_block(block_table, max_blocks, num_blocks, bs, b, t) < 0) return -2;
  }
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#else
  nthreads = 1;
#endif
  const int64_t n_work = (int64_t)n_seqs * Hq;
#pragma omp parallel num_threads(nthreads)
  {
    int64_t cap = 0;
    double* s = NULL;
#pragma omp for schedule(dynamic, 1)
    for (int64_t wi = 0; wi < n_work; ++wi) {
      const int i = (int)(wi / Hq), h = (int)(wi % Hq);
      const int b = seqs ? seqs[i] : i;
      const int g = h / G;
      const int t0 = kv_begin[b], t1 = kv_end[b];
      double* o = out + ((int64_t)i * Hq + h) * D;
      for (int d = 0; d < D; ++d) o[d] = 0.0;
      if (t1 <= t0) {
        lse[(int64_t)i * Hq + h] = -INFINITY;
        continue;
      }
      if (t1 - t0 > cap) {
        free(s);
        cap = t1 - t0;
        s = (double*)malloc((size_t)cap * sizeof(double));
      }
      const uint16_t* qv = q + ((int64_t)b * Hq + h) * D;
      double m = -INFINITY;
      for (int t = t0; t < t1; ++t) {
        int64_t blk = phys_block(block_table, max_blocks, num_blocks, bs, b, t);
        const uint16_t* kt = k_cache + (blk * Hkv + g) * (int64_t)D * bs;
        const int slot = t % bs;
        double acc = 0.0;
        for (int d = 0; d < D; ++d) acc += bf16_to_f64(qv[d]) * bf16_to_f64(kt[((d / 8) * bs + slot) * 8 + d % 8]);
        s[t - t0] = acc;
        if (acc > m) m = acc;
      }
      double l = 0.0;
      for (int t = t0; t < t1; ++t) {
        int64_t blk = phys_block(block_table, max_blocks, num_blocks, bs, b, t);
        const uint16_t* vt = v_cache + (blk * Hkv + g) * (int64_t)D * bs;
        const int slot = t % bs;
        double w = exp(s[t - t0] - m);
        l += w;
        for (int d = 0; d < D; ++d) o[d] += w * bf16_to_f64(vt[(int64_t)d * bs + slot]);
      }
      for (int d = 0; d < D; ++d) o[d] /= l;
      lse[(int64_t)i * Hq + h] = m + log(l);
    }
    free(s);
  }
  return 0;
}

/*
 * Merge of n_parts partials per row (Sec. 4.1(2): O = O^(1) + O^(2) after the
 * exchange of the partial denominators), written as the log-sum-exp merge:
 *   J = { p : lse_p != -inf };  J empty -> out = 0, lse_out = -inf;
 *   M = max_J lse_p,  w_p = exp(lse_p - M),
 *   out = sum_J w_p out_p / sum_J w_p,  lse_out = M + ln sum_J w_p.
 * outs is [n_parts][rows][D], lses is [n_parts][rows].
 */
int oracle_merge(int n_parts, int64_t rows, int D, const double* outs, const double* lses,
                 double* out, double* lse_out) {
  if (n_parts < 1 || rows < 0 || D <= 0) return -1;
  for (int64_t r = 0; r < rows; ++r) {
    double M = -INFINITY;
    for (int p = 0; p < n_parts; ++p) {
      double v = lses[(int64_t)p * rows + r];
      if (v != -INFINITY && v > M) M = v;
    }
    double* o = out + r * D;
    for (int d = 0; d < D; ++d) o[d] = 0.0;
    if (M == -INFINITY) {
      lse_out[r] = -INFINITY;
      continue;
    }
    double wsum = 0.0;
    for (int p = 0; p < n_parts; ++p) {
      double v = lses[(int64_t)p * rows + r];
      if (v == -INFINITY) continue;
      double w = exp(v - M);
      wsum += w;
      const double* op = outs + ((int64_t)p * rows + r) * D;
      for (int d = 0; d < D; ++d) o[d] += w * op[d];
    }
    for (int d = 0; d < D; ++d) o[d] /= wsum;
    lse_out[r] = M + log(wsum);
  }
  return 0;
}

/*
 * Address generator written from the layout contract: for every sequence b,
 * kv head g and logical token t of the table's span, the (tile, slot) index
 * ((blk * Hkv + g) * bs + t % bs) of the key and value the attention must
 * read, with blk = block_table[b][t / bs], or -1 when t lies outside
 * [kv_begin[b], kv_end[b]).  rows is [B][Hkv][max_blocks * bs].
 */
int oracle_kv_rows(int B, int Hkv, int bs, int max_blocks, int64_t num_blocks, const int32_t* block_table,
                   const int32_t* kv_begin, const int32_t* kv_end, int64_t* rows) {
  if (B <= 0 || Hkv <= 0 || bs <= 0 || max_blocks <= 0) return -1;
  const int64_t span = (int64_t)max_blocks * bs;
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < Hkv; ++g)
      for (int64_t t = 0; t < span; ++t) {
        int64_t* r = rows + ((int64_t)b * Hkv + g) * span + t;
        if (t < kv_begin[b] || t >= kv_end[b]) {
          *r = -1;
          continue;
        }
        int64_t blk = phys_block(block_table, max_blocks, num_blocks, bs, b, (int)t);
        *r = blk < 0 ? -2 : (blk * Hkv + g) * bs + t % bs;
      }
  return 0;
}
