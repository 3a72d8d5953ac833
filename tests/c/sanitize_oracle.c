/*
 * sanitize_oracle.c -- the fp64 oracle (oracle/oracle.c) built for the CPU with
 * AddressSanitizer and UndefinedBehaviorSanitizer, driven by seeded random small workloads:
 * every buffer is allocated at exactly the size the oracle's interface states, so any read or
 * write outside it is reported.  Covers empty, one-token, unaligned and whole-sequence ranges,
 * subsets of sequences, merges with -inf parts, the address export, and the error returns for
 * a range past seq_len and a table entry outside the pool.  Exits non-zero on a sanitizer
 * report or an unexpected return code.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_partial(int B, int Hq, int Hkv, int D, int bs, int max_blocks, int64_t num_blocks, const uint16_t* q,
                   const uint16_t* k_cache, const uint16_t* v_cache, const int32_t* block_table,
                   const int32_t* seq_lens, const int32_t* kv_begin, const int32_t* kv_end, const int32_t* seqs,
                   int n_seqs, double* out, double* lse, int nthreads);
int oracle_merge(int n_parts, int64_t rows, int D, const double* outs, const double* lses, double* out,
                 double* lse_out);
int oracle_kv_rows(int B, int Hkv, int bs, int max_blocks, int64_t num_blocks, const int32_t* block_table,
                   const int32_t* kv_begin, const int32_t* kv_end, int64_t* rows);

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd32(void) { /* splitmix64 */
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return (uint32_t)((z ^ (z >> 31)) >> 32);
}
static int rnd(int lo, int hi) { return lo + (int)(rnd32() % (uint32_t)(hi - lo + 1)); }
static uint16_t rnd_bf16(void) { return (uint16_t)(0x3C00 + (rnd32() % 0x0700)) ^ (uint16_t)((rnd32() & 1) << 15); }

#define CHECK(c)                                                               \
  do {                                                                         \
    if (!(c)) {                                                                \
      fprintf(stderr, "check failed: %s (line %d, case %d)\n", #c, __LINE__, cs); \
      return 1;                                                                \
    }                                                                          \
  } while (0)

int main(int argc, char** argv) {
  const int n_cases = argc > 1 ? atoi(argv[1]) : 300;
  const int D = 128, bs = 16;
  long calls = 0;
  for (int cs = 0; cs < n_cases; ++cs) {
    const int B = rnd(1, 4), Hkv = rnd(1, 3), G = rnd(1, 4), Hq = Hkv * G;
    const int max_blocks = rnd(1, 6);
    const int64_t nb = rnd(max_blocks * B, max_blocks * B + 5);
    uint16_t* q = malloc(sizeof(uint16_t) * B * Hq * D);
    uint16_t* k = malloc(sizeof(uint16_t) * nb * Hkv * D * bs);
    uint16_t* v = malloc(sizeof(uint16_t) * nb * Hkv * D * bs);
    int32_t* table = malloc(sizeof(int32_t) * B * max_blocks);
    int32_t *lens = malloc(sizeof(int32_t) * B), *beg = malloc(sizeof(int32_t) * B), *end = malloc(sizeof(int32_t) * B);
    for (int64_t i = 0; i < (int64_t)B * Hq * D; ++i) q[i] = rnd_bf16();
    for (int64_t i = 0; i < nb * Hkv * D * bs; ++i) k[i] = rnd_bf16(), v[i] = rnd_bf16();
    for (int b = 0; b < B; ++b) {
      lens[b] = rnd(0, max_blocks * bs);
      const int kind = rnd(0, 4);
      beg[b] = kind == 0 ? lens[b] : rnd(0, lens[b]);
      end[b] = kind == 1 ? lens[b] : rnd(beg[b], lens[b]);
      for (int j = 0; j < max_blocks; ++j) table[b * max_blocks + j] = j * bs < lens[b] ? (b * max_blocks + j) : -1;
    }
    /* whole batch, then a subset in reverse order */
    double* out = malloc(sizeof(double) * B * Hq * D);
    double* lse = malloc(sizeof(double) * B * Hq);
    CHECK(oracle_partial(B, Hq, Hkv, D, bs, max_blocks, nb, q, k, v, table, lens, beg, end, NULL, 0, out, lse, 2) == 0);
    int32_t seqs[4];
    const int ns = rnd(1, B);
    for (int i = 0; i < ns; ++i) seqs[i] = B - 1 - i;
    double* out2 = malloc(sizeof(double) * ns * Hq * D);
    double* lse2 = malloc(sizeof(double) * ns * Hq);
    CHECK(oracle_partial(B, Hq, Hkv, D, bs, max_blocks, nb, q, k, v, table, lens, beg, end, seqs, ns, out2, lse2, 1) == 0);
    /* merge of the partial with itself and an all-empty part */
    const int n_parts = rnd(1, 4);
    double* outs = malloc(sizeof(double) * n_parts * B * Hq * D);
    double* lses = malloc(sizeof(double) * n_parts * B * Hq);
    for (int p = 0; p < n_parts; ++p)
      for (int64_t r = 0; r < (int64_t)B * Hq; ++r) {
        lses[(int64_t)p * B * Hq + r] = p == n_parts - 1 && n_parts > 1 ? -INFINITY : lse[r];
        for (int d = 0; d < D; ++d) outs[((int64_t)p * B * Hq + r) * D + d] = out[r * D + d];
      }
    double* mo = malloc(sizeof(double) * B * Hq * D);
    double* ml = malloc(sizeof(double) * B * Hq);
    CHECK(oracle_merge(n_parts, (int64_t)B * Hq, D, outs, lses, mo, ml) == 0);
    int64_t* rows = malloc(sizeof(int64_t) * B * Hkv * max_blocks * bs);
    CHECK(oracle_kv_rows(B, Hkv, bs, max_blocks, nb, table, beg, end, rows) == 0);
    /* error returns: a range past seq_len, then a covered table entry outside the pool */
    const int b0 = rnd(0, B - 1);
    const int32_t saved_end = end[b0];
    end[b0] = lens[b0] + 1;
    CHECK(oracle_partial(B, Hq, Hkv, D, bs, max_blocks, nb, q, k, v, table, lens, beg, end, NULL, 0, out, lse, 1) == -1);
    end[b0] = saved_end;
    if (end[b0] > beg[b0]) {
      const int j = beg[b0] / bs;
      const int32_t saved = table[b0 * max_blocks + j];
      table[b0 * max_blocks + j] = (int32_t)nb;
      CHECK(oracle_partial(B, Hq, Hkv, D, bs, max_blocks, nb, q, k, v, table, lens, beg, end, NULL, 0, out, lse, 1) == -2);
      table[b0 * max_blocks + j] = saved;
    }
    calls += 6;
    free(q), free(k), free(v), free(table), free(lens), free(beg), free(end), free(out), free(lse), free(out2),
        free(lse2), free(outs), free(lses), free(mo), free(ml), free(rows);
  }
  printf("sanitized oracle sweep: %d cases, %ld calls\n", n_cases, calls);
  return 0;
}
