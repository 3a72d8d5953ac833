/*
 * abi_roundtrip.c -- a plain C caller of libbana.so (no Python, no torch).
 *
 * Builds a small paged KV cache (3 sequences, 8 query / 2 kv heads, ragged
 * lengths, ranges split off block boundaries, a shuffled block table and NaN
 * in every unused slot), runs the per-partition calls, the merge and the fused
 * call through the C ABI on its own HIP stream, and checks them against the
 * fp64 CPU oracle (test infrastructure, linked only into this test program).
 * Also checks that host-visible argument errors come back as status codes.
 * Exit status 0 = pass.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "bana.h"

/* The oracle's entry points (oracle/oracle.c). */
int oracle_partial(int B, int Hq, int Hkv, int D, int bs, int max_blocks, int64_t num_blocks, const uint16_t* q,
                   const uint16_t* k_cache, const uint16_t* v_cache, const int32_t* block_table,
                   const int32_t* seq_lens, const int32_t* kv_begin, const int32_t* kv_end, const int32_t* seqs,
                   int n_seqs, double* out, double* lse, int nthreads);
int oracle_merge(int n_parts, int64_t rows, int D, const double* outs, const double* lses, double* out,
                 double* lse_out);

#define B 3
#define HQ 8
#define HKV 2
#define D 128
#define BS 16
#define MAXB 8
#define NPARTS 2
#define TILE (D * BS)

#define CHECK_HIP(x)                                                          \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return 2;                                                               \
    }                                                                         \
  } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) { /* xorshift64* */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}
static float uniform_pm1(void) { return (float)next_u32() / 2147483648.0f - 1.0f; }

static uint16_t to_bf16(float x) { /* round to nearest even */
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

int main(void) {
  const int lens[B] = {40, 100, 17};
  const int cut[B] = {23, 64, 5}; /* partition 0 = [0, cut), partition 1 = [cut, len) */
  int nblk_total = 0;
  for (int b = 0; b < B; ++b) nblk_total += (lens[b] + BS - 1) / BS;
  const int64_t nb = nblk_total + 3;

  /* Shuffled physical blocks. */
  int32_t perm[64];
  for (int i = 0; i < nb; ++i) perm[i] = i;
  for (int i = (int)nb - 1; i > 0; --i) {
    int j = (int)(next_u32() % (uint32_t)(i + 1));
    int32_t t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  int32_t table[B * MAXB], seq_lens[B], begin[NPARTS * B], end[NPARTS * B];
  int used = 0;
  for (int b = 0; b < B; ++b) {
    seq_lens[b] = lens[b];
    for (int j = 0; j < MAXB; ++j) table[b * MAXB + j] = j < (lens[b] + BS - 1) / BS ? perm[used++] : -1;
    begin[b] = 0;
    end[b] = cut[b];
    begin[B + b] = cut[b];
    end[B + b] = lens[b];
  }

  /* Pools: NaN everywhere, then values in the covered slots (scaled so scores stay moderate). */
  const size_t pool_elems = (size_t)nb * HKV * TILE;
  uint16_t* k = malloc(pool_elems * 2);
  uint16_t* v = malloc(pool_elems * 2);
  uint16_t* q = malloc((size_t)B * HQ * D * 2);
  for (size_t i = 0; i < pool_elems; ++i) k[i] = v[i] = 0x7FC0;
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < lens[b]; ++t) {
      const int64_t blk = table[b * MAXB + t / BS];
      const int slot = t % BS;
      for (int g = 0; g < HKV; ++g)
        for (int d = 0; d < D; ++d) {
          const int64_t tile = (blk * HKV + g) * TILE;
          k[tile + ((d / 8) * BS + slot) * 8 + d % 8] = to_bf16(uniform_pm1());
          v[tile + (int64_t)d * BS + slot] = to_bf16(uniform_pm1());
        }
    }
  for (int i = 0; i < B * HQ * D; ++i) q[i] = to_bf16(0.25f * uniform_pm1());

  /* Device copies. */
  void *dq, *dk, *dv, *dtab, *dlen, *dbeg, *dend, *dparts, *dlses, *dout, *dlse, *dfout, *dflse, *dws = NULL;
  CHECK_HIP(hipMalloc(&dq, (size_t)B * HQ * D * 2));
  CHECK_HIP(hipMalloc(&dk, pool_elems * 2));
  CHECK_HIP(hipMalloc(&dv, pool_elems * 2));
  CHECK_HIP(hipMalloc(&dtab, sizeof table));
  CHECK_HIP(hipMalloc(&dlen, sizeof seq_lens));
  CHECK_HIP(hipMalloc(&dbeg, sizeof begin));
  CHECK_HIP(hipMalloc(&dend, sizeof end));
  CHECK_HIP(hipMalloc(&dparts, (size_t)NPARTS * B * HQ * D * 4));
  CHECK_HIP(hipMalloc(&dlses, (size_t)NPARTS * B * HQ * 4));
  CHECK_HIP(hipMalloc(&dout, (size_t)B * HQ * D * 4));
  CHECK_HIP(hipMalloc(&dlse, (size_t)B * HQ * 4));
  CHECK_HIP(hipMalloc(&dfout, (size_t)B * HQ * D * 4));
  CHECK_HIP(hipMalloc(&dflse, (size_t)B * HQ * 4));
  CHECK_HIP(hipMemcpy(dq, q, (size_t)B * HQ * D * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dk, k, pool_elems * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dv, v, pool_elems * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dtab, table, sizeof table, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dlen, seq_lens, sizeof seq_lens, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dbeg, begin, sizeof begin, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dend, end, sizeof end, hipMemcpyHostToDevice));
  hipStream_t stream;
  CHECK_HIP(hipStreamCreate(&stream));

  bana_dims d;
  memset(&d, 0, sizeof d);
  d.batch = B;
  d.num_q_heads = HQ;
  d.num_kv_heads = HKV;
  d.head_dim = D;
  d.block_size = BS;
  d.max_blocks_per_seq = MAXB;
  d.num_blocks = nb;
  d.chunks_hint = 3; /* force chunk partials through the workspace */
  const size_t ws_bytes = bana_decode_attn_workspace_bytes(&d);
  if (ws_bytes == 0) {
    fprintf(stderr, "expected a workspace for a chunked plan\n");
    return 1;
  }
  CHECK_HIP(hipMalloc(&dws, ws_bytes));

  /* Host-visible argument errors. */
  int fails = 0;
  if (bana_decode_attn_partial(&d, NULL, dk, dv, dtab, dlen, dbeg, dend, dparts, dlses, dws, ws_bytes, stream) !=
      BANA_ERR_INVALID)
    ++fails;
  if (bana_merge_partials(&d, dparts, dlses, 0, dout, dlse, stream) != BANA_ERR_INVALID) ++fails;
  if (strcmp(bana_status_string(BANA_ERR_UNSUPPORTED), "unsupported configuration") != 0) ++fails;

  /* Per-partition calls, merge, fused call. */
  for (int p = 0; p < NPARTS; ++p) {
    bana_status st = bana_decode_attn_partial(&d, dq, dk, dv, dtab, dlen, (int32_t*)dbeg + p * B,
                                              (int32_t*)dend + p * B, (float*)dparts + (size_t)p * B * HQ * D,
                                              (float*)dlses + (size_t)p * B * HQ, dws, ws_bytes, stream);
    if (st != BANA_OK) {
      fprintf(stderr, "partial %d: %s %s\n", p, bana_status_string(st), bana_last_error());
      return 1;
    }
  }
  if (bana_merge_partials(&d, dparts, dlses, NPARTS, dout, dlse, stream) != BANA_OK) return 1;
  if (bana_decode_attn_fused(&d, dq, dk, dv, dtab, dlen, dbeg, dend, NPARTS, dfout, dflse, dws, ws_bytes, stream) !=
      BANA_OK)
    return 1;
  CHECK_HIP(hipStreamSynchronize(stream));

  float parts[NPARTS * B * HQ * D], lses[NPARTS * B * HQ], out[B * HQ * D], lse[B * HQ], fout[B * HQ * D],
      flse[B * HQ];
  CHECK_HIP(hipMemcpy(parts, dparts, sizeof parts, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(lses, dlses, sizeof lses, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(out, dout, sizeof out, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(lse, dlse, sizeof lse, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(fout, dfout, sizeof fout, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(flse, dflse, sizeof flse, hipMemcpyDeviceToHost));

  /* Oracle. */
  static double ro[NPARTS * B * HQ * D], rl[NPARTS * B * HQ], mo[B * HQ * D], ml[B * HQ];
  for (int p = 0; p < NPARTS; ++p)
    if (oracle_partial(B, HQ, HKV, D, BS, MAXB, nb, q, k, v, table, seq_lens, begin + p * B, end + p * B, NULL, 0,
                       ro + (size_t)p * B * HQ * D, rl + (size_t)p * B * HQ, 1) != 0)
      return 1;
  if (oracle_merge(NPARTS, B * HQ, D, ro, rl, mo, ml) != 0) return 1;

  double max_abs = 0, max_lse = 0;
  for (int i = 0; i < NPARTS * B * HQ * D; ++i) max_abs = fmax(max_abs, fabs(parts[i] - ro[i]));
  for (int i = 0; i < B * HQ * D; ++i) {
    max_abs = fmax(max_abs, fabs(out[i] - mo[i]));
    max_abs = fmax(max_abs, fabs(fout[i] - mo[i]));
  }
  for (int i = 0; i < NPARTS * B * HQ; ++i) max_lse = fmax(max_lse, fabs(lses[i] - rl[i]));
  for (int i = 0; i < B * HQ; ++i) {
    max_lse = fmax(max_lse, fabs(lse[i] - ml[i]));
    max_lse = fmax(max_lse, fabs(flse[i] - ml[i]));
  }
  printf("abi_roundtrip: max-abs %.3e, lse max-abs %.3e, argument-check failures %d\n", max_abs, max_lse, fails);
  const int ok = max_abs <= 2e-3 && max_lse <= 1e-4 && fails == 0 && isfinite(max_abs);
  hipFree(dq); hipFree(dk); hipFree(dv); hipFree(dtab); hipFree(dlen); hipFree(dbeg); hipFree(dend);
  hipFree(dparts); hipFree(dlses); hipFree(dout); hipFree(dlse); hipFree(dfout); hipFree(dflse); hipFree(dws);
  hipStreamDestroy(stream);
  free(k); free(v); free(q);
  return ok ? 0 : 1;
}
