/*
 * bana.h -- C ABI of the split paged decode-attention library (libbana.so).
 *
 * The operation is the data-parallel step of attention-level KV-cache
 * migration (paper: Sec. 4.1(2), "Attention-level migration"): a decode
 * query attends to a paged KV cache whose token blocks are split into a
 * local partition and one or more migrated partitions.  Each partition is
 * reduced on its own to a softmax-normalised partial output plus its
 * log-sum-exp (the per-partition S = Q K^T, A = exp S, l = sum A,
 * O = A / l . V equations of that section), and a merge turns the partials
 * into the exact softmax attention over all tokens (the section's final
 * sum O = O^(1) + O^(2), with each partial rescaled by its share of the
 * total denominator; l^(j) = exp(lse_j)).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - All tensor arguments are DEVICE pointers owned by the caller, resident
 *    on the current HIP device, 16-byte aligned and densely packed in the
 *    layouts stated below.  The library allocates no memory and keeps no
 *    per-call state; calls are thread-safe.  (One exception, for callers that
 *    cannot allocate: bana_decode_attn_partial_noalloc keeps its partials in a
 *    static device array of the library, shared by its calls on a device.)
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream).  Nothing synchronises.
 *  - Host-checkable argument errors return before any HIP call:
 *    BANA_ERR_INVALID for a NULL required pointer, a non-positive size,
 *    num_q_heads % num_kv_heads != 0, n_parts < 1 or a misaligned pointer;
 *    BANA_ERR_UNSUPPORTED for head_dim != 128, block_size != 16, a GQA
 *    group (num_q_heads / num_kv_heads) above 16, or sizes whose indices
 *    leave 32 bits (batch * max_blocks_per_seq or max_blocks_per_seq * 16
 *    above 2^31 - 1, or batch * num_q_heads of 2^26 or more: a launch counts
 *    its threads in 32 bits).
 *  - A failed launch returns BANA_ERR_DEVICE; bana_last_error() then holds
 *    the HIP error text (per calling thread).
 *  - Device-resident values are preconditions and are not checked per call:
 *    0 <= kv_range_begin[b] <= kv_range_end[b] <= seq_lens[b], and every
 *    block-table entry for a block that overlaps [begin, end) names a block
 *    of the pool.  Entries outside the covered blocks are never read.
 *    bana_validate_ranges checks them on the device when wanted.  The
 *    optional dispatch order (bana_dims.seq_order) must be a permutation of
 *    0..batch-1 for every row to be written; out-of-range entries are
 *    clamped, never followed.
 *
 * Layouts (bf16 = IEEE binary16-brain, stored as 2 bytes)
 * --------------------------------------------------------
 *   q            bf16  [batch][num_q_heads][head_dim]
 *   k_cache      bf16  [num_blocks][num_kv_heads][head_dim / 8][block_size][8]
 *                      4 KiB tile per (block, kv head) of 16-byte chunks of
 *                      8 dims, chunk-major then token: element (token t,
 *                      dim d) of a tile is at ((d / 8) * block_size + t) * 8 + d % 8
 *   v_cache      bf16  [num_blocks][num_kv_heads][head_dim][block_size]
 *                      dim-major 4 KiB tile per (block, kv head): element
 *                      (token t, dim d) at d * block_size + t
 *  (These are the key and value block layouts of the paged KV cache the
 *  paper's serving system builds on.)
 *   block_table  int32 [batch][max_blocks_per_seq]
 *                      logical block j of sequence b -> physical block
 *   seq_lens     int32 [batch]  tokens in the cache, current token included
 *   out_partial  fp32  [batch][num_q_heads][head_dim]
 *   lse          fp32  [batch][num_q_heads], natural log
 *  Query head h reads kv head h / (num_q_heads / num_kv_heads).  Logical
 *  token t of sequence b lives in block block_table[b][t / 16], slot t % 16.
 *  Scores are the unscaled dot products q.k (the paper's S = Q K^T has no
 *  1/sqrt(d) factor); a caller that wants a softmax scale pre-scales q.
 */
#ifndef BANA_H
#define BANA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BANA_OK = 0,
  BANA_ERR_INVALID = -1,
  BANA_ERR_UNSUPPORTED = -2,
  BANA_ERR_DEVICE = -3
} bana_status;

typedef struct {
  int32_t batch;              /* B > 0 */
  int32_t num_q_heads;        /* Hq > 0, a multiple of num_kv_heads */
  int32_t num_kv_heads;       /* Hkv > 0; Hq / Hkv <= 16 */
  int32_t head_dim;           /* 128 */
  int32_t block_size;         /* 16 tokens per KV block */
  int32_t max_blocks_per_seq; /* row stride of block_table */
  int64_t num_blocks;         /* physical blocks in each pool */
  /* Performance hints; 0 = let the library choose.  They never change
   * results beyond float rounding order and never limit coverage. */
  int32_t max_range_tokens;   /* upper bound of kv_range_end - kv_range_begin over sequences */
  int32_t waves_hint;         /* waves per (sequence, kv head, chunk): 1, 2, 4 or 8 */
  int32_t chunks_hint;        /* chunks a range may be split into (needs workspace) */
  int32_t plan_hint;          /* 0 = choose; 1 = chunked launch; 2 = balanced launch
                                 (equal block intervals per wavefront across
                                 sequences; needs workspace, batch <= 2048 and
                                 batch * 64 * max_blocks_per_seq <= 2^31 - 1,
                                 otherwise the chunked launch runs) */
  int64_t total_range_tokens; /* sum over sequences of kv_range_end - kv_range_begin */
  /* Optional device array [batch]: the order in which sequences are
   * dispatched (a permutation of 0..batch-1; longest range first lets the
   * short ones fill the end of the launch).  NULL = natural order.  Results
   * do not depend on it.  Followed only when the range hints show uneven
   * ranges (longest > 1.25 x the mean); otherwise the natural order saves
   * a lookup per workgroup. */
  const int32_t* seq_order;
  /* Sequences whose range (all ranges, for the fused call) covers at least
   * one token; with total_range_tokens it gives the mean range of the
   * sequences that have work.  0 = unknown (taken as batch). */
  int32_t nonempty_ranges;
} bana_dims;

/*
 * Partial attention of one partition (Sec. 4.1(2): one of "Atten for Local
 * Seq" / "Atten for Offload Seq").  For every sequence b and query head h,
 * over the logical tokens T = [kv_range_begin[b], kv_range_end[b]):
 *   out_partial[b][h] = sum_{t in T} exp(s_t - m) v_t / sum_{t in T} exp(s_t - m)
 *   lse[b][h]         = m + ln sum_{t in T} exp(s_t - m),   m = max_{t in T} s_t
 * with s_t = q[b][h] . k_t.  An empty T gives out_partial = 0, lse = -inf.
 * Ranges need not be block aligned.  bf16 inputs, fp32 accumulation.
 *
 * workspace: optional device scratch of workspace_bytes bytes, at least
 * bana_decode_attn_workspace_bytes(d) for ranges to be split across several
 * workgroups (long ranges, few sequences, or uneven lengths: with the range
 * hints the library may cut the call's blocks into equal intervals across
 * sequences, one per wavefront); with less (or NULL, 0) the call runs
 * unsplit, with the same results up to rounding order.  The contents
 * need no initialisation and are garbage afterwards.  Calls that may run at
 * the same time (on different streams without an event between them) must
 * not share a workspace: they would overwrite each other's partials and
 * give wrong results (never an access outside the caller's buffers).  Results are
 * bit-identical run to run for the same inputs and dims, and invariant to
 * the physical placement of blocks.
 */
bana_status bana_decode_attn_partial(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     const int32_t* kv_range_begin, const int32_t* kv_range_end,
                                     float* out_partial, float* lse, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Bytes of the library's static device scratch (see bana_decode_attn_partial_noalloc). */
#define BANA_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation:
 * bana_decode_attn_partial without a caller workspace.  Same arguments (less
 * the workspace), same results bit for bit and same errors as
 * bana_decode_attn_partial given a workspace of
 * bana_decode_attn_workspace_bytes(d) bytes.  Where that call would split
 * ranges, the partials live in a static device array of the library,
 * BANA_STATIC_SCRATCH_BYTES (64 MiB) on each device, held from the time the
 * library's code is loaded on that device until the process ends.  This call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine); its
 * first call on a device, with that device current, looks the array's device
 * address up once (hipGetSymbolAddress).
 *   - Limit: when the launch plan for d needs more workspace than the array
 *     holds (bana_decode_attn_workspace_bytes(d) > BANA_STATIC_SCRATCH_BYTES),
 *     the call returns BANA_ERR_UNSUPPORTED before any launch, and
 *     bana_last_error() names both sizes; use bana_decode_attn_partial with a
 *     workspace of your own for such dims.
 *   - Sharing: every call on one device uses the same array and leaves its
 *     partials there.  Nothing in it needs to start at zero, but calls that
 *     may overlap on one device (on different streams with no event between
 *     them, or from several host threads) race for it and give wrong results:
 *     serialise them, e.g. on one stream.
 */
bana_status bana_decode_attn_partial_noalloc(const bana_dims* d, const void* q, const void* k_cache,
                                             const void* v_cache, const int32_t* block_table,
                                             const int32_t* seq_lens, const int32_t* kv_range_begin,
                                             const int32_t* kv_range_end, float* out_partial, float* lse,
                                             void* stream);

/*
 * Head-split partition: the literal reading of Sec. 4.1(2), where the KV
 * cache is split along the attention heads -- KV_1 keeps some kv
 * heads on the hot device, KV_2 the others on the cold device.  Computes, for
 * the kv heads [kv_head_begin, kv_head_end) only, exactly what
 * bana_decode_attn_partial computes on the sub-problem made of those heads
 * alone, bit for bit: q, the pools, out and lse holding only those heads
 * (and their G query heads each), with dims whose num_kv_heads is
 * kv_head_end - kv_head_begin and num_q_heads G times that.  That is what the
 * device holding those heads computes after they migrate there, so the launch
 * is planned for that many heads and fills the GPU by itself.  Only the rows
 * of the range's query heads (h with h / G in the kv-head range) of out / lse
 * are written; other rows are left untouched.  With head partitions the
 * "merge" is the concatenation of rows: calls over complementary kv-head
 * ranges give the full result, up to float rounding order as the full call
 * may plan its launch differently; with the launch shape fixed by
 * waves_hint and chunks_hint (both non-zero, chunks_hint <= 4) the plan does
 * not depend on the number of heads and the concatenation equals the full
 * call bit for bit.  An empty kv-head range does nothing.
 * workspace: as for bana_decode_attn_partial, sized by
 * bana_decode_attn_workspace_bytes of the sub-problem's dims.  Other
 * arguments and errors as for bana_decode_attn_partial; a kv-head range
 * outside [0, num_kv_heads] gives BANA_ERR_INVALID.
 */
bana_status bana_decode_attn_heads(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   const int32_t* kv_range_begin, const int32_t* kv_range_end,
                                   int32_t kv_head_begin, int32_t kv_head_end, float* out, float* lse,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace bana_decode_attn_partial / bana_decode_attn_fused can
 * use for these dims (0 when they would not split ranges); 0 for invalid
 * dims.  For bana_decode_attn_heads, pass the sub-problem's dims (its kv
 * heads only). */
size_t bana_decode_attn_workspace_bytes(const bana_dims* d);

/*
 * All partitions and their merge in one launch (Sec. 4.1(2): the partitions'
 * attention followed by the final O = O^(1) + O^(2), fused).  Equals
 * bana_decode_attn_partial on each of the n_parts ranges followed by
 * bana_merge_partials, up to float rounding order:
 *   out[b][h] / lse_out[b][h] = softmax attention of q[b][h] over the tokens
 *   of all ranges [kv_range_begin[p][b], kv_range_end[p][b]), p < n_parts
 * (a token covered by two ranges counts twice, as the merge of the two
 * partials would count it).  No token at all gives out = 0, lse_out = -inf.
 *   kv_range_begin / kv_range_end  int32 [n_parts][batch], 1 <= n_parts <= 64
 *   out      fp32 [batch][num_q_heads][head_dim]
 *   lse_out  fp32 [batch][num_q_heads]
 * dims->max_range_tokens / total_range_tokens, when given, refer to the sum
 * over a sequence's ranges.  Per-partition partials are not produced (use
 * bana_decode_attn_partial for those).  Errors as for the partial call;
 * n_parts > 64 or n_parts * max_blocks_per_seq above 2^31 - 1 gives
 * BANA_ERR_UNSUPPORTED.
 */
bana_status bana_decode_attn_fused(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   const int32_t* kv_range_begin, const int32_t* kv_range_end, int32_t n_parts,
                                   float* out, float* lse_out, void* workspace, size_t workspace_bytes,
                                   void* stream);

/* One host <-> device copy (see bana_decode_attn_fused_copies). */
typedef struct {
  void* dst;       /* device or pinned host memory, 16-byte aligned */
  const void* src; /* device or pinned host memory, 16-byte aligned */
  size_t bytes;    /* a multiple of 16 */
} bana_copy;

/*
 * bana_decode_attn_fused with up to 8 copies carried by the same launch: the
 * layer-wise pipeline of Sec. 4.2, where the fetch of layer i+1's KV from
 * the host store and the store of layer i-1's KV back to it overlap the
 * attention of layer i.  The copies (each like bana_copy_async) run in the
 * launch's first workgroups, dispatched ahead of the attention's, so one
 * launch per layer on one stream overlaps all three stages and orders them
 * against the neighbouring layers' launches by the stream alone.  The
 * attention runs the chunked launch (as with plan_hint 1) and its results
 * equal bana_decode_attn_fused with plan_hint 1 bit for bit.  The copies must
 * not overlap one another or any buffer the attention reads or writes.  The
 * copy workgroups take CU slots first: a plan that fills a whole dispatch round
 * by itself then runs some attention workgroups in a second round, so such
 * callers pass waves_hint 4 (or fewer) to leave room.  workspace: as for the
 * fused call, sized by bana_decode_attn_workspace_bytes of d with plan_hint 1.
 * A zero-byte copy is skipped (its pointers are not looked at).  Errors as for
 * the fused call; more than 8 copies gives BANA_ERR_UNSUPPORTED, a copy of a
 * non-zero size with a NULL or misaligned pointer or a size that is not a
 * multiple of 16 BANA_ERR_INVALID.
 */
bana_status bana_decode_attn_fused_copies(const bana_dims* d, const void* q, const void* k_cache,
                                          const void* v_cache, const int32_t* block_table, const int32_t* seq_lens,
                                          const int32_t* kv_range_begin, const int32_t* kv_range_end,
                                          int32_t n_parts, float* out, float* lse_out, void* workspace,
                                          size_t workspace_bytes, const bana_copy* copies, int32_t n_copies,
                                          void* stream);

/*
 * Merge of n_parts partials (Sec. 4.1(2), final O = O^(1) + O^(2) with the
 * exchange of the partial denominators l^(j) = exp(lse_j)).  Per row
 * r = (b, h):  J = { p : lses[p][r] != -inf };  J empty -> out = 0,
 * lse_out = -inf;  otherwise M = max_J lses[p][r], w_p = exp(lses[p][r] - M),
 *   out[r]     = sum_J w_p out_partials[p][r] / sum_J w_p,
 *   lse_out[r] = M + ln sum_J w_p.
 * Rows of parts with lse = -inf never enter a sum: they may hold anything,
 * NaN included (they lie inside the buffer and may be loaded).  Summation
 * runs in an order fixed by n_parts alone, so results are deterministic.
 * Of d, only batch, num_q_heads and head_dim are read.
 *   out_partials fp32 [n_parts][batch][num_q_heads][head_dim]
 *   lses         fp32 [n_parts][batch][num_q_heads]
 *   out          fp32 [batch][num_q_heads][head_dim]
 *   lse_out      fp32 [batch][num_q_heads], or NULL
 */
bana_status bana_merge_partials(const bana_dims* d, const float* out_partials, const float* lses, int32_t n_parts,
                                float* out, float* lse_out, void* stream);

/*
 * KV-block migration (Sec. 4.1(2): the KV of the offloaded part moves to the
 * cold device, T_attn ~ S_kv / B_net; Alg. 1's MigrateKVHeads): for every
 * sequence b and logical block j in [blk_begin[b], blk_end[b]) (block
 * units), copy the K and V tiles of all kv heads, bit for bit, from source
 * block src_block_table[b][j] to destination block dst_block_table[b][j].
 * After the call, attention over the migrated range through
 * (dst pools, dst_block_table) equals attention through the source pools,
 * bit for bit.
 *   src pools     layouts as above, d->num_blocks blocks
 *   dst pools     same layouts, dst_num_blocks blocks
 *   tables        int32 [batch][max_blocks_per_seq]; only the entries of
 *                 migrated blocks are read (the caller assigns destination
 *                 blocks; they must not overlap blocks being read)
 *   blk_begin/end int32 [batch], 0 <= begin <= end <= max_blocks_per_seq
 * d->max_range_tokens, when given, is a hint for (blk_end - blk_begin) *
 * block_size that sizes the launch (every block is copied regardless).
 * Errors as for the other calls; more than 65535 sequences gives
 * BANA_ERR_UNSUPPORTED.
 */
bana_status bana_migrate_kv_blocks(const bana_dims* d, const void* src_k_cache, const void* src_v_cache,
                                   const int32_t* src_block_table, void* dst_k_cache, void* dst_v_cache,
                                   const int32_t* dst_block_table, int64_t dst_num_blocks,
                                   const int32_t* blk_begin, const int32_t* blk_end, void* stream);

/*
 * Device-side check of the preconditions the attention and migration calls
 * trust (they are not checked per call, to keep calls free of host
 * synchronisation).  Writes to *result (int32 in device memory) 0 when, for
 * every partition p < n_parts and sequence b,
 *   0 <= seq_lens[b] <= max_blocks_per_seq * block_size            (else 3)
 *   0 <= kv_range_begin[p][b] <= kv_range_end[p][b]                (else 1)
 *   kv_range_end[p][b] <= seq_lens[b]                               (else 2)
 *   every block overlapping the range maps into [0, num_blocks)     (else 4)
 * and otherwise the highest code found.  Asynchronous on `stream`; read
 * *result after synchronising.  Table entries outside checked ranges are
 * never read.  More than 65535 partitions gives BANA_ERR_UNSUPPORTED.
 */
bana_status bana_validate_ranges(const bana_dims* d, const int32_t* block_table, const int32_t* seq_lens,
                                 const int32_t* kv_range_begin, const int32_t* kv_range_end, int32_t n_parts,
                                 int32_t* result, void* stream);

/*
 * Stream-ordered copy of `bytes` bytes from src to dst by a small kernel
 * (at most 64 workgroups), for staging KV between a host-side store and the
 * device pools in the layer-wise pipeline of Sec. 4.2 (fetch of layer i+1
 * and store of layer i-1 beside the attention of layer i).  Either side may
 * be device memory or pinned host memory (hipHostMalloc, reached over the
 * host link).  Being a kernel, the copy is ordered on `stream` like the
 * attention calls and waits for other streams only through device-side
 * events.  bytes must be a multiple of 16 and both pointers 16-byte aligned
 * (else BANA_ERR_INVALID); the ranges must not overlap.
 */
bana_status bana_copy_async(void* dst, const void* src, size_t bytes, void* stream);

/* Static text for a status code. */
const char* bana_status_string(bana_status s);

/* Text of the last error a call on this thread described in detail: the HIP
 * error text of a failed launch, or the sizes behind a refused
 * bana_decode_attn_partial_noalloc call ("" if none). */
const char* bana_last_error(void);

/*
 * Test hook for the address generator the attention kernel uses: for every
 * sequence b, kv head g and logical token t < max_blocks_per_seq * 16,
 *   rows_out[b][g][t] = (block_table[b][t / 16] * num_kv_heads + g) * 16 + t % 16
 * (the pool-wide (tile, slot) index whose key and value the partial kernel
 * reads for that token) when kv_range_begin[b] <= t < kv_range_end[b], and
 * -1 otherwise.  rows_out: int64 [batch][num_kv_heads][max_blocks_per_seq * 16].
 */
bana_status bana_debug_kv_rows(const bana_dims* d, const int32_t* block_table, const int32_t* kv_range_begin,
                               const int32_t* kv_range_end, int64_t* rows_out, void* stream);

/*
 * Measurement hook: the K/V read of attention over the ranges
 * [kv_range_begin[p][b], kv_range_end[p][b]) (p < n_parts), with the same
 * table walk and load shapes and no arithmetic, giving the practical
 * bandwidth ceiling of that access pattern.  Every 4 KiB K and V tile of
 * every covered block is read whole (a block covered by two ranges is read
 * twice) and its 32-bit words are XOR-folded:
 *   sink[b][g] = XOR of all 32-bit words of the K and V tiles of kv head g
 *                of the covered blocks of sequence b
 * so the result is checkable on the host.  sink: uint32 [batch][num_kv_heads]
 * (device).  Ranges are preconditions as for the attention calls.  Errors as
 * for the other calls; n_parts < 1 gives BANA_ERR_INVALID.
 */
bana_status bana_debug_gather_read(const bana_dims* d, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* kv_range_begin,
                                   const int32_t* kv_range_end, int32_t n_parts, uint32_t* sink, void* stream);

/*
 * Measurement hook: a plain front-to-back read of `bytes` bytes at src
 * (device memory, 16-byte aligned, bytes a multiple of 16) by n_groups
 * workgroups of 256 threads, each thread loading 16 bytes per step with a
 * stride of n_groups * 256 * 16 bytes (the streaming-read ceiling of HBM, for
 * comparison with the tile gather above; 8 workgroups per compute unit keep
 * 32 wavefronts resident on each).  The words are XOR-folded so the loads
 * cannot be dropped: the XOR of sink[0..n_groups) equals the XOR of all
 * 32-bit words of the buffer.  sink: uint32 [n_groups] (device).
 * BANA_ERR_INVALID for a NULL pointer, misalignment, or n_groups outside
 * [1, 65536].
 */
bana_status bana_debug_stream_read(const void* src, size_t bytes, int32_t n_groups, uint32_t* sink, void* stream);

/*
 * Measurement hook of the wavefront-timeline build (libbana_timeline.so, the
 * library compiled with BANA_WAVE_TIMELINE; same kernels and results): lane 0
 * of every wavefront of the attention launches (chunked and balanced) stores
 * readings of the GPU's constant 100 MHz clock in slot
 *   (workgroup index * wavefronts per workgroup + wavefront) mod BANA_TIMELINE_SLOTS
 * of a device table: [0] entry, [1] schedule ready (its ranges read, or the
 * balanced launch's prefix scan done), [2] first KV block consumed (the
 * earliest over the wavefront's pieces), [3] exit.  Side-copy workgroups and
 * wavefronts without work leave [2] (and those that exit early [3]) as they
 * were.
 * bana_debug_wave_timeline_clear: sets every slot word to UINT64_MAX after the
 *   stream's earlier work; returns when done.
 * bana_debug_wave_timeline_read: copies slots [0, n_slots) to out (host
 *   memory, uint64 [n_slots][4]) after the stream's earlier work; returns when
 *   done.  BANA_ERR_INVALID for a NULL out or n_slots > BANA_TIMELINE_SLOTS.
 * The product library returns BANA_ERR_UNSUPPORTED from both.
 */
#define BANA_TIMELINE_SLOTS (1 << 18)
bana_status bana_debug_wave_timeline_clear(void* stream);
bana_status bana_debug_wave_timeline_read(uint64_t* out, size_t n_slots, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BANA_H */
