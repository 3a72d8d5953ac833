// bana_api.cpp -- C ABI of libbana.so: argument checks, launch planning, launches.
//
// Every entry point validates what the host can see before touching HIP, so
// a rejected call never reaches the device.  Launch plans are a pure
// function of the dims (never of device properties or data), which keeps
// results bit-identical across runs.
#include "bana.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <string>

#include "kernels.h"

namespace {

thread_local std::string g_last_error;

constexpr int kHeadDim = 128;
constexpr int kBlockSize = 16;
constexpr int kMaxGroup = 16;           // query heads per kv head handled by one MFMA column tile
constexpr int kTargetWaves = 256 * 16;  // 256 CUs x 16 resident wavefronts: one full dispatch round
// Wavefronts of a balanced launch: 8 per CU, each walking twice the blocks it would in a full round.
// Measured on MI355X (long and mixed workloads, cold caches): 2048 wavefronts beat 4096 (each
// wavefront's start-up is paid over more blocks) and 1024 (too few blocks in flight).
constexpr int kBalancedTargetWaves = 256 * 8;
constexpr int kMinBlocksPerWave = 8;    // below this a wavefront spends more time starting than streaming
constexpr int kMaxBlocksPerWave = 64;   // longest run of blocks one wavefront should walk (no hints)
constexpr int kMaxChunks = 256;
constexpr int kMaxFusedParts = 64;  // one range per lane of the segment table
// Workgroups of an attention launch given to its side copies.  Measured on MI355X (the llama3_8b
// layer pipeline, 4 MiB of copies beside 1 GiB of attention reads): the copies' host-memory
// requests slow the attention they run beside, so fewer requests in flight over the attention's
// duration cost less: 32 workgroups with one 16-byte unit in flight per thread 0.182 ms per
// layer, 16 or 64 of them 0.185 / 0.191 ms, four units in flight 0.188-0.243 ms.
constexpr int kMaxSideCopyGroups = 32;
constexpr int64_t kMaxRows = int64_t{1} << 26;  // batch x num_q_heads: 64 threads per row stay below 2^32
constexpr int64_t kMaxLaunchItems = UINT32_MAX;  // work-items of one launch (grid x workgroup size)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bana_status check_dims(const bana_dims* d) {
  if (d == nullptr) return BANA_ERR_INVALID;
  if (d->batch <= 0 || d->num_q_heads <= 0 || d->num_kv_heads <= 0 || d->head_dim <= 0 || d->block_size <= 0 ||
      d->max_blocks_per_seq <= 0 || d->num_blocks <= 0)
    return BANA_ERR_INVALID;
  if (d->num_q_heads % d->num_kv_heads != 0) return BANA_ERR_INVALID;
  if (d->max_range_tokens < 0 || d->chunks_hint < 0 || d->plan_hint < 0 || d->plan_hint > 2 ||
      d->total_range_tokens < 0 || d->nonempty_ranges < 0)
    return BANA_ERR_INVALID;
  if (d->waves_hint != 0 && d->waves_hint != 1 && d->waves_hint != 2 && d->waves_hint != 4 && d->waves_hint != 8)
    return BANA_ERR_INVALID;
  if (d->head_dim != kHeadDim || d->block_size != kBlockSize) return BANA_ERR_UNSUPPORTED;
  if (d->num_q_heads / d->num_kv_heads > kMaxGroup) return BANA_ERR_UNSUPPORTED;
  // Index arithmetic of the kernels: table rows and token indices are
  // 32-bit, and a launch counts its work-items in 32 bits (one wavefront per
  // (sequence, kv head) at least; 32 threads per output row in the merge).
  if ((int64_t)d->batch * d->max_blocks_per_seq > INT32_MAX ||
      (int64_t)d->max_blocks_per_seq * kBlockSize > INT32_MAX ||
      (int64_t)d->batch * d->num_q_heads >= kMaxRows)
    return BANA_ERR_UNSUPPORTED;
  return BANA_OK;
}

struct Plan {
  int waves;      // wavefronts per workgroup
  int nc;         // chunks per (sequence, kv head)
  int cmin;       // minimum blocks per chunk
  bool balanced;  // equal block intervals per wavefront across sequences
  int K;          // balanced: wavefronts per kv head
  int kp;         // balanced: thread groups per row of the piece merge
  bool ordered;   // follow the caller's dispatch order (uneven ranges only)
};

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Workgroups are (chunk, sequence, kv head) with `waves` wavefronts each.
// Aim for one full round of resident wavefronts (256 CUs x 16).  With the
// range hints (longest range, total tokens, sequences with a non-empty
// range -- the "active" ones; the others cost a workgroup that exits at once):
//  - uneven ranges (longest > 1.25 x the mean over active sequences) get 8
//    waves per workgroup, so the long ranges finish early while short ones
//    fill the rest of the GPU;
//  - when the active (sequence, kv head) pairs alone cannot fill the round,
//    every range is cut into chunks of one wavefront's even share of the
//    call's blocks, enlarged so the rounding of each range to whole chunks
//    still fits one round (a second, partly filled round would double the
//    time of its workgroups);
//  - otherwise a range is only cut when its workgroup would take more than
//    twice the even share, into chunks of twice the even share.
// Chunks need workspace; without it the call runs unsplit.  Without hints
// the table width bounds the range length.
//
// Balanced launch (batch <= kMaxBalancedBatch): kBalancedTargetWaves
// wavefronts split over the kv heads, each over an equal interval of the
// call's blocks in sequence order, the pieces of a sequence merged
// afterwards.  Chosen when the ranges are uneven (longest > 1.25 x the mean),
// the active (sequence, kv head) pairs number at most a quarter of a round's
// wavefronts and the call has at least kMinBlocksPerWave blocks per
// wavefront (or asked for by plan_hint 2): there the chunked plan has to
// round every range to whole chunks within one or two rounds.  With even
// ranges that rounding costs less than the piece merge, and with many pairs
// several dispatch rounds, longest range first, balance by themselves
// (measured on MI355X, cold caches: mixed's 2048-pair calls 193 / 251 us
// chunked against 214 / 263 us balanced; its 1024-pair head halves 317
// against 278 us; long's fused call, 1.3 x spread, 494 against 478 us).
Plan make_plan(const bana_dims* d) {
  const int64_t pairs = (int64_t)d->batch * d->num_kv_heads;
  const int64_t active = d->nonempty_ranges > 0 ? std::min<int64_t>(d->nonempty_ranges, d->batch) : d->batch;
  const int64_t active_pairs = active * d->num_kv_heads;
  int64_t bound = d->max_blocks_per_seq;  // blocks of the longest range
  if (d->max_range_tokens > 0)
    bound = std::min<int64_t>(bound, ((int64_t)d->max_range_tokens + kBlockSize - 1) / kBlockSize);
  bound = std::max<int64_t>(bound, 1);
  int64_t wpp = (kTargetWaves + active_pairs - 1) / active_pairs;
  wpp = std::max<int64_t>(1, std::min<int64_t>(wpp, std::max<int64_t>(1, bound / kMinBlocksPerWave)));
  const bool hinted = d->total_range_tokens > 0;
  // The mean range cannot exceed the longest one; hints that say otherwise are clamped (this
  // also keeps mean_blocks x pairs inside 64 bits).
  const int64_t mean_blocks =
      hinted ? std::max<int64_t>(1, std::min<int64_t>(bound + 1, d->total_range_tokens / (kBlockSize * active) + 1))
             : bound;
  const bool uneven = hinted && 4 * bound > 5 * mean_blocks;
  Plan p;
  p.balanced = false;
  // The dispatch order pays off only when ranges are uneven (long ones first, short ones
  // filling the end of the launch); with even or unknown lengths its lookup would add one
  // dependent load to every wavefront's start, so it is skipped.
  p.ordered = uneven;
  p.K = std::max(1, kBalancedTargetWaves / (bana::kBalancedWaves * d->num_kv_heads)) * bana::kBalancedWaves;
  p.kp = 1;
  // The balanced schedule counts the blocks of all ranges of all sequences in 32 bits.
  const bool fits32 = (int64_t)d->batch * kMaxFusedParts * d->max_blocks_per_seq <= INT32_MAX;
  if (d->batch <= bana::kMaxBalancedBatch && fits32 && d->waves_hint == 0 && d->chunks_hint == 0 &&
      d->plan_hint != 1) {
    const int64_t call_blocks = hinted ? d->total_range_tokens / kBlockSize + active : 0;
    const bool few_pairs = 4 * active_pairs <= kTargetWaves;
    p.balanced = d->plan_hint == 2 || (uneven && few_pairs && call_blocks >= (int64_t)kMinBlocksPerWave * p.K);
  }
  if (p.balanced) {
    // Pieces of the row with the most: its blocks over intervals of at least s_lo blocks, plus
    // the two partly covered intervals at its ends.  Few rows (long sequences of a small batch)
    // spread each row's pieces over 8 thread groups; with many rows, one group per row streams
    // best unless a row has very many pieces (measured on MI355X, cold caches: mixed's migrated
    // partition, 8,192 rows, 68 / 69 / 71 / 76 us with 1 / 2 / 4 / 8 groups; long's partitions,
    // 256 rows, fastest with 8).
    const int64_t u_lo = hinted ? std::max<int64_t>(1, d->total_range_tokens / kBlockSize) : 1;
    const int64_t s_lo = std::max<int64_t>(1, u_lo / p.K);
    const int64_t pieces = (bound + 1) / s_lo + 2;
    const int64_t rows = (int64_t)d->batch * d->num_q_heads;
    p.kp = rows < 4096 ? 8 : pieces >= 64 ? 2 : 1;
  }
  if (p.balanced) {
    p.waves = bana::kBalancedWaves;
    p.nc = 1;
    p.cmin = 1;
    return p;
  }
  if (d->waves_hint > 0)
    p.waves = d->waves_hint;
  else if (uneven && bound >= 8 * kMinBlocksPerWave)
    p.waves = 8;
  else
    p.waves = wpp >= 8 ? 8 : wpp >= 4 ? 4 : wpp >= 2 ? 2 : 1;
  // The cross-wave combine keeps W * G rows of 132 floats in LDS; stay within 64 KiB per workgroup.
  const int G = d->num_q_heads / d->num_kv_heads;
  while (p.waves > 1 && sizeof(float) * (size_t)(32 * p.waves + p.waves * G * (kHeadDim + 4)) > 65536) p.waves /= 2;
  while (p.waves > 1 && (pairs + kMaxSideCopyGroups) * 64 * p.waves > kMaxLaunchItems) p.waves /= 2;
  if (d->chunks_hint > 0) {
    p.nc = d->chunks_hint;
    p.cmin = 1;
  } else if (hinted) {
    // (block, kv head) units of the call and the blocks per wavefront if they
    // were spread evenly over one round of resident wavefronts.
    const int64_t units = mean_blocks * active_pairs;
    const int64_t even = (units + kTargetWaves - 1) / kTargetWaves;
    const int64_t slots = kTargetWaves / p.waves;
    int64_t per_wave;
    if (active_pairs < slots) {
      per_wave = std::max<int64_t>(
          even, (units + p.waves * (slots - active_pairs) - 1) / (p.waves * (slots - active_pairs)));
    } else if (bound > 2 * even * p.waves) {
      per_wave = 2 * even;
    } else {
      per_wave = bound;  // one chunk per range
    }
    per_wave = std::max<int64_t>(kMinBlocksPerWave, per_wave);
    const int64_t chunk = per_wave * p.waves;
    p.nc = ceil_div(bound, chunk);
    p.cmin = (int)std::min<int64_t>(chunk, INT32_MAX);
  } else {
    p.nc = std::max(ceil_div(wpp, p.waves), ceil_div(bound, (int64_t)p.waves * kMaxBlocksPerWave));
    p.cmin = p.waves * 16;
  }
  p.nc = std::max(1, std::min(p.nc, kMaxChunks));
  if (((int64_t)p.nc * pairs + kMaxSideCopyGroups) * 64 * p.waves > kMaxLaunchItems) p.nc = 1;
  return p;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace regions of a plan.  Chunked: chunk partials [nc][B][Hq][128] and
// [nc][B][Hq].  Balanced: piece partials [K + B][Hq][128] and [K + B][Hq],
// then the block-count prefix sums [B + 1].
struct WorkspaceLayout {
  size_t out, lse, prefix, total;
};

WorkspaceLayout layout_for(const bana_dims* d, const Plan& p) {
  WorkspaceLayout w{0, 0, 0, 0};
  size_t rows;
  if (p.balanced) rows = ((size_t)p.K + d->batch) * d->num_q_heads;
  else if (p.nc > 1) rows = (size_t)p.nc * d->batch * d->num_q_heads;
  else return w;
  w.lse = align256(rows * kHeadDim * sizeof(float));
  w.total = align256(w.lse + rows * sizeof(float));
  if (p.balanced) {
    w.prefix = w.total;
    w.total = align256(w.prefix + ((size_t)d->batch + 1) * sizeof(int32_t));
  }
  return w;
}

size_t workspace_for(const bana_dims* d, const Plan& p) { return layout_for(d, p).total; }

bana_status device_status(hipError_t e) {
  if (e == hipSuccess) return BANA_OK;
  g_last_error = hipGetErrorString(e);
  return BANA_ERR_DEVICE;
}

}  // namespace

extern "C" {

const char* bana_status_string(bana_status s) {
  switch (s) {
    case BANA_OK: return "ok";
    case BANA_ERR_INVALID: return "invalid argument";
    case BANA_ERR_UNSUPPORTED: return "unsupported configuration";
    case BANA_ERR_DEVICE: return "device error";
  }
  return "unknown status";
}

const char* bana_last_error(void) { return g_last_error.c_str(); }

size_t bana_decode_attn_workspace_bytes(const bana_dims* d) {
  if (check_dims(d) != BANA_OK) return 0;
  return workspace_for(d, make_plan(d));
}

}  // extern "C"

namespace {

// Shared by the per-partition, fused and head-range entry points: n_parts
// ranges per sequence ([n_parts][B] begin / end), result (merged over the
// ranges) into the rows of kv heads [g0, g0 + ng) of out / lse.  The plan and
// the workspace layout are those of the sub-problem made of those heads alone
// (dims with ng kv heads and ng x G query heads), so a head-range call does
// exactly what the full call does on a cache holding only its heads.  Chunked
// plans leave chunk partials in the workspace and merge them with the merge
// kernel.
bana_status run_attention(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* block_table, const int32_t* kv_range_begin, const int32_t* kv_range_end,
                          int n_parts, int g0, int ng, float* out, float* lse, void* workspace,
                          size_t workspace_bytes, void* stream, const bana::SideCopies* side = nullptr) {
  const int G = d->num_q_heads / d->num_kv_heads;
  bana_dims sub = *d;
  sub.num_kv_heads = ng;
  sub.num_q_heads = ng * G;
  Plan plan = make_plan(&sub);
  const WorkspaceLayout ws = layout_for(&sub, plan);
  if (ws.total > 0 && (workspace == nullptr || workspace_bytes < ws.total)) {
    if (plan.balanced) {  // the chunked plan's launch shape, unsplit
      sub.plan_hint = 1;
      plan = make_plan(&sub);
    }
    plan.nc = 1;
  }

  bana::PartialArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_cache);
  a.v = static_cast<const uint16_t*>(v_cache);
  a.table = block_table;
  a.begin = kv_range_begin;
  a.end = kv_range_end;
  a.n_parts = n_parts;
  a.seq_order = plan.ordered ? d->seq_order : nullptr;
  a.B = d->batch;
  a.Hq = d->num_q_heads;
  a.Hkv = d->num_kv_heads;
  a.G = G;
  a.max_blocks = d->max_blocks_per_seq;
  a.g0 = g0;
  a.ng = ng;
  a.nc = plan.nc;
  a.cmin = plan.cmin;
  // Workspace partials hold the call's heads only; merged rows go to their place in out / lse.
  a.out_hq = ng * G;
  a.out_h0 = g0 * G;
  a.copies = bana::SideCopies{};
  if (side != nullptr && side->n > 0) {
    // Enough copy workgroups for the bytes (one 16-byte unit per thread per step), at most
    // kMaxSideCopyGroups, and at least one per copy (copy k takes the workgroups wg with
    // wg % n == k).
    a.copies = *side;
    int64_t units = 0;
    for (int i = 0; i < side->n; ++i) units += side->n16[i];
    const int64_t per_wg = (int64_t)64 * plan.waves;
    a.copies.n_wg = (int)std::max<int64_t>(
        side->n, std::min<int64_t>(kMaxSideCopyGroups, (units + per_wg - 1) / per_wg));
    // The launch counts its work-items in 32 bits (only batches of nearly 2^26 (sequence, kv head)
    // pairs come close).
    if (((int64_t)plan.nc * d->batch * ng + a.copies.n_wg) * 64 * plan.waves > kMaxLaunchItems) {
      g_last_error = "bana_decode_attn_fused_copies: the copy workgroups would take the launch past 2^32 work-items";
      return BANA_ERR_UNSUPPORTED;
    }
  }
  bana::MergeRows m;
  m.B = d->batch;
  m.hn = ng * G;
  m.in_hq = ng * G;
  m.in_h0 = 0;
  m.out_hq = d->num_q_heads;
  m.out_h0 = g0 * G;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (plan.balanced) {
    char* base = static_cast<char*>(workspace);
    float* ws_out = reinterpret_cast<float*>(base + ws.out);
    float* ws_lse = reinterpret_cast<float*>(base + ws.lse);
    int32_t* prefix = reinterpret_cast<int32_t*>(base + ws.prefix);
    a.out = ws_out;
    a.lse = ws_lse;
    hipError_t e = bana::launch_balanced_attn(a, prefix, plan.K, s);
    if (e != hipSuccess) return device_status(e);
    return device_status(bana::launch_merge_pieces(ws_out, ws_lse, prefix, plan.K, plan.kp, m, out, lse, s));
  }
  if (plan.nc == 1) {
    a.out = out;
    a.lse = lse;
    a.out_hq = d->num_q_heads;
    a.out_h0 = 0;
    return device_status(bana::launch_partial_attn(a, plan.waves, s));
  }
  char* base = static_cast<char*>(workspace);
  float* ws_out = reinterpret_cast<float*>(base + ws.out);
  float* ws_lse = reinterpret_cast<float*>(base + ws.lse);
  a.out = ws_out;
  a.lse = ws_lse;
  hipError_t e = bana::launch_partial_attn(a, plan.waves, s);
  if (e != hipSuccess) return device_status(e);
  return device_status(bana::launch_merge(ws_out, ws_lse, plan.nc, m, out, lse, s));
}

bana_status check_partial_args(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                               const int32_t* block_table, const int32_t* seq_lens, const int32_t* kv_range_begin,
                               const int32_t* kv_range_end, const float* out_partial, const float* lse,
                               const void* workspace) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !kv_range_begin || !kv_range_end || !out_partial ||
      !lse)
    return BANA_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out_partial) ||
      (workspace != nullptr && !aligned16(workspace)))
    return BANA_ERR_INVALID;
  return BANA_OK;
}

}  // namespace

extern "C" {

bana_status bana_decode_attn_partial(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     const int32_t* kv_range_begin, const int32_t* kv_range_end,
                                     float* out_partial, float* lse, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  const bana_status st = check_partial_args(d, q, k_cache, v_cache, block_table, seq_lens, kv_range_begin,
                                            kv_range_end, out_partial, lse, workspace);
  if (st != BANA_OK) return st;
  return run_attention(d, q, k_cache, v_cache, block_table, kv_range_begin, kv_range_end, 1, 0, d->num_kv_heads,
                       out_partial, lse, workspace, workspace_bytes, stream);
}

bana_status bana_decode_attn_partial_noalloc(const bana_dims* d, const void* q, const void* k_cache,
                                             const void* v_cache, const int32_t* block_table,
                                             const int32_t* seq_lens, const int32_t* kv_range_begin,
                                             const int32_t* kv_range_end, float* out_partial, float* lse,
                                             void* stream) {
  const bana_status st = check_partial_args(d, q, k_cache, v_cache, block_table, seq_lens, kv_range_begin,
                                            kv_range_end, out_partial, lse, nullptr);
  if (st != BANA_OK) return st;
  // The plan and the workspace it needs are those of bana_decode_attn_partial with a
  // workspace of bana_decode_attn_workspace_bytes(d) bytes; a plan the static scratch
  // cannot hold is refused rather than run differently.
  const size_t need = workspace_for(d, make_plan(d));
  if (need > bana::kStaticScratchBytes) {
    g_last_error = "bana_decode_attn_partial_noalloc: the launch plan for these dims needs " + std::to_string(need) +
                   " bytes of scratch, the library's static scratch holds " +
                   std::to_string(bana::kStaticScratchBytes) +
                   " (call bana_decode_attn_partial with a workspace of that size instead)";
    return BANA_ERR_UNSUPPORTED;
  }
  void* scratch = nullptr;
  const hipError_t e = bana::static_scratch(&scratch);
  if (e != hipSuccess) return device_status(e);
  return run_attention(d, q, k_cache, v_cache, block_table, kv_range_begin, kv_range_end, 1, 0, d->num_kv_heads,
                       out_partial, lse, scratch, bana::kStaticScratchBytes, stream);
}

bana_status bana_decode_attn_fused(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   const int32_t* kv_range_begin, const int32_t* kv_range_end, int32_t n_parts,
                                   float* out, float* lse_out, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !kv_range_begin || !kv_range_end || !out ||
      !lse_out || n_parts < 1)
    return BANA_ERR_INVALID;
  if (n_parts > kMaxFusedParts) return BANA_ERR_UNSUPPORTED;
  // A sequence's blocks over all its ranges are counted in 32 bits.
  if ((int64_t)n_parts * d->max_blocks_per_seq > INT32_MAX) return BANA_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out) ||
      (workspace != nullptr && !aligned16(workspace)))
    return BANA_ERR_INVALID;
  return run_attention(d, q, k_cache, v_cache, block_table, kv_range_begin, kv_range_end, n_parts, 0,
                       d->num_kv_heads, out, lse_out, workspace, workspace_bytes, stream);
}

bana_status bana_decode_attn_fused_copies(const bana_dims* d, const void* q, const void* k_cache,
                                          const void* v_cache, const int32_t* block_table, const int32_t* seq_lens,
                                          const int32_t* kv_range_begin, const int32_t* kv_range_end,
                                          int32_t n_parts, float* out, float* lse_out, void* workspace,
                                          size_t workspace_bytes, const bana_copy* copies, int32_t n_copies,
                                          void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !kv_range_begin || !kv_range_end || !out ||
      !lse_out || n_parts < 1 || n_copies < 0 || (n_copies > 0 && copies == nullptr))
    return BANA_ERR_INVALID;
  if (n_parts > kMaxFusedParts || n_copies > bana::kMaxSideCopies) return BANA_ERR_UNSUPPORTED;
  if ((int64_t)n_parts * d->max_blocks_per_seq > INT32_MAX) return BANA_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out) ||
      (workspace != nullptr && !aligned16(workspace)))
    return BANA_ERR_INVALID;
  bana::SideCopies side{};
  for (int i = 0; i < n_copies; ++i) {
    const bana_copy& c = copies[i];
    if (c.bytes == 0) continue;  // nothing to move; its pointers are not looked at
    if (!c.dst || !c.src || c.bytes % 16 != 0 || !aligned16(c.dst) || !aligned16(c.src)) return BANA_ERR_INVALID;
    side.src[side.n] = c.src;
    side.dst[side.n] = c.dst;
    side.n16[side.n] = (int64_t)(c.bytes / 16);
    ++side.n;
  }
  // The side copies ride on the chunked launch, with or without bytes to move.
  bana_dims chunked = *d;
  chunked.plan_hint = 1;
  return run_attention(&chunked, q, k_cache, v_cache, block_table, kv_range_begin, kv_range_end, n_parts, 0,
                       d->num_kv_heads, out, lse_out, workspace, workspace_bytes, stream, &side);
}

bana_status bana_decode_attn_heads(const bana_dims* d, const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   const int32_t* kv_range_begin, const int32_t* kv_range_end,
                                   int32_t kv_head_begin, int32_t kv_head_end, float* out, float* lse,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !kv_range_begin || !kv_range_end || !out || !lse)
    return BANA_ERR_INVALID;
  if (kv_head_begin < 0 || kv_head_end > d->num_kv_heads || kv_head_begin > kv_head_end) return BANA_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out) ||
      (workspace != nullptr && !aligned16(workspace)))
    return BANA_ERR_INVALID;
  if (kv_head_begin == kv_head_end) return BANA_OK;
  return run_attention(d, q, k_cache, v_cache, block_table, kv_range_begin, kv_range_end, 1, kv_head_begin,
                       kv_head_end - kv_head_begin, out, lse, workspace, workspace_bytes, stream);
}

bana_status bana_merge_partials(const bana_dims* d, const float* out_partials, const float* lses, int32_t n_parts,
                                float* out, float* lse_out, void* stream) {
  // Only the row count (batch x num_q_heads) and head_dim matter to the merge.
  if (d == nullptr || d->batch <= 0 || d->num_q_heads <= 0 || d->head_dim <= 0) return BANA_ERR_INVALID;
  if (d->head_dim != kHeadDim || (int64_t)d->batch * d->num_q_heads >= kMaxRows) return BANA_ERR_UNSUPPORTED;
  if (!out_partials || !lses || !out || n_parts < 1) return BANA_ERR_INVALID;
  if (!aligned16(out_partials) || !aligned16(out)) return BANA_ERR_INVALID;
  bana::MergeRows m;
  m.B = d->batch;
  m.hn = d->num_q_heads;
  m.in_hq = d->num_q_heads;
  m.in_h0 = 0;
  m.out_hq = d->num_q_heads;
  m.out_h0 = 0;
  return device_status(bana::launch_merge(out_partials, lses, n_parts, m, out, lse_out,
                                          static_cast<hipStream_t>(stream)));
}

bana_status bana_migrate_kv_blocks(const bana_dims* d, const void* src_k_cache, const void* src_v_cache,
                                   const int32_t* src_block_table, void* dst_k_cache, void* dst_v_cache,
                                   const int32_t* dst_block_table, int64_t dst_num_blocks,
                                   const int32_t* blk_begin, const int32_t* blk_end, void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!src_k_cache || !src_v_cache || !src_block_table || !dst_k_cache || !dst_v_cache || !dst_block_table ||
      !blk_begin || !blk_end || dst_num_blocks <= 0)
    return BANA_ERR_INVALID;
  if (!aligned16(src_k_cache) || !aligned16(src_v_cache) || !aligned16(dst_k_cache) || !aligned16(dst_v_cache))
    return BANA_ERR_INVALID;
  if (d->batch > 65535) return BANA_ERR_UNSUPPORTED;  // one grid row per sequence
  // Blocks per sequence the grid must cover: the hint (in tokens) when given, else the table width.
  int64_t maxb = d->max_blocks_per_seq;
  if (d->max_range_tokens > 0)
    maxb = std::min<int64_t>(maxb, ((int64_t)d->max_range_tokens + kBlockSize - 1) / kBlockSize);
  return device_status(bana::launch_migrate(src_k_cache, src_v_cache, src_block_table, dst_k_cache, dst_v_cache,
                                            dst_block_table, blk_begin, blk_end, d->batch, d->max_blocks_per_seq,
                                            (int)maxb, d->num_kv_heads, static_cast<hipStream_t>(stream)));
}

bana_status bana_validate_ranges(const bana_dims* d, const int32_t* block_table, const int32_t* seq_lens,
                                 const int32_t* kv_range_begin, const int32_t* kv_range_end, int32_t n_parts,
                                 int32_t* result, void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!block_table || !seq_lens || !kv_range_begin || !kv_range_end || !result || n_parts < 1) return BANA_ERR_INVALID;
  if (n_parts > 65535) return BANA_ERR_UNSUPPORTED;  // one grid row per partition
  return device_status(bana::launch_validate(block_table, seq_lens, kv_range_begin, kv_range_end, n_parts, d->batch,
                                             d->max_blocks_per_seq, d->num_blocks, result,
                                             static_cast<hipStream_t>(stream)));
}

bana_status bana_copy_async(void* dst, const void* src, size_t bytes, void* stream) {
  if (!dst || !src || bytes % 16 != 0 || !aligned16(dst) || !aligned16(src)) return BANA_ERR_INVALID;
  return device_status(bana::launch_copy(dst, src, bytes, static_cast<hipStream_t>(stream)));
}

bana_status bana_debug_kv_rows(const bana_dims* d, const int32_t* block_table, const int32_t* kv_range_begin,
                               const int32_t* kv_range_end, int64_t* rows_out, void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!block_table || !kv_range_begin || !kv_range_end || !rows_out) return BANA_ERR_INVALID;
  return device_status(bana::launch_debug_rows(block_table, kv_range_begin, kv_range_end, d->batch, d->num_kv_heads,
                                               d->max_blocks_per_seq, rows_out, static_cast<hipStream_t>(stream)));
}

bana_status bana_debug_gather_read(const bana_dims* d, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* kv_range_begin,
                                   const int32_t* kv_range_end, int32_t n_parts, uint32_t* sink, void* stream) {
  const bana_status st = check_dims(d);
  if (st != BANA_OK) return st;
  if (!k_cache || !v_cache || !block_table || !kv_range_begin || !kv_range_end || !sink || n_parts < 1)
    return BANA_ERR_INVALID;
  if (!aligned16(k_cache) || !aligned16(v_cache)) return BANA_ERR_INVALID;
  return device_status(bana::launch_gather_read(k_cache, v_cache, block_table, kv_range_begin, kv_range_end, n_parts,
                                                d->batch, d->num_kv_heads, d->max_blocks_per_seq, sink,
                                                static_cast<hipStream_t>(stream)));
}

bana_status bana_debug_wave_timeline_clear(void* stream) {
  const hipError_t e = bana::timeline_clear(static_cast<hipStream_t>(stream));
  if (e == hipErrorNotSupported) return BANA_ERR_UNSUPPORTED;
  return device_status(e);
}

bana_status bana_debug_wave_timeline_read(uint64_t* out, size_t n_slots, void* stream) {
  if (!out || n_slots > (size_t)BANA_TIMELINE_SLOTS) return BANA_ERR_INVALID;
  const hipError_t e = bana::timeline_read(out, n_slots, static_cast<hipStream_t>(stream));
  if (e == hipErrorNotSupported) return BANA_ERR_UNSUPPORTED;
  return device_status(e);
}

bana_status bana_debug_stream_read(const void* src, size_t bytes, int32_t n_groups, uint32_t* sink, void* stream) {
  if (!src || !sink || bytes % 16 != 0 || !aligned16(src) || n_groups < 1 || n_groups > 65536)
    return BANA_ERR_INVALID;
  return device_status(bana::launch_stream_read(src, bytes, n_groups, sink, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
