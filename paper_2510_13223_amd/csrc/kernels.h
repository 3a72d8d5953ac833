// kernels.h -- host-side launchers of the HIP kernels (internal to libbana.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bana.h"

namespace bana {

// LDS race check (a build option for a test build only): before writing what other wavefronts of
// the workgroup read back through LDS, odd wavefronts sleep a few microseconds, and every
// read-back is preceded by one more barrier.  With the barriers the kernels already have, results
// must not change bit for bit; a read that raced a write would change them.
#ifdef BANA_LDS_RACE_CHECK
__device__ __forceinline__ void race_check_delay(int wave) {
  if (wave & 1) __builtin_amdgcn_s_sleep(127);
}
__device__ __forceinline__ void race_check_barrier() { __syncthreads(); }
#else
__device__ __forceinline__ void race_check_delay(int) {}
__device__ __forceinline__ void race_check_barrier() {}
#endif

// Wavefront timeline of the measurement build (BANA_WAVE_TIMELINE): set every slot to UINT64_MAX /
// copy the first n_slots slots (uint64 [n_slots][4]) to host memory, both after the stream's
// earlier work and synchronous with the host.  hipErrorNotSupported in the product build.
hipError_t timeline_clear(hipStream_t stream);
hipError_t timeline_read(uint64_t* out, size_t n_slots, hipStream_t stream);

// Host <-> device copies carried by extra workgroups of an attention launch: they take the
// launch's first n_wg workgroups, so they are dispatched before the attention's and run beside
// them (the layer-wise pipeline's fetch and store, inside the attention launch of a layer).
constexpr int kMaxSideCopies = 8;
struct SideCopies {
  int n;     // copies (0: none)
  int n_wg;  // workgroups given to them
  const void* src[kMaxSideCopies];
  void* dst[kMaxSideCopies];
  int64_t n16[kMaxSideCopies];  // 16-byte units of each copy
};

struct PartialArgs {
  const uint16_t* q;        // bf16 [B][Hq][128]
  const uint16_t* k;        // bf16 [num_blocks][Hkv][128/8][16][8]
  const uint16_t* v;        // bf16 [num_blocks][Hkv][128][16]
  const int32_t* table;     // [B][max_blocks]
  const int32_t* begin;     // [n_parts][B]
  const int32_t* end;       // [n_parts][B]
  int n_parts;              // ranges per sequence, 1..64
  const int32_t* seq_order; // optional [B] dispatch order of sequences (NULL: natural)
  float* out;               // nc == 1: final output [B][Hq][128]; nc > 1: chunk partials [nc][B][out_hq][128]
  float* lse;               // nc == 1: final lse [B][Hq];               nc > 1: chunk lses [nc][B][out_hq]
  int B, Hq, Hkv, G, max_blocks;
  int g0, ng;  // kv heads [g0, g0 + ng) of this launch
  int nc;    // chunks per (sequence, kv head)
  int cmin;  // minimum blocks per chunk
  // Destination rows: query head h of sequence b (chunk or piece slot c) goes to row
  // (c * B + b) * out_hq + h - out_h0 of out / lse.  Final output: out_hq = Hq, out_h0 = 0;
  // workspace partials of a kv-head range hold only its heads: out_hq = ng * G, out_h0 = g0 * G.
  int out_hq, out_h0;
  SideCopies copies;  // chunked launch only (the balanced launch takes none)
};

// Partial attention: one workgroup of `waves` wavefronts per (chunk, sequence, kv head).
hipError_t launch_partial_attn(const PartialArgs& a, int waves, hipStream_t stream);

constexpr int kBalancedWaves = 8;         // wavefronts per workgroup of the balanced launch
constexpr int kMaxBalancedBatch = 2048;  // sequences of the in-kernel schedule (prefix sums held in LDS)

// Balanced launch: K wavefronts per kv head, each over an equal interval of the call's virtual
// blocks; a.out / a.lse are piece buffers [K + B][out_hq][128] / [K + B][out_hq]; prefix [B + 1]
// receives the block-count prefix sums over sequences (for the merge).
hipError_t launch_balanced_attn(const PartialArgs& a, int32_t* prefix, int K, hipStream_t stream);

// Rows of a merge: hn heads of each of B sequences.  Head i of sequence b is row
// b * in_hq + in_h0 + i of every part (parts are [n_parts][B][in_hq]) and row
// b * out_hq + out_h0 + i of out / lse_out.
struct MergeRows {
  int64_t B;
  int hn, in_hq, in_h0, out_hq, out_h0;
};

// Merge of the balanced launch's pieces (slots [K + B][in_hq]) into out / lse_out; kp (1, 2, 4 or 8)
// thread groups per merged row share its pieces.
hipError_t launch_merge_pieces(const float* outs, const float* lses, const int32_t* prefix, int K, int kp,
                               MergeRows m, float* out, float* lse_out, hipStream_t stream);

// Log-sum-exp merge of n_parts partials ([n_parts][B][in_hq][128] / [n_parts][B][in_hq]) into out / lse_out.
// Kernel and summation order depend only on n_parts and B x hn.
hipError_t launch_merge(const float* outs, const float* lses, int n_parts, MergeRows m, float* out, float* lse_out,
                        hipStream_t stream);

// Copy of the K/V tiles (all kv heads) of logical blocks [blk_begin[b], blk_end[b]) from the
// src pool (src_table) to the dst pool (dst_table); max_migrated_blocks bounds blk_end - blk_begin.
// Up to kMaxFlatMigrateBatch sequences: one flat list of tiles over a round of resident
// workgroups; more: a grid row per sequence.
constexpr int kMaxFlatMigrateBatch = 4096;
hipError_t launch_migrate(const void* src_k, const void* src_v, const int32_t* src_table, void* dst_k, void* dst_v,
                          const int32_t* dst_table, const int32_t* blk_begin, const int32_t* blk_end, int B,
                          int max_blocks, int max_migrated_blocks, int Hkv, hipStream_t stream);

// Stream-ordered copy of `bytes` (a multiple of 16) between 16-byte aligned buffers in device or
// pinned host memory, by a small kernel.
hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

// Device-side check of ranges, lengths and table entries; writes 0 or the highest broken-rule code
// to *result (device memory).
hipError_t launch_validate(const int32_t* table, const int32_t* seq_lens, const int32_t* begin, const int32_t* end,
                           int n_parts, int B, int max_blocks, int64_t num_blocks, int32_t* result,
                           hipStream_t stream);

// K/V read of the attention ranges with no arithmetic (bandwidth ceiling of the access pattern);
// sink[b * Hkv + g] = XOR of the 32-bit words read for (b, g).
hipError_t launch_gather_read(const void* k, const void* v, const int32_t* table, const int32_t* begin,
                              const int32_t* end, int n_parts, int B, int Hkv, int max_blocks, uint32_t* sink,
                              hipStream_t stream);

// Sequential read of `bytes` (a multiple of 16) by n_groups workgroups of 256 threads;
// sink[w] = XOR of the 32-bit words workgroup w read.
hipError_t launch_stream_read(const void* src, size_t bytes, int n_groups, uint32_t* sink, hipStream_t stream);

// The library's static device scratch (bana_decode_attn_partial_noalloc): its size, and its
// address on the current device (looked up once per device, then cached).
constexpr size_t kStaticScratchBytes = BANA_STATIC_SCRATCH_BYTES;
hipError_t static_scratch(void** ptr);

// Address export for the tests (rows of the K pool visited per logical token).
hipError_t launch_debug_rows(const int32_t* table, const int32_t* begin, const int32_t* end, int B, int Hkv,
                             int max_blocks, int64_t* rows, hipStream_t stream);

}  // namespace bana
