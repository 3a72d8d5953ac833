// paged_addr.h -- device-side address generation for the paged KV cache.
//
// Shared by the partial-attention kernel and the address-export test kernel
// so that the slots the test sees are the slots the attention reads.  Layout
// of the two pools, one 4 KiB tile per (block, kv head):
// K pool [num_blocks][Hkv][128/8][16][8] (16-byte chunks of 8 dims, chunk-major, then token),
// V pool [num_blocks][Hkv][128][16]      (dim-major).
#pragma once

#include <stdint.h>

namespace bana {

constexpr int kHeadDim = 128;
constexpr int kBlockSize = 16;
constexpr int kTileElems = kHeadDim * kBlockSize;  // bf16 elements per (block, kv head) tile

// Physical block of logical block j of sequence b.  The table is read-only
// for the whole launch and b, j are wave-uniform, so the entry is read
// through the constant address space: one scalar load per wave, tracked
// apart from the vector loads of K and V (it never stalls their pipeline).
__device__ __forceinline__ int32_t table_lookup(const int32_t* __restrict__ table, int max_blocks, int b, int j) {
  typedef const __attribute__((address_space(4))) int32_t* const_ptr;
  return ((const_ptr)table)[(int64_t)b * max_blocks + j];
}

// Index of the (block, kv head) tile; the tile starts at tile * kTileElems in either pool.
__device__ __forceinline__ int64_t kv_tile(int32_t blk, int g, int num_kv_heads) {
  return (int64_t)blk * num_kv_heads + g;
}

// Pool-wide index of slot `slot` of a tile (the token a (tile, slot) pair holds).
__device__ __forceinline__ int64_t tile_slot(int64_t tile, int slot) { return tile * kBlockSize + slot; }

}  // namespace bana
