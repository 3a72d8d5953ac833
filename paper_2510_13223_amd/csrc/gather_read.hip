// gather_read.hip -- the paged K/V read of decode attention with no arithmetic (gfx950).
//
// Measurement kernel: reads every K and V tile that attention over the ranges
// [begin[p][b], end[p][b]) reads, through the same block table and with the
// same load shapes (16 bytes per lane, whole 1 KiB runs per instruction,
// non-temporal), and folds the words into an XOR so the loads cannot be
// dropped.  Its bandwidth is the practical ceiling of the attention kernel's
// access pattern on random 4 KiB tiles.  One workgroup of 8 wavefronts per
// (sequence, kv head); wavefront w takes the blocks w, w + 8, ... of each
// range, two blocks in flight per step.
//
// A second hook reads one buffer front to back (the streaming ceiling of HBM
// reads, for comparison with the gather above).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "kernels.h"
#include "paged_addr.h"

namespace bana {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kLoads = kTileElems * 2 / 16 / 64;  // 16-byte loads per lane per 4 KiB tile (4)

__device__ __forceinline__ void read_tile(const uint16_t* pool, int64_t tile, int lane, u32x4* r) {
  const u32x4* src = reinterpret_cast<const u32x4*>(pool + tile * kTileElems) + lane;
#pragma unroll
  for (int i = 0; i < kLoads; ++i) r[i] = __builtin_nontemporal_load(src + 64 * i);
}

__global__ __launch_bounds__(64 * kWaves) void gather_read_kernel(const uint16_t* __restrict__ k,
                                                                  const uint16_t* __restrict__ v,
                                                                  const int32_t* __restrict__ table,
                                                                  const int32_t* __restrict__ begin,
                                                                  const int32_t* __restrict__ end, int n_parts,
                                                                  int B, int Hkv, int max_blocks,
                                                                  uint32_t* __restrict__ sink) {
  __shared__ uint32_t sm[kWaves];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int lane = threadIdx.x & 63;
  // Workgroups stride over the (sequence, kv head) pairs (one pass when the grid covers them all).
  for (int64_t pair = blockIdx.x; pair < (int64_t)B * Hkv; pair += gridDim.x) {
    const int g = (int)(pair % Hkv);
    const int b = (int)(pair / Hkv);
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int p = 0; p < n_parts; ++p) {
      const int t0 = table_lookup(begin, B, p, b);
      const int t1 = table_lookup(end, B, p, b);
      if (t1 <= t0) continue;
      const int j1 = (t1 - 1) / kBlockSize + 1;
      for (int j = t0 / kBlockSize + wave; j < j1; j += 2 * kWaves) {
        u32x4 r[4 * kLoads];
        const int64_t tile0 = kv_tile(table_lookup(table, max_blocks, b, j), g, Hkv);
        read_tile(k, tile0, lane, r);
        read_tile(v, tile0, lane, r + kLoads);
        const bool two = j + kWaves < j1;
        if (two) {
          const int64_t tile1 = kv_tile(table_lookup(table, max_blocks, b, j + kWaves), g, Hkv);
          read_tile(k, tile1, lane, r + 2 * kLoads);
          read_tile(v, tile1, lane, r + 3 * kLoads);
        }
#pragma unroll
        for (int i = 0; i < 2 * kLoads; ++i) acc ^= r[i];
        if (two) {
#pragma unroll
          for (int i = 2 * kLoads; i < 4 * kLoads; ++i) acc ^= r[i];
        }
      }
    }
    uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
    for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off);
    if (lane == 0) sm[wave] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t y = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) y ^= sm[w];
      sink[pair] = y;
    }
    __syncthreads();  // sm is rewritten by the next pair
  }
}

// Plain sequential read of n16 16-byte units, grid-stride, non-temporal: workgroup w reads units
// w * 256 + t + i * gridDim.x * 256 and XOR-folds their words into sink[w].
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ src, int64_t n16,
                                                          uint32_t* __restrict__ sink) {
  __shared__ uint32_t sm[4];
  const int64_t stride = (int64_t)gridDim.x * 256;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride)
    acc ^= __builtin_nontemporal_load(src + i);
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off);
  if ((threadIdx.x & 63) == 0) sm[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = sm[0] ^ sm[1] ^ sm[2] ^ sm[3];
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, int n_groups, uint32_t* sink, hipStream_t stream) {
  hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)n_groups), dim3(256), 0, stream,
                     static_cast<const u32x4*>(src), (int64_t)(bytes / 16), sink);
  return hipGetLastError();
}

hipError_t launch_gather_read(const void* k, const void* v, const int32_t* table, const int32_t* begin,
                              const int32_t* end, int n_parts, int B, int Hkv, int max_blocks, uint32_t* sink,
                              hipStream_t stream) {
  const int64_t grid = std::min<int64_t>((int64_t)B * Hkv, 1 << 20);  // work-items stay below 2^32
  hipLaunchKernelGGL(gather_read_kernel, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream,
                     static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), table, begin, end, n_parts, B,
                     Hkv, max_blocks, sink);
  return hipGetLastError();
}

}  // namespace bana
