// debug_rows.hip -- export of the (tile, slot) pairs the partial-attention kernel reads (test hook).
//
// Uses the same address helpers as the attention kernel: for each sequence b,
// kv head g and logical token t of the table span, the pool-wide slot index of
// (tile (block_table[b][t / 16], g), slot t % 16) when t is inside
// [begin[b], end[b]), else -1.  Table entries outside the covered blocks are
// never read.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
#include "paged_addr.h"

namespace bana {
namespace {

__global__ __launch_bounds__(256) void debug_rows_kernel(const int32_t* __restrict__ table,
                                                         const int32_t* __restrict__ begin,
                                                         const int32_t* __restrict__ end, int B, int Hkv,
                                                         int max_blocks, int64_t* __restrict__ rows) {
  const int64_t span = (int64_t)max_blocks * kBlockSize;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= (int64_t)B * Hkv * span) return;
  const int t = (int)(tid % span);
  const int g = (int)((tid / span) % Hkv);
  const int b = (int)(tid / (span * Hkv));
  int64_t r = -1;
  if (t >= begin[b] && t < end[b]) {
    const int64_t tile = kv_tile(table_lookup(table, max_blocks, b, t / kBlockSize), g, Hkv);
    r = tile_slot(tile, t % kBlockSize);
  }
  rows[tid] = r;
}

}  // namespace

hipError_t launch_debug_rows(const int32_t* table, const int32_t* begin, const int32_t* end, int B, int Hkv,
                             int max_blocks, int64_t* rows, hipStream_t stream) {
  const int64_t n = (int64_t)B * Hkv * max_blocks * kBlockSize;
  if ((n + 255) / 256 > (int64_t)UINT32_MAX / 256) return hipErrorInvalidValue;  // grid x limit
  const unsigned grid = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(debug_rows_kernel, dim3(grid), dim3(256), 0, stream, table, begin, end, B, Hkv, max_blocks,
                     rows);
  return hipGetLastError();
}

}  // namespace bana
