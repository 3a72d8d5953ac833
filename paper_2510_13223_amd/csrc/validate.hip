// validate.hip -- device-side check of the preconditions of the attention and migration calls.
//
// The attention kernels trust the device-resident arguments (reading them back to the host would
// cost a synchronisation per call).  This kernel checks them on the device and folds the first
// broken rule per (partition, sequence) into one code with an atomic max, so a caller can verify
// a batch's ranges and tables once, asynchronously, before using them:
//   1  kv_range_begin < 0 or kv_range_begin > kv_range_end
//   2  kv_range_end > seq_lens
//   3  seq_lens < 0 or seq_lens > max_blocks_per_seq * block_size
//   4  a block overlapping [begin, end) maps to no block of the pool (entry < 0 or >= num_blocks)
// Table entries are read only for blocks of ranges that passed rules 1-3, so the check itself
// never reads outside the table.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
#include "paged_addr.h"

namespace bana {
namespace {

__global__ void zero_kernel(int32_t* result) { *result = 0; }

__global__ __launch_bounds__(256) void validate_kernel(const int32_t* __restrict__ table,
                                                       const int32_t* __restrict__ seq_lens,
                                                       const int32_t* __restrict__ begin,
                                                       const int32_t* __restrict__ end, int B, int max_blocks,
                                                       int64_t num_blocks, int32_t* result) {
  const int p = blockIdx.y;
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    const int t0 = begin[(int64_t)p * B + b];
    const int t1 = end[(int64_t)p * B + b];
    const int L = seq_lens[b];
    int code = 0;
    if (L < 0 || (int64_t)L > (int64_t)max_blocks * kBlockSize) code = 3;
    else if (t0 < 0 || t0 > t1) code = 1;
    else if (t1 > L) code = 2;
    if (code != 0) {
      if (threadIdx.x == 0) atomicMax(result, code);
      continue;
    }
    if (t1 == t0) continue;
    const int j0 = t0 / kBlockSize, j1 = (t1 - 1) / kBlockSize;
    bool bad = false;
    for (int j = j0 + (int)threadIdx.x; j <= j1; j += (int)blockDim.x) {
      const int32_t blk = table[(int64_t)b * max_blocks + j];
      bad |= blk < 0 || (int64_t)blk >= num_blocks;
    }
    if (bad) atomicMax(result, 4);
  }
}

}  // namespace

hipError_t launch_validate(const int32_t* table, const int32_t* seq_lens, const int32_t* begin, const int32_t* end,
                           int n_parts, int B, int max_blocks, int64_t num_blocks, int32_t* result,
                           hipStream_t stream) {
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(1), 0, stream, result);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Workgroups stride over the sequences; the row width only sets parallelism.
  const unsigned row = (unsigned)(B < (1 << 16) ? B : (1 << 16));
  hipLaunchKernelGGL(validate_kernel, dim3(row, (unsigned)n_parts), dim3(256), 0, stream, table, seq_lens,
                     begin, end, B, max_blocks, num_blocks, result);
  return hipGetLastError();
}

}  // namespace bana
