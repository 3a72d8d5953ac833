// merge.hip -- log-sum-exp merge of partition partials (gfx950).
//
// Paper Sec. 4.1(2): the final output is the sum of the partitions' partial
// outputs once each is weighted by its share of the global softmax
// denominator (l^(j) = exp(lse_j)).  Per row r = (sequence, query head):
//   M = max_p lse_p,  w_p = exp(lse_p - M),
//   out = sum_p w_p out_p / sum_p w_p,  lse_out = M + ln sum_p w_p,
// skipping parts with lse_p = -inf (their out_p is never read); no live part
// gives out = 0, lse_out = -inf.  Parts are summed in index order, so the
// result is deterministic.  HBM-bound: one thread per 16-byte slice of a
// 128-float row, 32 consecutive threads per row, so each part's row is read
// with one fully coalesced 512-byte access.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kernels.h"

namespace bana {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ outs, const float* __restrict__ lses,
                                                    int n_parts, int64_t rows, float* __restrict__ out,
                                                    float* __restrict__ lse_out) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = tid >> 5;
  const int d4 = (int)(tid & 31);
  if (row >= rows) return;
  float M = -INFINITY;
  for (int p = 0; p < n_parts; ++p) M = fmaxf(M, lses[(int64_t)p * rows + row]);
  f32x4* dst = reinterpret_cast<f32x4*>(out + row * 128) + d4;
  if (M == -INFINITY) {
    *dst = f32x4{0.f, 0.f, 0.f, 0.f};
    if (lse_out != nullptr && d4 == 0) lse_out[row] = -INFINITY;
    return;
  }
  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < n_parts; ++p) {
    const float l = lses[(int64_t)p * rows + row];
    if (l == -INFINITY) continue;
    const float w = expf(l - M);
    wsum += w;
    acc += w * reinterpret_cast<const f32x4*>(outs + ((int64_t)p * rows + row) * 128)[d4];
  }
  *dst = acc * (1.0f / wsum);
  if (lse_out != nullptr && d4 == 0) lse_out[row] = M + logf(wsum);
}

}  // namespace

hipError_t launch_merge(const float* outs, const float* lses, int n_parts, int64_t rows, float* out, float* lse_out,
                        hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  const int64_t threads = rows * 32;
  const unsigned grid = (unsigned)((threads + 255) / 256);
  hipLaunchKernelGGL(merge_kernel, dim3(grid), dim3(256), 0, stream, outs, lses, n_parts, rows, out, lse_out);
  return hipGetLastError();
}

}  // namespace bana
