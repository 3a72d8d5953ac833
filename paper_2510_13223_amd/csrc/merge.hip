// merge.hip -- log-sum-exp merge of partition partials (gfx950).
//
// Paper Sec. 4.1(2): the final output is the sum of the partitions' partial
// outputs once each is weighted by its share of the global softmax
// denominator (l^(j) = exp(lse_j)).  Per row r = (sequence, query head):
//   M = max_p lse_p,  w_p = exp(lse_p - M),
//   out = sum_p w_p out_p / sum_p w_p,  lse_out = M + ln sum_p w_p,
// skipping parts with lse_p = -inf (their out_p never enters a sum); no live part
// gives out = 0, lse_out = -inf.
//
// HBM-bound.  32 consecutive threads cover one 128-float row (16 bytes each,
// one coalesced 512-byte access per part).  With many parts per row (the
// chunk partials of a long range, or many migrated partitions) the parts of
// a row are spread over KP thread groups that load independently, so the
// merge is not a chain of dependent loads; the KP partial sums are added in
// group order through LDS.  With at most four parts (the usual local +
// migrated split) every lse and every partial row is loaded up front, before
// any of them is used, so the kernel waits on one round of memory latency
// instead of two.  The part-to-group assignment and every summation order
// depend only on n_parts, so results are deterministic.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kernels.h"

namespace bana {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int KP>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ outs, const float* __restrict__ lses,
                                                    int n_parts, int64_t B, int Hq, int h0, int hn,
                                                    float* __restrict__ out, float* __restrict__ lse_out) {
  constexpr int R = 256 / (32 * KP);  // rows per workgroup
  __shared__ f32x4 sm_acc[KP > 1 ? R * KP * 32 : 1];
  __shared__ float sm_w[KP > 1 ? R * KP : 1];
  const int t = threadIdx.x;
  const int d4 = t & 31;
  const int k = (t >> 5) % KP;  // part group
  const int rl = t / (32 * KP);
  const int64_t r = (int64_t)blockIdx.x * R + rl;  // row among the B x hn merged rows
  const int64_t rows = B * Hq;                      // row stride of one part
  const bool live = r < B * hn;
  const int64_t row = live ? (r / hn) * Hq + h0 + r % hn : 0;

  float M = -INFINITY;
  if (live)
    for (int p = 0; p < n_parts; ++p) M = fmaxf(M, lses[(int64_t)p * rows + row]);
  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (live && M != -INFINITY) {
    for (int p = k; p < n_parts; p += KP) {
      const float l = lses[(int64_t)p * rows + row];
      if (l == -INFINITY) continue;
      const float w = expf(l - M);
      wsum += w;
      acc += w * reinterpret_cast<const f32x4*>(outs + ((int64_t)p * rows + row) * 128)[d4];
    }
  }
  if (KP > 1) {
    sm_acc[(rl * KP + k) * 32 + d4] = acc;
    if (d4 == 0) sm_w[rl * KP + k] = wsum;
    __syncthreads();
    if (k != 0) return;
    acc = f32x4{0.f, 0.f, 0.f, 0.f};
    wsum = 0.f;
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      acc += sm_acc[(rl * KP + j) * 32 + d4];
      wsum += sm_w[rl * KP + j];
    }
  }
  if (!live) return;
  f32x4* dst = reinterpret_cast<f32x4*>(out + row * 128) + d4;
  if (M == -INFINITY) {
    *dst = f32x4{0.f, 0.f, 0.f, 0.f};
    if (lse_out != nullptr && d4 == 0) lse_out[row] = -INFINITY;
    return;
  }
  *dst = acc * (1.0f / wsum);
  if (lse_out != nullptr && d4 == 0) lse_out[row] = M + logf(wsum);
}

// At most NP parts, all loaded before use.  Parts with lse = -inf are loaded
// too (their rows lie inside the partial buffer) but never enter a sum.
template <int NP>
__global__ __launch_bounds__(256) void merge_few_kernel(const float* __restrict__ outs,
                                                        const float* __restrict__ lses, int n_parts, int64_t B,
                                                        int Hq, int h0, int hn, float* __restrict__ out,
                                                        float* __restrict__ lse_out) {
  const int t = threadIdx.x;
  const int d4 = t & 31;
  const int64_t r = (int64_t)blockIdx.x * 8 + (t >> 5);
  if (r >= B * hn) return;
  const int64_t rows = B * Hq;
  const int64_t row = (r / hn) * Hq + h0 + r % hn;
  float l[NP];
  f32x4 o[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    if (p < n_parts) {
      l[p] = lses[(int64_t)p * rows + row];
      o[p] = reinterpret_cast<const f32x4*>(outs + ((int64_t)p * rows + row) * 128)[d4];
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int p = 0; p < NP; ++p)
    if (p < n_parts) M = fmaxf(M, l[p]);
  f32x4* dst = reinterpret_cast<f32x4*>(out + row * 128) + d4;
  if (M == -INFINITY) {
    *dst = f32x4{0.f, 0.f, 0.f, 0.f};
    if (lse_out != nullptr && d4 == 0) lse_out[row] = -INFINITY;
    return;
  }
  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    if (p < n_parts && l[p] != -INFINITY) {
      const float w = expf(l[p] - M);
      wsum += w;
      acc += w * o[p];
    }
  }
  *dst = acc * (1.0f / wsum);
  if (lse_out != nullptr && d4 == 0) lse_out[row] = M + logf(wsum);
}

template <int KP>
hipError_t launch(const float* outs, const float* lses, int n_parts, int64_t B, int Hq, int h0, int hn, float* out,
                  float* lse_out, hipStream_t stream) {
  constexpr int R = 256 / (32 * KP);
  const int64_t rows = B * hn;
  const unsigned grid = (unsigned)((rows + R - 1) / R);
  hipLaunchKernelGGL(merge_kernel<KP>, dim3(grid), dim3(256), 0, stream, outs, lses, n_parts, B, Hq, h0, hn, out,
                     lse_out);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const float* outs, const float* lses, int n_parts, int64_t B, int Hq, int h0, int hn,
                        float* out, float* lse_out, hipStream_t stream) {
  const int64_t rows = B * hn;
  if (rows == 0) return hipSuccess;
  if (n_parts <= 4) {
    hipLaunchKernelGGL(merge_few_kernel<4>, dim3((unsigned)((rows + 7) / 8)), dim3(256), 0, stream, outs, lses,
                       n_parts, B, Hq, h0, hn, out, lse_out);
    return hipGetLastError();
  }
  // With enough rows to fill the GPU, one thread group per row streams best.
  // With few rows (long ranges of few sequences), spread a row's parts over
  // up to 8 thread groups, at least 2 parts each.
  if (rows < 4096) {
    if (n_parts >= 16) return launch<8>(outs, lses, n_parts, B, Hq, h0, hn, out, lse_out, stream);
    if (n_parts >= 8) return launch<4>(outs, lses, n_parts, B, Hq, h0, hn, out, lse_out, stream);
    if (n_parts >= 4) return launch<2>(outs, lses, n_parts, B, Hq, h0, hn, out, lse_out, stream);
  }
  return launch<1>(outs, lses, n_parts, B, Hq, h0, hn, out, lse_out, stream);
}

}  // namespace bana
