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
// one coalesced 512-byte access per part).  Two kernels:
//  * up to four parts (the usual local + migrated split): every lse and every
//    partial row is loaded up front, before any of them is used, so the
//    kernel waits on one round of memory latency;
//  * more parts (many migrated partitions, or the chunk partials of long
//    ranges): the 32 lanes of a row first read 32 parts' lse at once and
//    reduce their max with lane shuffles, then stream the partial rows with
//    loads that do not depend on any lse (the weights come from the lanes by
//    shuffle), so loads of consecutive parts overlap.  With few rows the parts
//    of a row are spread over KP thread groups; each group keeps its sums
//    relative to its own max and the KP groups are combined through LDS,
//    rescaled to the common max (the same log-sum-exp algebra once more).
// The part-to-group assignment and every summation order depend only on
// n_parts and the number of merged rows, so results are deterministic.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kernels.h"

namespace bana {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// At most NP parts, all loaded before use.  Parts with lse = -inf are loaded
// too (their rows lie inside the partial buffer) but never enter a sum.
template <int NP>
__global__ __launch_bounds__(256) void merge_few_kernel(const float* __restrict__ outs,
                                                        const float* __restrict__ lses, int n_parts, MergeRows mr,
                                                        float* __restrict__ out, float* __restrict__ lse_out) {
  const int t = threadIdx.x;
  const int d4 = t & 31;
  const int64_t r = (int64_t)blockIdx.x * 8 + (t >> 5);
  if (r >= mr.B * mr.hn) return;
  const int64_t rows = mr.B * mr.in_hq;
  const int64_t b = r / mr.hn, i = r % mr.hn;
  const int64_t row = b * mr.in_hq + mr.in_h0 + i;
  const int64_t orow = b * mr.out_hq + mr.out_h0 + i;
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
  f32x4* dst = reinterpret_cast<f32x4*>(out + orow * 128) + d4;
  if (M == -INFINITY) {
    *dst = f32x4{0.f, 0.f, 0.f, 0.f};
    if (lse_out != nullptr && d4 == 0) lse_out[orow] = -INFINITY;
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
  if (lse_out != nullptr && d4 == 0) lse_out[orow] = M + logf(wsum);
}

// Any number of parts.  Group k (of KP) of a row takes parts k, k + KP, ...;
// its q-th part is p = k + KP q.  Part p of merged row r (head i of sequence
// b) is row base + p * prow of the part buffers: base = b * in_hq + in_h0 + i
// and prow = B x in_hq for partials [n_parts][B][in_hq]; for the balanced
// launch's pieces, base is the head's row in the sequence's first piece slot
// and prow = in_hq (the slots of a sequence's pieces are consecutive), and the
// part count comes from the block-count prefix sums (pieces = intervals of S
// blocks that overlap the sequence's blocks [prefix[b], prefix[b + 1])).
//
// Rows stream in rounds of U parts, each round requested before the previous one is summed (the
// waits the compiler places keep about one round in flight per lane, its loads overlapping the
// sums of the round before).  The many-part merge of many rows takes one part per round: with fewer
// part streams in flight per wavefront the 16-part merge of 32,768 rows runs in 50 us instead of
// 57 (U = 4) or 62 (U = 8) on MI355X, cold caches; the piece merges, few pieces per row, keep
// U = 4 (U = 1 costs them 2 us).
template <int KP, bool PIECES, int U>
__global__ __launch_bounds__(256) void merge_many_kernel(const float* __restrict__ outs,
                                                         const float* __restrict__ lses, int n_parts, MergeRows mr,
                                                         float* __restrict__ out, float* __restrict__ lse_out,
                                                         const int32_t* __restrict__ prefix, int K) {
  constexpr int R = 256 / (32 * KP);  // rows per workgroup
  __shared__ f32x4 sm_acc[KP > 1 ? R * KP * 32 : 1];
  __shared__ float sm_m[KP > 1 ? R * KP : 1];
  __shared__ float sm_w[KP > 1 ? R * KP : 1];
  const int t = threadIdx.x;
  const int d4 = t & 31;
  const int k = (t >> 5) % KP;
  const int rl = t / (32 * KP);
  const int64_t r = (int64_t)blockIdx.x * R + rl;  // row among the B x hn merged rows
  const bool live = r < mr.B * mr.hn;
  const int64_t b = live ? r / mr.hn : 0;
  const int64_t i = live ? r % mr.hn : 0;
  const int64_t dst_row = b * mr.out_hq + mr.out_h0 + i;
  int64_t base = b * mr.in_hq + mr.in_h0 + i;
  int64_t prow = mr.B * mr.in_hq;
  int n = n_parts;
  if (PIECES) {
    n = 0;
    prow = mr.in_hq;
    if (live) {
      const int p0 = prefix[b], p1 = prefix[b + 1], total = prefix[mr.B];
      const int64_t S = total > K ? ((int64_t)total + K - 1) / K : 1;
      if (p1 > p0) {  // slots clamped to [b, K + b): prefix sums from another call cannot reach outside
        const int64_t first = min(max((int64_t)p0 / S, (int64_t)0), (int64_t)K - 1);
        const int64_t last = min(max((int64_t)(p1 - 1) / S, first), (int64_t)K - 1);
        n = (int)(last - first + 1);
        base = (first + b) * mr.in_hq + mr.in_h0 + i;
      }
    }
  }
  const int nq = live && n > k ? (n - k + KP - 1) / KP : 0;
  const int64_t lstride = (int64_t)KP * prow;                   // from the q-th part of the group to the next
  const float* lrow = lses + (int64_t)k * prow + base;           // lse of the q-th part: lrow[q * lstride]
  const float* orow = outs + ((int64_t)k * prow + base) * 128;  // its row: orow + q * lstride * 128

  // Group max: lane d4 reads parts q = d4, d4 + 32, ...  The first round of partial rows is
  // requested at the same time: rows do not depend on any lse (the weights reach them by
  // shuffle), so the group waits on one round of memory latency for both.  Then the rows stream
  // in rounds of U, the next round requested before the current one is summed.  Rows of
  // empty parts are loaded too (they lie inside the part buffer) but never enter a sum.
  float l0 = -INFINITY;
  if (d4 < nq) l0 = lrow[d4 * lstride];
  f32x4 o[U];
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (u < nq) o[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(orow + u * lstride * 128) + d4);
  float m = l0;
  for (int q = d4 + 32; q < nq; q += 32) m = fmaxf(m, lrow[q * lstride]);
#pragma unroll
  for (int off = 16; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 32));

  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (m != -INFINITY) {
    // Weight of part 32r + d4 on lane d4 for the current round r of 32 parts (0 past the end
    // and for empty parts).
    float wq = l0 == -INFINITY ? 0.f : expf(l0 - m);
#pragma unroll 1
    for (int q = 0; q < nq; q += U) {
      if (q > 0 && (q & 31) == 0) {
        const float lq = q + d4 < nq ? lrow[(q + d4) * lstride] : -INFINITY;
        wq = lq == -INFINITY ? 0.f : expf(lq - m);
      }
      f32x4 cur[U];
#pragma unroll
      for (int u = 0; u < U; ++u) cur[u] = o[u];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (q + U + u < nq)
          o[u] = __builtin_nontemporal_load(
              reinterpret_cast<const f32x4*>(orow + (q + U + u) * lstride * 128) + d4);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (q + u < nq) {
          const float w = __shfl(wq, (q + u) & 31, 32);
          wsum += w;
          if (w != 0.f) acc += w * cur[u];
        }
      }
    }
  }
  float M = m;
  if (KP > 1) {
    race_check_delay(t >> 6);
    sm_acc[(rl * KP + k) * 32 + d4] = acc;
    if (d4 == 0) {
      sm_m[rl * KP + k] = m;
      sm_w[rl * KP + k] = wsum;
    }
    __syncthreads();
    race_check_barrier();
    if (k != 0) return;
    M = -INFINITY;
#pragma unroll
    for (int j = 0; j < KP; ++j) M = fmaxf(M, sm_m[rl * KP + j]);
    acc = f32x4{0.f, 0.f, 0.f, 0.f};
    wsum = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        const float mj = sm_m[rl * KP + j];
        if (mj == -INFINITY) continue;
        const float s = expf(mj - M);
        acc += s * sm_acc[(rl * KP + j) * 32 + d4];
        wsum += s * sm_w[rl * KP + j];
      }
    }
  }
  if (!live) return;
  f32x4* dst = reinterpret_cast<f32x4*>(out + dst_row * 128) + d4;
  if (M == -INFINITY) {
    *dst = f32x4{0.f, 0.f, 0.f, 0.f};
    if (lse_out != nullptr && d4 == 0) lse_out[dst_row] = -INFINITY;
    return;
  }
  *dst = acc * (1.0f / wsum);
  if (lse_out != nullptr && d4 == 0) lse_out[dst_row] = M + logf(wsum);
}

template <int KP, bool PIECES = false>
hipError_t launch_many(const float* outs, const float* lses, int n_parts, const MergeRows& m, float* out,
                       float* lse_out, hipStream_t stream, const int32_t* prefix = nullptr, int K = 0) {
  constexpr int R = 256 / (32 * KP);
  const int64_t rows = m.B * m.hn;
  const unsigned grid = (unsigned)((rows + R - 1) / R);
  constexpr int U = KP == 1 && !PIECES ? 1 : 4;
  hipLaunchKernelGGL((merge_many_kernel<KP, PIECES, U>), dim3(grid), dim3(256), 0, stream, outs, lses, n_parts, m,
                     out, lse_out, prefix, K);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const float* outs, const float* lses, int n_parts, MergeRows m, float* out, float* lse_out,
                        hipStream_t stream) {
  const int64_t rows = m.B * m.hn;
  if (rows == 0) return hipSuccess;
  if (n_parts <= 4) {
    hipLaunchKernelGGL(merge_few_kernel<4>, dim3((unsigned)((rows + 7) / 8)), dim3(256), 0, stream, outs, lses,
                       n_parts, m, out, lse_out);
    return hipGetLastError();
  }
  // With enough rows to fill the GPU, one thread group per row streams best.
  // With few rows (long ranges of few sequences), spread a row's parts over
  // up to 8 thread groups, at least 4 parts each.
  if (rows < 4096) {
    if (n_parts >= 32) return launch_many<8>(outs, lses, n_parts, m, out, lse_out, stream);
    if (n_parts >= 16) return launch_many<4>(outs, lses, n_parts, m, out, lse_out, stream);
    if (n_parts >= 8) return launch_many<2>(outs, lses, n_parts, m, out, lse_out, stream);
  }
  return launch_many<1>(outs, lses, n_parts, m, out, lse_out, stream);
}

hipError_t launch_merge_pieces(const float* outs, const float* lses, const int32_t* prefix, int K, int kp,
                               MergeRows m, float* out, float* lse_out, hipStream_t stream) {
  const int64_t rows = m.B * m.hn;
  if (rows == 0) return hipSuccess;
  switch (kp) {
    case 1: return launch_many<1, true>(outs, lses, 0, m, out, lse_out, stream, prefix, K);
    case 2: return launch_many<2, true>(outs, lses, 0, m, out, lse_out, stream, prefix, K);
    case 4: return launch_many<4, true>(outs, lses, 0, m, out, lse_out, stream, prefix, K);
    case 8: return launch_many<8, true>(outs, lses, 0, m, out, lse_out, stream, prefix, K);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bana
