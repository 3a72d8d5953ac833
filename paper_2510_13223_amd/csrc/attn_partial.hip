// attn_partial.hip -- partial attention of one KV partition over a paged cache (gfx950).
//
// Computes, per (sequence b, query head h) and over the logical tokens of
// the ranges [begin[p][b], end[p][b]) of n_parts partitions, the softmax-
// normalised output and its log-sum-exp (paper Sec. 4.1(2): S = Q K^T,
// A = exp S, l = sum A, O = A / l . V; the max-subtracted online form keeps
// the same value in a finite range).  With one partition this is that
// partition's partial; with several it is their merge (the online softmax
// running over the partitions one after the other is the same log-sum-exp
// algebra as the final O = O^(1) + O^(2)), computed in one launch.
//
// Work decomposition.  The blocks of a sequence's ranges are concatenated
// into one virtual block sequence, mapped back to (range, logical block) by
// a segment cursor.  Two launch shapes:
//  * chunked: one workgroup per (chunk c, sequence b, kv head g),
//    linearised chunk-major so that every (b, g) has its first chunk in the
//    first wave of dispatch.  A workgroup of W wavefronts walks the virtual
//    blocks of its chunk round-robin (block jr goes to wave jr % W); each
//    wavefront keeps an online-softmax state for all G query heads of the
//    kv head, and the W states are combined through LDS at the end.  A range
//    longer than one chunk leaves one partial per chunk in caller workspace,
//    merged by the merge kernel with the same log-sum-exp algebra as the
//    partition merge.
//  * balanced (uneven ranges, up to 2048 sequences): the virtual blocks of all
//    sequences, in sequence order, form one list per kv head, cut into K
//    equal intervals of S = ceil(U / K) blocks (U = blocks of the whole call),
//    one per wavefront.  A wavefront walks its interval block by block,
//    leaving one partial per sequence piece it covers in workspace slot
//    (k + b), which is unique (an interval and a sequence that overlap bound
//    each other's position); the merge finds a sequence's pieces from the
//    prefix sums of the block counts.  Every wavefront gets the same number of
//    blocks whatever the lengths, so one long range no longer sets the time
//    of the launch, and no range has to be rounded to whole chunks.
//
// One KV block (16 tokens x 128 dims for one kv head) per wavefront step:
//   scores  S^T[16 tok x 16 col] = K[16 tok x 128] . Q^T[128 x 16 col]
//           4 x v_mfma_f32_16x16x32_bf16, A = K straight from HBM (lane =
//           token row; the chunked K tile makes each 16-byte-per-lane load
//           one contiguous 1 KiB), B = Q of the G heads of the group
//           (columns >= G are zero).  bf16 x bf16 products are exact in
//           fp32, accumulation is fp32.
//   softmax running max per column (4 values per lane + two cross-lane
//           shuffles), p = 2^((s - m) log2 e), rescale of the accumulator.
//   values  O^T[128 dim x 16 col] += V^T[128 x 16 tok] . P^T[16 tok x 16 col]
//           8 tiles of v_mfma_f32_16x16x16_bf16.  The score tile's output
//           layout (lane = column, 4 consecutive token rows per lane) is
//           exactly the B-operand layout of this product, so P never leaves
//           its registers; V comes from the dim-major V tile with 8-byte loads
//           (4 consecutive tokens of one dim).  P is split into a bf16 high
//           part and a bf16 residual (two MFMAs per tile) so PV keeps ~16
//           significant bits of P instead of bf16's 8.
// K and V are read exactly once, so their loads carry the non-temporal hint
// (streaming through the caches instead of allocating in them).  With every
// load instruction covering whole 128-byte lines (1 KiB for K, 512 bytes for
// V) this lifts sustained HBM read bandwidth on random 4 KiB tiles by about
// a tenth; loads that split lines across instructions do not gain.
// Tokens of a partly covered block are selected out (score -inf, value 0),
// never multiplied by zero, so NaN in unused slots cannot leak.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kernels.h"
#include "paged_addr.h"

namespace bana {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kDimTiles = kHeadDim / 16;  // 8 output tiles of 16 dims
constexpr int kRowPad = kHeadDim + 4;     // LDS row stride (floats) for the combine

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wavefront timeline (a measurement build only, BANA_WAVE_TIMELINE): lane 0 of every wavefront of
// the attention launches stores readings of the constant 100 MHz clock in its slot
// (workgroup * wavefronts per workgroup + wavefront, modulo the table): entry, schedule ready,
// first block consumed (the earliest over its pieces), exit.  The product build compiles the
// marks away.
#ifdef BANA_WAVE_TIMELINE
__device__ unsigned long long g_wave_timeline[(size_t)BANA_TIMELINE_SLOTS * 4];
__device__ __forceinline__ unsigned long long* timeline_slot() {
  const unsigned slot = (blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) % BANA_TIMELINE_SLOTS;
  return g_wave_timeline + (size_t)slot * 4;
}
#define BANA_TIMELINE_MARK(i)                                                      \
  do {                                                                             \
    const unsigned long long t_ = __builtin_amdgcn_s_memrealtime();                \
    if ((threadIdx.x & 63) == 0) timeline_slot()[i] = t_;                          \
  } while (0)
#define BANA_TIMELINE_FIRST()                                                      \
  do {                                                                             \
    const unsigned long long t_ = __builtin_amdgcn_s_memrealtime();                \
    if ((threadIdx.x & 63) == 0) atomicMin(timeline_slot() + 2, t_);               \
  } while (0)
#else
#define BANA_TIMELINE_MARK(i) ((void)0)
#define BANA_TIMELINE_FIRST() ((void)0)
#endif

// Max over the 4 lanes of a column (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float column_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

__device__ __forceinline__ float column_sum(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// p = hi + lo with hi = p truncated to bf16 (exact in fp32) and lo = bf16
// round-to-nearest-even of the exact residual p - hi.  p is finite, >= 0.
__device__ __forceinline__ void split_bf16(float p, uint32_t& hi, uint32_t& lo) {
  const uint32_t u = __builtin_bit_cast(uint32_t, p);
  hi = u >> 16;
  const float r = p - __builtin_bit_cast(float, u & 0xFFFF0000u);
  const uint32_t ur = __builtin_bit_cast(uint32_t, r);
  lo = (ur + 0x7FFFu + ((ur >> 16) & 1u)) >> 16;
}

// K tile of one (block, kv head), stored as 16 chunks of 8 dims x 16 tokens:
// lane (col, quad) takes token row col, dims 32kk + 8quad + [0, 8), which is
// chunk 4kk + quad, so instruction kk reads 1 KiB at lane * 16 bytes.
__device__ __forceinline__ void load_k(u32x4 (&kr)[4], const uint16_t* __restrict__ k, int64_t tile, int col,
                                       int quad) {
  const u32x4* src = reinterpret_cast<const u32x4*>(k + tile * kTileElems) + (quad * kBlockSize + col);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) kr[kk] = __builtin_nontemporal_load(src + 4 * kBlockSize * kk);
}

// V tile (dim-major): lane (col, quad) takes dim 16dt + col, token slots 4quad + [0, 4).
__device__ __forceinline__ void load_v(u32x2 (&vr)[kDimTiles], const uint16_t* __restrict__ v, int64_t tile, int col,
                                       int quad) {
  const u32x2* src = reinterpret_cast<const u32x2*>(v + tile * kTileElems + col * kBlockSize + 4 * quad);
#pragma unroll
  for (int dt = 0; dt < kDimTiles; ++dt) vr[dt] = __builtin_nontemporal_load(src + 4 * 16 * dt);
}

// B operand of the score product: Q^T, lane (col, quad) holds dims 32kk + 8quad + [0, 8)
// of head hq0 + col (zero for col >= G).
__device__ __forceinline__ void load_q(bf16x8 (&qop)[4], const uint16_t* __restrict__ q, int64_t row0, int col,
                                       int quad, int G) {
  const uint16_t* qrow = q + (row0 + (col < G ? col : 0)) * kHeadDim + 8 * quad;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    u32x4 v = *reinterpret_cast<const u32x4*>(qrow + 32 * kk);
    if (col >= G) v = u32x4{0u, 0u, 0u, 0u};
    qop[kk] = __builtin_bit_cast(bf16x8, v);
  }
}

// Scores of one block: s[i] = q(head col) . k(token slot 4*quad + i).
__device__ __forceinline__ f32x4 block_scores(const bf16x8 (&qop)[4], const u32x4 (&kr)[4]) {
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
    s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[kk]), qop[kk], s, 0, 0, 0);
  return s;
}

// Online-softmax state of one wavefront: acc[dt][i] = unnormalised output for
// dim 16dt + 4quad + i of head col; m = running max; lsum = this lane's share
// of the running sum (its token rows only, summed over the column at the end).
struct Online {
  f32x4 acc[kDimTiles];
  float m;
  float lsum;

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int dt = 0; dt < kDimTiles; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    m = -INFINITY;
    lsum = 0.f;
  }

  // Online-softmax update and value accumulation of logical block j of a
  // range [t0, t1) (j overlaps the range).
  __device__ __forceinline__ void update(f32x4 s, u32x2 (&vr)[kDimTiles], const int j, const int t0, const int t1,
                                         const int quad) {
    if (j * kBlockSize < t0 || j * kBlockSize + kBlockSize > t1) {  // partly covered block (wave-uniform)
      const int tok = j * kBlockSize + 4 * quad;
      const bool ok0 = tok + 0 >= t0 && tok + 0 < t1;
      const bool ok1 = tok + 1 >= t0 && tok + 1 < t1;
      const bool ok2 = tok + 2 >= t0 && tok + 2 < t1;
      const bool ok3 = tok + 3 >= t0 && tok + 3 < t1;
      s[0] = ok0 ? s[0] : -INFINITY;
      s[1] = ok1 ? s[1] : -INFINITY;
      s[2] = ok2 ? s[2] : -INFINITY;
      s[3] = ok3 ? s[3] : -INFINITY;
      const uint32_t mlo = (ok0 ? 0x0000FFFFu : 0u) | (ok1 ? 0xFFFF0000u : 0u);
      const uint32_t mhi = (ok2 ? 0x0000FFFFu : 0u) | (ok3 ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int dt = 0; dt < kDimTiles; ++dt) {
        vr[dt][0] &= mlo;
        vr[dt][1] &= mhi;
      }
    }

    const float mx = column_max(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
    const float m_new = fmaxf(m, mx);  // finite: every visited block covers >= 1 token
    const float alpha = fast_exp2((m - m_new) * kLog2e);
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = fast_exp2((s[i] - m_new) * kLog2e);
    lsum = lsum * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    m = m_new;

    uint32_t h0, l0, h1, l1, h2, l2, h3, l3;
    split_bf16(p[0], h0, l0);
    split_bf16(p[1], h1, l1);
    split_bf16(p[2], h2, l2);
    split_bf16(p[3], h3, l3);
    const i16x4 phi = __builtin_bit_cast(i16x4, u32x2{h0 | (h1 << 16), h2 | (h3 << 16)});
    const i16x4 plo = __builtin_bit_cast(i16x4, u32x2{l0 | (l1 << 16), l2 | (l3 << 16)});
#pragma unroll
    for (int dt = 0; dt < kDimTiles; ++dt) {
      f32x4 t = acc[dt] * alpha;
      const i16x4 va = __builtin_bit_cast(i16x4, vr[dt]);
      t = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, phi, t, 0, 0, 0);
      acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, plo, t, 0, 0, 0);
    }
  }

  // Normalised rows of the G heads (out_dst row = head in group) and their lse.
  __device__ __forceinline__ void emit(float* __restrict__ out_dst, float* __restrict__ lse_dst, int col, int quad,
                                       int G) {
    const float l = column_sum(lsum);
    if (col < G) {
      const float inv = 1.0f / l;
#pragma unroll
      for (int dt = 0; dt < kDimTiles; ++dt)
        *reinterpret_cast<f32x4*>(out_dst + col * kHeadDim + 16 * dt + 4 * quad) = acc[dt] * inv;
      if (quad == 0) lse_dst[col] = m + logf(l);
    }
  }
};

// The ranges ("segments") of one sequence, one per lane p < n_parts, with
// the inclusive prefix sum of their block counts: the segments' blocks,
// concatenated, are the sequence's virtual block sequence [0, nblk).
struct Segments {
  int t0, t1, jfirst, nblk, vend;

  __device__ __forceinline__ void load(const PartialArgs& a, int b, int lane, int n_parts) {
    t0 = t1 = jfirst = nblk = 0;
    if (lane < n_parts) {
      t0 = a.begin[(int64_t)lane * a.B + b];
      t1 = a.end[(int64_t)lane * a.B + b];
      if (t1 > t0) {
        jfirst = t0 >> 4;
        nblk = ((t1 - 1) >> 4) - jfirst + 1;
      }
    }
    vend = nblk;
    if (n_parts == 1) return;  // one range: lane 0 holds it, nothing to sum
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(vend, off);
      if (lane >= off) vend += y;
    }
  }
  __device__ __forceinline__ int total(int n_parts) const { return __builtin_amdgcn_readlane(vend, n_parts - 1); }
};

// Cursor over the segments (wave-uniform): the segment holding virtual block
// v, advanced monotonically with readlane from the segment lanes.
struct Seg {
  int p, vstart, vend, jfirst, t0, t1;
};

__device__ __forceinline__ Seg seg_at(const Segments& sg, int p) {
  Seg c;
  c.p = p;
  c.vend = __builtin_amdgcn_readlane(sg.vend, p);
  c.vstart = c.vend - __builtin_amdgcn_readlane(sg.nblk, p);
  c.jfirst = __builtin_amdgcn_readlane(sg.jfirst, p);
  c.t0 = __builtin_amdgcn_readlane(sg.t0, p);
  c.t1 = __builtin_amdgcn_readlane(sg.t1, p);
  return c;
}

__device__ __forceinline__ void seek(const Segments& sg, Seg& c, int v, int n_parts) {
  while (v >= c.vend && c.p + 1 < n_parts) c = seg_at(sg, c.p + 1);
}

// Software pipeline over the virtual blocks jr, jr + STEP, ... < jb1 of
// sequence b, kv head g, one register set each for K and V: the next block's
// K is requested as soon as the score product has consumed the current one,
// and the next V as soon as the value product has consumed the current one,
// so about one block (8 KiB) per wave stays in flight through the softmax and
// MFMA work.  Table entries are read two blocks ahead with scalar loads.
// A wavefront that walks every block of its range alone (STEP 1: one-wavefront workgroups of the
// chunked launch, and the balanced launch) raises its issue priority until its first block has been
// consumed.  While the memory pipeline is full the hardware favours the oldest wavefronts, which
// always have their next load ready, so the last-dispatched ones would wait up to ~25 us for their
// first block and then walk all their blocks at the end of the launch (the timeline of fine's
// calls).  Measured on MI355X, cold caches: fine's 16 calls plus merge 840 against 848 us; mixed's
// migrated partition 67 against 68 us; results unchanged (priority changes only the order of issue).
template <int STEP>
__device__ __forceinline__ void walk_blocks(Online& st, const bf16x8 (&qop)[4], const Segments& sg, int n_parts,
                                            const PartialArgs& a, int b, int g, int col, int quad, int jr, int jb1) {
  if (jr >= jb1) return;
  const int vlast = jb1 - 1;
  if (STEP == 1) __builtin_amdgcn_s_setprio(3);
  Seg cm = seg_at(sg, 0);  // segment of the block being computed
  Seg ct = cm;             // segment of the block whose table entry is read
  auto table_at = [&](int v) {
    seek(sg, ct, v, n_parts);
    return table_lookup(a.table, a.max_blocks, b, ct.jfirst + (v - ct.vstart));
  };
  const int32_t blk_first = table_at(jr);
  int32_t blk_next = table_at(min(jr + STEP, vlast));
  u32x4 kr[4];
  u32x2 vr[kDimTiles];
  {
    const int64_t tile = kv_tile(blk_first, g, a.Hkv);
    load_k(kr, a.k, tile, col, quad);
    load_v(vr, a.v, tile, col, quad);
  }
  // Every load inside the loop is unconditional (the last block is peeled),
  // so the in-order memory counter lets each wait cover exactly the tile
  // it needs while the other one stays in flight.
  while (jr + STEP < jb1) {
    const int32_t blk_after = table_at(min(jr + 2 * STEP, vlast));
    const int64_t tile_next = kv_tile(blk_next, g, a.Hkv);
    const f32x4 s = block_scores(qop, kr);
    load_k(kr, a.k, tile_next, col, quad);
    seek(sg, cm, jr, n_parts);
    st.update(s, vr, cm.jfirst + (jr - cm.vstart), cm.t0, cm.t1, quad);
    BANA_TIMELINE_FIRST();
    if (STEP == 1) __builtin_amdgcn_s_setprio(0);
    load_v(vr, a.v, tile_next, col, quad);
    jr += STEP;
    blk_next = blk_after;
  }
  seek(sg, cm, jr, n_parts);
  st.update(block_scores(qop, kr), vr, cm.jfirst + (jr - cm.vstart), cm.t0, cm.t1, quad);
  BANA_TIMELINE_FIRST();
}

// Side copies: copy k is moved by the copy workgroups wg with wg % n == k, so all copies (host to
// device and device to host alike) proceed at the same time, each direction of the host link
// busy at once.  Within copy k, workgroup j of its m workgroups moves 16-byte units
// j * threads + tid, advancing by m * threads, kSideCopyUnroll units in flight per thread.  Either side may be
// device memory or pinned host memory; the source is read once (non-temporal), the destination is
// not read back by this launch (non-temporal stores).
constexpr int kSideCopyUnroll = 1;  // 16-byte units in flight per thread of a copy workgroup

__device__ __forceinline__ void side_copy(const SideCopies& c, int wg, int tid, int threads) {
  const int k = wg % c.n;
  const int m = (c.n_wg - k + c.n - 1) / c.n;  // workgroups of copy k
  const int64_t stride = (int64_t)m * threads;
  const int64_t first = (int64_t)(wg / c.n) * threads + tid;
  {
    const u32x4* __restrict__ src = static_cast<const u32x4*>(c.src[k]);
    u32x4* __restrict__ dst = static_cast<u32x4*>(c.dst[k]);
    const int64_t n = c.n16[k];
    for (int64_t i0 = first; i0 < n; i0 += kSideCopyUnroll * stride) {
      u32x4 x[kSideCopyUnroll];
#pragma unroll
      for (int u = 0; u < kSideCopyUnroll; ++u)
        if (i0 + u * stride < n) x[u] = __builtin_nontemporal_load(src + i0 + u * stride);
#pragma unroll
      for (int u = 0; u < kSideCopyUnroll; ++u)
        if (i0 + u * stride < n) __builtin_nontemporal_store(x[u], dst + i0 + u * stride);
    }
  }
}

// MULTI: the call passes several ranges per sequence (the fused entry point); a
// single range (one partition) compiles the segment handling away.
template <int W, bool MULTI>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(4, 8))) void partial_attn_kernel(PartialArgs a) {
  extern __shared__ float smem[];
  const int n_parts = MULTI ? a.n_parts : 1;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int col = lane & 15;  // query head in group (score/output column); token row for K; dim for V
  const int quad = lane >> 4;

  if (blockIdx.x < (unsigned)a.copies.n_wg) {  // side-copy workgroups come first
    side_copy(a.copies, blockIdx.x, threadIdx.x, 64 * W);
    return;
  }
  BANA_TIMELINE_MARK(0);
  int wg = blockIdx.x - a.copies.n_wg;
  const int g = a.g0 + wg % a.ng;
  wg /= a.ng;
  // The dispatch order is a hint: an entry outside [0, B) is clamped, never followed.
  const int b = a.seq_order != nullptr ? min(max(table_lookup(a.seq_order, 0, 0, wg % a.B), 0), a.B - 1) : wg % a.B;
  const int c = wg / a.B;
  const int G = a.G;
  const int hq0 = g * G;

  Segments sg;
  sg.load(a, b, lane, n_parts);
  const int nblk = sg.total(n_parts);
  BANA_TIMELINE_MARK(1);
  int per = (nblk + a.nc - 1) / a.nc;
  if (per < a.cmin) per = a.cmin;
  const int nch = nblk > 0 ? (nblk + per - 1) / per : 0;

  // Destination of this workgroup's result.
  const int64_t row0 = ((int64_t)(a.nc == 1 ? 0 : c) * a.B + b) * a.out_hq + hq0 - a.out_h0;
  float* __restrict__ out_dst = a.out + row0 * kHeadDim;
  float* __restrict__ lse_dst = a.lse + row0;

  if (c >= nch) {  // empty range or chunk: out = 0, lse = -inf (chunk slots only need the lse)
    if (a.nc == 1) {
      for (int i = threadIdx.x; i < G * (kHeadDim / 4); i += 64 * W)
        reinterpret_cast<f32x4*>(out_dst)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int i = threadIdx.x; i < G; i += 64 * W) lse_dst[i] = -INFINITY;
    return;
  }
  const int jb0 = c * per;
  const int jb1 = min(nblk, jb0 + per);

  bf16x8 qop[4];
  load_q(qop, a.q, (int64_t)b * a.Hq + hq0, col, quad, G);
  Online st;
  st.init();
  walk_blocks<W>(st, qop, sg, n_parts, a, b, g, col, quad, jb0 + wave, jb1);

  if (W == 1) {
    st.emit(out_dst, lse_dst, col, quad, G);
    BANA_TIMELINE_MARK(3);
    return;
  }

  const float lsum = column_sum(st.lsum);
  float* sm_m = smem;               // [W][16]
  float* sm_l = smem + 16 * W;      // [W][16]
  float* sm_acc = smem + 32 * W;    // [W][G][kRowPad]
  race_check_delay(wave);
  if (quad == 0) {
    sm_m[wave * 16 + col] = st.m;   // -inf for a wave that saw no block
    sm_l[wave * 16 + col] = lsum;
  }
  if (col < G) {
#pragma unroll
    for (int dt = 0; dt < kDimTiles; ++dt)
      *reinterpret_cast<f32x4*>(sm_acc + (wave * G + col) * kRowPad + 16 * dt + 4 * quad) = st.acc[dt];
  }
  __syncthreads();
  race_check_barrier();
  for (int idx = threadIdx.x; idx < G * (kHeadDim / 4); idx += 64 * W) {
    const int h = idx >> 5;
    const int d4 = idx & 31;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, sm_m[w * 16 + h]);
    float L = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const float mw = sm_m[w * 16 + h];
      if (mw == -INFINITY) continue;
      const float e = fast_exp2((mw - M) * kLog2e);
      L += e * sm_l[w * 16 + h];
      o += e * *reinterpret_cast<const f32x4*>(sm_acc + (w * G + h) * kRowPad + 4 * d4);
    }
    *reinterpret_cast<f32x4*>(out_dst + h * kHeadDim + 4 * d4) = o * (1.0f / L);
    if (d4 == 0) lse_dst[h] = M + logf(L);
  }
  BANA_TIMELINE_MARK(3);
}

// Balanced launch: wavefront k of kv head g walks the blocks [k S, (k + 1) S)
// (clipped to U) of the call's virtual block list -- every sequence's blocks
// over all its ranges, in sequence order -- and leaves one partial per
// sequence piece in slot k + b of the piece buffers ([slot][out_hq][128] and
// [slot][out_hq]).  The schedule is computed by each workgroup in LDS: the
// block count N_b of every sequence, their inclusive prefix sums P_b by a
// workgroup-wide scan, U = P_{B-1} and S = ceil(U / K); the sequence holding
// block pos is the first b with P_b > pos (binary search).  The first
// workgroup also stores the prefix sums (prefix[0..B], exclusive) for the
// piece merge.
template <int W>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(4, 8))) void balanced_attn_kernel(
    PartialArgs a, int32_t* __restrict__ prefix, int K) {
  BANA_TIMELINE_MARK(0);
  constexpr int kThreads = 64 * W;
  constexpr int kPerThread = (kMaxBalancedBatch + kThreads - 1) / kThreads;
  __shared__ int32_t sm_incl[kMaxBalancedBatch];
  __shared__ int32_t sm_wave_sum[W];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15;
  const int quad = lane >> 4;
  const int B = a.B;

  // Thread t counts the blocks of sequences [t * per, t * per + per) (per <= kPerThread).
  const int per = (B + kThreads - 1) / kThreads;
  const int s0 = threadIdx.x * per;
  int cnt[kPerThread];
  int local = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    cnt[i] = 0;
    const int b = s0 + i;
    if (i < per && b < B) {
      for (int p = 0; p < a.n_parts; ++p) {
        const int t0 = a.begin[(int64_t)p * B + b];
        const int t1 = a.end[(int64_t)p * B + b];
        if (t1 > t0) cnt[i] += ((t1 - 1) >> 4) - (t0 >> 4) + 1;
      }
    }
    local += cnt[i];
  }
  // Workgroup-wide exclusive scan of the per-thread totals: within the wave by shuffles, then
  // across the W waves through LDS.
  int incl = local;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  race_check_delay(wave);
  if (lane == 63) sm_wave_sum[wave] = incl;
  __syncthreads();
  race_check_barrier();
  int before = incl - local;
  for (int w = 0; w < wave; ++w) before += sm_wave_sum[w];
  race_check_delay(wave);
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int b = s0 + i;
    before += cnt[i];
    if (i < per && b < B) sm_incl[b] = before;
  }
  __syncthreads();
  race_check_barrier();

  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i <= B; i += kThreads) prefix[i] = i == 0 ? 0 : sm_incl[i - 1];
  }
  BANA_TIMELINE_MARK(1);
  const int g = a.g0 + (int)(blockIdx.x % (unsigned)a.ng);
  const int k = (int)(blockIdx.x / (unsigned)a.ng) * W + wave;
  if (k >= K) return;
  const int G = a.G;
  const int hq0 = g * G;
  const int U = sm_incl[B - 1];
  const int64_t S = U > K ? ((int64_t)U + K - 1) / K : 1;
  const int u1 = (int)min((int64_t)U, (k + 1) * S);
  int pos = (int)min((int64_t)U, k * S);

  while (pos < u1) {
    // Sequence holding block pos: the first b with P_b > pos (wave-uniform binary search).
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sm_incl[mid] > pos) hi = mid;
      else lo = mid + 1;
    }
    const int b = __builtin_amdgcn_readfirstlane(lo);
    const int pb = b > 0 ? sm_incl[b - 1] : 0;
    Segments sg;
    sg.load(a, b, lane, a.n_parts);
    const int nb = sg.total(a.n_parts);
    const int v0 = pos - pb;
    const int v1 = min(u1 - pb, nb);

    bf16x8 qop[4];
    load_q(qop, a.q, (int64_t)b * a.Hq + hq0, col, quad, G);
    Online st;
    st.init();
    walk_blocks<1>(st, qop, sg, a.n_parts, a, b, g, col, quad, v0, v1);
    const int64_t row0 = (int64_t)(k + b) * a.out_hq + hq0 - a.out_h0;
    st.emit(a.out + row0 * kHeadDim, a.lse + row0, col, quad, G);
    pos = pb + v1;
  }
  BANA_TIMELINE_MARK(3);
}

}  // namespace

hipError_t launch_partial_attn(const PartialArgs& a, int waves, hipStream_t stream) {
  const unsigned nwg = (unsigned)a.copies.n_wg + (unsigned)a.nc * (unsigned)a.B * (unsigned)a.ng;
  const size_t smem = waves > 1 ? sizeof(float) * (size_t)(32 * waves + waves * a.G * kRowPad) : 0;
  const bool multi = a.n_parts > 1;
  switch (waves) {
    case 1:
      if (multi) hipLaunchKernelGGL((partial_attn_kernel<1, true>), dim3(nwg), dim3(64), smem, stream, a);
      else hipLaunchKernelGGL((partial_attn_kernel<1, false>), dim3(nwg), dim3(64), smem, stream, a);
      break;
    case 2:
      if (multi) hipLaunchKernelGGL((partial_attn_kernel<2, true>), dim3(nwg), dim3(128), smem, stream, a);
      else hipLaunchKernelGGL((partial_attn_kernel<2, false>), dim3(nwg), dim3(128), smem, stream, a);
      break;
    case 4:
      if (multi) hipLaunchKernelGGL((partial_attn_kernel<4, true>), dim3(nwg), dim3(256), smem, stream, a);
      else hipLaunchKernelGGL((partial_attn_kernel<4, false>), dim3(nwg), dim3(256), smem, stream, a);
      break;
    case 8:
      if (multi) hipLaunchKernelGGL((partial_attn_kernel<8, true>), dim3(nwg), dim3(512), smem, stream, a);
      else hipLaunchKernelGGL((partial_attn_kernel<8, false>), dim3(nwg), dim3(512), smem, stream, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t timeline_clear(hipStream_t stream) {
#ifdef BANA_WAVE_TIMELINE
  void* p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(g_wave_timeline));
  if (e == hipSuccess) e = hipMemsetAsync(p, 0xFF, sizeof(g_wave_timeline), stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  return e;
#else
  (void)stream;
  return hipErrorNotSupported;
#endif
}

hipError_t timeline_read(uint64_t* out, size_t n_slots, hipStream_t stream) {
#ifdef BANA_WAVE_TIMELINE
  void* p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(g_wave_timeline));
  if (e == hipSuccess) e = hipMemcpyAsync(out, p, n_slots * 4 * sizeof(uint64_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  return e;
#else
  (void)out;
  (void)n_slots;
  (void)stream;
  return hipErrorNotSupported;
#endif
}

hipError_t launch_balanced_attn(const PartialArgs& a, int32_t* prefix, int K, hipStream_t stream) {
  if (a.B < 1 || a.B > kMaxBalancedBatch || K < 1) return hipErrorInvalidValue;  // the LDS schedule's bounds
  const unsigned nwg = (unsigned)((K + kBalancedWaves - 1) / kBalancedWaves) * (unsigned)a.ng;
  hipLaunchKernelGGL(balanced_attn_kernel<kBalancedWaves>, dim3(nwg), dim3(64 * kBalancedWaves), 0, stream, a,
                     prefix, K);
  return hipGetLastError();
}

}  // namespace bana
