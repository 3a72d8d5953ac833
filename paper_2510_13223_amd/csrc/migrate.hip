// migrate.hip -- copy of the KV blocks of migrated ranges into another block pool (gfx950).
//
// The data movement behind attention-level migration (paper Sec. 4.1(2): the
// KV of the offloaded part moves to the cold device, T_attn ~ S_kv / B_net;
// Alg. 1's MigrateKVHeads step): for every sequence b and logical block j in
// [blk_begin[b], blk_end[b]), the block's K and V tiles of all kv heads are
// copied bit for bit from src block src_table[b][j] to dst block
// dst_table[b][j].  In both pools a block's tiles for all kv heads are one
// contiguous run (Hkv x 4 KiB for K, the same for V), so a block is two
// contiguous copies.  Two kernels: the flat one (up to 4096 sequences, below)
// splits the list of all migrated tiles evenly over one round of resident
// workgroups; beyond that, a grid row per sequence whose workgroups stride
// over the sequence's migrated blocks.  Non-temporal loads (the source is read
// once), plain stores (measured faster than non-temporal ones for this
// scatter).  HBM-bound: reads and writes Hkv x 8 KiB per block.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "kernels.h"
#include "paged_addr.h"

namespace bana {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

__global__ __launch_bounds__(kThreads) void migrate_kernel(const u32x4* __restrict__ src_k,
                                                           const u32x4* __restrict__ src_v,
                                                           const int32_t* __restrict__ src_table,
                                                           u32x4* __restrict__ dst_k, u32x4* __restrict__ dst_v,
                                                           const int32_t* __restrict__ dst_table,
                                                           const int32_t* __restrict__ blk_begin,
                                                           const int32_t* __restrict__ blk_end, int max_blocks,
                                                           int Hkv) {
  const int b = blockIdx.y;
  const int jend = blk_end[b];
  const int64_t n16 = (int64_t)Hkv * kTileElems / 8;  // 16-byte units per block and pool
  // Workgroup x of the row takes blocks begin + x, begin + x + gridDim.x, ...
  for (int j = blk_begin[b] + (int)blockIdx.x; j < jend; j += (int)gridDim.x) {
    const int64_t sblk = table_lookup(src_table, max_blocks, b, j);
    const int64_t dblk = table_lookup(dst_table, max_blocks, b, j);
    const u32x4* sk = src_k + sblk * n16;
    const u32x4* sv = src_v + sblk * n16;
    u32x4* dk = dst_k + dblk * n16;
    u32x4* dv = dst_v + dblk * n16;
    for (int64_t i0 = threadIdx.x; i0 < n16; i0 += (int64_t)kThreads * kUnroll) {
      u32x4 kx[kUnroll], vx[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = i0 + (int64_t)u * kThreads;
        if (i < n16) {
          kx[u] = __builtin_nontemporal_load(sk + i);
          vx[u] = __builtin_nontemporal_load(sv + i);
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = i0 + (int64_t)u * kThreads;
        if (i < n16) {  // plain stores: measured ~4 % faster than non-temporal ones for this scatter
          dk[i] = kx[u];
          dv[i] = vx[u];
        }
      }
    }
  }
}

// Flat form (batch <= kMaxFlatMigrateBatch): the migrated blocks of all sequences, in sequence
// order, form one list of N blocks, each 2 * Hkv tiles of 4 KiB (the K tiles of its kv heads, then
// the V tiles).  The grid is one round of resident workgroups; workgroup w copies the tiles
// [w T, (w + 1) T) of the list (T = ceil(tiles / grid)), 4 tiles per step: thread t moves bytes
// [16 t, 16 t + 16) of each of the 4 tiles, so every load and store instruction of a wavefront
// covers 1 KiB of one tile, and 4 loads are in flight per thread.  A workgroup finds the sequence
// holding its first block by a prefix scan of the block counts in LDS and then walks the list in
// order, so every workgroup moves the same number of bytes whatever the per-sequence counts.
// Measured on MI355X (llama3_8b's migrated partition, 323 MB, cold caches): 2 or 4 tiles per
// step 105-106 us (6.1 TB/s of HBM traffic, above a linear device copy of the same bytes at
// 114 us), 8 tiles 133 us, 16 tiles 138 us; 1024 workgroups 127 us, 4096 or 8192 107-109 us.
constexpr int kFlatTilesPerStep = 4;

__global__ __launch_bounds__(kThreads) void migrate_flat_kernel(const u32x4* __restrict__ src_k,
                                                                const u32x4* __restrict__ src_v,
                                                                const int32_t* __restrict__ src_table,
                                                                u32x4* __restrict__ dst_k, u32x4* __restrict__ dst_v,
                                                                const int32_t* __restrict__ dst_table,
                                                                const int32_t* __restrict__ blk_begin,
                                                                const int32_t* __restrict__ blk_end, int B,
                                                                int max_blocks, int Hkv) {
  constexpr int kPerThread = (kMaxFlatMigrateBatch + kThreads - 1) / kThreads;
  __shared__ int32_t sm_incl[kMaxFlatMigrateBatch];  // inclusive prefix sums of the block counts
  __shared__ int32_t sm_wave_sum[kThreads / 64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int per = (B + kThreads - 1) / kThreads;
  const int s0 = threadIdx.x * per;
  int cnt[kPerThread];
  int local = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    cnt[i] = 0;
    const int b = s0 + i;
    if (i < per && b < B) cnt[i] = max(0, blk_end[b] - blk_begin[b]);
    local += cnt[i];
  }
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

  const int tpb = 2 * Hkv;                                   // tiles per block
  const int64_t n_tiles = (int64_t)sm_incl[B - 1] * tpb;
  const int64_t T = (n_tiles + gridDim.x - 1) / gridDim.x;  // tiles per workgroup
  int64_t tile = (int64_t)blockIdx.x * T;
  const int64_t tile_end = min(n_tiles, tile + T);
  if (tile >= tile_end) return;
  // Sequence b and logical block j of the workgroup's first tile: the first b with P_b > n.
  const int n0 = (int)(tile / tpb);
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (sm_incl[mid] > n0) hi = mid;
    else lo = mid + 1;
  }
  int b = lo;
  int j = blk_begin[b] + (n0 - (b > 0 ? sm_incl[b - 1] : 0));
  int r = (int)(tile - (int64_t)n0 * tpb);  // tile within the block
  constexpr int kTile16 = kTileElems / 8;  // 16-byte units per 4 KiB tile
  int64_t sblk = table_lookup(src_table, max_blocks, b, j);
  int64_t dblk = table_lookup(dst_table, max_blocks, b, j);
  // Tile offsets (in 16-byte units) are the same for the whole workgroup; each thread adds its own
  // 16-byte slot only at the load and the store.  V tiles are addressed from the K pool's base
  // plus the distance between the two pools (both pools of a side hold the same number of tiles).
  const int64_t sv = (int64_t)(reinterpret_cast<uintptr_t>(src_v) - reinterpret_cast<uintptr_t>(src_k)) / 16;
  const int64_t dv = (int64_t)(reinterpret_cast<uintptr_t>(dst_v) - reinterpret_cast<uintptr_t>(dst_k)) / 16;
  const uintptr_t sbase = reinterpret_cast<uintptr_t>(src_k);
  const uintptr_t dbase = reinterpret_cast<uintptr_t>(dst_k);
  while (tile < tile_end) {
    int64_t soff[kFlatTilesPerStep], doff[kFlatTilesPerStep];
    const int nt = (int)min((int64_t)kFlatTilesPerStep, tile_end - tile);
#pragma unroll
    for (int u = 0; u < kFlatTilesPerStep; ++u) {
      soff[u] = 0;
      doff[u] = 0;
      if (u < nt) {
        const bool is_k = r < Hkv;
        const int g = is_k ? r : r - Hkv;
        soff[u] = (sblk * Hkv + g) * kTile16 + (is_k ? 0 : sv);
        doff[u] = (dblk * Hkv + g) * kTile16 + (is_k ? 0 : dv);
        if (++r == tpb && (u + 1 < nt || tile + nt < tile_end)) {  // next block of the list
          r = 0;
          ++j;
          while (j >= blk_end[b]) {
            ++b;
            j = blk_begin[b];
          }
          sblk = table_lookup(src_table, max_blocks, b, j);
          dblk = table_lookup(dst_table, max_blocks, b, j);
        }
      }
    }
    u32x4 x[kFlatTilesPerStep];
#pragma unroll
    for (int u = 0; u < kFlatTilesPerStep; ++u)
      if (u < nt)
        x[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(sbase + 16 * (soff[u] + threadIdx.x)));
#pragma unroll
    for (int u = 0; u < kFlatTilesPerStep; ++u)
      if (u < nt) *reinterpret_cast<u32x4*>(dbase + 16 * (doff[u] + threadIdx.x)) = x[u];
    tile += nt;
  }
}

// Stream-ordered copy of n16 16-byte units by a grid-stride loop; either side may be device memory
// or pinned host memory (reached over the host link).
__global__ __launch_bounds__(kThreads) void copy_kernel(u32x4* __restrict__ dst, const u32x4* __restrict__ src,
                                                        int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i0 = (int64_t)blockIdx.x * kThreads + threadIdx.x; i0 < n16; i0 += stride * kUnroll) {
    u32x4 x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (i0 + u * stride < n16) x[u] = __builtin_nontemporal_load(src + i0 + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (i0 + u * stride < n16) __builtin_nontemporal_store(x[u], dst + i0 + u * stride);
  }
}

}  // namespace

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 == 0) return hipSuccess;
  // A few workgroups only: enough to fill the host link, few enough to leave the CUs to the
  // attention kernel that runs beside the copy.
  const int64_t per_wg = (int64_t)kThreads * kUnroll;
  const unsigned grid = (unsigned)std::min<int64_t>(64, (n16 + per_wg - 1) / per_wg);
  hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kThreads), 0, stream, static_cast<u32x4*>(dst),
                     static_cast<const u32x4*>(src), n16);
  return hipGetLastError();
}

hipError_t launch_migrate(const void* src_k, const void* src_v, const int32_t* src_table, void* dst_k, void* dst_v,
                          const int32_t* dst_table, const int32_t* blk_begin, const int32_t* blk_end, int B,
                          int max_blocks, int max_migrated_blocks, int Hkv, hipStream_t stream) {
  if (max_migrated_blocks <= 0) return hipSuccess;
  if (B <= kMaxFlatMigrateBatch) {
    // One round of resident workgroups (256 CUs x 8 workgroups of 256 threads), fewer when the
    // hint bounds the tiles to move below 8 tiles per workgroup.
    const int64_t tiles_bound = (int64_t)B * max_migrated_blocks * 2 * Hkv;
    const unsigned grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>(2048, tiles_bound / kFlatTilesPerStep));
    hipLaunchKernelGGL(migrate_flat_kernel, dim3(grid), dim3(kThreads), 0, stream, static_cast<const u32x4*>(src_k),
                       static_cast<const u32x4*>(src_v), src_table, static_cast<u32x4*>(dst_k),
                       static_cast<u32x4*>(dst_v), dst_table, blk_begin, blk_end, B, max_blocks, Hkv);
    return hipGetLastError();
  }
  // The row width only sets parallelism (workgroups stride over the blocks); keep the row's
  // work-items well inside 32 bits.
  const unsigned row = (unsigned)std::min(max_migrated_blocks, 1 << 16);
  hipLaunchKernelGGL(migrate_kernel, dim3(row, (unsigned)B), dim3(kThreads), 0, stream,
                     static_cast<const u32x4*>(src_k), static_cast<const u32x4*>(src_v), src_table,
                     static_cast<u32x4*>(dst_k), static_cast<u32x4*>(dst_v), dst_table, blk_begin, blk_end,
                     max_blocks, Hkv);
  return hipGetLastError();
}

}  // namespace bana
