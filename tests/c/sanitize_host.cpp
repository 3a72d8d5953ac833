// sanitize_host.cpp -- the library's host code (argument checks, launch planning, workspace
// layout) built for the CPU with AddressSanitizer and UndefinedBehaviorSanitizer, driven by a
// seeded sweep of ordinary and extreme dims through every entry point.
//
// The kernel launchers are replaced by stubs that launch nothing: each checks that the launch
// the host code planned stays inside the buffers of the call (fake device addresses that are
// never dereferenced) and inside the 32-bit launch limits, then returns success.  A failed
// check, a sanitizer report or a status outside the enum ends the program with a non-zero code.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <random>
#include <vector>

#include "bana.h"
#include "kernels.h"

namespace {

long g_case = 0;
long g_launches = 0;

struct Region {
  uintptr_t lo, hi;
};
std::vector<Region> g_regions;  // buffers of the current call

void add_region(const void* p, size_t bytes) {
  if (p != nullptr) g_regions.push_back({reinterpret_cast<uintptr_t>(p), reinterpret_cast<uintptr_t>(p) + bytes});
}

#define REQUIRE(c)                                                                       \
  do {                                                                                   \
    if (!(c)) {                                                                          \
      fprintf(stderr, "check failed: %s (line %d, case %ld)\n", #c, __LINE__, g_case); \
      abort();                                                                           \
    }                                                                                    \
  } while (0)

bool inside(const void* p, unsigned __int128 bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  for (const Region& r : g_regions)
    if (a >= r.lo && (unsigned __int128)a + bytes <= r.hi) return true;
  return false;
}

constexpr unsigned __int128 kRow = 128 * sizeof(float);
constexpr uint64_t kMaxItems = UINT32_MAX;

}  // namespace

extern "C" const char* hipGetErrorString(hipError_t) { return "stub"; }

namespace bana {

hipError_t launch_partial_attn(const PartialArgs& a, int waves, hipStream_t) {
  ++g_launches;
  REQUIRE(waves == 1 || waves == 2 || waves == 4 || waves == 8);
  REQUIRE(a.nc >= 1 && a.nc <= 256 && a.cmin >= 1);
  REQUIRE(a.G >= 1 && a.G <= 16 && (int64_t)a.G * a.Hkv == a.Hq);
  REQUIRE(a.g0 >= 0 && a.ng >= 1 && a.g0 + a.ng <= a.Hkv);
  REQUIRE(a.n_parts >= 1 && a.n_parts <= 64);
  REQUIRE((uint64_t)a.nc * a.B * a.ng * 64 * waves <= kMaxItems);
  REQUIRE(sizeof(float) * (size_t)(32 * waves + waves * a.G * 132) <= 65536 || waves == 1);
  const unsigned __int128 rows = (unsigned __int128)(a.nc == 1 ? 1 : a.nc) * a.B * a.out_hq;
  REQUIRE(a.out_h0 >= 0 && a.out_h0 + a.ng * a.G <= a.out_hq + a.out_h0);
  REQUIRE(inside(a.out, rows * kRow) && inside(a.lse, rows * sizeof(float)));
  REQUIRE(inside(a.q, (unsigned __int128)a.B * a.Hq * 128 * 2));
  REQUIRE(inside(a.table, (unsigned __int128)a.B * a.max_blocks * 4));
  REQUIRE(inside(a.begin, (unsigned __int128)a.n_parts * a.B * 4) && inside(a.end, (unsigned __int128)a.n_parts * a.B * 4));
  REQUIRE(a.copies.n >= 0 && a.copies.n <= kMaxSideCopies && a.copies.n_wg >= 0 && a.copies.n_wg <= 64);
  REQUIRE((a.copies.n == 0) == (a.copies.n_wg == 0));
  REQUIRE(((uint64_t)a.nc * a.B * a.ng + a.copies.n_wg) * 64 * waves <= kMaxItems);
  for (int i = 0; i < a.copies.n; ++i)
    REQUIRE(a.copies.n16[i] > 0 && inside(a.copies.src[i], (unsigned __int128)a.copies.n16[i] * 16) &&
            inside(a.copies.dst[i], (unsigned __int128)a.copies.n16[i] * 16));
  return hipSuccess;
}

hipError_t launch_balanced_attn(const PartialArgs& a, int32_t* prefix, int K, hipStream_t) {
  ++g_launches;
  REQUIRE(a.B >= 1 && a.B <= kMaxBalancedBatch && K >= kBalancedWaves && K % kBalancedWaves == 0);
  REQUIRE((uint64_t)(K / kBalancedWaves) * a.ng * 64 * kBalancedWaves <= kMaxItems);
  const unsigned __int128 slots = (unsigned __int128)(K + a.B) * a.out_hq;
  REQUIRE(inside(a.out, slots * kRow) && inside(a.lse, slots * sizeof(float)));
  REQUIRE(inside(prefix, (unsigned __int128)(a.B + 1) * 4));
  REQUIRE(a.g0 + a.ng <= a.Hkv && (int64_t)a.ng * a.G == a.out_hq);
  return hipSuccess;
}

hipError_t launch_merge_pieces(const float* outs, const float* lses, const int32_t* prefix, int K, int kp,
                               MergeRows m, float* out, float* lse_out, hipStream_t) {
  ++g_launches;
  REQUIRE(kp == 1 || kp == 2 || kp == 4 || kp == 8);
  const unsigned __int128 slots = (unsigned __int128)(K + m.B) * m.in_hq;
  REQUIRE(inside(outs, slots * kRow) && inside(lses, slots * sizeof(float)) && inside(prefix, (m.B + 1) * 4));
  REQUIRE(m.out_h0 + m.hn <= m.out_hq && m.in_h0 + m.hn <= m.in_hq);
  REQUIRE(inside(out, (unsigned __int128)m.B * m.out_hq * kRow));
  REQUIRE(lse_out == nullptr || inside(lse_out, (unsigned __int128)m.B * m.out_hq * sizeof(float)));
  REQUIRE((uint64_t)m.B * m.hn * 32 * kp <= kMaxItems + 255);
  return hipSuccess;
}

hipError_t launch_merge(const float* outs, const float* lses, int n_parts, MergeRows m, float* out, float* lse_out,
                        hipStream_t) {
  ++g_launches;
  REQUIRE(n_parts >= 1);
  const unsigned __int128 parts = (unsigned __int128)n_parts * m.B * m.in_hq;
  REQUIRE(inside(outs, parts * kRow) && inside(lses, parts * sizeof(float)));
  REQUIRE(m.out_h0 + m.hn <= m.out_hq && m.in_h0 + m.hn <= m.in_hq);
  REQUIRE(inside(out, (unsigned __int128)m.B * m.out_hq * kRow));
  REQUIRE(lse_out == nullptr || inside(lse_out, (unsigned __int128)m.B * m.out_hq * sizeof(float)));
  REQUIRE((uint64_t)m.B * m.hn * 32 * 8 <= kMaxItems + 255 || (uint64_t)m.B * m.hn * 32 <= kMaxItems);
  return hipSuccess;
}

hipError_t launch_migrate(const void* src_k, const void* src_v, const int32_t* src_table, void* dst_k, void* dst_v,
                          const int32_t* dst_table, const int32_t* blk_begin, const int32_t* blk_end, int B,
                          int max_blocks, int max_migrated_blocks, int Hkv, hipStream_t) {
  ++g_launches;
  REQUIRE(B >= 1 && B <= 65535 && Hkv >= 1 && max_migrated_blocks <= max_blocks);
  REQUIRE(inside(src_table, (unsigned __int128)B * max_blocks * 4) && inside(dst_table, (unsigned __int128)B * max_blocks * 4));
  REQUIRE(inside(blk_begin, B * 4) && inside(blk_end, B * 4));
  REQUIRE(inside(src_k, 1) && inside(src_v, 1) && inside(dst_k, 1) && inside(dst_v, 1));
  return hipSuccess;
}

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t) {
  ++g_launches;
  REQUIRE(bytes % 16 == 0 && inside(dst, bytes) && inside(src, bytes));
  return hipSuccess;
}

hipError_t launch_validate(const int32_t* table, const int32_t* seq_lens, const int32_t* begin, const int32_t* end,
                           int n_parts, int B, int max_blocks, int64_t, int32_t* result, hipStream_t) {
  ++g_launches;
  REQUIRE(n_parts >= 1 && n_parts <= 65535 && inside(result, 4));
  REQUIRE(inside(table, (unsigned __int128)B * max_blocks * 4) && inside(seq_lens, B * 4));
  REQUIRE(inside(begin, (unsigned __int128)n_parts * B * 4) && inside(end, (unsigned __int128)n_parts * B * 4));
  return hipSuccess;
}

hipError_t launch_gather_read(const void* k, const void* v, const int32_t* table, const int32_t* begin,
                              const int32_t* end, int n_parts, int B, int Hkv, int max_blocks, uint32_t* sink,
                              hipStream_t) {
  ++g_launches;
  REQUIRE(inside(sink, (unsigned __int128)B * Hkv * 4) && inside(table, (unsigned __int128)B * max_blocks * 4));
  REQUIRE(inside(begin, (unsigned __int128)n_parts * B * 4) && inside(end, (unsigned __int128)n_parts * B * 4));
  REQUIRE(inside(k, 1) && inside(v, 1));
  return hipSuccess;
}

hipError_t launch_stream_read(const void* src, size_t bytes, int n_groups, uint32_t* sink, hipStream_t) {
  ++g_launches;
  REQUIRE(n_groups >= 1 && n_groups <= 65536 && inside(src, bytes) && inside(sink, (size_t)n_groups * 4));
  return hipSuccess;
}

hipError_t launch_debug_rows(const int32_t* table, const int32_t* begin, const int32_t* end, int B, int Hkv,
                             int max_blocks, int64_t* rows, hipStream_t) {
  ++g_launches;
  REQUIRE(inside(rows, (unsigned __int128)B * Hkv * max_blocks * 16 * 8));
  REQUIRE(inside(table, (unsigned __int128)B * max_blocks * 4) && inside(begin, B * 4) && inside(end, B * 4));
  return hipSuccess;
}

// The product build's timeline hooks: nothing recorded.
hipError_t timeline_clear(hipStream_t) { return hipErrorNotSupported; }
hipError_t timeline_read(uint64_t*, size_t, hipStream_t) { return hipErrorNotSupported; }

hipError_t static_scratch(void** ptr) {
  *ptr = reinterpret_cast<void*>(uintptr_t{40} << 44);  // apart from every fake buffer below
  add_region(*ptr, kStaticScratchBytes);
  return hipSuccess;
}

}  // namespace bana

namespace {

std::mt19937_64 g_rng(20251213);

template <typename T>
T pick(std::initializer_list<T> xs) {
  std::uniform_int_distribution<size_t> d(0, xs.size() - 1);
  return *(xs.begin() + d(g_rng));
}

int64_t rnd(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(g_rng); }

// Fake, 256-byte aligned device addresses, far apart; never dereferenced.
void* fake(int i) { return reinterpret_cast<void*>((uintptr_t)(i + 1) << 44); }

bool valid_status(bana_status s) {
  return s == BANA_OK || s == BANA_ERR_INVALID || s == BANA_ERR_UNSUPPORTED || s == BANA_ERR_DEVICE;
}

}  // namespace

#ifndef BANA_HOSTCHECK_LIBRARY  // built as a shared library, only the stub launchers are needed
int main(int argc, char** argv) {
  const long n_cases = argc > 1 ? atol(argv[1]) : 20000;
  long ok_calls = 0;
  for (g_case = 0; g_case < n_cases; ++g_case) {
    bana_dims d{};
    d.batch = (int32_t)pick<int64_t>({1, 2, 3, 7, 64, 65, 100, 256, 2048, 2049, 4096, 4097, 65535, 65536,
                                      1 << 20, (1 << 26) - 1, 0, -1});
    const int32_t hkv = (int32_t)pick<int64_t>({1, 2, 8, 40, 64, 128, 0});
    const int32_t g = (int32_t)pick<int64_t>({1, 2, 3, 4, 8, 16, 17});
    d.num_kv_heads = hkv;
    d.num_q_heads = pick<int>({0, 1}) ? hkv * g : hkv * g + 1;
    d.head_dim = pick<int32_t>({128, 128, 128, 64});
    d.block_size = pick<int32_t>({16, 16, 16, 32});
    d.max_blocks_per_seq = (int32_t)pick<int64_t>({1, 16, 256, 8192, 1 << 20, 1 << 23, INT32_MAX / 16,
                                                   INT32_MAX / 16 + 1, INT32_MAX, 0});
    d.num_blocks = pick<int64_t>({1, 1000, int64_t{1} << 31, int64_t{1} << 40, 0});
    d.max_range_tokens = (int32_t)pick<int64_t>({0, 1, 16, 4096, 131072, INT32_MAX, -5});
    d.waves_hint = pick<int32_t>({0, 0, 0, 1, 2, 3, 4, 8});
    d.chunks_hint = pick<int32_t>({0, 0, 0, 1, 2, 7, 256, 1000, -1});
    d.plan_hint = pick<int32_t>({0, 0, 1, 2, 2, 3});
    d.total_range_tokens = pick<int64_t>({0, 1, (int64_t)d.batch * 1000, (int64_t)d.batch * 131072,
                                          int64_t{1} << 50, INT64_MAX, -1});
    d.nonempty_ranges = (int32_t)pick<int64_t>({0, 1, 61, d.batch, (int64_t)d.batch * 2, -1});
    d.seq_order = pick<int>({0, 1}) ? static_cast<const int32_t*>(fake(20)) : nullptr;

    const size_t ws = bana_decode_attn_workspace_bytes(&d);
    const bool have_ws = ws > 0 && pick<int>({0, 1, 1});
    void* wsp = have_ws ? fake(30) : nullptr;
    const size_t ws_bytes = have_ws ? ws : 0;
    const int n_parts = (int)pick<int64_t>({1, 2, 4, 16, 64, 65, 0});

    // Buffers of a call, sized from the dims as the header states them.
    g_regions.clear();
    const int64_t B = d.batch > 0 ? d.batch : 1, Hq = d.num_q_heads > 0 ? d.num_q_heads : 1;
    const int64_t mb = d.max_blocks_per_seq > 0 ? d.max_blocks_per_seq : 1;
    add_region(fake(0), (size_t)B * Hq * 128 * 2);        // q
    add_region(fake(1), 1);                               // k_cache
    add_region(fake(2), 1);                               // v_cache
    add_region(fake(3), (size_t)B * mb * 4);              // block_table
    add_region(fake(4), (size_t)B * 4);                   // seq_lens
    add_region(fake(5), (size_t)B * 4 * 65);              // begin [n_parts][B]
    add_region(fake(6), (size_t)B * 4 * 65);              // end
    add_region(fake(7), (size_t)B * Hq * 128 * 4 * 65);   // out / out_partials
    add_region(fake(8), (size_t)B * Hq * 4 * 65);         // lse / lses
    add_region(fake(9), (size_t)B * Hq * 128 * 4);        // merged out
    add_region(fake(10), (size_t)B * Hq * 4);             // merged lse
    add_region(fake(20), (size_t)B * 4);                  // seq_order
    add_region(fake(21), (size_t)B * mb * 4);             // dst table
    add_region(fake(22), 1);                              // dst pools
    add_region(fake(23), 1);
    add_region(fake(24), (size_t)B * (d.num_kv_heads > 0 ? d.num_kv_heads : 1) * mb * 16 * 8);  // rows / sink
    add_region(fake(25), 4);                              // validation result
    if (wsp) add_region(wsp, ws);

    const int32_t* i32 = nullptr;
    auto I = [&](int i) { return static_cast<const int32_t*>(fake(i)); };
    auto F = [&](int i) { return static_cast<float*>(fake(i)); };
    bana_status st[10];
    st[0] = bana_decode_attn_partial(&d, fake(0), fake(1), fake(2), I(3), I(4), I(5), I(6), F(7), F(8), wsp,
                                     ws_bytes, nullptr);
    st[1] = bana_decode_attn_fused(&d, fake(0), fake(1), fake(2), I(3), I(4), I(5), I(6), n_parts, F(9), F(10), wsp,
                                   ws_bytes, nullptr);
    const int32_t h0 = (int32_t)rnd(-1, d.num_kv_heads > 0 ? d.num_kv_heads : 1);
    const int32_t h1 = (int32_t)rnd(h0, (d.num_kv_heads > 0 ? d.num_kv_heads : 1) + 1);
    st[2] = bana_decode_attn_heads(&d, fake(0), fake(1), fake(2), I(3), I(4), I(5), I(6), h0, h1, F(9), F(10), wsp,
                                   ws_bytes, nullptr);
    st[3] = bana_decode_attn_partial_noalloc(&d, fake(0), fake(1), fake(2), I(3), I(4), I(5), I(6), F(7), F(8),
                                             nullptr);
    st[4] = bana_merge_partials(&d, F(7), F(8), n_parts, F(9), pick<int>({0, 1}) ? F(10) : nullptr, nullptr);
    st[5] = bana_migrate_kv_blocks(&d, fake(1), fake(2), I(3), fake(22), fake(23), I(21), d.num_blocks, I(5), I(6),
                                   nullptr);
    st[6] = bana_validate_ranges(&d, I(3), I(4), I(5), I(6), n_parts, static_cast<int32_t*>(fake(25)), nullptr);
    st[7] = bana_debug_kv_rows(&d, I(3), I(5), I(6), static_cast<int64_t*>(fake(24)), nullptr);
    st[8] = bana_debug_gather_read(&d, fake(1), fake(2), I(3), I(5), I(6), n_parts,
                                   static_cast<uint32_t*>(fake(24)), nullptr);
    // the fused call with side copies (fake host / device buffers of the given sizes)
    bana_copy copies[9];
    const int n_copies = (int)rnd(0, 9);
    for (int i = 0; i < n_copies; ++i) {
      copies[i].bytes = (size_t)rnd(0, 1 << 20) * 16;
      copies[i].dst = fake(11 + 2 * (i % 4));
      copies[i].src = fake(12 + 2 * (i % 4));
      add_region(copies[i].dst, copies[i].bytes);
      add_region(copies[i].src, copies[i].bytes);
    }
    st[9] = bana_decode_attn_fused_copies(&d, fake(0), fake(1), fake(2), I(3), I(4), I(5), I(6), n_parts, F(9),
                                          F(10), wsp, ws_bytes, copies, n_copies, nullptr);
    (void)i32;
    for (bana_status s : st) {
      REQUIRE(valid_status(s));
      ok_calls += s == BANA_OK;
    }
    REQUIRE(bana_status_string(st[0]) != nullptr);
  }
  printf("sanitized host sweep: %ld cases, %ld calls accepted, %ld launches checked\n", n_cases, ok_calls,
         g_launches);
  return 0;
}
#endif
