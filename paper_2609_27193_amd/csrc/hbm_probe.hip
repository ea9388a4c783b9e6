// Practical HBM ceilings of the access patterns the library's kernels use,
// measured with no arithmetic in the way:
//   read1   one array read                    (a bound for any read stream)
//   read2   two arrays read                   (the SNAPSHOT score: W and S)
//   copy    one array read, another written   (pack and restore)
//   r2w1    two arrays read, the second written (the ACCUM score: W, S read, S <- W)
// Each block moves one tile per stream: `threads` lanes, `vec` 16-byte
// vectors per lane, all loads issued before any use, accessed through a
// buffer resource per tile with the non-temporal, device-scope cache policy,
// and the XCD-contiguous block mapping of the kernels.  The sweep covers
// vec in {2, 4, 8} and threads in {256, 512}, and for the kernels' tile
// (2 x 256) the number of blocks a CU may hold at once (an LDS reservation
// the kernel never touches: 2, 3, 4, 6, or as many as fit); the arrays can
// be placed so the streams sit at chosen offsets of the memory interleave:
//   skew    the second array starts `skew` bytes further into its allocation
//   offset  both arrays start `offset` bytes past an allocation boundary, so
//           tiles straddle the boundaries a caller's layout can put them across
// Prints one JSON line per (pattern, vec, threads) with the best of two
// rounds of `reps` launches.
//
//   lc_hbm_probe [GiB per array, default 16] [skew bytes, default 20480] [offset bytes, default 0]
//   lc_hbm_probe empty     (dispatch cost of blocks that find no work)
//   lc_hbm_probe pairs     (8 separately allocated pairs of 8 GiB arrays: two
//                           reads + one write and copy per pair, r2w1 with
//                           each first array against the next pair's second,
//                           and r2w1 with the second array entered 64 MiB and
//                           512 MiB later; three rounds: how much the rate
//                           depends on the physical pages an allocation
//                           receives, and whether offsets move it)
//   lc_hbm_probe tail      (two 16 GiB arrays, read2 and r2w1 with the kernels'
//                           tile at 2, 3, 4, 6 blocks per CU or as many as fit:
//                           bare; with the score kernel's two dependent table
//                           lookups per block; with those lookups and its
//                           end-of-block reduction to one fp64 pair; with the
//                           lookups and one fp64 pair per wave instead (no LDS,
//                           no barrier): what a block's own latency costs)
//   lc_hbm_probe persist   (two 16 GiB arrays, read2, r2w1 and copy: one tile
//                           per block against k resident blocks per CU that
//                           each walk tiles of their XCD's eighth, loading the
//                           next tile before consuming the current one, in
//                           grid-stride order or in contiguous runs)
//
// Built a second time as a shared library (without LC_PROBE_MAIN), it
// exports lc_probe_arrays: the kernels' own tile over arrays the caller
// already holds, at a chosen number of blocks per CU, so a kernel's rate can
// be set against the ceiling of the same placement.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "lc_device.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kPolicy = 2 | 16;  // nt | sc1

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile(const char* base, size_t t, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base) + t * bytes, 0, static_cast<int>(bytes),
                                           0x00020000);
}
template <int NT>
__device__ __forceinline__ u32x4 ld(__amdgpu_buffer_rsrc_t r, int k) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (threadIdx.x + k * NT) * 16, 0, kPolicy);
}
template <int NT>
__device__ __forceinline__ void st(__amdgpu_buffer_rsrc_t r, int k, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (threadIdx.x + k * NT) * 16, 0, kPolicy);
}

#define CK(x)                                                                  \
  do {                                                                         \
    hipError_t e_ = (x);                                                       \
    if (e_ != hipSuccess) {                                                    \
      std::fprintf(stderr, "lc_hbm_probe: %s: %s\n", #x, hipGetErrorString(e_)); \
      std::exit(1);                                                            \
    }                                                                          \
  } while (0)

// Block x of G walks one contiguous eighth of the tiles per XCD (a bijection
// on the first 8*floor(G/8) tiles, identity on the rest).
__device__ __forceinline__ size_t tile_of(unsigned x, unsigned G) {
  const unsigned full = G - G % 8u;
  return x < full ? static_cast<size_t>(x % 8u) * (full / 8u) + x / 8u : x;
}

// Dynamic LDS per block that leaves room for at most k blocks on a CU (0 for
// k = 0, or when the device's limits leave no such size): more than
// L / (k + 1) of the CU's L bytes, and at most L / k.
unsigned lds_for(int k) {
  if (k <= 0) return 0;
  int dev = 0, cu = 0, blk = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) != hipSuccess ||
      hipDeviceGetAttribute(&blk, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || cu <= 0)
    return 0;
  const long want = (cu / (k + 1) + 2048 + 511) / 512 * 512;
  return (want > cu / k - 1024 || want > blk) ? 0 : static_cast<unsigned>(want);
}

// PAT: 0 read1, 1 read2, 2 copy, 3 r2w1.  The xor into `sink` under a
// condition that never holds keeps the loads of the read patterns.
template <int PAT, int VEC, int NT>
__global__ __launch_bounds__(NT) void probe(const char* a, char* b, unsigned* sink) {
  constexpr unsigned kTile = NT * VEC * 16;
  const size_t t = tile_of(blockIdx.x, gridDim.x);
  const auto ra = tile(a, t, kTile), rb = tile(b, t, kTile);
  u32x4 v[VEC], w[VEC];
#pragma unroll
  for (int k = 0; k < VEC; ++k) {
    v[k] = ld<NT>(ra, k);
    if constexpr (PAT == 1 || PAT == 3) w[k] = ld<NT>(rb, k);
  }
  unsigned acc = 0;
#pragma unroll
  for (int k = 0; k < VEC; ++k) {
    if constexpr (PAT == 2 || PAT == 3) st<NT>(rb, k, v[k]);
    acc ^= v[k].x ^ v[k].w;
    if constexpr (PAT == 1 || PAT == 3) acc += w[k].y;
  }
  if (acc == 0x9e3779b9u) sink[threadIdx.x] = acc;
}

// Every block reads the amount of work from device memory and finds none:
// the cost of dispatching blocks that exit at once (a grid sized for the
// worst case whose work is decided on the device).
__global__ __launch_bounds__(256) void empty_blocks(const unsigned* n_work, unsigned* sink) {
  if (blockIdx.x < *n_work) sink[threadIdx.x] = blockIdx.x;
}

// ---- tail: the cost of a block's own latency at few blocks per CU ------------
// Tiles are grouped into segments of kTailSegTiles; LOOKUP 1 finds a tile's
// addresses through tile -> segment -> (a, b, first tile), two dependent
// loads like the score kernel's chunk -> segment tables.  REDUCE 1 forms the
// score kernel's terms (|w - s| and |s| of bf16 pairs, fp32 per vector, fp64
// per lane) and reduces them to one fp64 pair per block (wave sums, LDS
// combine, thread 0 stores); REDUCE 2 stores one pair per wave instead.
constexpr unsigned kTailSegTiles = 4096;
struct TailSeg {
  uint64_t a, b, first;
};
struct TailArgs {
  const char* a;
  char* b;
  const uint32_t* tile_seg;
  const TailSeg* segs;
  double2* partials;  // [tiles * 4]
  unsigned* sink;
};

template <int PAT, int LOOKUP, int REDUCE>
__global__ __launch_bounds__(256) void tail_probe(const TailArgs g) {
  constexpr unsigned kTile = 256 * 2 * 16;
  const size_t t = tile_of(blockIdx.x, gridDim.x);
  const char* pa;
  char* pb;
  if constexpr (LOOKUP == 0) {
    pa = g.a + t * kTile;
    pb = g.b + t * kTile;
  } else {
    const TailSeg sg = g.segs[g.tile_seg[t]];
    pa = reinterpret_cast<const char*>(sg.a) + (t - sg.first) * kTile;
    pb = reinterpret_cast<char*>(sg.b) + (t - sg.first) * kTile;
  }
  const auto ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(pa), 0, static_cast<int>(kTile), 0x00020000);
  const auto rb = __builtin_amdgcn_make_buffer_rsrc(pb, 0, static_cast<int>(kTile), 0x00020000);
  u32x4 v[2], w[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    v[k] = ld<256>(ra, k);
    w[k] = ld<256>(rb, k);
  }
  if constexpr (REDUCE == 0) {
    unsigned acc = 0;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      if constexpr (PAT == 3) st<256>(rb, k, v[k]);
      acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
      acc += w[k].x + w[k].y + w[k].z + w[k].w;
    }
    if (acc == 0x9e3779b9u) g.sink[threadIdx.x] = acc;
  } else {
    double a = 0.0, b = 0.0;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      float d[8], e[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float w0 = lc::bf_lo(v[k][q]), w1 = lc::bf_hi(v[k][q]);
        const float s0 = lc::bf_lo(w[k][q]), s1 = lc::bf_hi(w[k][q]);
        d[2 * q] = fabsf(w0 - s0);
        d[2 * q + 1] = fabsf(w1 - s1);
        e[2 * q] = fabsf(s0);
        e[2 * q + 1] = fabsf(s1);
      }
      a += static_cast<double>(((d[0] + d[1]) + (d[2] + d[3])) + ((d[4] + d[5]) + (d[6] + d[7])));
      b += static_cast<double>(((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7])));
      if constexpr (PAT == 3) st<256>(rb, k, v[k]);
    }
    if constexpr (REDUCE == 1) {
      lc::block_sum2<256>(a, b);
      if (threadIdx.x == 0) g.partials[t] = make_double2(a, b);
    } else {
      lc::wave_sum2(a, b);
      if ((threadIdx.x & 63) == 0) g.partials[t * 4 + (threadIdx.x >> 6)] = make_double2(a, b);
    }
  }
}

// ---- persist: resident blocks walking tiles against one tile per block --------
// G blocks (a multiple of 8; block x runs on XCD x mod 8) each walk `per`
// tiles of their XCD's eighth: ORDER 0 grid-stride (tile base + j + i G/8),
// ORDER 1 contiguous runs (tile base + j per + i).  The next tile's loads are
// issued before the current tile is consumed, into a second register set (no
// copies between the sets, so each wait is for the older tile only); past the
// last tile the descriptors cover zero bytes and the loads touch no memory.
template <int PAT, int ORDER>
__global__ __launch_bounds__(256) void persist_probe(const char* a, char* b, unsigned* sink, unsigned tiles) {
  constexpr unsigned kTile = 256 * 2 * 16;
  const unsigned B = gridDim.x / 8u, xcd = blockIdx.x % 8u, j = blockIdx.x / 8u;
  const unsigned per = tiles / 8u / B;
  const size_t base = static_cast<size_t>(xcd) * (tiles / 8u);
  auto tile_at = [&](unsigned i) -> size_t {
    return ORDER == 0 ? base + j + static_cast<size_t>(i) * B : base + static_cast<size_t>(j) * per + i;
  };
  u32x4 va[2], wa[2], vb[2], wb[2];
  auto issue = [&](unsigned i, u32x4* v, u32x4* w) {
    const bool ok = i < per;
    const size_t t = ok ? tile_at(i) : 0;
    const int n = ok ? static_cast<int>(kTile) : 0;
    const auto ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a) + t * kTile, 0, n, 0x00020000);
    const auto rb = __builtin_amdgcn_make_buffer_rsrc(b + t * kTile, 0, n, 0x00020000);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      v[k] = ld<256>(ra, k);
      if constexpr (PAT != 2) w[k] = ld<256>(rb, k);
    }
  };
  unsigned acc = 0;
  auto consume = [&](unsigned i, const u32x4* v, const u32x4* w) {
    const auto rb = tile(b, tile_at(i), kTile);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      if constexpr (PAT >= 2) st<256>(rb, k, v[k]);
      acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
      if constexpr (PAT != 2) acc += w[k].x + w[k].y + w[k].z + w[k].w;
    }
  };
  issue(0, va, wa);
  for (unsigned i = 0; i < per; i += 2) {  // per is even (host check)
    issue(i + 1, vb, wb);
    consume(i, va, wa);
    issue(i + 2, va, wa);
    consume(i + 1, vb, wb);
  }
  if (acc == 0x9e3779b9u) sink[threadIdx.x] = acc;
}

template <typename F>
double best_ms(F launch, int reps) {
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  launch();
  CK(hipDeviceSynchronize());
  double best = 1e30;
  for (int round = 0; round < 2; ++round) {
    CK(hipEventRecord(e0));
    for (int i = 0; i < reps; ++i) launch();
    CK(hipEventRecord(e1));
    CK(hipEventSynchronize(e1));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, e0, e1));
    if (ms / reps < best) best = ms / reps;
  }
  CK(hipEventDestroy(e0));
  CK(hipEventDestroy(e1));
  return best;
}

const char* const kNames[4] = {"read1", "read2", "copy", "r2w1"};
const int kStreams[4] = {1, 2, 2, 3};

template <int PAT, int VEC, int NT>
void run(const char* a, char* b, unsigned* sink, size_t bytes, long skew, long offset, int blocks_per_cu = 0) {
  constexpr unsigned kTile = NT * VEC * 16;
  const unsigned grid = static_cast<unsigned>(bytes / kTile);
  const unsigned lds = lds_for(blocks_per_cu);
  const double ms = best_ms(
      [&] { hipLaunchKernelGGL((probe<PAT, VEC, NT>), dim3(grid), dim3(NT), lds, 0, a, b, sink); }, 8);
  CK(hipGetLastError());
  std::printf("{\"pattern\": \"%s\", \"vec\": %d, \"threads\": %d, \"tile_bytes\": %u, \"bytes_per_array\": %zu, "
              "\"skew\": %ld, \"offset\": %ld, \"blocks_per_cu\": %d, \"lds\": %u, \"gbs\": %.1f}\n",
              kNames[PAT], VEC, NT, kTile, bytes, skew, offset, lds ? blocks_per_cu : 0, lds,
              kStreams[PAT] * static_cast<double>(bytes) / ms / 1e6);
  std::fflush(stdout);
}

template <int PAT>
void sweep(const char* a, char* b, unsigned* sink, size_t bytes, long skew, long offset) {
  for (int k : {0, 2, 3, 4, 6}) run<PAT, 2, 256>(a, b, sink, bytes, skew, offset, k);
  run<PAT, 4, 256>(a, b, sink, bytes, skew, offset);
  run<PAT, 8, 256>(a, b, sink, bytes, skew, offset);
  run<PAT, 2, 512>(a, b, sink, bytes, skew, offset);
  run<PAT, 4, 512>(a, b, sink, bytes, skew, offset);
}

}  // namespace

// Rate in GB/s of `pattern` (0 read1, 1 read2, 2 copy, 3 r2w1) with the
// kernels' tile (2 vectors x 256 lanes, 8 KiB per stream) over the first
// bytes - bytes % 8 KiB of `a` and `b` (device memory the caller owns; b is
// written by copy and r2w1, with a's bytes), on the null stream, with at most
// `blocks_per_cu` blocks per CU (0: as many as fit); the best of two rounds
// of `reps` launches.  Returns 0, or -1 for bad arguments or a HIP error
// (nothing is launched for bad arguments).
extern "C" int lc_probe_arrays(int pattern, const void* a, void* b, uint64_t bytes, int reps, int blocks_per_cu,
                               double* gbs_out) {
  constexpr unsigned kTile = 256 * 2 * 16;
  const uint64_t tiles = bytes / kTile;
  if (!a || !b || !gbs_out || pattern < 0 || pattern > 3 || reps < 1 || tiles == 0 || tiles > 0xFFFFFFFFull / 256 ||
      blocks_per_cu < 0 || blocks_per_cu > 32)
    return -1;
  const unsigned lds = lds_for(blocks_per_cu);
  unsigned* sink = nullptr;
  if (hipMalloc(&sink, 256 * sizeof(unsigned)) != hipSuccess) return -1;
  const char* pa = static_cast<const char*>(a);
  char* pb = static_cast<char*>(b);
  const dim3 grid(static_cast<unsigned>(tiles)), block(256);
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1;
  auto launch = [&] {
    switch (pattern) {
      case 0: hipLaunchKernelGGL((probe<0, 2, 256>), grid, block, lds, 0, pa, pb, sink); break;
      case 1: hipLaunchKernelGGL((probe<1, 2, 256>), grid, block, lds, 0, pa, pb, sink); break;
      case 2: hipLaunchKernelGGL((probe<2, 2, 256>), grid, block, lds, 0, pa, pb, sink); break;
      default: hipLaunchKernelGGL((probe<3, 2, 256>), grid, block, lds, 0, pa, pb, sink); break;
    }
  };
  launch();
  double best = 1e30;
  bool ok = hipDeviceSynchronize() == hipSuccess;
  for (int round = 0; ok && round < 2; ++round) {
    ok = hipEventRecord(e0) == hipSuccess;
    for (int i = 0; ok && i < reps; ++i) launch();
    ok = ok && hipEventRecord(e1) == hipSuccess && hipEventSynchronize(e1) == hipSuccess;
    float ms = 0.f;
    ok = ok && hipEventElapsedTime(&ms, e0, e1) == hipSuccess;
    if (ok && ms / reps < best) best = ms / reps;
  }
  ok = ok && hipGetLastError() == hipSuccess;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  (void)hipFree(sink);
  if (!ok) return -1;
  *gbs_out = kStreams[pattern] * static_cast<double>(tiles * kTile) / best / 1e6;
  return 0;
}

#ifdef LC_PROBE_MAIN
int main(int argc, char** argv) {
  if (argc > 1 && std::string(argv[1]) == "empty") {
    unsigned *n_work = nullptr, *sink = nullptr;
    CK(hipMalloc(&n_work, sizeof(unsigned)));
    CK(hipMalloc(&sink, 256 * sizeof(unsigned)));
    CK(hipMemset(n_work, 0, sizeof(unsigned)));
    for (unsigned grid : {1u << 16, 1u << 20, 1u << 22, 14u << 20}) {  // 14 M blocks: the 8B worst-case pack
      const double ms = best_ms([&] { hipLaunchKernelGGL(empty_blocks, dim3(grid), dim3(256), 0, 0, n_work, sink); }, 8);
      CK(hipGetLastError());
      std::printf("{\"pattern\": \"empty\", \"blocks\": %u, \"threads\": 256, \"us\": %.1f}\n", grid, ms * 1e3);
      std::fflush(stdout);
    }
    CK(hipFree(n_work));
    CK(hipFree(sink));
    return 0;
  }
  if (argc > 1 && std::string(argv[1]) == "pairs") {
    // grid = bytes / 8 KiB tiles, every tile inside [0, bytes) of both arrays
    constexpr int kPairs = 8;
    const size_t bytes = size_t{8} << 30;
    char *a[kPairs], *b[kPairs];
    unsigned* sink = nullptr;
    for (int i = 0; i < kPairs; ++i) {
      CK(hipMalloc(&a[i], bytes));
      CK(hipMalloc(&b[i], bytes));
      CK(hipMemset(a[i], 1, bytes));
      CK(hipMemset(b[i], 2, bytes));
    }
    CK(hipMalloc(&sink, 512 * sizeof(unsigned)));
    CK(hipDeviceSynchronize());
    const unsigned lds = lds_for(3);
    // the shifted runs cover bytes - 512 MiB, so the second array's tiles stay inside it
    constexpr size_t kMaxShift = size_t{512} << 20;
    auto rate = [&](int pat, const char* x, char* y, size_t n) {
      const unsigned g = static_cast<unsigned>(n / (256 * 2 * 16));
      const double ms = best_ms(
          [&] {
            if (pat == 3) hipLaunchKernelGGL((probe<3, 2, 256>), dim3(g), dim3(256), lds, 0, x, y, sink);
            else hipLaunchKernelGGL((probe<2, 2, 256>), dim3(g), dim3(256), lds, 0, x, y, sink);
          },
          6);
      CK(hipGetLastError());
      return kStreams[pat] * static_cast<double>(n) / ms / 1e6;
    };
    for (int round = 0; round < 3; ++round)
      for (int i = 0; i < kPairs; ++i) {
        const double r = rate(3, a[i], b[i], bytes), c = rate(2, a[i], b[i], bytes),
                     x = rate(3, a[i], b[(i + 1) % kPairs], bytes),
                     s0 = rate(3, a[i], b[i], bytes - kMaxShift),
                     s64 = rate(3, a[i], b[i] + (size_t{64} << 20), bytes - kMaxShift),
                     s512 = rate(3, a[i], b[i] + kMaxShift, bytes - kMaxShift);
        std::printf("{\"pattern\": \"pairs\", \"round\": %d, \"pair\": %d, \"blocks_per_cu\": %d, "
                    "\"r2w1_gbs\": %.1f, \"copy_gbs\": %.1f, \"r2w1_next_pair_gbs\": %.1f, "
                    "\"r2w1_shift0_gbs\": %.1f, \"r2w1_shift64m_gbs\": %.1f, \"r2w1_shift512m_gbs\": %.1f}\n",
                    round, i, lds ? 3 : 0, r, c, x, s0, s64, s512);
        std::fflush(stdout);
      }
    for (int i = 0; i < kPairs; ++i) {
      CK(hipFree(a[i]));
      CK(hipFree(b[i]));
    }
    CK(hipFree(sink));
    return 0;
  }
  if (argc > 1 && (std::string(argv[1]) == "tail" || std::string(argv[1]) == "persist")) {
    // two 16 GiB arrays; every block's tiles lie inside [0, bytes) of both
    const size_t bytes = size_t{16} << 30;
    constexpr unsigned kTile = 256 * 2 * 16;
    const unsigned tiles = static_cast<unsigned>(bytes / kTile);  // 2 M, a multiple of kTailSegTiles and of 8
    char *a = nullptr, *b = nullptr;
    unsigned* sink = nullptr;
    CK(hipMalloc(&a, bytes));
    CK(hipMalloc(&b, bytes));
    CK(hipMalloc(&sink, 256 * sizeof(unsigned)));
    CK(hipMemset(a, 1, bytes));
    CK(hipMemset(b, 2, bytes));
    if (std::string(argv[1]) == "tail") {
      const unsigned nseg = tiles / kTailSegTiles;
      std::vector<uint32_t> tile_seg(tiles);
      std::vector<TailSeg> segs(nseg);
      for (unsigned i = 0; i < nseg; ++i)
        segs[i] = TailSeg{reinterpret_cast<uint64_t>(a + static_cast<size_t>(i) * kTailSegTiles * kTile),
                          reinterpret_cast<uint64_t>(b + static_cast<size_t>(i) * kTailSegTiles * kTile),
                          static_cast<uint64_t>(i) * kTailSegTiles};
      for (unsigned i = 0; i < tiles; ++i) tile_seg[i] = i / kTailSegTiles;
      TailArgs g{a, b, nullptr, nullptr, nullptr, sink};
      uint32_t* d_ts = nullptr;
      TailSeg* d_segs = nullptr;
      double2* parts = nullptr;
      CK(hipMalloc(&d_ts, tiles * sizeof(uint32_t)));
      CK(hipMalloc(&d_segs, nseg * sizeof(TailSeg)));
      CK(hipMalloc(&parts, static_cast<size_t>(tiles) * 4 * sizeof(double2)));
      CK(hipMemcpy(d_ts, tile_seg.data(), tiles * sizeof(uint32_t), hipMemcpyHostToDevice));
      CK(hipMemcpy(d_segs, segs.data(), nseg * sizeof(TailSeg), hipMemcpyHostToDevice));
      CK(hipDeviceSynchronize());
      g.tile_seg = d_ts;
      g.segs = d_segs;
      g.partials = parts;
      const char* vname[4] = {"bare", "lookups", "lookups+block_reduce", "lookups+wave_partials"};
      auto one = [&](int pat, int variant, int k) {
        const unsigned lds = lds_for(k);
        if (k > 0 && lds == 0) return;
        auto launch = [&] {
          const dim3 grid(tiles), block(256);
          if (pat == 1) {
            if (variant == 0) hipLaunchKernelGGL((tail_probe<1, 0, 0>), grid, block, lds, 0, g);
            else if (variant == 1) hipLaunchKernelGGL((tail_probe<1, 1, 0>), grid, block, lds, 0, g);
            else if (variant == 2) hipLaunchKernelGGL((tail_probe<1, 1, 1>), grid, block, lds, 0, g);
            else hipLaunchKernelGGL((tail_probe<1, 1, 2>), grid, block, lds, 0, g);
          } else {
            if (variant == 0) hipLaunchKernelGGL((tail_probe<3, 0, 0>), grid, block, lds, 0, g);
            else if (variant == 1) hipLaunchKernelGGL((tail_probe<3, 1, 0>), grid, block, lds, 0, g);
            else if (variant == 2) hipLaunchKernelGGL((tail_probe<3, 1, 1>), grid, block, lds, 0, g);
            else hipLaunchKernelGGL((tail_probe<3, 1, 2>), grid, block, lds, 0, g);
          }
        };
        const double ms = best_ms(launch, 5);
        CK(hipGetLastError());
        std::printf("{\"pattern\": \"%s\", \"variant\": \"%s\", \"blocks_per_cu\": %d, \"gbs\": %.1f}\n",
                    kNames[pat], vname[variant], k, kStreams[pat] * static_cast<double>(bytes) / ms / 1e6);
        std::fflush(stdout);
      };
      for (int pat : {1, 3})
        for (int k : {2, 3, 4, 6, 0})
          for (int variant = 0; variant < 4; ++variant) one(pat, variant, k);
      CK(hipFree(d_ts));
      CK(hipFree(d_segs));
      CK(hipFree(parts));
    } else {
      int dev = 0, cus = 0;
      CK(hipGetDevice(&dev));
      CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
      CK(hipDeviceSynchronize());
      for (int pat : {1, 3, 2})
        for (int k : {1, 2, 4}) {
          const unsigned lds = lds_for(k);
          if (lds == 0) continue;
          const double ms1 = best_ms(
              [&] {
                if (pat == 1) hipLaunchKernelGGL((probe<1, 2, 256>), dim3(tiles), dim3(256), lds, 0, a, b, sink);
                else if (pat == 3) hipLaunchKernelGGL((probe<3, 2, 256>), dim3(tiles), dim3(256), lds, 0, a, b, sink);
                else hipLaunchKernelGGL((probe<2, 2, 256>), dim3(tiles), dim3(256), lds, 0, a, b, sink);
              },
              5);
          CK(hipGetLastError());
          // G blocks per launch, all resident at once (k per CU); each walks
          // per = tiles / G tiles, an even count
          const unsigned G = static_cast<unsigned>(k * cus);
          const bool fits = G > 0 && G % 8 == 0 && (tiles / 8) % (G / 8) == 0 && (tiles / G) % 2 == 0;
          double ms_stride = 0.0, ms_runs = 0.0;
          if (fits) {
            ms_stride = best_ms(
                [&] {
                  if (pat == 1) hipLaunchKernelGGL((persist_probe<1, 0>), dim3(G), dim3(256), lds, 0, a, b, sink, tiles);
                  else if (pat == 3) hipLaunchKernelGGL((persist_probe<3, 0>), dim3(G), dim3(256), lds, 0, a, b, sink, tiles);
                  else hipLaunchKernelGGL((persist_probe<2, 0>), dim3(G), dim3(256), lds, 0, a, b, sink, tiles);
                },
                5);
            CK(hipGetLastError());
            ms_runs = best_ms(
                [&] {
                  if (pat == 1) hipLaunchKernelGGL((persist_probe<1, 1>), dim3(G), dim3(256), lds, 0, a, b, sink, tiles);
                  else if (pat == 3) hipLaunchKernelGGL((persist_probe<3, 1>), dim3(G), dim3(256), lds, 0, a, b, sink, tiles);
                  else hipLaunchKernelGGL((persist_probe<2, 1>), dim3(G), dim3(256), lds, 0, a, b, sink, tiles);
                },
                5);
            CK(hipGetLastError());
          }
          const double rate = kStreams[pat] * static_cast<double>(bytes) / 1e6;
          std::printf("{\"pattern\": \"%s\", \"blocks_per_cu\": %d, \"one_tile_per_block_gbs\": %.1f, "
                      "\"persistent_grid_stride_gbs\": %.1f, \"persistent_runs_gbs\": %.1f}\n",
                      kNames[pat], k, rate / ms1, fits ? rate / ms_stride : 0.0, fits ? rate / ms_runs : 0.0);
          std::fflush(stdout);
        }
    }
    CK(hipFree(a));
    CK(hipFree(b));
    CK(hipFree(sink));
    return 0;
  }
  const long gib = argc > 1 ? std::atol(argv[1]) : 16;
  const long skew = argc > 2 ? std::atol(argv[2]) : 20480;
  const long offset = argc > 3 ? std::atol(argv[3]) : 0;
  if (gib < 1 || gib > 64 || skew < 0 || skew > (1l << 30) || skew % 16 || offset < 0 || offset > (1l << 21) ||
      offset % 16) {
    std::fprintf(stderr, "lc_hbm_probe: GiB per array in [1, 64]; skew a multiple of 16 in [0, 1 GiB]; "
                         "offset a multiple of 16 in [0, 2 MiB]\n");
    return 2;
  }
  // every tile of every sweep lies inside [0, bytes) of each array: bytes is a
  // multiple of the largest tile (64 KiB), and each allocation holds
  // offset (+ skew) + bytes
  const size_t bytes = static_cast<size_t>(gib) << 30;
  if (bytes / (256 * 2 * 16) > 0xFFFFFFFFull) return 2;
  char *a0 = nullptr, *b0 = nullptr;
  unsigned* sink = nullptr;
  CK(hipMalloc(&a0, bytes + offset));
  CK(hipMalloc(&b0, bytes + offset + skew));
  char* a = a0 + offset;
  char* b = b0 + offset + skew;
  CK(hipMalloc(&sink, 512 * sizeof(unsigned)));
  CK(hipMemset(a0, 1, bytes + offset));
  CK(hipMemset(b0, 2, bytes + offset + skew));
  CK(hipDeviceSynchronize());
  sweep<0>(a, b, sink, bytes, skew, offset);
  sweep<1>(a, b, sink, bytes, skew, offset);
  sweep<2>(a, b, sink, bytes, skew, offset);
  sweep<3>(a, b, sink, bytes, skew, offset);
  CK(hipFree(a0));
  CK(hipFree(b0));
  CK(hipFree(sink));
  return 0;
}
#endif  // LC_PROBE_MAIN
