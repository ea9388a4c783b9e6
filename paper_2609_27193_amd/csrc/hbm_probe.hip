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
