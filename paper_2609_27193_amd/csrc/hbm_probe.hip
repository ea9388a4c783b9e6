// Practical HBM ceilings of the access patterns the library's kernels use,
// measured with no arithmetic in the way: read-only, copy (one read and one
// write stream) and two reads plus one write (the ACCUM score pattern: W and
// S read, S written).  Same tile as the kernels (256 threads, two 16-byte
// vectors per thread and stream, so 8 KiB per stream per block, accessed
// through a buffer resource per tile with the non-temporal, device-scope
// cache policy) and the same XCD-contiguous block mapping.  The second array
// starts `skew` bytes into its allocation, so the two streams need not sit
// at the same offsets of the memory interleave.  Prints one JSON line.
//
//   lc_hbm_probe [GiB per array, default 16] [skew bytes, default 20480]
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr int kVec = 2;
constexpr unsigned kTile = kThreads * kVec * 16;  // 8 KiB
constexpr int kPolicy = 2 | 16;                   // nt | sc1

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile(const u32x4* base, size_t t) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<u32x4*>(base) + t * kThreads * kVec, 0, kTile, 0x00020000);
}
__device__ __forceinline__ u32x4 ld(__amdgpu_buffer_rsrc_t r, int k) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (threadIdx.x + k * kThreads) * 16, 0, kPolicy);
}
__device__ __forceinline__ void st(__amdgpu_buffer_rsrc_t r, int k, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (threadIdx.x + k * kThreads) * 16, 0, kPolicy);
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

__global__ __launch_bounds__(kThreads) void read_only(const u32x4* a, unsigned* sink) {
  const auto ra = tile(a, tile_of(blockIdx.x, gridDim.x));
  unsigned acc = 0;
  u32x4 v[kVec];
#pragma unroll
  for (int k = 0; k < kVec; ++k) v[k] = ld(ra, k);
#pragma unroll
  for (int k = 0; k < kVec; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  if (acc == 0x9e3779b9u) sink[threadIdx.x] = acc;  // keeps the loads; the pattern never occurs
}

__global__ __launch_bounds__(kThreads) void copy(const u32x4* a, u32x4* b) {
  const size_t t = tile_of(blockIdx.x, gridDim.x);
  const auto ra = tile(a, t), rb = tile(b, t);
  u32x4 v[kVec];
#pragma unroll
  for (int k = 0; k < kVec; ++k) v[k] = ld(ra, k);
#pragma unroll
  for (int k = 0; k < kVec; ++k) st(rb, k, v[k]);
}

__global__ __launch_bounds__(kThreads) void read2_write1(const u32x4* a, u32x4* b, unsigned* sink) {
  const size_t t = tile_of(blockIdx.x, gridDim.x);
  const auto ra = tile(a, t), rb = tile(b, t);
  u32x4 v[kVec], w[kVec];
  unsigned acc = 0;
#pragma unroll
  for (int k = 0; k < kVec; ++k) {
    v[k] = ld(ra, k);
    w[k] = ld(rb, k);
  }
#pragma unroll
  for (int k = 0; k < kVec; ++k) {
    acc += w[k].x ^ v[k].y;
    st(rb, k, v[k]);
  }
  if (acc == 0x9e3779b9u) sink[threadIdx.x] = acc;
}

template <typename F>
float mean_ms(F launch, int reps) {
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  launch();
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(e0));
  for (int i = 0; i < reps; ++i) launch();
  CK(hipEventRecord(e1));
  CK(hipEventSynchronize(e1));
  float ms = 0.f;
  CK(hipEventElapsedTime(&ms, e0, e1));
  CK(hipEventDestroy(e0));
  CK(hipEventDestroy(e1));
  return ms / reps;
}

}  // namespace

int main(int argc, char** argv) {
  const long gib = argc > 1 ? std::atol(argv[1]) : 16;
  const long skew = argc > 2 ? std::atol(argv[2]) : 20480;
  if (gib < 1 || gib > 64 || skew < 0 || skew > (1l << 30) || skew % 16) {
    std::fprintf(stderr, "lc_hbm_probe: GiB per array in [1, 64]; skew a multiple of 16 in [0, 1 GiB]\n");
    return 2;
  }
  const size_t bytes = static_cast<size_t>(gib) << 30;
  const size_t tiles = bytes / kTile;  // exact: GiB multiple
  if (tiles > 0xFFFFFFFFull) return 2;
  const unsigned grid = static_cast<unsigned>(tiles);
  u32x4 *a = nullptr, *b0 = nullptr, *b = nullptr;
  unsigned* sink = nullptr;
  CK(hipMalloc(&a, bytes));
  CK(hipMalloc(&b0, bytes + skew));
  b = reinterpret_cast<u32x4*>(reinterpret_cast<char*>(b0) + skew);
  CK(hipMalloc(&sink, kThreads * sizeof(unsigned)));
  CK(hipMemset(a, 1, bytes));
  CK(hipMemset(b, 2, bytes));
  CK(hipDeviceSynchronize());
  const int reps = 10;
  const double r = mean_ms([&] { hipLaunchKernelGGL(read_only, dim3(grid), dim3(kThreads), 0, 0, a, sink); }, reps);
  const double c = mean_ms([&] { hipLaunchKernelGGL(copy, dim3(grid), dim3(kThreads), 0, 0, a, b); }, reps);
  const double w = mean_ms([&] { hipLaunchKernelGGL(read2_write1, dim3(grid), dim3(kThreads), 0, 0, a, b, sink); },
                           reps);
  CK(hipGetLastError());
  std::printf("{\"bytes_per_array\": %zu, \"skew\": %ld, \"read_gbs\": %.1f, \"copy_gbs\": %.1f, "
              "\"read2_write1_gbs\": %.1f}\n",
              bytes, skew, bytes / r / 1e6, 2.0 * bytes / c / 1e6, 3.0 * bytes / w / 1e6);
  CK(hipFree(a));
  CK(hipFree(b0));
  CK(hipFree(sink));
  return 0;
}
