// Device helpers shared by the kernels of the LayerCheck HIP library
// (lc_kernels.hip: score, finalize, select, pack, restore; lc_optim.hip: the
// optimizer steps with drift).  Every definition has internal linkage, so
// each kernel file carries its own inlined copy.
#pragma once

#include "lc_internal.h"

namespace lc {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Every array the kernels stream is device (global) memory; accessing it
// through global-address-space pointers gives global_load/global_store
// instead of flat accesses (no aperture check, no LDS-counter coupling).
typedef __attribute__((address_space(1))) u32x4 g_u32x4;
__device__ __forceinline__ u32x4 ld_nt(const u32x4* p) {
  return __builtin_nontemporal_load((const g_u32x4*)p);
}
__device__ __forceinline__ void st_nt(u32x4* p, u32x4 v) { __builtin_nontemporal_store(v, (g_u32x4*)p); }

// bf16 -> fp32 is exact: the bf16 bits are the top half of the fp32 bits.
__device__ __forceinline__ float bf_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) u32x2 g_u32x2;
__device__ __forceinline__ u32x2 ld_nt2(const u32x2* p) { return __builtin_nontemporal_load((const g_u32x2*)p); }
__device__ __forceinline__ void st_nt2(u32x2* p, u32x2 v) { __builtin_nontemporal_store(v, (g_u32x2*)p); }

// Full tiles (a whole score chunk or copy piece) go through buffer resources
// built from the tile's base, which is uniform per block: the descriptor sits
// in scalar registers and each lane supplies a 32-bit byte offset.  Loads and
// stores carry the non-temporal, device-scope cache policy (nt sc1), which
// streamed-once data wants: on the kernels' access patterns it measured
// 0.2-2% above non-temporal global accesses.  The descriptor's record count
// is the tile size, so an offset past the tile reads zero and drops the
// store instead of reaching other memory.
typedef __amdgpu_buffer_rsrc_t tile_t;
constexpr int kStreamPolicy = 2 | 16;         // nt | sc1
constexpr int kRawBufferWord3 = 0x00020000;   // untyped access, 32-bit data format
__device__ __forceinline__ tile_t make_tile(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), kRawBufferWord3);
}
__device__ __forceinline__ u32x4 ld_tile(tile_t t, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(t, off, 0, kStreamPolicy);
}
__device__ __forceinline__ void st_tile(tile_t t, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, t, off, 0, kStreamPolicy);
}
__device__ __forceinline__ u32x2 ld_tile2(tile_t t, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(t, off, 0, kStreamPolicy);
}
__device__ __forceinline__ void st_tile2(tile_t t, uint32_t off, u32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, t, off, 0, kStreamPolicy);
}

__device__ __forceinline__ uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Work item x of a launch of G blocks.  Workgroups are dispatched round-robin
// over the 8 XCDs; with LC_XCD_REMAP each XCD instead walks one contiguous
// eighth of the items (a bijection on the first 8*floor(G/8) items, identity
// on the rest), which keeps each XCD's in-flight accesses within a narrow
// address window.
__device__ __forceinline__ uint32_t remap_xcd(uint32_t x, uint32_t G) {
#if LC_XCD_REMAP && LC_XCD_RUN > 0
  // runs of LC_XCD_RUN consecutive items per XCD, the XCDs' runs interleaved
  constexpr uint32_t R = 8u * LC_XCD_RUN;
  const uint32_t full = G - G % R;
  if (x >= full) return x;
  const uint32_t xcd = x % 8u, k = x / 8u;
  return (k / LC_XCD_RUN) * R + xcd * LC_XCD_RUN + k % LC_XCD_RUN;
#elif LC_XCD_REMAP
  const uint32_t full = G - G % 8u;
  return x < full ? (x % 8u) * (full / 8u) + x / 8u : x;
#else
  (void)G;
  return x;
#endif
}

// ---- wave64 / block reductions of an fp64 pair, fixed order ------------------
__device__ __forceinline__ double dpp_f64(double v, int ctrl_sel) {
  int lo = __double2loint(v), hi = __double2hiint(v);
  if (ctrl_sel == 0) {  // quad_perm [1,0,3,2]: partner = lane ^ 1
    lo = __builtin_amdgcn_update_dpp(0, lo, 0xB1, 0xF, 0xF, false);
    hi = __builtin_amdgcn_update_dpp(0, hi, 0xB1, 0xF, 0xF, false);
  } else {              // quad_perm [2,3,0,1]: partner = lane ^ 2
    lo = __builtin_amdgcn_update_dpp(0, lo, 0x4E, 0xF, 0xF, false);
    hi = __builtin_amdgcn_update_dpp(0, hi, 0x4E, 0xF, 0xF, false);
  }
  return __hiloint2double(hi, lo);
}

__device__ __forceinline__ void wave_sum2(double& a, double& b) {
  a += dpp_f64(a, 0);
  b += dpp_f64(b, 0);
  a += dpp_f64(a, 1);
  b += dpp_f64(b, 1);
#pragma unroll
  for (int m = 4; m < 64; m <<= 1) {
    a += __shfl_xor(a, m, 64);
    b += __shfl_xor(b, m, 64);
  }
}

// Sum of (a, b) over a block of NT threads; the result is valid in thread 0.
template <int NT>
__device__ __forceinline__ void block_sum2(double& a, double& b) {
  __shared__ double sa[NT / 64], sb[NT / 64];
  wave_sum2(a, b);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sa[wave] = a;
    sb[wave] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double x = sa[0], y = sb[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) {
      x += sa[w];
      y += sb[w];
    }
    a = x;
    b = y;
  }
}

// Blocks per launch: one per work item up to the dispatch limit of 2^32
// work-items per dimension.  Beyond it the score and copy kernels are launched
// again over the next range of items; the optimizer kernels loop.
__host__ inline uint32_t grid_for(uint64_t items, uint32_t threads) {
  uint64_t cap = (0xFFFFFFFFull / threads) & ~7ull;
  if (LC_MAX_GRID_BLOCKS > 0 && cap > LC_MAX_GRID_BLOCKS) cap = LC_MAX_GRID_BLOCKS;
  return static_cast<uint32_t>(items < cap ? items : cap);
}

}  // namespace
}  // namespace lc
