// HIP kernels of the optimizer steps that yield the drift statistic (Section
// 3.4: the drift is taken from the optimizer's own update): AdamW, as the
// paper trains, and plain SGD, which Section 4.7 notes the method carries
// over to.  One pass over the optimizer state per step; per chunk of the
// score layout the kernel updates the parameters and writes the Eq. 1
// partial sums of |p_new - p| and |p|, which the finalize kernel turns into
// u and Delta.  Streaming rules as in lc_kernels.hip (full chunks through
// buffer resources, ragged ones through global pointers).
#include "lc_device.h"

namespace lc {
namespace {

constexpr int kAdamW = 0;
constexpr int kSGD = 1;

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7FC0u;  // NaN stays a quiet NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// One AdamW element update in fp32, one rounding per operation, fixed order.
// The library is built with -ffp-contract=off (no fused multiply-adds), and
// fp32 division and sqrtf compile to their correctly rounded sequences
// (div_scale/div_fmas/div_fixup; v_sqrt with neighbour correction), so every
// operation below is the IEEE round-to-nearest-even result.
__device__ __forceinline__ float adamw_elem(float p, float& m, float& v, float g, const AdamScalars& sc,
                                            bool decay) {
  m = sc.b1 * m + sc.omb1 * g;
  v = sc.b2 * v + sc.omb2 * (g * g);
  const float mh = m * sc.c1;
  const float vh = v * sc.c2;
  const float den = sqrtf(vh) + sc.eps;
  const float upd = mh / den;
  const float p1 = decay ? p * sc.decay : p;
  return p1 - sc.lr * upd;
}

template <int WDT>
__device__ __forceinline__ float w_load(const uint8_t* w, uint64_t i) {
  if constexpr (WDT == 1) return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(w)[i]) << 16);
  else return reinterpret_cast<const float*>(w)[i];
}
template <int WDT>
__device__ __forceinline__ void w_store(uint8_t* w, uint64_t i, float x) {
  if constexpr (WDT == 1) reinterpret_cast<uint16_t*>(w)[i] = bf16_rne(x);
  else reinterpret_cast<float*>(w)[i] = x;
}
template <int GDT>
__device__ __forceinline__ float g_load(const uint8_t* g, uint64_t i) {
  if constexpr (GDT == 1) return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(g)[i]) << 16);
  else return reinterpret_cast<const float*>(g)[i];
}

// One SGD element update in fp32 with decoupled weight decay, one rounding
// per operation: p_new = p * (1 - lr wd) - lr g (the decay only for decayed
// segments).
__device__ __forceinline__ float sgd_elem(float p, float g, const SgdScalars& sc, bool decay) {
  const float p1 = decay ? p * sc.decay : p;
  return p1 - sc.lr * g;
}

// The tiles of one full chunk: the parameters (the fp32 master, else the
// weights), the weights, the gradient and, for AdamW, the moments.
struct ChunkTiles {
  tile_t p, w, g, m, v;
};

__device__ __forceinline__ u32x4 widen_bf16x4(u32x2 x) {
  return u32x4{x[0] << 16, x[0] & 0xffff0000u, x[1] << 16, x[1] & 0xffff0000u};
}
__device__ __forceinline__ u32x2 narrow_bf16x4(u32x4 p) {
  return u32x2{bf16_rne(__uint_as_float(p[0])) | (static_cast<uint32_t>(bf16_rne(__uint_as_float(p[1]))) << 16),
               bf16_rne(__uint_as_float(p[2])) | (static_cast<uint32_t>(bf16_rne(__uint_as_float(p[3]))) << 16)};
}

// Four consecutive elements (every array 4-element aligned): loaded through
// global pointers (group gi of the segment, ragged chunks) or through the
// chunk's tiles (group j of a full chunk), updated in place, stored the same
// way.  AdamW also streams m and v; SGD touches only the parameters.
template <int OPT, int WDT, int GDT, bool MASTER>
struct Group4 {
  u32x4 p, m, v;  // parameters as fp32 bits, moments
  float g[4];

  __device__ __forceinline__ void set_grad(u32x2 x) {
    g[0] = __uint_as_float(x[0] << 16); g[1] = __uint_as_float(x[0] & 0xffff0000u);
    g[2] = __uint_as_float(x[1] << 16); g[3] = __uint_as_float(x[1] & 0xffff0000u);
  }
  __device__ __forceinline__ void set_grad(u32x4 x) {
    for (int k = 0; k < 4; ++k) g[k] = __uint_as_float(x[k]);
  }
  __device__ __forceinline__ void load(const OptSeg& sg, const GradSeg& gs, uint64_t gi) {
    if constexpr (MASTER) p = ld_nt(reinterpret_cast<const u32x4*>(sg.master) + gi);
    else if constexpr (WDT == 1) p = widen_bf16x4(ld_nt2(reinterpret_cast<const u32x2*>(sg.w) + gi));
    else p = ld_nt(reinterpret_cast<const u32x4*>(sg.w) + gi);
    if constexpr (OPT == kAdamW) {
      m = ld_nt(reinterpret_cast<const u32x4*>(sg.m) + gi);
      v = ld_nt(reinterpret_cast<const u32x4*>(sg.v) + gi);
    }
    if constexpr (GDT == 1) set_grad(ld_nt2(reinterpret_cast<const u32x2*>(gs.grad) + gi));
    else set_grad(ld_nt(reinterpret_cast<const u32x4*>(gs.grad) + gi));
  }
  __device__ __forceinline__ void load(const ChunkTiles& t, uint32_t j) {
    if constexpr (MASTER) p = ld_tile(t.p, j * 16u);
    else if constexpr (WDT == 1) p = widen_bf16x4(ld_tile2(t.p, j * 8u));
    else p = ld_tile(t.p, j * 16u);
    if constexpr (OPT == kAdamW) {
      m = ld_tile(t.m, j * 16u);
      v = ld_tile(t.v, j * 16u);
    }
    if constexpr (GDT == 1) set_grad(ld_tile2(t.g, j * 8u));
    else set_grad(ld_tile(t.g, j * 16u));
  }
  // One optimizer step of the four elements in place; returns the drift terms
  // (sum|p_new - p|, sum|p|) of the group.
  template <typename SC>
  __device__ __forceinline__ void update(const SC& sc, bool decay, float& da, float& db) {
    float d[4], b[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float po = __uint_as_float(p[k]);
      float x;
      if constexpr (OPT == kAdamW) {
        float mm = __uint_as_float(m[k]), vv = __uint_as_float(v[k]);
        x = adamw_elem(po, mm, vv, g[k], sc, decay);
        m[k] = __float_as_uint(mm);
        v[k] = __float_as_uint(vv);
      } else {
        x = sgd_elem(po, g[k], sc, decay);
      }
      p[k] = __float_as_uint(x);
      d[k] = fabsf(x - po);
      b[k] = fabsf(po);
    }
    da = (d[0] + d[1]) + (d[2] + d[3]);
    db = (b[0] + b[1]) + (b[2] + b[3]);
  }
  __device__ __forceinline__ void store(const OptSeg& sg, uint64_t gi) const {
    if constexpr (OPT == kAdamW) {
      st_nt(reinterpret_cast<u32x4*>(sg.m) + gi, m);
      st_nt(reinterpret_cast<u32x4*>(sg.v) + gi, v);
    }
    if constexpr (MASTER) st_nt(reinterpret_cast<u32x4*>(sg.master) + gi, p);
    if constexpr (WDT == 1) st_nt2(reinterpret_cast<u32x2*>(sg.w) + gi, narrow_bf16x4(p));
    else st_nt(reinterpret_cast<u32x4*>(sg.w) + gi, p);
  }
  __device__ __forceinline__ void store(const ChunkTiles& t, uint32_t j) const {
    if constexpr (OPT == kAdamW) {
      st_tile(t.m, j * 16u, m);
      st_tile(t.v, j * 16u, v);
    }
    if constexpr (MASTER) st_tile(t.p, j * 16u, p);
    if constexpr (WDT == 1) st_tile2(t.w, j * 8u, narrow_bf16x4(p));
    else st_tile(t.w, j * 16u, p);
  }
};

template <int OPT, int WDT, int GDT, bool MASTER, typename SC>
__device__ __forceinline__ void optim_chunk(const DeviceTables& t, const SC& sc, uint32_t c) {
  constexpr uint32_t WSZ = WDT == 1 ? 2 : 4;
  constexpr uint32_t CE = kChunkBytes / WSZ;        // elements per chunk (the score chunks)
  constexpr uint32_t GPT = CE / 4 / kScoreThreads;  // 4-element groups per thread in a full chunk
  static_assert(GPT >= 1 && CE % (4 * kScoreThreads) == 0, "tiling");
  const uint32_t tid = threadIdx.x;
  const uint32_t si = t.chunk_seg[c];
  const OptSeg sg = t.opt_segs[si];
  const GradSeg gs = t.grad_segs[si];
  const uint64_t e0 = static_cast<uint64_t>(c - sg.chunk_begin) * CE;
  const uint64_t rem = sg.numel - e0;
  const uint32_t n = rem < CE ? static_cast<uint32_t>(rem) : CE;
  const bool decay = gs.decay != 0;
  double a = 0.0, b = 0.0;
  uint32_t scalar_from = 0;
  if (sg.vec_ok && gs.vec_ok) {
    const uint64_t g0 = e0 / 4;
    const uint32_t ng = n / 4;
    if (ng == GPT * kScoreThreads) {
      constexpr uint32_t GSZ = GDT == 1 ? 2 : 4;
      ChunkTiles tl;
      tl.w = make_tile(reinterpret_cast<const uint8_t*>(sg.w) + e0 * WSZ, CE * WSZ);
      tl.p = MASTER ? make_tile(reinterpret_cast<const float*>(sg.master) + e0, CE * 4) : tl.w;
      tl.g = make_tile(reinterpret_cast<const uint8_t*>(gs.grad) + e0 * GSZ, CE * GSZ);
      tl.m = tl.v = tl.p;
      if constexpr (OPT == kAdamW) {
        tl.m = make_tile(reinterpret_cast<const float*>(sg.m) + e0, CE * 4);
        tl.v = make_tile(reinterpret_cast<const float*>(sg.v) + e0, CE * 4);
      }
      Group4<OPT, WDT, GDT, MASTER> grp[GPT];
#pragma unroll
      for (uint32_t k = 0; k < GPT; ++k) grp[k].load(tl, tid + k * kScoreThreads);
#pragma unroll
      for (uint32_t k = 0; k < GPT; ++k) {
        float da, db;
        grp[k].update(sc, decay, da, db);
        grp[k].store(tl, tid + k * kScoreThreads);
        a += static_cast<double>(da);
        b += static_cast<double>(db);
      }
    } else {
      for (uint32_t i = tid; i < ng; i += kScoreThreads) {
        Group4<OPT, WDT, GDT, MASTER> grp;
        grp.load(sg, gs, g0 + i);
        float da, db;
        grp.update(sc, decay, da, db);
        grp.store(sg, g0 + i);
        a += static_cast<double>(da);
        b += static_cast<double>(db);
      }
    }
    scalar_from = ng * 4;
  }
  const uint8_t* wb = reinterpret_cast<const uint8_t*>(sg.w);
  for (uint32_t i = scalar_from + tid; i < n; i += kScoreThreads) {
    const uint64_t e = e0 + i;
    const float po = MASTER ? reinterpret_cast<const float*>(sg.master)[e] : w_load<WDT>(wb, e);
    const float gv = g_load<GDT>(reinterpret_cast<const uint8_t*>(gs.grad), e);
    float x;
    if constexpr (OPT == kAdamW) {
      float* mp = reinterpret_cast<float*>(sg.m) + e;
      float* vp = reinterpret_cast<float*>(sg.v) + e;
      float mm = *mp, vv = *vp;
      x = adamw_elem(po, mm, vv, gv, sc, decay);
      *mp = mm;
      *vp = vv;
    } else {
      x = sgd_elem(po, gv, sc, decay);
    }
    if constexpr (MASTER) reinterpret_cast<float*>(sg.master)[e] = x;
    w_store<WDT>(reinterpret_cast<uint8_t*>(sg.w), e, x);
    a += static_cast<double>(fabsf(x - po));
    b += static_cast<double>(fabsf(po));
  }
  block_sum2<kScoreThreads>(a, b);
  if (tid == 0) t.partials[c] = make_double2(a, b);
}

template <int OPT, int WDT, int GDT, bool MASTER, bool LOOP, typename SC>
__global__ __launch_bounds__(kScoreThreads) void optim_kernel(const DeviceTables t, const SC sc) {
  if constexpr (!LOOP) {
    optim_chunk<OPT, WDT, GDT, MASTER>(t, sc, remap_xcd(blockIdx.x, gridDim.x));
  } else {
    for (uint64_t base = 0; base < t.n_chunks; base += gridDim.x) {
      const uint64_t left = t.n_chunks - base;
      const uint32_t span = left < gridDim.x ? static_cast<uint32_t>(left) : gridDim.x;
      if (blockIdx.x >= span) return;
      optim_chunk<OPT, WDT, GDT, MASTER>(t, sc, static_cast<uint32_t>(base + remap_xcd(blockIdx.x, span)));
      __syncthreads();
    }
  }
}

template <int OPT, int WDT, int GDT, bool MASTER, typename SC>
void launch_optim_t(const DeviceTables& t, const SC& sc, hipStream_t st) {
  const uint32_t g = grid_for(t.n_chunks, kScoreThreads);
  const uint32_t lds = occupancy_lds(OPT == kAdamW ? LC_ADAMW_BLOCKS_PER_CU : LC_SGD_BLOCKS_PER_CU);
  if (g == t.n_chunks)
    hipLaunchKernelGGL((optim_kernel<OPT, WDT, GDT, MASTER, false, SC>), dim3(g), dim3(kScoreThreads), lds, st, t, sc);
  else
    hipLaunchKernelGGL((optim_kernel<OPT, WDT, GDT, MASTER, true, SC>), dim3(g), dim3(kScoreThreads), lds, st, t, sc);
}

template <int OPT, typename SC>
void launch_optim(const DeviceTables& t, int grad_dtype, int has_master, const SC& sc, hipStream_t st) {
  const bool gb = grad_dtype == 1;
  if (t.dtype == 1) {
    if (has_master) { if (gb) launch_optim_t<OPT, 1, 1, true>(t, sc, st); else launch_optim_t<OPT, 1, 2, true>(t, sc, st); }
    else { if (gb) launch_optim_t<OPT, 1, 1, false>(t, sc, st); else launch_optim_t<OPT, 1, 2, false>(t, sc, st); }
  } else {
    if (has_master) { if (gb) launch_optim_t<OPT, 2, 1, true>(t, sc, st); else launch_optim_t<OPT, 2, 2, true>(t, sc, st); }
    else { if (gb) launch_optim_t<OPT, 2, 1, false>(t, sc, st); else launch_optim_t<OPT, 2, 2, false>(t, sc, st); }
  }
}

}  // namespace

hipError_t launch_adamw(const DeviceTables& t, int grad_dtype, int has_master, const AdamScalars& sc,
                        hipStream_t st) {
  launch_optim<kAdamW>(t, grad_dtype, has_master, sc, st);
  return hipGetLastError();
}

hipError_t launch_sgd(const DeviceTables& t, int grad_dtype, int has_master, const SgdScalars& sc, hipStream_t st) {
  launch_optim<kSGD>(t, grad_dtype, has_master, sc, st);
  return hipGetLastError();
}

}  // namespace lc
