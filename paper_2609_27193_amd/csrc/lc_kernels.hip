// HIP kernels of the LayerCheck decision step for gfx950 (MI355X, CDNA4).
//
// Every kernel here is HBM-bound streaming work or a tiny O(N) step; nothing
// is a dense contraction, so there is no MFMA.  Design rules:
//  * 16-byte (dwordx4) coalesced loads/stores, several in flight per lane;
//    non-temporal hints because every byte is touched once per step and the
//    per-step stream (tens of GB) dwarfs the 256 MB Infinity Cache;
//  * reductions use no floating-point atomics: one fp64 pair per chunk, then a
//    fixed-order per-layer sum, so scores are bitwise reproducible;
//  * wave64 reductions (DPP quad permutes, then cross-row shuffles), LDS for
//    the cross-wave combine.
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

// |W - S| and |S| of one 16-byte vector, summed pairwise in fp32.
template <int DT>
__device__ __forceinline__ void vec_terms(const u32x4 w, const u32x4 s, float& da, float& sb) {
  if constexpr (DT == 1) {
    float d[8], b[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float w0 = bf_lo(w[k]), w1 = bf_hi(w[k]);
      const float s0 = bf_lo(s[k]), s1 = bf_hi(s[k]);
      d[2 * k] = fabsf(w0 - s0);
      d[2 * k + 1] = fabsf(w1 - s1);
      b[2 * k] = fabsf(s0);
      b[2 * k + 1] = fabsf(s1);
    }
    da = ((d[0] + d[1]) + (d[2] + d[3])) + ((d[4] + d[5]) + (d[6] + d[7]));
    sb = ((b[0] + b[1]) + (b[2] + b[3])) + ((b[4] + b[5]) + (b[6] + b[7]));
  } else {
    float d[4], b[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float wf = __uint_as_float(w[k]), sf = __uint_as_float(s[k]);
      d[k] = fabsf(wf - sf);
      b[k] = fabsf(sf);
    }
    da = (d[0] + d[1]) + (d[2] + d[3]);
    sb = (b[0] + b[1]) + (b[2] + b[3]);
  }
}

template <int DT>
__device__ __forceinline__ float elem_value(const uint8_t* base, uint64_t i) {
  if constexpr (DT == 1) {
    return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(base)[i]) << 16);
  } else {
    return reinterpret_cast<const float*>(base)[i];
  }
}

template <int DT>
__device__ __forceinline__ void elem_copy(const uint8_t* src, uint8_t* dst, uint64_t i) {
  if constexpr (DT == 1) {
    reinterpret_cast<uint16_t*>(dst)[i] = reinterpret_cast<const uint16_t*>(src)[i];
  } else {
    reinterpret_cast<float*>(dst)[i] = reinterpret_cast<const float*>(src)[i];
  }
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

// ---- score: one chunk per block and iteration ---------------------------------
// Streams W and S of one chunk once; writes (sum|W-S|, sum|S|) in fp64.  In
// ACCUM mode the same pass stores W into S (the next step's W(t-1)).
template <int DT, bool ACCUM>
__device__ __forceinline__ void score_chunk(const DeviceTables& t, uint32_t c) {
  constexpr uint32_t ESZ = DT == 1 ? 2 : 4;
  constexpr uint32_t CE = kChunkBytes / ESZ;  // elements per chunk
  constexpr uint32_t EPV = 16 / ESZ;          // elements per 16-B vector
  constexpr uint32_t NV = CE / EPV;           // vectors per full chunk
  constexpr uint32_t VPT = NV / kScoreThreads;
  constexpr uint32_t U = VPT < 4 ? VPT : 4;   // vectors per thread per round
  static_assert(VPT % U == 0, "tiling");
  const uint32_t tid = threadIdx.x;
  const ScoreSeg sg = t.segs[t.chunk_seg[c]];
  const uint64_t e0 = static_cast<uint64_t>(c - sg.chunk_begin) * CE;
  const uint64_t rem = sg.numel - e0;
  const uint32_t n = rem < CE ? static_cast<uint32_t>(rem) : CE;
  const uint8_t* wb = reinterpret_cast<const uint8_t*>(sg.w) + e0 * ESZ;
  uint8_t* sbp = reinterpret_cast<uint8_t*>(sg.s) + e0 * ESZ;

  double a = 0.0, b = 0.0;
  uint32_t scalar_from = 0;
  if (sg.vec_ok) {
    const u32x4* wv = reinterpret_cast<const u32x4*>(wb);
    u32x4* sv = reinterpret_cast<u32x4*>(sbp);
    if (n == CE) {
#pragma unroll
      for (uint32_t r = 0; r < VPT / U; ++r) {
        u32x4 w[U], s[U];
#pragma unroll
        for (uint32_t k = 0; k < U; ++k) {
          const uint32_t i = tid + (r * U + k) * kScoreThreads;
          w[k] = ld_nt(wv + i);
          s[k] = ld_nt(sv + i);
        }
#pragma unroll
        for (uint32_t k = 0; k < U; ++k) {
          float da, db;
          vec_terms<DT>(w[k], s[k], da, db);
          a += static_cast<double>(da);
          b += static_cast<double>(db);
          if constexpr (ACCUM) st_nt(sv + tid + (r * U + k) * kScoreThreads, w[k]);
        }
      }
      scalar_from = n;
    } else {
      const uint32_t nv = n / EPV;
      for (uint32_t i = tid; i < nv; i += kScoreThreads) {
        const u32x4 w = ld_nt(wv + i);
        const u32x4 s = ld_nt(sv + i);
        float da, db;
        vec_terms<DT>(w, s, da, db);
        a += static_cast<double>(da);
        b += static_cast<double>(db);
        if constexpr (ACCUM) st_nt(sv + i, w);
      }
      scalar_from = nv * EPV;
    }
  }
  for (uint32_t i = scalar_from + tid; i < n; i += kScoreThreads) {
    const float wf = elem_value<DT>(wb, i), sf = elem_value<DT>(sbp, i);
    a += static_cast<double>(fabsf(wf - sf));
    b += static_cast<double>(fabsf(sf));
    if constexpr (ACCUM) elem_copy<DT>(wb, sbp, i);
  }
  block_sum2<kScoreThreads>(a, b);
  if (tid == 0) t.partials[c] = make_double2(a, b);
}

// LOOP = false: one chunk per block (the common case; the chunk's tables are
// read before any store, so they stay on the scalar path).  LOOP = true: the
// grid is capped by the dispatch limit and blocks take several rounds.
template <int DT, bool ACCUM, bool LOOP>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(const DeviceTables t) {
  if constexpr (!LOOP) {
    score_chunk<DT, ACCUM>(t, remap_xcd(blockIdx.x, gridDim.x));
  } else {
    for (uint64_t base = 0; base < t.n_chunks; base += gridDim.x) {
      const uint64_t left = t.n_chunks - base;
      const uint32_t span = left < gridDim.x ? static_cast<uint32_t>(left) : gridDim.x;
      if (blockIdx.x >= span) return;
      score_chunk<DT, ACCUM>(t, static_cast<uint32_t>(base + remap_xcd(blockIdx.x, span)));
      __syncthreads();  // the block reduction's LDS is reused by the next round
    }
  }
}

// ---- finalize: Eq. 1 and Eq. 2 per layer, one block per layer -----------------
// Thread j sums partials j, j + NT, j + 2 NT, ... of its layer into four
// interleaved accumulators (independent loads in flight), combined in a fixed
// order, then a fixed-order block reduction: deterministic for a given layout.
__global__ __launch_bounds__(kFinalizeThreads) void finalize_kernel(const DeviceTables t) {
  const uint32_t l = blockIdx.x;
  const uint32_t c0 = t.layer_chunk_begin[l], c1 = t.layer_chunk_begin[l + 1];
  double a[4] = {0.0, 0.0, 0.0, 0.0}, b[4] = {0.0, 0.0, 0.0, 0.0};
  uint32_t c = c0 + threadIdx.x;
  for (; c + 3 * kFinalizeThreads < c1; c += 4 * kFinalizeThreads) {
    double2 p[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) p[k] = t.partials[c + k * kFinalizeThreads];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      a[k] += p[k].x;
      b[k] += p[k].y;
    }
  }
  // at most three partials remain for this thread
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (c < c1) {
      const double2 p = t.partials[c];
      a[k] += p.x;
      b[k] += p.y;
      c += kFinalizeThreads;
    }
  }
  double x = (a[0] + a[1]) + (a[2] + a[3]);
  double y = (b[0] + b[1]) + (b[2] + b[3]);
  block_sum2<kFinalizeThreads>(x, y);
  if (threadIdx.x == 0) {
    const double n = static_cast<double>(t.numel[l]);
    const double u = (x / n) / (y / n + t.eps_w);
    t.u[l] = u;
    t.delta[l] = (t.mode == 0) ? t.delta[l] + u : u;
  }
}

// ---- select: Eq. 3-5, reset, staleness stats, pack plan ------------------------
__global__ __launch_bounds__(kSelectThreads) void select_kernel(const DeviceTables t, int64_t step,
                                                                double lr_scale, int base_mode) {
  uint8_t* mask = reinterpret_cast<uint8_t*>(t.result + 1);
  const uint32_t N = t.n_layers;
  for (uint32_t l = threadIdx.x; l < N; l += kSelectThreads) {
    uint8_t code = 1;  // bit0 selected, bit1 selected by the staleness guard alone
    if (!base_mode) {
      const double K = t.k0[l] * lr_scale;
      const int64_t age = step - t.t_last[l];
      const bool by_drift = t.delta[l] >= K;
      const bool by_age = age >= t.s_max;
      code = static_cast<uint8_t>((by_drift || by_age) ? 1 : 0) |
             static_cast<uint8_t>((!by_drift && by_age) ? 2 : 0);
      if (code & 1) {
        t.delta[l] = 0.0;
        t.t_last[l] = step;
      }
    }
    mask[l] = code;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t ns = 0, nf = 0;
    uint64_t pay = 0, pieces = 0, num = 0, den = 0;
    int64_t max_age = 0;
    t.sel_rec_prefix[0] = 0;
    t.sel_piece_prefix[0] = 0;
    for (uint32_t l = 0; l < N; ++l) {
      const uint8_t code = mask[l];
      if (code & 1) {
        t.sel_layer[ns] = l;
        pay += t.rec_bytes[l];
        pieces += t.layer_pieces[l];
        ++ns;
        t.sel_rec_prefix[ns] = pay;
        t.sel_piece_prefix[ns] = pieces;
      }
      if (code & 2) ++nf;
      mask[l] = code & 1;
      const int64_t age = step - t.t_last[l];
      if (age > max_age) max_age = age;
      num += t.numel[l] * static_cast<uint64_t>(age);
      den += t.numel[l];
    }
    SelectHeader h;
    h.n_selected = ns;
    h.n_forced = nf;
    h.payload_bytes = pay;
    h.max_age = max_age;
    h.weighted_age = static_cast<double>(num) / static_cast<double>(den);
    h.total_pieces = pieces;
    h.age_numerator = num;
    h.reserved[0] = h.reserved[1] = 0;
    *t.result = h;
  }
}

// ---- byte movement of one piece ----------------------------------------------
// len is a multiple of 2; src/dst are at least 2-byte aligned; `vec` means
// src, dst and dst2 are 16-byte aligned.
__device__ __forceinline__ void copy_piece(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                           uint8_t* __restrict__ dst2, uint32_t len, bool vec) {
  const uint32_t tid = threadIdx.x;
  uint32_t done = 0;
  if (vec) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4* d4 = reinterpret_cast<u32x4*>(dst);
    u32x4* e4 = reinterpret_cast<u32x4*>(dst2);
    if (len == kPieceBytes) {
      constexpr uint32_t V = kPieceBytes / 16 / kCopyThreads;
      u32x4 v[V];
#pragma unroll
      for (uint32_t k = 0; k < V; ++k) v[k] = ld_nt(s4 + tid + k * kCopyThreads);
#pragma unroll
      for (uint32_t k = 0; k < V; ++k) st_nt(d4 + tid + k * kCopyThreads, v[k]);
      if (dst2) {
#pragma unroll
        for (uint32_t k = 0; k < V; ++k) st_nt(e4 + tid + k * kCopyThreads, v[k]);
      }
      return;
    }
    const uint32_t nv = len / 16;
    for (uint32_t i = tid; i < nv; i += kCopyThreads) {
      const u32x4 x = ld_nt(s4 + i);
      st_nt(d4 + i, x);
      if (dst2) st_nt(e4 + i, x);
    }
    done = nv * 16;
  }
  const uint16_t* s2 = reinterpret_cast<const uint16_t*>(src);
  uint16_t* d2 = reinterpret_cast<uint16_t*>(dst);
  uint16_t* f2 = reinterpret_cast<uint16_t*>(dst2);
  for (uint32_t i = done / 2 + tid; i < len / 2; i += kCopyThreads) {
    const uint16_t x = s2[i];
    d2[i] = x;
    if (dst2) f2[i] = x;
  }
}



// ---- pack: selected records into the staging buffer ---------------------------
// Work item q is piece q (relative to piece_base) of the selected records of
// ranks [first, last); records are written from staging offset
// sel_rec_prefix[first] - rec_base.
template <bool REFRESH>
__device__ __forceinline__ void pack_piece(const DeviceTables& t, uint32_t first, uint32_t last, uint64_t q,
                                           uint64_t rec_base, uint8_t* staging) {
  uint32_t lo = first, hi = last;  // sel_piece_prefix[lo] <= q < sel_piece_prefix[hi]
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (t.sel_piece_prefix[mid] <= q) lo = mid; else hi = mid;
  }
  const uint32_t l = t.sel_layer[lo];
  const uint64_t lp = q - t.sel_piece_prefix[lo];
  const CopyUnit u = t.units[t.piece_unit[t.layer_piece_begin[l] + lp]];
  const uint64_t off = (lp - u.piece0) * kPieceBytes;
  const uint64_t rem = u.bytes - off;
  const uint32_t len = rem < kPieceBytes ? static_cast<uint32_t>(rem) : kPieceBytes;
  uint8_t* dst = staging + (t.sel_rec_prefix[lo] - rec_base) + u.rec_off + off;
  const uint8_t* src = reinterpret_cast<const uint8_t*>(u.arr) + off;
  uint8_t* dst2 = (REFRESH && u.shadow) ? reinterpret_cast<uint8_t*>(u.shadow) + off : nullptr;
  copy_piece(src, dst, dst2, len, u.vec_ok != 0);
  if (off + len == u.bytes) {  // zero the block's padding
    const uint32_t pad = static_cast<uint32_t>(round_up(u.bytes, kRecordAlign) - u.bytes);
    uint16_t* z = reinterpret_cast<uint16_t*>(dst + len);
    for (uint32_t i = threadIdx.x; i < pad / 2; i += kCopyThreads) z[i] = 0;
  }
}

template <bool REFRESH, bool LOOP>
__global__ __launch_bounds__(kCopyThreads) void pack_kernel(const DeviceTables t, uint32_t first,
                                                            uint32_t last, uint64_t piece_base,
                                                            uint64_t n_pieces, uint64_t rec_base,
                                                            uint8_t* staging) {
  if constexpr (!LOOP) {
    pack_piece<REFRESH>(t, first, last, piece_base + remap_xcd(blockIdx.x, gridDim.x), rec_base, staging);
  } else {
    for (uint64_t base = 0; base < n_pieces; base += gridDim.x) {
      const uint64_t left = n_pieces - base;
      const uint32_t span = left < gridDim.x ? static_cast<uint32_t>(left) : gridDim.x;
      if (blockIdx.x >= span) return;
      pack_piece<REFRESH>(t, first, last, piece_base + base + remap_xcd(blockIdx.x, span), rec_base, staging);
    }
  }
}

// ---- unpack: composite restore from device-resident records --------------------
// rank r restores layer rank_layer[r] from the record at address rank_src[r];
// every W block also refreshes the shadow.
__device__ __forceinline__ void unpack_piece(const DeviceTables& t, uint32_t n_ranks, uint64_t q) {
  uint32_t lo = 0, hi = n_ranks;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (t.rank_piece_prefix[mid] <= q) lo = mid; else hi = mid;
  }
  const uint32_t l = t.rank_layer[lo];
  const uint64_t lp = q - t.rank_piece_prefix[lo];
  const CopyUnit u = t.units[t.piece_unit[t.layer_piece_begin[l] + lp]];
  const uint64_t off = (lp - u.piece0) * kPieceBytes;
  const uint64_t rem = u.bytes - off;
  const uint32_t len = rem < kPieceBytes ? static_cast<uint32_t>(rem) : kPieceBytes;
  const uint64_t rec = t.rank_src[lo];
  const uint8_t* src = reinterpret_cast<const uint8_t*>(rec) + u.rec_off + off;
  uint8_t* dst = reinterpret_cast<uint8_t*>(u.arr) + off;
  uint8_t* dst2 = u.shadow ? reinterpret_cast<uint8_t*>(u.shadow) + off : nullptr;
  copy_piece(src, dst, dst2, len, u.vec_ok != 0 && (rec & 15) == 0);
}

template <bool LOOP>
__global__ __launch_bounds__(kCopyThreads) void unpack_kernel(const DeviceTables t, uint32_t n_ranks,
                                                              uint64_t n_pieces) {
  if constexpr (!LOOP) {
    unpack_piece(t, n_ranks, remap_xcd(blockIdx.x, gridDim.x));
  } else {
    for (uint64_t base = 0; base < n_pieces; base += gridDim.x) {
      const uint64_t left = n_pieces - base;
      const uint32_t span = left < gridDim.x ? static_cast<uint32_t>(left) : gridDim.x;
      if (blockIdx.x >= span) return;
      unpack_piece(t, n_ranks, base + remap_xcd(blockIdx.x, span));
    }
  }
}

// ---- fused AdamW step + drift (Eq. 1-2 on the optimizer's parameters) -------
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) u32x2 g_u32x2;
__device__ __forceinline__ u32x2 ld_nt2(const u32x2* p) { return __builtin_nontemporal_load((const g_u32x2*)p); }
__device__ __forceinline__ void st_nt2(u32x2* p, u32x2 v) { __builtin_nontemporal_store(v, (g_u32x2*)p); }

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

// Four consecutive elements starting at element 4*gi (all arrays 4-element aligned).
template <int WDT, int GDT, bool MASTER>
struct Group4 {
  u32x4 p, m, v;
  float g[4];
  __device__ __forceinline__ void load(const OptSeg& sg, const GradSeg& gs, uint64_t gi) {
    if constexpr (MASTER) {
      p = ld_nt(reinterpret_cast<const u32x4*>(sg.master) + gi);
    } else if constexpr (WDT == 1) {
      const u32x2 w = ld_nt2(reinterpret_cast<const u32x2*>(sg.w) + gi);
      p = u32x4{w[0] << 16, w[0] & 0xffff0000u, w[1] << 16, w[1] & 0xffff0000u};
    } else {
      p = ld_nt(reinterpret_cast<const u32x4*>(sg.w) + gi);
    }
    m = ld_nt(reinterpret_cast<const u32x4*>(sg.m) + gi);
    v = ld_nt(reinterpret_cast<const u32x4*>(sg.v) + gi);
    if constexpr (GDT == 1) {
      const u32x2 x = ld_nt2(reinterpret_cast<const u32x2*>(gs.grad) + gi);
      g[0] = __uint_as_float(x[0] << 16); g[1] = __uint_as_float(x[0] & 0xffff0000u);
      g[2] = __uint_as_float(x[1] << 16); g[3] = __uint_as_float(x[1] & 0xffff0000u);
    } else {
      const u32x4 x = ld_nt(reinterpret_cast<const u32x4*>(gs.grad) + gi);
      for (int k = 0; k < 4; ++k) g[k] = __uint_as_float(x[k]);
    }
  }
  // update in place; returns the drift terms (sum|p_new - p|, sum|p|) of the group
  __device__ __forceinline__ void step_store(const OptSeg& sg, uint64_t gi, const AdamScalars& sc, bool decay,
                                             float& da, float& db) {
    float d[4], b[4];
    u32x4 pn, mn, vn;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float po = __uint_as_float(p[k]);
      float mm = __uint_as_float(m[k]), vv = __uint_as_float(v[k]);
      const float x = adamw_elem(po, mm, vv, g[k], sc, decay);
      pn[k] = __float_as_uint(x);
      mn[k] = __float_as_uint(mm);
      vn[k] = __float_as_uint(vv);
      d[k] = fabsf(x - po);
      b[k] = fabsf(po);
    }
    da = (d[0] + d[1]) + (d[2] + d[3]);
    db = (b[0] + b[1]) + (b[2] + b[3]);
    st_nt(reinterpret_cast<u32x4*>(sg.m) + gi, mn);
    st_nt(reinterpret_cast<u32x4*>(sg.v) + gi, vn);
    if constexpr (MASTER) st_nt(reinterpret_cast<u32x4*>(sg.master) + gi, pn);
    if constexpr (WDT == 1) {
      const uint32_t lo = bf16_rne(__uint_as_float(pn[0])) | (static_cast<uint32_t>(bf16_rne(__uint_as_float(pn[1]))) << 16);
      const uint32_t hi = bf16_rne(__uint_as_float(pn[2])) | (static_cast<uint32_t>(bf16_rne(__uint_as_float(pn[3]))) << 16);
      st_nt2(reinterpret_cast<u32x2*>(sg.w) + gi, u32x2{lo, hi});
    } else {
      st_nt(reinterpret_cast<u32x4*>(sg.w) + gi, pn);
    }
  }
};

template <int WDT, int GDT, bool MASTER>
__device__ __forceinline__ void adamw_chunk(const DeviceTables& t, const AdamScalars& sc, uint32_t c) {
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
      Group4<WDT, GDT, MASTER> grp[GPT];
#pragma unroll
      for (uint32_t k = 0; k < GPT; ++k) grp[k].load(sg, gs, g0 + tid + k * kScoreThreads);
#pragma unroll
      for (uint32_t k = 0; k < GPT; ++k) {
        float da, db;
        grp[k].step_store(sg, g0 + tid + k * kScoreThreads, sc, decay, da, db);
        a += static_cast<double>(da);
        b += static_cast<double>(db);
      }
    } else {
      for (uint32_t i = tid; i < ng; i += kScoreThreads) {
        Group4<WDT, GDT, MASTER> grp;
        grp.load(sg, gs, g0 + i);
        float da, db;
        grp.step_store(sg, g0 + i, sc, decay, da, db);
        a += static_cast<double>(da);
        b += static_cast<double>(db);
      }
    }
    scalar_from = ng * 4;
  }
  const uint8_t* wb = reinterpret_cast<const uint8_t*>(sg.w);
  for (uint32_t i = scalar_from + tid; i < n; i += kScoreThreads) {
    const uint64_t e = e0 + i;
    float* mp = reinterpret_cast<float*>(sg.m) + e;
    float* vp = reinterpret_cast<float*>(sg.v) + e;
    const float po = MASTER ? reinterpret_cast<const float*>(sg.master)[e] : w_load<WDT>(wb, e);
    float mm = *mp, vv = *vp;
    const float x = adamw_elem(po, mm, vv, g_load<GDT>(reinterpret_cast<const uint8_t*>(gs.grad), e), sc, decay);
    *mp = mm;
    *vp = vv;
    if constexpr (MASTER) reinterpret_cast<float*>(sg.master)[e] = x;
    w_store<WDT>(reinterpret_cast<uint8_t*>(sg.w), e, x);
    a += static_cast<double>(fabsf(x - po));
    b += static_cast<double>(fabsf(po));
  }
  block_sum2<kScoreThreads>(a, b);
  if (tid == 0) t.partials[c] = make_double2(a, b);
}

template <int WDT, int GDT, bool MASTER, bool LOOP>
__global__ __launch_bounds__(kScoreThreads) void adamw_kernel(const DeviceTables t, const AdamScalars sc) {
  if constexpr (!LOOP) {
    adamw_chunk<WDT, GDT, MASTER>(t, sc, remap_xcd(blockIdx.x, gridDim.x));
  } else {
    for (uint64_t base = 0; base < t.n_chunks; base += gridDim.x) {
      const uint64_t left = t.n_chunks - base;
      const uint32_t span = left < gridDim.x ? static_cast<uint32_t>(left) : gridDim.x;
      if (blockIdx.x >= span) return;
      adamw_chunk<WDT, GDT, MASTER>(t, sc, static_cast<uint32_t>(base + remap_xcd(blockIdx.x, span)));
      __syncthreads();
    }
  }
}

// Blocks per launch: one per work item up to the dispatch limit of 2^32
// work-items per dimension; beyond it the kernels loop.
__host__ inline uint32_t grid_for(uint64_t items, uint32_t threads) {
  uint64_t cap = (0xFFFFFFFFull / threads) & ~7ull;
  if (LC_MAX_GRID_BLOCKS > 0 && cap > LC_MAX_GRID_BLOCKS) cap = LC_MAX_GRID_BLOCKS;
  return static_cast<uint32_t>(items < cap ? items : cap);
}

template <int DT, bool ACCUM>
void launch_score_t(const DeviceTables& t, hipStream_t st) {
  const uint32_t g = grid_for(t.n_chunks, kScoreThreads);
  if (g == t.n_chunks)
    hipLaunchKernelGGL((score_kernel<DT, ACCUM, false>), dim3(g), dim3(kScoreThreads), 0, st, t);
  else
    hipLaunchKernelGGL((score_kernel<DT, ACCUM, true>), dim3(g), dim3(kScoreThreads), 0, st, t);
}

template <bool REFRESH>
void launch_pack_t(const DeviceTables& t, uint32_t first, uint32_t last, uint64_t piece_base, uint64_t n_pieces,
                   uint64_t rec_base, uint8_t* stg, hipStream_t st) {
  const uint32_t g = grid_for(n_pieces, kCopyThreads);
  if (g == n_pieces)
    hipLaunchKernelGGL((pack_kernel<REFRESH, false>), dim3(g), dim3(kCopyThreads), 0, st, t, first, last,
                       piece_base, n_pieces, rec_base, stg);
  else
    hipLaunchKernelGGL((pack_kernel<REFRESH, true>), dim3(g), dim3(kCopyThreads), 0, st, t, first, last,
                       piece_base, n_pieces, rec_base, stg);
}

}  // namespace

hipError_t launch_score(const DeviceTables& t, hipStream_t st) {
  if (t.dtype == 1) {
    if (t.mode == 0) launch_score_t<1, true>(t, st);
    else launch_score_t<1, false>(t, st);
  } else {
    if (t.mode == 0) launch_score_t<2, true>(t, st);
    else launch_score_t<2, false>(t, st);
  }
  hipLaunchKernelGGL(finalize_kernel, dim3(t.n_layers), dim3(kFinalizeThreads), 0, st, t);
  return hipGetLastError();
}

hipError_t launch_select(const DeviceTables& t, int64_t step, double lr_scale, int base_mode,
                         hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kSelectThreads), 0, st, t, step, lr_scale, base_mode);
  return hipGetLastError();
}

hipError_t launch_pack(const DeviceTables& t, uint32_t first_rank, uint32_t last_rank,
                       uint64_t piece_base, uint64_t n_pieces, uint64_t rec_base, void* staging,
                       int refresh_shadow, hipStream_t st) {
  uint8_t* stg = static_cast<uint8_t*>(staging);
  if (refresh_shadow) launch_pack_t<true>(t, first_rank, last_rank, piece_base, n_pieces, rec_base, stg, st);
  else launch_pack_t<false>(t, first_rank, last_rank, piece_base, n_pieces, rec_base, stg, st);
  return hipGetLastError();
}

template <int WDT, int GDT, bool MASTER>
void launch_adamw_t(const DeviceTables& t, const AdamScalars& sc, hipStream_t st) {
  const uint32_t g = grid_for(t.n_chunks, kScoreThreads);
  if (g == t.n_chunks)
    hipLaunchKernelGGL((adamw_kernel<WDT, GDT, MASTER, false>), dim3(g), dim3(kScoreThreads), 0, st, t, sc);
  else
    hipLaunchKernelGGL((adamw_kernel<WDT, GDT, MASTER, true>), dim3(g), dim3(kScoreThreads), 0, st, t, sc);
}

hipError_t launch_adamw(const DeviceTables& t, int grad_dtype, int has_master, const AdamScalars& sc,
                        hipStream_t st) {
  const bool gb = grad_dtype == 1;
  if (t.dtype == 1) {
    if (has_master) { if (gb) launch_adamw_t<1, 1, true>(t, sc, st); else launch_adamw_t<1, 2, true>(t, sc, st); }
    else { if (gb) launch_adamw_t<1, 1, false>(t, sc, st); else launch_adamw_t<1, 2, false>(t, sc, st); }
  } else {
    if (has_master) { if (gb) launch_adamw_t<2, 1, true>(t, sc, st); else launch_adamw_t<2, 2, true>(t, sc, st); }
    else { if (gb) launch_adamw_t<2, 1, false>(t, sc, st); else launch_adamw_t<2, 2, false>(t, sc, st); }
  }
  hipLaunchKernelGGL(finalize_kernel, dim3(t.n_layers), dim3(kFinalizeThreads), 0, st, t);
  return hipGetLastError();
}

hipError_t launch_unpack(const DeviceTables& t, uint32_t n_ranks, uint64_t n_pieces, hipStream_t st) {
  const uint32_t g = grid_for(n_pieces, kCopyThreads);
  if (g == n_pieces)
    hipLaunchKernelGGL(unpack_kernel<false>, dim3(g), dim3(kCopyThreads), 0, st, t, n_ranks, n_pieces);
  else
    hipLaunchKernelGGL(unpack_kernel<true>, dim3(g), dim3(kCopyThreads), 0, st, t, n_ranks, n_pieces);
  return hipGetLastError();
}

}  // namespace lc
