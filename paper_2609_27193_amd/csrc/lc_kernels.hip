// HIP kernels of the LayerCheck decision step for gfx950 (MI355X, CDNA4).
//
// Every kernel here is HBM-bound streaming work or a tiny O(N) step; nothing
// is a dense contraction, so there is no MFMA.  Design rules:
//  * 16-byte (dwordx4) coalesced loads/stores, several in flight per lane;
//    non-temporal, device-scope cache policy because every byte is touched
//    once per step and the per-step stream (tens of GB) dwarfs the 256 MB
//    Infinity Cache; full chunks and pieces go through buffer resources;
//  * reductions use no floating-point atomics: one fp64 pair per chunk, then a
//    fixed-order per-layer sum, so scores are bitwise reproducible;
//  * wave64 reductions (DPP quad permutes, then cross-row shuffles), LDS for
//    the cross-wave combine.
#include "lc_device.h"

#include <atomic>

namespace lc {
namespace {

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
    if (n == CE) {
      const tile_t tw = make_tile(wb, kChunkBytes), ts = make_tile(sbp, kChunkBytes);
#pragma unroll
      for (uint32_t r = 0; r < VPT / U; ++r) {
        u32x4 w[U], s[U];
#pragma unroll
        for (uint32_t k = 0; k < U; ++k) {
          const uint32_t off = (tid + (r * U + k) * kScoreThreads) * 16u;
          w[k] = ld_tile(tw, off);
          s[k] = ld_tile(ts, off);
        }
#pragma unroll
        for (uint32_t k = 0; k < U; ++k) {
          float da, db;
          vec_terms<DT>(w[k], s[k], da, db);
          a += static_cast<double>(da);
          b += static_cast<double>(db);
          if constexpr (ACCUM) st_tile(ts, (tid + (r * U + k) * kScoreThreads) * 16u, w[k]);
        }
      }
      scalar_from = n;
    } else {
      const u32x4* wv = reinterpret_cast<const u32x4*>(wb);
      u32x4* sv = reinterpret_cast<u32x4*>(sbp);
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

// One chunk per block: the chunk's tables are read before any store, so they
// stay on the scalar path.  A layout with more chunks than one dispatch takes
// (2^32 work-items) is scored by consecutive launches, each over the next
// range of chunks starting at chunk_base.
template <int DT, bool ACCUM>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(const DeviceTables t, uint32_t chunk_base) {
  score_chunk<DT, ACCUM>(t, chunk_base + remap_xcd(blockIdx.x, gridDim.x));
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
                                                                double lr_scale, int base_mode, uint64_t seq) {
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
    h.seq = 0;
    h.reserved = 0;
    *t.result = h;
    // The host's copy, read with no device-to-host copy and no stream
    // synchronisation: the mask, then the header with seq = 0, then -- once a
    // system-scope fence has made those visible -- the number the host waits
    // for.
    SelectHeader* hr = t.host_result;
    const uint32_t* m32 = reinterpret_cast<const uint32_t*>(mask);
    uint32_t* h32 = reinterpret_cast<uint32_t*>(hr + 1);
    for (uint32_t w = 0; w < N / 4; ++w) h32[w] = m32[w];
    uint8_t* h8 = reinterpret_cast<uint8_t*>(hr + 1);
    for (uint32_t l = N & ~3u; l < N; ++l) h8[l] = mask[l];
    *hr = h;
    __threadfence_system();
    hr->seq = seq;
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
    if (len == kPieceBytes) {
      constexpr uint32_t V = kPieceBytes / 16 / kCopyThreads;
      const tile_t ts = make_tile(src, kPieceBytes), td = make_tile(dst, kPieceBytes);
      u32x4 v[V];
#pragma unroll
      for (uint32_t k = 0; k < V; ++k) v[k] = ld_tile(ts, (tid + k * kCopyThreads) * 16u);
#pragma unroll
      for (uint32_t k = 0; k < V; ++k) st_tile(td, (tid + k * kCopyThreads) * 16u, v[k]);
      if (dst2) {
        const tile_t te = make_tile(dst2, kPieceBytes);
#pragma unroll
        for (uint32_t k = 0; k < V; ++k) st_tile(te, (tid + k * kCopyThreads) * 16u, v[k]);
      }
      return;
    }
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4* d4 = reinterpret_cast<u32x4*>(dst);
    u32x4* e4 = reinterpret_cast<u32x4*>(dst2);
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

// One piece per block; piece_base is the first piece of this launch (a pack
// with more pieces than one dispatch takes is split into consecutive launches).
template <bool REFRESH>
__global__ __launch_bounds__(kCopyThreads) void pack_kernel(const DeviceTables t, uint32_t first,
                                                            uint32_t last, uint64_t piece_base,
                                                            uint64_t rec_base, uint8_t* staging) {
  pack_piece<REFRESH>(t, first, last, piece_base + remap_xcd(blockIdx.x, gridDim.x), rec_base, staging);
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

// One piece per block, from piece_base on (split like the pack).
__global__ __launch_bounds__(kCopyThreads) void unpack_kernel(const DeviceTables t, uint32_t n_ranks,
                                                              uint64_t piece_base) {
  unpack_piece(t, n_ranks, piece_base + remap_xcd(blockIdx.x, gridDim.x));
}

// Each launch takes the largest grid one dispatch allows (grid_for) and the
// next range of work items; every block does exactly one item.
template <int DT, bool ACCUM>
void launch_score_t(const DeviceTables& t, hipStream_t st) {
  const uint32_t lds = occupancy_lds(ACCUM ? LC_SCORE_ACCUM_BLOCKS_PER_CU : LC_SCORE_SNAPSHOT_BLOCKS_PER_CU);
  for (uint64_t done = 0; done < t.n_chunks;) {
    const uint32_t g = grid_for(t.n_chunks - done, kScoreThreads);
    hipLaunchKernelGGL((score_kernel<DT, ACCUM>), dim3(g), dim3(kScoreThreads), lds, st, t,
                       static_cast<uint32_t>(done));
    done += g;
  }
}

template <bool REFRESH>
void launch_pack_t(const DeviceTables& t, uint32_t first, uint32_t last, uint64_t piece_base, uint64_t n_pieces,
                   uint64_t rec_base, uint8_t* stg, hipStream_t st) {
  const uint32_t lds = occupancy_lds(LC_COPY_BLOCKS_PER_CU);
  for (uint64_t done = 0; done < n_pieces;) {
    const uint32_t g = grid_for(n_pieces - done, kCopyThreads);
    hipLaunchKernelGGL((pack_kernel<REFRESH>), dim3(g), dim3(kCopyThreads), lds, st, t, first, last,
                       piece_base + done, rec_base, stg);
    done += g;
  }
}

}  // namespace

// A CU holds L bytes of LDS; a block that asks for more than L / (k + 1)
// leaves room for at most k blocks.  The reservation asks for 2 KiB more than
// that (rounded to 512 B) so the kernel's own few bytes of static LDS cannot
// push it past L / k.  Queried once per device.
uint32_t occupancy_lds(uint32_t blocks_per_cu) {
  if (blocks_per_cu == 0) return 0;
  constexpr int kMaxDevices = 64;
  static std::atomic<int64_t> lds_cu[kMaxDevices], lds_block[kMaxDevices];  // 0: not queried yet
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  if (lds_cu[dev].load(std::memory_order_relaxed) == 0) {
    int cu = 0, blk = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) != hipSuccess ||
        hipDeviceGetAttribute(&blk, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    lds_block[dev].store(blk, std::memory_order_relaxed);
    lds_cu[dev].store(cu > 0 ? cu : -1, std::memory_order_relaxed);
  }
  const int64_t cu = lds_cu[dev].load(std::memory_order_relaxed);
  const int64_t blk = lds_block[dev].load(std::memory_order_relaxed);
  if (cu <= 0) return 0;
  const int64_t k = blocks_per_cu;
  const int64_t want = (cu / (k + 1) + 2048 + 511) / 512 * 512;
  if (want > cu / k - 1024 || want > blk) return 0;
  return static_cast<uint32_t>(want);
}

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

hipError_t launch_finalize(const DeviceTables& t, hipStream_t st) {
  hipLaunchKernelGGL(finalize_kernel, dim3(t.n_layers), dim3(kFinalizeThreads), 0, st, t);
  return hipGetLastError();
}

hipError_t launch_select(const DeviceTables& t, int64_t step, double lr_scale, int base_mode, uint64_t seq,
                         hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kSelectThreads), 0, st, t, step, lr_scale, base_mode, seq);
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

hipError_t launch_unpack(const DeviceTables& t, uint32_t n_ranks, uint64_t n_pieces, hipStream_t st) {
  const uint32_t lds = occupancy_lds(LC_COPY_BLOCKS_PER_CU);
  for (uint64_t done = 0; done < n_pieces;) {
    const uint32_t g = grid_for(n_pieces - done, kCopyThreads);
    hipLaunchKernelGGL(unpack_kernel, dim3(g), dim3(kCopyThreads), lds, st, t, n_ranks, done);
    done += g;
  }
  return hipGetLastError();
}

}  // namespace lc
