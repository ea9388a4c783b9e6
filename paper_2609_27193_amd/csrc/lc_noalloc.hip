// lc_score_layers_static: Eq. 1 for every layer of a list of segments, with
// no context and no device allocation, for callers that cannot allocate
// device memory.  The device tables the score and finalize kernels need (the
// segment table, the chunk -> segment table, one fp64 pair per chunk and the
// per-layer counts) live in one file-scope device array of fixed size; a
// layout whose tables do not fit is scored in consecutive batches of whole
// layers, each batch reusing the array after the previous batch's kernels
// (stream order).  Same kernels, same chunking and the same fixed-order
// per-layer sum as lc_score_layers, so u is bit-identical to the u that
// lc_score_layers computes for the same weights and shadow.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "layercheck.h"
#include "lc_ctx.h"
#include "lc_internal.h"
#include "lc_trace.h"

#ifndef LC_NOALLOC_SCRATCH_BYTES
#define LC_NOALLOC_SCRATCH_BYTES (16u << 20)
#endif

// The allocation-free path's device memory, one copy per GPU for the life of
// the process.  Host code never uses this name as an address: it is a
// host-side stand-in there.  Each device's address comes from
// hipGetSymbolAddress (scratch_base below).  Nothing in it has to start at
// zero: every call uploads or writes every table entry its kernels read
// (segment table, per-layer counts, chunk table, one partial per chunk)
// before they read it, whatever an earlier call left there.
static __device__ __align__(256) uint8_t scratch[LC_NOALLOC_SCRATCH_BYTES];

using namespace lc;

namespace {

constexpr uint64_t kScratchBytes = LC_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch regions are 256-byte aligned");
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

uint64_t align256(uint64_t x) { return (x + 255) / 256 * 256; }

// Scratch layout of one batch of ns segments, nc chunks and nl layers.
struct Regions {
  uint64_t segs, chunk_seg, lcb, numel, partials, delta, end;
};

Regions regions(uint64_t ns, uint64_t nc, uint64_t nl) {
  Regions r;
  r.segs = 0;
  r.chunk_seg = r.segs + align256(ns * sizeof(ScoreSeg));
  r.lcb = r.chunk_seg + align256(nc * sizeof(uint32_t));
  r.numel = r.lcb + align256((nl + 1) * sizeof(uint32_t));
  r.partials = r.numel + align256(nl * sizeof(uint64_t));
  r.delta = r.partials + align256(nc * sizeof(double2));
  r.end = r.delta + align256(nl * sizeof(double));
  return r;
}

// The device address of `scratch` on device `dev` (the current device),
// looked up once per device.
lc_status scratch_base(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(LC_ERR_INVALID_ARG, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(LC_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = p;
  }
  *out = static_cast<uint8_t*>(g_scratch_ptr[dev]);
  return LC_OK;
}

// chunk -> segment table of one batch, built on the device from the segment
// table: block i writes i over segment i's chunk range.
__global__ __launch_bounds__(256) void chunk_table_kernel(const ScoreSeg* segs, uint32_t* chunk_seg,
                                                          uint32_t n_chunks) {
  const uint32_t i = blockIdx.x;
  const uint32_t c0 = segs[i].chunk_begin;
  const uint32_t c1 = i + 1 < gridDim.x ? segs[i + 1].chunk_begin : n_chunks;
  for (uint32_t c = c0 + threadIdx.x; c < c1; c += 256) chunk_seg[c] = i;
}

// One batch: segments [s0, s1) holding layers [l0, l1).
struct Batch {
  uint32_t s0, s1, l0, l1;
  uint64_t chunks;
  std::vector<ScoreSeg> segs;
  std::vector<uint32_t> lcb;
  std::vector<uint64_t> numel;
};

// Host tables feed asynchronous copies: wait for the stream before they go,
// also on an early error return.
struct DrainOnExit {
  hipStream_t st;
  bool armed = false;
  ~DrainOnExit() {
    if (armed) (void)hipStreamSynchronize(st);
  }
};

}  // namespace

extern "C" lc_status lc_score_layers_static(const lc_segment* segments, uint32_t n_segments, uint32_t n_layers,
                                            int32_t weight_dtype, double eps_w, double* u_out, void* stream) {
  lc::TraceRange trace_("lc_score_layers_static");
  // ---- arguments and sizes (host only: nothing below touches the GPU) --------
  if (!segments) return fail(LC_ERR_INVALID_ARG, "segments is NULL");
  if (!u_out) return fail(LC_ERR_INVALID_ARG, "u_out is NULL");
  if (n_layers == 0) return fail(LC_ERR_INVALID_ARG, "n_layers must be >= 1");
  if (n_segments < n_layers) return fail(LC_ERR_INVALID_ARG, "n_segments < n_layers");
  if (weight_dtype != LC_DT_BF16 && weight_dtype != LC_DT_F32)
    return fail(LC_ERR_INVALID_ARG, "unknown weight dtype %d", weight_dtype);
  if (!(eps_w >= 0.0) || !std::isfinite(eps_w)) return fail(LC_ERR_INVALID_ARG, "eps_w must be finite and >= 0");
  if (reinterpret_cast<uintptr_t>(u_out) % alignof(double)) return fail(LC_ERR_INVALID_ARG, "u_out is misaligned");
  const uint32_t esz = weight_dtype == LC_DT_BF16 ? 2 : 4;
  const uint64_t ce = kChunkBytes / esz;
  std::vector<uint32_t> seg_begin(n_layers + 1, 0);
  std::vector<uint64_t> layer_chunks(n_layers, 0);
  int64_t prev = -1;
  for (uint32_t i = 0; i < n_segments; ++i) {
    const lc_segment& s = segments[i];
    if (s.layer >= n_layers) return fail(LC_ERR_INVALID_ARG, "segment %u: layer %u out of range", i, s.layer);
    if (static_cast<int64_t>(s.layer) < prev)
      return fail(LC_ERR_INVALID_ARG, "segment %u: segments must be grouped by ascending layer", i);
    if (static_cast<int64_t>(s.layer) > prev + 1)
      return fail(LC_ERR_INVALID_ARG, "layer %lld has no segment", static_cast<long long>(prev + 1));
    if (s.reserved != 0) return fail(LC_ERR_INVALID_ARG, "segment %u: reserved field must be 0", i);
    if (s.numel == 0) return fail(LC_ERR_INVALID_ARG, "segment %u: numel is 0", i);
    if (s.numel > (1ull << 46)) return fail(LC_ERR_INVALID_ARG, "segment %u: numel too large", i);
    if (!s.weight || !s.shadow) return fail(LC_ERR_INVALID_ARG, "segment %u: NULL weight or shadow", i);
    if (reinterpret_cast<uintptr_t>(s.weight) % esz || reinterpret_cast<uintptr_t>(s.shadow) % esz)
      return fail(LC_ERR_INVALID_ARG, "segment %u: misaligned pointer", i);
    if (static_cast<int64_t>(s.layer) != prev) seg_begin[s.layer] = i;
    prev = s.layer;
    layer_chunks[s.layer] += (s.numel + ce - 1) / ce;
  }
  if (prev != static_cast<int64_t>(n_layers) - 1)
    return fail(LC_ERR_INVALID_ARG, "layer %lld has no segment", static_cast<long long>(prev + 1));
  seg_begin[n_layers] = n_segments;
  // batches of whole layers whose tables fit the scratch array
  std::vector<Batch> batches;
  for (uint32_t l = 0; l < n_layers;) {
    Batch b;
    b.l0 = l;
    b.s0 = seg_begin[l];
    b.chunks = 0;
    while (l < n_layers) {
      const uint64_t ns = seg_begin[l + 1] - b.s0, nc = b.chunks + layer_chunks[l], nl = l + 1 - b.l0;
      if (regions(ns, nc, nl).end > kScratchBytes) break;
      b.chunks = nc;
      ++l;
    }
    if (l == b.l0)
      return fail(LC_ERR_CAPACITY,
                  "layer %u needs %llu bytes of tables, more than the %llu-byte array of the allocation-free path",
                  l, static_cast<unsigned long long>(regions(seg_begin[l + 1] - seg_begin[l], layer_chunks[l], 1).end),
                  static_cast<unsigned long long>(kScratchBytes));
    b.l1 = l;
    b.s1 = seg_begin[l];
    batches.push_back(std::move(b));
  }

  // ---- device checks -------------------------------------------------------------
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(LC_ERR_HIP, "no HIP device");
  }
  if (st) {
    int sdev = -1;
    if (hipStreamGetDevice(st, &sdev) != hipSuccess) {
      (void)hipGetLastError();
      return fail(LC_ERR_INVALID_ARG, "stream is not a HIP stream");
    }
    if (sdev != dev) return fail(LC_ERR_INVALID_ARG, "the stream belongs to device %d, not the current %d", sdev, dev);
  }
  for (uint32_t i = 0; i < n_segments; ++i) {
    const lc_segment& s = segments[i];
    if (!device_range_ok(s.weight, s.numel * esz) || !device_range_ok(s.shadow, s.numel * esz))
      return fail(LC_ERR_INVALID_ARG, "segment %u: weight or shadow is not device memory of %llu elements", i,
                  static_cast<unsigned long long>(s.numel));
  }
  if (!device_range_ok(u_out, n_layers * sizeof(double)))
    return fail(LC_ERR_INVALID_ARG, "u_out is not device memory of %u doubles", n_layers);
  uint8_t* base = nullptr;
  lc_status status = scratch_base(dev, &base);
  if (status != LC_OK) return status;

  // ---- tables and kernels, one batch after the other on the caller's stream --------
  for (Batch& b : batches) {
    uint32_t c = 0;
    for (uint32_t i = b.s0; i < b.s1; ++i) {
      const lc_segment& s = segments[i];
      ScoreSeg ss;
      ss.w = reinterpret_cast<uint64_t>(s.weight);
      ss.s = reinterpret_cast<uint64_t>(s.shadow);
      ss.numel = s.numel;
      ss.chunk_begin = c;
      ss.vec_ok = (ss.w % 16 == 0 && ss.s % 16 == 0) ? 1u : 0u;
      c += static_cast<uint32_t>((s.numel + ce - 1) / ce);
      b.segs.push_back(ss);
    }
    b.lcb.assign(1, 0);
    for (uint32_t l = b.l0; l < b.l1; ++l) {
      b.lcb.push_back(b.lcb.back() + static_cast<uint32_t>(layer_chunks[l]));
      uint64_t n = 0;
      for (uint32_t i = seg_begin[l]; i < seg_begin[l + 1]; ++i) n += segments[i].numel;
      b.numel.push_back(n);
    }
  }
  DrainOnExit drain{st};
  for (const Batch& b : batches) {
    const uint32_t ns = b.s1 - b.s0, nl = b.l1 - b.l0;
    const Regions r = regions(ns, b.chunks, nl);
    DeviceTables t{};
    t.n_layers = nl;
    t.n_chunks = static_cast<uint32_t>(b.chunks);
    t.dtype = weight_dtype;
    t.mode = LC_MODE_SNAPSHOT;  // u only: no shadow write, Delta_l = u_l into scratch
    t.eps_w = eps_w;
    t.s_max = 1;
    t.segs = reinterpret_cast<const ScoreSeg*>(base + r.segs);
    t.chunk_seg = reinterpret_cast<const uint32_t*>(base + r.chunk_seg);
    t.layer_chunk_begin = reinterpret_cast<const uint32_t*>(base + r.lcb);
    t.numel = reinterpret_cast<const uint64_t*>(base + r.numel);
    t.partials = reinterpret_cast<double2*>(base + r.partials);
    t.delta = reinterpret_cast<double*>(base + r.delta);
    t.u = u_out + b.l0;
    drain.armed = true;
    hipError_t e = hipMemcpyAsync(base + r.segs, b.segs.data(), ns * sizeof(ScoreSeg), hipMemcpyHostToDevice, st);
    if (e == hipSuccess)
      e = hipMemcpyAsync(base + r.lcb, b.lcb.data(), b.lcb.size() * sizeof(uint32_t), hipMemcpyHostToDevice, st);
    if (e == hipSuccess)
      e = hipMemcpyAsync(base + r.numel, b.numel.data(), nl * sizeof(uint64_t), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) {
      hipLaunchKernelGGL(chunk_table_kernel, dim3(ns), dim3(256), 0, st, t.segs,
                         reinterpret_cast<uint32_t*>(base + r.chunk_seg), t.n_chunks);
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = launch_score(t, st);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(LC_ERR_HIP, "lc_score_layers_static: %s", hipGetErrorString(e));
    }
  }
  drain.armed = false;
  const hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(LC_ERR_HIP, "lc_score_layers_static: %s", hipGetErrorString(e));
  }
  return LC_OK;
}
