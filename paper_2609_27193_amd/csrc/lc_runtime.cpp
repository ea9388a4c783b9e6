// Host runtime of the LayerCheck HIP library: validation, layer-aligned
// tables, the call-order state machine and kernel launches behind the C
// interface declared in include/layercheck.h.
#include <dlfcn.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <vector>

#include "layercheck.h"
#include "lc_ctx.h"
#include "lc_internal.h"
#include "lc_trace.h"

using namespace lc;

thread_local std::string lc::g_error;

namespace {

uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

lc_status build_layout(const lc_layout_desc* d, HostLayout& L) {
  if (!d) return fail(LC_ERR_INVALID_ARG, "descriptor is NULL");
  if (d->n_layers == 0) return fail(LC_ERR_INVALID_ARG, "n_layers must be >= 1");
  if (d->n_segments < d->n_layers) return fail(LC_ERR_INVALID_ARG, "n_segments < n_layers");
  if (!d->segments) return fail(LC_ERR_INVALID_ARG, "segments is NULL");
  if (d->weight_dtype != LC_DT_BF16 && d->weight_dtype != LC_DT_F32)
    return fail(LC_ERR_INVALID_ARG, "unknown weight dtype %d", d->weight_dtype);
  if (d->has_master != 0 && d->has_master != 1) return fail(LC_ERR_INVALID_ARG, "has_master must be 0 or 1");
  if (d->mode != LC_MODE_ACCUM && d->mode != LC_MODE_SNAPSHOT)
    return fail(LC_ERR_INVALID_ARG, "unknown mode %d", d->mode);
  if (d->reserved != 0) return fail(LC_ERR_INVALID_ARG, "reserved field must be 0");
  if (!d->k0) return fail(LC_ERR_INVALID_ARG, "k0 is NULL");
  for (uint32_t l = 0; l < d->n_layers; ++l)
    if (!(d->k0[l] >= 0.0)) return fail(LC_ERR_INVALID_ARG, "k0[%u] must be >= 0", l);
  if (d->s_max < 1) return fail(LC_ERR_INVALID_ARG, "s_max must be >= 1");
  if (!(d->eps_w >= 0.0) || !std::isfinite(d->eps_w)) return fail(LC_ERR_INVALID_ARG, "eps_w must be finite and >= 0");

  const uint32_t N = d->n_layers;
  L.N = N;
  L.dtype = d->weight_dtype;
  L.esz = d->weight_dtype == LC_DT_BF16 ? 2 : 4;
  L.has_master = d->has_master != 0;
  L.segs.assign(d->segments, d->segments + d->n_segments);
  L.layer_seg_begin.assign(N + 1, 0);
  L.numel.assign(N, 0);
  int64_t prev = -1;
  L.has_shadow = d->segments[0].shadow != nullptr;
  L.has_moments = d->segments[0].exp_avg != nullptr;
  if (!L.has_shadow && d->mode != LC_MODE_ACCUM)
    return fail(LC_ERR_INVALID_ARG, "a layout without shadow copies needs LC_MODE_ACCUM");
  for (uint32_t i = 0; i < d->n_segments; ++i) {
    const lc_segment& s = L.segs[i];
    if (s.layer >= N) return fail(LC_ERR_INVALID_ARG, "segment %u: layer %u out of range", i, s.layer);
    if (static_cast<int64_t>(s.layer) < prev)
      return fail(LC_ERR_INVALID_ARG, "segment %u: segments must be grouped by ascending layer", i);
    if (static_cast<int64_t>(s.layer) > prev + 1)
      return fail(LC_ERR_INVALID_ARG, "layer %lld has no segment", static_cast<long long>(prev + 1));
    if (s.reserved != 0) return fail(LC_ERR_INVALID_ARG, "segment %u: reserved field must be 0", i);
    if (s.numel == 0) return fail(LC_ERR_INVALID_ARG, "segment %u: numel is 0", i);
    if (s.numel > (1ull << 46)) return fail(LC_ERR_INVALID_ARG, "segment %u: numel too large", i);
    if (!s.weight) return fail(LC_ERR_INVALID_ARG, "segment %u: NULL weight pointer", i);
    if ((s.exp_avg != nullptr) != L.has_moments || (s.exp_avg_sq != nullptr) != L.has_moments)
      return fail(LC_ERR_INVALID_ARG, "segment %u: Adam moments must be given for every segment or for none", i);
    if ((s.shadow != nullptr) != L.has_shadow)
      return fail(LC_ERR_INVALID_ARG, "segment %u: shadow must be given for every segment or for none", i);
    if ((s.master != nullptr) != L.has_master)
      return fail(LC_ERR_INVALID_ARG, "segment %u: master must be %s", i, L.has_master ? "non-NULL" : "NULL");
    const uintptr_t wa = reinterpret_cast<uintptr_t>(s.weight), sa = reinterpret_cast<uintptr_t>(s.shadow);
    if (wa % L.esz || sa % L.esz || reinterpret_cast<uintptr_t>(s.exp_avg) % 4 ||
        reinterpret_cast<uintptr_t>(s.exp_avg_sq) % 4 || reinterpret_cast<uintptr_t>(s.master) % 4)
      return fail(LC_ERR_INVALID_ARG, "segment %u: misaligned pointer", i);
    if (L.has_shadow && s.weight == s.shadow)
      return fail(LC_ERR_INVALID_ARG, "segment %u: weight and shadow alias", i);
    if (static_cast<int64_t>(s.layer) != prev) L.layer_seg_begin[s.layer] = i;
    prev = s.layer;
    L.numel[s.layer] += s.numel;
    if (L.numel[s.layer] > (1ull << 52)) return fail(LC_ERR_INVALID_ARG, "layer %u: too many elements", s.layer);
  }
  if (prev != static_cast<int64_t>(N) - 1)
    return fail(LC_ERR_INVALID_ARG, "layer %lld has no segment", static_cast<long long>(prev + 1));
  // The library writes every array (the shadow on each score, all of them on
  // a restore or an optimizer step), so no two may share a byte.
  {
    struct Span { uint64_t b, e; uint32_t seg; };
    std::vector<Span> spans;
    spans.reserve(5ull * d->n_segments);
    for (uint32_t i = 0; i < d->n_segments; ++i) {
      const lc_segment& s = L.segs[i];
      const void* arr[5] = {s.weight, s.shadow, s.master, s.exp_avg, s.exp_avg_sq};
      for (int a = 0; a < 5; ++a)
        if (arr[a]) {
          const uint64_t b = reinterpret_cast<uint64_t>(arr[a]);
          spans.push_back({b, b + s.numel * (a < 2 ? L.esz : 4u), i});
        }
    }
    std::sort(spans.begin(), spans.end(), [](const Span& x, const Span& y) { return x.b < y.b; });
    uint64_t reach = 0;
    uint32_t reach_seg = 0;
    for (const Span& sp : spans) {
      if (sp.b < reach)
        return fail(LC_ERR_INVALID_ARG, "segments %u and %u: arrays overlap in memory", reach_seg, sp.seg);
      reach = sp.e;
      reach_seg = sp.seg;
    }
  }
  L.layer_seg_begin[N] = d->n_segments;
  L.total_numel = 0;
  for (uint32_t l = 0; l < N; ++l) {
    L.total_numel += L.numel[l];
    if (L.total_numel > (1ull << 56)) return fail(LC_ERR_INVALID_ARG, "too many elements in all");
  }
  // the staleness numerator sum_l n_l * age_l (age <= S_max - 1) must fit in 64 bits
  if (L.total_numel > static_cast<uint64_t>(std::numeric_limits<int64_t>::max()) / static_cast<uint64_t>(d->s_max))
    return fail(LC_ERR_INVALID_ARG, "total elements times s_max overflows 63 bits");

  // score chunks
  const uint64_t ce = kChunkBytes / L.esz;
  L.layer_chunk_begin.assign(N + 1, 0);
  uint64_t nchunks = 0;
  for (uint32_t i = 0; i < d->n_segments; ++i) {
    const lc_segment& s = L.segs[i];
    ScoreSeg ss;
    ss.w = reinterpret_cast<uint64_t>(s.weight);
    ss.s = reinterpret_cast<uint64_t>(s.shadow);
    ss.numel = s.numel;
    ss.chunk_begin = static_cast<uint32_t>(nchunks);
    ss.vec_ok = (ss.w % 16 == 0 && ss.s % 16 == 0) ? 1u : 0u;
    const uint64_t k = (s.numel + ce - 1) / ce;
    if (nchunks + k > 0xFFFFFFF0ull) return fail(LC_ERR_INVALID_ARG, "too many chunks");
    for (uint64_t j = 0; j < k; ++j) L.chunk_seg.push_back(i);
    nchunks += k;
    L.score_segs.push_back(ss);
    OptSeg os;
    os.w = ss.w;
    os.master = reinterpret_cast<uint64_t>(s.master);
    os.m = reinterpret_cast<uint64_t>(s.exp_avg);
    os.v = reinterpret_cast<uint64_t>(s.exp_avg_sq);
    os.numel = s.numel;
    os.chunk_begin = ss.chunk_begin;
    os.vec_ok = (os.w % (4 * L.esz) == 0 && os.master % 16 == 0 && os.m % 16 == 0 && os.v % 16 == 0) ? 1u : 0u;
    L.opt_segs.push_back(os);
    L.layer_chunk_begin[s.layer + 1] = static_cast<uint32_t>(nchunks);
  }

  // copy units in record order: W blocks, master blocks, m blocks, v blocks
  L.rec_bytes.assign(N, 0);
  L.layer_pieces.assign(N, 0);
  L.layer_piece_begin.assign(N + 1, 0);
  for (uint32_t l = 0; l < N; ++l) {
    uint64_t rec = 0, pieces = 0;
    for (int arr = 0; arr < 4; ++arr) {
      if (arr == 1 && !L.has_master) continue;
      if (arr >= 2 && !L.has_moments) continue;
      for (uint32_t i = L.layer_seg_begin[l]; i < L.layer_seg_begin[l + 1]; ++i) {
        const lc_segment& s = L.segs[i];
        CopyUnit u{};
        const void* base = arr == 0 ? s.weight : arr == 1 ? static_cast<void*>(s.master)
                          : arr == 2 ? static_cast<void*>(s.exp_avg) : static_cast<void*>(s.exp_avg_sq);
        u.arr = reinterpret_cast<uint64_t>(base);
        u.shadow = arr == 0 ? reinterpret_cast<uint64_t>(s.shadow) : 0;
        u.elem = arr == 0 ? L.esz : 4;
        u.bytes = s.numel * u.elem;
        u.rec_off = rec;
        u.piece0 = static_cast<uint32_t>(pieces);
        u.vec_ok = (u.arr % 16 == 0 && u.shadow % 16 == 0) ? 1u : 0u;
        const uint64_t k = (u.bytes + kPieceBytes - 1) / kPieceBytes;
        const uint32_t uid = static_cast<uint32_t>(L.units.size());
        for (uint64_t j = 0; j < k; ++j) L.piece_unit.push_back(uid);
        pieces += k;
        rec += round_up(u.bytes, kRecordAlign);
        L.units.push_back(u);
      }
    }
    if (pieces > 0xFFFFFFF0ull) return fail(LC_ERR_INVALID_ARG, "layer %u record too large", l);
    L.rec_bytes[l] = rec;
    L.layer_pieces[l] = pieces;
    L.layer_piece_begin[l + 1] = L.layer_piece_begin[l] + pieces;
  }
  return LC_OK;
}

}  // namespace

namespace {

#define LC_HIP(ctx, call)                                                                  \
  do {                                                                                    \
    hipError_t e_ = (call);                                                               \
    if (e_ != hipSuccess) {                                                               \
      if (ctx) (ctx)->poisoned = true;                                                    \
      return fail(LC_ERR_HIP, "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, __LINE__); \
    }                                                                                     \
  } while (0)

template <typename T>
lc_status dev_alloc(lc_ctx* c, T** p, size_t count) {
  void* q = nullptr;
  const size_t bytes = count * sizeof(T) > 0 ? count * sizeof(T) : 16;
  hipError_t e = hipMalloc(&q, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(LC_ERR_OOM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
  }
  c->allocations.push_back(q);
  *p = static_cast<T*>(q);
  return LC_OK;
}

// Host vectors that feed asynchronous uploads must outlive the copies: a
// function that uploads from locals holds one of these, so that an early
// return (a failed call after some copies were enqueued) still waits for
// the stream before the vectors go.  On the normal path the stream has
// already been synchronised and the wait returns at once.
struct UploadsDrained {
  lc_ctx* c;
  ~UploadsDrained() { (void)hipStreamSynchronize(c->stream); }
};

template <typename T>
lc_status upload(lc_ctx* c, T* dst, const std::vector<T>& src) {
  if (src.empty()) return LC_OK;
  LC_HIP(c, hipMemcpyAsync(dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice, c->stream));
  return LC_OK;
}

void free_all(lc_ctx* c) {
  for (void* p : c->allocations) (void)hipFree(p);
  c->allocations.clear();
  if (c->h_result) (void)hipHostFree(c->h_result);
  c->h_result = nullptr;
  if (c->h_grad) (void)hipHostFree(c->h_grad);
  c->h_grad = nullptr;
  if (c->grad_event) (void)hipEventDestroy(c->grad_event);
  c->grad_event = nullptr;
}

lc_status check_ctx(lc_ctx* c) {
  if (!c) return fail(LC_ERR_INVALID_ARG, "context is NULL");
  if (c->poisoned) return fail(LC_ERR_BAD_STATE, "context is poisoned by an earlier HIP error");
  return LC_OK;
}

// Wait until the select kernel has written the pending selection into the
// pinned host mirror (its sequence number appears last, after a system-scope
// fence).  The flag is polled, so the host reacts within a microsecond or two
// of the kernel's store instead of after a device-to-host copy and a stream
// synchronisation; every 256 polls the stream is queried, so an error or a
// stream that drained without the flag ends the wait.
lc_status wait_result(lc_ctx* c) {
  const volatile uint64_t* flag = &c->h_result->seq;
  for (uint32_t spin = 1;; ++spin) {
    if (*flag == c->result_seq) break;
    if (spin % 256 == 0) {
      const hipError_t q = hipStreamQuery(c->stream);
      if (q == hipSuccess) {
        if (*flag == c->result_seq) break;
        c->poisoned = true;
        return fail(LC_ERR_HIP, "the selection never reached the host");
      }
      if (q != hipErrorNotReady) {
        (void)hipGetLastError();
        c->poisoned = true;
        return fail(LC_ERR_HIP, "waiting for the selection failed: %s", hipGetErrorString(q));
      }
    }
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  return LC_OK;
}

// Make the pending selection's mask available on the host.
lc_status fetch_result(lc_ctx* c) {
  if (c->result_on_host) return LC_OK;
  lc_status st = wait_result(c);
  if (st != LC_OK) return st;
  const uint32_t N = c->L.N;
  const uint8_t* mask = reinterpret_cast<const uint8_t*>(c->h_result + 1);
  c->sel.clear();
  c->sel_rec_prefix.assign(1, 0);
  c->sel_piece_prefix.assign(1, 0);
  for (uint32_t l = 0; l < N; ++l) {
    if (mask[l] > 1) {
      c->poisoned = true;
      return fail(LC_ERR_HIP, "corrupt selection mask");
    }
    if (mask[l]) {
      c->sel.push_back(l);
      c->sel_rec_prefix.push_back(c->sel_rec_prefix.back() + c->L.rec_bytes[l]);
      c->sel_piece_prefix.push_back(c->sel_piece_prefix.back() + c->L.layer_pieces[l]);
    }
  }
  if (c->sel.size() != c->h_result->n_selected || c->sel_rec_prefix.back() != c->h_result->payload_bytes) {
    c->poisoned = true;
    return fail(LC_ERR_HIP, "device selection plan disagrees with the host");
  }
  c->rank_packed.assign(c->sel.size(), 0);
  c->n_unpacked = static_cast<uint32_t>(c->sel.size());
  c->result_on_host = true;
  if (c->n_unpacked == 0) c->pending = false;
  return LC_OK;
}

lc_status enqueue_select(lc_ctx* c, int64_t step, double lr, int base_mode, bool persists) {
  ++c->result_seq;
  LC_HIP(c, launch_select(c->dt, step, lr, base_mode, c->result_seq, c->stream));
  c->have_selection = true;
  c->pending = true;
  c->pending_persists = persists;
  c->result_on_host = false;
  return LC_OK;
}

// Eq. 4 resets Delta_l and t_l of every selected layer as if it were already
// persisted.  A selection made by lc_select or lc_rebase therefore has to be
// packed in full before the state moves on: were it dropped, a recovery would
// fall back to an older record of those layers without any error and the
// staleness bound of Section 3.3 would no longer hold.  The base selected by
// lc_init_layout resets nothing, so in ACCUM mode a warm-up may leave it
// unpacked; SNAPSHOT mode needs it packed, since its pack refreshes the shadow.
lc_status require_packed(lc_ctx* c) {
  if (!c->pending || !(c->pending_persists || c->mode == LC_MODE_SNAPSHOT)) return LC_OK;
  if (!c->result_on_host) {
    lc_status st = fetch_result(c);
    if (st != LC_OK) return st;
  }
  if (c->pending)
    return fail(LC_ERR_BAD_STATE, "the previous selection is not fully packed (%u of its layers are not)",
                c->n_unpacked);
  return LC_OK;
}

}  // namespace

namespace lc {

bool device_range_ok(const void* p, uint64_t bytes) {
  if (!p) return false;
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) return false;
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return true;  // the extent is not known (a virtual-memory mapping, say): the type check stands
  }
  const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
  return q >= b && q - b <= size && bytes <= size - (q - b);
}

lc_status restore_range_from_host(lc_ctx* c, uint32_t l, uint64_t rec_off, uint64_t len, const uint8_t* bytes) {
  const HostLayout& L = c->L;
  const uint32_t per_seg = 1u + (L.has_master ? 1u : 0u) + (L.has_moments ? 2u : 0u);
  uint32_t ub = 0;
  for (uint32_t j = 0; j < l; ++j) ub += (L.layer_seg_begin[j + 1] - L.layer_seg_begin[j]) * per_seg;
  const uint32_t nu = (L.layer_seg_begin[l + 1] - L.layer_seg_begin[l]) * per_seg;
  const uint64_t end = rec_off + len;
  for (uint32_t k = 0; k < nu; ++k) {
    const CopyUnit& u = L.units[ub + k];
    const uint64_t a = std::max<uint64_t>(u.rec_off, rec_off), b = std::min<uint64_t>(u.rec_off + u.bytes, end);
    if (a >= b) continue;  // this block (or its padding only) lies outside the range
    void* dst = reinterpret_cast<void*>(u.arr + (a - u.rec_off));
    LC_HIP(c, hipMemcpyAsync(dst, bytes + (a - rec_off), b - a, hipMemcpyHostToDevice, c->stream));
    if (u.shadow)
      LC_HIP(c, hipMemcpyAsync(reinterpret_cast<void*>(u.shadow + (a - u.rec_off)), dst, b - a,
                               hipMemcpyDeviceToDevice, c->stream));
  }
  return LC_OK;
}

lc_status restore_finish(lc_ctx* c, int64_t t_fail, const std::vector<int64_t>& steps) {
  const uint32_t N = c->L.N;
  std::vector<double> zeros(N, 0.0);
  UploadsDrained drained{c};
  lc_status st = upload(c, c->dt.delta, zeros);
  if (st != LC_OK) return st;
  st = upload(c, c->dt.t_last, steps);
  if (st != LC_OK) return st;
  LC_HIP(c, hipStreamSynchronize(c->stream));
  c->last_step = t_fail;
  c->scored = false;
  c->have_selection = false;
  c->pending = false;
  c->pending_persists = false;
  c->shadow_valid = c->L.has_shadow;
  c->result_on_host = false;
  return LC_OK;
}

}  // namespace lc

namespace {

using RoctxPush = int (*)(const char*);
using RoctxPop = int (*)();
struct Roctx {
  RoctxPush push = nullptr;
  RoctxPop pop = nullptr;
};

// Resolved once per process (thread-safe static initialisation).
const Roctx& roctx() {
  static const Roctx r = [] {
    Roctx x;
    const char* on = std::getenv("LAYERCHECK_ROCTX");
    if (!on || std::strcmp(on, "1") != 0) return x;
    void* h = dlopen("librocprofiler-sdk-roctx.so.1", RTLD_NOW | RTLD_LOCAL);
    if (!h) return x;
    x.push = reinterpret_cast<RoctxPush>(dlsym(h, "roctxRangePushA"));
    x.pop = reinterpret_cast<RoctxPop>(dlsym(h, "roctxRangePop"));
    if (!x.push || !x.pop) x = Roctx{};
    return x;
  }();
  return r;
}

}  // namespace

lc::TraceRange::TraceRange(const char* name) : on_(roctx().push != nullptr) {
  if (on_) roctx().push(name);
}

lc::TraceRange::~TraceRange() {
  if (on_) roctx().pop();
}

extern "C" {

const char* lc_last_error(void) { return g_error.c_str(); }

lc_status lc_query_build(lc_build_info* out) {
  if (!out) return fail(LC_ERR_INVALID_ARG, "out is NULL");
  out->chunk_bytes = kChunkBytes;
  out->piece_bytes = kPieceBytes;
  out->record_align = kRecordAlign;
  out->reserved = 0;
  return LC_OK;
}

lc_status lc_query_layout(const lc_layout_desc* d, uint64_t* numel_out, uint64_t* record_bytes_out) {
  HostLayout L;
  lc_status st = build_layout(d, L);
  if (st != LC_OK) return st;
  for (uint32_t l = 0; l < L.N; ++l) {
    if (numel_out) numel_out[l] = L.numel[l];
    if (record_bytes_out) record_bytes_out[l] = L.rec_bytes[l];
  }
  return LC_OK;
}

lc_status lc_init_layout(const lc_layout_desc* d, lc_ctx** out) {
  lc::TraceRange trace_("lc_init_layout");
  if (!out) return fail(LC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  lc_ctx* c = new (std::nothrow) lc_ctx();
  if (!c) return fail(LC_ERR_OOM, "host allocation failed");
  lc_status st = build_layout(d, c->L);
  if (st != LC_OK) {
    delete c;
    return st;
  }
  // every array a kernel will stream must be device memory of its full
  // extent: refused here rather than faulting in a kernel
  for (uint32_t i = 0; i < c->L.segs.size(); ++i) {
    const lc_segment& sg = c->L.segs[i];
    const void* arr[5] = {sg.weight, sg.shadow, sg.master, sg.exp_avg, sg.exp_avg_sq};
    static const char* const kName[5] = {"weight", "shadow", "master", "exp_avg", "exp_avg_sq"};
    for (int a = 0; a < 5; ++a) {
      if (!arr[a]) continue;
      const uint64_t bytes = sg.numel * (a < 2 ? c->L.esz : 4u);
      if (!device_range_ok(arr[a], bytes)) {
        delete c;
        return fail(LC_ERR_INVALID_ARG, "segment %u: %s is not device memory holding %llu bytes", i, kName[a],
                    static_cast<unsigned long long>(bytes));
      }
    }
  }
  c->mode = d->mode;
  c->s_max = d->s_max;
  c->eps_w = d->eps_w;
  c->t_base = d->t_base;
  c->stream = static_cast<hipStream_t>(d->stream);
  c->last_step = d->t_base;
  const HostLayout& L = c->L;
  const uint32_t N = L.N;

  auto bail = [&](lc_status s) {
    (void)hipStreamSynchronize(c->stream);
    free_all(c);
    delete c;
    return s;
  };
#define LC_TRY(expr)                   \
  do {                                 \
    lc_status s_ = (expr);             \
    if (s_ != LC_OK) return bail(s_);  \
  } while (0)

  DeviceTables& t = c->dt;
  t.n_layers = N;
  t.n_chunks = static_cast<uint32_t>(L.chunk_seg.size());
  t.dtype = L.dtype;
  t.mode = d->mode;
  t.eps_w = d->eps_w;
  t.s_max = d->s_max;
  ScoreSeg* segs; uint32_t* chunk_seg; uint32_t* lcb; double2* partials; double* u; double* delta;
  int64_t* t_last; double* k0; uint64_t* numel; uint64_t* rec; uint64_t* lpieces; CopyUnit* units;
  uint32_t* piece_unit; uint64_t* lpb; uint32_t* sel_layer; uint64_t* srp; uint64_t* spp;
  SelectHeader* result; uint32_t* rank_layer; uint64_t* rank_src; uint64_t* rpp;
  LC_TRY(dev_alloc(c, &segs, L.score_segs.size()));
  LC_TRY(dev_alloc(c, &chunk_seg, L.chunk_seg.size()));
  LC_TRY(dev_alloc(c, &lcb, N + 1));
  LC_TRY(dev_alloc(c, &partials, L.chunk_seg.size()));
  LC_TRY(dev_alloc(c, &u, N));
  LC_TRY(dev_alloc(c, &delta, N));
  LC_TRY(dev_alloc(c, &t_last, N));
  LC_TRY(dev_alloc(c, &k0, N));
  LC_TRY(dev_alloc(c, &numel, N));
  LC_TRY(dev_alloc(c, &rec, N));
  LC_TRY(dev_alloc(c, &lpieces, N));
  LC_TRY(dev_alloc(c, &units, L.units.size()));
  LC_TRY(dev_alloc(c, &piece_unit, L.piece_unit.size()));
  LC_TRY(dev_alloc(c, &lpb, N + 1));
  LC_TRY(dev_alloc(c, &sel_layer, N));
  LC_TRY(dev_alloc(c, &srp, N + 1));
  LC_TRY(dev_alloc(c, &spp, N + 1));
  {
    uint8_t* r8;
    LC_TRY(dev_alloc(c, &r8, sizeof(SelectHeader) + N));
    result = reinterpret_cast<SelectHeader*>(r8);
  }
  OptSeg* opt_segs;
  LC_TRY(dev_alloc(c, &opt_segs, L.opt_segs.size()));
  LC_TRY(dev_alloc(c, &c->d_grad, L.opt_segs.size()));
  LC_TRY(dev_alloc(c, &rank_layer, N));
  LC_TRY(dev_alloc(c, &rank_src, N));
  LC_TRY(dev_alloc(c, &rpp, N + 1));
  {
    // the select kernel writes this mirror itself: coherent (fine-grained)
    // pinned memory, so its stores reach the host without a copy
    void* h = nullptr;
    hipError_t e = hipHostMalloc(&h, sizeof(SelectHeader) + N, hipHostMallocCoherent);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return bail(fail(LC_ERR_OOM, "hipHostMalloc failed: %s", hipGetErrorString(e)));
    }
    c->h_result = static_cast<SelectHeader*>(h);
    std::memset(h, 0, sizeof(SelectHeader) + N);
    void* dh = nullptr;
    e = hipHostGetDevicePointer(&dh, h, 0);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return bail(fail(LC_ERR_HIP, "hipHostGetDevicePointer failed: %s", hipGetErrorString(e)));
    }
    t.host_result = static_cast<SelectHeader*>(dh);
    h = nullptr;
    e = hipHostMalloc(&h, sizeof(GradSeg) * L.opt_segs.size(), hipHostMallocDefault);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return bail(fail(LC_ERR_OOM, "hipHostMalloc failed: %s", hipGetErrorString(e)));
    }
    c->h_grad = static_cast<GradSeg*>(h);
    e = hipEventCreateWithFlags(&c->grad_event, hipEventDisableTiming);
    if (e != hipSuccess) return bail(fail(LC_ERR_HIP, "hipEventCreate failed: %s", hipGetErrorString(e)));
  }
  t.segs = segs; t.chunk_seg = chunk_seg; t.layer_chunk_begin = lcb; t.partials = partials;
  t.u = u; t.delta = delta; t.t_last = t_last; t.k0 = k0; t.numel = numel; t.rec_bytes = rec;
  t.layer_pieces = lpieces; t.units = units; t.piece_unit = piece_unit; t.layer_piece_begin = lpb;
  t.sel_layer = sel_layer; t.sel_rec_prefix = srp; t.sel_piece_prefix = spp; t.result = result;
  t.rank_layer = rank_layer; t.rank_src = rank_src; t.rank_piece_prefix = rpp;
  t.opt_segs = opt_segs; t.grad_segs = c->d_grad;

  std::vector<double> zeros(N, 0.0), k0v(d->k0, d->k0 + N);
  std::vector<int64_t> tl(N, d->t_base);
  LC_TRY(upload(c, segs, L.score_segs));
  LC_TRY(upload(c, chunk_seg, L.chunk_seg));
  LC_TRY(upload(c, lcb, L.layer_chunk_begin));
  LC_TRY(upload(c, u, zeros));
  LC_TRY(upload(c, delta, zeros));
  LC_TRY(upload(c, t_last, tl));
  LC_TRY(upload(c, k0, k0v));
  LC_TRY(upload(c, numel, L.numel));
  LC_TRY(upload(c, rec, L.rec_bytes));
  LC_TRY(upload(c, lpieces, L.layer_pieces));
  LC_TRY(upload(c, units, L.units));
  LC_TRY(upload(c, piece_unit, L.piece_unit));
  LC_TRY(upload(c, lpb, L.layer_piece_begin));
  LC_TRY(upload(c, opt_segs, L.opt_segs));
  // S <- W for every segment (Section 3.2: drift is measured from the base)
  c->shadow_valid = L.has_shadow;
  for (const lc_segment& s : L.segs) {
    if (!L.has_shadow) break;
    hipError_t e = hipMemcpyAsync(s.shadow, s.weight, s.numel * L.esz, hipMemcpyDeviceToDevice, c->stream);
    if (e != hipSuccess) return bail(fail(LC_ERR_HIP, "shadow init copy failed: %s", hipGetErrorString(e)));
  }
  // base selection: every layer, at t_base
  LC_TRY(enqueue_select(c, d->t_base, 1.0, 1, false));
  {
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return bail(fail(LC_ERR_HIP, "init failed: %s", hipGetErrorString(e)));
  }
#undef LC_TRY
  *out = c;
  return LC_OK;
}

lc_status lc_score_layers(lc_ctx* c, int64_t step) {
  lc::TraceRange trace_("lc_score_layers");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (step <= c->last_step)
    return fail(LC_ERR_BAD_STATE, "step %lld must exceed the previous step %lld", static_cast<long long>(step),
                static_cast<long long>(c->last_step));
  if (!c->shadow_valid)
    return fail(LC_ERR_BAD_STATE, c->L.has_shadow
                                      ? "the shadow is stale after a fused optimizer step; a restore or "
                                        "lc_rebase re-synchronises it"
                                      : "the layout has no shadow copies; use a fused optimizer step");
  st = require_packed(c);
  if (st != LC_OK) return st;
  LC_HIP(c, launch_score(c->dt, c->stream));
  c->last_step = step;
  c->scored = true;
  c->scored_step = step;
  c->have_selection = false;
  c->pending = false;
  c->result_on_host = false;
  return LC_OK;
}

lc_status lc_select(lc_ctx* c, int64_t step, double lr_scale, uint8_t* mask_out, lc_select_stats* stats_out) {
  lc::TraceRange trace_("lc_select");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (!c->scored || c->scored_step != step)
    return fail(LC_ERR_BAD_STATE, "lc_select(%lld) must follow lc_score_layers at the same step",
                static_cast<long long>(step));
  if (!(lr_scale > 0.0) || !std::isfinite(lr_scale))
    return fail(LC_ERR_INVALID_ARG, "lr_scale must be positive and finite");
  st = enqueue_select(c, step, lr_scale, 0, true);
  if (st != LC_OK) return st;
  c->scored = false;
  if (mask_out || stats_out) {
    st = fetch_result(c);
    if (st != LC_OK) return st;
    if (mask_out) std::memcpy(mask_out, c->h_result + 1, c->L.N);
    if (stats_out) {
      const SelectHeader& h = *c->h_result;
      stats_out->n_selected = h.n_selected;
      stats_out->n_forced = h.n_forced;
      stats_out->payload_bytes = h.payload_bytes;
      stats_out->max_age = h.max_age;
      stats_out->weighted_age = h.weighted_age;
    }
  }
  return LC_OK;
}

lc_status lc_pack_selected(lc_ctx* c, void* staging, uint64_t capacity, uint32_t first_rank,
                           lc_pack_result* out) {
  lc::TraceRange trace_("lc_pack_selected");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (!out) return fail(LC_ERR_INVALID_ARG, "out is NULL");
  if (!c->have_selection) return fail(LC_ERR_BAD_STATE, "no selection to pack");
  st = fetch_result(c);
  if (st != LC_OK) return st;
  const uint32_t ns = static_cast<uint32_t>(c->sel.size());
  if (first_rank > ns) return fail(LC_ERR_INVALID_ARG, "first_rank %u > %u selected", first_rank, ns);
  uint32_t last = first_rank;
  while (last < ns && c->sel_rec_prefix[last + 1] - c->sel_rec_prefix[first_rank] <= capacity) ++last;
  if (last == first_rank && first_rank < ns)
    return fail(LC_ERR_CAPACITY, "record of layer %u (%llu B) exceeds capacity %llu", c->sel[first_rank],
                static_cast<unsigned long long>(c->L.rec_bytes[c->sel[first_rank]]),
                static_cast<unsigned long long>(capacity));
  const uint64_t bytes = c->sel_rec_prefix[last] - c->sel_rec_prefix[first_rank];
  if (last > first_rank) {
    if (!staging) return fail(LC_ERR_INVALID_ARG, "staging is NULL");
    if (reinterpret_cast<uintptr_t>(staging) % kRecordAlign)
      return fail(LC_ERR_INVALID_ARG, "staging must be %u-byte aligned", kRecordAlign);
    if (!device_range_ok(staging, bytes))
      return fail(LC_ERR_INVALID_ARG, "staging is not device memory holding the %llu bytes to pack",
                  static_cast<unsigned long long>(bytes));
    const uint64_t pieces = c->sel_piece_prefix[last] - c->sel_piece_prefix[first_rank];
    LC_HIP(c, launch_pack(c->dt, first_rank, last, c->sel_piece_prefix[first_rank], pieces,
                          c->sel_rec_prefix[first_rank], staging, c->mode == LC_MODE_SNAPSHOT, c->stream));
    for (uint32_t r = first_rank; r < last; ++r)
      if (!c->rank_packed[r]) {
        c->rank_packed[r] = 1;
        --c->n_unpacked;
      }
  }
  if (c->n_unpacked == 0) c->pending = false;
  out->bytes_written = bytes;
  out->n_packed = last - first_rank;
  out->next_rank = last;
  out->done = last == ns ? 1 : 0;
  out->reserved = 0;
  return LC_OK;
}

lc_status lc_restore_composite(lc_ctx* c, const lc_version* v, uint32_t n_versions, int64_t t_fail,
                               int64_t* chosen_step_out) {
  lc::TraceRange trace_("lc_restore_composite");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (!v || n_versions == 0) return fail(LC_ERR_INVALID_ARG, "no versions");
  const HostLayout& L = c->L;
  const uint32_t N = L.N;
  for (uint32_t i = 0; i < n_versions; ++i) {
    if (!v[i].mask) return fail(LC_ERR_INVALID_ARG, "version %u: mask is NULL", i);
    uint64_t need = 0;
    for (uint32_t l = 0; l < N; ++l) {
      if (v[i].mask[l] > 1) return fail(LC_ERR_INVALID_ARG, "version %u: mask must be 0/1", i);
      if (v[i].mask[l]) need += L.rec_bytes[l];
    }
    if (need != v[i].payload_bytes)
      return fail(LC_ERR_INVALID_ARG, "version %u: payload_bytes %llu != %llu for its mask", i,
                  static_cast<unsigned long long>(v[i].payload_bytes), static_cast<unsigned long long>(need));
    if (need && !v[i].payload) return fail(LC_ERR_INVALID_ARG, "version %u: payload is NULL", i);
  }
  // plan (Section 3.5): newest version <= t_fail holding the layer
  std::vector<int64_t> choice(N, -1);
  for (uint32_t l = 0; l < N; ++l) {
    int64_t best = -1;
    bool dup = false;
    for (uint32_t i = 0; i < n_versions; ++i) {
      if (v[i].step > t_fail || !v[i].mask[l]) continue;
      if (best < 0 || v[i].step > v[best].step) {
        best = i;
        dup = false;
      } else if (v[i].step == v[best].step) {
        dup = true;
      }
    }
    if (best < 0)
      return fail(LC_ERR_NO_VERSION, "layer %u: no persisted version at step <= %lld", l,
                  static_cast<long long>(t_fail));
    if (dup)
      return fail(LC_ERR_INVALID_ARG, "layer %u: two versions at step %lld", l,
                  static_cast<long long>(v[best].step));
    choice[l] = best;
  }
  // record address of each layer, and where each version's payload lives
  std::vector<int> kind(n_versions, -1);  // 0 device, 1 host
  std::vector<const uint8_t*> dev_base(n_versions, nullptr);
  std::vector<uint32_t> rank_layer;
  std::vector<uint64_t> rank_src, rank_pp(1, 0);
  std::vector<std::pair<uint32_t, const uint8_t*>> host_layers;
  for (uint32_t l = 0; l < N; ++l) {
    const uint32_t i = static_cast<uint32_t>(choice[l]);
    if (kind[i] < 0) {
      hipPointerAttribute_t attr;
      hipError_t e = hipPointerGetAttributes(&attr, v[i].payload);
      if (e == hipSuccess && attr.type == hipMemoryTypeDevice) {
        if (!device_range_ok(v[i].payload, v[i].payload_bytes))
          return fail(LC_ERR_INVALID_ARG, "version %u: the device payload is shorter than payload_bytes", i);
        kind[i] = 0;
        dev_base[i] = static_cast<const uint8_t*>(v[i].payload);
      } else {
        (void)hipGetLastError();
        kind[i] = 1;
      }
    }
    uint64_t off = 0;
    for (uint32_t j = 0; j < l; ++j)
      if (v[i].mask[j]) off += L.rec_bytes[j];
    if (kind[i] == 0) {
      rank_layer.push_back(l);
      rank_src.push_back(reinterpret_cast<uint64_t>(dev_base[i] + off));
      rank_pp.push_back(rank_pp.back() + L.layer_pieces[l]);
    } else {
      host_layers.emplace_back(l, static_cast<const uint8_t*>(v[i].payload) + off);
    }
  }
  UploadsDrained drained{c};  // declared after the tables it protects, so it runs first
  if (!rank_layer.empty()) {
    st = upload(c, c->dt.rank_layer, rank_layer);
    if (st != LC_OK) return st;
    st = upload(c, c->dt.rank_src, rank_src);
    if (st != LC_OK) return st;
    st = upload(c, c->dt.rank_piece_prefix, rank_pp);
    if (st != LC_OK) return st;
    const uint64_t pieces = rank_pp.back();
    LC_HIP(c, launch_unpack(c->dt, static_cast<uint32_t>(rank_layer.size()), pieces, c->stream));
  }
  // host-resident records: one copy per block, then S <- W
  for (const auto& hl : host_layers) {
    st = restore_range_from_host(c, hl.first, 0, L.rec_bytes[hl.first], hl.second);
    if (st != LC_OK) return st;
  }
  std::vector<int64_t> steps(N);
  for (uint32_t l = 0; l < N; ++l) steps[l] = v[choice[l]].step;
  st = restore_finish(c, t_fail, steps);
  if (st != LC_OK) return st;
  if (chosen_step_out) std::memcpy(chosen_step_out, steps.data(), N * sizeof(int64_t));
  return LC_OK;
}

lc_status lc_rebase(lc_ctx* c, int64_t step) {
  lc::TraceRange trace_("lc_rebase");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (step < c->last_step)
    return fail(LC_ERR_BAD_STATE, "the base step %lld precedes the last step %lld", static_cast<long long>(step),
                static_cast<long long>(c->last_step));
  const uint32_t N = c->L.N;
  std::vector<double> zeros(N, 0.0);
  std::vector<int64_t> tl(N, step);
  UploadsDrained drained{c};
  st = upload(c, c->dt.delta, zeros);
  if (st != LC_OK) return st;
  st = upload(c, c->dt.t_last, tl);
  if (st != LC_OK) return st;
  for (const lc_segment& sg : c->L.segs) {
    if (!c->L.has_shadow) break;
    LC_HIP(c, hipMemcpyAsync(sg.shadow, sg.weight, sg.numel * c->L.esz, hipMemcpyDeviceToDevice, c->stream));
  }
  c->shadow_valid = c->L.has_shadow;
  st = enqueue_select(c, step, 1.0, 1, true);
  if (st != LC_OK) return st;
  // the uploads read host vectors that end with this call
  LC_HIP(c, hipStreamSynchronize(c->stream));
  c->last_step = step;
  c->scored = false;
  return LC_OK;
}

}  // extern "C"

namespace {

// Shared by the optimizer steps: validation of the call and the gradient
// table, its upload, and the call-order state afterwards (the caller
// launches its kernel between the two halves).
lc_status optimizer_begin(lc_ctx* c, int64_t step, const void* const* grads, int32_t grad_dtype,
                          const uint8_t* decay_mask) {
  if (!grads) return fail(LC_ERR_INVALID_ARG, "grads must be non-NULL");
  if (grad_dtype != LC_DT_BF16 && grad_dtype != LC_DT_F32)
    return fail(LC_ERR_INVALID_ARG, "unknown gradient dtype %d", grad_dtype);
  if (c->mode != LC_MODE_ACCUM) return fail(LC_ERR_BAD_STATE, "the fused optimizer step needs LC_MODE_ACCUM");
  if (step <= c->last_step)
    return fail(LC_ERR_BAD_STATE, "step %lld must exceed the previous step %lld", static_cast<long long>(step),
                static_cast<long long>(c->last_step));
  lc_status st = require_packed(c);
  if (st != LC_OK) return st;
  const size_t ns = c->L.opt_segs.size();
  const uint32_t gsz = grad_dtype == LC_DT_BF16 ? 2 : 4;
  for (size_t i = 0; i < ns; ++i) {
    const uintptr_t g = reinterpret_cast<uintptr_t>(grads[i]);
    if (!g) return fail(LC_ERR_INVALID_ARG, "gradient of segment %zu is NULL", i);
    if (g % gsz) return fail(LC_ERR_INVALID_ARG, "gradient of segment %zu is misaligned", i);
    if (decay_mask && decay_mask[i] > 1) return fail(LC_ERR_INVALID_ARG, "decay_mask must be 0/1");
  }
  // the pinned table may still feed the previous call's upload
  if (c->grad_event_pending) LC_HIP(c, hipEventSynchronize(c->grad_event));
  for (size_t i = 0; i < ns; ++i) {
    const uint64_t g = reinterpret_cast<uint64_t>(grads[i]);
    c->h_grad[i].grad = g;
    c->h_grad[i].decay = decay_mask ? decay_mask[i] : 1u;
    c->h_grad[i].vec_ok = g % (4 * gsz) == 0 ? 1u : 0u;
  }
  LC_HIP(c, hipMemcpyAsync(c->d_grad, c->h_grad, sizeof(GradSeg) * ns, hipMemcpyHostToDevice, c->stream));
  LC_HIP(c, hipEventRecord(c->grad_event, c->stream));
  c->grad_event_pending = true;
  return LC_OK;
}

lc_status optimizer_end(lc_ctx* c, int64_t step) {
  LC_HIP(c, launch_finalize(c->dt, c->stream));
  c->last_step = step;
  c->scored = true;
  c->scored_step = step;
  c->have_selection = false;
  c->pending = false;
  c->result_on_host = false;
  c->shadow_valid = false;
  return LC_OK;
}

}  // namespace

extern "C" {

lc_status lc_adamw_step_score(lc_ctx* c, int64_t step, const void* const* grads, int32_t grad_dtype,
                              const uint8_t* decay_mask, const lc_adamw_params* p) {
  lc::TraceRange trace_("lc_adamw_step_score");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (!p) return fail(LC_ERR_INVALID_ARG, "params must be non-NULL");
  if (!(p->lr >= 0.0) || !std::isfinite(p->lr)) return fail(LC_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (!(p->beta1 >= 0.0 && p->beta1 < 1.0) || !(p->beta2 >= 0.0 && p->beta2 < 1.0))
    return fail(LC_ERR_INVALID_ARG, "betas must lie in [0, 1)");
  if (!(p->eps > 0.0) || !std::isfinite(p->eps)) return fail(LC_ERR_INVALID_ARG, "eps must be finite and > 0");
  if (!(p->weight_decay >= 0.0) || !std::isfinite(p->weight_decay))
    return fail(LC_ERR_INVALID_ARG, "weight_decay must be finite and >= 0");
  if (p->adam_step < 1) return fail(LC_ERR_INVALID_ARG, "adam_step must be >= 1");
  if (!c->L.has_moments) return fail(LC_ERR_BAD_STATE, "the layout has no Adam moments");
  st = optimizer_begin(c, step, grads, grad_dtype, decay_mask);
  if (st != LC_OK) return st;
  const double t = static_cast<double>(p->adam_step);
  AdamScalars sc;
  sc.b1 = static_cast<float>(p->beta1);
  sc.omb1 = static_cast<float>(1.0 - p->beta1);
  sc.b2 = static_cast<float>(p->beta2);
  sc.omb2 = static_cast<float>(1.0 - p->beta2);
  sc.c1 = static_cast<float>(1.0 / (1.0 - std::pow(p->beta1, t)));
  sc.c2 = static_cast<float>(1.0 / (1.0 - std::pow(p->beta2, t)));
  sc.eps = static_cast<float>(p->eps);
  sc.lr = static_cast<float>(p->lr);
  sc.decay = static_cast<float>(1.0 - p->lr * p->weight_decay);
  LC_HIP(c, launch_adamw(c->dt, grad_dtype, c->L.has_master ? 1 : 0, sc, c->stream));
  return optimizer_end(c, step);
}

lc_status lc_sgd_step_score(lc_ctx* c, int64_t step, const void* const* grads, int32_t grad_dtype,
                            const uint8_t* decay_mask, const lc_sgd_params* p) {
  lc::TraceRange trace_("lc_sgd_step_score");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  if (!p) return fail(LC_ERR_INVALID_ARG, "params must be non-NULL");
  if (!(p->lr >= 0.0) || !std::isfinite(p->lr)) return fail(LC_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (!(p->weight_decay >= 0.0) || !std::isfinite(p->weight_decay))
    return fail(LC_ERR_INVALID_ARG, "weight_decay must be finite and >= 0");
  st = optimizer_begin(c, step, grads, grad_dtype, decay_mask);
  if (st != LC_OK) return st;
  SgdScalars sc;
  sc.lr = static_cast<float>(p->lr);
  sc.decay = static_cast<float>(1.0 - p->lr * p->weight_decay);
  LC_HIP(c, launch_sgd(c->dt, grad_dtype, c->L.has_master ? 1 : 0, sc, c->stream));
  return optimizer_end(c, step);
}

lc_status lc_read_state(lc_ctx* c, double* u_out, double* delta_out, int64_t* t_last_out) {
  lc::TraceRange trace_("lc_read_state");
  lc_status st = check_ctx(c);
  if (st != LC_OK) return st;
  const size_t N = c->L.N;
  LC_HIP(c, hipStreamSynchronize(c->stream));
  if (u_out) LC_HIP(c, hipMemcpy(u_out, c->dt.u, N * sizeof(double), hipMemcpyDeviceToHost));
  if (delta_out) LC_HIP(c, hipMemcpy(delta_out, c->dt.delta, N * sizeof(double), hipMemcpyDeviceToHost));
  if (t_last_out) LC_HIP(c, hipMemcpy(t_last_out, c->dt.t_last, N * sizeof(int64_t), hipMemcpyDeviceToHost));
  return LC_OK;
}

uint64_t lc_record_bytes(const lc_ctx* c, uint32_t layer) {
  if (!c || layer >= c->L.N) return 0;
  return c->L.rec_bytes[layer];
}

lc_status lc_destroy(lc_ctx* c) {
  lc::TraceRange trace_("lc_destroy");
  if (!c) return LC_OK;
  hipError_t e = hipStreamSynchronize(c->stream);
  free_all(c);
  delete c;
  if (e != hipSuccess) return fail(LC_ERR_HIP, "stream synchronize failed: %s", hipGetErrorString(e));
  return LC_OK;
}

}  // extern "C"
