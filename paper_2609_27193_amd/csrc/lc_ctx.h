// Host-side state of a LayerCheck context, shared by the runtime
// (lc_runtime.cpp) and the persistence store (lc_store.cpp).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "layercheck.h"
#include "lc_internal.h"

namespace lc {

// Message of the last failing call on this thread (lc_last_error).
extern thread_local std::string g_error;

inline lc_status fail(lc_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return st;
}

// Host-side layout derived from a descriptor (no GPU work).
struct HostLayout {
  uint32_t N = 0;
  int dtype = 0;
  uint32_t esz = 0;
  bool has_master = false;
  std::vector<lc_segment> segs;
  std::vector<uint32_t> layer_seg_begin;  // [N+1]
  std::vector<uint64_t> numel;            // [N]
  std::vector<uint64_t> rec_bytes;        // [N]
  std::vector<uint64_t> layer_pieces;     // [N]
  std::vector<ScoreSeg> score_segs;
  std::vector<OptSeg> opt_segs;
  bool has_shadow = true;
  bool has_moments = true;
  std::vector<uint32_t> chunk_seg;
  std::vector<uint32_t> layer_chunk_begin;  // [N+1]
  std::vector<CopyUnit> units;
  std::vector<uint32_t> piece_unit;
  std::vector<uint64_t> layer_piece_begin;  // [N+1]
  uint64_t total_numel = 0;
};

}  // namespace lc

struct lc_ctx {
  using HostLayout = lc::HostLayout;
  using DeviceTables = lc::DeviceTables;
  using SelectHeader = lc::SelectHeader;
  using GradSeg = lc::GradSeg;
  HostLayout L;
  int mode = 0;
  int64_t s_max = 1;
  double eps_w = 0;
  int64_t t_base = 0;
  hipStream_t stream = nullptr;
  DeviceTables dt{};
  std::vector<void*> allocations;
  SelectHeader* h_result = nullptr;  // pinned, coherent: header + mask[N], written by the select kernel
  uint64_t result_seq = 0;           // sequence number of the last select kernel enqueued
  GradSeg* h_grad = nullptr;         // pinned: per-call gradient table
  GradSeg* d_grad = nullptr;
  hipEvent_t grad_event = nullptr;   // marks the upload of h_grad
  bool grad_event_pending = false;
  bool shadow_valid = false;         // S holds what the score pass expects

  // state machine
  bool poisoned = false;
  int64_t last_step = 0;
  bool scored = false;
  int64_t scored_step = 0;
  bool have_selection = false; // a selection (or the base) exists to pack
  bool pending = false;        // a selection whose records are not all packed
  bool pending_persists = false; // it came from lc_select or lc_rebase, which reset
                                 // Delta and t_l of its layers: it must be packed
  bool result_on_host = false; // h_result reflects the pending selection
  std::vector<uint32_t> sel;            // selected layers, ascending
  std::vector<uint64_t> sel_rec_prefix, sel_piece_prefix;
  std::vector<uint8_t> rank_packed;
  uint32_t n_unpacked = 0;
};


namespace lc {
// Restore helpers used by lc_restore_composite and the store.  The first
// enqueues the host-to-device copies of the bytes [rec_off, rec_off + len)
// of one layer's record, held at `bytes` in host memory, into the layer's
// arrays (only the parts of blocks inside the range, padding skipped) and
// refreshes the shadow from the copied weights; the whole record is
// [0, record bytes).  restore_finish sets Delta = 0, t_l = steps and the
// call-order state.
lc_status restore_range_from_host(lc_ctx* c, uint32_t layer, uint64_t rec_off, uint64_t len, const uint8_t* bytes);
// True when [p, p + bytes) is device (or managed) memory inside one
// allocation, as far as HIP can tell: pointers a kernel or a device copy
// could only fault on are refused before any work is enqueued.
bool device_range_ok(const void* p, uint64_t bytes);
lc_status restore_finish(lc_ctx* c, int64_t t_fail, const std::vector<int64_t>& steps);
}  // namespace lc
