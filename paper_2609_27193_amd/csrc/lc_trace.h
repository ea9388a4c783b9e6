// Optional roctx ranges around the library's entry points, so a profiler's
// marker trace (rocprofv3 --marker-trace) shows each call's host span beside
// the kernels it enqueues.  Off unless the environment sets
// LAYERCHECK_ROCTX=1 when the first range is opened; the roctx library is
// then loaded at run time (dlopen), so the library neither links against it
// nor pays more than a branch per call while tracing is off.  Ranges nest
// per host thread, as roctx ranges do.
#pragma once

namespace lc {

class TraceRange {
 public:
  explicit TraceRange(const char* name);
  ~TraceRange();
  TraceRange(const TraceRange&) = delete;
  TraceRange& operator=(const TraceRange&) = delete;

 private:
  bool on_;
};

}  // namespace lc
