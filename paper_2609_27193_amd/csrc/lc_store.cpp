// Persistence store: the durable side of selective persistence and the
// metadata-driven reconstruction of Section 3.5.
//
// A store is a directory of version files (one payload each: the records of
// the layers packed at one step, in the lc_pack_selected format) and an
// append-only manifest.  A version becomes visible only after its file is
// complete and fsync'ed and its manifest line is written and fsync'ed, so a
// crash leaves at most an ignored partial file.  Device payloads are drained
// through a ring of pinned host buffers on a store-owned stream; a small pool
// of writer threads writes each buffer as soon as its copy completes, so the
// caller's stream is released as soon as the staging buffer has been read.
// Versions are made durable in the order they were appended.
#include <dirent.h>
#include <fcntl.h>
#include <sys/file.h>
#include <sys/stat.h>
#include <sys/types.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <cstdlib>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "lc_ctx.h"
#include "lc_trace.h"

using namespace lc;

namespace {

constexpr int kWriters = 4;  // concurrent pwrite()s of drained buffers

struct StoredVersion {
  int64_t step = 0;
  std::vector<uint8_t> mask;
  uint64_t bytes = 0;
  std::string file;
  int fd = -1;              // open while being written
  int dfd = -1;             // the same file opened for direct I/O, or -1
  uint64_t remaining = 0;   // bytes not yet written (or abandoned)
  bool enqueued_all = false;
  bool failed = false;      // a write or the drain failed: the version is dropped
};

struct WriteJob {
  int fd = -1;
  int dfd = -1;                    // direct-I/O descriptor for block-aligned parts, or -1
  uint64_t file_off = 0;
  uint64_t len = 0;
  int slot = -1;                   // pinned ring slot, or -1 for a caller host buffer
  const uint8_t* host_src = nullptr;
  size_t version = 0;              // index into lc_store::writing
};

bool write_all(int fd, const uint8_t* p, uint64_t n, uint64_t off) {
  while (n > 0) {
    const ssize_t w = pwrite(fd, p, n > (1ull << 30) ? (1ull << 30) : n, static_cast<off_t>(off));
    if (w < 0) {
      if (errno == EINTR) continue;
      return false;
    }
    p += w;
    n -= static_cast<uint64_t>(w);
    off += static_cast<uint64_t>(w);
  }
  return true;
}

constexpr uint64_t kDirectBlock = 4096;  // O_DIRECT offset/length/address granule

// Writes the block-aligned head of a buffer with direct I/O (the data goes
// to the device, skipping the page cache) and the rest through the page
// cache; falls back to buffered writes if the file system refuses direct I/O.
bool write_slot(int fd, int dfd, const uint8_t* p, uint64_t n, uint64_t off) {
  uint64_t head = dfd >= 0 && off % kDirectBlock == 0 && reinterpret_cast<uintptr_t>(p) % kDirectBlock == 0
                      ? n / kDirectBlock * kDirectBlock
                      : 0;
  while (head > 0) {
    const uint64_t piece = head > (1ull << 30) ? (1ull << 30) : head;
    const ssize_t w = pwrite(dfd, p, piece, static_cast<off_t>(off));
    if (w < 0 && errno == EINTR) continue;
    if (w <= 0 || static_cast<uint64_t>(w) % kDirectBlock) {
      if (w > 0) {
        p += w, n -= static_cast<uint64_t>(w), off += static_cast<uint64_t>(w);
      }
      break;  // refused or short: the rest goes through the page cache
    }
    p += w, n -= static_cast<uint64_t>(w), off += static_cast<uint64_t>(w), head -= static_cast<uint64_t>(w);
  }
  return write_all(fd, p, n, off);
}

bool read_all(int fd, uint8_t* p, uint64_t n, uint64_t off) {
  while (n > 0) {
    const ssize_t r = pread(fd, p, n > (1ull << 30) ? (1ull << 30) : n, static_cast<off_t>(off));
    if (r < 0) {
      if (errno == EINTR) continue;
      return false;
    }
    if (r == 0) return false;
    p += r;
    n -= static_cast<uint64_t>(r);
    off += static_cast<uint64_t>(r);
  }
  return true;
}

std::string mask_string(const std::vector<uint8_t>& m) {
  std::string s(m.size(), '0');
  for (size_t i = 0; i < m.size(); ++i) s[i] = m[i] ? '1' : '0';
  return s;
}

std::string manifest_line(const StoredVersion& v) {
  return "LCV1 " + std::to_string(v.step) + " " + std::to_string(v.bytes) + " " + v.file + " " + mask_string(v.mask) +
         "\n";
}

// Makes the directory's entries (new files, renames, removals) durable.
bool fsync_dir(const std::string& dir) {
  const int fd = open(dir.c_str(), O_RDONLY | O_DIRECTORY);
  if (fd < 0) return false;
  const bool ok = fsync(fd) == 0;
  close(fd);
  return ok;
}

}  // namespace

struct lc_store {
  std::string dir;
  uint32_t N = 0;
  std::vector<uint64_t> R;
  std::vector<StoredVersion> durable;  // visible versions, manifest order
  std::vector<StoredVersion> writing;  // being written, append order (indices stay valid until idle)
  size_t next_final = 0;               // writing[] below this index are finalised
  bool finalising = false;             // one thread at a time makes versions durable
  int manifest_fd = -1;
  int lock_fd = -1;                    // holds the directory's exclusive lock while open
  uint64_t seq = 0;
  uint64_t skipped = 0;                // manifest lines ignored at open
  // drain pipeline
  uint64_t slot_bytes = 0;
  uint32_t n_slots = 0;
  bool gpu_ready = false;
  hipStream_t copy_stream = nullptr;
  hipEvent_t caller_ready = nullptr, copies_done = nullptr;
  std::vector<uint8_t*> slots;
  std::vector<hipEvent_t> slot_events;
  std::vector<int> slot_free;
  std::mutex mu;
  std::condition_variable cv;
  std::deque<WriteJob> queue;
  uint64_t outstanding = 0;            // jobs queued or being written
  bool stop = false;
  std::string writer_error;
  std::vector<std::thread> writers;
};

namespace {

// Makes a completed version durable: fsync its file and the directory entry,
// then append and fsync its manifest line.
std::string finalise(lc_store* s, const StoredVersion& v) {
  std::string err;
  if (v.dfd >= 0) close(v.dfd);
  if (fsync(v.fd) != 0) err = std::string("fsync failed: ") + std::strerror(errno);
  close(v.fd);
  if (err.empty() && !fsync_dir(s->dir)) err = std::string("directory fsync failed: ") + std::strerror(errno);
  if (!err.empty()) return err;
  const std::string line = manifest_line(v);
  const off_t end = lseek(s->manifest_fd, 0, SEEK_END);
  if (end < 0 ||
      !write_all(s->manifest_fd, reinterpret_cast<const uint8_t*>(line.data()), line.size(),
                 static_cast<uint64_t>(end)) ||
      fsync(s->manifest_fd) != 0)
    err = std::string("manifest write failed: ") + std::strerror(errno);
  return err;
}

bool complete(const StoredVersion& v) { return v.enqueued_all && v.remaining == 0; }

// Finalises complete versions in append order, so the manifest lists them in
// the order they were appended.  Called with s->mu held; drops it around the
// file system calls.  Only one thread finalises at a time; a version that
// completes meanwhile is picked up by that thread's next check.
void advance(lc_store* s, std::unique_lock<std::mutex>& lk) {
  if (s->finalising) return;
  s->finalising = true;
  while (s->next_final < s->writing.size() && complete(s->writing[s->next_final])) {
    const StoredVersion v = s->writing[s->next_final];
    lk.unlock();
    std::string err;
    if (v.failed) {
      close(v.fd);
      if (v.dfd >= 0) close(v.dfd);
    }
    else err = finalise(s, v);
    lk.lock();
    if (!err.empty() && s->writer_error.empty()) s->writer_error = err;
    if (err.empty() && !v.failed) s->durable.push_back(v);
    s->writing[s->next_final].fd = -1;
    ++s->next_final;
  }
  s->finalising = false;
}

void writer_loop(lc_store* s) {
  // Direct I/O cannot read pinned (device-mapped) host memory, so each writer
  // copies a drained slot into an ordinary page-aligned buffer of its own,
  // frees the slot at once and writes from there.
  uint8_t* bounce = nullptr;
  for (;;) {
    WriteJob job;
    {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv.wait(lk, [&] { return s->stop || !s->queue.empty(); });
      if (s->queue.empty()) break;
      job = s->queue.front();
      s->queue.pop_front();
    }
    std::string err;
    const uint8_t* src = job.host_src;
    int dfd = -1;
    bool slot_held = job.slot >= 0;
    if (slot_held) {
      const hipError_t e = hipEventSynchronize(s->slot_events[job.slot]);
      if (e != hipSuccess) err = std::string("device-to-host copy failed: ") + hipGetErrorString(e);
      src = s->slots[job.slot];
      if (err.empty() && job.dfd >= 0 && !bounce) {
        void* p = nullptr;
        if (posix_memalign(&p, kDirectBlock, s->slot_bytes) == 0) bounce = static_cast<uint8_t*>(p);
      }
      if (err.empty() && job.dfd >= 0 && bounce) {
        std::memcpy(bounce, src, job.len);
        src = bounce;
        dfd = job.dfd;
        {
          std::lock_guard<std::mutex> lk(s->mu);
          s->slot_free[job.slot] = 1;
        }
        s->cv.notify_all();
        slot_held = false;
      }
    }
    if (err.empty() && job.len && !write_slot(job.fd, dfd, src, job.len, job.file_off))
      err = std::string("write failed: ") + std::strerror(errno);
    std::unique_lock<std::mutex> lk(s->mu);
    StoredVersion& w = s->writing[job.version];
    w.remaining -= job.len;
    if (!err.empty()) {
      w.failed = true;
      if (s->writer_error.empty()) s->writer_error = err;
    }
    if (slot_held) s->slot_free[job.slot] = 1;
    advance(s, lk);
    --s->outstanding;
    lk.unlock();
    s->cv.notify_all();
  }
  free(bounce);
}

// An append that fails after registering its version: the bytes it did not
// queue are written off and the version is dropped once its queued writes end.
void abandon(lc_store* s, size_t vi, uint64_t unqueued, const char* why) {
  std::unique_lock<std::mutex> lk(s->mu);
  StoredVersion& w = s->writing[vi];
  w.remaining -= unqueued;
  w.enqueued_all = true;
  w.failed = true;
  if (s->writer_error.empty()) s->writer_error = why;
  ++s->outstanding;  // the in-line advance below counts as a job
  advance(s, lk);
  --s->outstanding;
  lk.unlock();
  s->cv.notify_all();
}

lc_status parse_manifest(lc_store* s) {
  std::string text;
  {
    char buf[1 << 16];
    for (;;) {
      const ssize_t r = read(s->manifest_fd, buf, sizeof(buf));
      if (r < 0) {
        if (errno == EINTR) continue;
        return fail(LC_ERR_IO, "cannot read the manifest: %s", std::strerror(errno));
      }
      if (r == 0) break;
      text.append(buf, static_cast<size_t>(r));
    }
  }
  size_t pos = 0;
  while (pos < text.size()) {
    const size_t nl = text.find('\n', pos);
    if (nl == std::string::npos) {  // torn last line: never durable, cut it off
      ++s->skipped;
      if (ftruncate(s->manifest_fd, static_cast<off_t>(pos)) != 0 || fsync(s->manifest_fd) != 0)
        return fail(LC_ERR_IO, "cannot repair the manifest: %s", std::strerror(errno));
      break;
    }
    const std::string line = text.substr(pos, nl - pos);
    pos = nl + 1;
    char tag[8] = {0}, file[256] = {0};
    long long step = 0;
    unsigned long long bytes = 0;
    if (s->N > (1u << 20) ||
        sscanf(line.c_str(), "%7s %lld %llu %255s", tag, &step, &bytes, file) != 4 || std::strcmp(tag, "LCV1")) {
      ++s->skipped;
      continue;
    }
    const size_t mp = line.rfind(' ');
    const std::string ms = mp == std::string::npos ? "" : line.substr(mp + 1);
    if (ms.size() != s->N) {
      ++s->skipped;
      continue;
    }
    StoredVersion v;
    v.step = step;
    v.bytes = bytes;
    v.file = file;
    // only a plain name of this store's own version files: a damaged line must
    // never lead a restore or a removal outside the directory
    if (v.file.find('/') != std::string::npos || v.file.size() < 5 ||
        v.file.compare(v.file.size() - 4, 4, ".lcr") != 0 || v.file[0] != 'v') {
      ++s->skipped;
      continue;
    }
    v.mask.resize(s->N);
    uint64_t need = 0;
    bool ok = true;
    for (uint32_t l = 0; l < s->N; ++l) {
      if (ms[l] != '0' && ms[l] != '1') ok = false;
      v.mask[l] = ms[l] == '1';
      if (v.mask[l]) need += s->R[l];
    }
    struct stat sb;
    const std::string path = s->dir + "/" + v.file;
    if (!ok || need != v.bytes || stat(path.c_str(), &sb) != 0 || static_cast<uint64_t>(sb.st_size) != v.bytes) {
      ++s->skipped;
      continue;
    }
    unsigned long long q = 0;
    if (sscanf(v.file.c_str(), "v%llu_", &q) == 1) s->seq = std::max<uint64_t>(s->seq, q + 1);
    s->durable.push_back(v);
  }
  return LC_OK;
}

// Releases the drain ring and its stream (nothing may be in flight on them).
void release_gpu(lc_store* s) {
  for (uint8_t* p : s->slots) (void)hipHostFree(p);
  for (hipEvent_t e : s->slot_events) (void)hipEventDestroy(e);
  if (s->caller_ready) (void)hipEventDestroy(s->caller_ready);
  if (s->copies_done) (void)hipEventDestroy(s->copies_done);
  if (s->copy_stream) (void)hipStreamDestroy(s->copy_stream);
  s->slots.clear();
  s->slot_events.clear();
  s->slot_free.clear();
  s->caller_ready = s->copies_done = nullptr;
  s->copy_stream = nullptr;
  s->gpu_ready = false;
}

// The drain ring and its stream, set up on the first device append; a failed
// set-up releases what it created, so a later append can try again.
lc_status ensure_gpu(lc_store* s) {
  if (s->gpu_ready) return LC_OK;
  hipError_t e = hipStreamCreateWithFlags(&s->copy_stream, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->caller_ready, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->copies_done, hipEventDisableTiming);
  if (e != hipSuccess) {
    release_gpu(s);
    return fail(LC_ERR_HIP, "store stream setup failed: %s", hipGetErrorString(e));
  }
  for (uint32_t k = 0; k < s->n_slots; ++k) {
    void* p = nullptr;
    e = hipHostMalloc(&p, s->slot_bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
      release_gpu(s);
      return fail(LC_ERR_OOM, "pinned drain buffer: %s", hipGetErrorString(e));
    }
    s->slots.push_back(static_cast<uint8_t*>(p));
    hipEvent_t ev = nullptr;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) {
      release_gpu(s);
      return fail(LC_ERR_HIP, "event create failed: %s", hipGetErrorString(e));
    }
    s->slot_events.push_back(ev);
    s->slot_free.push_back(1);
  }
  s->gpu_ready = true;
  return LC_OK;
}

// Per layer, the index of the durable version it is restored from (Section 3.5).
lc_status plan_store(lc_store* s, int64_t t_fail, std::vector<size_t>& choice) {
  choice.assign(s->N, 0);
  for (uint32_t l = 0; l < s->N; ++l) {
    long best = -1;
    bool dup = false;
    for (size_t i = 0; i < s->durable.size(); ++i) {
      const StoredVersion& v = s->durable[i];
      if (v.step > t_fail || !v.mask[l]) continue;
      if (best < 0 || v.step > s->durable[best].step) {
        best = static_cast<long>(i);
        dup = false;
      } else if (v.step == s->durable[best].step) {
        dup = true;
      }
    }
    if (best < 0)
      return fail(LC_ERR_NO_VERSION, "layer %u: no persisted version at step <= %lld", l,
                  static_cast<long long>(t_fail));
    if (dup) return fail(LC_ERR_INVALID_ARG, "layer %u: two stored versions at one step", l);
    choice[l] = static_cast<size_t>(best);
  }
  return LC_OK;
}

lc_status wait_idle(lc_store* s) {
  std::unique_lock<std::mutex> lk(s->mu);
  s->cv.wait(lk, [&] { return s->outstanding == 0 && s->next_final == s->writing.size(); });
  s->writing.clear();
  s->next_final = 0;
  if (!s->writer_error.empty()) return fail(LC_ERR_IO, "store failed: %s", s->writer_error.c_str());
  return LC_OK;
}

// Keeps the visible versions flagged in `keep` and removes the rest, plus any
// version file no manifest line names (a crash between a manifest rewrite and
// the removals, or a version that never became visible: nothing is in flight
// once the store is idle).  The new manifest replaces the old one atomically
// (temporary file, fsync, rename, directory fsync) before any file goes.
lc_status keep_only(lc_store* s, const std::vector<uint8_t>& keep, uint32_t* removed_out) {
  const size_t n = s->durable.size();
  std::vector<StoredVersion> kept;
  std::vector<std::string> gone;
  for (size_t i = 0; i < n; ++i) {
    if (keep[i]) kept.push_back(s->durable[i]);
    else gone.push_back(s->durable[i].file);
  }
  if (DIR* dp = opendir(s->dir.c_str())) {
    std::vector<std::string> named;
    for (const StoredVersion& v : s->durable) named.push_back(v.file);
    while (dirent* e = readdir(dp)) {
      const std::string f = e->d_name;
      if (f.size() > 4 && f.compare(f.size() - 4, 4, ".lcr") == 0 &&
          std::find(named.begin(), named.end(), f) == named.end())
        gone.push_back(f);
    }
    closedir(dp);
  }
  if (gone.empty()) return LC_OK;
  if (kept.size() != n) {
    const std::string mpath = s->dir + "/manifest.lcm", tpath = s->dir + "/manifest.lcm.tmp";
    // the descriptor of the new file becomes the manifest's once renamed
    const int fd = open(tpath.c_str(), O_RDWR | O_CREAT | O_TRUNC, 0644);
    if (fd < 0) return fail(LC_ERR_IO, "cannot create %s: %s", tpath.c_str(), std::strerror(errno));
    std::string text;
    for (const StoredVersion& v : kept) text += manifest_line(v);
    if (!write_all(fd, reinterpret_cast<const uint8_t*>(text.data()), text.size(), 0) || fsync(fd) != 0 ||
        rename(tpath.c_str(), mpath.c_str()) != 0) {
      const int err = errno;
      close(fd);
      (void)unlink(tpath.c_str());
      return fail(LC_ERR_IO, "rewriting the manifest failed: %s", std::strerror(err));
    }
    close(s->manifest_fd);
    s->manifest_fd = fd;
    s->durable = kept;
    if (!fsync_dir(s->dir))
      return fail(LC_ERR_IO, "directory fsync after the manifest rewrite failed: %s", std::strerror(errno));
  }
  uint32_t removed = 0;
  for (const std::string& f : gone)
    if (unlink((s->dir + "/" + f).c_str()) == 0) ++removed;
  (void)fsync_dir(s->dir);
  if (removed_out) *removed_out = removed;
  return LC_OK;
}

// Reads the chosen record of every layer and restores it (Section 3.5 steps
// 2-3) as one pipeline over fixed 64 MiB pieces of the records, in layer
// order: reader threads fill a ring of pinned slots, each as soon as the
// copies out of its previous piece have completed; the calling thread
// enqueues each piece's host-to-device copies (the parts of the array blocks
// the piece holds) as soon as it has been read, then records the slot's
// event.  Neither the disk nor the host link waits for a layer boundary.
lc_status restore_pipeline(lc_store* s, lc_ctx* c, const std::vector<size_t>& choice,
                           const std::vector<uint64_t>& off, std::map<size_t, int>& fds) {
  constexpr uint64_t kPiece = 64ull << 20;
  constexpr uint32_t kSlots = 32;  // 2 GiB of pinned read-ahead
  constexpr unsigned kReaders = 8;
  struct Piece { int fd; uint64_t src; uint32_t layer; uint64_t rec_off, len; };
  std::vector<Piece> pieces;
  for (uint32_t l = 0; l < s->N; ++l)
    for (uint64_t o = 0; o < s->R[l]; o += kPiece)
      pieces.push_back({fds[choice[l]], off[l] + o, l, o, std::min<uint64_t>(kPiece, s->R[l] - o)});
  const size_t np = pieces.size();
  uint8_t* ring = nullptr;
  {
    void* p = nullptr;
    const hipError_t e = hipHostMalloc(&p, kSlots * kPiece, hipHostMallocDefault);
    if (e != hipSuccess) return fail(LC_ERR_OOM, "pinned restore ring: %s", hipGetErrorString(e));
    ring = static_cast<uint8_t*>(p);
  }
  std::vector<hipEvent_t> ev(kSlots, nullptr);
  for (auto& e : ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
      for (auto& x : ev)
        if (x) (void)hipEventDestroy(x);
      (void)hipHostFree(ring);
      return fail(LC_ERR_HIP, "event create failed");
    }
  std::mutex mu;
  std::condition_variable cv;
  std::vector<uint8_t> read_done(np, 0), issued(np, 0);
  size_t next_piece = 0;
  bool stop = false, failed = false;
  std::vector<std::thread> readers;
  for (unsigned r = 0; r < kReaders; ++r)
    readers.emplace_back([&] {
      for (;;) {
        size_t j;
        {
          std::unique_lock<std::mutex> lk(mu);
          if (stop || next_piece >= np) return;
          j = next_piece++;
          // the slot is free once the copies out of piece j - kSlots are done
          if (j >= kSlots) cv.wait(lk, [&] { return stop || issued[j - kSlots]; });
          if (stop) return;
        }
        bool ok = j < kSlots || hipEventSynchronize(ev[j % kSlots]) == hipSuccess;
        const Piece& pc = pieces[j];
        ok = ok && read_all(pc.fd, ring + (j % kSlots) * kPiece, pc.len, pc.src);
        {
          std::lock_guard<std::mutex> lk(mu);
          if (ok) read_done[j] = 1;
          else failed = true;
        }
        cv.notify_all();
      }
    });
  lc_status st = LC_OK;
  for (size_t i = 0; i < np && st == LC_OK; ++i) {
    {
      std::unique_lock<std::mutex> lk(mu);
      cv.wait(lk, [&] { return failed || read_done[i]; });
      if (!read_done[i]) {
        st = fail(LC_ERR_IO, "reading a stored record failed");
        break;
      }
    }
    const Piece& pc = pieces[i];
    st = restore_range_from_host(c, pc.layer, pc.rec_off, pc.len, ring + (i % kSlots) * kPiece);
    if (st != LC_OK) break;
    if (hipEventRecord(ev[i % kSlots], c->stream) != hipSuccess) {
      c->poisoned = true;
      st = fail(LC_ERR_HIP, "event record failed");
      break;
    }
    {
      std::lock_guard<std::mutex> lk(mu);
      issued[i] = 1;
    }
    cv.notify_all();
  }
  {
    std::lock_guard<std::mutex> lk(mu);
    stop = true;
  }
  cv.notify_all();
  for (auto& th : readers) th.join();
  // the ring must outlive every copy that reads it
  if (hipStreamSynchronize(c->stream) != hipSuccess && st == LC_OK) {
    c->poisoned = true;
    st = fail(LC_ERR_HIP, "restore copies failed");
  }
  for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  (void)hipHostFree(ring);
  return st;
}

}  // namespace

extern "C" {

lc_status lc_store_open(const char* dir, uint32_t n_layers, const uint64_t* record_bytes, uint64_t buffer_bytes,
                        lc_store** out) {
  lc::TraceRange trace_("lc_store_open");
  if (!out) return fail(LC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!dir || !*dir || n_layers == 0 || !record_bytes) return fail(LC_ERR_INVALID_ARG, "bad store arguments");
  for (uint32_t l = 0; l < n_layers; ++l)
    if (record_bytes[l] == 0 || record_bytes[l] % kRecordAlign)
      return fail(LC_ERR_INVALID_ARG, "record_bytes[%u] must be a positive multiple of %u", l, kRecordAlign);
  if (mkdir(dir, 0755) != 0 && errno != EEXIST)
    return fail(LC_ERR_IO, "cannot create %s: %s", dir, std::strerror(errno));
  lc_store* s = new (std::nothrow) lc_store();
  if (!s) return fail(LC_ERR_OOM, "host allocation failed");
  s->dir = dir;
  s->N = n_layers;
  s->R.assign(record_bytes, record_bytes + n_layers);
  // the ring: buffer_bytes of pinned memory in slots of at most 64 MiB, at
  // least 2 per writer so copies run ahead of the writes
  const uint64_t ring = std::max<uint64_t>(buffer_bytes ? buffer_bytes : (1ull << 30), 1ull << 20);
  s->slot_bytes = std::min<uint64_t>(64ull << 20, ring / (2 * kWriters));
  s->slot_bytes = (s->slot_bytes + 4095) / 4096 * 4096;
  s->n_slots = static_cast<uint32_t>(std::max<uint64_t>(2 * kWriters, ring / s->slot_bytes));
  // One writer per directory: a lock on a file that is never replaced (the
  // manifest itself is, by compaction), held until lc_store_close.
  const std::string lpath = s->dir + "/store.lock";
  s->lock_fd = open(lpath.c_str(), O_RDWR | O_CREAT, 0644);
  if (s->lock_fd < 0) {
    delete s;
    return fail(LC_ERR_IO, "cannot open %s: %s", lpath.c_str(), std::strerror(errno));
  }
  if (flock(s->lock_fd, LOCK_EX | LOCK_NB) != 0) {
    const int err = errno;
    close(s->lock_fd);
    delete s;
    if (err == EWOULDBLOCK)
      return fail(LC_ERR_BAD_STATE, "store %s is already open (another store holds its lock)", dir);
    return fail(LC_ERR_IO, "cannot lock %s: %s", lpath.c_str(), std::strerror(err));
  }
  const std::string mpath = s->dir + "/manifest.lcm";
  s->manifest_fd = open(mpath.c_str(), O_RDWR | O_CREAT, 0644);
  if (s->manifest_fd < 0) {
    close(s->lock_fd);
    delete s;
    return fail(LC_ERR_IO, "cannot open %s: %s", mpath.c_str(), std::strerror(errno));
  }
  lc_status st = parse_manifest(s);
  if (st != LC_OK) {
    close(s->manifest_fd);
    close(s->lock_fd);
    delete s;
    return st;
  }
  for (int i = 0; i < kWriters; ++i) s->writers.emplace_back(writer_loop, s);
  *out = s;
  return LC_OK;
}

}  // extern "C"

namespace {

// Both appends.  caller_waits: `stream` waits for the copies out of a device
// payload (lc_store_append); otherwise `reuse_event` is recorded behind them
// on the store's stream and `stream` runs on (lc_store_append_async).
lc_status append_impl(lc_store* s, int64_t step, const uint8_t* mask, const void* payload, uint64_t bytes,
                      void* stream, bool caller_waits, void* reuse_event) {
  if (!s || !mask) return fail(LC_ERR_INVALID_ARG, "store and mask must be non-NULL");
  StoredVersion v;
  v.step = step;
  v.bytes = bytes;
  v.mask.assign(mask, mask + s->N);
  uint64_t need = 0;
  for (uint32_t l = 0; l < s->N; ++l) {
    if (mask[l] > 1) return fail(LC_ERR_INVALID_ARG, "mask must be 0/1");
    if (mask[l]) need += s->R[l];
  }
  if (need != bytes)
    return fail(LC_ERR_INVALID_ARG, "payload_bytes %llu != %llu for the mask",
                static_cast<unsigned long long>(bytes), static_cast<unsigned long long>(need));
  if (bytes && !payload) return fail(LC_ERR_INVALID_ARG, "payload is NULL");
  {
    std::lock_guard<std::mutex> lk(s->mu);
    if (!s->writer_error.empty()) return fail(LC_ERR_IO, "store failed earlier: %s", s->writer_error.c_str());
    for (const auto* list : {&s->durable, &s->writing})
      for (const StoredVersion& o : *list)
        if (o.step == step)
          for (uint32_t l = 0; l < s->N; ++l)
            if (o.mask[l] && mask[l]) return fail(LC_ERR_INVALID_ARG, "layer %u already stored at this step", l);
  }
  bool device = false;
  if (bytes) {
    hipPointerAttribute_t attr;
    const hipError_t e = hipPointerGetAttributes(&attr, payload);
    if (e == hipSuccess && attr.type == hipMemoryTypeDevice) device = true;
    else (void)hipGetLastError();
  }
  if (device && !device_range_ok(payload, bytes))
    return fail(LC_ERR_INVALID_ARG, "the device payload is shorter than payload_bytes");
  if (device && !caller_waits && !reuse_event)
    return fail(LC_ERR_INVALID_ARG, "a device payload needs reuse_event");
  char name[96];
  snprintf(name, sizeof(name), "v%010llu_s%lld.lcr", static_cast<unsigned long long>(s->seq++),
           static_cast<long long>(step));
  v.file = name;
  const std::string path = s->dir + "/" + v.file;
  const int fd = open(path.c_str(), O_WRONLY | O_CREAT | O_TRUNC, 0644);
  if (fd < 0) return fail(LC_ERR_IO, "cannot create %s: %s", path.c_str(), std::strerror(errno));
  size_t vi;
  v.fd = fd;
  // device payloads leave the pinned ring by direct I/O where the file system allows it
  v.dfd = device ? open(path.c_str(), O_WRONLY | O_DIRECT) : -1;
  v.remaining = bytes;
  v.enqueued_all = !device;
  {
    std::lock_guard<std::mutex> lk(s->mu);
    vi = s->writing.size();
    s->writing.push_back(v);
  }
  if (!device) {
    // host payload (or empty): written from the caller's buffer, in pieces
    // the writers share, before returning
    constexpr uint64_t kPiece = 64ull << 20;
    {
      std::lock_guard<std::mutex> lk(s->mu);
      uint64_t off = 0;
      do {
        WriteJob job;
        job.fd = fd;
        job.file_off = off;
        job.len = std::min<uint64_t>(kPiece, bytes - off);
        job.host_src = static_cast<const uint8_t*>(payload) + off;
        job.version = vi;
        s->queue.push_back(job);
        ++s->outstanding;
        off += job.len;
      } while (off < bytes);
    }
    s->cv.notify_all();
    lc_status st = wait_idle(s);
    if (st == LC_OK && !caller_waits && reuse_event) {
      // the payload was written before this call returns: the event only
      // has to follow the caller's work
      const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(reuse_event), static_cast<hipStream_t>(stream));
      if (e != hipSuccess) return fail(LC_ERR_HIP, "event record failed: %s", hipGetErrorString(e));
    }
    return st;
  }
  lc_status st = ensure_gpu(s);
  if (st != LC_OK) {
    abandon(s, vi, bytes, "drain buffers could not be set up");
    return st;
  }
  hipStream_t cs = static_cast<hipStream_t>(stream);
  hipError_t e = hipEventRecord(s->caller_ready, cs);
  if (e == hipSuccess) e = hipStreamWaitEvent(s->copy_stream, s->caller_ready, 0);
  if (e != hipSuccess) {
    abandon(s, vi, bytes, "stream ordering failed");
    return fail(LC_ERR_HIP, "stream ordering failed: %s", hipGetErrorString(e));
  }
  const uint8_t* src = static_cast<const uint8_t*>(payload);
  for (uint64_t off = 0; off < bytes; off += s->slot_bytes) {
    const uint64_t len = std::min<uint64_t>(s->slot_bytes, bytes - off);
    int slot = -1;
    {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv.wait(lk, [&] {
        if (!s->writer_error.empty()) return true;
        for (uint32_t k = 0; k < s->n_slots; ++k)
          if (s->slot_free[k]) return true;
        return false;
      });
      if (!s->writer_error.empty()) {
        const std::string why = s->writer_error;
        lk.unlock();
        abandon(s, vi, bytes - off, why.c_str());
        (void)hipStreamSynchronize(s->copy_stream);  // nothing reads the payload after an error return
        return fail(LC_ERR_IO, "store: %s", why.c_str());
      }
      for (uint32_t k = 0; k < s->n_slots; ++k)
        if (s->slot_free[k]) {
          slot = static_cast<int>(k);
          s->slot_free[k] = 0;
          break;
        }
    }
    e = hipMemcpyAsync(s->slots[slot], src + off, len, hipMemcpyDeviceToHost, s->copy_stream);
    if (e == hipSuccess) e = hipEventRecord(s->slot_events[slot], s->copy_stream);
    if (e != hipSuccess) {
      {
        std::lock_guard<std::mutex> lk(s->mu);
        s->slot_free[slot] = 1;  // nothing was queued on it
      }
      abandon(s, vi, bytes - off, "drain copy failed");
      (void)hipStreamSynchronize(s->copy_stream);  // nothing reads the payload after an error return
      return fail(LC_ERR_HIP, "drain copy failed: %s", hipGetErrorString(e));
    }
    WriteJob job;
    job.fd = fd;
    job.dfd = v.dfd;
    job.file_off = off;
    job.len = len;
    job.slot = slot;
    job.version = vi;
    {
      std::lock_guard<std::mutex> lk(s->mu);
      if (off + len == bytes) s->writing[vi].enqueued_all = true;
      s->queue.push_back(job);
      ++s->outstanding;
    }
    s->cv.notify_all();
  }
  if (caller_waits) {
    // the caller's later work (the next pack into the same staging) waits for the copies
    e = hipEventRecord(s->copies_done, s->copy_stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(cs, s->copies_done, 0);
  } else {
    e = hipEventRecord(static_cast<hipEvent_t>(reuse_event), s->copy_stream);
  }
  if (e != hipSuccess) {
    (void)hipStreamSynchronize(s->copy_stream);
    return fail(LC_ERR_HIP, "stream ordering failed: %s", hipGetErrorString(e));
  }
  return LC_OK;
}

}  // namespace

extern "C" {

lc_status lc_store_append(lc_store* s, int64_t step, const uint8_t* mask, const void* payload, uint64_t bytes,
                          void* stream) {
  lc::TraceRange trace_("lc_store_append");
  return append_impl(s, step, mask, payload, bytes, stream, true, nullptr);
}

lc_status lc_store_append_async(lc_store* s, int64_t step, const uint8_t* mask, const void* payload,
                                uint64_t bytes, void* stream, void* reuse_event) {
  lc::TraceRange trace_("lc_store_append_async");
  return append_impl(s, step, mask, payload, bytes, stream, false, reuse_event);
}

lc_status lc_store_sync(lc_store* s) {
  lc::TraceRange trace_("lc_store_sync");
  if (!s) return fail(LC_ERR_INVALID_ARG, "store is NULL");
  return wait_idle(s);
}

lc_status lc_store_count(lc_store* s, uint32_t* n_out) {
  if (!s || !n_out) return fail(LC_ERR_INVALID_ARG, "bad arguments");
  std::lock_guard<std::mutex> lk(s->mu);
  *n_out = static_cast<uint32_t>(s->durable.size());
  return LC_OK;
}

lc_status lc_store_entry(lc_store* s, uint32_t i, int64_t* step_out, uint8_t* mask_out, uint64_t* bytes_out) {
  if (!s) return fail(LC_ERR_INVALID_ARG, "store is NULL");
  std::lock_guard<std::mutex> lk(s->mu);
  if (i >= s->durable.size()) return fail(LC_ERR_INVALID_ARG, "entry %u out of range", i);
  const StoredVersion& v = s->durable[i];
  if (step_out) *step_out = v.step;
  if (mask_out) std::memcpy(mask_out, v.mask.data(), s->N);
  if (bytes_out) *bytes_out = v.bytes;
  return LC_OK;
}

lc_status lc_store_plan(lc_store* s, int64_t t_fail, int64_t* chosen_step_out) {
  if (!s) return fail(LC_ERR_INVALID_ARG, "store is NULL");
  lc_status st = wait_idle(s);
  if (st != LC_OK) return st;
  std::vector<size_t> choice;
  st = plan_store(s, t_fail, choice);
  if (st != LC_OK) return st;
  if (chosen_step_out)
    for (uint32_t l = 0; l < s->N; ++l) chosen_step_out[l] = s->durable[choice[l]].step;
  return LC_OK;
}

lc_status lc_store_restore(lc_store* s, lc_ctx* c, int64_t t_fail, int64_t* chosen_step_out) {
  lc::TraceRange trace_("lc_store_restore");
  if (!s || !c) return fail(LC_ERR_INVALID_ARG, "store and context must be non-NULL");
  if (c->poisoned) return fail(LC_ERR_BAD_STATE, "context is poisoned by an earlier HIP error");
  if (c->L.N != s->N || c->L.rec_bytes != s->R)
    return fail(LC_ERR_INVALID_ARG, "the context's layout differs from the store's");
  lc_status st = wait_idle(s);
  if (st != LC_OK) return st;
  std::vector<size_t> choice;
  st = plan_store(s, t_fail, choice);
  if (st != LC_OK) return st;
  // offset of each layer's record inside its chosen version file
  std::vector<uint64_t> off(s->N, 0);
  for (uint32_t l = 0; l < s->N; ++l) {
    const StoredVersion& v = s->durable[choice[l]];
    uint64_t o = 0;
    for (uint32_t j = 0; j < l; ++j)
      if (v.mask[j]) o += s->R[j];
    off[l] = o;
  }
  std::map<size_t, int> fds;
  for (size_t i : choice) {
    if (fds.count(i)) continue;
    const std::string path = s->dir + "/" + s->durable[i].file;
    const int fd = open(path.c_str(), O_RDONLY);
    if (fd < 0) {
      for (auto& kv : fds) close(kv.second);
      return fail(LC_ERR_IO, "cannot open %s: %s", path.c_str(), std::strerror(errno));
    }
    fds[i] = fd;
  }
  st = restore_pipeline(s, c, choice, off, fds);
  for (auto& kv : fds) close(kv.second);
  if (st != LC_OK) return st;
  std::vector<int64_t> steps(s->N);
  for (uint32_t j = 0; j < s->N; ++j) steps[j] = s->durable[choice[j]].step;
  st = restore_finish(c, t_fail, steps);
  if (st != LC_OK) return st;
  if (chosen_step_out) std::memcpy(chosen_step_out, steps.data(), s->N * sizeof(int64_t));
  return LC_OK;
}

lc_status lc_store_compact(lc_store* s, int64_t t_keep, uint32_t* removed_out) {
  lc::TraceRange trace_("lc_store_compact");
  if (removed_out) *removed_out = 0;
  if (!s) return fail(LC_ERR_INVALID_ARG, "store is NULL");
  lc_status st = wait_idle(s);
  if (st != LC_OK) return st;
  // needed: every non-empty version after t_keep, and per layer the newest
  // version at or before t_keep holding it
  const size_t n = s->durable.size();
  std::vector<uint8_t> keep(n, 0);
  for (size_t i = 0; i < n; ++i) {
    const StoredVersion& v = s->durable[i];
    if (v.step > t_keep)
      for (uint32_t l = 0; l < s->N && !keep[i]; ++l) keep[i] = v.mask[l];
  }
  for (uint32_t l = 0; l < s->N; ++l) {
    long best = -1;
    for (size_t i = 0; i < n; ++i) {
      const StoredVersion& v = s->durable[i];
      if (v.step <= t_keep && v.mask[l] && (best < 0 || v.step > s->durable[best].step)) best = static_cast<long>(i);
    }
    if (best >= 0) keep[best] = 1;
  }
  return keep_only(s, keep, removed_out);
}

lc_status lc_store_discard_after(lc_store* s, int64_t step, uint32_t* removed_out) {
  lc::TraceRange trace_("lc_store_discard_after");
  if (removed_out) *removed_out = 0;
  if (!s) return fail(LC_ERR_INVALID_ARG, "store is NULL");
  lc_status st = wait_idle(s);
  if (st != LC_OK) return st;
  std::vector<uint8_t> keep(s->durable.size(), 0);
  for (size_t i = 0; i < keep.size(); ++i) keep[i] = s->durable[i].step <= step;
  return keep_only(s, keep, removed_out);
}

lc_status lc_store_close(lc_store* s) {
  lc::TraceRange trace_("lc_store_close");
  if (!s) return LC_OK;
  lc_status st = wait_idle(s);
  {
    std::lock_guard<std::mutex> lk(s->mu);
    s->stop = true;
  }
  s->cv.notify_all();
  for (auto& w : s->writers)
    if (w.joinable()) w.join();
  if (s->gpu_ready) {
    (void)hipStreamSynchronize(s->copy_stream);
    release_gpu(s);
  }
  if (s->manifest_fd >= 0) close(s->manifest_fd);
  if (s->lock_fd >= 0) close(s->lock_fd);  // releases the directory
  delete s;
  return st;
}

}  // extern "C"
