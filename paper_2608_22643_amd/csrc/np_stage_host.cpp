// np_stage_host.cpp -- staging through pinned host memory (Sec. 3.5, I/O
// path): incoming ids are walked layer by layer in ascending order, adjacent
// ids are coalesced into one contiguous source range, records are packed
// into a capacity-bounded pinned staging area, and each packed piece (its
// records followed by their destination rows) goes to the device with one
// hipMemcpyAsync on the side stream; a kernel on another stream then
// scatters the landed records into their slots.  The staging area is a ring
// of pieces so that packing one piece overlaps the copy of the previous
// ones, and the landing area is a ring of landed pieces, so the copies run
// back to back on the copy engine, with no kernel between two of them; a
// delta larger than the landing area wraps the ring.  The source is
// the storage tier in host memory (np_stage_rows: the ranges are copied by a
// thread pool) or in a file (np_stage_file: the ranges are read through
// io_uring, np_file.cpp).
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <map>
#include <condition_variable>
#include <mutex>
#include <thread>
#include <vector>

#include "np_internal.hpp"

namespace np {

// Persistent worker pool for the host pack (memcpy of coalesced runs).  One
// pool per process; concurrent callers take turns (run() holds a lock), so
// two pipelines staging at once share the packing threads.  Between jobs the
// workers spin on the job counter for a while before they sleep, so the next
// piece's job starts within a microsecond instead of a thread wake-up (a
// token's staging runs a few dozen jobs in quick succession).
class PackPool {
 public:
  struct Task {
    char* dst;
    const char* src;
    size_t n;
  };

  explicit PackPool(int nthreads) {
    for (int i = 0; i < nthreads; ++i) workers_.emplace_back([this] { loop(); });
  }

  void run(const std::vector<Task>& tasks) {
    if (workers_.empty() || tasks.size() < 2) {
      for (const Task& t : tasks) memcpy(t.dst, t.src, t.n);
      return;
    }
    std::lock_guard<std::mutex> turn(run_mu_);
    tasks_ = &tasks;
    next_.store(0);
    active_.store((int)workers_.size());
    {
      std::lock_guard<std::mutex> lk(mu_);  // a worker about to sleep sees the new job
      gen_.fetch_add(1, std::memory_order_release);
    }
    cv_start_.notify_all();
    drain();
    for (int i = 0; active_.load(std::memory_order_acquire) != 0 && i < kSpin; ++i) relax();
    if (active_.load(std::memory_order_acquire) != 0) {
      std::unique_lock<std::mutex> lk(mu_);
      cv_done_.wait(lk, [this] { return active_.load(std::memory_order_acquire) == 0; });
    }
    tasks_ = nullptr;
  }

 private:
  static constexpr int kSpin = 1 << 16;  // polls before sleeping (a few hundred us)
  static void relax() { __builtin_ia32_pause(); }
  void drain() {
    const std::vector<Task>& t = *tasks_;
    for (;;) {
      size_t i = next_.fetch_add(1);
      if (i >= t.size()) break;
      memcpy(t[i].dst, t[i].src, t[i].n);
    }
  }
  void loop() {
    uint64_t seen = 0;
    for (;;) {
      uint64_t g = gen_.load(std::memory_order_acquire);
      for (int i = 0; g == seen && i < kSpin; ++i) {
        relax();
        g = gen_.load(std::memory_order_acquire);
      }
      if (g == seen) {
        std::unique_lock<std::mutex> lk(mu_);
        cv_start_.wait(lk, [&] { return gen_.load(std::memory_order_acquire) != seen; });
        g = gen_.load(std::memory_order_acquire);
      }
      seen = g;
      drain();
      if (active_.fetch_sub(1, std::memory_order_acq_rel) == 1) {
        std::lock_guard<std::mutex> lk(mu_);
        cv_done_.notify_all();
      }
    }
  }

  std::vector<std::thread> workers_;
  std::mutex run_mu_;
  std::mutex mu_;
  std::condition_variable cv_start_, cv_done_;
  const std::vector<Task>* tasks_ = nullptr;
  std::atomic<size_t> next_{0};
  std::atomic<int> active_{0};
  std::atomic<uint64_t> gen_{0};
};

// Created on first use and kept for the life of the process (never joined).
// 8 threads including the caller: on the MI355X host, 8 packing threads
// (87 GB/s) leave the DMA engine its pinned-memory bandwidth; 16 packed
// faster alone (105 GB/s) but slowed the overlapped copies.
static PackPool* pack_pool() {
  static PackPool* pool = [] {
    int n = 8;
    if (const char* v = getenv("NP_PACK_THREADS")) n = atoi(v);
    unsigned hw = std::thread::hardware_concurrency();
    if (hw && n > (int)hw) n = (int)hw;
    if (n < 0) n = 0;
    // the calling thread also packs, so n - 1 helpers
    return new PackPool(n > 1 ? n - 1 : 0);
  }();
  return pool;
}

// State of one pinned staging buffer (keyed by device and base address):
// an event per staging piece (its copy has finished: the piece may be
// packed again, and its scatter may start) and the scatter stream with its
// last event.  Copies run on the caller's side stream back to back; each
// landed piece's scatter runs on the buffer's own scatter stream (default
// priority) once the piece's event has fired, so the copy engine never waits
// for a kernel between two copies.  ev_scattered
// marks the last scatter: the side stream waits on it before copies reuse
// the landing area and at the end of each call, so work the caller puts on
// `side` later follows the scatters.
// Calls on different staging buffers share nothing but the packing threads;
// calls on one buffer are serialised by its lock.
constexpr int MAX_PIECES = 8;
struct StageCtx {
  std::mutex mu;
  hipEvent_t ev[MAX_PIECES] = {};
  bool pending[MAX_PIECES] = {};
  int next_piece = 0;  // the piece ring continues across calls
  hipStream_t scat = nullptr;
  hipEvent_t ev_scattered = nullptr;
  bool scattered = false;  // ev_scattered has been recorded
  // the landing area is a ring of landed pieces (byte positions, each piece
  // at a 16-byte boundary) that continues across calls; the copies wait for
  // the scatters only when the ring wraps
  const void* land_ptr = nullptr;
  size_t land_bytes = 0, land_pos = 0;
};

static StageCtx* stage_ctx(int dev, const void* staging) {
  static std::mutex mu;
  static std::map<std::pair<int, uintptr_t>, StageCtx*> ctx;
  std::lock_guard<std::mutex> g(mu);
  StageCtx*& c = ctx[{dev, (uintptr_t)staging}];
  if (!c) c = new StageCtx();
  return c;
}

// Where the records come from: host memory (`host`) or a file (`fd` >= 0,
// the storage tier starting at byte `file_offset`), read into `io_buf`
// (ordinary host memory of io_bytes bytes; nullptr: straight into staging).
struct StageSource {
  const char* host;
  int fd;
  int64_t file_offset;
  char* io_buf;
  size_t io_bytes;
};

// Layout of the areas (rec = record bytes):
//   staging:  n_pieces pieces; a piece of n records is packed as [n records]
//             with the rows gathered at [piece_cap records ...] and moved to
//             just after the records when the piece is sent:
//             [n records | n int32 destination rows]
//   landing:  a ring of such landed pieces, each at a 16-byte boundary
// A token's records are packed piece by piece (the pieces form a ring: a
// piece is reused once its copy has finished), and each piece goes to the
// next free position of the landing ring with ONE hipMemcpyAsync on `side`
// (a second, small copy for the rows would be sent as a kernel, and every
// switch between the copy engine and a kernel on `side` costs tens of
// microseconds), then one scatter kernel on the scatter stream moves its
// records into their slots (layer * C + slot).  With layer_ready, at a layer
// boundary once the layers since the last event hold enough bytes, the open
// piece is sent and the events of those layers are recorded behind its
// scatter.  Pieces start small and grow (by default 2 MiB, then doubling)
// so the first copy starts after little packing; packing piece i + 1
// overlaps the copy of piece i.
static np_status stage_common(const char* fn, const np_shape* s, const np_stage_plan* plan,
                              int32_t lb, int32_t le, const StageSource& src, void* dev_resident,
                              void* host_staging, size_t staging_bytes, void* dev_landing,
                              size_t landing_bytes, hipStream_t side, hipEvent_t wait_before,
                              hipEvent_t* layer_ready) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (lb < 0 || le > s->layers || lb > le)
    return fail(NP_ERR_INVALID_ARG, "layer range [%d, %d) outside [0, %d)", lb, le, s->layers);
  if (!plan || !plan->counts || !plan->in_ids || !plan->in_slots)
    return fail(NP_ERR_INVALID_ARG, "%s: plan arrays must be non-NULL", fn);
  if ((src.fd < 0 && !src.host) || !host_staging || !aligned16(dev_resident) ||
      !aligned16(dev_landing) || !aligned16(host_staging))
    return fail(NP_ERR_INVALID_ARG, "%s: buffers must be non-NULL and 16-byte aligned", fn);
  if ((st = check_resident(fn, dev_resident)) != NP_OK) return st;
  const size_t rec = (size_t)3 * s->d_model * dtype_size(s->wdtype);
  const size_t rec_row = rec + sizeof(int32_t);  // landing bytes per record
  // pieces on 4 KiB boundaries, so that direct file reads land aligned
  int n_pieces = 4;
  while (n_pieces > 1 && ((staging_bytes / n_pieces) & ~(size_t)4095) < rec + sizeof(int32_t))
    --n_pieces;
  const size_t piece_bytes = (staging_bytes / n_pieces) & ~(size_t)4095;
  size_t piece_cap = piece_bytes / (rec + sizeof(int32_t));
  if (src.fd >= 0 && src.io_buf) piece_cap = std::min(piece_cap, src.io_bytes / rec);
  if (landing_bytes < rec_row || piece_cap < 1)
    return fail(NP_ERR_CAPACITY,
                "%s: the landing area (%zu B) or a staging piece (%zu B of %zu B) holds no "
                "record of %zu B and its row index", fn, landing_bytes, piece_bytes,
                staging_bytes, rec);
  const void* read_target = src.io_buf ? (const void*)src.io_buf : host_staging;
  if (src.fd >= 0 && file_is_direct(src.fd) &&
      (rec % IO_ALIGN || src.file_offset % IO_ALIGN || (uintptr_t)read_target % IO_ALIGN))
    return fail(NP_ERR_INVALID_ARG,
                "%s: an O_DIRECT file needs records (%zu B), the file offset and the read "
                "buffer aligned to %d bytes", fn, rec, IO_ALIGN);
  // validate the whole plan before enqueueing anything
  for (int l = lb; l < le; ++l) {
    const int n = plan->counts[(size_t)l * 4];
    if (n < 0 || n > s->k) return fail(NP_ERR_INVALID_ARG, "layer %d: n_in %d outside [0, k]", l, n);
    for (int j = 0; j < n; ++j) {
      const int id = plan->in_ids[(size_t)l * s->k + j];
      const int slot = plan->in_slots[(size_t)l * s->k + j];
      if (id < 0 || id >= s->d_ffn || slot < 0 || slot >= s->capacity)
        return fail(NP_ERR_INVALID_ARG, "layer %d entry %d: id %d / slot %d out of range", l, j,
                    id, slot);
    }
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  StageCtx* cx = stage_ctx(dev, host_staging);
  std::lock_guard<std::mutex> guard(cx->mu);
  for (int i = 0; i < MAX_PIECES; ++i)
    if (!cx->ev[i]) {
      e = hipEventCreateWithFlags(&cx->ev[i], hipEventDisableTiming);
      if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
    }
  if (!cx->ev_scattered) {
    e = hipEventCreateWithFlags(&cx->ev_scattered, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
  }
  if (!cx->scat) {
    e = hipStreamCreateWithFlags(&cx->scat, hipStreamNonBlocking);
    if (e != hipSuccess) return hip_fail(e, "hipStreamCreateWithFlags (scatter stream)");
  }
  int fail_after = -1;  // test hook: fail after this many pieces
  if (const char* v = getenv("NP_TEST_FAIL_STAGE_AFTER")) fail_after = atoi(v);
  // with layer_ready: at a layer boundary, once the layers since the last
  // recorded event hold this many bytes (NP_STAGE_GROUP_MIB, default 8 MiB),
  // the open piece is sent and their events are recorded
  size_t group_bytes = (size_t)8 << 20;
  if (const char* v = getenv("NP_STAGE_GROUP_MIB"))
    if (atoi(v) > 0) group_bytes = (size_t)atoi(v) << 20;

  // scatters write the resident buffer: they wait for wait_before; copies
  // into the landing area wait for the previous call's last scatter
  if (wait_before) {
    e = hipStreamWaitEvent(cx->scat, wait_before, 0);
    if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
  }
  if (cx->land_ptr != dev_landing || cx->land_bytes != landing_bytes) {
    // another landing area (or size): start its ring at 0 after every
    // scatter that may still read the previous one
    if (cx->scattered) {
      e = hipStreamWaitEvent(side, cx->ev_scattered, 0);
      if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
    }
    cx->land_ptr = dev_landing;
    cx->land_bytes = landing_bytes;
    cx->land_pos = 0;
  }

  char* const landing = (char*)dev_landing;
  std::vector<PackPool::Task> tasks;
  std::vector<ReadRun> reads;
  int32_t* piece_rows = nullptr;  // the open piece's destination rows
  int h = cx->next_piece % n_pieces, pieces = 0;
  char* stg = nullptr;
  // the open piece lands at byte `pos` of the landing ring and holds at most
  // piece_limit records; group_n: records sent since the last layer_ready
  // event
  size_t n_piece = 0, group_n = 0, pos = cx->land_pos, piece_limit = 1;
  // the first piece is small (NP_STAGE_FIRST_KIB, default 2 MiB) so that the
  // copy engine starts early, unless it is still busy with the previous
  // call's pieces; each later piece is NP_STAGE_GROWTH_PCT percent of the
  // one before (default 200; 100 keeps every piece at the first size), up
  // to the piece capacity
  size_t first_bytes = (size_t)2 << 20, growth_pct = 200;
  if (const char* v = getenv("NP_STAGE_FIRST_KIB"))
    if (atoi(v) > 0) first_bytes = (size_t)atoi(v) << 10;
  if (const char* v = getenv("NP_STAGE_GROWTH_PCT"))
    if (atoi(v) >= 100) growth_pct = (size_t)atoi(v);
  size_t cur_cap = std::min(piece_cap, std::max<size_t>(1, first_bytes / rec));
  {
    const int ph = (h + n_pieces - 1) % n_pieces;
    if (cx->pending[ph] && hipEventQuery(cx->ev[ph]) == hipErrorNotReady) cur_cap = piece_cap;
    (void)hipGetLastError();
  }
  // run being extended: source byte offset in the storage tier, length in
  // records, first record's index in the piece
  uint64_t run_src = 0;
  size_t run_len = 0, run_dst = 0;
  const size_t chunk = (size_t)256 << 10;
  int ready_from = lb;  // first layer whose layer_ready event is not recorded yet

  auto close_run = [&]() {
    if (!run_len) return;
    const size_t bytes = run_len * rec;
    if (src.fd >= 0) {
      char* target = src.io_buf ? src.io_buf : stg;
      reads.push_back({target + run_dst * rec, (uint64_t)src.file_offset + run_src, bytes});
    } else {
      for (size_t off = 0; off < bytes; off += chunk)
        tasks.push_back({stg + run_dst * rec + off, src.host + run_src + off,
                         std::min(chunk, bytes - off)});
    }
    run_len = 0;
  };
  auto begin_piece = [&]() -> np_status {
    if (cx->pending[h]) {
      hipError_t ee = hipEventSynchronize(cx->ev[h]);
      if (ee != hipSuccess) return hip_fail(ee, "hipEventSynchronize (staging reuse)");
      cx->pending[h] = false;
    }
    stg = (char*)host_staging + (size_t)h * piece_bytes;
    piece_rows = (int32_t*)(stg + piece_cap * rec);
    tasks.clear();
    reads.clear();
    n_piece = 0;
    return NP_OK;
  };
  // packs (or reads) the open piece and copies it to the landing area
  auto flush_piece = [&]() -> np_status {
    close_run();
    if (n_piece == 0) return NP_OK;
    if (fail_after >= 0 && pieces >= fail_after)
      return fail(NP_ERR_HIP, "%s: injected staging failure after %d pieces", fn, pieces);
    if (src.fd >= 0) {
      // each piece read into io_buf goes on to the same offset of the pinned
      // piece as soon as it is complete, overlapping the copies with the
      // reads still in flight
      struct Ctx {
        char* io;
        char* stg;
      } c{src.io_buf, stg};
      PieceDone to_staging = [](void* p, char* dst, size_t n) {
        Ctx* x = (Ctx*)p;
        memcpy(x->stg + (dst - x->io), dst, n);
      };
      np_status rs = read_runs(src.fd, reads, io_depth(), src.io_buf ? to_staging : nullptr, &c);
      if (rs != NP_OK) return rs;
    } else {
      pack_pool()->run(tasks);
    }
    // the rows go right after the records: one copy carries both
    const size_t rec_bytes = n_piece * rec, bytes = rec_bytes + n_piece * sizeof(int32_t);
    if ((char*)piece_rows != stg + rec_bytes)
      memmove(stg + rec_bytes, piece_rows, n_piece * sizeof(int32_t));
    hipError_t ee = hipMemcpyAsync(landing + pos, stg, bytes, hipMemcpyHostToDevice, side);
    if (ee != hipSuccess) return hip_fail(ee, "hipMemcpyAsync (staging piece)");
    ee = hipEventRecord(cx->ev[h], side);
    if (ee != hipSuccess) return hip_fail(ee, "hipEventRecord");
    cx->pending[h] = true;
    // the piece's scatter, after its copy (the same event: each event
    // recorded behind a copy costs the side stream ~5 us), on the scatter
    // stream
    ee = hipStreamWaitEvent(cx->scat, cx->ev[h], 0);
    if (ee != hipSuccess) return hip_fail(ee, "scatter stream ordering");
    ee = launch_stage_scatter(*s, landing + pos, (const int32_t*)(landing + pos + rec_bytes),
                              (int)n_piece, dev_resident, cx->scat);
    if (ee != hipSuccess) return hip_fail(ee, "scatter launch");
    ee = hipEventRecord(cx->ev_scattered, cx->scat);
    if (ee != hipSuccess) return hip_fail(ee, "hipEventRecord");
    cx->scattered = true;
    ++pieces;
    h = (h + 1) % n_pieces;
    cx->next_piece = h;
    pos = (pos + bytes + 15) & ~(size_t)15;
    cx->land_pos = pos;
    group_n += n_piece;
    n_piece = 0;
    if (growth_pct > 100)  // at least one record more, so that small pieces grow too
      cur_cap = std::min(piece_cap, std::max(cur_cap + 1, cur_cap * growth_pct / 100));
    return NP_OK;
  };
  // before a piece is packed: its size (the current piece size, at most
  // what the whole ring holds), and a wrap of the ring when the rest of it
  // cannot hold that many records and their rows, so that a piece is never
  // cut short at the end of the ring; copies into the wrapped ring wait (on
  // the side stream) for every scatter that may still read it
  auto ring_room = [&]() -> np_status {
    piece_limit = std::min(cur_cap, landing_bytes / rec_row);
    const size_t room = pos < landing_bytes ? (landing_bytes - pos) / rec_row : 0;
    if (room >= piece_limit) return NP_OK;
    if (cx->scattered) {
      hipError_t ee = hipStreamWaitEvent(side, cx->ev_scattered, 0);
      if (ee != hipSuccess) return hip_fail(ee, "hipStreamWaitEvent (landing ring)");
    }
    pos = 0;
    cx->land_pos = 0;
    return NP_OK;
  };
  // a piece that fails (a HIP call, a read) ends the call; every piece
  // copied before it has its scatter enqueued already, so what was enqueued
  // lands (the caller marks the resident buffer in any case)
  auto bail = [&](np_status err) -> np_status { return err; };
  auto record_ready = [&](int upto) -> np_status {  // layers [ready_from, upto)
    for (; ready_from < upto; ++ready_from) {
      hipError_t ee = hipEventRecord(layer_ready[ready_from], cx->scat);
      if (ee != hipSuccess) return hip_fail(ee, "hipEventRecord (layer_ready)");
    }
    return NP_OK;
  };

  bool open = false;
  for (int l = lb; l < le; ++l) {
    const int n = plan->counts[(size_t)l * 4];
    const int32_t* ids = plan->in_ids + (size_t)l * s->k;
    const int32_t* slots = plan->in_slots + (size_t)l * s->k;
    for (int j = 0; j < n; ++j) {
      if (!open) {
        if ((st = ring_room()) != NP_OK) return bail(st);
        if ((st = begin_piece()) != NP_OK) return st;
        open = true;
      }
      const uint64_t at = ((uint64_t)l * s->d_ffn + ids[j]) * rec;
      if (run_len && at == run_src + run_len * rec) {
        ++run_len;  // adjacent id: extend the contiguous range
      } else {
        close_run();
        run_src = at;
        run_len = 1;
        run_dst = n_piece;
      }
      piece_rows[n_piece] = l * s->capacity + slots[j];
      ++n_piece;
      if (n_piece == piece_limit) {
        if ((st = flush_piece()) != NP_OK) return bail(st);
        open = false;
      }
    }
    if (layer_ready && (l == le - 1 || (group_n + n_piece) * rec >= group_bytes)) {
      if (open) {
        if ((st = flush_piece()) != NP_OK) return bail(st);
        open = false;
      }
      if ((st = record_ready(l + 1)) != NP_OK) return st;
      group_n = 0;
    }
  }
  if (open && (st = flush_piece()) != NP_OK) return bail(st);
  if (layer_ready) return record_ready(le);
  // without layer events, later work on `side` follows the whole staging
  if (cx->scattered) {
    e = hipStreamWaitEvent(side, cx->ev_scattered, 0);
    if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
  }
  return NP_OK;
}

// A staging that fails at run time (a HIP call, a file read) may have
// placed only part of the delta: the resident buffer is marked so that later
// calls on it report NP_ERR_STATE.  Argument errors enqueue nothing.
static np_status staged(const void* resident, np_status st) {
  if (st == NP_ERR_HIP || st == NP_ERR_IO || st == NP_ERR_UNSUPPORTED)
    mark_resident_incomplete(resident);
  return st;
}

}  // namespace np

using namespace np;

extern "C" np_status np_stage_rows(const np_shape* s, const np_stage_plan* plan, int32_t lb,
                                   int32_t le, const void* host_storage, void* dev_resident,
                                   void* host_staging, size_t staging_bytes, void* dev_landing,
                                   size_t landing_bytes, hipStream_t side, hipEvent_t wait_before,
                                   hipEvent_t* layer_ready) {
  if (!host_storage) return fail(NP_ERR_INVALID_ARG, "np_stage_rows: host_storage is NULL");
  return staged(dev_resident,
                stage_common("np_stage_rows", s, plan, lb, le,
                             {(const char*)host_storage, -1, 0, nullptr, 0}, dev_resident,
                             host_staging, staging_bytes, dev_landing, landing_bytes, side,
                             wait_before, layer_ready));
}

extern "C" np_status np_stage_file(const np_shape* s, const np_stage_plan* plan, int32_t lb,
                                   int32_t le, int32_t fd, int64_t file_offset,
                                   void* dev_resident, void* host_staging, size_t staging_bytes,
                                   void* io_buffer, size_t io_buffer_bytes, void* dev_landing,
                                   size_t landing_bytes, hipStream_t side,
                                   hipEvent_t wait_before, hipEvent_t* layer_ready) {
  if (fd < 0 || file_offset < 0)
    return fail(NP_ERR_INVALID_ARG, "np_stage_file: fd %d / file offset %lld", fd,
                (long long)file_offset);
  if (io_buffer && io_buffer_bytes == 0)
    return fail(NP_ERR_INVALID_ARG, "np_stage_file: io_buffer of 0 bytes");
  return staged(dev_resident,
                stage_common("np_stage_file", s, plan, lb, le,
                             {nullptr, fd, file_offset, (char*)io_buffer, io_buffer_bytes},
                             dev_resident, host_staging, staging_bytes, dev_landing,
                             landing_bytes, side, wait_before, layer_ready));
}
