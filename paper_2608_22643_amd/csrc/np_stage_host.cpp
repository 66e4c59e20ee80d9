// np_stage_host.cpp -- staging through pinned host memory (Sec. 3.5, I/O
// path): incoming ids are walked layer by layer in ascending order, adjacent
// ids are coalesced into one contiguous source range, records are packed
// into a capacity-bounded pinned staging area, and each chunk goes to the
// device with one hipMemcpyAsync on the side stream, followed by a kernel
// that scatters the chunk's records into their slots.  The staging area is
// used as two halves so that packing one chunk overlaps the copy of the
// previous one; a delta larger than a chunk runs as several independent
// submit-and-scatter chunks.  The source is the storage tier in host memory
// (np_stage_rows: the ranges are copied by a thread pool) or in a file
// (np_stage_file: the ranges are read through io_uring, np_file.cpp).
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <mutex>
#include <thread>
#include <vector>

#include "np_internal.hpp"

namespace np {

// Persistent worker pool for the host pack (memcpy of coalesced runs).
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
    {
      std::lock_guard<std::mutex> lk(mu_);
      tasks_ = &tasks;
      next_.store(0);
      active_ = (int)workers_.size();
      ++gen_;
    }
    cv_start_.notify_all();
    drain();
    std::unique_lock<std::mutex> lk(mu_);
    cv_done_.wait(lk, [this] { return active_ == 0; });
    tasks_ = nullptr;
  }

 private:
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
      std::unique_lock<std::mutex> lk(mu_);
      cv_start_.wait(lk, [&] { return gen_ != seen; });
      seen = gen_;
      lk.unlock();
      drain();
      lk.lock();
      if (--active_ == 0) cv_done_.notify_all();
    }
  }

  std::vector<std::thread> workers_;
  std::mutex mu_;
  std::condition_variable cv_start_, cv_done_;
  const std::vector<Task>* tasks_ = nullptr;
  std::atomic<size_t> next_{0};
  int active_ = 0;
  uint64_t gen_ = 0;
};

// Created on first use and kept for the life of the process (never joined).
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

struct DeviceStaging {
  std::mutex mu;
  hipEvent_t ev[2] = {nullptr, nullptr};
  bool pending[2] = {false, false};
};

static DeviceStaging* device_staging(int dev) {
  static DeviceStaging slots[64];
  return (dev >= 0 && dev < 64) ? &slots[dev] : nullptr;
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
      !aligned16(dev_landing))
    return fail(NP_ERR_INVALID_ARG, "%s: buffers must be non-NULL (device: aligned)", fn);
  if ((st = check_resident(fn, dev_resident)) != NP_OK) return st;
  const size_t rec = (size_t)3 * s->d_model * dtype_size(s->wdtype);
  // halves on 4 KiB boundaries, so that direct file reads land aligned
  const size_t half = (staging_bytes / 2) & ~(size_t)4095;
  const void* read_target = src.io_buf ? (const void*)src.io_buf : host_staging;
  if (src.fd >= 0 && file_is_direct(src.fd) &&
      (rec % IO_ALIGN || src.file_offset % IO_ALIGN || (uintptr_t)read_target % IO_ALIGN))
    return fail(NP_ERR_INVALID_ARG,
                "%s: an O_DIRECT file needs records (%zu B), the file offset and the read "
                "buffer aligned to %d bytes", fn, rec, IO_ALIGN);
  size_t cap_bytes = std::min(half, landing_bytes);
  if (src.fd >= 0 && src.io_buf) cap_bytes = std::min(cap_bytes, src.io_bytes);
  const size_t chunk_cap = cap_bytes / (rec + sizeof(int32_t));
  if (chunk_cap < 1)
    return fail(NP_ERR_CAPACITY,
                "staging half (%zu B) or landing area (%zu B) holds no record of %zu B", half,
                landing_bytes, rec + sizeof(int32_t));
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
  DeviceStaging* ds = device_staging(dev);
  if (!ds) return fail(NP_ERR_UNSUPPORTED, "device index %d", dev);
  std::lock_guard<std::mutex> guard(ds->mu);
  for (int i = 0; i < 2; ++i)
    if (!ds->ev[i]) {
      e = hipEventCreateWithFlags(&ds->ev[i], hipEventDisableTiming);
      if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
    }
  int fail_after = -1;  // test hook: fail after this many chunks
  if (const char* v = getenv("NP_TEST_FAIL_STAGE_AFTER")) fail_after = atoi(v);

  if (wait_before) {
    e = hipStreamWaitEvent(side, wait_before, 0);
    if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
  }

  std::vector<PackPool::Task> tasks;
  std::vector<ReadRun> reads;
  std::vector<int32_t> dst_rows;
  dst_rows.reserve(chunk_cap);
  int h = 0, chunks = 0;
  char* stg = nullptr;
  size_t n_in_chunk = 0;
  // run being extended: source byte offset in the storage tier and length
  // in records
  uint64_t run_src = 0;
  size_t run_len = 0, run_dst = 0;
  const size_t piece = (size_t)256 << 10;

  auto close_run = [&]() {
    if (!run_len) return;
    size_t bytes = run_len * rec, off = 0;
    if (src.fd >= 0) {
      char* target = src.io_buf ? src.io_buf : stg;
      reads.push_back({target + run_dst * rec, (uint64_t)src.file_offset + run_src, bytes});
    } else {
      while (off < bytes) {
        size_t n = std::min(piece, bytes - off);
        tasks.push_back({stg + run_dst * rec + off, src.host + run_src + off, n});
        off += n;
      }
    }
    run_len = 0;
  };
  auto begin_chunk = [&]() -> np_status {
    if (ds->pending[h]) {
      hipError_t ee = hipEventSynchronize(ds->ev[h]);
      if (ee != hipSuccess) return hip_fail(ee, "hipEventSynchronize (staging reuse)");
      ds->pending[h] = false;
    }
    stg = (char*)host_staging + (size_t)h * half;
    tasks.clear();
    reads.clear();
    dst_rows.clear();
    n_in_chunk = 0;
    return NP_OK;
  };
  auto flush = [&]() -> np_status {
    close_run();
    if (n_in_chunk == 0) return NP_OK;
    if (fail_after >= 0 && chunks >= fail_after)
      return fail(NP_ERR_HIP, "%s: injected staging failure after %d chunks", fn, chunks);
    if (src.fd >= 0) {
      // each piece read into io_buf goes on to the same offset of the pinned
      // half as soon as it is complete, overlapping the copies with the
      // reads still in flight
      struct Ctx {
        char* io;
        char* stg;
      } cx{src.io_buf, stg};
      PieceDone to_staging = [](void* c, char* dst, size_t n) {
        Ctx* x = (Ctx*)c;
        memcpy(x->stg + (dst - x->io), dst, n);
      };
      np_status rs = read_runs(src.fd, reads, io_depth(), src.io_buf ? to_staging : nullptr, &cx);
      if (rs != NP_OK) return rs;
    } else {
      pack_pool()->run(tasks);
    }
    memcpy(stg + n_in_chunk * rec, dst_rows.data(), n_in_chunk * sizeof(int32_t));
    const size_t bytes = n_in_chunk * (rec + sizeof(int32_t));
    hipError_t ee = hipMemcpyAsync(dev_landing, stg, bytes, hipMemcpyHostToDevice, side);
    if (ee != hipSuccess) return hip_fail(ee, "hipMemcpyAsync (staging chunk)");
    ee = hipEventRecord(ds->ev[h], side);
    if (ee != hipSuccess) return hip_fail(ee, "hipEventRecord");
    ds->pending[h] = true;
    ee = launch_stage_scatter(*s, dev_landing, (int)n_in_chunk, dev_resident, side);
    if (ee != hipSuccess) return hip_fail(ee, "scatter launch");
    ++chunks;
    h ^= 1;
    n_in_chunk = 0;
    return NP_OK;
  };

  bool open = false;
  for (int l = lb; l < le; ++l) {
    const int n = plan->counts[(size_t)l * 4];
    const int32_t* ids = plan->in_ids + (size_t)l * s->k;
    const int32_t* slots = plan->in_slots + (size_t)l * s->k;
    for (int j = 0; j < n; ++j) {
      if (!open) {
        if ((st = begin_chunk()) != NP_OK) return st;
        open = true;
      }
      const uint64_t at = ((uint64_t)l * s->d_ffn + ids[j]) * rec;
      if (run_len && at == run_src + run_len * rec) {
        ++run_len;  // adjacent id: extend the contiguous range
      } else {
        close_run();
        run_src = at;
        run_len = 1;
        run_dst = n_in_chunk;
      }
      dst_rows.push_back(l * s->capacity + slots[j]);
      ++n_in_chunk;
      if (n_in_chunk == chunk_cap) {
        if ((st = flush()) != NP_OK) return st;
        open = false;
      }
    }
    if (layer_ready) {
      if (open) {
        if ((st = flush()) != NP_OK) return st;
        open = false;
      }
      e = hipEventRecord(layer_ready[l], side);
      if (e != hipSuccess) return hip_fail(e, "hipEventRecord (layer_ready)");
    }
  }
  if (open && (st = flush()) != NP_OK) return st;
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
