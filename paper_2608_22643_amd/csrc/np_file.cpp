// np_file.cpp -- the storage tier as a file (Sec. 3.5, I/O path): record
// reads through Linux io_uring, with the queue depth held up to 256 requests
// and each request a coalesced range of consecutive records.  The ring is set
// up with the raw system calls (no liburing): one submission and one
// completion ring mapped from the kernel, filled and drained here.  A read
// that returns short is resubmitted for its remainder; an error or an early
// end of file fails the whole batch.
#include <errno.h>
#include <fcntl.h>
#include <linux/io_uring.h>
#include <stdlib.h>
#include <string.h>
#include <sys/mman.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "np_internal.hpp"

namespace np {

namespace {

class URing {
 public:
  ~URing() { close_ring(); }

  // 0 on success, else an errno value
  int open_ring(unsigned entries) {
    io_uring_params p;
    memset(&p, 0, sizeof p);
    int fd = (int)syscall(__NR_io_uring_setup, entries, &p);
    if (fd < 0) return errno;
    fd_ = fd;
    sq_bytes_ = p.sq_off.array + p.sq_entries * sizeof(unsigned);
    cq_bytes_ = p.cq_off.cqes + p.cq_entries * sizeof(io_uring_cqe);
    const bool single = p.features & IORING_FEAT_SINGLE_MMAP;
    if (single) sq_bytes_ = cq_bytes_ = sq_bytes_ > cq_bytes_ ? sq_bytes_ : cq_bytes_;
    sq_ = mmap(nullptr, sq_bytes_, PROT_READ | PROT_WRITE, MAP_SHARED | MAP_POPULATE, fd,
               IORING_OFF_SQ_RING);
    if (sq_ == MAP_FAILED) return fail_open();
    cq_ = single ? sq_
                 : mmap(nullptr, cq_bytes_, PROT_READ | PROT_WRITE, MAP_SHARED | MAP_POPULATE, fd,
                        IORING_OFF_CQ_RING);
    if (cq_ == MAP_FAILED) return fail_open();
    sqes_bytes_ = p.sq_entries * sizeof(io_uring_sqe);
    sqes_ = (io_uring_sqe*)mmap(nullptr, sqes_bytes_, PROT_READ | PROT_WRITE,
                                MAP_SHARED | MAP_POPULATE, fd, IORING_OFF_SQES);
    if (sqes_ == MAP_FAILED) return fail_open();
    char* s = (char*)sq_;
    sq_head_ = (unsigned*)(s + p.sq_off.head);
    sq_tail_ = (unsigned*)(s + p.sq_off.tail);
    sq_mask_ = *(unsigned*)(s + p.sq_off.ring_mask);
    sq_array_ = (unsigned*)(s + p.sq_off.array);
    char* c = (char*)cq_;
    cq_head_ = (unsigned*)(c + p.cq_off.head);
    cq_tail_ = (unsigned*)(c + p.cq_off.tail);
    cq_mask_ = *(unsigned*)(c + p.cq_off.ring_mask);
    cqes_ = (io_uring_cqe*)(c + p.cq_off.cqes);
    entries_ = p.sq_entries;
    return 0;
  }

  unsigned entries() const { return entries_; }

  // queue one read (the caller keeps at most entries() in flight)
  void push_read(int fd, void* buf, unsigned len, uint64_t off, uint64_t tag) {
    const unsigned tail = *sq_tail_;
    const unsigned idx = tail & sq_mask_;
    io_uring_sqe* e = &sqes_[idx];
    memset(e, 0, sizeof *e);
    e->opcode = IORING_OP_READ;
    e->fd = fd;
    e->addr = (uint64_t)(uintptr_t)buf;
    e->len = len;
    e->off = off;
    e->user_data = tag;
    sq_array_[idx] = idx;
    __atomic_store_n(sq_tail_, tail + 1, __ATOMIC_RELEASE);
    ++unsubmitted_;
  }

  // submits what is queued and waits for at least `wait` completions;
  // 0 or an errno value
  int enter(unsigned wait) {
    for (;;) {
      int r = (int)syscall(__NR_io_uring_enter, fd_, unsubmitted_, wait,
                           wait ? IORING_ENTER_GETEVENTS : 0, nullptr, 0);
      if (r >= 0) {
        unsubmitted_ -= (unsigned)r < unsubmitted_ ? (unsigned)r : unsubmitted_;
        return 0;
      }
      if (errno != EINTR) return errno;
    }
  }

  // takes one completion if there is one
  bool pop(uint64_t* tag, int* res) {
    const unsigned head = *cq_head_;
    if (head == __atomic_load_n(cq_tail_, __ATOMIC_ACQUIRE)) return false;
    const io_uring_cqe* c = &cqes_[head & cq_mask_];
    *tag = c->user_data;
    *res = c->res;
    __atomic_store_n(cq_head_, head + 1, __ATOMIC_RELEASE);
    return true;
  }

 private:
  int fail_open() {
    int e = errno;
    close_ring();
    return e;
  }
  void close_ring() {
    if (sqes_ && sqes_ != MAP_FAILED) munmap(sqes_, sqes_bytes_);
    if (cq_ && cq_ != MAP_FAILED && cq_ != sq_) munmap(cq_, cq_bytes_);
    if (sq_ && sq_ != MAP_FAILED) munmap(sq_, sq_bytes_);
    if (fd_ >= 0) close(fd_);
    sqes_ = nullptr;
    sq_ = cq_ = nullptr;
    fd_ = -1;
  }

  int fd_ = -1;
  void *sq_ = nullptr, *cq_ = nullptr;
  io_uring_sqe* sqes_ = nullptr;
  size_t sq_bytes_ = 0, cq_bytes_ = 0, sqes_bytes_ = 0;
  unsigned *sq_head_ = nullptr, *sq_tail_ = nullptr, *sq_array_ = nullptr;
  unsigned *cq_head_ = nullptr, *cq_tail_ = nullptr;
  unsigned sq_mask_ = 0, cq_mask_ = 0, entries_ = 0, unsubmitted_ = 0;
  io_uring_cqe* cqes_ = nullptr;
};

std::mutex g_ring_mu;

// The process's ring (created on first use, kept for the life of the
// process); nullptr with *err set when io_uring cannot be set up.
URing* ring(int* err) {
  static URing* r = nullptr;
  static int r_err = 0;
  if (!r && !r_err) {
    URing* u = new URing();
    r_err = u->open_ring(IO_QD_MAX);
    if (r_err) delete u;
    else r = u;
  }
  *err = r_err;
  return r;
}

}  // namespace

int io_depth() {
  int qd = IO_QD_MAX;
  if (const char* v = getenv("NP_IO_QD")) qd = atoi(v);
  return qd < 1 ? 1 : (qd > IO_QD_MAX ? IO_QD_MAX : qd);
}

bool file_is_direct(int fd) {
  int fl = fcntl(fd, F_GETFL);
  return fl >= 0 && (fl & O_DIRECT);
}

np_status read_runs(int fd, const std::vector<ReadRun>& runs, int qd, PieceDone done,
                    void* ctx) {
  if (runs.empty()) return NP_OK;
  std::lock_guard<std::mutex> g(g_ring_mu);
  int err = 0;
  URing* r = ring(&err);
  if (!r) return fail(NP_ERR_IO, "io_uring setup failed: %s", strerror(err));
  if (qd > (int)r->entries()) qd = (int)r->entries();
  // requests in flight; each a piece of a run, reissued for its remainder
  // when a read returns short
  struct Req {
    char* buf;
    uint64_t off;
    size_t left;
    char* start;  // the piece as issued, for `done`
    size_t bytes;
  };
  std::vector<Req> reqs;  // runs cut into pieces of at most IO_PIECE bytes
  reqs.reserve(runs.size());
  for (const ReadRun& rr : runs)
    for (size_t o = 0; o < rr.bytes; o += IO_PIECE) {
      const size_t n = rr.bytes - o < IO_PIECE ? rr.bytes - o : IO_PIECE;
      reqs.push_back({rr.dst + o, rr.offset + o, n, rr.dst + o, n});
    }
  size_t next = 0, ndone = 0;
  std::vector<size_t> ready;  // pieces read in full since the last hand-over
  int inflight = 0;
  np_status st = NP_OK;
  auto issue = [&](size_t i) {
    r->push_read(fd, reqs[i].buf, (unsigned)reqs[i].left, reqs[i].off, (uint64_t)i);
    ++inflight;
  };
  while (ndone < reqs.size()) {
    while (st == NP_OK && inflight < qd && next < reqs.size()) issue(next++);
    if (inflight == 0) break;  // an error stopped new reads and the rest are reaped
    int e = r->enter(1);
    if (e) {
      // nothing more can be waited for safely: drop the ring's state by
      // reaping what is there, then report
      st = fail(NP_ERR_IO, "io_uring_enter: %s", strerror(e));
      break;
    }
    uint64_t tag;
    int res;
    while (r->pop(&tag, &res)) {
      --inflight;
      Req& q = reqs[(size_t)tag];
      if (res < 0) {
        if (st == NP_OK) st = fail(NP_ERR_IO, "record read at offset %llu: %s",
                                   (unsigned long long)q.off, strerror(-res));
        ++ndone;
        continue;
      }
      if (res == 0) {
        if (st == NP_OK) st = fail(NP_ERR_IO, "record read at offset %llu: end of file",
                                   (unsigned long long)q.off);
        ++ndone;
        continue;
      }
      q.buf += res;
      q.off += (uint64_t)res;
      q.left -= (size_t)res;
      if (q.left == 0) {
        ++ndone;
        if (done) ready.push_back((size_t)tag);
      } else if (st == NP_OK) {
        issue((size_t)tag);  // a short read: the remainder
      } else {
        ++ndone;
      }
    }
    if (!ready.empty()) {
      // refill the queue first, then hand over the finished pieces while the
      // new reads are in flight
      while (st == NP_OK && inflight < qd && next < reqs.size()) issue(next++);
      if (st == NP_OK && r->enter(0)) st = fail(NP_ERR_IO, "io_uring_enter (submit)");
      if (st == NP_OK)
        for (size_t i : ready) done(ctx, reqs[i].start, reqs[i].bytes);
      ready.clear();
    }
  }
  // a failed enter leaves requests in flight: wait for them before the
  // caller's buffers can go away
  while (inflight > 0) {
    if (r->enter(1)) break;
    uint64_t tag;
    int res;
    while (r->pop(&tag, &res)) --inflight;
  }
  return st;
}

}  // namespace np

using namespace np;

extern "C" np_status np_read_records(int32_t fd, int64_t file_offset, int64_t record_bytes,
                                     const int32_t* ids, int32_t n, void* dst) {
  if (n < 0) return fail(NP_ERR_INVALID_ARG, "np_read_records: n %d < 0", n);
  if (n == 0) return NP_OK;
  if (fd < 0 || file_offset < 0 || record_bytes < 1 || !ids || !dst)
    return fail(NP_ERR_INVALID_ARG, "np_read_records: bad fd, offset, record size or pointer");
  if (fcntl(fd, F_GETFL) < 0) return fail(NP_ERR_INVALID_ARG, "np_read_records: fd %d: %s", fd,
                                          strerror(errno));
  if (file_is_direct(fd) && ((file_offset | record_bytes) % IO_ALIGN || (uintptr_t)dst % IO_ALIGN))
    return fail(NP_ERR_INVALID_ARG,
                "np_read_records: an O_DIRECT file needs offset, record size and dst aligned to %d",
                IO_ALIGN);
  std::vector<ReadRun> runs;
  const size_t rec = (size_t)record_bytes;
  for (int j = 0; j < n; ++j) {
    if (ids[j] < 0) return fail(NP_ERR_INVALID_ARG, "np_read_records: id %d < 0", ids[j]);
    char* d = (char*)dst + (size_t)j * rec;
    const uint64_t off = (uint64_t)file_offset + (uint64_t)ids[j] * rec;
    if (j > 0 && ids[j] == ids[j - 1] + 1) runs.back().bytes += rec;  // adjacent: one range
    else runs.push_back({d, off, rec});
  }
  return read_runs(fd, runs, io_depth(), nullptr, nullptr);
}
