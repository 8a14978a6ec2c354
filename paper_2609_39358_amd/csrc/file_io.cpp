// Record files: the disk tier under the host tier. Records of one context are
// kept back to back in one file (record id i at byte offset i * record_bytes);
// batches of records are read into (or written from) caller memory, normally
// pinned host memory that tl_load reads directly, by several threads issuing
// positional reads of whole records. Paper Sec. 4.3: the saved blocks live on
// disk and are streamed in for a restore, then dropped.
#include <errno.h>
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <new>
#include <thread>
#include <vector>

#include "internal.h"

struct tl_file {
  int fd;
  uint64_t record_bytes;
  int n_threads;
  bool writable;
};

namespace {

// Moves len bytes at offset through fd, retrying short transfers and EINTR.
bool transfer(int fd, char* buf, uint64_t len, uint64_t off, bool write) {
  while (len) {
    const size_t chunk = len < (1ull << 30) ? (size_t)len : (size_t)1 << 30;
    const ssize_t r = write ? pwrite(fd, buf, chunk, (off_t)off) : pread(fd, buf, chunk, (off_t)off);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;  // error, or end of file on a read
    buf += r;
    off += (uint64_t)r;
    len -= (uint64_t)r;
  }
  return true;
}

// Runs transfer() for n records on up to f->n_threads threads; records are
// handed out one at a time so that threads stay busy until the end.
int batch(const tl_file* f, const uint64_t* ids, size_t n, char* mem, bool write) {
  std::atomic<size_t> next{0};
  std::atomic<bool> ok{true};
  auto work = [&] {
    for (size_t i; ok.load(std::memory_order_relaxed) && (i = next.fetch_add(1)) < n;) {
      if (!transfer(f->fd, mem + i * f->record_bytes, f->record_bytes, ids[i] * f->record_bytes, write))
        ok = false;
    }
  };
  const size_t nt = std::min<size_t>((size_t)f->n_threads, n);
  std::vector<std::thread> pool;
  try {
    for (size_t t = 1; t < nt; ++t) pool.emplace_back(work);
  } catch (...) {
    ok = false;
  }
  work();
  for (auto& t : pool) t.join();
  return ok ? TL_OK : TL_EIO;
}

}  // namespace

extern "C" {

tl_file* tl_file_open(const char* path, uint64_t record_bytes, int flags, int n_threads, int* status) {
  int st_local;
  int* st = status ? status : &st_local;
  if (!path || !record_bytes || n_threads < 1 || n_threads > 256 || (flags & ~(TL_FILE_WRITE | TL_FILE_CREATE))) {
    *st = TL_EINVAL;
    return nullptr;
  }
  int oflags = (flags & TL_FILE_WRITE) ? O_RDWR : O_RDONLY;
  if (flags & TL_FILE_CREATE) oflags |= O_CREAT | O_TRUNC;
  const int fd = open(path, oflags | O_CLOEXEC, 0644);
  if (fd < 0) {
    *st = TL_EIO;
    return nullptr;
  }
  tl_file* f = new (std::nothrow) tl_file{fd, record_bytes, n_threads, (flags & TL_FILE_WRITE) != 0};
  if (!f) {
    close(fd);
    *st = TL_ENOMEM;
    return nullptr;
  }
  *st = TL_OK;
  return f;
}

int tl_file_close(tl_file* f) {
  if (!f) return TL_OK;
  const int r = close(f->fd);
  delete f;
  return r == 0 ? TL_OK : TL_EIO;
}

uint64_t tl_file_records(const tl_file* f) {
  struct stat sb;
  if (!f || fstat(f->fd, &sb) != 0) return 0;
  return (uint64_t)sb.st_size / f->record_bytes;
}

int tl_file_read(const tl_file* f, const uint64_t* record_ids, size_t n, void* dst) {
  if (!f) return TL_EINVAL;
  if (n == 0) return TL_OK;
  if (!record_ids || !dst) return TL_EINVAL;
  const uint64_t have = tl_file_records(f);
  for (size_t i = 0; i < n; ++i)
    if (record_ids[i] >= have) return TL_ERANGE;
  return batch(f, record_ids, n, (char*)dst, false);
}

int tl_file_write(tl_file* f, const uint64_t* record_ids, size_t n, const void* src) {
  if (!f) return TL_EINVAL;
  if (n == 0) return TL_OK;
  if (!record_ids || !src || !f->writable) return TL_EINVAL;
  for (size_t i = 0; i < n; ++i)
    if (record_ids[i] > (UINT64_MAX - f->record_bytes) / f->record_bytes) return TL_ERANGE;
  return batch(f, record_ids, n, (char*)src, true);
}

int tl_file_drop_cache(tl_file* f) {
  if (!f) return TL_EINVAL;
  if (f->writable && fsync(f->fd) != 0) return TL_EIO;
  return posix_fadvise(f->fd, 0, 0, POSIX_FADV_DONTNEED) == 0 ? TL_OK : TL_EIO;
}

}  // extern "C"
