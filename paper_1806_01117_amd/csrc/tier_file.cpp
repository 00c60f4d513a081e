// The file tier below the pinned host tier: see tier_file.hpp.
#include "tier_file.hpp"

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <cerrno>
#include <chrono>
#include <cstring>

namespace ambptt {

namespace {

bool full_io(bool write, int fd, char* p, size_t n, off_t off) {
  while (n > 0) {
    const ssize_t r = write ? pwrite(fd, p, n, off) : pread(fd, p, n, off);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;
    p += r;
    n -= size_t(r);
    off += r;
  }
  return true;
}

}  // namespace

FileTier* FileTier::open(const std::string& dir, int64_t capacity, std::string* err) {
  if (capacity < 1) {
    *err = "file tier: capacity must be >= 1 slot";
    return nullptr;
  }
  std::string tmpl = (dir.empty() ? std::string(".") : dir) + "/ambptt-tier-XXXXXX";
  std::vector<char> name(tmpl.begin(), tmpl.end());
  name.push_back('\0');
  const int fd = mkstemp(name.data());
  if (fd < 0) {
    *err = "file tier: cannot create a file in " + dir + ": " + std::strerror(errno);
    return nullptr;
  }
  unlink(name.data());  // the file lives until it is closed
  FileTier* t = new FileTier();
  t->fd_ = fd;
  t->cap_ = capacity;
  t->io_ = std::thread([t] { t->loop(); });
  return t;
}

FileTier::~FileTier() {
  {
    std::lock_guard<std::mutex> lk(mu_);
    stop_ = true;
  }
  cv_.notify_all();
  if (io_.joinable()) io_.join();
  if (fd_ >= 0) close(fd_);
}

void FileTier::begin(char* base, int64_t ring, size_t stride, size_t bytes) {
  std::lock_guard<std::mutex> lk(mu_);
  base_ = base;
  ring_ = ring;
  stride_ = stride;
  bytes_ = bytes;
  holds_.assign(size_t(ring), -1);
  busy_.assign(size_t(ring), 0);
  failed_ = false;
  err_.clear();
}

bool FileTier::wait_until(std::unique_lock<std::mutex>& lk, const std::function<bool()>& ready) {
  cv_.wait(lk, [&] { return failed_ || ready(); });
  return !failed_;
}

char* FileTier::store_buffer(int64_t h) {
  if (h < 0 || h >= cap_) {
    std::lock_guard<std::mutex> lk(mu_);
    failed_ = true;
    err_ = "file tier: slot " + std::to_string(h) + " beyond its capacity";
    return nullptr;
  }
  const int64_t b = h % ring_;
  std::unique_lock<std::mutex> lk(mu_);
  if (!wait_until(lk, [&] { return busy_[size_t(b)] == 0; })) return nullptr;
  holds_[size_t(b)] = -1;
  return base_ + size_t(b) * stride_;
}

void FileTier::stored(int64_t h, std::function<bool()> wait) {
  const int64_t b = h % ring_;
  {
    std::lock_guard<std::mutex> lk(mu_);
    holds_[size_t(b)] = h;
    ++busy_[size_t(b)];
    jobs_.push_back({true, h, b, std::move(wait)});
  }
  cv_.notify_all();
}

char* FileTier::prefetch_buffer(int64_t h) {
  const int64_t b = h % ring_;
  std::unique_lock<std::mutex> lk(mu_);
  if (!wait_until(lk, [&] { return busy_[size_t(b)] == 0; })) return nullptr;
  if (holds_[size_t(b)] != h) {  // no queued read brings it: prefetches out of order
    failed_ = true;
    err_ = "file tier: slot " + std::to_string(h) + " is not in its buffer (prefetches must go in decreasing order)";
    return nullptr;
  }
  return base_ + size_t(b) * stride_;
}

void FileTier::prefetched(int64_t h, std::function<bool()> wait) {
  const int64_t prev = h - ring_;
  if (prev < 0) return;
  const int64_t b = h % ring_;
  {
    std::lock_guard<std::mutex> lk(mu_);
    ++busy_[size_t(b)];
    jobs_.push_back({false, prev, b, std::move(wait)});
  }
  cv_.notify_all();
}

bool FileTier::finish() {
  std::unique_lock<std::mutex> lk(mu_);
  cv_.wait(lk, [&] { return failed_ || (jobs_.empty() && !running_); });
  return !failed_;
}

double FileTier::time_write(const char* src, size_t bytes) {
  const auto t0 = std::chrono::steady_clock::now();
  const bool ok = full_io(true, fd_, const_cast<char*>(src), bytes, 0);
  const auto t1 = std::chrono::steady_clock::now();
  return ok ? std::chrono::duration<double>(t1 - t0).count() : -1.0;
}

void FileTier::loop() {
  for (;;) {
    Job j;
    {
      std::unique_lock<std::mutex> lk(mu_);
      cv_.wait(lk, [&] { return stop_ || !jobs_.empty(); });
      if (stop_) return;
      j = std::move(jobs_.front());
      jobs_.pop_front();
      running_ = true;
    }
    bool ok = j.wait();
    std::string why = ok ? "" : "file tier: waiting for a device copy failed";
    if (ok) {
      char* buf = base_ + size_t(j.b) * stride_;
      ok = full_io(j.write, fd_, buf, bytes_, off_t(j.h) * off_t(stride_));
      if (!ok) why = std::string("file tier: ") + (j.write ? "write" : "read") + " of slot " + std::to_string(j.h) +
                     " failed: " + std::strerror(errno);
    }
    {
      std::lock_guard<std::mutex> lk(mu_);
      running_ = false;
      if (!ok) {
        failed_ = true;
        err_ = why;
      } else if (j.write) {
        bytes_written += int64_t(bytes_);
      } else {
        holds_[size_t(j.b)] = j.h;
        bytes_read += int64_t(bytes_);
      }
      --busy_[size_t(j.b)];
    }
    cv_.notify_all();
  }
}

}  // namespace ambptt
