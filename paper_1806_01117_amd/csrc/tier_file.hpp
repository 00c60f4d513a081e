// A file below the pinned host tier (a third level of checkpoint storage).
//
// The schedule's slow slots h = 0, 1, 2, ... are stored in increasing order
// during the sweep and prefetched in decreasing order during the reverse
// (Section 2).  The pinned host tier becomes a ring of R buffers in front of
// an (unlinked) file: slot h is copied into buffer h % R and written behind
// to the file at offset h * stride by the tier's I/O thread, once the copy
// into the buffer has landed; a later store into the same buffer waits for
// that write.  In the reverse, once slot h has been copied out of its buffer,
// the I/O thread reads slot h - R back into it, so that the next R prefetches
// find their states in pinned memory.  Host-side waits order the thread's
// work against the device copies; `wait` callbacks block until a device copy
// has finished.  Pure C++ (the caller supplies the waits).
#pragma once

#include <condition_variable>
#include <cstdint>
#include <deque>
#include <functional>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

namespace ambptt {

class FileTier {
 public:
  // Opens a new file in `dir` (removed from the directory at once; it lives
  // until the tier is destroyed).  ring: pinned buffers of `stride` bytes
  // from `base`, each holding `bytes` of one state.  Returns nullptr and sets
  // *err on failure.
  static FileTier* open(const std::string& dir, int64_t capacity, std::string* err);
  ~FileTier();

  // Starts a pass over the given pinned ring (no buffer holds a slot).
  void begin(char* base, int64_t ring, size_t stride, size_t bytes);
  // Store of slot h: waits until its buffer is free, returns it (nullptr on error).
  char* store_buffer(int64_t h);
  // The copy of slot h into its buffer is enqueued: write it behind once wait() returns.
  void stored(int64_t h, std::function<bool()> wait);
  // Prefetch of slot h: waits until its buffer holds h, returns it (nullptr on error).
  char* prefetch_buffer(int64_t h);
  // The copy of slot h out of its buffer is enqueued (or not needed): read
  // slot h - R into the buffer once wait() returns.
  void prefetched(int64_t h, std::function<bool()> wait);
  // Waits until the thread is idle; false if any step failed (see error()).
  bool finish();
  // Seconds to write one state of `bytes` to the file (for the interval rule).
  double time_write(const char* src, size_t bytes);

  const std::string& error() const { return err_; }
  int64_t capacity() const { return cap_; }
  int64_t bytes_written = 0, bytes_read = 0;

 private:
  struct Job {
    bool write;
    int64_t h;
    int64_t b;
    std::function<bool()> wait;
  };
  FileTier() = default;
  void loop();
  bool wait_until(std::unique_lock<std::mutex>& lk, const std::function<bool()>& ready);

  int fd_ = -1;
  int64_t cap_ = 0;
  char* base_ = nullptr;
  int64_t ring_ = 0;
  size_t stride_ = 0, bytes_ = 0;
  std::vector<int64_t> holds_;  // slot held by each buffer, -1 if none
  std::vector<int> busy_;       // writes and reads of the buffer queued or running
  std::deque<Job> jobs_;
  bool running_ = false, stop_ = false, failed_ = false;
  std::string err_;
  std::mutex mu_;
  std::condition_variable cv_;
  std::thread io_;
};

}  // namespace ambptt
