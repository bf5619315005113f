// Library-owned side streams: a pool of kSidePool per device, default
// priority, created on first use and kept for the life of the process, each
// with a fork and a join event and a lock of its own.  A call that runs part
// of its work beside the caller's stream takes the next entry round robin and
// holds its lock from its fork to its join, since the entry's events are
// shared with the next call that takes it; calls holding different entries
// proceed (and run on the GPU) concurrently.
#include <atomic>

#include "internal.hpp"

namespace laep {
namespace {

constexpr int kMaxDevices = 64;
struct SideSlot {
  std::mutex mu;
  SideStream ss;
};
SideSlot g_side[kMaxDevices][kSidePool];
std::atomic<unsigned> g_next[kMaxDevices];

}  // namespace

hipError_t side_stream_acquire(SideStream*& out, std::unique_lock<std::mutex>& lock) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  SideSlot& slot = g_side[dev][g_next[dev].fetch_add(1, std::memory_order_relaxed) % kSidePool];
  lock = std::unique_lock<std::mutex>(slot.mu);
  SideStream& ss = slot.ss;
  if (!ss.stream) {
    if ((err = hipStreamCreateWithFlags(&ss.stream, hipStreamNonBlocking)) != hipSuccess) return err;
    if ((err = hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming)) != hipSuccess) return err;
    if ((err = hipEventCreateWithFlags(&ss.join, hipEventDisableTiming)) != hipSuccess) return err;
  }
  out = &ss;
  return hipSuccess;
}

hipError_t side_stream_fork(const SideStream& ss, hipStream_t s) {
  hipError_t err = hipEventRecord(ss.fork, s);
  return err == hipSuccess ? hipStreamWaitEvent(ss.stream, ss.fork, 0) : err;
}

hipError_t side_stream_join(const SideStream& ss, hipStream_t s) {
  hipError_t err = hipEventRecord(ss.join, ss.stream);
  return err == hipSuccess ? hipStreamWaitEvent(s, ss.join, 0) : err;
}

}  // namespace laep
