// Library-owned side streams: one per device, default priority, created on
// first use and kept for the life of the process, with a fork and a join event.
// A call that runs part of its work beside the caller's stream holds the lock
// from its fork to its join, since the events are shared.
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_side_mu;
SideStream g_side[kMaxDevices];

}  // namespace

std::unique_lock<std::mutex> side_stream_lock() { return std::unique_lock<std::mutex>(g_side_mu); }

hipError_t side_stream_get(SideStream*& out) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  SideStream& ss = g_side[dev];
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
