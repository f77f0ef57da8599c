// Host waits with a short wake-up. A host thread that sleeps in a stream
// synchronisation is woken some tens of microseconds after the GPU finishes,
// and a small copy into pageable memory waits the same way. The library
// waits after every stopping check of a solve and every few passes of the
// spectral iterations. So it records an event and polls it, with small
// read-backs landing in pinned host memory.
#pragma once

#include <string.h>

#include "common.h"

namespace optima {

constexpr int kMailboxDevices = 64;
constexpr size_t kMailboxBytes = 256;

// A pinned host buffer and a timing-free event for one host thread and one
// device, made on first use and kept until the process ends. Calls from one
// host thread run one after another, so they never share it at once.
struct HostMailbox {
  void* host = nullptr;
  hipEvent_t ev = nullptr;
};

inline hipError_t mailbox_for(hipStream_t s, HostMailbox** out) {
  int dev = 0;
  hipError_t e = hipStreamGetDevice(s, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMailboxDevices) return hipErrorInvalidDevice;
  thread_local HostMailbox boxes[kMailboxDevices];
  HostMailbox& b = boxes[dev];
  if (!b.ev) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* host = nullptr;
    hipEvent_t ev = nullptr;
    e = hipHostMalloc(&host, kMailboxBytes, hipHostMallocDefault);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess) {
      if (host) (void)hipHostFree(host);
      return e;
    }
    b.host = host;
    b.ev = ev;
  }
  *out = &b;
  return hipSuccess;
}

inline hipError_t poll_event(hipEvent_t ev) {
  hipError_t e;
  while ((e = hipEventQuery(ev)) == hipErrorNotReady) {
  }
  return e;
}

// Returns once the work queued on s so far has finished.
inline hipError_t wait_stream(hipStream_t s) {
  HostMailbox* b = nullptr;
  hipError_t e = mailbox_for(s, &b);
  if (e != hipSuccess) return e;
  if ((e = hipEventRecord(b->ev, s)) != hipSuccess) return e;
  return poll_event(b->ev);
}

// Copies `bytes` (at most kMailboxBytes) of device memory at src into dst
// once the work queued on s so far has finished.
inline hipError_t read_back(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (bytes > kMailboxBytes) return hipErrorInvalidValue;
  HostMailbox* b = nullptr;
  hipError_t e = mailbox_for(s, &b);
  if (e != hipSuccess) return e;
  if ((e = hipMemcpyAsync(b->host, src, bytes, hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
  if ((e = hipEventRecord(b->ev, s)) != hipSuccess) return e;
  if ((e = poll_event(b->ev)) != hipSuccess) return e;
  memcpy(dst, b->host, bytes);
  return hipSuccess;
}

}  // namespace optima
