// Host waits with a short wake-up. A host thread that sleeps in a stream
// synchronisation is woken some tens of microseconds after the GPU finishes,
// and a small copy into pageable memory waits the same way. The library
// waits after every stopping check of a solve and every few passes of the
// spectral iterations. So it records an event and polls it, with small
// read-backs landing in pinned host memory. The poll spins only briefly,
// then yields the core between polls, then sleeps between polls, so that a
// long wait (or a kernel that never ends) does not hold a host core.
#pragma once

#include <sched.h>
#include <string.h>
#include <time.h>

#include <mutex>
#include <vector>

#include "common.h"

namespace optima {

constexpr int kMailboxDevices = 64;
constexpr size_t kMailboxBytes = 256;
// Poll phases of a host wait: busy polls for the first kSpinUs, polls with a
// yield of the core in between up to kYieldUs, then a kNapNs sleep between
// polls. A solve's waits between checks are a few milliseconds at most on
// the layers measured, so they stay in the first two phases.
constexpr double kSpinUs = 50.0;
constexpr double kYieldUs = 20000.0;
constexpr long kNapNs = 100000;

// A pinned host buffer and a timing-free event for one host thread and one
// device. Calls from one host thread run one after another, so they never
// share it at once.
struct HostMailbox {
  void* host = nullptr;
  hipEvent_t ev = nullptr;
};

// Mailboxes of host threads that have ended, handed to the next thread that
// needs one: their count is bounded by the largest number of host threads
// that used the library at the same time. Nothing is released with a HIP
// call at thread or process exit (the runtime may already be gone then); the
// pool is left to the process's end.
struct MailboxPool {
  std::mutex mu;
  std::vector<HostMailbox> spare[kMailboxDevices];
};

inline MailboxPool& mailbox_pool() {
  static MailboxPool* pool = new MailboxPool;
  return *pool;
}

struct ThreadMailboxes {
  HostMailbox box[kMailboxDevices];
  ~ThreadMailboxes() {
    MailboxPool& p = mailbox_pool();
    std::lock_guard<std::mutex> g(p.mu);
    for (int d = 0; d < kMailboxDevices; ++d)
      if (box[d].ev) p.spare[d].push_back(box[d]);
  }
};

inline hipError_t mailbox_for(hipStream_t s, HostMailbox** out) {
  int dev = 0;
  hipError_t e = hipStreamGetDevice(s, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMailboxDevices) return hipErrorInvalidDevice;
  thread_local ThreadMailboxes mine;
  HostMailbox& b = mine.box[dev];
  if (!b.ev) {
    MailboxPool& p = mailbox_pool();
    std::lock_guard<std::mutex> g(p.mu);
    if (!p.spare[dev].empty()) {
      b = p.spare[dev].back();
      p.spare[dev].pop_back();
    }
  }
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

inline double elapsed_us(const timespec& t0) {
  timespec t;
  clock_gettime(CLOCK_MONOTONIC, &t);
  return double(t.tv_sec - t0.tv_sec) * 1e6 + double(t.tv_nsec - t0.tv_nsec) * 1e-3;
}

inline hipError_t poll_event(hipEvent_t ev) {
  hipError_t e = hipEventQuery(ev);
  if (e != hipErrorNotReady) return e;
  timespec t0;
  clock_gettime(CLOCK_MONOTONIC, &t0);
  while ((e = hipEventQuery(ev)) == hipErrorNotReady) {
    const double us = elapsed_us(t0);
    if (us < kSpinUs) continue;
    if (us < kYieldUs) {
      sched_yield();
    } else {
      const timespec nap{0, kNapNs};
      nanosleep(&nap, nullptr);
    }
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

// The same two waits without the pinned mailbox, for calls that may not
// allocate: the copy lands in the caller's host memory and the stream is
// synchronised (a longer wake-up, no allocation).
inline hipError_t read_back_plain(void* dst, const void* src, size_t bytes, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(s);
}

inline hipError_t wait_stream_plain(hipStream_t s) { return hipStreamSynchronize(s); }

}  // namespace optima
