// Stream-ordered workspace memory of the device entry points, from a memory
// pool the library creates once per device.  The pool keeps memory that was
// freed for the next call (its release threshold is unbounded), so a call's
// workspace is not mapped and unmapped again around every synchronisation,
// which the default pool does at a cost of milliseconds now and then.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>

namespace frog {

hipError_t ws_alloc(void** ptr, size_t bytes, hipStream_t stream);
hipError_t ws_free(void* ptr, hipStream_t stream);

// The search's workspace for work enqueued on `stream`: one buffer per
// (device, stream), kept between calls and grown (stream-ordered) only when a
// call needs more, so that the steady state allocates nothing.  A lease holds
// the buffer's lock while the caller enqueues (two threads on one stream take
// turns; other streams have buffers of their own).  Earlier uses of a
// stream's buffer were enqueued on the same stream, so stream order keeps
// them apart; no event or marker is added to the stream.
struct Slot;

class WsLease {
  public:
    WsLease() = default;
    WsLease(const WsLease&) = delete;
    WsLease& operator=(const WsLease&) = delete;
    ~WsLease() { release(); }
    // a buffer of at least `bytes` on `stream`; *ptr receives it
    hipError_t acquire(hipStream_t stream, size_t bytes, void** ptr);
    // after the call's last enqueue (also done by the destructor)
    void release();

  private:
    Slot* slot_ = nullptr;
};

}  // namespace frog
