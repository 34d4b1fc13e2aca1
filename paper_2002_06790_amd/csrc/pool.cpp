// Scratch sets handed to calls, so that calls on different streams that share
// one graph never use one copy of its scratch memory at the same time.
#include "sim.hpp"

namespace mlsim {

int ScratchPool::init(size_t nbytes, int n, bool with_capture, int (*fill)(void *ctx, char *base), void *ctx) {
  bytes = nbytes;
  sets.assign((size_t)n, Set{});
  auto make = [&](Set &s) -> int {
    if (hipMalloc((void **)&s.base, bytes ? bytes : 256) != hipSuccess) {
      s.base = nullptr;
      return SIM_E_NOMEM;
    }
    if (hipEventCreateWithFlags(&s.done, hipEventDisableTiming) != hipSuccess) {
      s.done = nullptr;
      return SIM_E_HIP;
    }
    return fill ? fill(ctx, s.base) : SIM_OK;
  };
  for (Set &s : sets)
    if (int rc = make(s)) return rc;
  if (with_capture)
    if (int rc = make(capture)) return rc;
  return hipDeviceSynchronize() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

void ScratchPool::destroy() {
  auto drop = [](Set &s) {
    if (s.base) (void)hipFree(s.base);
    if (s.done) (void)hipEventDestroy(s.done);
    s = Set{};
  };
  for (Set &s : sets) drop(s);
  drop(capture);
  sets.clear();
}

Lease::Lease(ScratchPool &pool, hipStream_t stream) : pool_(pool), lock_(pool.mu), stream_(stream) {
  if (pool_.sets.empty()) {
    rc_ = SIM_E_HIP;
    return;
  }
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
    rc_ = SIM_E_HIP;
    return;
  }
  if (cs != hipStreamCaptureStatusNone) {
    // a capture records no event and waits for none
    capturing_ = true;
    set_ = pool_.capture.base ? &pool_.capture : &pool_.sets[0];
    return;
  }
  ScratchPool::Set *pick = nullptr;
  for (auto &s : pool_.sets)  // last used on this stream: already ordered after it
    if (s.used && s.last == stream && (!pick || s.tick > pick->tick)) pick = &s;
  if (!pick)
    for (auto &s : pool_.sets)  // never used, or its last call has finished
      if (!s.used || hipEventQuery(s.done) == hipSuccess) {
        pick = &s;
        break;
      }
  if (!pick)
    for (auto &s : pool_.sets)  // least recently used
      if (!pick || s.tick < pick->tick) pick = &s;
  // order this call after the set's previous user (a no-op when it is this
  // stream's own earlier call or has finished)
  if (pick->used && hipStreamWaitEvent(stream, pick->done, 0) != hipSuccess) {
    rc_ = SIM_E_HIP;
    return;
  }
  set_ = pick;
}

Lease::~Lease() {
  if (!set_ || capturing_) return;
  // after the call's last launch; a failed launch enqueued nothing, so the
  // event then completes with the stream's earlier work
  if (hipEventRecord(set_->done, stream_) == hipSuccess) {
    set_->used = true;
    set_->last = stream_;
    set_->tick = ++pool_.clock;
  }
}

}  // namespace mlsim
