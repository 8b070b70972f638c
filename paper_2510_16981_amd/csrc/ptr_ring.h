// Device table of the caller's per-step (param, grad) pointers, shared by
// the optimizer contexts.  The table is uploaded from pinned host memory
// only when the pointers differ from the previous step's; uploads rotate
// through kSlots slots, and a slot's pinned copy is rewritten only after the
// event recorded behind its last upload has completed.
#pragma once
#include <hip/hip_runtime_api.h>

#include <vector>

#include "device_types.h"

namespace muonbp {

struct PtrRing {
  static constexpr int kSlots = 8;
  size_t n = 0;
  MatPtrs* dev[kSlots] = {};
  MatPtrs* host[kSlots] = {};  // pinned
  hipEvent_t ev[kSlots] = {};
  bool ev_used[kSlots] = {};
  int slot = -1;
  std::vector<MatPtrs> last;
  bool valid = false;

  hipError_t init(size_t count) {
    n = count;
    for (int i = 0; i < kSlots; ++i) {
      void* p = nullptr;
      hipError_t e = hipMalloc(&p, n * sizeof(MatPtrs));
      if (e != hipSuccess) return e;
      dev[i] = static_cast<MatPtrs*>(p);
      if ((e = hipHostMalloc(&p, n * sizeof(MatPtrs), 0)) != hipSuccess) return e;
      host[i] = static_cast<MatPtrs*>(p);
      if ((e = hipEventCreateWithFlags(&ev[i], hipEventDisableTiming)) != hipSuccess) return e;
    }
    return hipSuccess;
  }

  // Frees what init allocated (the owner has synchronised its stream).
  void release() {
    for (int i = 0; i < kSlots; ++i) {
      if (dev[i]) (void)hipFree(dev[i]);
      if (host[i]) (void)hipHostFree(host[i]);
      if (ev[i]) (void)hipEventDestroy(ev[i]);
      dev[i] = nullptr;
      host[i] = nullptr;
      ev[i] = nullptr;
    }
  }

  // Forget the last upload (the next stage() uploads again), e.g. after a
  // change of stream.
  void invalidate() { valid = false; }

  // Make the table of this step current on stream s.  Refused while s is
  // capturing a graph: the graph would record a copy from a pinned slot
  // that later uploads rewrite (a captured step must reuse the table of the
  // step before it).
  hipError_t stage(void* const* params, const void* const* grads, hipStream_t s) {
    bool same = valid;
    for (size_t i = 0; same && i < n; ++i) same = last[i].param == params[i] && last[i].grad == grads[i];
    if (same) return hipSuccess;
    hipError_t e;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if ((e = hipStreamIsCapturing(s, &cap)) != hipSuccess) return e;
    if (cap != hipStreamCaptureStatusNone) return hipErrorStreamCaptureUnsupported;
    const int next = (slot + 1) % kSlots;
    if (ev_used[next] && (e = hipEventSynchronize(ev[next])) != hipSuccess) return e;
    for (size_t i = 0; i < n; ++i) host[next][i] = MatPtrs{params[i], grads[i]};
    if ((e = hipMemcpyAsync(dev[next], host[next], n * sizeof(MatPtrs), hipMemcpyHostToDevice, s)) !=
        hipSuccess)
      return e;
    if ((e = hipEventRecord(ev[next], s)) != hipSuccess) return e;
    ev_used[next] = true;
    slot = next;
    last.assign(host[next], host[next] + n);
    valid = true;
    return hipSuccess;
  }

  const MatPtrs* current() const { return dev[slot]; }
};

}  // namespace muonbp
