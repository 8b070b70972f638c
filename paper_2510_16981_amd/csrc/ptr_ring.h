// Device table of the caller's per-step (param, grad) pointers, shared by
// the optimizer contexts.  The table is uploaded from pinned host memory
// only when the pointers differ from the previous step's; uploads rotate
// through the slots, and a slot's pinned copy is rewritten only after the
// event recorded behind its last upload has completed.
//
// A step captured into a HIP graph bakes the device address of the slot
// current at capture time into its kernels.  That slot is then pinned: no
// later upload writes it, so a replay after any number of eager steps with
// other pointers still reads the captured step's tensors.  When every slot
// is pinned a new one is allocated (outside capture only).
#pragma once
#include <hip/hip_runtime_api.h>

#include <vector>

#include "device_types.h"

namespace muonbp {

struct PtrRing {
  static constexpr int kInitialSlots = 8;
  static constexpr int kMaxSlots = 4096;
  struct Slot {
    MatPtrs* dev = nullptr;
    MatPtrs* host = nullptr;  // pinned
    hipEvent_t ev = nullptr;
    bool ev_used = false;
    bool pinned = false;      // referenced by a captured graph: never rewritten
  };
  size_t n = 0;
  std::vector<Slot> slots;
  int slot = -1;
  std::vector<MatPtrs> last;
  bool valid = false;

  hipError_t add_slot() {
    Slot s;
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, n * sizeof(MatPtrs));
    if (e != hipSuccess) return e;
    s.dev = static_cast<MatPtrs*>(p);
    slots.push_back(s);  // owned from here on (release frees what is set)
    if ((e = hipHostMalloc(&p, n * sizeof(MatPtrs), 0)) != hipSuccess) return e;
    slots.back().host = static_cast<MatPtrs*>(p);
    return hipEventCreateWithFlags(&slots.back().ev, hipEventDisableTiming);
  }

  hipError_t init(size_t count) {
    n = count;
    for (int i = 0; i < kInitialSlots; ++i) {
      hipError_t e = add_slot();
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }

  // Frees what init and add_slot allocated (the owner has synchronised its
  // stream).
  void release() {
    for (Slot& s : slots) {
      if (s.dev) (void)hipFree(s.dev);
      if (s.host) (void)hipHostFree(s.host);
      if (s.ev) (void)hipEventDestroy(s.ev);
    }
    slots.clear();
    slot = -1;
    valid = false;
  }

  // Forget the last upload (the next stage() uploads again), e.g. after a
  // change of stream.
  void invalidate() { valid = false; }

  // Make the table of this step current on stream s.  While s captures a
  // graph the table must be the one already current (the graph would
  // otherwise record a copy from a pinned host slot that later uploads
  // rewrite): new pointers are refused, and the current slot is pinned.
  hipError_t stage(void* const* params, const void* const* grads, hipStream_t s) {
    bool same = valid;
    for (size_t i = 0; same && i < n; ++i) same = last[i].param == params[i] && last[i].grad == grads[i];
    hipError_t e;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if ((e = hipStreamIsCapturing(s, &cap)) != hipSuccess) return e;
    if (cap != hipStreamCaptureStatusNone) {
      if (!same) return hipErrorStreamCaptureUnsupported;
      slots[size_t(slot)].pinned = true;
      return hipSuccess;
    }
    if (same) return hipSuccess;
    // The next slot after the current one that no graph holds.
    const int ns = int(slots.size());
    int next = -1;
    for (int k = 1; k <= ns && next < 0; ++k) {
      const int cand = (slot + k + ns) % ns;
      if (!slots[size_t(cand)].pinned) next = cand;
    }
    if (next < 0) {
      if (ns >= kMaxSlots) return hipErrorOutOfMemory;
      if ((e = add_slot()) != hipSuccess) return e;
      next = ns;
    }
    Slot& sl = slots[size_t(next)];
    if (sl.ev_used && (e = hipEventSynchronize(sl.ev)) != hipSuccess) return e;
    for (size_t i = 0; i < n; ++i) sl.host[i] = MatPtrs{params[i], grads[i]};
    if ((e = hipMemcpyAsync(sl.dev, sl.host, n * sizeof(MatPtrs), hipMemcpyHostToDevice, s)) !=
        hipSuccess)
      return e;
    if ((e = hipEventRecord(sl.ev, s)) != hipSuccess) return e;
    sl.ev_used = true;
    slot = next;
    last.assign(sl.host, sl.host + n);
    valid = true;
    return hipSuccess;
  }

  const MatPtrs* current() const { return slots[size_t(slot)].dev; }
};

}  // namespace muonbp
