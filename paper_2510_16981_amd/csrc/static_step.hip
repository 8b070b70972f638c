// Allocation-free MuonBP step (muonbp_step_static, declared in
// include/muonbp.h): the step of muonbp_step with every buffer the step
// needs besides the caller's tensors held in one file-scope device array.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is taken once per GPU with hipGetSymbolAddress (with that
// GPU current) and only that address is ever handed to kernels or copies.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/muonbp.h"
#include "kernels.h"
#include "plan.h"
#include "step_core.h"

// The step's scratch memory on every GPU the library runs on.
static __device__ __align__(256) unsigned char scratch[MUONBP_STATIC_SCRATCH_BYTES];

namespace muonbp {
namespace {

constexpr int64_t kStaticScratchBytes = MUONBP_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this GPU's scratch array (the current device's),
// looked up on the first call on that GPU.
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

template <typename T>
hipError_t copy_in(char* base, int64_t off, const std::vector<T>& v, hipStream_t s) {
  if (v.empty()) return hipSuccess;
  return hipMemcpyAsync(base + off, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice, s);
}

muonbp_status hip_status(hipError_t e) {
  return e == hipSuccess ? MUONBP_OK : MUONBP_E_HIP;
}

}  // namespace
}  // namespace muonbp

using namespace muonbp;

extern "C" muonbp_status muonbp_step_static(const muonbp_matrix* mats, int32_t n_mats,
                                            void* const* params, const void* const* grads,
                                            void* momentum, int64_t step, int64_t period,
                                            float lr_block, float lr_full, float momentum_mu,
                                            float weight_decay, const muonbp_options* opt,
                                            void* hip_stream) {
  // Host-side checks and planning, before any HIP call.
  muonbp_options o;
  muonbp_options_default(&o);
  if (opt) o = *opt;
  if (!params || !grads || !momentum || step < 0 || period < 0) return MUONBP_E_INVALID;
  if (!std::isfinite(lr_block) || !std::isfinite(lr_full) || !std::isfinite(momentum_mu) ||
      !std::isfinite(weight_decay))
    return MUONBP_E_INVALID;
  if (!validate_opts(o).empty()) return MUONBP_E_INVALID;
  if (!dtype_ok(o.param_dtype) || !dtype_ok(o.state_dtype) || !dtype_ok(o.ns_dtype))
    return MUONBP_E_DTYPE;
  std::vector<MatrixShape> shapes;
  if (!check_mats(mats, n_mats, &shapes).empty()) return MUONBP_E_INVALID;
  const size_t pb = dtype_size(o.param_dtype), sb = dtype_size(o.state_dtype);
  bool aligned = reinterpret_cast<uintptr_t>(momentum) % 16 == 0;
  if (reinterpret_cast<uintptr_t>(momentum) % sb) return MUONBP_E_INVALID;
  for (int32_t i = 0; i < n_mats; ++i) {
    if (!params[i] || !grads[i]) return MUONBP_E_INVALID;
    if (reinterpret_cast<uintptr_t>(params[i]) % pb || reinterpret_cast<uintptr_t>(grads[i]) % pb)
      return MUONBP_E_INVALID;
    aligned = aligned && reinterpret_cast<uintptr_t>(params[i]) % 16 == 0 &&
              reinterpret_cast<uintptr_t>(grads[i]) % 16 == 0;
  }
  const int full = (period > 0 && step % period == 0) ? 1 : 0;
  Layout lay;
  ScratchPlan sp;
  PlanHostTables h;
  std::vector<BlockDesc> bd;
  try {
    bool shape_err = false;
    if (!layout_for(shapes, o, &lay, &shape_err, reinterpret_cast<uintptr_t>(momentum) % 16 == 0).empty())
      return shape_err ? MUONBP_E_SHAPE : MUONBP_E_INVALID;
    sp = scratch_plan(lay, full, o);
    if (sp.total > kStaticScratchBytes) return MUONBP_E_TOO_LARGE;
    bd = block_descs(lay);
  } catch (const std::bad_alloc&) {
    return MUONBP_E_NOMEM;
  }
  aligned = aligned && layout_vectorizable(lay);

  // Device side: the scratch array of the current GPU.
  void* base_v = nullptr;
  hipError_t e = scratch_address(&base_v);
  if (e != hipSuccess) return hip_status(e);
  char* base = static_cast<char*>(base_v);
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const Plan& plan = lay.plan[full];
  std::vector<MatPtrs> ptrs(static_cast<size_t>(n_mats));
  std::vector<const TileRef*> phase_tiles(plan.phases.size());
  try {
    build_plan_host_tables(lay, o, full, base + sp.ws, momentum, reinterpret_cast<const float*>(base + sp.scales),
                           &h);
  } catch (const std::bad_alloc&) {
    return MUONBP_E_NOMEM;
  }
  for (int32_t i = 0; i < n_mats; ++i) ptrs[size_t(i)] = MatPtrs{params[i], grads[i]};
  // Tables into the scratch array; the host vectors are the copies' sources,
  // so every return from here on waits for the stream first.
  auto done = [&](hipError_t err) {
    const hipError_t w = hipStreamSynchronize(s);
    return hip_status(err != hipSuccess ? err : w);
  };
  if ((e = copy_in(base, sp.segs, lay.segs, s)) != hipSuccess ||
      (e = copy_in(base, sp.blocks, bd, s)) != hipSuccess ||
      (e = copy_in(base, sp.scale_d, h.scale, s)) != hipSuccess ||
      (e = copy_in(base, sp.pack_d, h.pack, s)) != hipSuccess ||
      (e = copy_in(base, sp.pack_tiles, plan.pack_tiles, s)) != hipSuccess ||
      (e = copy_in(base, sp.descs, h.descs, s)) != hipSuccess ||
      (e = copy_in(base, sp.upd, h.upd, s)) != hipSuccess ||
      (e = copy_in(base, sp.ptrs, ptrs, s)) != hipSuccess)
    return done(e);
  for (size_t ph = 0; ph < plan.phases.size(); ++ph) {
    if ((e = copy_in(base, sp.phase_tiles[ph], plan.phases[ph].tiles, s)) != hipSuccess)
      return done(e);
    phase_tiles[ph] = reinterpret_cast<const TileRef*>(base + sp.phase_tiles[ph]);
  }
  // The K-split counters must start at zero (the kernels leave them zeroed,
  // but an earlier call may have stopped short of that).
  if (plan.split_slots > 0 &&
      (e = hipMemsetAsync(base + sp.kcount, 0, size_t(plan.split_slots) * 4, s)) != hipSuccess)
    return done(e);

  StepBuffers b;
  b.mom = momentum;
  b.partials = reinterpret_cast<float*>(base + sp.partials);
  b.scales = reinterpret_cast<float*>(base + sp.scales);
  b.ksum = reinterpret_cast<float*>(base + sp.ksum);
  b.kcount = reinterpret_cast<int*>(base + sp.kcount);
  b.segs = reinterpret_cast<const SegDesc*>(base + sp.segs);
  b.blocks = reinterpret_cast<const BlockDesc*>(base + sp.blocks);
  b.mats = reinterpret_cast<const MatPtrs*>(base + sp.ptrs);
  b.n_segs = int(lay.segs.size());
  StepScalars sc;
  sc.mu = momentum_mu;
  sc.eta = full ? lr_full : lr_block;
  sc.wd = weight_decay;
  sc.vec = aligned;
  sc.nt = stream_nontemporal(lay, o);
  PlanView pv;
  pv.scale = reinterpret_cast<const ScaleDesc*>(base + sp.scale_d);
  pv.pack = reinterpret_cast<const PackDesc*>(base + sp.pack_d);
  pv.pack_tiles = reinterpret_cast<const TileRef*>(base + sp.pack_tiles);
  pv.descs = reinterpret_cast<const GemmDesc*>(base + sp.descs);
  pv.phase_tiles = phase_tiles.data();
  pv.upd = reinterpret_cast<const UpdDesc*>(base + sp.upd);
  pv.fuse_scale = h.fuse_scale;

  auto wrap = [](int, auto&& launch) { return launch(); };
  if ((e = enqueue_momentum(o, b, sc, s, wrap)) != hipSuccess) return done(e);
  if (o.check_finite) {
    int flag = 0;
    int* dflag = reinterpret_cast<int*>(base + sp.scales);  // scales are written after this
    if ((e = launch_check_finite(b.n_segs, b.partials, dflag, s)) != hipSuccess ||
        (e = hipMemcpyAsync(&flag, dflag, sizeof(int), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
      return done(e);
    if (flag != 0) return MUONBP_E_NONFINITE;
  }
  const char* what = "";
  e = enqueue_after_momentum(o, plan, pv, b, sc, s, wrap, [](bool, int) { return hipSuccess; }, &what);
  // The wait also completes the step.
  return done(e);
}
