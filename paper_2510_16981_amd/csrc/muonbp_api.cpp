// C ABI of the MuonBP optimizer step (declared in include/muonbp.h).
//
// The host side of Algorithm 1 (Sec. 3.2): it owns the momentum buffers and
// the NS workspace, picks the block or the full plan by step mod P, and
// enqueues the kernels of kernels.hip on the caller's stream.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "../../include/muonbp.h"
#include "kernels.h"
#include "plan.h"
#include "ptr_ring.h"
#include "step_core.h"

using namespace muonbp;

namespace {

struct PlanDev {
  ScaleDesc* scale = nullptr;
  PackDesc* pack = nullptr;
  TileRef* pack_tiles = nullptr;
  GemmDesc* descs = nullptr;             // Layout::desc_per_problem per problem
  std::vector<TileRef*> phase_tiles;     // one tile list per launch phase
  UpdDesc* upd = nullptr;
  std::vector<UpdDesc> upd_host;  // for muonbp_get_update
  bool fuse_scale = false;        // the pack computes the scales (no k_scale launch)

  PlanView view() const {
    PlanView v;
    v.scale = scale;
    v.pack = pack;
    v.pack_tiles = pack_tiles;
    v.descs = descs;
    v.phase_tiles = phase_tiles.data();
    v.upd = upd;
    v.fuse_scale = fuse_scale;
    return v;
  }
};

struct ProfRec {
  int kind;
  int full;      // launched by a full step
  int launches;  // launches between the two events
  hipEvent_t start, stop;
};

}  // namespace

struct muonbp_ctx {
  Layout lay;
  muonbp_options opt{};
  int64_t period = 0;
  float lr_block = 0, lr_full = 0, mu = 0, wd = 0;
  hipStream_t stream = nullptr;
  int device = 0;

  void* mom = nullptr;
  void* ws = nullptr;
  float* partials = nullptr;
  float* scales = nullptr;
  float* ksum = nullptr;   // fp32 partial sums of K-split NS GEMM launches
  int* kcount = nullptr;   // one arrival counter per tile of such a launch (kept zeroed)
  int* finite_flag = nullptr;       // check_finite: 1 when a partial sum is not finite
  int* finite_host = nullptr;       // pinned copy of it
  SegDesc* segs = nullptr;
  BlockDesc* blocks = nullptr;
  PlanDev pd[2];
  std::vector<void*> allocs;
  int64_t allocated = 0;  // bytes in allocs (device_memory_limit)

  PtrRing ptrs;  // caller's param / grad pointers of the current step

  bool vec_layout = false;
  bool stream_nt = false;  // nontemporal momentum / update accesses
  int last_plan = -1;
  bool poisoned = false;
  std::string err;

  int prof = 0;  // 0 off, 1 every launch, 2 one span over the NS GEMM launches
  std::vector<ProfRec> prof_recs;
  std::vector<hipEvent_t> ev_pool;
  int prof_full = 0;  // kind of the step being enqueued
};

namespace {

muonbp_status fail(muonbp_ctx* c, muonbp_status s, const std::string& msg) {
  if (c) c->err = msg;
  return s;
}

muonbp_status hip_fail(muonbp_ctx* c, hipError_t e, const char* what) {
  if (c) {
    c->poisoned = true;
    c->err = std::string(what) + ": " + hipGetErrorString(e);
  }
  return MUONBP_E_HIP;
}

// Copies a host table into new device memory on the context's stream and
// waits for that stream only (no device-wide synchronisation, which would
// also wait for, or break a graph capture on, the caller's other streams).
hipError_t dev_alloc(muonbp_ctx* c, void** p, size_t bytes);

template <typename T>
hipError_t upload(muonbp_ctx* c, T** dst, const std::vector<T>& src) {
  *dst = nullptr;
  if (src.empty()) return hipSuccess;
  void* p = nullptr;
  hipError_t e = dev_alloc(c, &p, src.size() * sizeof(T));
  if (e != hipSuccess) return e;
  *dst = static_cast<T*>(p);
  e = hipMemcpyAsync(p, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice, c->stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(c->stream);
}

// hipMalloc within the context's device_memory_limit (over it: out of
// memory, without calling hipMalloc).
hipError_t dev_alloc(muonbp_ctx* c, void** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  const int64_t limit = c->opt.device_memory_limit;
  if (limit > 0 && int64_t(bytes) > limit - c->allocated) return hipErrorOutOfMemory;
  hipError_t e = hipMalloc(p, bytes);
  if (e == hipSuccess) {
    c->allocs.push_back(*p);
    c->allocated += int64_t(bytes);
  }
  return e;
}

// Device tables of one plan (needs c->ws allocated).
hipError_t build_plan_tables(muonbp_ctx* c, int full) {
  const Plan& plan = c->lay.plan[full];
  PlanDev& pd = c->pd[full];
  PlanHostTables h;
  build_plan_host_tables(c->lay, c->opt, full, c->ws, c->mom, c->scales, &h);
  pd.fuse_scale = h.fuse_scale;
  pd.upd_host = h.upd;
  const std::vector<ScaleDesc>& sd = h.scale;
  const std::vector<PackDesc>& pk = h.pack;
  const std::vector<GemmDesc>& descs = h.descs;
  hipError_t e;
  if ((e = upload(c, &pd.scale, sd)) != hipSuccess) return e;
  if ((e = upload(c, &pd.pack, pk)) != hipSuccess) return e;
  if ((e = upload(c, &pd.pack_tiles, plan.pack_tiles)) != hipSuccess) return e;
  if ((e = upload(c, &pd.descs, descs)) != hipSuccess) return e;
  pd.phase_tiles.assign(plan.phases.size(), nullptr);
  for (size_t ph = 0; ph < plan.phases.size(); ++ph)
    if ((e = upload(c, &pd.phase_tiles[ph], plan.phases[ph].tiles)) != hipSuccess) return e;
  if ((e = upload(c, &pd.upd, pd.upd_host)) != hipSuccess) return e;
  return hipSuccess;
}

void free_ctx(muonbp_ctx* c) {
  if (!c) return;
  for (void* p : c->allocs) (void)hipFree(p);
  c->ptrs.release();
  for (auto& r : c->prof_recs) {
    (void)hipEventDestroy(r.start);
    if (r.stop) (void)hipEventDestroy(r.stop);
  }
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->finite_host) (void)hipHostFree(c->finite_host);
  delete c;
}

// Profiling helpers: bracket a launch with events when enabled.
hipEvent_t take_event(muonbp_ctx* c) {
  if (!c->ev_pool.empty()) {
    hipEvent_t e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
hipError_t timed(muonbp_ctx* c, int kind, F&& launch) {
  if (c->prof != 1) return launch();
  hipEvent_t a = take_event(c), b = take_event(c);
  hipError_t e = (a && b) ? hipEventRecord(a, c->stream) : hipErrorOutOfMemory;
  if (e == hipSuccess) e = launch();
  if (e == hipSuccess) e = hipEventRecord(b, c->stream);
  if (e != hipSuccess) {  // the events go back to the pool
    if (a) c->ev_pool.push_back(a);
    if (b) c->ev_pool.push_back(b);
    return e;
  }
  c->prof_recs.push_back(ProfRec{kind, c->prof_full, 1, a, b});
  return hipSuccess;
}

// Span mode: one event before the first and one after the last NS GEMM
// launch of a step (kind 7); the launches in between run back to back.
hipError_t span_mark(muonbp_ctx* c, bool begin, int launches) {
  if (c->prof != 2 || launches == 0) return hipSuccess;
  // The end mark closes the open span its begin mark left last.
  if (!begin && (c->prof_recs.empty() || c->prof_recs.back().kind != 7 || c->prof_recs.back().stop))
    return hipErrorInvalidValue;
  hipEvent_t ev = take_event(c);
  if (!ev) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(ev, c->stream);
  if (e != hipSuccess) {
    c->ev_pool.push_back(ev);
    return e;
  }
  if (begin) {
    c->prof_recs.push_back(ProfRec{7, c->prof_full, launches, ev, nullptr});
  } else {
    c->prof_recs.back().stop = ev;
  }
  return hipSuccess;
}

}  // namespace

extern "C" {

void muonbp_options_default(muonbp_options* o) {
  if (!o) return;
  std::memset(o, 0, sizeof(*o));
  o->ns_steps = 5;
  o->a = 2.0f;
  o->b = -1.5f;
  o->c = 0.5f;
  o->eps = 1e-7f;
  o->nesterov = 0;
  o->scale_mode = 0;
  o->rms_beta = 1.0f;
  o->param_dtype = MUONBP_BF16;
  o->state_dtype = MUONBP_BF16;
  o->ns_dtype = MUONBP_BF16;
  o->tile_policy = 0;
  o->k_split = 0;
}

const char* muonbp_status_string(muonbp_status s) {
  switch (s) {
    case MUONBP_OK: return "ok";
    case MUONBP_E_INVALID: return "invalid argument";
    case MUONBP_E_SHAPE: return "invalid shape or grid";
    case MUONBP_E_DTYPE: return "unsupported dtype";
    case MUONBP_E_NOMEM: return "out of memory";
    case MUONBP_E_HIP: return "HIP error";
    case MUONBP_E_STATE: return "context unusable after an earlier HIP error";
    case MUONBP_E_NONFINITE: return "non-finite orthogonalization input";
    case MUONBP_E_TOO_LARGE: return "step needs more than the static scratch array";
  }
  return "unknown status";
}

const char* muonbp_last_error(const muonbp_ctx* c) {
  if (!c) return "no context";
  return c->err.c_str();
}

muonbp_status muonbp_describe_plan(const muonbp_matrix* mats, int32_t n_mats,
                                   const muonbp_options* opt, int32_t full,
                                   muonbp_plan_info* out) {
  if (!out || (full != 0 && full != 1)) return MUONBP_E_INVALID;
  muonbp_options o;
  muonbp_options_default(&o);
  if (opt) o = *opt;
  if (!validate_opts(o).empty()) return MUONBP_E_INVALID;
  if (!dtype_ok(o.param_dtype) || !dtype_ok(o.state_dtype) || !dtype_ok(o.ns_dtype))
    return MUONBP_E_DTYPE;
  std::vector<MatrixShape> shapes;
  if (!check_mats(mats, n_mats, &shapes).empty()) return MUONBP_E_INVALID;
  Layout lay;
  bool shape_err = false;
  try {
    if (!layout_for(shapes, o, &lay, &shape_err).empty())
      return shape_err ? MUONBP_E_SHAPE : MUONBP_E_INVALID;
  } catch (const std::bad_alloc&) {
    return MUONBP_E_NOMEM;
  }
  const Plan& p = lay.plan[full];
  std::memset(out, 0, sizeof(*out));
  out->n_problems = int64_t(p.probs.size());
  out->n_elements = lay.total_elems;
  for (int k = 0; k < 3; ++k) {
    out->gemm_tiles[k] = p.tiles_per_iter[k];
    out->gemm_tile_rows[k] = kGemmTileRows[p.variant[k]];
    out->gemm_tile_cols[k] = kGemmTileCols[p.variant[k]];
    out->gemm_split[k] = p.nsplit[k];
  }
  out->gemm_launches = int64_t(p.phases.size());
  out->apply_nn = p.nn_apply ? 1 : 0;
  out->ns_flops = p.ns_flops;
  out->ns_dense_flops = p.ns_dense_flops;
  const double pb = double(dtype_size(o.param_dtype)), sb = double(dtype_size(o.state_dtype)),
               nb = double(dtype_size(o.ns_dtype));
  // momentum: read G, M, write M; update: read X, U, write X.
  out->elementwise_bytes = double(lay.total_elems) * ((pb + 2 * sb) + (2 * pb + nb));
  out->workspace_bytes = p.ws_elems * int64_t(nb);
  out->static_scratch_bytes = scratch_plan(lay, full, o).total;
  out->device_bytes = context_bulk_bytes(lay, o);
  for (const Problem& q : p.probs) {
    out->gram_units += q.gram ? 1 : 0;
    out->pack_elements += q.in_place ? 0 : q.rows * q.cols;
  }
  return MUONBP_OK;
}

muonbp_status muonbp_create(const muonbp_matrix* mats, int32_t n_mats, int64_t period,
                            float lr_block, float lr_full, float momentum, float weight_decay,
                            const muonbp_options* opt, void* hip_stream, muonbp_ctx** out) {
  if (!out) return MUONBP_E_INVALID;
  *out = nullptr;
  muonbp_options o;
  muonbp_options_default(&o);
  if (opt) o = *opt;
  if (period < 0) return MUONBP_E_INVALID;
  if (!std::isfinite(lr_block) || !std::isfinite(lr_full) || !std::isfinite(momentum) ||
      !std::isfinite(weight_decay))
    return MUONBP_E_INVALID;
  if (!validate_opts(o).empty()) return MUONBP_E_INVALID;
  if (!dtype_ok(o.param_dtype) || !dtype_ok(o.state_dtype) || !dtype_ok(o.ns_dtype))
    return MUONBP_E_DTYPE;
  std::vector<MatrixShape> shapes;
  if (!check_mats(mats, n_mats, &shapes).empty()) return MUONBP_E_INVALID;

  muonbp_ctx* c = new (std::nothrow) muonbp_ctx();
  if (!c) return MUONBP_E_NOMEM;
  try {
    bool shape_err = false;
    std::string msg = layout_for(shapes, o, &c->lay, &shape_err);
    if (!msg.empty()) {
      free_ctx(c);
      return shape_err ? MUONBP_E_SHAPE : MUONBP_E_INVALID;
    }
  } catch (const std::bad_alloc&) {
    free_ctx(c);
    return MUONBP_E_NOMEM;
  }
  if (o.device_memory_limit > 0 && context_bulk_bytes(c->lay, o) > o.device_memory_limit) {
    free_ctx(c);
    return MUONBP_E_NOMEM;
  }
  c->opt = o;
  c->period = period;
  c->lr_block = lr_block;
  c->lr_full = lr_full;
  c->mu = momentum;
  c->wd = weight_decay;
  c->stream = static_cast<hipStream_t>(hip_stream);

  // 16-byte vector paths need 8-element aligned windows and strides.
  c->vec_layout = layout_vectorizable(c->lay);
  c->stream_nt = stream_nontemporal(c->lay, o);

  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) {
    hip_fail(c, e, "hipGetDevice");
    free_ctx(c);
    return MUONBP_E_HIP;
  }
  auto bail = [&](hipError_t err, const char* what) {
    const muonbp_status st = (err == hipErrorOutOfMemory) ? MUONBP_E_NOMEM : MUONBP_E_HIP;
    free_ctx(c);
    (void)what;
    return st;
  };
  const size_t sb = dtype_size(o.state_dtype), nb = dtype_size(o.ns_dtype);
  const int64_t ws_elems = std::max(c->lay.plan[0].ws_elems, c->lay.plan[1].ws_elems);
  const size_t n_probs = std::max(c->lay.plan[0].probs.size(), c->lay.plan[1].probs.size());
  if ((e = dev_alloc(c, &c->mom, size_t(c->lay.total_elems) * sb)) != hipSuccess) return bail(e, "momentum");
  if ((e = dev_alloc(c, &c->ws, size_t(ws_elems) * nb)) != hipSuccess) return bail(e, "workspace");
  void* p = nullptr;
  if ((e = dev_alloc(c, &p, c->lay.segs.size() * sizeof(float))) != hipSuccess) return bail(e, "partials");
  c->partials = static_cast<float*>(p);
  if ((e = dev_alloc(c, &p, n_probs * sizeof(float))) != hipSuccess) return bail(e, "scales");
  c->scales = static_cast<float*>(p);
  const int64_t split_floats = std::max(c->lay.plan[0].split_floats, c->lay.plan[1].split_floats);
  const int64_t split_slots = std::max(c->lay.plan[0].split_slots, c->lay.plan[1].split_slots);
  if (split_slots > 0) {
    if ((e = dev_alloc(c, &p, size_t(split_floats) * sizeof(float))) != hipSuccess) return bail(e, "split sums");
    c->ksum = static_cast<float*>(p);
    if ((e = dev_alloc(c, &p, size_t(split_slots) * sizeof(int))) != hipSuccess) return bail(e, "split counters");
    c->kcount = static_cast<int*>(p);
    if ((e = hipMemsetAsync(c->kcount, 0, size_t(split_slots) * sizeof(int), c->stream)) !=
        hipSuccess)
      return bail(e, "split counters");
  }
  if ((e = upload(c, &c->segs, c->lay.segs)) != hipSuccess) return bail(e, "segments");
  if ((e = upload(c, &c->blocks, block_descs(c->lay))) != hipSuccess) return bail(e, "blocks");
  for (int full = 0; full < 2; ++full)
    if ((e = build_plan_tables(c, full)) != hipSuccess) return bail(e, "plan tables");
  if ((e = c->ptrs.init(shapes.size())) != hipSuccess) return bail(e, "pointer tables");
  if (o.check_finite) {
    if ((e = dev_alloc(c, &p, sizeof(int))) != hipSuccess) return bail(e, "finite flag");
    c->finite_flag = static_cast<int*>(p);
    if ((e = hipHostMalloc(&p, sizeof(int), 0)) != hipSuccess) return bail(e, "finite flag");
    c->finite_host = static_cast<int*>(p);
  }
  // Algorithm 1: M_{-1} = 0.
  if ((e = hipMemsetAsync(c->mom, 0, size_t(c->lay.total_elems) * sb, c->stream)) != hipSuccess)
    return bail(e, "memset");
  if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) return bail(e, "sync");
  *out = c;
  return MUONBP_OK;
}

muonbp_status muonbp_step(muonbp_ctx* c, void* const* params, const void* const* grads, int64_t step) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  if (!params || !grads) return fail(c, MUONBP_E_INVALID, "params and grads must not be NULL");
  if (step < 0) return fail(c, MUONBP_E_INVALID, "step must be >= 0");
  const size_t n = c->lay.mats.size();
  const size_t pb = dtype_size(c->opt.param_dtype);
  bool aligned = c->vec_layout;
  for (size_t i = 0; i < n; ++i) {
    if (!params[i] || !grads[i]) return fail(c, MUONBP_E_INVALID, "NULL param or grad pointer");
    if (reinterpret_cast<uintptr_t>(params[i]) % pb || reinterpret_cast<uintptr_t>(grads[i]) % pb)
      return fail(c, MUONBP_E_INVALID, "param or grad pointer not element-aligned");
    aligned = aligned && reinterpret_cast<uintptr_t>(params[i]) % 16 == 0 &&
              reinterpret_cast<uintptr_t>(grads[i]) % 16 == 0;
  }
  if (c->prof != 0 || c->opt.check_finite) {
    // Profiling events and the finite check's wait cannot be part of a graph.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(c->stream, &cap) == hipSuccess && cap != hipStreamCaptureStatusNone)
      return fail(c, MUONBP_E_STATE,
                  "profiling or check_finite is enabled while the stream captures a graph");
  }
  hipError_t e = c->ptrs.stage(params, grads, c->stream);
  if (e == hipErrorStreamCaptureUnsupported)  // nothing enqueued: the context stays usable
    return fail(c, MUONBP_E_STATE,
                "param / grad pointers differ from the previous step's while the stream captures a "
                "graph; run one step with these pointers before capturing");
  if (e != hipSuccess) return hip_fail(c, e, "pointer upload");
  const MatPtrs* mats = c->ptrs.current();

  // Algorithm 1: full orthogonalization iff t mod P = 0 (P = 0 means infinity).
  const int full = (c->period > 0 && step % c->period == 0) ? 1 : 0;
  const muonbp_options& o = c->opt;
  const hipStream_t s = c->stream;
  c->prof_full = full;
  StepBuffers b;
  b.mom = c->mom;
  b.partials = c->partials;
  b.scales = c->scales;
  b.ksum = c->ksum;
  b.kcount = c->kcount;
  b.segs = c->segs;
  b.blocks = c->blocks;
  b.mats = mats;
  b.n_segs = int(c->lay.segs.size());
  StepScalars sc;
  sc.mu = c->mu;
  sc.eta = full ? c->lr_full : c->lr_block;
  sc.wd = c->wd;
  sc.vec = aligned;
  sc.nt = c->stream_nt;
  auto wrap = [&](int kind, auto&& launch) { return timed(c, kind, launch); };
  if ((e = enqueue_momentum(o, b, sc, s, wrap)) != hipSuccess) return hip_fail(c, e, "momentum");
  if (o.check_finite) {
    // Debug check: any non-finite per-segment sum of squares of the NS input.
    if ((e = launch_check_finite(b.n_segs, c->partials, c->finite_flag, s)) != hipSuccess ||
        (e = hipMemcpyAsync(c->finite_host, c->finite_flag, sizeof(int), hipMemcpyDeviceToHost, s)) !=
            hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
      return hip_fail(c, e, "finite check");
    if (*c->finite_host != 0)
      return fail(c, MUONBP_E_NONFINITE,
                  "NaN or Inf in the orthogonalization input (momentum of this step) of some unit; "
                  "params not updated");
  }
  const char* what = "";
  e = enqueue_after_momentum(o, c->lay.plan[full], c->pd[full].view(), b, sc, s, wrap,
                             [&](bool begin, int n_launches) { return span_mark(c, begin, n_launches); },
                             &what);
  if (e != hipSuccess) return hip_fail(c, e, what);
  c->last_plan = full;
  return MUONBP_OK;
}

muonbp_status muonbp_set_lr(muonbp_ctx* c, float lr_block, float lr_full) {
  if (!c) return MUONBP_E_INVALID;
  if (!std::isfinite(lr_block) || !std::isfinite(lr_full))
    return fail(c, MUONBP_E_INVALID, "learning rates must be finite");
  c->lr_block = lr_block;
  c->lr_full = lr_full;
  return MUONBP_OK;
}

muonbp_status muonbp_set_period(muonbp_ctx* c, int64_t period) {
  if (!c) return MUONBP_E_INVALID;
  if (period < 0) return fail(c, MUONBP_E_INVALID, "period must be >= 0 (0 = infinity)");
  c->period = period;
  return MUONBP_OK;
}

muonbp_status muonbp_set_stream(muonbp_ctx* c, void* hip_stream) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  // Order the new stream after everything enqueued so far.
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->ptrs.invalidate();
  return MUONBP_OK;
}

static muonbp_status momentum_copy(muonbp_ctx* c, int32_t mat, void* dst, const void* src) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  if (mat < 0 || size_t(mat) >= c->lay.mats.size()) return fail(c, MUONBP_E_INVALID, "bad matrix index");
  if (!dst && !src) return fail(c, MUONBP_E_INVALID, "NULL pointer");
  const MatrixShape& m = c->lay.mats[mat];
  const size_t sb = dtype_size(c->opt.state_dtype);
  char* mom = static_cast<char*>(c->mom) + c->lay.mat_off[mat] * int64_t(sb);
  const size_t bytes = size_t(m.rows * m.cols) * sb;
  hipError_t e = dst ? hipMemcpyAsync(dst, mom, bytes, hipMemcpyDeviceToDevice, c->stream)
                     : hipMemcpyAsync(mom, src, bytes, hipMemcpyDeviceToDevice, c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "momentum copy");
  return MUONBP_OK;
}

muonbp_status muonbp_get_momentum(muonbp_ctx* c, int32_t mat, void* dst) {
  if (c && !dst) return fail(c, MUONBP_E_INVALID, "dst is NULL");
  return momentum_copy(c, mat, dst, nullptr);
}

muonbp_status muonbp_set_momentum(muonbp_ctx* c, int32_t mat, const void* src) {
  if (c && !src) return fail(c, MUONBP_E_INVALID, "src is NULL");
  return momentum_copy(c, mat, nullptr, src);
}

muonbp_status muonbp_get_update(muonbp_ctx* c, int32_t mat, void* dst) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  if (mat < 0 || size_t(mat) >= c->lay.mats.size()) return fail(c, MUONBP_E_INVALID, "bad matrix index");
  if (!dst) return fail(c, MUONBP_E_INVALID, "dst is NULL");
  if (c->last_plan < 0) return fail(c, MUONBP_E_STATE, "no step has run yet");
  const MatrixShape& m = c->lay.mats[mat];
  const size_t es = dtype_size(c->opt.ns_dtype);
  const PlanDev& pd = c->pd[c->last_plan];
  for (size_t b = 0; b < c->lay.blocks.size(); ++b) {
    const BlockPlan& bp = c->lay.blocks[b];
    if (bp.mat != mat) continue;
    const UpdDesc& u = pd.upd_host[b];
    char* d = static_cast<char*>(dst) + (bp.row0 * m.cols + bp.col0) * int64_t(es);
    hipError_t e = hipMemcpy2DAsync(d, size_t(m.cols) * es, u.u, size_t(u.ldu) * es, size_t(bp.cols) * es,
                                    size_t(bp.rows), hipMemcpyDeviceToDevice, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "update copy");
  }
  return MUONBP_OK;
}

muonbp_status muonbp_synchronize(muonbp_ctx* c) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  return MUONBP_OK;
}

muonbp_status muonbp_profile_enable(muonbp_ctx* c, int32_t enable) {
  if (!c) return MUONBP_E_INVALID;
  if (enable < 0 || enable > 2) return fail(c, MUONBP_E_INVALID, "profile mode must be 0, 1 or 2");
  c->prof = enable;
  return MUONBP_OK;
}

muonbp_status muonbp_profile_read(muonbp_ctx* c, muonbp_profile* out) {
  if (!c || !out) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  *out = muonbp_profile{};
  for (ProfRec& r : c->prof_recs) {
    if (!r.stop) {  // span left open by a failed step
      c->ev_pool.push_back(r.start);
      continue;
    }
    hipError_t e = hipEventSynchronize(r.stop);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventElapsedTime");
    out->ms[r.kind] += ms;
    out->launches[r.kind] += r.launches;
    if (r.full) {
      out->ms_full_steps[r.kind] += ms;
      out->launches_full_steps[r.kind] += r.launches;
    }
    c->ev_pool.push_back(r.start);
    c->ev_pool.push_back(r.stop);
  }
  c->prof_recs.clear();
  return MUONBP_OK;
}

void muonbp_destroy(muonbp_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  free_ctx(c);
}

}  // extern "C"
