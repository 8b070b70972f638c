// C ABI of the scalar optimizer (AdamW with global-norm clipping) that the
// paper's training setup applies to the parameters MuonBP does not
// orthogonalize (Appendix B), or Lion (the scalar optimizer of its 160M
// comparison, Sec. 4), and of the learning-rate schedules of its runs.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <vector>

#include "../../include/muonbp.h"
#include "kernels.h"
#include "plan.h"
#include "ptr_ring.h"

using namespace muonbp;

struct muonbp_adamw_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  muonbp_adamw_options opt{};
  std::vector<int64_t> sizes;
  std::vector<int64_t> state_off;  // element offset of each tensor in the moment arenas
  int64_t state_elems = 0;
  int32_t n_segs = 0;
  ScalarSeg* segs = nullptr;
  float* m = nullptr;
  float* v = nullptr;
  float* partials = nullptr;
  float* clip = nullptr;  // [0] clipping factor, [1] global norm
  PtrRing ptrs;
  bool stream_nt = false;
  bool norm_valid = false;
  bool poisoned = false;
  std::string err;
  std::vector<void*> allocs;
};

namespace {

size_t elem_size(muonbp_dtype d) { return d == MUONBP_F32 ? 4 : 2; }

muonbp_status fail(muonbp_adamw_ctx* c, muonbp_status st, const std::string& msg) {
  if (c) c->err = msg;
  return st;
}

muonbp_status hip_fail(muonbp_adamw_ctx* c, hipError_t e, const char* what) {
  c->poisoned = true;
  c->err = std::string(what) + ": " + hipGetErrorString(e);
  return MUONBP_E_HIP;
}

void free_ctx(muonbp_adamw_ctx* c) {
  if (!c) return;
  for (void* p : c->allocs) (void)hipFree(p);
  c->ptrs.release();
  delete c;
}

hipError_t dev_alloc(muonbp_adamw_ctx* c, void** p, size_t bytes) {
  *p = nullptr;
  hipError_t e = hipMalloc(p, std::max<size_t>(bytes, 256));
  if (e == hipSuccess) c->allocs.push_back(*p);
  return e;
}

std::string validate(const muonbp_adamw_options& o) {
  const float f[] = {o.beta1, o.beta2, o.eps, o.weight_decay, o.max_grad_norm};
  for (float x : f)
    if (!std::isfinite(x)) return "options must be finite";
  if (o.beta1 < 0.f || o.beta1 >= 1.f || o.beta2 < 0.f || o.beta2 >= 1.f) return "betas in [0, 1)";
  if (o.eps < 0.f) return "eps must be >= 0";
  if (o.max_grad_norm < 0.f) return "max_grad_norm must be >= 0";
  if (o.stream_hint < 0 || o.stream_hint > 2) return "stream_hint out of range";
  if (o.algorithm != 0 && o.algorithm != 1) return "algorithm must be 0 (AdamW) or 1 (Lion)";
  return "";
}

}  // namespace

extern "C" {

void muonbp_adamw_options_default(muonbp_adamw_options* o) {
  if (!o) return;
  std::memset(o, 0, sizeof(*o));
  o->beta1 = 0.9f;
  o->beta2 = 0.95f;
  o->eps = 1e-8f;
  o->weight_decay = 0.1f;
  o->max_grad_norm = 1.0f;
  o->param_dtype = MUONBP_BF16;
  o->stream_hint = 0;
}

muonbp_status muonbp_adamw_create(const int64_t* sizes, int32_t n, const muonbp_adamw_options* opt,
                                  void* hip_stream, muonbp_adamw_ctx** out) {
  if (!out) return MUONBP_E_INVALID;
  *out = nullptr;
  if (!sizes || n <= 0) return MUONBP_E_INVALID;
  muonbp_adamw_options o;
  muonbp_adamw_options_default(&o);
  if (opt) o = *opt;
  if (!validate(o).empty()) return MUONBP_E_INVALID;
  if (o.param_dtype != MUONBP_F32 && o.param_dtype != MUONBP_BF16) return MUONBP_E_DTYPE;
  for (int32_t i = 0; i < n; ++i)
    if (sizes[i] <= 0) return MUONBP_E_SHAPE;

  muonbp_adamw_ctx* c = new (std::nothrow) muonbp_adamw_ctx();
  if (!c) return MUONBP_E_NOMEM;
  std::vector<ScalarSeg> segs;
  try {
    c->opt = o;
    c->stream = static_cast<hipStream_t>(hip_stream);
    c->sizes.assign(sizes, sizes + n);
    // Moments of each tensor start at a multiple of 8 elements (32 bytes), and
    // segments of kSegTarget elements (a multiple of 8) tile each tensor.
    int64_t off = 0;
    for (int32_t i = 0; i < n; ++i) {
      c->state_off.push_back(off);
      for (int64_t b = 0; b < sizes[i]; b += kSegTarget)
        segs.push_back(ScalarSeg{i, int32_t(std::min<int64_t>(kSegTarget, sizes[i] - b)), b, off + b});
      if (sizes[i] > std::numeric_limits<int64_t>::max() / 2 - off) {
        delete c;
        return MUONBP_E_SHAPE;
      }
      off += (sizes[i] + 7) / 8 * 8;
    }
    if (segs.size() > size_t(std::numeric_limits<int32_t>::max())) {
      delete c;
      return MUONBP_E_SHAPE;
    }
    c->state_elems = off;
  } catch (const std::bad_alloc&) {
    delete c;
    return MUONBP_E_NOMEM;
  }
  c->n_segs = int32_t(segs.size());
  // Nontemporal accesses once a step streams more than the last-level cache
  // holds: params, grads, m and v read, params, m and v written (Lion: no v).
  const int64_t streamed =
      c->state_elems * int64_t(2 * elem_size(o.param_dtype) + (o.algorithm == 1 ? 8 : 16));
  c->stream_nt = o.stream_hint == 2 || (o.stream_hint == 0 && streamed > kStreamNtBytes);

  hipError_t e;
  auto bail = [&](hipError_t err) {
    const muonbp_status st = err == hipErrorOutOfMemory ? MUONBP_E_NOMEM : MUONBP_E_HIP;
    free_ctx(c);
    return st;
  };
  if ((e = hipGetDevice(&c->device)) != hipSuccess) return bail(e);
  void* p = nullptr;
  if ((e = dev_alloc(c, &p, size_t(c->state_elems) * 4)) != hipSuccess) return bail(e);
  c->m = static_cast<float*>(p);
  if (o.algorithm == 0) {  // Lion keeps no second moment
    if ((e = dev_alloc(c, &p, size_t(c->state_elems) * 4)) != hipSuccess) return bail(e);
    c->v = static_cast<float*>(p);
  }
  if ((e = dev_alloc(c, &p, segs.size() * sizeof(ScalarSeg))) != hipSuccess) return bail(e);
  c->segs = static_cast<ScalarSeg*>(p);
  if ((e = dev_alloc(c, &p, segs.size() * sizeof(float))) != hipSuccess) return bail(e);
  c->partials = static_cast<float*>(p);
  if ((e = dev_alloc(c, &p, 2 * sizeof(float))) != hipSuccess) return bail(e);
  c->clip = static_cast<float*>(p);
  if ((e = c->ptrs.init(size_t(n))) != hipSuccess) return bail(e);
  // Table upload and m_0 = v_0 = 0 on the context's stream; the call waits
  // for that stream only (not for the device's other streams).
  if ((e = hipMemcpyAsync(c->segs, segs.data(), segs.size() * sizeof(ScalarSeg),
                          hipMemcpyHostToDevice, c->stream)) != hipSuccess)
    return bail(e);
  if ((e = hipMemsetAsync(c->m, 0, size_t(c->state_elems) * 4, c->stream)) != hipSuccess) return bail(e);
  if (c->v && (e = hipMemsetAsync(c->v, 0, size_t(c->state_elems) * 4, c->stream)) != hipSuccess)
    return bail(e);
  if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) return bail(e);
  *out = c;
  return MUONBP_OK;
}

muonbp_status muonbp_adamw_step(muonbp_adamw_ctx* c, void* const* params, const void* const* grads,
                                int64_t step, float lr) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  if (!params || !grads) return fail(c, MUONBP_E_INVALID, "params and grads must not be NULL");
  if (step < 0) return fail(c, MUONBP_E_INVALID, "step must be >= 0");
  if (!std::isfinite(lr)) return fail(c, MUONBP_E_INVALID, "lr must be finite");
  const size_t es = elem_size(c->opt.param_dtype);
  bool aligned = true;
  for (size_t i = 0; i < c->sizes.size(); ++i) {
    if (!params[i] || !grads[i]) return fail(c, MUONBP_E_INVALID, "NULL param or grad pointer");
    const uintptr_t a = reinterpret_cast<uintptr_t>(params[i]), b = reinterpret_cast<uintptr_t>(grads[i]);
    if (a % es || b % es) return fail(c, MUONBP_E_INVALID, "param or grad pointer not element-aligned");
    aligned = aligned && a % 16 == 0 && b % 16 == 0;
  }
  hipError_t e = c->ptrs.stage(params, grads, c->stream);
  if (e == hipErrorStreamCaptureUnsupported)  // nothing enqueued: the context stays usable
    return fail(c, MUONBP_E_STATE,
                "param / grad pointers differ from the previous step's while the stream captures a graph");
  if (e != hipSuccess) return hip_fail(c, e, "pointer upload");
  const DType tp = c->opt.param_dtype == MUONBP_F32 ? DType::F32 : DType::BF16;
  const bool clipping = c->opt.max_grad_norm > 0.f;
  if (clipping) {
    if ((e = launch_adamw_sumsq(tp, aligned, c->stream_nt, c->n_segs, c->segs, c->ptrs.current(),
                                c->partials, c->stream)) != hipSuccess)
      return hip_fail(c, e, "gradient norm");
    if ((e = launch_adamw_clip(c->partials, adamw_norm_blocks(c->n_segs), c->opt.max_grad_norm, c->clip,
                               c->stream)) !=
        hipSuccess)
      return hip_fail(c, e, "clipping factor");
  }
  // Bias corrections of step t = step + 1 (AdamW), in double on the host.
  const bool lion = c->opt.algorithm == 1;
  const double t = double(step) + 1.0;
  const double bc1 = 1.0 - std::pow(double(c->opt.beta1), t);
  const double bc2 = 1.0 - std::pow(double(c->opt.beta2), t);
  AdamwArgs a;
  a.beta1 = c->opt.beta1;
  a.beta2 = c->opt.beta2;
  a.eps = c->opt.eps;
  a.decay = float(1.0 - double(lr) * double(c->opt.weight_decay));
  a.step = lion ? lr : float(double(lr) / bc1);
  a.inv_sqrt_bc2 = float(1.0 / std::sqrt(bc2));
  if ((e = launch_adamw(tp, aligned, c->stream_nt, c->n_segs, c->segs, c->ptrs.current(), c->m, c->v,
                        clipping ? c->clip : nullptr, a, lion, c->stream)) != hipSuccess)
    return hip_fail(c, e, lion ? "Lion update" : "AdamW update");
  c->norm_valid = clipping;
  return MUONBP_OK;
}

muonbp_status muonbp_adamw_grad_norm(muonbp_adamw_ctx* c, float* out) {
  if (!c || !out) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  if (!c->norm_valid) return fail(c, MUONBP_E_STATE, "no step with clipping has run");
  float h[2];
  hipError_t e = hipMemcpyAsync(h, c->clip, sizeof(h), hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "gradient norm copy");
  *out = h[1];
  return MUONBP_OK;
}

static muonbp_status state_copy(muonbp_adamw_ctx* c, int32_t i, void* m_dst, void* v_dst,
                                const void* m_src, const void* v_src) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  if (i < 0 || size_t(i) >= c->sizes.size()) return fail(c, MUONBP_E_INVALID, "tensor index out of range");
  const size_t bytes = size_t(c->sizes[size_t(i)]) * 4;
  float* m = c->m + c->state_off[size_t(i)];
  float* v = c->v ? c->v + c->state_off[size_t(i)] : nullptr;  // no v under Lion
  hipError_t e = hipSuccess;
  if (m_dst) e = hipMemcpyAsync(m_dst, m, bytes, hipMemcpyDeviceToDevice, c->stream);
  if (e == hipSuccess && v_dst)
    e = v ? hipMemcpyAsync(v_dst, v, bytes, hipMemcpyDeviceToDevice, c->stream)
          : hipMemsetAsync(v_dst, 0, bytes, c->stream);
  if (e == hipSuccess && m_src) e = hipMemcpyAsync(m, m_src, bytes, hipMemcpyDeviceToDevice, c->stream);
  if (e == hipSuccess && v_src && v) e = hipMemcpyAsync(v, v_src, bytes, hipMemcpyDeviceToDevice, c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "state copy");
  return MUONBP_OK;
}

muonbp_status muonbp_adamw_get_state(muonbp_adamw_ctx* c, int32_t i, void* m_dst, void* v_dst) {
  return state_copy(c, i, m_dst, v_dst, nullptr, nullptr);
}

muonbp_status muonbp_adamw_set_state(muonbp_adamw_ctx* c, int32_t i, const void* m_src,
                                     const void* v_src) {
  return state_copy(c, i, nullptr, nullptr, m_src, v_src);
}

muonbp_status muonbp_adamw_set_stream(muonbp_adamw_ctx* c, void* hip_stream) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->ptrs.invalidate();
  return MUONBP_OK;
}

muonbp_status muonbp_adamw_synchronize(muonbp_adamw_ctx* c) {
  if (!c) return MUONBP_E_INVALID;
  if (c->poisoned) return fail(c, MUONBP_E_STATE, "context poisoned: " + c->err);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  return MUONBP_OK;
}

const char* muonbp_adamw_last_error(const muonbp_adamw_ctx* c) {
  if (!c) return "NULL context";
  return c->err.c_str();
}

void muonbp_adamw_destroy(muonbp_adamw_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  free_ctx(c);
}

double muonbp_lr_cosine(int64_t t, int64_t total, double lr_max, double lr_min, int64_t warmup) {
  if (t < warmup) return lr_max * double(t + 1) / double(warmup);
  const double span = double(std::max<int64_t>(1, total - warmup));
  const double x = std::min(1.0, double(t - warmup) / span);
  return lr_min + (lr_max - lr_min) * 0.5 * (1.0 + std::cos(M_PI * x));
}

double muonbp_lr_wsd(int64_t t, int64_t total, double lr_max, double lr_min, int64_t warmup,
                     int64_t decay) {
  if (t < warmup) return lr_max * double(t + 1) / double(warmup);
  if (decay <= 0 || t < total - decay) return lr_max;
  if (t >= total) return lr_min;
  return lr_max + (lr_min - lr_max) * (double(t - (total - decay)) / double(decay));
}

}  // extern "C"
