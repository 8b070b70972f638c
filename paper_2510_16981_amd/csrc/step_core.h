// The parts of one MuonBP step (Algorithm 1, Sec. 3.2) shared by the
// context API (muonbp_api.cpp) and the allocation-free entry point
// (static_step.hip): option checks, the host form of one plan's device
// tables, the scratch layout of the allocation-free step, and the launch
// sequence momentum -> scale -> pack -> K x (Gram, poly, apply) -> update.
#pragma once
#include <hip/hip_runtime_api.h>

#include <string>
#include <vector>

#include "../../include/muonbp.h"
#include "kernels.h"
#include "plan.h"

namespace muonbp {

size_t dtype_size(muonbp_dtype d);
DType to_dtype(muonbp_dtype d);
bool dtype_ok(muonbp_dtype d);

// Polynomial descriptors per problem: one for the constant quintic, else one
// per table entry that some iteration uses.
int poly_slots(const muonbp_options& o);

// "" when the options are valid, else the reason.
std::string validate_opts(const muonbp_options& o);

// Device bytes of a context's momentum, NS workspace (the larger plan's)
// and K-split partial sums.
int64_t context_bulk_bytes(const Layout& lay, const muonbp_options& o);

// Copies the shapes (E_INVALID text on a NULL array or a bad count).
std::string check_mats(const muonbp_matrix* mats, int32_t n_mats, std::vector<MatrixShape>* out);

// build_layout with the NS settings of the options.  momentum_aligned: the
// momentum arena starts on a 16-byte boundary (always for a context's own
// arena), a condition for reading it in place as the NS input.
std::string layout_for(const std::vector<MatrixShape>& shapes, const muonbp_options& o, Layout* out,
                       bool* shape_error, bool momentum_aligned = true);

// Host form of one plan's device tables, the NS workspace starting at `ws`,
// the momentum arena at `mom` and the per-problem scales at `scales` (both
// device addresses; the units read in place point their first products
// there).
struct PlanHostTables {
  std::vector<ScaleDesc> scale;  // one per problem
  std::vector<PackDesc> pack;    // one per problem
  std::vector<GemmDesc> descs;   // Layout::desc_per_problem per problem
  std::vector<UpdDesc> upd;      // one per block
  bool fuse_scale = false;       // the pack computes the scales (no k_scale launch)
};
void build_plan_host_tables(const Layout& lay, const muonbp_options& o, int full, void* ws,
                            const void* mom, const float* scales, PlanHostTables* out);

std::vector<BlockDesc> block_descs(const Layout& lay);

// The 16-byte vector paths of the elementwise kernels apply (every block
// window, leading dimension and matrix offset a multiple of 8 elements).
bool layout_vectorizable(const Layout& lay);

// Nontemporal streaming of the momentum and update accesses.
bool stream_nontemporal(const Layout& lay, const muonbp_options& o);

// Byte offsets of everything the allocation-free step keeps in its static
// scratch array for one plan (each 256-byte aligned), and the total.
struct ScratchPlan {
  int64_t ws = 0, partials = 0, scales = 0, ksum = 0, kcount = 0, segs = 0, blocks = 0;
  int64_t scale_d = 0, pack_d = 0, pack_tiles = 0, descs = 0, upd = 0, ptrs = 0;
  std::vector<int64_t> phase_tiles;  // one tile list per launch phase
  int64_t total = 0;
};
ScratchPlan scratch_plan(const Layout& lay, int full, const muonbp_options& o);

// Device view of one plan's tables.
struct PlanView {
  const ScaleDesc* scale = nullptr;
  const PackDesc* pack = nullptr;
  const TileRef* pack_tiles = nullptr;
  const GemmDesc* descs = nullptr;
  const TileRef* const* phase_tiles = nullptr;  // host array: one device pointer per phase
  const UpdDesc* upd = nullptr;
  bool fuse_scale = false;
};

// Device buffers of one step besides the caller's tensors.
struct StepBuffers {
  void* mom = nullptr;
  float* partials = nullptr;
  float* scales = nullptr;
  float* ksum = nullptr;
  int* kcount = nullptr;
  const SegDesc* segs = nullptr;
  const BlockDesc* blocks = nullptr;
  const MatPtrs* mats = nullptr;
  int n_segs = 0;
};

struct StepScalars {
  float mu = 0, eta = 0, wd = 0;
  bool vec = false, nt = false;
};

// Kinds of launches, as muonbp_profile numbers them.
enum LaunchKind { kKindMomentum = 0, kKindScale = 1, kKindPack = 2, kKindGram = 3, kKindPoly = 4,
                  kKindApply = 5, kKindUpdate = 6 };

// M <- mu M + G with the per-segment sums of squares (eq. NTR).
// wrap(kind, launch) runs one launch and returns its status.
template <typename Wrap>
hipError_t enqueue_momentum(const muonbp_options& o, const StepBuffers& b, const StepScalars& sc,
                            hipStream_t s, Wrap&& wrap) {
  return wrap(kKindMomentum, [&] {
    return launch_momentum(to_dtype(o.param_dtype), to_dtype(o.state_dtype), sc.vec, sc.nt, b.n_segs,
                           b.segs, b.blocks, b.mats, b.mom, sc.mu, o.nesterov, b.partials, s);
  });
}

// The rest of the step after the momentum: scales (unless the pack computes
// them), pack, the grouped NS GEMM launches (span(true / false, launches)
// brackets them), update.  *what names the failing stage.
template <typename Wrap, typename Span>
hipError_t enqueue_after_momentum(const muonbp_options& o, const Plan& plan, const PlanView& pv,
                                  const StepBuffers& b, const StepScalars& sc, hipStream_t s,
                                  Wrap&& wrap, Span&& span, const char** what) {
  const DType tp = to_dtype(o.param_dtype), tm = to_dtype(o.state_dtype), tn = to_dtype(o.ns_dtype);
  hipError_t e;
  if (!pv.fuse_scale) {
    *what = "scale";
    e = wrap(kKindScale, [&] {
      return launch_scale(int(plan.probs.size()), pv.scale, b.partials, b.scales, o.eps, s);
    });
    if (e != hipSuccess) return e;
  }
  *what = "pack";
  e = wrap(kKindPack, [&] {
    return launch_pack(tm, tp, tn, sc.vec, int(plan.pack_tiles.size()), pv.pack_tiles, pv.pack, b.mats,
                       b.mom, b.scales, b.partials, o.eps, pv.fuse_scale, sc.mu, o.nesterov, s);
  });
  if (e != hipSuccess) return e;
  const int nphases = int(plan.phases.size());
  *what = "profiling event";
  if ((e = span(true, nphases)) != hipSuccess) return e;
  *what = "NS GEMM";
  for (int ph = 0; ph < nphases; ++ph) {
    const GemmPhase& P = plan.phases[ph];
    e = wrap(kKindGram + P.kind, [&] {
      return launch_ns_gemm(tn, P.variant, P.nn, int(P.tiles.size()), pv.descs, pv.phase_tiles[ph],
                            P.nsplit, b.ksum, b.kcount, s, P.long_k);
    });
    if (e != hipSuccess) return e;
  }
  *what = "profiling event";
  if ((e = span(false, nphases)) != hipSuccess) return e;
  *what = "update";
  return wrap(kKindUpdate, [&] {
    return launch_update(tp, tn, sc.vec, sc.nt, b.n_segs, b.segs, b.blocks, b.mats, pv.upd, sc.eta,
                         sc.wd, s);
  });
}

}  // namespace muonbp
