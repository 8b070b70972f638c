// Host-only sweep of the planner under AddressSanitizer and UBSan (built by
// tests/test_sanitize_host.py with g++; no GPU, no HIP call): build_layout
// over the benchmark workloads' shapes, every tile policy, K split and apply
// mode, both NS dtypes, ragged and degenerate shapes and the bad-argument
// cases, then the host form of both plans' device tables and the scratch
// layout of the allocation-free step.  Prints one line per case family and
// "ok" at the end; any sanitizer report aborts with a non-zero status.
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "plan.h"
#include "step_core.h"

using namespace muonbp;

namespace {

std::vector<MatrixShape> repeat(const std::vector<MatrixShape>& m, int layers) {
  std::vector<MatrixShape> out;
  for (int l = 0; l < layers; ++l) out.insert(out.end(), m.begin(), m.end());
  return out;
}

muonbp_options defaults() {
  muonbp_options o;
  muonbp_options_default(&o);
  return o;
}

int64_t checksum = 0;

// One plan set: layout, both plans' host tables, both scratch layouts.
bool one(const std::vector<MatrixShape>& mats, const muonbp_options& o, bool expect_ok) {
  Layout lay;
  bool shape_err = false;
  const std::string msg = layout_for(mats, o, &lay, &shape_err);
  if (msg.empty() != expect_ok) {
    std::printf("unexpected result (%s): %s\n", expect_ok ? "want ok" : "want error", msg.c_str());
    return false;
  }
  if (!msg.empty()) return true;
  static char fake_ws[256];
  for (int full = 0; full < 2; ++full) {
    PlanHostTables h;
    build_plan_host_tables(lay, o, full, fake_ws, fake_ws, reinterpret_cast<const float*>(fake_ws), &h);
    const ScratchPlan sp = scratch_plan(lay, full, o);
    checksum += int64_t(h.descs.size()) + int64_t(h.upd.size()) + sp.total;
    for (const GemmPhase& ph : lay.plan[full].phases)
      for (const TileRef& t : ph.tiles) checksum += t.prob ^ t.ij;
  }
  checksum += int64_t(block_descs(lay).size()) + (layout_vectorizable(lay) ? 1 : 0);
  return true;
}

}  // namespace

// muonbp_options_default lives in muonbp_api.cpp, which this host-only
// build leaves out (it makes HIP calls); the same defaults are restated here.
extern "C" void muonbp_options_default(muonbp_options* o) {
  std::memset(o, 0, sizeof(*o));
  o->ns_steps = 5;
  o->a = 2.0f;
  o->b = -1.5f;
  o->c = 0.5f;
  o->eps = 1e-7f;
  o->rms_beta = 1.0f;
  o->param_dtype = MUONBP_BF16;
  o->state_dtype = MUONBP_BF16;
  o->ns_dtype = MUONBP_BF16;
}

int main() {
  const std::vector<std::vector<MatrixShape>> big = {
      {{2048, 6144, 1, 8}},
      repeat({{2048, 2048, 1, 8}, {2048, 2048, 1, 8}, {2048, 2048, 1, 8}, {2048, 2048, 1, 8},
              {2048, 8192, 1, 8}, {2048, 8192, 1, 8}, {8192, 2048, 1, 8}}, 16),
      repeat({{4096, 4096, 1, 8}, {4096, 1024, 1, 8}, {4096, 1024, 1, 8}, {4096, 4096, 8, 1},
              {4096, 14336, 1, 8}, {4096, 14336, 1, 8}, {14336, 4096, 8, 1}}, 32),
      {{4096, 14336, 4, 2}, {14336, 4096, 4, 2}},
  };
  const std::vector<std::vector<MatrixShape>> small = {
      {{256, 512, 1, 2}},
      {{272, 528, 2, 2}, {528, 272, 2, 2}, {129, 1000, 1, 1}, {8, 40, 1, 1}},
      {{300, 520, 2, 4}, {520, 300, 4, 2}, {64, 12, 1, 12}, {1, 40, 1, 1}, {3, 5, 1, 1}},
      {{264, 1040, 1, 2}, {1040, 264, 2, 1}, {296, 296, 1, 1}, {136, 2048, 1, 1}},
      {{1, 1, 1, 1}},
      {{7, 1, 7, 1}, {1, 9, 1, 9}},
  };
  int cases = 0;
  bool ok = true;
  // The benchmark workloads with the planner's choices and a few forced ones.
  for (const auto& m : big)
    for (int tp : {0, 9, 14})
      for (int ks : {0, 1, 3}) {
        muonbp_options o = defaults();
        o.tile_policy = tp;
        o.k_split = ks;
        ok = one(m, o, true) && ok;
        ++cases;
      }
  std::printf("benchmark workloads: %d cases\n", cases);
  // Every tile policy, K split, apply mode, dtype and iteration count on
  // small and ragged shapes.
  int n = 0;
  for (const auto& m : small)
    for (int tp = 0; tp <= kNumGemmVariants; ++tp)
      for (int ks = 0; ks <= kMaxKSplit; ks += 2)
        for (int am = 0; am < 2; ++am)
          for (int dt = 0; dt < 2; ++dt)
            for (int K : {0, 1, 5}) {
              muonbp_options o = defaults();
              o.tile_policy = tp;
              o.k_split = ks;
              o.apply_mode = am;
              o.ns_dtype = dt ? MUONBP_BF16 : MUONBP_F32;
              o.ns_steps = K;
              o.coeff_count = (tp % 3 == 0) ? 3 : 0;
              ok = one(m, o, true) && ok;
              ++n;
            }
  std::printf("small and ragged shapes: %d cases\n", n);
  // Refusals: bad grids and sizes, operands of 2^31 bytes, bad arguments.
  const std::vector<std::vector<MatrixShape>> bad = {
      {{10, 8, 3, 1}}, {{0, 8, 1, 1}}, {{8, 8, 0, 1}}, {{8, -8, 1, 1}}, {{8, 8, 1, 9}},
      {{4096, 600000, 1, 1}}, {{40000, 40000, 8, 8}}, {{int64_t(1) << 31, 8, 1, 1}},
  };
  for (const auto& m : bad) ok = one(m, defaults(), false) && ok;
  {
    Layout lay;
    bool se = false;
    ok = !build_layout(nullptr, 1, 2, 5, 1, 0, 0, 0, &lay, &se).empty() && ok;
    MatrixShape m{8, 8, 1, 1};
    ok = !build_layout(&m, 0, 2, 5, 1, 0, 0, 0, &lay, &se).empty() && ok;
    ok = !build_layout(&m, 1, 2, -1, 1, 0, 0, 0, &lay, &se).empty() && ok;
    ok = !build_layout(&m, 1, 2, 5, 0, 0, 0, 0, &lay, &se).empty() && ok;
    ok = !build_layout(&m, 1, 2, 5, 1, kNumGemmVariants + 1, 0, 0, &lay, &se).empty() && ok;
    ok = !build_layout(&m, 1, 2, 5, 1, 0, kMaxKSplit + 1, 0, &lay, &se).empty() && ok;
  }
  std::printf("refusals checked\n");
  std::printf("checksum %lld\n", static_cast<long long>(checksum));
  if (!ok) return 1;
  std::printf("ok\n");
  return 0;
}
