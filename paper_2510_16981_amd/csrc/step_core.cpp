// Shared host side of one MuonBP step (see step_core.h).  No HIP call.
#include "step_core.h"

#include <algorithm>
#include <cmath>

namespace muonbp {

size_t dtype_size(muonbp_dtype d) { return d == MUONBP_F32 ? 4 : 2; }
DType to_dtype(muonbp_dtype d) { return d == MUONBP_F32 ? DType::F32 : DType::BF16; }
bool dtype_ok(muonbp_dtype d) { return d == MUONBP_F32 || d == MUONBP_BF16; }

int poly_slots(const muonbp_options& o) {
  if (o.coeff_count <= 0) return 1;
  return std::max(1, std::min(o.coeff_count, o.ns_steps));
}

namespace {

// Iteration k's (a, b, c) (Alg. 2; a table's last entry repeats).
void ns_coeffs(const muonbp_options& o, int k, float* a, float* b, float* c) {
  if (o.coeff_count <= 0) {
    *a = o.a, *b = o.b, *c = o.c;
    return;
  }
  const int e = std::min(k, o.coeff_count - 1);
  *a = o.coeff_table[3 * e], *b = o.coeff_table[3 * e + 1], *c = o.coeff_table[3 * e + 2];
}

int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

}  // namespace

std::string validate_opts(const muonbp_options& o) {
  if (o.ns_steps < 0 || o.ns_steps > 1000) return "ns_steps must be in [0, 1000]";
  if (!(o.eps >= 0.f) || !std::isfinite(o.eps)) return "eps must be finite and >= 0";
  if (!std::isfinite(o.a) || !std::isfinite(o.b) || !std::isfinite(o.c))
    return "NS coefficients must be finite";
  if (o.nesterov != 0 && o.nesterov != 1) return "nesterov must be 0 or 1";
  if (o.scale_mode != 0 && o.scale_mode != 1) return "scale_mode must be 0 or 1";
  if (!std::isfinite(o.rms_beta)) return "rms_beta must be finite";
  if (o.tile_policy < 0 || o.tile_policy > kNumGemmVariants) return "tile_policy out of range";
  if (o.k_split < 0 || o.k_split > kMaxKSplit) return "k_split out of range";
  if (o.coeff_count < 0 || o.coeff_count > MUONBP_MAX_COEFFS) return "coeff_count out of range";
  if (o.stream_hint < 0 || o.stream_hint > 2) return "stream_hint out of range";
  if (o.apply_mode < 0 || o.apply_mode > 1) return "apply_mode out of range";
  if (o.check_finite != 0 && o.check_finite != 1) return "check_finite must be 0 or 1";
  if (o.device_memory_limit < 0) return "device_memory_limit must be >= 0";
  if (o.gram_iteration < 0 || o.gram_iteration > 2) return "gram_iteration must be 0, 1 or 2";
  for (int i = 0; i < 3 * o.coeff_count; ++i)
    if (!std::isfinite(o.coeff_table[i])) return "coefficients must be finite";
  return "";
}

int64_t context_bulk_bytes(const Layout& lay, const muonbp_options& o) {
  const int64_t ws = std::max(lay.plan[0].ws_elems, lay.plan[1].ws_elems);
  const int64_t split = std::max(lay.plan[0].split_floats, lay.plan[1].split_floats);
  return lay.total_elems * int64_t(dtype_size(o.state_dtype)) + ws * int64_t(dtype_size(o.ns_dtype)) +
         split * int64_t(sizeof(float));
}

std::string check_mats(const muonbp_matrix* mats, int32_t n_mats, std::vector<MatrixShape>* out) {
  if (!mats) return "mats is NULL";
  if (n_mats <= 0) return "n_mats must be > 0";
  out->clear();
  for (int32_t i = 0; i < n_mats; ++i)
    out->push_back(MatrixShape{mats[i].rows, mats[i].cols, mats[i].grid_rows, mats[i].grid_cols});
  return "";
}

std::string layout_for(const std::vector<MatrixShape>& shapes, const muonbp_options& o, Layout* out,
                       bool* shape_error, bool momentum_aligned) {
  // The NS input is the momentum itself when it is stored as the NS dtype
  // and no Nesterov blend is formed.
  const bool in_place = momentum_aligned && o.state_dtype == MUONBP_BF16 && o.ns_dtype == MUONBP_BF16 &&
                        o.nesterov == 0;
  return build_layout(shapes.data(), int32_t(shapes.size()), int(dtype_size(o.ns_dtype)), o.ns_steps,
                      poly_slots(o), o.tile_policy, o.k_split, o.apply_mode, out, shape_error,
                      o.gram_iteration, in_place);
}

void build_plan_host_tables(const Layout& lay, const muonbp_options& o, int full, void* ws_base,
                            const void* mom_base, const float* scales, PlanHostTables* out) {
  const Plan& plan = lay.plan[full];
  const size_t es = dtype_size(o.ns_dtype);
  char* ws = static_cast<char*>(ws_base);
  auto at = [&](int64_t off) { return static_cast<void*>(ws + off * int64_t(es)); };
  *out = PlanHostTables{};

  std::vector<int64_t> pack_tiles_of(plan.probs.size(), 0);
  for (const TileRef& t : plan.pack_tiles) ++pack_tiles_of[size_t(t.prob)];
  int64_t fused_reads = 0;
  bool any_in_place = false;
  for (size_t i = 0; i < plan.probs.size(); ++i) {
    fused_reads += pack_tiles_of[i] * (plan.probs[i].seg_end - plan.probs[i].seg_begin);
    any_in_place = any_in_place || plan.probs[i].in_place;
  }
  // Units read in place have no pack tiles to compute their scale.
  out->fuse_scale = !any_in_place && fused_reads <= kFuseScaleMaxReads;
  for (size_t pi = 0; pi < plan.probs.size(); ++pi) {
    const Problem& p = plan.probs[pi];
    const size_t desc0 = out->descs.size();
    out->scale.push_back(ScaleDesc{p.seg_begin, p.seg_end});
    const MatrixShape& m = lay.mats[p.mat];
    PackDesc d{};
    d.in_mat_off = p.row0 * m.cols + p.col0;
    d.mom_off = lay.mat_off[p.mat] + d.in_mat_off;
    d.ld = m.cols;
    d.mat = p.mat;
    d.rows = int32_t(p.rows);
    d.cols = int32_t(p.cols);
    d.tiles_c = int32_t((p.cols + kPackTile - 1) / kPackTile);
    d.seg_begin = p.seg_begin;
    d.seg_end = p.seg_end;
    // Z = Y (S = rows) or Y^T (S = cols); Z^T the other way round, needed
    // by the NT apply.  The apply that reads Z row-major needs Z only, and
    // with no iterations the straight copy is U itself (in the matrix's
    // orientation, where the update reads it).
    const bool z_only = plan.nn_apply && o.ns_steps > 0;
    const bool u_only = plan.nn_apply && o.ns_steps == 0;
    if (!p.trans) {
      d.dst_s = at(p.off_z[0]);
      d.ld_s = p.Lp;
      d.dst_t = (z_only || u_only) ? nullptr : at(p.off_zt[0]);
      d.ld_t = p.Sp;
    } else {
      d.dst_s = z_only ? nullptr : at(p.off_zt[0]);
      d.ld_s = p.Sp;
      d.dst_t = u_only ? nullptr : at(p.off_z[0]);
      d.ld_t = p.Lp;
    }
    out->pack.push_back(d);
    const int32_t S = int32_t(p.S), Lr = int32_t(p.L), Sp = int32_t(p.Sp), Lp = int32_t(p.Lp);
    // Slots in DescSlot order.  Gram: A = Z_q Z_q^T (symmetric).
    for (int q = 0; q < 2; ++q)
      out->descs.push_back(GemmDesc{at(p.off_z[q]), at(p.off_z[q]), nullptr, at(p.off_a), at(p.off_a),
                                    S, S, Lr, Lp, Lp, 0, Sp, Sp, 1.f, 0.f, 0.f, 1});
    // Apply: Z_{1-q} = (a I + B) Z_q (= a Z_q + B Z_q).  NT: Y = Z_q^T and
    // Z_{1-q} also stored transposed.  NN: Y = Z_q itself, and only the last
    // apply of a transposed unit writes Z^T (as U, where the update reads it).
    auto apply_desc = [&](int q, bool last) {
      if (!plan.nn_apply)
        return GemmDesc{at(p.off_b), at(p.off_zt[q]), nullptr, at(p.off_z[1 - q]), at(p.off_zt[1 - q]),
                        S, Lr, S, Sp, Sp, 0, Lp, Sp, 1.f, 0.f, 0.f, 0};
      const bool t_only = last && p.trans;
      return GemmDesc{at(p.off_b), at(p.off_z[q]), nullptr, t_only ? nullptr : at(p.off_z[1 - q]),
                      t_only ? at(p.off_zt[1 - q]) : nullptr, S, Lr, S, Sp, Lp, 0, Lp, Sp,
                      1.f, 0.f, 0.f, 0};
    };
    for (int q = 0; q < 2; ++q) out->descs.push_back(apply_desc(q, false));
    out->descs.push_back(apply_desc((o.ns_steps + 1) & 1, true));  // iteration K - 1 reads Z_{(K-1) mod 2}
    // Gram-space products (kSlotT0 .. kSlotGApply0 + 7; placeholders that
    // no tile refers to on a unit that iterates as printed).  All but the
    // applies are S x S x S products of symmetric matrices that commute
    // (polynomials in the Gram matrix a segment starts from), so the result
    // is symmetric and only its upper tiles are computed.
    {
      const int32_t ld = Sp;
      auto sym_desc = [&](int64_t x, int64_t y, int64_t c) {
        return GemmDesc{at(x), at(y), nullptr, at(c), at(c), S, S, S, ld, ld, 0, ld, ld, 1.f, 0.f, 0.f, 1};
      };
      if (!p.gram) {
        const GemmDesc unused = out->descs.front();
        for (int k = kSlotT0; k < kSlotGramM; ++k) out->descs.push_back(unused);
      } else {
        const int64_t q0 = p.off_q[0], q1 = p.off_q[1], t = p.off_t;
        out->descs.push_back(sym_desc(p.off_a, q0, t));       // kSlotT0
        out->descs.push_back(sym_desc(p.off_a, p.off_b, t));  // kSlotT
        out->descs.push_back(sym_desc(t, q0, p.off_a));       // kSlotA0
        out->descs.push_back(sym_desc(t, p.off_b, p.off_a));  // kSlotA
        out->descs.push_back(sym_desc(p.off_b, q1, q0));      // kSlotQ0
        out->descs.push_back(sym_desc(p.off_b, q0, q1));      // kSlotQ1
        // Z[1 - z] = Q[q] Z[z]; the final segment of a transposed unit writes
        // Z^T[1 - z] instead (U in the matrix's orientation, where the update
        // reads it).
        for (int last = 0; last < 2; ++last)
          for (int q = 0; q < 2; ++q)
            for (int z = 0; z < 2; ++z) {
              const bool t_only = last && p.trans;
              out->descs.push_back(GemmDesc{at(p.off_q[q]), at(p.off_z[z]), nullptr,
                                            t_only ? nullptr : at(p.off_z[1 - z]),
                                            t_only ? at(p.off_zt[1 - z]) : nullptr, S, Lr, S, Sp, Lp, 0,
                                            Lp, Sp, 1.f, 0.f, 0.f, 0});  // kSlotGApply0 + z + 2 q + 4 last
            }
      }
    }
    // The first Gram and the first apply of a unit read in place: the slots
    // they replace, with the momentum window as Z_0 and alpha scaled by s^2
    // (Gram) and s (apply).  Placeholders on other units.
    if (!p.in_place) {
      const GemmDesc unused = out->descs.front();
      out->descs.push_back(unused);
      out->descs.push_back(unused);
    } else {
      const void* mw = static_cast<const char*>(mom_base) +
                       (lay.mat_off[p.mat] + p.row0 * m.cols + p.col0) * int64_t(dtype_size(o.state_dtype));
      const int32_t ldm = int32_t(m.cols);
      GemmDesc g = out->descs[desc0 + kSlotGram0];
      g.X = g.Y = mw;
      g.ldx = g.ldy = ldm;
      g.scale = scales + pi;
      g.scale_sq = 1;
      out->descs.push_back(g);  // kSlotGramM
      // The apply the first iteration (segment) would run on Z_0.
      GemmDesc a = out->descs[desc0 + size_t(first_apply_slot(p, o.ns_steps))];
      a.Y = mw;
      a.ldy = ldm;
      a.scale = scales + pi;
      a.scale_sq = 0;
      out->descs.push_back(a);  // kSlotApplyM
    }
    // Polynomial of iteration k: B = c_k A A^T + b_k A + a_k I (A symmetric;
    // the a I term carries Algorithm 2's a X into the apply).
    // Then the same polynomials into Q[0] (a Gram-space segment's first;
    // placeholders on a unit that iterates as printed).
    for (int into_q = 0; into_q < 2; ++into_q)
      for (int k = 0; k < lay.poly_slots; ++k) {
        float a, b, cc;
        ns_coeffs(o, k, &a, &b, &cc);
        const int64_t dst = into_q && p.gram ? p.off_q[0] : p.off_b;
        out->descs.push_back(GemmDesc{at(p.off_a), at(p.off_a), at(p.off_a), at(dst), at(dst), S, S, S, Sp,
                                      Sp, Sp, Sp, Sp, cc, b, a, 1});
      }
  }
  // Update table: U of every block after K iterations (buffer K mod 2).
  const int fin = o.ns_steps & 1;
  for (const Problem& p : plan.probs) {
    float s = 1.f;
    if (o.scale_mode == 1) s = o.rms_beta * std::sqrt(float(std::max(p.rows, p.cols)));
    // A Gram-space unit's last segment writes Z[number of segments mod 2].
    const int u = p.gram ? ((o.ns_steps + kGramSegment - 1) / kGramSegment) & 1 : fin;
    const int64_t base = p.trans ? p.off_zt[u] : p.off_z[u];
    const int64_t ldu = p.trans ? p.Sp : p.Lp;
    for (int32_t b = p.first_block; b < p.first_block + p.n_blocks; ++b) {
      const BlockPlan& bp = lay.blocks[b];
      const int64_t off = base + (bp.row0 - p.row0) * ldu + (bp.col0 - p.col0);
      out->upd.push_back(UpdDesc{at(off), ldu, s, 0});
    }
  }
}

std::vector<BlockDesc> block_descs(const Layout& lay) {
  std::vector<BlockDesc> bd;
  for (const BlockPlan& b : lay.blocks) {
    const MatrixShape& m = lay.mats[b.mat];
    BlockDesc d{};
    d.in_mat_off = b.row0 * m.cols + b.col0;
    d.mom_off = lay.mat_off[b.mat] + d.in_mat_off;
    d.ld = m.cols;
    d.mat = b.mat;
    d.cols = int32_t(b.cols);
    bd.push_back(d);
  }
  return bd;
}

bool layout_vectorizable(const Layout& lay) {
  bool vec = true;
  for (const BlockPlan& b : lay.blocks) {
    const MatrixShape& m = lay.mats[b.mat];
    vec = vec && b.cols % 8 == 0 && b.col0 % 8 == 0 && m.cols % 8 == 0 && lay.mat_off[b.mat] % 8 == 0;
  }
  return vec;
}

bool stream_nontemporal(const Layout& lay, const muonbp_options& o) {
  // Nontemporal streaming once a step's momentum and update data cannot
  // stay in the last-level cache anyway.
  const int64_t streamed =
      lay.total_elems * int64_t(2 * dtype_size(o.param_dtype) + dtype_size(o.state_dtype));
  return o.stream_hint == 2 || (o.stream_hint == 0 && streamed > kStreamNtBytes);
}

ScratchPlan scratch_plan(const Layout& lay, int full, const muonbp_options& o) {
  const Plan& plan = lay.plan[full];
  ScratchPlan sp;
  int64_t cur = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = cur;
    cur = align256(cur + std::max<int64_t>(bytes, 1));
    return at;
  };
  sp.ws = take(plan.ws_elems * int64_t(dtype_size(o.ns_dtype)));
  sp.partials = take(int64_t(lay.segs.size()) * 4);
  sp.scales = take(int64_t(plan.probs.size()) * 4);
  sp.ksum = take(plan.split_floats * 4);
  sp.kcount = take(plan.split_slots * 4);
  sp.segs = take(int64_t(lay.segs.size() * sizeof(SegDesc)));
  sp.blocks = take(int64_t(lay.blocks.size() * sizeof(BlockDesc)));
  sp.scale_d = take(int64_t(plan.probs.size() * sizeof(ScaleDesc)));
  sp.pack_d = take(int64_t(plan.probs.size() * sizeof(PackDesc)));
  sp.pack_tiles = take(int64_t(plan.pack_tiles.size() * sizeof(TileRef)));
  sp.descs = take(int64_t(plan.probs.size()) * lay.desc_per_problem * int64_t(sizeof(GemmDesc)));
  for (const GemmPhase& ph : plan.phases)
    sp.phase_tiles.push_back(take(int64_t(ph.tiles.size() * sizeof(TileRef))));
  sp.upd = take(int64_t(lay.blocks.size() * sizeof(UpdDesc)));
  sp.ptrs = take(int64_t(lay.mats.size() * sizeof(MatPtrs)));
  sp.total = cur;
  return sp;
}

}  // namespace muonbp
