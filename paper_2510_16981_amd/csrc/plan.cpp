// Host planner (see plan.h).  Builds, for a list of matrices and shard grids
// (Sec. 3, "How blocks align with model-parallel shards"), the tables used by
// the kernels.  No HIP call is made here.
#include "plan.h"

#include <algorithm>
#include <limits>
#include <utility>

namespace muonbp {

namespace {

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int64_t kMaxDim = int64_t(1) << 30;    // int32 leading dims stay valid
constexpr int64_t kMaxTiles = int64_t(1) << 16;  // tile index packs in 16 bits

// Byte offsets inside one NS operand are 32-bit in the GEMM kernels (buffer
// descriptors and per-lane offsets), so no operand may reach 2^31 bytes.
constexpr int64_t kMaxOperandBytes = int64_t(1) << 31;

// Appends the workspace buffers of one problem; returns false on overflow.
// nn (the apply reads Z row-major, so no Z^T is kept between iterations):
// Z[0], Z[1], A, B, with each Z buffer large enough for either layout (S x
// Lp or L x Sp); U of a transposed unit is written as Z^T into the buffer
// the last apply would otherwise fill (off_zt aliases off_z).  Otherwise
// (the transposed-copy apply, or the register-loop kernels): Z[2], Z^T[2],
// A, B.  A Gram-space unit adds Q[2] and T (S x Sp each).
bool place_problem(Problem* p, int64_t* cursor, int64_t align_elems, bool nn) {
  auto take = [&](int64_t n) {
    int64_t at = *cursor;
    *cursor = round_up(at + n, align_elems);
    return at;
  };
  const int64_t zs = p->S * p->Lp, zts = p->L * p->Sp, as = p->S * p->Sp;
  if (nn) {
    const int64_t both = std::max(zs, zts);
    p->off_z[0] = p->off_zt[0] = take(both);
    p->off_z[1] = p->off_zt[1] = take(both);
  } else {
    p->off_z[0] = take(zs);
    p->off_z[1] = take(zs);
    p->off_zt[0] = take(zts);
    p->off_zt[1] = take(zts);
  }
  p->off_a = take(as);
  p->off_b = take(as);
  if (p->gram) {
    p->off_q[0] = take(as);
    p->off_q[1] = take(as);
    p->off_t = take(as);
  }
  return *cursor > 0 && *cursor < (int64_t(1) << 46);
}

// Largest operand of a problem in bytes (Z in either layout, A, B).
int64_t max_operand_bytes(const Problem& p, int es) {
  return std::max(std::max(p.S * p.Lp, p.L * p.Sp), p.S * p.Sp) * int64_t(es);
}

void add_pack_tiles(Plan* plan, int32_t prob) {
  const Problem& p = plan->probs[prob];
  const int64_t pr = ceil_div(p.rows, kPackTile), pc = ceil_div(p.cols, kPackTile);
  for (int64_t i = 0; i < pr; ++i)
    for (int64_t j = 0; j < pc; ++j)
      plan->pack_tiles.push_back(TileRef{prob, int32_t((i << 16) | j)});
}

// Rows x columns of C for one product of problem p.
void gemm_dims(const Problem& p, GemmKind kind, int64_t* m, int64_t* n, int64_t* k) {
  *m = p.S;
  *n = kind == kApply ? p.L : p.S;
  *k = kind == kGram ? p.L : p.S;
}

int64_t count_tiles(const std::vector<Problem>& probs, GemmKind kind, int v) {
  int64_t n = 0;
  for (const Problem& p : probs) {
    int64_t m, c, k;
    gemm_dims(p, kind, &m, &c, &k);
    const int64_t tm = ceil_div(m, kGemmTileRows[v]), tn = ceil_div(c, kGemmTileCols[v]);
    n += kind == kApply ? tm * tn : tm * (tm + 1) / 2;
  }
  return n;
}

// Logical tile order of one product of one problem: bands of `group` tile
// rows, each band walked column by column (rows inside a column first).  An
// XCD's concurrent tiles then form a group x (tiles / group) block of C that
// shares `group` X panels and as many Y panels as it has columns, instead of
// one X panel and a Y panel per tile.  Tiles taller than 128 rows take
// bands of 4, or of 8 for the polynomial and apply products of a unit with
// at least 16 rows of tiles (measured on the 8B-shaped model: bands of 8
// make the full-step apply, 16 x 56 tiles, 1.7% faster; on the block
// steps' 7-row units they leave the time unchanged and raise the apply's
// traffic by 60%, and the Gram is 2% slower with them; bands of 2 make the
// apply 5% slower).
void append_tiles(const Problem& p, GemmKind kind, int v, int32_t desc,
                  std::vector<TileRef>* out) {
  int64_t m, c, k;
  gemm_dims(p, kind, &m, &c, &k);
  const int64_t tm = ceil_div(m, kGemmTileRows[v]), tn = ceil_div(c, kGemmTileCols[v]);
  const bool small_tiles = kGemmTileRows[v] == 128 && v != kGemm128x128Split2;
  const int64_t group = small_tiles || (kind != kGram && tm >= 16) ? 8 : 4;
  for (int64_t g0 = 0; g0 < tm; g0 += group)
    for (int64_t j = (kind == kApply ? 0 : g0); j < tn; ++j)
      for (int64_t i = g0; i < std::min(tm, g0 + group); ++i)
        if (kind == kApply || i <= j) out->push_back(TileRef{desc, int32_t((i << 16) | j)});
}

}  // namespace

int32_t gram_apply_slot(int ns_steps, int sg) {
  const int n = std::min(kGramSegment, ns_steps - sg * kGramSegment);
  const int nseg = (ns_steps + kGramSegment - 1) / kGramSegment;
  return kSlotGApply0 + (sg & 1) + 2 * ((n - 1) & 1) + 4 * (sg == nseg - 1);
}

int32_t first_apply_slot(const Problem& p, int ns_steps) {
  if (p.gram) return gram_apply_slot(ns_steps, 0);
  return ns_steps == 1 ? kSlotApplyLast : kSlotApply0;
}

namespace {

int32_t slot_of(GemmKind kind, int iter, int ns_steps, int poly_slots) {
  const int q = iter & 1;
  return kind == kGram   ? kSlotGram0 + q
         : kind == kPoly ? kSlotPoly0 + std::min(iter, poly_slots - 1)
         : iter == ns_steps - 1 ? kSlotApplyLast
                                : kSlotApply0 + q;
}

// Launch schedule of the K NS iterations.  Per iteration: the Gram (every
// unit that iterates as printed; a Gram-space unit at the start of each
// segment), the polynomial (every unit; a segment's first into Q[0]), then
// for the Gram-space units the products Q_j = P_j Q_{j-1} and T = A_j P_j
// together, and A_{j+1} = T P_j (none in a segment's last iteration), then
// the apply (every unit that iterates as printed; a Gram-space unit's Z <-
// Q Z at the end of each segment).  The Gram-space products take the
// polynomial's tile shape (all are S x S x S).
void build_phases(Plan* plan, int ns_steps, int poly_slots, int desc_per_problem, int ns_elem_bytes) {
  plan->phases.clear();
  plan->split_floats = plan->split_slots = 0;
  const int32_t np = int32_t(plan->probs.size());
  using Item = std::pair<int32_t, int32_t>;  // (problem, descriptor slot)
  auto add_phase = [&](GemmKind kind, const std::vector<Item>& items) {
    if (items.empty()) return;
    GemmPhase phase;
    phase.variant = plan->variant[kind];
    phase.kind = kind;
    phase.nsplit = plan->nsplit[kind];
    phase.nn = kind == kApply && plan->nn_apply;
    std::vector<TileRef> logical;
    for (const Item& it : items) {
      const Problem& p = plan->probs[size_t(it.first)];
      if (ns_elem_bytes == 4 && !gemm_is_dmap(phase.variant)) {
        int64_t m, n, k;
        gemm_dims(p, kind, &m, &n, &k);
        phase.long_k = phase.long_k || k > kLongK;
      }
      append_tiles(p, kind, phase.variant, it.first * desc_per_problem + it.second, &logical);
    }
    if (phase.nsplit > 1) {
      // The shares of one tile are adjacent, so that the XCD order below
      // keeps them on one XCD (one L2) as a rule.
      std::vector<TileRef> parts;
      parts.reserve(logical.size() * size_t(phase.nsplit));
      for (size_t ti = 0; ti < logical.size(); ++ti)
        for (int32_t q = 0; q < phase.nsplit; ++q)
          parts.push_back(TileRef{logical[ti].prob, logical[ti].ij, int32_t(ti), q});
      plan->split_slots = std::max<int64_t>(plan->split_slots, int64_t(logical.size()));
      plan->split_floats = std::max<int64_t>(
          plan->split_floats, int64_t(logical.size()) * phase.nsplit *
                                  kGemmTileRows[phase.variant] * kGemmTileCols[phase.variant]);
      logical.swap(parts);
    }
    phase.tiles = xcd_order(logical);
    plan->phases.push_back(std::move(phase));
  };
  for (int iter = 0; iter < ns_steps; ++iter) {
    std::vector<Item> gram, poly, qt, upd, apply;
    for (int32_t pi = 0; pi < np; ++pi) {
      const Problem& p = plan->probs[size_t(pi)];
      // An in-place unit's first Gram and first apply read the momentum.
      const bool first_m = p.in_place && iter == 0;
      if (!p.gram) {
        gram.push_back({pi, first_m ? kSlotGramM : slot_of(kGram, iter, ns_steps, poly_slots)});
        poly.push_back({pi, slot_of(kPoly, iter, ns_steps, poly_slots)});
        apply.push_back({pi, first_m ? kSlotApplyM : slot_of(kApply, iter, ns_steps, poly_slots)});
        continue;
      }
      // Segment sg of n iterations, j-th of them.
      const int sg = iter / kGramSegment, j = iter % kGramSegment;
      const int n = std::min(kGramSegment, ns_steps - sg * kGramSegment);
      const int32_t poly_b = slot_of(kPoly, iter, ns_steps, poly_slots);
      if (j == 0) gram.push_back({pi, first_m ? kSlotGramM : kSlotGram0 + (sg & 1)});
      poly.push_back({pi, j == 0 ? poly_b + poly_slots : poly_b});
      if (j > 0) qt.push_back({pi, (j & 1) ? kSlotQ1 : kSlotQ0});
      if (j < n - 1) {
        qt.push_back({pi, j == 0 ? kSlotT0 : kSlotT});
        upd.push_back({pi, j == 0 ? kSlotA0 : kSlotA});
      } else {
        apply.push_back({pi, p.in_place && sg == 0 ? kSlotApplyM : gram_apply_slot(ns_steps, sg)});
      }
    }
    add_phase(kGram, gram);
    add_phase(kPoly, poly);
    add_phase(kPoly, qt);
    add_phase(kPoly, upd);
    add_phase(kApply, apply);
  }
}

}  // namespace

std::vector<TileRef> xcd_order(const std::vector<TileRef>& logical) {
  const int64_t n = int64_t(logical.size());
  const int64_t q = n / kNumXCDs, r = n % kNumXCDs;
  std::vector<TileRef> out(logical.size());
  for (int64_t w = 0; w < n; ++w) {
    const int64_t x = w % kNumXCDs, j = w / kNumXCDs;
    out[w] = logical[x * q + std::min(x, r) + j];
  }
  return out;
}

bool dma_allowed(const std::vector<Problem>& probs, GemmKind kind, int ns_elem_bytes) {
  if (ns_elem_bytes != 2) return false;
  for (const Problem& p : probs) {
    int64_t m, n, k;
    gemm_dims(p, kind, &m, &n, &k);
    if (k % 8 != 0) return false;
  }
  return true;
}

// Time model of one launch of the interleaved DMA kernel, in microseconds,
// fitted to per-launch measurements on MI355X (engine clock about 1.7 GHz
// under sustained MFMA load): rounds of resident workgroups x (fixed cost +
// K slices x time per 32-deep slice).  The fixed cost (launch, ring fill,
// epilogue) is 6.5 us.  A slice costs the tile's MFMA cycles over an
// efficiency that grows with the MFMAs per wave and K step: 4 (128 x 128):
// 0.49, 8: 0.55, 16 (256 x 256): 0.61.  128 x 128 tiles fit two per CU,
// and then take 0.65 us per slice each; larger tiles fit one.
double dmap_launch_us(const std::vector<Problem>& probs, GemmKind kind, int v) {
  int64_t tiles = 0;
  double slices = 0;
  for (const Problem& p : probs) {
    int64_t m, c, k;
    gemm_dims(p, kind, &m, &c, &k);
    const int64_t tm = ceil_div(m, kGemmTileRows[v]), tn = ceil_div(c, kGemmTileCols[v]);
    const int64_t nt = kind == kApply ? tm * tn : tm * (tm + 1) / 2;
    tiles += nt;
    slices += double(nt) * double(ceil_div(k, 32));
  }
  if (tiles == 0) return 0;
  slices /= double(tiles);
  const int nm = (kGemmTileRows[v] / 64) * (kGemmTileCols[v] / 64);
  const double eff = nm <= 4 ? 0.49 : nm <= 8 ? 0.49 + 0.015 * (nm - 4)
                                              : std::min(0.61, 0.55 + 0.0075 * (nm - 8));
  const double slice_us = nm * 2 * 32 / eff / 1700.0;
  constexpr double kFixedUs = 6.5;
  const double one = kFixedUs + slices * slice_us;  // a round with one tile per CU
  if (v != kGemmDmaP128x128) return double(ceil_div(tiles, kNumCUs)) * one;
  const double two = kFixedUs + slices * 0.65;      // a round with two tiles per CU
  const int64_t full = tiles / (2 * kNumCUs), rest = tiles % (2 * kNumCUs);
  return double(full) * two + (rest == 0 ? 0.0 : rest <= kNumCUs ? one : two);
}

int32_t choose_variant(const std::vector<Problem>& probs, GemmKind kind, int tile_policy,
                       int ns_elem_bytes) {
  const bool sym = kind != kApply;
  const bool dma = dma_allowed(probs, kind, ns_elem_bytes);
  if (tile_policy > 0) {
    int v = tile_policy - 1;
    // The block-ordered LDS-DMA loop these variants named was removed (the
    // interleaved loop of the same tile shape was 20-25% faster on every
    // launch): they select the interleaved kernel.
    if (v >= kGemmDma128x128 && v <= kGemmDma256x256) v += kGemmDmaP128x128 - kGemmDma128x128;
    // Symmetric products take square tiles; without the DMA path, the
    // register K loop on the same (or, for 192-wide tiles, the nearest) shape.
    if (sym && kGemmTileRows[v] != kGemmTileCols[v]) {
      static const int32_t square[kNumGemmVariants] = {0, 0, 2, 3, 3, 5, 6, 7, 7, 9, 12, 12, 12, 13,
                                                        12, 12};
      v = square[v];
    }
    if (kGemmIsDma[v] && !dma) {
      static const int32_t twin[kNumGemmVariants] = {0, 1, 2, 0, 1, 2, 6, 0, 1, 2, 2, 2, 0, 2,
                                                      2, 2};
      v = twin[v];
    }
    return v;
  }
  // With the interleaved DMA loop (bf16, K a multiple of 8): the tile shape
  // the time model above puts first (square shapes for the symmetric
  // products).  Register K loop otherwise (rules from per-launch
  // measurements on MI355X):
  // symmetric products on 128 x 128 tiles (split over two K groups below two
  // tiles per CU), the apply product on 256 x 256 tiles from two per CU.
  if (dma) {
    // 256 x 256 tiles run on the 8-wave kernel (two waves per SIMD): 4-19%
    // faster than the 4-wave one on every measured launch, never slower.
    // 192 x 256 and 256 x 192 tiles too, since the two waves of a SIMD swap
    // issue priority every slice: the 2048 x 768 shards' apply 700 against
    // 649 TFLOP/s, the 2048 x 6144 step 2.5% faster (before the swap the
    // launches after them ran slower and the step did not gain).
    static const int32_t sym_cands[] = {kGemmDmaP128x128, kGemmDmaP192x192, kGemmDmaP256x256W8};
    static const int32_t gen_cands[] = {kGemmDmaP128x128, kGemmDmaP256x128, kGemmDmaP192x256,
                                        kGemmDmaP256x192, kGemmDmaP256x256W8};
    int32_t best = kGemmDmaP128x128;
    double best_us = dmap_launch_us(probs, kind, best);
    const int32_t* c = sym ? sym_cands : gen_cands;
    const int nc = sym ? 3 : 5;
    for (int i = 1; i < nc; ++i) {
      const double us = dmap_launch_us(probs, kind, c[i]);
      if (us < best_us) {
        best = c[i];
        best_us = us;
      }
    }
    if (best == kGemmDmaP192x256) best = kGemmDmaP192x256W8;
    if (best == kGemmDmaP256x192) best = kGemmDmaP256x192W8;
    return best;
  }
  const int64_t n128 = count_tiles(probs, kind, kGemm128x128);
  const int32_t small = n128 < 2 * kNumCUs ? kGemm128x128Split2 : kGemm128x128;
  if (sym) return small;
  if (count_tiles(probs, kind, kGemm256x256) >= 2 * kNumCUs) return kGemm256x256;
  return small;
}

// K split of the interleaved DMA kernels: each tile shared by q workgroups,
// each on about 1/q of the K slices, the last to finish adding the partial
// sums.  Only on request (k_split > 0): the partial sums have to cross the
// per-XCD caches, and on MI355X that traffic (a full fp32 tile per share)
// cost more than the extra CUs gained on every launch measured (the 2048 x
// 6144 shards' Gram: 35 us split 3 ways against 27 us unsplit).
// With k_split = 0 the planner splits 3 ways only a launch that leaves
// most CUs idle and has a long K loop everywhere (fewer tiles than 0.6 x
// the CUs, at least 128 K slices per product): there the extra CUs win
// over the partial-sum traffic (the whole 2048 x 6144 matrix's Gram, 136
// tiles at K = 6144: 56 against 60 us a launch).
int32_t choose_split(const std::vector<Problem>& probs, GemmKind kind, int32_t v, int k_split) {
  if (!gemm_is_dmap(v)) return 1;
  if (k_split > 0) return k_split;
  const int64_t tiles = count_tiles(probs, kind, v);
  if (tiles == 0 || 10 * tiles > 6 * kNumCUs) return 1;
  for (const Problem& p : probs) {
    int64_t m, c, k;
    gemm_dims(p, kind, &m, &c, &k);
    if (ceil_div(k, 32) < 128) return 1;
  }
  return 3;
}

double ns_unit_flops(int64_t S, int64_t L, int K, bool gram) {
  const double s = double(S), l = double(L);
  // Gram Z Z^T: S(S+1)/2 distinct entries x 2L; a symmetric S x S x S
  // product (A A, and the Gram-space Q, T and A products): S(S+1)/2 x 2S;
  // B Z (the apply): S x L entries x 2S.
  const double gram_zz = s * (s + 1) * l, sym = s * s * (s + 1), apply = 2 * s * s * l;
  if (!gram || K == 0) return double(K) * (gram_zz + sym + apply);
  // Per segment of n iterations: one Gram, n polynomials, n - 1 Q products,
  // 2 (n - 1) A updates, one apply.
  double f = 0;
  for (int k0 = 0; k0 < K; k0 += kGramSegment) {
    const int n = std::min(kGramSegment, K - k0);
    f += gram_zz + (4.0 * n - 3.0) * sym + apply;
  }
  return f;
}

double ns_unit_dense_flops(int64_t S, int64_t L, int K) {
  const double s = double(S), l = double(L);
  return 2.0 * K * (2.0 * l * s * s + s * s * s);
}

std::string build_layout(const MatrixShape* mats, int32_t n_mats,
                         int ns_elem_bytes, int ns_steps, int poly_slots, int tile_policy,
                         int k_split, int apply_mode, Layout* out, bool* shape_error, int gram_mode,
                         bool in_place_input) {
  *shape_error = false;
  if (!mats || n_mats <= 0) return "mats must be a non-empty array";
  if (ns_steps < 0) return "ns_steps must be >= 0";
  if (poly_slots < 1 || poly_slots > 64) return "poly_slots out of range";
  if (tile_policy < 0 || tile_policy > kNumGemmVariants) return "tile_policy out of range";
  if (k_split < 0 || k_split > kMaxKSplit) return "k_split out of range";
  if (gram_mode < 0 || gram_mode > 2) return "gram_mode out of range";
  Layout L;
  L.mats.assign(mats, mats + n_mats);
  int64_t elems = 0;
  for (int32_t k = 0; k < n_mats; ++k) {
    const MatrixShape& m = mats[k];
    if (m.rows <= 0 || m.cols <= 0 || m.grid_rows <= 0 || m.grid_cols <= 0 ||
        m.rows > kMaxDim || m.cols > kMaxDim || m.rows % m.grid_rows ||
        m.cols % m.grid_cols) {
      *shape_error = true;
      return "matrix " + std::to_string(k) + ": sizes must be positive, at most 2^30, "
             "and the grid must divide rows and cols";
    }
    if (ceil_div(std::max(m.rows, m.cols), 64) >= kMaxTiles) {
      *shape_error = true;
      return "matrix " + std::to_string(k) + " is too large";
    }
    L.mat_off.push_back(elems);
    elems += m.rows * m.cols;
  }
  L.total_elems = elems;
  L.poly_slots = poly_slots;
  L.desc_per_problem = kSlotPoly0 + 2 * poly_slots;

  // Blocks in matrix order, row-major inside each grid; segments per block.
  for (int32_t k = 0; k < n_mats; ++k) {
    const MatrixShape& m = mats[k];
    const int64_t br = m.rows / m.grid_rows, bc = m.cols / m.grid_cols;
    const int64_t rows_per_seg = std::max<int64_t>(1, std::min(br, kSegTarget / bc));
    for (int32_t i = 0; i < m.grid_rows; ++i)
      for (int32_t j = 0; j < m.grid_cols; ++j) {
        BlockPlan b{k, i * br, j * bc, br, bc, int32_t(L.segs.size()), 0};
        for (int64_t r = 0; r < br; r += rows_per_seg) {
          if (L.segs.size() >= size_t(std::numeric_limits<int32_t>::max()))
            return "too many segments";
          L.segs.push_back(SegDesc{int32_t(L.blocks.size()), int32_t(r),
                                   int32_t(std::min(rows_per_seg, br - r)),
                                   int32_t(L.segs.size())});
        }
        b.seg_end = int32_t(L.segs.size());
        L.blocks.push_back(b);
      }
  }
  // Launch order: the r-th segment of every block of one block row of a
  // matrix, then the (r+1)-th, ...  For a column-sharded matrix the
  // workgroups that run together then cover whole rows of the matrix instead
  // of one block's narrow row pieces (a 4096 x 1024 matrix in 8 shards has
  // 256-byte pieces of 2 KB rows); for a single column of blocks it is the
  // block order.
  {
    std::vector<SegDesc> order;
    order.reserve(L.segs.size());
    int32_t bi = 0;
    for (int32_t k = 0; k < n_mats; ++k) {
      const MatrixShape& m = mats[k];
      for (int32_t i = 0; i < m.grid_rows; ++i) {
        const int32_t b0 = bi + i * m.grid_cols;
        const int32_t nseg = L.blocks[b0].seg_end - L.blocks[b0].seg_begin;
        for (int32_t r = 0; r < nseg; ++r)
          for (int32_t j = 0; j < m.grid_cols; ++j) order.push_back(L.segs[L.blocks[b0 + j].seg_begin + r]);
      }
      bi += m.grid_rows * m.grid_cols;
    }
    L.segs.swap(order);
  }

  const int64_t align_elems = kWsAlignBytes / ns_elem_bytes;
  for (int full = 0; full < 2; ++full) {
    Plan& plan = L.plan[full];
    plan.full = full != 0;
    int32_t bi = 0;
    // The units: every block (block plan) or every matrix (full plan).
    for (int32_t k = 0; k < n_mats; ++k) {
      const MatrixShape& m = mats[k];
      const int32_t nb = m.grid_rows * m.grid_cols;
      auto add = [&](int64_t r0, int64_t c0, int64_t rows, int64_t cols, int32_t first_block,
                     int32_t n_blocks) {
        Problem p{};
        p.mat = k;
        p.row0 = r0;
        p.col0 = c0;
        p.rows = rows;
        p.cols = cols;
        p.trans = rows > cols;
        p.S = std::min(rows, cols);
        p.L = std::max(rows, cols);
        p.Sp = round_up(p.S, 8);
        p.Lp = round_up(p.L, 8);
        p.first_block = first_block;
        p.n_blocks = n_blocks;
        p.seg_begin = L.blocks[first_block].seg_begin;
        p.seg_end = L.blocks[first_block + n_blocks - 1].seg_end;
        plan.probs.push_back(p);
      };
      if (full) {
        add(0, 0, m.rows, m.cols, bi, nb);
      } else {
        for (int32_t b = 0; b < nb; ++b) {
          const BlockPlan& bp = L.blocks[bi + b];
          add(bp.row0, bp.col0, bp.rows, bp.cols, bi + b, 1);
        }
      }
      bi += nb;
    }
    for (const Problem& p : plan.probs)
      if (max_operand_bytes(p, ns_elem_bytes) >= kMaxOperandBytes) {
        *shape_error = true;
        return "matrix " + std::to_string(p.mat) + (full ? "" : " (one block)") + ": a " +
               std::to_string(p.S) + " x " + std::to_string(p.L) +
               " orthogonalization operand reaches 2^31 bytes, beyond the 32-bit byte offsets "
               "of the NS kernels";
      }
    for (int kind = 0; kind < 3; ++kind) {
      plan.variant[kind] = choose_variant(plan.probs, GemmKind(kind), tile_policy, ns_elem_bytes);
      plan.nsplit[kind] = choose_split(plan.probs, GemmKind(kind), plan.variant[kind], k_split);
      plan.tiles_per_iter[kind] = count_tiles(plan.probs, GemmKind(kind), plan.variant[kind]);
      if (plan.tiles_per_iter[kind] * plan.nsplit[kind] > int64_t(std::numeric_limits<int32_t>::max() / 2))
        return "too many tiles";
    }
    plan.nn_apply = apply_mode == 0 && gemm_is_dmap(plan.variant[kApply]);
    int64_t cursor = 0;
    for (int32_t pi = 0; pi < int32_t(plan.probs.size()); ++pi) {
      Problem& p = plan.probs[pi];
      p.gram = gram_mode != 1 && ns_elem_bytes == 2 && plan.nn_apply && ns_steps >= 2 &&
               (gram_mode == 2 || (p.S >= kGramMinS && 4 * p.L >= 5 * p.S));
      // The momentum window as a GEMM operand: rows of 16-byte chunks (the
      // arena is 16-byte aligned), within the kernels' 32-bit byte offsets.
      const MatrixShape& mm = mats[p.mat];
      const int64_t mom_off = L.mat_off[p.mat] + p.row0 * mm.cols + p.col0;
      p.in_place = in_place_input && ns_elem_bytes == 2 && ns_steps >= 1 && plan.nn_apply && !p.trans &&
                   mm.cols % 8 == 0 && mom_off % 8 == 0 && p.rows * mm.cols * ns_elem_bytes < kMaxOperandBytes;
      if (!place_problem(&p, &cursor, align_elems, plan.nn_apply)) return "workspace too large";
      if (!p.in_place) add_pack_tiles(&plan, pi);
      plan.ns_flops += ns_unit_flops(p.S, p.L, ns_steps, p.gram);
      plan.ns_dense_flops += ns_unit_dense_flops(p.S, p.L, ns_steps);
    }
    plan.ws_elems = cursor;
    build_phases(&plan, ns_steps, poly_slots, L.desc_per_problem, ns_elem_bytes);
    if (plan.pack_tiles.size() > size_t(std::numeric_limits<int32_t>::max() / 2))
      return "too many tiles";
  }
  *out = std::move(L);
  return "";
}

}  // namespace muonbp
