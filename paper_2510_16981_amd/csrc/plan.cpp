// Host planner (see plan.h).  Builds, for a list of matrices and shard grids
// (Sec. 3, "How blocks align with model-parallel shards"), the tables used by
// the kernels.  No HIP call is made here.
#include "plan.h"

#include <algorithm>
#include <limits>

namespace muonbp {

namespace {

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int64_t kMaxDim = int64_t(1) << 30;    // int32 leading dims stay valid
constexpr int64_t kMaxTiles = int64_t(1) << 16;  // tile index packs in 16 bits

// Appends the workspace buffers of one problem; returns false on overflow.
bool place_problem(Problem* p, int64_t* cursor, int64_t align_elems) {
  auto take = [&](int64_t n) {
    int64_t at = *cursor;
    *cursor = round_up(at + n, align_elems);
    return at;
  };
  const int64_t zs = p->S * p->Lp, zts = p->L * p->Sp, as = p->S * p->Sp;
  p->off_z[0] = take(zs);
  p->off_z[1] = take(zs);
  p->off_zt[0] = take(zts);
  p->off_zt[1] = take(zts);
  p->off_a = take(as);
  p->off_b = take(as);
  return *cursor > 0 && *cursor < (int64_t(1) << 46);
}

void add_tiles(Plan* plan, int32_t prob) {
  const Problem& p = plan->probs[prob];
  const int64_t ts = ceil_div(p.S, kGemmTile), tl = ceil_div(p.L, kGemmTile);
  for (int64_t i = 0; i < ts; ++i)
    for (int64_t j = i; j < ts; ++j) {
      TileRef t{prob, int32_t((i << 16) | j)};
      plan->gram_tiles.push_back(t);
      plan->poly_tiles.push_back(t);
    }
  for (int64_t i = 0; i < ts; ++i)
    for (int64_t j = 0; j < tl; ++j)
      plan->apply_tiles.push_back(TileRef{prob, int32_t((i << 16) | j)});
  const int64_t pr = ceil_div(p.rows, kPackTile), pc = ceil_div(p.cols, kPackTile);
  for (int64_t i = 0; i < pr; ++i)
    for (int64_t j = 0; j < pc; ++j)
      plan->pack_tiles.push_back(TileRef{prob, int32_t((i << 16) | j)});
}

}  // namespace

double ns_unit_flops(int64_t S, int64_t L, int K) {
  const double s = double(S), l = double(L);
  // Gram Z Z^T: S(S+1)/2 distinct entries x 2L; A A: S(S+1)/2 x 2S;
  // B Z: S x L entries x 2S.
  return double(K) * (s * (s + 1) * l + s * s * (s + 1) + 2 * s * s * l);
}

double ns_unit_dense_flops(int64_t S, int64_t L, int K) {
  const double s = double(S), l = double(L);
  return 2.0 * K * (2.0 * l * s * s + s * s * s);
}

std::string build_layout(const MatrixShape* mats, int32_t n_mats,
                         int ns_elem_bytes, int ns_steps, Layout* out,
                         bool* shape_error) {
  *shape_error = false;
  if (!mats || n_mats <= 0) return "mats must be a non-empty array";
  if (ns_steps < 0) return "ns_steps must be >= 0";
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
    if (ceil_div(std::max(m.rows, m.cols), kGemmTile) >= kMaxTiles) {
      *shape_error = true;
      return "matrix " + std::to_string(k) + " is too large";
    }
    L.mat_off.push_back(elems);
    elems += m.rows * m.cols;
  }
  L.total_elems = elems;

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
                                   int32_t(std::min(rows_per_seg, br - r)), 0});
        }
        b.seg_end = int32_t(L.segs.size());
        L.blocks.push_back(b);
      }
  }

  const int64_t align_elems = kWsAlignBytes / ns_elem_bytes;
  for (int full = 0; full < 2; ++full) {
    Plan& plan = L.plan[full];
    plan.full = full != 0;
    int64_t cursor = 0;
    int32_t bi = 0;
    for (int32_t k = 0; k < n_mats; ++k) {
      const MatrixShape& m = mats[k];
      const int32_t nb = m.grid_rows * m.grid_cols;
      auto add = [&](int64_t r0, int64_t c0, int64_t rows, int64_t cols,
                     int32_t first_block, int32_t n_blocks) -> bool {
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
        if (!place_problem(&p, &cursor, align_elems)) return false;
        plan.probs.push_back(p);
        add_tiles(&plan, int32_t(plan.probs.size() - 1));
        plan.ns_flops += ns_unit_flops(p.S, p.L, ns_steps);
        plan.ns_dense_flops += ns_unit_dense_flops(p.S, p.L, ns_steps);
        return true;
      };
      if (full) {
        if (!add(0, 0, m.rows, m.cols, bi, nb)) return "workspace too large";
      } else {
        for (int32_t b = 0; b < nb; ++b) {
          const BlockPlan& bp = L.blocks[bi + b];
          if (!add(bp.row0, bp.col0, bp.rows, bp.cols, bi + b, 1))
            return "workspace too large";
        }
      }
      bi += nb;
    }
    plan.ws_elems = cursor;
    if (plan.gram_tiles.size() > size_t(std::numeric_limits<int32_t>::max() / 2) ||
        plan.apply_tiles.size() > size_t(std::numeric_limits<int32_t>::max() / 2) ||
        plan.pack_tiles.size() > size_t(std::numeric_limits<int32_t>::max() / 2))
      return "too many tiles";
  }
  *out = std::move(L);
  return "";
}

}  // namespace muonbp
