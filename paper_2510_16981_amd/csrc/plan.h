// Host-side planner of the MuonBP step: block table, elementwise segments,
// the two orthogonalization plans (blocks / whole matrices) with their NS
// workspace layout and the tile lists of every grouped launch.  Pure C++ with
// no HIP call, so it runs (and is tested) without a GPU.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "device_types.h"

namespace muonbp {

constexpr int kPackTile = 64;           // square tile of the pack kernel
constexpr int kNumCUs = 256;            // MI355X compute units
constexpr int kNumXCDs = 8;             // dies; workgroups are dealt round-robin
constexpr int64_t kSegTarget = 16384;   // elements per elementwise workgroup
constexpr int64_t kWsAlignBytes = 256;  // alignment of every workspace buffer
constexpr int kMaxKSplit = 8;           // workgroups that may share one tile's K loop
constexpr int64_t kStreamNtBytes = int64_t(256) << 20;  // last-level cache (MALL) size

struct MatrixShape {
  int64_t rows, cols;
  int32_t grid_rows, grid_cols;
};

struct BlockPlan {
  int32_t mat;
  int64_t row0, col0, rows, cols;  // window inside the matrix
  int32_t seg_begin, seg_end;
};

// One orthogonalized unit: a block (block plan) or a whole matrix (full
// plan).  NS runs on the S x L matrix Z = Y (or Y^T when rows > cols).
struct Problem {
  int32_t mat;
  int64_t row0, col0, rows, cols;
  bool trans;
  int64_t S, L;    // S = min(rows, cols), L = max(rows, cols)
  int64_t Sp, Lp;  // leading dimensions (multiples of 8 elements)
  // Element offsets inside the NS workspace arena.
  int64_t off_z[2];   // Z (S x Lp), ping-pong
  int64_t off_zt[2];  // Z^T (L x Sp), ping-pong; the same buffers as off_z
                      // when the plan's apply reads Z row-major (Plan::nn_apply):
                      // then only U of a transposed unit is stored this way
  int64_t off_a;      // A = Z Z^T (S x Sp)
  int64_t off_b;      // B = b A + c A^2 (S x Sp)
  int32_t seg_begin, seg_end;
  int32_t first_block, n_blocks;
  // Gram-space iteration: every polynomial of Alg. 2 is a polynomial in
  // the Gram matrix of the iterate it starts from, so n iterations can run
  // on S x S matrices only -- P_j = a I + b A_j + c A_j^2, A_{j+1} = A_j
  // P_j^2 (as (A_j P_j) P_j), Q_j = P_j Q_{j-1} -- and one apply Z <- Q_{n-1}
  // Z ends them.  The K iterations run in segments of at most
  // kGramSegment such iterations, each starting from a fresh Gram of the
  // current Z (segment s reads Z[s mod 2] and writes Z[(s + 1) mod 2]).
  bool gram = false;
  int64_t off_q[2] = {0, 0};  // Q ping-pong (S x Sp), Gram-space units only
  int64_t off_t = 0;          // A_j P_j (S x Sp), Gram-space units only
  // NS input read in place: an untransposed unit whose input is the bf16
  // momentum itself (no Nesterov blend) skips the pack; its first Gram and
  // first apply read the momentum window (leading dimension = the matrix's
  // columns) and fold the Frobenius scale s into alpha (s^2 and s).
  bool in_place = false;
};

// The three grouped products of one NS iteration.
enum GemmKind { kGram = 0, kPoly = 1, kApply = 2 };

// GEMM descriptors per problem: Gram reading Z[0] / Z[1], apply reading
// Z[0] / Z[1], the apply of the last iteration (which writes U where the
// update reads it), the products of the Gram-space iteration (Problem::gram;
// T is the Z[1] buffer), then one polynomial per distinct iteration
// coefficient set (kSlotPoly0 + k for iteration k, the last one repeated).
// TileRef::prob of a GEMM tile is problem * Layout::desc_per_problem + slot.
enum DescSlot {
  kSlotGram0 = 0,
  kSlotGram1 = 1,
  kSlotApply0 = 2,
  kSlotApply1 = 3,
  kSlotApplyLast = 4,
  kSlotT0 = 5,       // Gram-space: T = A Q[0] (first iteration of a segment, P_0 in Q[0])
  kSlotT = 6,        // T = A B
  kSlotA0 = 7,       // A = T Q[0]
  kSlotA = 8,        // A = T B
  kSlotQ0 = 9,       // Q[0] = B Q[1]
  kSlotQ1 = 10,      // Q[1] = B Q[0]
  // Z[1 - z] = Q[q] Z[z] at slot kSlotGApply0 + z + 2 q + 4 last (last: the
  // final segment, which writes Z^T, i.e. U, for a transposed unit).
  kSlotGApply0 = 11,
  kSlotGramM = 19,   // Problem::in_place: the first Gram, reading the momentum
  kSlotApplyM = 20,  // Problem::in_place: the first apply, reading the momentum
  kSlotPoly0 = 21    // then poly_slots polynomials into B, poly_slots into Q[0]
};

// Gram-space iterations per segment: with longer runs the product chain's
// bf16 rounding outgrows the iteration as printed (emulated, 1792 x 4096
// after 48 momentum steps: 1.16% for one run of 5 against 0.75% as
// printed), with runs of at most 3 it stays below it (0.63%).
constexpr int kGramSegment = 3;

// Gram-space iteration where it saves work (bf16 NS, the row-major apply,
// K >= 2): on units with S >= kGramMinS and L >= 1.25 S.  A segment of n
// iterations costs one Gram (S x S x L), 4n - 3 symmetric S x S x S
// products and one apply (S x L x S) against n of each of the Gram, the
// polynomial and the apply; with segments of 3 the measured kernel rates
// break even at L = 1.26 S.  In segments of at most 3 its bf16 error is at
// or below the printed iteration's from S = 128 to 4096 (emulated, rank-128
// gradients, 48 momentum steps: 0.91 / 0.80 / 0.63% at S = 128 / 512 /
// 1792 against 1.06 / 0.95 / 0.75%).  Below the floor a unit's products
// are mostly tile padding; from S = 128 (the 8B-shaped model's k / v
// shards) the fewer Gram and apply launches still win (block step 0.8%
// faster than with the floor at 256).
constexpr int64_t kGramMinS = 128;

// One grouped GEMM launch of a step.
struct GemmPhase {
  int32_t variant = 0;         // GemmVariant of every tile
  int32_t kind = 0;            // GemmKind
  int32_t nsplit = 1;          // workgroups per tile, each on a share of K
  bool nn = false;             // apply reading Z row-major (no Z^T operand)
  // fp32 register-loop kernel with a product over more than kLongK terms:
  // the variant that restarts its sums every 2048 terms (see k_ns_gemm).
  bool long_k = false;
  std::vector<TileRef> tiles;  // workgroup order
};

constexpr int64_t kLongK = 65536;

struct Plan {
  bool full = false;
  std::vector<Problem> probs;
  int64_t ws_elems = 0;
  std::vector<TileRef> pack_tiles;
  int32_t variant[3] = {0, 0, 0};     // GemmVariant per GemmKind
  int32_t nsplit[3] = {1, 1, 1};      // K split per GemmKind
  // Apply products read Z row-major through LDS transpose reads (the
  // interleaved DMA kernel runs them): no Z^T is kept between iterations;
  // only the last apply of a transposed unit writes Z^T, as U.
  bool nn_apply = false;
  int64_t tiles_per_iter[3] = {0, 0, 0};
  int64_t split_floats = 0;           // fp32 partial sums of the largest split launch
  int64_t split_slots = 0;            // tiles of the largest split launch (one counter each)
  std::vector<GemmPhase> phases;      // in launch order, 3 per NS iteration
  double ns_flops = 0, ns_dense_flops = 0;
};

struct Layout {
  std::vector<MatrixShape> mats;
  std::vector<int64_t> mat_off;  // element offset of each matrix (momentum arena)
  std::vector<BlockPlan> blocks;
  std::vector<SegDesc> segs;
  int64_t total_elems = 0;
  int32_t poly_slots = 1;        // distinct polynomial descriptors per problem
  int32_t desc_per_problem = kSlotPoly0 + 2;  // kSlotPoly0 + 2 poly_slots
  Plan plan[2];  // [0] block plan, [1] full plan
};

// Validates shapes and builds every table.  ns_elem_bytes sizes the
// workspace alignment and allows the bf16-only LDS-DMA kernels; ns_steps
// only feeds the flop counts; tile_policy 0 picks each launch's tile shape
// from its tile counts, 1 + GemmVariant forces one (square shapes only for
// the symmetric products; the register K loop where DMA is not allowed).
// Returns "" on success, else a message (with *shape_error telling shape
// vs. argument).
// gram_mode: 0 = the Gram-space iteration where it saves work (above),
// 1 = never, 2 = on every unit that allows it (bf16, row-major apply,
// K >= 2) whatever its shape.
// in_place_input: the NS input is the momentum itself, stored as the NS
// dtype (bf16 state, bf16 NS, no Nesterov blend); untransposed units whose
// momentum window is 16-byte aligned then read it in place
// (Problem::in_place).
std::string build_layout(const MatrixShape* mats, int32_t n_mats,
                         int ns_elem_bytes, int ns_steps, int poly_slots, int tile_policy,
                         int k_split, int apply_mode,
                         Layout* out, bool* shape_error, int gram_mode = 0,
                         bool in_place_input = false);

// Descriptor slot of segment sg's apply on a Gram-space unit (Z[1 - z] =
// Q[q] Z[z] with z = sg mod 2, q the buffer of the segment's last Q, and
// the final segment writing U), and the slot of a unit's first apply.
int32_t gram_apply_slot(int ns_steps, int sg);
int32_t first_apply_slot(const Problem& p, int ns_steps);

// Tile shape the planner picks for one grouped product.
int32_t choose_variant(const std::vector<Problem>& probs, GemmKind kind, int tile_policy,
                       int ns_elem_bytes);

int32_t choose_split(const std::vector<Problem>& probs, GemmKind kind, int32_t variant,
                     int k_split);

// Workgroup order for a logical tile order: workgroup w runs on XCD w % 8, so
// each XCD receives a contiguous run of logical tiles (shared operands stay
// in that XCD's L2).
std::vector<TileRef> xcd_order(const std::vector<TileRef>& logical);

// Per-step flops of NS on one S x L unit for K iterations.
double ns_unit_flops(int64_t S, int64_t L, int K, bool gram = false);  // symmetric-aware, as computed
double ns_unit_dense_flops(int64_t S, int64_t L, int K);  // Sec. 2.2 model

}  // namespace muonbp
