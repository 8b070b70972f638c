// Plain descriptors shared by the host planner and the HIP kernels.
// Every table lives in device memory, built once per context; the kernels
// read one entry per workgroup.
#pragma once
#include <stdint.h>

namespace muonbp {

// Row segment of one block, the unit of work of the elementwise kernels
// (momentum, update).  One workgroup per segment, in launch order; `slot` is
// where the segment's sum of squares goes (the segments of one block have
// consecutive slots, whatever their launch order).
struct SegDesc {
  int32_t block;      // index into the block table
  int32_t row_begin;  // first row inside the block
  int32_t nrows;      // rows in this segment
  int32_t slot;       // index of its partial sum
};

// One block of the shard grid (Sec. 3): a rows x cols window of a matrix.
struct BlockDesc {
  int64_t in_mat_off;  // row0 * ld + col0: element offset inside its matrix
  int64_t mom_off;     // element offset of the block origin in the momentum arena
  int64_t ld;          // leading dimension of the matrix (= its cols)
  int32_t mat;         // matrix index
  int32_t cols;        // block width
};

// Caller pointers of one matrix for the current step.
struct MatPtrs {
  void* param;
  const void* grad;
};

// Sum-of-squares range of one orthogonalized unit (problem).
struct ScaleDesc {
  int32_t seg_begin, seg_end;  // partial sums [seg_begin, seg_end)
};

// Where the pack kernel reads one problem (a block or a whole matrix) and
// where it writes the two layouts of the scaled NS input.
struct PackDesc {
  int64_t mom_off;     // momentum arena offset of the problem origin
  int64_t in_mat_off;  // same origin inside the matrix (for grads)
  int64_t ld;          // matrix leading dimension
  void* dst_s;         // straight copy: dst_s[r * ld_s + c] = s * Y[r][c]
  void* dst_t;         // transposed copy: dst_t[c * ld_t + r] = s * Y[r][c]
  int64_t ld_s, ld_t;
  int32_t mat, rows, cols, tiles_c;  // tiles_c: 64-wide column tiles
  int32_t seg_begin, seg_end;        // the problem's sum-of-squares partials
};

// One product of a grouped NS launch, all row-major with K contiguous:
//   C[i][j] = alpha * sum_k X[i][k] Y[j][k] + beta * D[i][j] + gamma [i == j]
// and, when Ct is set, Ct[j][i] = the same value.  With both Ct and D set,
// D must be symmetric (the transposed tile reuses D's tile).
// sym: the product is symmetric; its tile list holds upper tiles only and
// the mirror write (Ct = C) is skipped on diagonal tiles.
// scale: when set, alpha is multiplied by scale[0] (by scale[0]^2 with
// scale_sq) -- Alg. 2's Frobenius normalisation folded into the first Gram
// and apply of a unit that reads its NS input (the momentum) in place.
struct GemmDesc {
  const void* X;
  const void* Y;
  const void* D;
  void* C;
  void* Ct;
  int32_t M, N, K;
  int32_t ldx, ldy, ldd, ldc, ldct;
  float alpha, beta, gamma;
  int32_t sym;
  const float* scale;
  int32_t scale_sq;
};

// Workgroup tile shapes of the NS GEMM (rows x columns of C per workgroup):
// register-staged K loop (any dtype, any K) or LDS-DMA K loop (bf16, K a
// multiple of 8).
// kGemm128x128Split2 runs two K halves of each tile in one 8-wave
// workgroup.  kGemmDma128x128 .. kGemmDma256x256 are kept as numbers only:
// the planner turns them into the interleaved kernels of the same shapes.
enum GemmVariant : int32_t {
  kGemm128x128 = 0, kGemm256x128 = 1, kGemm256x256 = 2,
  kGemmDma128x128 = 3, kGemmDma256x128 = 4, kGemmDma256x256 = 5,
  kGemm128x128Split2 = 6,
  kGemmDmaP128x128 = 7, kGemmDmaP256x128 = 8, kGemmDmaP256x256 = 9,
  kGemmDmaP192x256 = 10, kGemmDmaP256x192 = 11, kGemmDmaP192x192 = 12,
  kGemmDmaP256x256W8 = 13, kGemmDmaP192x256W8 = 14, kGemmDmaP256x192W8 = 15,
  kNumGemmVariants = 16
};
constexpr int kGemmTileRows[kNumGemmVariants] = {128, 256, 256, 128, 256, 256, 128, 128,
                                                 256, 256, 192, 256, 192, 256, 192, 256};
constexpr int kGemmTileCols[kNumGemmVariants] = {128, 128, 256, 128, 128, 256, 128, 128,
                                                 128, 256, 256, 192, 192, 256, 256, 192};
constexpr bool kGemmIsDma[kNumGemmVariants] = {false, false, false, true, true, true, false, true,
                                               true,  true,  true,  true, true, true, true,  true};
// Interleaved DMA kernels (k_ns_gemm_dmap).
constexpr bool gemm_is_dmap(int v) { return v >= kGemmDmaP128x128; }

// One workgroup tile of a grouped launch: problem index and packed
// (tile row << 16 | tile column).
struct TileRef {
  int32_t prob;
  int32_t ij;
  int32_t slot;  // K-split launches: index of the tile's partial sums and counter
  int32_t part;  // K-split launches: which share of the K slices
};

// Update source of one block for one plan: U window and RMS scale.
struct UpdDesc {
  const void* u;  // U element (0, 0) of this block
  int64_t ldu;
  float s;        // 1, or beta * sqrt(max(p, q))
  int32_t pad;
};

// Scalar optimizer (AdamW): one workgroup's contiguous element range of one
// tensor, and where that range's moments sit in the state arenas.
struct ScalarSeg {
  int32_t tensor;  // index into the pointer table
  int32_t count;   // elements
  int64_t begin;   // first element inside the tensor
  int64_t state;   // arena offset of element `begin`
};

// Per-step scalars of the AdamW and Lion kernels (computed on the host in
// double).
struct AdamwArgs {
  float beta1, beta2, eps;
  float decay;         // 1 - lr * weight_decay
  float step;          // AdamW: lr / (1 - beta1^t); Lion: lr
  float inv_sqrt_bc2;  // AdamW: 1 / sqrt(1 - beta2^t)
};

}  // namespace muonbp
