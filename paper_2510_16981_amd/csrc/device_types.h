// Plain descriptors shared by the host planner and the HIP kernels.
// Every table lives in device memory, built once per context; the kernels
// read one entry per workgroup.
#pragma once
#include <stdint.h>

namespace muonbp {

// Row segment of one block, the unit of work of the elementwise kernels
// (momentum, update).  One workgroup per segment.
struct SegDesc {
  int32_t block;      // index into the block table
  int32_t row_begin;  // first row inside the block
  int32_t nrows;      // rows in this segment
  int32_t pad;
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
};

// One product of a grouped NS launch, all row-major with K contiguous:
//   C[i][j] = alpha * sum_k X[i][k] Y[j][k] + beta * D[i][j]
// and, when Ct is set, Ct[j][i] = alpha * sum_k X[i][k] Y[j][k] + beta * Dt[j][i]
// where Dt holds D transposed (the same values, so Ct = C^T).
struct GemmDesc {
  const void* X;
  const void* Y;
  const void* D;
  const void* Dt;
  void* C;
  void* Ct;
  int32_t M, N, K;
  int32_t ldx, ldy, ldd, lddt, ldc, ldct;
};

// Workgroup tile shapes of the NS GEMM (rows x columns of C per workgroup).
enum GemmVariant : int32_t { kGemm128x128 = 0, kGemm256x128 = 1, kGemm256x256 = 2 };
constexpr int kGemmTileRows[3] = {128, 256, 256};
constexpr int kGemmTileCols[3] = {128, 128, 256};

// One workgroup tile of a grouped launch: problem index and packed
// (tile row << 16 | tile column).
struct TileRef {
  int32_t prob;
  int32_t ij;
};

// Update source of one block for one plan: U window and RMS scale.
struct UpdDesc {
  const void* u;  // U element (0, 0) of this block
  int64_t ldu;
  float s;        // 1, or beta * sqrt(max(p, q))
  int32_t pad;
};

}  // namespace muonbp
