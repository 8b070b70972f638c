// Launchers of the MuonBP HIP kernels (gfx950).  Each returns the launch
// status; tables are device pointers built by the planner.
#pragma once
#include <hip/hip_runtime_api.h>

#include "device_types.h"

namespace muonbp {

enum class DType { F32 = 0, BF16 = 1 };

// M <- mu M + G over every block segment (eq. NTR); partials[seg] = sum of
// squares of the NS input of that segment (M, or G + mu M with Nesterov).
hipError_t launch_momentum(DType grad_t, DType mom_t, bool vec, bool nt, int n_segs,
                           const SegDesc* segs, const BlockDesc* blocks,
                           const MatPtrs* mats, void* mom, float mu,
                           int nesterov, float* partials, hipStream_t s);

// flag[0] = 1 if any of partials[0 .. n) is NaN or Inf, else 0 (one
// workgroup; the debug check of muonbp_options.check_finite).
hipError_t launch_check_finite(int n, const float* partials, int* flag, hipStream_t s);

// scales[p] = 1 / (sqrt(sum of its partials) + eps)  (Algorithm 2, first line).
hipError_t launch_scale(int n_probs, const ScaleDesc* sd, const float* partials,
                        float* scales, float eps, hipStream_t s);

// Z0 = s_p Y_p written straight and/or transposed into the NS workspace.
// s_p comes from scales, or (fuse_scale) is computed in the kernel from the
// problem's partial sums exactly as launch_scale would.
hipError_t launch_pack(DType mom_t, DType grad_t, DType ns_t, bool vec, int n_tiles,
                       const TileRef* tiles, const PackDesc* pd,
                       const MatPtrs* mats, const void* mom,
                       const float* scales, const float* partials, float eps,
                       bool fuse_scale, float mu, int nesterov, hipStream_t s);

// The pack computes the scales itself (no separate scale launch) when its
// workgroups would read at most this many partial sums in all: every pack
// workgroup reads all the partials of its unit, so the cost grows with
// tiles x partials per unit.  Measured: 0.3 M reads (2048x768 shards) add
// 1.3 us to the pack against 6 us for the scale launch; 2.4 M reads (the
// whole 2048x6144 matrix) add 7 us; 8.4 M add 17 us and 268 M 266 us.
constexpr int64_t kFuseScaleMaxReads = int64_t(1) << 20;

// Grouped C = alpha X Y^T + beta D + gamma I (+ transposed copy) over a
// tile list whose tile shape is `variant` (GemmVariant in device_types.h);
// each tile names its problem descriptor, which carries the coefficients.
// nn (interleaved DMA variants only): Y is K x N row-major instead, so C =
// alpha X Y + ...; C may then be NULL when only the transposed copy is
// wanted.
// nsplit > 1 (interleaved DMA variants only): n_tiles workgroups share
// their tiles' K loops as the tile table says; ksum holds the fp32 partial
// sums (tiles x nsplit x tile area floats) and kcount one zeroed counter per
// tile (left zeroed on return).
// long_k (fp32 register-loop 128 x 128 variants): sums restarted every
// 2048 terms, for products over very long K.
hipError_t launch_ns_gemm(DType ns_t, int variant, bool nn, int n_tiles, const GemmDesc* probs,
                          const TileRef* tiles, int nsplit, float* ksum, int* kcount,
                          hipStream_t s, bool long_k = false);

// X <- X (1 - eta lambda) - eta s_b U_b over every block segment.
hipError_t launch_update(DType param_t, DType ns_t, bool vec, bool nt, int n_segs,
                         const SegDesc* segs, const BlockDesc* blocks,
                         const MatPtrs* mats, const UpdDesc* upd, float eta,
                         float lambda, hipStream_t s);

// Scalar optimizer (AdamW with global-norm clipping) over segments of the
// tensors MuonBP does not orthogonalize.
// Workgroups of the gradient-norm pass (and partial sums it writes).
constexpr int kAdamwNormBlocks = 1024;
int adamw_norm_blocks(int n_segs);
// partials[b] (b < adamw_norm_blocks(n_segs)) = sum of squares of the
// gradients of segments b, b + nb, ...
hipError_t launch_adamw_sumsq(DType param_t, bool vec, bool nt, int n_segs, const ScalarSeg* segs,
                              const MatPtrs* ptrs, float* partials, hipStream_t s);
// clip[0] = min(1, max_norm / (||g|| + 1e-6)) (1 when max_norm <= 0),
// clip[1] = ||g||, from the n partial sums of the norm pass.
hipError_t launch_adamw_clip(const float* partials, int n, float max_norm, float* clip,
                             hipStream_t s);
// The AdamW update of params and of the fp32 moments m and v, or (lion) the
// Lion update of params and m; gradients are scaled by clip[0] when clip is
// not NULL.
hipError_t launch_adamw(DType param_t, bool vec, bool nt, int n_segs, const ScalarSeg* segs,
                        const MatPtrs* ptrs, float* m, float* v, const float* clip,
                        const AdamwArgs& a, bool lion, hipStream_t s);

}  // namespace muonbp
