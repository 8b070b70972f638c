// HIP kernels of the MuonBP optimizer step for CDNA4 (gfx950, wave64).
//
//  * k_momentum  -- M <- mu M + G (eq. NTR / Algorithm 1), fused with the
//                   per-segment sum of squares of the NS input.
//  * k_scale     -- 1 / (||Y||_F + eps) per orthogonalized unit (Algorithm 2).
//  * k_pack      -- scaled NS input, written row-major and/or transposed.
//  * k_ns_gemm   -- grouped MFMA GEMM C = alpha X Y^T + beta D used for the
//                   three products of every NS iteration (Algorithm 2):
//                   A = Z Z^T, B = b A + c A A, Z' = a Z + B Z.
//  * k_update    -- X <- X (1 - eta lambda) - eta s U (Algorithm 1).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace muonbp {

typedef __bf16 bf16;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Global-address-space views of device pointers: accesses through them
// compile to global_load / global_store.  A generic (flat) access counts
// against the LDS wait counter as well as the memory one, so every LDS wait
// issued after it (the GEMM epilogue's staged reads, the pack's transpose,
// the K loop's fragment reads) would also wait for that memory access to
// complete.  The integer round trip makes the compiler take the address
// space.
typedef __attribute__((address_space(1))) u32x4_t g_u32x4_t;
__device__ __forceinline__ g_u32x4_t* gvec(const void* p) {
  return (g_u32x4_t*)(reinterpret_cast<uintptr_t>(p));
}
template <typename T>
__device__ __forceinline__ void gstore1(T* p, T v) {
  *(__attribute__((address_space(1))) T*)(reinterpret_cast<uintptr_t>(p)) = v;
}

constexpr int kThreads = 256;

// ---------------------------------------------------------------- helpers

template <typename T> __device__ __forceinline__ float to_f(T x);
template <> __device__ __forceinline__ float to_f<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 x) { return float(x); }

template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float x) { return bf16(x); }

// Value after a round trip through storage type T.
template <typename T> __device__ __forceinline__ float rt(float x) {
  return to_f<T>(from_f<T>(x));
}

// Eight consecutive elements <-> floats (pointer 16-byte aligned).
__device__ __forceinline__ void load8(const bf16* p, float f[8]) {
  const u32x4_t v = *gvec(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float f[8]) {
  const u32x4_t a = gvec(p)[0], b = gvec(p)[1];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = __uint_as_float(a[i]);
    f[4 + i] = __uint_as_float(b[i]);
  }
}
__device__ __forceinline__ void store8(bf16* p, const float f[8]) {
  union {
    bf16 h[8];
    u32x4_t v;
  } u;
#pragma unroll
  for (int i = 0; i < 8; ++i) u.h[i] = bf16(f[i]);
  *gvec(p) = u.v;
}
__device__ __forceinline__ void store8(float* p, const float f[8]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    u32x4_t v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __float_as_uint(f[4 * i + k]);
    gvec(p)[i] = v;
  }
}

// Eight consecutive elements as raw 16-byte words.  NT: loaded and stored
// with the nontemporal hint, for steps whose streamed data (read once or
// written once per step) is far larger than the last-level cache; smaller
// steps keep plain accesses, whose data stays cache-resident between the
// kernels of a step.
template <typename T> struct Raw8 {
  u32x4_t w[sizeof(T) / 2];
};
template <bool NT, typename T> __device__ __forceinline__ Raw8<T> load8r(const T* p) {
  Raw8<T> r;
  g_u32x4_t* q = gvec(p);
#pragma unroll
  for (int i = 0; i < int(sizeof(T) / 2); ++i) r.w[i] = NT ? __builtin_nontemporal_load(q + i) : q[i];
  return r;
}
__device__ __forceinline__ void unpack8(const Raw8<bf16>& r, float f[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(r.w[0][i] << 16);
    f[2 * i + 1] = __uint_as_float(r.w[0][i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack8(const Raw8<float>& r, float f[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = __uint_as_float(r.w[i >> 2][i & 3]);
}
template <bool NT> __device__ __forceinline__ void store_w(u32x4_t* p, u32x4_t v) {
  if (NT)
    __builtin_nontemporal_store(v, gvec(p));
  else
    *gvec(p) = v;
}
template <bool NT> __device__ __forceinline__ void store8r(bf16* p, const float f[8]) {
  union {
    bf16 h[8];
    u32x4_t v;
  } u;
#pragma unroll
  for (int i = 0; i < 8; ++i) u.h[i] = bf16(f[i]);
  store_w<NT>(reinterpret_cast<u32x4_t*>(p), u.v);
}
template <bool NT> __device__ __forceinline__ void store8r(float* p, const float f[8]) {
  u32x4_t* q = reinterpret_cast<u32x4_t*>(p);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    u32x4_t v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __float_as_uint(f[4 * i + k]);
    store_w<NT>(q + i, v);
  }
}

// Chunks of 8 elements each thread of an elementwise kernel loads before it
// does any arithmetic (memory-level parallelism of the streaming loops).
constexpr int kStreamUnroll = 8;

// Deterministic workgroup sum (fixed butterfly inside each wave, fixed
// wave order across the workgroup).
__device__ __forceinline__ float block_sum(float v) {
  __shared__ float red[kThreads / 64];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = 0.f;
  if (threadIdx.x == 0)
    for (int w = 0; w < kThreads / 64; ++w) s += red[w];
  return s;  // valid in thread 0
}

// ---------------------------------------------------------------- momentum

template <typename TG, typename TM, bool VEC, bool NT>
__global__ __launch_bounds__(kThreads) void k_momentum(
    const SegDesc* __restrict__ segs, const BlockDesc* __restrict__ blocks,
    const MatPtrs* __restrict__ mats, TM* __restrict__ mom, float mu,
    int nesterov, float* __restrict__ partials) {
  const SegDesc sd = segs[blockIdx.x];
  const BlockDesc bd = blocks[sd.block];
  const int64_t row_off = int64_t(sd.row_begin) * bd.ld;
  const TG* g = static_cast<const TG*>(mats[bd.mat].grad) + bd.in_mat_off + row_off;
  TM* m = mom + bd.mom_off + row_off;
  const int cols = bd.cols;
  float acc = 0.f;
  if (VEC) {
    const int vpr = cols >> 3;
    const int nv = sd.nrows * vpr;
    for (int v0 = threadIdx.x; v0 < nv; v0 += kThreads * kStreamUnroll) {
      Raw8<TG> gr[kStreamUnroll];
      Raw8<TM> mr[kStreamUnroll];
      int64_t o[kStreamUnroll];
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u) {
        const int v = v0 + kThreads * u;
        if (v < nv) {
          const int r = v / vpr;
          o[u] = int64_t(r) * bd.ld + ((v - r * vpr) << 3);
          gr[u] = load8r<NT>(g + o[u]);
          mr[u] = load8r<NT>(m + o[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u) {
        if (v0 + kThreads * u < nv) {
          float gf[8], mf[8];
          unpack8(gr[u], gf);
          unpack8(mr[u], mf);
#pragma unroll
          for (int i = 0; i < 8; ++i) mf[i] = fmaf(mu, mf[i], gf[i]);
          store8r<NT>(m + o[u], mf);
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const float mq = rt<TM>(mf[i]);
            const float y = nesterov ? fmaf(mu, mq, gf[i]) : mq;
            acc = fmaf(y, y, acc);
          }
        }
      }
    }
  } else {
    const int n = sd.nrows * cols;
    for (int e = threadIdx.x; e < n; e += kThreads) {
      const int r = e / cols;
      const int64_t o = int64_t(r) * bd.ld + (e - r * cols);
      const float gv = to_f<TG>(g[o]);
      const float mv = rt<TM>(fmaf(mu, to_f<TM>(m[o]), gv));
      m[o] = from_f<TM>(mv);
      const float y = nesterov ? fmaf(mu, mv, gv) : mv;
      acc = fmaf(y, y, acc);
    }
  }
  acc = block_sum(acc);
  if (threadIdx.x == 0) partials[sd.slot] = acc;
}

// ---------------------------------------------------------------- finite check

// flag[0] = 1 when some partial sum is NaN or Inf (a NaN or Inf anywhere in a
// segment's NS input makes its sum of squares non-finite).  One workgroup,
// so the flag is written once, by thread 0, with no atomics.
__global__ __launch_bounds__(kThreads) void k_check_finite(const float* __restrict__ partials, int n,
                                                           int* __restrict__ flag) {
  __shared__ int any[kThreads / 64];
  int bad = 0;
  for (int i = threadIdx.x; i < n; i += kThreads) bad |= !isfinite(partials[i]);
  bad = __any(bad) ? 1 : 0;
  if ((threadIdx.x & 63) == 0) any[threadIdx.x >> 6] = bad;
  __syncthreads();
  if (threadIdx.x == 0) {
    int f = 0;
    for (int w = 0; w < kThreads / 64; ++w) f |= any[w];
    flag[0] = f;
  }
}

// ---------------------------------------------------------------- scale

__global__ __launch_bounds__(64) void k_scale(const ScaleDesc* __restrict__ sd,
                                              const float* __restrict__ partials,
                                              float* __restrict__ scales, float eps) {
  const ScaleDesc d = sd[blockIdx.x];
  double acc = 0.0;
  for (int i = d.seg_begin + int(threadIdx.x); i < d.seg_end; i += 64) acc += partials[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (threadIdx.x == 0) scales[blockIdx.x] = float(1.0 / (sqrt(acc) + double(eps)));
}

// ---------------------------------------------------------------- pack

// Z = s Y (straight) and Z^T = s Y^T (transposed) for one 64 x 64 tile of a
// problem, Y = M (or G + mu M with Nesterov).  The transposed copy goes
// through LDS.  VEC: columns, windows and leading dimensions are multiples
// of 8 elements and the pointers 16-byte aligned, so every access is one
// 16-byte chunk of 8 elements (the last chunk of a Z^T row may be cut by the
// problem's row count).
// fuse_scale: s is computed here from the problem's partial sums, exactly
// as k_scale computes it (same lanes, same order), instead of read from
// scales (small problems: the separate launch costs more than the sum).
template <typename TM, typename TG, typename TN, bool VEC>
__global__ __launch_bounds__(kThreads) void k_pack(
    const TileRef* __restrict__ tiles, const PackDesc* __restrict__ pd,
    const MatPtrs* __restrict__ mats, const TM* __restrict__ mom,
    const float* __restrict__ scales, const float* __restrict__ partials, float eps,
    int fuse_scale, float mu, int nesterov) {
  __shared__ float tile[64][65];
  __shared__ float s_fused;
  const TileRef t = tiles[blockIdx.x];
  const PackDesc d = pd[t.prob];
  const int r0 = (t.ij >> 16) * 64, c0 = (t.ij & 0xffff) * 64;
  if (fuse_scale) {  // uniform
    if (threadIdx.x < 64) {
      double acc = 0.0;
      for (int i = d.seg_begin + int(threadIdx.x); i < d.seg_end; i += 64) acc += partials[i];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
      if (threadIdx.x == 0) s_fused = float(1.0 / (sqrt(acc) + double(eps)));
    }
    __syncthreads();
  }
  const float s = fuse_scale ? s_fused : scales[t.prob];
  const TM* m = mom + d.mom_off;
  const TG* g = static_cast<const TG*>(mats[d.mat].grad) + d.in_mat_off;
  TN* ds = static_cast<TN*>(d.dst_s);
  TN* dt = static_cast<TN*>(d.dst_t);
  if (VEC) {
    // Straight copy: 64 rows x 8 chunks, two chunks per thread.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = threadIdx.x + kThreads * i, rr = q >> 3, ch = q & 7;
      const int r = r0 + rr, c = c0 + 8 * ch;
      float y[8];
      if (r < d.rows && c < d.cols) {
        const int64_t o = int64_t(r) * d.ld + c;
        load8(m + o, y);
        if (nesterov) {
          float gv[8];
          load8(g + o, gv);
#pragma unroll
          for (int e = 0; e < 8; ++e) y[e] = fmaf(mu, y[e], gv[e]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] *= s;
        if (ds) store8(ds + int64_t(r) * d.ld_s + c, y);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) tile[rr][8 * ch + e] = y[e];
    }
    if (!dt) return;  // uniform: no transposed copy wanted
    __syncthreads();
    // Transposed copy: Z^T rows c0 .. c0 + 63, chunks of 8 rows of Y.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = threadIdx.x + kThreads * i, cc = q >> 3, j = q & 7;
      const int c = c0 + cc, r = r0 + 8 * j;
      if (c < d.cols && r < d.rows) {
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = tile[8 * j + e][cc];
        TN* p = dt + int64_t(c) * d.ld_t + r;
        if (r + 8 <= d.rows) {
          store8(p, y);
        } else {
          for (int e = 0; e < d.rows - r; ++e) gstore1(p + e, from_f<TN>(y[e]));
        }
      }
    }
    return;
  }
  const int lc = threadIdx.x & 63, lr = threadIdx.x >> 6;
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = r0 + lr + 4 * i, c = c0 + lc;
    float y = 0.f;
    if (r < d.rows && c < d.cols) {
      const int64_t o = int64_t(r) * d.ld + c;
      y = to_f<TM>(m[o]);
      if (nesterov) y = fmaf(mu, y, to_f<TG>(g[o]));
      y *= s;
      if (ds) gstore1(ds + int64_t(r) * d.ld_s + c, from_f<TN>(y));
    }
    tile[lr + 4 * i][lc] = y;
  }
  if (!dt) return;  // uniform: no transposed copy wanted
  __syncthreads();
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int c = c0 + lr + 4 * i, r = r0 + lc;
    if (r < d.rows && c < d.cols) gstore1(dt + int64_t(c) * d.ld_t + r, from_f<TN>(tile[lc][lr + 4 * i]));
  }
}

// ---------------------------------------------------------------- NS GEMM
//
// Grouped C = alpha X Y^T + beta D + gamma I over a tile list (alpha, beta,
// gamma and the symmetry flag per problem), both operands row-major
// with K contiguous.  Workgroup tile BM x BN, 256 threads = 4 waves in a
// 2 x 2 layout, (BM/2) x (BN/2) per wave as TM x TN MFMA 32x32 tiles.  The K
// loop stages 128-byte K slices of X and Y rows through double-buffered LDS
// (row pitch 144 B to spread banks); global loads for slice k+1 are issued
// before the MFMAs of slice k.  Each 16-byte LDS read feeds one
// v_mfma_f32_32x32x16_bf16 (bf16) or four v_mfma_f32_32x32x2f32 (fp32).
// Lanes 0-31 take the even 16-byte chunk of a 32-byte K step, lanes 32-63 the
// odd one, identically for both operands, so every k is summed exactly once.

constexpr int kLdsRow = 144;

template <typename T> struct Mfma;
template <> struct Mfma<bf16> {
  static __device__ __forceinline__ f32x16_t step(uint4 a, uint4 b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static __device__ __forceinline__ f32x16_t step(uint4 a, uint4 b, f32x16_t c) {
    const f32x4_t af = __builtin_bit_cast(f32x4_t, a);
    const f32x4_t bf = __builtin_bit_cast(f32x4_t, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(af[e], bf[e], c, 0, 0, 0);
    return c;
  }
};

// 16-byte load through the global address space (the register-staged K
// loop's prefetch: a flat load would make its LDS waits wait for it).
__device__ __forceinline__ uint4 gld16(const void* p) {
  const u32x4_t v = *gvec(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Word 3 of a raw buffer descriptor on CDNA (gfx9 family): 32-bit data
// format, no swizzle, bounds checked against the byte count in word 2.
constexpr int kBufferWord3 = 0x00020000;

// 16-byte buffer load at byte offset voff + soff; reads past the
// descriptor's byte count (checked on voff) return zero.
__device__ __forceinline__ uint4 bld16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Zero the elements of a 16-byte slice at positions >= nv (nv in [0, EPV]).
template <typename T>
__device__ __forceinline__ uint4 mask_tail(uint4 v, int nv) {
  if (sizeof(T) == 2) {
    v.x &= (nv > 0 ? 0xffffu : 0u) | (nv > 1 ? 0xffff0000u : 0u);
    v.y &= (nv > 2 ? 0xffffu : 0u) | (nv > 3 ? 0xffff0000u : 0u);
    v.z &= (nv > 4 ? 0xffffu : 0u) | (nv > 5 ? 0xffff0000u : 0u);
    v.w &= (nv > 6 ? 0xffffu : 0u) | (nv > 7 ? 0xffff0000u : 0u);
  } else {
    v.x = nv > 0 ? v.x : 0u;
    v.y = nv > 1 ? v.y : 0u;
    v.z = nv > 2 ? v.z : 0u;
    v.w = nv > 3 ? v.w : 0u;
  }
  return v;
}

// f[e] += beta * element e of the 8-element chunk held in v (one 16-byte
// slice for bf16, two for fp32).
template <typename T>
__device__ __forceinline__ void add8(float f[8], const uint4* v, float beta);
template <>
__device__ __forceinline__ void add8<bf16>(float f[8], const uint4* v, float beta) {
  const uint32_t w[4] = {v[0].x, v[0].y, v[0].z, v[0].w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = fmaf(beta, __uint_as_float(w[i] << 16), f[2 * i]);
    f[2 * i + 1] = fmaf(beta, __uint_as_float(w[i] & 0xffff0000u), f[2 * i + 1]);
  }
}
template <>
__device__ __forceinline__ void add8<float>(float f[8], const uint4* v, float beta) {
  const uint32_t w[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = fmaf(beta, __uint_as_float(w[i]), f[i]);
}

// f[e] += gamma where row == col + e (the diagonal crosses this chunk).
__device__ __forceinline__ void add_diag(float f[8], int row, int col, float gamma) {
#pragma unroll
  for (int e = 0; e < 8; ++e) f[e] += (row == col + e) ? gamma : 0.f;
}

// Store 8 values at out[row * ld + col ..]: one 16-byte (bf16) or two
// 16-byte (fp32) stores when the chunk is inside [0, nr) x [0, nc), else the
// in-range elements one by one.
template <typename T>
__device__ __forceinline__ void store_chunk(T* out, int ld, int row, int col, int nr, int nc,
                                            const float f[8]) {
  if (row >= nr || col >= nc) return;
  T* p = out + int64_t(row) * ld + col;
  if (col + 8 <= nc) {
    store8(p, f);
  } else {
    for (int e = 0; e < nc - col; ++e) gstore1(p + e, from_f<T>(f[e]));
  }
}

// Epilogue shared by the NS GEMM kernels: writes the workgroup tile at
// (m0, n0) from the accumulators of its WM x WN waves (row-major layout,
// TM x TN MFMA 32x32 tiles each; wave w sits at (w / WN, w % WN), taken
// modulo WM WN so that the second K group of a split workgroup mirrors the
// first).  st: this wave's free LDS block of 32 * (32 TN + 1) floats.
// gamma is added on the diagonal of C (row == column).  Waves with
// active == false only take part in the workgroup barriers.  WG_SYNC =
// false: no workgroup barrier between the passes (every wave stages in its
// own block and the LDS runs one wave's accesses in order, so a wave needs
// no other wave to reach a pass boundary).
template <typename T, int TM, int TN, int WM = 2, int WN = 2, bool WG_SYNC = true>
__device__ __forceinline__ void gemm_epilogue(f32x16_t (&acc)[TM][TN], float* st,
                                              const GemmDesc& d, int m0, int n0, bool diag,
                                              float alpha, float beta, float gamma,
                                              bool active = true) {
  constexpr int ES = sizeof(T);
  const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) % (WM * WN);
  const int wm = wave / WN, wn = wave % WN;
  // One pass per MFMA row of the wave's sub-tile (32 x 32TN): alpha * acc
  // is staged in a wave-private LDS block (odd pitch), then each lane
  // writes 8-element (16-byte) chunks of C rows and, for the transposed
  // copy, of Ct rows read down the staged columns.  beta * D arrives as
  // bounds-checked buffer loads (rows past the matrix read zero; columns
  // past N only feed values that are not stored), issued one pass ahead so
  // their latency overlaps the previous pass.  D is added to the staged
  // rows in place, and the Ct chunks are read after that, so the transposed
  // tile needs no loads of its own (D is symmetric whenever Ct is written).
  // C == NULL: only the transposed copy is written.
  // 32x32 accumulator layout: lane l holds column l % 32 and, for register
  // v, row 8 (v / 4) + 4 (l / 32) + v % 4.
  constexpr int P = 32 * TN + 1;
  constexpr int NCH = 4 * TN;           // 8-element chunks per staged row
  constexpr int CPL = 32 * NCH / 64;    // chunks per lane, C and Ct alike
  constexpr int VPC = ES / 2;           // 16-byte slices per 8-element chunk
  const bool mirror = d.Ct != nullptr && !diag;
  const bool has_d = d.D != nullptr;
  const int wr0 = m0 + wm * 32 * TM, wc0 = n0 + wn * 32 * TN;
  const __amdgpu_buffer_rsrc_t dr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(has_d ? d.D : d.X), 0, has_d ? d.M * d.ldd * ES : 0, kBufferWord3);
  // Rows past M take the out-of-range offset (no 32-bit product past 2^31).
  T* C = static_cast<T*>(d.C);
  T* Ct = static_cast<T*>(d.Ct);
  uint4 dv[2][CPL][VPC];
  const int dbytes = has_d ? d.M * d.ldd * ES : 0;
  auto load_d = [&](int i, uint4 (&buf)[CPL][VPC]) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int q = lane + 64 * c, r = q / NCH, ch = q - r * NCH;
      const int row = wr0 + 32 * i + r;
      const int o = row < d.M ? (row * d.ldd + wc0 + 8 * ch) * ES : dbytes;
#pragma unroll
      for (int h = 0; h < VPC; ++h) buf[c][h] = bld16(dr, o + 16 * h, 0);
    }
  };
  if (has_d && active) load_d(0, dv[0]);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r0 = wr0 + 32 * i;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        st[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * P + j * 32 + (lane & 31)] = alpha * acc[i][j][v];
    if (i + 1 < TM && has_d && active) load_d(i + 1, dv[(i + 1) & 1]);
    if constexpr (WG_SYNC) __syncthreads();
#pragma unroll
    for (int c = 0; c < CPL && active; ++c) {
      const int q = lane + 64 * c, r = q / NCH, ch = q - r * NCH;
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = st[r * P + 8 * ch + e];
      if (has_d) add8<T>(f, dv[i & 1][c], beta);
      if (gamma != 0.f) add_diag(f, r0 + r, wc0 + 8 * ch, gamma);
      if (C) store_chunk<T>(C, d.ldc, r0 + r, wc0 + 8 * ch, d.M, d.N, f);
      if (mirror && has_d) {
#pragma unroll
        for (int e = 0; e < 8; ++e) st[r * P + 8 * ch + e] = f[e];
      }
    }
    if (WG_SYNC && mirror && has_d) __syncthreads();
    if (mirror && active) {
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int q = lane + 64 * c, rr = q >> 2, cc = q & 3;
        float f[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = st[(8 * cc + e) * P + rr];
        store_chunk<T>(Ct, d.ldct, wc0 + rr, r0 + 8 * cc, d.N, d.M, f);
      }
    }
    if constexpr (WG_SYNC) __syncthreads();
  }
}

// 16-byte buffer store at byte offset voff; a store at or past the
// descriptor's byte count is dropped.
__device__ __forceinline__ void bst16(__amdgpu_buffer_rsrc_t r, u32x4_t v, uint32_t voff) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, 0, 0);
}

__device__ __forceinline__ u32x4_t pack_bf16x8(const float f[8]) {
  union {
    bf16 h[8];
    u32x4_t v;
  } u;
#pragma unroll
  for (int i = 0; i < 8; ++i) u.h[i] = bf16(f[i]);
  return u.v;
}

// alpha of a product, with the unit's Frobenius scale when the descriptor
// carries one (a scalar load; read at the start of a tile, so that its
// latency is hidden by the K loop).
__device__ __forceinline__ float desc_alpha(const GemmDesc& d) {
  if (d.scale == nullptr) return d.alpha;
  const float s = d.scale[0];
  return d.alpha * (d.scale_sq ? s * s : s);
}

// Epilogue of the LDS-DMA kernel (bf16 C and Ct): the arithmetic of
// gemm_epilogue in the same order (alpha acc, then + beta D, then + gamma
// on the diagonal, one rounding to bf16), with the per-chunk work cut
// down for tiles whose rows of C (and of Ct) are whole 8-element chunks:
// buffer stores whose offset splits into a per-lane part fixed for the
// tile and a wave-uniform part per pass, rows past the matrix sent past
// the descriptor's byte count (the hardware drops them), the diagonal
// term only on passes that cross the diagonal, and no workgroup barriers
// (every wave stages in its own block, and the LDS runs one wave's
// accesses in order).  Other tiles take gemm_epilogue.
template <int TM, int TN, int WM, int WN>
__device__ __forceinline__ void dma_epilogue(f32x16_t (&acc)[TM][TN], float* st, const GemmDesc& d, int m0,
                                             int n0, bool diag, float alpha) {
  constexpr int ES = 2;
  constexpr int P = 32 * TN + 1;
  constexpr int NCH = 4 * TN;         // 8-element chunks per staged row
  constexpr int CPL = 32 * NCH / 64;  // chunks per lane, C and Ct alike
  const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) % (WM * WN);
  const int wm = wave / WN, wn = wave % WN;
  const int wr0 = m0 + wm * 32 * TM, wc0 = n0 + wn * 32 * TN;
  const bool mirror = d.Ct != nullptr && !diag;
  const bool has_d = d.D != nullptr;
  const float beta = d.beta, gamma = d.gamma;
  if (d.N % 8 != 0 || (mirror && d.M % 8 != 0)) {
    gemm_epilogue<bf16, TM, TN, WM, WN, false>(acc, st, d, m0, n0, diag, alpha, beta, gamma);
    return;
  }
  // Byte offsets as the sum of a per-lane part fixed for the tile (row and
  // column within the wave block) and a wave-uniform part per pass (the
  // block's origin).  A chunk outside the matrix takes the byte count
  // itself as its offset, so that no offset reaches 2^31 (the bounds check
  // does not drop offsets from 2^31 up).
  const uint32_t cbytes = d.C ? uint32_t(d.M) * uint32_t(d.ldc) * ES : 0u;
  const uint32_t tbytes = mirror ? uint32_t(d.N) * uint32_t(d.ldct) * ES : 0u;
  const uint32_t dbytes = has_d ? uint32_t(d.M) * uint32_t(d.ldd) * ES : 0u;
  const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(d.C ? d.C : d.Ct, 0, cbytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t tr = __builtin_amdgcn_make_buffer_rsrc(d.Ct ? d.Ct : d.C, 0, tbytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t dr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(has_d ? d.D : d.X), 0, dbytes, kBufferWord3);
  // Per lane: row and column of each C chunk within the 32-row block of a
  // pass, and of each Ct chunk within the wave's block of Ct; whether a C
  // chunk's columns (a Ct chunk's rows) lie inside the matrix.
  int crow[CPL], ccol[CPL], trow[CPL], tcol[CPL];
  bool cin[CPL], tin[CPL];
  uint32_t coff[CPL], doff[CPL], toff[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int q = lane + 64 * c;
    crow[c] = q / NCH;
    ccol[c] = 8 * (q - crow[c] * NCH);
    trow[c] = q >> 2;
    tcol[c] = 8 * (q & 3);
    cin[c] = wc0 + ccol[c] < d.N;
    tin[c] = wc0 + trow[c] < d.N;
    coff[c] = uint32_t(crow[c] * d.ldc + ccol[c]) * ES;
    doff[c] = uint32_t(crow[c] * d.ldd + ccol[c]) * ES;
    toff[c] = uint32_t(trow[c] * d.ldct + tcol[c]) * ES;
  }
  uint4 dv[2][CPL];
  auto load_d = [&](int i, uint4 (&buf)[CPL]) {
    const int r0 = wr0 + 32 * i;
    const uint32_t so = r0 < d.M ? uint32_t(r0 * d.ldd + wc0) * ES : 0u;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const bool in = cin[c] && r0 + crow[c] < d.M;
      const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(dr, in ? doff[c] + so : dbytes, 0, 0);
      buf[c] = make_uint4(v.x, v.y, v.z, v.w);
    }
  };
  if (has_d) load_d(0, dv[0]);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r0 = wr0 + 32 * i;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        st[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * P + j * 32 + (lane & 31)] = alpha * acc[i][j][v];
    if (i + 1 < TM && has_d) load_d(i + 1, dv[(i + 1) & 1]);
    // The diagonal crosses this pass's 32 x 32 TN block.
    const bool dg = gamma != 0.f && r0 < wc0 + 32 * TN && wc0 < r0 + 32;
    if (d.C || (mirror && (has_d || dg))) {
      const uint32_t so = r0 < d.M ? uint32_t(r0 * d.ldc + wc0) * ES : 0u;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        float f[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = st[crow[c] * P + ccol[c] + e];
        if (has_d) add8<bf16>(f, &dv[i & 1][c], beta);
        if (dg) add_diag(f, r0 + crow[c], wc0 + ccol[c], gamma);
        if (d.C) bst16(cr, pack_bf16x8(f), cin[c] && r0 + crow[c] < d.M ? coff[c] + so : cbytes);
        if (mirror && (has_d || dg)) {
#pragma unroll
          for (int e = 0; e < 8; ++e) st[crow[c] * P + ccol[c] + e] = f[e];
        }
      }
    }
    if (mirror) {
      const uint32_t so = wc0 < d.N ? uint32_t(wc0 * d.ldct + r0) * ES : 0u;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        float f[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = st[(tcol[c] + e) * P + trow[c]];
        bst16(tr, pack_bf16x8(f), tin[c] && r0 + tcol[c] < d.M ? toff[c] + so : tbytes);
      }
    }
  }
}

template <typename T, int BM, int BN, int KS>
struct GemmShape {
  static constexpr int EPV = 16 / sizeof(T);  // elements per 16-byte slice
  static constexpr int BK = 8 * EPV;          // elements per 128-byte K slice
  static constexpr int TM = BM / 64;          // MFMA tiles per wave, rows
  static constexpr int TN = BN / 64;          // MFMA tiles per wave, columns
  static constexpr int QX = BM * 8 / 256;     // 16-byte X slices per thread per stage
  static constexpr int QY = BN * 8 / 256;
  static constexpr int LDS_X = BM * kLdsRow;
  static constexpr int LDS_STAGE = (BM + BN) * kLdsRow;
  static constexpr int ST_PITCH = 32 * TN + 1;  // epilogue staging pitch (floats)
  static constexpr int LDS_EPI = KS * 4 * 32 * ST_PITCH * 4;
  static constexpr int LDS_RED = (KS - 1) * 4 * TM * TN * 16 * 64 * 4;  // split-K partials
  static constexpr int LDS_LOOP = KS * 2 * LDS_STAGE;
  static constexpr int LDS_BYTES = LDS_LOOP > LDS_EPI ? (LDS_LOOP > LDS_RED ? LDS_LOOP : LDS_RED)
                                                      : (LDS_EPI > LDS_RED ? LDS_EPI : LDS_RED);
};

//
// KS > 1 splits K inside the workgroup: KS groups of 4 waves each run the
// K loop over every KS-th slice with their own LDS buffers, and the partial
// sums are added in LDS (a fixed order) before the epilogue.  Used when a
// launch has too few tiles to give every CU two workgroups.
template <typename T, int BM, int BN, int KS, bool TWO = false>
__global__ __launch_bounds__(kThreads * KS) void k_ns_gemm(const GemmDesc* __restrict__ probs,
                                                           const TileRef* __restrict__ tiles) {
  using G = GemmShape<T, BM, BN, KS>;
  constexpr int EPV = G::EPV, BK = G::BK, TM = G::TM, TN = G::TN, QX = G::QX, QY = G::QY;
  __shared__ __attribute__((aligned(16))) unsigned char lds[G::LDS_BYTES];

  const TileRef t = tiles[blockIdx.x];
  const GemmDesc d = probs[t.prob];
  const float alpha = desc_alpha(d);
  const int ti = t.ij >> 16, tj = t.ij & 0xffff;
  const int m0 = ti * BM, n0 = tj * BN;
  const int grp = threadIdx.x >> 8;       // K group
  const int tid = threadIdx.x & 255;      // thread inside the group
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  unsigned char* glds = lds + grp * 2 * G::LDS_STAGE;

  // Operands are read with buffer loads: one 32-bit offset per 16-byte slice
  // (constant over the K loop) plus the K position as a uniform scalar
  // offset.  Rows at or beyond M (N) take an offset past the descriptor's
  // byte count (never a row product, which could pass 2^31 for the last
  // tile of a unit just under the operand limit) and read as zero; columns
  // at or beyond K are masked to zero in the last K
  // slice, which may straddle K (rows are padded to a multiple of 8 elements,
  // so the read stays inside the row).
  constexpr int ES = sizeof(T);
  const int xbytes = d.M * d.ldx * ES, ybytes = d.N * d.ldy * ES;
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(d.X), 0, xbytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(d.Y), 0, ybytes, kBufferWord3);
  const int kc = (tid & 7) * EPV;  // this thread's column inside a K slice
  int xo[QX], yo[QY];
#pragma unroll
  for (int q = 0; q < QX; ++q) {
    const int r = m0 + (tid >> 3) + 32 * q;
    xo[q] = r < d.M ? (r * d.ldx + kc) * ES : xbytes;
  }
#pragma unroll
  for (int q = 0; q < QY; ++q) {
    const int r = n0 + (tid >> 3) + 32 * q;
    yo[q] = r < d.N ? (r * d.ldy + kc) * ES : ybytes;
  }
  uint4 rx[QX], ry[QY];
  auto gload = [&](int k0) {
#pragma unroll
    for (int q = 0; q < QX; ++q) rx[q] = bld16(xr, xo[q], k0 * ES);
#pragma unroll
    for (int q = 0; q < QY; ++q) ry[q] = bld16(yr, yo[q], k0 * ES);
  };
  // A slice entirely past K is read through an out-of-range offset: the
  // bounds check covers the per-lane offset only (not the scalar K offset),
  // so this is what keeps such lanes from touching memory past the row.
  auto gload_tail = [&](int k0) {
    const int nv = max(0, min(d.K - (k0 + kc), EPV));
#pragma unroll
    for (int q = 0; q < QX; ++q) rx[q] = mask_tail<T>(bld16(xr, nv > 0 ? xo[q] : xbytes, k0 * ES), nv);
#pragma unroll
    for (int q = 0; q < QY; ++q) ry[q] = mask_tail<T>(bld16(yr, nv > 0 ? yo[q] : ybytes, k0 * ES), nv);
  };
  auto lstore = [&](int buf) {
    unsigned char* base = glds + buf * G::LDS_STAGE;
    const int off = (tid >> 3) * kLdsRow + (tid & 7) * 16;
#pragma unroll
    for (int q = 0; q < QX; ++q)
      *reinterpret_cast<uint4*>(base + off + q * 32 * kLdsRow) = rx[q];
#pragma unroll
    for (int q = 0; q < QY; ++q)
      *reinterpret_cast<uint4*>(base + G::LDS_X + off + q * 32 * kLdsRow) = ry[q];
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  // TWO (fp32, launches over a very long K): the accumulators are added
  // into a second set every kFlush iterations (kFlush x 32 K) and
  // restarted, so that no fp32 sum runs over more than 2048 products.  Over
  // a long K one accumulator per output loses most of each product's bits
  // once the products are a few units in the last place of the running sum
  // (a 124-row unit's U was 6.9e-4 from the fp64 result at K = 4065000).
  // The second set costs 64 registers (one workgroup per CU instead of
  // two), so shorter launches keep the single set.
  constexpr bool kTwoLevel = TWO && std::is_same<T, float>::value && TM * TN <= 4;
  constexpr int kFlush = 64;
  f32x16_t hi[kTwoLevel ? TM : 1][kTwoLevel ? TN : 1];
  if constexpr (kTwoLevel) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) hi[i][j][v] = 0.f;
  }

  // Group grp handles K slices kt = KS it + grp, it < niter (the same count
  // in every group, so all threads meet every barrier); slices past K load
  // as zeros.
  const int nk = (d.K + BK - 1) / BK;
  const int niter = (nk + KS - 1) / KS;
  auto fetch = [&](int kt) {
    if ((kt + 1) * BK <= d.K) gload(kt * BK); else gload_tail(kt * BK);
  };
  fetch(grp);
  lstore(0);
  __syncthreads();
  const int xoff = (wm * 32 * TM + (lane & 31)) * kLdsRow;
  const int yoff = G::LDS_X + (wn * 32 * TN + (lane & 31)) * kLdsRow;
  for (int it = 0; it < niter; ++it) {
    const int buf = it & 1;
    if (it + 1 < niter) fetch((it + 1) * KS + grp);
    // Fragments of K step s + 1 are read from LDS before the MFMAs of step s
    // (two register sets), so LDS latency overlaps the matrix pipeline.
    const unsigned char* S = glds + buf * G::LDS_STAGE;
    uint4 a[2][TM], b[2][TN];
    auto frag = [&](int s, uint4* fa, uint4* fb) {
      const int koff = (2 * s + (lane >> 5)) * 16;
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const uint4*>(S + xoff + i * 32 * kLdsRow + koff);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const uint4*>(S + yoff + j * 32 * kLdsRow + koff);
    };
    frag(0, a[0], b[0]);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s < 3) frag(s + 1, a[(s + 1) & 1], b[(s + 1) & 1]);
      // Keep the reads above where they are: the scheduler would otherwise
      // sink each read next to its first use and expose its latency.
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = Mfma<T>::step(a[s & 1][i], b[s & 1][j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (kTwoLevel) {
      if (it % kFlush == kFlush - 1) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            hi[i][j] += acc[i][j];
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
          }
      }
    }
    if (it + 1 < niter) lstore(buf ^ 1);
    __syncthreads();
  }
  if constexpr (kTwoLevel) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = hi[i][j] + acc[i][j];
  }
  if (KS > 1) {
    // Groups 1.. hand their partial sums to group 0 through LDS, register by
    // register (same lane layout), and group 0 adds them in group order.
    float* red = reinterpret_cast<float*>(lds);
    constexpr int PER_WAVE = TM * TN * 16 * 64;
    if (grp > 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            red[((grp - 1) * 4 + wave) * PER_WAVE + ((i * TN + j) * 16 + v) * 64 + lane] = acc[i][j][v];
    }
    __syncthreads();
    if (grp == 0) {
      for (int g = 1; g < KS; ++g)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
              acc[i][j][v] += red[((g - 1) * 4 + wave) * PER_WAVE + ((i * TN + j) * 16 + v) * 64 + lane];
    }
    __syncthreads();
  }

  gemm_epilogue<T, TM, TN>(acc, reinterpret_cast<float*>(lds) + (threadIdx.x >> 6) * 32 * (32 * TN + 1),
                           d, m0, n0, ti == tj && d.sym, alpha, d.beta, d.gamma, grp == 0);
}

// ---------------------------------------------------------------- NS GEMM, LDS-DMA staging
//
// The bf16 kernel below serves units whose K is a multiple of 8.  Operand
// slices go straight from global memory into LDS (buffer_load_dwordx4 ...
// lds: lane l of a wave writes 16 bytes at the wave's LDS window + 16 l),
// through a ring of NS stages of 32-element (64-byte) K slices, NS - 1
// slices ahead of the MFMAs; no registers hold prefetched data.  Inside
// a stage a row occupies 64 bytes as four 16-byte chunks, chunk c stored at
// position c ^ swz(row), swz(row) = ((row >> 1) & 3) ^ ((row >> 3) & 1), so
// that any 8 (or 16) consecutive rows read at the same chunk by one MFMA
// operand fetch hit distinct LDS banks.  Rows past M (N) and chunks past K
// are read through an out-of-range offset and land as zeros.

constexpr int kDmaRow = 64;  // bytes per staged row (32 bf16)

// s_waitcnt immediate that waits until at most n vector-memory operations
// of this wave are outstanding (exp and lgkm counters left at their maxima).
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

template <int BM, int BN, int NS>
struct DmaShape {
  static constexpr int TM = BM / 64, TN = BN / 64;
  static constexpr int STAGE = (BM + BN) * kDmaRow;     // bytes per stage
  static constexpr int LPW = (BM + BN) / 64;            // 1 KB loads per wave per stage
  static constexpr int ST_PITCH = 32 * TN + 1;
  static constexpr int LDS_EPI = 4 * 32 * ST_PITCH * 4;
  static constexpr int LDS_BYTES = NS * STAGE > LDS_EPI ? NS * STAGE : LDS_EPI;
};

typedef __attribute__((address_space(3))) void lds_void_t;

// One 16-byte buffer load per lane straight into LDS: lane l writes at
// dst + 16 l; offsets past the descriptor's byte count write zeros.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, lds_void_t* dst, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
}

__device__ __forceinline__ int swz(int row) { return ((row >> 1) & 3) ^ ((row >> 3) & 1); }


// 16-byte LDS read issued without a compiler-inserted wait: the compiler
// would otherwise make every LDS read wait for all copies into LDS still in
// flight (it cannot tell the stages apart).  lds_wait() must complete the
// reads before their registers are used; it takes the fragments as in/out
// operands so that no use can be scheduled above it.
__device__ __forceinline__ u32x4_t lds_read16(uint32_t addr) {
  u32x4_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

// LDS transpose read (gfx950 ds_read_b64_tr_b16), issued without a
// compiler-inserted wait like lds_read16.  Each group of 16 lanes reads a 4 x
// 16 block of 16-bit elements: lane i of the group supplies the address of
// elements 4 (i % 4) .. 4 (i % 4) + 3 of row i / 4, and receives column i of
// the block, rows 0..3 (measured lane layout).  With a row-major K x N tile
// that gives each lane four consecutive k of one n: half of an MFMA B
// operand.
__device__ __forceinline__ u32x2_t lds_read8_tr(uint32_t addr) {
  u32x2_t v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t (&f)[N]) {
  static_assert(N >= 4 && N <= 8, "fragment count");
  if constexpr (N == 4)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]));
  else if constexpr (N == 5)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]));
  else if constexpr (N == 6)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]));
  else if constexpr (N == 7)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]),
                   "+v"(f[6]));
  else
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]),
                   "+v"(f[6]), "+v"(f[7]));
}

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every copy into LDS still in flight, including the ones the
// pipeline keeps ahead on purpose.  Completion of the copies that matter is
// waited for explicitly before it; the memory clobber keeps the compiler from
// moving memory operations across it.
__device__ __forceinline__ void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void_t*)p));
}

// ---------------------------------------------------------------- NS GEMM, interleaved DMA pipeline
//
// The operands are staged as described above (a 4-stage ring of 32-element
// K slices, straight from global memory into LDS), and the loop is
// scheduled so that the matrix pipeline never drains at a slice boundary:
//
//   * both K steps of a slice are read from LDS one step ahead, each read
//     issued between two MFMAs of the previous step;
//   * the barrier that publishes the next slice sits right after the first
//     MFMA of the current slice's second step (that MFMA keeps running);
//   * right after it, the copy that refills the slot just consumed and the
//     reads of the next slice's first step are spread over the remaining
//     MFMAs.
//
// Slices past K are copied too (as zeros, through an out-of-range offset),
// so the loop has no branches and every wait is a constant count.
//
// Waves: WM x WN, row-major; 2 x 2 (one wave per SIMD), or 8 waves as
// 2 x 4 / 4 x 2 so that each SIMD holds two waves whose MFMAs cover each
// other's waits (the sub-tile then needs half the accumulator registers).
//
// K split (nsplit > 1): the workgroups of one tile each run about 1/nsplit
// of its K slices (share t.part), store their fp32 sums at
// ksum[(t.slot * nsplit + part) * BM * BN] (MFMA register order), and count
// themselves in kcount[t.slot].  The last to arrive adds the nsplit sums in
// share order (the result does not depend on the arrival order), resets
// the counter for the next launch and runs the epilogue; the others exit.
// No workgroup waits for another.
//
// NN (Y row-major K x N, ldy its row pitch; the apply product reads Z this
// way, so no transposed copy of Z is needed): a stage holds the Y slice as
// 32 k-rows of BN elements, 16-byte chunk c of k-row r stored at position
// c ^ nn_swz<BN>(r), and the B operands come from LDS transpose reads, two
// per fragment (k 0..3 and 4..7 of the lane's 8).  Y chunks past N and
// k-rows past K are copied as zeros.
// Chunk swizzle of the NN Y stage.  The 32 lanes of one LDS transpose-read
// pass fetch k-rows r0 .. r0 + 3 (r0 % 4 == 0) x four aligned 16-byte chunks
// of each row.  With a row pitch of 512 or 256 bytes every row starts on
// the same banks, so row r's chunks move by 4 (r % 4) (64 bytes): the 16
// chunks land on 16 different 16-byte bank groups.  With 384 bytes odd rows
// already start 128 bytes over, and 4 ((r % 4) / 2) separates the rest while
// staying inside each aligned group of 8 chunks (a row has 24).
template <int BN>
__device__ __forceinline__ int nn_swz(int r) {
  return BN % 128 == 0 ? 4 * (r & 3) : 4 * ((r & 3) >> 1);
}

template <int BM, int BN, bool NN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void k_ns_gemm_dmap(const GemmDesc* __restrict__ probs,
                                                           const TileRef* __restrict__ tiles,
                                                           int nsplit, float* __restrict__ ksum,
                                                           int* __restrict__ kcount) {
  constexpr int NS = 4;
  using G = DmaShape<BM, BN, NS>;
  using T = bf16;
  // WM x WN waves, each owning a (BM / WM) x (BN / WN) sub-tile of TM x TN
  // MFMA tiles.  A slice is RG copies of 1 KB (16 rows of X or Y, or two NN
  // k-rows); wave w issues copies w, w + W, ...  When W does not divide RG,
  // a wave past the last copy repeats its previous one (same bytes to the
  // same LDS place), so that every wave has LPW copies per slice in flight
  // and the waits stay constant counts.
  constexpr int W = WM * WN;
  constexpr int TM = BM / (32 * WM), TN = BN / (32 * WN), ES = 2, NF = TM + TN;
  constexpr int RG = (BM + BN) / 16;
  constexpr int LPW = (RG + W - 1) / W;
  static_assert(TM * 32 * WM == BM && TN * 32 * WN == BN && RG * 16 == BM + BN, "wave layout");
  constexpr int NM = TM * TN;  // MFMAs per K step
  // LDS read instructions per K step: one per X fragment; one per Y
  // fragment (NT) or two (NN).
  constexpr int NR = NN ? TM + 2 * TN : NF;
  constexpr int RPM = (NR + NM - 1) / NM;  // reads issued after each MFMA of a step
  constexpr int CPR = BN / 8;  // NN: 16-byte chunks per staged k-row
  static_assert(!NN || (BN % 128 == 0 ? CPR % 16 == 0 : CPR % 8 == 0), "NN chunk swizzle range");
  static_assert(BM % 16 == 0, "copies hold X rows or Y rows, not both");
  // MFMAs of the second step issued before the barrier: one keeps the
  // matrix pipeline busy while the barrier resolves, and leaves the rest of
  // the step to hide the next slice's reads (measured: 2-4% faster than
  // half the step on every tile shape).
  constexpr int H = 1;
  constexpr int EPI = W * 32 * (32 * TN + 1) * 4;  // epilogue staging, one block per wave
  __shared__ __attribute__((aligned(1024))) unsigned char lds[NS * G::STAGE > EPI ? NS * G::STAGE : EPI];

  const TileRef t = tiles[blockIdx.x];
  const GemmDesc d = probs[t.prob];
  const float alpha = desc_alpha(d);
  const int ti = t.ij >> 16, tj = t.ij & 0xffff;
  const int m0 = ti * BM, n0 = tj * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  const int xbytes = d.M * d.ldx * ES, ybytes = (NN ? d.K : d.N) * d.ldy * ES;
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(d.X), 0, xbytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(d.Y), 0, ybytes, kBufferWord3);

  // cu[jj]: which of the slice's RG copies copy jj is (wave-uniform);
  // chunk[jj]: K chunk of an X (or NT Y) row; NN Y: the k-row in the slice.
  // holds_x(jj): copy jj holds X rows.  With 4 waves (every copy index
  // jj is all X or all Y) the tests are the ones the kernel has always
  // used; with 8 the W copies of one index may straddle the X / Y boundary,
  // and the test is then made per wave.
  constexpr int XG = BM / 16;  // copies of X rows per slice
  constexpr bool EVEN = RG % W == 0;
  static_assert(W == 8 || (W == 4 && EVEN && BM % (16 * W) == 0), "4-wave copy layout");
  int voff[LPW], chunk[LPW], cu[LPW];
  auto holds_x = [&](int jj) {
    if constexpr (W == 4) {
      return NN ? jj < BM / 64 : wave + 4 * jj < BM / 16;
    } else {
      const int lo = (!EVEN && jj == LPW - 1) ? W * (jj - 1) : W * jj;  // lowest copy index
      if (W * jj + W <= XG) return true;
      if (lo >= XG) return false;
      return cu[jj] < XG;
    }
  };
#pragma unroll
  for (int jj = 0; jj < LPW; ++jj) {
    const int u = (EVEN || wave + W * jj < RG) ? wave + W * jj : wave + W * (jj - 1);
    cu[jj] = u;
    if (NN && !holds_x(jj)) {  // Y slice copy
      const int q = 64 * (u - BM / 16) + lane, kr = q / CPR;
      const int cn = (q - kr * CPR) ^ nn_swz<BN>(kr);
      chunk[jj] = kr;
      // k-row kr of every slice: past K in all of them when kr >= K.
      voff[jj] = n0 + 8 * cn < d.N && kr < d.K ? (kr * d.ldy + n0 + 8 * cn) * ES : ybytes;
    } else {
      const int row = 16 * u + (lane >> 2);
      const int c = (lane & 3) ^ swz(row);
      chunk[jj] = c;
      // Rows past M (N) take the out-of-range offset, not a row product
      // (which could pass 2^31 in the last tile of a unit near the limit).
      if (row < BM)
        voff[jj] = m0 + row < d.M ? ((m0 + row) * d.ldx + 8 * c) * ES : xbytes;
      else
        voff[jj] = n0 + row - BM < d.N ? ((n0 + row - BM) * d.ldy + 8 * c) * ES : ybytes;
    }
  }
  const int nk_all = (d.K + 31) / 32;
  const int kb = nsplit > 1 ? t.part * nk_all / nsplit : 0;
  const int ke = nsplit > 1 ? (t.part + 1) * nk_all / nsplit : nk_all;
  // Copy jj of slice kt into its ring slot (slices outside [kb, ke) as zeros).
  auto copy = [&](int kt, int jj) {
    unsigned char* base = lds + (kt % NS) * G::STAGE;
    const int k0 = kt * 32;
    lds_void_t* dst = (lds_void_t*)(base + (W == 4 ? wave + 4 * jj : cu[jj]) * 1024);
    if constexpr (NN) {
      if (holds_x(jj)) {  // uniform: X rows
        const bool kin = kt < ke && k0 + 8 * chunk[jj] < d.K;
        dma16(xr, dst, kin ? voff[jj] : xbytes, k0 * ES);
      } else {
        const bool kin = kt < ke && k0 + chunk[jj] < d.K;
        // The slice's k-row offset only for slices that start inside K
        // (k0 ldy < K ldy, so the product stays below the byte count).
        dma16(yr, dst, kin ? voff[jj] : ybytes, (k0 < d.K ? k0 : 0) * d.ldy * ES);
      }
    } else {
      const bool kin = kt < ke && k0 + 8 * chunk[jj] < d.K;
      if (holds_x(jj))  // uniform: X rows
        dma16(xr, dst, kin ? voff[jj] : xbytes, k0 * ES);
      else
        dma16(yr, dst, kin ? voff[jj] : ybytes, k0 * ES);
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  uint32_t fa[NF];
  int fsw[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int r = f < TM ? wm * 32 * TM + 32 * f + (lane & 31) : BM + wn * 32 * TN + 32 * (f - TM) + (lane & 31);
    fa[f] = lds_addr(lds) + r * kDmaRow;
    fsw[f] = swz(r);
  }
  if (NN) {
    // Y fragment j: n = wn 32 TN + 32 j + 16 ((lane / 16) % 2) + 4 (lane % 4)
    // .. + 3, k-row 8 (lane / 32) + (lane % 16) / 4 (+ 16 s + 4 r); the
    // k-row % 4 the swizzle depends on is (lane % 16) / 4.
    const int si = lane & 15, g = lane >> 4;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = wn * 32 * TN + 32 * j + 16 * (g & 1) + 4 * (si & 3);
      const int kr = 8 * (g >> 1) + (si >> 2);
      fa[TM + j] = lds_addr(lds) + BM * kDmaRow + kr * (2 * BN) + (((n >> 3) ^ nn_swz<BN>(si >> 2)) << 4) +
                   8 * (si & 1);
    }
  }
  // A diagonal tile of a product whose two operands are the same rows of
  // the same matrix (the Gram Z Z^T, the polynomial's A A) needs only the X
  // panel: the Y fragments are read from the X rows (fas), and the slice's
  // copies are the X copies alone (the first XG / W of every wave).
  constexpr bool kShareXY = !NN && EVEN && XG % W == 0;
  const bool share_xy = kShareXY && ti == tj && d.X == d.Y && d.ldx == d.ldy && d.M == d.N;
  uint32_t fas[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) fas[f] = f < TM ? fa[f] : fa[f] - BM * kDmaRow;
  auto read1 = [&](auto sh, int kt, int s, int f) {
    const uint32_t sbase = (kt % NS) * G::STAGE;
    const int c = 2 * s + (lane >> 5);
    const uint32_t base = decltype(sh)::value ? fas[f] : fa[f];
    return lds_read16(base + sbase + ((c ^ fsw[f]) << 4));
  };
  // Fragments of one K step: f (X, and Y when NT) from 16-byte reads; NN Y
  // fragments from two transpose reads each, held as halves (yl, yh) until
  // their wait and then joined into f[TM + j].
  constexpr int YH = NN ? TN : 1;
  using Fr = u32x4_t[NF];
  using Yh = u32x2_t[YH];
  // Read instruction o (0 <= o < NR) of K step s of slice kt.
  auto read_op = [&](auto sh, Fr& f, Yh& yl, Yh& yh, int kt, int s, int o) {
    if constexpr (!NN) {
      f[o] = read1(sh, kt, s, o);
    } else {
      if (o < TM) {
        f[o] = read1(sh, kt, s, o);
      } else {
        const int j = (o - TM) >> 1, r = (o - TM) & 1;
        const uint32_t a = fa[TM + j] + (kt % NS) * G::STAGE + (16 * s + 4 * r) * (2 * BN);
        if (r == 0)
          yl[j] = lds_read8_tr(a);
        else
          yh[j] = lds_read8_tr(a);
      }
    }
  };
  auto frag_wait = [&](Fr& f, Yh& yl, Yh& yh) {
    if constexpr (!NN) {
      lds_wait(f);
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int i = 0; i < TM; ++i) asm volatile("" : "+v"(f[i]));
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        asm volatile("" : "+v"(yl[j]), "+v"(yh[j]));
        f[TM + j] = __builtin_shufflevector(yl[j], yh[j], 0, 1, 2, 3);
      }
    }
  };
  auto mfma = [&](const Fr& fr, int q) {
    const int i = q / TN, j = q % TN;
    acc[i][j] = Mfma<T>::step(__builtin_bit_cast(uint4, fr[i]), __builtin_bit_cast(uint4, fr[TM + j]),
                              acc[i][j]);
  };

  // Idle waves run the K loop's copies, waits and barriers but no MFMAs or
  // fragment reads, and store nothing.  In a diagonal tile of a symmetric
  // product those are the waves whose sub-tile lies strictly below the
  // diagonal, and the waves whose sub-tile lies strictly above it write
  // their block's transpose there (Ct = C): with 2 x 4 or 2 x 2 waves on a
  // square tile the blocks below are exactly the transposes of the blocks
  // above.  (Not where the epilogue takes the general path: rows of C not
  // whole 8-element chunks.)
  constexpr bool kDiagSkip = BM == BN && WM == 2 && (WN == 4 || WN == 2);
  const bool dtile = kDiagSkip && ti == tj && d.sym && d.Ct == d.C && d.M % 8 == 0 && d.N % 8 == 0;
  const int lr0 = wm * 32 * TM, lc0 = wn * 32 * TN;  // the wave's sub-tile inside the tile
  const bool below = dtile && lr0 >= lc0 + 32 * TN;
  const bool above = dtile && lc0 >= lr0 + 32 * TM;
  // So is a wave whose whole sub-tile lies past M or N (a unit smaller than
  // the tile), whose rows or columns of C are never stored.
  const bool idle = below || m0 + lr0 >= d.M || n0 + lc0 >= d.N;

  u32x4_t f0[NF], f1[NF];
  u32x2_t y0l[YH], y0h[YH], y1l[YH], y1h[YH];
  auto kloop = [&](auto math, auto sh) {
    constexpr bool MATH = decltype(math)::value;
    // Copies per wave and slice: all LPW, or the X copies alone.
    constexpr int LP = decltype(sh)::value ? XG / W : LPW;
    // Prologue: fill the ring, publish slice kb, read its first K step.
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int jj = 0; jj < LP; ++jj) copy(kb + s, jj);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 1) * LP));
    barrier_no_fence();
    if constexpr (MATH)
#pragma unroll
      for (int o = 0; o < NR; ++o) read_op(sh, f0, y0l, y0h, kb, 0, o);
    frag_wait(f0, y0l, y0h);

    for (int kt = kb; kt < ke; ++kt) {
      // 8 waves: waves w and w + 4 share a SIMD.  Their issue priority swaps
      // every slice, so that neither falls behind the other on every slice
      // and holds up the barrier (measured: Gram 2%, step 0.7-0.9% faster
      // than equal priorities; swapping every K step was 2% slower).
      if constexpr (W == 8) {
        if (((kt + (wave >> 2)) & 1) != 0)
          __builtin_amdgcn_s_setprio(1);
        else
          __builtin_amdgcn_s_setprio(0);
      }
      // Step 0 of slice kt, with the reads of its step 1.
#pragma unroll
      for (int q = 0; q < NM; ++q) {
        if constexpr (MATH) {
          mfma(f0, q);
#pragma unroll
          for (int o = q * RPM; o < (q + 1) * RPM && o < NR; ++o) read_op(sh, f1, y1l, y1h, kt, 1, o);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      frag_wait(f1, y1l, y1h);
      // Step 1, first part.
#pragma unroll
      for (int q = 0; q < H; ++q) {
        if constexpr (MATH) mfma(f1, q);
        __builtin_amdgcn_sched_barrier(0);
      }
      // Slice kt + 1 has landed for this wave (two later slices may still be
      // in flight); after the barrier it has landed for every wave, and no
      // wave reads slice kt any more, so its slot takes slice kt + NS.
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LP));
      barrier_no_fence();
      // Step 1, rest, with the reads of slice kt + 1 and the refill copies.
      constexpr int OPS = LP + NR;
#pragma unroll
      for (int q = H; q < NM; ++q) {
        if constexpr (MATH) mfma(f1, q);
        constexpr int R = NM - H;
        const int lo = (q - H) * OPS / R, hi = (q - H + 1) * OPS / R;
#pragma unroll
        for (int o = lo; o < hi; ++o) {
          if (o < NR) {
            if constexpr (MATH) read_op(sh, f0, y0l, y0h, kt + 1, 0, o);
          } else
            copy(kt + NS, o - NR);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      frag_wait(f0, y0l, y0h);
    }
  };
  if (share_xy) {
    if constexpr (kShareXY) {
      if (idle)
        kloop(std::false_type{}, std::true_type{});
      else
        kloop(std::true_type{}, std::true_type{});
    }
  } else if (idle) {
    kloop(std::false_type{}, std::false_type{});
  } else {
    kloop(std::true_type{}, std::false_type{});
  }
  // Zero-filled copies past the share may still be in flight: let them land
  // before the epilogue reuses the ring.
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  if (nsplit > 1) {
    // The sums are stored and loaded as device-coherent relaxed atomics
    // (they bypass the per-XCD caches), and every store has completed before
    // the share is counted.  A device-scope fence would do the same for
    // plain accesses but writes back and invalidates the whole L2, which
    // costs the other workgroups their cached operands.
    constexpr int PER_WAVE = NM * 16 * 64;
    float* mine = ksum + (size_t(t.slot) * nsplit + t.part) * (BM * BN) + wave * PER_WAVE;
#pragma unroll
    for (int q = 0; q < NM; ++q)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        __hip_atomic_store(mine + (q * 16 + v) * 64 + lane, acc[q / TN][q % TN][v], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __shared__ int last;
    __syncthreads();
    if (tid == 0)
      last = __hip_atomic_fetch_add(kcount + t.slot, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
             nsplit - 1;
    __syncthreads();
    if (!last) return;
    const float* all = ksum + size_t(t.slot) * nsplit * (BM * BN) + wave * PER_WAVE;
    for (int p = 0; p < nsplit; ++p)
#pragma unroll
      for (int q = 0; q < NM; ++q)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float x = __hip_atomic_load(all + size_t(p) * (BM * BN) + (q * 16 + v) * 64 + lane,
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          acc[q / TN][q % TN][v] = p == 0 ? x : acc[q / TN][q % TN][v] + x;
        }
    if (tid == 0) __hip_atomic_store(kcount + t.slot, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (idle) return;
  dma_epilogue<TM, TN, WM, WN>(acc, reinterpret_cast<float*>(lds) + wave * 32 * (32 * TN + 1), d, m0, n0,
                              ti == tj && d.sym && !above, alpha);
}

// ---------------------------------------------------------------- update

template <typename TP, typename TU, bool VEC, bool NT>
__global__ __launch_bounds__(kThreads) void k_update(
    const SegDesc* __restrict__ segs, const BlockDesc* __restrict__ blocks,
    const MatPtrs* __restrict__ mats, const UpdDesc* __restrict__ upd, float eta,
    float lambda) {
  const SegDesc sd = segs[blockIdx.x];
  const BlockDesc bd = blocks[sd.block];
  const UpdDesc ud = upd[sd.block];
  TP* x = static_cast<TP*>(mats[bd.mat].param) + bd.in_mat_off + int64_t(sd.row_begin) * bd.ld;
  const TU* u = static_cast<const TU*>(ud.u) + int64_t(sd.row_begin) * ud.ldu;
  const float decay = 1.f - eta * lambda, step = eta * ud.s;
  const int cols = bd.cols;
  if (VEC) {
    const int vpr = cols >> 3;
    const int nv = sd.nrows * vpr;
    for (int v0 = threadIdx.x; v0 < nv; v0 += kThreads * kStreamUnroll) {
      Raw8<TP> xr[kStreamUnroll];
      Raw8<TU> ur[kStreamUnroll];
      int64_t ox[kStreamUnroll];
#pragma unroll
      for (int k = 0; k < kStreamUnroll; ++k) {
        const int v = v0 + kThreads * k;
        if (v < nv) {
          const int r = v / vpr, c = (v - r * vpr) << 3;
          ox[k] = int64_t(r) * bd.ld + c;
          xr[k] = load8r<NT>(x + ox[k]);
          ur[k] = load8r<NT>(u + int64_t(r) * ud.ldu + c);
        }
      }
#pragma unroll
      for (int k = 0; k < kStreamUnroll; ++k) {
        if (v0 + kThreads * k < nv) {
          float xf[8], uf[8];
          unpack8(xr[k], xf);
          unpack8(ur[k], uf);
#pragma unroll
          for (int i = 0; i < 8; ++i) xf[i] = fmaf(decay, xf[i], -step * uf[i]);
          store8r<NT>(x + ox[k], xf);
        }
      }
    }
  } else {
    const int n = sd.nrows * cols;
    for (int e = threadIdx.x; e < n; e += kThreads) {
      const int r = e / cols, c = e - r * cols;
      const int64_t ox = int64_t(r) * bd.ld + c;
      x[ox] = from_f<TP>(fmaf(decay, to_f<TP>(x[ox]), -step * to_f<TU>(u[int64_t(r) * ud.ldu + c])));
    }
  }
}

// ---------------------------------------------------------------- AdamW
//
// The parameters MuonBP does not orthogonalize (1D parameters and the input
// embedding in the paper's training setup, Appendix B) take AdamW steps with
// global-norm gradient clipping.  One workgroup per segment (a contiguous
// element range of one tensor); VEC: the tensor pointers are 16-byte aligned
// and every segment starts at a multiple of 8 elements, so full 8-element
// chunks are 16-byte accesses (the segment's last partial chunk goes one
// element at a time).

// Workgroup b sums the squares of segments b, b + gridDim.x, ... (a fixed
// assignment, so the result does not depend on scheduling); partials[b].
template <typename TP, bool VEC, bool NT>
__global__ __launch_bounds__(kThreads) void k_adamw_sumsq(const ScalarSeg* __restrict__ segs,
                                                          int n_segs,
                                                          const MatPtrs* __restrict__ ptrs,
                                                          float* __restrict__ partials) {
  float acc = 0.f;
  for (int si = blockIdx.x; si < n_segs; si += gridDim.x) {
    const ScalarSeg sg = segs[si];
    const TP* g = static_cast<const TP*>(ptrs[sg.tensor].grad) + sg.begin;
    const int n = sg.count, nv = VEC ? n >> 3 : 0;
    for (int c0 = threadIdx.x; c0 < nv; c0 += kThreads * kStreamUnroll) {
      Raw8<TP> gr[kStreamUnroll];
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u)
        if (c0 + kThreads * u < nv) gr[u] = load8r<NT>(g + 8 * (c0 + kThreads * u));
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u)
        if (c0 + kThreads * u < nv) {
          float f[8];
          unpack8(gr[u], f);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc = fmaf(f[i], f[i], acc);
        }
    }
    for (int e = 8 * nv + threadIdx.x; e < n; e += kThreads) {
      const float x = to_f<TP>(g[e]);
      acc = fmaf(x, x, acc);
    }
  }
  acc = block_sum(acc);
  if (threadIdx.x == 0) partials[blockIdx.x] = acc;
}

// One workgroup: the global norm from the partial sums (in double, fixed
// order) and the clipping factor.
__global__ __launch_bounds__(kThreads) void k_adamw_clip(const float* __restrict__ partials, int n,
                                                         float max_norm, float* __restrict__ clip) {
  __shared__ double red[kThreads / 64];
  double acc = 0.0;
  for (int i = threadIdx.x; i < n; i += kThreads) acc += partials[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double total = 0.0;
    for (int w = 0; w < kThreads / 64; ++w) total += red[w];
    const double norm = sqrt(total);
    clip[0] = max_norm > 0.f ? float(fmin(1.0, double(max_norm) / (norm + 1e-6))) : 1.f;
    clip[1] = float(norm);
  }
}

// p <- p (1 - lr wd) - lr m_hat / (sqrt(v_hat) + eps) with the moments of
// the clipped gradient (Adam's bias-corrected moments, decoupled decay).
__device__ __forceinline__ void adamw_elem(float& p, float g, float& m, float& v, const AdamwArgs& a) {
  m = fmaf(a.beta1, m, (1.f - a.beta1) * g);
  v = fmaf(a.beta2, v, (1.f - a.beta2) * g * g);
  p = fmaf(p, a.decay, -a.step * (m / fmaf(sqrtf(v), a.inv_sqrt_bc2, a.eps)));
}

// Lion (Chen et al., 2023): c = b1 m + (1 - b1) g; p <- p (1 - lr wd) -
// lr sign(c); m <- b2 m + (1 - b2) g.  sign(0) = 0, and a NaN in c stays NaN.
__device__ __forceinline__ void lion_elem(float& p, float g, float& m, const AdamwArgs& a) {
  const float c = fmaf(a.beta1, m, (1.f - a.beta1) * g);
  const float sg = c > 0.f ? 1.f : (c < 0.f ? -1.f : c * 0.f);
  p = fmaf(p, a.decay, -a.step * sg);
  m = fmaf(a.beta2, m, (1.f - a.beta2) * g);
}

constexpr int kAdamwUnroll = 4;  // chunks of 8 elements in flight per thread

// LION: the Lion update (v is neither read nor written).
template <typename TP, bool VEC, bool NT, bool LION>
__global__ __launch_bounds__(kThreads) void k_adamw(const ScalarSeg* __restrict__ segs,
                                                    const MatPtrs* __restrict__ ptrs,
                                                    float* __restrict__ m, float* __restrict__ v,
                                                    const float* __restrict__ clip, AdamwArgs a) {
  const ScalarSeg sg = segs[blockIdx.x];
  TP* p = static_cast<TP*>(ptrs[sg.tensor].param) + sg.begin;
  const TP* g = static_cast<const TP*>(ptrs[sg.tensor].grad) + sg.begin;
  float* ms = m + sg.state;
  float* vs = LION ? nullptr : v + sg.state;  // Lion: no v arena
  const float c = clip ? clip[0] : 1.f;
  const int n = sg.count, nv = VEC ? n >> 3 : 0;
  for (int c0 = threadIdx.x; c0 < nv; c0 += kThreads * kAdamwUnroll) {
    Raw8<TP> pr[kAdamwUnroll], gr[kAdamwUnroll];
    Raw8<float> mr[kAdamwUnroll], vr[kAdamwUnroll];
#pragma unroll
    for (int u = 0; u < kAdamwUnroll; ++u) {
      const int k = c0 + kThreads * u;
      if (k < nv) {
        pr[u] = load8r<NT>(p + 8 * k);
        gr[u] = load8r<NT>(g + 8 * k);
        mr[u] = load8r<NT>(ms + 8 * k);
        if (!LION) vr[u] = load8r<NT>(vs + 8 * k);
      }
    }
#pragma unroll
    for (int u = 0; u < kAdamwUnroll; ++u) {
      const int k = c0 + kThreads * u;
      if (k < nv) {
        float pf[8], gf[8], mf[8], vf[8];
        unpack8(pr[u], pf);
        unpack8(gr[u], gf);
        unpack8(mr[u], mf);
        if (LION) {
#pragma unroll
          for (int i = 0; i < 8; ++i) lion_elem(pf[i], c * gf[i], mf[i], a);
        } else {
          unpack8(vr[u], vf);
#pragma unroll
          for (int i = 0; i < 8; ++i) adamw_elem(pf[i], c * gf[i], mf[i], vf[i], a);
        }
        store8r<NT>(p + 8 * k, pf);
        store8r<NT>(ms + 8 * k, mf);
        if (!LION) store8r<NT>(vs + 8 * k, vf);
      }
    }
  }
  for (int e = 8 * nv + threadIdx.x; e < n; e += kThreads) {
    float pf = to_f<TP>(p[e]), mf = ms[e];
    if (LION) {
      lion_elem(pf, c * to_f<TP>(g[e]), mf, a);
    } else {
      float vf = vs[e];
      adamw_elem(pf, c * to_f<TP>(g[e]), mf, vf, a);
      vs[e] = vf;
    }
    p[e] = from_f<TP>(pf);
    ms[e] = mf;
  }
}

// ---------------------------------------------------------------- launchers

namespace {
template <typename F>
hipError_t dispatch1(DType a, F&& f) {
  if (a == DType::F32) return f(float{});
  return f(bf16{});
}
}  // namespace

hipError_t launch_momentum(DType grad_t, DType mom_t, bool vec, bool nt, int n_segs,
                           const SegDesc* segs, const BlockDesc* blocks,
                           const MatPtrs* mats, void* mom, float mu, int nesterov,
                           float* partials, hipStream_t s) {
  if (n_segs <= 0) return hipSuccess;
  return dispatch1(grad_t, [&](auto g) {
    return dispatch1(mom_t, [&](auto m) {
      using TG = decltype(g);
      using TM = decltype(m);
      if (vec && nt)
        hipLaunchKernelGGL((k_momentum<TG, TM, true, true>), dim3(n_segs), dim3(kThreads), 0, s,
                           segs, blocks, mats, static_cast<TM*>(mom), mu, nesterov, partials);
      else if (vec)
        hipLaunchKernelGGL((k_momentum<TG, TM, true, false>), dim3(n_segs), dim3(kThreads), 0, s,
                           segs, blocks, mats, static_cast<TM*>(mom), mu, nesterov, partials);
      else
        hipLaunchKernelGGL((k_momentum<TG, TM, false, false>), dim3(n_segs), dim3(kThreads), 0, s,
                           segs, blocks, mats, static_cast<TM*>(mom), mu, nesterov, partials);
      return hipGetLastError();
    });
  });
}

hipError_t launch_check_finite(int n, const float* partials, int* flag, hipStream_t s) {
  hipLaunchKernelGGL(k_check_finite, dim3(1), dim3(kThreads), 0, s, partials, n, flag);
  return hipGetLastError();
}

hipError_t launch_scale(int n_probs, const ScaleDesc* sd, const float* partials, float* scales,
                        float eps, hipStream_t s) {
  if (n_probs <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_scale, dim3(n_probs), dim3(64), 0, s, sd, partials, scales, eps);
  return hipGetLastError();
}

hipError_t launch_pack(DType mom_t, DType grad_t, DType ns_t, bool vec, int n_tiles,
                       const TileRef* tiles, const PackDesc* pd, const MatPtrs* mats,
                       const void* mom, const float* scales, const float* partials, float eps,
                       bool fuse_scale, float mu, int nesterov, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  return dispatch1(mom_t, [&](auto m) {
    return dispatch1(grad_t, [&](auto g) {
      return dispatch1(ns_t, [&](auto n) {
        using TM = decltype(m);
        using TG = decltype(g);
        using TN = decltype(n);
        const int fuse = fuse_scale ? 1 : 0;
        if (vec)
          hipLaunchKernelGGL((k_pack<TM, TG, TN, true>), dim3(n_tiles), dim3(kThreads), 0, s, tiles,
                             pd, mats, static_cast<const TM*>(mom), scales, partials, eps, fuse, mu,
                             nesterov);
        else
          hipLaunchKernelGGL((k_pack<TM, TG, TN, false>), dim3(n_tiles), dim3(kThreads), 0, s, tiles,
                             pd, mats, static_cast<const TM*>(mom), scales, partials, eps, fuse, mu,
                             nesterov);
        return hipGetLastError();
      });
    });
  });
}

hipError_t launch_ns_gemm(DType ns_t, int variant, bool nn, int n_tiles, const GemmDesc* probs,
                          const TileRef* tiles, int nsplit, float* ksum, int* kcount,
                          hipStream_t s, bool long_k) {
  if (nsplit > 1 && (!ksum || !kcount || !gemm_is_dmap(variant))) return hipErrorInvalidValue;
  if (nn && !gemm_is_dmap(variant)) return hipErrorInvalidValue;
  if (n_tiles <= 0) return hipSuccess;
  return dispatch1(ns_t, [&](auto n) {
    using TN = decltype(n);
    switch (variant) {
      case kGemm128x128:
        if (long_k && std::is_same<TN, float>::value)
          hipLaunchKernelGGL((k_ns_gemm<TN, 128, 128, 1, true>), dim3(n_tiles), dim3(kThreads), 0, s,
                             probs, tiles);
        else
          hipLaunchKernelGGL((k_ns_gemm<TN, 128, 128, 1>), dim3(n_tiles), dim3(kThreads), 0, s, probs,
                             tiles);
        break;
      case kGemm256x128:
        hipLaunchKernelGGL((k_ns_gemm<TN, 256, 128, 1>), dim3(n_tiles), dim3(kThreads), 0, s, probs,
                           tiles);
        break;
      case kGemm256x256:
        hipLaunchKernelGGL((k_ns_gemm<TN, 256, 256, 1>), dim3(n_tiles), dim3(kThreads), 0, s, probs,
                           tiles);
        break;
      case kGemm128x128Split2:
        if (long_k && std::is_same<TN, float>::value)
          hipLaunchKernelGGL((k_ns_gemm<TN, 128, 128, 2, true>), dim3(n_tiles), dim3(2 * kThreads), 0,
                             s, probs, tiles);
        else
          hipLaunchKernelGGL((k_ns_gemm<TN, 128, 128, 2>), dim3(n_tiles), dim3(2 * kThreads), 0, s,
                             probs, tiles);
        break;
      case kGemmDmaP128x128:
      case kGemmDmaP256x128:
      case kGemmDmaP256x256:
      case kGemmDmaP192x256:
      case kGemmDmaP256x192:
      case kGemmDmaP192x192:
      case kGemmDmaP256x256W8:
      case kGemmDmaP192x256W8:
      case kGemmDmaP256x192W8:
        if constexpr (std::is_same<TN, bf16>::value) {
#define MUONBP_DMAP(BM_, BN_, WM_, WN_)                                                        \
  if (nn)                                                                                      \
    hipLaunchKernelGGL((k_ns_gemm_dmap<BM_, BN_, true, WM_, WN_>), dim3(n_tiles),              \
                       dim3(64 * WM_ * WN_), 0, s, probs, tiles, nsplit, ksum, kcount);        \
  else                                                                                         \
    hipLaunchKernelGGL((k_ns_gemm_dmap<BM_, BN_, false, WM_, WN_>), dim3(n_tiles),             \
                       dim3(64 * WM_ * WN_), 0, s, probs, tiles, nsplit, ksum, kcount)
          switch (variant) {
            case kGemmDmaP128x128: MUONBP_DMAP(128, 128, 2, 2); break;
            case kGemmDmaP256x128: MUONBP_DMAP(256, 128, 2, 2); break;
            case kGemmDmaP256x256: MUONBP_DMAP(256, 256, 2, 2); break;
            case kGemmDmaP192x256: MUONBP_DMAP(192, 256, 2, 2); break;
            case kGemmDmaP256x192: MUONBP_DMAP(256, 192, 2, 2); break;
            case kGemmDmaP256x256W8: MUONBP_DMAP(256, 256, 2, 4); break;
            case kGemmDmaP192x256W8: MUONBP_DMAP(192, 256, 2, 4); break;
            case kGemmDmaP256x192W8: MUONBP_DMAP(256, 192, 4, 2); break;
            default: MUONBP_DMAP(192, 192, 2, 2); break;
          }
#undef MUONBP_DMAP
          break;
        } else {
          return hipErrorInvalidValue;
        }
      default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
  });
}

hipError_t launch_update(DType param_t, DType ns_t, bool vec, bool nt, int n_segs,
                         const SegDesc* segs,
                         const BlockDesc* blocks, const MatPtrs* mats, const UpdDesc* upd,
                         float eta, float lambda, hipStream_t s) {
  if (n_segs <= 0) return hipSuccess;
  return dispatch1(param_t, [&](auto p) {
    return dispatch1(ns_t, [&](auto n) {
      using TP = decltype(p);
      using TU = decltype(n);
      if (vec && nt)
        hipLaunchKernelGGL((k_update<TP, TU, true, true>), dim3(n_segs), dim3(kThreads), 0, s,
                           segs, blocks, mats, upd, eta, lambda);
      else if (vec)
        hipLaunchKernelGGL((k_update<TP, TU, true, false>), dim3(n_segs), dim3(kThreads), 0, s,
                           segs, blocks, mats, upd, eta, lambda);
      else
        hipLaunchKernelGGL((k_update<TP, TU, false, false>), dim3(n_segs), dim3(kThreads), 0, s,
                           segs, blocks, mats, upd, eta, lambda);
      return hipGetLastError();
    });
  });
}

int adamw_norm_blocks(int n_segs) { return n_segs < kAdamwNormBlocks ? n_segs : kAdamwNormBlocks; }

hipError_t launch_adamw_sumsq(DType param_t, bool vec, bool nt, int n_segs, const ScalarSeg* segs,
                              const MatPtrs* ptrs, float* partials, hipStream_t s) {
  if (n_segs <= 0) return hipSuccess;
  const int nb = adamw_norm_blocks(n_segs);
  return dispatch1(param_t, [&](auto p) {
    using TP = decltype(p);
    if (vec && nt)
      hipLaunchKernelGGL((k_adamw_sumsq<TP, true, true>), dim3(nb), dim3(kThreads), 0, s, segs,
                         n_segs, ptrs, partials);
    else if (vec)
      hipLaunchKernelGGL((k_adamw_sumsq<TP, true, false>), dim3(nb), dim3(kThreads), 0, s, segs,
                         n_segs, ptrs, partials);
    else
      hipLaunchKernelGGL((k_adamw_sumsq<TP, false, false>), dim3(nb), dim3(kThreads), 0, s, segs,
                         n_segs, ptrs, partials);
    return hipGetLastError();
  });
}

hipError_t launch_adamw_clip(const float* partials, int n, float max_norm, float* clip,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_adamw_clip, dim3(1), dim3(kThreads), 0, s, partials, n, max_norm, clip);
  return hipGetLastError();
}

hipError_t launch_adamw(DType param_t, bool vec, bool nt, int n_segs, const ScalarSeg* segs,
                        const MatPtrs* ptrs, float* m, float* v, const float* clip,
                        const AdamwArgs& a, bool lion, hipStream_t s) {
  if (n_segs <= 0) return hipSuccess;
  return dispatch1(param_t, [&](auto p) {
    using TP = decltype(p);
    auto go = [&](auto lion_tag) {
      constexpr bool L = decltype(lion_tag)::value;
      if (vec && nt)
        hipLaunchKernelGGL((k_adamw<TP, true, true, L>), dim3(n_segs), dim3(kThreads), 0, s, segs, ptrs,
                           m, v, clip, a);
      else if (vec)
        hipLaunchKernelGGL((k_adamw<TP, true, false, L>), dim3(n_segs), dim3(kThreads), 0, s, segs,
                           ptrs, m, v, clip, a);
      else
        hipLaunchKernelGGL((k_adamw<TP, false, false, L>), dim3(n_segs), dim3(kThreads), 0, s, segs,
                           ptrs, m, v, clip, a);
      return hipGetLastError();
    };
    return lion ? go(std::true_type{}) : go(std::false_type{});
  });
}

}  // namespace muonbp
