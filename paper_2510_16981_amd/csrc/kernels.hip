// HIP kernels of the MuonBP optimizer step for CDNA4 (gfx950, wave64).
//
//  * k_momentum  -- M <- mu M + G (eq. NTR / Algorithm 1), fused with the
//                   per-segment sum of squares of the NS input.
//  * k_scale     -- 1 / (||Y||_F + eps) per orthogonalized unit (Algorithm 2).
//  * k_pack      -- scaled NS input, written row-major and transposed.
//  * k_ns_gemm   -- grouped MFMA GEMM C = alpha X Y^T + beta D used for the
//                   three products of every NS iteration (Algorithm 2):
//                   A = Z Z^T, B = b A + c A A, Z' = a Z + B Z.
//  * k_update    -- X <- X (1 - eta lambda) - eta s U (Algorithm 1).
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace muonbp {

typedef __bf16 bf16;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float f[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
  f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}
__device__ __forceinline__ void store8(bf16* p, const float f[8]) {
  union {
    bf16 h[8];
    uint4 v;
  } u;
#pragma unroll
  for (int i = 0; i < 8; ++i) u.h[i] = bf16(f[i]);
  *reinterpret_cast<uint4*>(p) = u.v;
}
__device__ __forceinline__ void store8(float* p, const float f[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(f[0], f[1], f[2], f[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(f[4], f[5], f[6], f[7]);
}

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

template <typename TG, typename TM, bool VEC>
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
    for (int v = threadIdx.x; v < nv; v += kThreads) {
      const int r = v / vpr;
      const int64_t o = int64_t(r) * bd.ld + ((v - r * vpr) << 3);
      float gf[8], mf[8];
      load8(g + o, gf);
      load8(m + o, mf);
#pragma unroll
      for (int i = 0; i < 8; ++i) mf[i] = fmaf(mu, mf[i], gf[i]);
      store8(m + o, mf);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float mr = rt<TM>(mf[i]);
        const float y = nesterov ? fmaf(mu, mr, gf[i]) : mr;
        acc = fmaf(y, y, acc);
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
  if (threadIdx.x == 0) partials[blockIdx.x] = acc;
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

template <typename TM, typename TG, typename TN>
__global__ __launch_bounds__(kThreads) void k_pack(
    const TileRef* __restrict__ tiles, const PackDesc* __restrict__ pd,
    const MatPtrs* __restrict__ mats, const TM* __restrict__ mom,
    const float* __restrict__ scales, float mu, int nesterov) {
  __shared__ float tile[64][65];
  const TileRef t = tiles[blockIdx.x];
  const PackDesc d = pd[t.prob];
  const int r0 = (t.ij >> 16) * 64, c0 = (t.ij & 0xffff) * 64;
  const float s = scales[t.prob];
  const TM* m = mom + d.mom_off;
  const TG* g = static_cast<const TG*>(mats[d.mat].grad) + d.in_mat_off;
  TN* ds = static_cast<TN*>(d.dst_s);
  TN* dt = static_cast<TN*>(d.dst_t);
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
      ds[int64_t(r) * d.ld_s + c] = from_f<TN>(y);
    }
    tile[lr + 4 * i][lc] = y;
  }
  __syncthreads();
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int c = c0 + lr + 4 * i, r = r0 + lc;
    if (r < d.rows && c < d.cols) dt[int64_t(c) * d.ld_t + r] = from_f<TN>(tile[lc][lr + 4 * i]);
  }
}

// ---------------------------------------------------------------- NS GEMM
//
// Grouped C = alpha X Y^T + beta D over a tile list, both operands row-major
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

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4_t gu32x4_t;

// 16-byte load through the global address space (global_load rather than
// flat_load: flat loads also count against the LDS wait counter, so every
// LDS wait in the K loop would also wait for the prefetch).  The integer
// round trip makes the compiler emit an address-space-1 access.
__device__ __forceinline__ uint4 gld16(const void* p) {
  const u32x4_t v = *(gu32x4_t*)(reinterpret_cast<uintptr_t>(p));
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

// Writes nrows x (8 * nchunk) of one wave's staged fp32 rows to out,
// adding beta * add; `st` row pitch `pitch` floats.  Output row r, chunk c
// of the staged block is element (r0 + r, c0 + 8c) of out; with `transposed`
// the staged value is read at st[(8c + e) * pitch + r].
template <typename T>
__device__ __forceinline__ void store_rows(const float* st, int pitch, int nrows, int nchunk,
                                           T* out, int ldo, const T* add, int lda, float beta,
                                           int r0, int c0, int nr, int nc, bool transposed,
                                           int lane) {
  for (int q = lane; q < nrows * nchunk; q += 64) {
    const int r = q / nchunk, c = (q - r * nchunk) * 8;
    const int gr = r0 + r, gc = c0 + c;
    if (gr >= nr || gc >= nc) continue;
    float f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = transposed ? st[(c + e) * pitch + r] : st[r * pitch + c + e];
    const int64_t oo = int64_t(gr) * ldo + gc, oa = int64_t(gr) * lda + gc;
    if (gc + 8 <= nc) {
      if (add) {
        float a8[8];
        load8(add + oa, a8);
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = fmaf(beta, a8[e], f[e]);
      }
      store8(out + oo, f);
    } else {
      for (int e = 0; e < nc - gc; ++e) {
        float v = f[e];
        if (add) v = fmaf(beta, to_f<T>(add[oa + e]), v);
        out[oo + e] = from_f<T>(v);
      }
    }
  }
}

template <typename T, int BM, int BN>
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
  static constexpr int LDS_EPI = 4 * 32 * ST_PITCH * 4;
  static constexpr int LDS_BYTES = 2 * LDS_STAGE > LDS_EPI ? 2 * LDS_STAGE : LDS_EPI;
};

template <typename T, int BM, int BN>
__global__ __launch_bounds__(kThreads) void k_ns_gemm(const GemmDesc* __restrict__ probs,
                                                      const TileRef* __restrict__ tiles,
                                                      float alpha, float beta, int sym) {
  using G = GemmShape<T, BM, BN>;
  constexpr int EPV = G::EPV, BK = G::BK, TM = G::TM, TN = G::TN, QX = G::QX, QY = G::QY;
  __shared__ __attribute__((aligned(16))) unsigned char lds[G::LDS_BYTES];

  const TileRef t = tiles[blockIdx.x];
  const GemmDesc d = probs[t.prob];
  const int ti = t.ij >> 16, tj = t.ij & 0xffff;
  const int m0 = ti * BM, n0 = tj * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Rows beyond M (N) are clamped to a valid row: they only feed output rows
  // (columns) that are never stored.  Columns at or beyond K are masked to
  // zero in the last K slice, which may straddle K (rows are padded to a
  // multiple of 8 elements, so the 16-byte read stays inside the row).
  const int kc = (tid & 7) * EPV;  // this thread's column inside a K slice
  const T* xrow[QX];
  const T* yrow[QY];
#pragma unroll
  for (int q = 0; q < QX; ++q)
    xrow[q] = static_cast<const T*>(d.X) + int64_t(min(m0 + ((tid + kThreads * q) >> 3), d.M - 1)) * d.ldx;
#pragma unroll
  for (int q = 0; q < QY; ++q)
    yrow[q] = static_cast<const T*>(d.Y) + int64_t(min(n0 + ((tid + kThreads * q) >> 3), d.N - 1)) * d.ldy;
  uint4 rx[QX], ry[QY];
  auto gload = [&](int k0) {
#pragma unroll
    for (int q = 0; q < QX; ++q) rx[q] = gld16(xrow[q] + k0 + kc);
#pragma unroll
    for (int q = 0; q < QY; ++q) ry[q] = gld16(yrow[q] + k0 + kc);
  };
  auto gload_tail = [&](int k0) {
    const int kk = k0 + kc;
    const int nv = max(0, min(d.K - kk, EPV));
    const int o = nv > 0 ? kk : 0;
#pragma unroll
    for (int q = 0; q < QX; ++q) rx[q] = mask_tail<T>(gld16(xrow[q] + o), nv);
#pragma unroll
    for (int q = 0; q < QY; ++q) ry[q] = mask_tail<T>(gld16(yrow[q] + o), nv);
  };
  auto lstore = [&](int buf) {
    unsigned char* base = lds + buf * G::LDS_STAGE;
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

  const int nk = (d.K + BK - 1) / BK;
  if (BK <= d.K) gload(0); else gload_tail(0);
  lstore(0);
  __syncthreads();
  const int xoff = (wm * 32 * TM + (lane & 31)) * kLdsRow;
  const int yoff = G::LDS_X + (wn * 32 * TN + (lane & 31)) * kLdsRow;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      if ((kt + 2) * BK <= d.K) gload((kt + 1) * BK); else gload_tail((kt + 1) * BK);
    }
    const unsigned char* S = lds + buf * G::LDS_STAGE;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int koff = (2 * s + (lane >> 5)) * 16;
      uint4 a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        a[i] = *reinterpret_cast<const uint4*>(S + xoff + i * 32 * kLdsRow + koff);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        b[j] = *reinterpret_cast<const uint4*>(S + yoff + j * 32 * kLdsRow + koff);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = Mfma<T>::step(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue, one MFMA row of the wave's sub-tile at a time.  32x32
  // accumulator layout: lane l holds column l % 32 and, for register v, row
  // 8 (v / 4) + 4 (l / 32) + v % 4.  alpha * acc is staged in a wave-private
  // LDS block (32 rows x 32 TN columns, odd pitch), then written as 16-byte
  // chunks of C rows and, for the transposed copy, of Ct rows, adding
  // beta * D (or beta * Dt) in fp32.
  constexpr int P = G::ST_PITCH;
  float* st = reinterpret_cast<float*>(lds) + wave * 32 * P;
  const bool mirror = d.Ct != nullptr && !(sym && ti == tj);
  const int wr0 = m0 + wm * 32 * TM, wc0 = n0 + wn * 32 * TN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        st[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * P + j * 32 + (lane & 31)] = alpha * acc[i][j][v];
    __syncthreads();
    store_rows<T>(st, P, 32, 4 * TN, static_cast<T*>(d.C), d.ldc, static_cast<const T*>(d.D), d.ldd,
                  beta, wr0 + 32 * i, wc0, d.M, d.N, false, lane);
    if (mirror)
      store_rows<T>(st, P, 32 * TN, 4, static_cast<T*>(d.Ct), d.ldct, static_cast<const T*>(d.Dt),
                    d.lddt, beta, wc0, wr0 + 32 * i, d.N, d.M, true, lane);
    __syncthreads();
  }
}

// ---------------------------------------------------------------- update

template <typename TP, typename TU, bool VEC>
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
    for (int v = threadIdx.x; v < nv; v += kThreads) {
      const int r = v / vpr, c = (v - r * vpr) << 3;
      const int64_t ox = int64_t(r) * bd.ld + c, ou = int64_t(r) * ud.ldu + c;
      float xf[8], uf[8];
      load8(x + ox, xf);
      load8(u + ou, uf);
#pragma unroll
      for (int i = 0; i < 8; ++i) xf[i] = fmaf(decay, xf[i], -step * uf[i]);
      store8(x + ox, xf);
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

// ---------------------------------------------------------------- launchers

namespace {
template <typename F>
hipError_t dispatch1(DType a, F&& f) {
  if (a == DType::F32) return f(float{});
  return f(bf16{});
}
}  // namespace

hipError_t launch_momentum(DType grad_t, DType mom_t, bool vec, int n_segs,
                           const SegDesc* segs, const BlockDesc* blocks,
                           const MatPtrs* mats, void* mom, float mu, int nesterov,
                           float* partials, hipStream_t s) {
  if (n_segs <= 0) return hipSuccess;
  return dispatch1(grad_t, [&](auto g) {
    return dispatch1(mom_t, [&](auto m) {
      using TG = decltype(g);
      using TM = decltype(m);
      if (vec)
        hipLaunchKernelGGL((k_momentum<TG, TM, true>), dim3(n_segs), dim3(kThreads), 0, s, segs,
                           blocks, mats, static_cast<TM*>(mom), mu, nesterov, partials);
      else
        hipLaunchKernelGGL((k_momentum<TG, TM, false>), dim3(n_segs), dim3(kThreads), 0, s, segs,
                           blocks, mats, static_cast<TM*>(mom), mu, nesterov, partials);
      return hipGetLastError();
    });
  });
}

hipError_t launch_scale(int n_probs, const ScaleDesc* sd, const float* partials, float* scales,
                        float eps, hipStream_t s) {
  if (n_probs <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_scale, dim3(n_probs), dim3(64), 0, s, sd, partials, scales, eps);
  return hipGetLastError();
}

hipError_t launch_pack(DType mom_t, DType grad_t, DType ns_t, int n_tiles, const TileRef* tiles,
                       const PackDesc* pd, const MatPtrs* mats, const void* mom,
                       const float* scales, float mu, int nesterov, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  return dispatch1(mom_t, [&](auto m) {
    return dispatch1(grad_t, [&](auto g) {
      return dispatch1(ns_t, [&](auto n) {
        using TM = decltype(m);
        using TG = decltype(g);
        using TN = decltype(n);
        hipLaunchKernelGGL((k_pack<TM, TG, TN>), dim3(n_tiles), dim3(kThreads), 0, s, tiles, pd,
                           mats, static_cast<const TM*>(mom), scales, mu, nesterov);
        return hipGetLastError();
      });
    });
  });
}

hipError_t launch_ns_gemm(DType ns_t, int variant, int n_tiles, const GemmDesc* probs,
                          const TileRef* tiles, float alpha, float beta, int sym, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  return dispatch1(ns_t, [&](auto n) {
    using TN = decltype(n);
    switch (variant) {
      case kGemm128x128:
        hipLaunchKernelGGL((k_ns_gemm<TN, 128, 128>), dim3(n_tiles), dim3(kThreads), 0, s, probs,
                           tiles, alpha, beta, sym);
        break;
      case kGemm256x128:
        hipLaunchKernelGGL((k_ns_gemm<TN, 256, 128>), dim3(n_tiles), dim3(kThreads), 0, s, probs,
                           tiles, alpha, beta, sym);
        break;
      case kGemm256x256:
        hipLaunchKernelGGL((k_ns_gemm<TN, 256, 256>), dim3(n_tiles), dim3(kThreads), 0, s, probs,
                           tiles, alpha, beta, sym);
        break;
      default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
  });
}

hipError_t launch_update(DType param_t, DType ns_t, bool vec, int n_segs, const SegDesc* segs,
                         const BlockDesc* blocks, const MatPtrs* mats, const UpdDesc* upd,
                         float eta, float lambda, hipStream_t s) {
  if (n_segs <= 0) return hipSuccess;
  return dispatch1(param_t, [&](auto p) {
    return dispatch1(ns_t, [&](auto n) {
      using TP = decltype(p);
      using TU = decltype(n);
      if (vec)
        hipLaunchKernelGGL((k_update<TP, TU, true>), dim3(n_segs), dim3(kThreads), 0, s, segs,
                           blocks, mats, upd, eta, lambda);
      else
        hipLaunchKernelGGL((k_update<TP, TU, false>), dim3(n_segs), dim3(kThreads), 0, s, segs,
                           blocks, mats, upd, eta, lambda);
      return hipGetLastError();
    });
  });
}

}  // namespace muonbp
