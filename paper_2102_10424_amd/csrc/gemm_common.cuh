// Operand / output views and tile ordering shared by the GEMM kernels.
#pragma once

#include <climits>
#include <cstdint>

#include "gist_internal.h"

namespace gist {

// Device view of an Operand (see gist_internal.h): logical R x K matrix,
// optionally concatenated from two pointers at `split`.
struct OpView {
  const float* p0;
  const float* p1;
  int64_t ld0, ld1, split;

  static OpView from(const Operand& o) {
    return OpView{o.p0, o.p1 ? o.p1 : o.p0, o.ld0, o.p1 ? o.ld1 : o.ld0,
                  o.p1 ? o.split : INT64_MAX};
  }
  // Element (r, k); KMAJ: K contiguous (split along K), else R contiguous
  // (split along R).
  template <bool KMAJ>
  __device__ __forceinline__ float at(int64_t r, int64_t k) const {
    if constexpr (KMAJ) return k < split ? p0[r * ld0 + k] : p1[r * ld1 + (k - split)];
    else return r < split ? p0[k * ld0 + r] : p1[k * ld1 + (r - split)];
  }
  // Four consecutive elements along the contiguous dimension, starting at
  // (r, k); the caller guarantees 16-byte alignment and that the four do
  // not straddle `split`.
  template <bool KMAJ>
  __device__ __forceinline__ float4 at4(int64_t r, int64_t k) const {
    const float* p;
    if constexpr (KMAJ) p = k < split ? p0 + r * ld0 + k : p1 + r * ld1 + (k - split);
    else p = r < split ? p0 + k * ld0 + r : p1 + k * ld1 + (r - split);
    return *reinterpret_cast<const float4*>(p);
  }
  // Two consecutive elements along the contiguous dimension (8-byte aligned,
  // not straddling `split`).
  template <bool KMAJ>
  __device__ __forceinline__ float2 at2(int64_t r, int64_t k) const {
    const float* p;
    if constexpr (KMAJ) p = k < split ? p0 + r * ld0 + k : p1 + r * ld1 + (k - split);
    else p = r < split ? p0 + k * ld0 + r : p1 + k * ld1 + (r - split);
    return *reinterpret_cast<const float2*>(p);
  }
};

// Device view of a GemmOut: optional ReLU, columns >= c_split go to c1,
// optional fused SGD step (C <- fmaf(-lr, product, C)).
struct OutView {
  float* c0;
  float* c1;
  int64_t ldc0, ldc1, c_split;
  int relu;
  int sgd;
  float lr;
  const float* mask;   // store 0 where mask <= 0 (c0 columns only), or null
  int64_t ldm;

  static OutView from(const GemmOut& c) {
    return OutView{c.c0, c.c1, c.ldc0, c.ldc1, c.c_split, c.relu ? 1 : 0, c.sgd ? 1 : 0, c.lr,
                   c.mask, c.ldm};
  }
  template <bool SPLIT>
  __device__ __forceinline__ float* ptr(int64_t row, int64_t col) const {
    return (SPLIT && col >= c_split) ? c1 + row * ldc1 + (col - c_split) : c0 + row * ldc0 + col;
  }
  template <bool SPLIT>
  __device__ __forceinline__ void store(int64_t row, int64_t col, float v) const {
    if (relu) v = fmaxf(v, 0.f);
    if (mask && (!SPLIT || col < c_split) && !(mask[row * ldm + col] > 0.f)) v = 0.f;
    float* p = ptr<SPLIT>(row, col);
    if (sgd) v = fmaf(-lr, v, *p);
    *p = v;
  }
};

// Tile id -> (tile_m, tile_n): column-major in bands of 8 tile rows, so the
// tiles an XCD runs together share B columns and a narrow band of A rows.
__device__ __forceinline__ void tile_coords_banded(int64_t t, int tiles_m, int tiles_n, int& tm,
                                                   int& tn) {
  constexpr int kBand = 8;
  const int band = static_cast<int>(t / (static_cast<int64_t>(kBand) * tiles_n));
  const int rows_in_band = min(kBand, tiles_m - band * kBand);
  const int64_t in_band = t - static_cast<int64_t>(band) * kBand * tiles_n;
  tm = band * kBand + static_cast<int>(in_band % rows_in_band);
  tn = static_cast<int>(in_band / rows_in_band);
}

bool gemm_bf16_packed_eligible(int64_t M, int64_t N, int64_t K);
size_t gemm_bf16_packed_workspace(int64_t M, int64_t N, int64_t K);
gist_status gemm_bf16_packed(hipStream_t st, int64_t M, int64_t N, int64_t K, const Operand& A,
                             const Operand& B, const GemmOut& C, void* ws, size_t ws_bytes);

}  // namespace gist
