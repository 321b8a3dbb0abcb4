// CSR aggregation Y = Abar X (+ Add) (ReLU), the sparse half of eq. (2).
//
// One row of Abar is handled by a group of LPR lanes of a wave (LPR = 64 for
// wide features, fewer for narrow ones, so a wave covers 64 / LPR rows);
// each lane owns VEC consecutive feature columns and walks the row's
// nonzeros, so every nonzero costs one coalesced gather of LPR * VEC floats
// of X.  The row's (col, val) pairs are read cooperatively, one per lane, and
// broadcast within the lane group, so each nonzero's index is loaded once
// per group instead of once per lane.  Features wider than 64 * VEC are split
// into column tiles.  Blocks are ordered XCD-major, column tile major: each
// XCD's L2 sees a contiguous range of rows of one column slab at a time
// (block-ordered graphs keep neighbours close).
// No atomics: every output element is written by exactly one lane, and the
// nonzeros of a row are summed in storage order, so results are bitwise
// reproducible.

#include <cstdio>

#include "common.cuh"
#include "gist_internal.h"

namespace gist {

namespace {

template <int VEC>
struct VecT;
template <>
struct VecT<1> { using T = float; };
template <>
struct VecT<2> { using T = float2; };
template <>
struct VecT<4> { using T = float4; };

template <int VEC>
__device__ __forceinline__ void load_vec(const float* p, float (&x)[VEC]) {
  using T = typename VecT<VEC>::T;
  T v = *reinterpret_cast<const T*>(p);
  if constexpr (VEC == 1) {
    x[0] = v;
  } else if constexpr (VEC == 2) {
    x[0] = v.x; x[1] = v.y;
  } else {
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float* p, const float (&x)[VEC]) {
  using T = typename VecT<VEC>::T;
  T v;
  if constexpr (VEC == 1) {
    v = x[0];
  } else if constexpr (VEC == 2) {
    v.x = x[0]; v.y = x[1];
  } else {
    v.x = x[0]; v.y = x[1]; v.z = x[2]; v.w = x[3];
  }
  *reinterpret_cast<T*>(p) = v;
}

constexpr int kWaves = 4;  // waves per block

template <int VEC, int LPR>
__global__ __launch_bounds__(256) void spmm_kernel(
    int n, const int* __restrict__ rowptr, const int* __restrict__ col,
    const float* __restrict__ val, const float* __restrict__ X, int64_t ldx, int width,
    float* Y, int64_t ldy, const float* add, int64_t ld_add, int relu, int col_tiles,
    int64_t nblocks, const float* mask, int64_t ldm) {
  constexpr int RPW = 64 / LPR;  // rows per wave
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = lane / LPR;       // row slot inside the wave
  const int gl = lane % LPR;        // lane inside the row group
  const int64_t logical = xcd_remap(blockIdx.x, nblocks);
  // column tile major: an XCD's contiguous range of blocks covers all rows
  // of one or a few column slabs, whose gathered rows then fit its L2
  const int64_t rblocks = nblocks / col_tiles;
  const int ctile = static_cast<int>(logical / rblocks);
  const int64_t rblock = logical - static_cast<int64_t>(ctile) * rblocks;
  const int64_t row = (rblock * kWaves + wave) * RPW + grp;
  const int c0 = ctile * (LPR * VEC) + gl * VEC;
  const bool active = row < n && c0 < width;

  int e0 = 0, e1 = 0;
  if (row < n) {
    e0 = rowptr[row];
    e1 = rowptr[row + 1];
  }
  // The epilogue's Add and mask values load before the row's gathers, so
  // their latency overlaps them (row and column clamped into the matrix:
  // every load is in bounds; an inactive lane's values are never stored).
  float a[VEC], mv[VEC];
  {
    const int64_t rr = min(row, static_cast<int64_t>(n) - 1);
    const int cc = min(c0, width - VEC);
    if (add) load_vec<VEC>(add + rr * ld_add + cc, a);
    if (mask) load_vec<VEC>(mask + rr * ldm + cc, mv);
  }
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;

  // Walk the row in windows of LPR nonzeros: lane gl of the group loads
  // nonzero (base + gl), then the group reads them back by shuffle.
  for (int base = e0; base < e1; base += LPR) {
    const int cnt = min(LPR, e1 - base);
    int my_c = 0;
    float my_v = 0.f;
    if (gl < cnt) {
      my_c = col[base + gl];
      my_v = val[base + gl];
    }
    int j = 0;
    for (; j + 4 <= cnt; j += 4) {
      int cj[4];
      float vj[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        cj[u] = __shfl(my_c, grp * LPR + j + u, 64);
        vj[u] = __shfl(my_v, grp * LPR + j + u, 64);
      }
      if (active) {
        float x[4][VEC];
#pragma unroll
        for (int u = 0; u < 4; ++u) load_vec<VEC>(X + static_cast<int64_t>(cj[u]) * ldx + c0, x[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[v] = fmaf(vj[u], x[u][v], acc[v]);
      }
    }
    for (; j < cnt; ++j) {
      const int cj = __shfl(my_c, grp * LPR + j, 64);
      const float vj = __shfl(my_v, grp * LPR + j, 64);
      if (active) {
        float x[VEC];
        load_vec<VEC>(X + static_cast<int64_t>(cj) * ldx + c0, x);
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[v] = fmaf(vj, x[v], acc[v]);
      }
    }
  }
  if (!active) return;
  if (add) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] += a[v];
  }
  if (relu) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = fmaxf(acc[v], 0.f);
  }
  if (mask) {   // the ReLU derivative of the layer whose output is `mask`
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = mv[v] > 0.f ? acc[v] : 0.f;
  }
  store_vec<VEC>(Y + row * ldy + c0, acc);
}

// Wide rows (64 lanes per row): the row index is wave-uniform, so each
// nonzero's (col, val) is broadcast with readlane into scalar registers and
// the gather address is a scalar base plus the lane's column offset; eight
// gathers are kept in flight per wave.
template <int VEC>
__global__ __launch_bounds__(256) void spmm_wide_kernel(
    int n, const int* __restrict__ rowptr, const int* __restrict__ col,
    const float* __restrict__ val, const float* __restrict__ X, int64_t ldx, int width,
    float* Y, int64_t ldy, const float* add, int64_t ld_add, int relu, int col_tiles,
    int64_t nblocks, const float* mask, int64_t ldm) {
  constexpr int kUnroll = 8;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t logical = xcd_remap(blockIdx.x, nblocks);
  // column tile major: an XCD's contiguous range of blocks covers all rows
  // of one or a few column slabs, whose gathered rows then fit its L2
  const int64_t rblocks = nblocks / col_tiles;
  const int ctile = static_cast<int>(logical / rblocks);
  const int64_t rblock = logical - static_cast<int64_t>(ctile) * rblocks;
  const int64_t row = rblock * kWaves + wave;
  if (row >= n) return;
  const int c0 = ctile * (64 * VEC) + lane * VEC;
  const bool active = c0 < width;
  const int e0 = rowptr[row], e1 = rowptr[row + 1];
  // Add and mask values load before the gathers (column clamped into the
  // row: every load is in bounds; an inactive lane's values are never stored)
  float a[VEC], mv[VEC];
  {
    const int cc = min(c0, width - VEC);
    if (add) load_vec<VEC>(add + row * ld_add + cc, a);
    if (mask) load_vec<VEC>(mask + row * ldm + cc, mv);
  }
  const float* Xc = X + c0;
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  for (int base = e0; base < e1; base += 64) {
    const int cnt = min(64, e1 - base);
    int my_c = 0;
    float my_v = 0.f;
    if (lane < cnt) {
      my_c = col[base + lane];
      my_v = val[base + lane];
    }
    int j = 0;
    for (; j + kUnroll <= cnt; j += kUnroll) {
      int cj[kUnroll];
      float vj[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        cj[u] = __builtin_amdgcn_readlane(my_c, j + u);
        vj[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), j + u));
      }
      if (active) {
        float x[kUnroll][VEC];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) load_vec<VEC>(Xc + static_cast<int64_t>(cj[u]) * ldx, x[u]);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[v] = fmaf(vj[u], x[u][v], acc[v]);
      }
    }
    for (; j < cnt; ++j) {
      const int cj = __builtin_amdgcn_readlane(my_c, j);
      const float vj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), j));
      if (active) {
        float x[VEC];
        load_vec<VEC>(Xc + static_cast<int64_t>(cj) * ldx, x);
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[v] = fmaf(vj, x[v], acc[v]);
      }
    }
  }
  if (!active) return;
  if (add) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] += a[v];
  }
  if (relu) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = fmaxf(acc[v], 0.f);
  }
  if (mask) {   // the ReLU derivative of the layer whose output is `mask`
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = mv[v] > 0.f ? acc[v] : 0.f;
  }
  store_vec<VEC>(Y + row * ldy + c0, acc);
}

template <int VEC, int LPR>
gist_status launch(hipStream_t st, int64_t n, int64_t nnz, const int32_t* rowptr, const int32_t* col,
                   const float* val, const float* X, int64_t ldx, int width, float* Y,
                   int64_t ldy, const float* add, int64_t ld_add, bool relu, const float* mask,
                   int64_t ldm) {
  constexpr int RPW = 64 / LPR;
  const int col_tiles = (width + LPR * VEC - 1) / (LPR * VEC);
  const int64_t rblocks = (n + kWaves * RPW - 1) / (kWaves * RPW);
  const int64_t nblocks = rblocks * col_tiles;
  if (nblocks > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "spmm: grid too large");
  char name[32];
  snprintf(name, sizeof(name), "spmm_v%d_l%d", VEC, LPR);
  // algorithmic bytes: rowptr, (col, val) per nonzero, X read once, Y written
  // once (and Add read once)
  const double bytes = 4.0 * (n + 1) + 8.0 * static_cast<double>(nnz) +
                       4.0 * static_cast<double>(n) * width * (2.0 + (add ? 1.0 : 0.0) +
                                                                (mask ? 1.0 : 0.0));
  ProfScope ps(st, name, 2.0 * static_cast<double>(nnz) * width, bytes);
  if constexpr (LPR == 64) {
    hipLaunchKernelGGL((spmm_wide_kernel<VEC>), dim3(static_cast<unsigned>(nblocks)), dim3(256),
                       0, st, static_cast<int>(n), rowptr, col, val, X, ldx, width, Y, ldy, add,
                       ld_add, relu ? 1 : 0, col_tiles, nblocks, mask, ldm);
  } else {
    hipLaunchKernelGGL((spmm_kernel<VEC, LPR>), dim3(static_cast<unsigned>(nblocks)), dim3(256),
                       0, st, static_cast<int>(n), rowptr, col, val, X, ldx, width, Y, ldy, add,
                       ld_add, relu ? 1 : 0, col_tiles, nblocks, mask, ldm);
  }
  return check_launch("spmm");
}

template <int VEC>
gist_status launch_vec(hipStream_t st, int64_t n, int64_t nnz, const int32_t* rowptr, const int32_t* col,
                       const float* val, const float* X, int64_t ldx, int width, float* Y,
                       int64_t ldy, const float* add, int64_t ld_add, bool relu,
                       const float* mask, int64_t ldm) {
  // lanes per row: the smallest power of two covering the row, at most 64
  const int chunks = (width + VEC - 1) / VEC;
  if (chunks > 32)
    return launch<VEC, 64>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add, ld_add,
                               relu, mask, ldm);
  if (chunks > 16)
    return launch<VEC, 32>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add, ld_add,
                               relu, mask, ldm);
  if (chunks > 8)
    return launch<VEC, 16>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add, ld_add,
                               relu, mask, ldm);
  if (chunks > 4)
    return launch<VEC, 8>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add, ld_add,
                               relu, mask, ldm);
  return launch<VEC, 4>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add, ld_add,
                             relu, mask, ldm);
}

}  // namespace

gist_status spmm(hipStream_t st, int64_t n, int64_t nnz, const int32_t* rowptr, const int32_t* col,
                 const float* val, const float* X, int64_t ldx, int width, float* Y,
                 int64_t ldy, const float* add, int64_t ld_add, bool relu, const float* mask,
                 int64_t ldm) {
  if (n <= 0 || width <= 0) return GIST_OK;
  const bool v4 = width % 4 == 0 && ldx % 4 == 0 && ldy % 4 == 0 && aligned16(X) &&
                  aligned16(Y) && (!add || (ld_add % 4 == 0 && aligned16(add))) &&
                  (!mask || (ldm % 4 == 0 && aligned16(mask)));
  const bool v2 = width % 2 == 0 && ldx % 2 == 0 && ldy % 2 == 0 && aligned8(X) &&
                  aligned8(Y) && (!add || (ld_add % 2 == 0 && aligned8(add))) &&
                  (!mask || (ldm % 2 == 0 && aligned8(mask)));
  // Prefer the widest vector that still fills a 64-lane row; a row that
  // would need fewer than 33 lanes at 16 bytes uses 8-byte vectors instead
  // when that gives a full-wave row (e.g. width 100: 50 lanes x 2 floats).
  if (v4 && (width > 128 || width <= 64))
    return launch_vec<4>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add,
                         ld_add, relu, mask, ldm);
  if (v2) return launch_vec<2>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add,
                         ld_add, relu, mask, ldm);
  if (v4) return launch_vec<4>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add,
                         ld_add, relu, mask, ldm);
  return launch_vec<1>(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add,
                         ld_add, relu, mask, ldm);
}

}  // namespace gist
