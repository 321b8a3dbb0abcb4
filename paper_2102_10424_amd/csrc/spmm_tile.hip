// Aggregation Y = Abar X (+ Add) (ReLU) for a cluster mini-batch, on the
// matrix cores -- the sparse half of eq. (2) when Abar is nearly block
// diagonal.
//
// A cluster mini-batch over block-contiguous node ids (Section 2.2: a batch
// is a union of clusters) has almost every entry of row r inside its own
// cluster's block around the diagonal.  The gather kernel (spmm.hip) moves
// one X row from cache to the CUs per entry -- nnz * width * 4 bytes, twenty
// times the algorithmic bytes at the c5 shape -- so it is bound by cache
// bandwidth, not HBM.  Here a workgroup takes 32 rows and one 256-column
// slab of X, four workgroups per CU:
//
//   1. window: [clo, clo + K) spans the columns of the tile's entries that
//      lie within kNear of their row's diagonal, K <= kMaxK, rounded up to
//      the MFMA depth and kept inside the matrix;
//   2. the entries inside the window are expanded into a dense 32 x K tile
//      in LDS, each value split into two bf16 halves, hi = bf16(v) and
//      lo = bf16(v - hi) (both rounded to nearest even);
//   3. each wave streams its 64 columns of X rows clo .. clo + K - 1 from
//      memory straight into MFMA operand registers (a lane holds 8
//      consecutive rows of one column), three 16-row steps ahead, splits them
//      the same way and multiplies on v_mfma_f32_32x32x16_bf16 with fp32
//      accumulation: hi*hi + hi*lo + lo*hi.  The dense tile is the only LDS
//      operand and read-only here, so the loop has no barrier and the waves
//      run independently.  Each X row of the window is read once per 32
//      output rows instead of once per entry;
//   steps 1-3 run a second time, over a second window, for the near-diagonal
//      entries the first could not hold (rows straddling two clusters);
//   4. the entries outside both windows (edges between clusters) are listed
//      per wave, gathered one X row each and added in storage order; then
//      Add, ReLU, the ReLU derivative of the layer below, and the store.
//
// Accuracy: a value's hi + lo carries 16 significant bits, so each split
// operand is within 2^-17 of its value, and the dropped lo*lo term is below
// 2^-16 of the product: every product enters the fp32 sum with a relative
// error below 2^-15 (3.1e-5).  The sum order is fixed (the MFMA k order of
// the first window, then of the second, then the remaining entries in
// storage order): results are deterministic.  Correct for any matrix and
// finite X; fast when most entries sit near the diagonal.

#include <climits>
#include <cstdio>

#include "common.cuh"
#include "gist_internal.h"

namespace gist {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned uint4v __attribute__((ext_vector_type(4)));
typedef unsigned short ushort8 __attribute__((ext_vector_type(8)));

constexpr int kRows = 32;          // output rows per workgroup (the MFMA's M)
constexpr int kCols = 256;         // output columns per workgroup: 4 waves x 64
constexpr int kMaxK = 288;         // widest dense window (a multiple of kKs)
constexpr int kNear = 192;         // an entry within this of its row's diagonal sets the window
constexpr int kKs = 16;            // window rows per step (the MFMA's K)
constexpr int kDepth = 3;          // X steps in flight ahead of the one multiplied
constexpr int kALd = kMaxK + 8;    // bf16 per row of the dense tile (16 B pad)
constexpr int kBlocksPerCU = 4;    // resident workgroups per CU (LDS and registers sized for it)
constexpr int kYLd = kCols + 4;    // floats per row of the result tile
constexpr int kChunk = 8;          // 64-entry chunks a wave loads at once
constexpr int kBatch = 16;         // outside-window entries gathered at once
constexpr int kList = 64;          // outside-window entries a wave lists before gathering


__device__ __forceinline__ unsigned short bf16_bits(float f) {
  return __builtin_bit_cast(unsigned short, static_cast<__bf16>(f));
}
__device__ __forceinline__ float bf16_value(unsigned short h) {
  return __uint_as_float(static_cast<unsigned>(h) << 16);
}
// Two values to packed bf16 (a in the low half), rounded to nearest even.
__device__ __forceinline__ unsigned bf16_pair(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector((float2v){a, b}, bf16x2));
}
// Split 8 values into bf16 halves hi = bf16(v), lo = bf16(v - hi), packed as
// MFMA operands (element i in half i of the fragment).
__device__ __forceinline__ void split8(const float (&v)[8], bf16x8& hi, bf16x8& lo) {
  uint4v h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const unsigned hp = bf16_pair(v[2 * i], v[2 * i + 1]);
    h[i] = hp;
    l[i] = bf16_pair(v[2 * i] - __uint_as_float(hp << 16),
                     v[2 * i + 1] - __uint_as_float(hp & 0xffff0000u));
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

// Wave-uniform row (relative to the wave's first row) of entry e, given the
// wave's row pointers rp[0..8].
__device__ __forceinline__ int row_of(int e, const int (&rp)[9]) {
  int rl = 0;
#pragma unroll
  for (int i = 1; i < 8; ++i) rl += e >= rp[i] ? 1 : 0;
  return rl;
}

__global__ __launch_bounds__(256, kBlocksPerCU) void spmm_tile_kernel(
    int n, int n_in, const int* __restrict__ rowptr, const int* __restrict__ col,
    const float* __restrict__ val, const float* __restrict__ X, int64_t ldx, int width,
    float* Y, int64_t ldy, const float* add, int64_t ld_add, int relu, int tiles,
    int64_t nblocks, const float* mask, int64_t ldm, int vec) {
  // dense tile (hi, lo), later the fp32 result tile
  __shared__ __attribute__((aligned(16))) unsigned short Atile[2 * kRows * kALd];
  __shared__ int red[8];
  static_assert(sizeof(float) * kRows * kYLd + 4 * sizeof(int) * 3 * kList <=
                    sizeof(unsigned short) * 2 * kRows * kALd,
                "result tile and outside-entry lists must fit in the dense tile's space");
  // steps run kDepth at a time: the padded steps stay inside the zeroed tile
  static_assert(kMaxK % (kKs * kDepth) == 0 && kALd % 8 == 0, "tile layout");

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int li = lane & 31, lh = lane >> 5;
  const int64_t logical = xcd_remap(blockIdx.x, nblocks);
  const int slab = static_cast<int>(logical / tiles);
  const int tile = static_cast<int>(logical - static_cast<int64_t>(slab) * tiles);
  const int r0 = tile * kRows;
  const int cs = slab * kCols;
  const int rw = r0 + 8 * wave;   // this wave's first row

  // this wave's rows rw .. rw + 7 and their entries [rp[0], rp[8])
  int rp[9];
#pragma unroll
  for (int i = 0; i <= 8; ++i) rp[i] = rowptr[min(rw + i, n)];
  // When the wave's entries fit in kChunk chunks of 64 they stay in
  // registers for all three passes; longer rows (hubs) are re-read per pass.
  const bool fit = rp[8] - rp[0] <= 64 * kChunk;
  int cc[kChunk];
  float vv[kChunk];
  auto load_chunks = [&](int base) {
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const int e = base + 64 * u + lane;
      cc[u] = e < rp[8] ? col[e] : INT_MIN / 2;
      vv[u] = e < rp[8] ? val[e] : 0.f;
    }
  };
  if (fit) load_chunks(rp[0]);

  auto zero_tile = [&]() {
    uint4v* z = reinterpret_cast<uint4v*>(Atile);
    constexpr int units = 2 * kRows * kALd / 8;
    for (int u = t; u < units; u += 256) z[u] = uint4v{0u, 0u, 0u, 0u};
  };
  // pass 0 zeroes the dense tile while the entries arrive
  zero_tile();

  // X operand: lane (li, lh) of this wave holds window rows 16 j + 8 lh .. + 7
  // of columns c0 + li and c0 + 32 + li.  Columns past the matrix read its
  // last column (their results are never stored) and steps past the window
  // re-read its last step (multiplied by the tile's zero columns), so every
  // load is unconditional and in bounds: one uniform 64-bit base per step and
  // 32-bit lane offsets, no address selects (loads behind branches or
  // selects would make the compiler drain them before each step).
  const int c0 = cs + wave * 64 + li;
  const int ld4 = static_cast<int>(ldx * 4);
  const unsigned off0 = static_cast<unsigned>(8 * lh * ld4 + 4 * min(c0, width - 1));
  const unsigned off1 = static_cast<unsigned>(8 * lh * ld4 + 4 * min(c0 + 32, width - 1));
  float xr[kDepth][2][8];
  floatx16 acc[2];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;

  // Up to two windows, each a pass of steps 1-3: the first spans the
  // entries near their row's diagonal, the second those of them outside the
  // first (a tile whose rows straddle two clusters needs about twice kMaxK
  // columns; two passes keep the tile, and so the workgroups per CU, at one
  // window's size).  Window p is [lo_p, lo_p + kw_p); an entry belongs to
  // the first window that holds it, or to step 4.
  int lo0 = 0, kw0 = 0, lo1 = 0, kw1 = 0;
  for (int pass = 0; pass < 2; ++pass) {
    // ---- 1. window: columns of the near entries no earlier window holds
    int cmin = INT_MAX, cmax = -1;
    for (int base = rp[0]; base < rp[8]; base += 64 * kChunk) {
      if (!fit) load_chunks(base);
#pragma unroll
      for (int u = 0; u < kChunk; ++u) {
        const int e = base + 64 * u + lane;
        if (e < rp[8]) {
          const int r = rw + row_of(e, rp);
          const bool fresh =
              static_cast<unsigned>(cc[u] - lo0) >= static_cast<unsigned>(kw0);
          if (cc[u] >= r - kNear && cc[u] <= r + kNear && fresh) {
            cmin = min(cmin, cc[u]);
            cmax = max(cmax, cc[u]);
          }
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      cmin = min(cmin, __shfl_xor(cmin, o, 64));
      cmax = max(cmax, __shfl_xor(cmax, o, 64));
    }
    if (lane == 0) {
      red[wave] = cmin;
      red[4 + wave] = cmax;
    }
    // (pass 1: also every wave is past pass 0's reads of the dense tile)
    __syncthreads();
    cmin = min(min(red[0], red[1]), min(red[2], red[3]));
    cmax = max(max(red[4], red[5]), max(red[6], red[7]));
    // The window [clo, clo + K) lies inside the matrix's columns, K a
    // multiple of kKs (shifted left from cmin where it would pass n_in,
    // which keeps [cmin, cmax] inside it unless K was capped).  Every
    // window row is then a real row of X.
    int clo = 0, K = 0;
    if (cmax >= cmin) {
      K = min(min(kMaxK, (cmax - cmin + kKs) / kKs * kKs), n_in / kKs * kKs);
      clo = min(cmin, n_in - K);
    }
    clo = __builtin_amdgcn_readfirstlane(clo);
    K = __builtin_amdgcn_readfirstlane(K);
    const int nk = K / kKs;
    if (nk == 0) break;
    if (pass == 0) {
      lo0 = clo;
      kw0 = K;
    } else {
      lo1 = clo;
      kw1 = K;
    }

    auto gload = [&](float (&dst)[2][8], int j) {
      const int jj = min(j, nk - 1);
      const char* base =
          reinterpret_cast<const char*>(X + static_cast<int64_t>(clo + jj * kKs) * ldx);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        dst[0][i] = *reinterpret_cast<const float*>(base + i * ld4 + off0);
        dst[1][i] = *reinterpret_cast<const float*>(base + i * ld4 + off1);
      }
    };
    // the first steps load while the dense tile is built
#pragma unroll
    for (int p = 0; p < kDepth; ++p) gload(xr[p], p);
    if (pass > 0) {
      zero_tile();
      __syncthreads();
    }

    // ---- 2. this window's entries as a dense 32 x K tile (bf16 hi, lo)
    for (int base = rp[0]; base < rp[8]; base += 64 * kChunk) {
      if (!fit) load_chunks(base);
#pragma unroll
      for (int u = 0; u < kChunk; ++u) {
        const int e = base + 64 * u + lane;
        const unsigned k = static_cast<unsigned>(cc[u] - clo);
        const bool fresh =
            pass == 0 || static_cast<unsigned>(cc[u] - lo0) >= static_cast<unsigned>(kw0);
        if (e < rp[8] && k < static_cast<unsigned>(K) && fresh) {
          const int rl = 8 * wave + row_of(e, rp);
          const unsigned short hi = bf16_bits(vv[u]);
          Atile[rl * kALd + k] = hi;
          Atile[(kRows + rl) * kALd + k] = bf16_bits(vv[u] - bf16_value(hi));
        }
      }
    }
    __syncthreads();

    // ---- 3. Y_tile += A_tile X[clo .. clo + K) on the matrix cores, no barriers
    auto mfma = [&](const float (&src)[2][8], int j) {
      // A fragment: tile row li, window columns 16 j + 8 lh .. + 7
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(Atile + li * kALd + j * kKs + 8 * lh);
      const bf16x8 al =
          *reinterpret_cast<const bf16x8*>(Atile + (kRows + li) * kALd + j * kKs + 8 * lh);
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        bf16x8 bh, bl;
        split8(src[b], bh, bl);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc[b], 0, 0, 0);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc[b], 0, 0, 0);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc[b], 0, 0, 0);
      }
    };
    // steps nk .. (padded to a multiple of kDepth) multiply the tile's zero
    // columns with the window's last rows
    for (int j0 = 0; j0 < nk; j0 += kDepth) {
#pragma unroll
      for (int p = 0; p < kDepth; ++p) {
        mfma(xr[p], j0 + p);
        gload(xr[p], j0 + p + kDepth);
      }
    }
  }
  __syncthreads();   // every wave is past its last read of the dense tile

  // the result tile takes the dense tile's space
  float* Ys = reinterpret_cast<float*>(Atile);
  // acc[b] register r of lane l: tile row 8 (r / 4) + 4 (l / 32) + r % 4,
  // column wave 64 + 32 b + l % 32
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      Ys[(8 * (r / 4) + 4 * lh + (r % 4)) * kYLd + wave * 64 + 32 * b + li] = acc[b][r];
  __syncthreads();

  // ---- 4. entries outside both windows, in storage order, then the store.
  // This wave owns tile rows 8 wave .. + 7; lane owns columns cs + lane + 64 q.
  // The wave's outside entries are listed in LDS (behind the result tile)
  // in storage order, up to kList at a time, and their X rows gathered
  // kBatch at a time: a wave with a few outside entries in each 64-entry
  // chunk then waits once per kBatch entries, not once per chunk.
  int* lst_c = reinterpret_cast<int*>(Atile) + kRows * kYLd + wave * 3 * kList;
  int* lst_r = lst_c + kList;
  float* lst_v = reinterpret_cast<float*>(lst_r + kList);
  const int cl0 = min(cs + lane, width - 1), cl1 = min(cs + lane + 64, width - 1);
  const int cl2 = min(cs + lane + 128, width - 1), cl3 = min(cs + lane + 192, width - 1);
  int cnt = 0;
  auto flush = [&]() {
    for (int q0 = 0; q0 < cnt; q0 += kBatch) {
      const int nb = min(kBatch, cnt - q0);
      int ec[kBatch], er[kBatch];
      float ev[kBatch];
#pragma unroll
      for (int q = 0; q < kBatch; ++q) {
        const int i = min(q0 + q, cnt - 1);   // past the batch: a listed entry, not added
        ec[q] = __builtin_amdgcn_readfirstlane(lst_c[i]);
        er[q] = __builtin_amdgcn_readfirstlane(lst_r[i]);
        ev[q] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(lst_v[i])));
      }
      // every load in bounds and unconditional (columns past the matrix read
      // its last column and are never stored)
      float xv[kBatch][4];
#pragma unroll
      for (int q = 0; q < kBatch; ++q) {
        const float* xrow = X + static_cast<int64_t>(ec[q]) * ldx;
        xv[q][0] = xrow[cl0];
        xv[q][1] = xrow[cl1];
        xv[q][2] = xrow[cl2];
        xv[q][3] = xrow[cl3];
      }
#pragma unroll
      for (int q = 0; q < kBatch; ++q) {
        if (q < nb) {
          float* yrow = Ys + (8 * wave + er[q]) * kYLd + lane;
#pragma unroll
          for (int p = 0; p < 4; ++p) yrow[64 * p] = fmaf(ev[q], xv[q][p], yrow[64 * p]);
        }
      }
    }
    cnt = 0;
  };
  for (int base = rp[0]; base < rp[8]; base += 64 * kChunk) {
    if (!fit) load_chunks(base);
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const int e = base + 64 * u + lane;
      const bool out = e < rp[8] &&
                       static_cast<unsigned>(cc[u] - lo0) >= static_cast<unsigned>(kw0) &&
                       static_cast<unsigned>(cc[u] - lo1) >= static_cast<unsigned>(kw1);
      const uint64_t m = __ballot(out);
      const int pc = __builtin_popcountll(m);
      if (pc == 0) continue;
      if (cnt + pc > kList) flush();
      if (out) {
        const int i = cnt + __builtin_amdgcn_mbcnt_hi(static_cast<unsigned>(m >> 32),
                                                      __builtin_amdgcn_mbcnt_lo(static_cast<unsigned>(m), 0u));
        lst_c[i] = cc[u];
        lst_r[i] = row_of(e, rp);
        lst_v[i] = vv[u];
      }
      cnt += pc;
    }
  }
  flush();
  // store this wave's rows (Add, ReLU, the layer below's ReLU derivative)
  if (vec) {
    // 16-byte accesses, lane owning columns cs + 4 lane .. + 3: all eight
    // rows' Add and mask values are read before any row is stored (Add may
    // alias Y element for element), rows and columns past the matrix
    // clamped so every load is in bounds and unconditional
    const int c = cs + 4 * lane;
    const int ccl = min(c, width - 4);
    floatx4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      v[i] = *reinterpret_cast<const floatx4*>(Ys + (8 * wave + i) * kYLd + 4 * lane);
    if (add) {
      floatx4 a[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        a[i] = *reinterpret_cast<const floatx4*>(add + static_cast<int64_t>(min(rw + i, n - 1)) * ld_add + ccl);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] += a[i];
    }
    if (relu) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) v[i][q] = fmaxf(v[i][q], 0.f);
    }
    if (mask) {
      floatx4 mk[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        mk[i] = *reinterpret_cast<const floatx4*>(mask + static_cast<int64_t>(min(rw + i, n - 1)) * ldm + ccl);
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (!(mk[i][q] > 0.f)) v[i][q] = 0.f;
    }
    if (c < width) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (rw + i < n) *reinterpret_cast<floatx4*>(Y + static_cast<int64_t>(rw + i) * ldy + c) = v[i];
    }
    return;
  }
  for (int i = 0; i < 8; ++i) {
    const int64_t r = rw + i;
    if (r >= n) break;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int c = cs + lane + 64 * p;
      if (c < width) {
        float y = Ys[(8 * wave + i) * kYLd + lane + 64 * p];
        if (add) y += add[r * ld_add + c];
        if (relu) y = fmaxf(y, 0.f);
        if (mask && !(mask[r * ldm + c] > 0.f)) y = 0.f;   // ReLU derivative of the layer below
        Y[r * ldy + c] = y;
      }
    }
  }
}

}  // namespace

gist_status spmm_clustered(hipStream_t st, int64_t n, int64_t n_in, int64_t nnz,
                           const int32_t* rowptr, const int32_t* col, const float* val,
                           const float* X, int64_t ldx, int width, float* Y, int64_t ldy,
                           const float* add, int64_t ld_add, bool relu, const float* mask,
                           int64_t ldm) {
  if (n <= 0 || width <= 0) return GIST_OK;
  // The X loads use 32-bit byte offsets of up to 16 rows: wider rows, or a
  // matrix with fewer columns than one window step, take the gather kernel.
  if (ldx > INT32_MAX / 64 || n_in < kKs)
    return spmm(st, n, nnz, rowptr, col, val, X, ldx, width, Y, ldy, add, ld_add, relu, mask,
                ldm);
  const int64_t tiles = (n + kRows - 1) / kRows;
  const int64_t slabs = (width + kCols - 1) / kCols;
  const int64_t nblocks = tiles * slabs;
  if (nblocks > INT32_MAX || tiles > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, "spmm_clustered: grid too large");
  const double bytes = 4.0 * (n + 1) + 8.0 * static_cast<double>(nnz) +
                       4.0 * static_cast<double>(n) * width * (2.0 + (add ? 1.0 : 0.0) +
                                                                (mask ? 1.0 : 0.0));
  // 16-byte result stores (and Add / mask reads) where every row allows them
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  const bool vec = width % 4 == 0 && ldy % 4 == 0 && al16(Y) &&
                   (!add || (ld_add % 4 == 0 && al16(add))) &&
                   (!mask || (ldm % 4 == 0 && al16(mask)));
  ProfScope ps(st, "spmm_tile", 2.0 * static_cast<double>(nnz) * width, bytes);
  hipLaunchKernelGGL(spmm_tile_kernel, dim3(static_cast<unsigned>(nblocks)), dim3(256), 0, st,
                     static_cast<int>(n), static_cast<int>(n_in), rowptr, col, val, X, ldx, width,
                     Y, ldy, add, ld_add, relu ? 1 : 0, static_cast<int>(tiles), nblocks, mask,
                     ldm, vec ? 1 : 0);
  return check_launch("spmm_clustered");
}

}  // namespace gist
