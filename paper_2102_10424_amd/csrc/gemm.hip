// Dense contractions of the sub-GCN layer on the MFMA matrix cores.
//
// C (M x N) = act(A (M x K) * B (K x N)) for the three products of eq. (2)
// and its backward pass: the forward transform (Abar H) W (for GraphSAGE
// [H | Abar H] [W_self; W_neigh]), the weight gradient (Abar H)^T dZ and the
// input gradient dZ W^T.  Operands are read straight from the row-major
// activations and weights in whichever orientation the product needs (see
// Operand in gist_internal.h), so no transpose is ever materialised.
//
// Tiling (gfx950, wave64): a 256-thread block computes a 128 x 128 tile of C;
// each of its four waves owns a 64 x 64 quadrant = 2 x 2 MFMA tiles of
// 32 x 32.  K advances in steps of 32 through double-buffered LDS tiles that
// always hold both operands K-contiguous ([row][k], padded), so every lane
// fetches its MFMA operands with one 16-byte LDS read per 4 MFMAs.
//
// fp32: v_mfma_f32_32x32x2_f32.  For step s of an 8-wide K chunk, lane l
// supplies A[i][4 h + s] and B[4 h + s][j] with i = j = l mod 32, h = l / 32:
// the two K slots of the instruction are mapped onto K columns 4h + s, which
// is a relabelling of the K sum and leaves the product unchanged.
//
// bf16-input: the same tile walk, operands rounded to bf16 (nearest-even)
// when staged into LDS, v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
//
// Small output grids split K over blocks (grid z); each split writes its
// partial tile to the workspace and a second kernel sums the splits in a
// fixed order, so results never depend on scheduling.

#include <algorithm>
#include <cstdio>

#include "common.cuh"
#include "gist_internal.h"

namespace gist {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDK = BK + 4;        // fp32 LDS row stride (floats)
constexpr int LDKH = BK + 8;       // bf16 LDS row stride (halves)
constexpr int kThreads = 256;

struct OpDev {
  const float* p0;
  const float* p1;
  int64_t ld0, ld1, split;
};

struct OutDev {
  float* c0;
  float* c1;
  int64_t ldc0, ldc1, c_split;
  int relu;
};

// Element (r, k) of an operand; r < R and k < K are checked by the caller.
template <bool KMAJ>
__device__ __forceinline__ float op_elem(const OpDev& o, int64_t r, int64_t k) {
  if constexpr (KMAJ) {
    return k < o.split ? o.p0[r * o.ld0 + k] : o.p1[r * o.ld1 + (k - o.split)];
  } else {
    return r < o.split ? o.p0[k * o.ld0 + r] : o.p1[k * o.ld1 + (r - o.split)];
  }
}

// Stage a 128 x 32 tile (rows r0.., k0..) of an operand into registers:
// 4 groups of 4 consecutive K values per thread.
template <bool KMAJ, bool VEC>
__device__ __forceinline__ void load_tile(const OpDev& o, int64_t R, int64_t K, int64_t r0,
                                          int64_t k0, floatx4 (&reg)[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int rr, kk;
    if constexpr (KMAJ) {  // 8 threads read one row's 32 K values (128 B)
      const int idx = t + kThreads * i;
      rr = idx >> 3;
      kk = (idx & 7) * 4;
    } else {  // consecutive threads read consecutive rows at fixed K
      const int idx = t + kThreads * i;
      rr = idx & 127;
      kk = (idx >> 7) * 4;
    }
    const int64_t r = r0 + rr, k = k0 + kk;
    floatx4 v = {0.f, 0.f, 0.f, 0.f};
    if (r < R) {
      if constexpr (KMAJ && VEC) {
        if (k + 3 < K) {
          const float* p = k < o.split ? o.p0 + r * o.ld0 + k : o.p1 + r * o.ld1 + (k - o.split);
          v = *reinterpret_cast<const floatx4*>(p);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (k + q < K) v[q] = op_elem<KMAJ>(o, r, k + q);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (k + q < K) v[q] = op_elem<KMAJ>(o, r, k + q);
      }
    }
    reg[i] = v;
  }
}

template <bool KMAJ>
__device__ __forceinline__ void tile_coord(int i, int& rr, int& kk) {
  const int idx = threadIdx.x + kThreads * i;
  if constexpr (KMAJ) {
    rr = idx >> 3;
    kk = (idx & 7) * 4;
  } else {
    rr = idx & 127;
    kk = (idx >> 7) * 4;
  }
}

template <bool KMAJ>
__device__ __forceinline__ void store_tile_f32(float* lds, const floatx4 (&reg)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int rr, kk;
    tile_coord<KMAJ>(i, rr, kk);
    *reinterpret_cast<floatx4*>(lds + rr * LDK + kk) = reg[i];
  }
}

// Round-to-nearest-even fp32 -> bf16 (NaN kept quiet).
__device__ __forceinline__ unsigned short f2bf(float f) {
  unsigned int u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<unsigned short>((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<unsigned short>(u >> 16);
}

template <bool KMAJ>
__device__ __forceinline__ void store_tile_bf16(unsigned short* lds, const floatx4 (&reg)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int rr, kk;
    tile_coord<KMAJ>(i, rr, kk);
    ushort4 h;
    h.x = f2bf(reg[i][0]);
    h.y = f2bf(reg[i][1]);
    h.z = f2bf(reg[i][2]);
    h.w = f2bf(reg[i][3]);
    *reinterpret_cast<ushort4*>(lds + rr * LDKH + kk) = h;
  }
}

// Map a linear tile id to (tile_m, tile_n): XCD-major, then column-major in
// bands of 8 tile rows so the blocks an XCD runs together share B columns
// and a narrow band of A rows.
__device__ __forceinline__ void tile_of(int64_t bid, int64_t tiles, int tiles_m, int& tm,
                                        int& tn) {
  const int64_t l = xcd_remap(bid, tiles);
  constexpr int kBand = 8;
  const int tiles_n = static_cast<int>(tiles / tiles_m);
  const int band = static_cast<int>(l / (static_cast<int64_t>(kBand) * tiles_n));
  const int rows_in_band = min(kBand, tiles_m - band * kBand);
  const int64_t in_band = l - static_cast<int64_t>(band) * kBand * tiles_n;
  tm = band * kBand + static_cast<int>(in_band % rows_in_band);
  tn = static_cast<int>(in_band / rows_in_band);
}

template <bool AK, bool BK_, bool AV, bool BV, bool BF16>
__global__ __launch_bounds__(kThreads) void gemm_kernel(int64_t M, int64_t N, int64_t K,
                                                        OpDev A, OpDev B, OutDev C,
                                                        int64_t k_per_split, float* partials,
                                                        int tiles_m) {
  constexpr int kStage = BF16 ? 0 : 2 * BM * LDK;  // floats per fp32 stage (A + B)
  constexpr int kStageH = BF16 ? 2 * BM * LDKH : 0;
  __shared__ __attribute__((aligned(16))) float lds_f[BF16 ? 1 : 2 * kStage];
  __shared__ __attribute__((aligned(16))) unsigned short lds_h[BF16 ? 2 * kStageH : 1];

  const int64_t tiles = static_cast<int64_t>(gridDim.x);
  int tm, tn;
  tile_of(blockIdx.x, tiles, tiles_m, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * BM, n0 = static_cast<int64_t>(tn) * BN;
  const int64_t kbeg = static_cast<int64_t>(blockIdx.z) * k_per_split;
  const int64_t kend = min(K, kbeg + k_per_split);
  const int nk = static_cast<int>((kend - kbeg + BK - 1) / BK);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, lh = lane >> 5;

  floatx16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  floatx4 ra[4], rb[4];
  if (nk > 0) {
    load_tile<AK, AV>(A, M, kend, m0, kbeg, ra);
    load_tile<BK_, BV>(B, N, kend, n0, kbeg, rb);
    if constexpr (BF16) {
      store_tile_bf16<AK>(lds_h, ra);
      store_tile_bf16<BK_>(lds_h + BM * LDKH, rb);
    } else {
      store_tile_f32<AK>(lds_f, ra);
      store_tile_f32<BK_>(lds_f + BM * LDK, rb);
    }
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t kn = kbeg + static_cast<int64_t>(kt + 1) * BK;
      load_tile<AK, AV>(A, M, kend, m0, kn, ra);
      load_tile<BK_, BV>(B, N, kend, n0, kn, rb);
    }
    if constexpr (BF16) {
      const unsigned short* As = lds_h + buf * kStageH;
      const unsigned short* Bs = As + BM * LDKH;
      // two K chunks of 16; lane half h supplies K values 8h .. 8h+7
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8 av[2], bv[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          av[t] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + t * 32 + li) * LDKH + 16 * c + 8 * lh);
          bv[t] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + t * 32 + li) * LDKH + 16 * c + 8 * lh);
        }
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[a], bv[b], acc[a][b], 0, 0, 0);
      }
    } else {
      const float* As = lds_f + buf * kStage;
      const float* Bs = As + BM * LDK;
#pragma unroll
      for (int c = 0; c < BK / 8; ++c) {
        floatx4 av[2], bv[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          av[t] = *reinterpret_cast<const floatx4*>(As + (wm * 64 + t * 32 + li) * LDK + 8 * c + 4 * lh);
          bv[t] = *reinterpret_cast<const floatx4*>(Bs + (wn * 64 + t * 32 + li) * LDK + 8 * c + 4 * lh);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
              acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[a][s], bv[b][s], acc[a][b], 0, 0, 0);
      }
    }
    if (more) {
      const int nb = buf ^ 1;
      if constexpr (BF16) {
        store_tile_bf16<AK>(lds_h + nb * kStageH, ra);
        store_tile_bf16<BK_>(lds_h + nb * kStageH + BM * LDKH, rb);
      } else {
        store_tile_f32<AK>(lds_f + nb * kStage, ra);
        store_tile_f32<BK_>(lds_f + nb * kStage + BM * LDK, rb);
      }
    }
    __syncthreads();
  }

  // Epilogue.  Accumulator register r of lane l holds C row
  // 8 (r / 4) + 4 (l / 32) + (r mod 4), column l mod 32 of its 32 x 32 tile.
  const bool split = gridDim.z > 1;
  float* part = split ? partials + static_cast<int64_t>(blockIdx.z) * M * N : nullptr;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t col = n0 + wn * 64 + b * 32 + li;
      if (col >= N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row >= M) continue;
        float v = acc[a][b][r];
        if (split) {
          part[row * N + col] = v;
        } else {
          if (C.relu) v = fmaxf(v, 0.f);
          if (col < C.c_split) C.c0[row * C.ldc0 + col] = v;
          else C.c1[row * C.ldc1 + (col - C.c_split)] = v;
        }
      }
    }
}

// Sum the K splits in order z = 0, 1, ... and apply the epilogue.
__global__ __launch_bounds__(256) void splitk_reduce(int64_t M, int64_t N, int splits,
                                                     const float* __restrict__ partials,
                                                     OutDev C) {
  const int64_t total = M * N;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < total; i += 256ll * gridDim.x) {
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += partials[static_cast<int64_t>(z) * total + i];
    if (C.relu) s = fmaxf(s, 0.f);
    const int64_t row = i / N, col = i % N;
    if (col < C.c_split) C.c0[row * C.ldc0 + col] = s;
    else C.c1[row * C.ldc1 + (col - C.c_split)] = s;
  }
}

struct Plan {
  int64_t tiles_m, tiles_n, splits, k_per_split;
};

Plan make_plan(int64_t M, int64_t N, int64_t K) {
  Plan p;
  p.tiles_m = (M + BM - 1) / BM;
  p.tiles_n = (N + BN - 1) / BN;
  const int64_t tiles = p.tiles_m * p.tiles_n;
  constexpr int64_t kTargetBlocks = 512;  // two rounds over 256 CUs
  int64_t s = 1;
  if (tiles < kTargetBlocks) {
    s = std::max<int64_t>(1, kTargetBlocks / tiles);
    s = std::min<int64_t>(s, std::max<int64_t>(1, K / 256));  // >= 256 of K per split
  }
  int64_t kps = (K + s - 1) / s;
  kps = (kps + BK - 1) / BK * BK;
  p.k_per_split = std::max<int64_t>(kps, BK);
  p.splits = (K + p.k_per_split - 1) / p.k_per_split;
  if (p.splits < 1) p.splits = 1;
  return p;
}

bool op_vec_ok(const Operand& o) {
  if (!o.k_major) return false;
  if (o.ld0 % 4 || !aligned16(o.p0)) return false;
  if (o.p1 && (o.ld1 % 4 || !aligned16(o.p1) || o.split % 4)) return false;
  return true;
}

template <bool AK, bool BK_, bool BF16>
void launch_kernel(hipStream_t st, bool av, bool bv, dim3 grid, int64_t M, int64_t N, int64_t K,
                   const OpDev& A, const OpDev& B, const OutDev& C, int64_t kps, float* part,
                   int tiles_m) {
#define GIST_GEMM_LAUNCH(AV_, BV_)                                                         \
  hipLaunchKernelGGL((gemm_kernel<AK, BK_, AV_, BV_, BF16>), grid, dim3(kThreads), 0, st, \
                     M, N, K, A, B, C, kps, part, tiles_m)
  if (av && bv) GIST_GEMM_LAUNCH(true, true);
  else if (av) GIST_GEMM_LAUNCH(true, false);
  else if (bv) GIST_GEMM_LAUNCH(false, true);
  else GIST_GEMM_LAUNCH(false, false);
#undef GIST_GEMM_LAUNCH
}

template <bool BF16>
void dispatch(hipStream_t st, const Operand& A, const Operand& B, bool av, bool bv, dim3 grid,
              int64_t M, int64_t N, int64_t K, const OpDev& a, const OpDev& b, const OutDev& c,
              int64_t kps, float* part, int tiles_m) {
  // Only the K-contiguous orientation has a vector path (VEC implies KMAJ).
  if (A.k_major && B.k_major)
    launch_kernel<true, true, BF16>(st, av, bv, grid, M, N, K, a, b, c, kps, part, tiles_m);
  else if (A.k_major)
    launch_kernel<true, false, BF16>(st, av, false, grid, M, N, K, a, b, c, kps, part, tiles_m);
  else if (B.k_major)
    launch_kernel<false, true, BF16>(st, false, bv, grid, M, N, K, a, b, c, kps, part, tiles_m);
  else
    launch_kernel<false, false, BF16>(st, false, false, grid, M, N, K, a, b, c, kps, part,
                                      tiles_m);
}

}  // namespace

size_t gemm_workspace(int64_t M, int64_t N, int64_t K, int /*dtype*/) {
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  const Plan p = make_plan(M, N, K);
  if (p.splits <= 1) return 0;
  return static_cast<size_t>(p.splits) * static_cast<size_t>(M) * static_cast<size_t>(N) *
         sizeof(float);
}

gist_status gemm(hipStream_t st, int64_t M, int64_t N, int64_t K, const Operand& A,
                 const Operand& B, const GemmOut& C, int dtype, void* ws, size_t ws_bytes) {
  if (M <= 0 || N <= 0) return GIST_OK;
  OutDev c{C.c0, C.c1, C.ldc0, C.ldc1, C.c_split, C.relu ? 1 : 0};
  if (K <= 0) {
    return set_error(GIST_E_UNSUPPORTED, "gemm: K == 0");
  }
  const Plan p = make_plan(M, N, K);
  if (p.tiles_m * p.tiles_n > INT32_MAX || p.splits > 65535)
    return set_error(GIST_E_UNSUPPORTED, "gemm: grid too large");
  float* part = nullptr;
  if (p.splits > 1) {
    const size_t need = gemm_workspace(M, N, K, dtype);
    if (!ws || ws_bytes < need) return set_error(GIST_E_NOMEM, "gemm: split-K workspace too small");
    part = static_cast<float*>(ws);
  }
  OpDev a{A.p0, A.p1 ? A.p1 : A.p0, A.ld0, A.p1 ? A.ld1 : A.ld0, A.p1 ? A.split : INT64_MAX};
  OpDev b{B.p0, B.p1 ? B.p1 : B.p0, B.ld0, B.p1 ? B.ld1 : B.ld0, B.p1 ? B.split : INT64_MAX};
  const bool av = op_vec_ok(A), bv = op_vec_ok(B);
  dim3 grid(static_cast<unsigned>(p.tiles_m * p.tiles_n), 1, static_cast<unsigned>(p.splits));
  const int tm = static_cast<int>(p.tiles_m);
  {
    // variant name: dtype, then the K-contiguous (K) / row-contiguous (R)
    // orientation of A and B as read from memory
    char name[32];
    snprintf(name, sizeof(name), "gemm_%s_%c%c", dtype == GIST_DTYPE_BF16_IN ? "bf16" : "f32",
             A.k_major ? 'K' : 'R', B.k_major ? 'K' : 'R');
    const double md = static_cast<double>(M), nd = static_cast<double>(N),
                 kd = static_cast<double>(K);
    ProfScope ps(st, name, 2.0 * md * nd * kd, 4.0 * (md * kd + kd * nd + md * nd));
    if (dtype == GIST_DTYPE_BF16_IN)
      dispatch<true>(st, A, B, av, bv, grid, M, N, K, a, b, c, p.k_per_split, part, tm);
    else
      dispatch<false>(st, A, B, av, bv, grid, M, N, K, a, b, c, p.k_per_split, part, tm);
  }
  {
    gist_status s = check_launch("gemm");
    if (s != GIST_OK) return s;
  }
  if (p.splits > 1) {
    const int64_t total = M * N;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 4096);
    ProfScope ps(st, "gemm_splitk_reduce", static_cast<double>(p.splits) * total,
                 4.0 * static_cast<double>(p.splits + 1) * total);
    hipLaunchKernelGGL(splitk_reduce, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, M,
                       N, static_cast<int>(p.splits), part, c);
    return check_launch("gemm split-K reduce");
  }
  return GIST_OK;
}

}  // namespace gist
