// bf16-input GEMM for large products: operands are rounded to bf16 once,
// into padded K-contiguous copies, then multiplied on the bf16 MFMA units
// with fp32 accumulation.
//
// Why a separate path: the bf16 matrix cores run 16x faster than fp32 ones,
// so a kernel that streams fp32 operands (4 bytes per element) into a
// 128 x 128 tile and rounds them while staging cannot feed them -- it is
// bound by L2 traffic and conversion instructions.  Here
//
//   1. cvt_bf16_kernel rounds an operand (nearest-even, in hardware) into a
//      bf16 buffer [Rp][Kp], K contiguous, zero-padded to the tile grid
//      (row-contiguous operands are transposed through LDS on the way);
//   2. gemm_bf16_kernel multiplies the padded copies: 128 x 256 tiles (twice
//      the arithmetic per byte of a 128 x 128 tile), K steps of 64, four
//      waves each owning 128 rows x 64 columns (4 x 2 MFMA tiles of 32 x 32,
//      v_mfma_f32_32x32x16_bf16), double-buffered LDS, no bounds checks in
//      the loads thanks to the padding;
//   3. stream-K over one workgroup per CU with the same deterministic
//      partial-tile fix-up as the fp32 path.
//
// The result equals the in-kernel-rounding path's: both round the same fp32
// values to bf16 with round-to-nearest-even and accumulate in fp32.

#include <algorithm>
#include <cstdio>

#include "common.cuh"
#include "gemm_common.cuh"
#include "gist_internal.h"

namespace gist {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short ushort8 __attribute__((ext_vector_type(8)));

constexpr int TM = 128, TN = 256, TK = 64;
constexpr int LDH = TK + 8;          // LDS row stride in halves (144 B)
constexpr int kThr = 256;
constexpr int kStreamGroups = 256;   // one 256-thread workgroup per CU

__device__ __forceinline__ unsigned short bf16_bits(float f) {
  return __builtin_bit_cast(unsigned short, static_cast<__bf16>(f));
}

// ---- 1. conversion ---------------------------------------------------------

// dst[r][k] = bf16(src(r, k)) for r < Rp, k < Kp; zero outside R x K.
// One 64 x 64 tile per block, through LDS so both source orientations read
// and write coalesced.
template <bool KMAJ>
__global__ __launch_bounds__(256) void cvt_bf16_kernel(OpView src, int64_t R, int64_t K,
                                                       unsigned short* __restrict__ dst,
                                                       int64_t Kp, int64_t tiles_k) {
  __shared__ float tile[64][65];
  const int64_t tr = blockIdx.x / tiles_k, tk = blockIdx.x % tiles_k;
  const int64_t r0 = tr * 64, k0 = tk * 64;
  const int t = threadIdx.x;
  // load: 64 x 64 floats, 16 per thread
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int e = t + 256 * i;
    int rr, kk;
    if constexpr (KMAJ) { rr = e >> 6; kk = e & 63; }   // consecutive threads along K
    else { kk = e >> 6; rr = e & 63; }                  // consecutive threads along R
    const int64_t r = r0 + rr, k = k0 + kk;
    tile[rr][kk] = (r < R && k < K) ? src.at<KMAJ>(r, k) : 0.f;
  }
  __syncthreads();
  // store: 8 halves (16 B) per thread, K contiguous
  const int rr = t >> 2, kk = (t & 3) * 16;
  ushort8 lo, hi;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    lo[q] = bf16_bits(tile[rr][kk + q]);
    hi[q] = bf16_bits(tile[rr][kk + 8 + q]);
  }
  unsigned short* d = dst + (r0 + rr) * Kp + k0 + kk;
  *reinterpret_cast<ushort8*>(d) = lo;
  *reinterpret_cast<ushort8*>(d + 8) = hi;
}

// ---- 2. the product ----------------------------------------------------------

struct SchedB {
  int64_t T, ipw;
  int nk, tiles_m, tiles_n;
};

template <bool SPLIT_OUT>
__global__ __launch_bounds__(kThr) void gemm_bf16_kernel(int64_t M, int64_t N,
                                                         const unsigned short* __restrict__ A,
                                                         const unsigned short* __restrict__ B,
                                                         int64_t Kp, OutView C, SchedB S,
                                                         float* __restrict__ partials) {
  __shared__ __attribute__((aligned(16))) unsigned short lds[2][(TM + TN) * LDH];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int li = lane & 31, lh = lane >> 5;

  floatx16 acc[4][2];
  ushort8 ra[4], rb[8];
  int64_t m0 = 0, n0 = 0;

  // loads: 8 threads cover one row's 64 halves (128 B); 32 rows per pass
  const int lrow = t >> 3, lchunk = (t & 7) * 8;
  auto load = [&](int64_t k) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      ra[i] = *reinterpret_cast<const ushort8*>(A + (m0 + lrow + 32 * i) * Kp + k + lchunk);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      rb[i] = *reinterpret_cast<const ushort8*>(B + (n0 + lrow + 32 * i) * Kp + k + lchunk);
  };
  auto stage = [&](int buf) {
    unsigned short* As = lds[buf];
    unsigned short* Bs = As + TM * LDH;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<ushort8*>(As + (lrow + 32 * i) * LDH + lchunk) = ra[i];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<ushort8*>(Bs + (lrow + 32 * i) * LDH + lchunk) = rb[i];
  };
  auto compute = [&](int buf) {
    const unsigned short* As = lds[buf];
    const unsigned short* Bs = As + TM * LDH;
#pragma unroll
    for (int c = 0; c < TK / 16; ++c) {
      bf16x8 av[4], bv[2];
#pragma unroll
      for (int a = 0; a < 4; ++a)
        av[a] = *reinterpret_cast<const bf16x8*>(As + (a * 32 + li) * LDH + 16 * c + 8 * lh);
#pragma unroll
      for (int b = 0; b < 2; ++b)
        bv[b] = *reinterpret_cast<const bf16x8*>(Bs + (wave * 64 + b * 32 + li) * LDH + 16 * c +
                                                 8 * lh);
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[a], bv[b], acc[a][b], 0, 0, 0);
    }
  };

  const int64_t w = xcd_remap(blockIdx.x, gridDim.x);
  int64_t it = w * S.ipw;
  const int64_t it_end = min(S.T, it + S.ipw);
  const int64_t first_tile = it / S.nk;
  while (it < it_end) {
    const int64_t tile = it / S.nk;
    const int kb = static_cast<int>(it % S.nk);
    const int ke = static_cast<int>(min<int64_t>(S.nk, kb + (it_end - it)));
    int tm, tn;
    tile_coords_banded(tile, S.tiles_m, S.tiles_n, tm, tn);
    m0 = static_cast<int64_t>(tm) * TM;
    n0 = static_cast<int64_t>(tn) * TN;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
    __syncthreads();
    load(static_cast<int64_t>(kb) * TK);
    stage(0);
    __syncthreads();
    for (int j = kb; j + 1 < ke; ++j) {
      load(static_cast<int64_t>(j + 1) * TK);
      __builtin_amdgcn_sched_barrier(0);
      compute((j - kb) & 1);
      __builtin_amdgcn_sched_barrier(0);
      stage((j + 1 - kb) & 1);
      __syncthreads();
    }
    compute((ke - 1 - kb) & 1);

    // acc[a][b] register r of lane l: row a*32 + 8(r/4) + 4(l/32) + r%4,
    // column wave*64 + b*32 + l%32 of the tile
    if (kb == 0 && ke == S.nk) {
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int64_t col = n0 + wave * 64 + b * 32 + li;
          if (col >= N) continue;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t row = m0 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
            if (row < M) C.store<SPLIT_OUT>(row, col, acc[a][b][r]);
          }
        }
    } else {
      float* part = partials + (w * 2 + (tile == first_tile ? 0 : 1)) * (TM * TN);
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            part[(a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3)) * TN + wave * 64 + b * 32 + li] =
                acc[a][b][r];
    }
    it += ke - kb;
  }
}

// Sum split tiles' partials in workgroup order (one block per tile).
__global__ __launch_bounds__(256) void fixup_bf16_kernel(int64_t M, int64_t N, SchedB S,
                                                         const float* __restrict__ partials,
                                                         OutView C) {
  constexpr int kMaxParts = 512;
  __shared__ int64_t slot_off[kMaxParts];
  const int64_t t = blockIdx.x;
  const int64_t w_first = (t * S.nk) / S.ipw;
  const int64_t w_last = ((t + 1) * S.nk - 1) / S.ipw;
  if (w_first == w_last) return;
  const int parts = static_cast<int>(w_last - w_first + 1);
  for (int j = threadIdx.x; j < parts; j += 256) {
    const int64_t w = w_first + j;
    slot_off[j] = (w * 2 + (((w * S.ipw) / S.nk) == t ? 0 : 1)) * (TM * TN);
  }
  __syncthreads();
  int tm, tn;
  tile_coords_banded(t, S.tiles_m, S.tiles_n, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * TM, n0 = static_cast<int64_t>(tn) * TN;
  for (int e4 = threadIdx.x; e4 < TM * TN / 4; e4 += 256) {
    const int e = e4 * 4;
    const int64_t row = m0 + e / TN, col = n0 + e % TN;
    if (row >= M || col >= N) continue;
    floatx4 s = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < parts; ++j) s += *reinterpret_cast<const floatx4*>(partials + slot_off[j] + e);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (col + q < N) C.store<true>(row, col + q, s[q]);
  }
}

struct Layout {
  int64_t Mp, Np, Kp;
  size_t a_bytes, b_bytes, part_bytes;
  SchedB S;
  bool split;
  size_t total() const { return a_bytes + b_bytes + part_bytes; }
};

size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

Layout make_layout(int64_t M, int64_t N, int64_t K) {
  Layout L;
  L.Mp = (M + TM - 1) / TM * TM;
  L.Np = (N + TN - 1) / TN * TN;
  L.Kp = (K + TK - 1) / TK * TK;
  L.a_bytes = up256(static_cast<size_t>(L.Mp) * L.Kp * 2);
  L.b_bytes = up256(static_cast<size_t>(L.Np) * L.Kp * 2);
  SchedB& s = L.S;
  s.tiles_m = static_cast<int>(L.Mp / TM);
  s.tiles_n = static_cast<int>(L.Np / TN);
  s.nk = static_cast<int>(L.Kp / TK);
  const int64_t tiles = static_cast<int64_t>(s.tiles_m) * s.tiles_n;
  s.T = tiles * s.nk;
  s.ipw = tiles >= 4 * kStreamGroups ? s.nk : (s.T + kStreamGroups - 1) / kStreamGroups;
  L.split = s.ipw % s.nk != 0;
  const int64_t groups = (s.T + s.ipw - 1) / s.ipw;
  L.part_bytes = L.split ? static_cast<size_t>(groups) * 2 * TM * TN * sizeof(float) : 0;
  return L;
}

gist_status convert(hipStream_t st, const Operand& o, int64_t R, int64_t K, int64_t Rp,
                    int64_t Kp, unsigned short* dst) {
  OpView v = OpView::from(o);
  const int64_t tiles_k = Kp / 64;
  const int64_t blocks = (Rp / 64) * tiles_k;
  ProfScope ps(st, o.k_major ? "cvt_bf16_K" : "cvt_bf16_R", 0.0,
               4.0 * static_cast<double>(R) * K + 2.0 * static_cast<double>(Rp) * Kp);
  if (o.k_major)
    hipLaunchKernelGGL(cvt_bf16_kernel<true>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                       v, R, K, dst, Kp, tiles_k);
  else
    hipLaunchKernelGGL(cvt_bf16_kernel<false>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                       st, v, R, K, dst, Kp, tiles_k);
  return check_launch("bf16 conversion");
}

}  // namespace

bool gemm_bf16_packed_eligible(int64_t M, int64_t N, int64_t K) {
  // big enough that the conversion pass pays for itself
  return M >= 512 && N >= 512 && K >= 256;
}

size_t gemm_bf16_packed_workspace(int64_t M, int64_t N, int64_t K) {
  return make_layout(M, N, K).total();
}

gist_status gemm_bf16_packed(hipStream_t st, int64_t M, int64_t N, int64_t K, const Operand& A,
                             const Operand& B, const GemmOut& Cout, void* ws, size_t ws_bytes) {
  const Layout L = make_layout(M, N, K);
  if (!ws || ws_bytes < L.total()) return set_error(GIST_E_NOMEM, "gemm bf16: workspace too small");
  const int64_t groups = (L.S.T + L.S.ipw - 1) / L.S.ipw;
  if (groups > INT32_MAX || L.Mp % 64 || L.Np % 64)
    return set_error(GIST_E_UNSUPPORTED, "gemm bf16: grid too large");
  char* base = static_cast<char*>(ws);
  auto* a16 = reinterpret_cast<unsigned short*>(base);
  auto* b16 = reinterpret_cast<unsigned short*>(base + L.a_bytes);
  float* part = reinterpret_cast<float*>(base + L.a_bytes + L.b_bytes);
  gist_status s = convert(st, A, M, K, L.Mp, L.Kp, a16);
  if (s != GIST_OK) return s;
  s = convert(st, B, N, K, L.Np, L.Kp, b16);
  if (s != GIST_OK) return s;
  OutView c = OutView::from(Cout);
  const bool split_out = Cout.c1 != nullptr;
  {
    ProfScope ps(st, "gemm_bf16_packed", 2.0 * static_cast<double>(M) * N * K,
                 2.0 * (static_cast<double>(M) * K + static_cast<double>(N) * K) +
                     4.0 * static_cast<double>(M) * N);
    if (split_out)
      hipLaunchKernelGGL(gemm_bf16_kernel<true>, dim3(static_cast<unsigned>(groups)), dim3(kThr), 0,
                         st, M, N, a16, b16, L.Kp, c, L.S, part);
    else
      hipLaunchKernelGGL(gemm_bf16_kernel<false>, dim3(static_cast<unsigned>(groups)), dim3(kThr),
                         0, st, M, N, a16, b16, L.Kp, c, L.S, part);
  }
  s = check_launch("gemm bf16");
  if (s != GIST_OK) return s;
  if (L.split) {
    const int64_t tiles = static_cast<int64_t>(L.S.tiles_m) * L.S.tiles_n;
    ProfScope ps(st, "gemm_bf16_fixup", 0.0, 0.0);
    hipLaunchKernelGGL(fixup_bf16_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, st, M, N,
                       L.S, part, c);
    return check_launch("gemm bf16 fix-up");
  }
  return GIST_OK;
}

}  // namespace gist
