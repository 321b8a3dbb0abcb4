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
// Work distribution (stream-K): the (tile, K step) iterations of the whole
// product are dealt out in equal contiguous ranges to a fixed grid of 512
// workgroups (two per CU on 256 CUs), so the machine stays evenly loaded
// whatever the tile count -- M = 1,633 gives only 416 or 832 tiles, which
// whole-tile scheduling would spread over 1.6 rounds.  A tile whose K range
// is split between workgroups is written as partial tiles to the workspace
// and summed by a second kernel in workgroup order: deterministic, and no
// workgroup ever waits on another.  Products with plenty of tiles use one
// whole tile per workgroup and skip the second kernel.  Products with few
// tiles and a long K (a weight gradient reduced over many nodes) split K
// into slices dealt out slice-major, so that the workgroups an XCD runs
// together share each K range's operand rows in L2.  For N <= 64 the two
// waves whose columns would lie past the matrix take the second half of
// every K step instead (see NARROW below).

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

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDK = BK + 4;        // fp32 LDS row stride, [row][k] layout (floats)
constexpr int kTileF = BM * LDK;   // floats per fp32 operand tile
constexpr int KSH = 64;            // bf16 K step: two 32-wide load sub-tiles
constexpr int LDKH = KSH + 8;      // bf16 LDS row stride (halves)
constexpr int kThreads = 256;

struct OpDev {
  const float* p0;
  const float* p1;
  int64_t ld0, ld1, split;
  int64_t gs0, gs1;   // group strides of p0 / p1

  __device__ __forceinline__ OpDev group(int64_t g) const {
    OpDev o = *this;
    o.p0 += g * gs0;
    o.p1 += g * gs1;
    return o;
  }
};

struct OutDev {
  float* c0;
  float* c1;
  int64_t ldc0, ldc1, c_split;
  int relu;
  int64_t gs0, gs1;
  int sgd;     // C <- fmaf(-lr, product, C): a fused SGD step on weights in C
  float lr;
  const float* mask;   // C <- 0 where mask <= 0 (c0 columns only), or null
  int64_t ldm, gsm;

  __device__ __forceinline__ OutDev group(int64_t g) const {
    OutDev o = *this;
    o.c0 += g * gs0;
    o.c1 += g * gs1;
    if (mask) o.mask += g * gsm;
    return o;
  }
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

// Thread -> (row, k) of the 4-float group it stages, for a 128 x 32 tile.
//   K-contiguous operands: 8 threads cover one row's 32 K values (128 B).
//   Row-contiguous, scalar: consecutive threads take consecutive rows at one
//     K and read 4 K values each.
//   Row-contiguous, vector: each thread owns a 4 x 4 block (rows 4g..4g+3,
//     K values 4q..4q+3) and loads it as 4 row vectors, one per K value;
//     group i is the vector at K value 4q + i, transposed into rows when
//     staged.  Lane bits (0 | 1-2 | 3-5) of a wave pick (g mod 2 | q mod 4 |
//     g / 2 mod 8); the wave picks g / 16 and q / 4.  Each run of eight
//     lanes (one LDS write pass) then holds both row-block parities times
//     four K groups, so its 16-byte stores into the [row][k] tile (row
//     stride LDK = 36 floats) land in eight distinct groups of four banks;
//     with consecutive row blocks per run they fell into two (4-way
//     conflicts).  Sixteen lanes still read 256 contiguous bytes per K value.
template <bool KMAJ, bool VEC>
__device__ __forceinline__ void tile_coord(int i, int& rr, int& kk) {
  const int idx = threadIdx.x + kThreads * i;
  if constexpr (KMAJ) {
    rr = idx >> 3;
    kk = (idx & 7) * 4;
  } else if constexpr (VEC) {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    rr = 4 * ((l & 1) + 2 * ((l >> 3) & 7) + 16 * (w & 1));
    kk = 4 * (((l >> 1) & 3) + 4 * (w >> 1)) + i;
  } else {
    rr = idx & 127;
    kk = (idx >> 7) * 4;
  }
}

// Stage a 128 x 32 tile (rows r0.., k0..) of an operand into registers:
// 4 groups of 4 consecutive K values per thread.
//
// Full K tiles (FULLK: k0 + 32 <= K) take a branch-free path: rows past the
// operand's edge read a clamped (valid) row, so the loads of a tile issue
// back to back with no wait.  Only the last, partial K tile of a split checks
// every element (it must contribute exact zeros beyond K).
template <bool KMAJ, bool VEC, bool FULLK>
__device__ __forceinline__ void load_tile(const OpDev& o, int64_t R, int64_t K, int64_t r0,
                                          int64_t k0, floatx4 (&reg)[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int rr, kk;
    tile_coord<KMAJ, VEC>(i, rr, kk);
    const int64_t r = r0 + rr, k = k0 + kk;
    floatx4 v = {0.f, 0.f, 0.f, 0.f};
    if constexpr (!KMAJ && VEC) {
      // 4 consecutive rows at one K: a 16-byte load along the contiguous dim.
      // The vector path requires split % 128 == 0, so the whole tile lies on
      // one side of the split and the pointer choice is uniform.
      const bool lo = r0 < o.split;
      const float* base = lo ? o.p0 : o.p1 - o.split;
      const int64_t ld = lo ? o.ld0 : o.ld1;
      if constexpr (FULLK) {
        const int64_t rc = r < R ? r : R - 4;  // R % 4 == 0 on this path
        v = *reinterpret_cast<const floatx4*>(base + k * ld + rc);
      } else {
        if (k < K) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (r + q < R) v[q] = base[k * ld + r + q];
        }
      }
    } else {
      const bool rin = r < R;
      const int64_t rc = rin ? r : R - 1;
      if constexpr (FULLK) {
        if constexpr (KMAJ && VEC) {
          // split % 128 == 0: the whole K step lies on one side of the split
          const bool lo = k0 < o.split;
          const float* base = lo ? o.p0 : o.p1 - o.split;
          const int64_t ld = lo ? o.ld0 : o.ld1;
          v = *reinterpret_cast<const floatx4*>(base + rc * ld + k);
        } else if constexpr (KMAJ) {
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = op_elem<KMAJ>(o, rc, k + q);
        } else {
          const float* base = rc < o.split ? o.p0 + rc : o.p1 + (rc - o.split);
          const int64_t ld = rc < o.split ? o.ld0 : o.ld1;
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = base[(k + q) * ld];
        }
        // rows past the edge keep the clamped row's (finite) values: they only
        // feed output rows / columns the epilogue never stores
      } else {
        if (rin) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (k + q < K) v[q] = op_elem<KMAJ>(o, r, k + q);
        }
      }
    }
    reg[i] = v;
    (void)t;
  }
}

// Transpose a row-vector 4 x 4 block (reg[i][j] = element (rr + j, kk + i))
// into row order (out[j][i]).
__device__ __forceinline__ void transpose4(const floatx4 (&reg)[4], floatx4 (&out)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) out[j][i] = reg[i][j];
}

template <bool KMAJ, bool VEC>
__device__ __forceinline__ void store_tile_f32(float* lds, const floatx4 (&reg)[4]) {
  if constexpr (!KMAJ && VEC) {
    floatx4 rows[4];
    transpose4(reg, rows);
    int rr, kk;
    tile_coord<KMAJ, VEC>(0, rr, kk);
#pragma unroll
    for (int j = 0; j < 4; ++j) *reinterpret_cast<floatx4*>(lds + (rr + j) * LDK + kk) = rows[j];
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int rr, kk;
      tile_coord<KMAJ, VEC>(i, rr, kk);
      *reinterpret_cast<floatx4*>(lds + rr * LDK + kk) = reg[i];
    }
  }
}

// MFMA operand fragment: the 4 K values k0 .. k0+3 of tile row `row`.
__device__ __forceinline__ floatx4 frag_f32(const float* lds, int row, int k0) {
  return *reinterpret_cast<const floatx4*>(lds + row * LDK + k0);
}

// Round-to-nearest-even fp32 -> bf16 (gfx950 converts in hardware).
__device__ __forceinline__ unsigned short f2bf(float f) {
  return __builtin_bit_cast(unsigned short, static_cast<__bf16>(f));
}

template <bool KMAJ, bool VEC>
__device__ __forceinline__ void store_tile_bf16(unsigned short* lds, const floatx4 (&reg)[4],
                                                int koff) {
  auto put = [&](int rr, int kk, const floatx4& v) {
    ushort4 h;
    h.x = f2bf(v[0]);
    h.y = f2bf(v[1]);
    h.z = f2bf(v[2]);
    h.w = f2bf(v[3]);
    *reinterpret_cast<ushort4*>(lds + rr * LDKH + koff + kk) = h;
  };
  if constexpr (!KMAJ && VEC) {
    floatx4 rows[4];
    transpose4(reg, rows);
    int rr, kk;
    tile_coord<KMAJ, VEC>(0, rr, kk);
#pragma unroll
    for (int j = 0; j < 4; ++j) put(rr + j, kk, rows[j]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int rr, kk;
      tile_coord<KMAJ, VEC>(i, rr, kk);
      put(rr, kk, reg[i]);
    }
  }
}

struct Sched {
  int64_t T;        // total iterations = tiles * nk (tiles of all groups)
  int64_t ipw;      // iterations per workgroup (stream-K)
  int nk;           // K steps per tile
  int tiles_m, tiles_n;
  int64_t tpg;      // tiles per group (tiles_m * tiles_n)
  int64_t tiles;    // tiles of all groups
  int64_t spu;      // > 0: K-slice-major split, K steps per slice; 0: stream-K
};

__device__ __forceinline__ float* out_ptr(const OutDev& C, int64_t row, int64_t col) {
  return col < C.c_split ? C.c0 + row * C.ldc0 + col : C.c1 + row * C.ldc1 + (col - C.c_split);
}

__device__ __forceinline__ void store_out(const OutDev& C, int64_t row, int64_t col, float v) {
  if (C.relu) v = fmaxf(v, 0.f);
  if (C.mask && col < C.c_split && !(C.mask[row * C.ldm + col] > 0.f)) v = 0.f;
  float* p = out_ptr(C, row, col);
  if (C.sgd) v = fmaf(-C.lr, v, *p);
  *p = v;
}

// Two resident blocks per CU where that fits in registers without spilling
// (fp32 with vector loads on both operands, or both K-contiguous).
template <bool AK, bool BK_, bool AV, bool BV, bool BF16>
constexpr int min_blocks() { return (!BF16 && ((AV && BV) || (AK && BK_))) ? 2 : 1; }

// Double-buffered MFMA fragments (16 more VGPRs) where the variant still
// fits two waves per SIMD with them.
template <bool AK, bool BK_, bool AV, bool BV>
constexpr bool kPipeFrag() { return AV && BV && AK == BK_; }

// NARROW (fp32, N <= 64): the tile's columns 64..127 lie past the matrix, so
// the two waves that would own them take half of every K step instead --
// waves wn = 0 the step's 8-wide K chunks 0-1, waves wn = 1 chunks 2-3, all
// on columns 0..63 -- and the two halves are added through LDS before the
// epilogue (a split of K inside the workgroup, always summed in the same
// order).  Each step then costs half the MFMA time per wave.
template <bool AK, bool BK_, bool AV, bool BV, bool BF16, bool NARROW>
__global__ __launch_bounds__(kThreads, (min_blocks<AK, BK_, AV, BV, BF16>())) void gemm_kernel(int64_t M, int64_t N, int64_t K,
                                                        OpDev A, OpDev B, OutDev C, Sched S,
                                                        float* partials) {
  static_assert(!(NARROW && BF16), "the narrow split is an fp32 variant");
  constexpr int kStage = BF16 ? 0 : 2 * kTileF;    // floats per fp32 stage (A + B)
  constexpr int kStageH = BF16 ? 2 * BM * LDKH : 0;
  __shared__ __attribute__((aligned(16))) float lds_f[BF16 ? 1 : 2 * kStage];
  __shared__ __attribute__((aligned(16))) unsigned short lds_h[BF16 ? 2 * kStageH : 1];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, lh = lane >> 5;
  constexpr int NC = NARROW ? 2 : BK / 8;   // 8-wide K chunks per wave per fp32 step
  const int cb = NARROW ? 2 * wn : 0;       // this wave's first chunk
  const int bw = NARROW ? 0 : wn;           // this wave's 64-column block of the tile

  // K per pipeline step: one 32-wide load sub-tile for fp32, two for bf16
  constexpr int KS = BF16 ? KSH : BK;
  constexpr int SUB = KS / BK;
  floatx16 acc[2][2];
  floatx4 ra[SUB][4], rb[SUB][4];
  int64_t m0 = 0, n0 = 0;
  OpDev Ag = A, Bg = B;   // this tile's group of A, B and C
  OutDev Cg = C;

  auto stage = [&](int buf) {
    if constexpr (BF16) {
#pragma unroll
      for (int s = 0; s < SUB; ++s) {
        store_tile_bf16<AK, AV>(lds_h + buf * kStageH, ra[s], s * BK);
        store_tile_bf16<BK_, BV>(lds_h + buf * kStageH + BM * LDKH, rb[s], s * BK);
      }
    } else {
      store_tile_f32<AK, AV>(lds_f + buf * kStage, ra[0]);
      store_tile_f32<BK_, BV>(lds_f + buf * kStage + kTileF, rb[0]);
    }
  };
  auto load_full = [&](int64_t k) {
#pragma unroll
    for (int s = 0; s < SUB; ++s) {
      load_tile<AK, AV, true>(Ag, M, K, m0, k + s * BK, ra[s]);
      load_tile<BK_, BV, true>(Bg, N, K, n0, k + s * BK, rb[s]);
    }
  };
  auto load_edge = [&](int64_t k) {
#pragma unroll
    for (int s = 0; s < SUB; ++s) {
      load_tile<AK, AV, false>(Ag, M, K, m0, k + s * BK, ra[s]);
      load_tile<BK_, BV, false>(Bg, N, K, n0, k + s * BK, rb[s]);
    }
  };
  auto compute = [&](int buf) {
    if constexpr (BF16) {
      const unsigned short* As = lds_h + buf * kStageH;
      const unsigned short* Bs = As + BM * LDKH;
      // K chunks of 16; lane half h supplies K values 8h .. 8h+7
#pragma unroll
      for (int c = 0; c < KS / 16; ++c) {
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
      const float* Bs = As + kTileF;
      if constexpr (kPipeFrag<AK, BK_, AV, BV>()) {
        // fragments of chunk c+1 are read while chunk c multiplies
        floatx4 av[2][2], bv[2][2];
        auto rd = [&](int c, int p) {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            av[p][t] = frag_f32(As, wm * 64 + t * 32 + li, 8 * c + 4 * lh);
            bv[p][t] = frag_f32(Bs, bw * 64 + t * 32 + li, 8 * c + 4 * lh);
          }
        };
        rd(cb, 0);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          if (c + 1 < NC) rd(cb + c + 1, (c + 1) & 1);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
              for (int b = 0; b < 2; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[c & 1][a][s], bv[c & 1][b][s],
                                                                 acc[a][b], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      } else {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          floatx4 av[2], bv[2];
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            av[t] = frag_f32(As, wm * 64 + t * 32 + li, 8 * (cb + c) + 4 * lh);
            bv[t] = frag_f32(Bs, bw * 64 + t * 32 + li, 8 * (cb + c) + 4 * lh);
          }
#pragma unroll
          for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
              for (int b = 0; b < 2; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[a][s], bv[b][s], acc[a][b], 0, 0, 0);
          // one K chunk's fragments live at a time (keeps two waves per SIMD)
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // fp32 step j with step j+1's staging (its registers to LDS buffer nbuf,
  // free since the barrier that ended step j-1) placed among the MFMAs of
  // chunk 2: the transposes and LDS writes issue while the matrix core runs,
  // instead of after the last MFMA, when the other wave of the SIMD may be
  // staging too.  Same arithmetic, same order as compute then stage.
  auto compute_staged = [&](int buf, int nbuf) {
    const float* As = lds_f + buf * kStage;
    const float* Bs = As + kTileF;
    auto mfma16 = [&](const floatx4 (&av)[2], const floatx4 (&bv)[2]) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[a][q], bv[b][q], acc[a][b], 0, 0, 0);
    };
    auto interleave = [&]() {
#pragma unroll
      for (int g = 0; g < 8; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);   // up to four VALU
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);   // an LDS write
      }
    };
    if constexpr (kPipeFrag<AK, BK_, AV, BV>()) {
      floatx4 av[2][2], bv[2][2];
      auto rd = [&](int c, int p) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          av[p][t] = frag_f32(As, wm * 64 + t * 32 + li, 8 * c + 4 * lh);
          bv[p][t] = frag_f32(Bs, bw * 64 + t * 32 + li, 8 * c + 4 * lh);
        }
      };
      rd(cb, 0);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        if (c + 1 < NC) rd(cb + c + 1, (c + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
        if (c == 1) stage(nbuf);
        mfma16(av[c & 1], bv[c & 1]);
        if (c == 1) interleave();
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        floatx4 av[2], bv[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          av[t] = frag_f32(As, wm * 64 + t * 32 + li, 8 * (cb + c) + 4 * lh);
          bv[t] = frag_f32(Bs, bw * 64 + t * 32 + li, 8 * (cb + c) + 4 * lh);
        }
        if (c == 1) stage(nbuf);
        mfma16(av, bv);
        if (c == 1) interleave();
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  const int64_t w = xcd_remap(blockIdx.x, gridDim.x);
  int64_t it, it_end;
  if (S.spu > 0) {
    // K-slice-major: workgroup w takes K slice w / tiles of tile w % tiles,
    // so the workgroups an XCD runs together (consecutive w) cover every
    // tile of the same K range and share its operand rows in L2
    const int64_t q = w / S.tiles, t = w - q * S.tiles;
    const int64_t kb = q * S.spu;
    it = t * S.nk + kb;
    it_end = t * S.nk + min<int64_t>(S.nk, kb + S.spu);
  } else {
    it = w * S.ipw;
    it_end = min(S.T, it + S.ipw);
  }
  const int64_t first_tile = it / S.nk;
  const bool k_ragged = K % KS != 0;

  while (it < it_end) {
    const int64_t tile = it / S.nk;
    const int kb = static_cast<int>(it % S.nk);
    const int ke = static_cast<int>(min<int64_t>(S.nk, kb + (it_end - it)));
    const int64_t grp = tile / S.tpg;
    int tm, tn;
    tile_coords_banded(tile - grp * S.tpg, S.tiles_m, S.tiles_n, tm, tn);
    m0 = static_cast<int64_t>(tm) * BM;
    n0 = static_cast<int64_t>(tn) * BN;
    Ag = A.group(grp);
    Bg = B.group(grp);
    Cg = C.group(grp);
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    // K steps [kb, ke) of this tile; the tile's last step may be partial
    const bool tail = ke == S.nk && k_ragged;
    const int full_end = tail ? ke - 1 : ke;
    __syncthreads();  // LDS of the previous segment fully consumed
    if (kb < full_end) {
      load_full(static_cast<int64_t>(kb) * KS);
      stage(0);
      __syncthreads();
      // steady state: prefetch step j+1 into registers while step j computes
      for (int j = kb; j + 1 < full_end; ++j) {
        load_full(static_cast<int64_t>(j + 1) * KS);
        // keep the prefetch at the top of the iteration: without the fence
        // the scheduler sinks the loads next to their LDS stores, and their
        // latency is no longer hidden behind the step's MFMAs
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (BF16) {
          compute((j - kb) & 1);
          __builtin_amdgcn_sched_barrier(0);
          stage((j + 1 - kb) & 1);
        } else {
          compute_staged((j - kb) & 1, (j + 1 - kb) & 1);
        }
        __syncthreads();
      }
      compute((full_end - 1 - kb) & 1);
    }
    if (tail) {
      const int buf = (full_end - kb) & 1;
      load_edge(static_cast<int64_t>(full_end) * KS);
      __syncthreads();
      stage(buf);
      __syncthreads();
      compute(buf);
    }

    if constexpr (NARROW) {
      // each wave adds its partner's K half (waves 2i and 2i+1 hold the two
      // halves of the same 64 x 64 block; a + b == b + a, so both end with
      // the same sums), without a branch on the wave
      __syncthreads();   // every wave is done reading this segment's tiles
      float* mine = lds_f + wave * 4096;
      const float* other = lds_f + (wave ^ 1) * 4096;
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) mine[((a * 2 + b) * 16 + r) * 64 + lane] = acc[a][b][r];
      __syncthreads();
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[a][b][r] += other[((a * 2 + b) * 16 + r) * 64 + lane];
          __builtin_amdgcn_sched_barrier(0);
        }
    }

    // Epilogue.  Accumulator register r of lane l holds C row
    // 8 (r / 4) + 4 (l / 32) + (r mod 4), column l mod 32 of its 32 x 32 tile.
    // (NARROW: the waves of column block 1 hold columns 64.. >= N and store
    // nothing.)
    if (kb == 0 && ke == S.nk) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int64_t col = n0 + wn * 64 + b * 32 + li;
          if (col >= N) continue;
          if (Cg.sgd) {
            // fused SGD step: the sub-tile's 16 weights are read before any is
            // written (one memory latency, not sixteen; reading the next
            // sub-tile's ahead would need registers these kernels lack)
            float w[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int64_t row = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
              w[r] = row < M ? *out_ptr(Cg, row, col) : 0.f;
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int64_t row = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
              if (row < M) *out_ptr(Cg, row, col) = fmaf(-Cg.lr, acc[a][b][r], w[r]);
            }
            continue;
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t row = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
            if (row < M) store_out(Cg, row, col, acc[a][b][r]);
          }
        }
    } else if (!NARROW || wn == 0) {
      // partial tile: slot 0 holds this workgroup's first tile, slot 1 its last
      float* part = partials + (w * 2 + (tile == first_tile ? 0 : 1)) * (BM * BN);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int rr = wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
            const int cc = wn * 64 + b * 32 + li;
            part[rr * BN + cc] = acc[a][b][r];
          }
    }
    it += ke - kb;
  }
}

// Sum the partial tiles of every tile split between workgroups, in
// workgroup order, and apply the epilogue.  Grid: (tile, 8-row chunk of the
// tile), so that a tile split over many workgroups (a thin dW = H^T dZ with
// a long K) is still summed by 16 blocks; each thread sums one float4 of
// every partial, in workgroup order (bitwise the same for any grid shape).
constexpr int kMaxFixupParts = 1024;
constexpr int kFixRows = 8;
constexpr int kFixChunks = BM / kFixRows;
static_assert(kFixRows * BN == 4 * 256, "one float4 per thread per partial");

__global__ __launch_bounds__(256) void streamk_fixup(int64_t M, int64_t N, Sched S,
                                                     const float* __restrict__ partials,
                                                     OutDev C) {
  __shared__ int64_t slot_off[kMaxFixupParts];
  const int64_t t = blockIdx.x;
  const int chunk = blockIdx.y;
  const bool sliced = S.spu > 0;
  const int64_t w_first = sliced ? 0 : (t * S.nk) / S.ipw;
  const int64_t w_last = sliced ? (S.nk + S.spu - 1) / S.spu - 1 : ((t + 1) * S.nk - 1) / S.ipw;
  if (w_first == w_last) return;  // computed whole and stored by one workgroup
  const int64_t grp = t / S.tpg;
  int tm, tn;
  tile_coords_banded(t - grp * S.tpg, S.tiles_m, S.tiles_n, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * BM, n0 = static_cast<int64_t>(tn) * BN;
  if (m0 + chunk * kFixRows >= M) return;   // the chunk lies below the matrix
  const int parts = static_cast<int>(w_last - w_first + 1);
  for (int j = threadIdx.x; j < parts; j += 256) {
    // sliced: slice j of tile t is workgroup j * tiles + t, its only tile
    const int64_t w = w_first + j;
    slot_off[j] = sliced ? (j * S.tiles + t) * 2 * (BM * BN)
                         : (w * 2 + (((w * S.ipw) / S.nk) == t ? 0 : 1)) * (BM * BN);
  }
  __syncthreads();
  const OutDev Cg = C.group(grp);
  const int e = chunk * kFixRows * BN + threadIdx.x * 4;
  const int64_t row = m0 + e / BN, col = n0 + e % BN;
  if (row >= M || col >= N) return;
  floatx4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int j = 0; j < parts; ++j) s += *reinterpret_cast<const floatx4*>(partials + slot_off[j] + e);
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (col + q < N) store_out(Cg, row, col + q, s[q]);
}

constexpr int64_t kStreamWG = 512;   // two resident 256-thread blocks per CU, 256 CUs
constexpr int64_t kMinSteps = 8;     // fewest K steps a stream-K workgroup takes

Sched make_sched(int64_t M, int64_t N, int64_t K, int dtype, int64_t groups = 1) {
  const int ks = dtype == GIST_DTYPE_BF16_IN ? KSH : BK;
  Sched s;
  s.tiles_m = static_cast<int>((M + BM - 1) / BM);
  s.tiles_n = static_cast<int>((N + BN - 1) / BN);
  s.nk = static_cast<int>((K + ks - 1) / ks);
  s.tpg = static_cast<int64_t>(s.tiles_m) * s.tiles_n;
  const int64_t tiles = s.tpg * groups;
  s.tiles = tiles;
  s.T = tiles * s.nk;
  s.spu = 0;
  if (tiles >= 4 * kStreamWG) {
    s.ipw = s.nk;   // enough tiles: one whole tile per workgroup
  } else if (tiles * 8 <= kStreamWG && s.nk >= 2 * kMinSteps) {
    // few tiles, long K (a weight gradient over many nodes): the K range in
    // slices, K-slice-major over the grid, at least kMinSteps steps each
    const int64_t slices = std::min<int64_t>(kStreamWG / tiles, s.nk / kMinSteps);
    s.spu = (s.nk + slices - 1) / slices;
    s.ipw = s.spu;
  } else {
    // stream-K over kStreamWG workgroups, but at least kMinSteps K steps
    // each: a small product (a narrow slice, few tiles) split one step per
    // workgroup would write a 64 KB partial tile per step for the fix-up to
    // read back
    s.ipw = std::max<int64_t>((s.T + kStreamWG - 1) / kStreamWG,
                              std::min<int64_t>(s.nk, kMinSteps));
  }
  return s;
}

int64_t sched_slices(const Sched& s) { return (s.nk + s.spu - 1) / s.spu; }
int64_t sched_groups(const Sched& s) {
  return s.spu > 0 ? sched_slices(s) * s.tiles : (s.T + s.ipw - 1) / s.ipw;
}
bool sched_split(const Sched& s) { return s.spu > 0 ? sched_slices(s) > 1 : s.ipw % s.nk != 0; }

// 16-byte loads along the operand's contiguous dimension are legal when the
// leading dimensions and base addresses are multiples of 4 floats (and, for
// row-contiguous operands, the row count too).  A concatenation split must
// fall on a 128 boundary, so that every K step and every tile lies on one
// side of it and the pointer choice stays uniform.
bool op_vec_ok(const Operand& o, int64_t R) {
  if (o.ld0 % 4 || !aligned16(o.p0) || o.gs0 % 4) return false;
  if (o.p1 && (o.ld1 % 4 || !aligned16(o.p1) || o.split % 128 || o.gs1 % 4)) return false;
  if (!o.k_major && R % 4) return false;
  return true;
}

template <bool AK, bool BK_, bool BF16, bool NARROW>
void launch_kernel(hipStream_t st, bool av, bool bv, dim3 grid, int64_t M, int64_t N, int64_t K,
                   const OpDev& A, const OpDev& B, const OutDev& C, const Sched& S,
                   float* part) {
#define GIST_GEMM_LAUNCH(AV_, BV_)                                                         \
  hipLaunchKernelGGL((gemm_kernel<AK, BK_, AV_, BV_, BF16, NARROW>), grid, dim3(kThreads), 0, \
                     st, M, N, K, A, B, C, S, part)
  if (av && bv) GIST_GEMM_LAUNCH(true, true);
  else if (av) GIST_GEMM_LAUNCH(true, false);
  else if (bv) GIST_GEMM_LAUNCH(false, true);
  else GIST_GEMM_LAUNCH(false, false);
#undef GIST_GEMM_LAUNCH
}

template <bool BF16, bool NARROW>
void dispatch(hipStream_t st, const Operand& A, const Operand& B, bool av, bool bv, dim3 grid,
              int64_t M, int64_t N, int64_t K, const OpDev& a, const OpDev& b, const OutDev& c,
              const Sched& S, float* part) {
  if (A.k_major && B.k_major)
    launch_kernel<true, true, BF16, NARROW>(st, av, bv, grid, M, N, K, a, b, c, S, part);
  else if (A.k_major)
    launch_kernel<true, false, BF16, NARROW>(st, av, bv, grid, M, N, K, a, b, c, S, part);
  else if (B.k_major)
    launch_kernel<false, true, BF16, NARROW>(st, av, bv, grid, M, N, K, a, b, c, S, part);
  else
    launch_kernel<false, false, BF16, NARROW>(st, av, bv, grid, M, N, K, a, b, c, S, part);
}

}  // namespace

size_t gemm_workspace(int64_t M, int64_t N, int64_t K, int dtype, int64_t groups) {
  if (M <= 0 || N <= 0 || K <= 0 || groups <= 0) return 0;
  if (dtype == GIST_DTYPE_BF16_IN && gemm_bf16_packed_eligible(M, N, K))
    return gemm_bf16_packed_workspace(M, N, K);   // groups run one after another
  const Sched s = make_sched(M, N, K, dtype, groups);
  if (!sched_split(s)) return 0;
  return static_cast<size_t>(sched_groups(s)) * 2 * BM * BN * sizeof(float);
}

gist_status gemm(hipStream_t st, int64_t M, int64_t N, int64_t K, const Operand& A,
                 const Operand& B, const GemmOut& C, int dtype, void* ws, size_t ws_bytes,
                 int64_t ngroups, int64_t k_alg) {
  if (M <= 0 || N <= 0 || ngroups <= 0) return GIST_OK;
  OutDev c{C.c0, C.c1, C.ldc0, C.ldc1, C.c_split, C.relu ? 1 : 0, C.gs0, C.gs1,
           C.sgd ? 1 : 0, C.lr, C.mask, C.ldm, C.gsm};
  if (K <= 0) return set_error(GIST_E_UNSUPPORTED, "gemm: K == 0");
  if (dtype == GIST_DTYPE_BF16_IN && gemm_bf16_packed_eligible(M, N, K)) {
    // the packed path converts each group's operands; groups run in turn
    for (int64_t g = 0; g < ngroups; ++g) {
      Operand ag = A, bg = B;
      GemmOut cg = C;
      ag.p0 += g * A.gs0;
      if (A.p1) ag.p1 += g * A.gs1;
      bg.p0 += g * B.gs0;
      if (B.p1) bg.p1 += g * B.gs1;
      cg.c0 += g * C.gs0;
      if (C.c1) cg.c1 += g * C.gs1;
      if (C.mask) cg.mask += g * C.gsm;
      gist_status s = gemm_bf16_packed(st, M, N, K, ag, bg, cg, ws, ws_bytes);
      if (s != GIST_OK) return s;
    }
    return GIST_OK;
  }
  if (K > (static_cast<int64_t>(INT32_MAX) - KSH) * BK)
    return set_error(GIST_E_UNSUPPORTED, "gemm: K too large");
  const Sched S = make_sched(M, N, K, dtype, ngroups);
  const int64_t groups = sched_groups(S);
  const int64_t tiles = S.tpg * ngroups;
  if (groups > INT32_MAX || tiles > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, "gemm: grid too large");
  float* part = nullptr;
  const bool split = sched_split(S);
  if (split) {
    // a tile's iterations span at most ceil(nk / ipw) + 1 workgroups
    if ((S.spu > 0 ? sched_slices(S) : (S.nk + S.ipw - 1) / S.ipw + 1) > kMaxFixupParts)
      return set_error(GIST_E_UNSUPPORTED, "gemm: too many partial tiles per tile");
    const size_t need = gemm_workspace(M, N, K, dtype, ngroups);
    if (!ws || ws_bytes < need) return set_error(GIST_E_NOMEM, "gemm: workspace too small");
    part = static_cast<float*>(ws);
  }
  OpDev a{A.p0, A.p1 ? A.p1 : A.p0, A.ld0, A.p1 ? A.ld1 : A.ld0, A.p1 ? A.split : INT64_MAX,
          A.gs0, A.p1 ? A.gs1 : A.gs0};
  OpDev b{B.p0, B.p1 ? B.p1 : B.p0, B.ld0, B.p1 ? B.ld1 : B.ld0, B.p1 ? B.split : INT64_MAX,
          B.gs0, B.p1 ? B.gs1 : B.gs0};
  const bool bf = dtype == GIST_DTYPE_BF16_IN;
  const bool av = op_vec_ok(A, M);
  const bool bv = op_vec_ok(B, N);
  const bool narrow = !bf && N <= BN / 2;
  dim3 grid(static_cast<unsigned>(groups));
  {
    // variant name: dtype, the K-contiguous (K) / row-contiguous (R)
    // orientation of A and B as read from memory, whether each is read
    // with 16-byte vector loads (v) or scalar loads (s), and _n for the
    // narrow split -- one name per kernel instantiation
    char name[32];
    snprintf(name, sizeof(name), "gemm_%s_%c%c_%c%c%s", bf ? "bf16" : "f32",
             A.k_major ? 'K' : 'R', B.k_major ? 'K' : 'R', av ? 'v' : 's', bv ? 'v' : 's',
             narrow ? "_n" : "");
    const double md = static_cast<double>(M), nd = static_cast<double>(N),
                 kd = static_cast<double>(k_alg > 0 ? k_alg : K);
    const double gd = static_cast<double>(ngroups);
    ProfScope ps(st, name, 2.0 * md * nd * kd * gd, 4.0 * (md * kd + kd * nd + md * nd) * gd);
    if (bf) dispatch<true, false>(st, A, B, av, bv, grid, M, N, K, a, b, c, S, part);
    else if (narrow) dispatch<false, true>(st, A, B, av, bv, grid, M, N, K, a, b, c, S, part);
    else dispatch<false, false>(st, A, B, av, bv, grid, M, N, K, a, b, c, S, part);
  }
  {
    gist_status s = check_launch("gemm");
    if (s != GIST_OK) return s;
  }
  if (split) {
    ProfScope ps(st, "gemm_streamk_fixup", 0.0,
                 4.0 * static_cast<double>(groups) * 2 * BM * BN + 4.0 * M * N * ngroups);
    hipLaunchKernelGGL(streamk_fixup, dim3(static_cast<unsigned>(tiles), kFixChunks), dim3(256), 0,
                       st, M, N, S, part, c);
    return check_launch("gemm stream-K fix-up");
  }
  return GIST_OK;
}

}  // namespace gist
