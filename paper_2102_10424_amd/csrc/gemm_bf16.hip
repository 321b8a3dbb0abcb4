// bf16-input GEMM for large products: operands rounded to bf16 (nearest
// even), multiplied on the bf16 MFMA units with fp32 accumulation, in
// 256 x 256 tiles.
//
//   1. The product kernel: eight waves (two per SIMD, so one wave's MFMAs
//      run while the other waits on memory), each owning 128 rows x 64
//      columns (4 x 2 MFMA tiles of 32 x 32, v_mfma_f32_32x32x16_bf16), K
//      steps of 32, three LDS tile buffers [row][k] with 64-byte rows
//      whose 16-byte chunks are XOR-swizzled so that neither the staging
//      writes nor the fragment reads meet bank conflicts, the next step's
//      operands loaded into registers while the current one multiplies.
//   2. Direct staging (the usual path): each step's operand tiles are read
//      straight from the fp32 operands and rounded in registers on their way
//      to LDS -- K-contiguous operands with 16-byte loads, row-contiguous
//      ones with one row per lane (256 contiguous bytes per wave load),
//      written K-major into the tile either way.  No conversion pass and no
//      bf16 copies: each operand byte is read once from memory per tile that
//      uses it, instead of read, written as bf16 and read back.
//   3. Packed staging (operands the direct loads cannot take: K not a
//      multiple of 32 for a K-contiguous operand, unaligned bases, a
//      concatenation split inside a tile): cvt_bf16_kernel first rounds
//      each operand into a zero-padded K-contiguous bf16 copy [Rp][Kp]
//      (row-contiguous ones transposed through LDS), which the same product
//      kernel then reads.
//   4. Work units are (K slice, tile) pairs, K-slice-major, so the units an
//      XCD runs together cover neighbouring tiles over the same K range at
//      the same time and share their operands in L2.  Shapes with too few
//      tiles to fill the GPU split K into up to kMaxSplit slices whose fp32
//      partials a fix-up kernel sums in slice order (deterministic).
//
// Both stagings put the same bf16 values in the same LDS tiles and run the
// same MFMA sequence, so they give bitwise the same result.

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

constexpr int TM = 256, TN = 256, TK = 32;
constexpr int LDH = TK;              // LDS row stride in halves (64 B, swizzled)
constexpr int kThr = 512;            // 8 waves: 2 along M x 4 along N
constexpr int kCUs = 256;            // MI355X compute units (one workgroup each)
constexpr int kMaxSplit = 8;
constexpr int kPad = 256;            // row padding of the bf16 copies (tile edge)
constexpr int kPadK = 64;            // K padding (conversion tile)

// Workgroup barrier that orders LDS only: waits for this wave's LDS
// accesses, not its global loads, so prefetches stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ unsigned short bf16_bits(float f) {
  return __builtin_bit_cast(unsigned short, static_cast<__bf16>(f));
}

// ---- 1. conversion ---------------------------------------------------------

// dst[r][k] = bf16(src(r, k)) for r < Rp, k < Kp; zero outside R x K.
// One 64 x 64 tile per block.  K-contiguous sources go straight from
// registers to the packed rows; row-contiguous ones are transposed through
// LDS.  VEC: 16-byte source loads (strides, bases and the concatenation
// split are multiples of 4 floats, and the contiguous extent is too, so a
// group of four is wholly inside or outside the matrix).
template <bool KMAJ, bool VEC>
__global__ __launch_bounds__(256) void cvt_bf16_kernel(OpView src, int64_t R, int64_t K,
                                                       unsigned short* __restrict__ dst,
                                                       int64_t Kp, int64_t tiles_k) {
  const int64_t tr = blockIdx.x / tiles_k, tk = blockIdx.x % tiles_k;
  const int64_t r0 = tr * 64, k0 = tk * 64;
  const int t = threadIdx.x;
  const int rr = t >> 2, kk = (t & 3) * 16;   // output: row rr, K kk .. kk+15
  float v[16];
  if constexpr (KMAJ) {
    const int64_t r = r0 + rr;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int64_t k = k0 + kk + 4 * g;
      if constexpr (VEC) {
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (r < R && k < K) x = src.at4<true>(r, k);
        v[4 * g] = x.x; v[4 * g + 1] = x.y; v[4 * g + 2] = x.z; v[4 * g + 3] = x.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * g + q] = (r < R && k + q < K) ? src.at<true>(r, k + q) : 0.f;
      }
    }
  } else {
    __shared__ float tile[64][65];   // [r][k]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = t + 256 * i;
      const int lk = e >> 4, lr = (e & 15) * 4;   // consecutive threads along R
      const int64_t k = k0 + lk, r = r0 + lr;
      if constexpr (VEC) {
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (k < K && r < R) x = src.at4<false>(r, k);
        tile[lr][lk] = x.x; tile[lr + 1][lk] = x.y; tile[lr + 2][lk] = x.z; tile[lr + 3][lk] = x.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) tile[lr + q][lk] = (k < K && r + q < R) ? src.at<false>(r + q, k) : 0.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = tile[rr][kk + q];
  }
  ushort8 lo, hi;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    lo[q] = bf16_bits(v[q]);
    hi[q] = bf16_bits(v[8 + q]);
  }
  unsigned short* d = dst + (r0 + rr) * Kp + k0 + kk;
  *reinterpret_cast<ushort8*>(d) = lo;
  *reinterpret_cast<ushort8*>(d + 8) = hi;
}

// ---- 2. the product ----------------------------------------------------------

struct SchedB {
  int64_t tiles;          // tiles_m * tiles_n
  int tiles_m, tiles_n;
  int nk;                 // K steps of the whole product
  int split;              // K slices
  int spu;                // K steps per slice
};

typedef float float2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef unsigned uint4v __attribute__((ext_vector_type(4)));

// Two values to packed bf16 (a in the low half), rounded to nearest even.
__device__ __forceinline__ unsigned bf16_pair(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector((float2v){a, b}, bf16x2));
}
__device__ __forceinline__ uint4v pack8(const float* v) {
  uint4v u;
#pragma unroll
  for (int i = 0; i < 4; ++i) u[i] = bf16_pair(v[2 * i], v[2 * i + 1]);
  return u;
}

// LDS tiles [row][k]: 64-byte rows of four 16-byte chunks (8 K each), chunk
// q of row r stored at position q ^ ((r ^ (r >> 2)) & 3).  With this
// swizzle the three access patterns -- staging writes with four lanes per
// row (chunks 0..3 of 16 rows), staging writes with one row per lane (64
// rows, one chunk) and MFMA fragment reads (32 rows, one chunk) -- each put
// every group of lanes the LDS serves together on distinct banks, whether
// it serves 8 lanes of 16 bytes over 32 banks or 16 lanes over 64.  (Padded
// 80-byte rows left the four-lanes-per-row writes with bank conflicts.)
__device__ __forceinline__ int lds_at(int row, int q) {
  return row * LDH + 8 * (q ^ ((row ^ (row >> 2)) & 3));
}

// Lane map of K-contiguous staging: rows (t >> 2) + 128 i, chunk t & 3.  Four
// consecutive lanes read one row's 64 contiguous bytes (bf16) or 128 (fp32),
// which the load unit merges into whole cache lines.
__device__ __forceinline__ int kstage_row(int t) { return t >> 2; }
__device__ __forceinline__ int kstage_q(int t) { return t & 3; }

// Staging of one operand's 256 x 32 tile per K step: `load` fetches this
// thread's share from memory into registers, `store` writes it to the LDS
// tile [row][k] (the lds_at layout) as bf16.

// From a padded bf16 copy [Rp][Kp]: rows kstage_row(t) + 128 i, K chunk kstage_q(t).
struct PackedOp {
  const unsigned short* p;
  int64_t Kp;
};
struct PackedStage {
  ushort8 r[2];
  const unsigned short* row;   // this thread's first row, at its K offset
  __device__ __forceinline__ void init(const PackedOp& o, int64_t, int64_t, int64_t r0, int t) {
    row = o.p + (r0 + kstage_row(t)) * o.Kp + 8 * kstage_q(t);
  }
  __device__ __forceinline__ void load(const PackedOp& o, int64_t k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
      r[i] = *reinterpret_cast<const ushort8*>(row + 128 * i * o.Kp + k0);
  }
  __device__ __forceinline__ void store(unsigned short* S, int t) const {
#pragma unroll
    for (int i = 0; i < 2; ++i)
      *reinterpret_cast<ushort8*>(S + lds_at(kstage_row(t) + 128 * i, kstage_q(t))) = r[i];
  }
};

// Straight from the fp32 operand, rounded to bf16 (nearest even) on the way
// to LDS.  Rows past the operand's end read its last rows (they only feed
// output rows or columns that are never stored).  Each thread's rows are
// fixed for the whole product, so their offsets are formed once, as 32-bit
// byte offsets from a per-step base that is the same for the whole wave
// (scalar address arithmetic, one vector register per load address).
template <bool KMAJ>
struct DirectStage;

// K contiguous: rows kstage_row(t) + 128 i, K chunk kstage_q(t) (two
// 16-byte loads per row).  Needs K and the concatenation split to be multiples of
// the K step (every step full and on one side of the split), leading
// dimensions that are multiples of 4 floats and 16-byte bases.
template <>
struct DirectStage<true> {
  float4 x[4];                 // row i: x[2i], x[2i+1] (K kc .. kc+7)
  unsigned off0[2], off1[2];   // byte offsets of this thread's rows in p0 / p1
  __device__ __forceinline__ void init(const OpView& o, int64_t R, int64_t, int64_t r0, int t) {
    const int kc = 8 * kstage_q(t);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int64_t r = min(r0 + kstage_row(t) + 128 * i, R - 1);
      off0[i] = static_cast<unsigned>((r * o.ld0 + kc) * 4);
      off1[i] = static_cast<unsigned>((r * o.ld1 + kc) * 4);
    }
  }
  __device__ __forceinline__ void load(const OpView& o, int64_t k0) {
    const bool first = k0 < o.split;
    const char* base = reinterpret_cast<const char*>(first ? o.p0 + k0 : o.p1 + (k0 - o.split));
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const char* q = base + (first ? off0[i] : off1[i]);
      x[2 * i] = *reinterpret_cast<const float4*>(q);
      x[2 * i + 1] = *reinterpret_cast<const float4*>(q + 16);
    }
  }
  __device__ __forceinline__ void store(unsigned short* S, int t) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const float4 a = x[2 * i], b = x[2 * i + 1];
      const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      *reinterpret_cast<uint4v*>(S + lds_at(kstage_row(t) + 128 * i, kstage_q(t))) = pack8(v);
    }
  }
};

// Row-contiguous: row t & 255, K (t >> 8) * 16 .. +15 (the same sixteen K
// for the whole wave), one 4-byte load per K, so that each wave's load
// covers 256 contiguous bytes and every loaded value sits in a register of
// its own (pairs or quads of loaded values that the conversion does not use
// together would make the compiler move them across the loop, waiting for
// the loads).  Two 16-byte LDS writes per thread fill the [row][k] tile.
// K past the end reads zero.  Needs a concatenation split on a tile
// boundary (a tile on one side of it).
template <>
struct DirectStage<false> {
  float v[16];   // K kc + i of this thread's row
  const float* p;
  int64_t ld, kend, kl;
  unsigned off;   // byte offset of this thread's row
  int kc;
  __device__ __forceinline__ void init(const OpView& o, int64_t R, int64_t K, int64_t r0, int t) {
    const bool first = r0 < o.split;
    p = first ? o.p0 : o.p1;
    ld = first ? o.ld0 : o.ld1;
    const int64_t r = min(r0 + (t & 255), R - 1);
    off = static_cast<unsigned>((first ? r : r - o.split) * 4);
    kc = __builtin_amdgcn_readfirstlane((t >> 8) * 16);
    kend = K;
  }
  __device__ __forceinline__ void load(const OpView&, int64_t k0) {
    kl = k0;
    // K rows kb .. kb+15, those past the end clamped to the last one: one
    // 64-bit base per step and a 32-bit step per row, no branch (a branch
    // here would make the compiler wait for the loads where its paths join)
    const int64_t kb = k0 + kc;
    const char* base = reinterpret_cast<const char*>(p + kb * ld);
    const int last = static_cast<int>(kend - 1 - kb);   // >= -31
    const int ld4 = static_cast<int>(ld * 4);
#pragma unroll
    for (int i = 0; i < 16; ++i)
      v[i] = *reinterpret_cast<const float*>(base + min(i, last) * ld4 + off);
  }
  // The zeros past K are applied here, where the loaded values are first
  // used, so that the loads stay in flight until then.
  __device__ __forceinline__ void store(unsigned short* S, int t) const {
    const int r = t & 255, q = (t >> 8) * 2;
    uint4v* d0 = reinterpret_cast<uint4v*>(S + lds_at(r, q));
    uint4v* d1 = reinterpret_cast<uint4v*>(S + lds_at(r, q + 1));
    if (kl + kc + 15 < kend) {
      *d0 = pack8(&v[0]);
      *d1 = pack8(&v[8]);
      return;
    }
    float w[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) w[i] = kl + kc + i < kend ? v[i] : 0.f;
    *d0 = pack8(&w[0]);
    *d1 = pack8(&w[8]);
  }
};

// Padded bf16 copies need no set-up.
// One work unit (K slice, 256 x 256 tile) of C = A B^T with A staged by SA
// from OA and B by SB from OB.
template <class SA, class SB, class OA, class OB, bool SPLIT_OUT>
__device__ __forceinline__ void gemm_bf16_body(int64_t M, int64_t N, int64_t K, const OA& A,
                                               const OB& B, const OutView& C, const SchedB& S,
                                               float* __restrict__ partials) {
  __shared__ __attribute__((aligned(16))) unsigned short lds[3][(TM + TN) * LDH];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int li = lane & 31, lh = lane >> 5;
  const int wm = wave >> 2, wn = wave & 3;   // this wave's 128 x 64 block of the tile

  const int64_t u = xcd_remap(blockIdx.x, gridDim.x);
  const int ks = static_cast<int>(u / S.tiles);
  const int64_t tile = u - static_cast<int64_t>(ks) * S.tiles;
  int tm, tn;
  tile_coords_banded(tile, S.tiles_m, S.tiles_n, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * TM, n0 = static_cast<int64_t>(tn) * TN;
  const int kb = ks * S.spu;
  const int ke = min(S.nk, kb + S.spu);

  floatx16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  SA sa;
  SB sb;
  sa.init(A, M, K, m0, t);
  sb.init(B, N, K, n0, t);
  auto gload = [&](int64_t k) {
    sa.load(A, k);
    sb.load(B, k);
  };
  auto swrite = [&](int buf) {
    sa.store(lds[buf], t);
    sb.store(lds[buf] + TM * LDH, t);
  };
  // MFMA fragments of one 16-wide K chunk: A rows wm*128 + a*32 + lane%32,
  // B rows wn*64 + b*32 + lane%32; lane half lh holds K elements 8*lh .. +7.
  struct Frag { bf16x8 a[4], b[2]; };
  auto rfrag = [&](int buf, int c, Frag& f) {
    const unsigned short* As = lds[buf];
    const unsigned short* Bs = As + TM * LDH;
#pragma unroll
    for (int a = 0; a < 4; ++a)
      f.a[a] = *reinterpret_cast<const bf16x8*>(As + lds_at(wm * 128 + a * 32 + li, 2 * c + lh));
#pragma unroll
    for (int b = 0; b < 2; ++b)
      f.b[b] = *reinterpret_cast<const bf16x8*>(Bs + lds_at(wn * 64 + b * 32 + li, 2 * c + lh));
  };
  auto mfma8 = [&](const Frag& f) {
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
  };

  // Pipeline over three LDS buffers (32 KB each), step j in buffer
  // (j - kb) % 3, written two steps ahead:
  //   - chunk 0's fragments of step j were read during step j-1; chunk 1's
  //     are read while chunk 0 multiplies;
  //   - then step j+2's staging registers (loaded during step j-1) go to the
  //     buffer step j-1 used -- whose reads all completed before the barrier
  //     that ended step j-1 -- and are reloaded at once with step j+3, a
  //     whole step before they are needed again;
  //   - chunk 0 of step j+1 is read from its buffer, whole since that same
  //     barrier, while chunk 1 multiplies; the barrier ends the step.
  // So no wave waits for fragments after a barrier, and the barrier sits
  // after both chunks.
  gload(static_cast<int64_t>(kb) * TK);
  swrite(0);
  if (kb + 1 < ke) {
    gload(static_cast<int64_t>(kb + 1) * TK);
    swrite(1);
  }
  if (kb + 2 < ke) gload(static_cast<int64_t>(kb + 2) * TK);
  __syncthreads();
  Frag f0, f1;
  rfrag(0, 0, f0);
  int cur = 0;
  for (int j = kb; j < ke; ++j) {
    const int nxt = cur == 2 ? 0 : cur + 1;
    const int prev = nxt == 2 ? 0 : nxt + 1;   // the buffer step j-1 used
    rfrag(cur, 1, f1);
    __builtin_amdgcn_sched_barrier(0);
    // chunk 0's MFMAs interleaved with the staging work (conversion, LDS
    // writes, next loads, next fragment reads): the two waves of a SIMD
    // reach this phase together, so staging work left between the chunks
    // would leave the matrix core idle
    mfma8(f0);
    // unconditional: on the last two steps these write a buffer no later
    // step reads and read one whose fragments go unused, and a branch here
    // would leave the LDS counter unknown where the paths join, so that the
    // compiler would wait for these reads before chunk 1
    swrite(prev);
    if (j + 3 < ke) gload(static_cast<int64_t>(j + 3) * TK);
    rfrag(nxt, 0, f0);
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);   // up to six VALU
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);   // an LDS write
      __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);   // up to four loads
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // an LDS read
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma8(f1);
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    cur = nxt;
  }

  // acc[a][b] register r of lane l: tile row wm*128 + a*32 + 8(r/4) +
  // 4(l/32) + r%4, tile column wn*64 + b*32 + l%32
  if (S.split == 1 && C.sgd) {
    // fused SGD step, C <- fmaf(-lr, acc, C): the weights of the next 32 x 32
    // sub-tile are read while the current one is written, so a tile waits for
    // memory once, not once per weight
    float w[2][16];
    auto fetch = [&](int t, float (&dst)[16]) {
      const int a = t >> 1, b = t & 1;
      const int64_t col = n0 + wn * 64 + b * 32 + li;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * 128 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        dst[r] = (row < M && col < N) ? *C.ptr<SPLIT_OUT>(row, col) : 0.f;
      }
    };
    fetch(0, w[0]);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      if (t + 1 < 8) fetch(t + 1, w[(t + 1) & 1]);
      const int a = t >> 1, b = t & 1;
      const int64_t col = n0 + wn * 64 + b * 32 + li;
      if (col >= N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * 128 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row < M) *C.ptr<SPLIT_OUT>(row, col) = fmaf(-C.lr, acc[a][b][r], w[t & 1][r]);
      }
    }
  } else if (S.split == 1) {
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int64_t col = n0 + wn * 64 + b * 32 + li;
        if (col >= N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = m0 + wm * 128 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
          if (row < M) C.store<SPLIT_OUT>(row, col, acc[a][b][r]);
        }
      }
  } else {
    float* part = partials + u * static_cast<int64_t>(TM * TN);   // slot (ks, tile)
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          part[(wm * 128 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3)) * TN + wn * 64 + b * 32 +
               li] = acc[a][b][r];
  }
}

// Both operands from their padded bf16 copies.
template <bool SPLIT_OUT>
__global__ __launch_bounds__(kThr) void gemm_bf16_kernel(int64_t M, int64_t N, int64_t K,
                                                         PackedOp A, PackedOp B, OutView C,
                                                         SchedB S, float* __restrict__ partials) {
  gemm_bf16_body<PackedStage, PackedStage, PackedOp, PackedOp, SPLIT_OUT>(M, N, K, A, B, C, S,
                                                                          partials);
}

// Both operands straight from fp32 memory (AK / BK: K contiguous).
template <bool AK, bool BK, bool SPLIT_OUT>
__global__ __launch_bounds__(kThr) void gemm_bf16_direct_kernel(int64_t M, int64_t N, int64_t K,
                                                                OpView A, OpView B, OutView C,
                                                                SchedB S,
                                                                float* __restrict__ partials) {
  gemm_bf16_body<DirectStage<AK>, DirectStage<BK>, OpView, OpView, SPLIT_OUT>(M, N, K, A, B, C,
                                                                              S, partials);
}

// Sum the K slices' partials of one tile in slice order.  One block per
// kFixRows rows of a tile (a tile alone would leave most CUs idle).
constexpr int kFixRows = 16;

__global__ __launch_bounds__(256) void fixup_bf16_kernel(int64_t M, int64_t N, SchedB S,
                                                         const float* __restrict__ partials,
                                                         OutView C) {
  constexpr int kChunks = TM / kFixRows;
  const int64_t tile = blockIdx.x / kChunks;
  const int r0 = static_cast<int>(blockIdx.x % kChunks) * kFixRows;
  int tm, tn;
  tile_coords_banded(tile, S.tiles_m, S.tiles_n, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * TM, n0 = static_cast<int64_t>(tn) * TN;
  const int64_t slot = static_cast<int64_t>(TM * TN);
#pragma unroll
  for (int i = 0; i < kFixRows * TN / 4 / 256; ++i) {
    const int e = r0 * TN + (threadIdx.x + 256 * i) * 4;
    const int64_t row = m0 + e / TN, col = n0 + e % TN;
    if (row >= M || col >= N) continue;
    floatx4 s = *reinterpret_cast<const floatx4*>(partials + tile * slot + e);
    for (int k = 1; k < S.split; ++k)
      s += *reinterpret_cast<const floatx4*>(partials + (k * S.tiles + tile) * slot + e);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (col + q < N) C.store<true>(row, col + q, s[q]);
  }
}

struct Layout {
  int64_t Mp, Np, Kp;
  size_t a_bytes, b_bytes, part_bytes;
  SchedB S;
  size_t total() const { return a_bytes + b_bytes + part_bytes; }
};

size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

// K slices for a product of `tiles` tiles and nk K steps: the fewest rounds
// of kCUs workgroups times the steps per slice, plus the fix-up's traffic
// (split + 1 partial tiles per output tile at ~4 TB/s) priced in K steps of
// one workgroup (~0.8 us each at the measured rate).
int choose_split(int64_t tiles, int nk) {
  int best = 1;
  double best_cost = 0.0;
  for (int s = 1; s <= kMaxSplit; ++s) {
    const int spu = (nk + s - 1) / s;
    if (s > 1 && (spu < 8 || (s - 1) * spu >= nk)) break;
    const double rounds = static_cast<double>((tiles * s + kCUs - 1) / kCUs);
    double cost = rounds * spu;
    if (s > 1) cost += static_cast<double>(tiles) * (s + 1) * TM * TN * 4.0 / 4e12 / 0.8e-6;
    if (s == 1 || cost < best_cost) { best = s; best_cost = cost; }
  }
  return best;
}

Layout make_layout(int64_t M, int64_t N, int64_t K) {
  Layout L;
  L.Mp = (M + kPad - 1) / kPad * kPad;
  L.Np = (N + kPad - 1) / kPad * kPad;
  L.Kp = (K + kPadK - 1) / kPadK * kPadK;
  L.a_bytes = up256(static_cast<size_t>(L.Mp) * L.Kp * 2);
  L.b_bytes = up256(static_cast<size_t>(L.Np) * L.Kp * 2);
  SchedB& s = L.S;
  s.tiles_m = static_cast<int>(L.Mp / TM);
  s.tiles_n = static_cast<int>(L.Np / TN);
  s.tiles = static_cast<int64_t>(s.tiles_m) * s.tiles_n;
  s.nk = static_cast<int>(L.Kp / TK);
  s.split = choose_split(s.tiles, s.nk);
  s.spu = (s.nk + s.split - 1) / s.split;
  L.part_bytes = s.split > 1 ? static_cast<size_t>(s.split) * s.tiles * TM * TN * sizeof(float) : 0;
  return L;
}

gist_status convert(hipStream_t st, const Operand& o, int64_t R, int64_t K, int64_t Rp,
                    int64_t Kp, unsigned short* dst) {
  OpView v = OpView::from(o);
  const int64_t tiles_k = Kp / 64;
  const int64_t blocks = (Rp / 64) * tiles_k;
  const bool vec = o.ld0 % 4 == 0 && aligned16(o.p0) &&
                   (!o.p1 || (o.ld1 % 4 == 0 && aligned16(o.p1) && o.split % 4 == 0)) &&
                   (o.k_major ? K % 4 == 0 : R % 4 == 0);
  ProfScope ps(st, o.k_major ? "cvt_bf16_K" : "cvt_bf16_R", 0.0,
               4.0 * static_cast<double>(R) * K + 2.0 * static_cast<double>(Rp) * Kp);
  const dim3 g(static_cast<unsigned>(blocks));
  if (o.k_major && vec)
    hipLaunchKernelGGL((cvt_bf16_kernel<true, true>), g, dim3(256), 0, st, v, R, K, dst, Kp, tiles_k);
  else if (o.k_major)
    hipLaunchKernelGGL((cvt_bf16_kernel<true, false>), g, dim3(256), 0, st, v, R, K, dst, Kp, tiles_k);
  else if (vec)
    hipLaunchKernelGGL((cvt_bf16_kernel<false, true>), g, dim3(256), 0, st, v, R, K, dst, Kp, tiles_k);
  else
    hipLaunchKernelGGL((cvt_bf16_kernel<false, false>), g, dim3(256), 0, st, v, R, K, dst, Kp,
                       tiles_k);
  return check_launch("bf16 conversion");
}

// The direct kernel's operand requirements (DirectStage), plus 32-bit byte
// offsets for every row it reads.
bool direct_ok(const Operand& o, int64_t R, int64_t K) {
  auto al = [](const float* p, unsigned a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; };
  const int64_t lim = int64_t(1) << 30;   // floats addressable by a 32-bit byte offset
  if (o.k_major) {
    if (K % TK || o.ld0 % 4 || !al(o.p0, 16) || R * o.ld0 >= lim) return false;
    return !o.p1 || (o.ld1 % 4 == 0 && al(o.p1, 16) && o.split % TK == 0 && R * o.ld1 < lim);
  }
  // (and K-row steps of +-31 leading dimensions within a 32-bit byte offset)
  const int64_t ldlim = int64_t(1) << 24;
  if (R >= lim || o.ld0 >= ldlim) return false;
  return !o.p1 || (o.ld1 < ldlim && o.split % TM == 0);
}

template <bool SPLIT_OUT>
void launch_direct(hipStream_t st, dim3 g, int64_t M, int64_t N, int64_t K, const Operand& A,
                   const Operand& B, const OutView& c, const SchedB& S, float* part) {
  const OpView a = OpView::from(A), b = OpView::from(B);
#define GIST_BF16_DIRECT(AK_, BK_)                                                        \
  hipLaunchKernelGGL((gemm_bf16_direct_kernel<AK_, BK_, SPLIT_OUT>), g, dim3(kThr), 0, st, M, \
                     N, K, a, b, c, S, part)
  if (A.k_major && B.k_major) GIST_BF16_DIRECT(true, true);
  else if (A.k_major) GIST_BF16_DIRECT(true, false);
  else if (B.k_major) GIST_BF16_DIRECT(false, true);
  else GIST_BF16_DIRECT(false, false);
#undef GIST_BF16_DIRECT
}

}  // namespace

bool gemm_bf16_packed_eligible(int64_t M, int64_t N, int64_t K) {
  // big enough for 256 x 256 tiles to pay
  return M >= 512 && N >= 512 && K >= 256;
}

size_t gemm_bf16_packed_workspace(int64_t M, int64_t N, int64_t K) {
  return make_layout(M, N, K).total();
}

gist_status gemm_bf16_packed(hipStream_t st, int64_t M, int64_t N, int64_t K, const Operand& A,
                             const Operand& B, const GemmOut& Cout, void* ws, size_t ws_bytes) {
  const Layout L = make_layout(M, N, K);
  if (!ws || ws_bytes < L.total()) return set_error(GIST_E_NOMEM, "gemm bf16: workspace too small");
  const int64_t units = L.S.tiles * L.S.split;
  if (units > INT32_MAX || L.S.tiles * (TM / kFixRows) > INT32_MAX || L.Kp / TK > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, "gemm bf16: grid too large");
  char* base = static_cast<char*>(ws);
  auto* a16 = reinterpret_cast<unsigned short*>(base);
  auto* b16 = reinterpret_cast<unsigned short*>(base + L.a_bytes);
  float* part = reinterpret_cast<float*>(base + L.a_bytes + L.b_bytes);
  OutView c = OutView::from(Cout);
  const bool split_out = Cout.c1 != nullptr;
  const dim3 g(static_cast<unsigned>(units));
  const double flops = 2.0 * static_cast<double>(M) * N * K;
  if (direct_ok(A, M, K) && direct_ok(B, N, K)) {
    // operands rounded while staged: no conversion pass, no bf16 copies
    // variant name: the K-contiguous (K) / row-contiguous (R) orientation of
    // A and B as read from memory
    static const char* const kNames[4] = {"gemm_bf16_direct_RR", "gemm_bf16_direct_RK",
                                          "gemm_bf16_direct_KR", "gemm_bf16_direct_KK"};
    ProfScope ps(st, kNames[(A.k_major ? 2 : 0) + (B.k_major ? 1 : 0)], flops,
                 4.0 * (static_cast<double>(M) * K + static_cast<double>(N) * K) +
                     4.0 * static_cast<double>(M) * N);
    if (split_out) launch_direct<true>(st, g, M, N, K, A, B, c, L.S, part);
    else launch_direct<false>(st, g, M, N, K, A, B, c, L.S, part);
  } else {
    gist_status s = convert(st, A, M, K, L.Mp, L.Kp, a16);
    if (s != GIST_OK) return s;
    s = convert(st, B, N, K, L.Np, L.Kp, b16);
    if (s != GIST_OK) return s;
    const PackedOp pa{a16, L.Kp}, pb{b16, L.Kp};
    ProfScope ps(st, "gemm_bf16_packed", flops,
                 2.0 * (static_cast<double>(M) * K + static_cast<double>(N) * K) +
                     4.0 * static_cast<double>(M) * N);
    if (split_out)
      hipLaunchKernelGGL(gemm_bf16_kernel<true>, g, dim3(kThr), 0, st, M, N, K, pa, pb, c, L.S,
                         part);
    else
      hipLaunchKernelGGL(gemm_bf16_kernel<false>, g, dim3(kThr), 0, st, M, N, K, pa, pb, c, L.S,
                         part);
  }
  gist_status s = check_launch("gemm bf16");
  if (s != GIST_OK) return s;
  if (L.S.split > 1) {
    ProfScope ps(st, "gemm_bf16_fixup", 0.0,
                 4.0 * static_cast<double>(L.S.split) * L.S.tiles * TM * TN +
                     4.0 * static_cast<double>(M) * N);
    hipLaunchKernelGGL(fixup_bf16_kernel, dim3(static_cast<unsigned>(L.S.tiles * (TM / kFixRows))),
                       dim3(256), 0, st, M, N, L.S, part, c);
    return check_launch("gemm bf16 fix-up");
  }
  return GIST_OK;
}

}  // namespace gist
