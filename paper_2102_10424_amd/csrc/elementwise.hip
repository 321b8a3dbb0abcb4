// Bandwidth-bound kernels of the step: ReLU derivative, softmax
// cross-entropy, slice gather (subGCNs), slice scatter (subAgg), SGD.

#include "common.cuh"
#include "gist_internal.h"

namespace gist {

namespace {

constexpr int kBlock = 256;

unsigned grid_for(int64_t work, int64_t per_block, int64_t cap = 1 << 20) {
  int64_t b = (work + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<unsigned>(b);
}

// dZ = dH * 1[Hout > 0]: the ReLU derivative, read from the layer output.
__global__ __launch_bounds__(kBlock) void relu_mask_kernel(int64_t count, const float* __restrict__ dH,
                                                           const float* __restrict__ Hout,
                                                           float* __restrict__ dZ, int vec) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  if (vec) {
    const int64_t c4 = count / 4;
    const float4* d4 = reinterpret_cast<const float4*>(dH);
    const float4* h4 = reinterpret_cast<const float4*>(Hout);
    float4* z4 = reinterpret_cast<float4*>(dZ);
    for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < c4; i += stride) {
      const float4 d = d4[i], h = h4[i];
      float4 z;
      z.x = h.x > 0.f ? d.x : 0.f;
      z.y = h.y > 0.f ? d.y : 0.f;
      z.z = h.z > 0.f ? d.z : 0.f;
      z.w = h.w > 0.f ? d.w : 0.f;
      z4[i] = z;
    }
    for (int64_t i = c4 * 4 + blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < count;
         i += stride)
      dZ[i] = Hout[i] > 0.f ? dH[i] : 0.f;
    return;
  }
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < count; i += stride)
    dZ[i] = Hout[i] > 0.f ? dH[i] : 0.f;
}

// W -= lr * dW with a single rounding per element.
__global__ __launch_bounds__(kBlock) void sgd_kernel(int64_t n, float* __restrict__ W,
                                                     const float* __restrict__ dW, float lr) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < n; i += stride)
    W[i] = fmaf(-lr, dW[i], W[i]);
}

// Adam: four elements per thread per pass (16-byte accesses when the four
// arrays are aligned), the scalar tail by the first threads.  step_size =
// lr / (1 - beta1^k) and inv_sqrt_bc2 = 1 / sqrt(1 - beta2^k) come from
// the host, so  W -= step_size m / (sqrt(v) inv_sqrt_bc2 + eps).
struct AdamCoef {
  float step_size, inv_sqrt_bc2, beta1, beta2, eps;
};

__device__ __forceinline__ void adam_one(float& w, float g, float& m, float& v, const AdamCoef& c,
                                         bool fresh) {
  const float m0 = fresh ? 0.f : m, v0 = fresh ? 0.f : v;
  m = c.beta1 * m0 + (1.f - c.beta1) * g;
  v = c.beta2 * v0 + (1.f - c.beta2) * (g * g);
  w = w - c.step_size * m / (sqrtf(v) * c.inv_sqrt_bc2 + c.eps);
}

// coef_dev (optional): {step_size, inv_sqrt_bc2, fresh} read from device
// memory instead of the arguments, so that a replayed step advances them.
template <bool VEC4>
__global__ __launch_bounds__(kBlock) void adam_kernel(int64_t n, float* __restrict__ W,
                                                      const float* __restrict__ dW,
                                                      float* __restrict__ M, float* __restrict__ V,
                                                      AdamCoef c, int fresh,
                                                      const float* __restrict__ coef_dev) {
  if (coef_dev) {
    c.step_size = coef_dev[0];
    c.inv_sqrt_bc2 = coef_dev[1];
    fresh = coef_dev[2] != 0.f;
  }
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  const int64_t t0 = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if constexpr (VEC4) {
    const int64_t n4 = n / 4;
    for (int64_t i = t0; i < n4; i += stride) {
      float4 w = reinterpret_cast<float4*>(W)[i], m = reinterpret_cast<float4*>(M)[i],
             v = reinterpret_cast<float4*>(V)[i];
      const float4 g = reinterpret_cast<const float4*>(dW)[i];
      adam_one(w.x, g.x, m.x, v.x, c, fresh);
      adam_one(w.y, g.y, m.y, v.y, c, fresh);
      adam_one(w.z, g.z, m.z, v.z, c, fresh);
      adam_one(w.w, g.w, m.w, v.w, c, fresh);
      reinterpret_cast<float4*>(W)[i] = w;
      reinterpret_cast<float4*>(M)[i] = m;
      reinterpret_cast<float4*>(V)[i] = v;
    }
    if (t0 < n - 4 * n4) {
      const int64_t i = 4 * n4 + t0;
      adam_one(W[i], dW[i], M[i], V[i], c, fresh);
    }
  } else {
    for (int64_t i = t0; i < n; i += stride) adam_one(W[i], dW[i], M[i], V[i], c, fresh);
  }
}

// One block per output row; threads stride over the row's columns.  The
// global row is read in ascending column order, so the lines of a row are
// streamed once.
__global__ __launch_bounds__(kBlock) void gather_kernel(const float* __restrict__ Wg, int64_t ldg,
                                                        const int* __restrict__ rows, int nr,
                                                        const int* __restrict__ cols, int nc,
                                                        float* __restrict__ Ws, int64_t lds) {
  const int64_t i = xcd_remap(blockIdx.x, gridDim.x);
  if (i >= nr) return;
  const int64_t r = rows ? rows[i] : i;
  const float* src = Wg + r * ldg;
  float* dst = Ws + i * lds;
  if (cols) {
    for (int j = threadIdx.x; j < nc; j += kBlock) dst[j] = src[cols[j]];
  } else {
    for (int j = threadIdx.x; j < nc; j += kBlock) dst[j] = src[j];
  }
}

__global__ __launch_bounds__(kBlock) void scatter_kernel(float* __restrict__ Wg, int64_t ldg,
                                                         const int* __restrict__ rows, int nr,
                                                         const int* __restrict__ cols, int nc,
                                                         const float* __restrict__ Ws, int64_t lds) {
  const int64_t i = xcd_remap(blockIdx.x, gridDim.x);
  if (i >= nr) return;
  const int64_t r = rows ? rows[i] : i;
  float* dst = Wg + r * ldg;
  const float* src = Ws + i * lds;
  if (cols) {
    for (int j = threadIdx.x; j < nc; j += kBlock) dst[cols[j]] = src[j];
  } else {
    for (int j = threadIdx.x; j < nc; j += kBlock) dst[j] = src[j];
  }
}

// Wg[r][c] = mean over the m slices, summed in double in slice order.
__global__ __launch_bounds__(kBlock) void subagg_mean_kernel(float* __restrict__ Wg, int64_t rows,
                                                             int64_t cols, int64_t ldg, int m,
                                                             const float* const* __restrict__ slices,
                                                             int64_t lds) {
  const int64_t count = rows * cols;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; e < count; e += stride) {
    const int64_t r = e / cols, c = e - r * cols;
    double s = 0.0;
    for (int i = 0; i < m; ++i) s += static_cast<double>(slices[i][r * lds + c]);
    Wg[r * ldg + c] = static_cast<float>(s / m);
  }
}

__global__ __launch_bounds__(kBlock) void zero_kernel(float* __restrict__ p, int64_t count) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < count; i += stride)
    p[i] = 0.f;
}

__global__ void zero_int_kernel(int* p) {
  if (threadIdx.x == 0 && blockIdx.x == 0) p[0] = 0;
}

// dst (cols x rows, leading dimension ldd) = transpose of src (rows x cols,
// leading dimension lds), through a 64 x 65 LDS tile (the extra column keeps
// the column reads of the tile free of bank conflicts), and zeros in columns
// rows .. ldd-1 of every dst row.  Both the reads and the writes go along the
// contiguous dimension, 64 floats per wave row.
__global__ __launch_bounds__(kBlock) void transpose_kernel(const float* __restrict__ src,
                                                           int64_t rows, int64_t cols,
                                                           int64_t lds, float* __restrict__ dst,
                                                           int64_t ldd) {
  __shared__ float tile[64][65];
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += kBlock / 64) {
    const int64_t r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = src[r * lds + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += kBlock / 64) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < cols && r < ldd) dst[c * ldd + r] = r < rows ? tile[tx][i] : 0.f;
  }
}

// The same with 16-byte accesses on both sides (lds, cols and ldd multiples of
// 4 floats, 16-byte aligned bases): a thread loads four consecutive columns
// of a source row and stores four consecutive entries of a destination row
// (rows past `rows` as zeros), so each wave moves whole 256-byte runs.
__global__ __launch_bounds__(kBlock) void transpose4_kernel(const float* __restrict__ src,
                                                            int64_t rows, int64_t cols,
                                                            int64_t lds, float* __restrict__ dst,
                                                            int64_t ldd) {
  __shared__ float tile[64][65];
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int q = threadIdx.x & 15, g = threadIdx.x >> 4;   // 16 float4 per 64-float row
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lr = g + 16 * i;
    const int64_t r = r0 + lr, c = c0 + 4 * q;
    if (r < rows && c < cols) {   // cols % 4 == 0: the four columns are all in
      const float4 v = *reinterpret_cast<const float4*>(src + r * lds + c);
      tile[lr][4 * q] = v.x;
      tile[lr][4 * q + 1] = v.y;
      tile[lr][4 * q + 2] = v.z;
      tile[lr][4 * q + 3] = v.w;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lc = g + 16 * i;
    const int64_t c = c0 + lc, r = r0 + 4 * q;
    if (c < cols && r < ldd) {    // ldd % 4 == 0: the four entries are all in
      float4 o;
      o.x = r < rows ? tile[4 * q][lc] : 0.f;
      o.y = r + 1 < rows ? tile[4 * q + 1][lc] : 0.f;
      o.z = r + 2 < rows ? tile[4 * q + 2][lc] : 0.f;
      o.w = r + 3 < rows ? tile[4 * q + 3][lc] : 0.f;
      *reinterpret_cast<float4*>(dst + c * ldd + r) = o;
    }
  }
}

// Copy of `n16` 16-byte words, then `tail` single bytes, from `src` (which
// may be pinned host memory: the reads then cross the host link) to `dst`.
__global__ __launch_bounds__(kBlock) void pull_kernel(uint4* __restrict__ dst,
                                                      const uint4* __restrict__ src, int64_t n16,
                                                      int64_t tail) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  const int64_t t0 = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  for (int64_t i = t0; i < n16; i += stride) dst[i] = src[i];
  if (t0 < tail)
    reinterpret_cast<unsigned char*>(dst + n16)[t0] =
        reinterpret_cast<const unsigned char*>(src + n16)[t0];
}

__global__ __launch_bounds__(kBlock) void pull_bytes_kernel(unsigned char* __restrict__ dst,
                                                            const unsigned char* __restrict__ src,
                                                            int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

__global__ __launch_bounds__(kBlock) void nonfinite_kernel(const float* __restrict__ Ws, int64_t lds,
                                                           int nr, int nc, int* flag) {
  const int64_t total = static_cast<int64_t>(nr) * nc;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  int bad = 0;
  for (int64_t t = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; t < total; t += stride) {
    const float v = Ws[(t / nc) * lds + (t % nc)];
    bad |= !isfinite(v);
  }
  if (bad) atomicOr(flag, 1);
}

// Softmax cross-entropy: one wave per row (classes strided over lanes);
// per-block partial sums of the row losses, summed in order afterwards.
// Rows at or past the valid count (n, or *n_dev when given, clamped to
// [0, n]) are padding: their gradient rows are zero and they add nothing.
__device__ __forceinline__ int valid_rows(int n, const int* n_dev) {
  if (!n_dev) return n;
  const int v = *n_dev;
  return v < 0 ? 0 : (v > n ? n : v);
}

__global__ __launch_bounds__(kBlock) void xent_rows_kernel(int n, int C,
                                                           const float* __restrict__ Z,
                                                           const int* __restrict__ y,
                                                           float* __restrict__ dZ,
                                                           float* __restrict__ partials,
                                                           const int* __restrict__ n_dev) {
  __shared__ float wloss[kBlock / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave;
  const int nv = valid_rows(n, n_dev);
  float row_loss = 0.f;
  if (row >= nv && row < n) {
    for (int j = lane; j < C; j += 64) dZ[row * C + j] = 0.f;
  } else if (row < n) {
    const float* z = Z + row * C;
    float* g = dZ + row * C;
    const int label = y[row];
    float mx = -INFINITY;
    for (int j = lane; j < C; j += 64) mx = fmaxf(mx, z[j]);
    mx = wave_max(mx);
    float s = 0.f;
    for (int j = lane; j < C; j += 64) s += expf(z[j] - mx);
    s = wave_sum(s);
    const float lse = mx + logf(s);
    const float inv_n = 1.0f / static_cast<float>(nv);
    float zy = 0.f;
    for (int j = lane; j < C; j += 64) {
      const float p = expf(z[j] - lse);
      g[j] = (p - (j == label ? 1.f : 0.f)) * inv_n;
      if (j == label) zy = z[j];
    }
    zy = wave_sum(zy);
    row_loss = (label >= 0 && label < C) ? lse - zy : __int_as_float(0x7fc00000);
  }
  if (lane == 0) wloss[wave] = row_loss;
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int w = 0; w < kBlock / 64; ++w) s += wloss[w];
    partials[blockIdx.x] = s;
  }
}

__global__ __launch_bounds__(kBlock) void xent_finish_kernel(int nparts, const float* __restrict__ partials,
                                                             int n, float* loss,
                                                             const int* __restrict__ n_dev) {
  n = valid_rows(n, n_dev);
  __shared__ float sh[kBlock];
  float s = 0.f;
  for (int i = threadIdx.x; i < nparts; i += kBlock) s += partials[i];
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int o = kBlock / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = n > 0 ? sh[0] / static_cast<float>(n) : 0.f;
}


// subAgg of one round fused with the gather of the next.  One block per
// (row, 4*kBlock-column chunk) of the global matrix, one 4-column group per
// thread and no loop: every load a thread issues (the matrix, the columns'
// ranks, the trained values) is independent of its stores, so the latency
// chain is paid once per thread and hidden by the other resident waves.
// Every entry owned by a sub-GCN of `done` takes its trained value, the
// group is written back whole (full-line writes), and the entries owned by
// a sub-GCN of `next` are copied into its slice.
//
// A partitioned row belongs to one block b, found once per thread; its
// slice row and block b's column-rank range [col_offs[b], col_offs[b+1])
// then place each column with one compare.  Only an unpartitioned row (the
// input width at layer 0) looks up each column's block.
struct SliceSetDev {
  const int* row_rank;
  const int64_t* row_offs;
  const int* col_rank;
  const int64_t* col_offs;
  float* const* slices;
  int64_t ld;
};

// Block b of a partition with offs[b] <= k < offs[b+1] (empty blocks allowed).
__device__ __forceinline__ int block_of(const int64_t* offs, int m, int64_t k) {
  int lo = 0, hi = m;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (offs[mid] <= k) lo = mid; else hi = mid;
  }
  return lo;
}

struct RowSel {
  float* base;     // partitioned row: its row in the owner's slice
  int64_t lo, hi;  // the owner's column-rank range
};

__device__ __forceinline__ RowSel row_select(const SliceSetDev& s, int m, int64_t r) {
  RowSel q{nullptr, 0, 0};
  if (s.row_rank) {
    const int64_t kr = s.row_rank[r];
    const int b = block_of(s.row_offs, m, kr);
    q.base = s.slices[b] + (kr - s.row_offs[b]) * s.ld;
    if (s.col_rank) { q.lo = s.col_offs[b]; q.hi = s.col_offs[b + 1]; }
  }
  return q;
}

// Address of element (r, c), column rank kc, in its owner's slice; nullptr
// when no sub-GCN owns it.
__device__ __forceinline__ float* slot_of(const SliceSetDev& s, int m, const RowSel& q, int64_t r,
                                          int64_t c, int kc) {
  if (s.row_rank) {
    if (!s.col_rank) return q.base + c;
    return (kc >= q.lo && kc < q.hi) ? q.base + (kc - q.lo) : nullptr;
  }
  if (!s.col_rank) return s.slices[0] + r * s.ld + c;   // m == 1
  const int b = block_of(s.col_offs, m, kc);
  return s.slices[b] + r * s.ld + (kc - s.col_offs[b]);
}

template <bool VEC4>
__device__ __forceinline__ void ranks4(const int* rank, int64_t c0, int nq, int (&k)[4]) {
  if (!rank) {
#pragma unroll
    for (int q = 0; q < 4; ++q) k[q] = 0;
    return;
  }
  if constexpr (VEC4) {
    const int4 t = *reinterpret_cast<const int4*>(rank + c0);
    k[0] = t.x; k[1] = t.y; k[2] = t.z; k[3] = t.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) k[q] = q < nq ? rank[c0 + q] : 0;
  }
}

__device__ __forceinline__ int wave_min_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ int wave_max_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}

// Fast path, used when every given set partitions the rows and the widths
// are float4-aligned.  A row then has one owner per set, and the columns it
// owns are block b's members: with ascending blocks (as gist_partition
// returns them) the owned columns inside one wave's 256 consecutive columns
// are consecutive members, i.e. one contiguous run of slice positions.  The
// gather half stages that run in LDS at (position - first) and stores it
// with consecutive lanes instead of one sparse store per column; a wave
// whose owned positions are not contiguous stores them one by one.
//
// A block covers kRowChunks chunks of 1024 columns of one row: every
// thread issues its kRowChunks Theta loads before the row's owner is
// resolved (a chain of dependent loads: rank, block search, slice
// pointer), which is done once per block, so each block keeps 16 KB in
// flight behind one latency chain.
constexpr int kRowChunks = 4;
// The model's rows are read once and written once per pass (gigabytes):
// non-temporal accesses keep them from displacing cached data (the slice
// index tables, the staged runs); 1.91 against 1.98 ms per c4 matrix.
// Eight chunks per block (more loads in flight, 32 KB of LDS) ran at 2.26 ms.
typedef float ntx4 __attribute__((ext_vector_type(4)));

template <bool DONE, bool NEXT>
__global__ __launch_bounds__(kBlock) void subagg_gather_rows_kernel(
    float* __restrict__ Wg, int64_t rows, int64_t cols, int64_t ldg, int64_t groups, int m,
    SliceSetDev done, SliceSetDev next) {
  __shared__ float stage[kRowChunks][kBlock / 64][256];
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t r = b / groups;
  if (r >= rows) return;   // block-uniform
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t g0 = (b - r * groups) * (kRowChunks * 4 * kBlock) + 4 * static_cast<int64_t>(threadIdx.x);
  float* __restrict__ wrow = Wg + r * ldg;
  float v[kRowChunks][4];
  bool in[kRowChunks];
#pragma unroll
  for (int j = 0; j < kRowChunks; ++j) {
    const int64_t c0 = g0 + j * (4 * kBlock);
    in[j] = c0 < cols;   // cols % 4 == 0: a group is wholly in or out
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
    if (in[j]) {
      const ntx4 u = __builtin_nontemporal_load(reinterpret_cast<const ntx4*>(wrow + c0));
      t = make_float4(u[0], u[1], u[2], u[3]);
    }
    v[j][0] = t.x; v[j][1] = t.y; v[j][2] = t.z; v[j][3] = t.w;
  }
  // Column keys: the rank when the columns are partitioned, else the
  // column itself (owned by every row owner); -1 outside the matrix.
  int kd[kRowChunks][4], kn[kRowChunks][4];
  RowSel qd{nullptr, 0, 0}, qn{nullptr, 0, 0};
#pragma unroll
  for (int j = 0; j < kRowChunks; ++j) {
    const int64_t c0 = g0 + j * (4 * kBlock);
    if (DONE) {
      if (done.col_rank && in[j]) ranks4<true>(done.col_rank, c0, 4, kd[j]);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (!done.col_rank || !in[j]) kd[j][q] = in[j] ? static_cast<int>(c0 + q) : -1;
    }
    if (NEXT) {
      if (next.col_rank && in[j]) ranks4<true>(next.col_rank, c0, 4, kn[j]);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (!next.col_rank || !in[j]) kn[j][q] = in[j] ? static_cast<int>(c0 + q) : -1;
    }
  }
  if (DONE) {
    qd = row_select(done, m, r);
    if (!done.col_rank) { qd.lo = 0; qd.hi = cols; }
  }
  if (NEXT) {
    qn = row_select(next, m, r);
    if (!next.col_rank) { qn.lo = 0; qn.hi = cols; }
  }
  if (DONE) {
#pragma unroll
    for (int j = 0; j < kRowChunks; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (kd[j][q] >= qd.lo && kd[j][q] < qd.hi) v[j][q] = qd.base[kd[j][q] - qd.lo];
      if (in[j])
        __builtin_nontemporal_store(ntx4{v[j][0], v[j][1], v[j][2], v[j][3]},
                                    reinterpret_cast<ntx4*>(wrow + g0 + j * (4 * kBlock)));
    }
  }
  if (NEXT) {
    int first[kRowChunks], cnt[kRowChunks];
    bool run[kRowChunks];
#pragma unroll
    for (int j = 0; j < kRowChunks; ++j) {
      int f = INT32_MAX, l = -1, c = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool own = kn[j][q] >= qn.lo && kn[j][q] < qn.hi;
        if (own) { f = min(f, kn[j][q]); l = max(l, kn[j][q]); }
        c += __popcll(__ballot(own));
      }
      f = wave_min_int(f);
      l = wave_max_int(l);
      first[j] = f;
      cnt[j] = c;
      run[j] = c > 0 && l - f + 1 == c;   // wave-uniform
      if (run[j]) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (kn[j][q] >= qn.lo && kn[j][q] < qn.hi) stage[j][wv][kn[j][q] - f] = v[j][q];
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (kn[j][q] >= qn.lo && kn[j][q] < qn.hi) qn.base[kn[j][q] - qn.lo] = v[j][q];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kRowChunks; ++j) {
      if (run[j]) {
        float* dst = qn.base + (first[j] - qn.lo);
        for (int i = lane; i < cnt[j]; i += 64) dst[i] = stage[j][wv][i];
      }
    }
  }
}

template <bool VEC4>
__global__ __launch_bounds__(kBlock) void subagg_gather_kernel(float* __restrict__ Wg, int64_t rows,
                                                              int64_t cols, int64_t ldg,
                                                              int64_t chunks, int m,
                                                              SliceSetDev done, int has_done,
                                                              SliceSetDev next, int has_next) {
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t r = b / chunks;
  const int64_t c0 = (b - r * chunks) * (4 * kBlock) + 4 * static_cast<int64_t>(threadIdx.x);
  if (r >= rows || c0 >= cols) return;
  const int nq = cols - c0 < 4 ? static_cast<int>(cols - c0) : 4;
  float* __restrict__ w = Wg + r * ldg + c0;
  float v[4];
  if constexpr (VEC4) {
    const float4 t = *reinterpret_cast<const float4*>(w);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = q < nq ? w[q] : 0.f;
  }
  int kd[4], kn[4];
  RowSel qd{nullptr, 0, 0}, qn{nullptr, 0, 0};
  if (has_done) {
    ranks4<VEC4>(done.col_rank, c0, nq, kd);
    qd = row_select(done, m, r);
  }
  if (has_next) {
    ranks4<VEC4>(next.col_rank, c0, nq, kn);
    qn = row_select(next, m, r);
  }
  if (has_done) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float* p = q < nq ? slot_of(done, m, qd, r, c0 + q, kd[q]) : nullptr;
      if (p) v[q] = *p;
    }
    if constexpr (VEC4) {
      *reinterpret_cast<float4*>(w) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q < nq) w[q] = v[q];
    }
  }
  if (has_next) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float* p = q < nq ? slot_of(next, m, qn, r, c0 + q, kn[q]) : nullptr;
      if (p) *p = v[q];
    }
  }
}

}  // namespace

gist_status subagg_gather(hipStream_t st, float* Wg, int64_t rows, int64_t cols, int64_t ldg,
                          int m, const gist_slice_set* done, const gist_slice_set* next,
                          double bytes) {
  SliceSetDev d{}, n{};
  if (done) d = SliceSetDev{done->row_rank, done->row_offs, done->col_rank, done->col_offs,
                            done->slices, done->ld};
  if (next) n = SliceSetDev{next->row_rank, next->row_offs, next->col_rank, next->col_offs,
                            next->slices, next->ld};
  const int64_t chunks = (cols + 4 * kBlock - 1) / (4 * kBlock);
  if (rows * chunks > static_cast<int64_t>(UINT32_MAX))
    return set_error(GIST_E_UNSUPPORTED, "subagg_gather: matrix too large for one launch");
  bool vec = cols % 4 == 0 && ldg % 4 == 0 && aligned16(Wg);
  for (const SliceSetDev* s : {&d, &n})
    if (s->col_rank) vec = vec && aligned16(s->col_rank);
  const dim3 grid(static_cast<unsigned>(rows * chunks));
  const bool rows_part = (!done || done->row_rank) && (!next || next->row_rank);
  ProfScope ps(st, vec && rows_part ? "subagg_gather_rows" : "subagg_gather", 0.0, bytes);
  if (vec && rows_part) {
    const int dn = done ? 1 : 0, nx = next ? 1 : 0;
    const int64_t groups = (chunks + kRowChunks - 1) / kRowChunks;
    const dim3 rgrid(static_cast<unsigned>(rows * groups));
    if (dn && nx)
      hipLaunchKernelGGL((subagg_gather_rows_kernel<true, true>), rgrid, dim3(kBlock), 0, st, Wg,
                         rows, cols, ldg, groups, m, d, n);
    else if (dn)
      hipLaunchKernelGGL((subagg_gather_rows_kernel<true, false>), rgrid, dim3(kBlock), 0, st, Wg,
                         rows, cols, ldg, groups, m, d, n);
    else
      hipLaunchKernelGGL((subagg_gather_rows_kernel<false, true>), rgrid, dim3(kBlock), 0, st, Wg,
                         rows, cols, ldg, groups, m, d, n);
  } else if (vec) {
    hipLaunchKernelGGL(subagg_gather_kernel<true>, grid, dim3(kBlock), 0, st, Wg, rows, cols, ldg,
                       chunks, m, d, done ? 1 : 0, n, next ? 1 : 0);
  } else {
    hipLaunchKernelGGL(subagg_gather_kernel<false>, grid, dim3(kBlock), 0, st, Wg, rows, cols, ldg,
                       chunks, m, d, done ? 1 : 0, n, next ? 1 : 0);
  }
  return check_launch("subagg_gather");
}

gist_status relu_mask(hipStream_t st, int64_t count, const float* dH, const float* Hout,
                      float* dZ) {
  if (count <= 0) return GIST_OK;
  const int vec = aligned16(dH) && aligned16(Hout) && aligned16(dZ);
  ProfScope ps(st, "relu_mask", 0.0, 12.0 * static_cast<double>(count));
  hipLaunchKernelGGL(relu_mask_kernel, dim3(grid_for(count / 4 + 1, kBlock, 8192)), dim3(kBlock),
                     0, st, count, dH, Hout, dZ, vec);
  return check_launch("relu_mask");
}

gist_status fill_zero(hipStream_t st, float* p, int64_t count) {
  if (count <= 0) return GIST_OK;
  ProfScope ps(st, "fill_zero", 0.0, 4.0 * static_cast<double>(count));
  hipLaunchKernelGGL(zero_kernel, dim3(grid_for(count, kBlock, 8192)), dim3(kBlock), 0, st, p,
                     count);
  return check_launch("fill_zero");
}

gist_status transpose(hipStream_t st, const float* src, int64_t rows, int64_t cols, int64_t lds,
                      float* dst, int64_t ldd) {
  if (rows <= 0 || cols <= 0) return GIST_OK;
  if (ldd < rows) return set_error(GIST_E_INVAL, "transpose: ldd < rows");
  const int64_t gx = (cols + 63) / 64, gy = (ldd + 63) / 64;
  if (gx > INT32_MAX || gy > 65535)
    return set_error(GIST_E_UNSUPPORTED, "transpose: matrix too large");
  ProfScope ps(st, "transpose", 0.0, 4.0 * static_cast<double>(rows + ldd) * cols);
  const bool vec = lds % 4 == 0 && cols % 4 == 0 && ldd % 4 == 0 && aligned16(src) &&
                   aligned16(dst);
  if (vec)
    hipLaunchKernelGGL(transpose4_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)),
                       dim3(kBlock), 0, st, src, rows, cols, lds, dst, ldd);
  else
    hipLaunchKernelGGL(transpose_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)),
                       dim3(kBlock), 0, st, src, rows, cols, lds, dst, ldd);
  return check_launch("transpose");
}

gist_status pull_copy(hipStream_t st, void* dst, const void* src, int64_t bytes) {
  if (bytes <= 0) return GIST_OK;
  ProfScope ps(st, "pull_copy", 0.0, 2.0 * static_cast<double>(bytes));
  const bool a16 = (reinterpret_cast<uintptr_t>(dst) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(src) % 16 == 0);
  if (a16) {
    const int64_t n16 = bytes / 16, tail = bytes % 16;
    hipLaunchKernelGGL(pull_kernel, dim3(grid_for(n16 > 0 ? n16 : 1, kBlock, 2048)), dim3(kBlock),
                       0, st, static_cast<uint4*>(dst), static_cast<const uint4*>(src), n16, tail);
  } else {
    hipLaunchKernelGGL(pull_bytes_kernel, dim3(grid_for(bytes, kBlock, 2048)), dim3(kBlock), 0, st,
                       static_cast<unsigned char*>(dst), static_cast<const unsigned char*>(src),
                       bytes);
  }
  return check_launch("pull_copy");
}

gist_status subagg_mean(hipStream_t st, float* Wg, int64_t rows, int64_t cols, int64_t ldg, int m,
                        const float* const* slices, int64_t lds) {
  const int64_t count = rows * cols;
  if (count <= 0) return GIST_OK;
  ProfScope ps(st, "subagg_mean", static_cast<double>(m) * count, 4.0 * (m + 1.0) * count);
  hipLaunchKernelGGL(subagg_mean_kernel, dim3(grid_for(count, kBlock, 8192)), dim3(kBlock), 0, st,
                     Wg, rows, cols, ldg, m, slices, lds);
  return check_launch("subagg_mean");
}

gist_status sgd(hipStream_t st, float* W, const float* dW, int64_t n, float lr) {
  ProfScope ps(st, "sgd_update", 2.0 * static_cast<double>(n), 12.0 * static_cast<double>(n));
  hipLaunchKernelGGL(sgd_kernel, dim3(grid_for(n, kBlock, 8192)), dim3(kBlock), 0, st, n, W, dW,
                     lr);
  return check_launch("sgd_update");
}

gist_status adam(hipStream_t st, float* W, const float* dW, float* m, float* v, int64_t n,
                 float step_size, float inv_sqrt_bc2, float beta1, float beta2, float eps,
                 bool fresh, const float* coef_dev) {
  const AdamCoef c{step_size, inv_sqrt_bc2, beta1, beta2, eps};
  const bool vec = aligned16(W) && aligned16(dW) && aligned16(m) && aligned16(v);
  ProfScope ps(st, "adam_update", 0.0, (fresh ? 12.0 : 20.0) * static_cast<double>(n));
  if (vec)
    hipLaunchKernelGGL(adam_kernel<true>, dim3(grid_for((n + 3) / 4, kBlock, 8192)), dim3(kBlock), 0,
                       st, n, W, dW, m, v, c, fresh ? 1 : 0, coef_dev);
  else
    hipLaunchKernelGGL(adam_kernel<false>, dim3(grid_for(n, kBlock, 8192)), dim3(kBlock), 0, st, n,
                       W, dW, m, v, c, fresh ? 1 : 0, coef_dev);
  return check_launch("adam_update");
}

gist_status gather(hipStream_t st, const float* Wg, int64_t ldg, const int32_t* rows,
                   int32_t nr, const int32_t* cols, int32_t nc, float* Ws, int64_t lds) {
  ProfScope ps(st, "gather_slice", 0.0,
               8.0 * static_cast<double>(nr) * nc + 4.0 * ((rows ? nr : 0) + (cols ? nc : 0)));
  hipLaunchKernelGGL(gather_kernel, dim3(static_cast<unsigned>(nr)), dim3(kBlock), 0, st, Wg, ldg,
                     rows, nr, cols, nc, Ws, lds);
  return check_launch("gather_slice");
}

gist_status scatter(hipStream_t st, float* Wg, int64_t ldg, const int32_t* rows, int32_t nr,
                    const int32_t* cols, int32_t nc, const float* Ws, int64_t lds) {
  ProfScope ps(st, "subagg_scatter", 0.0,
               8.0 * static_cast<double>(nr) * nc + 4.0 * ((rows ? nr : 0) + (cols ? nc : 0)));
  hipLaunchKernelGGL(scatter_kernel, dim3(static_cast<unsigned>(nr)), dim3(kBlock), 0, st, Wg,
                     ldg, rows, nr, cols, nc, Ws, lds);
  return check_launch("subagg");
}

gist_status count_nonfinite(hipStream_t st, const float* Ws, int64_t lds, int32_t nr, int32_t nc,
                            int* d_count) {
  hipLaunchKernelGGL(zero_int_kernel, dim3(1), dim3(64), 0, st, d_count);
  hipLaunchKernelGGL(nonfinite_kernel,
                     dim3(grid_for(static_cast<int64_t>(nr) * nc, kBlock, 4096)), dim3(kBlock),
                     0, st, Ws, lds, nr, nc, d_count);
  return check_launch("subagg finite check");
}

gist_status softmax_xent(hipStream_t st, int64_t n, int C, const float* logits,
                         const int32_t* labels, float* loss, float* dlogits, float* partials,
                         const int32_t* n_dev) {
  const int rows_per_block = kBlock / 64;
  const int nparts = static_cast<int>((n + rows_per_block - 1) / rows_per_block);
  if (n > 0) {
    ProfScope ps(st, "softmax_xent_rows", 0.0, 8.0 * static_cast<double>(n) * C + 4.0 * n);
    hipLaunchKernelGGL(xent_rows_kernel, dim3(static_cast<unsigned>(nparts)), dim3(kBlock), 0,
                       st, static_cast<int>(n), C, logits, labels, dlogits, partials, n_dev);
  }
  hipLaunchKernelGGL(xent_finish_kernel, dim3(1), dim3(kBlock), 0, st, nparts, partials,
                     static_cast<int>(n), loss, n_dev);
  return check_launch("softmax_xent");
}

}  // namespace gist
