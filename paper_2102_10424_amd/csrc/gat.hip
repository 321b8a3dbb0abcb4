// Graph attention layer (the GAT models the paper trains with GIST,
// Section 2.3 and Table 2; single head as Velickovic et al. define it):
//   P = H W,  u = P a_src,  v = P a_dst,  e_ij = LeakyReLU(u_i + v_j),
//   alpha = row softmax of e over the pattern N(i) u {i},  Z = A_alpha P.
// The GEMMs and the alpha-weighted aggregation reuse the library's GEMM and
// SpMM; the kernels here are the attention-specific steps.  Every
// reduction runs in a fixed order (wave butterflies, sequential chunks), so
// results are bitwise reproducible.

#include <cmath>

#include "common.cuh"
#include "gist_internal.h"

namespace gist {

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ float leaky(float x, float slope) { return x > 0.f ? x : slope * x; }

// u_i = P_i . a_src, v_i = P_i . a_dst: one wave per row.
__global__ __launch_bounds__(kBlock) void gat_scores_kernel(int64_t n, int s, const float* __restrict__ P,
                                                            int64_t ldp, const float* __restrict__ a_src,
                                                            const float* __restrict__ a_dst,
                                                            float* __restrict__ u, float* __restrict__ v) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
  if (i >= n) return;
  const float* p = P + i * ldp;
  float su = 0.f, sv = 0.f;
  for (int k = lane; k < s; k += 64) {
    su = fmaf(p[k], a_src[k], su);
    sv = fmaf(p[k], a_dst[k], sv);
  }
  su = wave_sum(su);
  sv = wave_sum(sv);
  if (lane == 0) { u[i] = su; v[i] = sv; }
}

// alpha over row i's entries: one wave per row, entries in chunks of 64
// (the row maximum and the exponential sum accumulate chunk by chunk).
__global__ __launch_bounds__(kBlock) void gat_softmax_kernel(int64_t n, const int* __restrict__ rowptr,
                                                             const int* __restrict__ col,
                                                             const float* __restrict__ u,
                                                             const float* __restrict__ v, float slope,
                                                             float* __restrict__ alpha) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
  if (i >= n) return;
  const int e0 = rowptr[i], e1 = rowptr[i + 1];
  const float ui = u[i];
  float mx = -INFINITY;
  for (int b = e0; b < e1; b += 64) {
    const int p = b + lane;
    const float e = p < e1 ? leaky(ui + v[col[p]], slope) : -INFINITY;
    mx = fmaxf(mx, wave_max(e));
  }
  float sum = 0.f;
  for (int b = e0; b < e1; b += 64) {
    const int p = b + lane;
    const float x = p < e1 ? expf(leaky(ui + v[col[p]], slope) - mx) : 0.f;
    sum += wave_sum(x);
  }
  const float inv = 1.f / sum;
  for (int b = e0; b < e1; b += 64) {
    const int p = b + lane;
    if (p < e1) alpha[p] = expf(leaky(ui + v[col[p]], slope) - mx) * inv;
  }
}

// Backward through the attention of row i (one wave per row):
//   dalpha_ij = dZ_i . P_j,  c_i = sum_j alpha_ij dalpha_ij,
//   t_ij = alpha_ij (dalpha_ij - c_i),
//   dpre_ij = t_ij * LeakyReLU'(u_i + v_j),   du_i = sum_j dpre_ij.
// Since sum_j t_ij = c_i (1 - sum_j alpha_ij) = 0, du_i equals
// (1 - slope) T+ = -(1 - slope) T- with T+ / T- the sums of t over the
// entries with positive / non-positive scores; the kernel takes the form
// over the smaller of the two sets.  A row whose scores all lie on one side
// then has du_i = 0 exactly (a_src cannot change its attention, whatever
// the rounding of alpha), where the plain sum would leave a rounding
// residue that an optimizer normalising by |g| (Adam) would turn into a
// full-size step.
//
// The dot products dZ_i . P_j are computed by groups of G lanes (G a power
// of two sized to the feature width, each lane covering about 16 features
// with float4 loads where rows are 16-byte aligned), 64 / G entries per
// pass.  The first kKeep dalpha of a row are kept in LDS for the second
// pass (one lane per entry); a longer row's remaining entries recompute
// theirs in the second pass, so nothing is read back from global memory.
constexpr int kKeep = 512;
constexpr int kWaves = kBlock / 64;

template <int VEC>
__device__ __forceinline__ float group_dot(const float* __restrict__ a, const float* __restrict__ b,
                                           int s, int gl, int G) {
  float part = 0.f;
  if constexpr (VEC == 4) {
    for (int k = gl * 4; k < s; k += G * 4) {
      const float4 x = *reinterpret_cast<const float4*>(a + k);
      const float4 y = *reinterpret_cast<const float4*>(b + k);
      part = fmaf(x.x, y.x, part);
      part = fmaf(x.y, y.y, part);
      part = fmaf(x.z, y.z, part);
      part = fmaf(x.w, y.w, part);
    }
  } else {
    for (int k = gl; k < s; k += G) part = fmaf(a[k], b[k], part);
  }
  for (int off = G >> 1; off > 0; off >>= 1) part += __shfl_xor(part, off);
  return part;    // every lane of the group holds the group's sum
}

template <int VEC>
__global__ __launch_bounds__(kBlock) void gat_edge_grad_kernel(
    int64_t n, int s, int G, const int* __restrict__ rowptr, const int* __restrict__ col,
    const float* __restrict__ alpha, const float* __restrict__ dZ, int64_t ldz,
    const float* __restrict__ P, int64_t ldp, const float* __restrict__ u,
    const float* __restrict__ v, float slope, float* __restrict__ dpre, float* __restrict__ du) {
  __shared__ float keep_lds[kWaves][kKeep];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
  const bool active = i < n;
  const int e0 = active ? rowptr[i] : 0, e1 = active ? rowptr[i + 1] : 0;
  const int len = e1 - e0;
  const int E = 64 / G;                 // entries per pass
  const int gi = lane / G, gl = lane % G;
  const float* dz = dZ + (active ? i : 0) * ldz;
  float* keep = keep_lds[wave];
  // pass 1: dalpha of every entry, c_i
  float cpart = 0.f;
  for (int b = 0; b < len; b += E) {
    const int q = b + gi;
    const bool valid = q < len;
    const int p = e0 + (valid ? q : 0);
    const float da = group_dot<VEC>(dz, P + static_cast<int64_t>(col[p]) * ldp, s, gl, G);
    if (valid && gl == 0) {
      if (q < kKeep) keep[q] = da;
      cpart = fmaf(alpha[p], da, cpart);
    }
  }
  const float c = wave_sum(cpart);
  __syncthreads();   // the kept dalpha are visible to every lane of the wave
  // pass 2: t, dpre, and the one-sided sums for du
  const float ui = active ? u[i] : 0.f;
  float tpos = 0.f, tneg = 0.f;
  int npos = 0;
  const int nkeep = min(len, kKeep);
  for (int q = lane; q < nkeep; q += 64) {
    const int p = e0 + q;
    const bool pos = ui + v[col[p]] > 0.f;
    const float t = alpha[p] * (keep[q] - c);
    dpre[p] = pos ? t : slope * t;
    if (pos) { tpos += t; ++npos; } else { tneg += t; }
  }
  for (int b = kKeep; b < len; b += E) {    // rows longer than kKeep: recompute
    const int q = b + gi;
    const bool valid = q < len;
    const int p = e0 + (valid ? q : 0);
    const float da = group_dot<VEC>(dz, P + static_cast<int64_t>(col[p]) * ldp, s, gl, G);
    if (valid && gl == 0) {
      const bool pos = ui + v[col[p]] > 0.f;
      const float t = alpha[p] * (da - c);
      dpre[p] = pos ? t : slope * t;
      if (pos) { tpos += t; ++npos; } else { tneg += t; }
    }
  }
  tpos = wave_sum(tpos);
  tneg = wave_sum(tneg);
  for (int off = 32; off > 0; off >>= 1) npos += __shfl_xor(npos, off);
  const int nneg = len - npos;
  if (active && lane == 0) du[i] = npos <= nneg ? (1.f - slope) * tpos : -((1.f - slope) * tneg);
}

// tpos[q] = p where entry q of row j is (j, i) and entry p of row i is
// (i, j): the position of each entry's mirror in a symmetric pattern (one
// wave per row i, binary search in row j).  Mirrors that do not exist keep
// the -1 the caller filled in.
__global__ __launch_bounds__(kBlock) void gat_mirror_kernel(int64_t n, const int* __restrict__ rowptr,
                                                            const int* __restrict__ col,
                                                            int* __restrict__ tpos) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
  if (i >= n) return;
  const int e0 = rowptr[i], e1 = rowptr[i + 1];
  const int ii = static_cast<int>(i);
  for (int p = e0 + lane; p < e1; p += 64) {
    const int j = col[p];
    int lo = rowptr[j], hi = rowptr[j + 1];
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (col[mid] < ii) lo = mid + 1; else hi = mid;
    }
    if (lo < rowptr[j + 1] && col[lo] == ii) tpos[lo] = p;
  }
}

// dv_j = sum over row j's entries q of dpre[tpos[q]]; alpha_t[q] =
// alpha[tpos[q]] (the transposed attention in row j's order).  One wave per
// row, entries in chunks of 64.
__global__ __launch_bounds__(kBlock) void gat_mirror_sums_kernel(int64_t n, const int* __restrict__ rowptr,
                                                                 const int* __restrict__ tpos,
                                                                 const float* __restrict__ dpre,
                                                                 const float* __restrict__ alpha,
                                                                 float* __restrict__ dv,
                                                                 float* __restrict__ alpha_t) {
  const int lane = threadIdx.x & 63;
  const int64_t j = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
  if (j >= n) return;
  const int e0 = rowptr[j], e1 = rowptr[j + 1];
  float sum = 0.f;
  for (int b = e0; b < e1; b += 64) {
    const int q = b + lane;
    float x = 0.f;
    if (q < e1) {
      const int p = tpos[q];
      x = p >= 0 ? dpre[p] : 0.f;
      alpha_t[q] = p >= 0 ? alpha[p] : 0.f;
    }
    sum += wave_sum(x);
  }
  if (lane == 0) dv[j] = sum;
}

// dP_ik += du_i a_src_k + dv_i a_dst_k.
__global__ __launch_bounds__(kBlock) void gat_rank2_kernel(int64_t n, int s, float* __restrict__ dP,
                                                           int64_t ld, const float* __restrict__ du,
                                                           const float* __restrict__ dv,
                                                           const float* __restrict__ a_src,
                                                           const float* __restrict__ a_dst) {
  const int64_t total = n * s;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; e < total; e += stride) {
    const int64_t i = e / s;
    const int k = static_cast<int>(e - i * s);
    float* d = dP + i * ld + k;
    *d = fmaf(dv[i], a_dst[k], fmaf(du[i], a_src[k], *d));
  }
}

// da_src = P^T du, da_dst = P^T dv in two deterministic stages.  Stage 1:
// one block per (64-column group, chunk of rows); wave w sums rows
// r0 + w, r0 + w + 4, ... of the chunk (lane = column), then the four wave
// sums are added in wave order.  Stage 2: per column, the chunk sums in
// chunk order.  At most kMaxChunks chunks, each a multiple of 4 rows.
constexpr int kMaxChunks = 1024;

__host__ __device__ inline int64_t gemv_rows_per_chunk(int64_t n) {
  int64_t r = (n + kMaxChunks - 1) / kMaxChunks;
  r = r < 64 ? 64 : r;
  return (r + 3) / 4 * 4;
}

__global__ __launch_bounds__(kBlock) void gat_gemv_partial_kernel(int64_t n, int s, int64_t rpc,
                                                                  const float* __restrict__ P,
                                                                  int64_t ldp, const float* __restrict__ du,
                                                                  const float* __restrict__ dv,
                                                                  float* __restrict__ part) {
  __shared__ float red[2][kWaves][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int k = blockIdx.x * 64 + lane;
  const int64_t chunk = blockIdx.y;
  const int64_t r0 = chunk * rpc;
  const int64_t r1 = min<int64_t>(n, r0 + rpc);
  float a = 0.f, b = 0.f;
  if (k < s) {
    for (int64_t r = r0 + wave; r < r1; r += kWaves) {
      const float x = P[r * ldp + k];
      a = fmaf(x, du[r], a);
      b = fmaf(x, dv[r], b);
    }
  }
  red[0][wave][lane] = a;
  red[1][wave][lane] = b;
  __syncthreads();
  if (wave == 0 && k < s) {
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      sa += red[0][w][lane];
      sb += red[1][w][lane];
    }
    part[(chunk * 2) * s + k] = sa;
    part[(chunk * 2 + 1) * s + k] = sb;
  }
}

__global__ __launch_bounds__(kBlock) void gat_gemv_final_kernel(int64_t chunks, int s,
                                                                const float* __restrict__ part,
                                                                float* __restrict__ da_src,
                                                                float* __restrict__ da_dst) {
  const int k = blockIdx.x * kBlock + threadIdx.x;
  if (k >= s) return;
  float a = 0.f, b = 0.f;
#pragma unroll 8
  for (int64_t c = 0; c < chunks; ++c) {
    a += part[(c * 2) * s + k];
    b += part[(c * 2 + 1) * s + k];
  }
  da_src[k] = a;
  da_dst[k] = b;
}

__global__ __launch_bounds__(kBlock) void fill_int_kernel(int* p, int64_t count, int value) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; e < count; e += stride)
    p[e] = value;
}

unsigned rows_grid(int64_t n) { return static_cast<unsigned>((n * 64 + kBlock - 1) / kBlock); }
unsigned flat_grid(int64_t count) {
  return static_cast<unsigned>(std::min<int64_t>((count + kBlock - 1) / kBlock, 8192));
}

}  // namespace

gist_status gat_scores(hipStream_t st, int64_t n, int s, const float* P, int64_t ldp,
                       const float* a_src, const float* a_dst, float* u, float* v) {
  ProfScope ps(st, "gat_scores", 4.0 * n * s, 4.0 * (static_cast<double>(n) * s + 2 * s + 2 * n));
  hipLaunchKernelGGL(gat_scores_kernel, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, s, P, ldp,
                     a_src, a_dst, u, v);
  return check_launch("gat_scores");
}

gist_status gat_softmax(hipStream_t st, int64_t n, int64_t nnz, const int* rowptr, const int* col,
                        const float* u, const float* v, float slope, float* alpha) {
  ProfScope ps(st, "gat_softmax", 0.0, 4.0 * (n + 1) + 12.0 * nnz + 4.0 * n);
  hipLaunchKernelGGL(gat_softmax_kernel, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, rowptr, col,
                     u, v, slope, alpha);
  return check_launch("gat_softmax");
}

gist_status gat_edge_grad(hipStream_t st, int64_t n, int64_t nnz, int s, const int* rowptr,
                          const int* col, const float* alpha, const float* dZ, int64_t ldz,
                          const float* P, int64_t ldp, const float* u, const float* v, float slope,
                          float* dpre, float* du) {
  ProfScope ps(st, "gat_edge_grad", 2.0 * nnz * s,
               4.0 * (static_cast<double>(nnz) * s + static_cast<double>(n) * s) + 16.0 * nnz);
  // lanes per entry: a power of two giving each lane about 16 features
  const bool vec = s % 4 == 0 && ldz % 4 == 0 && ldp % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(dZ) % 16 == 0 && reinterpret_cast<uintptr_t>(P) % 16 == 0;
  int G = 1;
  while (G < 64 && G * 16 < s) G <<= 1;
  if (vec)
    hipLaunchKernelGGL(gat_edge_grad_kernel<4>, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, s, G,
                       rowptr, col, alpha, dZ, ldz, P, ldp, u, v, slope, dpre, du);
  else
    hipLaunchKernelGGL(gat_edge_grad_kernel<1>, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, s, G,
                       rowptr, col, alpha, dZ, ldz, P, ldp, u, v, slope, dpre, du);
  return check_launch("gat_edge_grad");
}

gist_status gat_mirror(hipStream_t st, int64_t n, int64_t nnz, const int* rowptr, const int* col,
                       int* tpos) {
  ProfScope ps(st, "gat_mirror", 0.0, 12.0 * nnz);
  if (nnz > 0)
    hipLaunchKernelGGL(fill_int_kernel, dim3(flat_grid(nnz)), dim3(kBlock), 0, st, tpos, nnz, -1);
  hipLaunchKernelGGL(gat_mirror_kernel, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, rowptr, col,
                     tpos);
  return check_launch("gat_mirror");
}

gist_status gat_mirror_sums(hipStream_t st, int64_t n, int64_t nnz, const int* rowptr, const int* tpos,
                            const float* dpre, const float* alpha, float* dv, float* alpha_t) {
  ProfScope ps(st, "gat_mirror_sums", 0.0, 16.0 * nnz + 4.0 * n);
  hipLaunchKernelGGL(gat_mirror_sums_kernel, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, rowptr,
                     tpos, dpre, alpha, dv, alpha_t);
  return check_launch("gat_mirror_sums");
}

gist_status gat_rank2(hipStream_t st, int64_t n, int s, float* dP, int64_t ld, const float* du,
                      const float* dv, const float* a_src, const float* a_dst) {
  ProfScope ps(st, "gat_rank2", 4.0 * n * s, 8.0 * static_cast<double>(n) * s);
  hipLaunchKernelGGL(gat_rank2_kernel, dim3(flat_grid(n * s)), dim3(kBlock), 0, st, n, s, dP, ld,
                     du, dv, a_src, a_dst);
  return check_launch("gat_rank2");
}

size_t gat_gemv_workspace(int64_t n, int s) {
  const int64_t rpc = gemv_rows_per_chunk(n);
  const int64_t chunks = (n + rpc - 1) / rpc;
  return static_cast<size_t>(chunks) * 2 * s * sizeof(float);
}

gist_status gat_gemv_t(hipStream_t st, int64_t n, int s, const float* P, int64_t ldp, const float* du,
                       const float* dv, float* da_src, float* da_dst, float* part) {
  const int64_t rpc = gemv_rows_per_chunk(n);
  const int64_t chunks = (n + rpc - 1) / rpc;
  ProfScope ps(st, "gat_gemv_t", 4.0 * n * s, 4.0 * static_cast<double>(n) * s);
  const unsigned cx = static_cast<unsigned>((s + 63) / 64);
  hipLaunchKernelGGL(gat_gemv_partial_kernel, dim3(cx, static_cast<unsigned>(chunks)), dim3(kBlock),
                     0, st, n, s, rpc, P, ldp, du, dv, part);
  hipLaunchKernelGGL(gat_gemv_final_kernel, dim3(static_cast<unsigned>((s + kBlock - 1) / kBlock)),
                     dim3(kBlock), 0, st, chunks, s, part, da_src, da_dst);
  return check_launch("gat_gemv_t");
}

}  // namespace gist
