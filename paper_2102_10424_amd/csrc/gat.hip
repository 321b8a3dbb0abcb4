// Graph attention layer (the GAT models the paper trains with GIST,
// Section 3 and Table 2; single head as Velickovic et al. define it):
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
// The first kKeep * 64 dalpha of a row stay in registers (lane l keeps
// entry 64 c + l of chunk c); a longer row's remaining entries recompute
// theirs in the second pass, so nothing is read back from memory.
constexpr int kKeep = 8;

__device__ __forceinline__ float dot_row(const float* __restrict__ a, const float* __restrict__ b, int s,
                                         int lane) {
  float part = 0.f;
  for (int k = lane; k < s; k += 64) part = fmaf(a[k], b[k], part);
  return wave_sum(part);
}

__global__ __launch_bounds__(kBlock) void gat_edge_grad_kernel(
    int64_t n, int s, const int* __restrict__ rowptr, const int* __restrict__ col,
    const float* __restrict__ alpha, const float* __restrict__ dZ, int64_t ldz,
    const float* __restrict__ P, int64_t ldp, const float* __restrict__ u,
    const float* __restrict__ v, float slope, float* __restrict__ dpre, float* __restrict__ du) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
  if (i >= n) return;
  const int e0 = rowptr[i], e1 = rowptr[i + 1];
  const float* dz = dZ + i * ldz;
  float keep[kKeep];
  float c = 0.f;
#pragma unroll
  for (int cc = 0; cc < kKeep; ++cc) {
    keep[cc] = 0.f;
    const int b = e0 + 64 * cc;
    if (b >= e1) continue;
    const int end = min(e1, b + 64);
    for (int p = b; p < end; ++p) {
      const float da = dot_row(dz, P + static_cast<int64_t>(col[p]) * ldp, s, lane);
      if (lane == p - b) keep[cc] = da;
      c = fmaf(alpha[p], da, c);
    }
  }
  for (int p = e0 + 64 * kKeep; p < e1; ++p)
    c = fmaf(alpha[p], dot_row(dz, P + static_cast<int64_t>(col[p]) * ldp, s, lane), c);
  const float ui = u[i];
  float tpos = 0.f, tneg = 0.f;
  int npos = 0;
#pragma unroll
  for (int cc = 0; cc < kKeep; ++cc) {
    const int p = e0 + 64 * cc + lane;
    float t = 0.f;
    bool pos = false;
    if (p < e1) {
      pos = ui + v[col[p]] > 0.f;
      t = alpha[p] * (keep[cc] - c);
      dpre[p] = pos ? t : slope * t;
    }
    npos += __popcll(__ballot(pos));
    tpos += wave_sum(pos ? t : 0.f);
    tneg += wave_sum(pos ? 0.f : t);
  }
  for (int p = e0 + 64 * kKeep; p < e1; ++p) {
    const float da = dot_row(dz, P + static_cast<int64_t>(col[p]) * ldp, s, lane);
    const bool pos = ui + v[col[p]] > 0.f;
    const float t = alpha[p] * (da - c);
    if (lane == 0) dpre[p] = pos ? t : slope * t;
    if (pos) { tpos += t; ++npos; } else { tneg += t; }
  }
  const int nneg = (e1 - e0) - npos;
  if (lane == 0) du[i] = npos <= nneg ? (1.f - slope) * tpos : -((1.f - slope) * tneg);
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
// alpha[tpos[q]] (the transposed attention in row j's order).  One thread
// per row.
__global__ __launch_bounds__(kBlock) void gat_mirror_sums_kernel(int64_t n, const int* __restrict__ rowptr,
                                                                 const int* __restrict__ tpos,
                                                                 const float* __restrict__ dpre,
                                                                 const float* __restrict__ alpha,
                                                                 float* __restrict__ dv,
                                                                 float* __restrict__ alpha_t) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (j >= n) return;
  float s = 0.f;
  for (int q = rowptr[j]; q < rowptr[j + 1]; ++q) {
    const int p = tpos[q];
    s += p >= 0 ? dpre[p] : 0.f;
    alpha_t[q] = p >= 0 ? alpha[p] : 0.f;
  }
  dv[j] = s;
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

// da_src = P^T du, da_dst = P^T dv in two deterministic stages: partial sums
// over chunks of kRowsPerChunk rows (one thread per column), then the chunks
// summed in order.
constexpr int kRowsPerChunk = 128;

__global__ __launch_bounds__(kBlock) void gat_gemv_partial_kernel(int64_t n, int s, const float* __restrict__ P,
                                                                  int64_t ldp, const float* __restrict__ du,
                                                                  const float* __restrict__ dv,
                                                                  float* __restrict__ part) {
  const int k = blockIdx.x * kBlock + threadIdx.x;
  const int64_t chunk = blockIdx.y;
  if (k >= s) return;
  const int64_t r0 = chunk * kRowsPerChunk;
  const int64_t r1 = min<int64_t>(n, r0 + kRowsPerChunk);
  float a = 0.f, b = 0.f;
  for (int64_t i = r0; i < r1; ++i) {
    const float x = P[i * ldp + k];
    a = fmaf(x, du[i], a);
    b = fmaf(x, dv[i], b);
  }
  part[(chunk * 2) * s + k] = a;
  part[(chunk * 2 + 1) * s + k] = b;
}

__global__ __launch_bounds__(kBlock) void gat_gemv_final_kernel(int64_t chunks, int s,
                                                                const float* __restrict__ part,
                                                                float* __restrict__ da_src,
                                                                float* __restrict__ da_dst) {
  const int k = blockIdx.x * kBlock + threadIdx.x;
  if (k >= s) return;
  float a = 0.f, b = 0.f;
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
  hipLaunchKernelGGL(gat_edge_grad_kernel, dim3(rows_grid(n)), dim3(kBlock), 0, st, n, s, rowptr,
                     col, alpha, dZ, ldz, P, ldp, u, v, slope, dpre, du);
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
  hipLaunchKernelGGL(gat_mirror_sums_kernel, dim3(static_cast<unsigned>((n + kBlock - 1) / kBlock)),
                     dim3(kBlock), 0, st, n, rowptr, tpos, dpre, alpha, dv, alpha_t);
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
  const int64_t chunks = (n + kRowsPerChunk - 1) / kRowsPerChunk;
  return static_cast<size_t>(chunks) * 2 * s * sizeof(float);
}

gist_status gat_gemv_t(hipStream_t st, int64_t n, int s, const float* P, int64_t ldp, const float* du,
                       const float* dv, float* da_src, float* da_dst, float* part) {
  const int64_t chunks = (n + kRowsPerChunk - 1) / kRowsPerChunk;
  if (chunks > 65535) return set_error(GIST_E_UNSUPPORTED, "gat: too many rows");
  ProfScope ps(st, "gat_gemv_t", 4.0 * n * s, 4.0 * static_cast<double>(n) * s);
  const unsigned cx = static_cast<unsigned>((s + kBlock - 1) / kBlock);
  hipLaunchKernelGGL(gat_gemv_partial_kernel, dim3(cx, static_cast<unsigned>(chunks)), dim3(kBlock),
                     0, st, n, s, P, ldp, du, dv, part);
  hipLaunchKernelGGL(gat_gemv_final_kernel, dim3(cx), dim3(kBlock), 0, st, chunks, s, part, da_src,
                     da_dst);
  return check_launch("gat_gemv_t");
}

}  // namespace gist
