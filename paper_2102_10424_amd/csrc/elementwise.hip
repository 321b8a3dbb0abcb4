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

__global__ __launch_bounds__(kBlock) void zero_kernel(float* __restrict__ p, int64_t count) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < count; i += stride)
    p[i] = 0.f;
}

__global__ void zero_int_kernel(int* p) {
  if (threadIdx.x == 0 && blockIdx.x == 0) p[0] = 0;
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
__global__ __launch_bounds__(kBlock) void xent_rows_kernel(int n, int C,
                                                           const float* __restrict__ Z,
                                                           const int* __restrict__ y,
                                                           float* __restrict__ dZ,
                                                           float* __restrict__ partials) {
  __shared__ float wloss[kBlock / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave;
  float row_loss = 0.f;
  if (row < n) {
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
    const float inv_n = 1.0f / static_cast<float>(n);
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
                                                             int n, float* loss) {
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

}  // namespace

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

gist_status sgd(hipStream_t st, float* W, const float* dW, int64_t n, float lr) {
  ProfScope ps(st, "sgd_update", 2.0 * static_cast<double>(n), 12.0 * static_cast<double>(n));
  hipLaunchKernelGGL(sgd_kernel, dim3(grid_for(n, kBlock, 8192)), dim3(kBlock), 0, st, n, W, dW,
                     lr);
  return check_launch("sgd_update");
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
                         const int32_t* labels, float* loss, float* dlogits, float* partials) {
  const int rows_per_block = kBlock / 64;
  const int nparts = static_cast<int>((n + rows_per_block - 1) / rows_per_block);
  if (n > 0) {
    ProfScope ps(st, "softmax_xent_rows", 0.0, 8.0 * static_cast<double>(n) * C + 4.0 * n);
    hipLaunchKernelGGL(xent_rows_kernel, dim3(static_cast<unsigned>(nparts)), dim3(kBlock), 0,
                       st, static_cast<int>(n), C, logits, labels, dlogits, partials);
  }
  hipLaunchKernelGGL(xent_finish_kernel, dim3(1), dim3(kBlock), 0, st, nparts, partials,
                     static_cast<int>(n), loss);
  return check_launch("softmax_xent");
}

}  // namespace gist
