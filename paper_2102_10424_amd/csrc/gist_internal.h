// Internal declarations shared by the libgist sources (not part of the ABI).
#pragma once

#include <cstddef>
#include <climits>
#include <cstdint>
#include <string>

#include "../../include/gist.h"

struct ihipStream_t;
typedef struct ihipStream_t* hipStream_t;

namespace gist {
struct Profiler;
}

struct gist_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  int* d_flag = nullptr;   // 4 ints of device memory owned by the context
  float* loss_scratch = nullptr;   // this device's copy of the static loss buffer
  gist::Profiler* prof = nullptr;
};

namespace gist {

// Launch timing (gist_profile_*).  The entry points install the calling
// context's profiler for the duration of the call (ProfBind); launchers wrap
// each kernel launch in a ProfScope, which records an event pair on the
// launch stream when a profiler is recording.
class ProfBind {
 public:
  explicit ProfBind(gist_ctx* ctx);
  ~ProfBind();
 private:
  Profiler* prev_;
};

class ProfScope {
 public:
  ProfScope(hipStream_t st, const char* name, double flops, double bytes);
  ~ProfScope();
 private:
  int slot_ = -1;
  hipStream_t st_;
};

// SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): the state advances by the golden-ratio
// increment and each output is the state through the variant-13 finaliser.
// The host-side random streams (feature partition, LADIES draws) use it.
class SplitMix64 {
 public:
  explicit SplitMix64(uint64_t seed) : s_(seed) {}
  uint64_t next() {
    s_ += 0x9E3779B97F4A7C15ull;
    uint64_t z = s_;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  // Uniform on [0, bound): reject the incomplete top range of 2^64.
  uint64_t below(uint64_t bound) {
    const uint64_t rem = (0ull - bound) % bound;  // 2^64 mod bound
    for (;;) {
      const uint64_t r = next();
      if (rem == 0 || r < 0ull - rem) return r % bound;
    }
  }
 private:
  uint64_t s_;
};

// Thread-local error message; set_error returns the status for chaining.
gist_status set_error(gist_status s, const std::string& msg);
void clear_error();

// Convert the last HIP error of a launch into GIST_E_DEVICE.
gist_status check_launch(const char* what);

// Make `ctx->device` current for the duration of a call.
class DeviceGuard {
 public:
  explicit DeviceGuard(int dev);
  ~DeviceGuard();
 private:
  int prev_ = -1;
  bool changed_ = false;
};

// ---- kernel launchers (implemented in the .hip files) -------------------

// Y[r, c] = sum_e val[e] * X[col[e], c]  (+ Add[r, c]) (ReLU optional),
// r < n, c < width.  Row-major with leading dimensions.  `add` may alias Y.
// With `mask` (leading dimension ldm), Y[r, c] is stored as 0 where
// mask[r, c] > 0 fails: the ReLU derivative of the layer whose output mask is.
gist_status spmm(hipStream_t st, int64_t n, int64_t nnz, const int32_t* rowptr,
                 const int32_t* col, const float* val, const float* X,
                 int64_t ldx, int width, float* Y, int64_t ldy,
                 const float* add, int64_t ld_add, bool relu,
                 const float* mask = nullptr, int64_t ldm = 0);

// The same on the matrix cores for a matrix (n x n_in) whose entries sit
// mostly near the diagonal (a cluster mini-batch): dense bf16-split tiles
// for the entries near the diagonal, a gather for the rest (spmm_tile.hip).
// Requires no repeated (row, column) entry.  `add` may alias Y.
gist_status spmm_clustered(hipStream_t st, int64_t n, int64_t n_in, int64_t nnz,
                           const int32_t* rowptr, const int32_t* col, const float* val,
                           const float* X, int64_t ldx, int width, float* Y, int64_t ldy,
                           const float* add, int64_t ld_add, bool relu,
                           const float* mask = nullptr, int64_t ldm = 0);

// Operand of a GEMM: logical R x K matrix (R = M for A, N for B).
//   k_major == true : element (r, k) at p[r * ld + k]   (K contiguous)
//   k_major == false: element (r, k) at p[k * ld + r]   (R contiguous)
// A second pointer p1 takes over from index `split` along the concatenated
// dimension: along K when k_major, along R otherwise (SAGE's [H | Abar H]).
struct Operand {
  const float* p0 = nullptr;
  const float* p1 = nullptr;
  int64_t ld0 = 0, ld1 = 0;
  int64_t split = INT64_MAX;
  bool k_major = true;
  int64_t gs0 = 0, gs1 = 0;   // element offsets of p0 / p1 between GEMM groups
};

// C (M x N) = act(A (M x K) * B (K x N)), with B given as an N x K operand.
// Columns >= c_split go to C1 (column index minus c_split).
// `sgd`: C holds weights that take one SGD step with the product as their
// gradient, C <- fmaf(-lr, A B, C) (gist_sgd_update's arithmetic), instead of
// C <- A B; every element of C is written exactly once, so the step is
// applied once.
struct GemmOut {
  float* c0 = nullptr;
  float* c1 = nullptr;
  int64_t ldc0 = 0, ldc1 = 0;
  int64_t c_split = INT64_MAX;
  bool relu = false;
  int64_t gs0 = 0, gs1 = 0;   // element offsets of c0 / c1 between GEMM groups
  bool sgd = false;
  float lr = 0.f;
  // C[r, c] is stored as 0 where mask[r, c] > 0 fails (the ReLU derivative of
  // the layer below, applied as its input gradient is written); c0 only
  const float* mask = nullptr;
  int64_t ldm = 0, gsm = 0;
};

// `groups` independent products of the same shape: group g reads A and B
// and writes C at the pointers offset by g times their group strides.
size_t gemm_workspace(int64_t M, int64_t N, int64_t K, int dtype, int64_t groups = 1);
// k_alg: the reduction length the profiler counts (flops, bytes) when K
// includes zero padding (0: K itself).
gist_status gemm(hipStream_t st, int64_t M, int64_t N, int64_t K,
                 const Operand& A, const Operand& B, const GemmOut& C, int dtype,
                 void* ws, size_t ws_bytes, int64_t groups = 1, int64_t k_alg = 0);

// dZ[i] = dH[i] * (Hout[i] > 0) over n x w (ld = w).
gist_status relu_mask(hipStream_t st, int64_t count, const float* dH,
                      const float* Hout, float* dZ);

gist_status gather(hipStream_t st, const float* Wg, int64_t ldg,
                   const int32_t* rows, int32_t nr, const int32_t* cols,
                   int32_t nc, float* Ws, int64_t lds);
gist_status scatter(hipStream_t st, float* Wg, int64_t ldg, const int32_t* rows,
                    int32_t nr, const int32_t* cols, int32_t nc, const float* Ws,
                    int64_t lds);
gist_status count_nonfinite(hipStream_t st, const float* Ws, int64_t lds,
                            int32_t nr, int32_t nc, int* d_count);
gist_status fill_zero(hipStream_t st, float* p, int64_t count);
// dst (cols x rows, ld ldd >= rows) = src^T (src rows x cols, ld lds); columns
// rows .. ldd-1 of every dst row are set to zero.
gist_status transpose(hipStream_t st, const float* src, int64_t rows, int64_t cols, int64_t lds,
                      float* dst, int64_t ldd);
// dst <- src (bytes), by a kernel on the stream; src may be pinned host memory.
gist_status pull_copy(hipStream_t st, void* dst, const void* src, int64_t bytes);
gist_status subagg_gather(hipStream_t st, float* Wg, int64_t rows, int64_t cols, int64_t ldg,
                          int m, const gist_slice_set* done, const gist_slice_set* next, double bytes);
gist_status sgd(hipStream_t st, float* W, const float* dW, int64_t n, float lr);
gist_status subagg_mean(hipStream_t st, float* Wg, int64_t rows, int64_t cols, int64_t ldg, int m,
                        const float* const* slices, int64_t lds);
// graph attention steps (gat.hip)
gist_status gat_scores(hipStream_t st, int64_t n, int s, const float* P, int64_t ldp,
                       const float* a_src, const float* a_dst, float* u, float* v);
gist_status gat_softmax(hipStream_t st, int64_t n, int64_t nnz, const int* rowptr, const int* col,
                        const float* u, const float* v, float slope, float* alpha);
gist_status gat_edge_grad(hipStream_t st, int64_t n, int64_t nnz, int s, const int* rowptr,
                          const int* col, const float* alpha, const float* dZ, int64_t ldz,
                          const float* P, int64_t ldp, const float* u, const float* v, float slope,
                          float* dpre, float* du);
gist_status gat_mirror(hipStream_t st, int64_t n, int64_t nnz, const int* rowptr, const int* col,
                       int* tpos);
gist_status gat_mirror_sums(hipStream_t st, int64_t n, int64_t nnz, const int* rowptr,
                            const int* tpos, const float* dpre, const float* alpha, float* dv,
                            float* alpha_t);
gist_status gat_rank2(hipStream_t st, int64_t n, int s, float* dP, int64_t ld, const float* du,
                      const float* dv, const float* a_src, const float* a_dst);
size_t gat_gemv_workspace(int64_t n, int s);
gist_status gat_gemv_t(hipStream_t st, int64_t n, int s, const float* P, int64_t ldp,
                       const float* du, const float* dv, float* da_src, float* da_dst, float* part);
gist_status adam(hipStream_t st, float* W, const float* dW, float* m, float* v, int64_t n,
                 float step_size, float inv_sqrt_bc2, float beta1, float beta2, float eps,
                 bool fresh, const float* coef_dev = nullptr);
gist_status softmax_xent(hipStream_t st, int64_t n, int C, const float* logits,
                         const int32_t* labels, float* loss, float* dlogits,
                         float* partials, const int32_t* n_dev = nullptr);

}  // namespace gist
