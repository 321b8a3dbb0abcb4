// Context, error state and the device entry points of libgist.
//
// The layer entry points only validate arguments and sequence kernels on
// the context's stream; the arithmetic lives in spmm.hip, gemm.hip and
// elementwise.hip.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "gist_internal.h"

// Partial sums of gist_softmax_xent_noalloc: one float per 4-row block of
// logits, for at most GIST_NOALLOC_LOSS_MAX_ROWS rows (4 MiB).  Every GPU the
// library runs on holds its own copy until the process ends.  Host code never
// passes this array's name to a kernel: its device address is looked up once
// per device (noalloc_scratch below) and only that address is used.
static __device__ __align__(256) float scratch[GIST_NOALLOC_LOSS_MAX_ROWS / 4 + 1];

namespace gist {

namespace {
std::mutex g_scratch_mu;
std::vector<float*> g_scratch_ptr;   // device id -> address of that device's copy
}

// The device address of `scratch` on `device`, which must be current.  Looked
// up once per device (hipGetSymbolAddress), then cached.
static gist_status noalloc_scratch(int device, float** out) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (device < 0) return set_error(GIST_E_INVAL, "noalloc: bad device");
  if (static_cast<size_t>(device) >= g_scratch_ptr.size()) g_scratch_ptr.resize(device + 1, nullptr);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(GIST_E_DEVICE, std::string("noalloc: cannot resolve the loss buffer: ") +
                                          hipGetErrorString(e));
    g_scratch_ptr[device] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[device];
  return GIST_OK;
}

namespace {
thread_local std::string t_err;
}

gist_status set_error(gist_status s, const std::string& msg) {
  t_err = msg;
  return s;
}

void clear_error() { t_err.clear(); }

gist_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return set_error(GIST_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
  return GIST_OK;
}

DeviceGuard::DeviceGuard(int dev) {
  if (hipGetDevice(&prev_) == hipSuccess && prev_ != dev) {
    changed_ = hipSetDevice(dev) == hipSuccess;
  }
}

DeviceGuard::~DeviceGuard() {
  if (changed_) (void)hipSetDevice(prev_);
}

// ---- launch timing ---------------------------------------------------------

struct Profiler {
  std::vector<hipEvent_t> ev;   // 2 per slot
  std::vector<std::string> name;
  std::vector<double> flops, bytes;
  int64_t used = 0, dropped = 0;
};

namespace {
thread_local Profiler* t_prof = nullptr;
}

ProfBind::ProfBind(gist_ctx* ctx) : prev_(t_prof) { t_prof = ctx ? ctx->prof : nullptr; }
ProfBind::~ProfBind() { t_prof = prev_; }

ProfScope::ProfScope(hipStream_t st, const char* name, double flops, double bytes) : st_(st) {
  Profiler* p = t_prof;
  if (!p) return;
  if (p->used >= static_cast<int64_t>(p->name.size())) {
    ++p->dropped;
    return;
  }
  slot_ = static_cast<int>(p->used++);
  p->name[slot_] = name;
  p->flops[slot_] = flops;
  p->bytes[slot_] = bytes;
  (void)hipEventRecord(p->ev[2 * slot_], st);
}

ProfScope::~ProfScope() {
  if (slot_ >= 0 && t_prof) (void)hipEventRecord(t_prof->ev[2 * slot_ + 1], st_);
}

}  // namespace gist

using gist::set_error;

#define GIST_TRY(expr)                 \
  do {                                 \
    gist_status _s = (expr);           \
    if (_s != GIST_OK) return _s;      \
  } while (0)

extern "C" const char* gist_last_error(void) { return gist::t_err.c_str(); }

extern "C" const char* gist_status_str(gist_status s) {
  switch (s) {
    case GIST_OK: return "GIST_OK";
    case GIST_E_INVAL: return "GIST_E_INVAL";
    case GIST_E_NOMEM: return "GIST_E_NOMEM";
    case GIST_E_DEVICE: return "GIST_E_DEVICE";
    case GIST_E_UNSUPPORTED: return "GIST_E_UNSUPPORTED";
    case GIST_E_NONFINITE: return "GIST_E_NONFINITE";
  }
  return "GIST_E_UNKNOWN";
}

extern "C" gist_status gist_create(int device, void* hip_stream, gist_ctx** out) {
  gist::clear_error();
  if (!out) return set_error(GIST_E_INVAL, "gist_create: NULL out");
  int count = 0;
  hipError_t e = hipGetDeviceCount(&count);
  if (e != hipSuccess || device < 0 || device >= count)
    return set_error(GIST_E_DEVICE, "gist_create: no such HIP device");
  gist::DeviceGuard g(device);
  gist_ctx* c = new (std::nothrow) gist_ctx;
  if (!c) return set_error(GIST_E_NOMEM, "gist_create: out of host memory");
  c->device = device;
  c->stream = static_cast<hipStream_t>(hip_stream);
  if (hipMalloc(&c->d_flag, 4 * sizeof(int)) != hipSuccess) {
    delete c;
    return set_error(GIST_E_DEVICE, "gist_create: cannot allocate context flag");
  }
  // with `device` current: this device's copy of the no-allocation loss buffer
  const gist_status ss = gist::noalloc_scratch(device, &c->loss_scratch);
  if (ss != GIST_OK) {
    (void)hipFree(c->d_flag);
    delete c;
    return ss;
  }
  *out = c;
  return GIST_OK;
}

extern "C" gist_status gist_destroy(gist_ctx* ctx) {
  gist::clear_error();
  if (!ctx) return GIST_OK;
  gist_profile_end(ctx);
  {
    gist::DeviceGuard g(ctx->device);
    if (ctx->d_flag) (void)hipFree(ctx->d_flag);
  }
  delete ctx;
  return GIST_OK;
}

extern "C" gist_status gist_set_stream(gist_ctx* ctx, void* hip_stream) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "gist_set_stream: NULL ctx");
  ctx->stream = static_cast<hipStream_t>(hip_stream);
  return GIST_OK;
}

// ---------------------------------------------------------------------------
// Layer forward / backward
// ---------------------------------------------------------------------------

namespace {

size_t fbytes(int64_t a, int64_t b) { return static_cast<size_t>(a) * static_cast<size_t>(b) * 4; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int resolve_order(const gist_layer_desc* L) {
  if (L->kind == GIST_LAYER_SAGE_MEAN) return GIST_ORDER_AGG_FIRST;
  if (L->order != GIST_ORDER_AUTO) return L->order;
  return L->s_in <= L->s_out ? GIST_ORDER_AGG_FIRST : GIST_ORDER_XFORM_FIRST;
}

gist_status check_desc(const gist_layer_desc* L) {
  if (!L) return set_error(GIST_E_INVAL, "layer: NULL descriptor");
  if (L->kind != GIST_LAYER_GCN && L->kind != GIST_LAYER_SAGE_MEAN)
    return set_error(GIST_E_INVAL, "layer: unknown kind");
  if (L->act != GIST_ACT_NONE && L->act != GIST_ACT_RELU)
    return set_error(GIST_E_INVAL, "layer: unknown activation");
  if (L->dtype != GIST_DTYPE_F32 && L->dtype != GIST_DTYPE_BF16_IN)
    return set_error(GIST_E_INVAL, "layer: unknown dtype");
  if (L->order < GIST_ORDER_AUTO || L->order > GIST_ORDER_XFORM_FIRST)
    return set_error(GIST_E_INVAL, "layer: unknown order");
  if (L->kind == GIST_LAYER_SAGE_MEAN && L->order == GIST_ORDER_XFORM_FIRST)
    return set_error(GIST_E_INVAL, "layer: SAGE-mean aggregates first");
  if (L->n < 0 || L->s_in < 1 || L->s_out < 1 || L->groups < 0)
    return set_error(GIST_E_INVAL, "layer: bad sizes");
  if (L->flags & ~static_cast<uint32_t>(GIST_LAYER_SHARED_INPUT | GIST_LAYER_GROUP_MAJOR_OUT |
                                         GIST_LAYER_CLUSTERED | GIST_LAYER_DZ_IN |
                                         GIST_LAYER_MASK_DH))
    return set_error(GIST_E_INVAL, "layer: unknown flags");
  if (L->n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "layer: n exceeds int32 rows");
  if (L->n_in < 0) return set_error(GIST_E_INVAL, "layer: bad n_in");
  if (L->n_in > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "layer: n_in exceeds int32 rows");
  const int64_t n_in = L->n_in > 0 ? L->n_in : L->n;
  if (n_in != L->n && L->kind != GIST_LAYER_GCN)
    return set_error(GIST_E_INVAL, "layer: only GCN layers may be rectangular (n_in != n)");
  const int64_t G = L->groups > 1 ? L->groups : 1;
  if (G * L->s_in > INT32_MAX || G * L->s_out > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, "layer: batched width exceeds int32");
  return GIST_OK;
}

// Layout of a (possibly batched) layer: leading dimensions and per-group
// element offsets of the input-side (H, agg, dH) and output-side (H_out,
// dH_out, dZ) tensors and of the weight slices.
struct Lay {
  int64_t G, n, n_in, si, so, wrows;
  bool shared, gmajor, clustered;
  int64_t ld_in, gs_in, ld_out, gs_out, gs_w;
  int64_t gs_out_in;   // group stride of an output-width tensor with n_in rows
  int64_t w_in() const { return shared ? si : G * si; }   // aggregation width on the input side
};

Lay layout(const gist_layer_desc* L) {
  Lay y;
  y.G = L->groups > 1 ? L->groups : 1;
  y.n = L->n; y.n_in = L->n_in > 0 ? L->n_in : L->n; y.si = L->s_in; y.so = L->s_out;
  y.wrows = (L->kind == GIST_LAYER_SAGE_MEAN ? 2 : 1) * y.si;
  y.shared = (L->flags & GIST_LAYER_SHARED_INPUT) != 0;
  y.gmajor = (L->flags & GIST_LAYER_GROUP_MAJOR_OUT) != 0;
  y.clustered = (L->flags & GIST_LAYER_CLUSTERED) != 0;
  y.ld_in = y.shared ? y.si : y.G * y.si;
  y.gs_in = y.shared ? 0 : y.si;
  y.ld_out = y.gmajor ? y.so : y.G * y.so;
  y.gs_out = y.gmajor ? y.n * y.so : y.so;
  y.gs_out_in = y.gmajor ? y.n_in * y.so : y.so;
  y.gs_w = y.wrows * y.so;
  return y;
}

// Abar X (+ Add) (ReLU) for a layer's matrix A (rows x cols): the matrix-core
// tile kernel for a cluster mini-batch (GIST_LAYER_CLUSTERED), else the
// gather kernel.
gist_status aggregate(hipStream_t st, const Lay& y, const gist_csr_dev* A, int64_t rows,
                      int64_t cols, const float* X, int64_t ldx, int width, float* Y,
                      int64_t ldy, const float* add, int64_t ld_add, bool relu,
                      const float* mask = nullptr, int64_t ldm = 0) {
  if (y.clustered)
    return gist::spmm_clustered(st, rows, cols, A->nnz, A->rowptr, A->col, A->val, X, ldx, width,
                                Y, ldy, add, ld_add, relu, mask, ldm);
  return gist::spmm(st, rows, A->nnz, A->rowptr, A->col, A->val, X, ldx, width, Y, ldy, add,
                    ld_add, relu, mask, ldm);
}

// A X over output-width tensors (dZ-like layout), A with `rows` rows: one
// full-width call, or one per group when the groups are stored one after
// another (group strides gx of X and gy of Y).
gist_status spmm_out(hipStream_t st, const Lay& y, const gist_csr_dev* A, int64_t rows,
                     int64_t cols, const float* X, int64_t gx, float* Y, int64_t gy, bool relu) {
  if (!y.gmajor)
    return aggregate(st, y, A, rows, cols, X, y.ld_out, int(y.G * y.so), Y, y.ld_out, nullptr, 0,
                     relu);
  for (int64_t g = 0; g < y.G; ++g)
    GIST_TRY(aggregate(st, y, A, rows, cols, X + g * gx, y.so, int(y.so), Y + g * gy, y.so,
                       nullptr, 0, relu));
  return GIST_OK;
}

gist_status check_csr(const gist_csr_dev* A, int64_t n, const char* what) {
  if (!A) return set_error(GIST_E_INVAL, std::string(what) + ": NULL CSR");
  if (A->n != n) return set_error(GIST_E_INVAL, std::string(what) + ": CSR rows != n");
  if (A->nnz < 0 || A->nnz > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, std::string(what) + ": nnz outside int32");
  if (n > 0 && (!A->rowptr || (A->nnz > 0 && (!A->col || !A->val))))
    return set_error(GIST_E_INVAL, std::string(what) + ": NULL CSR arrays");
  return GIST_OK;
}

// The weight gradient dW = X^T D reads both of its operands across their
// rows (X and D are node-major, the reduction runs over nodes), which the
// GEMM stages through register transposes at a lower MFMA rate.  For large
// fp32 products both operands are first transposed into node-contiguous
// copies, zero-padded to a multiple of 32 nodes, so the GEMM reads
// K-contiguous tiles and every K step is whole (a ragged last step would
// take the per-element edge loads); the zero columns add nothing.
// The copies cost one read and one write of X and D; at c4 sizes (8192 x
// 4096 x 1633) the product took 921 instead of 1046 us, for three
// transposes of 18 us each.
bool transposed_dw(const gist_layer_desc* L, int64_t M, int64_t N, int64_t K) {
  const int64_t G = L->groups > 1 ? L->groups : 1;
  return L->dtype == GIST_DTYPE_F32 && G == 1 && M >= 1024 && N >= 1024 && K >= 256 &&
         (K + 31) / 32 * 32 <= 65535 * 64;   // the transpose grid: padded K in 64-row blocks
}

int64_t round32(int64_t x) { return (x + 31) / 32 * 32; }

// Workspace layout of the backward pass: [dZ | tmp | gemm scratch | X^T | D^T].
struct BwdPlan {
  size_t dz = 0, tmp = 0, gemm = 0, ta = 0, tb = 0;
  bool tdw = false;
  size_t total() const { return align256(dz) + align256(tmp) + align256(gemm) + align256(ta) + tb; }
};

BwdPlan plan_bwd(const gist_layer_desc* L) {
  BwdPlan p;
  const Lay y = layout(L);
  const int64_t n = y.n, n_in = y.n_in, si = y.si, so = y.so, G = y.G;
  if (L->act == GIST_ACT_RELU && !(L->flags & GIST_LAYER_DZ_IN)) p.dz = fbytes(n, G * so);
  const int order = resolve_order(L);
  int64_t wm, wk;   // dW = X^T D: M x so, reduced over K nodes
  if (L->kind == GIST_LAYER_SAGE_MEAN || order == GIST_ORDER_AGG_FIRST) {
    p.tmp = fbytes(n, G * si);  // dP = dZ W^T (W_neigh for SAGE)
    p.gemm = std::max(gist::gemm_workspace(y.wrows, so, n, L->dtype, G),
                      gist::gemm_workspace(n, y.wrows, so, L->dtype, G));
    wm = y.wrows;
    wk = n;
  } else {
    p.tmp = fbytes(n_in, G * so);  // Abar^T dZ
    p.gemm = std::max(gist::gemm_workspace(si, so, n_in, L->dtype, G),
                      gist::gemm_workspace(n_in, si, so, L->dtype, G));
    wm = si;
    wk = n_in;
  }
  p.tdw = transposed_dw(L, wm, so, wk);
  if (p.tdw) {
    p.ta = fbytes(wm, round32(wk));
    p.tb = fbytes(so, round32(wk));
  }
  return p;
}

size_t plan_fwd(const gist_layer_desc* L) {
  const Lay y = layout(L);
  const int order = resolve_order(L);
  if (L->kind == GIST_LAYER_GCN && order == GIST_ORDER_XFORM_FIRST)
    return align256(fbytes(y.n_in, y.G * y.so)) +
           gist::gemm_workspace(y.n_in, y.so, y.si, L->dtype, y.G);
  return gist::gemm_workspace(y.n, y.so, y.wrows, L->dtype, y.G);
}

}  // namespace

extern "C" gist_status gist_layer_workspace_size(const gist_layer_desc* L,
                                                 size_t* fwd_bytes, size_t* bwd_bytes) {
  gist::clear_error();
  GIST_TRY(check_desc(L));
  if (fwd_bytes) *fwd_bytes = plan_fwd(L);
  if (bwd_bytes) *bwd_bytes = plan_bwd(L).total();
  return GIST_OK;
}

extern "C" gist_status gist_gcn_layer_fwd(gist_ctx* ctx, const gist_layer_desc* L,
                                          const gist_csr_dev* A, const float* H,
                                          const float* W, float* agg_save,
                                          float* H_out, void* ws, size_t ws_bytes) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "layer_fwd: NULL ctx");
  gist::ProfBind pb(ctx);
  GIST_TRY(check_desc(L));
  GIST_TRY(check_csr(A, L->n, "layer_fwd"));
  const Lay y = layout(L);
  const int64_t n = y.n, n_in = y.n_in, si = y.si, so = y.so, G = y.G;
  const int order = resolve_order(L);
  const bool sage = L->kind == GIST_LAYER_SAGE_MEAN;
  if (n > 0 && (!H || !W || !H_out)) return set_error(GIST_E_INVAL, "layer_fwd: NULL pointer");
  if (n > 0 && (sage || order == GIST_ORDER_AGG_FIRST) && !agg_save)
    return set_error(GIST_E_INVAL, "layer_fwd: agg_save required");
  const size_t need = plan_fwd(L);
  if (ws_bytes < need || (need > 0 && !ws))
    return set_error(GIST_E_NOMEM, "layer_fwd: workspace too small");
  if (n == 0) return GIST_OK;
  gist::DeviceGuard dg(ctx->device);
  hipStream_t st = ctx->stream;
  const bool relu = L->act == GIST_ACT_RELU;
  gist::Operand b;  // W_g is (K x s_out) row-major: an N x K operand, N contiguous
  b.p0 = W; b.ld0 = so; b.k_major = false; b.gs0 = y.gs_w;
  if (sage || order == GIST_ORDER_AGG_FIRST) {
    // one aggregation over every group's columns (or the shared input once)
    GIST_TRY(aggregate(st, y, A, n, n_in, H, y.ld_in, int(y.w_in()), agg_save, y.ld_in, nullptr,
                       0, false));
    gist::Operand a;
    a.k_major = true;
    if (sage) {  // [H_g | Abar H_g], concatenated along K
      a.p0 = H; a.ld0 = y.ld_in; a.gs0 = y.gs_in;
      a.p1 = agg_save; a.ld1 = y.ld_in; a.gs1 = y.gs_in; a.split = si;
    } else {
      a.p0 = agg_save; a.ld0 = y.ld_in; a.gs0 = y.gs_in;
    }
    gist::GemmOut out;
    out.c0 = H_out; out.ldc0 = y.ld_out; out.gs0 = y.gs_out; out.relu = relu;
    return gist::gemm(st, n, so, y.wrows, a, b, out, L->dtype, ws, ws_bytes, G);
  }
  // transform first: T_g = H_g W_g over the n_in input rows (workspace, laid out
  // like H_out), H_out = act(Abar T)
  float* T = static_cast<float*>(ws);
  const size_t tb = align256(fbytes(n_in, G * so));
  void* gws = static_cast<char*>(ws) + tb;
  gist::Operand a;
  a.p0 = H; a.ld0 = y.ld_in; a.gs0 = y.gs_in; a.k_major = true;
  gist::GemmOut t;
  t.c0 = T; t.ldc0 = y.ld_out; t.gs0 = y.gs_out_in;
  GIST_TRY(gist::gemm(st, n_in, so, si, a, b, t, L->dtype, gws, ws_bytes - tb, G));
  return spmm_out(st, y, A, n, n_in, T, y.gs_out_in, H_out, y.gs_out, relu);
}

namespace {

// The backward pass of eq. (2).  W_sgd == nullptr: dW is written.  Else the
// SGD step W_sgd <- W_sgd - lr dW is applied by the weight-gradient GEMM's
// epilogue (W == W_sgd, dW == nullptr), after the input gradient has read W.
gist_status layer_bwd(gist_ctx* ctx, const gist_layer_desc* L, const gist_csr_dev* A,
                      const gist_csr_dev* A_T, const float* H, const float* agg_save,
                      const float* H_out, const float* W, const float* dH_out, float* dW,
                      float* W_sgd, float lr, float* dH, void* ws, size_t ws_bytes,
                      const std::string& what) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, what + ": NULL ctx");
  gist::ProfBind pb(ctx);
  GIST_TRY(check_desc(L));
  GIST_TRY(check_csr(A, L->n, what.c_str()));
  const bool sage = L->kind == GIST_LAYER_SAGE_MEAN;
  const Lay y = layout(L);
  const int64_t n = y.n, n_in = y.n_in, si = y.si, so = y.so, G = y.G;
  const std::string wt = what + " (transpose)";
  if (sage || n_in != n) GIST_TRY(check_csr(A_T, n_in, wt.c_str()));
  else if (A_T) GIST_TRY(check_csr(A_T, n_in, wt.c_str()));
  const int order = resolve_order(L);
  const bool relu = L->act == GIST_ACT_RELU;
  // dH_out already carries this layer's ReLU derivative (the layer above
  // applied it with GIST_LAYER_MASK_DH); dH takes the layer below's
  const bool dz_in = (L->flags & GIST_LAYER_DZ_IN) != 0;
  const float* dh_mask = (L->flags & GIST_LAYER_MASK_DH) ? H : nullptr;
  const bool fused = W_sgd != nullptr;
  if (!W || (!fused && !dW)) return set_error(GIST_E_INVAL, what + ": NULL dW or W");
  if (fused && !std::isfinite(lr)) return set_error(GIST_E_INVAL, what + ": lr not finite");
  if (dH && y.shared)
    return set_error(GIST_E_INVAL, what + ": a shared input has no per-group dH");
  if (n > 0 && (!H || !dH_out || (relu && !dz_in && !H_out)))
    return set_error(GIST_E_INVAL, what + ": NULL pointer");
  if (n > 0 && (sage || order == GIST_ORDER_AGG_FIRST) && !agg_save)
    return set_error(GIST_E_INVAL, what + ": agg_save required");
  const BwdPlan p = plan_bwd(L);
  if (ws_bytes < p.total() || (p.total() > 0 && !ws))
    return set_error(GIST_E_NOMEM, what + ": workspace too small");
  gist::DeviceGuard dg(ctx->device);
  hipStream_t st = ctx->stream;
  if (n == 0) {  // no output rows: zero gradients (a zero step leaves W as it is)
    if (!fused) GIST_TRY(gist::fill_zero(st, dW, G * y.wrows * so));
    return dH && n_in > 0 ? gist::fill_zero(st, dH, n_in * G * si) : GIST_OK;
  }
  char* base = static_cast<char*>(ws);
  float* dZbuf = reinterpret_cast<float*>(base);
  float* tmp = reinterpret_cast<float*>(base + align256(p.dz));
  void* gws = base + align256(p.dz) + align256(p.tmp);
  const size_t gbytes = p.gemm;
  float* tA = reinterpret_cast<float*>(base + align256(p.dz) + align256(p.tmp) +
                                       align256(p.gemm));
  float* tB = reinterpret_cast<float*>(reinterpret_cast<char*>(tA) + align256(p.ta));
  const float* dZ = dH_out;
  if (relu && !dz_in) {
    GIST_TRY(gist::relu_mask(st, n * G * so, dH_out, H_out, dZbuf));
    dZ = dZbuf;
  }
  const gist_csr_dev* AT = A_T ? A_T : A;

  gist::Operand dz_as_b;  // dZ_g (n x s_out): B operand of the weight gradient, N = s_out, K = n
  dz_as_b.p0 = dZ; dz_as_b.ld0 = y.ld_out; dz_as_b.gs0 = y.gs_out; dz_as_b.k_major = false;
  gist::GemmOut wout;     // dW_g, or the SGD step on W_g
  wout.c0 = fused ? W_sgd : dW; wout.ldc0 = so; wout.gs0 = y.gs_w;
  wout.sgd = fused; wout.lr = lr;
  gist::Operand w_as_b;   // W_g^T as an N x K operand is W_g itself (rows = N, K contiguous)
  w_as_b.p0 = W; w_as_b.ld0 = so; w_as_b.gs0 = y.gs_w; w_as_b.k_major = true;
  const int64_t ld_p = G * si;   // dP: n x (G s_in); dH: n_in x (G s_in)

  if (sage || order == GIST_ORDER_AGG_FIRST) {
    // dW_g = [H_g | Abar H_g]^T dZ_g (SAGE) or (Abar H_g)^T dZ_g: element (r, k) of the
    // transposed activation is act[k * ld + r]
    auto weight_grad = [&]() -> gist_status {
      if (p.tdw) {   // node-contiguous copies: [H | Abar H]^T (wrows x n) and dZ^T (so x n)
        const int64_t n32 = round32(n);
        if (sage) {
          GIST_TRY(gist::transpose(st, H, n, si, y.ld_in, tA, n32));
          GIST_TRY(gist::transpose(st, agg_save, n, si, y.ld_in, tA + si * n32, n32));
        } else {
          GIST_TRY(gist::transpose(st, agg_save, n, si, y.ld_in, tA, n32));
        }
        GIST_TRY(gist::transpose(st, dZ, n, so, y.ld_out, tB, n32));
        gist::Operand at, bt;
        at.p0 = tA; at.ld0 = n32; at.k_major = true;
        bt.p0 = tB; bt.ld0 = n32; bt.k_major = true;
        return gist::gemm(st, y.wrows, so, n32, at, bt, wout, L->dtype, gws, gbytes, 1, n);
      }
      gist::Operand a;
      a.k_major = false;
      if (sage) {
        a.p0 = H; a.ld0 = y.ld_in; a.gs0 = y.gs_in;
        a.p1 = agg_save; a.ld1 = y.ld_in; a.gs1 = y.gs_in; a.split = si;
      } else {
        a.p0 = agg_save; a.ld0 = y.ld_in; a.gs0 = y.gs_in;
      }
      return gist::gemm(st, y.wrows, so, n, a, dz_as_b, wout, L->dtype, gws, gbytes, G);
    };
    auto input_grad = [&]() -> gist_status {
      if (!dH) return GIST_OK;
      // [dH_self | dP]_g = dZ_g W_g^T (SAGE), dP_g = dZ_g W_g^T (GCN)
      gist::Operand a2;
      a2.p0 = dZ; a2.ld0 = y.ld_out; a2.gs0 = y.gs_out; a2.k_major = true;
      gist::GemmOut o2;
      if (sage) {
        o2.c0 = dH; o2.ldc0 = ld_p; o2.gs0 = si;
        o2.c1 = tmp; o2.ldc1 = ld_p; o2.gs1 = si; o2.c_split = si;
      } else {
        o2.c0 = tmp; o2.ldc0 = ld_p; o2.gs0 = si;
      }
      GIST_TRY(gist::gemm(st, n, y.wrows, so, a2, w_as_b, o2, L->dtype, gws, gbytes, G));
      // dH (+)= Abar^T dP, every group at once (times the layer below's
      // ReLU derivative with GIST_LAYER_MASK_DH)
      return aggregate(st, y, AT, n_in, n, tmp, ld_p, int(ld_p), dH, ld_p, sage ? dH : nullptr,
                       ld_p, false, dh_mask, y.ld_in);
    };
    if (fused) {
      GIST_TRY(input_grad());
      return weight_grad();
    }
    GIST_TRY(weight_grad());
    return input_grad();
  }
  // GCN transform-first: T = Abar^T dZ (n_in rows, laid out like dZ); dW_g = H_g^T T_g;
  // dH_g = T_g W_g^T
  GIST_TRY(spmm_out(st, y, AT, n_in, n, dZ, y.gs_out, tmp, y.gs_out_in, false));
  auto weight_grad = [&]() -> gist_status {
    if (p.tdw) {   // node-contiguous copies H^T (si x n_in) and T^T (so x n_in)
      const int64_t n32 = round32(n_in);
      GIST_TRY(gist::transpose(st, H, n_in, si, y.ld_in, tA, n32));
      GIST_TRY(gist::transpose(st, tmp, n_in, so, y.ld_out, tB, n32));
      gist::Operand at, bt;
      at.p0 = tA; at.ld0 = n32; at.k_major = true;
      bt.p0 = tB; bt.ld0 = n32; bt.k_major = true;
      return gist::gemm(st, si, so, n32, at, bt, wout, L->dtype, gws, gbytes, 1, n_in);
    }
    gist::Operand a;
    a.p0 = H; a.ld0 = y.ld_in; a.gs0 = y.gs_in; a.k_major = false;
    gist::Operand g;
    g.p0 = tmp; g.ld0 = y.ld_out; g.gs0 = y.gs_out_in; g.k_major = false;
    return gist::gemm(st, si, so, n_in, a, g, wout, L->dtype, gws, gbytes, G);
  };
  auto input_grad = [&]() -> gist_status {
    if (!dH) return GIST_OK;
    gist::Operand a2;
    a2.p0 = tmp; a2.ld0 = y.ld_out; a2.gs0 = y.gs_out_in; a2.k_major = true;
    gist::GemmOut o2;
    o2.c0 = dH; o2.ldc0 = ld_p; o2.gs0 = si;
    o2.mask = dh_mask; o2.ldm = y.ld_in; o2.gsm = y.gs_in;
    return gist::gemm(st, n_in, si, so, a2, w_as_b, o2, L->dtype, gws, gbytes, G);
  };
  if (fused) {
    GIST_TRY(input_grad());
    return weight_grad();
  }
  GIST_TRY(weight_grad());
  return input_grad();
}

}  // namespace

extern "C" gist_status gist_gcn_layer_bwd(gist_ctx* ctx, const gist_layer_desc* L,
                                          const gist_csr_dev* A, const gist_csr_dev* A_T,
                                          const float* H, const float* agg_save,
                                          const float* H_out, const float* W,
                                          const float* dH_out, float* dW, float* dH,
                                          void* ws, size_t ws_bytes) {
  return layer_bwd(ctx, L, A, A_T, H, agg_save, H_out, W, dH_out, dW, nullptr, 0.f, dH, ws,
                   ws_bytes, "layer_bwd");
}

extern "C" gist_status gist_gcn_layer_bwd_sgd(gist_ctx* ctx, const gist_layer_desc* L,
                                              const gist_csr_dev* A, const gist_csr_dev* A_T,
                                              const float* H, const float* agg_save,
                                              const float* H_out, float* W, const float* dH_out,
                                              float lr, float* dH, void* ws, size_t ws_bytes) {
  return layer_bwd(ctx, L, A, A_T, H, agg_save, H_out, W, dH_out, nullptr, W, lr, dH, ws,
                   ws_bytes, "layer_bwd_sgd");
}

// ---------------------------------------------------------------------------
// Graph attention layer
// ---------------------------------------------------------------------------

namespace {

gist_status check_gat(const gist_gat_desc* D, const gist_csr_dev* A, const char* what) {
  if (!D) return set_error(GIST_E_INVAL, std::string(what) + ": NULL descriptor");
  if (D->n < 0 || D->nnz < 0 || D->s_in < 1 || D->s_out < 1 ||
      (D->flags & ~static_cast<uint32_t>(GIST_GAT_MIRROR_IN_WS)))
    return set_error(GIST_E_INVAL, std::string(what) + ": bad sizes");
  if (D->act != GIST_ACT_NONE && D->act != GIST_ACT_RELU)
    return set_error(GIST_E_INVAL, std::string(what) + ": unknown activation");
  if (D->dtype != GIST_DTYPE_F32 && D->dtype != GIST_DTYPE_BF16_IN)
    return set_error(GIST_E_INVAL, std::string(what) + ": unknown dtype");
  if (!std::isfinite(D->slope)) return set_error(GIST_E_INVAL, std::string(what) + ": bad slope");
  if (D->n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, std::string(what) + ": n exceeds int32");
  if (A) {
    GIST_TRY(check_csr(A, D->n, what));
    if (A->nnz != D->nnz) return set_error(GIST_E_INVAL, std::string(what) + ": CSR nnz != desc nnz");
  }
  return GIST_OK;
}

// backward workspace: [tpos | dZ | u | v | dpre | du | dv | alpha_t | dP | gemv | gemm];
// the mirror map tpos comes first, so that it stays in place for the next
// layer's call on the same pattern (GIST_GAT_MIRROR_IN_WS)
struct GatPlan {
  size_t dz, uv, dpre, dudv, tpos, alpha_t, dp, gemv, gemm;
  size_t total() const {
    return align256(tpos) + align256(dz) + align256(uv) + align256(dpre) + align256(dudv) +
           align256(alpha_t) + align256(dp) + align256(gemv) + gemm;
  }
};

GatPlan plan_gat_bwd(const gist_gat_desc* D) {
  GatPlan p{};
  const int64_t n = D->n, si = D->s_in, so = D->s_out;
  p.dz = D->act == GIST_ACT_RELU ? fbytes(n, so) : 0;
  p.uv = fbytes(2, n);
  p.dpre = fbytes(1, D->nnz);
  p.dudv = fbytes(2, n);
  p.tpos = static_cast<size_t>(D->nnz) * sizeof(int);
  p.alpha_t = fbytes(1, D->nnz);
  p.dp = fbytes(n, so);
  p.gemv = gist::gat_gemv_workspace(n, static_cast<int>(so));
  p.gemm = std::max(gist::gemm_workspace(si, so, n, D->dtype),
                    gist::gemm_workspace(n, si, so, D->dtype));
  return p;
}

size_t plan_gat_fwd(const gist_gat_desc* D) {
  return align256(fbytes(2, D->n)) + gist::gemm_workspace(D->n, D->s_out, D->s_in, D->dtype);
}

}  // namespace

extern "C" gist_status gist_gat_workspace_size(const gist_gat_desc* D, size_t* fwd_bytes,
                                               size_t* bwd_bytes) {
  gist::clear_error();
  GIST_TRY(check_gat(D, nullptr, "gat_workspace_size"));
  if (fwd_bytes) *fwd_bytes = plan_gat_fwd(D);
  if (bwd_bytes) *bwd_bytes = plan_gat_bwd(D).total();
  return GIST_OK;
}

extern "C" gist_status gist_gat_scores(gist_ctx* ctx, int64_t n, int32_t s, const float* P,
                                       int64_t ldp, const float* a_src, const float* a_dst,
                                       float* u, float* v) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "gat_scores: NULL ctx");
  gist::ProfBind pb(ctx);
  if (n < 0 || s < 1 || ldp < s) return set_error(GIST_E_INVAL, "gat_scores: bad sizes");
  if (n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "gat_scores: n exceeds int32");
  if (n == 0) return GIST_OK;
  if (!P || !a_src || !a_dst || !u || !v) return set_error(GIST_E_INVAL, "gat_scores: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  return gist::gat_scores(ctx->stream, n, s, P, ldp, a_src, a_dst, u, v);
}

extern "C" gist_status gist_gat_layer_fwd(gist_ctx* ctx, const gist_gat_desc* D,
                                          const gist_csr_dev* A, const float* H, const float* W,
                                          const float* a_src, const float* a_dst, float* P_save,
                                          float* alpha_save, float* H_out, void* ws,
                                          size_t ws_bytes) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "gat_fwd: NULL ctx");
  gist::ProfBind pb(ctx);
  GIST_TRY(check_gat(D, A, "gat_fwd"));
  const int64_t n = D->n, si = D->s_in, so = D->s_out;
  if (n > 0 && (!H || !W || !a_src || !a_dst || !P_save || !H_out || (D->nnz > 0 && !alpha_save)))
    return set_error(GIST_E_INVAL, "gat_fwd: NULL pointer");
  const size_t need = plan_gat_fwd(D);
  if (ws_bytes < need || (need > 0 && !ws)) return set_error(GIST_E_NOMEM, "gat_fwd: workspace too small");
  if (n == 0) return GIST_OK;
  gist::DeviceGuard dg(ctx->device);
  hipStream_t st = ctx->stream;
  float* u = static_cast<float*>(ws);
  float* v = u + n;
  void* gws = static_cast<char*>(ws) + align256(fbytes(2, n));
  const size_t gbytes = ws_bytes - align256(fbytes(2, n));
  // P = H W
  gist::Operand a;
  a.p0 = H; a.ld0 = si; a.k_major = true;
  gist::Operand b;
  b.p0 = W; b.ld0 = so; b.k_major = false;
  gist::GemmOut pc;
  pc.c0 = P_save; pc.ldc0 = so;
  GIST_TRY(gist::gemm(st, n, so, si, a, b, pc, D->dtype, gws, gbytes));
  GIST_TRY(gist::gat_scores(st, n, static_cast<int>(so), P_save, so, a_src, a_dst, u, v));
  GIST_TRY(gist::gat_softmax(st, n, D->nnz, A->rowptr, A->col, u, v, D->slope, alpha_save));
  // H_out = act(A_alpha P)
  return gist::spmm(st, n, D->nnz, A->rowptr, A->col, alpha_save, P_save, so, int(so), H_out, so,
                    nullptr, 0, D->act == GIST_ACT_RELU);
}

extern "C" gist_status gist_gat_layer_bwd(gist_ctx* ctx, const gist_gat_desc* D,
                                          const gist_csr_dev* A, const float* H,
                                          const float* P_save, const float* alpha_save,
                                          const float* H_out, const float* W, const float* a_src,
                                          const float* a_dst, const float* dH_out, float* dW,
                                          float* da_src, float* da_dst, float* dH, void* ws,
                                          size_t ws_bytes) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "gat_bwd: NULL ctx");
  gist::ProfBind pb(ctx);
  GIST_TRY(check_gat(D, A, "gat_bwd"));
  const int64_t n = D->n, si = D->s_in, so = D->s_out;
  const bool relu = D->act == GIST_ACT_RELU;
  if (!dW || !W || !a_src || !a_dst || !da_src || !da_dst)
    return set_error(GIST_E_INVAL, "gat_bwd: NULL pointer");
  if (n > 0 && (!H || !P_save || !dH_out || (relu && !H_out) || (D->nnz > 0 && !alpha_save)))
    return set_error(GIST_E_INVAL, "gat_bwd: NULL pointer");
  const GatPlan p = plan_gat_bwd(D);
  if (ws_bytes < p.total() || (p.total() > 0 && !ws))
    return set_error(GIST_E_NOMEM, "gat_bwd: workspace too small");
  gist::DeviceGuard dg(ctx->device);
  hipStream_t st = ctx->stream;
  if (n == 0) {   // empty batch: zero gradients
    GIST_TRY(gist::fill_zero(st, dW, si * so));
    GIST_TRY(gist::fill_zero(st, da_src, so));
    return gist::fill_zero(st, da_dst, so);
  }
  char* c = static_cast<char*>(ws);
  auto take = [&](size_t bytes) { char* r = c; c += align256(bytes); return r; };
  int* tpos = reinterpret_cast<int*>(take(p.tpos));
  float* dZbuf = reinterpret_cast<float*>(take(p.dz));
  float* u = reinterpret_cast<float*>(take(p.uv));
  float* v = u + n;
  float* dpre = reinterpret_cast<float*>(take(p.dpre));
  float* du = reinterpret_cast<float*>(take(p.dudv));
  float* dv = du + n;
  float* alpha_t = reinterpret_cast<float*>(take(p.alpha_t));
  float* dP = reinterpret_cast<float*>(take(p.dp));
  float* part = reinterpret_cast<float*>(take(p.gemv));
  void* gws = c;
  const float* dZ = dH_out;
  if (relu) {
    GIST_TRY(gist::relu_mask(st, n * so, dH_out, H_out, dZbuf));
    dZ = dZbuf;
  }
  const int s = static_cast<int>(so);
  GIST_TRY(gist::gat_scores(st, n, s, P_save, so, a_src, a_dst, u, v));
  GIST_TRY(gist::gat_edge_grad(st, n, D->nnz, s, A->rowptr, A->col, alpha_save, dZ, so, P_save, so,
                               u, v, D->slope, dpre, du));
  if (!(D->flags & GIST_GAT_MIRROR_IN_WS))
    GIST_TRY(gist::gat_mirror(st, n, D->nnz, A->rowptr, A->col, tpos));
  GIST_TRY(gist::gat_mirror_sums(st, n, D->nnz, A->rowptr, tpos, dpre, alpha_save, dv, alpha_t));
  // dP = A_alpha^T dZ (the pattern is symmetric: row j lists the i with alpha_ij)
  GIST_TRY(gist::spmm(st, n, D->nnz, A->rowptr, A->col, alpha_t, dZ, so, s, dP, so, nullptr, 0,
                      false));
  GIST_TRY(gist::gat_gemv_t(st, n, s, P_save, so, du, dv, da_src, da_dst, part));
  GIST_TRY(gist::gat_rank2(st, n, s, dP, so, du, dv, a_src, a_dst));
  // dW = H^T dP; dH = dP W^T
  gist::Operand a;
  a.p0 = H; a.ld0 = si; a.k_major = false;
  gist::Operand g;
  g.p0 = dP; g.ld0 = so; g.k_major = false;
  gist::GemmOut wout;
  wout.c0 = dW; wout.ldc0 = so;
  GIST_TRY(gist::gemm(st, si, so, n, a, g, wout, D->dtype, gws, p.gemm));
  if (!dH) return GIST_OK;
  gist::Operand a2;
  a2.p0 = dP; a2.ld0 = so; a2.k_major = true;
  gist::Operand b2;
  b2.p0 = W; b2.ld0 = so; b2.k_major = true;
  gist::GemmOut o2;
  o2.c0 = dH; o2.ldc0 = si;
  return gist::gemm(st, n, si, so, a2, b2, o2, D->dtype, gws, p.gemm);
}

// ---------------------------------------------------------------------------
// Loss, gather, SGD, subAgg
// ---------------------------------------------------------------------------

extern "C" size_t gist_softmax_xent_workspace(int64_t n) {
  // one partial sum per 4-row block (one wave per row)
  if (n < 0) n = 0;
  return align256(static_cast<size_t>((n + 3) / 4 + 1) * sizeof(float));
}

extern "C" gist_status gist_softmax_xent(gist_ctx* ctx, int64_t n, int32_t C,
                                         const float* logits, const int32_t* labels,
                                         float* loss_dev, float* dlogits, void* ws,
                                         size_t ws_bytes) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "softmax_xent: NULL ctx");
  gist::ProfBind pb(ctx);
  if (n < 0 || C < 1) return set_error(GIST_E_INVAL, "softmax_xent: bad sizes");
  if (!loss_dev || (n > 0 && (!logits || !labels || !dlogits)))
    return set_error(GIST_E_INVAL, "softmax_xent: NULL pointer");
  if (n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "softmax_xent: n exceeds int32");
  if (ws_bytes < gist_softmax_xent_workspace(n) || !ws)
    return set_error(GIST_E_NOMEM, "softmax_xent: workspace too small");
  gist::DeviceGuard dg(ctx->device);
  return gist::softmax_xent(ctx->stream, n, C, logits, labels, loss_dev, dlogits,
                            static_cast<float*>(ws));
}

extern "C" gist_status gist_softmax_xent_noalloc(gist_ctx* ctx, int64_t n, int32_t C,
                                                 const float* logits, const int32_t* labels,
                                                 float* loss_dev, float* dlogits) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "softmax_xent_noalloc: NULL ctx");
  gist::ProfBind pb(ctx);
  if (n < 0 || C < 1) return set_error(GIST_E_INVAL, "softmax_xent_noalloc: bad sizes");
  if (n > GIST_NOALLOC_LOSS_MAX_ROWS)
    return set_error(GIST_E_INVAL, "softmax_xent_noalloc: n exceeds GIST_NOALLOC_LOSS_MAX_ROWS "
                                   "(4194304 rows); use gist_softmax_xent with a workspace");
  if (!loss_dev || (n > 0 && (!logits || !labels || !dlogits)))
    return set_error(GIST_E_INVAL, "softmax_xent_noalloc: NULL pointer");
  if (!ctx->loss_scratch) return set_error(GIST_E_DEVICE, "softmax_xent_noalloc: no loss buffer");
  gist::DeviceGuard dg(ctx->device);
  // the rows kernel writes every partial the finishing kernel reads, so the
  // buffer needs no clearing between calls
  return gist::softmax_xent(ctx->stream, n, C, logits, labels, loss_dev, dlogits,
                            ctx->loss_scratch);
}

extern "C" gist_status gist_softmax_xent_padded(gist_ctx* ctx, int64_t n, int32_t C,
                                                const float* logits, const int32_t* labels,
                                                const int32_t* n_valid_dev, float* loss_dev,
                                                float* dlogits, void* ws, size_t ws_bytes) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "softmax_xent_padded: NULL ctx");
  if (!n_valid_dev) return set_error(GIST_E_INVAL, "softmax_xent_padded: NULL row count");
  gist::ProfBind pb(ctx);
  if (n < 0 || C < 1) return set_error(GIST_E_INVAL, "softmax_xent_padded: bad sizes");
  if (!loss_dev || (n > 0 && (!logits || !labels || !dlogits)))
    return set_error(GIST_E_INVAL, "softmax_xent_padded: NULL pointer");
  if (n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "softmax_xent_padded: n exceeds int32");
  if (ws_bytes < gist_softmax_xent_workspace(n) || !ws)
    return set_error(GIST_E_NOMEM, "softmax_xent_padded: workspace too small");
  gist::DeviceGuard dg(ctx->device);
  return gist::softmax_xent(ctx->stream, n, C, logits, labels, loss_dev, dlogits,
                            static_cast<float*>(ws), n_valid_dev);
}

extern "C" gist_status gist_gather_slice(gist_ctx* ctx, const float* Wg, int64_t ldg,
                                         const int32_t* rows, int32_t nr,
                                         const int32_t* cols, int32_t nc, float* Ws,
                                         int64_t lds) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "gather_slice: NULL ctx");
  gist::ProfBind pb(ctx);
  if (nr < 0 || nc < 0 || lds < nc || ldg < 1 || (!cols && ldg < nc))
    return set_error(GIST_E_INVAL, "gather_slice: bad sizes");
  if (nr == 0 || nc == 0) return GIST_OK;
  if (!Wg || !Ws) return set_error(GIST_E_INVAL, "gather_slice: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  return gist::gather(ctx->stream, Wg, ldg, rows, nr, cols, nc, Ws, lds);
}

extern "C" gist_status gist_sgd_update(gist_ctx* ctx, float* W, const float* dW, int64_t n,
                                       float lr) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "sgd_update: NULL ctx");
  gist::ProfBind pb(ctx);
  if (n < 0) return set_error(GIST_E_INVAL, "sgd_update: n < 0");
  if (n == 0) return GIST_OK;
  if (!W || !dW) return set_error(GIST_E_INVAL, "sgd_update: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  return gist::sgd(ctx->stream, W, dW, n, lr);
}

extern "C" gist_status gist_subagg_mean(gist_ctx* ctx, float* Wg, int64_t rows, int64_t cols,
                                        int64_t ldg, int32_t m, const float* const* slices,
                                        int64_t lds) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "subagg_mean: NULL ctx");
  gist::ProfBind pb(ctx);
  if (rows < 0 || cols < 0 || m < 1 || ldg < cols || lds < cols)
    return set_error(GIST_E_INVAL, "subagg_mean: bad sizes");
  if (rows == 0 || cols == 0) return GIST_OK;
  if (!Wg || !slices) return set_error(GIST_E_INVAL, "subagg_mean: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  return gist::subagg_mean(ctx->stream, Wg, rows, cols, ldg, m, slices, lds);
}

namespace {
// The step-dependent Adam coefficients, formed in double and rounded once:
// {lr / (1 - beta1^k), 1 / sqrt(1 - beta2^k), fresh}.
gist_status adam_coef(const char* what, float lr, float beta1, float beta2, float eps,
                      int64_t step, uint32_t flags, float* out) {
  if (step < 1) return set_error(GIST_E_INVAL, std::string(what) + ": step counts from 1");
  if (!(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f))
    return set_error(GIST_E_INVAL, std::string(what) + ": beta outside [0, 1)");
  if (!(eps >= 0.f) || !std::isfinite(lr) || !std::isfinite(eps))
    return set_error(GIST_E_INVAL, std::string(what) + ": bad lr or eps");
  if (flags & ~static_cast<uint32_t>(GIST_ADAM_FRESH))
    return set_error(GIST_E_INVAL, std::string(what) + ": unknown flags");
  const double bc1 = 1.0 - std::pow(static_cast<double>(beta1), static_cast<double>(step));
  const double bc2 = 1.0 - std::pow(static_cast<double>(beta2), static_cast<double>(step));
  if (!(bc1 > 0.0) || !(bc2 > 0.0))
    return set_error(GIST_E_INVAL,
                     std::string(what) + ": zero bias correction (beta = 0 needs no step)");
  out[0] = static_cast<float>(lr / bc1);
  out[1] = static_cast<float>(1.0 / std::sqrt(bc2));
  out[2] = (flags & GIST_ADAM_FRESH) ? 1.f : 0.f;
  return GIST_OK;
}
}  // namespace

extern "C" gist_status gist_adam_coefficients(float lr, float beta1, float beta2, float eps,
                                              int64_t step, uint32_t flags, float* coef3) {
  gist::clear_error();
  if (!coef3) return set_error(GIST_E_INVAL, "adam_coefficients: NULL out");
  return adam_coef("adam_coefficients", lr, beta1, beta2, eps, step, flags, coef3);
}

extern "C" gist_status gist_adam_update(gist_ctx* ctx, float* W, const float* dW, float* m,
                                        float* v, int64_t n, float lr, float beta1, float beta2,
                                        float eps, int64_t step, uint32_t flags) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "adam_update: NULL ctx");
  gist::ProfBind pb(ctx);
  if (n < 0) return set_error(GIST_E_INVAL, "adam_update: n < 0");
  float c[3];
  GIST_TRY(adam_coef("adam_update", lr, beta1, beta2, eps, step, flags, c));
  if (n == 0) return GIST_OK;
  if (!W || !dW || !m || !v) return set_error(GIST_E_INVAL, "adam_update: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  return gist::adam(ctx->stream, W, dW, m, v, n, c[0], c[1], beta1, beta2, eps, c[2] != 0.f);
}

extern "C" gist_status gist_adam_update_dev(gist_ctx* ctx, float* W, const float* dW, float* m,
                                            float* v, int64_t n, float beta1, float beta2,
                                            float eps, const float* coef_dev) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "adam_update_dev: NULL ctx");
  gist::ProfBind pb(ctx);
  if (n < 0) return set_error(GIST_E_INVAL, "adam_update_dev: n < 0");
  if (!(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f))
    return set_error(GIST_E_INVAL, "adam_update_dev: beta outside [0, 1)");
  if (!(eps >= 0.f) || !std::isfinite(eps))
    return set_error(GIST_E_INVAL, "adam_update_dev: bad eps");
  if (!coef_dev) return set_error(GIST_E_INVAL, "adam_update_dev: NULL coefficients");
  if (n == 0) return GIST_OK;
  if (!W || !dW || !m || !v) return set_error(GIST_E_INVAL, "adam_update_dev: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  return gist::adam(ctx->stream, W, dW, m, v, n, 0.f, 0.f, beta1, beta2, eps, false, coef_dev);
}

extern "C" gist_status gist_subagg(gist_ctx* ctx, float* Wg, int64_t ldg,
                                   const int32_t* rows, int32_t nr, const int32_t* cols,
                                   int32_t nc, const float* Ws, int64_t lds, uint32_t flags) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "subagg: NULL ctx");
  gist::ProfBind pb(ctx);
  if (flags & ~GIST_SUBAGG_CHECK_FINITE) return set_error(GIST_E_INVAL, "subagg: unknown flags");
  if (nr < 0 || nc < 0 || lds < nc || ldg < 1 || (!cols && ldg < nc))
    return set_error(GIST_E_INVAL, "subagg: bad sizes");
  if (nr == 0 || nc == 0) return GIST_OK;
  if (!Wg || !Ws) return set_error(GIST_E_INVAL, "subagg: NULL pointer");
  gist::DeviceGuard dg(ctx->device);
  if (flags & GIST_SUBAGG_CHECK_FINITE) {
    GIST_TRY(gist::count_nonfinite(ctx->stream, Ws, lds, nr, nc, ctx->d_flag));
    int bad = 0;
    if (hipMemcpyAsync(&bad, ctx->d_flag, sizeof(int), hipMemcpyDeviceToHost, ctx->stream) !=
            hipSuccess ||
        hipStreamSynchronize(ctx->stream) != hipSuccess)
      return gist::check_launch("subagg: finite check");
    if (bad) return set_error(GIST_E_NONFINITE, "subagg: slice holds NaN or Inf; nothing written");
  }
  return gist::scatter(ctx->stream, Wg, ldg, rows, nr, cols, nc, Ws, lds);
}

extern "C" gist_status gist_subagg_gather(gist_ctx* ctx, float* Wg, int64_t rows, int64_t cols,
                                          int64_t ldg, int32_t m, const gist_slice_set* done,
                                          const gist_slice_set* next) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "subagg_gather: NULL ctx");
  gist::ProfBind pb(ctx);
  if (rows < 0 || cols < 0 || m < 1 || ldg < cols) return set_error(GIST_E_INVAL, "subagg_gather: bad sizes");
  if (rows > INT32_MAX || cols > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, "subagg_gather: dimension exceeds int32 ranks");
  if (rows == 0 || cols == 0 || (!done && !next)) return GIST_OK;
  if (!Wg) return set_error(GIST_E_INVAL, "subagg_gather: NULL matrix");
  for (const gist_slice_set* s : {done, next}) {
    if (!s) continue;
    if (!s->slices || s->ld < 1) return set_error(GIST_E_INVAL, "subagg_gather: bad slice set");
    if (!s->row_rank != !s->row_offs || !s->col_rank != !s->col_offs)
      return set_error(GIST_E_INVAL, "subagg_gather: ranks and offsets come in pairs");
    if (m > 1 && !s->row_rank && !s->col_rank)
      return set_error(GIST_E_INVAL, "subagg_gather: m > 1 needs a partitioned dimension");
  }
  if (done && next && done->slices == next->slices)
    return set_error(GIST_E_INVAL, "subagg_gather: done and next share one slice table");
  gist::DeviceGuard dg(ctx->device);
  // algorithmic bytes: the matrix read once (and written once with `done`),
  // plus the slices' elements read (done) and written (next)
  double bytes = (done ? 8.0 : 4.0) * static_cast<double>(rows) * cols;
  auto slice_elems = [&](const gist_slice_set* s) {
    const double fr = s->row_rank ? 1.0 / m : 1.0, fc = s->col_rank ? 1.0 / m : 1.0;
    return static_cast<double>(rows) * cols * fr * fc * m;
  };
  if (done) bytes += 4.0 * slice_elems(done);
  if (next) bytes += 4.0 * slice_elems(next);
  return gist::subagg_gather(ctx->stream, Wg, rows, cols, ldg, m, done, next, bytes);
}

// ---------------------------------------------------------------------------
// Instrumentation
// ---------------------------------------------------------------------------

extern "C" gist_status gist_profile_begin(gist_ctx* ctx, int64_t cap) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "profile_begin: NULL ctx");
  if (cap < 1 || cap > (1 << 22)) return set_error(GIST_E_INVAL, "profile_begin: bad capacity");
  gist_profile_end(ctx);
  gist::DeviceGuard dg(ctx->device);
  auto* p = new (std::nothrow) gist::Profiler;
  if (!p) return set_error(GIST_E_NOMEM, "profile_begin: out of host memory");
  p->ev.resize(static_cast<size_t>(2 * cap));
  for (auto& e : p->ev) {
    if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
      for (auto& f : p->ev)
        if (f) (void)hipEventDestroy(f);
      delete p;
      return set_error(GIST_E_DEVICE, "profile_begin: hipEventCreate failed");
    }
  }
  p->name.resize(static_cast<size_t>(cap));
  p->flops.assign(static_cast<size_t>(cap), 0.0);
  p->bytes.assign(static_cast<size_t>(cap), 0.0);
  ctx->prof = p;
  return GIST_OK;
}

extern "C" gist_status gist_profile_read(gist_ctx* ctx, gist_prof_entry* out, int32_t out_cap,
                                         int32_t* n, int64_t* dropped) {
  gist::clear_error();
  if (!ctx || !n) return set_error(GIST_E_INVAL, "profile_read: NULL argument");
  *n = 0;
  gist::Profiler* p = ctx->prof;
  if (!p) return set_error(GIST_E_INVAL, "profile_read: profiling not started");
  gist::DeviceGuard dg(ctx->device);
  if (hipStreamSynchronize(ctx->stream) != hipSuccess) return gist::check_launch("profile_read");
  std::map<std::string, gist_prof_entry> agg;
  for (int64_t i = 0; i < p->used; ++i) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p->ev[2 * i], p->ev[2 * i + 1]) != hipSuccess)
      return gist::check_launch("profile_read: elapsed time");
    gist_prof_entry& e = agg[p->name[i]];
    std::strncpy(e.name, p->name[i].c_str(), sizeof(e.name) - 1);
    e.launches += 1;
    e.ms += ms;
    e.flops += p->flops[i];
    e.bytes += p->bytes[i];
  }
  if (dropped) *dropped = p->dropped;
  int32_t k = 0;
  for (auto& kv : agg) {
    if (k >= out_cap) break;
    if (out) out[k] = kv.second;
    ++k;
  }
  *n = k;
  p->used = 0;
  p->dropped = 0;
  return GIST_OK;
}

extern "C" gist_status gist_profile_end(gist_ctx* ctx) {
  if (!ctx) return set_error(GIST_E_INVAL, "profile_end: NULL ctx");
  gist::Profiler* p = ctx->prof;
  if (!p) return GIST_OK;
  gist::DeviceGuard dg(ctx->device);
  (void)hipStreamSynchronize(ctx->stream);
  for (auto& e : p->ev)
    if (e) (void)hipEventDestroy(e);
  delete p;
  ctx->prof = nullptr;
  return GIST_OK;
}

// ---------------------------------------------------------------------------
// Replays: HIP graphs of library calls, and events
// ---------------------------------------------------------------------------

struct gist_replay {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

struct gist_event {
  hipEvent_t ev = nullptr;
};

namespace {
gist_status hip_fail(const char* what, hipError_t e) {
  (void)hipGetLastError();   // clear the runtime's record of it
  return set_error(GIST_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}
}  // namespace

extern "C" gist_status gist_capture_begin(gist_ctx* ctx) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "capture_begin: NULL ctx");
  if (!ctx->stream)
    return set_error(GIST_E_INVAL, "capture_begin: the context's stream is the default stream");
  if (ctx->prof)
    return set_error(GIST_E_INVAL, "capture_begin: the context is recording a profile");
  gist::DeviceGuard dg(ctx->device);
  hipError_t e = hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) return hip_fail("capture_begin", e);
  return GIST_OK;
}

extern "C" gist_status gist_capture_end(gist_ctx* ctx, gist_replay** out) {
  gist::clear_error();
  if (!ctx || !out) return set_error(GIST_E_INVAL, "capture_end: NULL argument");
  *out = nullptr;
  gist::DeviceGuard dg(ctx->device);
  hipGraph_t g = nullptr;
  if (hipStreamEndCapture(ctx->stream, &g) != hipSuccess || !g) {
    if (g) (void)hipGraphDestroy(g);
    (void)hipGetLastError();
    return set_error(GIST_E_DEVICE, "capture_end: the capture failed (a call made during it "
                                    "is not capturable, or the capture was invalidated)");
  }
  hipGraphExec_t e = nullptr;
  const hipError_t ie = hipGraphInstantiate(&e, g, nullptr, nullptr, 0);
  if (ie != hipSuccess) {
    (void)hipGraphDestroy(g);
    return hip_fail("capture_end (instantiate)", ie);
  }
  gist_replay* r = new (std::nothrow) gist_replay;
  if (!r) {
    (void)hipGraphExecDestroy(e);
    (void)hipGraphDestroy(g);
    return set_error(GIST_E_NOMEM, "capture_end: out of host memory");
  }
  r->graph = g;
  r->exec = e;
  *out = r;
  return GIST_OK;
}

extern "C" gist_status gist_replay_launch(gist_ctx* ctx, gist_replay* r, void* dst,
                                          const void* src, size_t bytes, gist_event* copied) {
  gist::clear_error();
  if (!ctx || !r) return set_error(GIST_E_INVAL, "replay_launch: NULL argument");
  if (bytes && (!dst || !src)) return set_error(GIST_E_INVAL, "replay_launch: NULL copy buffer");
  gist::DeviceGuard dg(ctx->device);
  gist::ProfBind pb(ctx);
  hipError_t e = hipSuccess;
  // the copy is a kernel on the stream reading the pinned source over the
  // host link: unlike a copy-engine transfer it needs no hand-off between
  // engines before the replay starts
  if (bytes) GIST_TRY(gist::pull_copy(ctx->stream, dst, src, static_cast<int64_t>(bytes)));
  if (copied && (e = hipEventRecord(copied->ev, ctx->stream)) != hipSuccess)
    return hip_fail("replay_launch (event)", e);
  if ((e = hipGraphLaunch(r->exec, ctx->stream)) != hipSuccess)
    return hip_fail("replay_launch", e);
  return GIST_OK;
}

extern "C" gist_status gist_copy(gist_ctx* ctx, void* dst, const void* src, size_t bytes,
                                 gist_event* copied) {
  gist::clear_error();
  if (!ctx) return set_error(GIST_E_INVAL, "copy: NULL ctx");
  if (bytes && (!dst || !src)) return set_error(GIST_E_INVAL, "copy: NULL buffer");
  gist::ProfBind pb(ctx);
  gist::DeviceGuard dg(ctx->device);
  if (bytes) GIST_TRY(gist::pull_copy(ctx->stream, dst, src, static_cast<int64_t>(bytes)));
  if (copied) {
    const hipError_t e = hipEventRecord(copied->ev, ctx->stream);
    if (e != hipSuccess) return hip_fail("copy (event)", e);
  }
  return GIST_OK;
}

extern "C" gist_status gist_replay_destroy(gist_replay* r) {
  gist::clear_error();
  if (!r) return GIST_OK;
  if (r->exec) (void)hipGraphExecDestroy(r->exec);
  if (r->graph) (void)hipGraphDestroy(r->graph);
  delete r;
  return GIST_OK;
}

extern "C" gist_status gist_event_create(gist_event** out) {
  gist::clear_error();
  if (!out) return set_error(GIST_E_INVAL, "event_create: NULL out");
  gist_event* e = new (std::nothrow) gist_event;
  if (!e) return set_error(GIST_E_NOMEM, "event_create: out of host memory");
  const hipError_t he = hipEventCreateWithFlags(&e->ev, hipEventDisableTiming);
  if (he != hipSuccess) {
    delete e;
    return hip_fail("event_create", he);
  }
  *out = e;
  return GIST_OK;
}

extern "C" gist_status gist_event_synchronize(gist_event* e) {
  gist::clear_error();
  if (!e) return set_error(GIST_E_INVAL, "event_synchronize: NULL event");
  const hipError_t he = hipEventSynchronize(e->ev);
  if (he != hipSuccess) return hip_fail("event_synchronize", he);
  return GIST_OK;
}

extern "C" gist_status gist_event_destroy(gist_event* e) {
  gist::clear_error();
  if (!e) return GIST_OK;
  if (e->ev) (void)hipEventDestroy(e->ev);
  delete e;
  return GIST_OK;
}
