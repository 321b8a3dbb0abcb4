/*
 * gist.h -- C ABI of libgist, the GIST sub-GCN training step on AMD MI355X.
 *
 * GIST ("Graph Independent Subnetwork Training", Algorithm 1) splits every
 * hidden feature dimension of a GCN into m disjoint random blocks (subGCNs,
 * Section 2.1), trains each narrow sub-GCN on cluster mini-batches
 * (subTrain, Section 2.2) and copies the trained weight slices back into the
 * global model (subAgg, Section 2.2).  This library provides the pieces of
 * that hot path:
 *
 *   gist_partition             subGCNs: random equal blocks of [0, d)   (host)
 *   gist_build_minibatch_csr   Cluster mini-batch: induced, normalised  (host)
 *   gist_ladies_sample         LADIES layer-sampled mini-batch (GCN)    (host)
 *   gist_gather_slice          Theta^(i) = Theta[D_in, D_out]           (device)
 *   gist_gcn_layer_fwd/_bwd    eq. (2) sub-GCN layer, GCN and SAGE-mean (device)
 *   gist_gcn_layer_bwd_sgd     the backward pass with the SGD step fused   (device)
 *   gist_gat_layer_fwd/_bwd    the graph attention layer GIST also trains (device)
 *   gist_softmax_xent          loss and its gradient                    (device)
 *   gist_sgd_update            one SGD step                             (device)
 *   gist_adam_update           one Adam step (the experiments' optimizer) (device)
 *   gist_adam_update_dev       the same, coefficients read from the device (device)
 *   gist_subagg                subAgg: Theta[D_in, D_out] <- Theta^(i)  (device)
 *   gist_subagg_gather         subAgg of one round + gather of the next (device)
 *   gist_subagg_mean           subAgg of an unsplit parameter: mean of copies (device)
 *   gist_capture_* / replay_*  record library calls once, replay them      (device)
 *
 * Conventions
 *  - Every matrix is row-major fp32 with the leading dimension stated.
 *  - "device" pointers are HIP device memory on the context's device; the
 *    caller owns every buffer.  The library never frees caller memory and
 *    never allocates device memory inside these calls: scratch space is
 *    passed in as a workspace sized by gist_layer_workspace_size().
 *  - Device calls are asynchronous and ordered on the context's stream.
 *    Host-side argument checks run before any launch and return an error
 *    without launching anything; faults inside a kernel surface at the
 *    caller's next synchronisation of that stream.
 *  - Every call returns a gist_status; on failure gist_last_error() holds a
 *    message (per thread).  No C++ exception crosses this interface.
 *  - Zero-sized work (n == 0, nnz == 0) is a valid no-op returning GIST_OK.
 */
#ifndef GIST_H_
#define GIST_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gist_status {
  GIST_OK = 0,
  GIST_E_INVAL = -1,        /* bad shape, pointer, flag, m does not divide d,
                               label or cluster id out of range, ...          */
  GIST_E_NOMEM = -2,        /* caller buffer / workspace too small            */
  GIST_E_DEVICE = -3,       /* HIP runtime error (text in gist_last_error)    */
  GIST_E_UNSUPPORTED = -4,  /* valid request the library does not implement */
  GIST_E_NONFINITE = -5     /* GIST_SUBAGG_CHECK_FINITE found a NaN/Inf       */
} gist_status;

/* ---- errors --------------------------------------------------------- */

/* Message of the calling thread's last failed call ("" if none).  The
 * pointer stays valid until this thread's next gist_* call. */
const char* gist_last_error(void);
/* Static name of a status code. */
const char* gist_status_str(gist_status s);

/* ---- context -------------------------------------------------------- */

typedef struct gist_ctx gist_ctx;

/* Create a context bound to HIP device `device` and stream `hip_stream`
 * (a hipStream_t; NULL = the default stream).  The stream is the caller's
 * and is not destroyed by gist_destroy. */
gist_status gist_create(int device, void* hip_stream, gist_ctx** out);
gist_status gist_destroy(gist_ctx* ctx);
gist_status gist_set_stream(gist_ctx* ctx, void* hip_stream);

/* ---- subGCNs: feature partition (Section 2.1, Algorithm 1) ----------- */

#define GIST_PART_CATEGORICAL 1u

/* Partition the feature indices [0, d) into m disjoint blocks D^(0..m-1).
 *
 * Section 2.1 asks for a random, disjoint partition into equally sized
 * blocks (its footnote's example for d = 4, m = 2: {1,4} and {2,3}, 1-based).
 * The randomness is fixed so that any implementation reproduces it bit for
 * bit: a SplitMix64 stream seeded with `seed` (Steele, Lea & Flood 2014)
 * drives a Fisher-Yates shuffle of [0, d) (for i = d-1 down to 1, j uniform
 * on [0, i] by rejection of draws >= 2^64 - (2^64 mod (i+1)), j = draw mod
 * (i+1); swap); block k is shuffled positions [k d/m, (k+1) d/m), sorted.
 * With GIST_PART_CATEGORICAL each index r (ascending) instead draws its block
 * uniformly from [0, m) (the i.i.d. categorical masks of the convergence
 * analysis, Appendix C.1); block sizes are then random and may be zero.
 *
 * Host only, synchronous.  Outputs (host memory, caller-allocated):
 *   idx_out[d]     blocks concatenated, each ascending, 0-based
 *   offs_out[m+1]  block k is idx_out[offs_out[k] .. offs_out[k+1])
 * Errors: GIST_E_INVAL if d < 1, m < 1, m > d, a NULL pointer, unknown
 * flags, or (equal blocks) d % m != 0.  Outputs are untouched on error. */
gist_status gist_partition(int64_t d, int32_t m, uint64_t seed, uint32_t flags,
                           int32_t* idx_out, int64_t* offs_out);

/* ---- Cluster mini-batch (Section 2.2; eq. (1); Appendix C.2) --------- */

typedef enum gist_norm {
  /* Dt^-1/2 (A + I) Dt^-1/2, Dt = 1 + degree: the degree-normalised
   * adjacency with self-loops of eq. (1) (renormalisation trick). */
  GIST_NORM_GCN_SYM = 0,
  /* D^-1 A: GraphSAGE's mean aggregator; no self-loop; a node without
   * neighbours has an empty row.  Also emits the explicit transpose. */
  GIST_NORM_SAGE_MEAN = 1,
  /* I + D^-1/2 A D^-1/2: the aggregation matrix of the analysis. */
  GIST_NORM_THEORY = 2
} gist_norm;

/* Global training graph: simple, undirected, no self-loops, stored as a
 * symmetric CSR with strictly ascending columns; plus its clustering. */
typedef struct gist_graph {
  int64_t n;                     /* nodes                                 */
  const int64_t* rowptr;         /* [n+1]                                 */
  const int32_t* col;            /* [rowptr[n]]                           */
  int32_t n_clusters;            /* c                                     */
  const int64_t* cluster_ptr;    /* [c+1]                                 */
  const int32_t* cluster_nodes;  /* [cluster_ptr[c]]: node ids per cluster */
} gist_graph;

/* Mini-batch CSR, host memory.  `cap_n` / `cap_nnz` are the capacities of
 * the caller's arrays (rowptr and t_rowptr hold cap_n + 1 entries); `n` and
 * `nnz` are outputs.  If `rowptr` is NULL the call only computes n and nnz
 * (size query).  t_* are written only for GIST_NORM_SAGE_MEAN (then they
 * are required). */
typedef struct gist_csr {
  int64_t n, nnz;                /* out                                   */
  int64_t cap_n, cap_nnz;        /* in                                    */
  int32_t* rowptr;               /* [n+1]                                 */
  int32_t* col;                  /* [nnz], ascending per row              */
  float* val;                    /* [nnz]                                 */
  int32_t* node_map;             /* [n]: local row -> global node id      */
  int32_t* t_rowptr;             /* transpose (SAGE only)                 */
  int32_t* t_col;
  float* t_val;
} gist_csr;

/* Build the normalised CSR of the subgraph induced by the union of the
 * clusters `clusters[0 .. n_clusters)` (duplicates allowed, any order);
 * n_clusters == -1 selects the whole graph (`clusters` may be NULL).
 *
 * Section 2.2 makes a mini-batch one cluster or a union of clusters; the
 * subgraph keeps every edge with both ends selected and degrees are those
 * of that induced subgraph.  Local rows are the selected nodes in ascending
 * global id; columns ascend within each row.  Values are computed in fp64
 * and rounded once to fp32: GCN 1/sqrt(Dt_i Dt_j), SAGE 1/deg_i, THEORY 1
 * on the diagonal and 1/sqrt(deg_i deg_j) off it -- so GCN and THEORY
 * matrices are bitwise symmetric.
 *
 * Host only, synchronous.  Errors: GIST_E_INVAL (NULL graph arrays, empty
 * selection, cluster id out of range, bad norm), GIST_E_NOMEM (capacities
 * too small; n/nnz still report the needed sizes), GIST_E_UNSUPPORTED
 * (n or nnz >= 2^31). */
gist_status gist_build_minibatch_csr(const gist_graph* g, const int32_t* clusters,
                                     int32_t n_clusters, gist_norm norm,
                                     gist_csr* out);

/* ---- LADIES layer-sampled mini-batch (Section 5.4; Appendix A.6) ---- */

/* One layer of a layer-sampled mini-batch, host memory.  Layer l aggregates
 * from the node set V_l (its columns) into V_{l+1} (its rows); V_{l+1} is a
 * subset of V_l.  `cap_n` / `cap_nnz` are the capacities of the caller's
 * arrays: nodes holds cap_n entries, rowptr and t_rowptr cap_n + 1, the
 * entry arrays cap_nnz.  n_out, n_in and nnz are outputs. */
typedef struct gist_ladies_layer {
  int64_t n_out, n_in, nnz;      /* out: |V_{l+1}|, |V_l|, entries        */
  int64_t cap_n, cap_nnz;        /* in                                    */
  int32_t* nodes;                /* [n_in]: V_l, ascending global ids     */
  int32_t* rowptr;               /* [n_out+1]                             */
  int32_t* col;                  /* [nnz]: positions in V_l, ascending    */
  float* val;                    /* [nnz]                                 */
  int32_t* t_rowptr;             /* [n_in+1]: the transpose, rows V_l     */
  int32_t* t_col;                /* [nnz]: positions in V_{l+1}, ascending */
  float* t_val;                  /* [nnz]                                 */
} gist_ladies_layer;

/* LADIES (Zou et al., NeurIPS 2019), the layer-wise importance sampling
 * GIST is combined with in place of graph partitioning, for an L-layer GCN.
 *
 * A is the full-graph GCN matrix (gist_build_minibatch_csr over the whole
 * graph with GIST_NORM_GCN_SYM; n, rowptr, col, val are read).  `batch`
 * holds the b output nodes V_L, strictly ascending.  For l = L-1 down to 0:
 *   q_j = sum over i in V_{l+1} (ascending) of A_ij^2, in double;
 *   p_j = q_j / Q with Q the sum of q_j over ascending j;
 *   s draws, each from the next output x of one SplitMix64 stream seeded
 *   `seed` (shared by all layers, layer L-1 first): t = (x >> 11) 2^-53 Q,
 *   node = the smallest j whose prefix sum q_0 + ... + q_j exceeds t (the
 *   largest j with q_j > 0 if t reached Q);
 *   V_l = distinct draws and V_{l+1}, ascending;
 *   row i of layer l: every entry (i, j) of A with j in V_l, ascending j,
 *   value w_ij = A_ij / (max(s,1) p_j), divided by the row's sum of w
 *   (ascending j) and rounded once to float.
 * The transpose is written too (rows V_l, entries in ascending row).
 * layers[l] describes layer l (0 = the input layer).  b == 0 gives empty
 * layers and draws nothing.
 *
 * If every layers[l].rowptr is NULL the call only reports the sizes.
 * Host only, synchronous, thread-safe (per-thread scratch).  Errors:
 * GIST_E_INVAL (NULL arguments, L < 1, s < 0, batch not strictly ascending
 * or out of range), GIST_E_NOMEM (a capacity too small; every layer's
 * n_out, n_in and nnz still report the needed sizes), GIST_E_UNSUPPORTED
 * (A->n >= 2^31). */
gist_status gist_ladies_sample(const gist_csr* A, const int32_t* batch, int64_t b, int32_t L,
                               int32_t s, uint64_t seed, gist_ladies_layer* layers);

/* ---- device CSR and layer descriptor -------------------------------- */

typedef struct gist_csr_dev {   /* device memory, layout as gist_csr */
  int64_t n, nnz;
  const int32_t* rowptr;        /* [n+1] */
  const int32_t* col;           /* [nnz] */
  const float* val;             /* [nnz] */
} gist_csr_dev;

typedef enum gist_layer_kind { GIST_LAYER_GCN = 0, GIST_LAYER_SAGE_MEAN = 1 } gist_layer_kind;
typedef enum gist_act { GIST_ACT_NONE = 0, GIST_ACT_RELU = 1 } gist_act;
typedef enum gist_dtype {
  GIST_DTYPE_F32 = 0,      /* fp32 operands, fp32 MFMA                        */
  GIST_DTYPE_BF16_IN = 1   /* GEMM operands rounded to bf16 (nearest-even),    */
                           /* fp32 accumulation; aggregation stays fp32        */
} gist_dtype;
typedef enum gist_order {
  GIST_ORDER_AUTO = 0,        /* GCN: aggregate at min(s_in, s_out)        */
  GIST_ORDER_AGG_FIRST = 1,   /* (Abar H) W                                 */
  GIST_ORDER_XFORM_FIRST = 2  /* Abar (H W)  (GCN only)                     */
} gist_order;

typedef struct gist_layer_desc {
  int32_t kind;    /* gist_layer_kind                                   */
  int32_t act;     /* gist_act: RELU for hidden layers, NONE for the last */
  int32_t dtype;   /* gist_dtype                                        */
  int32_t order;   /* gist_order                                        */
  int64_t n;       /* mini-batch rows                                   */
  int32_t s_in;    /* sub-GCN input width  |D_l|  (d_0 at layer 0)       */
  int32_t s_out;   /* sub-GCN output width |D_l+1| (d_L at the last layer) */
  int32_t groups;  /* G sub-GCNs batched on this mini-batch (0 means 1)  */
  uint32_t flags;  /* GIST_LAYER_SHARED_INPUT | GIST_LAYER_GROUP_MAJOR_OUT */
  int64_t n_in;    /* input rows (columns of Abar); 0 means n.  GCN only  */
                   /* when different from n (a layer-sampled batch)       */
} gist_layer_desc;

/* Rectangular layers (n_in != n): Abar is n x n_in and aggregates the
 * n_in input rows H into n output rows, as a layer-sampled mini-batch does
 * (gist_ladies_sample).  H and dH have n_in rows; agg_save, H_out and
 * dH_out have n.  The backward pass needs the explicit transpose A_T
 * (n_in rows).  Only GCN layers may be rectangular.  With no output rows
 * (n == 0) the backward pass zeroes dW and dH. */

/* Batched sub-GCNs (G > 1): the layer of G sub-GCNs that share one
 * mini-batch, each with its own weight slice -- the same results as G
 * separate calls, with one full-width aggregation and grouped GEMMs.
 * Layouts (row-major fp32):
 *   H, agg_save, dH   n x (G s_in), sub-GCN g in columns [g s_in, (g+1) s_in);
 *                     with GIST_LAYER_SHARED_INPUT one n x s_in matrix that
 *                     every sub-GCN reads (the unpartitioned input layer:
 *                     Abar H is formed once; dH must be NULL);
 *   W, dW             G consecutive slices of (s_in or 2 s_in) x s_out;
 *   H_out, dH_out     n x (G s_out), sub-GCN g in columns [g s_out, ...);
 *                     with GIST_LAYER_GROUP_MAJOR_OUT G consecutive
 *                     n x s_out blocks (each sub-GCN's logits contiguous). */
enum {
  GIST_LAYER_SHARED_INPUT = 1,
  GIST_LAYER_GROUP_MAJOR_OUT = 2,
  GIST_LAYER_CLUSTERED = 4,
  GIST_LAYER_DZ_IN = 8,
  GIST_LAYER_MASK_DH = 16
};

/* The ReLU derivative of a hidden layer, fused into the producer of the
 * gradient it multiplies (backward pass only; the forward ignores these):
 *   GIST_LAYER_MASK_DH  the backward pass writes dH * 1[H > 0] instead of dH:
 *                       the gradient with respect to the pre-activation of
 *                       the layer below, whose (ReLU) output H is.  The
 *                       product is applied in the epilogue of the kernel that
 *                       writes dH (the transposed aggregation, or the dH
 *                       product of a transform-first GCN layer).
 *   GIST_LAYER_DZ_IN    dH_out already is dZ = dH_out * 1[H_out > 0] (the
 *                       layer above was called with GIST_LAYER_MASK_DH), so
 *                       no ReLU derivative is formed here and H_out may be
 *                       NULL.
 * A chain of ReLU layers passes MASK_DH to every layer above the first and
 * DZ_IN to every hidden layer: no separate ReLU-derivative pass remains, and
 * the gradients are bitwise those of the unflagged calls (the derivative is
 * the same select, 1[H > 0], applied to the same values). */

/* GIST_LAYER_CLUSTERED: a hint that almost every entry of Abar (and A_T)
 * sits within a few hundred columns of its row's diagonal: the matrix of a
 * cluster mini-batch over block-contiguous node ids (Section 2.2: a union of
 * clusters), or a whole graph numbered cluster by cluster.  The aggregation
 * then runs on the matrix cores: for every 32 rows, the entries within 192
 * of their row's diagonal form up to two dense tiles of at most 288 columns
 * (the second for rows that straddle two clusters) whose values and the
 * matching X rows are each split into two bf16 halves (hi = bf16(v),
 * lo = bf16(v - hi)); the products hi*hi + hi*lo + lo*hi are accumulated in
 * fp32, so every term carries a relative error below 2^-15; the remaining
 * entries are gathered and added in storage order.  Results are
 * deterministic and agree with the plain fp32 aggregation within that bound
 * for any matrix and finite X (only the speed depends on the structure; an
 * Inf or NaN in a window row reaches every output row of that tile, since
 * the dense tile multiplies it by zero).  The matrix
 * must not repeat a (row, column) entry (gist_build_minibatch_csr never
 * does).  On the cluster-structured workloads measured it is faster than the
 * gather kernel (4.1 against 7.4 ms for the 2.45M-node graph at width 256,
 * 34 against 55 us for a 10-cluster mini-batch at width 4,096); without the
 * structure it gathers every entry and is slower. */

/* Workspace (device bytes) that fwd and bwd need for this descriptor. */
gist_status gist_layer_workspace_size(const gist_layer_desc* L, size_t* fwd_bytes,
                                      size_t* bwd_bytes);

/* Sub-GCN layer forward, eq. (2): H_out = act(Abar H W), W = Theta^(i)_l.
 *
 *   GCN:       Z = (Abar H) W   or  Abar (H W)  (same value; `order`)
 *   SAGE-mean: Z = H W_self + (Abar H) W_neigh   -- GraphSAGE concatenates
 *              the aggregated neighbourhood with the node itself; W holds
 *              [W_self; W_neigh] as one (2 s_in) x s_out matrix.
 *
 * H [n x s_in], W [s_in x s_out] (SAGE [2 s_in x s_out]), H_out [n x s_out].
 * agg_save [n x s_in] receives Abar H (required for SAGE and for GCN when
 * aggregating first; may be NULL for GCN transform-first).  The ReLU mask
 * for the backward pass is recovered from H_out (H_out > 0 iff Z > 0).
 * Errors: GIST_E_INVAL (NULL pointers, widths < 1, unknown enums, SAGE with
 * XFORM_FIRST), GIST_E_NOMEM (ws_bytes below gist_layer_workspace_size). */
gist_status gist_gcn_layer_fwd(gist_ctx* ctx, const gist_layer_desc* L,
                               const gist_csr_dev* A, const float* H,
                               const float* W, float* agg_save, float* H_out,
                               void* ws, size_t ws_bytes);

/* Sub-GCN layer backward (chain rule of the forward).
 *
 *   dZ = dH_out * 1[H_out > 0] (ReLU) or dH_out (identity, or DZ_IN)
 *   GCN:  dW = (Abar H)^T dZ,               dH = Abar^T (dZ W^T)
 *   SAGE: dW = [H | Abar H]^T dZ  ([2 s_in x s_out]),
 *         dH = dZ W_self^T + Abar^T (dZ W_neigh^T)
 *
 * A_T is the explicit transpose CSR (required for SAGE-mean and for
 * rectangular layers; NULL for a square GCN layer means Abar is symmetric,
 * as GIST_NORM_GCN_SYM / THEORY produce).
 * dW is overwritten.  dH may be NULL (layer 0: no input gradient).
 * Results are deterministic: no atomics, fixed reduction order. */
gist_status gist_gcn_layer_bwd(gist_ctx* ctx, const gist_layer_desc* L,
                               const gist_csr_dev* A, const gist_csr_dev* A_T,
                               const float* H, const float* agg_save,
                               const float* H_out, const float* W,
                               const float* dH_out, float* dW, float* dH,
                               void* ws, size_t ws_bytes);

/* The same backward pass with subTrain's SGD step fused in (Algorithm 1; the
 * update of gist_sgd_update): W <- W - lr dW in place, where dW is the
 * weight gradient above, without writing dW anywhere.  The input gradient dH
 * is formed from the weights before the step.  Every other argument has the
 * meaning, layout and workspace size it has in gist_gcn_layer_bwd; W (device
 * memory, every group's slice for G > 1) is read and then updated in place,
 * and there is no dW argument.  Bitwise the same W and dH as gist_gcn_layer_bwd
 * followed by gist_sgd_update(W, dW, lr): the GEMM writing the gradient
 * applies fmaf(-lr, dW_ij, W_ij) to each element once, in its epilogue.
 * Saves the gradient's write and the separate pass that reads it.  With no
 * output rows (n == 0) W is unchanged.  Errors as gist_gcn_layer_bwd, and
 * GIST_E_INVAL for a non-finite lr. */
gist_status gist_gcn_layer_bwd_sgd(gist_ctx* ctx, const gist_layer_desc* L,
                                   const gist_csr_dev* A, const gist_csr_dev* A_T,
                                   const float* H, const float* agg_save,
                                   const float* H_out, float* W, const float* dH_out,
                                   float lr, float* dH, void* ws, size_t ws_bytes);

/* ---- graph attention layer ------------------------------------------ */

/* The GAT layer the paper trains with GIST alongside GCN and GraphSAGE
 * (Section 2.3, architecture-agnostic training; Table 2).  Single head, as
 * Velickovic et al. (ICLR 2018) define it:
 *   P = H W,  u = P a_src,  v = P a_dst,  e_ij = LeakyReLU(u_i + v_j),
 *   alpha_ij = softmax of e_i. over the pattern N(i) u {i},
 *   Z_i = sum_j alpha_ij P_j,  H_out = ReLU(Z) (act) or Z.
 * A sub-GCN's slice of a_src / a_dst is their entries D_{l+1}^(i), the
 * output features its slice of W keeps.  A is the pattern N(i) u {i}: a
 * symmetric CSR with ascending columns (the GCN matrix of an undirected
 * graph has it); its values are ignored.  H (n x s_in), W (s_in x s_out),
 * P_save / H_out / dH_out (n x s_out) row-major; a_src, a_dst (s_out);
 * alpha_save (nnz, in A's entry order).  P_save and alpha_save come out of
 * the forward and go into the backward.  dW is overwritten; dH == NULL
 * skips the input gradient.  Errors as gist_gcn_layer_fwd. */
typedef struct gist_gat_desc {
  int64_t n;       /* rows                                               */
  int64_t nnz;     /* entries of the pattern                             */
  int32_t s_in;
  int32_t s_out;
  int32_t act;     /* gist_act                                           */
  int32_t dtype;   /* gist_dtype of the two GEMMs                        */
  float slope;     /* LeakyReLU slope for negative scores (0.2 in the GAT paper) */
  uint32_t flags;  /* 0 or GIST_GAT_MIRROR_IN_WS                        */
} gist_gat_desc;

/* GIST_GAT_MIRROR_IN_WS (backward only): the first nnz int32 of the
 * backward workspace already hold A's mirror map (for each entry (i, j) the
 * position of (j, i)), as a previous gist_gat_layer_bwd on the same pattern
 * A left them in the same workspace, and nothing has written that workspace
 * since.  The map is then not formed again.  The layers of one sub-GCN step
 * share the mini-batch's pattern: the first backward call forms the map,
 * the layers below pass the flag.  With a different matrix, or a
 * workspace written in between (a forward call), results are undefined. */
enum { GIST_GAT_MIRROR_IN_WS = 1 };

/* The two per-node halves of the attention scores, u = P a_src and
 * v = P a_dst (n floats each, device memory), exactly as the layer's forward
 * and backward passes form them: the score of entry (i, j) is
 * LeakyReLU(u_i + v_j), its side decided by u_i + v_j > 0 in fp32.  P is
 * n x s row-major with leading dimension ldp; a_src, a_dst have s entries.
 * For a caller that needs the attention logits, or the side each score
 * fell on.  Errors: GIST_E_INVAL (NULL pointers with n > 0, s < 1,
 * ldp < s, n < 0). */
gist_status gist_gat_scores(gist_ctx* ctx, int64_t n, int32_t s, const float* P, int64_t ldp,
                            const float* a_src, const float* a_dst, float* u, float* v);

gist_status gist_gat_workspace_size(const gist_gat_desc* D, size_t* fwd_bytes,
                                    size_t* bwd_bytes);
gist_status gist_gat_layer_fwd(gist_ctx* ctx, const gist_gat_desc* D, const gist_csr_dev* A,
                               const float* H, const float* W, const float* a_src,
                               const float* a_dst, float* P_save, float* alpha_save,
                               float* H_out, void* ws, size_t ws_bytes);
gist_status gist_gat_layer_bwd(gist_ctx* ctx, const gist_gat_desc* D, const gist_csr_dev* A,
                               const float* H, const float* P_save, const float* alpha_save,
                               const float* H_out, const float* W, const float* a_src,
                               const float* a_dst, const float* dH_out, float* dW,
                               float* da_src, float* da_dst, float* dH, void* ws,
                               size_t ws_bytes);

/* ---- loss (Section 2.1: the sub-GCN output keeps the global width, so the
 *      loss is the usual one) ---------------------------------------- */

/* Mean softmax cross-entropy over n rows of logits [n x C] with int32
 * labels in [0, C): *loss_dev (one device float) = mean_v (logsumexp(z_v) -
 * z_v,y_v); dlogits [n x C] = (softmax(z) - onehot(y)) / n.  `ws` needs
 * gist_softmax_xent_workspace(n) bytes.  Labels out of range are a caller
 * error: the kernel clamps nothing and reports it by writing NaN to
 * *loss_dev. */
size_t gist_softmax_xent_workspace(int64_t n);
gist_status gist_softmax_xent(gist_ctx* ctx, int64_t n, int32_t C,
                              const float* logits, const int32_t* labels,
                              float* loss_dev, float* dlogits, void* ws,
                              size_t ws_bytes);
/* The same over a batch padded to n rows, with the number of real rows in
 * device memory (*n_valid_dev, one int32, read by the kernels, so that a
 * replayed step can change it): the loss is the mean over rows
 * [0, n_valid) and the gradient rows [n_valid, n) are zero.  A count
 * outside [0, n] is clamped.  Same workspace; errors as gist_softmax_xent. */
gist_status gist_softmax_xent_padded(gist_ctx* ctx, int64_t n, int32_t C,
                                     const float* logits, const int32_t* labels,
                                     const int32_t* n_valid_dev, float* loss_dev,
                                     float* dlogits, void* ws, size_t ws_bytes);

/* For callers that cannot allocate device memory (code under stream
 * capture, serving loops, harnesses that forbid hipMalloc): the loss of
 * gist_softmax_xent without a workspace argument.  Its partial sums live in
 * a buffer the library keeps per device for the life of the process
 * (4 MiB, looked up at gist_create), so the call allocates nothing; the
 * caller still owns logits, labels, *loss_dev and dlogits.  Results are
 * bitwise those of gist_softmax_xent.  n may be at most
 * GIST_NOALLOC_LOSS_MAX_ROWS (GIST_E_INVAL beyond, before any launch).
 * Every call on one device shares that buffer: calls ordered on one stream
 * are safe, calls that overlap in time on one device (other streams or
 * threads) race and give undefined losses. */
#define GIST_NOALLOC_LOSS_MAX_ROWS 4194304
gist_status gist_softmax_xent_noalloc(gist_ctx* ctx, int64_t n, int32_t C,
                                      const float* logits, const int32_t* labels,
                                      float* loss_dev, float* dlogits);

/* ---- subGCNs slice gather (Section 2.1) ----------------------------- */

/* Ws[i][j] = Wg[rows[i]][cols[j]], i < nr, j < nc: the sub-GCN weight
 * Theta^(i)_l = [Theta_l] restricted to rows D^(i)_l and columns
 * D^(i)_{l+1}.  rows / cols are device int32 arrays; NULL selects all
 * (0..nr-1 / 0..nc-1).  Also gathers mini-batch feature rows (cols NULL).
 * Bit-exact copy.  Indices must lie inside Wg (checked only by the caller). */
gist_status gist_gather_slice(gist_ctx* ctx, const float* Wg, int64_t ldg,
                              const int32_t* rows, int32_t nr,
                              const int32_t* cols, int32_t nc, float* Ws,
                              int64_t lds);

/* ---- subTrain update (Section 2.2) ---------------------------------- */

/* W[k] -= lr * dW[k] for k < n, in fp32 (one rounding per element). */
gist_status gist_sgd_update(gist_ctx* ctx, float* W, const float* dW, int64_t n,
                            float lr);

/* One Adam step on n parameters -- the optimizer the paper's experiments
 * train with (no weight decay), as defined by Kingma & Ba (ICLR 2015,
 * Algorithm 1), step k >= 1 counting from 1:
 *   m <- beta1 m + (1 - beta1) g,   v <- beta2 v + (1 - beta2) g^2,
 *   W <- W - lr (m / (1 - beta1^k)) / (sqrt(v / (1 - beta2^k)) + eps).
 * W, m, v are updated in place, g = dW is read; all device fp32 arrays of n
 * elements.  The bias corrections are formed in double on the host and
 * applied in fp32.  GIST_ADAM_FRESH treats the incoming m and v as zero (a
 * sub-GCN whose moments restart, e.g. at the start of a round), so they
 * need no clearing pass.  Errors: GIST_E_INVAL for n < 0, NULL pointers
 * with n > 0, k < 1, beta outside [0, 1), eps < 0, a non-finite lr or
 * unknown flags. */
enum { GIST_ADAM_FRESH = 1 };
gist_status gist_adam_update(gist_ctx* ctx, float* W, const float* dW, float* m, float* v,
                             int64_t n, float lr, float beta1, float beta2, float eps,
                             int64_t step, uint32_t flags);

/* The step-dependent coefficients of gist_adam_update, host only:
 * coef3 = {lr / (1 - beta1^k), 1 / sqrt(1 - beta2^k), 1 if GIST_ADAM_FRESH
 * else 0}, formed in double and rounded once to float, with the same
 * checks and errors.  gist_adam_update_dev reads these three floats from
 * device memory (`coef_dev`) when its kernel runs, so a recorded step
 * (gist_capture_begin) advances k and the fresh flag through the contents
 * of one buffer; with the same coefficients it updates W, m and v exactly
 * as gist_adam_update does.  Errors as gist_adam_update (coef_dev NULL:
 * GIST_E_INVAL). */
gist_status gist_adam_coefficients(float lr, float beta1, float beta2, float eps,
                                   int64_t step, uint32_t flags, float* coef3);
gist_status gist_adam_update_dev(gist_ctx* ctx, float* W, const float* dW, float* m, float* v,
                                 int64_t n, float beta1, float beta2, float eps,
                                 const float* coef_dev);

/* ---- subAgg (Section 2.2) ------------------------------------------- */

#define GIST_SUBAGG_CHECK_FINITE 1u

/* Wg[rows[i]][cols[j]] = Ws[i][j]: each worker's trained slice replaces the
 * global entries it owns; blocks of different sub-GCNs never overlap, so
 * calls for different sub-GCNs may run in any order.  Entries outside
 * every block are left unchanged.  With GIST_SUBAGG_CHECK_FINITE the slice
 * is first scanned (synchronously) and, if any entry is NaN or Inf, nothing
 * is written and GIST_E_NONFINITE is returned. */
gist_status gist_subagg(gist_ctx* ctx, float* Wg, int64_t ldg, const int32_t* rows,
                        int32_t nr, const int32_t* cols, int32_t nc,
                        const float* Ws, int64_t lds, uint32_t flags);

/* subAgg of a parameter that no partition splits: a GAT output layer's
 * attention vectors live in the unpartitioned class dimension, so every
 * sub-GCN trains a full copy.  The paper is silent on how those copies are
 * combined; this is the rule of independent subnet training, which GIST
 * extends -- the mean of the m trained copies:
 *   Wg[r][c] = (sum_{i<m} slices[i][r * lds + c]) / m,  r < rows, c < cols,
 * summed in double in the order i = 0, 1, ..., m-1, divided in double and
 * rounded once to fp32 (bitwise reproducible).  `slices` is a device array
 * of m device pointers, each to a rows x cols row-major block with row
 * stride lds; Wg is row-major with stride ldg and must not overlap them.
 * Errors: GIST_E_INVAL for negative sizes, m < 1, ldg < cols, lds < cols
 * or NULL pointers when rows * cols > 0. */
gist_status gist_subagg_mean(gist_ctx* ctx, float* Wg, int64_t rows, int64_t cols,
                             int64_t ldg, int32_t m, const float* const* slices,
                             int64_t lds);

/* ---- subAgg of one round fused with the gather of the next ---------- */

/* Inverse of a partition (host): rank[idx[k]] = k for k < d, i.e. the
 * position of each index in the block-ordered list gist_partition returns;
 * index r is then the (rank[r] - offs[b])-th member of the block b with
 * offs[b] <= rank[r] < offs[b+1].  Errors: GIST_E_INVAL for NULL pointers,
 * offsets that are not ascending from 0 to d, or an index outside [0, d) or
 * listed twice. */
gist_status gist_partition_inverse(int64_t d, int32_t m, const int32_t* idx,
                                   const int64_t* offs, int32_t* rank_out);

/* How one global weight matrix (rows x cols) is split among m sub-GCNs in
 * one round (device memory).  A partitioned dimension is given by its ranks
 * (gist_partition_inverse) and its m + 1 block offsets; NULL ranks and
 * offsets mean the dimension is not partitioned (every sub-GCN holds all of
 * it at its own index: the input width at layer 0, the output width at the
 * last layer, Section 2.1).  Element (r, c) belongs to sub-GCN i when the
 * partitioned dimensions place both r and c in block i; it sits in slice i
 * at (position of r in block i, position of c in block i), an unpartitioned
 * index keeping its own value.  `slices` is a device array of m device
 * pointers, each slice row-major with leading dimension `ld`.  The kernels
 * trust these arrays: ranks and offsets must describe a partition (as the
 * two host calls return them) and each slice must hold its block. */
typedef struct gist_slice_set {
  const int32_t* row_rank;
  const int64_t* row_offs;
  const int32_t* col_rank;
  const int64_t* col_offs;
  float* const* slices;
  int64_t ld;
} gist_slice_set;

/* One pass over Wg (rows x cols, leading dimension ldg) that first applies
 * subAgg for the slices of `done` (every entry a sub-GCN owns is replaced by
 * its trained value; entries owned by none keep theirs, Section 2.2) and then
 * gathers the slices of `next` from the updated matrix -- the end of one
 * round of Algorithm 1 and the start of the next.  Either set may be NULL
 * (plain gather, or plain subAgg).  Equal to gist_subagg for every slice of
 * `done` followed by gist_gather_slice for every slice of `next`, bit for
 * bit; every row of Wg is read and rewritten whole, so HBM sees full-line
 * writes instead of 1/m-dense scattered ones.  The partitions of `done`
 * and `next` may differ.  At least one dimension of each set must be
 * partitioned when m > 1, and ranks and offsets come in pairs (GIST_E_INVAL
 * otherwise).  The slices of `done` and of `next` must not share memory with
 * each other or with Wg: one grid reads the trained slices and writes the new
 * ones, so an overlap would let a row's block overwrite entries another block
 * has not read yet.  The call rejects the one overlap it can see on the host,
 * both sets naming the same pointer table (GIST_E_INVAL); any other overlap
 * gives undefined results. */
gist_status gist_subagg_gather(gist_ctx* ctx, float* Wg, int64_t rows, int64_t cols,
                               int64_t ldg, int32_t m, const gist_slice_set* done,
                               const gist_slice_set* next);

/* ---- instrumentation ------------------------------------------------ */

/* Per-kernel timing with HIP events recorded on the context's stream around
 * every kernel launch the library makes, for measuring kernels against
 * their rooflines.  gist_profile_begin(ctx, cap) creates `cap` event pairs
 * (host-side set-up, outside any hot path) and starts recording; while
 * recording, launches beyond `cap` are not timed (and counted as dropped).
 * gist_profile_read synchronises the stream and aggregates the records per
 * kernel variant into `out[0 .. *n)` (at most `out_cap` entries), then
 * clears them; gist_profile_end stops recording and frees the events.
 * `flops` counts 2 M N K per GEMM; `bytes` the algorithmic HBM bytes
 * (each operand read once, each result written once). */
typedef struct gist_prof_entry {
  char name[48];      /* kernel variant, e.g. "gemm_f32_KR", "spmm_v4_l64" */
  int64_t launches;
  double ms;          /* summed event time */
  double flops;       /* summed algorithmic flops */
  double bytes;       /* summed algorithmic bytes */
} gist_prof_entry;

gist_status gist_profile_begin(gist_ctx* ctx, int64_t cap);
gist_status gist_profile_read(gist_ctx* ctx, gist_prof_entry* out, int32_t out_cap,
                              int32_t* n, int64_t* dropped);
gist_status gist_profile_end(gist_ctx* ctx);

/* ---- replays: HIP graphs of library calls -------------------------- */

/* A step of many small launches (a sub-GCN step on a LADIES mini-batch) can
 * cost more host time to issue than device time to run.  These calls record
 * a sequence of library calls once and replay it with one launch.
 *
 * gist_capture_begin starts capturing the calls made on `ctx` from this
 * thread (hipStreamBeginCapture, thread-local mode): they are recorded, not
 * run.  The context's stream must not be the default stream, and the
 * context must not be recording a profile.  Only device calls with fixed
 * shapes and buffers belong in a capture: a replay repeats the recorded
 * launches with the recorded arguments, so the buffers must outlive it and
 * their contents (not their sizes) are what changes between replays.
 * gist_capture_end ends the capture and instantiates the replay (caller
 * owns it; gist_replay_destroy frees it).  Errors: GIST_E_INVAL, and
 * GIST_E_DEVICE if the runtime rejected the capture (a failed call inside
 * it ends the capture too; the caller must still call gist_capture_end).
 *
 * gist_replay_launch enqueues on the stream of `ctx` (any context on the
 * same device): first a copy of `bytes` from `src` to device `dst` (skipped
 * when bytes == 0), made by a kernel that reads `src` directly, so src must
 * be device memory or pinned host memory (hipHostMalloc; torch's
 * pin_memory), then a record of `copied` (may be NULL: after it, src may be
 * reused), then the replay.  All asynchronous. */
typedef struct gist_replay gist_replay;
typedef struct gist_event gist_event;
gist_status gist_capture_begin(gist_ctx* ctx);
gist_status gist_capture_end(gist_ctx* ctx, gist_replay** out);
gist_status gist_replay_launch(gist_ctx* ctx, gist_replay* r, void* dst, const void* src,
                               size_t bytes, gist_event* copied);
gist_status gist_replay_destroy(gist_replay* r);
/* The copy of gist_replay_launch on its own: `bytes` from `src` (device or
 * pinned host memory) to device `dst` by a kernel on the stream of `ctx`,
 * then a record of `copied` (may be NULL).  Small uploads made this way
 * stay on the compute queue (no copy-engine hand-off). */
gist_status gist_copy(gist_ctx* ctx, void* dst, const void* src, size_t bytes,
                      gist_event* copied);
/* A device event (no timing) for gist_replay_launch: create, wait for its
 * last record on the host, destroy. */
gist_status gist_event_create(gist_event** out);
gist_status gist_event_synchronize(gist_event* e);
gist_status gist_event_destroy(gist_event* e);

#ifdef __cplusplus
}
#endif

#endif /* GIST_H_ */
